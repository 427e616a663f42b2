"""Parity at the full sizes of the sweep and long-context workloads.

The whole batch runs on the GPU; sampled prompts are checked against the
float64 oracle (batch independence makes a prompt's result independent of
the others).  A full oracle step per prompt is too slow at these sizes, so
each sampled prompt is checked on the parts that define the step:
  a1  the beam heads of the prefill (top-k of s_0, near-ties allowed),
  a3-a5  the verification of a seeded k x d lookahead block fed with the
      oracle's heads (the verify is stateless with respect to the beams),
  a2  the greedy rollout of the first beams from the oracle's heads.
"""
import numpy as np
import pytest
import torch

import oracle
from cdsl_harness import TOK_MARGIN, lp_tol, make_engine, make_setup

pytestmark = pytest.mark.gpu


def _check_prompt_heads(g_beams, g_hlp, heads, hlp, margins, tol):
    for u in range(len(heads)):
        if int(g_beams[u]) != int(heads[u]):
            near = margins[u] <= TOK_MARGIN or (u > 0 and margins[u - 1] <= TOK_MARGIN)
            assert near, (u, list(g_beams), list(heads), margins)
        else:
            assert abs(float(g_hlp[u]) - float(hlp[u])) <= tol


def _full_size(name, k, d, check, roll_beams=2, **over):
    s = make_setup(name, **over)
    wl = s.wl
    B = wl.batch
    tol = lp_tol(wl.dtype)
    eng = make_engine(s, B=B, max_steps=2, k=k, d=d)
    try:
        prompts = s.prompts(B)
        st = eng.start(torch.from_numpy(prompts).cuda(), k=k)
        beams = st.beams.cpu().numpy().copy()
        head_lp = st.head_lp.cpu().numpy().copy()
        rng = np.random.default_rng(11)
        look = np.zeros((B, k, d + 1), np.int32)
        look[:, :, 0] = beams
        look[:, :, 1:] = rng.integers(0, wl.target.vocab, (B, k, d))
        ost, oheads, ohlp = {}, {}, {}
        for b in check:
            ost[b] = oracle.prefill(s.odraft, s.otarget, prompts[b])
            heads, hlp, margins = oracle.beam_heads(ost[b], k)
            _check_prompt_heads(beams[b], head_lp[b], heads, hlp, margins, tol)
            oheads[b], ohlp[b] = heads, hlp
            look[b, :, 0] = heads
            beams[b] = heads
            head_lp[b] = hlp
        # a3-a5 on the seeded block
        out = eng.ctx.cdsl_verify(st.prefix, torch.from_numpy(look).cuda(), k, d,
                                  torch.from_numpy(head_lp.astype(np.float32)).cuda())
        g = {kk: v.cpu().numpy() for kk, v in out.items() if v is not None}
        for b in check:
            ve = oracle.verify(s.otarget, ost[b], oheads[b], ohlp[b], look[b, :, 1:])
            err = np.max(np.abs(g["logprobs"][b] - ve.logprobs))
            print(f"{name} k={k} d={d} prompt {b}: verify max |dlp| {err:.2e}")
            assert err <= tol
            ok = ve.margin > TOK_MARGIN
            assert np.array_equal(g["target_argmax"][b][ok], ve.y[ok])
            if np.all(ok):
                assert np.array_equal(g["n_accept"][b], ve.n)
            assert np.max(np.abs(g["scores"][b] - ve.scores)) <= tol * (d + 1)
        # a2 from the oracle's heads
        la = eng.ctx.cdsl_rollout(st.prefix, torch.from_numpy(beams).cuda(), k, d).cpu().numpy()
        for b in check:
            assert np.array_equal(la[b, :, 0], oheads[b])
            ro = oracle.rollout(s.odraft, ost[b], oheads[b][:roll_beams], d)
            for i in range(roll_beams):
                diff = np.nonzero(la[b, i, 1:] != ro.x[i])[0]
                if diff.size:
                    u = int(diff[0])
                    assert ro.margin[i, u] <= TOK_MARGIN, (b, i, u, la[b, i], ro.x[i], ro.margin[i])
                    print(f"{name} prompt {b} beam {i}: draft near tie at j={u + 1}")
        st.prefix.free()
    finally:
        eng.close()


@pytest.mark.timeout(900)
def test_sweep_full_size_widest_block():
    """7B/1B pair at batch 32 with 512-token prompts, the sweep's largest
    block (k=10 beams x d=20: two suffix blocks per beam, 6400 verify rows)."""
    _full_size("sweep", k=10, d=20, check=[0, 31])


@pytest.mark.timeout(900)
def test_long_context_full_size():
    """7B GQA-8 target, V=128256, batch 64 with 2048-token prompts, k=8, d=8."""
    _full_size("long", k=8, d=8, check=[0])
