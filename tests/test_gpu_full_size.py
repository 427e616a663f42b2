"""Parity at the full sizes of the sweep and long-context workloads.

The whole batch runs on the GPU; sampled prompts are checked against the
float64 oracle (batch independence makes a prompt's result independent of
the others).  Each sampled prompt is checked on the parts that define the
step at every (k, d) point:
  a1  the beam heads of the prefill (top-k of s_0, near-ties allowed),
  a3-a5  the verification of a seeded k x d lookahead block fed with the
      oracle's heads (the verify is stateless with respect to the beams),
  a2  the greedy rollout of the first beams from the oracle's heads,
and by whole steps (rollout, verification, linear reward, selection,
commit, next heads) compared step by step as in the smaller workloads.
"""
import numpy as np
import pytest
import torch

import oracle
from cdsl_harness import (TOK_MARGIN, Report, assert_full_or_tie, compare_step, lp_tol, make_engine,
                          make_setup)

pytestmark = pytest.mark.gpu

SWEEP_K = (2, 5, 10)
SWEEP_D = (2, 5, 10, 20)


def _check_prompt_heads(g_beams, g_hlp, heads, hlp, margins, tol):
    for u in range(len(heads)):
        if int(g_beams[u]) != int(heads[u]):
            near = margins[u] <= TOK_MARGIN or (u > 0 and margins[u - 1] <= TOK_MARGIN)
            assert near, (u, list(g_beams), list(heads), margins)
        else:
            assert abs(float(g_hlp[u]) - float(hlp[u])) <= tol


def _block_checks(s, eng, st, ost, check, k, d, roll_beams, seed):
    """Heads, a seeded verification block and the rollout of the first
    beams at one (k, d) point, on a prefix prefilled with at least k heads."""
    wl = s.wl
    B = st.prefix.B
    tol = lp_tol(wl.dtype)
    beams = st.beams.cpu().numpy()[:, :k].copy()
    head_lp = st.head_lp.cpu().numpy()[:, :k].copy()
    rng = np.random.default_rng([seed, k, d])
    look = np.zeros((B, k, d + 1), np.int32)
    look[:, :, 0] = beams
    look[:, :, 1:] = rng.integers(0, wl.target.vocab, (B, k, d))
    oheads, ohlp = {}, {}
    for b in check:
        heads, hlp, margins = oracle.beam_heads(ost[b], k)
        _check_prompt_heads(beams[b], head_lp[b], heads, hlp, margins, tol)
        oheads[b], ohlp[b] = heads, hlp
        look[b, :, 0] = heads
        beams[b] = heads
        head_lp[b] = hlp
    out = eng.ctx.cdsl_verify(st.prefix, torch.from_numpy(look).cuda(), k, d,
                              torch.from_numpy(head_lp.astype(np.float32)).cuda())
    g = {kk: v.cpu().numpy() for kk, v in out.items() if v is not None}
    for b in check:
        ve = oracle.verify(s.otarget, ost[b], oheads[b], ohlp[b], look[b, :, 1:])
        err = np.max(np.abs(g["logprobs"][b] - ve.logprobs))
        print(f"{wl.name} k={k} d={d} prompt {b}: verify max |dlp| {err:.2e}", flush=True)
        assert err <= tol
        ok = ve.margin > TOK_MARGIN
        assert np.array_equal(g["target_argmax"][b][ok], ve.y[ok])
        if np.all(ok):
            assert np.array_equal(g["n_accept"][b], ve.n)
        assert np.max(np.abs(g["scores"][b] - ve.scores)) <= tol * (d + 1)
    la = eng.ctx.cdsl_rollout(st.prefix, torch.from_numpy(beams).cuda(), k, d).cpu().numpy()
    for b in check:
        assert np.array_equal(la[b, :, 0], oheads[b])
        nr = min(roll_beams, k)
        ro = oracle.rollout(s.odraft, ost[b], oheads[b][:nr], d)
        for i in range(nr):
            diff = np.nonzero(la[b, i, 1:] != ro.x[i])[0]
            if diff.size:
                u = int(diff[0])
                assert ro.margin[i, u] <= TOK_MARGIN, (b, i, u, la[b, i], ro.x[i], ro.margin[i])
                print(f"{wl.name} prompt {b} beam {i}: draft near tie at j={u + 1}")


def _whole_steps(s, eng, st, ost, check, k, d, steps):
    """`steps` whole steps of the batch on the GPU, each sampled prompt
    compared with its own oracle step."""
    wl = s.wl
    tol = lp_tol(wl.dtype)
    rw_t = torch.from_numpy(s.rw).cuda() if s.rw is not None else None
    kw_t = torch.from_numpy(s.kws[:st.prefix.B]).cuda() if s.kws is not None else None
    reps = {b: Report() for b in check}
    live = set(check)
    cur = dict(ost)
    for _ in range(steps):
        heads = st.beams.cpu().numpy().copy()
        head_lp = st.head_lp.cpu().numpy().copy()
        bf = eng.step(st, keywords=kw_t, reward_w=rw_t, k=k, d=d)
        look = bf.lookaheads.cpu().numpy()
        ver = {kk: (v.cpu().numpy() if v is not None else None) for kk, v in bf.verify.items()}
        rew = bf.reward.cpu().numpy()
        beam = bf.beam.cpu().numpy()
        for b in list(live):
            o = oracle.step(s.odraft, s.otarget, cur[b], k, d, wl.alpha, wl.reward,
                            kws=s.kws[b] if s.kws is not None else None, w=s.rw)
            gv = {kk: (x[b] if x is not None else None) for kk, x in ver.items()}
            cont = compare_step(reps[b], wl, k, d, o, heads[b], head_lp[b], look[b], gv, rew[b], beam[b],
                                eng._last_emitted[b], tol, alpha=wl.alpha, w=s.rw)
            if cont:
                reps[b].steps_compared += 1
                cur[b] = o.state
            if cont is not True:
                live.discard(b)
    for b, r in reps.items():
        print(f"{wl.name} k={k} d={d} whole steps, prompt {b}: {r.steps_compared} compared, "
              f"max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}", flush=True)
    assert_full_or_tie(reps, steps)


def _full_size(name, points, check, roll_beams=2, step_at=(), steps=1, **over):
    """points: the (k, d) grid checked on one prefill with the largest k;
    step_at: the (k, d) points of whole steps, each from a fresh prefill."""
    s = make_setup(name, **over)
    wl = s.wl
    B = wl.batch
    kmax = max(k for k, _ in list(points) + list(step_at))
    dmax = max(d for _, d in list(points) + list(step_at))
    eng = make_engine(s, B=B, max_steps=steps + 1, k=kmax, d=dmax)
    try:
        prompts = s.prompts(B)
        ost = {b: oracle.prefill(s.odraft, s.otarget, prompts[b]) for b in check}
        st = eng.start(torch.from_numpy(prompts).cuda(), k=kmax)
        for k, d in points:
            _block_checks(s, eng, st, ost, check, k, d, roll_beams, seed=11)
        st.prefix.free()
        for k, d in step_at:
            st = eng.start(torch.from_numpy(prompts).cuda(), k=k)
            _whole_steps(s, eng, st, ost, check, k, d, steps)
            st.prefix.free()
    finally:
        eng.close()


@pytest.mark.timeout(1000)
def test_sweep_full_size_every_point():
    """7B/1B pair at batch 32 with 512-token prompts: every point of the
    k in {2, 5, 10} x d in {2, 5, 10, 20} grid (the widest, k=10 x d=20, has
    two suffix blocks per beam and 6400 verify rows), and whole steps at
    k=2 d=20 (two suffix blocks per beam, 64 draft rows on the skinny
    kernel), k=5 d=10 and k=10 d=2 (320 draft rows on the dense kernel)."""
    points = [(k, d) for k in SWEEP_K for d in SWEEP_D]
    _full_size("sweep", points, check=[0, 31], roll_beams=1, step_at=[(2, 20), (5, 10), (10, 2)], steps=1)


@pytest.mark.timeout(1000)
def test_long_context_full_size():
    """7B GQA-8 target, V=128256, batch 64 with 2048-token prompts, k=8,
    d=8: the block checks and one whole step (linear reward, selection,
    commit, next heads over the 128256-token vocabulary), two of them."""
    _full_size("long", [(8, 8)], check=[0], step_at=[(8, 8)], steps=2)
