"""Speculative sampling (soft rejection) on the GPU, through the C ABI,
against the float64 oracle: the row kernel (draft log-prob of the drafted
token, residual draw from the normalised max(0, p - q)) on given logits, and
whole CDSL steps with soft rejection on seeded uniforms.

Decisions that floating point takes (an acceptance test near its bound, a
residual draw near a cumulative boundary) are compared exactly where the
oracle's margin exceeds what the log-prob tolerance allows; closer to the
boundary the GPU's choice must still be a valid one (its interval of the
oracle's residual distribution holds v within that margin), and the
trajectory comparison ends there."""
import numpy as np
import pytest
import torch

import cdsl_inputs as ci
import oracle
from cdsl_harness import assert_full_or_tie, make_engine, make_setup, run_and_compare

pytestmark = pytest.mark.gpu


def _soft_rows_case(M, d, V, seed):
    rng = np.random.default_rng([seed, M, V])
    zp = (rng.standard_normal((M, V)) * 2.0).astype(np.float32)
    zq = (rng.standard_normal((M, V)) * 2.0).astype(np.float32)
    zq[0] = zp[0]                       # p = q: no residual mass, argmax p
    zp[1, :] = 0.0                      # uniform p ...
    zq[1, 7 % V] = 30.0                 # ... and a q with all its mass on one token
    if M > 2:
        zp[2, V - 1] = 25.0             # the mass at the last id
    look = rng.integers(0, V, (M // d, d + 1)).astype(np.int32)
    v = rng.random(M).astype(np.float32)
    v[min(3, M - 1)] = 0.0
    v[M - 1] = np.nextafter(np.float32(1.0), np.float32(0.0))
    return zp, zq, look, v


@pytest.mark.parametrize("M,d,V", [(12, 4, 1024), (6, 3, 32000), (4, 2, 128256), (10, 10, 997)])
def test_soft_rows_match_oracle(M, d, V):
    from paper_2412_10418_amd.binding import cdsl_op_soft_rows
    zp, zq, look, v = _soft_rows_case(M, d, V, 1)
    t = lambda a: torch.from_numpy(a).cuda()
    dlp, rid, rlp = cdsl_op_soft_rows(t(zp), t(zq), d, t(look), t(v))
    dlp, rid, rlp = (x.cpu().numpy() for x in (dlp, rid, rlp))
    exact = 0
    for m in range(M):
        x = look[m // d, m % d + 1]
        assert abs(dlp[m] - oracle.log_softmax(zq[m].astype(np.float64))[x]) < 5e-5
        tok, lp, mg = oracle.residual_sample(zp[m].astype(np.float64), zq[m].astype(np.float64), float(v[m]))
        if m == 0:
            assert rid[m] == tok == oracle.argmax_lowest(zp[m])
        if rid[m] == tok:
            exact += 1
            assert abs(rlp[m] - lp) < 5e-5
            continue
        # inputs are the same fp32 values: only summation order differs
        lo, hi, Z = oracle.residual_interval(zp[m].astype(np.float64), zq[m].astype(np.float64), int(rid[m]))
        assert mg < 1e-4 and hi > lo and lo - 1e-4 <= v[m] <= hi + 1e-4, (m, rid[m], tok, mg, lo, hi, v[m])
    assert exact >= M - 1


@pytest.fixture(scope="module")
def tiny():
    s = make_setup("tiny")
    make_engine(s, B=3, max_steps=10)
    yield s
    s.engine.close()


def test_tiny_soft_steps_match_oracle(tiny):
    """fp32: 8 whole steps for 3 prompts with soft rejection; the uniforms
    come from the seeded generator both sides read."""
    st, reps = run_and_compare(tiny, B=3, steps=8, check_prompts=[0, 1, 2], soft=True)
    total = 0
    for b, r in reps.items():
        print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
        total += r.steps_compared
    assert total >= 12
    assert_full_or_tie(reps, 8)
    st.prefix.free()


def test_soft_acceptance_depends_on_u(tiny):
    """u = 0 keeps every drafted token (n = d); u just below 1 keeps only
    tokens the target likes at least as much as the draft."""
    s, eng = tiny, tiny.engine
    k, d = s.wl.k, s.wl.d
    kw = torch.from_numpy(s.kws[:3]).cuda()
    for fill, expect_all in ((0.0, True), (np.nextafter(np.float32(1.0), np.float32(0.0)), False)):
        st = eng.start(torch.from_numpy(s.prompts(3)).cuda())
        u = torch.full((3, k, d), float(fill), dtype=torch.float32, device="cuda")
        v = torch.full((3, k, d), 0.5, dtype=torch.float32, device="cuda")
        bf = eng.step(st, keywords=kw, u=u, v=v)
        n = bf.verify["n_accept"].cpu().numpy()
        lp = bf.verify["logprobs"].cpu().numpy()
        lq = bf.verify["draft_lp"].cpu().numpy()
        if expect_all:
            assert (n == d).all()
        else:
            # n lies between the run of tokens surely kept (p/q >= 1 by a
            # clear margin) and the run of tokens not surely rejected
            def run(mask):
                r = 0
                while r < d and mask[r]:
                    r += 1
                return r
            for b in range(3):
                for i in range(k):
                    diff = lp[b, i] - lq[b, i]
                    assert run(diff >= 1e-5) <= n[b, i] <= run(diff >= -1e-5), (diff, n[b, i])
        st.prefix.free()


def test_tiny_soft_draft_equal_to_target_accepts_all():
    s = make_setup("tiny", draft_is_target=True)
    make_engine(s, B=2, max_steps=6)
    try:
        st, reps = run_and_compare(s, B=2, steps=3, check_prompts=[0, 1], soft=True)
        for r in reps.values():
            assert r.steps_compared == 3, r.stopped
        st.prefix.free()
    finally:
        s.engine.close()


def test_soft_error_paths(tiny):
    import ctypes
    from paper_2412_10418_amd import binding
    from paper_2412_10418_amd.binding import CDSLError
    s, eng = tiny, tiny.engine
    k, d = s.wl.k, s.wl.d
    st = eng.start(torch.from_numpy(s.prompts(1)).cuda())
    bf = eng.buffers(1, k, d)
    sb = eng._soft_buffers(1, k, d, bf)
    u = torch.zeros((1, k, d), dtype=torch.float32, device="cuda")
    c = eng.ctx
    # soft verification needs the logits of a keeping rollout
    c.cdsl_rollout(st.prefix, st.beams, k, d, bf.lookaheads)
    with pytest.raises(CDSLError):
        c.cdsl_verify_soft(st.prefix, bf.lookaheads, k, d, st.head_lp, sb["draft_logits"], u, u, bf.verify)
    # a soft verification is committed by cdsl_commit_soft only, and back
    c.cdsl_rollout_keep(st.prefix, st.beams, k, d, bf.lookaheads, sb["draft_logits"])
    c.cdsl_verify_soft(st.prefix, bf.lookaheads, k, d, st.head_lp, sb["draft_logits"], u, u, bf.verify)
    with pytest.raises(CDSLError):
        c.cdsl_commit(st.prefix, bf.lookaheads, bf.beam.zero_(), bf.verify["n_accept"], bf.verify["row_topk_ids"],
                      bf.verify["row_topk_lp"], k, d, bf.next_beams, bf.next_head_lp)
    c.cdsl_verify(st.prefix, bf.lookaheads, k, d, st.head_lp, out=bf.verify)
    with pytest.raises(CDSLError):
        c.cdsl_commit_soft(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"], bf.verify["row_topk_ids"],
                           bf.verify["row_topk_lp"], bf.verify["res_ids"], bf.verify["res_lp"], k, d,
                           bf.next_beams, bf.next_head_lp)
    # the commit's next-head width must be the soft verification's top-k
    # width: the binding refuses buffers of another width, and the library
    # refuses the call itself (before it reads anything)
    c.cdsl_rollout_keep(st.prefix, st.beams, k, d, bf.lookaheads, sb["draft_logits"])
    c.cdsl_verify_soft(st.prefix, bf.lookaheads, k, d, st.head_lp, sb["draft_logits"], u, u, bf.verify)
    nb = torch.zeros((1, k - 1), dtype=torch.int32, device="cuda")
    nl = torch.zeros((1, k - 1), dtype=torch.float32, device="cuda")
    with pytest.raises(ValueError):
        c.cdsl_commit_soft(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"], bf.verify["row_topk_ids"],
                           bf.verify["row_topk_lp"], bf.verify["res_ids"], bf.verify["res_lp"], k, d, nb, nl)
    em, ne = (ctypes.c_int32 * (d + 1))(), (ctypes.c_int32 * 1)()
    vb = bf.verify
    rc = binding.lib().cdsl_commit_soft(c.handle, st.prefix.handle, bf.lookaheads.data_ptr(), bf.beam.data_ptr(),
                                        vb["n_accept"].data_ptr(), vb["row_topk_ids"].data_ptr(),
                                        vb["row_topk_lp"].data_ptr(), vb["res_ids"].data_ptr(),
                                        vb["res_lp"].data_ptr(), k, d, k - 1, em, ne, nb.data_ptr(), nl.data_ptr())
    assert rc == binding.CDSL_ESTATE
    # top-k buffers of another width are refused before any launch
    with pytest.raises(ValueError):
        c.cdsl_verify_soft(st.prefix, bf.lookaheads, k, d, st.head_lp, sb["draft_logits"], u, u, bf.verify,
                           kk=k - 1)
    st.prefix.free()


@pytest.mark.timeout(900)
def test_small_bf16_soft_steps_match_oracle():
    """bf16 12L/24L pair, 2 prompts, 2 soft steps."""
    s = make_setup("small")
    make_engine(s, B=2, max_steps=4)
    try:
        st, reps = run_and_compare(s, B=2, steps=2, check_prompts=[0, 1], soft=True)
        for b, r in reps.items():
            print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
        assert_full_or_tie(reps, 2)
        st.prefix.free()
    finally:
        s.engine.close()
