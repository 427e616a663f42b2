"""End-to-end parity of the CDSL step on the GPU (C ABI) against the
float64 CPU oracle, on the seeded workloads."""
import math

import numpy as np
import pytest
import torch

import cdsl_inputs as ci
import oracle
from cdsl_harness import TOK_MARGIN, assert_full_or_tie, lp_tol, make_engine, make_setup, run_and_compare

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    s = make_setup("tiny")
    make_engine(s, B=3, max_steps=12)
    yield s
    s.engine.close()


def test_tiny_fp32_eight_steps_match_oracle(tiny):
    """The fp32 workload (k=4, d=4, 8 steps) for 3 prompts, every prompt
    compared with its own oracle run; log-probs within 1e-4."""
    st, reps = run_and_compare(tiny, B=3, steps=8, check_prompts=[0, 1, 2])
    for b, r in reps.items():
        print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
    assert_full_or_tie(reps, 8)
    lens = st.prefix.lengths()
    assert lens == [tiny.wl.prompt_len + len(e) for e in st.emitted]
    st.prefix.free()


def test_tiny_alpha_infinity_and_zero(tiny):
    for alpha in (math.inf, 0.0):
        st, reps = run_and_compare(tiny, B=2, steps=3, check_prompts=[0, 1], alpha=alpha)
        assert_full_or_tie(reps, 3)
        st.prefix.free()


def test_tiny_batch_independence_is_bitwise(tiny):
    """A prompt's outputs do not depend on the other prompts of the batch."""
    eng = tiny.engine
    outs = []
    for B in (1, 3):
        p = torch.from_numpy(tiny.prompts(B)).cuda()
        st = eng.start(p)
        kw = torch.from_numpy(tiny.kws[:B]).cuda()
        bf = eng.step(st, keywords=kw)
        outs.append((bf.lookaheads[0].cpu().clone(), bf.verify["logprobs"][0].cpu().clone(), st.emitted[0][:]))
        st.prefix.free()
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])
    assert outs[0][2] == outs[1][2]


def test_tiny_deterministic(tiny):
    res = []
    for _ in range(2):
        p = torch.from_numpy(tiny.prompts(3)).cuda()
        st = tiny.engine.start(p)
        kw = torch.from_numpy(tiny.kws[:3]).cuda()
        for _ in range(3):
            bf = tiny.engine.step(st, keywords=kw)
        res.append((bf.verify["logprobs"].cpu().clone(), [e[:] for e in st.emitted]))
        st.prefix.free()
    assert torch.equal(res[0][0], res[1][0]) and res[0][1] == res[1][1]


def test_verify_is_stateless_on_oracle_lookaheads(tiny):
    """Feed the oracle's own lookaheads to cdsl_verify: every verification
    output matches the oracle's verification of the same tokens."""
    s = tiny
    eng = s.engine
    k, d = s.wl.k, s.wl.d
    prompts = s.prompts(2)
    st = eng.start(torch.from_numpy(prompts).cuda())
    look = np.zeros((2, k, d + 1), np.int32)
    ovs = []
    for b in range(2):
        ost = oracle.prefill(s.odraft, s.otarget, prompts[b])
        heads, hlp, _ = oracle.beam_heads(ost, k)
        # a lookahead that is NOT the draft's: random tokens
        x = np.random.default_rng(b).integers(0, s.wl.target.vocab, (k, d))
        look[b, :, 0] = heads
        look[b, :, 1:] = x
        ovs.append(oracle.verify(s.otarget, ost, heads, hlp, x))
    out = eng.ctx.cdsl_verify(st.prefix, torch.from_numpy(look).cuda(), k, d, st.head_lp)
    for b in range(2):
        ve = ovs[b]
        assert np.max(np.abs(out["logprobs"][b].cpu().numpy() - ve.logprobs)) < 1e-4
        ok = ve.margin > TOK_MARGIN
        assert np.array_equal(out["target_argmax"][b].cpu().numpy()[ok], ve.y[ok])
        rtk = out["row_topk_ids"][b].cpu().numpy()
        for i in range(k):
            for j in range(d):
                z = np.sort(ve.logits[i, j])[::-1][:k + 1]
                if np.all(-np.diff(z) > TOK_MARGIN):
                    assert list(rtk[i, j]) == list(ve.row_topk[i, j])
    st.prefix.free()


def test_draft_equal_to_target_accepts_all_and_catches_up():
    """Draft = target: every lookahead token is accepted (n = d), d + 1
    tokens are emitted per step and the catch-up pass completes the
    prefix; the trajectory matches the oracle."""
    s = make_setup("tiny", draft_is_target=True)
    make_engine(s, B=2, max_steps=6)
    try:
        st, reps = run_and_compare(s, B=2, steps=4, check_prompts=[0, 1])
        assert_full_or_tie(reps, 4)
        assert all(len(e) >= 3 * (s.wl.d + 1) for e in st.emitted)
        st.prefix.free()
    finally:
        s.engine.close()


def test_k1_is_greedy_decoding_of_target():
    s = make_setup("tiny")
    make_engine(s, B=1, max_steps=10, k=1, d=3)
    try:
        st, reps = run_and_compare(s, B=1, steps=5, check_prompts=[0], k=1, d=3)
        assert_full_or_tie(reps, 5)
        # the oracle's k=1 result is itself pinned to greedy decoding
        seq = list(s.prompts(1)[0])
        from oracle.decoder import Decoder
        out = []
        for _ in range(len(st.emitted[0])):
            z = s.otarget.full(seq).logits[-1]
            seq.append(int(np.argmax(z)))
        greedy = seq[s.wl.prompt_len:]
        assert st.emitted[0][:len(greedy)] == greedy
        st.prefix.free()
    finally:
        s.engine.close()


def test_error_paths(tiny):
    from paper_2412_10418_amd.binding import CDSLError, CDSL_ERANGE, CDSL_EINVAL, CDSL_ESTATE
    eng = tiny.engine
    p = torch.from_numpy(tiny.prompts(1)).cuda()
    st = eng.start(p)
    wide = torch.zeros((1, tiny.wl.k + 1), dtype=torch.int32, device="cuda")
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_rollout(st.prefix, wide, tiny.wl.k + 1, tiny.wl.d)
    assert e.value.code == CDSL_ERANGE
    with pytest.raises(ValueError):       # buffers of the wrong size never reach the library
        eng.ctx.cdsl_rollout(st.prefix, st.beams, tiny.wl.k + 1, tiny.wl.d)
    bf = eng.buffers(1, tiny.wl.k, tiny.wl.d)
    with pytest.raises(CDSLError) as e:   # commit before rollout/verify
        eng.ctx.cdsl_commit(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                            bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], tiny.wl.k, tiny.wl.d)
    assert e.value.code == CDSL_ESTATE
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_select(bf.verify["scores"], bf.reward, -math.inf, bf.beam)
    assert e.value.code == CDSL_EINVAL
    # NaN score -> beam -1 -> commit reports EINVAL
    eng.ctx.cdsl_rollout(st.prefix, st.beams, tiny.wl.k, tiny.wl.d, bf.lookaheads)
    eng.ctx.cdsl_verify(st.prefix, bf.lookaheads, tiny.wl.k, tiny.wl.d, st.head_lp, out=bf.verify)
    bf.verify["scores"][0, 1] = float("nan")
    eng.ctx.cdsl_select(bf.verify["scores"], bf.reward, 1.0, bf.beam)
    assert int(bf.beam[0]) == -1
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_commit(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                            bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], tiny.wl.k, tiny.wl.d)
    assert e.value.code == CDSL_EINVAL
    st.prefix.free()


@pytest.fixture(scope="module")
def small():
    s = make_setup("small")
    make_engine(s, B=8, max_steps=4)
    yield s
    s.engine.close()


def test_small_bf16_steps_match_oracle(small):
    """bf16 12L/24L pair at its full batch (8 prompts x 128 tokens, k=5,
    d=5); prompts 0 and 5 are compared with the oracle."""
    st, reps = run_and_compare(small, B=8, steps=3, check_prompts=[0, 5])
    for b, r in reps.items():
        print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
    assert_full_or_tie(reps, 3)
    st.prefix.free()


def test_small_bf16_verify_on_oracle_lookaheads(small):
    s = small
    k, d = s.wl.k, s.wl.d
    prompts = s.prompts(8)
    st = s.engine.start(torch.from_numpy(prompts).cuda())
    look = np.zeros((8, k, d + 1), np.int32)
    rng = np.random.default_rng(3)
    ost = oracle.prefill(s.odraft, s.otarget, prompts[6])
    heads, hlp, _ = oracle.beam_heads(ost, k)
    look[:, :, 0] = st.beams.cpu().numpy()
    look[:, :, 1:] = rng.integers(0, s.wl.target.vocab, (8, k, d))
    look[6, :, 0] = heads
    out = s.engine.ctx.cdsl_verify(st.prefix, torch.from_numpy(look).cuda(), k, d, st.head_lp)
    ve = oracle.verify(s.otarget, ost, heads, hlp, look[6, :, 1:])
    err = np.max(np.abs(out["logprobs"][6].cpu().numpy() - ve.logprobs))
    print("bf16 verify max |dlp|", err)
    assert err < 2e-2
    st.prefix.free()


@pytest.mark.timeout(900)
def test_small_bf16_draft_equal_to_target_catches_up():
    """bf16 with the 24-layer target as its own draft: the lookaheads are
    accepted (n = d up to near ties between the rollout's and the
    verification's rounding), so the commit promotes d rows of the hi / lo
    KV planes and feeds x_d as the catch-up row through both models."""
    s = make_setup("small", draft_is_target=True)
    make_engine(s, B=2, max_steps=4)
    try:
        st, reps = run_and_compare(s, B=2, steps=2, check_prompts=[0])
        for b, r in reps.items():
            print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
        assert_full_or_tie(reps, 2)
        assert len(st.emitted[0]) == 2 * (s.wl.d + 1) or reps[0].stopped
        st.prefix.free()
    finally:
        s.engine.close()


@pytest.mark.timeout(900)
def test_small_bf16_k1_matches_oracle():
    """bf16, one beam (k = 1): the step is greedy speculative decoding of the
    target with no bonus token, compared with the oracle for 3 steps."""
    s = make_setup("small")
    make_engine(s, B=2, max_steps=4, k=1, d=5)
    try:
        st, reps = run_and_compare(s, B=2, steps=3, check_prompts=[1], k=1, d=5)
        assert_full_or_tie(reps, 3)
        st.prefix.free()
    finally:
        s.engine.close()


@pytest.mark.parametrize("same", [False, True])
def test_one_lookahead_token_matches_oracle(same):
    """d = 1, the smallest lookahead: one draft pass per beam, one verified
    row per beam, with k = 4 beams and with a single beam, hard and soft
    rejection.  With draft = target every token is accepted, so n = d = 1
    and every step feeds the catch-up row."""
    s = make_setup("tiny", draft_is_target=same)
    make_engine(s, B=3, max_steps=10, k=4, d=1)
    try:
        for k in (4, 1):
            for soft in (False, True):
                st, reps = run_and_compare(s, B=3, steps=6, check_prompts=[0, 1, 2], k=k, d=1, soft=soft)
                for b, r in reps.items():
                    print(f"same={same} k={k} soft={soft} prompt {b}: {r.steps_compared} steps, "
                          f"max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
                assert_full_or_tie(reps, 6)
                if same:
                    assert all(len(e) == 6 * 2 for e in st.emitted)   # c + x_1 every step
                st.prefix.free()
    finally:
        s.engine.close()


def test_largest_k_and_d_match_oracle():
    """The largest beam count and lookahead depth the library takes (k = 16,
    d = 32: two suffix blocks per beam, 512 verified rows per prompt, top-16
    rows), hard and soft rejection, against the oracle."""
    s = make_setup("tiny")
    make_engine(s, B=2, max_steps=6, k=16, d=32)
    try:
        st, reps = run_and_compare(s, B=2, steps=2, check_prompts=[0, 1], k=16, d=32)
        for b, r in reps.items():
            print(f"hard, prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
        assert_full_or_tie(reps, 2)
        st.prefix.free()
        st, reps = run_and_compare(s, B=2, steps=2, check_prompts=[0, 1], k=16, d=32, soft=True)
        for b, r in reps.items():
            print(f"soft, prompt {b}: {r.steps_compared} steps, stop: {r.stopped or '-'}")
        assert_full_or_tie(reps, 2)
        st.prefix.free()
    finally:
        s.engine.close()


def test_batch_and_context_limits(tiny):
    """An empty batch, a batch or prompt beyond the limits, and a context
    that runs out are reported as errors (nothing is launched for them),
    and the prefix never grows past max_ctx."""
    from paper_2412_10418_amd.binding import CDSLError, CDSL_ERANGE, CDSL_EINVAL
    eng = tiny.engine
    L = tiny.wl.prompt_len
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_prefill(torch.zeros((0, L), dtype=torch.int32, device="cuda"), tiny.wl.k)
    assert e.value.code == CDSL_EINVAL
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_prefill(torch.zeros((7, L), dtype=torch.int32, device="cuda"), tiny.wl.k)
    assert e.value.code == CDSL_ERANGE
    with pytest.raises(CDSLError) as e:
        eng.ctx.cdsl_prefill(torch.zeros((1, L + 1), dtype=torch.int32, device="cuda"), tiny.wl.k)
    assert e.value.code == CDSL_ERANGE
    # the tiny engine holds prompt + 8 steps of d + 1 tokens: keep stepping
    # until the next lookahead would not fit
    st = eng.start(torch.from_numpy(tiny.prompts(1)).cuda())
    kw = torch.from_numpy(tiny.kws[:1]).cuda()
    max_ctx = eng.ctx.limits["max_ctx"]
    raised = False
    for _ in range(200):
        try:
            eng.step(st, keywords=kw)
        except CDSLError as err:
            assert err.code == CDSL_ERANGE
            raised = True
            break
        assert max(st.prefix.lengths()) <= max_ctx
    assert raised
    assert max(st.prefix.lengths()) + tiny.wl.d + 1 > max_ctx
    st.prefix.free()
