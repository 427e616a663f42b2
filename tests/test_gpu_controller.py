"""The paper's baselines (CDLH, CDLH-appx.) and its full controller (Alg. 1
states S1..S4) on the GPU, through the C ABI, against the float64 oracle.

Every token choice is compared.  Where the GPU and the oracle choose
differently, the oracle's deciding margin there (top-k boundary, greedy draw,
acceptance test) must be within the margin of the workload's precision (1e-3
for fp32, whose logits match the oracle to ~1e-6; TOK_MARGIN for bf16):
either choice is then correct, and that prompt's comparison ends.  Rewards
are concept counts, exact on both sides."""
import math

import numpy as np
import pytest
import torch

import cdsl_inputs as ci
import oracle
from cdsl_harness import (TOK_MARGIN, assert_full_or_tie, lp_tol, make_engine, make_setup, run_and_compare,
                          soft_margins)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    s = make_setup("tiny")
    make_engine(s, B=6, max_steps=24)
    yield s
    s.engine.close()


@pytest.fixture(scope="module")
def tiny_same():
    """Draft = target: every lookahead is accepted (a = 1), so the reward
    threshold alone decides between S1 and S4."""
    s = make_setup("tiny", draft_is_target=True)
    make_engine(s, B=3, max_steps=24)
    yield s
    s.engine.close()


def _margin(s):
    return 1e-3 if s.wl.dtype == "f32" else TOK_MARGIN


def _oracle_states(s, B):
    """Prefilled oracle states of the first B prompts, kept on the setup (the
    oracle's states are immutable values)."""
    cache = s.__dict__.setdefault("_ost", {})
    if B not in cache:
        cache[B] = [oracle.prefill(s.odraft, s.otarget, p) for p in s.prompts(B)]
    return list(cache[B])


def _first_diff(a, b):
    for u, (x, y) in enumerate(zip(a, b)):
        if int(x) != int(y):
            return u
    return -1


def _cmp_head_step(M, look, rew, tok, hs, check_token=True):
    """One prompt's one-token lookahead step (GPU lookaheads [k, d+1],
    rewards [k], token) against the oracle's HeadStep.  Returns "" when
    everything matched, else the near tie that ended the comparison."""
    u = _first_diff(look[:, 0], hs.heads)
    if u >= 0:
        assert hs.head_margin <= M, (list(look[:, 0]), list(hs.heads), hs.head_margin)
        return f"head near tie ({hs.head_margin:.1e})"
    for i in range(len(hs.heads)):
        u = _first_diff(look[i, 1:], hs.x[i])
        if u >= 0:
            assert hs.margin[i, u] <= M, (i, u, list(look[i]), list(hs.x[i]), hs.margin[i])
            return f"rollout near tie ({hs.margin[i, u]:.1e})"
    assert np.allclose(rew, hs.reward, rtol=0, atol=1e-6), (rew, hs.reward)
    if check_token:
        assert tok == hs.token
    return ""


def _cmp_soft(s, sv, cs):
    """Speculative sampling's test of one prompt's iteration (sv: its
    verification buffers on the host): the draft log-probs and the
    acceptance count.  Returns "" when they match, else the near tie that
    ends the comparison."""
    am, _ = soft_margins(s.wl.dtype)
    tol = lp_tol(s.wl.dtype)
    so = cs.soft
    assert np.max(np.abs(sv["draft_lp"] - cs.roll.lq[0])) <= tol
    gn, on = int(sv["n"]), int(so.n[0])
    if gn != on:
        j = min(gn, on)
        assert so.accept_margin[0, j] <= am, (gn, on, so.accept_margin[0])
        return f"soft acceptance near tie ({so.accept_margin[0, j]:.1e})"
    return ""


def _cmp_controller(s, M, look, y, lp, out, b, cs, st, r_t, bb, it_emitted, sv=None):
    """One prompt's Alg. 1 iteration: the GPU's lookahead row [d+1] (the
    prefix's last token, then x_1..x_d), the target argmax [d] and log-probs
    [d] of the verification, the engine's outputs and the tokens the
    iteration emitted, against the oracle's ControllerStep (cs) from state
    st.  The action after x_1..x_n is compared with the oracle's candidate
    table there (for b = 1 with Step-1 folded in as the first-candidate
    rule, the form the GPU computes; a CPU pin shows it equals Step-1 then
    Step-2), and with b >= 2 every further Step-1 round with the oracle's."""
    assert look[0] == st.tokens[-1]
    u = _first_diff(look[1:], cs.x)
    if u >= 0:
        assert cs.draft_margin[u] <= M, (u, list(look), list(cs.x), cs.draft_margin)
        return f"draft near tie ({cs.draft_margin[u]:.1e})"
    assert np.max(np.abs(lp - cs.ver.logprobs[0])) <= lp_tol(s.wl.dtype)
    if cs.soft is not None:
        why = _cmp_soft(s, sv, cs)
        if why:
            return why
    else:
        u = _first_diff(y, cs.ver.y[0])
        if u >= 0:
            assert cs.ver.margin[0, u] <= M, (u, list(y), list(cs.ver.y[0]), cs.ver.margin[0])
            if out["n"][b] != cs.n:
                return f"acceptance near tie ({cs.ver.margin[0, u]:.1e})"
    assert out["n"][b] == cs.n
    assert out["r"][b] == pytest.approx(cs.r, abs=1e-6)
    assert out["states"][b] == cs.state
    acc = [int(t) for t in cs.x[:cs.n]]
    assert list(out["emitted"][b]) == acc
    ex = out["extra"]
    if cs.state == "S1":
        assert ex is None or ex["tokens"][b] < 0
        assert it_emitted == acc == cs.emitted
        return ""
    assert ex is not None and ex["tokens"][b] >= 0
    st1 = oracle.commit(s.odraft, s.otarget, st, acc)
    multi = cs.state == "S2/S3" and bb >= 2
    hs = oracle.cdlh_step(False, s.odraft, s.otarget, st1, s.wl.k, s.wl.d, s.wl.reward, s.kws[b],
                          prefer_first_at=r_t if (cs.state == "S2/S3" and bb == 1) else None)
    why = _cmp_head_step(M, ex["lookaheads"][b].cpu().numpy(), ex["reward"][b].cpu().numpy(), ex["tokens"][b], hs,
                         check_token=not multi)
    if why:
        return why
    if multi:
        # round 1 is candidate 0 of the table; rounds 2.. come from the engine
        assert cs.step1[0].X == [int(hs.heads[0])] and cs.step1[0].reward == pytest.approx(hs.reward[0])
        for ri, rd in enumerate(out["rounds"]):
            if not rd["active"][b]:
                break
            t = cs.step1[ri + 1]
            if rd["X"][b] != t.X[-1]:
                assert t.x_margin <= M, (rd["X"][b], t.X, t.x_margin)
                return f"step-1 token near tie ({t.x_margin:.1e})"
            u = _first_diff(rd["lookaheads"][b, 0, 1:].cpu().numpy(), t.lh)
            if u >= 0:
                assert t.lh_margin[u] <= M, (u, t.lh, t.lh_margin)
                return f"step-1 lookahead near tie ({t.lh_margin[u]:.1e})"
            assert rd["reward"][b] == pytest.approx(t.reward, abs=1e-6)
    assert it_emitted == cs.emitted, (it_emitted, cs.emitted)
    return ""


def _run_head_steps(s, B, steps, roller):
    eng = s.engine
    k, d = s.wl.k, s.wl.d
    st = eng.start(torch.from_numpy(s.prompts(B)).cuda())
    kw = torch.from_numpy(s.kws[:B]).cuda()
    ost = _oracle_states(s, B)
    alive = [True] * B
    compared = 0
    for _ in range(steps):
        out = eng.head_step(st, kw, roller)
        look = out["lookaheads"].cpu().numpy()
        rew = out["reward"].cpu().numpy()
        for b in range(B):
            if not alive[b]:
                continue
            hs = oracle.cdlh_step(roller == 1, s.odraft, s.otarget, ost[b], k, d, s.wl.reward, s.kws[b])
            why = _cmp_head_step(_margin(s), look[b], rew[b], out["tokens"][b], hs)
            if why:
                print(f"prompt {b}: stopped after {compared} compared steps: {why}")
                alive[b] = False
                continue
            ost[b] = hs.state
            compared += 1
    for b in range(B):
        if alive[b]:
            assert st.emitted[b] == ost[b].generated
    assert st.prefix.lengths() == [s.wl.prompt_len + len(e) for e in st.emitted]
    st.prefix.free()
    print("compared", compared)
    return compared


def _run_controller(s, B, steps, a_t, r_t, bb, soft=False):
    eng = s.engine
    k, d = s.wl.k, s.wl.d
    st = eng.start(torch.from_numpy(s.prompts(B)).cuda())
    kw = torch.from_numpy(s.kws[:B]).cuda()
    ost = _oracle_states(s, B)
    alive = [True] * B
    stopped = {}
    seen = set()
    compared = 0
    cb = eng._controller_buffers(B, k, d)
    for t in range(steps):
        u = None
        if soft:
            # uniforms of the one lookahead per prompt: [B, d]
            u = ci.uniforms(s.wl.seed, 0, t, B, 1, d)[:, 0]
        before = [len(e) for e in st.emitted]
        out = eng.controller_step(st, kw, a_t, r_t, bb, u=torch.from_numpy(np.ascontiguousarray(u)).cuda()
                                  if soft else None)
        look = cb["look"].cpu().numpy()
        y = cb["verify"]["target_argmax"].cpu().numpy()
        lp = cb["verify"]["logprobs"].cpu().numpy()
        if soft:
            sv = {nm: cb["verify"][nm].cpu().numpy() for nm in ("draft_lp", "n_accept")}
        for b in range(B):
            if not alive[b]:
                continue
            cs = oracle.controller_step(s.odraft, s.otarget, ost[b], k, d, a_t, r_t, bb, s.wl.reward, s.kws[b],
                                        rejection="soft" if soft else "hard", u=u[b][None] if soft else None)
            svb = {"draft_lp": sv["draft_lp"][b], "n": sv["n_accept"][b]} if soft else None
            why = _cmp_controller(s, _margin(s), look[b], y[b], lp[b], out, b, cs, ost[b], r_t, bb,
                                  [int(t) for t in st.emitted[b][before[b]:]], svb)
            if why:
                print(f"prompt {b}: stopped after {compared} compared steps: {why}")
                alive[b] = False
                stopped[b] = why
                continue
            seen.add(cs.state)
            if cs.n > 0:
                seen.add("accepted")
            if len(cs.step1) > 1:
                seen.add("step1 round 2")
                if cs.extra is None:
                    seen.add("step1 round 2 kept")
                else:
                    seen.add("step1 withdrawn")
            ost[b] = cs.after
            compared += 1
    for b in range(B):
        if alive[b]:
            assert st.emitted[b] == ost[b].generated
    assert st.prefix.lengths() == [s.wl.prompt_len + len(e) for e in st.emitted]
    st.prefix.free()
    # every prompt ran every iteration, or ended at a logged near tie
    assert all(alive[b] or b in stopped for b in range(B))
    print("compared", compared, "states seen:", sorted(seen), "stopped:", stopped)
    return compared, seen, stopped


@pytest.mark.parametrize("roller", [0, 1])
def test_head_steps_match_oracle(tiny, roller):
    """CDLH (roller 1, the target) and CDLH-appx. (roller 0, the draft):
    8 one-token steps for 6 prompts."""
    assert _run_head_steps(tiny, 6, 8, roller) >= 10


@pytest.mark.parametrize("which,a_t,r_t,bb,state", [
    ("tiny", 0.5, 1.0, 1, "S2/S3"), ("tiny", 0.5, 1.0, 0, "S2/S3"),
    ("tiny_same", 0.5, 0.0, 0, "S1"), ("tiny_same", 0.5, 1.0, 1, "S4")])
def test_controller_steps_match_oracle(request, which, a_t, r_t, bb, state):
    """Alg. 1 with hard rejection, 5 iterations for 3 prompts: the draft
    from the prefix, the verification, n, r, the state, the Step-1 / Step-2
    token and the emitted tokens."""
    compared, seen, stopped = _run_controller(request.getfixturevalue(which), 3, 5, a_t, r_t, bb)
    assert compared >= 5
    assert compared == 15 or stopped
    assert state in seen


@pytest.mark.parametrize("which,a_t,r_t,bb,state", [
    ("tiny", 0.5, 1.0, 1, "S2/S3"), ("tiny", 0.3, 0.0, 0, "S2/S3"),
    ("tiny_same", 0.5, 0.0, 0, "S1"), ("tiny_same", 0.5, 1.0, 1, "S4")])
def test_soft_controller_steps_match_oracle(request, which, a_t, r_t, bb, state):
    """Alg. 1 with speculative sampling's test in the rejection loop, 5
    iterations for 3 prompts on seeded uniforms: the draft, its log-probs,
    the acceptance count, r, the state and the emitted tokens.  With draft =
    target every token is accepted (p = q)."""
    compared, seen, stopped = _run_controller(request.getfixturevalue(which), 3, 5, a_t, r_t, bb, soft=True)
    assert compared >= 5
    assert compared == 15 or stopped
    assert state in seen


@pytest.mark.parametrize("r_t", [1.0, 2.0])
def test_controller_step1_two_rounds_match_oracle(tiny, r_t):
    """Alg. 1 with b = 2 (a_t = 2 keeps every prompt in S2/S3): when M_p's
    first token misses r_t, it is appended tentatively and its successor is
    scored; a second miss withdraws it and Step-2 decides.  6 prompts, 5
    iterations, every round compared with the oracle's."""
    compared, seen, stopped = _run_controller(tiny, 6, 5, 2.0, r_t, 2)
    assert compared >= 10
    assert compared == 30 or stopped
    assert "step1 round 2" in seen and "step1 withdrawn" in seen
    if r_t == 1.0:
        assert "step1 round 2 kept" in seen


def test_one_token_prompts():
    """Prompts of a single token: the beam step, and Alg. 1 drafting from
    the prefix, whose first pass re-feeds that token at position 0 over an
    empty prefix; 4 iterations for 3 prompts each, against the oracle."""
    s = make_setup("tiny", prompt_len=1)
    make_engine(s, B=3, max_steps=12)
    try:
        st, reps = run_and_compare(s, B=3, steps=4, check_prompts=[0, 1, 2])
        assert_full_or_tie(reps, 4)
        st.prefix.free()
        compared, seen, stopped = _run_controller(s, 3, 4, 0.5, 1.0, 1)
        assert compared == 12 or stopped
        assert "S2/S3" in seen
    finally:
        s.engine.close()


def test_controller_error_paths(tiny):
    from paper_2412_10418_amd.binding import CDSLError
    s, eng = tiny, tiny.engine
    st = eng.start(torch.from_numpy(s.prompts(1)).cuda())
    kw = torch.from_numpy(s.kws[:1]).cuda()
    with pytest.raises(ValueError):
        eng.controller_step(st, kw, 0.5, 1.0, -1)
    with pytest.raises(ValueError):
        eng.controller_step(st, kw, 0.0, 1.0, 1)
    # a head-only commit without a rollout is out of order
    with pytest.raises(CDSLError):
        eng.ctx.cdsl_commit_heads(st.prefix, torch.zeros(1, s.wl.k, s.wl.d + 1, dtype=torch.int32, device="cuda"),
                                  torch.zeros(1, dtype=torch.int32, device="cuda"), s.wl.k, s.wl.d, None,
                                  st.beams, st.head_lp)
    # an Alg. 1 commit needs a draft and a verification from the prefix
    d = s.wl.d
    look = torch.zeros(1, d + 1, dtype=torch.int32, device="cuda")
    z = lambda *sh, dt=torch.float32: torch.zeros(sh, dtype=dt, device="cuda")
    with pytest.raises(CDSLError):
        eng.ctx.cdsl_commit_prefix(st.prefix, look, z(1, dt=torch.int32), d, z(1, d, s.wl.k, dt=torch.int32),
                                   z(1, d, s.wl.k), st.beams, st.head_lp)
    # a beam verification does not commit as an Alg. 1 iteration
    eng.ctx.cdsl_draft_prefix(st.prefix, d, look)
    vb = eng.ctx.cdsl_verify(st.prefix, torch.zeros(1, 1, d + 1, dtype=torch.int32, device="cuda"), 1, d,
                             z(1, 1), kk=s.wl.k)
    with pytest.raises(CDSLError):
        eng.ctx.cdsl_commit_prefix(st.prefix, look, vb["n_accept"].view(1), d, vb["row_topk_ids"].view(1, d, -1),
                                   vb["row_topk_lp"].view(1, d, -1), st.beams, st.head_lp)
    st.prefix.free()


@pytest.fixture(scope="module")
def small():
    s = make_setup("small")
    make_engine(s, B=2, max_steps=12)
    yield s
    s.engine.close()


# the float64 oracle of the 24-layer target takes ~15 s per step on the host
@pytest.mark.timeout(900)
@pytest.mark.parametrize("roller", [0, 1])
def test_small_bf16_head_steps_match_oracle(small, roller):
    """bf16 weights: CDLH rolls with the hd = 128 target (4 key groups do
    not fit, so 2 key groups and both row tiles per workgroup), CDLH-appx.
    with the hd = 64 draft; 2 one-token steps for 2 prompts."""
    assert _run_head_steps(small, 2, 2, roller) >= 1


@pytest.mark.timeout(900)
def test_small_bf16_controller_matches_oracle(small):
    compared, _, stopped = _run_controller(small, 2, 2, 0.4, 0.3, 1)
    assert compared == 4 or stopped


@pytest.mark.timeout(900)
def test_small_bf16_controller_step1_two_rounds_match_oracle(small):
    """b = 2 on the bf16 pair (a_t = 2 keeps every prompt in S2/S3): the
    tentative append of M_p's token into the hi/lo KV pool, the second
    round's rollout and reward, and the withdrawal; 2 iterations for 2
    prompts."""
    compared, seen, stopped = _run_controller(small, 2, 2, 2.0, 1.0, 2)
    assert compared == 4 or stopped
    assert "step1 round 2" in seen or stopped


@pytest.mark.timeout(900)
def test_small_bf16_soft_controller_matches_oracle(small):
    """Alg. 1 with speculative sampling's test on the bf16 pair: 2
    iterations for 2 prompts."""
    compared, _, stopped = _run_controller(small, 2, 2, 0.4, 0.3, 1, soft=True)
    assert compared == 4 or stopped
