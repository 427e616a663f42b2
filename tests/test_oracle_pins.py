"""Pins for the CPU oracle: every check compares it with something other than
itself (an independent library decoder, brute force, closed forms, the
paper's worked example, algebraic invariants of the method)."""
import json
import math
import os

import numpy as np
import pytest

import cdsl_inputs as ci
import oracle
from oracle import decoder as odec

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

GQA = ci.ModelShape(2, 32, 4, 2, 48, 64)      # G = 2
MHA = ci.ModelShape(3, 48, 3, 3, 64, 64)      # hd = 16


def _weights(shape, model_id, gains=True, seed=7):
    w = ci.model_weights(shape, seed, model_id, "f32", threads=1)
    # scale so the random model has sharp distributions, and random gains so a
    # dropped norm gain cannot go unnoticed
    rng = np.random.default_rng([seed, 99, model_id])
    for lw in w["layers"]:
        for nm in ci.LAYER_MATS:
            lw[nm] = lw[nm] * 10.0
        if gains:
            lw["attn_norm"] = rng.uniform(0.5, 1.5, shape.d_model)
            lw["mlp_norm"] = rng.uniform(0.5, 1.5, shape.d_model)
    w["tok_emb"] = w["tok_emb"] * 10.0
    w["lm_head"] = w["lm_head"] * 10.0
    if gains:
        w["final_norm"] = rng.uniform(0.5, 1.5, shape.d_model)
    return w


@pytest.fixture(scope="module")
def models():
    from hf_ref import hf_llama
    out = {}
    for nm, shape, mid in (("gqa", GQA, 0), ("mha", MHA, 1)):
        w = _weights(shape, mid)
        out[nm] = (shape, w, odec.Decoder(shape, w), hf_llama(shape, w))
    return out


def _prompt(n, V, seed=3):
    return np.random.default_rng(seed).integers(0, V, n)


# ---------------------------------------------------------------------------
# the decoder against an independent implementation
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("which", ["gqa", "mha"])
def test_decoder_matches_library_llama(models, which):
    from hf_ref import hf_logits
    shape, w, dec, hf = models[which]
    toks = _prompt(21, shape.vocab)
    ours = dec.full(toks).logits
    ref = hf_logits(hf, toks)
    # the library evaluates the rotary angles in float32 (its only non-fp64
    # step), hence 2e-5 rather than 1e-12; planted mistakes below give > 1e-3
    assert np.max(np.abs(ours - ref)) < 2e-5 * max(1.0, np.max(np.abs(ref)))


def test_plausible_mistakes_fail_the_library_pin(models, monkeypatch):
    """Planted oracle mistakes (in the oracle, on the CPU) are caught."""
    from hf_ref import hf_logits
    shape, w, dec, hf = models["gqa"]
    toks = _prompt(12, shape.vocab)
    ref = hf_logits(hf, toks)

    def wrong_rope(x, pos, theta):  # interleaved pairing instead of rotate-half
        hd = x.shape[-1]
        inv = theta ** (-(np.arange(hd // 2) * 2.0) / hd)
        ang = np.asarray(pos, float)[:, None] * inv[None, :]
        c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        x1, x2 = x[..., 0::2], x[..., 1::2]
        o = np.empty_like(x)
        o[..., 0::2] = x1 * c - x2 * s
        o[..., 1::2] = x2 * c + x1 * s
        return o

    def no_gain_norm(x, g, eps):
        return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)

    for name, fn in (("rope", wrong_rope), ("rms_norm", no_gain_norm)):
        with monkeypatch.context() as m:
            m.setattr(odec, name, fn)
            bad = dec.full(toks).logits
        assert np.max(np.abs(bad - ref)) > 1e-3, name


@pytest.mark.parametrize("which", ["gqa", "mha"])
def test_hidden_state_matches_library_final_normed_state(models, which, monkeypatch):
    """The hidden state the linear reward reads is the final-normed one: it
    matches the library model's last (normed) hidden state; a planted
    mistake that skips the final norm (the pre-norm residual stream) fails."""
    from hf_ref import hf_hidden
    shape, w, dec, hf = models[which]
    toks = _prompt(15, shape.vocab)
    ref = hf_hidden(hf, toks)
    ours = dec.full(toks).hidden
    assert np.max(np.abs(ours - ref)) < 2e-5 * max(1.0, np.max(np.abs(ref)))
    calls = {"n": 0}
    real = odec.rms_norm

    def skip_final(x, g, eps):
        calls["n"] += 1
        return x if calls["n"] == 2 * shape.n_layers + 1 else real(x, g, eps)

    monkeypatch.setattr(odec, "rms_norm", skip_final)
    bad = dec.full(toks).hidden
    assert np.max(np.abs(bad - ref)) > 1e-2


def test_linear_reward_reads_the_last_fed_row(models):
    """The linear reward of beam i is w . h, h the final-normed state of the
    last fed row (i, d-1), i.e. after pfx + c_i + x_{i,1..d-1}: checked by a
    full forward of the library model; the previous row fails."""
    from hf_ref import hf_hidden
    draft, target, st = _state(models, n=8)
    hf_t = models["mha"][3]
    k, d = 3, 4
    w = np.random.default_rng(4).standard_normal(models["mha"][0].d_model)
    r = oracle.step(draft, target, st, k, d, 1.0, "linear", w=w)
    for i in range(k):
        seq = list(st.tokens) + [int(r.heads[i])] + [int(t) for t in r.roll.x[i, :d - 1]]
        hs = hf_hidden(hf_t, seq)
        # the library's float32 rotary angles bound each state entry's error
        # to ~2e-5 (see the decoder pin); a wrong row is off by O(1)
        tol = 2e-5 * float(np.sum(np.abs(w))) * max(1.0, float(np.max(np.abs(hs[-1]))))
        assert abs(r.reward[i] - float(hs[-1] @ w)) < tol
        assert abs(float(hs[-2] @ w) - r.reward[i]) > 100 * tol


def test_top2_margin_against_sorting_by_hand():
    """The near-tie gate: the largest value minus the largest of the rest
    (one copy of the maximum removed), so exact ties give 0."""
    rng = np.random.default_rng(8)
    for _ in range(200):
        V = int(rng.integers(2, 40))
        z = rng.normal(0.0, 1.0, V)
        if rng.random() < 0.3:
            z[rng.integers(0, V)] = z.max()            # planted tie
        rest = [float(v) for v in z]
        top = max(rest)
        rest.remove(top)
        assert oracle.top2_margin(z) == top - max(rest)
    assert oracle.top2_margin([1.0, 3.0, 3.0]) == 0.0


def test_soft_accept_margins_closed_form():
    """Distance of u from min(1, p/q), element by element with scalar
    math; zero exactly at the bound."""
    rng = np.random.default_rng(9)
    lt, ld = rng.uniform(-8.0, 0.0, 50), rng.uniform(-8.0, 0.0, 50)
    u = rng.random(50)
    got = oracle.soft_accept_margins(lt, ld, u)
    for j in range(50):
        bound = min(1.0, math.exp(lt[j] - ld[j]))
        assert abs(got[j] - abs(u[j] - bound)) < 1e-15
    assert oracle.soft_accept_margins([-1.0], [-0.5], [math.exp(-0.5)])[0] < 1e-15
    assert oracle.soft_accept_margins([0.0], [-2.0], [1.0])[0] == 0.0


def test_residual_interval_is_the_cumulative_sum():
    """Token t's interval of v is [sum_{s<t} w_s, sum_{s<=t} w_s] / Z for w =
    max(0, p - q), summed here with scalar math; the intervals tile [0, 1),
    and a draw at an interval's midpoint returns its token."""
    rng = np.random.default_rng(10)
    for _ in range(20):
        V = int(rng.integers(3, 30))
        zp, zq = rng.normal(0, 2, V), rng.normal(0, 2, V)
        ep = [math.exp(v - max(zp)) for v in zp]
        eq = [math.exp(v - max(zq)) for v in zq]
        p = [e / math.fsum(ep) for e in ep]
        q = [e / math.fsum(eq) for e in eq]
        w = [max(0.0, a - b) for a, b in zip(p, q)]
        Z = math.fsum(w)
        prev_hi = 0.0
        for t in range(V):
            lo, hi, Zo = oracle.residual_interval(zp, zq, t)
            assert abs(Zo - Z) < 1e-12
            assert abs(lo - math.fsum(w[:t]) / Z) < 1e-12 and abs(hi - math.fsum(w[:t + 1]) / Z) < 1e-12
            assert abs(lo - prev_hi) < 1e-12
            prev_hi = hi
            if w[t] > 0:
                assert oracle.residual_sample(zp, zq, (lo + hi) / 2)[0] == t
        assert abs(prev_hi - 1.0) < 1e-12
    assert oracle.residual_interval([1.0, 2.0], [1.0, 2.0], 1) == (0.0, 0.0, 0.0)


# ---------------------------------------------------------------------------
# caching and verification invariants
# ---------------------------------------------------------------------------
def test_incremental_equals_full_recompute(models):
    shape, w, dec, _ = models["gqa"]
    toks = _prompt(17, shape.vocab)
    full = dec.full(toks).logits
    cache = dec.empty_cache()
    rows = []
    for t in toks:
        out, cache = dec.extend(cache, [t])
        rows.append(out.logits[0])
    assert np.max(np.abs(np.stack(rows) - full)) < 1e-10


def _state(models, which_d="gqa", which_t="mha", n=9):
    sd, wd, dd, _ = models[which_d]
    st_, wt, dt, _ = models[which_t]
    return dd, dt, oracle.prefill(dd, dt, _prompt(n, sd.vocab, seed=11))


def test_tree_verify_equals_per_beam_and_full(models):
    draft, target, st = _state(models)
    k, d = 3, 4
    heads = oracle.topk_ids(st.s_logits, k)
    x = oracle.rollout(draft, st, heads, d).x
    lt, ht = oracle.verify_rows_tree(target, st, heads, x)
    lb, hb = oracle.verify_rows_per_beam(target, st, heads, x)
    assert np.max(np.abs(lt - lb)) < 1e-10 and np.max(np.abs(ht - hb)) < 1e-10
    for i in range(k):
        seq = st.tokens + [int(heads[i])] + [int(t) for t in x[i, :d - 1]]
        full = target.full(seq).logits[-d:]
        assert np.max(np.abs(full - lt[i])) < 1e-10


def test_shared_prefix_equals_duplicated_prefix(models):
    """Rollout of every beam from one shared prefix cache equals rollouts
    from independent full recomputes (no state leaks between beams)."""
    draft, target, st = _state(models)
    heads = oracle.topk_ids(st.s_logits, 4)
    ro = oracle.rollout(draft, st, heads, 3)
    for i, c in enumerate(heads):
        seq = list(st.tokens) + [int(c)]
        for j in range(3):
            z = draft.full(seq).logits[-1]
            assert ro.x[i, j] == int(np.argmax(z))
            seq.append(int(ro.x[i, j]))


def test_rollout_is_argmax_of_library_forward(models):
    from hf_ref import hf_logits
    sd, wd, dd, hf_d = models["gqa"]
    _, _, dt, _ = models["mha"]
    st = oracle.prefill(dd, dt, _prompt(8, sd.vocab, seed=5))
    heads = oracle.topk_ids(st.s_logits, 3)
    ro = oracle.rollout(dd, st, heads, 4)
    for i, c in enumerate(heads):
        seq = list(st.tokens) + [int(c)]
        for j in range(4):
            assert ro.x[i, j] == int(np.argmax(hf_logits(hf_d, seq)[-1]))
            seq.append(int(ro.x[i, j]))


# ---------------------------------------------------------------------------
# special cases of the whole step
# ---------------------------------------------------------------------------
def test_k1_reduces_to_greedy_decoding_of_target(models):
    """With one beam the emitted tokens are exactly the target's greedy
    continuation (greedy speculative decoding is lossless), for any draft."""
    from hf_ref import hf_greedy
    draft, target, st0 = _state(models, n=7)
    hf_t = models["mha"][3]
    st = st0
    out = []
    for _ in range(5):
        r = oracle.step(draft, target, st, 1, 3, 1.0, "keyword_count", kws=[1, 2, 3])
        out += r.emitted
        st = r.state
    assert out == hf_greedy(hf_t, st0.tokens, len(out))


def test_draft_equal_to_target_accepts_every_token(models):
    _, _, dt, _ = models["mha"]
    st = oracle.prefill(dt, dt, _prompt(6, 64, seed=2))
    k, d = 3, 4
    r = oracle.step(dt, dt, st, k, d, 1.0, "keyword_count", kws=[5, 6, 7])
    assert list(r.ver.n) == [d] * k
    for i in range(k):
        for j in range(d):
            z = r.ver.logits[i, j]
            assert abs(r.ver.logprobs[i, j] - oracle.log_softmax(z).max()) < 1e-12
    # n = d: all d+1 tokens are emitted and the next head distribution is the
    # target's distribution after x_d
    assert len(r.emitted) == d + 1
    full = dt.full(r.state.tokens).logits[-1]
    assert np.max(np.abs(r.state.s - oracle.log_softmax(full))) < 1e-10


TINY = ci.ModelShape(1, 16, 2, 1, 32, 16)


def test_select_matches_brute_force_enumeration():
    """k = V: every possible head is a beam.  Enumerate all heads, roll out
    and score by full recompute, and check the step's choice."""
    wt = _weights(TINY, 1, seed=21)
    wd = _weights(TINY, 0, seed=22)
    T, Dm = odec.Decoder(TINY, wt), odec.Decoder(TINY, wd)
    V = TINY.vocab
    prompt = [3, 9, 1, 14]
    st = oracle.prefill(Dm, T, prompt)
    kws = [2, 5, 11]
    for d in (1, 2, 3):
        for alpha in (0.0, 0.7, math.inf):
            r = oracle.step(Dm, T, st, V, d, alpha, "keyword_count", kws=kws)
            best, best_val, rows = None, -math.inf, []
            s0 = oracle.log_softmax(T.full(prompt).logits[-1])
            for c in range(V):
                seq = prompt + [c]
                for _ in range(d):
                    seq.append(int(np.argmax(Dm.full(seq).logits[-1])))
                ls = oracle.log_softmax(T.full(seq[:-1]).logits[-d:])
                x = seq[len(prompt) + 1:]
                score = s0[c] + sum(ls[j, x[j]] for j in range(d))
                rew = oracle.keyword_hits([c] + x, kws)
                val = rew if math.isinf(alpha) else score + alpha * rew
                rows.append((c, val))
            ordered = sorted(rows, key=lambda cv: (-cv[1], [h for h in r.heads].index(cv[0])))
            assert int(r.heads[r.beam]) == ordered[0][0]
            assert abs(r.combined[r.beam] - ordered[0][1]) < 1e-9


def test_alpha_infinity_is_the_lookahead_heuristic_rule():
    """alpha = inf keeps the first beam with the strictly largest reward."""
    scores = np.array([-1.0, -9.0, -2.0, -0.5])
    reward = np.array([0.25, 0.75, 0.75, 0.5])
    best, best_r = None, -math.inf
    for i, r in enumerate(reward):   # the CDLH update, written out
        if r > best_r:
            best, best_r = i, r
    assert oracle.select_beam(scores, reward, math.inf) == best == 1
    assert oracle.select_beam(scores, reward, 0.0) == 3


# ---------------------------------------------------------------------------
# reward, rows, rejection
# ---------------------------------------------------------------------------
def test_reward_worked_example_from_the_paper():
    g = json.load(open(os.path.join(GOLDEN, "reward_worked_example.json")))
    concepts = list(range(100, 100 + g["concepts"]))
    window = [7, concepts[0], 8, concepts[3], concepts[3], 9]
    assert oracle.keyword_hits(window, concepts) == g["covered"]
    assert abs(oracle.keyword_coverage(window, concepts) - g["reward"]) < 1e-15


def test_log_softmax_and_topk_rows():
    rng = np.random.default_rng(0)
    z = rng.standard_normal(50) * 3
    ls = oracle.log_softmax(z)
    assert abs(np.sum(np.exp(ls)) - 1.0) < 1e-13
    assert np.allclose(ls - ls[0], z - z[0], atol=1e-12)
    # forced ties: equal values resolve to the lower id
    z = np.array([1.0, 3.0, 2.0, 3.0, 2.0, -1.0, 3.0])
    assert list(oracle.topk_ids(z, 5)) == [1, 3, 6, 2, 4]
    assert oracle.argmax_lowest(z) == 1
    brute = sorted(range(len(z)), key=lambda i: (-z[i], i))
    assert list(oracle.topk_ids(z, 7)) == brute


def test_hard_rejection_counts_leading_matches():
    assert oracle.leading_matches([1, 2, 3], [1, 2, 3]) == 3
    assert oracle.leading_matches([1, 2, 3], [1, 5, 3]) == 1
    assert oracle.leading_matches([4, 2, 3], [1, 2, 3]) == 0


# ---------------------------------------------------------------------------
# resume and batch independence
# ---------------------------------------------------------------------------
def test_resume_by_reprefill_equals_uninterrupted_run(models):
    draft, target, st = _state(models, n=6)
    a = st
    for _ in range(4):
        a = oracle.step(draft, target, a, 3, 2, 1.0, "keyword_count", kws=[1, 2]).state
    b = oracle.prefill(draft, target, a.tokens)
    b.n_prompt = st.n_prompt
    for _ in range(3):
        a = oracle.step(draft, target, a, 3, 2, 1.0, "keyword_count", kws=[1, 2]).state
        b = oracle.step(draft, target, b, 3, 2, 1.0, "keyword_count", kws=[1, 2]).state
    assert a.tokens == b.tokens


def test_inputs_do_not_depend_on_batch_size():
    a = ci.prompts(0, 5, 9, 1000)
    b = ci.prompts(0, 2, 9, 1000, first=3)
    assert np.array_equal(a[3:], b)
    ka = ci.keywords(0, 4, 3, 1000)
    assert all(len(set(r)) == 3 for r in ka)
    assert np.array_equal(ka[2:], ci.keywords(0, 2, 3, 1000, first=2))


# ---------------------------------------------------------------------------
# the baselines (CDLH, CDLH-appx.) and the Alg. 1 controller
# ---------------------------------------------------------------------------
def _hf_greedy_tail(hf, seq, d):
    """d greedy tokens after seq by full recomputation (independent path)."""
    return [int(t) for t in _hf_greedy(hf, seq, d)]


def _hf_greedy(hf, seq, n):
    from hf_ref import hf_greedy
    return hf_greedy(hf, seq, n)


def _brute_cdlh(hf_roller, hf_target, tokens, n_prompt, k, d, kws, kind):
    """The appendix algorithm written out with full forwards: candidates =
    top-k of the target (value desc, id asc), each extended by d greedy
    tokens of the roller, scored by the concept count over generated +
    candidate + lookahead; first best wins."""
    from hf_ref import hf_logits
    z = hf_logits(hf_target, tokens)[-1]
    order = sorted(range(len(z)), key=lambda v: (-z[v], v))[:k]
    scores = []
    for c in order:
        look = _hf_greedy_tail(hf_roller, list(tokens) + [c], d)
        window = list(tokens[n_prompt:]) + [c] + look
        hits = len(set(window) & set(kws))
        scores.append(hits / len(set(kws)) if kind == "keyword_coverage" else float(hits))
    best = max(range(k), key=lambda i: (scores[i], -i))
    return order, scores, best


@pytest.mark.parametrize("roller_is_target", [False, True])
def test_lookahead_heuristic_k1_is_greedy_decoding(models, roller_is_target):
    """One candidate: CDLH and CDLH-appx. emit the target's greedy tokens."""
    draft, target, st0 = _state(models, n=6)
    hf_t = models["mha"][3]
    st, out = st0, []
    for _ in range(4):
        hs = oracle.cdlh_step(roller_is_target, draft, target, st, 1, 3, "keyword_count", [1, 2, 3])
        out.append(hs.token)
        st = hs.state
    assert out == _hf_greedy(hf_t, st0.tokens, 4)


@pytest.mark.parametrize("roller_is_target", [False, True])
def test_lookahead_heuristic_choice_matches_full_recompute(models, roller_is_target):
    draft, target, st = _state(models, n=8)
    hf_d, hf_t = models["gqa"][3], models["mha"][3]
    k, d = 4, 3
    # concepts taken from the third candidate's own lookahead, so that the
    # rewards differ and the choice is not the first candidate by default
    from hf_ref import hf_logits
    z = hf_logits(hf_t, st.tokens)[-1]
    c3 = sorted(range(len(z)), key=lambda v: (-z[v], v))[2]
    roller = hf_t if roller_is_target else hf_d
    kws = _hf_greedy_tail(roller, list(st.tokens) + [c3], d)[:2] + [63]
    for kind in ("keyword_count", "keyword_coverage"):
        hs = oracle.cdlh_step(roller_is_target, draft, target, st, k, d, kind, kws)
        order, scores, best = _brute_cdlh(roller, hf_t, st.tokens, st.n_prompt, k, d, kws, kind)
        assert list(hs.heads) == order
        assert np.allclose(hs.reward, scores)
        assert hs.pick == best and hs.token == order[best]
        # the emitted token extends the prefix and the next distribution is
        # the target's after it
        full = target.full(hs.state.tokens).logits[-1]
        assert hs.state.tokens == list(st.tokens) + [order[best]]
        assert np.max(np.abs(hs.state.s - oracle.log_softmax(full))) < 1e-10


def _hf_alg1_draft_verify(hf_d, hf_t, tokens, d):
    """Alg. 1's drafting loop and hard rejection by full recomputation: d
    greedy draft tokens after the prefix, then the leading matches with the
    target's argmax after pfx + x_1..x_{j-1}."""
    from hf_ref import hf_logits
    x = _hf_greedy_tail(hf_d, tokens, d)
    zt = hf_logits(hf_t, list(tokens) + x[:-1])[len(tokens) - 1:]
    n = 0
    for j in range(d):
        if int(np.argmax(zt[j])) != x[j]:
            break
        n += 1
    return x, n, zt


def _near_draft(models, scale=0.03, seed=5):
    """A draft that mostly agrees with the "mha" target: its weights plus
    3% noise, so that 0 < n < d occurs."""
    shape, w, _, _ = models["mha"]
    rng = np.random.default_rng(seed)
    nw = {k: (v + scale * np.std(v) * rng.standard_normal(v.shape) if isinstance(v, np.ndarray) and v.ndim == 2 else v)
          for k, v in w.items() if k != "layers"}
    nw["layers"] = [{k: (v + scale * np.std(v) * rng.standard_normal(v.shape) if v.ndim == 2 else v)
                     for k, v in lw.items()} for lw in w["layers"]]
    return odec.Decoder(shape, nw)


@pytest.mark.parametrize("which,a_t,b", [("random", 2.0, 1), ("random", 1e-9, 1), ("same", 1e-9, 0),
                                         ("near", 1e-9, 1), ("near", 2.0, 1)])
def test_controller_greedy_settings_reproduce_greedy_decoding(models, which, a_t, b):
    """r_t = -inf makes every reward check pass.  Then S1 emits the accepted
    tokens, which are the target's greedy tokens, and S2/S3's Step-1 (b = 1)
    emits the target's greedy token after them (a_t = 2 forces S2/S3 every
    time).  With draft = target every token is accepted (n = d, S1).  Either
    way Alg. 1 is greedy decoding of the target."""
    _, _, dt, hf_t = models["mha"]
    draft = {"random": models["gqa"][2], "same": dt, "near": None}[which] or _near_draft(models)
    st0 = oracle.prefill(draft, dt, _prompt(7, 64, seed=11))
    st, out, seen = st0, [], set()
    for _ in range(5):
        cs = oracle.controller_step(draft, dt, st, 3, 3, a_t, -math.inf, b, "keyword_count", [4, 5])
        seen.add((cs.state, cs.n))
        out += cs.emitted
        st = cs.after
    assert out == _hf_greedy(hf_t, st0.tokens, len(out))
    if which == "same":
        assert seen == {("S1", 3)}
    if a_t > 1:
        assert {s for s, _ in seen} == {"S2/S3"}


def test_controller_without_acceptance_emits_exactly_one_token(models):
    """n = 0 with a_t = 0.3: a = 0 < a_t, so S2/S3, and the iteration emits
    one token: Step-1's X_1 if its lookahead reaches r_t, else Step-2's."""
    draft, target, st = _state(models, n=9)
    hit = 0
    for b in (0, 1):
        for r_t in (0.0, 1.0, math.inf):
            cur = st
            for _ in range(3):
                cs = oracle.controller_step(draft, target, cur, 3, 4, 0.3, r_t, b, "keyword_count", [7, 11, 40])
                if cs.n == 0:
                    hit += 1
                    assert cs.state == "S2/S3" and len(cs.emitted) == 1
                    assert (cs.extra is None) == (b == 1 and cs.step1[0].reward >= r_t)
                cur = cs.after
    assert hit >= 6


def test_controller_after_partial_s1_accepts_nothing(models):
    """A property of the printed algorithm with greedy drafts and hard
    rejection: after an S1 that accepted n < d tokens the next draft starts
    with x_{n+1} again, which the target rejected, so that iteration has
    n = 0."""
    _, _, dt, _ = models["mha"]
    draft = _near_draft(models)
    seen = 0
    for seed in (11, 12, 13):
        st = oracle.prefill(draft, dt, _prompt(7, 64, seed=seed))
        prev = None
        for _ in range(8):
            cs = oracle.controller_step(draft, dt, st, 3, 4, 1e-9, -math.inf, 1, "keyword_count", [4])
            if prev is not None and prev.state == "S1" and prev.n < 4:
                assert cs.n == 0 and int(cs.x[0]) == int(prev.x[prev.n])
                seen += 1
            prev, st = cs, cs.after
    assert seen >= 2


@pytest.mark.parametrize("a_t,r_t,b,state", [(1e-9, -math.inf, 0, "S1"), (2.0, -math.inf, 0, "S2/S3"),
                                             (2.0, math.inf, 1, "S2/S3"), (2.0, 0.0, 1, "S2/S3"),
                                             (1e-9, math.inf, 1, "S4")])
def test_controller_matches_full_recompute(models, a_t, r_t, b, state):
    """Every quantity of one Alg. 1 iteration by full recomputation with the
    library models: x drafted from the prefix, n, a, r, the state, Step-1's
    X_1 and its lookahead reward, and the Step-2 / S4 token (the appendix
    algorithm after x_1..x_n).  The near draft makes n > 0 for S1 and S4."""
    from hf_ref import hf_logits
    _, _, dt, hf_t = models["mha"]
    draft = _near_draft(models)
    from hf_ref import hf_llama
    hf_d = hf_llama(models["mha"][0], draft.w)
    st = oracle.prefill(draft, dt, _prompt(9, 64, seed=12))
    k, d, kws = 3, 4, [7, 11, 13, 40]
    cs = oracle.controller_step(draft, dt, st, k, d, a_t, r_t, b, "keyword_count", kws)
    assert cs.state == state
    x, n, _ = _hf_alg1_draft_verify(hf_d, hf_t, st.tokens, d)
    assert list(cs.x) == x and cs.n == n and cs.a == n / d
    if state != "S2/S3":
        assert n > 0
    acc = x[:n]
    assert cs.r == float(len(set(acc) & set(kws)))
    base = list(st.tokens) + acc
    if state == "S1":
        assert cs.emitted == acc and cs.extra is None
        return
    tail = None
    if state == "S2/S3" and b == 1:
        X1 = int(np.argmax(hf_logits(hf_t, base)[-1]))
        lh = _hf_greedy_tail(hf_d, base + [X1], d)
        rr = float(len(set(acc + [X1] + lh) & set(kws)))
        assert cs.step1[0].X == [X1] and list(cs.step1[0].lh) == lh and cs.step1[0].reward == rr
        if rr >= r_t:
            tail = [X1]
    if tail is None:
        order, scores, best = _brute_cdlh(hf_d, hf_t, base, st.n_prompt, k, d, kws, "keyword_count")
        tail = [order[best]]
        assert cs.extra is not None and list(cs.extra.heads) == order
    assert cs.emitted == acc + tail


def test_step1_with_two_rounds(models):
    """b = 2: when the first M_p token's lookahead misses r_t, Step-1 takes
    M_p's greedy token after it and tries again; O = x_1..x_n + X_1 + X_2 if
    that window reaches r_t.  If neither does, both are dropped and Step-2
    adds the appendix algorithm's token after x_1..x_n."""
    from hf_ref import hf_logits
    draft, target, st = _state(models, n=9)
    hf_d, hf_t = models["gqa"][3], models["mha"][3]
    d, k = 3, 3
    x, n, _ = _hf_alg1_draft_verify(hf_d, hf_t, st.tokens, d)
    acc = x[:n]
    base = list(st.tokens) + acc
    X1 = int(np.argmax(hf_logits(hf_t, base)[-1]))
    lh1 = _hf_greedy_tail(hf_d, base + [X1], d)
    X2 = int(np.argmax(hf_logits(hf_t, base + [X1])[-1]))
    lh2 = _hf_greedy_tail(hf_d, base + [X1, X2], d)
    before = set(st.tokens[st.n_prompt:]) | set(acc) | {X1} | set(lh1)
    fresh = [t for t in [X2] + lh2 if t not in before]
    assert fresh, "the seeded prompt has no token that only the second round reaches"
    cs = oracle.controller_step(draft, target, st, k, d, 2.0, 1.0, 2, "keyword_count", [fresh[0]])
    assert [t.X for t in cs.step1] == [[X1], [X1, X2]] and list(cs.step1[1].lh) == lh2
    assert cs.extra is None and cs.emitted == acc + [X1, X2]
    assert cs.after.tokens == base + [X1, X2]
    # no round reaches r_t: the X are dropped, Step-2 after x_1..x_n
    absent = [t for t in range(64) if t not in set(st.tokens) | set(acc) | {X1, X2} | set(lh1) | set(lh2)]
    cs = oracle.controller_step(draft, target, st, k, d, 2.0, 1.0, 2, "keyword_count", [absent[0]])
    order, scores, best = _brute_cdlh(hf_d, hf_t, base, st.n_prompt, k, d, [absent[0]], "keyword_count")
    assert len(cs.step1) == 2 and cs.emitted == acc + [order[best]]


@pytest.mark.parametrize("r_t", [0.0, 1.0, 2.0])
def test_step1_b1_equals_the_first_candidate_rule(models, r_t):
    """With b = 1, Step-1's token and lookahead are the appendix algorithm's
    first candidate and its lookahead, so Step-1 then Step-2 equals one
    candidate table in which candidate 0 wins once it reaches r_t (the form
    the GPU path computes)."""
    draft, target, st = _state(models, n=10)
    kws = [3, 9, 17, 30, 41]
    cur = st
    for _ in range(3):
        cs = oracle.controller_step(draft, target, cur, 4, 3, 2.0, r_t, 1, "keyword_count", kws)
        acc = [int(t) for t in cs.x[:cs.n]]
        st1 = oracle.commit(draft, target, cur, acc)
        hs = oracle.cdlh_step(False, draft, target, st1, 4, 3, "keyword_count", kws, prefer_first_at=r_t)
        assert cs.emitted == acc + [hs.token]
        cur = cs.after


def test_controller_visits_every_state_on_the_tiny_workload():
    """On the seeded `tiny` workload the controller settings of the GPU
    parity tests reach S1, S2/S3 and S4 (S1 and S4 with the target as its
    own draft, where every lookahead is accepted), so every branch is
    compared."""
    wl = ci.workload("tiny")
    tw = ci.model_weights(wl.target, wl.seed, 1, wl.dtype)
    dw = ci.model_weights(wl.draft, wl.seed, 0, wl.dtype)
    od, ot = oracle.Decoder(wl.draft, dw), oracle.Decoder(wl.target, tw)
    kws = ci.keywords(wl.seed, 64, wl.n_keywords, wl.target.vocab)
    prompts = ci.prompts(wl.seed, 3, wl.prompt_len, wl.target.vocab)
    seen = {}
    for dm, a_t, r_t, bb in [(od, 0.5, 1.0, 1), (od, 0.5, 1.0, 0), (ot, 0.5, 0.0, 0), (ot, 0.5, 1.0, 1)]:
        for b in range(3):
            st = oracle.prefill(dm, ot, prompts[b])
            for _ in range(3):
                cs = oracle.controller_step(dm, ot, st, wl.k, wl.d, a_t, r_t, bb, wl.reward, kws[b])
                seen[cs.state] = seen.get(cs.state, 0) + 1
                st = cs.after
    assert set(seen) == {"S1", "S2/S3", "S4"}, seen


def test_controller_rejects_non_positive_acceptance_threshold(models):
    draft, target, st = _state(models, n=6)
    with pytest.raises(ValueError):
        oracle.controller_step(draft, target, st, 3, 3, 0.0, 0.0, 1, "keyword_count", [1])


# ---------------------------------------------------------------------------
# speculative sampling (soft rejection)
# ---------------------------------------------------------------------------
def _grid(N):
    """Stratified points of U[0, 1): every cell of width 1/N once."""
    return (np.arange(N) + 0.5) / N


def _softmax(z):
    e = np.exp(np.asarray(z, np.float64) - np.max(z))
    return e / e.sum()


def test_soft_acceptance_rate_is_min_one_ratio():
    """Over a stratified grid of u the accepted fraction equals min(1, p/q)
    (to the grid's 1/N), and a run ends at its first rejection."""
    N = 2000
    rng = np.random.default_rng(5)
    for _ in range(12):
        lt, ld = rng.uniform(-6.0, 0.0, 2)
        acc = sum(oracle.soft_accept_count([lt], [ld], [u]) for u in _grid(N)) / N
        assert abs(acc - min(1.0, math.exp(lt - ld))) <= 1.0 / N
    assert oracle.soft_accept_count([0.0, -9.0, 0.0], [0.0, 0.0, 0.0], [0.5, 0.5, 0.0]) == 1
    assert oracle.soft_accept_count([-1.0, -1.0], [-2.0, -2.0], [0.999, 0.999]) == 2   # p > q: always kept
    assert oracle.soft_accept_count([-1.0], [-1.0], [0.0]) == 1


def test_residual_draw_is_the_inverse_cdf_of_the_positive_part():
    """Each draw equals a library inverse-CDF lookup on the normalised
    max(0, p - q); over a stratified grid of v the frequencies match it and
    tokens with p <= q are never drawn.  Equal logits fall back to argmax p."""
    rng = np.random.default_rng(6)
    V = 9
    zp, zq = rng.normal(0.0, 2.0, V), rng.normal(0.0, 2.0, V)
    p, q = _softmax(zp), _softmax(zq)
    w = np.maximum(0.0, p - q)
    w /= w.sum()
    cdf = np.cumsum(w)
    N = 5000
    counts = np.zeros(V)
    for v in _grid(N):
        t, lp, mg = oracle.residual_sample(zp, zq, v)
        counts[t] += 1
        assert t == int(np.searchsorted(cdf, v, side="right"))
        assert abs(lp - math.log(p[t])) < 1e-12
        assert 0.0 <= mg <= w[t] / 2 + 1e-12
    assert np.max(np.abs(counts / N - w)) <= 1.0 / N + 1e-12
    assert np.all(counts[w == 0.0] == 0)
    t, _, _ = oracle.residual_sample(zp, zp, 0.3)
    assert t == int(np.argmax(zp))


def _output_distribution(zp, zq, residual=None):
    """Distribution of speculative sampling's output token when the draft
    token x is drawn from q: accepted with the oracle's test, else replaced
    by the oracle's residual draw; enumerated over x and stratified u, v."""
    residual = residual or oracle.residual_sample
    lp, lq = oracle.log_softmax(zp), oracle.log_softmax(zq)
    V = len(zp)
    Nu = Nv = 1000
    R = np.zeros(V)
    for v in _grid(Nv):
        R[residual(zp, zq, v)[0]] += 1.0 / Nv
    out = np.zeros(V)
    for x in range(V):
        acc = sum(oracle.soft_accept_count([lp[x]], [lq[x]], [u]) for u in _grid(Nu)) / Nu
        out[x] += math.exp(lq[x]) * acc
        out += math.exp(lq[x]) * (1.0 - acc) * R
    return out


def test_speculative_sampling_reproduces_the_target_distribution():
    """The theorem speculative sampling rests on (Leviathan et al., 2023):
    with x ~ q, accept-or-resample outputs tokens distributed exactly as p."""
    rng = np.random.default_rng(7)
    for V in (2, 6):
        zp, zq = rng.normal(0.0, 1.5, V), rng.normal(0.0, 1.5, V)
        out = _output_distribution(zp, zq)
        assert np.max(np.abs(out - _softmax(zp))) < 3e-3


def test_swapped_residual_fails_the_distribution_pin():
    """A planted mistake in the oracle (drawing from max(0, q - p)) breaks
    the theorem check above."""
    rng = np.random.default_rng(7)
    zp, zq = rng.normal(0.0, 1.5, 6), rng.normal(0.0, 1.5, 6)
    swapped = lambda a, b, v: oracle.residual_sample(b, a, v)
    out = _output_distribution(zp, zq, swapped)
    assert np.max(np.abs(out - _softmax(zp))) > 3e-2


def test_soft_step_with_draft_equal_to_target_accepts_every_token(models):
    _, _, dt, _ = models["mha"]
    st = oracle.prefill(dt, dt, _prompt(6, 64, seed=2))
    k, d = 3, 4
    u = np.full((k, d), np.nextafter(np.float32(1.0), np.float32(0.0)), np.float32)
    r = oracle.step(dt, dt, st, k, d, 1.0, "keyword_count", kws=[5, 6, 7], rejection="soft", u=u, v=u)
    assert list(r.soft.n) == [d] * k
    assert r.soft.lead is None and r.state.lead is None
    assert len(r.emitted) == d + 1


def test_soft_step_matches_full_recompute(models):
    """Every beam's soft count from p and q recomputed by the library models
    on the full sequences; the selected beam's lead token is the residual
    draw from those logits at its rejected position, and it heads the next
    beams, followed by the target's top tokens without it."""
    from hf_ref import hf_logits
    draft, target, st = _state(models, n=8)
    hf_d, hf_t = models["gqa"][3], models["mha"][3]
    k, d = 3, 4
    rng = np.random.default_rng(12)
    seen_lead = 0
    cur = st
    for it in range(4):
        u = rng.random((k, d)).astype(np.float32)
        v = rng.random((k, d)).astype(np.float32)
        r = oracle.step(draft, target, cur, k, d, 1.0, "keyword_count", kws=[1, 2, 3], rejection="soft", u=u, v=v)
        for i in range(k):
            seq = list(cur.tokens) + [int(r.heads[i])] + [int(t) for t in r.roll.x[i]]
            L = len(cur.tokens)
            zt = hf_logits(hf_t, seq[:-1])[L:]          # p_j for x_{i,j}, j = 1..d
            zd = hf_logits(hf_d, seq[:-1])[L:]
            lt = [oracle.log_softmax(zt[j])[r.roll.x[i, j]] for j in range(d)]
            ld = [oracle.log_softmax(zd[j])[r.roll.x[i, j]] for j in range(d)]
            assert oracle.soft_accept_count(lt, ld, u[i]) == r.soft.n[i]
            if i == r.beam and r.soft.n[i] < d:
                n = int(r.soft.n[i])
                t, _, _ = oracle.residual_sample(zt[n], zd[n], v[i, n])
                assert t == r.soft.lead
                seen_lead += 1
        nxt, _, _ = oracle.beam_heads(r.state, k)
        if r.soft.lead is not None:
            zn = hf_logits(hf_t, r.state.tokens)[-1]
            rest = [int(x) for x in sorted(range(len(zn)), key=lambda x: (-zn[x], x)) if x != r.soft.lead][:k - 1]
            assert list(nxt) == [r.soft.lead] + rest
        cur = r.state
    assert seen_lead >= 1


def test_soft_controller_matches_full_recompute(models):
    """Alg. 1 with speculative sampling's test in the rejection loop: x
    drafted greedily from the prefix, n from p_j and q_j recomputed by the
    library models on pfx + x_1..x_{j-1}; the accepted tokens are emitted
    first (a_t = 2 forces S2/S3, Step-1 with r_t = -inf then adds M_p's
    greedy token after them)."""
    from hf_ref import hf_logits
    _, _, dt, hf_t = models["mha"]
    draft = _near_draft(models, scale=0.3)
    from hf_ref import hf_llama
    hf_d = hf_llama(models["mha"][0], draft.w)
    cur = oracle.prefill(draft, dt, _prompt(8, 64, seed=13))
    d = 3
    rng = np.random.default_rng(21)
    ns = []
    for _ in range(5):
        u = rng.random((1, d)).astype(np.float32)
        cs = oracle.controller_step(draft, dt, cur, 3, d, 2.0, -math.inf, 1, "keyword_count", [1, 2, 3],
                                    rejection="soft", u=u)
        assert cs.state == "S2/S3"
        x = _hf_greedy_tail(hf_d, cur.tokens, d)
        assert list(cs.x) == x
        L = len(cur.tokens)
        zt = hf_logits(hf_t, list(cur.tokens) + x[:-1])[L - 1:]
        zd = hf_logits(hf_d, list(cur.tokens) + x[:-1])[L - 1:]
        lt = [oracle.log_softmax(zt[j])[x[j]] for j in range(d)]
        ld = [oracle.log_softmax(zd[j])[x[j]] for j in range(d)]
        n = oracle.soft_accept_count(lt, ld, u[0])
        assert n == cs.n
        ns.append(n)
        X1 = int(np.argmax(hf_logits(hf_t, list(cur.tokens) + x[:n])[-1]))
        assert cs.emitted == x[:n] + [X1]
        cur = cs.after
    assert max(ns) > 0
