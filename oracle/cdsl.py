"""CPU oracle, part 2: one lookahead step of constrained decoding with
speculative lookaheads (CDSL), computed from the definitions in float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/decoder.py``).

One step for one prompt, in the paper's order (Sec. 3.2, Alg. 1; the beam
heads and the reward selection follow CDLH, Alg. 2 and Sec. 2.1):

a1  beam heads: c_1..c_k = top-k of s_t = log_softmax(M_p(pfx)) (Alg. 2,
    the top-k selection; Step-2 of Sec. 3.2.3); head_lp_i = s_t[c_i].
a2  draft rollout: x_{i,j} = argmax q_j, q_j = M_q(pfx + c_i + x_{i,<j}),
    j = 1..d, greedy (Alg. 1, drafting loop; Sec. 3.2.1).
a3  verification: p_j = M_p(pfx + c_i + x_{i,<j}), j = 1..d, all k*d rows
    in one pass (Alg. 1, parallel verification; Sec. 3.2.2).
a4  l_{i,j} = log p_j(x_{i,j}); y_{i,j} = argmax p_j.
a5  hard rejection: n_i = number of leading j with y_{i,j} = x_{i,j}
    (Alg. 1, rejection loop); a_i = n_i / d; score_i = head_lp_i + sum_j l_{i,j}.
    Soft rejection (speculative sampling, Sec. 3.2.2): x_{i,j} is rejected
    when u_{i,j} > min(1, p_j(x_{i,j}) / q_j(x_{i,j})) with u ~ U[0, 1); n_i
    counts the positions before the first rejection.
a6  reward r_i over generated-so-far + c_i + x_{i,1..d} (Sec. 3.2.2,
    validation by R; lexical rewards of Sec. 4.1).
a7  select i* = argmax_i (score_i + alpha * r_i); alpha = inf means the
    reward alone, ties to the lowest index (Alg. 2's strict ">" update).
a8  commit: emit O = [c_i*, x_i*,1..n_i*] (S1 action, no bonus token from
    M_p; Sec. 3.2.3), pfx <- pfx + O, and s_{t+1} = log_softmax(M_p(pfx)).
    With soft rejection and n_i* < d, the token drawn at the rejected
    position from the adjusted distribution (normalised max(0, p - q),
    Sec. 3.2.2) leads the next beam heads, in place of M_p's greedy token.

Readings where the paper is silent or garbled are listed in the design doc and
restated next to the code that takes them.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence

import numpy as np

from .decoder import Decoder, KVCache


# ----------------------------------------------------------------------------
# row operations on one distribution
# ----------------------------------------------------------------------------
def log_softmax(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    return z - (m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True)))


def argmax_lowest(z: np.ndarray) -> int:
    """argmax; equal maxima resolve to the lowest token id."""
    return int(np.argmax(z))


def topk_ids(z: np.ndarray, k: int) -> np.ndarray:
    """The k largest entries: value descending, then token id ascending."""
    z = np.asarray(z)
    order = np.lexsort((np.arange(z.shape[-1]), -z))
    return order[:k].astype(np.int64)


def top2_margin(z: np.ndarray) -> float:
    """Gap between the largest and the second-largest entry."""
    s = np.sort(np.asarray(z, dtype=np.float64))
    return float(s[-1] - s[-2])


def leading_matches(y: Sequence[int], x: Sequence[int]) -> int:
    """Hard rejection: count positions before the first y_j != x_j."""
    n = 0
    for yj, xj in zip(y, x):
        if yj != xj:
            break
        n += 1
    return n


# ----------------------------------------------------------------------------
# rewards (stand-ins; see module docstring of cdsl_inputs)
# ----------------------------------------------------------------------------
def keyword_hits(window: Sequence[int], kws: Sequence[int]) -> int:
    """Number of distinct keywords that occur in ``window``."""
    present = set(int(t) for t in window)
    return sum(1 for kw in set(int(k) for k in kws) if kw in present)


def keyword_coverage(window: Sequence[int], kws: Sequence[int]) -> float:
    """Fraction of the keyword set covered (concept counting, Sec. 4.1)."""
    kws = list(set(int(k) for k in kws))
    return keyword_hits(window, kws) / len(kws)


def select_beam(scores: np.ndarray, reward: np.ndarray, alpha: float) -> int:
    """argmax_i (score_i + alpha r_i), lowest i on ties; alpha = inf: reward only."""
    scores = np.asarray(scores, np.float64)
    reward = np.asarray(reward, np.float64)
    if math.isinf(alpha) and alpha > 0:
        comb = reward
    else:
        comb = scores + alpha * reward
    return int(np.argmax(comb))


# ----------------------------------------------------------------------------
# per-prompt state and the step
# ----------------------------------------------------------------------------
@dataclass
class PromptState:
    tokens: List[int]          # prompt + everything emitted so far
    n_prompt: int
    draft_cache: KVCache
    target_cache: KVCache
    s: np.ndarray              # log_softmax of M_p at the end of the prefix
    s_logits: np.ndarray       # the raw target logits of that row
    lead: Optional[int] = None  # soft rejection's resampled token: the first next head
    q_logits: Optional[np.ndarray] = None   # the raw draft logits at the end of the prefix

    @property
    def generated(self) -> List[int]:
        return self.tokens[self.n_prompt:]

    @property
    def length(self) -> int:
        return len(self.tokens)


def prefill(draft: Decoder, target: Decoder, prompt: Sequence[int]) -> PromptState:
    prompt = [int(t) for t in prompt]
    dout, dc = draft.extend(draft.empty_cache(), prompt)
    out, tc = target.extend(target.empty_cache(), prompt)
    z = out.logits[-1]
    return PromptState(list(prompt), len(prompt), dc, tc, log_softmax(z), z, q_logits=dout.logits[-1])


@dataclass
class Rollout:
    x: np.ndarray              # [k, d] lookahead tokens
    margin: np.ndarray         # [k, d] top-2 margin of the draft logits at each draw
    lq: Optional[np.ndarray] = None      # [k, d] log q_j(x_{i,j}), the draft's own log-prob
    logits: Optional[np.ndarray] = None  # [k, d, V] the draft logits of every draw


def rollout(draft: Decoder, st: PromptState, heads: Sequence[int], d: int) -> Rollout:
    """a2: greedy lookahead of d tokens from each head, one token at a time,
    each beam on its own copy of the prefix cache."""
    k = len(heads)
    x = np.zeros((k, d), np.int64)
    mg = np.zeros((k, d))
    lq = np.zeros((k, d))
    zs = np.zeros((k, d, draft.shape.vocab))
    for i, c in enumerate(heads):
        cache = st.draft_cache
        fed = int(c)
        for j in range(d):
            out, cache = draft.extend(cache, [fed])
            z = out.logits[0]
            x[i, j] = argmax_lowest(z)
            mg[i, j] = top2_margin(z)
            lq[i, j] = log_softmax(z)[x[i, j]]
            zs[i, j] = z
            fed = int(x[i, j])
    return Rollout(x, mg, lq, zs)


@dataclass
class Verify:
    logits: np.ndarray         # [k, d, V] target logits of the fed rows
    hidden: np.ndarray         # [k, d, D] final-normed hidden states
    logprobs: np.ndarray       # [k, d]  l_{i,j} = log p_j(x_{i,j})
    y: np.ndarray              # [k, d]  argmax p_j
    margin: np.ndarray         # [k, d]  top-2 margin of p_j logits
    n: np.ndarray              # [k]     leading matches
    scores: np.ndarray         # [k]     head_lp + sum_j l
    row_topk: np.ndarray       # [k, d, k] top-k ids of every fed row
    row_topk_lp: np.ndarray    # [k, d, k]


def verify_rows_tree(target: Decoder, st: PromptState, heads, x) -> tuple:
    """a3 as one pass: rows (i, j) feed [c_i, x_{i,1..d-1}] at positions
    L + j; row (i, j) sees the whole prefix and rows (i, 0..j) of its beam."""
    k, d = x.shape
    L = st.length
    fed = np.concatenate([np.asarray(heads, np.int64)[:, None], x[:, :d - 1]], 1)  # [k, d]
    toks = fed.reshape(-1)
    pos = np.tile(L + np.arange(d), k)
    beam_of = np.repeat(np.arange(k), d)
    j_of = np.tile(np.arange(d), k)
    tree = (beam_of[:, None] == beam_of[None, :]) & (j_of[None, :] <= j_of[:, None])
    allowed = np.concatenate([np.ones((k * d, L), bool), tree], 1)
    out = target.forward(toks, pos, st.target_cache, allowed)
    return out.logits.reshape(k, d, -1), out.hidden.reshape(k, d, -1)


def verify_rows_per_beam(target: Decoder, st: PromptState, heads, x) -> tuple:
    """a3 with one causal pass per beam on a duplicated prefix cache."""
    k, d = x.shape
    lg, hd = [], []
    for i in range(k):
        fed = [int(heads[i])] + [int(t) for t in x[i, :d - 1]]
        out, _ = target.extend(st.target_cache.copy(), fed)
        lg.append(out.logits)
        hd.append(out.hidden)
    return np.stack(lg), np.stack(hd)


def verify(target: Decoder, st: PromptState, heads, head_lp, x, tree: bool = True) -> Verify:
    x = np.asarray(x, np.int64)
    k, d = x.shape
    logits, hidden = (verify_rows_tree if tree else verify_rows_per_beam)(target, st, heads, x)
    lp = np.zeros((k, d))
    y = np.zeros((k, d), np.int64)
    mg = np.zeros((k, d))
    rtk = np.zeros((k, d, k), np.int64)
    rtl = np.zeros((k, d, k))
    for i in range(k):
        for j in range(d):
            z = logits[i, j]
            ls = log_softmax(z)
            lp[i, j] = ls[x[i, j]]
            y[i, j] = argmax_lowest(z)
            mg[i, j] = top2_margin(z)
            ids = topk_ids(z, k)
            rtk[i, j] = ids
            rtl[i, j] = ls[ids]
    n = np.array([leading_matches(y[i], x[i]) for i in range(k)], np.int64)
    scores = np.asarray(head_lp, np.float64) + lp.sum(1)
    return Verify(logits, hidden, lp, y, mg, n, scores, rtk, rtl)


def reward_for(kind: str, generated: Sequence[int], heads, x, hidden, kws=None, w=None) -> np.ndarray:
    """a6: one reward per beam.  Keyword rewards look at generated-so-far
    + c_i + x_{i,1..d} (the prompt is excluded: prompts carry the concepts);
    the linear reward reads the final-normed hidden state of row (i, d-1)."""
    k, d = np.asarray(x).shape
    r = np.zeros(k)
    for i in range(k):
        window = list(generated) + [int(heads[i])] + [int(t) for t in x[i]]
        if kind == "keyword_count":
            r[i] = keyword_hits(window, kws)
        elif kind == "keyword_coverage":
            r[i] = keyword_coverage(window, kws)
        elif kind == "linear":
            r[i] = float(np.dot(np.asarray(hidden[i, d - 1], np.float64), np.asarray(w, np.float64)))
        else:
            raise ValueError(kind)
    return r


def commit(draft: Decoder, target: Decoder, st: PromptState, emitted: Sequence[int],
           lead: Optional[int] = None) -> PromptState:
    """a8: pfx <- pfx + O; both caches are extended by feeding O, and the
    next head distribution is read at the last emitted token.  ``lead`` (soft
    rejection) is the token that heads the next beams."""
    emitted = [int(t) for t in emitted]
    if not emitted:      # pfx + [] = pfx (an Alg. 1 iteration that accepted nothing)
        return PromptState(list(st.tokens), st.n_prompt, st.draft_cache, st.target_cache, st.s, st.s_logits,
                           None if lead is None else int(lead), st.q_logits)
    dout, dc = draft.extend(st.draft_cache, emitted)
    out, tc = target.extend(st.target_cache, emitted)
    z = out.logits[-1]
    return PromptState(st.tokens + emitted, st.n_prompt, dc, tc, log_softmax(z), z,
                       None if lead is None else int(lead), dout.logits[-1])


# ----------------------------------------------------------------------------
# speculative sampling (soft rejection), Sec. 3.2.2
# ----------------------------------------------------------------------------
def soft_accept_count(lp_target: Sequence[float], lp_draft: Sequence[float], u: Sequence[float]) -> int:
    """Speculative sampling's test on one lookahead: x_j is rejected when
    u_j > min(1, p_j(x_j) / q_j(x_j)), with u_j ~ U[0, 1) given and the
    ratio formed from the two log-probs; returns the number of positions
    before the first rejection."""
    n = 0
    for lt, ld, uj in zip(lp_target, lp_draft, u):
        if float(uj) > min(1.0, math.exp(float(lt) - float(ld))):
            break
        n += 1
    return n


def soft_accept_margins(lp_target, lp_draft, u) -> np.ndarray:
    """Distance of every u_j from its acceptance bound min(1, p/q)."""
    lt = np.asarray(lp_target, np.float64)
    ld = np.asarray(lp_draft, np.float64)
    return np.abs(np.asarray(u, np.float64) - np.minimum(1.0, np.exp(lt - ld)))


def residual_sample(zp: np.ndarray, zq: np.ndarray, v: float):
    """The new token at a rejected position: a draw from the adjusted
    distribution w = max(0, p - q) / Z, Z = sum(w), with p and q the
    softmaxes of the target and draft logits there.  The draw inverts the
    cumulative sum over token ids in ascending order at v * Z: the smallest
    t with w_0 + ... + w_t > v * Z.  When Z = 0 (p <= q everywhere, which
    after a rejection only rounding can cause) it is argmax p.  Returns
    (token, log p(token), margin) with margin = the distance of v * Z from
    the nearest cumulative boundary, over Z."""
    p = np.exp(log_softmax(zp))
    q = np.exp(log_softmax(zq))
    w = np.maximum(0.0, p - q)
    Z = float(np.sum(w))
    lp = np.log(p)
    if Z <= 0.0:
        t = argmax_lowest(zp)
        return t, float(lp[t]), 0.0
    target = float(v) * Z
    run = 0.0
    t = -1
    for tok in range(len(w)):
        if w[tok] <= 0.0:
            continue
        nxt = run + float(w[tok])
        if nxt > target:
            t = tok
            break
        run = nxt
    if t < 0:            # v * Z beyond the rounded total: the last token with mass
        t = int(np.nonzero(w > 0.0)[0][-1])
        return t, float(lp[t]), 0.0
    margin = min(target - run, run + float(w[t]) - target) / Z
    return t, float(lp[t]), margin


def residual_interval(zp: np.ndarray, zq: np.ndarray, t: int):
    """The part of [0, 1) that draws token t in ``residual_sample``: the
    cumulative sums of w / Z before and after t (equal when w_t = 0), and Z."""
    p = np.exp(log_softmax(zp))
    q = np.exp(log_softmax(zq))
    w = np.maximum(0.0, p - q)
    Z = float(np.sum(w))
    if Z <= 0.0:
        return 0.0, 0.0, 0.0
    lo = float(np.sum(w[:t])) / Z
    return lo, lo + float(w[t]) / Z, Z


@dataclass
class SoftResult:
    n: np.ndarray              # [k] positions before the first soft rejection
    accept_margin: np.ndarray  # [k, d] |u - min(1, p/q)|
    lead: Optional[int]        # residual draw of the selected beam (None when n = d)
    lead_lp: Optional[float]
    lead_margin: float


@dataclass
class StepResult:
    heads: np.ndarray          # [k]
    head_lp: np.ndarray        # [k]
    head_margins: np.ndarray   # [k] gap between consecutive top-(k+1) values of s_t
    roll: Rollout
    ver: Verify
    reward: np.ndarray         # [k]
    combined: np.ndarray       # [k]
    beam: int
    emitted: List[int]
    state: PromptState         # state after the commit
    soft: Optional[SoftResult] = None


def beam_heads(st: PromptState, k: int):
    """a1: top-k of s_t (value descending, id ascending) and their log-probs.
    After a soft rejection the resampled token ``st.lead`` comes first and
    the other k - 1 heads are the top of s_t without it.  The margins are
    the gaps between consecutive values of the ranked part (inf for the
    lead, which the residual draw decides)."""
    if st.lead is None:
        ids = topk_ids(st.s_logits, k)
        srt = np.sort(st.s_logits)[::-1][:k + 1]
        return ids, st.s[ids], -np.diff(srt)
    rest = [int(t) for t in topk_ids(st.s_logits, k) if int(t) != st.lead][:k - 1]
    ids = np.array([st.lead] + rest, np.int64)
    others = np.delete(np.asarray(st.s_logits, np.float64), st.lead)
    srt = np.sort(others)[::-1][:k]
    return ids, st.s[ids], np.concatenate([[math.inf], -np.diff(srt)])


def step(draft: Decoder, target: Decoder, st: PromptState, k: int, d: int, alpha: float,
         reward_kind: str, kws=None, w=None, tree: bool = True, rejection: str = "hard",
         u: Optional[np.ndarray] = None, v: Optional[np.ndarray] = None) -> StepResult:
    """One CDSL step.  rejection = "soft" takes speculative sampling's test
    with the given uniforms u [k, d] and draws the next lead token with
    v [k, d] (the entry of the selected beam at its rejected position)."""
    heads, head_lp, hm = beam_heads(st, k)
    ro = rollout(draft, st, heads, d)
    ve = verify(target, st, heads, head_lp, ro.x, tree=tree)
    r = reward_for(reward_kind, st.generated, heads, ro.x, ve.hidden, kws, w)
    comb = r if (math.isinf(alpha) and alpha > 0) else ve.scores + alpha * r
    b = select_beam(ve.scores, r, alpha)
    soft = None
    if rejection == "soft":
        ns = np.array([soft_accept_count(ve.logprobs[i], ro.lq[i], u[i]) for i in range(k)], np.int64)
        am = np.stack([soft_accept_margins(ve.logprobs[i], ro.lq[i], u[i]) for i in range(k)])
        n = int(ns[b])
        lead, lead_lp, lm = None, None, math.inf
        if n < d:
            lead, lead_lp, lm = residual_sample(ve.logits[b, n], ro.logits[b, n], v[b, n])
        soft = SoftResult(ns, am, lead, lead_lp, lm)
    elif rejection == "hard":
        n = int(ve.n[b])
        lead = None
    else:
        raise ValueError(rejection)
    emitted = [int(heads[b])] + [int(t) for t in ro.x[b, :n]]
    nst = commit(draft, target, st, emitted, lead)
    return StepResult(heads, head_lp, hm, ro, ve, r, comb, b, emitted, nst, soft)


# ----------------------------------------------------------------------------
# the baselines (CDLH, CDLH-appx.) and the full controller (Alg. 1 states)
# ----------------------------------------------------------------------------
def keyword_reward(kind: str, window: Sequence[int], kws: Sequence[int]) -> float:
    """The lexical reward R of Sec. 4.1 on one token window: the number of
    distinct concepts present, or that number over the number of concepts."""
    if kind == "keyword_count":
        return float(keyword_hits(window, kws))
    if kind == "keyword_coverage":
        return keyword_coverage(window, kws)
    raise ValueError(f"the controller and the baselines take a lexical reward, not {kind!r}")


def argmax_first(values: Sequence[float]) -> int:
    """Index of the largest value, the first one on ties (the strict '>'
    update of the appendix algorithm)."""
    best = 0
    for i in range(1, len(values)):
        if values[i] > values[best]:
            best = i
    return best


@dataclass
class HeadStep:
    heads: np.ndarray          # [k] top-k of M_p at the prefix end
    x: np.ndarray              # [k, d] greedy lookahead of every head (by the roller)
    margin: np.ndarray         # [k, d] top-2 margin of the roller at each draw
    reward: np.ndarray         # [k]
    pick: int
    token: int                 # the one emitted token
    state: PromptState         # after it
    head_margin: float         # smallest gap among the target's top-(k+1) logits


def lookahead_heads(roller: Decoder, roller_cache: KVCache, st: PromptState, k: int, d: int):
    """The k candidate tokens of the appendix algorithm -- the top-k of M_p
    at the prefix end, value descending, lowest id first on ties (after a
    soft rejection, the resampled token first: ``beam_heads``) -- each
    followed by d greedy tokens of the roller on its own copy of the cache."""
    heads = beam_heads(st, k)[0]
    x = np.zeros((k, d), np.int64)
    mg = np.zeros((k, d))
    for i, c in enumerate(heads):
        cache = roller_cache
        fed = int(c)
        for j in range(d):
            out, cache = roller.extend(cache, [fed])
            z = out.logits[0]
            x[i, j] = argmax_lowest(z)
            mg[i, j] = top2_margin(z)
            fed = int(x[i, j])
    return heads, x, mg


def cdlh_step(roller_is_target: bool, draft: Decoder, target: Decoder, st: PromptState, k: int, d: int,
              reward_kind: str, kws: Sequence[int], prefer_first_at: Optional[float] = None) -> HeadStep:
    """One token of lookahead-heuristic decoding (Sec. 2.1 and the appendix
    algorithm): every top-k candidate of M_p is extended by d greedy tokens,
    by M_p itself (CDLH) or by the draft M_q (CDLH-appx., Sec. 3.1); R scores
    generated-so-far + candidate + lookahead (the prompt is left out, as in
    the step), and the best candidate is the one token emitted.

    prefer_first_at = r_t folds Step-1 of Alg. 1 with b = 1 into the same
    candidate table: the first candidate (M_p's greedy token; after a soft
    rejection of the beam step, the resampled token) is taken when its
    lookahead reaches the threshold, else the best.  With b = 1 Step-1's
    X_1 and its lookahead are exactly candidate 0 and its lookahead, so this
    equals Step-1 followed by Step-2 (``controller_step`` computes them
    apart, in the paper's order)."""
    roller = target if roller_is_target else draft
    cache = st.target_cache if roller_is_target else st.draft_cache
    heads, x, mg = lookahead_heads(roller, cache, st, k, d)
    r = np.array([keyword_reward(reward_kind, list(st.generated) + [int(heads[i])] + [int(t) for t in x[i]], kws)
                  for i in range(k)])
    if prefer_first_at is not None and r[0] >= prefer_first_at:
        pick = 0
    else:
        pick = argmax_first(r)
    tok = int(heads[pick])
    hm = float(np.min(beam_heads(st, k)[2]))
    return HeadStep(heads, x, mg, r, pick, tok, commit(draft, target, st, [tok]), hm)


# ----------------------------------------------------------------------------
# Alg. 1 itself: lookaheads drafted from the prefix, no beam heads
# ----------------------------------------------------------------------------
def draft_from_prefix(draft: Decoder, st: PromptState, d: int) -> Rollout:
    """Alg. 1, drafting loop: q_1 = M_q(pfx) is the draft's distribution at
    the end of the prefix, x_j = argmax q_j (lowest id on ties) and
    q_{j+1} = M_q(pfx + x_1..x_j), for j = 1..d (one sequence: k = 1)."""
    x = np.zeros((1, d), np.int64)
    mg = np.zeros((1, d))
    lq = np.zeros((1, d))
    zs = np.zeros((1, d, draft.shape.vocab))
    z = np.asarray(st.q_logits, np.float64)
    cache = st.draft_cache
    for j in range(d):
        x[0, j] = argmax_lowest(z)
        mg[0, j] = top2_margin(z)
        lq[0, j] = log_softmax(z)[x[0, j]]
        zs[0, j] = z
        if j + 1 < d:
            out, cache = draft.extend(cache, [int(x[0, j])])
            z = out.logits[0]
    return Rollout(x, mg, lq, zs)


def verify_from_prefix(target: Decoder, st: PromptState, x: Sequence[int], kk: int) -> Verify:
    """Alg. 1, verification: p_1 = M_p(pfx) (the target's distribution at
    the end of the prefix) and p_j = M_p(pfx + x_1..x_{j-1}) for j = 2..d,
    the last d - 1 in one causal pass over x_1..x_{d-1}; then per row the
    log-prob of x_j, the argmax y_j, the top-kk (the candidates that Step-2
    needs after n accepted tokens are those of row n + 1) and the leading
    matches n (the rejection loop).  One sequence: the outputs are [1, d]."""
    x = np.asarray(x, np.int64).reshape(-1)
    d = x.shape[0]
    rows = [np.asarray(st.s_logits, np.float64)]
    if d > 1:
        out, _ = target.extend(st.target_cache, [int(t) for t in x[:d - 1]])
        rows += list(out.logits)
    logits = np.stack(rows)[None]                    # [1, d, V]
    lp = np.zeros((1, d))
    y = np.zeros((1, d), np.int64)
    mg = np.zeros((1, d))
    rtk = np.zeros((1, d, kk), np.int64)
    rtl = np.zeros((1, d, kk))
    for j in range(d):
        z = logits[0, j]
        ls = log_softmax(z)
        lp[0, j] = ls[x[j]]
        y[0, j] = argmax_lowest(z)
        mg[0, j] = top2_margin(z)
        rtk[0, j] = topk_ids(z, kk)
        rtl[0, j] = ls[rtk[0, j]]
    n = np.array([leading_matches(y[0], x)], np.int64)
    return Verify(logits, None, lp, y, mg, n, lp.sum(1), rtk, rtl)


@dataclass
class Step1Try:
    """One round of Step-1 (S2/S3): M_p's greedy token X_i after
    pfx + x_1..x_n + X_1..X_{i-1}, the draft's d-token lookahead after it, and
    the reward of the whole window."""
    X: List[int]               # X_1..X_i
    x_margin: float            # top-2 margin of M_p's logits at the choice of X_i
    lh: np.ndarray             # [d] the lookahead
    lh_margin: np.ndarray      # [d] top-2 margins of its draws
    reward: float              # R(generated + x_1..x_n + X_1..X_i + lh)


@dataclass
class ControllerStep:
    x: np.ndarray              # [d] x_1..x_d drafted from the prefix
    draft_margin: np.ndarray   # [d] top-2 margins of the draft draws
    ver: Verify                # p_1..p_d of the verification, [1, d]
    n: int                     # accepted tokens (hard: leading matches; soft: speculative sampling)
    a: float                   # n / d
    r: float                   # R(generated + x_1..x_n)
    state: str                 # "S1", "S2/S3" or "S4"
    step1: List[Step1Try]      # the Step-1 rounds tried (S2/S3 with b > 0)
    extra: Optional[HeadStep]  # the CDLH-appx. token of Step-2 / S4
    emitted: List[int]
    after: PromptState
    soft: Optional[SoftResult] = None   # speculative sampling's test on x_1..x_d
    roll: Optional[Rollout] = None


def controller_step(draft: Decoder, target: Decoder, st: PromptState, k: int, d: int, a_t: float, r_t: float,
                    b: int, reward_kind: str, kws: Sequence[int], rejection: str = "hard",
                    u: Optional[np.ndarray] = None) -> ControllerStep:
    """One iteration of Alg. 1 (Sec. 3.2.1-3.2.3) with hard rejection, or
    with speculative sampling's test in the rejection loop (rejection =
    "soft", uniforms u of shape [1, d]: x_j is kept while u_j <= min(1,
    p_j(x_j) / q_j(x_j))).

    Draft x_1..x_d greedily from pfx; verify them with p_1..p_d; n = the
    accepted count, a = n / d, r = R(generated + x_1..x_n).  Then:
      S1 (a >= a_t and r >= r_t): O = [x_1..x_n].
      S2/S3 (a < a_t): Step-1 tries up to b tokens of M_p: X_i = argmax
          M_p(pfx + x_1..x_n + X_1..X_{i-1}), a d-token draft lookahead lh
          after it, and if R(generated + x_1..x_n + X_1..X_i + lh) >= r_t
          then O = [x_1..x_n] + X_1..X_i.  If no round reaches r_t the X are
          dropped and Step-2 adds the CDLH-appx. token after x_1..x_n.
      S4 (a >= a_t, r < r_t): O = [x_1..x_n] + the CDLH-appx. token.
    The reward windows leave the prompt out, as the step's do.  a_t must be
    positive: with a_t <= 0 an iteration that accepts nothing would be S1
    and emit nothing, and the deterministic loop would stand still (the
    paper's settings use a_t >= 0.3).  With soft rejection only the
    acceptance count changes: the S1 action emits no token beyond the
    accepted ones and Step-1 takes M_p's greedy tokens, so the residual
    draw at the rejected position plays no part."""
    if not a_t > 0:
        raise ValueError("a_t must be positive")
    if b < 0:
        raise ValueError("b must be >= 0")
    ro = draft_from_prefix(draft, st, d)
    x = ro.x[0]
    ve = verify_from_prefix(target, st, x, k)
    soft = None
    if rejection == "soft":
        n = soft_accept_count(ve.logprobs[0], ro.lq[0], u[0])
        soft = SoftResult(np.array([n]), soft_accept_margins(ve.logprobs[0], ro.lq[0], u[0])[None], None, None,
                          math.inf)
    elif rejection == "hard":
        n = int(ve.n[0])
    else:
        raise ValueError(rejection)
    a = n / d
    acc = [int(t) for t in x[:n]]
    r = keyword_reward(reward_kind, list(st.generated) + acc, kws)
    st1 = commit(draft, target, st, acc)
    if a >= a_t and r >= r_t:
        return ControllerStep(x, ro.margin[0], ve, n, a, r, "S1", [], None, acc, st1, soft, ro)
    state = "S2/S3" if a < a_t else "S4"
    tries: List[Step1Try] = []
    if state == "S2/S3":
        cur, X = st1, []
        for _ in range(b):
            Xi = argmax_lowest(cur.s_logits)
            xm = top2_margin(cur.s_logits)
            X.append(Xi)
            cur = commit(draft, target, cur, [Xi])
            lh = draft_from_prefix(draft, cur, d)
            rr = keyword_reward(reward_kind, list(st.generated) + acc + X + [int(t) for t in lh.x[0]], kws)
            tries.append(Step1Try(list(X), xm, lh.x[0], lh.margin[0], rr))
            if rr >= r_t:
                return ControllerStep(x, ro.margin[0], ve, n, a, r, state, tries, None, acc + X, cur, soft, ro)
    hs = cdlh_step(False, draft, target, st1, k, d, reward_kind, kws)
    return ControllerStep(x, ro.margin[0], ve, n, a, r, state, tries, hs, acc + [hs.token], hs.state, soft, ro)
