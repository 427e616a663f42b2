"""Test harness: the same seeded workload on the GPU library and on the CPU
oracle, and the step-by-step comparison rules.

Comparison rules (for the GPU against the float64 oracle):
* token ids (beam heads, draft argmax, target argmax) are bit-exact wherever
  the oracle's deciding margin exceeds TOK_MARGIN; below it either choice is
  correct, and since every later quantity then depends on that choice, the
  trajectory comparison stops there (logged; every prompt either runs all
  its steps or ends at such a tie, see assert_full_or_tie);
* the selected beam is bit-exact wherever the oracle's best-vs-second gap of
  score + alpha * reward exceeds max(TOK_MARGIN, 2 * the largest difference
  between the GPU's and the oracle's combined values of that step): when
  every combined value is within e of the oracle's, only a gap below 2e can
  reorder the best two;
* log-probs within LP_TOL (1e-4 fp32, 2e-2 bf16), beam scores within
  (d + 1) * LP_TOL;
* the linear reward's hidden state within LP_TOL per entry, and the reward
  within |w|_1 times the measured hidden-state error (plus fp32 rounding of
  the dot product), the bound that error implies.
No GPU value is ever fed into the oracle.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import cdsl_inputs as ci
import oracle

TOK_MARGIN = 1e-2


def lp_tol(dtype):
    return 1e-4 if dtype == "f32" else 2e-2


@dataclass
class Setup:
    wl: object
    draft_np: dict
    target_np: dict
    odraft: object
    otarget: object
    engine: object = None
    kws: Optional[np.ndarray] = None
    rw: Optional[np.ndarray] = None

    def prompts(self, B, first=0):
        return ci.prompts(self.wl.seed, B, self.wl.prompt_len, self.wl.target.vocab, first=first)


def make_setup(name, draft_is_target=False, B=None, max_steps=8, k=None, d=None, **wl_over):
    wl = ci.workload(name)
    if wl_over:
        wl = wl.with_(**wl_over)
    if draft_is_target:
        wl = wl.with_(draft=wl.target)
    tw = ci.model_weights(wl.target, wl.seed, 1, wl.dtype)
    dw = tw if draft_is_target else ci.model_weights(wl.draft, wl.seed, 0, wl.dtype)
    s = Setup(wl, dw, tw, oracle.Decoder(wl.draft, dw), oracle.Decoder(wl.target, tw))
    B = max(B or wl.batch, 64)
    if wl.reward.startswith("keyword"):
        s.kws = ci.keywords(wl.seed, B, wl.n_keywords, wl.target.vocab)
    else:
        s.rw = ci.reward_head(wl.seed, wl.target.d_model)
    return s


def make_engine(s: Setup, B, max_steps=8, k=None, d=None):
    import torch
    from paper_2412_10418_amd.engine import Engine
    dwd, twd = Engine.upload(s.wl, s.draft_np, s.target_np)
    s.engine = Engine(s.wl, dwd, twd, max_steps=max_steps, max_batch=B, k=k, d=d)
    return s.engine


@dataclass
class Report:
    steps_compared: int = 0
    stopped: str = ""
    max_lp_err: float = 0.0
    max_score_err: float = 0.0
    checks: int = 0


def _first_diff(a, b):
    for u, (x, y) in enumerate(zip(a, b)):
        if int(x) != int(y):
            return u
    return -1


def soft_margins(dtype):
    """(acceptance, residual) margins below which either soft decision is
    correct, from the log-prob tolerance e: the bound min(1, p/q) moves by up
    to e^(2e) - 1 ~ 2e; a cumulative boundary of the residual by up to
    sum |dp| + sum |dq| ~ 2e in probability, i.e. 2e / Z in the units of v."""
    e = lp_tol(dtype)
    return 2.0 * e, 2.0 * e


def assert_full_or_tie(reps, steps):
    """Every compared prompt ran all ``steps`` steps, or its comparison
    ended at a logged near tie (whose oracle margin compare_step checked)."""
    for b, r in reps.items():
        assert r.steps_compared >= 1, (b, r)
        assert r.steps_compared == steps or r.stopped, (b, r)


def compare_step(rep: Report, wl, k, d, o_step, g_heads, g_head_lp, g_look, g_ver, g_reward, g_beam, g_emit,
                 tol, g_v=None, alpha=None, w=None) -> bool:
    """Compare one prompt's step; returns False when a legal near-tie
    divergence ends the trajectory comparison (raises on a real mismatch),
    "last" when the step matched but the trajectories part after it.
    With soft rejection (o_step.soft set), the acceptance counts, the draft
    log-probs and the residual draw are compared too; g_v is the prompt's
    v [k, d]."""
    # a1 beam heads: ordered top-k of s_t
    oh = o_step.heads
    u = _first_diff(g_heads, oh)
    if u >= 0:
        assert o_step.head_margins[u] <= TOK_MARGIN, (u, list(g_heads), list(oh), o_step.head_margins)
        rep.stopped = f"beam-head near tie (margin {o_step.head_margins[u]:.2e})"
        return False
    assert np.max(np.abs(g_head_lp - o_step.head_lp)) <= tol
    # a2 rollout
    ox = o_step.roll.x
    assert np.array_equal(g_look[:, 0], oh)
    for i in range(k):
        u = _first_diff(g_look[i, 1:], ox[i])
        if u >= 0:
            assert o_step.roll.margin[i, u] <= TOK_MARGIN, (i, u, g_look[i], ox[i], o_step.roll.margin[i])
            rep.stopped = f"draft near tie (beam {i}, j {u}, margin {o_step.roll.margin[i, u]:.2e})"
            return False
    # a3-a5 verification of identical inputs
    ve = o_step.ver
    lp_err = np.max(np.abs(g_ver["logprobs"] - ve.logprobs))
    assert lp_err <= tol, lp_err
    rep.max_lp_err = max(rep.max_lp_err, lp_err)
    ok = ve.margin > TOK_MARGIN
    assert np.array_equal(g_ver["target_argmax"][ok], ve.y[ok])
    so = o_step.soft
    if so is not None:
        am, rm = soft_margins(wl.dtype)
        assert np.max(np.abs(g_ver["draft_lp"] - o_step.roll.lq)) <= tol
        for i in range(k):
            gn, on = int(g_ver["n_accept"][i]), int(so.n[i])
            if gn != on:
                j = min(gn, on)
                assert so.accept_margin[i, j] <= am, (i, gn, on, so.accept_margin[i])
                rep.stopped = f"soft acceptance near tie (beam {i}, j {j}, margin {so.accept_margin[i, j]:.1e})"
                return False
    elif np.all(ok) or np.array_equal(g_ver["target_argmax"], ve.y):
        assert np.array_equal(g_ver["n_accept"], ve.n)
    elif not np.array_equal(g_ver["n_accept"], ve.n):
        rep.stopped = "target argmax near tie"
        return False
    sc_err = np.max(np.abs(g_ver["scores"] - ve.scores))
    assert sc_err <= tol * (d + 1), sc_err
    rep.max_score_err = max(rep.max_score_err, sc_err)
    # a6 reward
    if wl.reward.startswith("keyword"):
        assert np.array_equal(g_reward, o_step.reward)
    else:
        oh = o_step.ver.hidden[:, d - 1]
        h_err = float(np.max(np.abs(g_ver["hidden"] - oh)))
        assert h_err <= tol, h_err
        w64 = np.asarray(w, np.float64)
        bound = float(np.sum(np.abs(w64))) * h_err + 1e-5 * float(np.max(np.abs(oh) @ np.abs(w64)))
        r_err = float(np.max(np.abs(g_reward - o_step.reward)))
        assert r_err <= bound, (r_err, bound, h_err)
    # a7 select
    alpha = wl.alpha if alpha is None else alpha
    g_comb = (np.asarray(g_reward, np.float64) if (math.isinf(alpha) and alpha > 0)
              else np.asarray(g_ver["scores"], np.float64) + alpha * np.asarray(g_reward, np.float64))
    comb_err = float(np.max(np.abs(g_comb - o_step.combined)))
    window = max(TOK_MARGIN, 2.0 * comb_err)
    comb = np.sort(o_step.combined)[::-1]
    gap = comb[0] - comb[1] if len(comb) > 1 else math.inf
    if int(g_beam) != o_step.beam:
        assert gap <= window, (g_beam, o_step.beam, o_step.combined, window)
        rep.stopped = f"selection near tie (gap {gap:.2e}, window {window:.2e})"
        return False
    # a8 commit
    assert list(g_emit) == list(o_step.emitted)
    if so is not None and so.lead is not None:
        i, n = int(g_beam), int(so.n[int(g_beam)])
        g_res = int(g_ver["res_ids"][i, n])
        assert abs(float(g_ver["res_lp"][i, n]) - so.lead_lp) <= tol or g_res != so.lead
        if g_res != so.lead:
            # a different draw must still sit at v in the oracle's residual
            # distribution, within the residual margin
            lo, hi, Z = oracle.residual_interval(o_step.ver.logits[i, n], o_step.roll.logits[i, n], g_res)
            vv = float(g_v[i, n])
            win = rm / Z
            assert hi > lo and lo - win <= vv <= hi + win, (g_res, so.lead, lo, hi, vv, Z)
            assert so.lead_margin <= win, (g_res, so.lead, so.lead_margin, Z)
            # this step matched; the next one starts from another lead token
            rep.stopped = f"after this step: residual draw near a boundary (margin {so.lead_margin:.1e})"
            rep.checks += 1
            return "last"
    rep.checks += 1
    return True


def run_and_compare(s: Setup, B: int, steps: int, check_prompts, k=None, d=None, alpha=None, soft=False):
    """Run ``steps`` GPU steps on a batch of B prompts and compare the listed
    prompts step by step with independent oracle runs.  soft: speculative
    sampling's rejection with seeded uniforms of the workload."""
    import torch
    wl = s.wl
    k = k or wl.k
    d = d or wl.d
    alpha = wl.alpha if alpha is None else alpha
    eng = s.engine
    prompts = s.prompts(B)
    st = eng.start(torch.from_numpy(prompts).cuda(), k=k)
    kw_t = torch.from_numpy(s.kws[:B]).cuda() if s.kws is not None else None
    rw_t = torch.from_numpy(s.rw).cuda() if s.rw is not None else None
    ost = {b: oracle.prefill(s.odraft, s.otarget, prompts[b]) for b in check_prompts}
    reps = {b: Report() for b in check_prompts}
    live = set(check_prompts)
    tol = lp_tol(wl.dtype)
    for t in range(steps):
        heads = st.beams.cpu().numpy().copy()
        head_lp = st.head_lp.cpu().numpy().copy()
        u = v = None
        if soft:
            u = ci.uniforms(wl.seed, 0, t, B, k, d)
            v = ci.uniforms(wl.seed, 1, t, B, k, d)
        bf = eng.step(st, keywords=kw_t, reward_w=rw_t, alpha=alpha, k=k, d=d,
                      u=torch.from_numpy(u).cuda() if soft else None, v=torch.from_numpy(v).cuda() if soft else None)
        look = bf.lookaheads.cpu().numpy()
        ver = {kk: (v.cpu().numpy() if v is not None else None) for kk, v in bf.verify.items()}
        rew = bf.reward.cpu().numpy()
        beam = bf.beam.cpu().numpy()
        for b in list(live):
            o = oracle.step(s.odraft, s.otarget, ost[b], k, d, alpha, wl.reward,
                            kws=s.kws[b] if s.kws is not None else None, w=s.rw,
                            rejection="soft" if soft else "hard",
                            u=u[b] if soft else None, v=v[b] if soft else None)
            gv = {kk: (x[b] if x is not None else None) for kk, x in ver.items()}
            cont = compare_step(reps[b], wl, k, d, o, heads[b], head_lp[b], look[b], gv, rew[b], beam[b],
                                eng._last_emitted[b], tol, g_v=v[b] if soft else None, alpha=alpha, w=s.rw)
            if cont:
                reps[b].steps_compared += 1
                ost[b] = o.state
            if cont is not True:
                live.discard(b)
    return st, reps
