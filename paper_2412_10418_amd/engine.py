"""One CDSL lookahead step on the GPU, driven through the C ABI.

A step is rollout -> verify -> reward -> select -> commit on the context
stream, with the step's device buffers allocated once per (B, k, d) so the
steady-state loop allocates nothing.

Also the paper's baselines and its full controller on the same calls:
``head_step`` emits one token of lookahead-heuristic decoding (CDLH with the
target as the roller, CDLH-appx. with the draft; Sec. 2.1, 3.1 and the
appendix algorithm), and ``controller_step`` runs one iteration of Alg. 1:
lookaheads drafted from the prefix, then states S1 .. S4 of Sec. 3.2.3 with
thresholds a_t, r_t and b <= 1.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import torch

from .binding import Context, Prefix, upload_weights

# state codes of cdsl_controller_states
STATE_NAMES = {1: "S1", 2: "S2/S3", 4: "S4"}


@dataclass
class StepBuffers:
    lookaheads: torch.Tensor
    verify: Dict[str, torch.Tensor]
    reward: torch.Tensor
    beam: torch.Tensor
    next_beams: torch.Tensor
    next_head_lp: torch.Tensor


@dataclass
class DecodeState:
    prefix: Prefix
    beams: torch.Tensor
    head_lp: torch.Tensor
    emitted: List[List[int]] = field(default_factory=list)


class Engine:
    def __init__(self, workload, draft_w, target_w, max_steps: int, device="cuda",
                 max_batch: Optional[int] = None, k: Optional[int] = None, d: Optional[int] = None,
                 max_prompt: Optional[int] = None, max_prefixes: int = 1):
        wl = workload
        self.wl = wl
        self.k = k or wl.k
        self.d = d or wl.d
        self.device = device
        B = max_batch or wl.batch
        mp = max_prompt or wl.prompt_len
        limits = dict(max_batch=B, max_prompt=mp,
                      max_ctx=max(mp, wl.prompt_len + max_steps * (self.d + 1) + 2),
                      max_k=self.k, max_d=self.d, max_prefixes=max_prefixes)
        self.ctx = Context(wl.draft, draft_w, wl.target, target_w, wl.dtype, limits)
        self._bufs: Dict[tuple, StepBuffers] = {}

    @staticmethod
    def upload(workload, draft_np, target_np, device="cuda"):
        return (upload_weights(draft_np, workload.dtype, device),
                upload_weights(target_np, workload.dtype, device))

    def buffers(self, B: int, k: int, d: int) -> StepBuffers:
        key = (B, k, d)
        if key not in self._bufs:
            dev = self.device
            z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=dev)
            i32 = torch.int32
            want_hidden = self.wl.reward == "linear"
            self._bufs[key] = StepBuffers(
                lookaheads=z(B, k, d + 1, dt=i32),
                verify={
                    "logprobs": z(B, k, d), "target_argmax": z(B, k, d, dt=i32), "n_accept": z(B, k, dt=i32),
                    "scores": z(B, k), "row_topk_ids": z(B, k, d, k, dt=i32), "row_topk_lp": z(B, k, d, k),
                    "hidden": z(B, k, self.wl.target.d_model) if want_hidden else None,
                },
                reward=z(B, k), beam=z(B, dt=i32), next_beams=z(B, k, dt=i32), next_head_lp=z(B, k))
        return self._bufs[key]

    def start(self, prompts: torch.Tensor, k: Optional[int] = None) -> DecodeState:
        k = k or self.k
        prefix, beams, head_lp = self.ctx.cdsl_prefill(prompts, k)
        return DecodeState(prefix, beams, head_lp, [[] for _ in range(prompts.shape[0])])

    def _soft_buffers(self, B: int, k: int, d: int, bf: StepBuffers):
        key = ("soft", B, k, d)
        if key not in self._bufs:
            dev = self.device
            z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=dev)
            self._bufs[key] = {"draft_logits": z(B, k, d, self.wl.draft.vocab)}
            bf.verify.update(draft_lp=z(B, k, d), res_ids=z(B, k, d, dt=torch.int32), res_lp=z(B, k, d))
        return self._bufs[key]

    def step(self, st: DecodeState, keywords: Optional[torch.Tensor] = None,
             reward_w: Optional[torch.Tensor] = None, alpha: Optional[float] = None,
             k: Optional[int] = None, d: Optional[int] = None, marks: Optional[list] = None,
             reward: Optional[str] = None, u: Optional[torch.Tensor] = None,
             v: Optional[torch.Tensor] = None) -> StepBuffers:
        """One lookahead step.  Updates ``st`` in place; returns the step's
        buffers (valid until the next step with the same shape).  With a list
        ``marks``, timing events are appended before the rollout, after it,
        after the verification and after the commit.  ``reward`` overrides the
        workload's reward kind.  With uniforms u and v ([B, k, d] device
        float32) the step uses speculative sampling's soft rejection."""
        def mark():
            if marks is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append(e)

        k = k or self.k
        d = d or self.d
        alpha = self.wl.alpha if alpha is None else alpha
        B = st.prefix.B
        bf = self.buffers(B, k, d)
        c = self.ctx
        soft = u is not None
        if soft:
            if v is None:
                raise ValueError("soft rejection takes both u and v")
            sb = self._soft_buffers(B, k, d, bf)
        mark()
        if soft:
            c.cdsl_rollout_keep(st.prefix, st.beams, k, d, bf.lookaheads, sb["draft_logits"])
        else:
            c.cdsl_rollout(st.prefix, st.beams, k, d, bf.lookaheads)
        mark()
        if soft:
            c.cdsl_verify_soft(st.prefix, bf.lookaheads, k, d, st.head_lp, sb["draft_logits"], u, v, bf.verify,
                               want_hidden=bf.verify["hidden"] is not None)
        else:
            c.cdsl_verify(st.prefix, bf.lookaheads, k, d, st.head_lp, out=bf.verify)
        mark()
        kind = reward or self.wl.reward
        if kind == "linear":
            c.cdsl_reward_linear(bf.verify["hidden"], reward_w, bf.reward)
        else:
            c.cdsl_reward_keywords(st.prefix, bf.lookaheads, k, d, keywords,
                                   normalize=(kind == "keyword_coverage"), reward=bf.reward)
        c.cdsl_select(bf.verify["scores"], bf.reward, alpha, bf.beam)
        # commit writes the next heads into separate buffers, then they swap
        if soft:
            em = c.cdsl_commit_soft(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                                    bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], bf.verify["res_ids"],
                                    bf.verify["res_lp"], k, d, bf.next_beams, bf.next_head_lp)
        else:
            em, _, _ = c.cdsl_commit(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                                     bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], k, d,
                                     bf.next_beams, bf.next_head_lp)
        mark()
        for b in range(B):
            st.emitted[b].extend(em[b])
        st.beams, bf.next_beams = bf.next_beams, st.beams
        st.head_lp, bf.next_head_lp = bf.next_head_lp, st.head_lp
        self._last_emitted = em
        return bf

    # -- the baselines and the full controller ---------------------------------
    def _heads_buffers(self, B: int, k: int, d: int):
        key = ("heads", B, k, d)
        if key not in self._bufs:
            dev = self.device
            self._bufs[key] = {"look": torch.zeros(B, k, d + 1, dtype=torch.int32, device=dev),
                               "reward": torch.zeros(B, k, device=dev),
                               "beam": torch.zeros(B, dtype=torch.int32, device=dev)}
        return self._bufs[key]

    def _controller_buffers(self, B: int, k: int, d: int):
        key = ("ctrl", B, k, d)
        if key not in self._bufs:
            dev = self.device
            z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=dev)
            i32 = torch.int32
            self._bufs[key] = {
                "look": z(B, d + 1, dt=i32),
                "verify": {"logprobs": z(B, d), "target_argmax": z(B, d, dt=i32), "n_accept": z(B, dt=i32),
                           "scores": z(B), "row_topk_ids": z(B, d, k, dt=i32), "row_topk_lp": z(B, d, k)},
                "reward": z(B), "next_beams": z(B, k, dt=i32), "next_head_lp": z(B, k),
                "state": z(B, dt=i32), "first_at": z(B)}
        return self._bufs[key]

    def _controller_soft_buffers(self, B: int, k: int, d: int, cb: dict):
        key = ("ctrl_soft", B, k, d)
        if key not in self._bufs:
            dev = self.device
            z = lambda *s, dt=torch.float32: torch.zeros(s, dtype=dt, device=dev)
            self._bufs[key] = {"draft_logits": z(B, d, self.wl.draft.vocab)}
            cb["verify"].update(draft_lp=z(B, d), res_ids=z(B, d, dt=torch.int32), res_lp=z(B, d))
        return self._bufs[key]

    def head_step(self, st: DecodeState, keywords: torch.Tensor, roller: int, k: Optional[int] = None,
                  d: Optional[int] = None, mask: Optional[List[bool]] = None,
                  first_at: Optional[torch.Tensor] = None,
                  normalize: Optional[bool] = None) -> dict:
        """One token of lookahead-heuristic decoding for every prompt (or the
        prompts with mask[b]): the k heads of ``st`` (top-k of the target) are
        rolled d tokens by the roller (1 = target: CDLH, 0 = draft:
        CDLH-appx.), scored by the lexical reward, and the best head is
        emitted.  first_at (device [B], NaN = off) makes prompt b take head 0
        when its reward reaches first_at[b] (Step-1 of Alg. 1 with b = 1)."""
        k = k or self.k
        d = d or self.d
        B = st.prefix.B
        hb = self._heads_buffers(B, k, d)
        c = self.ctx
        if normalize is None:
            normalize = self.wl.reward == "keyword_coverage"
        c.cdsl_rollout_with(st.prefix, st.beams, k, d, roller, hb["look"])
        c.cdsl_reward_keywords(st.prefix, hb["look"], k, d, keywords, normalize=normalize, reward=hb["reward"])
        if first_at is None:
            c.cdsl_select(hb["reward"], hb["reward"], math.inf, hb["beam"])
        else:
            c.cdsl_select_first(hb["reward"], first_at, hb["beam"])
        toks = c.cdsl_commit_heads(st.prefix, hb["look"], hb["beam"], k, d, mask, st.beams, st.head_lp)
        for b in range(B):
            if toks[b] >= 0:
                st.emitted[b].append(toks[b])
        return {"tokens": toks, "lookaheads": hb["look"], "reward": hb["reward"], "beam": hb["beam"]}

    def controller_step(self, st: DecodeState, keywords: torch.Tensor, a_t: float, r_t: float, b: int,
                        k: Optional[int] = None, d: Optional[int] = None,
                        normalize: Optional[bool] = None, u: Optional[torch.Tensor] = None) -> dict:
        """One iteration of Alg. 1 for every prompt, as the oracle's
        ``controller_step`` computes it: d draft tokens from the prefix
        (cdsl_draft_prefix), their verification p_1..p_d, n accepted (hard
        rejection, or speculative sampling's test with uniforms u [B, d]),
        a = n / d, r = R(generated + x_1..x_n), the state, and the commit of
        x_1..x_n.  Prompts not in S1 then take their action with the k
        candidates after x_1..x_n (the target's top-k, each with a d-token
        draft lookahead and its reward):
          S2/S3, Step-1: M_p's greedy token X_1 is candidate 0; it is taken
            when its lookahead reaches r_t.  With b >= 2 the prompts whose
            X_1 missed append it tentatively (cdsl_append), take X_2 = M_p's
            greedy token after it with a fresh lookahead, and so on for up to
            b tokens; the first round that reaches r_t keeps its X_1..X_i.
            If none does, the tentative tokens are withdrawn (cdsl_withdraw)
            and Step-2 follows.
          Step-2 and S4: the candidate with the best reward (CDLH-appx.).
        The host reads the state codes and, between Step-1 rounds, the
        round's rewards against r_t, to know which prompts continue."""
        if not a_t > 0:
            raise ValueError("a_t must be positive")
        if b < 0:
            raise ValueError("b must be >= 0")
        k = k or self.k
        d = d or self.d
        B = st.prefix.B
        cb = self._controller_buffers(B, k, d)
        c = self.ctx
        soft = u is not None
        if normalize is None:
            normalize = self.wl.reward == "keyword_coverage"
        ver = cb["verify"]
        if soft:
            sb = self._controller_soft_buffers(B, k, d, cb)
            c.cdsl_draft_prefix(st.prefix, d, cb["look"], sb["draft_logits"])
            # the residual draws (at v = u) are computed by the soft test but
            # play no part in Alg. 1
            c.cdsl_verify_prefix(st.prefix, cb["look"], d, k, ver, sb["draft_logits"], u, u)
        else:
            c.cdsl_draft_prefix(st.prefix, d, cb["look"])
            c.cdsl_verify_prefix(st.prefix, cb["look"], d, k, ver)
        c.cdsl_reward_keywords_prefix(st.prefix, cb["look"], d, ver["n_accept"], keywords, normalize, cb["reward"])
        c.cdsl_controller_states(ver["n_accept"], cb["reward"], d, a_t, r_t, min(b, 1), cb["state"],
                                 cb["first_at"])
        em = c.cdsl_commit_prefix(st.prefix, cb["look"], ver["n_accept"], d, ver["row_topk_ids"],
                                  ver["row_topk_lp"], cb["next_beams"], cb["next_head_lp"])
        # the commit has synchronised the stream: these reads only copy
        codes = cb["state"].cpu().tolist()
        n = ver["n_accept"].cpu().tolist()
        r = cb["reward"].cpu().tolist()
        states = [STATE_NAMES[x] for x in codes]
        for i in range(B):
            st.emitted[i].extend(em[i])
        st.beams.copy_(cb["next_beams"])
        st.head_lp.copy_(cb["next_head_lp"])
        extra, rounds = None, None
        need = [x != 1 for x in codes]
        if any(need):
            extra, rounds = self._step1_step2(st, keywords, codes, b, r_t, k, d, normalize, cb["first_at"])
        return {"states": states, "n": n, "r": r, "emitted": em, "extra": extra, "rounds": rounds}

    def _step1_step2(self, st: DecodeState, keywords, codes, b, r_t, k, d, normalize, first_at):
        """The one-token actions of the prompts not in S1 (see
        controller_step).  Returns the candidate table (heads, lookaheads,
        rewards, the chosen index and the emitted token per prompt) and the
        Step-1 rounds beyond the first: a list of {"X": [B] tokens,
        "lookaheads": [B, 1, d+1], "reward": [B], "active": [B] bool}."""
        B = st.prefix.B
        c = self.ctx
        hb = self._heads_buffers(B, k, d)
        need = [x != 1 for x in codes]
        c.cdsl_rollout_with(st.prefix, st.beams, k, d, 0, hb["look"])
        c.cdsl_reward_keywords(st.prefix, hb["look"], k, d, keywords, normalize=normalize, reward=hb["reward"])
        c.cdsl_select_first(hb["reward"], first_at, hb["beam"])
        table = {"lookaheads": hb["look"].clone(), "reward": hb["reward"].clone(), "beam": hb["beam"].clone(),
                 "tokens": [-1] * B}
        pending = [False] * B
        if b >= 2:
            r0 = hb["reward"][:, 0].cpu().tolist()
            pending = [codes[i] == 2 and not (r0[i] >= r_t) for i in range(B)]
        final = [need[i] and not pending[i] for i in range(B)]
        if any(final):
            toks = c.cdsl_commit_heads(st.prefix, hb["look"], hb["beam"], k, d, final, st.beams, st.head_lp)
            for i in range(B):
                if final[i]:
                    st.emitted[i].append(toks[i])
                    table["tokens"][i] = toks[i]
        rounds = []
        if not any(pending):
            return table, rounds
        # Step-2's choice for the prompts still in Step-1, should every round miss
        s2_tok = torch.gather(table["lookaheads"][:, :, 0], 1, table["beam"].long().view(B, 1)).view(B).contiguous()
        tentative = [[] for _ in range(B)]
        look1 = torch.zeros(B, 1, d + 1, dtype=torch.int32, device=st.beams.device)
        rew1 = torch.zeros(B, 1, device=st.beams.device)
        zeros = torch.zeros(B, dtype=torch.int32, device=st.beams.device)
        for _ in range(2, b + 1):
            if not any(pending):
                break
            # take M_p's greedy token tentatively; its next greedy token leads the round
            xt = st.beams[:, 0].contiguous()
            got = c.cdsl_append(st.prefix, xt, pending, st.beams, st.head_lp)
            for i in range(B):
                if pending[i]:
                    tentative[i].append(got[i])
            c.cdsl_rollout_with(st.prefix, st.beams[:, :1].contiguous(), 1, d, 0, look1)
            c.cdsl_reward_keywords(st.prefix, look1, 1, d, keywords, normalize=normalize, reward=rew1)
            rr = rew1[:, 0].cpu().tolist()
            ok = [pending[i] and rr[i] >= r_t for i in range(B)]
            rounds.append({"X": look1[:, 0, 0].cpu().tolist(), "lookaheads": look1.clone(), "reward": rr,
                           "active": list(pending)})
            if any(ok):
                toks = c.cdsl_commit_heads(st.prefix, look1, zeros, 1, d, ok, st.beams, st.head_lp)
                for i in range(B):
                    if ok[i]:
                        st.emitted[i].extend(tentative[i] + [toks[i]])
                        table["tokens"][i] = toks[i]
            pending = [pending[i] and not ok[i] for i in range(B)]
        if any(pending):
            c.cdsl_withdraw(st.prefix, [len(tentative[i]) if pending[i] else 0 for i in range(B)])
            toks = c.cdsl_append(st.prefix, s2_tok, pending, st.beams, st.head_lp)
            for i in range(B):
                if pending[i]:
                    st.emitted[i].append(toks[i])
                    table["tokens"][i] = toks[i]
        return table, rounds

    def close(self):
        self.ctx.close()
