"""One CDSL lookahead step on the GPU, driven through the C ABI.

A step is rollout -> verify -> reward -> select -> commit on the context
stream, with the step's device buffers allocated once per (B, k, d) so the
steady-state loop allocates nothing.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import torch

from .binding import Context, Prefix, upload_weights


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
                 max_batch: Optional[int] = None, k: Optional[int] = None, d: Optional[int] = None):
        wl = workload
        self.wl = wl
        self.k = k or wl.k
        self.d = d or wl.d
        self.device = device
        B = max_batch or wl.batch
        limits = dict(max_batch=B, max_prompt=wl.prompt_len,
                      max_ctx=wl.prompt_len + max_steps * (self.d + 1) + 2,
                      max_k=self.k, max_d=self.d, max_prefixes=1)
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

    def step(self, st: DecodeState, keywords: Optional[torch.Tensor] = None,
             reward_w: Optional[torch.Tensor] = None, alpha: Optional[float] = None,
             k: Optional[int] = None, d: Optional[int] = None, marks: Optional[list] = None) -> StepBuffers:
        """One lookahead step.  Updates ``st`` in place; returns the step's
        buffers (valid until the next step with the same shape).  With a list
        ``marks``, timing events are appended before the rollout, after it,
        after the verification and after the commit."""
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
        mark()
        c.cdsl_rollout(st.prefix, st.beams, k, d, bf.lookaheads)
        mark()
        c.cdsl_verify(st.prefix, bf.lookaheads, k, d, st.head_lp, out=bf.verify)
        mark()
        kind = self.wl.reward
        if kind == "linear":
            c.cdsl_reward_linear(bf.verify["hidden"], reward_w, bf.reward)
        else:
            c.cdsl_reward_keywords(st.prefix, bf.lookaheads, k, d, keywords,
                                   normalize=(kind == "keyword_coverage"), reward=bf.reward)
        c.cdsl_select(bf.verify["scores"], bf.reward, alpha, bf.beam)
        # commit writes the next heads into separate buffers, then they swap
        em, nb, nlp = c.cdsl_commit(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                                    bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], k, d,
                                    bf.next_beams, bf.next_head_lp)
        mark()
        for b in range(B):
            st.emitted[b].extend(em[b])
        st.beams, bf.next_beams = bf.next_beams, st.beams
        st.head_lp, bf.next_head_lp = bf.next_head_lp, st.head_lp
        self._last_emitted = em
        return bf

    def close(self):
        self.ctx.close()
