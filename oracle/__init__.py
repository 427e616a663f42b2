"""CPU oracle for the CDSL lookahead step (float64 numpy).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the product path.  It
shares no code with the HIP library; the only module both sides use is the
seeded input generator ``cdsl_inputs``.

Pins (tests marked ``not gpu``): the decoder against an independent library
implementation of the same architecture; incremental = full recompute =
tree-parallel verification; greedy rollout = argmax of a full forward; k = 1
reduces to plain greedy decoding of the target; draft = target accepts every
lookahead token; beam selection against brute-force enumeration on a tiny
vocabulary; the paper's worked reward value (2 of 5 concepts -> 0.4); the
lookahead-heuristic baselines and the Alg. 1 controller against greedy
decoding of the target and against full recomputation; speculative
sampling's acceptance rate and residual draw against their closed forms, and
the pair against the theorem that it reproduces the target distribution.
"""
from .decoder import Decoder, KVCache, ForwardOut, rms_norm, rope  # noqa: F401
from .cdsl import (  # noqa: F401
    PromptState, StepResult, prefill, step, rollout, verify, commit, beam_heads,
    log_softmax, argmax_lowest, topk_ids, top2_margin, leading_matches,
    keyword_hits, keyword_coverage, select_beam, reward_for,
    verify_rows_tree, verify_rows_per_beam,
    keyword_reward, argmax_first, lookahead_heads, cdlh_step, controller_step, HeadStep, ControllerStep,
    draft_from_prefix, verify_from_prefix, Step1Try,
    soft_accept_count, soft_accept_margins, residual_sample, residual_interval, SoftResult,
)
