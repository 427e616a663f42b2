"""End-to-end parity on shapes the named small workloads do not reach:
grouped-query attention in bf16 (4 query heads per KV head, head dims 64
and 128), lookaheads that span two suffix blocks, ragged prompt lengths,
and the full-size 7B / 1B pair (sampled prompts of the whole batch)."""
import numpy as np
import pytest
import torch

import cdsl_inputs as ci
from cdsl_harness import assert_full_or_tie, make_engine, make_setup, run_and_compare

pytestmark = pytest.mark.gpu

# draft head_dim 64, target head_dim 128, both with 4 query heads per KV head
GQA_DRAFT = ci.ModelShape(2, 512, 8, 2, 1024, 4096)
GQA_TARGET = ci.ModelShape(3, 1024, 8, 2, 2048, 4096)


def _report(reps, steps):
    for b, r in reps.items():
        print(f"prompt {b}: {r.steps_compared} steps, max |dlp| {r.max_lp_err:.2e}, stop: {r.stopped or '-'}")
    assert_full_or_tie(reps, steps)


@pytest.mark.parametrize("k,d,L", [(4, 6, 40), (3, 18, 37)])
def test_gqa_bf16_steps_match_oracle(k, d, L):
    """bf16 GQA pair; d=18 puts every beam's lookahead rows in two suffix
    blocks; prompt lengths 40 and 37 leave ragged last prefix blocks."""
    s = make_setup("small", draft=GQA_DRAFT, target=GQA_TARGET, batch=4, prompt_len=L, k=k, d=d)
    make_engine(s, B=4, max_steps=6, k=k, d=d)
    try:
        st, reps = run_and_compare(s, B=4, steps=4, check_prompts=[0, 3], k=k, d=d)
        _report(reps, 4)
        st.prefix.free()
    finally:
        s.engine.close()


@pytest.fixture(scope="module")
def full7b():
    s = make_setup("7b1b")
    make_engine(s, B=16, max_steps=4)
    yield s
    s.engine.close()


@pytest.mark.timeout(600)
def test_7b1b_full_size_sampled_parity(full7b):
    """The 7B / 1B pair at its full batch (16 prompts x 256 tokens, k=5,
    d=10) in the launch configuration the benchmark times; prompts 0 and 11
    of the batch are compared with the oracle for two steps."""
    st, reps = run_and_compare(full7b, B=16, steps=2, check_prompts=[0, 11])
    _report(reps, 2)
    st.prefix.free()


@pytest.mark.timeout(600)
def test_7b1b_full_size_soft_rejection(full7b):
    """The same configuration with speculative sampling's soft rejection
    (kept draft logits of 16 x 5 x 10 rows over 32000 tokens, the residual
    draw): prompts 0 and 11, two steps."""
    st, reps = run_and_compare(full7b, B=16, steps=2, check_prompts=[0, 11], soft=True)
    _report(reps, 2)
    st.prefix.free()
