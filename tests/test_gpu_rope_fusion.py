"""The q/k/v projection's rotary epilogue against the separate rotary +
KV-write kernel.  Both apply the same arithmetic to the same product, so
with the same inputs every output of a run is bitwise the same.  The
epilogue applies where the projection runs on the dense kernel without a K
split: the prompt prefill of both models (head sizes 128 and 64, prefix
positions) and, with 64 prompts of the `small` workload (1600 rows), the
verification (beam suffix slots, the tree of k beams).  A grouped-query
draft (8 query heads, 2 KV heads of 64 dims) puts key and value heads in
one output tile of its prefill."""
import numpy as np
import pytest
import torch

import cdsl_inputs as ci
from cdsl_harness import make_engine, make_setup

pytestmark = pytest.mark.gpu

B = 64
GQA_DRAFT = ci.ModelShape(2, 512, 8, 2, 1024, 4096)
GQA_TARGET = ci.ModelShape(3, 1024, 8, 2, 2048, 4096)


def _run(s, eng, steps, B=B):
    prompts = torch.from_numpy(s.prompts(B)).cuda()
    kws = torch.from_numpy(s.kws[:B]).cuda()
    st = eng.start(prompts)
    outs = [("heads", st.beams.clone()), ("head_lp", st.head_lp.clone())]
    for t in range(steps):
        bf = eng.step(st, keywords=kws)
        outs.append((f"lookaheads {t}", bf.lookaheads.clone()))
        outs += [(f"{n} {t}", v.clone()) for n, v in bf.verify.items() if v is not None]
        outs += [(f"reward {t}", bf.reward.clone()), (f"beam {t}", bf.beam.clone())]
        outs += [(f"next heads {t}", st.beams.clone()), (f"next head_lp {t}", st.head_lp.clone())]
    emitted = [list(e) for e in st.emitted]
    lens = st.prefix.lengths()
    st.prefix.free()
    return outs, emitted, lens


@pytest.mark.parametrize("case", ["small", "gqa"])
def test_rotary_epilogue_matches_the_rotary_kernel(monkeypatch, case):
    if case == "small":
        nb, s = B, make_setup("small", B=B)
    else:
        # 32 prompts x 256 tokens: the draft's q/k/v output tile 2 holds
        # its 2 key heads and its 2 value heads
        nb = 32
        s = make_setup("small", draft=GQA_DRAFT, target=GQA_TARGET, batch=nb, prompt_len=256, B=nb)
    eng = make_engine(s, B=nb, max_steps=3)
    try:
        monkeypatch.setenv("CDSL_UNFUSED_ROPE", "1")
        ref, em_ref, len_ref = _run(s, eng, 2, nb)
        monkeypatch.delenv("CDSL_UNFUSED_ROPE")
        got, em, lens = _run(s, eng, 2, nb)
        for (name, a), (_, b) in zip(ref, got):
            assert a.dtype == b.dtype and a.shape == b.shape, name
            same = a.view(torch.int32) == b.view(torch.int32) if a.dtype == torch.float32 else a == b
            assert bool(same.all()), (name, int((~same).sum()))
        assert em == em_ref
        assert lens == len_ref
        # the comparison is not vacuous: the lookaheads differ between prompts
        la = ref[2][1].cpu().numpy()
        assert len({la[b].tobytes() for b in range(nb)}) > 1
    finally:
        eng.close()
