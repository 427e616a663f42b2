"""The q/k/v projection's rotary epilogue against the separate rotary +
KV-write kernel.  Both apply the same arithmetic to the same product, so
with the same inputs every output of a run is bitwise the same.  The
epilogue applies where the projection runs on the dense kernel without a K
split: the prompt prefill of both models (head sizes 128 and 64, prefix
positions) and, with 64 prompts of the `small` workload (1600 rows), the
verification (beam suffix slots, the tree of k beams)."""
import numpy as np
import pytest
import torch

from cdsl_harness import make_engine, make_setup

pytestmark = pytest.mark.gpu

B = 64


def _run(s, eng, steps):
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


def test_rotary_epilogue_matches_the_rotary_kernel(monkeypatch):
    s = make_setup("small", B=B)
    eng = make_engine(s, B=B, max_steps=3)
    try:
        monkeypatch.setenv("CDSL_UNFUSED_ROPE", "1")
        ref, em_ref, len_ref = _run(s, eng, 2)
        monkeypatch.delenv("CDSL_UNFUSED_ROPE")
        got, em, lens = _run(s, eng, 2)
        for (name, a), (_, b) in zip(ref, got):
            assert a.dtype == b.dtype and a.shape == b.shape, name
            same = a.view(torch.int32) == b.view(torch.int32) if a.dtype == torch.float32 else a == b
            assert bool(same.all()), (name, int((~same).sum()))
        assert em == em_ref
        assert lens == len_ref
        # the comparison is not vacuous: the lookaheads differ between prompts
        la = ref[2][1].cpu().numpy()
        assert len({la[b].tobytes() for b in range(B)}) > 1
    finally:
        eng.close()
