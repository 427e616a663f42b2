"""Failure handling and resume on the GPU, through the C ABI: token ids
outside the vocabulary, a commit that fails validation (the prefix and its
generated tokens stay as they were), destroyed contexts and freed prefix
handles, limits beyond device memory, misaligned borrowed weights, a run
resumed by re-prefilling its tokens, and two live prefix handles.  Every error is forced from the host; no kernel faults."""
import math

import numpy as np
import pytest
import torch

import cdsl_inputs as ci
import oracle
from cdsl_harness import make_engine, make_setup

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    s = make_setup("tiny")
    make_engine(s, B=3, max_steps=12)
    yield s
    s.engine.close()


def _bad_code(fn):
    from paper_2412_10418_amd.binding import CDSLError
    with pytest.raises(CDSLError) as e:
        fn()
    return e.value.code


def test_prompt_token_outside_the_vocabulary(tiny):
    from paper_2412_10418_amd.binding import CDSL_EINVAL
    eng = tiny.engine
    p = torch.from_numpy(tiny.prompts(2)).cuda()
    p[1, 5] = tiny.wl.target.vocab          # one past the last id
    assert _bad_code(lambda: eng.start(p)) == CDSL_EINVAL
    p[1, 5] = -3
    assert _bad_code(lambda: eng.start(p)) == CDSL_EINVAL
    # no handle was left behind: the one allowed prefix can still be made
    st = eng.start(torch.from_numpy(tiny.prompts(2)).cuda())
    st.prefix.free()


def test_lookahead_token_outside_the_vocabulary_fails_the_commit(tiny):
    """A verification fed an id >= V returns (it is asynchronous) with NaN
    at that gathered log-prob; the commit after it reports EINVAL and the
    prefix is unchanged, so the step can be redone."""
    from paper_2412_10418_amd.binding import CDSL_EINVAL
    eng, wl = tiny.engine, tiny.wl
    k, d = wl.k, wl.d
    st = eng.start(torch.from_numpy(tiny.prompts(2)).cuda())
    kw = torch.from_numpy(tiny.kws[:2]).cuda()
    bf = eng.buffers(2, k, d)
    c = eng.ctx
    c.cdsl_rollout(st.prefix, st.beams, k, d, bf.lookaheads)
    bad = bf.lookaheads.clone()
    bad[1, 2, d] = wl.target.vocab + 7      # only gathered (x_d is never fed)
    c.cdsl_verify(st.prefix, bad, k, d, st.head_lp, out=bf.verify)
    assert torch.isnan(bf.verify["logprobs"][1, 2, d - 1]).item()
    c.cdsl_reward_keywords(st.prefix, bad, k, d, kw, normalize=False, reward=bf.reward)
    c.cdsl_select(bf.verify["scores"], bf.reward, 0.0, bf.beam)
    lens = st.prefix.lengths()
    assert _bad_code(lambda: c.cdsl_commit(st.prefix, bad, bf.beam, bf.verify["n_accept"],
                                           bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], k, d)) == CDSL_EINVAL
    assert st.prefix.lengths() == lens
    # the flag was cleared: the same step with valid ids commits
    bf2 = eng.step(st, keywords=kw)
    assert st.prefix.lengths() == [l + len(e) for l, e in zip(lens, st.emitted)]
    st.prefix.free()


def test_failed_commit_changes_no_prompt(tiny):
    """B = 2 with a NaN score for prompt 1: the commit reports EINVAL before
    prompt 0's tokens reach the generated sequence.  Checked through the
    keyword reward, which reads the generated tokens: a keyword equal to
    prompt 0's selected head stays absent."""
    from paper_2412_10418_amd.binding import CDSL_EINVAL
    eng, wl = tiny.engine, tiny.wl
    k, d = wl.k, wl.d
    st = eng.start(torch.from_numpy(tiny.prompts(2)).cuda())
    bf = eng.buffers(2, k, d)
    c = eng.ctx
    c.cdsl_rollout(st.prefix, st.beams, k, d, bf.lookaheads)
    c.cdsl_verify(st.prefix, bf.lookaheads, k, d, st.head_lp, out=bf.verify)
    bf.verify["scores"][1, 0] = float("nan")
    zero = torch.zeros(2, k, device="cuda")
    c.cdsl_select(bf.verify["scores"], zero, 1.0, bf.beam)
    beam = bf.beam.cpu().tolist()
    assert beam[0] >= 0 and beam[1] == -1
    head0 = int(bf.lookaheads[0, beam[0], 0])
    nb_before = st.beams.clone()
    lens = st.prefix.lengths()
    assert _bad_code(lambda: c.cdsl_commit(st.prefix, bf.lookaheads, bf.beam, bf.verify["n_accept"],
                                           bf.verify["row_topk_ids"], bf.verify["row_topk_lp"], k, d,
                                           st.beams, st.head_lp)) == CDSL_EINVAL
    torch.cuda.synchronize()
    assert st.prefix.lengths() == lens
    assert torch.equal(st.beams, nb_before)
    # a window without that token: the reward sees no keyword unless the
    # failed commit had appended it to the generated tokens
    other = (head0 + 1) % wl.target.vocab
    look = torch.full((2, k, d + 1), other, dtype=torch.int32, device="cuda")
    kw = torch.tensor([[head0], [head0]], dtype=torch.int32, device="cuda")
    r = c.cdsl_reward_keywords(st.prefix, look, k, d, kw, normalize=False)
    assert r.abs().sum().item() == 0.0
    st.prefix.free()


def test_destroyed_context_and_freed_prefix_are_refused(tiny):
    from paper_2412_10418_amd import binding as bd
    from paper_2412_10418_amd.engine import Engine
    eng = tiny.engine
    st = eng.start(torch.from_numpy(tiny.prompts(1)).cuda())
    handle = st.prefix.handle
    st.prefix.free()
    L = bd.lib()
    out = (bd.C.c_int32 * 1)()
    assert L.cdsl_prefix_lengths(eng.ctx.handle, handle, out) == bd.CDSL_ESTATE
    assert L.cdsl_free_prefix(eng.ctx.handle, handle) == bd.CDSL_ESTATE
    assert L.cdsl_rollout(eng.ctx.handle, handle, st.beams.data_ptr(), tiny.wl.k, tiny.wl.d,
                          st.beams.data_ptr()) == bd.CDSL_ESTATE
    # a second context, destroyed: every call refuses it, a second destroy too
    dwd, twd = Engine.upload(tiny.wl, tiny.draft_np, tiny.target_np)
    e2 = Engine(tiny.wl, dwd, twd, max_steps=2, max_batch=1)
    h = e2.ctx.handle
    e2.close()
    assert L.cdsl_destroy(h) == bd.CDSL_ESTATE
    assert L.cdsl_prefix_lengths(h, handle, out) == bd.CDSL_ESTATE
    assert L.cdsl_select(h, st.head_lp.data_ptr(), st.head_lp.data_ptr(), 1.0, 1, tiny.wl.k,
                         st.beams.data_ptr()) == bd.CDSL_ESTATE
    assert b"destroyed" in L.cdsl_last_error(h)


def test_limits_beyond_device_memory(tiny):
    """A KV pool larger than the free device memory is refused at init
    (ENOMEM) before it is allocated."""
    from paper_2412_10418_amd import binding as bd
    from paper_2412_10418_amd.engine import Engine
    dwd, twd = Engine.upload(tiny.wl, tiny.draft_np, tiny.target_np)
    with pytest.raises(bd.CDSLError) as e:
        Engine(tiny.wl, dwd, twd, max_steps=2, max_batch=4096, max_prompt=65536)
    assert e.value.code == bd.CDSL_ENOMEM
    assert "exceeds free device memory" in str(e.value)


def test_borrowed_weights_must_be_aligned(tiny):
    """The embedding, LM head, norm gains, wo and w_down are read in place
    with 16-byte loads: a pointer off that alignment is refused at init
    (EINVAL) before any kernel reads it."""
    from paper_2412_10418_amd import binding as bd
    from paper_2412_10418_amd.engine import Engine
    dwd, twd = Engine.upload(tiny.wl, tiny.draft_np, tiny.target_np)
    emb = twd["tok_emb"]
    shifted = torch.empty(emb.numel() + 1, dtype=emb.dtype, device=emb.device)[1:].view(emb.shape)
    shifted.copy_(emb)
    assert shifted.data_ptr() % 16 != 0
    twd = dict(twd, tok_emb=shifted)
    with pytest.raises(bd.CDSLError) as e:
        Engine(tiny.wl, dwd, twd, max_steps=2, max_batch=2)
    assert e.value.code == bd.CDSL_EINVAL
    assert "aligned" in str(e.value)


def test_resume_by_reprefill_matches_uninterrupted(tiny):
    """8 steps equal 4 steps, a prefill of prompt + the 4 steps' tokens as a
    new prompt, and 4 more steps (the fp32 workload, 2 prompts, each resumed
    on its own since the resumed prompts differ in length).  Selection by
    the scores alone (alpha = 0): the keyword reward reads the generated
    tokens, which a re-prefill turns into prompt tokens."""
    from paper_2412_10418_amd.engine import Engine
    wl = tiny.wl
    B = 2
    dwd, twd = Engine.upload(wl, tiny.draft_np, tiny.target_np)
    eng = Engine(wl, dwd, twd, max_steps=12, max_batch=B, max_prompt=wl.prompt_len + 8 * (wl.d + 1))
    kw = torch.from_numpy(tiny.kws[:B]).cuda()
    prompts = tiny.prompts(B)
    runs = {}
    for n in (8, 4):
        st = eng.start(torch.from_numpy(prompts).cuda())
        for _ in range(n):
            eng.step(st, keywords=kw, alpha=0.0)
        runs[n] = [list(e) for e in st.emitted]
        st.prefix.free()
    for b in range(B):
        toks = np.concatenate([prompts[b], np.array(runs[4][b], np.int32)])[None]
        st = eng.start(torch.from_numpy(np.ascontiguousarray(toks)).cuda())
        for _ in range(4):
            eng.step(st, keywords=kw[b:b + 1], alpha=0.0)
        print(f"prompt {b}: {len(runs[4][b])} + {len(st.emitted[0])} tokens resumed, {len(runs[8][b])} straight")
        assert runs[4][b] + st.emitted[0] == runs[8][b]
        st.prefix.free()
    eng.close()


def test_second_prefix_leaves_the_first_unchanged(tiny):
    """Two live prefix handles on one context: prompt set A steps, set B is
    prefilled right after A's commit (the shared pinned block-table buffer
    is refilled for B while A's table upload was queued), then both step in
    turn.  A's tokens and log-probs equal a run of A alone, bitwise, and B's
    equal a run of B alone."""
    from paper_2412_10418_amd.engine import Engine
    wl = tiny.wl
    B = 2
    dwd, twd = Engine.upload(wl, tiny.draft_np, tiny.target_np)
    eng = Engine(wl, dwd, twd, max_steps=8, max_batch=B, max_prefixes=2)
    kw = torch.from_numpy(tiny.kws[:B]).cuda()
    pa = torch.from_numpy(tiny.prompts(B)).cuda()
    pb = torch.from_numpy(tiny.prompts(B, first=B)).cuda()

    def run(prompts, n):
        st = eng.start(prompts)
        lps = []
        for _ in range(n):
            bf = eng.step(st, keywords=kw)
            lps.append(bf.verify["logprobs"].cpu().clone())
        out = ([list(e) for e in st.emitted], lps)
        st.prefix.free()
        return out

    alone_a, alone_b = run(pa, 4), run(pb, 3)
    sa = eng.start(pa)
    lpa, lpb = [], []
    bf = eng.step(sa, keywords=kw)
    lpa.append(bf.verify["logprobs"].cpu().clone())
    sb = eng.start(pb)
    for t in range(3):
        bf = eng.step(sa, keywords=kw)
        lpa.append(bf.verify["logprobs"].cpu().clone())
        bf = eng.step(sb, keywords=kw)
        lpb.append(bf.verify["logprobs"].cpu().clone())
    assert [list(e) for e in sa.emitted] == alone_a[0]
    assert [list(e) for e in sb.emitted] == alone_b[0]
    assert all(torch.equal(x, y) for x, y in zip(lpa, alone_a[1]))
    assert all(torch.equal(x, y) for x, y in zip(lpb, alone_b[1]))
    sa.prefix.free()
    sb.prefix.free()
    eng.close()
