"""The numeric contract measured at the full-size targets: the 7B target
with a 256-token prompt and the GQA-8 long-context target (V = 128256) with a
2048-token prompt.  Same emulation as the CPU measurement on the small
target (bf16 activations, hi + lo activations, bf16 keys and values with
fp32 activations, each against float64), run in torch float64 on the GPU
because the CPU would take minutes per forward at these sizes.

Measured (max |dlogprob| over seeded tokens at every prompt position):
  7B, 256 tokens:      bf16 1.5e-1   kv16 8.8e-2   hilo 2.3e-4
  long, 2048 tokens:   bf16 2.6e-1   kv16 1.1e-1   hilo 2.8e-4
so a bf16 KV cache misses the 2e-2 log-prob bar by four to five times at
both sizes (at the long context its median error is already 1.8e-2), and the
hi + lo planes meet it with about two orders of magnitude to spare.

Measurement, not a parity test: no library code runs here.
"""
import numpy as np
import pytest
import torch

import cdsl_inputs as ci

pytestmark = pytest.mark.gpu

BAR = 2e-2
F = torch.float64


def _bf(x):
    return x.to(torch.bfloat16).to(F)


def _hilo(x):
    h = _bf(x)
    return h + _bf(x - h)


def _rms(x, eps):
    return x / torch.sqrt((x * x).mean(-1, keepdim=True) + eps)


def _rope(x, pos, theta):
    """Rotate-half rotary embedding; x [T, heads, hd]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-(torch.arange(half, dtype=F, device=x.device) * 2.0) / hd)
    ang = pos.to(F)[:, None] * inv[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], -1)


def _contract_errors(name):
    wl = ci.workload(name)
    sh = wl.target
    dev = "cuda"
    w = ci.model_weights(sh, wl.seed, 1, wl.dtype)
    L = wl.prompt_len
    toks = ci.prompts(wl.seed, 1, L, sh.vocab)[0]
    H, Hkv, hd = sh.n_heads, sh.n_kv_heads, sh.head_dim
    G = H // Hkv
    ident = lambda x: x
    variants = {"exact": (ident, ident), "bf16": (_bf, ident), "hilo": (_hilo, ident), "kv16": (ident, _bf)}
    pos = torch.arange(L, device=dev)
    emb = torch.from_numpy(w["tok_emb"][toks]).to(dev).to(F)
    h = {v: emb.clone() for v in variants}
    visible = torch.ones(L, L, dtype=torch.bool, device=dev).tril()
    for lw in w["layers"]:
        W = {nm: torch.from_numpy(lw[nm]).to(dev).to(F) for nm in ci.LAYER_MATS}
        for v, (act, kv) in variants.items():
            u = act(_rms(h[v], sh.rms_eps))
            q = _rope((u @ W["wq"].T).reshape(L, H, hd), pos, sh.rope_theta)
            k = _rope((u @ W["wk"].T).reshape(L, Hkv, hd), pos, sh.rope_theta)
            vv = (u @ W["wv"].T).reshape(L, Hkv, hd)
            q, k, vv = act(q), kv(act(k)), kv(act(vv))
            kt = k.repeat_interleave(G, dim=1).permute(1, 2, 0).contiguous()        # [H, hd, L]
            sc = torch.bmm(q.permute(1, 0, 2).contiguous(), kt) / hd ** 0.5         # [H, L, L]
            sc = sc.masked_fill(~visible, float("-inf"))
            p = torch.exp(sc - sc.max(-1, keepdim=True).values)
            vh = vv.repeat_interleave(G, dim=1).permute(1, 0, 2).contiguous()       # [H, L, hd]
            o = (torch.bmm(act(p), vh) / p.sum(-1, keepdim=True)).permute(1, 0, 2).reshape(L, H * hd)
            h[v] = h[v] + act(o) @ W["wo"].T
            u = act(_rms(h[v], sh.rms_eps))
            g = u @ W["w_gate"].T
            h[v] = h[v] + act(g / (1 + torch.exp(-g)) * (u @ W["w_up"].T)) @ W["w_down"].T
        del W
    lm = torch.from_numpy(w["lm_head"]).to(dev).to(F)
    pick = torch.from_numpy(np.random.default_rng([wl.seed, 77]).integers(0, sh.vocab, L)).to(dev)
    rows = torch.arange(L, device=dev)
    lp = {v: torch.log_softmax(act(_rms(h[v], sh.rms_eps)) @ lm.T, -1)[rows, pick]
          for v, (act, _) in variants.items()}
    err = {v: float((lp[v] - lp["exact"]).abs().max()) for v in ("bf16", "hilo", "kv16")}
    print(name, "max |dlogprob| vs float64:", err)
    return err


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["7b1b", "long"])
def test_bf16_kv_misses_the_bar_at_full_size(name):
    err = _contract_errors(name)
    assert err["bf16"] > BAR and err["kv16"] > BAR
    assert err["hilo"] < BAR / 50
