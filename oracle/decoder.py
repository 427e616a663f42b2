"""CPU oracle, part 1: a plain Llama-style decoder in float64.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP path.

The paper fixes no architecture (its models are OPT / Bloomz / Qwen, Sec. 4.2).
The workloads are "Llama-style" decoders, read as: pre-norm RMSNorm
(x / sqrt(mean(x^2) + eps) * g), rotary position embedding with the
rotate-half pairing (i, i + hd/2) and frequencies theta^(-2i/hd) at 0-based
absolute positions, grouped-query attention (query head h reads KV head
floor(h / (H / Hkv))), softmax(q k^T / sqrt(hd)) v, SwiGLU MLP
(silu(u Wg^T) * (u Wu^T)) Wd^T, no biases, untied embedding and LM head.

Everything is computed in float64 with no blocking or fusion; the KV cache is a
plain list of per-layer arrays.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

F64 = np.float64


def _f64(a):
    return np.asarray(a, dtype=F64)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * _f64(g)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotary embedding, rotate-half form.  x: [T, n_heads, hd]; pos: [T]."""
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = theta ** (-(np.arange(half, dtype=F64) * 2.0) / hd)
    ang = _f64(pos)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


@dataclass
class KVCache:
    """Per-layer keys/values, each [P, Hkv, hd] float64 (post-RoPE keys)."""
    k: List[np.ndarray]
    v: List[np.ndarray]

    @staticmethod
    def empty(n_layers: int, n_kv: int, hd: int) -> "KVCache":
        return KVCache([np.zeros((0, n_kv, hd)) for _ in range(n_layers)],
                       [np.zeros((0, n_kv, hd)) for _ in range(n_layers)])

    @property
    def length(self) -> int:
        return self.k[0].shape[0]

    def copy(self) -> "KVCache":
        return KVCache([a.copy() for a in self.k], [a.copy() for a in self.v])

    def extended(self, new_k: List[np.ndarray], new_v: List[np.ndarray]) -> "KVCache":
        return KVCache([np.concatenate([a, b]) for a, b in zip(self.k, new_k)],
                       [np.concatenate([a, b]) for a, b in zip(self.v, new_v)])


@dataclass
class ForwardOut:
    logits: np.ndarray        # [T, V]
    hidden: np.ndarray        # [T, D]  final-normed hidden state
    new_k: List[np.ndarray]   # per layer [T, Hkv, hd]
    new_v: List[np.ndarray]


class Decoder:
    """A decoder over given weights (any float dtype; computed in float64)."""

    def __init__(self, shape, weights):
        self.shape = shape
        self.w = weights
        self._f64 = {}

    def mat(self, layer, name):
        """Weight as float64, converted once and kept."""
        key = (layer, name)
        if key not in self._f64:
            src = self.w[name] if layer is None else self.w["layers"][layer][name]
            self._f64[key] = _f64(src)
        return self._f64[key]

    @property
    def n_layers(self):
        return self.shape.n_layers

    def empty_cache(self) -> KVCache:
        s = self.shape
        return KVCache.empty(s.n_layers, s.n_kv_heads, s.head_dim)

    def forward(self, tokens, positions, cache: KVCache, allowed: np.ndarray) -> ForwardOut:
        """Run the new tokens against ``cache`` plus themselves.

        allowed[t, c] says whether new row t may attend to column c, where
        columns 0..P-1 are the cached positions and P..P+T-1 the new rows.
        """
        s = self.shape
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.asarray(positions, dtype=np.int64)
        T = tokens.shape[0]
        H, Hkv, hd = s.n_heads, s.n_kv_heads, s.head_dim
        G = H // Hkv
        P = cache.length
        assert allowed.shape == (T, P + T)
        h = _f64(self.w["tok_emb"][tokens])
        new_k, new_v = [], []
        for l, lw in enumerate(self.w["layers"]):
            u = rms_norm(h, lw["attn_norm"], s.rms_eps)
            q = (u @ self.mat(l, "wq").T).reshape(T, H, hd)
            k = (u @ self.mat(l, "wk").T).reshape(T, Hkv, hd)
            v = (u @ self.mat(l, "wv").T).reshape(T, Hkv, hd)
            q = rope(q, positions, s.rope_theta)
            k = rope(k, positions, s.rope_theta)
            new_k.append(k)
            new_v.append(v)
            K = np.concatenate([cache.k[l], k])     # [P+T, Hkv, hd]
            V = np.concatenate([cache.v[l], v])
            o = np.empty((T, H, hd))
            for hq in range(H):
                kv = hq // G
                sc = (q[:, hq, :] @ K[:, kv, :].T) / np.sqrt(hd)
                sc = np.where(allowed, sc, -np.inf)
                o[:, hq, :] = softmax_rows(sc) @ V[:, kv, :]
            h = h + o.reshape(T, H * hd) @ self.mat(l, "wo").T
            u = rms_norm(h, lw["mlp_norm"], s.rms_eps)
            a = silu(u @ self.mat(l, "w_gate").T) * (u @ self.mat(l, "w_up").T)
            h = h + a @ self.mat(l, "w_down").T
        hf = rms_norm(h, self.w["final_norm"], s.rms_eps)
        logits = hf @ self.mat(None, "lm_head").T
        return ForwardOut(logits, hf, new_k, new_v)

    # -- convenience wrappers -------------------------------------------------
    def full(self, tokens) -> ForwardOut:
        """Full recompute of a sequence from scratch with a causal mask."""
        T = len(tokens)
        allowed = np.tril(np.ones((T, T), dtype=bool))
        return self.forward(tokens, np.arange(T), self.empty_cache(), allowed)

    def extend(self, cache: KVCache, tokens) -> tuple:
        """Append tokens after ``cache`` (causal); returns (out, new cache)."""
        P, T = cache.length, len(tokens)
        allowed = np.concatenate([np.ones((T, P), bool), np.tril(np.ones((T, T), bool))], 1)
        out = self.forward(tokens, P + np.arange(T), cache, allowed)
        return out, cache.extended(out.new_k, out.new_v)
