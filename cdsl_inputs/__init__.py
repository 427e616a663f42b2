"""Seeded synthetic inputs for the CDSL lookahead step.

This module is shared by the CPU oracle and the GPU path and holds none of the
method's arithmetic: it only defines the workload shapes and draws the random
inputs (weights, prompts, keyword sets, the reward head) from fixed seeds.

The paper evaluates on CommonGen and HH-RLHF with OPT / Bloomz / Qwen models
(Sec. 4.1-4.2).  None of those datasets or checkpoints are used here; seeded,
random-init Llama-style decoders and uniform-random prompts of the stated
shapes stand in for them.

Recipe (every draw is reproducible from the seed alone):

* Every weight matrix (token embedding, q/k/v/o, gate/up/down, lm_head) is
  N(0, 0.02^2).  Tensor ``tau`` of model ``model_id`` (0 = draft,
  1 = target) is flattened and drawn in chunks of 2**20 elements; chunk ``c``
  comes from ``numpy.random.default_rng([seed, model_id, tau, c])
  .standard_normal(n, float32) * 0.02``.  Norm gains are all ones.
* For bf16 workloads every weight is rounded to bf16 (round to nearest even)
  and both sides consume the rounded values.
* Prompt ``b`` is ``default_rng([seed, 1, b]).integers(0, V, L)``: a prompt
  does not depend on the batch size.
* Keyword set of prompt ``b``: ``default_rng([seed, 2, b]).choice(V, n_kw,
  replace=False)``.
* Linear reward head: ``default_rng([seed, 3]).standard_normal(D, float32) *
  0.02`` (fp32, not rounded).
"""
from __future__ import annotations

import concurrent.futures as _cf
import math
import os
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional

import numpy as np

__all__ = [
    "ModelShape", "Workload", "WORKLOADS", "workload",
    "model_weights", "weight_names", "prompts", "keywords", "reward_head",
    "f32_to_bf16_bits", "bf16_bits_to_f32", "round_to_bf16",
]

CHUNK = 1 << 20
LAYER_MATS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


@dataclass(frozen=True)
class ModelShape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    ffn_dim: int
    vocab: int
    rope_theta: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def n_params(self, with_embeddings: bool = True) -> int:
        D, hd = self.d_model, self.head_dim
        per = (self.n_heads * hd * D + 2 * self.n_kv_heads * hd * D + D * self.n_heads * hd
               + 3 * self.ffn_dim * D + 2 * D)
        tot = self.n_layers * per + D + self.vocab * D
        if with_embeddings:
            tot += self.vocab * D
        return tot


@dataclass(frozen=True)
class Workload:
    """One synthetic CDSL workload: a draft/target pair and step shape."""
    name: str
    draft: ModelShape
    target: ModelShape
    dtype: str            # "f32" or "bf16": the arithmetic type of the path
    batch: int
    prompt_len: int
    k: int
    d: int
    steps: int
    reward: str           # "keyword_count" | "keyword_coverage" | "linear"
    n_keywords: int = 0
    alpha: float = 1.0    # weight of the reward in the beam selection score
    seed: int = 0
    description: str = ""

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


_TINY_DRAFT = ModelShape(2, 128, 4, 4, 512, 1024)
_TINY_TARGET = ModelShape(4, 256, 8, 8, 1024, 1024)
_SMALL_DRAFT = ModelShape(12, 1024, 16, 16, 4096, 32000)
_SMALL_TARGET = ModelShape(24, 2048, 16, 16, 5632, 32000)
_DRAFT_1B = ModelShape(16, 2048, 32, 8, 8192, 32000)
_TARGET_7B = ModelShape(32, 4096, 32, 32, 11008, 32000)

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        "tiny", _TINY_DRAFT, _TINY_TARGET, "f32", batch=1, prompt_len=32, k=4, d=4,
        steps=8, reward="keyword_count", n_keywords=3,
        description="fp32 plumbing case: 2L/128 draft, 4L/256 target, V=1024"),
    "small": Workload(
        "small", _SMALL_DRAFT, _SMALL_TARGET, "bf16", batch=8, prompt_len=128, k=5, d=5,
        steps=64, reward="keyword_coverage", n_keywords=4,
        description="bf16 12L/1024 draft, 24L/2048 target, V=32000"),
    "7b1b": Workload(
        "7b1b", _DRAFT_1B, _TARGET_7B, "bf16", batch=16, prompt_len=256, k=5, d=10,
        steps=128, reward="linear",
        description="bf16 1B-shaped draft (GQA 32/8) with a Llama-7B-shaped target, V=32000"),
    "sweep": Workload(
        "sweep", _DRAFT_1B, _TARGET_7B, "bf16", batch=32, prompt_len=512, k=5, d=10,
        steps=8, reward="linear",
        description="7B/1B pair at batch 32, 512-token prompts; k and d are swept"),
    "long": Workload(
        "long", _DRAFT_1B, replace(_TARGET_7B, n_kv_heads=8, vocab=128256),
        "bf16", batch=64, prompt_len=2048, k=8, d=8, steps=4, reward="linear",
        description="7B GQA-8 target, V=128256, 2048-token prompts"),
}
# the long-context draft shares the target's 128256-token vocabulary
WORKLOADS["long"] = WORKLOADS["long"].with_(draft=replace(_DRAFT_1B, vocab=128256))

SWEEP_KD = [(k, d) for k in (2, 5, 10) for d in (2, 5, 10, 20)]


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# ----------------------------------------------------------------------------
# bf16 helpers (bit manipulation only)
# ----------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------
def weight_names(shape: ModelShape) -> List[tuple]:
    """(name, tau, shape) for every random tensor of a model, in tau order."""
    D, hd, H, Hkv, F, V = (shape.d_model, shape.head_dim, shape.n_heads,
                          shape.n_kv_heads, shape.ffn_dim, shape.vocab)
    out = [("tok_emb", 0, (V, D))]
    dims = {"wq": (H * hd, D), "wk": (Hkv * hd, D), "wv": (Hkv * hd, D), "wo": (D, H * hd),
            "w_gate": (F, D), "w_up": (F, D), "w_down": (D, F)}
    for l in range(shape.n_layers):
        for t, nm in enumerate(LAYER_MATS):
            out.append((f"layers.{l}.{nm}", 1 + 7 * l + t, dims[nm]))
    out.append(("lm_head", 1 + 7 * shape.n_layers, (V, D)))
    return out


def _fill_chunk(out_flat: np.ndarray, seed: int, model_id: int, tau: int, c: int, bf16: bool):
    lo = c * CHUNK
    hi = min(lo + CHUNK, out_flat.size)
    g = np.random.default_rng([seed, model_id, tau, c])
    x = g.standard_normal(hi - lo, dtype=np.float32)
    x *= np.float32(0.02)
    if bf16:
        x = round_to_bf16(x)
    out_flat[lo:hi] = x


def _draw(shape_t, seed, model_id, tau, bf16, pool) -> np.ndarray:
    arr = np.empty(int(np.prod(shape_t)), dtype=np.float32)
    nchunk = (arr.size + CHUNK - 1) // CHUNK
    if pool is None or nchunk == 1:
        for c in range(nchunk):
            _fill_chunk(arr, seed, model_id, tau, c, bf16)
    else:
        list(pool.map(lambda c: _fill_chunk(arr, seed, model_id, tau, c, bf16), range(nchunk)))
    return arr.reshape(shape_t)


def model_weights(shape: ModelShape, seed: int, model_id: int, dtype: str,
                  threads: Optional[int] = None) -> Dict[str, object]:
    """All weights of one model as float32 arrays (bf16-rounded for bf16 runs).

    Returns {"tok_emb", "layers": [ {attn_norm, wq, wk, wv, wo, mlp_norm,
    w_gate, w_up, w_down}, ...], "final_norm", "lm_head"}; matrices are
    [out_features, in_features].
    """
    bf16 = dtype == "bf16"
    threads = threads or min(16, os.cpu_count() or 1)
    pool = _cf.ThreadPoolExecutor(threads) if threads > 1 else None
    try:
        flat = {nm: _draw(sh, seed, model_id, tau, bf16, pool)
                for nm, tau, sh in weight_names(shape)}
    finally:
        if pool is not None:
            pool.shutdown()
    D = shape.d_model
    layers = []
    for l in range(shape.n_layers):
        lw = {nm: flat.pop(f"layers.{l}.{nm}") for nm in LAYER_MATS}
        lw["attn_norm"] = np.ones(D, np.float32)
        lw["mlp_norm"] = np.ones(D, np.float32)
        layers.append(lw)
    return {"tok_emb": flat.pop("tok_emb"), "layers": layers,
            "final_norm": np.ones(D, np.float32), "lm_head": flat.pop("lm_head")}


# ----------------------------------------------------------------------------
# prompts, keywords, reward head
# ----------------------------------------------------------------------------
def prompts(seed: int, batch: int, length: int, vocab: int, first: int = 0) -> np.ndarray:
    """int32 [batch, length]; row i is prompt number ``first + i``."""
    out = np.empty((batch, length), dtype=np.int32)
    for i in range(batch):
        g = np.random.default_rng([seed, 1, first + i])
        out[i] = g.integers(0, vocab, size=length)
    return out


def keywords(seed: int, batch: int, n_kw: int, vocab: int, first: int = 0) -> np.ndarray:
    """int32 [batch, n_kw] distinct keyword token ids per prompt."""
    out = np.empty((batch, n_kw), dtype=np.int32)
    for i in range(batch):
        g = np.random.default_rng([seed, 2, first + i])
        out[i] = g.choice(vocab, size=n_kw, replace=False)
    return out


def reward_head(seed: int, d_model: int) -> np.ndarray:
    g = np.random.default_rng([seed, 3])
    return g.standard_normal(d_model, dtype=np.float32) * np.float32(0.02)


def uniforms(seed: int, which: int, step: int, batch: int, k: int, d: int, first: int = 0) -> np.ndarray:
    """float32 [batch, k, d] draws from U[0, 1) for speculative sampling:
    which = 0 for the acceptance tests, 1 for the residual draws; row i
    belongs to prompt ``first + i`` at decoding step ``step``.  Both sides
    read these float32 values, so the oracle's draws equal the kernels'."""
    out = np.empty((batch, k, d), dtype=np.float32)
    for i in range(batch):
        g = np.random.default_rng([seed, 4 + which, step, first + i])
        out[i] = g.random((k, d), dtype=np.float32)
    return out
