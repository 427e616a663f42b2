"""ctypes binding of libcdsl.so: the calls of include/cdsl.h and
include/cdsl_ops.h with the same names, marshalling torch device tensors to
plain pointers.  Every step of the computation runs in the HIP library; if
the library is missing, loading fails loudly (there is no fallback)."""
from __future__ import annotations

import ctypes as C
import math
import os
from typing import Dict, List, Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "_lib", "libcdsl.so")

CDSL_OK, CDSL_EINVAL, CDSL_ERANGE, CDSL_ENOMEM, CDSL_EDEVICE, CDSL_ESTATE = 0, -1, -2, -3, -4, -5
CDSL_F32, CDSL_BF16 = 0, 1
CDSL_EPI_STORE, CDSL_EPI_RESIDUAL = 0, 1
ERR_NAMES = {0: "OK", -1: "EINVAL", -2: "ERANGE", -3: "ENOMEM", -4: "EDEVICE", -5: "ESTATE"}

EXPORTS = [
    "cdsl_init", "cdsl_prefill", "cdsl_rollout", "cdsl_rollout_with", "cdsl_rollout_keep", "cdsl_verify",
    "cdsl_verify_kk", "cdsl_verify_soft", "cdsl_commit_soft", "cdsl_op_soft_rows",
    "cdsl_op_lm_head_rows_workspace", "cdsl_op_lm_head_rows",
    "cdsl_reward_keywords",
    "cdsl_reward_keywords_upto", "cdsl_reward_linear", "cdsl_select", "cdsl_select_first", "cdsl_controller_states",
    "cdsl_commit", "cdsl_commit_kk",
    "cdsl_commit_heads",
    "cdsl_draft_prefix", "cdsl_verify_prefix", "cdsl_verify_prefix_soft", "cdsl_reward_keywords_prefix",
    "cdsl_commit_prefix", "cdsl_append", "cdsl_withdraw",
    "cdsl_prefix_lengths",
    "cdsl_free_prefix", "cdsl_destroy", "cdsl_last_error", "cdsl_profile_enable", "cdsl_profile_read",
    "cdsl_op_gemm_workspace", "cdsl_op_gemm", "cdsl_op_gemm_static", "cdsl_op_logit_rows",
]


class CDSLError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class ModelConfig(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("ffn_dim", C.c_int32), ("vocab", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float), ("dtype", C.c_int32)]


class Model(C.Structure):
    _fields_ = [("cfg", ModelConfig), ("tok_emb", C.c_void_p), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p), ("layer_ptrs", C.POINTER(C.c_void_p))]


KERNEL_CLASSES = ["gemm_dense", "gemm_skinny", "attention", "attn_combine", "logit_rows", "rowwise", "step",
                  "gemm_f32", "splitk_reduce"]


class KernelStats(C.Structure):
    _fields_ = [("launches", C.c_int64 * len(KERNEL_CLASSES)), ("ms", C.c_double * len(KERNEL_CLASSES)),
                ("flops", C.c_double * len(KERNEL_CLASSES)), ("bytes", C.c_double * len(KERNEL_CLASSES))]


class Limits(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("max_ctx", C.c_int32), ("max_k", C.c_int32),
                ("max_d", C.c_int32), ("max_prompt", C.c_int32), ("max_prefixes", C.c_int32)]


_lib = None


def lib():
    """Load libcdsl.so (built in-tree by ``paper_2412_10418_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2412_10418_amd.build` (no CPU fallback exists)")
    L = C.CDLL(LIB_PATH)
    vp, i32, f32 = C.c_void_p, C.c_int32, C.c_float
    sig = {
        "cdsl_init": ([C.POINTER(Model), C.POINTER(Model), C.POINTER(Limits), vp, C.POINTER(vp)], i32),
        "cdsl_prefill": ([vp, vp, i32, i32, i32, C.POINTER(vp), vp, vp], i32),
        "cdsl_rollout": ([vp, vp, vp, i32, i32, vp], i32),
        "cdsl_rollout_with": ([vp, vp, vp, i32, i32, i32, vp], i32),
        "cdsl_rollout_keep": ([vp, vp, vp, i32, i32, vp, vp], i32),
        "cdsl_verify_soft": ([vp, vp, vp, i32, i32, i32] + [vp] * 14, i32),
        "cdsl_commit_soft": ([vp, vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp], i32),
        "cdsl_op_soft_rows": ([vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp], i32),
        "cdsl_op_lm_head_rows_workspace": ([i32, i32, i32, i32, i32], C.c_size_t),
        "cdsl_op_lm_head_rows": ([vp, vp, i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp, C.c_size_t, vp], i32),
        "cdsl_reward_keywords_upto": ([vp, vp, vp, i32, i32, vp, vp, i32, i32, vp], i32),
        "cdsl_commit_heads": ([vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp], i32),
        "cdsl_draft_prefix": ([vp, vp, i32, vp, vp], i32),
        "cdsl_verify_prefix": ([vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp], i32),
        "cdsl_verify_prefix_soft": ([vp, vp, vp, i32, i32] + [vp] * 12, i32),
        "cdsl_reward_keywords_prefix": ([vp, vp, vp, i32, vp, vp, i32, i32, vp], i32),
        "cdsl_commit_prefix": ([vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp], i32),
        "cdsl_append": ([vp, vp, vp, vp, i32, vp, vp, vp], i32),
        "cdsl_withdraw": ([vp, vp, vp], i32),
        "cdsl_verify_kk": ([vp, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp], i32),
        "cdsl_commit_kk": ([vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp], i32),
        "cdsl_verify": ([vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp], i32),
        "cdsl_reward_keywords": ([vp, vp, vp, i32, i32, vp, i32, i32, vp], i32),
        "cdsl_reward_linear": ([vp, vp, vp, i32, i32, i32, vp], i32),
        "cdsl_select": ([vp, vp, vp, f32, i32, i32, vp], i32),
        "cdsl_select_first": ([vp, vp, vp, i32, i32, vp], i32),
        "cdsl_controller_states": ([vp, vp, vp, i32, i32, C.c_double, C.c_double, i32, vp, vp], i32),
        "cdsl_commit": ([vp, vp, vp, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp], i32),
        "cdsl_prefix_lengths": ([vp, vp, vp], i32),
        "cdsl_free_prefix": ([vp, vp], i32),
        "cdsl_destroy": ([vp], i32),
        "cdsl_last_error": ([vp], C.c_char_p),
        "cdsl_profile_enable": ([vp, i32], i32),
        "cdsl_profile_read": ([vp, C.POINTER(KernelStats)], i32),
        "cdsl_op_gemm_workspace": ([i32, i32, i32, i32], C.c_size_t),
        "cdsl_op_gemm": ([vp, vp, vp, i32, i32, i32, i32, i32, vp, C.c_size_t, vp], i32),
        "cdsl_op_gemm_static": ([vp, vp, vp, i32, i32, i32, i32, i32, vp], i32),
        "cdsl_op_logit_rows": ([vp, i32, i32, vp, i32, vp, vp, vp, vp, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor"):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _sized(t: Optional[torch.Tensor], n: int, dtype, name="tensor"):
    """_ptr of a buffer the library reads or writes n elements of: a device
    tensor of that many elements is required (the C ABI cannot check)."""
    if t is None:
        raise ValueError(f"{name} is required")
    if t.numel() != n:
        raise ValueError(f"{name} must hold {n} elements, got {tuple(t.shape)}")
    return _ptr(t, dtype, name)


def _verify_out_ptrs(out: dict, B: int, k: int, d: int, kk: int, D: int):
    """Pointers of cdsl_verify's output buffers, each checked for its size."""
    hid = out.get("hidden")
    return (_sized(out["logprobs"], B * k * d, torch.float32, "logprobs"),
            _sized(out["target_argmax"], B * k * d, torch.int32, "target_argmax"),
            _sized(out["n_accept"], B * k, torch.int32, "n_accept"),
            _sized(out["scores"], B * k, torch.float32, "scores"),
            _sized(out["row_topk_ids"], B * k * d * kk, torch.int32, "row_topk_ids"),
            _sized(out["row_topk_lp"], B * k * d * kk, torch.float32, "row_topk_lp"),
            _sized(hid, B * k * D, torch.float32, "hidden") if hid is not None else None)


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _check(rc, ctx=None):
    if rc != CDSL_OK:
        msg = lib().cdsl_last_error(ctx)
        raise CDSLError(rc, msg.decode() if msg else "")


# ---------------------------------------------------------------------------
# kernel-level entry points
# ---------------------------------------------------------------------------
_GEMM_WS = {}


def cdsl_op_gemm(A: torch.Tensor, B: torch.Tensor, C_out: Optional[torch.Tensor] = None,
                 residual: bool = False) -> torch.Tensor:
    M, K = A.shape
    N = B.shape[0]
    dt = CDSL_BF16 if B.dtype == torch.bfloat16 else CDSL_F32
    if C_out is None:
        C_out = torch.zeros((M, N), dtype=torch.float32, device=A.device)
    need = lib().cdsl_op_gemm_workspace(M, N, K, dt)
    ws = _GEMM_WS.get(A.device)
    if ws is None or ws.numel() < need:
        ws = torch.zeros(max(need, 256), dtype=torch.uint8, device=A.device)
        _GEMM_WS[A.device] = ws
    rc = lib().cdsl_op_gemm(_ptr(A, torch.float32, "A"), _ptr(B, B.dtype, "B"), _ptr(C_out, torch.float32, "C"),
                            M, N, K, dt, CDSL_EPI_RESIDUAL if residual else CDSL_EPI_STORE,
                            ws.data_ptr(), ws.numel(), _stream())
    _check(rc)
    return C_out


def cdsl_op_logit_rows(logits: torch.Tensor, gather: Optional[torch.Tensor], kk: int):
    M, V = logits.shape
    dev = logits.device
    lp = torch.zeros(M, dtype=torch.float32, device=dev)
    amax = torch.zeros(M, dtype=torch.int32, device=dev)
    tk = torch.zeros((M, max(kk, 1)), dtype=torch.int32, device=dev)
    tl = torch.zeros((M, max(kk, 1)), dtype=torch.float32, device=dev)
    rc = lib().cdsl_op_logit_rows(_ptr(logits, torch.float32, "logits"), M, V,
                                  _ptr(gather, torch.int32, "gather"), kk, lp.data_ptr(),
                                  amax.data_ptr(), tk.data_ptr(), tl.data_ptr(), _stream())
    _check(rc)
    return lp, amax, tk[:, :kk], tl[:, :kk]


def cdsl_op_lm_head_rows(A: torch.Tensor, B: torch.Tensor, gather: Optional[torch.Tensor], kk: int):
    """The LM head with the fused row epilogue; returns (lp, amax, topk_ids,
    topk_lp) as cdsl_op_logit_rows does for the logits A @ B.T."""
    M, K = A.shape
    V = B.shape[0]
    dt = CDSL_BF16 if B.dtype == torch.bfloat16 else CDSL_F32
    dev = A.device
    need = lib().cdsl_op_lm_head_rows_workspace(M, V, K, dt, kk)
    if need == 0:
        raise ValueError("shape not covered by the fused LM-head epilogue")
    ws = torch.zeros(need, dtype=torch.uint8, device=dev)
    lp = torch.zeros(M, dtype=torch.float32, device=dev)
    amax = torch.zeros(M, dtype=torch.int32, device=dev)
    tk = torch.zeros((M, max(kk, 1)), dtype=torch.int32, device=dev)
    tl = torch.zeros((M, max(kk, 1)), dtype=torch.float32, device=dev)
    rc = lib().cdsl_op_lm_head_rows(_ptr(A, torch.float32, "A"), _ptr(B, B.dtype, "B"), M, V, K, dt,
                                    _ptr(gather, torch.int32, "gather"), kk, lp.data_ptr(), amax.data_ptr(),
                                    tk.data_ptr(), tl.data_ptr(), ws.data_ptr(), need, _stream())
    _check(rc)
    return lp, amax, tk[:, :kk], tl[:, :kk]


def cdsl_op_soft_rows(target_logits: torch.Tensor, draft_logits: torch.Tensor, d: int, lookaheads: torch.Tensor,
                      v: torch.Tensor):
    """Returns (draft_lp, res_ids, res_lp), each [M]."""
    M, V = target_logits.shape
    if draft_logits.shape != (M, V) or v.shape != (M,) or lookaheads.shape != (M // d, d + 1) or M % d:
        raise ValueError("shapes: logits [M, V] twice, lookaheads [M/d, d+1], v [M]")
    dev = target_logits.device
    dlp = torch.empty(M, dtype=torch.float32, device=dev)
    rid = torch.empty(M, dtype=torch.int32, device=dev)
    rlp = torch.empty(M, dtype=torch.float32, device=dev)
    rc = lib().cdsl_op_soft_rows(_ptr(target_logits, torch.float32, "target_logits"),
                                 _ptr(draft_logits, torch.float32, "draft_logits"), M, V, d,
                                 _ptr(lookaheads, torch.int32, "lookaheads"), _ptr(v, torch.float32, "v"),
                                 dlp.data_ptr(), rid.data_ptr(), rlp.data_ptr(), _stream())
    _check(rc)
    return dlp, rid, rlp


# ---------------------------------------------------------------------------
# context
# ---------------------------------------------------------------------------
def _model_struct(shape, dtype_code, tensors: Dict[str, object]):
    cfg = ModelConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.ffn_dim,
                      shape.vocab, shape.rope_theta, shape.rms_eps, dtype_code)
    order = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")
    ptrs = []
    for lw in tensors["layers"]:
        for nm in order:
            ptrs.append(_ptr(lw[nm], None, nm))
    arr = (C.c_void_p * len(ptrs))(*ptrs)
    m = Model(cfg, _ptr(tensors["tok_emb"], None, "tok_emb"), _ptr(tensors["final_norm"], torch.float32, "final_norm"),
              _ptr(tensors["lm_head"], None, "lm_head"), C.cast(arr, C.POINTER(C.c_void_p)))
    return m, arr


class Prefix:
    def __init__(self, ctx: "Context", handle, B: int):
        self.ctx, self.handle, self.B = ctx, handle, B

    def lengths(self) -> List[int]:
        out = (C.c_int32 * self.B)()
        _check(lib().cdsl_prefix_lengths(self.ctx.handle, self.handle, out), self.ctx.handle)
        return list(out)

    def free(self):
        if self.handle:
            _check(lib().cdsl_free_prefix(self.ctx.handle, self.handle), self.ctx.handle)
            self.handle = None


class Context:
    """One draft/target pair behind cdsl_init.  Weights are dicts of device
    tensors laid out like ``cdsl_inputs.model_weights`` (matrices
    [out, in] in the model dtype, norm gains fp32)."""

    def __init__(self, draft_shape, draft_w, target_shape, target_w, dtype: str, limits: Dict[str, int]):
        code = CDSL_BF16 if dtype == "bf16" else CDSL_F32
        dm, dkeep = _model_struct(draft_shape, code, draft_w)
        tm, tkeep = _model_struct(target_shape, code, target_w)
        lim = Limits(limits["max_batch"], limits["max_ctx"], limits["max_k"], limits["max_d"],
                     limits["max_prompt"], limits.get("max_prefixes", 1))
        h = C.c_void_p()
        rc = lib().cdsl_init(C.byref(dm), C.byref(tm), C.byref(lim), _stream(), C.byref(h))
        _check(rc)
        self.handle = h
        self.draft_shape, self.target_shape = draft_shape, target_shape
        self.dtype = dtype
        self.limits = {"max_batch": lim.max_batch, "max_ctx": lim.max_ctx, "max_k": lim.max_k,
                       "max_d": lim.max_d, "max_prompt": lim.max_prompt, "max_prefixes": lim.max_prefixes}
        # the library borrows the embedding, LM head, norm gains, wo and
        # w_down: their tensors live as long as the context
        self._borrowed = (draft_w, target_w, dkeep, tkeep)

    def close(self):
        if self.handle:
            lib().cdsl_destroy(self.handle)
            self.handle = None
        self._borrowed = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- measurement -----------------------------------------------------------
    def profile_enable(self, on: bool = True):
        _check(lib().cdsl_profile_enable(self.handle, 1 if on else 0), self.handle)

    def profile_read(self) -> Dict[str, dict]:
        st = KernelStats()
        _check(lib().cdsl_profile_read(self.handle, C.byref(st)), self.handle)
        return {nm: {"launches": int(st.launches[i]), "ms": float(st.ms[i]), "flops": float(st.flops[i]),
                     "bytes": float(st.bytes[i])} for i, nm in enumerate(KERNEL_CLASSES)}

    # -- the step ------------------------------------------------------------
    def cdsl_prefill(self, tokens: torch.Tensor, k: int):
        B, L = tokens.shape
        dev = tokens.device
        beams = torch.empty((B, k), dtype=torch.int32, device=dev)
        head_lp = torch.empty((B, k), dtype=torch.float32, device=dev)
        h = C.c_void_p()
        rc = lib().cdsl_prefill(self.handle, _ptr(tokens, torch.int32, "tokens"), B, L, k, C.byref(h),
                                beams.data_ptr(), head_lp.data_ptr())
        _check(rc, self.handle)
        return Prefix(self, h, B), beams, head_lp

    def cdsl_rollout(self, prefix: Prefix, beams: torch.Tensor, k: int, d: int,
                     lookaheads: Optional[torch.Tensor] = None) -> torch.Tensor:
        if lookaheads is None:
            lookaheads = torch.empty((prefix.B, k, d + 1), dtype=torch.int32, device=beams.device)
        rc = lib().cdsl_rollout(self.handle, prefix.handle, _sized(beams, prefix.B * k, torch.int32, "beams"), k, d,
                                _sized(lookaheads, prefix.B * k * (d + 1), torch.int32, "lookaheads"))
        _check(rc, self.handle)
        return lookaheads

    def cdsl_rollout_with(self, prefix: Prefix, beams: torch.Tensor, k: int, d: int, roller: int,
                          lookaheads: Optional[torch.Tensor] = None) -> torch.Tensor:
        if lookaheads is None:
            lookaheads = torch.empty((prefix.B, k, d + 1), dtype=torch.int32, device=beams.device)
        rc = lib().cdsl_rollout_with(self.handle, prefix.handle, _sized(beams, prefix.B * k, torch.int32, "beams"),
                                     k, d, int(roller),
                                     _sized(lookaheads, prefix.B * k * (d + 1), torch.int32, "lookaheads"))
        _check(rc, self.handle)
        return lookaheads

    def cdsl_rollout_keep(self, prefix: Prefix, beams: torch.Tensor, k: int, d: int, lookaheads: torch.Tensor,
                          draft_logits: torch.Tensor) -> torch.Tensor:
        if draft_logits.numel() != prefix.B * k * d * self.draft_shape.vocab:
            raise ValueError("draft_logits must be [B, k, d, V]")
        rc = lib().cdsl_rollout_keep(self.handle, prefix.handle, _sized(beams, prefix.B * k, torch.int32, "beams"),
                                     k, d, _sized(lookaheads, prefix.B * k * (d + 1), torch.int32, "lookaheads"),
                                     _ptr(draft_logits, torch.float32, "draft_logits"))
        _check(rc, self.handle)
        return lookaheads

    def cdsl_verify_soft(self, prefix: Prefix, lookaheads: torch.Tensor, k: int, d: int, head_lp: torch.Tensor,
                         draft_logits: torch.Tensor, u: torch.Tensor, v: torch.Tensor, out: dict,
                         want_hidden: bool = False, kk: Optional[int] = None) -> dict:
        """out: the buffers of cdsl_verify plus draft_lp, res_ids, res_lp ([B, k, d]);
        kk: top-k width of row_topk (default k)."""
        B = prefix.B
        kk = k if kk is None else kk
        for nm, t in (("u", u), ("v", v)):
            if t.shape != (B, k, d):
                raise ValueError(f"{nm} must be [B, k, d]")
        o = dict(out)
        if not want_hidden:
            o["hidden"] = None
        lp, y, na, sc, ti, tl, hid = _verify_out_ptrs(o, B, k, d, kk, self.target_shape.d_model)
        rc = lib().cdsl_verify_soft(self.handle, prefix.handle,
                                    _sized(lookaheads, B * k * (d + 1), torch.int32, "lookaheads"), k, d, kk,
                                    _sized(head_lp, B * k, torch.float32, "head_lp"),
                                    _sized(draft_logits, B * k * d * self.draft_shape.vocab, torch.float32,
                                           "draft_logits"),
                                    _ptr(u, torch.float32, "u"), _ptr(v, torch.float32, "v"), lp,
                                    _sized(out["draft_lp"], B * k * d, torch.float32, "draft_lp"), y, na, sc, ti, tl,
                                    _sized(out["res_ids"], B * k * d, torch.int32, "res_ids"),
                                    _sized(out["res_lp"], B * k * d, torch.float32, "res_lp"), hid)
        _check(rc, self.handle)
        return out

    def cdsl_commit_soft(self, prefix: Prefix, lookaheads, beam, n_accept, row_topk_ids, row_topk_lp, res_ids,
                         res_lp, k, d, next_beams: torch.Tensor, next_head_lp: torch.Tensor):
        """kk (the next-head width) is next_beams.shape[1]."""
        B = prefix.B
        kk = next_beams.shape[1]
        emitted = (C.c_int32 * (B * (d + 1)))()
        n_emit = (C.c_int32 * B)()
        rc = lib().cdsl_commit_soft(self.handle, prefix.handle,
                                    _sized(lookaheads, B * k * (d + 1), torch.int32, "lookaheads"),
                                    _sized(beam, B, torch.int32, "beam"),
                                    _sized(n_accept, B * k, torch.int32, "n_accept"),
                                    _sized(row_topk_ids, B * k * d * kk, torch.int32, "row_topk_ids"),
                                    _sized(row_topk_lp, B * k * d * kk, torch.float32, "row_topk_lp"),
                                    _sized(res_ids, B * k * d, torch.int32, "res_ids"),
                                    _sized(res_lp, B * k * d, torch.float32, "res_lp"),
                                    k, d, kk, emitted, n_emit, _sized(next_beams, B * kk, torch.int32, "next_beams"),
                                    _sized(next_head_lp, B * kk, torch.float32, "next_head_lp"))
        _check(rc, self.handle)
        return [[emitted[b * (d + 1) + t] for t in range(n_emit[b])] for b in range(B)]

    def cdsl_verify(self, prefix: Prefix, lookaheads: torch.Tensor, k: int, d: int, head_lp: torch.Tensor,
                    want_hidden: bool = False, out: Optional[dict] = None, kk: Optional[int] = None) -> dict:
        """kk: top-k width of row_topk (default k; another value uses cdsl_verify_kk)."""
        B = prefix.B
        dev = lookaheads.device
        kk = k if kk is None else kk
        if out is None:
            out = {
                "logprobs": torch.empty((B, k, d), dtype=torch.float32, device=dev),
                "target_argmax": torch.empty((B, k, d), dtype=torch.int32, device=dev),
                "n_accept": torch.empty((B, k), dtype=torch.int32, device=dev),
                "scores": torch.empty((B, k), dtype=torch.float32, device=dev),
                "row_topk_ids": torch.empty((B, k, d, kk), dtype=torch.int32, device=dev),
                "row_topk_lp": torch.empty((B, k, d, kk), dtype=torch.float32, device=dev),
                "hidden": (torch.empty((B, k, self.target_shape.d_model), dtype=torch.float32, device=dev)
                           if want_hidden else None),
            }
        outs = _verify_out_ptrs(out, B, k, d, kk, self.target_shape.d_model)
        look = _sized(lookaheads, B * k * (d + 1), torch.int32, "lookaheads")
        hl = _sized(head_lp, B * k, torch.float32, "head_lp")
        if kk != k:
            rc = lib().cdsl_verify_kk(self.handle, prefix.handle, look, k, d, kk, hl, *outs)
            _check(rc, self.handle)
            return out
        rc = lib().cdsl_verify(self.handle, prefix.handle, look, k, d, hl, *outs)
        _check(rc, self.handle)
        return out

    def cdsl_reward_keywords(self, prefix: Prefix, lookaheads, k, d, keywords, normalize: bool,
                             reward: Optional[torch.Tensor] = None):
        if reward is None:
            reward = torch.empty((prefix.B, k), dtype=torch.float32, device=lookaheads.device)
        rc = lib().cdsl_reward_keywords(self.handle, prefix.handle, _ptr(lookaheads, torch.int32, "lookaheads"),
                                        k, d, _ptr(keywords, torch.int32, "keywords"), keywords.shape[1],
                                        1 if normalize else 0, reward.data_ptr())
        _check(rc, self.handle)
        return reward

    def cdsl_reward_keywords_upto(self, prefix: Prefix, lookaheads, k, d, upto: Optional[torch.Tensor], keywords,
                                  normalize: bool, reward: Optional[torch.Tensor] = None):
        if reward is None:
            reward = torch.empty((prefix.B, k), dtype=torch.float32, device=lookaheads.device)
        rc = lib().cdsl_reward_keywords_upto(self.handle, prefix.handle,
                                             _ptr(lookaheads, torch.int32, "lookaheads"), k, d,
                                             _ptr(upto, torch.int32, "upto") if upto is not None else None,
                                             _ptr(keywords, torch.int32, "keywords"), keywords.shape[1],
                                             1 if normalize else 0, reward.data_ptr())
        _check(rc, self.handle)
        return reward

    def cdsl_reward_linear(self, hidden: torch.Tensor, w: torch.Tensor, reward: Optional[torch.Tensor] = None):
        B, k, D = hidden.shape
        if reward is None:
            reward = torch.empty((B, k), dtype=torch.float32, device=hidden.device)
        rc = lib().cdsl_reward_linear(self.handle, _ptr(hidden, torch.float32, "hidden"),
                                      _ptr(w, torch.float32, "w"), B, k, D, reward.data_ptr())
        _check(rc, self.handle)
        return reward

    def cdsl_select(self, scores: torch.Tensor, reward: torch.Tensor, alpha: float,
                    beam: Optional[torch.Tensor] = None) -> torch.Tensor:
        B, k = scores.shape
        if beam is None:
            beam = torch.empty(B, dtype=torch.int32, device=scores.device)
        rc = lib().cdsl_select(self.handle, _ptr(scores, torch.float32, "scores"),
                               _ptr(reward, torch.float32, "reward"), float(alpha), B, k, beam.data_ptr())
        _check(rc, self.handle)
        return beam

    def cdsl_select_first(self, reward: torch.Tensor, first_at: torch.Tensor,
                          beam: Optional[torch.Tensor] = None) -> torch.Tensor:
        B, k = reward.shape
        if first_at.shape != (B,):
            raise ValueError("first_at must be [B]")
        if beam is None:
            beam = torch.empty(B, dtype=torch.int32, device=reward.device)
        rc = lib().cdsl_select_first(self.handle, _ptr(reward, torch.float32, "reward"),
                                     _ptr(first_at, torch.float32, "first_at"), B, k, beam.data_ptr())
        _check(rc, self.handle)
        return beam

    def cdsl_controller_states(self, n_accept: torch.Tensor, reward: torch.Tensor, d: int, a_t: float,
                               r_t: float, b: int, state: Optional[torch.Tensor] = None,
                               first_at: Optional[torch.Tensor] = None):
        """n_accept / reward: [B] (or [B, 1]) k = 1 outputs; returns (state, first_at)."""
        B = n_accept.numel()
        if reward.numel() != B:
            raise ValueError("n_accept and reward must have B elements")
        if state is None:
            state = torch.empty(B, dtype=torch.int32, device=n_accept.device)
        if first_at is None:
            first_at = torch.empty(B, dtype=torch.float32, device=n_accept.device)
        rc = lib().cdsl_controller_states(self.handle, _ptr(n_accept, torch.int32, "n_accept"),
                                          _ptr(reward, torch.float32, "reward"), B, d, float(a_t), float(r_t),
                                          int(b), state.data_ptr(), first_at.data_ptr())
        _check(rc, self.handle)
        return state, first_at

    def cdsl_commit(self, prefix: Prefix, lookaheads, beam, n_accept, row_topk_ids, row_topk_lp, k, d,
                    next_beams: Optional[torch.Tensor] = None, next_head_lp: Optional[torch.Tensor] = None,
                    kk: Optional[int] = None):
        """kk: top-k width of row_topk and of the next heads (default k; another
        value uses cdsl_commit_kk)."""
        B = prefix.B
        dev = lookaheads.device
        kk = k if kk is None else kk
        if next_beams is None:
            next_beams = torch.empty((B, kk), dtype=torch.int32, device=dev)
        if next_head_lp is None:
            next_head_lp = torch.empty((B, kk), dtype=torch.float32, device=dev)
        emitted = (C.c_int32 * (B * (d + 1)))()
        n_emit = (C.c_int32 * B)()
        args = (_sized(lookaheads, B * k * (d + 1), torch.int32, "lookaheads"),
                _sized(beam, B, torch.int32, "beam"), _sized(n_accept, B * k, torch.int32, "n_accept"),
                _sized(row_topk_ids, B * k * d * kk, torch.int32, "row_topk_ids"),
                _sized(row_topk_lp, B * k * d * kk, torch.float32, "row_topk_lp"))
        nb = _sized(next_beams, B * kk, torch.int32, "next_beams")
        nl = _sized(next_head_lp, B * kk, torch.float32, "next_head_lp")
        if kk != k:
            rc = lib().cdsl_commit_kk(self.handle, prefix.handle, *args, k, d, kk, emitted, n_emit, nb, nl)
        else:
            rc = lib().cdsl_commit(self.handle, prefix.handle, *args, k, d, emitted, n_emit, nb, nl)
        _check(rc, self.handle)
        em = [[emitted[b * (d + 1) + t] for t in range(n_emit[b])] for b in range(B)]
        return em, next_beams, next_head_lp

    def cdsl_commit_heads(self, prefix: Prefix, lookaheads, beam, k, d, mask: Optional[List[int]],
                          next_beams: torch.Tensor, next_head_lp: torch.Tensor) -> List[int]:
        """Head-only commit; returns the emitted token per prompt (-1: none).
        next_beams / next_head_lp [B, kk] are updated in place for emitting
        prompts."""
        B = prefix.B
        kk = next_beams.shape[1]
        m = None
        if mask is not None:
            m = (C.c_int32 * B)(*[1 if v else 0 for v in mask])
        emitted = (C.c_int32 * B)()
        rc = lib().cdsl_commit_heads(self.handle, prefix.handle, _ptr(lookaheads, torch.int32, "lookaheads"),
                                     _ptr(beam, torch.int32, "beam"), k, d, kk, m, emitted,
                                     _ptr(next_beams, torch.int32, "next_beams"),
                                     _ptr(next_head_lp, torch.float32, "next_head_lp"))
        _check(rc, self.handle)
        return [emitted[b] for b in range(B)]

    # -- Alg. 1 from the prefix (one lookahead per prompt) -------------------
    def cdsl_draft_prefix(self, prefix: Prefix, d: int, lookaheads: torch.Tensor,
                          draft_logits: Optional[torch.Tensor] = None) -> torch.Tensor:
        """lookaheads [B, d+1] (or [B, 1, d+1]); draft_logits [B, d, V] or None."""
        B = prefix.B
        dl = None
        if draft_logits is not None:
            dl = _sized(draft_logits, B * d * self.draft_shape.vocab, torch.float32, "draft_logits")
        rc = lib().cdsl_draft_prefix(self.handle, prefix.handle, d,
                                     _sized(lookaheads, B * (d + 1), torch.int32, "lookaheads"), dl)
        _check(rc, self.handle)
        return lookaheads

    def cdsl_verify_prefix(self, prefix: Prefix, lookaheads: torch.Tensor, d: int, kk: int, out: dict,
                           draft_logits: Optional[torch.Tensor] = None, u: Optional[torch.Tensor] = None,
                           v: Optional[torch.Tensor] = None) -> dict:
        """out: logprobs [B, d], target_argmax [B, d], n_accept [B], scores [B],
        row_topk_ids / row_topk_lp [B, d, kk]; with u (speculative sampling)
        also draft_lp, res_ids, res_lp [B, d], and draft_logits / v."""
        B = prefix.B
        look = _sized(lookaheads, B * (d + 1), torch.int32, "lookaheads")
        base = (_sized(out["logprobs"], B * d, torch.float32, "logprobs"),
                _sized(out["target_argmax"], B * d, torch.int32, "target_argmax"),
                _sized(out["n_accept"], B, torch.int32, "n_accept"),
                _sized(out["scores"], B, torch.float32, "scores"),
                _sized(out["row_topk_ids"], B * d * kk, torch.int32, "row_topk_ids"),
                _sized(out["row_topk_lp"], B * d * kk, torch.float32, "row_topk_lp"))
        if u is None:
            rc = lib().cdsl_verify_prefix(self.handle, prefix.handle, look, d, kk, *base)
        else:
            lp, y, na, sc, ti, tl = base
            rc = lib().cdsl_verify_prefix_soft(
                self.handle, prefix.handle, look, d, kk,
                _sized(draft_logits, B * d * self.draft_shape.vocab, torch.float32, "draft_logits"),
                _sized(u, B * d, torch.float32, "u"), _sized(v, B * d, torch.float32, "v"), lp,
                _sized(out["draft_lp"], B * d, torch.float32, "draft_lp"), y, na, sc, ti, tl,
                _sized(out["res_ids"], B * d, torch.int32, "res_ids"),
                _sized(out["res_lp"], B * d, torch.float32, "res_lp"))
        _check(rc, self.handle)
        return out

    def cdsl_reward_keywords_prefix(self, prefix: Prefix, lookaheads, d, upto: Optional[torch.Tensor], keywords,
                                    normalize: bool, reward: torch.Tensor):
        B = prefix.B
        rc = lib().cdsl_reward_keywords_prefix(self.handle, prefix.handle,
                                               _sized(lookaheads, B * (d + 1), torch.int32, "lookaheads"), d,
                                               _sized(upto, B, torch.int32, "upto") if upto is not None else None,
                                               _ptr(keywords, torch.int32, "keywords"), keywords.shape[1],
                                               1 if normalize else 0, _sized(reward, B, torch.float32, "reward"))
        _check(rc, self.handle)
        return reward

    def cdsl_commit_prefix(self, prefix: Prefix, lookaheads, n_accept, d, row_topk_ids, row_topk_lp,
                           next_beams: torch.Tensor, next_head_lp: torch.Tensor) -> List[List[int]]:
        """Emits x_1..x_n per prompt; kk = next_beams.shape[1]."""
        B = prefix.B
        kk = next_beams.shape[1]
        emitted = (C.c_int32 * (B * d))()
        n_emit = (C.c_int32 * B)()
        rc = lib().cdsl_commit_prefix(self.handle, prefix.handle,
                                      _sized(lookaheads, B * (d + 1), torch.int32, "lookaheads"),
                                      _sized(n_accept, B, torch.int32, "n_accept"), d, kk,
                                      _sized(row_topk_ids, B * d * kk, torch.int32, "row_topk_ids"),
                                      _sized(row_topk_lp, B * d * kk, torch.float32, "row_topk_lp"),
                                      emitted, n_emit, _sized(next_beams, B * kk, torch.int32, "next_beams"),
                                      _sized(next_head_lp, B * kk, torch.float32, "next_head_lp"))
        _check(rc, self.handle)
        return [[emitted[b * d + t] for t in range(n_emit[b])] for b in range(B)]

    def cdsl_append(self, prefix: Prefix, tokens: torch.Tensor, mask: Optional[List[bool]],
                    next_beams: torch.Tensor, next_head_lp: torch.Tensor) -> List[int]:
        """Emit tokens[b] for the masked prompts; next heads [B, kk] updated
        in place for them.  Returns the emitted token per prompt (-1: none)."""
        B = prefix.B
        kk = next_beams.shape[1]
        m = None if mask is None else (C.c_int32 * B)(*[1 if v else 0 for v in mask])
        emitted = (C.c_int32 * B)()
        rc = lib().cdsl_append(self.handle, prefix.handle, _sized(tokens, B, torch.int32, "tokens"), m, kk, emitted,
                               _sized(next_beams, B * kk, torch.int32, "next_beams"),
                               _sized(next_head_lp, B * kk, torch.float32, "next_head_lp"))
        _check(rc, self.handle)
        return [emitted[b] for b in range(B)]

    def cdsl_withdraw(self, prefix: Prefix, counts: List[int]):
        B = prefix.B
        arr = (C.c_int32 * B)(*[int(x) for x in counts])
        _check(lib().cdsl_withdraw(self.handle, prefix.handle, arr), self.handle)


# ---------------------------------------------------------------------------
# weight upload (marshalling of the seeded host arrays)
# ---------------------------------------------------------------------------
def upload_weights(w: Dict[str, object], dtype: str, device="cuda") -> Dict[str, object]:
    """Host float32 arrays (bf16-representable for bf16) -> device tensors."""
    import numpy as np
    from cdsl_inputs import f32_to_bf16_bits

    def mat(a):
        if dtype == "bf16":
            bits = torch.from_numpy(f32_to_bf16_bits(a).view(np.int16))
            return bits.to(device).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)

    def vec(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)

    out = {"tok_emb": mat(w["tok_emb"]), "lm_head": mat(w["lm_head"]), "final_norm": vec(w["final_norm"]),
           "layers": []}
    for lw in w["layers"]:
        out["layers"].append({nm: (vec(v) if nm.endswith("norm") else mat(v)) for nm, v in lw.items()})
    return out
