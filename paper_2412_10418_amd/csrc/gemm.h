// Internal interface of the projection kernels (gemm.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

#include "common.h"

namespace cdsl {

enum GemmEpilogue { kEpiStore = 0, kEpiResidual = 1, kEpiSwiGLU = 2, kEpiRowStats = 3, kEpiRope = 4 };

// kEpiRope: the q/k/v projection of pass p (W packs H query heads, then Hkv
// key heads, then Hkv value heads, hd columns each) finishes in its
// epilogue what the rotary + KV-write kernel does with the stored product:
// q heads rotated into qout (fp32 [M][H][hd]), key heads rotated and value
// heads as they are into the layer's units of the bf16 KV pool (hi / lo
// planes; K [16][hd], V [hd][16] per block and KV head), at the block, slot
// and position of each row.  cos_t / sin_t: [position][hd / 2].  rowinfo:
// [M] (block * 16 + slot, position) of each row of p.  hd is 64 or 128.
struct RopeEpi {
  PassDesc p;
  const int2* rowinfo;
  float* qout;
  KVPool pool;
  int layer;
  const float* cos_t;
  const float* sin_t;
  int H, Hkv, hd;
};

// The activation operand: bf16 hi / lo planes [M, K] (bf16-weight models) or
// one fp32 matrix [M, K] (fp32-weight models).
struct GemmOperand {
  const bf16* hi;
  const bf16* lo;
  const float* f32;
};

// Where the product goes: fp32 [M, ldc] for kEpiStore / kEpiResidual, the
// bf16 hi / lo planes [M, ldc] of silu(gate) * up for kEpiSwiGLU.
struct GemmOut {
  float* f32;
  bf16* hi;
  bf16* lo;
  int ldc;
};

// C = A[M,K] * W[N,K]^T, fp32 accumulate.  dtype 1: W bf16 (A as hi / lo
// planes, two MFMA products per step); dtype 0: W fp32 (A fp32).
//   kEpiStore:    C  = product
//   kEpiResidual: C += product
//   kEpiSwiGLU:   (bf16 only) W packs, per group of 32 rows, 16 gate rows
//                 then the 16 matching up rows; the output (ldc = N/2)
//                 receives silu(gate) * up as hi / lo planes.
//   kEpiRowStats: no C; the product's row statistics per column tile go to
//                 *rs (RowStats in common.h), whose tiles field the launch
//                 sets.  The K dimension is never split for it.
//   kEpiRope:     no C; see RopeEpi (*rope).  Only where gemm_rope_fusable
//                 holds: the dense kernel with no K split, whose output tile
//                 holds whole heads.
size_t gemm_workspace_bytes(int M, int N, int K, int dtype);
int gemm_check(int M, int N, int K, int dtype);
// 0: dense bf16 kernel, 1: skinny bf16 kernel, 2: fp32 kernel
int gemm_kind(int M, int N, int K, int dtype);
// Column tiles of a kEpiRowStats launch of this shape (0: not supported).
int gemm_rowstats_tiles(int M, int N, int K, int dtype);
// Whether a kEpiRope launch of this shape and head size is supported.
bool gemm_rope_fusable(int M, int N, int K, int dtype, int hd);
// Called between the main kernel and the split-K reduce, when there is one
// (lets the caller time the two kernels separately).
struct GemmHook {
  virtual void before_reduce(int ksplit) = 0;
};
// prefill selects a separately named instantiation of the dense kernel.
// With deferred != null, a K split is left unreduced: the ksplit fp32
// planes [ksplit][M][N] stay at the start of ws for the caller to consume
// (before the next projection), the epilogue is not applied, and *deferred
// receives ksplit (1: no split, the epilogue was applied as usual).
// kEpiSwiGLU is never deferred.
hipError_t gemm_launch(const GemmOperand& A, const void* B, const GemmOut& out, int M, int N, int K, int dtype,
                       int epi, void* ws, size_t ws_bytes, hipStream_t st, bool prefill = false,
                       GemmHook* hook = nullptr, int* deferred = nullptr, RowStats* rs = nullptr,
                       const RopeEpi* rope = nullptr);
hipError_t swiglu_f32_launch(const float* gu, float* act, int M, int F, hipStream_t st);
hipError_t split_planes_launch(const float* x, bf16* hi, bf16* lo, long long n, hipStream_t st);

}  // namespace cdsl
