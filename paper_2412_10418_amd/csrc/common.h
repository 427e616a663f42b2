// Shared device/host definitions of the CDSL library (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cdsl {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2v;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
// native 16-byte vector for raw copies (HIP's uint4 wraps a union, which
// keeps the optimizer from holding it in registers)
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 16;        // tokens per KV block (= one MFMA key tile)
constexpr int kMaxK = 16;         // beams
constexpr int kMaxD = 32;         // lookahead depth
constexpr int kWave = 64;

// --------------------------------------------------------------------------
// One forward pass of a decoder over a set of rows.
//
// Rows are grouped by prompt: row m = (bi * kp + i) * R + j for prompt slot
// bi < nb (batch index b = prompt_ids ? prompt_ids[bi] : bi), beam i < kp and
// row j < R of that beam.
//   mode kAppend: the rows extend the prefix (prompt prefill, catch-up).
//                 Row j sits at position Lp[b] + j, writes its K/V into the
//                 prefix blocks and attends causally to prefix [0, pos].
//   mode kSuffix: the rows are beam continuations (rollout, verification).
//                 Row (i, j) sits at position Lp[b] + j0 + j, writes its K/V
//                 into slot j0 + j of beam i's suffix blocks and attends to
//                 the prefix [0, Lp[b]) plus its beam's slots [0, j0 + j].
// --------------------------------------------------------------------------
enum PassMode { kAppend = 0, kSuffix = 1 };

struct PassDesc {
  int mode;
  int nb, kp, R, j0;
  const int* prompt_ids;   // [nb] or null (identity)
  const int* Lp;           // [B] prefix length before this pass
  const int* ptable;       // [B][ptable_stride] prefix block ids
  int ptable_stride;
  const int* stable;       // [Bmax][kmax][sblocks] suffix block ids
  int s_stride_b, s_stride_i, sblocks;
  // token of row m: tok[(b * kp + i) * tok_stride + tok_off + j]
  const int* tok;
  int tok_stride, tok_off;
  int* bad;                // set to 1 when a fed token id lies outside [0, V) (may be null)
  int M() const { return nb * kp * R; }
};

__host__ __device__ inline int pass_batch(const PassDesc& p, int bi) {
  return p.prompt_ids ? p.prompt_ids[bi] : bi;
}

// Row m of a pass as (prompt slot bi, batch index b, beam i, row j).
__device__ __forceinline__ void row_decode(const PassDesc& p, int m, int& bi, int& b, int& i, int& j) {
  j = m % p.R;
  const int t = m / p.R;
  i = t % p.kp;
  bi = t / p.kp;
  b = pass_batch(p, bi);
}

// KV block, slot in the block, and position of row (b, i, j) of a pass whose
// prompt b has Lp prefix tokens: a suffix slot j0 + j of beam i, or prefix
// position Lp + j.
__device__ __forceinline__ void kv_slot(const PassDesc& p, int b, int i, int j, int Lp, int& blk, int& slot,
                                        int& pos) {
  if (p.mode == kSuffix) {
    const int s = p.j0 + j;
    pos = Lp + s;
    blk = p.stable[(long long)b * p.s_stride_b + i * p.s_stride_i + s / kBlock];
    slot = s % kBlock;
  } else {
    pos = Lp + j;
    blk = p.ptable[(long long)b * p.ptable_stride + pos / kBlock];
    slot = pos % kBlock;
  }
}

// Rotary embedding of the pair (x1, x2) = (x[d], x[d + hd/2]) at angle
// theta with c = cos(theta), s = sin(theta):
//   y1 = x1 c - x2 s,  y2 = x2 c + x1 s.
// Written with explicit fused multiply-adds so that every kernel that
// rotates (the rotary kernels and the q/k/v projection's epilogue) rounds
// the same way.
__device__ __forceinline__ float rope_first(float x1, float x2, float c, float s) { return fmaf(x1, c, -(x2 * s)); }
__device__ __forceinline__ float rope_second(float x1, float x2, float c, float s) { return fmaf(x2, c, x1 * s); }

// Index of row m of a pass into a [B][kp][stride] token array:
// (b * kp + i) * stride + off + j.  Disabled: index = m.
struct RowMap {
  int enabled;
  PassDesc p;
  int stride, off;
};

__host__ __device__ inline long long rowmap_index(const RowMap& r, int m) {
  if (!r.enabled) return m;
  const int j = m % r.p.R;
  const int t = m / r.p.R;
  const int i = t % r.p.kp;
  const int bi = t / r.p.kp;
  const int b = r.p.prompt_ids ? r.p.prompt_ids[bi] : bi;
  return (long long)(b * r.p.kp + i) * r.stride + r.off + j;
}

// Per-row statistics of a logit matrix, kept per column tile so that the
// logits themselves never reach memory (the LM-head GEMM writes these in
// its epilogue; a merge kernel folds the tiles).  For row m and tile t:
//   mx[m * tiles + t]   largest value of the tile's columns
//   se[m * tiles + t]   sum of exp(v - mx) over them
//   am[m * tiles + t]   lowest column holding mx
//   tv/tc[(m * tiles + t) * kk + u]  the tile's kk best (value descending,
//                        column ascending), kk <= 16; unused slots -inf
//   zx[m]               the value at column gather_tok[rowmap(gather_map, m)]
//                        (written by the tile that holds it; gather_tok null:
//                        no gather)
struct RowStats {
  float* mx;
  float* se;
  int* am;
  float* tv;
  int* tc;
  int kk;
  int tiles;
  float* zx;
  const int* gather_tok;
  RowMap gather_map;
};

// KV pool of one model: per layer, per block, per KV head:
//   K: [16 tokens][hd]            (key-major, hd contiguous)
//   V: [hd][16 tokens]            (transposed: token contiguous)
// so that both MFMA operands of attention read 8/16-byte runs.
struct KVPool {
  void* k;                 // base of layer 0
  void* v;
  long long layer_elems;   // elements per layer = nblocks * Hkv * 16 * hd
  int Hkv, hd;
};

// KV pool format of bf16-weight models.  A unit (layer, block, KV head) has
// the byte size of the fp32 unit (16 * hd * 4 bytes) and holds each fp32
// value as a bf16 (hi, lo) pair, plane by plane:
//   K unit: [hi | lo][16 tokens][hd]
//   V unit: [hi | lo][hd][16 tokens]
__host__ __device__ inline long long split_unit_elems(int hd) { return 2LL * kBlock * hd; }

template <typename T>
__device__ __forceinline__ float to_f32(T x);
template <>
__device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f32<bf16>(bf16 x) { return (float)x; }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// An fp32 activation as the bf16 pair (hi, lo) with x ~= hi + lo to about
// 2^-17 relative.  Weights are exactly bf16, so a projection over split
// activations (hi * W + lo * W, two MFMA products) keeps fp32-level accuracy.
__device__ __forceinline__ void split_bf16(float x, bf16& hi, bf16& lo) {
  hi = (bf16)x;
  lo = (bf16)(x - (float)hi);
}

// Slots [slot, slot + n) of one dim row of a V unit in the split KV format
// (hi plane at row[0..16), lo plane at row[plane..plane + 16)), from vv[t]
// for slot t; entries outside the run are ignored.  The widest stores that
// stay inside the run: whole 8-slot halves as 16 bytes, else slot pairs as
// 4 bytes, else single slots.
__device__ __forceinline__ void store_v_run(bf16* row, long long plane, const float (&vv)[kBlock], int slot, int n) {
  bf16 vh[kBlock], vlo[kBlock];
#pragma unroll
  for (int t = 0; t < kBlock; ++t) {
    bf16 h, l;
    split_bf16(vv[t], h, l);
    const bool in = t >= slot && t < slot + n;
    vh[t] = in ? h : (bf16)0.f;
    vlo[t] = in ? l : (bf16)0.f;
  }
#pragma unroll
  for (int h8 = 0; h8 < 2; ++h8) {
    const int t0 = h8 * 8;
    if (t0 >= slot && t0 + 8 <= slot + n) {
      bf16x8 a, c;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a[e] = vh[t0 + e];
        c[e] = vlo[t0 + e];
      }
      *(bf16x8*)(row + t0) = a;
      *(bf16x8*)(row + plane + t0) = c;
    } else {
#pragma unroll
      for (int t = t0; t < t0 + 8; t += 2) {
        const bool in0 = t >= slot && t < slot + n, in1 = t + 1 >= slot && t + 1 < slot + n;
        if (in0 && in1) {
          bf16x2v a = {vh[t], vh[t + 1]}, c = {vlo[t], vlo[t + 1]};
          *(bf16x2v*)(row + t) = a;
          *(bf16x2v*)(row + plane + t) = c;
        } else if (in0) {
          row[t] = vh[t];
          row[plane + t] = vlo[t];
        } else if (in1) {
          row[t + 1] = vh[t + 1];
          row[plane + t + 1] = vlo[t + 1];
        }
      }
    }
  }
}

// (value, id) ordering used by every argmax / top-k: larger value first,
// then smaller id.
__device__ __forceinline__ bool vi_better(float a, int ia, float b, int ib) {
  return a > b || (a == b && ia < ib);
}

}  // namespace cdsl
