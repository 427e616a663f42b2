// Projections of the decoders: C[M,N] = A[M,K] * B[N,K]^T, fp32 accumulate.
//
// Both operands are K-contiguous ([rows][K] row-major), which is what the
// CDNA4 MFMA fragments want: lane (r, g) of v_mfma_f32_16x16x32_bf16 holds 8
// consecutive K elements of row r, so every fragment is one 16-byte load.
//
// Two bf16 kernels:
//   dense  (M > 128): 128x128 tiles, 4 waves (2x2) of 64x64, BK = 64, both
//          operands staged through double-buffered LDS.  Arithmetic
//          intensity ~M flop/B: the verification block and prefill.
//   skinny (M <= 128): the decode shape of the draft rollout.  Weight
//          streaming bound: every weight byte is read once, straight into
//          registers with 8-deep prefetch, while the small activation tile
//          sits in LDS and is shared by the 4 waves of a workgroup.
// Both split K across workgroups when the tile grid alone cannot fill the
// 256 CUs.  Split partials go to a workspace and the LAST workgroup to
// arrive on a tile (arrival counter) sums them in split order, so results are
// bitwise deterministic, then applies the epilogue.
#include "common.h"
#include "gemm.h"

namespace cdsl {

namespace {

constexpr int kPad = 8;
// Workspace layout: arrival counters first (a fixed region shared by every
// shape, so one GEMM's partials never land on another's counters), then the
// split partials.  Counters return to zero after each use.
constexpr int kMaxCounters = 4096;
constexpr size_t kCounterBytes = kMaxCounters * sizeof(int);

struct GemmArgs {
  const float* A;
  const bf16* B;
  int M, N, K;
  void* C;
  int ldc;
  int epi;
  int ksplit, kchunk;
  float* partial;
  int* counters;
  int tiles_n;
};

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }

// Epilogue for one output element pair.  For kSwiGLU the packed weight puts
// 16 gate rows then the 16 matching up rows in every group of 32, so the
// accumulator tiles tn (gate) and tn+1 (up) of a lane hold the same feature.
__device__ __forceinline__ void epi_store(const GemmArgs& a, int row, int col, float v) {
  if (row >= a.M || col >= a.N) return;
  float* C = (float*)a.C;
  long long idx = (long long)row * a.ldc + col;
  if (a.epi == kEpiResidual) C[idx] += v;
  else C[idx] = v;
}

__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, int row, int col_gate, float g, float u) {
  if (row >= a.M || col_gate >= a.N) return;
  int f = (col_gate >> 5) * 16 + (col_gate & 15);
  ((float*)a.C)[(long long)row * a.ldc + f] = silu(g) * u;
}

// Split-K fixup.  Every workgroup of a tile stores its NV accumulator
// vectors to partial[(tile * S + z) * (NV * 4 * 256) + (v * 4 + c) * 256 +
// tid]; the last to arrive returns true with acc[] replaced by the in-order
// sum over splits.
template <int NV>
__device__ __forceinline__ bool splitk_reduce(const GemmArgs& a, int tile, f32x4* acc) {
  if (a.ksplit == 1) return true;
  const int tid = threadIdx.x;
  const int z = blockIdx.z;
  constexpr int NE = NV * 4 * 256;
  float* mine = a.partial + ((long long)tile * a.ksplit + z) * NE;
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int c = 0; c < 4; ++c) mine[(v * 4 + c) * 256 + tid] = acc[v][c];
  __threadfence();
  __syncthreads();
  __shared__ int s_last;
  if (tid == 0) {
    int prev = atomicAdd(&a.counters[tile], 1);
    s_last = (prev == a.ksplit - 1);
  }
  __syncthreads();
  if (!s_last) return false;
  __threadfence();
  f32x4 sum[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) sum[v] = (f32x4){0.f, 0.f, 0.f, 0.f};
  for (int zz = 0; zz < a.ksplit; ++zz) {
    const float* p = a.partial + ((long long)tile * a.ksplit + zz) * NE;
    if (zz == z) {
#pragma unroll
      for (int v = 0; v < NV; ++v) sum[v] += acc[v];
    } else {
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[v][c] += __builtin_nontemporal_load(p + (v * 4 + c) * 256 + tid);
    }
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) acc[v] = sum[v];
  if (tid == 0) atomicExch(&a.counters[tile], 0);
  return true;
}

// Split an fp32 value into bf16 hi + lo with x ~= hi + lo to ~2^-17
// relative: the activation operand keeps fp32-level precision while both
// MFMA operands stay bf16 (weights are exactly bf16).
__device__ __forceinline__ void split_bf16(float x, bf16& hi, bf16& lo) {
  hi = (bf16)x;
  lo = (bf16)(x - (float)hi);
}

__device__ __forceinline__ void split4(const float4& v, bf16x4& hi, bf16x4& lo) {
  bf16 h0, h1, h2, h3, l0, l1, l2, l3;
  split_bf16(v.x, h0, l0);
  split_bf16(v.y, h1, l1);
  split_bf16(v.z, h2, l2);
  split_bf16(v.w, h3, l3);
  hi = (bf16x4){h0, h1, h2, h3};
  lo = (bf16x4){l0, l1, l2, l3};
}

// ---------------------------------------------------------------------------
// dense kernel: 128 x 128 x 32 tiles, 2 x 2 waves of 64 x 64
// ---------------------------------------------------------------------------
constexpr int DBM = 128, DBN = 128, DBK = 32;
constexpr int DTM = 4, DTN = 4;   // 16x16 tiles per wave
constexpr int DLD = DBK + kPad;   // LDS row stride (conflict-free fragment reads)

__global__ __launch_bounds__(256) void gemm_bf16_dense(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) bf16 Ah[2][DBM][DLD];
  __shared__ __attribute__((aligned(16))) bf16 Al[2][DBM][DLD];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][DBN][DLD];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int tile = blockIdx.x;
  const int tm_blk = tile / a.tiles_n, tn_blk = tile % a.tiles_n;
  const int m0 = tm_blk * DBM, n0 = tn_blk * DBN;
  const int kbeg = blockIdx.z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nk = (kend - kbeg) / DBK;

  // global -> registers: A 128 x 32 fp32 (4 x 16 B per thread),
  // B 128 x 32 bf16 (2 x 16 B per thread)
  float4 ra[4];
  uint4 rb[2];
  auto gload = [&](int kt) {
    const int k0 = kbeg + kt * DBK;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u;
      const int row = c >> 3, cc = c & 7;
      const int gm = m0 + row;
      ra[u] = gm < a.M ? *(const float4*)(a.A + (long long)gm * a.K + k0 + cc * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = tid + 256 * u;
      const int row = c >> 2, cc = c & 3;
      const int gn = n0 + row;
      rb[u] = gn < a.N ? *(const uint4*)(a.B + (long long)gn * a.K + k0 + cc * 8) : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u;
      const int row = c >> 3, cc = c & 7;
      bf16x4 hi, lo;
      split4(ra[u], hi, lo);
      *(bf16x4*)&Ah[buf][row][cc * 4] = hi;
      *(bf16x4*)&Al[buf][row][cc * 4] = lo;
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = tid + 256 * u;
      const int row = c >> 2, cc = c & 3;
      *(uint4*)&Bs[buf][row][cc * 8] = rb[u];
    }
  };

  f32x4 acc[DTM * DTN];
#pragma unroll
  for (int v = 0; v < DTM * DTN; ++v) acc[v] = (f32x4){0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lg = lane >> 4;
  if (nk > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
    bf16x8 ah[DTM], al[DTM], bw[DTN];
#pragma unroll
    for (int i = 0; i < DTM; ++i) {
      ah[i] = *(const bf16x8*)&Ah[cur][wm * 64 + i * 16 + lr][lg * 8];
      al[i] = *(const bf16x8*)&Al[cur][wm * 64 + i * 16 + lr][lg * 8];
    }
#pragma unroll
    for (int j = 0; j < DTN; ++j) bw[j] = *(const bf16x8*)&Bs[cur][wn * 64 + j * 16 + lr][lg * 8];
#pragma unroll
    for (int i = 0; i < DTM; ++i)
#pragma unroll
      for (int j = 0; j < DTN; ++j) {
        acc[i * DTN + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[i], bw[j], acc[i * DTN + j], 0, 0, 0);
        acc[i * DTN + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], bw[j], acc[i * DTN + j], 0, 0, 0);
      }
    if (kt + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  if (!splitk_reduce<DTM * DTN>(a, tile, acc)) return;

#pragma unroll
  for (int i = 0; i < DTM; ++i) {
#pragma unroll
    for (int j = 0; j < DTN; ++j) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = m0 + wm * 64 + i * 16 + lg * 4 + e;
        const int col = n0 + wn * 64 + j * 16 + lr;
        if (a.epi == kEpiSwiGLU) {
          if ((j & 1) == 0) epi_swiglu(a, row, col, acc[i * DTN + j][e], acc[i * DTN + j + 1][e]);
        } else {
          epi_store(a, row, col, acc[i * DTN + j][e]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// skinny kernel: MT x 16 rows, 64 columns per workgroup (16 per wave)
// ---------------------------------------------------------------------------
template <int MT>
struct SkinnyCfg {
  static constexpr int KC = MT <= 4 ? 256 : 128;   // K per chunk (LDS budget)
};

template <int MT>
__global__ __launch_bounds__(256) void gemm_bf16_skinny(GemmArgs a) {
  constexpr int BM = MT * 16;
  constexpr int KC = SkinnyCfg<MT>::KC;
  constexpr int KS = KC / 32;   // MFMA k-steps per chunk
  constexpr int LD = KC + kPad;
  __shared__ __attribute__((aligned(16))) bf16 Ah[BM][LD];
  __shared__ __attribute__((aligned(16))) bf16 Al[BM][LD];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int tile = blockIdx.x;                  // column block
  const int m0 = blockIdx.y * BM;
  const int n0 = tile * 64 + wave * 16;
  const int kbeg = blockIdx.z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nchunk = (kend - kbeg) / KC;

  const int brow = n0 + lr;
  const bf16* bptr = a.B + (long long)min(brow, a.N - 1) * a.K + lg * 8;

  bf16x8 bcur[KS], bnxt[KS];
  auto bload = [&](bf16x8* dst, int c) {
    const int k0 = kbeg + c * KC;
#pragma unroll
    for (int s = 0; s < KS; ++s) dst[s] = *(const bf16x8*)(bptr + k0 + s * 32);
  };

  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = (f32x4){0.f, 0.f, 0.f, 0.f};

  if (nchunk > 0) bload(bcur, 0);
  for (int c = 0; c < nchunk; ++c) {
    if (c + 1 < nchunk) bload(bnxt, c + 1);
    // activation chunk (fp32) -> hi/lo bf16 in LDS
    const int k0 = kbeg + c * KC;
    constexpr int CH = BM * (KC / 4);
#pragma unroll
    for (int u = 0; u < (CH + 255) / 256; ++u) {
      const int ci = tid + 256 * u;
      if (ci < CH) {
        const int row = ci / (KC / 4), cc = ci % (KC / 4);
        const int gm = m0 + row;
        float4 v = gm < a.M ? *(const float4*)(a.A + (long long)gm * a.K + k0 + cc * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
        bf16x4 hi, lo;
        split4(v, hi, lo);
        *(bf16x4*)&Ah[row][cc * 4] = hi;
        *(bf16x4*)&Al[row][cc * 4] = lo;
      }
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < KS; ++s) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const bf16x8 ah = *(const bf16x8*)&Ah[i * 16 + lr][s * 32 + lg * 8];
        const bf16x8 al = *(const bf16x8*)&Al[i * 16 + lr][s * 32 + lg * 8];
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bcur[s], acc[i], 0, 0, 0);
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bcur[s], acc[i], 0, 0, 0);
      }
    }
    __syncthreads();
    if (c + 1 < nchunk) {
#pragma unroll
      for (int s = 0; s < KS; ++s) bcur[s] = bnxt[s];
    }
  }

  const int tile_id = blockIdx.y * gridDim.x + tile;
  if (!splitk_reduce<MT>(a, tile_id, acc)) return;

  if (a.epi == kEpiSwiGLU) {
    // gate = wave tile with (wave & 1) == 0, up = the next wave's tile: swap
    // through LDS (the activation buffer is free by now) so the gate wave
    // owns both.
    static_assert(sizeof(float) * 2 * MT * 4 * 64 <= sizeof(Ah), "exchange fits");
    float (*xch)[MT * 4][64] = reinterpret_cast<float (*)[MT * 4][64]>(&Ah[0][0]);
    if (wave & 1) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) xch[wave >> 1][i * 4 + e][lane] = acc[i][e];
    }
    __syncthreads();
    if ((wave & 1) == 0) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int row = m0 + i * 16 + lg * 4 + e;
          epi_swiglu(a, row, n0 + lr, acc[i][e], xch[wave >> 1][i * 4 + e][lane]);
        }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) epi_store(a, m0 + i * 16 + lg * 4 + e, n0 + lr, acc[i][e]);
}

// ---------------------------------------------------------------------------
// fp32 kernel (the fp32 workload): 64x64 tiles, 4x4 outputs per thread
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemm_f32_tiled(const float* __restrict__ A, const float* __restrict__ B,
                                                       float* __restrict__ C, int M, int N, int K, int ldc,
                                                       int epi) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      int idx = tid + 256 * u;        // 64 rows x 16 k
      int r = idx >> 4, kk = idx & 15;
      int gm = m0 + r, gn = n0 + r;
      As[kk][r] = gm < M ? A[(long long)gm * K + k0 + kk] : 0.f;
      Bs[kk][r] = gn < N ? B[(long long)gn * K + k0 + kk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
      if (row < M && col < N) {
        long long idx = (long long)row * ldc + col;
        if (epi == kEpiResidual) C[idx] += acc[i][j];
        else C[idx] = acc[i][j];
      }
    }
}

// act[m, f] = silu(g) * u for the fp32 path, reading the packed [M, 2F]
// product (groups of 16 gate columns followed by their 16 up columns).
__global__ void swiglu_f32(const float* __restrict__ gu, float* __restrict__ act, int M, int F) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (long long)M * F) return;
  int m = (int)(i / F), f = (int)(i % F);
  int col = (f >> 4) * 32 + (f & 15);
  float g = gu[(long long)m * 2 * F + col], u = gu[(long long)m * 2 * F + col + 16];
  act[i] = silu(g) * u;
}

struct Plan {
  int kind;          // 0 dense, 1 skinny, 2 f32
  int mt;            // skinny row tiles
  int tiles_m, tiles_n;
  int ksplit, kchunk;
  size_t ws_bytes;
};

Plan make_plan(int M, int N, int K, int dtype) {
  Plan p{};
  if (dtype == 0) {
    p.kind = 2;
    return p;
  }
  const int target_wg = 512;
  const int mt = (M + 15) / 16;
  const int kc = mt <= 4 ? 256 : 128;   // SkinnyCfg<mt>::KC
  if (M <= 128 && K % kc == 0) {
    p.kind = 1;
    p.mt = mt;
    p.tiles_m = 1;
    p.tiles_n = (N + 63) / 64;
    const int nchunks = K / kc;
    int s = (target_wg + p.tiles_n - 1) / p.tiles_n;
    s = max(1, min(s, nchunks));
    const int per = (nchunks + s - 1) / s;
    s = (nchunks + per - 1) / per;
    p.ksplit = s;
    p.kchunk = per * kc;
    if (s > 1) p.ws_bytes = kCounterBytes + (size_t)p.tiles_n * s * (p.mt * 4 * 256) * sizeof(float);
  } else {
    p.kind = 0;
    p.tiles_m = (M + DBM - 1) / DBM;
    p.tiles_n = (N + DBN - 1) / DBN;
    const int tiles = p.tiles_m * p.tiles_n;
    const int nk = K / DBK;
    int s = 1;
    if (tiles < 256) s = min((target_wg + tiles - 1) / tiles, max(1, nk / 8));
    const int per = (nk + s - 1) / s;
    s = (nk + per - 1) / per;
    p.ksplit = s;
    p.kchunk = per * DBK;
    if (s > 1) p.ws_bytes = kCounterBytes + (size_t)tiles * s * (DTM * DTN * 4 * 256) * sizeof(float);
  }
  return p;
}

}  // namespace

size_t gemm_workspace_bytes(int M, int N, int K, int dtype) {
  if (dtype == 0 || M <= 0) return 0;
  size_t b = make_plan(M, N, K, dtype).ws_bytes;
  return (b + 255) & ~(size_t)255;
}

int gemm_kind(int M, int N, int K, int dtype) { return make_plan(M, N, K, dtype).kind; }

int gemm_check(int M, int N, int K, int dtype) {
  if (M < 0 || N <= 0 || K <= 0) return -1;
  if (dtype == 1 && K % 32 != 0) return -1;
  if (dtype == 0 && K % 16 != 0) return -1;
  return 0;
}

hipError_t gemm_launch(const void* A, const void* B, void* C, int M, int N, int K, int ldc, int dtype, int epi,
                       void* ws, size_t ws_bytes, hipStream_t st) {
  if (M == 0) return hipSuccess;
  Plan p = make_plan(M, N, K, dtype);
  if (p.kind == 2) {
    if (epi == kEpiSwiGLU) return hipErrorInvalidValue;  // fp32 path: store + swiglu_f32
    dim3 grid((N + 63) / 64, (M + 63) / 64);
    gemm_f32_tiled<<<grid, 256, 0, st>>>((const float*)A, (const float*)B, (float*)C, M, N, K, ldc, epi);
    return hipGetLastError();
  }
  if (p.ws_bytes > ws_bytes) return hipErrorInvalidValue;
  GemmArgs a;
  a.A = (const float*)A;
  a.B = (const bf16*)B;
  a.M = M;
  a.N = N;
  a.K = K;
  a.C = C;
  a.ldc = ldc;
  a.epi = epi;
  a.ksplit = p.ksplit;
  a.kchunk = p.kchunk;
  a.tiles_n = p.tiles_n;
  const int tiles = p.tiles_m * p.tiles_n;
  if (p.ksplit > 1 && tiles > kMaxCounters) return hipErrorInvalidValue;
  a.counters = (int*)ws;
  a.partial = (float*)((char*)ws + kCounterBytes);
  if (p.kind == 0) {
    dim3 grid(tiles, 1, p.ksplit);
    gemm_bf16_dense<<<grid, 256, 0, st>>>(a);
  } else {
    dim3 grid(p.tiles_n, 1, p.ksplit);
    switch (p.mt) {
      case 1: gemm_bf16_skinny<1><<<grid, 256, 0, st>>>(a); break;
      case 2: gemm_bf16_skinny<2><<<grid, 256, 0, st>>>(a); break;
      case 3: gemm_bf16_skinny<3><<<grid, 256, 0, st>>>(a); break;
      case 4: gemm_bf16_skinny<4><<<grid, 256, 0, st>>>(a); break;
      case 5: gemm_bf16_skinny<5><<<grid, 256, 0, st>>>(a); break;
      case 6: gemm_bf16_skinny<6><<<grid, 256, 0, st>>>(a); break;
      case 7: gemm_bf16_skinny<7><<<grid, 256, 0, st>>>(a); break;
      default: gemm_bf16_skinny<8><<<grid, 256, 0, st>>>(a); break;
    }
  }
  return hipGetLastError();
}

hipError_t swiglu_f32_launch(const float* gu, float* act, int M, int F, hipStream_t st) {
  long long n = (long long)M * F;
  if (n == 0) return hipSuccess;
  swiglu_f32<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(gu, act, M, F);
  return hipGetLastError();
}

}  // namespace cdsl
