// Projections of the decoders: C[M,N] = A[M,K] * W[N,K]^T, fp32 accumulate.
//
// For bf16-weight models the activation operand arrives as two bf16 planes,
// A = A_hi + A_lo (written that way by the kernel that produced it), and
// every MFMA step is done twice (A_hi * W, A_lo * W) into one fp32
// accumulator: the weights are exactly bf16, so the product keeps
// fp32-level accuracy at twice the MFMA work of a plain bf16 product.
//
// Both operands are K-contiguous ([rows][K] row-major), which is what the
// CDNA4 MFMA fragments want: lane (r, g) of v_mfma_f32_16x16x32_bf16 holds 8
// consecutive K elements of row r, so every fragment is one 16-byte load.
//
//   dense  (M > 128): 128 x 128 tiles, 4 waves (2 x 2) of 64 x 64, K step
//          32, double-buffered LDS fed from registers two K steps ahead.
//          Arithmetic intensity ~M flop/B: the verification block, prefill.
//   skinny (M <= 128): the decode rows of the draft rollout.  Weight
//          streaming bound: each wave owns 16 columns and keeps four K
//          stages of weight fragments in flight in registers, straight from
//          HBM; the small activation block is staged once per K stage in
//          LDS and shared by the 4 waves.  Loads are issued in the order they
//          are consumed so the in-order vmcnt waits never stall on a later
//          prefetch.
// When the tile grid cannot fill the 256 CUs, K is split across workgroups;
// each split writes its own fp32 plane and a reduce kernel sums the planes
// in split order and applies the epilogue (bitwise deterministic).
#include <stdlib.h>

#include <type_traits>

#include "common.h"
#include "gemm.h"

namespace cdsl {

namespace {

constexpr int kPad = 8;

struct GemmArgs {
  const bf16* Ahi;
  const bf16* Alo;
  const bf16* B;
  int M, N, K;
  void* C;          // fp32 [M, ldc] (store / residual)
  bf16* Chi;        // SwiGLU output planes [M, ldc]
  bf16* Clo;
  int ldc;
  int epi;
  int ksplit, kchunk;
  float* partial;   // split planes [ksplit][M][N]
  int tiles_m, tiles_n;
};

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }

__device__ __forceinline__ void epi_store(const GemmArgs& a, int row, int col, float v) {
  if (row >= a.M || col >= a.N) return;
  float* C = (float*)a.C;
  long long idx = (long long)row * a.ldc + col;
  if (a.epi == kEpiResidual) C[idx] += v;
  else C[idx] = v;
}

// The packed gate/up weight puts 16 gate rows then the 16 matching up rows in
// every group of 32, so output column f of silu(gate) * up pairs packed
// columns 32*(f/16) + f%16 and that + 16.
__device__ __forceinline__ void epi_swiglu(const GemmArgs& a, int row, int col_gate, float g, float u) {
  if (row >= a.M || col_gate >= a.N) return;
  const int f = (col_gate >> 5) * 16 + (col_gate & 15);
  bf16 h, l;
  split_bf16(silu(g) * u, h, l);
  a.Chi[(long long)row * a.ldc + f] = h;
  a.Clo[(long long)row * a.ldc + f] = l;
}

__device__ __forceinline__ void part_store(const GemmArgs& a, int row, int col, float v) {
  if (row >= a.M || col >= a.N) return;
  a.partial[((long long)blockIdx.z * a.M + row) * a.N + col] = v;
}

__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long plane = (long long)a.M * a.N;
  if (a.epi == kEpiSwiGLU) {
    const int F = a.N / 2;
    if (i >= (long long)a.M * F) return;
    const int row = (int)(i / F), f = (int)(i % F);
    const int cg = (f >> 4) * 32 + (f & 15);
    const long long ig = (long long)row * a.N + cg;
    float g = 0.f, u = 0.f;
    for (int z = 0; z < a.ksplit; ++z) {
      g += a.partial[z * plane + ig];
      u += a.partial[z * plane + ig + 16];
    }
    bf16 h, l;
    split_bf16(silu(g) * u, h, l);
    a.Chi[(long long)row * a.ldc + f] = h;
    a.Clo[(long long)row * a.ldc + f] = l;
    return;
  }
  if (i >= plane) return;
  float v = 0.f;
  for (int z = 0; z < a.ksplit; ++z) v += a.partial[z * plane + i];
  const int row = (int)(i / a.N), col = (int)(i % a.N);
  float* C = (float*)a.C + (long long)row * a.ldc + col;
  if (a.epi == kEpiResidual) *C += v;
  else *C = v;
}

template <int I>
using ic = std::integral_constant<int, I>;

// ---------------------------------------------------------------------------
// dense kernel: WM x WN waves, each owning TM x TN tiles of 16 x 16; K step 32
//
// Block tile BM x BN = (WM * TM * 16) x (WN * TN * 16).  A_hi, A_lo and W
// tiles of one K step are staged through double-buffered LDS in an
// XOR-swizzled layout (16-byte chunk c of row r stored at chunk
// c ^ ((r >> 1) & 3) of a 64-byte row): any 8 consecutive rows then cover
// all 32 banks once, so both the staging writes and the fragment reads are
// free of bank conflicts; the staging itself runs two
// K steps ahead in registers.  Large tiles matter here because the
// activation operand costs 4 bytes per element (hi + lo planes) and is
// re-read once per column block.
// ---------------------------------------------------------------------------
constexpr int DBK = 32;   // K granularity of splits (one MFMA k-step)

// 16-byte chunk c of row r (rows of KC bf16 = KC/8 chunks) sits at chunk
// c ^ (r & (KC/8 - 1)) for 128-byte rows, c ^ ((r >> 1) & 3) for 64-byte
// rows: 8 consecutive rows then cover the 32 banks exactly once.
template <int KC>
__device__ __forceinline__ int swz(int row, int chunk) {
  if constexpr (KC == 64) return row * KC + ((chunk ^ (row & 7)) << 3);
  else return row * KC + ((chunk ^ ((row >> 1) & 3)) << 3);
}

template <int WM, int WN, int TM, int TN, int KC>
struct DenseCfg {
  static constexpr int NT = 64 * WM * WN;          // threads
  static constexpr int BM = WM * TM * 16, BN = WN * TN * 16;
  static constexpr int CPR = KC / 8;               // 16-byte chunks per row
  static constexpr int ACH = BM * CPR, BCH = BN * CPR;
  static constexpr int CH = 2 * ACH + BCH;         // hi + lo + weights
  static constexpr int PER = (CH + NT - 1) / NT;   // chunks per thread
};

template <int WM, int WN, int TM, int TN, int KC, int PREFILL>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_dense(GemmArgs a) {
  using C = DenseCfg<WM, WN, TM, TN, KC>;
  constexpr int BM = C::BM, BN = C::BN, PER = C::PER, CPR = C::CPR;
  // one LDS stage: A_hi [BM][KC], A_lo [BM][KC], W [BN][KC], then one
  // 16-byte slot per thread for the padding chunks of the staging pattern
  constexpr int OFF_LO = BM * KC, OFF_B = 2 * BM * KC, OFF_PAD = (2 * BM + BN) * KC;
  constexpr int STAGE = OFF_PAD + C::NT * 8;
  __shared__ __attribute__((aligned(16))) bf16 lds[2][STAGE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lr = lane & 15, lg = lane >> 4;
  // XCD-aware tile order.  Workgroups are dispatched round-robin over the 8
  // XCDs (each with its own L2), so workgroup p runs on XCD p % 8.  Give each
  // XCD a contiguous range of logical tiles, ordered with the row block
  // fastest: the tiles an XCD runs together then share weight column blocks
  // (and the few activation row blocks) through its L2 instead of fetching
  // them once per tile (measured: 894 MB -> 224 MB of HBM reads for the
  // 800 x 22016 x 4096 projection).
  const int T = a.tiles_m * a.tiles_n;
  const int p = blockIdx.x, xcd = p & 7, slot = p >> 3;
  const int per = T >> 3, rem = T & 7;
  const int tile = xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
  const int tm_blk = tile % a.tiles_m, tn_blk = tile / a.tiles_m;
  const int m0 = tm_blk * BM, n0 = tn_blk * BN;
  const int kbeg = blockIdx.z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nk = (kend - kbeg) / KC;

  // staging assignment: chunk q of the K stage -> plane, row, 16-byte column.
  // Rows past M (N) are clamped to the last row: they only feed outputs the
  // epilogue discards.  Threads without a chunk in some slot load a valid
  // dummy and store it to their pad slot, so the loop has no branches around
  // memory operations.
  const bf16* src[PER];
  int dst[PER];   // LDS element offset within a stage
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int q = tid + C::NT * u;
    int plane, row, ch;
    if (q < C::ACH) {
      plane = 0; row = q / CPR; ch = q % CPR;
    } else if (q < 2 * C::ACH) {
      plane = 1; row = (q - C::ACH) / CPR; ch = q % CPR;
    } else if (q < C::CH) {
      plane = 2; row = (q - 2 * C::ACH) / CPR; ch = q % CPR;
    } else {
      plane = -1; row = 0; ch = 0;
    }
    dst[u] = plane == 0 ? swz<KC>(row, ch)
             : plane == 1 ? OFF_LO + swz<KC>(row, ch)
             : plane == 2 ? OFF_B + swz<KC>(row, ch)
                          : OFF_PAD + tid * 8;
    const bf16* base = plane == 1 ? a.Alo : plane == 2 ? a.B : a.Ahi;
    const int lim = plane == 2 ? a.N - 1 : a.M - 1;
    const int r0 = plane == 2 ? n0 : m0;
    src[u] = base + (long long)min(r0 + row, lim) * a.K + kbeg + ch * 8;
  }

  u32x4 r0[PER], r1[PER];
  auto gload = [&](u32x4* r, int kt) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PER; ++u) r[u] = *(const u32x4*)(src[u] + kt * KC);
  };
  auto sstore = [&](const u32x4* r, int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < PER; ++u) *(u32x4*)&lds[buf][dst[u]] = r[u];
  };

  f32x4 acc[TM * TN];
#pragma unroll
  for (int v = 0; v < TM * TN; ++v) acc[v] = (f32x4){0.f, 0.f, 0.f, 0.f};

  // all fragments of a 32-deep k-step are read before its MFMAs (one LDS
  // latency per k-step instead of one per row tile)
  auto mma = [&](int cur) __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < KC / 32; ++s) {
      bf16x8 bf[TN], ah[TM], al[TM];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *(const bf16x8*)&lds[cur][OFF_B + swz<KC>(wn * TN * 16 + j * 16 + lr, s * 4 + lg)];
#pragma unroll
      for (int t = 0; t < TM; ++t) {
        const int row = wm * TM * 16 + t * 16 + lr;
        ah[t] = *(const bf16x8*)&lds[cur][swz<KC>(row, s * 4 + lg)];
        al[t] = *(const bf16x8*)&lds[cur][OFF_LO + swz<KC>(row, s * 4 + lg)];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[t * TN + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[t], bf[j], acc[t * TN + j], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[t * TN + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[t], bf[j], acc[t * TN + j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // K stage kt: LDS buffer kt & 1; staging set (kt & 1) receives stage kt + 2
  // (clamped to the last stage: those loads are never stored) while the other
  // set, holding stage kt + 1, moves to the other buffer
  if (nk > 0) {
    gload(r0, 0);
    gload(r1, min(1, nk - 1));
    sstore(r0, 0);
    __syncthreads();
  }
  // the scheduling barriers keep each prefetch issued ahead of the MFMAs
  // (left alone, the scheduler sinks the loads below them, which shortens
  // the prefetch distance to a single stage)
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    gload(r0, min(kt + 2, nk - 1));
    __builtin_amdgcn_sched_barrier(0);
    mma(0);
    __builtin_amdgcn_sched_barrier(0);
    sstore(r1, 1);
    __syncthreads();
    gload(r1, min(kt + 3, nk - 1));
    __builtin_amdgcn_sched_barrier(0);
    mma(1);
    __builtin_amdgcn_sched_barrier(0);
    sstore(r0, 0);
    __syncthreads();
  }
  if (kt < nk) mma(0);   // odd number of stages: the last one is in buffer 0

  const int rbase = m0 + wm * TM * 16 + lg * 4, cbase = n0 + wn * TN * 16 + lr;
  if (a.ksplit > 1) {
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) part_store(a, rbase + t * 16 + e, cbase + j * 16, acc[t * TN + j][e]);
    return;
  }
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = rbase + t * 16 + e, col = cbase + j * 16;
        if (a.epi == kEpiSwiGLU) {
          if ((j & 1) == 0) epi_swiglu(a, row, col, acc[t * TN + j][e], acc[t * TN + j + 1][e]);
        } else {
          epi_store(a, row, col, acc[t * TN + j][e]);
        }
      }
}

// ---------------------------------------------------------------------------
// skinny kernel: MT x 16 rows, 64 columns per workgroup (16 per wave)
// ---------------------------------------------------------------------------
constexpr int SKC = 64;            // K per stage (2 MFMA k-steps)
constexpr int SRING = 4;           // weight stages in flight per wave
constexpr int SLD = SKC + kPad;

template <int MT>
__global__ __launch_bounds__(256) void gemm_bf16_skinny(GemmArgs a) {
  constexpr int BM = MT * 16;
  constexpr int ACH = BM * (SKC / 8);            // 16-B chunks per plane per stage
  constexpr int APT = 2 * ACH / 256;              // per thread (hi + lo) = MT
  static_assert(2 * ACH % 256 == 0, "whole chunks per thread");
  __shared__ __attribute__((aligned(16))) bf16 Ah[2][BM][SLD];
  __shared__ __attribute__((aligned(16))) bf16 Al[2][BM][SLD];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int tile = blockIdx.x;
  const int n0 = tile * 64 + wave * 16;
  const int kbeg = blockIdx.z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nst = (kend - kbeg) / SKC;

  const bf16* bptr = a.B + (long long)min(n0 + lr, a.N - 1) * a.K + kbeg + lg * 8;

  bf16x8 ring[SRING][2];
  u32x4 ar[APT];
  auto bload = [&](int c, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
    ring[sl][0] = *(const bf16x8*)(bptr + c * SKC);
    ring[sl][1] = *(const bf16x8*)(bptr + c * SKC + 32);
  };
  // activation rows past M are clamped to the last row (their outputs are
  // discarded)
  auto aload = [&](int c) __attribute__((always_inline)) {
    const int k0 = kbeg + c * SKC;
#pragma unroll
    for (int u = 0; u < APT; ++u) {
      const int ci = tid + 256 * u;
      const int pl = ci >= ACH;
      const int cc = ci - pl * ACH;
      const int row = min(cc / (SKC / 8), a.M - 1), col = (cc % (SKC / 8)) * 8;
      const bf16* src = pl ? a.Alo : a.Ahi;
      ar[u] = *(const u32x4*)(src + (long long)row * a.K + k0 + col);
    }
  };
  auto astore = [&](auto buf_c) __attribute__((always_inline)) {
    constexpr int bb = decltype(buf_c)::value;
#pragma unroll
    for (int u = 0; u < APT; ++u) {
      const int ci = tid + 256 * u;
      const int pl = ci >= ACH;
      const int cc = ci - pl * ACH;
      const int row = cc / (SKC / 8), col = (cc % (SKC / 8)) * 8;
      if (pl) *(u32x4*)&Al[bb][row][col] = ar[u];
      else *(u32x4*)&Ah[bb][row][col] = ar[u];
    }
  };

  f32x4 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = (f32x4){0.f, 0.f, 0.f, 0.f};

  // prologue: A(0) -> LDS, weights of stages 0..SRING-1, A(1) in registers
  if (nst > 0) {
    aload(0);
    astore(ic<0>{});
    bload(0, ic<0>{});
    if (1 < nst) bload(1, ic<1>{});
    if (2 < nst) bload(2, ic<2>{});
    if (3 < nst) bload(3, ic<3>{});
    if (1 < nst) aload(1);
    __syncthreads();
  }
  // stage c: MFMAs on LDS buffer c & 1 and ring slot c % SRING; then refill
  // that slot with stage c + SRING, move A(c + 1) to LDS and fetch A(c + 2)
  auto stage = [&](int c, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
    constexpr int cur = sl & 1;
#pragma unroll
    for (int s = 0; s < 2; ++s) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const bf16x8 ah = *(const bf16x8*)&Ah[cur][i * 16 + lr][s * 32 + lg * 8];
        const bf16x8 al = *(const bf16x8*)&Al[cur][i * 16 + lr][s * 32 + lg * 8];
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, ring[sl][s], acc[i], 0, 0, 0);
        acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, ring[sl][s], acc[i], 0, 0, 0);
      }
    }
    if (c + SRING < nst) bload(c + SRING, slot_c);
    if (c + 1 < nst) astore(ic<cur ^ 1>{});
    if (c + 2 < nst) aload(c + 2);
    __syncthreads();
  };
  for (int c = 0; c < nst; c += SRING) {
    stage(c, ic<0>{});
    if (c + 1 < nst) stage(c + 1, ic<1>{});
    if (c + 2 < nst) stage(c + 2, ic<2>{});
    if (c + 3 < nst) stage(c + 3, ic<3>{});
  }

  if (a.ksplit > 1) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) part_store(a, i * 16 + lg * 4 + e, n0 + lr, acc[i][e]);
    return;
  }
  if (a.epi == kEpiSwiGLU) {
    // gate = wave tile with (wave & 1) == 0, up = the next wave's tile: swap
    // through LDS (the activation buffers are free by now) so the gate wave
    // owns both.
    static_assert(sizeof(float) * 2 * MT * 4 * 64 <= sizeof(Ah), "exchange fits");
    float (*xch)[MT * 4][64] = reinterpret_cast<float (*)[MT * 4][64]>(&Ah[0][0][0]);
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
        for (int e = 0; e < 4; ++e)
          epi_swiglu(a, i * 16 + lg * 4 + e, n0 + lr, acc[i][e], xch[wave >> 1][i * 4 + e][lane]);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) epi_store(a, i * 16 + lg * 4 + e, n0 + lr, acc[i][e]);
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

// split an fp32 matrix into its bf16 hi / lo planes (for operands that do not
// come from a library kernel, e.g. the kernel-level entry point)
__global__ void split_planes(const float* __restrict__ x, bf16* __restrict__ hi, bf16* __restrict__ lo, long long n) {
  long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  bf16 h, l;
  split_bf16(x[i], h, l);
  hi[i] = h;
  lo[i] = l;
}

// dense tile configurations (wave grid x wave tile)
struct DenseShape {
  int wm, wn, tm, tn, kc, bm, bn;
};
constexpr DenseShape kDense[] = {
    {2, 4, 5, 4, 32, 160, 256},   // 0: 8 waves of 80 x 64, K stage 32
    {2, 4, 5, 4, 64, 160, 256},   // 1: 8 waves of 80 x 64, K stage 64
    {2, 4, 4, 4, 64, 128, 256},   // 2: 8 waves of 64 x 64, K stage 64
    {2, 2, 4, 4, 64, 128, 128},   // 3: 4 waves of 64 x 64, K stage 64
};

int dense_cfg() {
  static int cfg = [] {
    const char* e = getenv("CDSL_DENSE_CFG");
    int v = e ? atoi(e) : 1;
    return (v >= 0 && v < 4) ? v : 1;
  }();
  return cfg;
}

struct Plan {
  int kind;          // 0 dense, 1 skinny, 2 f32
  int cfg;           // dense tile configuration
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
  if (M <= 128 && K % SKC == 0) {
    p.kind = 1;
    p.mt = (M + 15) / 16;
    p.tiles_m = 1;
    p.tiles_n = (N + 63) / 64;
    // ~2 workgroups per CU, each streaming >= 2 * SRING stages
    const int nst = K / SKC;
    int s = (512 + p.tiles_n - 1) / p.tiles_n;
    s = max(1, min(s, nst / (2 * SRING)));
    const int per = (nst + s - 1) / s;
    s = (nst + per - 1) / per;
    p.ksplit = s;
    p.kchunk = per * SKC;
  } else {
    p.kind = 0;
    p.cfg = dense_cfg();
    if (K % kDense[p.cfg].kc != 0) p.cfg = 0;   // the K-32 configuration
    const DenseShape& d = kDense[p.cfg];
    p.tiles_m = (M + d.bm - 1) / d.bm;
    p.tiles_n = (N + d.bn - 1) / d.bn;
    const int tiles = p.tiles_m * p.tiles_n;
    const int kc = d.kc;
    const int nk = K / kc;
    int s = 1;
    if (tiles < 200) s = min((400 + tiles - 1) / tiles, max(1, nk / 8));
    const int per = (nk + s - 1) / s;
    s = (nk + per - 1) / per;
    p.ksplit = s;
    p.kchunk = per * kc;
  }
  if (p.ksplit > 1) p.ws_bytes = (size_t)p.ksplit * M * N * sizeof(float);
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
  if (dtype == 1 && K % DBK != 0) return -1;
  if (dtype == 0 && K % 16 != 0) return -1;
  return 0;
}

hipError_t gemm_launch(const GemmOperand& A, const void* B, const GemmOut& out, int M, int N, int K, int dtype,
                       int epi, void* ws, size_t ws_bytes, hipStream_t st, bool prefill, GemmHook* hook) {
  if (M == 0) return hipSuccess;
  Plan p = make_plan(M, N, K, dtype);
  if (p.kind == 2) {
    if (epi == kEpiSwiGLU) return hipErrorInvalidValue;  // fp32 path: store + swiglu_f32
    dim3 grid((N + 63) / 64, (M + 63) / 64);
    gemm_f32_tiled<<<grid, 256, 0, st>>>(A.f32, (const float*)B, out.f32, M, N, K, out.ldc, epi);
    return hipGetLastError();
  }
  if (p.ws_bytes > ws_bytes) return hipErrorInvalidValue;
  GemmArgs a;
  a.Ahi = A.hi;
  a.Alo = A.lo;
  a.B = (const bf16*)B;
  a.M = M;
  a.N = N;
  a.K = K;
  a.C = out.f32;
  a.Chi = out.hi;
  a.Clo = out.lo;
  a.ldc = out.ldc;
  a.epi = epi;
  a.ksplit = p.ksplit;
  a.kchunk = p.kchunk;
  a.tiles_m = p.tiles_m;
  a.tiles_n = p.tiles_n;
  a.partial = (float*)ws;
  if (p.kind == 0) {
    dim3 grid(p.tiles_m * p.tiles_n, 1, p.ksplit);
    const DenseShape& d = kDense[p.cfg];
    const int nt = 64 * d.wm * d.wn;
#define CDSL_DENSE(I, WM, WN, TM, TN, KC)                                                  \
  case I:                                                                                  \
    if (prefill) gemm_bf16_dense<WM, WN, TM, TN, KC, 1><<<grid, nt, 0, st>>>(a);           \
    else gemm_bf16_dense<WM, WN, TM, TN, KC, 0><<<grid, nt, 0, st>>>(a);                   \
    break;
    switch (p.cfg) {
      CDSL_DENSE(0, 2, 4, 5, 4, 32)
      CDSL_DENSE(1, 2, 4, 5, 4, 64)
      CDSL_DENSE(2, 2, 4, 4, 4, 64)
      default: CDSL_DENSE(3, 2, 2, 4, 4, 64)
    }
#undef CDSL_DENSE
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
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.ksplit == 1) return e;
  const long long outs = epi == kEpiSwiGLU ? (long long)M * (N / 2) : (long long)M * N;
  if (hook) hook->before_reduce(p.ksplit);
  splitk_reduce_kernel<<<(unsigned)((outs + 255) / 256), 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t swiglu_f32_launch(const float* gu, float* act, int M, int F, hipStream_t st) {
  long long n = (long long)M * F;
  if (n == 0) return hipSuccess;
  swiglu_f32<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(gu, act, M, F);
  return hipGetLastError();
}

hipError_t split_planes_launch(const float* x, bf16* hi, bf16* lo, long long n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  split_planes<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(x, hi, lo, n);
  return hipGetLastError();
}

}  // namespace cdsl
