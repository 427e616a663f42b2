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
//   dense  (M > 128): 160 x 256 block tiles, 8 waves (2 x 4) of 80 x 64,
//          64-deep K stages, double-buffered LDS fed from registers two
//          stages ahead, XCD-aware tile order.  The verification block, the
//          prefill, and draft passes of more than 128 rows.
//   skinny (M <= 128): the decode rows of the draft rollout.  Weight
//          streaming bound: each wave owns 16 or 32 columns and keeps a ring
//          of 4 or 8 K stages of weight fragments in flight in registers,
//          straight from HBM; the small activation block is staged once per
//          K stage in LDS and shared by the 4 waves.  Loads are issued in the
//          order they are consumed so the in-order vmcnt waits never stall on
//          a later prefetch.
// When the tile grid cannot fill the 256 CUs, K is split across workgroups;
// each split writes its own fp32 plane, summed in split order (bitwise
// deterministic) by a reduce kernel or by the kernel that consumes the
// result.
#include <stdlib.h>

#include <type_traits>
#include <utility>

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
  RowStats rs;      // kEpiRowStats: per-tile row statistics instead of C
  RopeEpi re;       // kEpiRope: rotary + KV write instead of C
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

// kEpiRowStats: statistics of the rows of an fp32 tile [BM][BN] held in LDS
// (rows m0 + r, columns n0 + c; rows >= M and columns >= N left out).  P
// adjacent lanes share a row, each owning a run of CW columns.  The tile is
// stored with the columns of each run XOR-permuted by a row- and
// run-dependent mask (RsLayout::at), so that when every lane reads the
// same position of its own run, the lanes of a wave hit at most two lanes
// per LDS bank.  A lane reads its run into registers once, in column
// order; then branch-free passes over the registers: maximum and argmax
// (strict comparison in column order keeps the lowest column on ties), the
// sum of exp, and one pass per further top-k place picking the best entry
// ordered after the previous pick (the first place is the maximum), each
// followed by a merge over the P lanes with shuffles.  t is the column
// tile's index in the RowStats layout.
template <int NT, int BM, int BN>
struct RsLayout {
  static constexpr int P = BN >= 64 ? 4 : (BN >= 32 ? 2 : 1);            // lanes per row, divides 64
  static constexpr int CW = BN / P;                                     // columns per lane
  static constexpr int XM = (CW < 32 ? CW : 32) - 1;
  static_assert(BN % P == 0 && (CW & (CW - 1)) == 0, "power-of-two column runs");
  __device__ static int at(int r, int c) { return r * BN + (c ^ ((r + 8 * (c / CW)) & XM)); }
};

template <int NT, int BM, int BN>
__device__ void tile_row_stats(const float* tile, int m0, int n0, int M, int N, int t, const RowStats& s) {
  using L = RsLayout<NT, BM, BN>;
  constexpr int P = L::P, CW = L::CW;
  constexpr int RPP = NT / P;                                     // rows per pass
  const int part = threadIdx.x % P;
  const int c0 = part * CW;
  const int cbase = n0 + c0;
  const int nv = N - cbase;                                       // valid columns of this lane if < CW
  auto row_best = [&](float& v, int& id) {
#pragma unroll
    for (int o = 1; o < P; o <<= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(id, o, 64);
      if (vi_better(ov, oi, v, id)) {
        v = ov;
        id = oi;
      }
    }
  };
#pragma unroll 1
  for (int r0 = 0; r0 < BM; r0 += RPP) {
    // a wave whose first row is past the tile has no live row (uniform)
    if (r0 + (int)(threadIdx.x & ~63u) / P >= BM) continue;
    const int r = min(r0 + (int)threadIdx.x / P, BM - 1);
    const int m = m0 + r;
    const bool live = r0 + (int)threadIdx.x / P < BM && m < M;
    const float* rowp = tile + r * BN + c0;
    const int g = (r + 8 * part) & L::XM;
    float v[CW];   // v[i]: column cbase + i (-inf past N)
#pragma unroll
    for (int i = 0; i < CW; ++i) v[i] = i < nv ? rowp[i ^ g] : -INFINITY;
    float av = -INFINITY;
    int al = -1;
#pragma unroll
    for (int i = 0; i < CW; ++i) {
      const bool b = v[i] > av;
      av = b ? v[i] : av;
      al = b ? i : al;
    }
    int ai = al >= 0 ? cbase + al : 0x7fffffff;
    row_best(av, ai);
    // sum of exp(v - max) as 2^(v log2 e - max log2 e): one FMA per value
    constexpr float kL2e = 1.4426950408889634f;
    const float nb = -av * kL2e;
    float se = 0.f;
#pragma unroll
    for (int i = 0; i < CW; ++i) se += __builtin_amdgcn_exp2f(fmaf(v[i], kL2e, nb));   // 2^-inf = 0 past N
#pragma unroll
    for (int o = 1; o < P; o <<= 1) se += __shfl_xor(se, o, 64);
    const long long o = (long long)m * s.tiles + t;
    if (live && part == 0) {
      s.mx[o] = av;
      s.se[o] = se;
      s.am[o] = ai;
      if (s.kk > 0) {
        s.tv[o * s.kk] = av;
        s.tc[o * s.kk] = ai;
      }
    }
    // top-kk: place 0 is the maximum; place u is the best entry ordered
    // after place u - 1 (value descending, column ascending).  The fast
    // passes take the best value strictly below the previous pick.  That is
    // the same order unless some value equals an earlier pick at another
    // column, which shows as more than kk values >= the last pick in the
    // row (a last pick of -inf counts every column); then the wave redoes
    // the places with the tie-aware order, overwriting the stored ones.
    if (s.kk > 1) {
      float pv = av;
#pragma unroll 1
      for (int u = 1; u < s.kk; ++u) {
        float cv = -INFINITY;
        int cl = -1;
#pragma unroll
        for (int i = 0; i < CW; ++i) {
          const float x = v[i];
          const bool b = (x < pv) & (x > cv);
          cv = b ? x : cv;
          cl = b ? i : cl;
        }
        int ci = cl >= 0 ? cbase + cl : 0x7fffffff;
        row_best(cv, ci);
        if (live && part == 0) {
          s.tv[o * s.kk + u] = cv;
          s.tc[o * s.kk + u] = ci;
        }
        pv = cv;
      }
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < CW; ++i) cnt += v[i] >= pv ? 1 : 0;
#pragma unroll
      for (int q = 1; q < P; q <<= 1) cnt += __shfl_xor(cnt, q, 64);
      if (__any(live && cnt > s.kk)) {
        pv = av;
        int pc = ai;
#pragma unroll 1
        for (int u = 1; u < s.kk; ++u) {
          const int pl = pc - cbase;   // the previous pick as a local position (any value)
          float cv = -INFINITY;
          int cl = -1;
#pragma unroll
          for (int i = 0; i < CW; ++i) {
            const float x = v[i];
            // bitwise, not short-circuit, so the pass stays free of branches
            const bool after = (x < pv) | ((x == pv) & (i > pl));
            const bool b = after & (x > cv);
            cv = b ? x : cv;
            cl = b ? i : cl;
          }
          int ci = cl >= 0 ? cbase + cl : 0x7fffffff;
          row_best(cv, ci);
          if (live && part == 0) {
            s.tv[o * s.kk + u] = cv;
            s.tc[o * s.kk + u] = ci;
          }
          pv = cv;
          pc = ci;
        }
      }
    }
    if (live && s.gather_tok) {
      const int x = min(max(s.gather_tok[rowmap_index(s.gather_map, m)], 0), N - 1);
      const int c = x - cbase;
      if (c >= 0 && c < CW) s.zx[m] = rowp[c ^ g];
    }
  }
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

// kEpiRope.  The tile holds whole heads.  For its rotary heads the fp32
// output tile [BM][BN] is staged in LDS (rope_at: 16-column groups
// XOR-permuted by (row / 4) % 4, so that the four row groups of an MFMA
// fragment write different banks; float4 runs stay whole), and:
//  - rotary heads (q, then k): unit = (row, head, 8 dims of the first half)
//    with its 8 partners; BM * BN / 16 units, a fixed number per thread, so
//    every row record and cos / sin load of a thread is issued before the
//    tile is staged.  q goes out as 16-byte fp32 runs, K as 16-byte runs of
//    each bf16 plane.
//  - value heads: straight from the accumulators, which hold four
//    consecutive rows (slots) of one dim per lane; a tile without rotary
//    heads is not staged.
template <int BN>
__device__ __forceinline__ int rope_at(int r, int c) {
  return r * BN + (c ^ (((r >> 2) & 3) << 4));
}

template <int NT, int BM, int BN, int HD, int TM, int TN>
__device__ __forceinline__ void rope_epilogue(const GemmArgs& a, const f32x4 (&acc)[TM * TN], float* tile, int m0,
                                              int n0, int wm, int wn, int lr, int lg) {
  constexpr int HALF = HD / 2, C8 = HALF / 8, UPT = BM * BN / 16 / NT;
  static_assert(BN % HD == 0 && HALF % 8 == 0 && BM * BN % (16 * NT) == 0, "rotary units per thread");
  const RopeEpi& re = a.re;
  const int H = re.H, Hkv = re.Hkv, Hqk = H + Hkv;
  const long long unit = split_unit_elems(HD), plane = (long long)kBlock * HD;
  bf16* kl = (bf16*)re.pool.k + (long long)re.layer * 2 * re.pool.layer_elems;
  bf16* vl = (bf16*)re.pool.v + (long long)re.layer * 2 * re.pool.layer_elems;
  const int2* __restrict__ rinfo = re.rowinfo;
  const int rows = min(BM, a.M - m0);
  const int h0 = n0 / HD, nh = min(BN, a.N - n0) / HD;
  const int nrot = max(0, min(nh, Hqk - h0));
  auto tile4 = [&](int r, int c) { return *(const float4*)&tile[rope_at<BN>(r, c)]; };

  // value columns (below) come straight from the accumulators: this lane's
  // rows' KV places are loaded up front
  const int nv = nh - nrot;
  const int rw = wm * TM * 16 + lg * 4;   // first local row of this lane
  int kvr[TM][4];
#pragma unroll
  for (int t = 0; t < TM; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e) kvr[t][e] = nv > 0 ? rinfo[m0 + min(rw + t * 16 + e, rows - 1)].x : 0;

  // rotary units u = tid + NT * w: chunk fastest, then head, then row
  if (nrot > 0) {
    int2 ri[UPT];
    float4 cs[UPT][4];
    bool live[UPT];
#pragma unroll
    for (int w = 0; w < UPT; ++w) {
      const int u = threadIdx.x + NT * w;
      const int r = u / (C8 * (BN / HD)), hh = u / C8 % (BN / HD);
      live[w] = r < rows && hh < nrot;
      ri[w] = rinfo[m0 + min(r, rows - 1)];
    }
#pragma unroll
    for (int w = 0; w < UPT; ++w) {
      const int d = (threadIdx.x + NT * w) % C8 * 8;
      const float* ct = re.cos_t + (long long)ri[w].y * HALF + d;
      const float* st = re.sin_t + (long long)ri[w].y * HALF + d;
      cs[w][0] = *(const float4*)ct;
      cs[w][1] = *(const float4*)(ct + 4);
      cs[w][2] = *(const float4*)st;
      cs[w][3] = *(const float4*)(st + 4);
    }
    // the loads above are in flight while the tile goes to LDS (the K
    // stages' buffers are free once every wave has left the K loop)
    __syncthreads();
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          tile[rope_at<BN>(wm * TM * 16 + t * 16 + lg * 4 + e, wn * TN * 16 + j * 16 + lr)] = acc[t * TN + j][e];
    __syncthreads();
#pragma unroll
    for (int w = 0; w < UPT; ++w) {
      if (!live[w]) continue;
      const int u = threadIdx.x + NT * w;
      const int r = u / (C8 * (BN / HD)), hh = u / C8 % (BN / HD), d = u % C8 * 8;
      const int m = m0 + r, head = h0 + hh, lc = hh * HD + d;
      const float4 x1a = tile4(r, lc), x1b = tile4(r, lc + 4), x2a = tile4(r, lc + HALF), x2b = tile4(r, lc + HALF + 4);
      const float x1[8] = {x1a.x, x1a.y, x1a.z, x1a.w, x1b.x, x1b.y, x1b.z, x1b.w};
      const float x2[8] = {x2a.x, x2a.y, x2a.z, x2a.w, x2b.x, x2b.y, x2b.z, x2b.w};
      const float c[8] = {cs[w][0].x, cs[w][0].y, cs[w][0].z, cs[w][0].w, cs[w][1].x, cs[w][1].y, cs[w][1].z, cs[w][1].w};
      const float sn[8] = {cs[w][2].x, cs[w][2].y, cs[w][2].z, cs[w][2].w, cs[w][3].x, cs[w][3].y, cs[w][3].z, cs[w][3].w};
      float y1[8], y2[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        y1[e] = rope_first(x1[e], x2[e], c[e], sn[e]);
        y2[e] = rope_second(x1[e], x2[e], c[e], sn[e]);
      }
      if (head < H) {
        float* q = re.qout + ((long long)m * H + head) * HD + d;
        *(float4*)q = make_float4(y1[0], y1[1], y1[2], y1[3]);
        *(float4*)(q + 4) = make_float4(y1[4], y1[5], y1[6], y1[7]);
        *(float4*)(q + HALF) = make_float4(y2[0], y2[1], y2[2], y2[3]);
        *(float4*)(q + HALF + 4) = make_float4(y2[4], y2[5], y2[6], y2[7]);
      } else {
        bf16x8 h1, l1, h2, l2;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          bf16 h, l;
          split_bf16(y1[e], h, l);
          h1[e] = h;
          l1[e] = l;
          split_bf16(y2[e], h, l);
          h2[e] = h;
          l2[e] = l;
        }
        bf16* kr = kl + ((long long)(ri[w].x / kBlock) * Hkv + (head - H)) * unit + (long long)(ri[w].x % kBlock) * HD + d;
        *(bf16x8*)kr = h1;
        *(bf16x8*)(kr + plane) = l1;
        *(bf16x8*)(kr + HALF) = h2;
        *(bf16x8*)(kr + plane + HALF) = l2;
      }
    }
  }

  if (nv <= 0) return;
  // value heads.  V is stored [hd][16 slots] per block and KV head, so a lane's four
  // consecutive rows of one dim are four consecutive slots of its dim row
  // when they lie in one block from a slot that is a multiple of 4: one
  // 8-byte store per plane; otherwise slot by slot
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int col = n0 + wn * TN * 16 + j * 16 + lr;
    const int head = col / HD;
    if (col >= a.N || head < Hqk) continue;
    const int d = col - head * HD;
    bf16* vh0 = vl + (long long)(head - Hqk) * unit + (long long)d * kBlock;
#pragma unroll
    for (int t = 0; t < TM; ++t) {
      const int k0 = kvr[t][0];
      const bool live0 = rw + t * 16 < rows;
      const bool run = rw + t * 16 + 3 < rows && (k0 & 3) == 0 && kvr[t][1] == k0 + 1 && kvr[t][2] == k0 + 2 &&
                       kvr[t][3] == k0 + 3;
      if (run) {
        bf16x4 hv, lv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bf16 h, l;
          split_bf16(acc[t * TN + j][e], h, l);
          hv[e] = h;
          lv[e] = l;
        }
        bf16* vr = vh0 + (long long)(k0 / kBlock) * Hkv * unit + k0 % kBlock;
        *(bf16x4*)vr = hv;
        *(bf16x4*)(vr + plane) = lv;
      } else if (live0) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (rw + t * 16 + e >= rows) continue;
          bf16 h, l;
          split_bf16(acc[t * TN + j][e], h, l);
          bf16* vr = vh0 + (long long)(kvr[t][e] / kBlock) * Hkv * unit + kvr[t][e] % kBlock;
          vr[0] = h;
          vr[plane] = l;
        }
      }
    }
  }
}

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
  // them once per tile (measured: 894 MB -> about 420 MB of HBM reads for the
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
  if constexpr ((size_t)BM * BN * sizeof(float) <= sizeof(lds)) {
    if (a.epi == kEpiRowStats) {
      // the stages are consumed: the tile goes through LDS for the row pass
      float* tile = reinterpret_cast<float*>(&lds[0][0]);
      __syncthreads();
#pragma unroll
      for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            tile[RsLayout<C::NT, BM, BN>::at(wm * TM * 16 + t * 16 + lg * 4 + e, wn * TN * 16 + j * 16 + lr)] =
                acc[t * TN + j][e];
      __syncthreads();
      tile_row_stats<C::NT, BM, BN>(tile, m0, n0, a.M, a.N, tn_blk, a.rs);
      return;
    }
    if (a.epi == kEpiRope) {
      float* tile = reinterpret_cast<float*>(&lds[0][0]);
      if (a.re.hd == 128) rope_epilogue<C::NT, BM, BN, 128, TM, TN>(a, acc, tile, m0, n0, wm, wn, lr, lg);
      else rope_epilogue<C::NT, BM, BN, 64, TM, TN>(a, acc, tile, m0, n0, wm, wn, lr, lg);
      return;
    }
  }
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
// skinny kernel: MT x 16 rows, CT x 16 columns per wave, 4 waves
//
// Weight streaming.  Each wave keeps RING K stages of its weight fragments in
// flight in registers, straight from HBM (one 16-byte load per column tile
// and k-step).  The activation stage (hi and lo planes, MT x 16 rows x 64 K)
// goes through double-buffered LDS, XOR-swizzled like the dense kernel, and
// each activation fragment feeds CT MFMA column tiles.  The main loop is
// free of branches around memory operations: prefetches past the last stage
// re-read it (L2 hits), so the compiler's in-order vmcnt accounting stays
// exact and the ring is never drained early.
// ---------------------------------------------------------------------------
constexpr int SKC = 64;            // K per stage (2 MFMA k-steps)

template <int MT, int CT, int RING, int NWV>
__global__ __launch_bounds__(64 * NWV) void gemm_bf16_skinny(GemmArgs a) {
  constexpr int NT = 64 * NWV;
  constexpr int BM = MT * 16;
  constexpr int BN = NWV * CT * 16;               // columns per workgroup
  constexpr int ACH = BM * (SKC / 8);             // 16-B chunks per plane per stage
  constexpr int APT = 2 * ACH / NT;               // per thread (hi + lo)
  static_assert(2 * ACH % NT == 0, "whole chunks per thread");
  __shared__ __attribute__((aligned(16))) bf16 As[2][2][BM * SKC];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int n0 = blockIdx.x * BN + wave * CT * 16;
  const int kbeg = blockIdx.z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nst = (kend - kbeg) / SKC;

  const bf16* bptr[CT];
#pragma unroll
  for (int j = 0; j < CT; ++j) bptr[j] = a.B + (long long)min(n0 + j * 16 + lr, a.N - 1) * a.K + kbeg + lg * 8;

  bf16x8 ring[RING][CT][2];
  auto bload = [&](int c, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < CT; ++j) ring[sl][j][s] = *(const bf16x8*)(bptr[j] + c * SKC + s * 32);
  };
  // activation chunk q of a stage: plane q / ACH, row (q % ACH) / 8, 16-byte
  // column q % 8; rows past M are clamped to the last row (their outputs are
  // discarded).  NA register sets: A(c + NA) is fetched at stage c and
  // written to LDS at stage c + NA - 1, so each activation load has NA - 1
  // stages to arrive.
  // (the split narrow projections, a ring of 4 at 16 columns per wave:
  // two sets, which frees the registers those short chunks do not need)
  constexpr int NA = (NWV == 4 && !(CT == 1 && RING == 4)) ? 4 : 2;
  static_assert(RING % NA == 0, "register sets rotate with the ring");
  u32x4 ar[NA][APT];
  auto aload = [&](int c, auto set_c) __attribute__((always_inline)) {
    constexpr int st = decltype(set_c)::value;
    const int k0 = kbeg + c * SKC;
#pragma unroll
    for (int u = 0; u < APT; ++u) {
      const int q = tid + NT * u;
      const int pl = q / ACH, cc = q % ACH;
      const int row = min(cc / 8, a.M - 1), col = (cc % 8) * 8;
      ar[st][u] = *(const u32x4*)((pl ? a.Alo : a.Ahi) + (long long)row * a.K + k0 + col);
    }
  };
  auto astore = [&](int buf, auto set_c) __attribute__((always_inline)) {
    constexpr int st = decltype(set_c)::value;
#pragma unroll
    for (int u = 0; u < APT; ++u) {
      const int q = tid + NT * u;
      const int pl = q / ACH, cc = q % ACH;
      const int row = cc / 8, c = cc % 8;
      *(u32x4*)&As[buf][pl][row * SKC + ((c ^ (row & 7)) << 3)] = ar[st][u];
    }
  };

  f32x4 acc[MT][CT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < CT; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};

  // The fragments of a stage (both k-steps when they fit the registers,
  // else one k-step at a time) are all read before the MFMAs that use them,
  // and consecutive MFMAs go to different accumulators (the hi planes of
  // every row tile, then the lo planes).  With one wave per SIMD nothing
  // else hides an LDS round trip or a dependent MFMA, so reading and
  // multiplying fragment by fragment would serialise them.
  constexpr int KB = MT <= 5 ? 2 : 1;          // k-steps per fragment batch
  auto mma = [&](int cur, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
#pragma unroll
    for (int s0 = 0; s0 < 2; s0 += KB) {
      bf16x8 af[KB][2][MT];
#pragma unroll
      for (int u = 0; u < KB; ++u)
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int row = i * 16 + lr;
          const int off = row * SKC + ((((s0 + u) * 4 + lg) ^ (row & 7)) << 3);
          af[u][0][i] = *(const bf16x8*)&As[cur][0][off];
          af[u][1][i] = *(const bf16x8*)&As[cur][1][off];
        }
#pragma unroll
      for (int u = 0; u < KB; ++u)
#pragma unroll
        for (int pl = 0; pl < 2; ++pl)
#pragma unroll
          for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < CT; ++j)
              acc[i][j] =
                  __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[u][pl][i], ring[sl][j][s0 + u], acc[i][j], 0, 0, 0);
      // the first k-step's reads, then its MFMAs interleaved with the
      // second k-step's reads, then the second k-step's MFMAs
      if constexpr (KB == 2) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * MT, 0);
#pragma unroll
        for (int q = 0; q < 2 * MT; ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, CT, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * MT * CT, 0);
      } else {
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * KB * MT, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * KB * MT * CT, 0);
      }
    }
  };

  // stage c (ring slot c % RING, register set c % NA): MFMAs on LDS buffer
  // c & 1; refill the ring slot with stage c + RING; write A(c + 1) (set
  // (c + 1) % NA) to the other buffer; fetch A(c + NA) into the set freed by
  // A(c)
  auto stage = [&](int c, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
    mma(c & 1, slot_c);
    bload(min(c + RING, nst - 1), slot_c);
    astore((c + 1) & 1, ic<(sl + 1) % NA>{});
    aload(min(c + NA, nst - 1), ic<sl % NA>{});
    __syncthreads();
  };
  auto stage_tail = [&](int c, auto slot_c) __attribute__((always_inline)) {
    constexpr int sl = decltype(slot_c)::value;
    if (c < nst) {
      mma(c & 1, slot_c);
      if (c + 1 < nst) astore((c + 1) & 1, ic<(sl + 1) % NA>{});
      if (c + NA < nst) aload(c + NA, ic<sl % NA>{});
      __syncthreads();
    }
  };

  if (nst > 0) {
    [&]<int... U>(std::integer_sequence<int, U...>) {
      (aload(min(U, nst - 1), ic<U>{}), ...);
    }(std::make_integer_sequence<int, NA>{});
    [&]<int... U>(std::integer_sequence<int, U...>) {
      (bload(min(U, nst - 1), ic<U>{}), ...);
    }(std::make_integer_sequence<int, RING>{});
    astore(0, ic<0>{});
    __syncthreads();
  }
  int c = 0;
  for (; c + RING <= nst; c += RING) {
    [&]<int... U>(std::integer_sequence<int, U...>) {
      (stage(c + U, ic<U>{}), ...);
    }(std::make_integer_sequence<int, RING>{});
  }
  // tail stages (fewer than RING left)
  [&]<int... U>(std::integer_sequence<int, U...>) {
    (stage_tail(c + U, ic<U>{}), ...);
  }(std::make_integer_sequence<int, RING>{});

  if (a.ksplit > 1) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < CT; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e) part_store(a, i * 16 + lg * 4 + e, n0 + j * 16 + lr, acc[i][j][e]);
    return;
  }
  if (a.epi == kEpiRowStats) {
    static_assert((size_t)BM * BN * sizeof(float) <= sizeof(As), "the tile fits the activation buffers");
    float* tile = reinterpret_cast<float*>(&As[0][0][0]);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int j = 0; j < CT; ++j)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          tile[RsLayout<NT, BM, BN>::at(i * 16 + lg * 4 + e, wave * CT * 16 + j * 16 + lr)] = acc[i][j][e];
    __syncthreads();
    tile_row_stats<NT, BM, BN>(tile, 0, blockIdx.x * BN, a.M, a.N, blockIdx.x, a.rs);
    return;
  }
  if (a.epi == kEpiSwiGLU) {
    if constexpr (CT % 2 == 0) {
      // column tiles 2t (gate) and 2t + 1 (up) of the packed weight are in
      // this wave
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < CT; j += 2)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            epi_swiglu(a, i * 16 + lg * 4 + e, n0 + j * 16 + lr, acc[i][j][e], acc[i][j + 1][e]);
    } else {
      // gate = wave tile with (wave & 1) == 0, up = the next wave's tile:
      // swap through LDS (the activation buffers are free by now) so the
      // gate wave owns both
      static_assert(sizeof(float) * 2 * MT * 4 * 64 <= sizeof(As), "exchange fits");
      float (*xch)[MT * 4][64] = reinterpret_cast<float (*)[MT * 4][64]>(&As[0][0][0]);
      if (wave & 1) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) xch[wave >> 1][i * 4 + e][lane] = acc[i][0][e];
      }
      __syncthreads();
      if ((wave & 1) == 0) {
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            epi_swiglu(a, i * 16 + lg * 4 + e, n0 + lr, acc[i][0][e], xch[wave >> 1][i * 4 + e][lane]);
      }
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < CT; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) epi_store(a, i * 16 + lg * 4 + e, n0 + j * 16 + lr, acc[i][j][e]);
}

// ---------------------------------------------------------------------------
// fp32 kernel (the fp32 workload): 64x64 tiles, 4x4 outputs per thread
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemm_f32_tiled(const float* __restrict__ A, const float* __restrict__ B,
                                                       float* __restrict__ C, int M, int N, int K, int ldc,
                                                       int epi, RowStats rs) {
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
  if (epi == kEpiRowStats) {
    __shared__ float tile[64 * 64];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) tile[RsLayout<256, 64, 64>::at(ty * 4 + i, tx * 4 + j)] = acc[i][j];
    __syncthreads();
    tile_row_stats<256, 64, 64>(tile, m0, n0, M, N, blockIdx.x, rs);
    return;
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
  int mt, ct, nwv;   // skinny row tiles, 16-column tiles per wave, waves
  bool wide;         // skinny: unsplit wide projection
  int tiles_m, tiles_n;
  int ksplit, kchunk;
  size_t ws_bytes;
};

// K stages of weights in flight per wave: 8 for the unsplit wide
// projections at 16 columns per wave, else 4 (which also lets a narrow
// projection split K into twice as many chunks)
constexpr int skinny_ring(int ct, bool wide) { return ct == 1 && wide ? 8 : 4; }

Plan make_plan(int M, int N, int K, int dtype, bool no_split = false) {
  Plan p{};
  if (dtype == 0) {
    p.kind = 2;
    return p;
  }
  if (M <= 128 && K % SKC == 0) {
    p.kind = 1;
    p.mt = (M + 15) / 16;
    // Wide projections (>= 200 tiles of 64 columns: gate/up, LM head) run
    // with no K split, so no partial planes are written: 32 columns per
    // wave (each activation fragment feeds two MFMA tiles) when that still
    // gives >= 200 workgroups, else 16.  Narrow ones run 16 columns per wave
    // with K split to about 256 workgroups, each streaming whole rings of K
    // stages: twice the column tiles of 32 columns per wave, hence half the
    // split planes for the consumer to fold (measured 1-2 us faster per
    // projection at 80 rows).
    const int nst = K / SKC;
    const bool wide = (N + 63) / 64 >= 200;
    p.ct = (wide && (N + 127) / 128 >= 200) ? 2 : 1;
    p.nwv = 4;
    p.wide = wide;
    const int ring = skinny_ring(p.ct, wide);
    p.tiles_m = 1;
    p.tiles_n = (N + p.nwv * p.ct * 16 - 1) / (p.nwv * p.ct * 16);
    int s = wide ? 1 : (256 + p.tiles_n - 1) / p.tiles_n;
    s = max(1, min(s, nst / ring));
    int per = (nst + s - 1) / s;
    if (nst >= ring) per = (per + ring - 1) / ring * ring;
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
    // One workgroup fits per CU.  Pick the K split s that minimises
    // rounds(s) x (stages(s) + 2) -- whole rounds of 256 workgroups, so a
    // split that leaves the last round half empty is avoided, and each
    // workgroup pays about two stages of prologue and epilogue -- plus the
    // traffic of the s fp32 planes (written, then read by the fold),
    // expressed in stage times (about 2 us per stage of this tile, ~5 TB/s
    // for planes).  Splits keep at least two stages each: few row blocks
    // (the draft rollout of more than 128 rows) would otherwise leave most
    // CUs idle (the o projection at 160 rows: 8 tiles).
    int s = 1;
    double best = 1e300;
    for (int c = 1; c <= 32 && c <= max(1, nk / 2); ++c) {
      const int per = (nk + c - 1) / c;
      const double rounds = (double)((tiles * c + 255) / 256);
      const double planes = c > 1 ? (c + 1.0) * M * N * 4.0 / 5e12 / 2e-6 : 0.0;
      // a split must gain more than 5% over the unsplit launch
      const double t = (rounds * (per + 2.0) + planes) * (c > 1 ? 1.05 : 1.0);
      if (t < best - 1e-9) {
        best = t;
        s = c;
      }
    }
    const int per = (nk + s - 1) / s;
    s = (nk + per - 1) / per;
    p.ksplit = s;
    p.kchunk = per * kc;
  }
  if (no_split) {
    p.ksplit = 1;
    p.kchunk = K;
  }
  if (p.ksplit > 1) p.ws_bytes = (size_t)p.ksplit * M * N * sizeof(float);
  return p;
}

// Whether a dense configuration's fp32 output tile fits the LDS of its K
// stages (the row-statistics and rotary epilogues stage it there).
bool tile_fits_lds(const DenseShape& d) {
  const size_t lds = 2 * 2 * ((size_t)(2 * d.bm + d.bn) * d.kc + 64 * d.wm * d.wn * 8);
  return (size_t)d.bm * d.bn * sizeof(float) <= lds;
}

// Column tiles of a row-statistics launch (0: the shape's kernel cannot
// stage its output tile through LDS).
int rowstats_tiles(const Plan& p, int N) {
  if (p.kind == 2) return (N + 63) / 64;
  if (p.kind == 1) return p.tiles_n;
  return tile_fits_lds(kDense[p.cfg]) ? p.tiles_n : 0;
}

bool rope_fusable(const Plan& p, int N, int hd) {
  if (p.kind != 0 || p.ksplit != 1 || (hd != 64 && hd != 128) || N % hd != 0) return false;
  const DenseShape& d = kDense[p.cfg];
  return d.bn % hd == 0 && tile_fits_lds(d);
}

}  // namespace

size_t gemm_workspace_bytes(int M, int N, int K, int dtype) {
  if (dtype == 0 || M <= 0) return 0;
  size_t b = make_plan(M, N, K, dtype).ws_bytes;
  return (b + 255) & ~(size_t)255;
}

int gemm_kind(int M, int N, int K, int dtype) { return make_plan(M, N, K, dtype).kind; }

int gemm_rowstats_tiles(int M, int N, int K, int dtype) {
  if (M <= 0) return 0;
  return rowstats_tiles(make_plan(M, N, K, dtype, true), N);
}

bool gemm_rope_fusable(int M, int N, int K, int dtype, int hd) {
  if (M <= 0 || dtype != 1) return false;
  return rope_fusable(make_plan(M, N, K, dtype), N, hd);
}

int gemm_check(int M, int N, int K, int dtype) {
  if (M < 0 || N <= 0 || K <= 0) return -1;
  if (dtype == 1 && K % DBK != 0) return -1;
  if (dtype == 0 && K % 16 != 0) return -1;
  return 0;
}

hipError_t gemm_launch(const GemmOperand& A, const void* B, const GemmOut& out, int M, int N, int K, int dtype,
                       int epi, void* ws, size_t ws_bytes, hipStream_t st, bool prefill, GemmHook* hook,
                       int* deferred, RowStats* rs, const RopeEpi* rope) {
  if (deferred) *deferred = 1;
  if (M == 0) return hipSuccess;
  const bool stats = epi == kEpiRowStats;
  if (stats != (rs != nullptr)) return hipErrorInvalidValue;
  if ((epi == kEpiRope) != (rope != nullptr)) return hipErrorInvalidValue;
  Plan p = make_plan(M, N, K, dtype, stats);
  if (rope && !rope_fusable(p, N, rope->hd)) return hipErrorInvalidValue;
  if (stats) {
    rs->tiles = rowstats_tiles(p, N);
    if (rs->tiles == 0 || rs->kk < 0 || rs->kk > 16) return hipErrorInvalidValue;
  }
  if (p.kind == 2) {
    if (epi == kEpiSwiGLU) return hipErrorInvalidValue;  // fp32 path: store + swiglu_f32
    dim3 grid((N + 63) / 64, (M + 63) / 64);
    gemm_f32_tiled<<<grid, 256, 0, st>>>(A.f32, (const float*)B, out.f32, M, N, K, out.ldc, epi,
                                         stats ? *rs : RowStats{});
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
  a.rs = stats ? *rs : RowStats{};
  a.re = rope ? *rope : RopeEpi{};
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
#define CDSL_SKINNY(MT)                                                                     \
  case MT:                                                                                  \
    if (p.ct == 2) gemm_bf16_skinny<MT, 2, skinny_ring(2, true), 4><<<grid, 256, 0, st>>>(a);  \
    else if (p.wide) gemm_bf16_skinny<MT, 1, skinny_ring(1, true), 4><<<grid, 256, 0, st>>>(a); \
    else gemm_bf16_skinny<MT, 1, skinny_ring(1, false), 4><<<grid, 256, 0, st>>>(a);           \
    break;
    switch (p.mt) {
      CDSL_SKINNY(1)
      CDSL_SKINNY(2)
      CDSL_SKINNY(3)
      CDSL_SKINNY(4)
      CDSL_SKINNY(5)
      CDSL_SKINNY(6)
      CDSL_SKINNY(7)
      default: CDSL_SKINNY(8)
    }
#undef CDSL_SKINNY
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.ksplit == 1) return e;
  if (deferred && epi != kEpiSwiGLU) {
    *deferred = p.ksplit;
    return hipSuccess;
  }
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
