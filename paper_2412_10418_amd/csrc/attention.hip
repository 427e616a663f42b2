// Attention of one decoder layer over the paged KV cache.
//
// Workgroup = (key split, prompt x KV head, group of 16-row tiles).  The
// query rows of one prompt and one KV head are ALL beams x all rows of the
// beam x the G query heads sharing that KV head, so every shared-prefix KV
// block is read once for all k beams (speculative lookaheads of every beam
// share the prompt and the committed tokens).  Each beam's own lookahead
// tokens live in its suffix blocks, masked so that row (i, j) sees only
// slots 0..j0+j of beam i: the tree mask of the verification pass, and the
// causal mask of one rollout step.
//
// bf16-weight models (attn_split): the KV pool holds fp32 values as bf16
// (hi, lo) planes.  The workgroup first lists the key blocks its rows can
// see, then streams them in pairs (32 keys) through double-buffered LDS,
// the next pair's global loads in flight while the current pair is
// computed.  Per wave: 16 query rows.  Scores are computed transposed, per
// block of 16 keys,
//   S^T[16 keys, 16 rows] = K[16, hd] . Q^T[hd, 16]      (MFMA 16x16x32)
// so that lane (row r, group g) holds keys 4g..4g+3 of both blocks of the
// pair -- exactly its B fragment of
//   O^T[16 dims, 16 rows] += V^T[16 dims, 32 keys] . P^T[32 keys, 16 rows]
// once V's slots are stored in that key order: no shuffles or LDS round
// trip between the two products.  Every product takes three
// MFMAs (hi*hi + hi*lo + lo*hi), keeping fp32-level accuracy.  Online
// softmax in the log2 domain; the row max / sum combine the two lanes of a
// row with one xor shuffle.  Key splits write (m, l, unnormalised O)
// partials that a combine kernel merges in split order (deterministic).
#include <algorithm>

#include "attention.h"
#include "common.h"

namespace cdsl {

namespace {

struct RowInfo {
  int valid, i, j, m, h, pos;
};

__device__ __forceinline__ RowInfo decode_row(const PassDesc& p, int r, int nrows, int bi, int kvh, int G, int Lp) {
  RowInfo ri;
  ri.valid = r < nrows;
  int rr = ri.valid ? r : 0;
  int g = rr % G;
  int t = rr / G;
  ri.j = t % p.R;
  ri.i = t / p.R;
  ri.m = (bi * p.kp + ri.i) * p.R + ri.j;
  ri.h = kvh * G + g;
  ri.pos = Lp + (p.mode == kSuffix ? p.j0 + ri.j : ri.j);
  return ri;
}

// Key block q of prompt b: q < nP are prefix blocks, then kp * nS suffix
// blocks (beam-major).  Returns the pool block id; owner = -1 for prefix.
__device__ __forceinline__ int key_block(const PassDesc& p, int b, int q, int nP, int nS, int& owner, int& base) {
  if (q < nP) {
    owner = -1;
    base = q * kBlock;
    return p.ptable[(long long)b * p.ptable_stride + q];
  }
  int qq = q - nP;
  owner = qq / nS;
  int sub = qq % nS;
  base = sub * kBlock;
  return p.stable[(long long)b * p.s_stride_b + owner * p.s_stride_i + sub];
}

__device__ __forceinline__ bool key_valid(const PassDesc& p, int owner, int slot, const RowInfo& ri, int Lp) {
  if (!ri.valid) return false;
  if (owner < 0) return p.mode == kSuffix ? slot < Lp : slot <= ri.pos;
  return owner == ri.i && slot <= p.j0 + ri.j;
}

// fp32 -> (hi, lo) bf16 pairs, 8 values
__device__ __forceinline__ void split8(const float4& a, const float4& b, bf16x8& hi, bf16x8& lo) {
  const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const bf16 h = (bf16)v[e];
    hi[e] = h;
    lo[e] = (bf16)(v[e] - (float)h);
  }
}

// x . y for fp32 data held as bf16 (hi, lo) pairs: hi*hi + hi*lo + lo*hi,
// ~2^-16 relative (the lo*lo term is below fp32 rounding of the sum)
__device__ __forceinline__ f32x4 mfma3(const bf16x8& ah, const bf16x8& al, const bf16x8& bh, const bf16x8& bl,
                                       f32x4 c) {
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, c, 0, 0, 0);
  return c;
}

// The beams, prefix-key limit and suffix-slot limit that rows [ra, rb] of a
// (prompt, KV head) can see.  Rows of one beam have increasing j, so the
// largest j of the range is that of rb unless the range crosses a beam.
struct Window {
  int i_lo, i_hi, key_lim, slot_lim;
};

__device__ __forceinline__ Window row_window(const PassDesc& p, int ra, int rb, int G, int Lp) {
  const int t_lo = ra / G, t_hi = rb / G;
  const int jmax = (t_lo / p.R == t_hi / p.R) ? t_hi % p.R : p.R - 1;
  Window w;
  w.i_lo = t_lo / p.R;
  w.i_hi = t_hi / p.R;
  w.key_lim = p.mode == kSuffix ? Lp : Lp + jmax + 1;
  w.slot_lim = p.j0 + jmax;
  return w;
}

__device__ __forceinline__ bool window_sees(const Window& w, int owner, int base) {
  if (owner < 0) return base < w.key_lim;
  return owner >= w.i_lo && owner <= w.i_hi && base <= w.slot_lim;
}

// KW = key groups: the NW waves are (NW / KW) row tiles x KW key groups,
// and one iteration stages KW pairs of key blocks: wave (rt, kw) computes
// pair kw of it for row tile rt, and the key groups of a row tile merge
// their (m, l, O) states at the end.  KW > 1 keeps every wave busy, and
// the grid full, when a (prompt, KV head) has few row tiles (the rollout:
// k beams x G heads); the chain of dependent memory round trips (block
// table, then one per iteration) is then short.  Eight waves put up to
// four row tiles of a (prompt, KV head) in one workgroup, so its keys are
// read from memory once for all of them.
template <int HD, int KW, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void attn_split(AttnArgs a) {
  constexpr int NT = 64 * NW;
  constexpr int RTW = NW / KW;                 // row tiles per workgroup
  constexpr int NPI = KW;                      // pairs per iteration
  constexpr int KCH = HD / 8;                  // 16-byte chunks per K row
  constexpr int KPL = 2 * kBlock * HD;         // LDS K plane: 2 blocks x 16 keys x HD
  constexpr int VPL = 2 * HD * kBlock;         // LDS V plane: HD x (4 groups x (4 keys of A, 4 of B))
  constexpr int BUF = 2 * KPL + 2 * VPL;       // K hi, K lo, V hi, V lo
  constexpr int UNIT = 2 * kBlock * HD;        // pool unit (both planes), bf16
  constexpr int UCH = UNIT / 8;                // 16-byte chunks per unit
  constexpr int PER = 4 * UCH / NT;            // chunks per thread per pair (UCH is a multiple of 64)
  constexpr int KS = HD / 32;                  // k-steps of the score product
  constexpr int DT = HD / 16;                  // 16-dim output tiles
  static_assert((4 * UCH) % NT == 0 && UCH % 64 == 0, "whole chunks per thread, one region per wave");
  __shared__ __attribute__((aligned(16))) bf16 lds[2][NPI][BUF];
  __shared__ int lblk[kAttnMaxList];
  __shared__ int lmeta[kAttnMaxList];   // base * 32 + owner + 1
  __shared__ int lcount;

  const PassDesc& p = a.p;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // (key split, prompt x KV head, row group) of this workgroup.  With key
  // splits the grid is (split, pair, row group).  Without, it is one
  // dimension of pairs x row groups: the row groups of one (prompt, KV head)
  // read the same keys, and workgroup p runs on XCD p % 8, so the row groups
  // of a pair take consecutive slots of one XCD (ids xcd + 8 t) and the
  // second read of each key block finds it in that XCD's L2; the pairs past
  // the last multiple of 8 follow in order.
  int split, pq, rg;
  if (a.nsplit > 1) {
    split = blockIdx.x;
    pq = blockIdx.y;
    rg = blockIdx.z;
  } else {
    split = 0;
    const int NQ = p.nb * a.Hkv;
    const int NR = gridDim.x / NQ;   // row groups per pair
    const int full = NQ & ~7;
    const int L = blockIdx.x;
    if (L < full * NR) {
      const int t = L >> 3;
      pq = (L & 7) + 8 * (t / NR);
      rg = t % NR;
    } else {
      const int l2 = L - full * NR;
      pq = full + l2 / NR;
      rg = l2 % NR;
    }
  }
  const int bi = pq / a.Hkv, kvh = pq % a.Hkv;
  const int b = pass_batch(p, bi);
  const int G = a.G;
  const int nrows = p.kp * p.R * G;
  const int wg_r0 = rg * 16 * RTW;
  if (wg_r0 >= nrows) return;   // uniform over the workgroup
  const int Lp = p.Lp[b];

  const int nS = p.mode == kSuffix ? (p.j0 + p.R + kBlock - 1) / kBlock : 0;
  const int nP = p.mode == kSuffix ? (Lp + kBlock - 1) / kBlock : (Lp + p.R + kBlock - 1) / kBlock;
  const int nK = nP + p.kp * nS;
  const int qbeg = split * a.blocks_per_split;
  // the host keeps blocks_per_split <= kAttnMaxList; the clamp only guards LDS
  const int qend = min(min(nK, qbeg + a.blocks_per_split), qbeg + kAttnMaxList);

  // this wave's rows (a wave past the last row still stages key blocks)
  const int rt = wave / KW, kw = wave % KW;
  const int rw0 = wg_r0 + rt * 16;
  const bool wave_has_rows = rw0 < nrows;
  const RowInfo ri = decode_row(p, rw0 + lr, nrows, bi, kvh, G, Lp);
  const Window wwin = row_window(p, min(rw0, nrows - 1), min(rw0 + 15, nrows - 1), G, Lp);

  // Q^T fragments (B operand): row lr, dims 32s + 8lg .. +8, as hi / lo;
  // issued before the key-block list so the two latencies overlap
  float4 qx[KS][2];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    qx[s][0] = qx[s][1] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (ri.valid) {
      const float* qrow = a.Q + ((long long)ri.m * a.H + ri.h) * HD + s * 32 + lg * 8;
      qx[s][0] = *(const float4*)qrow;
      qx[s][1] = *(const float4*)(qrow + 4);
    }
  }

  // list of the key blocks that some row of the workgroup can see
  if (wave == 0) {
    const Window ww = row_window(p, wg_r0, min(wg_r0 + 16 * RTW, nrows) - 1, G, Lp);
    int n = 0;
    for (int c0 = qbeg; c0 < qend; c0 += 64) {
      const int q = c0 + lane;
      int owner = -1, base = 0, blk = 0;
      bool rel = false;
      if (q < qend) {
        blk = key_block(p, b, q, nP, nS, owner, base);
        rel = window_sees(ww, owner, base);
      }
      const unsigned long long m = __ballot(rel);
      const int pos = n + __popcll(m & ((1ull << lane) - 1ull));
      if (rel) {
        lblk[pos] = blk;
        lmeta[pos] = base * 32 + owner + 1;
      }
      n += __popcll(m);
    }
    if (lane == 0) lcount = n;
  }
  __syncthreads();
  const int n = lcount;
  const int npairs = (n + 1) / 2;
  const int niters = (npairs + NPI - 1) / NPI;

  bf16x8 qh[KS], ql[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) split8(qx[s][0], qx[s][1], qh[s], ql[s]);

  // staging: chunk q = tid + NT * u of a pair is region q / UCH (K of block
  // A, K of block B, V of A, V of B) at 16-byte offset q % UCH of the unit.
  // K rows are XOR-swizzled by 16-byte chunk (c ^ (row & 7)).  A V row of
  // the pair (one dim, 64 bytes) holds, for key group g = 0..3, keys
  // 4g..4g+3 of block A then of block B: the V^T fragment of one lane.
  const bf16* kpool = (const bf16*)a.pool.k + (long long)a.layer * 2 * a.pool.layer_elems;
  const bf16* vpool = (const bf16*)a.pool.v + (long long)a.layer * 2 * a.pool.layer_elems;
  auto dst_of = [&](int u) __attribute__((always_inline)) {
    const int region = (tid + NT * u) / UCH, w = (tid + NT * u) % UCH;
    const int plane = w / (UCH / 2), wp = w % (UCH / 2);
    if (region < 2) {
      const int row = region * kBlock + wp / KCH, c = wp % KCH;
      return plane * KPL + row * HD + ((c ^ (row & 7)) << 3);
    }
    // 16-byte chunk wp = (dim, half h) holds keys 8h..8h+7 of one block
    const int dim = wp >> 1, h = wp & 1;
    return 2 * KPL + plane * VPL + dim * 32 + h * 16 + (region - 2) * 4;
  };
  // staging registers: the pairs of iteration it + 1 are in flight while
  // those of iteration it are computed (pairs past the last one re-read
  // the last block and are not computed)
  u32x4 stg[NPI][PER];
  auto gload = [&](int it) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NPI; ++q) {
      const int pi = it * NPI + q;
      const int eA = min(2 * pi, n - 1);
      const int eB = min(2 * pi + 1, n - 1);
      const long long ua = ((long long)lblk[eA] * a.Hkv + kvh) * UNIT;
      const long long ub = ((long long)lblk[eB] * a.Hkv + kvh) * UNIT;
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int region = (tid + NT * u) / UCH;   // uniform over a wave
        const bf16* base = (region < 2 ? kpool : vpool) + ((region & 1) ? ub : ua);
        stg[q][u] = *(const u32x4*)(base + ((tid + NT * u) % UCH) * 8);
      }
    }
  };
  auto sstore = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NPI; ++q)
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int region = (tid + NT * u) / UCH;
        bf16* d = &lds[buf][q][dst_of(u)];
        if (region < 2) {
          *(u32x4*)d = stg[q][u];
        } else {
          // keys 8h..8h+3 -> group 2h, keys 8h+4..8h+7 -> group 2h + 1
          *(uint2*)d = make_uint2(stg[q][u].x, stg[q][u].y);
          *(uint2*)(d + 8) = make_uint2(stg[q][u].z, stg[q][u].w);
        }
      }
  };

  f32x4 acc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
  // Running max m_run (log2 units) and sum l_run of this lane's row.  The
  // exponentials use a possibly stale max: it is only raised (and O, l
  // rescaled) once the true max exceeds it by more than kLazy, so
  // probabilities stay below 2^kLazy and the rescale is rare.  O / l does
  // not depend on which max was used.
  constexpr float kLazy = 8.f;
  float m_run = -INFINITY, l_run = 0.f;
  // Visibility of a key at absolute slot x of a block of owner o to this
  // lane's row: x <= lim_pre for prefix blocks (o < 0), x <= lim_own for
  // the suffix blocks of the row's own beam, never for other beams.
  const int lim_pre = !ri.valid ? -1 : (p.mode == kSuffix ? Lp - 1 : ri.pos);
  const int lim_own = ri.valid ? p.j0 + ri.j : -1;
  auto limit = [&](int owner, int base) __attribute__((always_inline)) {
    return (owner < 0 ? lim_pre : (owner == ri.i ? lim_own : -1)) - base;
  };

  // One pair of key blocks (A, B) from LDS buffer buf.  Scores transposed:
  // S^T[16 keys, 16 rows] = K . Q^T per block, so lane (row lr, group lg)
  // holds keys 4lg..4lg+3 of A and of B -- which, in that order, is the
  // lane's B fragment of O^T[16 dims, 16 rows] += V^T[16 dims, 32 keys] .
  // P^T[32 keys, 16 rows] when the V^T fragment takes the same keys.
  auto compute = [&](int buf, int slot, int pi) __attribute__((always_inline)) {
    const int eA = 2 * pi, eB = 2 * pi + 1;
    if (eA >= n) return;   // past the last pair (uniform over the wave)
    const bool hasB = eB < n;
    const int mA = lmeta[eA], mB = hasB ? lmeta[eB] : 0;
    const int ownA = (mA & 31) - 1, baseA = mA >> 5;
    const int ownB = (mB & 31) - 1, baseB = mB >> 5;
    const bool relA = window_sees(wwin, ownA, baseA);
    const bool relB = hasB && window_sees(wwin, ownB, baseB);
    if (!wave_has_rows || (!relA && !relB)) return;
    const bf16* L = lds[buf][slot];
    f32x4 sA = {0.f, 0.f, 0.f, 0.f}, sB = sA;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int rowA = lr, rowB = kBlock + lr;
      const int offA = rowA * HD + (((4 * s + lg) ^ (rowA & 7)) << 3);
      const int offB = rowB * HD + (((4 * s + lg) ^ (rowB & 7)) << 3);
      const bf16x8 kah = *(const bf16x8*)(L + offA), kal = *(const bf16x8*)(L + KPL + offA);
      const bf16x8 kbh = *(const bf16x8*)(L + offB), kbl = *(const bf16x8*)(L + KPL + offB);
      sA = mfma3(kah, kal, qh[s], ql[s], sA);
      sB = mfma3(kbh, kbl, qh[s], ql[s], sB);
    }
    const int tA = limit(ownA, baseA) - 4 * lg;
    const int tB = (hasB ? limit(ownB, baseB) : -1) - 4 * lg;
    float sv[8];
    float mt = -INFINITY;
    if (__all(tA >= 3 && tB >= 3)) {   // every key of both blocks visible
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sv[e] = sA[e] * a.scale_log2;
        sv[4 + e] = sB[e] * a.scale_log2;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sv[e] = e <= tA ? sA[e] * a.scale_log2 : -INFINITY;
        sv[4 + e] = e <= tB ? sB[e] * a.scale_log2 : -INFINITY;
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) mt = fmaxf(mt, sv[e]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const bool raise = mt > m_run + kLazy;   // true for the first visible key
    if (__ballot(raise)) {
      const float m_to = raise ? mt : m_run;
      const float corr = m_to == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run - m_to);
      l_run *= corr;
#pragma unroll
      for (int t = 0; t < DT; ++t) acc[t] *= corr;
      m_run = m_to;
    }
    const float m_use = m_run == -INFINITY ? 0.f : m_run;
    float psum = 0.f;
    bf16x8 ph, pl;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float pv = __builtin_amdgcn_exp2f(sv[e] - m_use);
      psum += pv;
      const bf16 h = (bf16)pv;
      ph[e] = h;
      pl[e] = (bf16)(pv - (float)h);
    }
    l_run += psum;
    // V^T fragment: dim 16t + lr, keys 4lg..4lg+3 of A then of B
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const int voff = 2 * KPL + (t * 16 + lr) * 32 + lg * 8;
      const bf16x8 vh = *(const bf16x8*)(L + voff), vl = *(const bf16x8*)(L + VPL + voff);
      acc[t] = mfma3(vh, vl, ph, pl, acc[t]);
    }
  };

  // iteration it (pairs it * NPI .. + NPI - 1) sits in LDS buffer it & 1
  if (niters > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
  }
  for (int it = 0; it < niters; ++it) {
    const bool more = it + 1 < niters;
    if (more) gload(it + 1);
    compute(it & 1, kw, it * NPI + kw);
    if (more) sstore((it + 1) & 1);
    __syncthreads();
  }

  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if constexpr (KW > 1) {
    // key groups 1.. hand (m, l, O) to group 0 of their row tile through
    // LDS (free after the loop's last barrier); group 0 merges them in
    // group order
    constexpr int SLOT = (2 + 4 * DT) * 64;   // floats per wave
    float* X = (float*)&lds[0][0][0];
    if (wave_has_rows && kw > 0) {
      float* x = X + (rt * (KW - 1) + kw - 1) * SLOT;
      x[lane] = m_run;
      x[64 + lane] = l_run;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) x[(2 + 4 * t + e) * 64 + lane] = acc[t][e];
    }
    __syncthreads();
    if (kw > 0 || !wave_has_rows) return;
#pragma unroll
    for (int q = 1; q < KW; ++q) {
      const float* x = X + (rt * (KW - 1) + q - 1) * SLOT;
      const float mq = x[lane], lq = x[64 + lane];
      const float mn = fmaxf(m_run, mq);
      const float s0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mn);
      const float s1 = mq == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mq - mn);
      l_run = l_run * s0 + lq * s1;
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[t][e] = acc[t][e] * s0 + x[(2 + 4 * t + e) * 64 + lane] * s1;
      m_run = mn;
    }
  }
  if (!wave_has_rows || !ri.valid) return;
  const long long rowid = (long long)ri.m * a.H + ri.h;
  // lane (row lr, lg) holds dims 16t + 4lg .. +3
  if (a.nsplit == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      bf16x4 hv, lv;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bf16 h, l;
        split_bf16(acc[t][e] * inv, h, l);
        hv[e] = h;
        lv[e] = l;
      }
      const long long o = rowid * HD + t * 16 + lg * 4;
      *(bf16x4*)(a.Ohi + o) = hv;
      *(bf16x4*)(a.Olo + o) = lv;
    }
  } else {
    const long long prow = (long long)split * a.rows_total + rowid;
    float* po = a.part_o + prow * HD + lg * 4;
#pragma unroll
    for (int t = 0; t < DT; ++t) *(f32x4*)(po + t * 16) = acc[t];
    if (lg == 0) {
      a.part_ml[prow * 2] = m_run;
      a.part_ml[prow * 2 + 1] = l_run;
    }
  }
}

// Merge the split partials of every (row, head): one wave per row.  Lane s
// reads split s's (m, l); every partial O load is issued before the weights
// exp2(m_s - max) are formed, so a row costs two memory round trips.
template <int HD>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows_total) return;
  constexpr int PER = (HD + 63) / 64;
  const int ns = a.nsplit;   // <= kAttnMaxSplits (the plan guarantees it)
  float ms = -INFINITY, ls = 0.f;
  if (lane < ns) {
    const long long pr = (long long)lane * a.rows_total + row;
    ms = a.part_ml[pr * 2];
    ls = a.part_ml[pr * 2 + 1];
  }
  float o[kAttnMaxSplits][PER];
#pragma unroll
  for (int s = 0; s < kAttnMaxSplits; ++s)
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int d = lane + 64 * u;
      o[s][u] = (s < ns && d < HD) ? a.part_o[((long long)s * a.rows_total + row) * HD + d] : 0.f;
    }
  const float mx = wave_max(ms);
  const float mu = mx == -INFINITY ? 0.f : mx;
  const float ws = lane < ns ? exp2f(ms - mu) : 0.f;
  const float l = wave_sum(ws * ls);
  float acc[PER] = {};
#pragma unroll
  for (int s = 0; s < kAttnMaxSplits; ++s) {
    const float w = __shfl(ws, s, 64);
#pragma unroll
    for (int u = 0; u < PER; ++u) acc[u] = fmaf(w, o[s][u], acc[u]);
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int d = lane + 64 * u;
    if (d < HD) {
      bf16 h, lo;
      split_bf16(acc[u] * inv, h, lo);
      a.Ohi[row * HD + d] = h;
      a.Olo[row * HD + d] = lo;
    }
  }
}

// Plain path for fp32 models: one wave per (row, head), 64 keys per chunk
// (one per lane), online softmax, no MFMA.  Same cache layout and masks.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32(AttnArgs a) {
  const PassDesc& p = a.p;
  const int lane = threadIdx.x;
  const long long rowid = blockIdx.x;   // (m, h)
  const int m = (int)(rowid / a.H), h = (int)(rowid % a.H);
  const int kvh = h / a.G;
  const int j = m % p.R;
  const int i = (m / p.R) % p.kp;
  const int bi = m / (p.R * p.kp);
  const int b = pass_batch(p, bi);
  const int Lp = p.Lp[b];
  RowInfo ri;
  ri.valid = 1;
  ri.i = i;
  ri.j = j;
  ri.m = m;
  ri.h = h;
  ri.pos = Lp + (p.mode == kSuffix ? p.j0 + j : j);
  const int nS = p.mode == kSuffix ? (p.j0 + p.R + kBlock - 1) / kBlock : 0;
  const int nP = p.mode == kSuffix ? (Lp + kBlock - 1) / kBlock : (Lp + p.R + kBlock - 1) / kBlock;
  const int nkeys = (nP + p.kp * nS) * kBlock;
  const float* q = a.Q + ((long long)m * a.H + h) * HD;
  const float* kbase = (const float*)a.pool.k + (long long)a.layer * a.pool.layer_elems;
  const float* vbase = (const float*)a.pool.v + (long long)a.layer * a.pool.layer_elems;
  constexpr int PER = (HD + 63) / 64;
  float acc[PER] = {};
  float m_run = -INFINITY, l_run = 0.f;
  for (int c0 = 0; c0 < nkeys; c0 += 64) {
    const int key = c0 + lane;
    float s = -INFINITY;
    int blk = 0, t = 0;
    bool ok = false;
    if (key < nkeys) {
      int owner, base;
      blk = key_block(p, b, key / kBlock, nP, nS, owner, base);
      t = key % kBlock;
      ok = key_valid(p, owner, base + t, ri, Lp);
      if (ok) {
        const float* kr = kbase + ((long long)blk * a.Hkv + kvh) * (kBlock * HD) + t * HD;
        float dot = 0.f;
        for (int d = 0; d < HD; ++d) dot = fmaf(q[d], kr[d], dot);
        s = dot * a.scale_log2;
      }
    }
    const float cm = wave_max(s);
    const float m_new = fmaxf(m_run, cm);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float corr = exp2f(m_run - m_use);
    const float pk = ok ? exp2f(s - m_use) : 0.f;
    l_run = l_run * corr + wave_sum(pk);
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < PER; ++u) acc[u] *= corr;
    for (int kk = 0; kk < 64; ++kk) {
      const float pv = __shfl(pk, kk, 64);
      const int bk = __shfl(blk, kk, 64), tk = __shfl(t, kk, 64);
      if (pv != 0.f) {
        const float* vr = vbase + ((long long)bk * a.Hkv + kvh) * (HD * kBlock) + tk;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          int d = lane + 64 * u;
          if (d < HD) acc[u] = fmaf(pv, vr[d * kBlock], acc[u]);
        }
      }
    }
  }
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    int d = lane + 64 * u;
    if (d < HD) a.O[rowid * HD + d] = acc[u] * inv;
  }
}

}  // namespace

AttnPlan attn_plan(const PassDesc& p, int H, int Hkv, int hd, int dtype, int max_prefix_len, int max_splits) {
  AttnPlan pl{};
  const int G = H / Hkv;
  const int nrows = p.kp * p.R * G;
  const int nS = p.mode == kSuffix ? (p.j0 + p.R + kBlock - 1) / kBlock : 0;
  const int nP = p.mode == kSuffix ? (max_prefix_len + kBlock - 1) / kBlock
                                   : (max_prefix_len + p.R + kBlock - 1) / kBlock;
  const int nK = nP + p.kp * nS;
  if (dtype == 0) {
    pl.nsplit = 1;
    pl.blocks_per_split = nK;
    return pl;
  }
  // 16-row tiles, 4 or 8 waves per workgroup (a wave without rows still
  // stages its share of the key blocks).  At most 2 row tiles: the waves
  // become key groups instead -- 4 of them per row tile at hd = 64; 2, with
  // both row tiles in one workgroup, at hd = 128 (LDS: 2 x 32 KB per key
  // group).
  pl.row_tiles = (nrows + 15) / 16;
  pl.threads = 256;
  pl.kw = pl.row_tiles <= 2 ? (hd == 64 ? 4 : 2) : 1;
  if (hd == 64 && pl.row_tiles >= 2 && pl.row_tiles <= 4 && p.nb * Hkv >= 256) {
    // eight waves: 2 row tiles x 4 key groups, or 4 x 2; the keys are read
    // once per (prompt, KV head) instead of once per row tile.  With fewer
    // than 256 (prompt, KV head) pairs the pass is latency-bound and twice
    // the workgroups (one per row tile) finish sooner (measured at 16
    // prompts x 8 KV heads: the eight-wave form cost 0.1 ms more per step)
    pl.threads = 512;
    pl.kw = pl.row_tiles == 2 ? 4 : 2;
  } else if (pl.row_tiles > 4) {
    // eight row tiles per workgroup: each key block is read once per 128
    // rows (the verification of long prefixes) instead of once per 64
    pl.threads = 512;
    pl.kw = 1;
  }
  const int rtw = pl.threads / 64 / pl.kw;
  pl.row_groups = (pl.row_tiles + rtw - 1) / rtw;
  // enough workgroups for two per CU, >= 1 key-block pair per split, and at
  // most kAttnMaxList key blocks per split; no split (and no combine
  // launch) when the grid already holds two workgroups per CU or when a
  // workgroup's chain of pair iterations is short
  const int base = p.nb * Hkv * pl.row_groups;
  const int iters1 = ((nK + 1) / 2 + pl.kw - 1) / pl.kw;
  int s = (base >= 512 || iters1 <= 8) ? 1 : (1024 + base - 1) / base;
  s = std::min(s, (nK + 1) / 2);
  s = std::max(s, (nK + kAttnMaxList - 1) / kAttnMaxList);
  s = std::max(1, std::min(s, std::min(max_splits, kAttnMaxSplits)));
  int bps = (nK + s - 1) / s;
  bps += bps & 1;
  s = std::max(1, (nK + bps - 1) / bps);
  pl.nsplit = s;
  pl.blocks_per_split = bps;
  return pl;
}

hipError_t attn_launch(const AttnArgs& args, const AttnPlan& pl, int hd, int dtype, hipStream_t st) {
  AttnArgs a = args;
  a.nsplit = pl.nsplit;
  a.blocks_per_split = pl.blocks_per_split;
  if (a.rows_total == 0) return hipSuccess;
  if (dtype == 0) {
    dim3 grid((unsigned)a.rows_total);
    switch (hd) {
      case 32: attn_f32<32><<<grid, 64, 0, st>>>(a); break;
      case 64: attn_f32<64><<<grid, 64, 0, st>>>(a); break;
      case 128: attn_f32<128><<<grid, 64, 0, st>>>(a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  if (pl.blocks_per_split > kAttnMaxList) return hipErrorInvalidValue;
  const dim3 grid = pl.nsplit > 1 ? dim3(pl.nsplit, a.p.nb * a.Hkv, pl.row_groups)
                                   : dim3(a.p.nb * a.Hkv * pl.row_groups);
  // LDS: 2 buffers x KW pairs of 16 KB (hd 64) or 32 KB (hd 128)
  if (hd == 64) {
    if (pl.threads == 512) {
      if (pl.kw == 4) attn_split<64, 4, 8><<<grid, 512, 0, st>>>(a);
      else if (pl.kw == 2) attn_split<64, 2, 8><<<grid, 512, 0, st>>>(a);
      else attn_split<64, 1, 8><<<grid, 512, 0, st>>>(a);
    } else if (pl.kw == 4) {
      attn_split<64, 4, 4><<<grid, 256, 0, st>>>(a);
    } else {
      attn_split<64, 1, 4><<<grid, 256, 0, st>>>(a);
    }
  } else if (hd == 128) {
    if (pl.threads == 512) attn_split<128, 1, 8><<<grid, 512, 0, st>>>(a);
    else if (pl.kw == 2) attn_split<128, 2, 4><<<grid, 256, 0, st>>>(a);
    else attn_split<128, 1, 4><<<grid, 256, 0, st>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t attn_combine_launch(const AttnArgs& args, const AttnPlan& pl, int hd, hipStream_t st) {
  if (pl.nsplit == 1 || args.rows_total == 0) return hipSuccess;
  AttnArgs a = args;
  a.nsplit = pl.nsplit;
  a.blocks_per_split = pl.blocks_per_split;
  dim3 cg((unsigned)((a.rows_total + 3) / 4));
  switch (hd) {
    case 32: attn_combine<32><<<cg, 256, 0, st>>>(a); break;
    case 64: attn_combine<64><<<cg, 256, 0, st>>>(a); break;
    case 128: attn_combine<128><<<cg, 256, 0, st>>>(a); break;
  }
  return hipGetLastError();
}

}  // namespace cdsl
