// Attention of one decoder layer over the paged KV cache.
//
// Workgroup = (key split, prompt x KV head, group of 4 row tiles).  The
// query rows of one prompt and one KV head are ALL beams x all rows of the
// beam x the G query heads sharing that KV head, so every shared-prefix KV
// block is read once for all k beams (speculative lookaheads of every beam
// share the prompt and the committed tokens).  Each beam's own lookahead
// tokens live in its suffix blocks, masked so that row (i, j) sees only
// slots 0..j0+j of beam i: the tree mask of the verification pass, and the
// causal mask of one rollout step.
//
// Per wave: 16 query rows.  Scores are computed transposed,
//   S^T[16 keys, 16 rows] = K[16, hd] . Q^T[hd, 16]      (MFMA 16x16x32)
// so that lane (row r, group g) ends up holding P[r][keys 4g..4g+3] of two
// consecutive blocks -- exactly the B fragment of
//   O^T[hd, 16 rows] += V^T[hd, 32 keys] . P^T[32 keys, 16 rows]
// with V stored transposed per block ([hd][16 tokens]): no shuffles or LDS
// round trip between the two products.  Q, K, V and P are fp32, each MFMA
// operand is split into bf16 hi + lo and a product takes three MFMAs
// (hi*hi + hi*lo + lo*hi), keeping fp32-level accuracy.  Online softmax in
// the log2 domain;
// the row max / sum are reduced across the 4 lanes of a row with xor
// shuffles.  Key splits write (m, l, unnormalised O) partials that a
// combine kernel merges in split order (deterministic).
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

template <int HD>
__global__ __launch_bounds__(256) void attn_mfma(AttnArgs a) {
  constexpr int KS = HD / 32;   // k-steps of the score product
  constexpr int DT = HD / 16;   // output tiles of 16 dims
  const PassDesc& p = a.p;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int split = blockIdx.x;
  const int bi = blockIdx.y / a.Hkv, kvh = blockIdx.y % a.Hkv;
  const int b = pass_batch(p, bi);
  const int G = a.G;
  const int nrows = p.kp * p.R * G;
  const int r0 = (blockIdx.z * 4 + wave) * 16;
  if (r0 >= nrows) return;
  const int Lp = p.Lp[b];

  const RowInfo ri = decode_row(p, r0 + lr, nrows, bi, kvh, G, Lp);

  // key blocks of this prompt and this split
  const int nS = p.mode == kSuffix ? (p.j0 + p.R + kBlock - 1) / kBlock : 0;
  const int nP = p.mode == kSuffix ? (Lp + kBlock - 1) / kBlock : (Lp + p.R + kBlock - 1) / kBlock;
  const int nK = nP + p.kp * nS;
  const int qbeg = split * a.blocks_per_split;
  const int qend = min(nK, qbeg + a.blocks_per_split);

  // wave-uniform relevance: beams and positions covered by this wave's rows
  const int rlast = min(r0 + 15, nrows - 1);
  const int t_lo = r0 / G, t_hi = rlast / G;
  const int i_lo = t_lo / p.R, i_hi = t_hi / p.R;
  int jmax = 0;
  for (int t = t_lo; t <= t_hi; ++t) jmax = max(jmax, t % p.R);
  const int key_lim = p.mode == kSuffix ? Lp : Lp + jmax + 1;       // prefix keys < key_lim
  const int slot_lim = p.j0 + jmax;                                 // suffix slots <= slot_lim
  auto relevant = [&](int q) -> bool {
    if (q < nP) return q * kBlock < key_lim;
    int qq = q - nP;
    int owner = qq / nS, sub = qq % nS;
    return owner >= i_lo && owner <= i_hi && sub * kBlock <= slot_lim;
  };
  auto next_rel = [&](int q) -> int {
    while (q < qend && !relevant(q)) ++q;
    return q;
  };

  // Q^T fragments (B operand): row lr, dims 32s + 8lg .. +8, as hi/lo
  bf16x8 qh[KS], ql[KS];
  {
    const float* qrow = a.Q + ((long long)ri.m * a.H + ri.h) * HD + lg * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      float4 x0 = make_float4(0.f, 0.f, 0.f, 0.f), x1 = x0;
      if (ri.valid) {
        x0 = *(const float4*)(qrow + s * 32);
        x1 = *(const float4*)(qrow + s * 32 + 4);
      }
      split8(x0, x1, qh[s], ql[s]);
    }
  }

  const float* kbase = (const float*)a.pool.k + (long long)a.layer * a.pool.layer_elems;
  const float* vbase = (const float*)a.pool.v + (long long)a.layer * a.pool.layer_elems;

  f32x4 acc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t) acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  int q = next_rel(qbeg);
  while (q < qend) {
    const int qa = q;
    const int qb = next_rel(qa + 1);
    q = qb < qend ? next_rel(qb + 1) : qend;
    const bool hasB = qb < qend;

    int ownA, baseA, ownB = -2, baseB = 0;
    const int blkA = key_block(p, b, qa, nP, nS, ownA, baseA);
    const int blkB = hasB ? key_block(p, b, qb, nP, nS, ownB, baseB) : 0;

    // scores of the two blocks
    f32x4 sA = {0.f, 0.f, 0.f, 0.f}, sB = {0.f, 0.f, 0.f, 0.f};
    {
      const float* kA = kbase + ((long long)blkA * a.Hkv + kvh) * (kBlock * HD) + lr * HD + lg * 8;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 kh, kl;
        split8(*(const float4*)(kA + s * 32), *(const float4*)(kA + s * 32 + 4), kh, kl);
        sA = mfma3(kh, kl, qh[s], ql[s], sA);
      }
      if (hasB) {
        const float* kB = kbase + ((long long)blkB * a.Hkv + kvh) * (kBlock * HD) + lr * HD + lg * 8;
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          bf16x8 kh, kl;
          split8(*(const float4*)(kB + s * 32), *(const float4*)(kB + s * 32 + 4), kh, kl);
          sB = mfma3(kh, kl, qh[s], ql[s], sB);
        }
      }
    }
    float sv[8];
    float mt = -INFINITY;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int t = lg * 4 + e;
      sv[e] = key_valid(p, ownA, baseA + t, ri, Lp) ? sA[e] * a.scale_log2 : -INFINITY;
      sv[4 + e] = (hasB && key_valid(p, ownB, baseB + t, ri, Lp)) ? sB[e] * a.scale_log2 : -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) mt = fmaxf(mt, sv[e]);
    mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
    mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
    const float m_new = fmaxf(m_run, mt);
    const float m_use = m_new == -INFINITY ? 0.f : m_new;
    const float corr = exp2f(m_run - m_use);
    float psum = 0.f;
    float pv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv[e] = exp2f(sv[e] - m_use);
      psum += pv[e];
    }
    bf16x8 ph, pl;
    split8(make_float4(pv[0], pv[1], pv[2], pv[3]), make_float4(pv[4], pv[5], pv[6], pv[7]), ph, pl);
    l_run = l_run * corr + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      acc[t][0] *= corr;
      acc[t][1] *= corr;
      acc[t][2] *= corr;
      acc[t][3] *= corr;
    }
    // O^T += V^T . P^T
    const float* vA = vbase + ((long long)blkA * a.Hkv + kvh) * (HD * kBlock) + lr * kBlock + lg * 4;
    const float* vB = vbase + ((long long)blkB * a.Hkv + kvh) * (HD * kBlock) + lr * kBlock + lg * 4;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const float4 va = *(const float4*)(vA + t * 16 * kBlock);
      const float4 vb = hasB ? *(const float4*)(vB + t * 16 * kBlock) : make_float4(0.f, 0.f, 0.f, 0.f);
      bf16x8 vh, vl;
      split8(va, vb, vh, vl);
      acc[t] = mfma3(vh, vl, ph, pl, acc[t]);
    }
  }

  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  if (!ri.valid) return;
  const long long rowid = (long long)ri.m * a.H + ri.h;
  if (a.nsplit == 1) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    const long long o = rowid * HD + lg * 4;
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
      *(bf16x4*)(a.Ohi + o + t * 16) = hv;
      *(bf16x4*)(a.Olo + o + t * 16) = lv;
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

// Merge the split partials of every (row, head): one wave per row.
template <int HD>
__global__ __launch_bounds__(256) void attn_combine(AttnArgs a) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= a.rows_total) return;
  float mx = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) mx = fmaxf(mx, a.part_ml[((long long)s * a.rows_total + row) * 2]);
  const float mu = mx == -INFINITY ? 0.f : mx;
  constexpr int PER = (HD + 63) / 64;
  float o[PER] = {};
  float l = 0.f;
  for (int s = 0; s < a.nsplit; ++s) {
    const long long pr = (long long)s * a.rows_total + row;
    const float w = exp2f(a.part_ml[pr * 2] - mu);
    l += w * a.part_ml[pr * 2 + 1];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      int d = lane + 64 * u;
      if (d < HD) o[u] += w * a.part_o[pr * HD + d];
    }
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    int d = lane + 64 * u;
    if (d < HD) {
      bf16 h, lo;
      split_bf16(o[u] * inv, h, lo);
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
  pl.row_tiles = (nrows + 15) / 16;
  pl.row_groups = (pl.row_tiles + 3) / 4;
  pl.threads = 64 * (pl.row_tiles < 4 ? pl.row_tiles : 4);
  const int nS = p.mode == kSuffix ? (p.j0 + p.R + kBlock - 1) / kBlock : 0;
  const int nP = p.mode == kSuffix ? (max_prefix_len + kBlock - 1) / kBlock
                                   : (max_prefix_len + p.R + kBlock - 1) / kBlock;
  const int nK = nP + p.kp * nS;
  if (dtype == 0) {
    pl.nsplit = 1;
    pl.blocks_per_split = nK;
    return pl;
  }
  // enough workgroups to cover the CUs several times, >= 2 blocks per split
  const int base = p.nb * Hkv * pl.row_groups;
  int want = (1024 + base - 1) / base;
  int maxs = (nK + 1) / 2;
  int s = want < maxs ? want : maxs;
  if (s > max_splits) s = max_splits;
  if (s < 1) s = 1;
  int bps = (nK + s - 1) / s;
  bps += bps & 1;
  s = (nK + bps - 1) / bps;
  if (s < 1) s = 1;
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
  dim3 grid(pl.nsplit, a.p.nb * a.Hkv, pl.row_groups);
  switch (hd) {
    case 32: attn_mfma<32><<<grid, pl.threads, 0, st>>>(a); break;
    case 64: attn_mfma<64><<<grid, pl.threads, 0, st>>>(a); break;
    case 128: attn_mfma<128><<<grid, pl.threads, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
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
