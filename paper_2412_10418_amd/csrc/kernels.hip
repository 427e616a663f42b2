// Row-wise kernels of the CDSL step: embedding gather, RMSNorm, rotary
// embedding + KV write, the fused log-softmax / gather / argmax / top-k of a
// logits row, hard rejection and beam scores, rewards, beam selection, and
// the commit (emit, next beams, prefix promotion).
#include <float.h>

#include "block_pool.h"
#include "common.h"
#include "kernels.h"

namespace cdsl {

namespace {

template <int NW>
__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int u = 0; u < NW; ++u) t += sh[u];
  return t;
}

// ---------------------------------------------------------------------------
// A token id outside [0, V) sets *bad (the library reports it as an invalid
// argument at its next synchronisation) and is clamped for the read, so it
// never reads out of bounds.
// With rowinfo, row m's KV place is also recorded for the pass's layers:
// rowinfo[m] = (block * 16 + slot, position).
template <typename T>
__global__ __launch_bounds__(256) void embed_rows(PassDesc p, const T* __restrict__ emb, float* __restrict__ h,
                                                  int D, int V, int* __restrict__ bad, int2* __restrict__ rowinfo) {
  const int m = blockIdx.x;
  int bi, b, i, j;
  row_decode(p, m, bi, b, i, j);
  if (rowinfo && threadIdx.x == 0) {
    int blk, slot, pos;
    kv_slot(p, b, i, j, p.Lp[b], blk, slot, pos);
    rowinfo[m] = make_int2(blk * kBlock + slot, pos);
  }
  const int raw = p.tok[(long long)(b * p.kp + i) * p.tok_stride + p.tok_off + j];
  if ((raw < 0 || raw >= V) && threadIdx.x == 0 && bad) *bad = 1;
  const int tok = min(max(raw, 0), V - 1);
  const T* e = emb + (long long)tok * D;
  float* o = h + (long long)m * D;
  for (int c = threadIdx.x; c < D; c += 256) o[c] = to_f32<T>(e[c]);
}

// out[r] = x[src(r)] / sqrt(mean(x^2) + eps) * g.  src(r) = r, or the last
// row of beam r when last_only (prompt prefill: only the last position needs
// logits).  The result goes to out32 (fp32) or, for bf16-weight models, to
// the hi / lo planes that the next projection consumes.  hid (fp32)
// additionally receives the normed row of every beam's last row (the reward
// reads it).
//
// With S > 0 split planes part[S][rows][D] of a residual projection, the
// row is first completed: x[r] += sum of the planes in split order (the
// same arithmetic as the split-K reduce), written back to x.  g == null
// then only folds.
// The row stays in registers between the two phases: float4 column groups
// threadIdx.x + NT * u, u < kNormU (D <= 4 * NT * kNormU).
constexpr int kNormU = 8;

template <int NT>
__global__ __launch_bounds__(NT) void rmsnorm_rows(float* __restrict__ x, const float* __restrict__ g,
                                                    float* __restrict__ out32, bf16* __restrict__ ohi,
                                                    bf16* __restrict__ olo, int D, float eps, int last_only, int R,
                                                    float* __restrict__ hid, const float* __restrict__ part, int S,
                                                    int rows) {
  __shared__ float sh[NT / 64];
  const int r = blockIdx.x;
  const int src = last_only ? r * R + (R - 1) : r;
  float* xr = x + (long long)src * D;
  float4 v[kNormU];
  float ss = 0.f;
  const long long plane = (long long)rows * D;
  const float* pr = part + (long long)src * D;
#pragma unroll
  for (int u = 0; u < kNormU; ++u) {
    const int c = (threadIdx.x + NT * u) * 4;
    v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (c >= D) continue;
    if (S > 0) {
      // the planes are loaded eight at a time (independent loads in flight)
      // and added in split order
      float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int z0 = 0; z0 < S; z0 += 8) {
        float4 t[8];
#pragma unroll
        for (int e = 0; e < 8; ++e)
          t[e] = z0 + e < S ? *(const float4*)(pr + (z0 + e) * plane + c) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (z0 + e < S) {
            a.x += t[e].x;
            a.y += t[e].y;
            a.z += t[e].z;
            a.w += t[e].w;
          }
      }
      const float4 h = *(const float4*)(xr + c);
      a.x += h.x;
      a.y += h.y;
      a.z += h.z;
      a.w += h.w;
      *(float4*)(xr + c) = a;
      v[u] = a;
    } else {
      v[u] = *(const float4*)(xr + c);
    }
    ss = fmaf(v[u].x, v[u].x, ss);
    ss = fmaf(v[u].y, v[u].y, ss);
    ss = fmaf(v[u].z, v[u].z, ss);
    ss = fmaf(v[u].w, v[u].w, ss);
  }
  if (!g) return;
  ss = block_sum<NT / 64>(ss, sh);
  const float inv = rsqrtf(ss / (float)D + eps);
  const long long o = (long long)r * D;
  const bool want_hid = hid && (last_only || (r % R) == R - 1);
  float* hr = want_hid ? hid + (long long)(last_only ? r : r / R) * D : nullptr;
#pragma unroll
  for (int u = 0; u < kNormU; ++u) {
    const int c = (threadIdx.x + NT * u) * 4;
    if (c >= D) continue;
    const float4 gg = *(const float4*)(g + c);
    const float4 y = make_float4(v[u].x * inv * gg.x, v[u].y * inv * gg.y, v[u].z * inv * gg.z, v[u].w * inv * gg.w);
    if (out32) {
      *(float4*)(out32 + o + c) = y;
    } else {
      bf16x4 h4, l4;
      const float yy[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        bf16 h, l;
        split_bf16(yy[e], h, l);
        h4[e] = h;
        l4[e] = l;
      }
      *(bf16x4*)(ohi + o + c) = h4;
      *(bf16x4*)(olo + o + c) = l4;
    }
    if (hr) *(float4*)(hr + c) = y;
  }
}

// Rotary embedding of q and k (rotate-half pairs (d, d + hd/2), angle
// pos * theta^(-2d/hd) from the host-built tables), then q -> Q buffer and
// k, v -> the row's KV slot: prefix block for kAppend, the beam's suffix
// block for kSuffix.
template <typename T>
__global__ __launch_bounds__(256) void rope_kv_write(PassDesc p, const float* __restrict__ qkv, T* __restrict__ qout,
                                                     KVPool pool, int layer, const float* __restrict__ cos_t,
                                                     const float* __restrict__ sin_t, int H, int Hkv, int hd) {
  const int m = blockIdx.x;
  int bi, b, i, j;
  row_decode(p, m, bi, b, i, j);
  int pos, blk, slot;
  kv_slot(p, b, i, j, p.Lp[b], blk, slot, pos);
  const int half = hd / 2;
  const float* row = qkv + (long long)m * (H + 2 * Hkv) * hd;
  const float* ct = cos_t + (long long)pos * half;
  const float* stt = sin_t + (long long)pos * half;
  T* kb = (T*)pool.k + (long long)layer * pool.layer_elems + ((long long)blk * Hkv) * kBlock * hd;
  T* vb = (T*)pool.v + (long long)layer * pool.layer_elems + ((long long)blk * Hkv) * kBlock * hd;
  // q and k heads: pairs
  const int npairs = (H + Hkv) * half;
  for (int u = threadIdx.x; u < npairs; u += 256) {
    const int hh = u / half, d = u % half;
    const float x1 = row[hh * hd + d], x2 = row[hh * hd + d + half];
    const float c = ct[d], s = stt[d];
    const float y1 = rope_first(x1, x2, c, s), y2 = rope_second(x1, x2, c, s);
    if (hh < H) {
      T* q = qout + ((long long)m * H + hh) * hd;
      q[d] = from_f32<T>(y1);
      q[d + half] = from_f32<T>(y2);
    } else {
      T* kr = kb + ((long long)(hh - H) * kBlock + slot) * hd;
      kr[d] = from_f32<T>(y1);
      kr[d + half] = from_f32<T>(y2);
    }
  }
  // v: transposed [hd][16] per block and head
  const float* vrow = row + (long long)(H + Hkv) * hd;
  for (int u = threadIdx.x; u < Hkv * hd; u += 256) {
    const int hh = u / hd, d = u % hd;
    vb[((long long)hh * hd + d) * kBlock + slot] = from_f32<T>(vrow[u]);
  }
}

// Same for bf16-weight models, whose KV pool holds each fp32 value as a
// bf16 (hi, lo) pair in the split unit format (K [plane][16][hd], V
// [plane][hd][16]).  q stays fp32.  With S > 0, qkv holds S split planes
// [S][M][(H + 2 Hkv) hd] of the projection, summed here in split order.
//
// Workgroups 0..M-1 take one row each (rotary q and k, the K write).
// Workgroups M.. take one (beam, KV head) each, one thread per head dim,
// and write V: the rows of a beam sit in consecutive slots, so each thread
// writes a run of slots of its dim row with wide stores instead of one
// 2-byte store per row into a different 32-byte row.
struct QkvRow {
  const float* qkv;
  long long split_plane;
  int S;
  // four consecutive values of row m at column idx (summed over the split
  // planes in split order, eight planes' loads in flight at a time)
  __device__ __forceinline__ float4 val4(long long m, int W, int idx) const {
    const float* row = qkv + m * W;
    if (S <= 0) return *(const float4*)(row + idx);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int z0 = 0; z0 < S; z0 += 8) {
      float4 t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        t[u] = z0 + u < S ? *(const float4*)(row + (z0 + u) * split_plane + idx) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (z0 + u < S) {
          v.x += t[u].x;
          v.y += t[u].y;
          v.z += t[u].z;
          v.w += t[u].w;
        }
    }
    return v;
  }
  __device__ __forceinline__ float val(long long m, int W, int idx) const {
    const float* row = qkv + m * W;
    if (S <= 0) return row[idx];
    float v = 0.f;
    for (int z = 0; z < S; ++z) v += row[z * split_plane + idx];
    return v;
  }
};

template <int NT>
__global__ __launch_bounds__(NT) void rope_kv_write_split(PassDesc p, const float* __restrict__ qkv,
                                                           float* __restrict__ qout, KVPool pool, int layer,
                                                           const float* __restrict__ cos_t,
                                                           const float* __restrict__ sin_t, int H, int Hkv, int hd,
                                                           int S) {
  const int M = p.nb * p.kp * p.R;
  const int W = (H + 2 * Hkv) * hd;
  const QkvRow src{qkv, (long long)M * W, S};
  const int half = hd / 2;
  const long long unit = split_unit_elems(hd);
  const long long plane = (long long)kBlock * hd;
  bf16* kl = (bf16*)pool.k + (long long)layer * 2 * pool.layer_elems;
  bf16* vl = (bf16*)pool.v + (long long)layer * 2 * pool.layer_elems;
  if ((int)blockIdx.x < M) {
    const int m = blockIdx.x;
    int bi, b, i, j;
    row_decode(p, m, bi, b, i, j);
    int blk, slot, pos;
    kv_slot(p, b, i, j, p.Lp[b], blk, slot, pos);
    const float* ct = cos_t + (long long)pos * half;
    const float* stt = sin_t + (long long)pos * half;
    bf16* kb = kl + (long long)blk * Hkv * unit;
    // q and k heads: rotate-half pairs (d, d + hd/2), four d at a time
    const int q4 = half / 4;
    for (int u = threadIdx.x; u < (H + Hkv) * q4; u += NT) {
      const int hh = u / q4, d = (u % q4) * 4;
      const float4 x1 = src.val4(m, W, hh * hd + d), x2 = src.val4(m, W, hh * hd + d + half);
      const float4 c = *(const float4*)(ct + d), sn = *(const float4*)(stt + d);
      const float y1[4] = {rope_first(x1.x, x2.x, c.x, sn.x), rope_first(x1.y, x2.y, c.y, sn.y),
                           rope_first(x1.z, x2.z, c.z, sn.z), rope_first(x1.w, x2.w, c.w, sn.w)};
      const float y2[4] = {rope_second(x1.x, x2.x, c.x, sn.x), rope_second(x1.y, x2.y, c.y, sn.y),
                           rope_second(x1.z, x2.z, c.z, sn.z), rope_second(x1.w, x2.w, c.w, sn.w)};
      if (hh < H) {
        float* q = qout + ((long long)m * H + hh) * hd + d;
        *(float4*)q = make_float4(y1[0], y1[1], y1[2], y1[3]);
        *(float4*)(q + half) = make_float4(y2[0], y2[1], y2[2], y2[3]);
      } else {
        bf16* kr = kb + (long long)(hh - H) * unit + (long long)slot * hd + d;
        bf16x4 h1, l1, h2, l2;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          bf16 h, l;
          split_bf16(y1[e], h, l);
          h1[e] = h;
          l1[e] = l;
          split_bf16(y2[e], h, l);
          h2[e] = h;
          l2[e] = l;
        }
        *(bf16x4*)kr = h1;
        *(bf16x4*)(kr + plane) = l1;
        *(bf16x4*)(kr + half) = h2;
        *(bf16x4*)(kr + plane + half) = l2;
      }
    }
    return;
  }
  // V of (beam group, KV head) tasks, NT / hd of them per workgroup: thread
  // d < hd of a task owns dim row d
  const int per = NT / hd;
  const int task = ((int)blockIdx.x - M) * per + (int)threadIdx.x / hd;
  const int d = (int)threadIdx.x % hd;
  if ((int)threadIdx.x >= per * hd || task >= p.nb * p.kp * Hkv) return;
  const int g = task / Hkv, hh = task % Hkv;
  const int bi = g / p.kp, i = g % p.kp;
  const int b = pass_batch(p, bi);
  const int Lp = p.Lp[b];
  const int voff = (H + Hkv) * hd + hh * hd + d;
  const long long m0 = (long long)g * p.R;
  int j = 0;
  while (j < p.R) {
    int blk, slot, pos;
    kv_slot(p, b, i, j, Lp, blk, slot, pos);
    const int n = min(p.R - j, kBlock - slot);   // rows of this block: slots [slot, slot + n)
    // every row's load is issued before any is used (the rows are
    // independent; one latency per block instead of one per row)
    float vv[kBlock];
#pragma unroll
    for (int t = 0; t < kBlock; ++t) vv[t] = (t >= slot && t < slot + n) ? src.val(m0 + j + (t - slot), W, voff) : 0.f;
    store_v_run(vl + ((long long)blk * Hkv + hh) * unit + (long long)d * kBlock, plane, vv, slot, n);
    j += n;
  }
}

// ---------------------------------------------------------------------------
// Logits row statistics, one workgroup per row, one read of the row:
// online logsumexp, argmax, thread-local top-KK lists merged by KK rounds of
// block argmax.  Ordering: value descending, then id ascending.
// A token id that indexes the vocabulary even for a row without a finite
// logit (all NaN), so that the next pass's embedding never reads out of
// bounds; the NaN still reaches the scores and makes the selection fail.
__device__ __forceinline__ int vocab_id(int id, int V) { return (id >= 0 && id < V) ? id : 0; }

template <int KKMAX>
__global__ __launch_bounds__(256) void logit_rows_kernel(LogitArgs a) {
  __shared__ float shv[4];
  __shared__ int shi[4];
  __shared__ float shs[4];
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* z = a.logits + (long long)m * (a.ld ? a.ld : (long long)a.V);

  float mloc = -INFINITY, sloc = 0.f;
  float bv = -INFINITY;
  int bid = 0x7fffffff;
  float lv[KKMAX > 0 ? KKMAX : 1];
  int li[KKMAX > 0 ? KKMAX : 1];
#pragma unroll
  for (int s = 0; s < (KKMAX > 0 ? KKMAX : 1); ++s) {
    lv[s] = -INFINITY;
    li[s] = 0x7fffffff;
  }
  auto visit = [&](float v, int id) {
    if (a.want_lse) {
      if (v > mloc) {
        sloc = sloc * __expf(mloc - v) + 1.f;
        mloc = v;
      } else {
        sloc += __expf(v - mloc);
      }
    }
    if (vi_better(v, id, bv, bid)) {
      bv = v;
      bid = id;
    }
    // keep the best KKMAX (>= kk) so every list index is static
    if (KKMAX > 0 && vi_better(v, id, lv[(KKMAX > 0 ? KKMAX : 1) - 1], li[(KKMAX > 0 ? KKMAX : 1) - 1])) {
      float cv = v;
      int ci = id;
#pragma unroll
      for (int s = 0; s < KKMAX; ++s) {
        if (vi_better(cv, ci, lv[s], li[s])) {
          float tv = lv[s];
          int ti = li[s];
          lv[s] = cv;
          li[s] = ci;
          cv = tv;
          ci = ti;
        }
      }
    }
  };
  const int V4 = (a.V & 3) == 0 ? a.V / 4 : 0;
  const float4* z4 = (const float4*)z;
  for (int c = tid; c < V4; c += 256) {
    float4 v = z4[c];
    visit(v.x, 4 * c);
    visit(v.y, 4 * c + 1);
    visit(v.z, 4 * c + 2);
    visit(v.w, 4 * c + 3);
  }
  for (int c = 4 * V4 + tid; c < a.V; c += 256) visit(z[c], c);

  // argmax
  {
    float v = bv;
    int id = bid;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      float ov = __shfl_xor(v, o, 64);
      int oi = __shfl_xor(id, o, 64);
      if (vi_better(ov, oi, v, id)) {
        v = ov;
        id = oi;
      }
    }
    if (lane == 0) {
      shv[w] = v;
      shi[w] = id;
    }
    __syncthreads();
    if (tid == 0) {
      float fv = shv[0];
      int fi = shi[0];
      for (int u = 1; u < 4; ++u)
        if (vi_better(shv[u], shi[u], fv, fi)) {
          fv = shv[u];
          fi = shi[u];
        }
      shi[0] = fi;
      shv[0] = fv;
    }
    __syncthreads();
    if (tid == 0 && a.amax) a.amax[rowmap_index(a.amax_map, m)] = vocab_id(shi[0], a.V);
    __syncthreads();
  }
  if (!a.want_lse) return;
  // logsumexp
  float lse;
  {
    float mm = wave_max(mloc);
    if (lane == 0) shv[w] = mm;
    __syncthreads();
    const float M = fmaxf(fmaxf(shv[0], shv[1]), fmaxf(shv[2], shv[3]));
    float sv = mloc == -INFINITY ? 0.f : sloc * __expf(mloc - M);
    sv = wave_sum(sv);
    if (lane == 0) shs[w] = sv;
    __syncthreads();
    lse = M + __logf(shs[0] + shs[1] + shs[2] + shs[3]);
    __syncthreads();
  }
  if (a.lp && tid == 0) {
    const int tok = a.gather_tok[rowmap_index(a.gather_map, m)];
    const bool in = tok >= 0 && tok < a.V;
    if (!in && a.bad) *a.bad = 1;
    a.lp[m] = in ? z[tok] - lse : __int_as_float(0x7fc00000);
  }
  if (KKMAX == 0 || a.kk == 0) return;
  const int dst = a.topk_rows ? a.topk_rows[m] : m;
  for (int r = 0; r < a.kk; ++r) {
    float v = lv[0];
    int id = li[0];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      float ov = __shfl_xor(v, o, 64);
      int oi = __shfl_xor(id, o, 64);
      if (vi_better(ov, oi, v, id)) {
        v = ov;
        id = oi;
      }
    }
    if (lane == 0) {
      shv[w] = v;
      shi[w] = id;
    }
    __syncthreads();
    float fv = shv[0];
    int fi = shi[0];
    for (int u = 1; u < 4; ++u)
      if (vi_better(shv[u], shi[u], fv, fi)) {
        fv = shv[u];
        fi = shi[u];
      }
    if (tid == 0) {
      a.topk_ids[(long long)dst * a.kk + r] = vocab_id(fi, a.V);
      a.topk_lp[(long long)dst * a.kk + r] = fv - lse;
    }
    if (li[0] == fi) {   // ids are unique: exactly one thread pops
#pragma unroll
      for (int s = 0; s + 1 < (KKMAX > 0 ? KKMAX : 1); ++s) {
        lv[s] = lv[s + 1];
        li[s] = li[s + 1];
      }
      lv[(KKMAX > 0 ? KKMAX : 1) - 1] = -INFINITY;
      li[(KKMAX > 0 ? KKMAX : 1) - 1] = 0x7fffffff;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Hard rejection (leading matches of target argmax and lookahead) and beam
// scores, one thread per (b, i).
// With lq and u (soft rejection, speculative sampling): x_j is kept while
// u_j <= min(1, p_j(x_j) / q_j(x_j)), the ratio formed from the two log-probs.
__global__ void beam_scores_kernel(int BK, int d, const int* __restrict__ look, const int* __restrict__ y,
                                   const float* __restrict__ lp, const float* __restrict__ head_lp,
                                   const float* __restrict__ lq, const float* __restrict__ u,
                                   int* __restrict__ n_accept, float* __restrict__ scores) {
  const int bk = blockIdx.x * blockDim.x + threadIdx.x;
  if (bk >= BK) return;
  int n = 0;
  bool run = true;
  float s = head_lp ? head_lp[bk] : 0.f;
  for (int j = 0; j < d; ++j) {
    const long long r = (long long)bk * d + j;
    bool keep;
    if (lq) keep = u[r] <= fminf(1.f, expf(lp[r] - lq[r]));
    else keep = y[r] == look[(long long)bk * (d + 1) + j + 1];
    if (run && keep) ++n;
    else run = false;
    s += lp[r];
  }
  n_accept[bk] = n;
  scores[bk] = s;
}

// first_at (optional, [B]): Step-1 of the controller with b = 1 keeps the
// greedy head (beam 0) when its reward reaches first_at[b]; NaN = no such rule.
__global__ void select_kernel(int B, int k, const float* __restrict__ scores, const float* __restrict__ reward,
                              float alpha, int reward_only, const float* __restrict__ first_at,
                              int* __restrict__ beam) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  if (first_at) {
    const float t = first_at[b], r0 = reward[b * k];
    if (isnan(r0)) {
      beam[b] = -1;
      return;
    }
    if (!isnan(t) && r0 >= t) {
      beam[b] = 0;
      return;
    }
  }
  int best = -1;
  float bv = -INFINITY;
  bool bad = false;
  for (int i = 0; i < k; ++i) {
    const float sc = scores[b * k + i], r = reward[b * k + i];
    if (isnan(sc) || isnan(r)) bad = true;
    const float v = reward_only ? r : sc + alpha * r;
    if (best < 0 || v > bv) {
      best = i;
      bv = v;
    }
  }
  beam[b] = bad ? -1 : best;
}

// Speculative sampling rows (Sec. 3.2.2), one workgroup per fed row m of a
// verification (rows ordered (b, i, j), both logit arrays [M][V]):
//   draft_lp[m] = log q(x), x the row's lookahead token;
//   res_ids[m]  = the draw at v[m] from w = max(0, p - q) / Z, inverting the
//                 cumulative sum over token ids in ascending order (argmax p
//                 when Z = 0), and res_lp[m] = log p of it.
// Three passes over the rows: both logsumexps and argmax p; per-wave sums
// of w over four contiguous id segments; one wave walks the segment that
// holds v * Z with a 64-lane scan per chunk.
__global__ __launch_bounds__(256) void soft_rows_kernel(const float* __restrict__ zp_all,
                                                        const float* __restrict__ zq_all, int V, int d,
                                                        const int* __restrict__ look, const float* __restrict__ v,
                                                        float* __restrict__ draft_lp, int* __restrict__ res_ids,
                                                        float* __restrict__ res_lp) {
  __shared__ float sh_m[2][4], sh_s[2][4], sh_bv[4], part[4];
  __shared__ int sh_bi[4];
  __shared__ int sh_res;
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float* zp = zp_all + (long long)m * V;
  const float* zq = zq_all + (long long)m * V;

  float mp = -INFINITY, sp = 0.f, mq = -INFINITY, sq = 0.f, bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t = tid; t < V; t += 256) {
    const float a = zp[t], b = zq[t];
    if (a > mp) {
      sp = sp * __expf(mp - a) + 1.f;
      mp = a;
    } else {
      sp += __expf(a - mp);
    }
    if (b > mq) {
      sq = sq * __expf(mq - b) + 1.f;
      mq = b;
    } else {
      sq += __expf(b - mq);
    }
    if (vi_better(a, t, bv, bi)) {
      bv = a;
      bi = t;
    }
  }
  {
    float ov;
    int oi;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      ov = __shfl_xor(bv, o, 64);
      oi = __shfl_xor(bi, o, 64);
      if (vi_better(ov, oi, bv, bi)) {
        bv = ov;
        bi = oi;
      }
    }
    const float Mp = wave_max(mp), Mq = wave_max(mq);
    const float s1 = wave_sum(mp == -INFINITY ? 0.f : sp * __expf(mp - Mp));
    const float s2 = wave_sum(mq == -INFINITY ? 0.f : sq * __expf(mq - Mq));
    if (lane == 0) {
      sh_m[0][wv] = Mp;
      sh_s[0][wv] = s1;
      sh_m[1][wv] = Mq;
      sh_s[1][wv] = s2;
      sh_bv[wv] = bv;
      sh_bi[wv] = bi;
    }
  }
  __syncthreads();
  float lse[2];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const float M = fmaxf(fmaxf(sh_m[r][0], sh_m[r][1]), fmaxf(sh_m[r][2], sh_m[r][3]));
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u) sum += sh_m[r][u] == -INFINITY ? 0.f : sh_s[r][u] * __expf(sh_m[r][u] - M);
    lse[r] = M + __logf(sum);
  }
  int amax = sh_bi[0];
  {
    float av = sh_bv[0];
    for (int u = 1; u < 4; ++u)
      if (vi_better(sh_bv[u], sh_bi[u], av, amax)) {
        av = sh_bv[u];
        amax = sh_bi[u];
      }
  }
  // per-wave sums of w over contiguous segments (multiples of 64 ids)
  const int seg = ((V + 255) / 256) * 64;
  const int s0 = wv * seg, s1 = min(V, s0 + seg);
  float acc = 0.f;
  for (int t = s0 + lane; t < s1; t += 64) acc += fmaxf(0.f, __expf(zp[t] - lse[0]) - __expf(zq[t] - lse[1]));
  acc = wave_sum(acc);
  if (lane == 0) part[wv] = acc;
  if (tid == 0) sh_res = -1;
  __syncthreads();
  const float Z = part[0] + part[1] + part[2] + part[3];
  const float T = v[m] * Z;
  // segment holding T (the last one with mass when rounding leaves T past the total)
  int sg = -1;
  float before = 0.f;
  {
    float run = 0.f;
    for (int u = 0; u < 4; ++u) {
      if (part[u] > 0.f) {
        if (run + part[u] > T) {
          sg = u;
          before = run;
          break;
        }
        sg = u;
        before = run;
      }
      run += part[u];
    }
  }
  if (Z > 0.f && wv == sg) {
    const int g0 = sg * seg, g1 = min(V, g0 + seg);
    const float Tl = T - before;
    float run = 0.f;
    int last = -1;
    int found = -1;
    for (int c0 = g0; c0 < g1; c0 += 64) {
      const int t = c0 + lane;
      const float wt = t < g1 ? fmaxf(0.f, __expf(zp[t] - lse[0]) - __expf(zq[t] - lse[1])) : 0.f;
      float sc = wt;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const float n = __shfl_up(sc, o, 64);
        if (lane >= o) sc += n;
      }
      const unsigned long long hit = __ballot(wt > 0.f && run + sc > Tl);
      if (hit) {
        found = c0 + __builtin_ctzll(hit);
        break;
      }
      const unsigned long long mass = __ballot(wt > 0.f);
      if (mass) last = c0 + 63 - __builtin_clzll(mass);
      run += __shfl(sc, 63, 64);
    }
    if (lane == 0) sh_res = found >= 0 ? found : last;
  }
  __syncthreads();
  if (tid == 0) {
    int res = (Z > 0.f && sh_res >= 0) ? sh_res : amax;
    const bool ok = res >= 0 && res < V;   // false only for rows without a finite logit
    if (!ok) res = 0;
    const int x = look[(long long)(m / d) * (d + 1) + (m % d) + 1];
    draft_lp[m] = (x >= 0 && x < V) ? zq[x] - lse[1] : __int_as_float(0x7fc00000);
    res_ids[m] = res;
    res_lp[m] = ok ? zp[res] - lse[0] : __int_as_float(0x7fc00000);
  }
}

// Alg. 1 state of each prompt after a k = 1 lookahead: a = n / d (float64,
// as the thresholds are given), r = the accepted window's reward.
// state: 1 = S1 (a >= a_t and r >= r_t), 2 = S2/S3 (a < a_t), 4 = S4.
// first_at[b] = r_t where Step-1 with b = 1 applies (state 2, b1 set), else NaN.
__global__ void controller_states_kernel(int B, int d, const int* __restrict__ n_accept,
                                         const float* __restrict__ reward, double a_t, double r_t, int b1,
                                         int* __restrict__ state, float* __restrict__ first_at) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const double a = (double)n_accept[b] / (double)d;
  const double r = (double)reward[b];
  const int s = a < a_t ? 2 : (r >= r_t ? 1 : 4);
  state[b] = s;
  first_at[b] = (s == 2 && b1) ? (float)r_t : __int_as_float(0x7fc00000);
}

// Keyword reward, one workgroup per (b, i): distinct keywords present in
// generated-so-far + the row's head (when head is set) + its first
// upto[b, i] lookahead tokens (all d when upto is null).
__global__ __launch_bounds__(256) void reward_keywords_kernel(int k, int d, const int* __restrict__ gen,
                                                              int gen_stride, const int* __restrict__ gen_len,
                                                              const int* __restrict__ look,
                                                              const int* __restrict__ upto, int head,
                                                              const int* __restrict__ kws, int n_kw, int normalize,
                                                              float* __restrict__ reward) {
  __shared__ int hit[64];
  __shared__ int uniq[64];
  const int bk = blockIdx.x;
  const int b = bk / k;
  for (int u = threadIdx.x; u < 64; u += 256) hit[u] = 0;
  __syncthreads();
  const int* kw = kws + (long long)b * n_kw;
  const int gl = gen_len[b];
  const int nx = upto ? min(max(upto[bk], 0), d) : d;
  const int skip = head ? 0 : 1;
  const int total = gl + nx + 1 - skip;
  for (int t = threadIdx.x; t < total; t += 256) {
    const int tok = t < gl ? gen[(long long)b * gen_stride + t] : look[(long long)bk * (d + 1) + skip + (t - gl)];
    for (int u = 0; u < n_kw; ++u)
      if (kw[u] == tok) atomicOr(&hit[u], 1);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int cnt = 0, nd = 0;
    for (int u = 0; u < n_kw; ++u) {
      bool dup = false;
      for (int v = 0; v < u; ++v) dup |= kw[v] == kw[u];
      if (dup) continue;
      ++nd;
      cnt += hit[u];
    }
    reward[bk] = normalize ? (float)cnt / (float)(nd > 0 ? nd : 1) : (float)cnt;
  }
}

__global__ __launch_bounds__(256) void reward_linear_kernel(const float* __restrict__ hidden,
                                                            const float* __restrict__ w, int D,
                                                            float* __restrict__ reward) {
  __shared__ float sh[4];
  const int bk = blockIdx.x;
  const float* h = hidden + (long long)bk * D;
  float s = 0.f;
  for (int c = threadIdx.x; c < D; c += 256) s = fmaf(h[c], w[c], s);
  s = block_sum<4>(s, sh);
  if (threadIdx.x == 0) reward[bk] = s;
}

// The commit kernels only stage their decisions, one record per prompt (see
// the layout in kernels.h); commit_apply_kernel carries a record out after
// the host has checked every prompt's record, so a commit that fails
// validation changes no generated tokens and no next heads.
__device__ __forceinline__ void stage_heads(int* st, int tcap, int kk, int u, int id, float lp) {
  st[kStageHdr + tcap + u] = id;
  st[kStageHdr + tcap + kk + u] = __float_as_int(lp);
}

// Beam commit, one thread per prompt: emit [c_i*, x_i*,1..n] of the selected
// beam.  res_ids / res_lp (soft rejection, [B, k, d]): when n < d the
// residual draw at the rejected position leads the next heads, followed by
// the row's top tokens without it.
__global__ void commit_kernel(int B, int k, int d, int kk, const int* __restrict__ look, const int* __restrict__ beam,
                              const int* __restrict__ n_accept, const int* __restrict__ rtk_ids,
                              const float* __restrict__ rtk_lp, const int* __restrict__ res_ids,
                              const float* __restrict__ res_lp, int* __restrict__ stage, int stage_stride,
                              int tcap) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int* st = stage + (long long)b * stage_stride;
  const int i = beam[b];
  const int n = (i >= 0 && i < k) ? n_accept[b * k + i] : -1;
  if (i < 0 || i >= k || n < 0 || n > d) {
    st[0] = -1;
    return;
  }
  const int bk = b * k + i;
  const int* row = look + (long long)bk * (d + 1);
  st[0] = n + 1;
  st[1] = n == d;
  st[2] = i;
  st[3] = n < d;
  for (int t = 0; t <= n; ++t) st[kStageHdr + t] = row[t];
  if (n < d && res_ids) {
    const long long q = (long long)bk * d + n;
    const long long r = q * kk;
    const int lead = res_ids[q];
    stage_heads(st, tcap, kk, 0, lead, res_lp[q]);
    int o = 1;
    for (int u = 0; u < kk && o < kk; ++u) {
      if (rtk_ids[r + u] == lead) continue;
      stage_heads(st, tcap, kk, o, rtk_ids[r + u], rtk_lp[r + u]);
      ++o;
    }
  } else if (n < d) {
    const long long r = ((long long)bk * d + n) * kk;
    for (int u = 0; u < kk; ++u) stage_heads(st, tcap, kk, u, rtk_ids[r + u], rtk_lp[r + u]);
  }
}

// Alg. 1 commit of a lookahead drafted from the prefix (one sequence per
// prompt, lookahead row [last prefix token, x_1..x_d]): emit x_1..x_n.  The
// next heads are row n's top-kk (the target after x_1..x_n) when n < d;
// when n = d, x_d is fed as a catch-up row.  n = 0 emits nothing.
__global__ void commit_prefix_kernel(int B, int d, int kk, const int* __restrict__ look,
                                     const int* __restrict__ n_accept, const int* __restrict__ rtk_ids,
                                     const float* __restrict__ rtk_lp, int* __restrict__ stage, int stage_stride,
                                     int tcap) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int* st = stage + (long long)b * stage_stride;
  const int n = n_accept[b];
  if (n < 0 || n > d) {
    st[0] = -1;
    return;
  }
  const int* row = look + (long long)b * (d + 1);
  st[0] = n;
  st[1] = n == d;
  st[2] = 0;
  st[3] = n < d;
  for (int t = 0; t < n; ++t) st[kStageHdr + t] = row[1 + t];
  if (n < d) {
    const long long r = ((long long)b * d + n) * kk;
    for (int u = 0; u < kk; ++u) stage_heads(st, tcap, kk, u, rtk_ids[r + u], rtk_lp[r + u]);
  }
}

// Head-only commit, one thread per prompt: prompts with mask[b] != 0 emit
// the head of their selected beam, fed afterwards as a one-row append pass
// that yields the next heads; the others emit nothing (n_emit = 0).
__global__ void commit_heads_kernel(int B, int k, int d, const int* __restrict__ look, const int* __restrict__ beam,
                                    const int* __restrict__ mask, int* __restrict__ stage, int stage_stride) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int* st = stage + (long long)b * stage_stride;
  st[1] = 0;
  st[3] = 0;
  if (!mask[b]) {
    st[0] = 0;
    return;
  }
  const int i = beam[b];
  if (i < 0 || i >= k) {
    st[0] = -1;
    return;
  }
  st[0] = 1;
  st[1] = 1;
  st[2] = i;
  st[kStageHdr] = look[(long long)(b * k + i) * (d + 1)];
}

// Append of given tokens, one thread per prompt: prompts with mask[b] != 0
// emit tokens[b] (checked against [0, V): an id outside it invalidates the
// record), fed afterwards as one appended row; the others emit nothing.
__global__ void commit_tokens_kernel(int B, const int* __restrict__ tokens, const int* __restrict__ mask, int V,
                                     int* __restrict__ stage, int stage_stride) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  int* st = stage + (long long)b * stage_stride;
  st[1] = 0;
  st[3] = 0;
  if (!mask[b]) {
    st[0] = 0;
    return;
  }
  const int tok = tokens[b];
  if (tok < 0 || tok >= V) {
    st[0] = -1;
    return;
  }
  st[0] = 1;
  st[1] = 1;
  st[2] = 0;
  st[kStageHdr] = tok;
}

// Withdraw the last cnt[b] tokens of prompt b's prefix (its length and its
// generated tokens).
__global__ void withdraw_kernel(int B, const int* __restrict__ cnt, int* __restrict__ Lp, int* __restrict__ gen_len) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  Lp[b] -= cnt[b];
  gen_len[b] -= cnt[b];
}

// Carries out the checked records: append the emitted tokens to the
// generated tokens, write the staged next heads, and queue the last emitted
// token of catch-up prompts.
__global__ void commit_apply_kernel(int B, const int* __restrict__ stage, int stage_stride, int tcap, int kk,
                                    int* __restrict__ gen, int gen_stride, int* __restrict__ gen_len,
                                    int* __restrict__ next_beams, float* __restrict__ next_head_lp,
                                    int* __restrict__ catch_tok) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int* st = stage + (long long)b * stage_stride;
  const int ne = st[0];
  if (ne > 0) {
    const int gl = gen_len[b];
    for (int t = 0; t < ne; ++t) gen[(long long)b * gen_stride + gl + t] = st[kStageHdr + t];
    gen_len[b] = gl + ne;
    if (st[1]) catch_tok[b] = st[kStageHdr + ne - 1];
  }
  if (ne >= 0 && st[3] && !st[1]) {
    for (int u = 0; u < kk; ++u) {
      next_beams[b * kk + u] = st[kStageHdr + tcap + u];
      next_head_lp[b * kk + u] = __int_as_float(st[kStageHdr + tcap + kk + u]);
    }
  }
}

// Alg. 1 passes from the prefix: the lookahead row starts with the last
// token of the prefix (the prompt's last token until something is
// generated), and those passes see a prefix one token shorter: Lm1 = Lp - 1.
__global__ void prefix_tail_kernel(int B, const int* __restrict__ gen, int gen_stride, const int* __restrict__ gen_len,
                                   const int* __restrict__ ptail, const int* __restrict__ Lp, int* __restrict__ Lm1,
                                   int* __restrict__ look, int look_stride) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  Lm1[b] = Lp[b] - 1;
  if (look) {
    const int gl = gen_len[b];
    look[(long long)b * look_stride] = gl > 0 ? gen[(long long)b * gen_stride + gl - 1] : ptail[b];
  }
}

__global__ void last_tokens_kernel(int B, const int* __restrict__ tokens, int L, int* __restrict__ out) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) out[b] = tokens[(long long)b * L + L - 1];
}

// Copy cnt suffix slots of the selected beam, from slot soff on, into the
// prefix at positions Lp[b] .. Lp[b] + cnt - 1, for every layer and KV head
// (cnt = min(n_emit, dlim)).
template <typename T>
__global__ __launch_bounds__(256) void promote_kernel(int k, KVPool pool, int n_layers, const int* __restrict__ stage,
                                                      int stage_stride, int dlim, int soff, const int* __restrict__ Lp,
                                                      const int* __restrict__ ptable, int ptable_stride,
                                                      const int* __restrict__ stable, int s_stride_b,
                                                      int s_stride_i) {
  const int b = blockIdx.x;
  const int layer = blockIdx.y;
  const int* st = stage + (long long)b * stage_stride;
  const int ne = st[0];
  if (ne <= 0) return;
  const int cnt = min(ne, dlim);
  const int i = st[2];
  const int L0 = Lp[b];
  const int hd = pool.hd, Hkv = pool.Hkv;
  T* kl = (T*)pool.k + (long long)layer * pool.layer_elems;
  T* vl = (T*)pool.v + (long long)layer * pool.layer_elems;
  const int per_tok = Hkv * hd;
  for (int u = threadIdx.x; u < cnt * per_tok; u += 256) {
    const int t = u / per_tok, rem = u % per_tok;
    const int hh = rem / hd, dd = rem % hd;
    const PromoteIndex ix = promote_index(stable + (long long)b * s_stride_b + i * s_stride_i,
                                          ptable + (long long)b * ptable_stride, L0, t, soff);
    const int sblk = ix.sblk, sslot = ix.sslot, pblk = ix.pblk, pslot = ix.pslot;
    kl[(((long long)pblk * Hkv + hh) * kBlock + pslot) * hd + dd] =
        kl[(((long long)sblk * Hkv + hh) * kBlock + sslot) * hd + dd];
    vl[(((long long)pblk * Hkv + hh) * hd + dd) * kBlock + pslot] =
        vl[(((long long)sblk * Hkv + hh) * hd + dd) * kBlock + sslot];
  }
}

// promote_kernel for the split bf16 pool format
__global__ __launch_bounds__(256) void promote_split_kernel(int k, KVPool pool, int n_layers,
                                                            const int* __restrict__ stage, int stage_stride, int dlim,
                                                            int soff, const int* __restrict__ Lp,
                                                            const int* __restrict__ ptable,
                                                            int ptable_stride, const int* __restrict__ stable,
                                                            int s_stride_b, int s_stride_i) {
  const int b = blockIdx.x;
  const int layer = blockIdx.y;
  const int* st = stage + (long long)b * stage_stride;
  const int ne = st[0];
  if (ne <= 0) return;
  const int cnt = min(ne, dlim);
  const int i = st[2];
  const int L0 = Lp[b];
  const int hd = pool.hd, Hkv = pool.Hkv;
  const long long unit = split_unit_elems(hd);
  const long long plane = (long long)kBlock * hd;
  bf16* kl = (bf16*)pool.k + (long long)layer * 2 * pool.layer_elems;
  bf16* vl = (bf16*)pool.v + (long long)layer * 2 * pool.layer_elems;
  const int per_tok = Hkv * hd;
  for (int u = threadIdx.x; u < cnt * per_tok; u += 256) {
    const int t = u / per_tok, rem = u % per_tok;
    const int hh = rem / hd, dd = rem % hd;
    const PromoteIndex ix = promote_index(stable + (long long)b * s_stride_b + i * s_stride_i,
                                          ptable + (long long)b * ptable_stride, L0, t, soff);
    const int sblk = ix.sblk, sslot = ix.sslot, pblk = ix.pblk, pslot = ix.pslot;
    const bf16* ks = kl + ((long long)sblk * Hkv + hh) * unit + (long long)sslot * hd + dd;
    bf16* kd = kl + ((long long)pblk * Hkv + hh) * unit + (long long)pslot * hd + dd;
    kd[0] = ks[0];
    kd[plane] = ks[plane];
    const bf16* vs = vl + ((long long)sblk * Hkv + hh) * unit + (long long)dd * kBlock + sslot;
    bf16* vd = vl + ((long long)pblk * Hkv + hh) * unit + (long long)dd * kBlock + pslot;
    vd[0] = vs[0];
    vd[plane] = vs[plane];
  }
}

__global__ void advance_kernel(int B, const int* __restrict__ stage, int stage_stride, int dlim,
                               int* __restrict__ Lp) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const int ne = stage[(long long)b * stage_stride];
  if (ne > 0) Lp[b] += min(ne, dlim);
}

__global__ void add_kernel(int n, const int* __restrict__ ids, int* __restrict__ v, int delta) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u < n) v[ids ? ids[u] : u] += delta;
}

__global__ void fill_int_kernel(int* __restrict__ p, int v, long long n) {
  long long u = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (u < n) p[u] = v;
}

__global__ void heads_to_lookaheads(int BK, int d, const int* __restrict__ beams, int* __restrict__ look) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u < BK) look[(long long)u * (d + 1)] = beams[u];
}

}  // namespace

// ---------------------------------------------------------------------------
hipError_t embed_launch(const PassDesc& p, const void* emb, float* h, int D, int V, int dtype, hipStream_t st,
                        int2* rowinfo) {
  const int M = p.M();
  if (M == 0) return hipSuccess;
  if (dtype == 1) embed_rows<bf16><<<M, 256, 0, st>>>(p, (const bf16*)emb, h, D, V, p.bad, rowinfo);
  else embed_rows<float><<<M, 256, 0, st>>>(p, (const float*)emb, h, D, V, p.bad, rowinfo);
  return hipGetLastError();
}

hipError_t rmsnorm_launch(float* x, const float* g, float* out32, bf16* ohi, bf16* olo, int rows, int D,
                          float eps, int last_only, int R, float* hid, hipStream_t st, const float* part, int S) {
  if (rows == 0) return hipSuccess;
  if (S > 0 && last_only) return hipErrorInvalidValue;
  if (D % 4 != 0 || D > 4 * 256 * kNormU) return hipErrorInvalidValue;
  // few rows (the rollout): more threads per row keep more split planes'
  // loads in flight
  if (rows < 256)
    rmsnorm_rows<1024><<<rows, 1024, 0, st>>>(x, g, out32, ohi, olo, D, eps, last_only, R, hid, part, S, rows);
  else
    rmsnorm_rows<256><<<rows, 256, 0, st>>>(x, g, out32, ohi, olo, D, eps, last_only, R, hid, part, S, rows);
  return hipGetLastError();
}

hipError_t rope_kv_launch(const PassDesc& p, const float* qkv, void* qout, const KVPool& pool, int layer,
                          const float* cos_t, const float* sin_t, int H, int Hkv, int hd, int dtype, hipStream_t st,
                          int S) {
  const int M = p.M();
  if (M == 0) return hipSuccess;
  // q is fp32 for every weight dtype; the KV pool is fp32 or split bf16
  if (dtype == 1) {
    if (hd <= 0 || hd > 256) return hipErrorInvalidValue;
    const int tasks = p.nb * p.kp * Hkv;   // V: (beam group, KV head) tasks, NT / hd per workgroup
    // few rows (the rollout): wider row tasks keep more split planes' loads
    // in flight
    if (M < 256)
      rope_kv_write_split<512><<<M + (tasks + 512 / hd - 1) / (512 / hd), 512, 0, st>>>(
          p, qkv, (float*)qout, pool, layer, cos_t, sin_t, H, Hkv, hd, S);
    else
      rope_kv_write_split<256><<<M + (tasks + 256 / hd - 1) / (256 / hd), 256, 0, st>>>(
          p, qkv, (float*)qout, pool, layer, cos_t, sin_t, H, Hkv, hd, S);
  }
  else if (S > 1)
    return hipErrorInvalidValue;
  else
    rope_kv_write<float><<<M, 256, 0, st>>>(p, qkv, (float*)qout, pool, layer, cos_t, sin_t, H, Hkv, hd);
  return hipGetLastError();
}

// The outputs of logit_rows_kernel from the per-tile row statistics the
// LM-head GEMM wrote (RowStats) instead of from the logits: argmax, the
// log-prob of the gathered token, and the top-kk as log-probs.  One
// workgroup per row.  The top-kk come in kk rounds over the tiles' lists,
// each taking the best candidate ordered after the previous pick (value
// descending, id ascending; ids are unique).
__global__ __launch_bounds__(256) void rowstats_merge_kernel(RowStats s, LogitArgs a) {
  __shared__ float shv[4];
  __shared__ int shi[4];
  __shared__ float shs[4];
  const int m = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const long long base = (long long)m * s.tiles;
  auto block_best = [&](float v, int id, float& fv, int& fi) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(id, o, 64);
      if (vi_better(ov, oi, v, id)) {
        v = ov;
        id = oi;
      }
    }
    if (lane == 0) {
      shv[w] = v;
      shi[w] = id;
    }
    __syncthreads();
    fv = shv[0];
    fi = shi[0];
    for (int u = 1; u < 4; ++u)
      if (vi_better(shv[u], shi[u], fv, fi)) {
        fv = shv[u];
        fi = shi[u];
      }
    __syncthreads();
  };
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int t = tid; t < s.tiles; t += 256)
    if (vi_better(s.mx[base + t], s.am[base + t], bv, bi)) {
      bv = s.mx[base + t];
      bi = s.am[base + t];
    }
  float G;
  int amax;
  block_best(bv, bi, G, amax);
  if (tid == 0 && a.amax) a.amax[rowmap_index(a.amax_map, m)] = vocab_id(amax, a.V);
  if (!a.want_lse) return;
  float sv = 0.f;
  for (int t = tid; t < s.tiles; t += 256) {
    const float mx = s.mx[base + t];
    if (mx != -INFINITY) sv += s.se[base + t] * __expf(mx - G);
  }
  sv = wave_sum(sv);
  if (lane == 0) shs[w] = sv;
  __syncthreads();
  const float lse = G + __logf(shs[0] + shs[1] + shs[2] + shs[3]);
  if (a.lp && tid == 0) {
    const int tok = s.gather_tok ? s.gather_tok[rowmap_index(s.gather_map, m)] : 0;
    const bool in = tok >= 0 && tok < a.V;
    if (!in && a.bad) *a.bad = 1;
    a.lp[m] = in ? s.zx[m] - lse : __int_as_float(0x7fc00000);
  }
  if (a.kk == 0) return;
  const int dst = a.topk_rows ? a.topk_rows[m] : m;
  const int nc = s.tiles * s.kk;
  const long long cb = base * s.kk;
  float pv = INFINITY;
  int pi = -1;
  for (int r = 0; r < a.kk; ++r) {
    float cv = -INFINITY;
    int ci = 0x7fffffff;
    for (int q = tid; q < nc; q += 256) {
      const float v = s.tv[cb + q];
      const int id = s.tc[cb + q];
      if ((v < pv || (v == pv && id > pi)) && vi_better(v, id, cv, ci)) {
        cv = v;
        ci = id;
      }
    }
    float fv;
    int fi;
    block_best(cv, ci, fv, fi);
    if (tid == 0) {
      a.topk_ids[(long long)dst * a.kk + r] = vocab_id(fi, a.V);
      a.topk_lp[(long long)dst * a.kk + r] = fv - lse;
    }
    pv = fv;
    pi = fi;
  }
}

hipError_t rowstats_merge_launch(const RowStats& s, const LogitArgs& a, int M, hipStream_t st) {
  if (M == 0) return hipSuccess;
  if (a.kk != s.kk || a.kk < 0 || a.kk > 16 || s.tiles <= 0) return hipErrorInvalidValue;
  rowstats_merge_kernel<<<M, 256, 0, st>>>(s, a);
  return hipGetLastError();
}

hipError_t logit_rows_launch(const LogitArgs& a, int M, hipStream_t st) {
  if (M == 0) return hipSuccess;
  if (a.kk > 16 || a.kk < 0) return hipErrorInvalidValue;
  if (a.kk == 0) logit_rows_kernel<0><<<M, 256, 0, st>>>(a);
  else if (a.kk <= 4) logit_rows_kernel<4><<<M, 256, 0, st>>>(a);
  else if (a.kk <= 8) logit_rows_kernel<8><<<M, 256, 0, st>>>(a);
  else logit_rows_kernel<16><<<M, 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t beam_scores_launch(int BK, int d, const int* look, const int* y, const float* lp, const float* head_lp,
                              const float* lq, const float* u, int* n_accept, float* scores, hipStream_t st) {
  if (BK == 0) return hipSuccess;
  beam_scores_kernel<<<(BK + 127) / 128, 128, 0, st>>>(BK, d, look, y, lp, head_lp, lq, u, n_accept, scores);
  return hipGetLastError();
}

hipError_t select_launch(int B, int k, const float* scores, const float* reward, float alpha, int reward_only,
                         const float* first_at, int* beam, hipStream_t st) {
  if (B == 0) return hipSuccess;
  select_kernel<<<(B + 127) / 128, 128, 0, st>>>(B, k, scores, reward, alpha, reward_only, first_at, beam);
  return hipGetLastError();
}

hipError_t soft_rows_launch(const float* zp, const float* zq, int M, int V, int d, const int* look, const float* v,
                            float* draft_lp, int* res_ids, float* res_lp, hipStream_t st) {
  if (M == 0) return hipSuccess;
  soft_rows_kernel<<<M, 256, 0, st>>>(zp, zq, V, d, look, v, draft_lp, res_ids, res_lp);
  return hipGetLastError();
}

hipError_t controller_states_launch(int B, int d, const int* n_accept, const float* reward, double a_t, double r_t,
                                    int b1, int* state, float* first_at, hipStream_t st) {
  if (B == 0) return hipSuccess;
  controller_states_kernel<<<(B + 127) / 128, 128, 0, st>>>(B, d, n_accept, reward, a_t, r_t, b1, state, first_at);
  return hipGetLastError();
}

hipError_t reward_keywords_launch(int B, int k, int d, const int* gen, int gen_stride, const int* gen_len,
                                  const int* look, const int* upto, int head, const int* kws, int n_kw, int normalize,
                                  float* reward, hipStream_t st) {
  if (B * k == 0) return hipSuccess;
  reward_keywords_kernel<<<B * k, 256, 0, st>>>(k, d, gen, gen_stride, gen_len, look, upto, head, kws, n_kw,
                                                normalize, reward);
  return hipGetLastError();
}

hipError_t reward_linear_launch(int BK, const float* hidden, const float* w, int D, float* reward, hipStream_t st) {
  if (BK == 0) return hipSuccess;
  reward_linear_kernel<<<BK, 256, 0, st>>>(hidden, w, D, reward);
  return hipGetLastError();
}

hipError_t commit_heads_launch(int B, int k, int d, const int* look, const int* beam, const int* mask, int* stage,
                               int stage_stride, hipStream_t st) {
  commit_heads_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, k, d, look, beam, mask, stage, stage_stride);
  return hipGetLastError();
}

hipError_t commit_tokens_launch(int B, const int* tokens, const int* mask, int V, int* stage, int stage_stride,
                                hipStream_t st) {
  commit_tokens_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, tokens, mask, V, stage, stage_stride);
  return hipGetLastError();
}

hipError_t withdraw_launch(int B, const int* cnt, int* Lp, int* gen_len, hipStream_t st) {
  withdraw_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, cnt, Lp, gen_len);
  return hipGetLastError();
}

hipError_t commit_launch(int B, int k, int d, int kk, const int* look, const int* beam, const int* n_accept,
                         const int* rtk_ids, const float* rtk_lp, const int* res_ids, const float* res_lp, int* stage,
                         int stage_stride, int tcap, hipStream_t st) {
  commit_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, k, d, kk, look, beam, n_accept, rtk_ids, rtk_lp, res_ids, res_lp,
                                              stage, stage_stride, tcap);
  return hipGetLastError();
}

hipError_t commit_prefix_launch(int B, int d, int kk, const int* look, const int* n_accept, const int* rtk_ids,
                                const float* rtk_lp, int* stage, int stage_stride, int tcap, hipStream_t st) {
  commit_prefix_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, d, kk, look, n_accept, rtk_ids, rtk_lp, stage, stage_stride,
                                                     tcap);
  return hipGetLastError();
}

hipError_t commit_apply_launch(int B, const int* stage, int stage_stride, int tcap, int kk, int* gen, int gen_stride,
                               int* gen_len, int* next_beams, float* next_head_lp, int* catch_tok, hipStream_t st) {
  commit_apply_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, stage, stage_stride, tcap, kk, gen, gen_stride, gen_len,
                                                    next_beams, next_head_lp, catch_tok);
  return hipGetLastError();
}

hipError_t prefix_tail_launch(int B, const int* gen, int gen_stride, const int* gen_len, const int* ptail,
                              const int* Lp, int* Lm1, int* look, int look_stride, hipStream_t st) {
  prefix_tail_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, gen, gen_stride, gen_len, ptail, Lp, Lm1, look, look_stride);
  return hipGetLastError();
}

hipError_t last_tokens_launch(int B, const int* tokens, int L, int* out, hipStream_t st) {
  last_tokens_kernel<<<(B + 63) / 64, 64, 0, st>>>(B, tokens, L, out);
  return hipGetLastError();
}

hipError_t promote_launch(int B, int k, const KVPool& pool, int n_layers, const int* stage, int stage_stride, int dlim,
                          int soff, const int* Lp, const int* ptable, int ptable_stride, const int* stable,
                          int s_stride_b, int s_stride_i, int dtype, hipStream_t st) {
  dim3 grid(B, n_layers);
  if (dtype == 1)
    promote_split_kernel<<<grid, 256, 0, st>>>(k, pool, n_layers, stage, stage_stride, dlim, soff, Lp, ptable,
                                                ptable_stride, stable, s_stride_b, s_stride_i);
  else
    promote_kernel<float><<<grid, 256, 0, st>>>(k, pool, n_layers, stage, stage_stride, dlim, soff, Lp, ptable,
                                                ptable_stride, stable, s_stride_b, s_stride_i);
  return hipGetLastError();
}

hipError_t advance_launch(int B, const int* stage, int stage_stride, int dlim, int* Lp, hipStream_t st) {
  advance_kernel<<<(B + 127) / 128, 128, 0, st>>>(B, stage, stage_stride, dlim, Lp);
  return hipGetLastError();
}

hipError_t add_launch(int n, const int* ids, int* v, int delta, hipStream_t st) {
  if (n == 0) return hipSuccess;
  add_kernel<<<(n + 127) / 128, 128, 0, st>>>(n, ids, v, delta);
  return hipGetLastError();
}

hipError_t fill_int_launch(int* p, int v, long long n, hipStream_t st) {
  if (n == 0) return hipSuccess;
  fill_int_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(p, v, n);
  return hipGetLastError();
}

hipError_t heads_to_lookaheads_launch(int BK, int d, const int* beams, int* look, hipStream_t st) {
  if (BK == 0) return hipSuccess;
  heads_to_lookaheads<<<(BK + 127) / 128, 128, 0, st>>>(BK, d, beams, look);
  return hipGetLastError();
}

}  // namespace cdsl
