// Host runtime and C ABI of the CDSL library: weight packing, the paged KV
// pool and its block allocator, the per-pass model runner, and the entry
// points declared in include/cdsl.h and include/cdsl_ops.h.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <unordered_set>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "../../include/cdsl.h"
#include "../../include/cdsl_ops.h"
#include "attention.h"
#include "block_pool.h"
#include "common.h"
#include "gemm.h"
#include "kernels.h"

using namespace cdsl;

static_assert(kBlock == kPoolBlock, "KV blocks and the pool bookkeeping agree on the block size");

namespace {

// A roctx range around each library call (shown by rocprofv3 --marker-trace
// and correlated with the kernels it launches); a no-op without a tool.
struct Range {
  explicit Range(const char* name) { roctxRangePushA(name); }
  ~Range() { roctxRangePop(); }
  Range(const Range&) = delete;
  Range& operator=(const Range&) = delete;
};

constexpr int kMaxSplits = kAttnMaxSplits;

struct Fail {
  int code;
};

struct Model {
  cdsl_model_config c{};
  int hd = 0, G = 0, qkv_n = 0;
  size_t esz = 0;
  void* emb = nullptr;
  void* lm = nullptr;
  float* gf = nullptr;
  std::vector<void*> wqkv, wo, wgu, wd;
  std::vector<float*> g1, g2;
  KVPool pool{};
  float* cos_t = nullptr;
  float* sin_t = nullptr;
};

struct Workspace {
  int Mmax = 0, Mlog = 0;
  float* h = nullptr;        // residual stream [M, D]
  float* qkv = nullptr;      // [M, (H + 2 Hkv) hd]
  float* q = nullptr;        // [M, H, hd] after rotary
  int2* rowinfo = nullptr;   // [M] (block * 16 + slot, position) of each row of the pass
  // projection inputs: hi / lo bf16 planes (bf16 weights) or fp32
  bf16 *uh = nullptr, *ul = nullptr, *oh = nullptr, *ol = nullptr, *ah = nullptr, *al = nullptr;
  float *u32 = nullptr, *o32 = nullptr, *act32 = nullptr;
  float* gu32 = nullptr;
  float* logits = nullptr;
  // LM-head row statistics per column tile (the fused epilogue); rs_cap rows
  // x tiles, times the top-k width for the candidate lists
  float *rs_mx = nullptr, *rs_se = nullptr, *rs_tv = nullptr, *rs_zx = nullptr;
  int *rs_am = nullptr, *rs_tc = nullptr;
  size_t rs_cap = 0;
  float* part_o = nullptr;
  float* part_ml = nullptr;
  size_t part_rows = 0;     // capacity in (row, head) units for one split
  void* gemm_ws = nullptr;
  size_t gemm_ws_bytes = 0;
};

}  // namespace

struct cdsl_prefix {
  int B = 0;
  int L0 = 0;                   // prompt length
  std::vector<int> len;        // host copy of prefix lengths
  std::vector<int> table;      // [B][pstride] prefix block ids
  std::vector<int> owned;      // blocks to return on free
  int* Lp = nullptr;           // device [B]
  int* table_dev = nullptr;    // device [B][pstride]
  int* gen = nullptr;          // device [B][gen_stride] emitted tokens
  int* gen_len = nullptr;      // device [B]
  int* ptail = nullptr;        // device [B] last prompt token
  int* Lm1 = nullptr;          // device [B] Lp - 1 (the passes that re-feed the last prefix token)
  int rolled_k = 0, rolled_d = 0;
  int rolled_pfx = 0, verified_pfx = 0;   // the last rollout / verify started from the prefix itself
  int verified_k = 0, verified_d = 0, verified_kk = 0;
  const float* kept_logits = nullptr;   // draft logits of the last rollout (cdsl_rollout_keep)
  int verified_soft = 0;
};

struct cdsl_ctx {
  hipStream_t st = nullptr;
  cdsl_limits lim{};
  Model m[2];                  // 0 draft, 1 target
  int dtype = 0;
  Workspace ws;
  int nblocks = 0;
  int pstride = 0;             // prefix blocks per prompt
  int sblocks = 0;             // suffix blocks per beam
  BlockPool pool_blocks;       // free list of the prefix blocks
  int* stable = nullptr;       // device [max_B][max_k][sblocks]
  int* iota = nullptr;         // device [max_B] = 0..max_B-1
  int* stage = nullptr;        // device [max_B][stage_stride]
  int stage_stride = 0;
  int* stage_host = nullptr;   // pinned
  int* table_host = nullptr;   // pinned [max_B][pstride]
  int* ids_host = nullptr;     // pinned [max_B] prompt ids of an appended row (written after a sync)
  int* mask_host = nullptr;    // pinned [max_B] append mask (its own buffer: written before the call syncs)
  int* cnt_host = nullptr;     // pinned [max_B] withdrawn counts
  int* ids_dev = nullptr;      // device [max_B]
  int* catch_tok = nullptr;    // device [max_B]
  int* mask_dev = nullptr;     // device [max_B] (head-only commit mask)
  int* cnt_dev = nullptr;      // device [max_B] (withdrawn counts)
  int* bad = nullptr;          // device flag: a token id outside [0, V) was fed or gathered
  int* bad_host = nullptr;     // pinned copy of it
  int stage_tcap = 0;          // token capacity of a commit record
  std::unordered_set<cdsl_prefix*> prefixes;
  int live_prefixes = 0;
  std::vector<void*> allocs;
  std::string err;
  // per-kernel-class timing (cdsl_profile_*)
  bool prof = false;
  cdsl_kernel_stats acc{};
  std::vector<hipEvent_t> ev_free;
  struct Pending {
    hipEvent_t a, b;
    int cls;
  };
  std::vector<Pending> pend;
};

namespace {

thread_local std::string g_err;

int fail(cdsl_ctx* c, int code, const std::string& msg) {
  if (c) c->err = msg;
  g_err = msg;
  return code;
}

// Contexts and prefix handles alive, so that a call with a destroyed
// context or a freed prefix is refused instead of touching freed memory.
std::mutex g_live_mu;
std::unordered_set<const cdsl_ctx*> g_live;

bool ctx_live(const cdsl_ctx* c) {
  std::lock_guard<std::mutex> g(g_live_mu);
  return g_live.count(c) != 0;
}

#define CTX_CHECK(c)                                                                         \
  do {                                                                                       \
    if (!(c)) return fail(nullptr, CDSL_EINVAL, "null context");                             \
    if (!ctx_live(c)) return fail(nullptr, CDSL_ESTATE, "unknown or destroyed context");     \
  } while (0)

#define PX_CHECK(c, px)                                                                      \
  do {                                                                                       \
    if ((px) && !(c)->prefixes.count(px)) return fail((c), CDSL_ESTATE, "unknown or freed prefix handle"); \
  } while (0)

#define CK(call)                                                                             \
  do {                                                                                       \
    hipError_t e_ = (call);                                                                  \
    if (e_ != hipSuccess) {                                                                  \
      throw_dev(#call, e_);                                                                  \
    }                                                                                        \
  } while (0)

[[noreturn]] void throw_dev(const char* what, hipError_t e) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  throw Fail{CDSL_EDEVICE};
}

template <typename T>
T* dev_alloc(cdsl_ctx* c, size_t count) {
  if (count == 0) count = 1;
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, count * sizeof(T));
  if (e != hipSuccess) {
    g_err = "hipMalloc of " + std::to_string(count * sizeof(T)) + " bytes failed";
    throw Fail{CDSL_ENOMEM};
  }
  c->allocs.push_back(p);
  return (T*)p;
}

void* dev_alloc_bytes(cdsl_ctx* c, size_t bytes) { return dev_alloc<char>(c, bytes); }

// ---------------------------------------------------------------------------
// profiling: a pair of events around a launch, harvested after a sync
// ---------------------------------------------------------------------------
hipEvent_t take_event(cdsl_ctx* c) {
  if (!c->ev_free.empty()) {
    hipEvent_t e = c->ev_free.back();
    c->ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) {
    g_err = "hipEventCreate failed";
    throw Fail{CDSL_EDEVICE};
  }
  return e;
}

void harvest(cdsl_ctx* c) {
  for (auto& p : c->pend) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) c->acc.ms[p.cls] += ms;
    c->ev_free.push_back(p.a);
    c->ev_free.push_back(p.b);
  }
  c->pend.clear();
}

struct Span {
  cdsl_ctx* c;
  int cls;
  hipEvent_t a = nullptr;
  Span(cdsl_ctx* cc, int k, double flops, double bytes) : c(cc), cls(k) {
    if (!c->prof) return;
    a = take_event(c);
    (void)hipEventRecord(a, c->st);
    c->acc.launches[cls] += 1;
    c->acc.flops[cls] += flops;
    c->acc.bytes[cls] += bytes;
  }
  // records the end event now (idempotent)
  void close() {
    if (!a) return;
    hipEvent_t b = nullptr;
    if (!c->ev_free.empty()) {
      b = c->ev_free.back();
      c->ev_free.pop_back();
    } else if (hipEventCreate(&b) != hipSuccess) {
      c->ev_free.push_back(a);
      a = nullptr;
      return;
    }
    (void)hipEventRecord(b, c->st);
    c->pend.push_back({a, b, cls});
    a = nullptr;
  }
  ~Span() { close(); }
};

bool cfg_ok(const cdsl_model_config& c, std::string& why) {
  if (c.n_layers <= 0 || c.d_model <= 0 || c.n_heads <= 0 || c.n_kv_heads <= 0 || c.ffn_dim <= 0 || c.vocab <= 0) {
    why = "non-positive model dimension";
    return false;
  }
  if (c.d_model % c.n_heads != 0 || c.n_heads % c.n_kv_heads != 0) {
    why = "d_model % n_heads or n_heads % n_kv_heads != 0";
    return false;
  }
  int hd = c.d_model / c.n_heads;
  if (hd != 32 && hd != 64 && hd != 128) {
    why = "head_dim must be 32, 64 or 128";
    return false;
  }
  if (c.dtype == CDSL_BF16 && hd == 32) {
    why = "bf16 models need head_dim 64 or 128";
    return false;
  }
  if (c.dtype != CDSL_F32 && c.dtype != CDSL_BF16) {
    why = "dtype must be CDSL_F32 or CDSL_BF16";
    return false;
  }
  if (c.d_model > 8192) {
    why = "d_model must be at most 8192";
    return false;
  }
  if (c.ffn_dim % 16 != 0) {
    why = "ffn_dim must be a multiple of 16";
    return false;
  }
  int kmul = c.dtype == CDSL_BF16 ? 64 : 16;
  if (c.d_model % kmul != 0 || c.ffn_dim % kmul != 0) {
    why = "d_model and ffn_dim must be multiples of 64 (bf16) or 16 (fp32)";
    return false;
  }
  if (c.dtype == CDSL_BF16 && c.ffn_dim % 32 != 0) {
    why = "bf16 ffn_dim must be a multiple of 32";
    return false;
  }
  if (!(c.rms_eps > 0.f) || !(c.rope_theta > 0.f)) {
    why = "rms_eps and rope_theta must be positive";
    return false;
  }
  return true;
}

void load_model(cdsl_ctx* c, Model& md, const cdsl_model& src, int max_pos) {
  md.c = src.cfg;
  const auto& k = md.c;
  md.hd = k.d_model / k.n_heads;
  md.G = k.n_heads / k.n_kv_heads;
  md.qkv_n = (k.n_heads + 2 * k.n_kv_heads) * md.hd;
  md.esz = k.dtype == CDSL_BF16 ? 2 : 4;
  const size_t D = k.d_model, F = k.ffn_dim, V = k.vocab, hd = md.hd;
  const size_t Hq = k.n_heads * hd, Hk = k.n_kv_heads * hd;
  const size_t es = md.esz;
  hipStream_t st = c->st;
  if (!src.tok_emb || !src.lm_head || !src.final_norm || !src.layer_ptrs) {
    g_err = "null weight pointer";
    throw Fail{CDSL_EINVAL};
  }
  // Matrices the kernels read as given are borrowed (used in place; the
  // caller keeps them alive until cdsl_destroy).  Their rows are read with
  // 16-byte vector loads, so every pointer must be 16-byte aligned.
  auto borrow = [&](const void* p) {
    if (((uintptr_t)p & 15) != 0) {
      g_err = "weight pointers must be 16-byte aligned";
      throw Fail{CDSL_EINVAL};
    }
    return const_cast<void*>(p);
  };
  md.emb = borrow(src.tok_emb);
  md.lm = borrow(src.lm_head);
  md.gf = (float*)borrow(src.final_norm);
  for (int l = 0; l < k.n_layers; ++l) {
    const void* const* lp = src.layer_ptrs + 9 * l;
    for (int u = 0; u < 9; ++u)
      if (!lp[u]) {
        g_err = "null layer weight pointer";
        throw Fail{CDSL_EINVAL};
      }
    md.g1.push_back((float*)borrow(lp[0]));
    md.g2.push_back((float*)borrow(lp[5]));
    char* qkv = (char*)dev_alloc_bytes(c, (Hq + 2 * Hk) * D * es);
    CK(hipMemcpyAsync(qkv, lp[1], Hq * D * es, hipMemcpyDeviceToDevice, st));
    CK(hipMemcpyAsync(qkv + Hq * D * es, lp[2], Hk * D * es, hipMemcpyDeviceToDevice, st));
    CK(hipMemcpyAsync(qkv + (Hq + Hk) * D * es, lp[3], Hk * D * es, hipMemcpyDeviceToDevice, st));
    md.wqkv.push_back(qkv);
    md.wo.push_back(borrow(lp[4]));
    // gate/up interleaved in groups of 16 rows: [g0..g15, u0..u15, g16..]
    char* gu = (char*)dev_alloc_bytes(c, 2 * F * D * es);
    CK(hipMemcpy2DAsync(gu, 32 * D * es, lp[6], 16 * D * es, 16 * D * es, F / 16, hipMemcpyDeviceToDevice, st));
    CK(hipMemcpy2DAsync(gu + 16 * D * es, 32 * D * es, lp[7], 16 * D * es, 16 * D * es, F / 16,
                        hipMemcpyDeviceToDevice, st));
    md.wgu.push_back(gu);
    md.wd.push_back(borrow(lp[8]));
  }
  // rotary tables in double precision, stored fp32: [max_pos][hd/2]
  const int half = md.hd / 2;
  std::vector<float> ct((size_t)max_pos * half), stt((size_t)max_pos * half);
  for (int p = 0; p < max_pos; ++p)
    for (int d = 0; d < half; ++d) {
      double inv = pow((double)k.rope_theta, -2.0 * d / (double)md.hd);
      double ang = (double)p * inv;
      ct[(size_t)p * half + d] = (float)cos(ang);
      stt[(size_t)p * half + d] = (float)sin(ang);
    }
  md.cos_t = dev_alloc<float>(c, ct.size());
  md.sin_t = dev_alloc<float>(c, stt.size());
  CK(hipMemcpy(md.cos_t, ct.data(), ct.size() * 4, hipMemcpyHostToDevice));
  CK(hipMemcpy(md.sin_t, stt.data(), stt.size() * 4, hipMemcpyHostToDevice));
}

void alloc_pool(cdsl_ctx* c, Model& md) {
  const long long per_layer = (long long)c->nblocks * md.c.n_kv_heads * kBlock * md.hd;
  md.pool.Hkv = md.c.n_kv_heads;
  md.pool.hd = md.hd;
  md.pool.layer_elems = per_layer;
  const size_t bytes = (size_t)per_layer * md.c.n_layers * sizeof(float);   // fp32 KV
  size_t free_b = 0, total_b = 0;
  CK(hipMemGetInfo(&free_b, &total_b));
  if (2 * bytes > free_b) {
    g_err = "the KV pool the limits ask for (" + std::to_string(2 * bytes) + " bytes) exceeds free device memory (" +
            std::to_string(free_b) + " bytes)";
    throw Fail{CDSL_ENOMEM};
  }
  md.pool.k = dev_alloc_bytes(c, bytes);
  md.pool.v = dev_alloc_bytes(c, bytes);
  // zero once: stale slots are then always finite (masked weights are 0)
  CK(hipMemsetAsync(md.pool.k, 0, bytes, c->st));
  CK(hipMemsetAsync(md.pool.v, 0, bytes, c->st));
}

int prefill_chunk_prompts(const cdsl_limits& l) {
  int per = std::max(1, 8192 / std::max(1, l.max_prompt));
  return std::min(per, l.max_batch);
}

void alloc_workspace(cdsl_ctx* c) {
  const cdsl_limits& l = c->lim;
  const int verify_rows = l.max_batch * l.max_k * l.max_d;
  const int roll_rows = l.max_batch * l.max_k;
  const int pre_rows = prefill_chunk_prompts(l) * l.max_prompt;
  Workspace& w = c->ws;
  w.Mmax = std::max({verify_rows, roll_rows, pre_rows, l.max_batch});
  w.Mlog = std::max({verify_rows, roll_rows, l.max_batch});
  size_t Dm = 0, QKVm = 0, HQm = 0, Fm = 0, Vm = 0, Hm = 0, HDm = 0;
  for (auto& md : c->m) {
    Dm = std::max<size_t>(Dm, md.c.d_model);
    QKVm = std::max<size_t>(QKVm, md.qkv_n);
    HQm = std::max<size_t>(HQm, (size_t)md.c.n_heads * md.hd);
    Fm = std::max<size_t>(Fm, md.c.ffn_dim);
    Vm = std::max<size_t>(Vm, md.c.vocab);
    Hm = std::max<size_t>(Hm, md.c.n_heads);
    HDm = std::max<size_t>(HDm, md.hd);
  }
  const size_t M = w.Mmax;
  w.h = dev_alloc<float>(c, M * Dm);
  w.qkv = dev_alloc<float>(c, M * QKVm);
  w.q = dev_alloc<float>(c, M * HQm);
  w.rowinfo = dev_alloc<int2>(c, M);
  if (c->dtype == CDSL_BF16) {
    w.uh = dev_alloc<bf16>(c, M * Dm);
    w.ul = dev_alloc<bf16>(c, M * Dm);
    w.oh = dev_alloc<bf16>(c, M * HQm);
    w.ol = dev_alloc<bf16>(c, M * HQm);
    w.ah = dev_alloc<bf16>(c, M * Fm);
    w.al = dev_alloc<bf16>(c, M * Fm);
  } else {
    w.u32 = dev_alloc<float>(c, M * Dm);
    w.o32 = dev_alloc<float>(c, M * HQm);
    w.act32 = dev_alloc<float>(c, M * Fm);
    w.gu32 = dev_alloc<float>(c, M * 2 * Fm);
  }
  w.logits = dev_alloc<float>(c, (size_t)w.Mlog * Vm);
  for (auto& md : c->m)
    for (int mm = 1; mm <= w.Mlog; ++mm)
      w.rs_cap = std::max(w.rs_cap, (size_t)mm * gemm_rowstats_tiles(mm, md.c.vocab, md.c.d_model, c->dtype));
  w.rs_mx = dev_alloc<float>(c, w.rs_cap);
  w.rs_se = dev_alloc<float>(c, w.rs_cap);
  w.rs_am = dev_alloc<int>(c, w.rs_cap);
  w.rs_tv = dev_alloc<float>(c, w.rs_cap * l.max_k);
  w.rs_tc = dev_alloc<int>(c, w.rs_cap * l.max_k);
  w.rs_zx = dev_alloc<float>(c, w.Mlog);
  // attention split partials sized for the verification / rollout passes
  w.part_rows = (size_t)std::max(verify_rows, roll_rows) * Hm;
  if (c->dtype == CDSL_BF16) {
    w.part_o = dev_alloc<float>(c, kMaxSplits * w.part_rows * HDm);
    w.part_ml = dev_alloc<float>(c, kMaxSplits * w.part_rows * 2);
  }
  // GEMM split-K workspace: the largest need over every shape and row count
  size_t need = 0;
  for (auto& md : c->m) {
    const int D = md.c.d_model, F = md.c.ffn_dim, V = md.c.vocab, HQ = md.c.n_heads * md.hd;
    const int shapes[5][2] = {{md.qkv_n, D}, {D, HQ}, {2 * F, D}, {D, F}, {V, D}};
    for (int mm = 1; mm <= w.Mmax; ++mm)
      for (auto& s : shapes) need = std::max(need, gemm_workspace_bytes(mm, s[0], s[1], c->dtype));
  }
  w.gemm_ws_bytes = need;
  if (need) {
    w.gemm_ws = dev_alloc_bytes(c, need);
    CK(hipMemsetAsync(w.gemm_ws, 0, need, c->st));
  }
}

// ---------------------------------------------------------------------------
// model runner
// ---------------------------------------------------------------------------
// Returns the number of split planes left in the GEMM workspace for the
// caller to fold (1: none) when defer is set.
int gemm(cdsl_ctx* c, const GemmOperand& A, const void* W, const GemmOut& out, int M, int N, int K, int epi,
         bool prefill, bool defer = false, RowStats* rs = nullptr, const RopeEpi* rope = nullptr) {
  const double wes = c->dtype == CDSL_BF16 ? 2.0 : 4.0;   // weight element size
  // output bytes: fp32 store (also the rotary epilogue's fp32 q and hi / lo
  // K, V), fp32 read-modify-write, the two bf16 planes of the half-width
  // SwiGLU output, or the per-tile row statistics
  const double outb =
      epi == kEpiSwiGLU     ? (double)M * (N / 2) * 4.0
      : epi == kEpiRowStats ? (double)M * gemm_rowstats_tiles(M, N, K, c->dtype) * (3.0 + 2.0 * rs->kk) * 4.0
                            : (double)M * N * 4.0 * (epi == kEpiResidual ? 2.0 : 1.0);
  const int kind = gemm_kind(M, N, K, c->dtype);
  const int cls = kind == 0 ? CDSL_K_GEMM_DENSE : kind == 1 ? CDSL_K_GEMM_SKINNY : CDSL_K_GEMM_F32;
  // with split-K, the main kernel writes fp32 partial planes and the reduce
  // kernel (timed as its own class) reads them and applies the epilogue
  struct Hook : GemmHook {
    cdsl_ctx* c = nullptr;
    Span* main = nullptr;
    double outb = 0.0, plane = 0.0;
    Span* red = nullptr;
    alignas(Span) unsigned char buf[sizeof(Span)];
    void before_reduce(int ksplit) override {
      main->close();
      red = new (buf) Span(c, CDSL_K_SPLITK_REDUCE, 0.0, ksplit * plane + outb);
    }
    ~Hook() {
      if (red) red->~Span();
    }
  };
  Span sp(c, cls, 2.0 * M * N * (double)K, (double)M * K * 4.0 + (double)N * K * wes + outb);
  Hook hk;
  hk.c = c;
  hk.main = &sp;
  hk.outb = outb;
  hk.plane = (double)M * N * 4.0;
  int planes = 1;
  CK(gemm_launch(A, W, out, M, N, K, c->dtype, epi, c->ws.gemm_ws, c->ws.gemm_ws_bytes, c->st, prefill,
                 c->prof ? &hk : nullptr, defer ? &planes : nullptr, rs, rope));
  return planes;
}

void logit_rows(cdsl_ctx* c, const LogitArgs& la, int M);

// Forward pass of one model over the rows of p.  With want_logits, the
// final-normed rows (all, or the last row of each beam with last_only) go
// through the LM head into ws.logits (or logits_out at row stride
// logits_ld); hid receives fp32 final-normed rows of every beam's last row
// when non-null.  fuse names the row outputs wanted from the logits
// (argmax, gathered log-prob, top-k): the LM head then leaves per-tile row
// statistics and a merge kernel writes those outputs, so no logits reach
// memory.  Without fuse (speculative sampling, which reads whole rows) the
// head writes the logits.
void run_pass(cdsl_ctx* c, Model& md, const PassDesc& p, int max_prefix_len, long long sum_prefix_len,
              bool want_logits, bool last_only, float* hid, bool prefill = false, float* logits_out = nullptr,
              int logits_ld = 0, const LogitArgs* fuse = nullptr) {
  Workspace& w = c->ws;
  const auto& k = md.c;
  const int M = p.M();
  const int D = k.d_model, F = k.ffn_dim, H = k.n_heads, Hkv = k.n_kv_heads, hd = md.hd;
  const int dt = k.dtype;
  if (M > w.Mmax) {
    g_err = "pass rows exceed the workspace";
    throw Fail{CDSL_ERANGE};
  }
  const double es = 4.0;   // fp32 activations and KV
  {
    Span sp(c, CDSL_K_ROWWISE, 0.0, (double)M * D * ((dt == CDSL_BF16 ? 2.0 : 4.0) + 4.0));
    CK(embed_launch(p, md.emb, w.h, D, k.vocab, dt, c->st, w.rowinfo));
  }
  // algorithmic attention work of this pass: the prefix KV of a prompt is
  // read once for all its rows; every query head sees its visible keys
  const double kvtok = (double)Hkv * hd * 2.0 * es;
  const double R = p.R, kp = p.kp;
  const double pre_tok = p.mode == kSuffix ? (double)sum_prefix_len : (double)sum_prefix_len + p.nb * R;
  const double suf_tok = p.mode == kSuffix ? (double)p.nb * kp * (p.j0 + R) : 0.0;
  const double attn_bytes = (pre_tok + suf_tok) * kvtok + 2.0 * M * (double)H * hd * es;
  const double vis = p.mode == kSuffix
                         ? kp * (R * ((double)sum_prefix_len + p.nb * (double)p.j0) + p.nb * R * (R + 1) / 2)
                         : R * (double)sum_prefix_len + p.nb * R * (R + 1) / 2;
  const double attn_flops = 4.0 * hd * (double)H * vis;
  AttnPlan pl = attn_plan(p, H, Hkv, hd, dt, max_prefix_len, kMaxSplits);
  if (pl.nsplit > 1 && (size_t)M * H > w.part_rows) {
    pl = attn_plan(p, H, Hkv, hd, dt, max_prefix_len, 1);
  }
  AttnArgs aa{};
  aa.p = p;
  aa.Q = w.q;
  aa.O = w.o32;
  aa.Ohi = w.oh;
  aa.Olo = w.ol;
  aa.pool = md.pool;
  aa.H = H;
  aa.Hkv = Hkv;
  aa.G = md.G;
  aa.rows_total = (long long)M * H;
  aa.scale_log2 = (float)(1.4426950408889634 / sqrt((double)hd));
  aa.part_o = w.part_o;
  aa.part_ml = w.part_ml;
  const double norm_bytes = (double)M * D * (4.0 + es);
  const double rope_bytes = (double)M * md.qkv_n * (4.0 + es);
  const double comb_bytes = (double)pl.nsplit * M * H * (hd + 2) * 4.0 + (double)M * H * hd * es;
  const bool bf = dt == CDSL_BF16;
  const GemmOperand Au{w.uh, w.ul, w.u32}, Ao{w.oh, w.ol, w.o32}, Aact{w.ah, w.al, w.act32};
  const GemmOut to_qkv{w.qkv, nullptr, nullptr, md.qkv_n}, to_h{w.h, nullptr, nullptr, D};
  const GemmOut to_act{nullptr, w.ah, w.al, F}, to_gu{w.gu32, nullptr, nullptr, 2 * F};
  // Residual projections (W_o, W_down) and the q/k/v projection may leave
  // their K split unreduced: the planes are folded by the kernel that
  // consumes the result (RMSNorm of the residual stream, rotary + KV
  // write), which saves a reduce launch per projection.
  const float* planes_ws = (const float*)w.gemm_ws;
  // Where the q/k/v projection is not split (the dense kernel at the
  // verification and prefill row counts), its epilogue applies the rotary
  // embedding and writes q and the KV pool itself: no q/k/v product in
  // memory and no rotary launch.  CDSL_UNFUSED_ROPE=1 keeps the separate
  // kernel (same arithmetic, for comparison).
  const char* unfused_env = getenv("CDSL_UNFUSED_ROPE");
  const bool fuse_rope = bf && !(unfused_env && unfused_env[0] == '1') &&
                         gemm_rope_fusable(M, md.qkv_n, D, c->dtype, hd);
  RopeEpi rope{p, w.rowinfo, w.q, md.pool, 0, md.cos_t, md.sin_t, H, Hkv, hd};
  {
    Span sp(c, CDSL_K_ROWWISE, 0.0, norm_bytes);
    CK(rmsnorm_launch(w.h, md.g1[0], w.u32, w.uh, w.ul, M, D, k.rms_eps, 0, 1, nullptr, c->st));
  }
  for (int l = 0; l < k.n_layers; ++l) {
    if (fuse_rope) {
      rope.layer = l;
      gemm(c, Au, md.wqkv[l], GemmOut{}, M, md.qkv_n, D, kEpiRope, prefill, false, nullptr, &rope);
    } else {
      const int sq = gemm(c, Au, md.wqkv[l], to_qkv, M, md.qkv_n, D, kEpiStore, prefill, bf);
      Span sp(c, CDSL_K_ROWWISE, 0.0, rope_bytes + (sq > 1 ? (double)sq * M * md.qkv_n * 4.0 : 0.0));
      CK(rope_kv_launch(p, sq > 1 ? planes_ws : w.qkv, w.q, md.pool, l, md.cos_t, md.sin_t, H, Hkv, hd, dt, c->st,
                        sq > 1 ? sq : 0));
    }
    aa.layer = l;
    {
      Span sp(c, CDSL_K_ATTENTION, attn_flops, attn_bytes);
      CK(attn_launch(aa, pl, hd, dt, c->st));
    }
    if (pl.nsplit > 1) {
      Span sp(c, CDSL_K_ATTN_COMBINE, 0.0, comb_bytes);
      CK(attn_combine_launch(aa, pl, hd, c->st));
    }
    const int so = gemm(c, Ao, md.wo[l], to_h, M, D, H * hd, kEpiResidual, prefill, bf);
    {
      Span sp(c, CDSL_K_ROWWISE, 0.0, norm_bytes + (so > 1 ? (double)(so + 1) * M * D * 4.0 : 0.0));
      CK(rmsnorm_launch(w.h, md.g2[l], w.u32, w.uh, w.ul, M, D, k.rms_eps, 0, 1, nullptr, c->st,
                        so > 1 ? planes_ws : nullptr, so > 1 ? so : 0));
    }
    if (bf) {
      gemm(c, Au, md.wgu[l], to_act, M, 2 * F, D, kEpiSwiGLU, prefill);
    } else {
      gemm(c, Au, md.wgu[l], to_gu, M, 2 * F, D, kEpiStore, prefill);
      Span sp(c, CDSL_K_ROWWISE, 0.0, (double)M * F * 12.0);
      CK(swiglu_f32_launch(w.gu32, w.act32, M, F, c->st));
    }
    const int sd = gemm(c, Aact, md.wd[l], to_h, M, D, F, kEpiResidual, prefill, bf);
    const bool last = l + 1 == k.n_layers;
    if (!last || sd > 1) {
      // next layer's attention norm (or, after the last layer, only the
      // fold: the final norm below may take just the last rows)
      Span sp(c, CDSL_K_ROWWISE, 0.0, (last ? 0.0 : norm_bytes) + (sd > 1 ? (double)(sd + 1) * M * D * 4.0 : 0.0));
      CK(rmsnorm_launch(w.h, last ? nullptr : md.g1[l + 1], w.u32, w.uh, w.ul, M, D, k.rms_eps, 0, 1, nullptr, c->st,
                        sd > 1 ? planes_ws : nullptr, sd > 1 ? sd : 0));
    }
  }
  if (!want_logits) return;
  const int rows = last_only ? p.nb * p.kp : M;
  {
    Span sp(c, CDSL_K_ROWWISE, 0.0, (double)rows * D * (4.0 + es));
    CK(rmsnorm_launch(w.h, md.gf, w.u32, w.uh, w.ul, rows, D, k.rms_eps, last_only ? 1 : 0, p.R, hid, c->st));
  }
  // Every head whose caller wants only row outputs takes the fused
  // epilogue: no logits reach memory.  Measured against writing the logits
  // and reducing them with logit_rows: 80 rows of a 32000-token head, top-5,
  // 97 vs 131 us; 800 rows, top-5, 497 vs 505 us; 4096 rows of a
  // 128256-token head, top-8, 8.30 vs 8.35 ms.
  if (fuse) {
    const int tiles = gemm_rowstats_tiles(rows, k.vocab, D, c->dtype);
    if (tiles > 0 && (size_t)rows * tiles <= w.rs_cap && fuse->kk <= c->lim.max_k) {
      RowStats rs{};
      rs.mx = w.rs_mx;
      rs.se = w.rs_se;
      rs.am = w.rs_am;
      rs.tv = w.rs_tv;
      rs.tc = w.rs_tc;
      rs.kk = fuse->kk;
      rs.zx = w.rs_zx;
      rs.gather_tok = fuse->lp ? fuse->gather_tok : nullptr;
      rs.gather_map = fuse->gather_map;
      gemm(c, Au, md.lm, GemmOut{nullptr, nullptr, nullptr, k.vocab}, rows, k.vocab, D, kEpiRowStats, prefill, false,
           &rs);
      Span sp(c, CDSL_K_LOGIT_ROWS, 0.0, (double)rows * rs.tiles * (3.0 + 2.0 * rs.kk) * 4.0);
      CK(rowstats_merge_launch(rs, *fuse, rows, c->st));
      return;
    }
  }
  gemm(c, Au, md.lm, GemmOut{logits_out ? logits_out : w.logits, nullptr, nullptr, logits_ld ? logits_ld : k.vocab},
       rows, k.vocab, D, kEpiStore, prefill);
  if (fuse) {
    LogitArgs la = *fuse;
    la.logits = w.logits;
    la.ld = 0;
    logit_rows(c, la, rows);
  }
}

void logit_rows(cdsl_ctx* c, const LogitArgs& la, int M) {
  Span sp(c, CDSL_K_LOGIT_ROWS, 0.0, (double)M * la.V * 4.0);
  CK(logit_rows_launch(la, M, c->st));
}

long long sum_len(const cdsl_prefix* px) {
  long long s = 0;
  for (int v : px->len) s += v;
  return s;
}

PassDesc base_pass(cdsl_ctx* c, cdsl_prefix* px) {
  PassDesc p{};
  p.Lp = px->Lp;
  p.ptable = px->table_dev;
  p.ptable_stride = c->pstride;
  p.stable = c->stable;
  p.sblocks = c->sblocks;
  p.s_stride_i = c->sblocks;
  p.s_stride_b = c->lim.max_k * c->sblocks;
  p.bad = c->bad;
  return p;
}

int max_len(const cdsl_prefix* px) {
  int m = 0;
  for (int v : px->len) m = std::max(m, v);
  return m;
}

// make sure prompt b owns blocks for positions [0, new_len)
void ensure_blocks(cdsl_ctx* c, cdsl_prefix* px, int b, int new_len) {
  const int r = c->pool_blocks.ensure(px->table, px->owned, c->pstride, b, new_len);
  if (r == BlockPool::kRange) {
    g_err = "prompt " + std::to_string(b) + " exceeds max_ctx";
    throw Fail{CDSL_ERANGE};
  }
  if (r == BlockPool::kExhausted) {
    g_err = "KV pool exhausted";
    throw Fail{CDSL_ENOMEM};
  }
}

// Callers synchronise the stream first: the staging buffer is shared by
// every prefix handle, and the previous copy from it may still be queued.
void upload_table(cdsl_ctx* c, cdsl_prefix* px) {
  const size_t n = (size_t)px->B * c->pstride;
  for (size_t u = 0; u < n; ++u) c->table_host[u] = px->table[u] < 0 ? 0 : px->table[u];
  CK(hipMemcpyAsync(px->table_dev, c->table_host, n * sizeof(int), hipMemcpyHostToDevice, c->st));
}

template <typename F>
int guarded(cdsl_ctx* c, F&& f) {
  try {
    return f();
  } catch (const Fail& e) {
    if (c) c->err = g_err;
    return e.code;
  } catch (const std::bad_alloc&) {
    return fail(c, CDSL_ENOMEM, "host allocation failed");
  } catch (...) {
    return fail(c, CDSL_EDEVICE, "unexpected exception");
  }
}

}  // namespace

void destroy_ctx(cdsl_ctx* c);

namespace {

// Queue the read-back of the token-range flag; after the stream has been
// synchronised, check_bad reports a token id outside [0, V) fed or gathered
// since the last check as an invalid argument (and clears the flag).
void queue_bad(cdsl_ctx* c) {
  CK(hipMemcpyAsync(c->bad_host, c->bad, sizeof(int), hipMemcpyDeviceToHost, c->st));
}

void check_bad(cdsl_ctx* c) {
  if (!*c->bad_host) return;
  *c->bad_host = 0;
  CK(fill_int_launch(c->bad, 0, 1, c->st));
  g_err = "a token id outside [0, vocab) was passed since the last synchronising call";
  throw Fail{CDSL_EINVAL};
}

// device buffers of a prefix handle (allocated by cdsl_prefill)
void free_px_buffers(cdsl_ctx* c, cdsl_prefix* px) {
  for (void* p : {(void*)px->Lp, (void*)px->table_dev, (void*)px->gen, (void*)px->gen_len, (void*)px->ptail,
                  (void*)px->Lm1}) {
    auto it = std::find(c->allocs.begin(), c->allocs.end(), p);
    if (p && it != c->allocs.end()) {
      (void)hipFree(p);
      c->allocs.erase(it);
    }
  }
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

int cdsl_init(const cdsl_model* draft, const cdsl_model* target, const cdsl_limits* limits, void* stream,
              cdsl_ctx** out) {
  if (!draft || !target || !limits || !out) return fail(nullptr, CDSL_EINVAL, "null argument");
  *out = nullptr;
  std::string why;
  if (!cfg_ok(draft->cfg, why)) return fail(nullptr, CDSL_EINVAL, "draft: " + why);
  if (!cfg_ok(target->cfg, why)) return fail(nullptr, CDSL_EINVAL, "target: " + why);
  if (draft->cfg.vocab != target->cfg.vocab)
    return fail(nullptr, CDSL_EINVAL, "draft and target vocabularies differ");
  if (draft->cfg.dtype != target->cfg.dtype) return fail(nullptr, CDSL_EINVAL, "draft and target dtypes differ");
  const cdsl_limits& l = *limits;
  if (l.max_batch <= 0 || l.max_ctx <= 0 || l.max_k <= 0 || l.max_k > kMaxK || l.max_d <= 0 || l.max_d > kMaxD ||
      l.max_prompt <= 0 || l.max_prompt > l.max_ctx || l.max_prefixes <= 0)
    return fail(nullptr, CDSL_EINVAL, "invalid limits (max_k <= 16, max_d <= 32, max_prompt <= max_ctx)");
  cdsl_ctx* c = new (std::nothrow) cdsl_ctx();
  if (!c) return fail(nullptr, CDSL_ENOMEM, "host allocation failed");
  c->st = (hipStream_t)stream;
  c->lim = l;
  c->dtype = draft->cfg.dtype;
  int rc = guarded(c, [&]() {
    const int max_pos = l.max_ctx + l.max_d + 2;
    load_model(c, c->m[0], *draft, max_pos);
    load_model(c, c->m[1], *target, max_pos);
    c->pstride = (l.max_ctx + l.max_d + 2 + kBlock - 1) / kBlock;
    c->sblocks = (l.max_d + kBlock - 1) / kBlock;
    const int suffix_blocks = l.max_batch * l.max_k * c->sblocks;
    const int prefix_blocks = l.max_prefixes * l.max_batch * c->pstride;
    c->nblocks = suffix_blocks + prefix_blocks;
    alloc_pool(c, c->m[0]);
    alloc_pool(c, c->m[1]);
    std::vector<int> st_ids(suffix_blocks);
    for (int u = 0; u < suffix_blocks; ++u) st_ids[u] = u;
    c->stable = dev_alloc<int>(c, suffix_blocks);
    CK(hipMemcpy(c->stable, st_ids.data(), suffix_blocks * sizeof(int), hipMemcpyHostToDevice));
    c->pool_blocks.reset(suffix_blocks, c->nblocks);
    std::vector<int> io(l.max_batch);
    for (int u = 0; u < l.max_batch; ++u) io[u] = u;
    c->iota = dev_alloc<int>(c, l.max_batch);
    CK(hipMemcpy(c->iota, io.data(), io.size() * sizeof(int), hipMemcpyHostToDevice));
    c->stage_tcap = l.max_d + 1;
    c->stage_stride = kStageHdr + c->stage_tcap + 2 * l.max_k;
    c->stage = dev_alloc<int>(c, (size_t)l.max_batch * c->stage_stride);
    c->bad = dev_alloc<int>(c, 1);
    CK(fill_int_launch(c->bad, 0, 1, c->st));
    c->ids_dev = dev_alloc<int>(c, l.max_batch);
    c->catch_tok = dev_alloc<int>(c, l.max_batch);
    c->mask_dev = dev_alloc<int>(c, l.max_batch);
    c->cnt_dev = dev_alloc<int>(c, l.max_batch);
    CK(hipHostMalloc((void**)&c->stage_host, (size_t)l.max_batch * c->stage_stride * sizeof(int), 0));
    CK(hipHostMalloc((void**)&c->table_host, (size_t)l.max_batch * c->pstride * sizeof(int), 0));
    CK(hipHostMalloc((void**)&c->ids_host, (size_t)l.max_batch * sizeof(int), 0));
    CK(hipHostMalloc((void**)&c->bad_host, sizeof(int), 0));
    CK(hipHostMalloc((void**)&c->mask_host, (size_t)l.max_batch * sizeof(int), 0));
    CK(hipHostMalloc((void**)&c->cnt_host, (size_t)l.max_batch * sizeof(int), 0));
    alloc_workspace(c);
    CK(hipStreamSynchronize(c->st));
    return CDSL_OK;
  });
  if (rc != CDSL_OK) {
    std::string msg = c->err;
    destroy_ctx(c);
    return fail(nullptr, rc, msg);
  }
  {
    std::lock_guard<std::mutex> g(g_live_mu);
    g_live.insert(c);
  }
  *out = c;
  return CDSL_OK;
}

int cdsl_destroy(cdsl_ctx* c) {
  if (!c) return CDSL_OK;
  {
    std::lock_guard<std::mutex> g(g_live_mu);
    if (!g_live.erase(c)) return fail(nullptr, CDSL_ESTATE, "unknown or destroyed context");
  }
  destroy_ctx(c);
  return CDSL_OK;
}

}  // extern "C"

void destroy_ctx(cdsl_ctx* c) {
  if (c->st) (void)hipStreamSynchronize(c->st);
  else (void)hipDeviceSynchronize();
  for (auto& p : c->pend) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  for (hipEvent_t e : c->ev_free) (void)hipEventDestroy(e);
  for (void* p : c->allocs) (void)hipFree(p);
  if (c->stage_host) (void)hipHostFree(c->stage_host);
  if (c->table_host) (void)hipHostFree(c->table_host);
  if (c->ids_host) (void)hipHostFree(c->ids_host);
  if (c->bad_host) (void)hipHostFree(c->bad_host);
  if (c->mask_host) (void)hipHostFree(c->mask_host);
  if (c->cnt_host) (void)hipHostFree(c->cnt_host);
  for (cdsl_prefix* px : c->prefixes) delete px;
  delete c;
}

extern "C" {

const char* cdsl_last_error(const cdsl_ctx* c) {
  if (c && ctx_live(c)) return c->err.c_str();
  return g_err.c_str();
}

int cdsl_prefill(cdsl_ctx* c, const int32_t* tokens, int32_t B, int32_t L, int32_t k, cdsl_prefix** out,
                 int32_t* beams, float* head_lp) {
  Range range_("cdsl_prefill");
  CTX_CHECK(c);
  if (!tokens || !out || !beams || !head_lp) return fail(c, CDSL_EINVAL, "null argument");
  if (B <= 0 || L <= 0 || k <= 0) return fail(c, CDSL_EINVAL, "B, L and k must be positive");
  if (B > c->lim.max_batch || L > c->lim.max_prompt || k > c->lim.max_k)
    return fail(c, CDSL_ERANGE, "B, L or k beyond the limits");
  if (k > c->m[1].c.vocab) return fail(c, CDSL_EINVAL, "k exceeds the vocabulary");
  if (c->live_prefixes >= c->lim.max_prefixes) return fail(c, CDSL_ERANGE, "too many live prefixes");
  *out = nullptr;
  cdsl_prefix* px = new (std::nothrow) cdsl_prefix();
  if (!px) return fail(c, CDSL_ENOMEM, "host allocation failed");
  int rc = guarded(c, [&]() {
    // the pinned block-table staging buffer may still feed the table copy
    // a commit queued for another prefix: let the stream drain before
    // upload_table refills it
    CK(hipStreamSynchronize(c->st));
    px->B = B;
    px->L0 = L;
    px->len.assign(B, 0);
    px->table.assign((size_t)B * c->pstride, -1);
    // per-handle device state (lengths, block table, emitted tokens)
    px->Lp = dev_alloc<int>(c, B);
    px->table_dev = dev_alloc<int>(c, (size_t)B * c->pstride);
    px->gen = dev_alloc<int>(c, (size_t)B * c->lim.max_ctx);
    px->gen_len = dev_alloc<int>(c, B);
    px->ptail = dev_alloc<int>(c, B);
    px->Lm1 = dev_alloc<int>(c, B);
    for (int b = 0; b < B; ++b) ensure_blocks(c, px, b, L);
    upload_table(c, px);
    CK(fill_int_launch(px->Lp, 0, B, c->st));
    CK(fill_int_launch(px->gen_len, 0, B, c->st));
    const int chunk = prefill_chunk_prompts(c->lim);
    for (int b0 = 0; b0 < B; b0 += chunk) {
      const int nb = std::min(chunk, B - b0);
      PassDesc p = base_pass(c, px);
      p.mode = kAppend;
      p.nb = nb;
      p.kp = 1;
      p.R = L;
      p.j0 = 0;
      p.prompt_ids = c->iota + b0;
      p.tok = tokens;
      p.tok_stride = L;
      p.tok_off = 0;
      LogitArgs la{};
      la.bad = c->bad;
      la.V = c->m[1].c.vocab;
      la.want_lse = 1;
      la.kk = k;
      la.topk_ids = beams;
      la.topk_lp = head_lp;
      la.topk_rows = c->iota + b0;
      run_pass(c, c->m[0], p, 0, 0, false, false, nullptr, true);
      run_pass(c, c->m[1], p, 0, 0, true, true, nullptr, true, nullptr, 0, &la);
    }
    CK(add_launch(B, nullptr, px->Lp, L, c->st));
    CK(last_tokens_launch(B, tokens, L, px->ptail, c->st));
    for (int b = 0; b < B; ++b) px->len[b] = L;
    queue_bad(c);
    CK(hipStreamSynchronize(c->st));
    check_bad(c);
    return CDSL_OK;
  });
  if (rc != CDSL_OK) {
    (void)hipStreamSynchronize(c->st);
    c->pool_blocks.release(px->owned);
    free_px_buffers(c, px);
    delete px;
    return rc;
  }
  c->live_prefixes++;
  c->prefixes.insert(px);
  *out = px;
  return CDSL_OK;
}

int cdsl_rollout(cdsl_ctx* c, cdsl_prefix* px, const int32_t* beams, int32_t k, int32_t d, int32_t* lookaheads) {
  return cdsl_rollout_with(c, px, beams, k, d, 0, lookaheads);
}

namespace {

// d sequential passes of the roller over all B*k beams; with keep, the
// logits of pass j land in keep[(b*k + i)*d + j][V] instead of the workspace
// pfx: Alg. 1's drafting loop from the prefix itself (k = 1, no beams):
// pass 0 re-feeds the last prefix token at position Lp - 1 into suffix slot 0
// (the pass sees the prefix minus that token), so its argmax is the draft's
// greedy token at the end of the prefix.
int rollout_impl(cdsl_ctx* c, cdsl_prefix* px, const int32_t* beams, int32_t k, int32_t d, int32_t roller,
                 int32_t* lookaheads, float* keep, bool pfx = false) {
  Range range_("cdsl_rollout");
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (roller != 0 && roller != 1) return fail(c, CDSL_EINVAL, "roller must be 0 (draft) or 1 (target)");
  if (!px || (!beams && !pfx) || !lookaheads) return fail(c, CDSL_EINVAL, "null argument");
  if (k <= 0 || d <= 0) return fail(c, CDSL_EINVAL, "k and d must be positive");
  if (k > c->lim.max_k || d > c->lim.max_d) return fail(c, CDSL_ERANGE, "k or d beyond the limits");
  if (max_len(px) + d + 1 > c->lim.max_ctx) return fail(c, CDSL_ERANGE, "context would exceed max_ctx");
  const int V = c->m[roller].c.vocab;
  if (keep && (long long)d * V > INT32_MAX) return fail(c, CDSL_ERANGE, "d * vocab too large for the kept logits");
  return guarded(c, [&]() {
    const int B = px->B;
    if (pfx)
      CK(prefix_tail_launch(B, px->gen, c->lim.max_ctx, px->gen_len, px->ptail, px->Lp, px->Lm1, lookaheads, d + 1,
                            c->st));
    else
      CK(heads_to_lookaheads_launch(B * k, d, beams, lookaheads, c->st));
    const int Lmax = max_len(px);
    for (int j0 = 0; j0 < d; ++j0) {
      PassDesc p = base_pass(c, px);
      if (pfx) p.Lp = px->Lm1;
      p.mode = kSuffix;
      p.nb = B;
      p.kp = k;
      p.R = 1;
      p.j0 = j0;
      p.tok = lookaheads;
      p.tok_stride = d + 1;
      p.tok_off = j0;
      float* dst = keep ? keep + (long long)j0 * V : nullptr;
      LogitArgs la{};
      la.bad = c->bad;
      la.V = V;
      la.want_lse = 0;
      la.kk = 0;
      la.amax = lookaheads;
      la.amax_map.enabled = 1;
      la.amax_map.p = p;
      la.amax_map.stride = d + 1;
      la.amax_map.off = j0 + 1;
      if (keep) {
        // the kept logits are an output: write them, then take the argmax
        run_pass(c, c->m[roller], p, Lmax, sum_len(px), true, false, nullptr, false, dst, d * V);
        la.logits = dst;
        la.ld = (long long)d * V;
        logit_rows(c, la, p.M());
      } else {
        run_pass(c, c->m[roller], p, Lmax, sum_len(px), true, false, nullptr, false, nullptr, 0, &la);
      }
    }
    px->rolled_k = k;
    px->rolled_d = d;
    px->rolled_pfx = pfx ? 1 : 0;
    px->verified_k = px->verified_d = 0;
    px->verified_pfx = 0;
    px->kept_logits = keep;
    return CDSL_OK;
  });
}

}  // namespace

int cdsl_rollout_with(cdsl_ctx* c, cdsl_prefix* px, const int32_t* beams, int32_t k, int32_t d, int32_t roller,
                      int32_t* lookaheads) {
  return rollout_impl(c, px, beams, k, d, roller, lookaheads, nullptr);
}

int cdsl_rollout_keep(cdsl_ctx* c, cdsl_prefix* px, const int32_t* beams, int32_t k, int32_t d, int32_t* lookaheads,
                      float* draft_logits) {
  CTX_CHECK(c);
  if (!draft_logits) return fail(c, CDSL_EINVAL, "null argument");
  return rollout_impl(c, px, beams, k, d, 0, lookaheads, draft_logits);
}

int cdsl_draft_prefix(cdsl_ctx* c, cdsl_prefix* px, int32_t d, int32_t* lookaheads, float* draft_logits) {
  return rollout_impl(c, px, nullptr, 1, d, 0, lookaheads, draft_logits, true);
}

int cdsl_verify(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d, const float* head_lp,
                float* logprobs, int32_t* target_argmax, int32_t* n_accept, float* scores, int32_t* row_topk_ids,
                float* row_topk_lp, float* hidden) {
  return cdsl_verify_kk(c, px, look, k, d, k, head_lp, logprobs, target_argmax, n_accept, scores, row_topk_ids,
                        row_topk_lp, hidden);
}

namespace {

struct SoftArgs {
  const float* draft_logits;   // [B, k, d, V] from cdsl_rollout_keep
  const float* u;              // [B, k, d]
  const float* v;              // [B, k, d]
  float* draft_lp;             // [B, k, d]
  int32_t* res_ids;            // [B, k, d]
  float* res_lp;               // [B, k, d]
};

// pfx: Alg. 1's verification of a lookahead drafted from the prefix (k = 1):
// row 0 re-feeds the last prefix token at position Lp - 1, so row j gives
// p_{j+1} = M_p(pfx + x_1..x_j); no head log-prob enters the score.
int verify_impl(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d, int32_t kk,
                const float* head_lp, float* logprobs, int32_t* target_argmax, int32_t* n_accept, float* scores,
                int32_t* row_topk_ids, float* row_topk_lp, float* hidden, const SoftArgs* soft, bool pfx = false) {
  Range range_("cdsl_verify");
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (kk <= 0 || kk > c->lim.max_k) return fail(c, CDSL_ERANGE, "top-k width beyond the limits");
  if (!px || !look || (!head_lp && !pfx) || !logprobs || !target_argmax || !n_accept || !scores || !row_topk_ids ||
      !row_topk_lp)
    return fail(c, CDSL_EINVAL, "null argument");
  if (k <= 0 || d <= 0) return fail(c, CDSL_EINVAL, "k and d must be positive");
  if (k > c->lim.max_k || d > c->lim.max_d) return fail(c, CDSL_ERANGE, "k or d beyond the limits");
  if (max_len(px) + d + 1 > c->lim.max_ctx) return fail(c, CDSL_ERANGE, "context would exceed max_ctx");
  if (soft) {
    if (!soft->draft_logits || !soft->u || !soft->v || !soft->draft_lp || !soft->res_ids || !soft->res_lp)
      return fail(c, CDSL_EINVAL, "null argument");
    if (c->m[0].c.vocab != c->m[1].c.vocab) return fail(c, CDSL_EINVAL, "soft rejection needs one vocabulary");
    if (soft->draft_logits != px->kept_logits || px->rolled_k != k || px->rolled_d != d || px->rolled_pfx != (pfx ? 1 : 0))
      return fail(c, CDSL_ESTATE, "soft verification needs the kept draft logits of the matching rollout (same k, d)");
  }
  return guarded(c, [&]() {
    const int B = px->B;
    if (pfx)
      CK(prefix_tail_launch(B, px->gen, c->lim.max_ctx, px->gen_len, px->ptail, px->Lp, px->Lm1, nullptr, 0, c->st));
    PassDesc p = base_pass(c, px);
    if (pfx) p.Lp = px->Lm1;
    p.mode = kSuffix;
    p.nb = B;
    p.kp = k;
    p.R = d;
    p.j0 = 0;
    p.tok = look;
    p.tok_stride = d + 1;
    p.tok_off = 0;
    LogitArgs la{};
    la.bad = c->bad;
    la.V = c->m[1].c.vocab;
    la.want_lse = 1;
    la.kk = kk;
    la.amax = target_argmax;
    la.lp = logprobs;
    la.gather_tok = look;
    la.gather_map.enabled = 1;
    la.gather_map.p = p;
    la.gather_map.stride = d + 1;
    la.gather_map.off = 1;
    la.topk_ids = row_topk_ids;
    la.topk_lp = row_topk_lp;
    if (soft) {
      // speculative sampling reads the target's logit rows: keep them
      run_pass(c, c->m[1], p, max_len(px), sum_len(px), true, false, hidden);
      la.logits = c->ws.logits;
      logit_rows(c, la, p.M());
    } else {
      run_pass(c, c->m[1], p, max_len(px), sum_len(px), true, false, hidden, false, nullptr, 0, &la);
    }
    if (soft) {
      Span sp(c, CDSL_K_LOGIT_ROWS, 0.0, (double)p.M() * la.V * 4.0 * 2.0);
      CK(soft_rows_launch(c->ws.logits, soft->draft_logits, p.M(), la.V, d, look, soft->v, soft->draft_lp,
                          soft->res_ids, soft->res_lp, c->st));
    }
    {
      Span sp(c, CDSL_K_STEP, 0.0, (double)B * k * d * (soft ? 20.0 : 12.0));
      CK(beam_scores_launch(B * k, d, look, target_argmax, logprobs, head_lp, soft ? soft->draft_lp : nullptr,
                            soft ? soft->u : nullptr, n_accept, scores, c->st));
    }
    px->verified_k = k;
    px->verified_d = d;
    px->verified_kk = kk;
    px->verified_soft = soft ? 1 : 0;
    px->verified_pfx = pfx ? 1 : 0;
    return CDSL_OK;
  });
}

}  // namespace

int cdsl_verify_kk(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d, int32_t kk,
                   const float* head_lp, float* logprobs, int32_t* target_argmax, int32_t* n_accept, float* scores,
                   int32_t* row_topk_ids, float* row_topk_lp, float* hidden) {
  return verify_impl(c, px, look, k, d, kk, head_lp, logprobs, target_argmax, n_accept, scores, row_topk_ids,
                     row_topk_lp, hidden, nullptr);
}

int cdsl_verify_soft(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d, int32_t kk,
                     const float* head_lp, const float* draft_logits, const float* u, const float* v,
                     float* logprobs, float* draft_lp, int32_t* target_argmax, int32_t* n_accept, float* scores,
                     int32_t* row_topk_ids, float* row_topk_lp, int32_t* res_ids, float* res_lp, float* hidden) {
  const SoftArgs sa{draft_logits, u, v, draft_lp, res_ids, res_lp};
  return verify_impl(c, px, look, k, d, kk, head_lp, logprobs, target_argmax, n_accept, scores, row_topk_ids,
                     row_topk_lp, hidden, &sa);
}

int cdsl_verify_prefix(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t d, int32_t kk, float* logprobs,
                       int32_t* target_argmax, int32_t* n_accept, float* scores, int32_t* row_topk_ids,
                       float* row_topk_lp) {
  return verify_impl(c, px, look, 1, d, kk, nullptr, logprobs, target_argmax, n_accept, scores, row_topk_ids,
                     row_topk_lp, nullptr, nullptr, true);
}

int cdsl_verify_prefix_soft(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t d, int32_t kk,
                            const float* draft_logits, const float* u, const float* v, float* logprobs,
                            float* draft_lp, int32_t* target_argmax, int32_t* n_accept, float* scores,
                            int32_t* row_topk_ids, float* row_topk_lp, int32_t* res_ids, float* res_lp) {
  const SoftArgs sa{draft_logits, u, v, draft_lp, res_ids, res_lp};
  return verify_impl(c, px, look, 1, d, kk, nullptr, logprobs, target_argmax, n_accept, scores, row_topk_ids,
                     row_topk_lp, nullptr, &sa, true);
}

int cdsl_reward_keywords(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d,
                         const int32_t* keywords, int32_t n_kw, int32_t normalize, float* reward) {
  return cdsl_reward_keywords_upto(c, px, look, k, d, nullptr, keywords, n_kw, normalize, reward);
}

namespace {
int reward_kw_impl(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d, const int32_t* upto,
                   int head, const int32_t* keywords, int32_t n_kw, int32_t normalize, float* reward) {
  Range range_("cdsl_reward_keywords");
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (!px || !look || !keywords || !reward) return fail(c, CDSL_EINVAL, "null argument");
  if (k <= 0 || d <= 0 || n_kw <= 0 || n_kw > 64) return fail(c, CDSL_EINVAL, "bad k, d or n_kw (1..64)");
  return guarded(c, [&]() {
    Span sp(c, CDSL_K_STEP, 0.0, (double)px->B * k * (d + 1) * 4.0);
    CK(reward_keywords_launch(px->B, k, d, px->gen, c->lim.max_ctx, px->gen_len, look, upto, head, keywords, n_kw,
                              normalize, reward, c->st));
    return CDSL_OK;
  });
}
}  // namespace

int cdsl_reward_keywords_upto(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t k, int32_t d,
                              const int32_t* upto, const int32_t* keywords, int32_t n_kw, int32_t normalize,
                              float* reward) {
  return reward_kw_impl(c, px, look, k, d, upto, 1, keywords, n_kw, normalize, reward);
}

int cdsl_reward_keywords_prefix(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, int32_t d, const int32_t* upto,
                                const int32_t* keywords, int32_t n_kw, int32_t normalize, float* reward) {
  return reward_kw_impl(c, px, look, 1, d, upto, 0, keywords, n_kw, normalize, reward);
}

int cdsl_reward_linear(cdsl_ctx* c, const float* hidden, const float* w, int32_t B, int32_t k, int32_t D,
                       float* reward) {
  Range range_("cdsl_reward_linear");
  CTX_CHECK(c);
  if (!hidden || !w || !reward || B <= 0 || k <= 0 || D <= 0) return fail(c, CDSL_EINVAL, "bad argument");
  return guarded(c, [&]() {
    Span sp(c, CDSL_K_STEP, 2.0 * B * k * D, (double)B * k * D * 4.0);
    CK(reward_linear_launch(B * k, hidden, w, D, reward, c->st));
    return CDSL_OK;
  });
}

int cdsl_select(cdsl_ctx* c, const float* scores, const float* reward, float alpha, int32_t B, int32_t k,
                int32_t* beam) {
  Range range_("cdsl_select");
  CTX_CHECK(c);
  if (!scores || !reward || !beam || B <= 0 || k <= 0) return fail(c, CDSL_EINVAL, "bad argument");
  if (isnan(alpha) || (isinf(alpha) && alpha < 0)) return fail(c, CDSL_EINVAL, "alpha must be finite or +inf");
  return guarded(c, [&]() {
    const int reward_only = isinf(alpha) ? 1 : 0;
    Span sp(c, CDSL_K_STEP, 0.0, (double)B * k * 8.0);
    CK(select_launch(B, k, scores, reward, reward_only ? 0.f : alpha, reward_only, nullptr, beam, c->st));
    return CDSL_OK;
  });
}

int cdsl_select_first(cdsl_ctx* c, const float* reward, const float* first_at, int32_t B, int32_t k,
                      int32_t* beam) {
  Range range_("cdsl_select_first");
  CTX_CHECK(c);
  if (!reward || !first_at || !beam || B <= 0 || k <= 0) return fail(c, CDSL_EINVAL, "bad argument");
  return guarded(c, [&]() {
    Span sp(c, CDSL_K_STEP, 0.0, (double)B * (k * 4.0 + 8.0));
    CK(select_launch(B, k, reward, reward, 0.f, 1, first_at, beam, c->st));
    return CDSL_OK;
  });
}

int cdsl_controller_states(cdsl_ctx* c, const int32_t* n_accept, const float* reward, int32_t B, int32_t d,
                           double a_t, double r_t, int32_t b, int32_t* state, float* first_at) {
  Range range_("cdsl_controller_states");
  CTX_CHECK(c);
  if (!n_accept || !reward || !state || !first_at || B <= 0 || d <= 0) return fail(c, CDSL_EINVAL, "bad argument");
  if (b != 0 && b != 1) return fail(c, CDSL_EINVAL, "b must be 0 or 1");
  if (isnan(a_t) || isnan(r_t)) return fail(c, CDSL_EINVAL, "thresholds must not be NaN");
  return guarded(c, [&]() {
    Span sp(c, CDSL_K_STEP, 0.0, (double)B * 16.0);
    CK(controller_states_launch(B, d, n_accept, reward, a_t, r_t, b, state, first_at, c->st));
    return CDSL_OK;
  });
}

int cdsl_commit(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, const int32_t* n_accept,
                const int32_t* rtk_ids, const float* rtk_lp, int32_t k, int32_t d, int32_t* emitted_host,
                int32_t* n_emit_host, int32_t* next_beams, float* next_head_lp) {
  return cdsl_commit_kk(c, px, look, beam, n_accept, rtk_ids, rtk_lp, k, d, k, emitted_host, n_emit_host,
                        next_beams, next_head_lp);
}

namespace {
int commit_impl(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, const int32_t* n_accept,
                const int32_t* rtk_ids, const float* rtk_lp, const int32_t* res_ids, const float* res_lp, int32_t k,
                int32_t d, int32_t kk, int32_t* emitted_host, int32_t* n_emit_host, int32_t* next_beams,
                float* next_head_lp, bool pfx);
}  // namespace

int cdsl_commit_kk(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, const int32_t* n_accept,
                   const int32_t* rtk_ids, const float* rtk_lp, int32_t k, int32_t d, int32_t kk,
                   int32_t* emitted_host, int32_t* n_emit_host, int32_t* next_beams, float* next_head_lp) {
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (px && px->verified_soft)
    return fail(c, CDSL_ESTATE, "the last verification was soft: commit it with cdsl_commit_soft");
  return commit_impl(c, px, look, beam, n_accept, rtk_ids, rtk_lp, nullptr, nullptr, k, d, kk, emitted_host,
                     n_emit_host, next_beams, next_head_lp, false);
}

int cdsl_commit_soft(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, const int32_t* n_accept,
                     const int32_t* rtk_ids, const float* rtk_lp, const int32_t* res_ids, const float* res_lp,
                     int32_t k, int32_t d, int32_t kk, int32_t* emitted_host, int32_t* n_emit_host,
                     int32_t* next_beams, float* next_head_lp) {
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (!res_ids || !res_lp) return fail(c, CDSL_EINVAL, "null argument");
  if (px && !px->verified_soft) return fail(c, CDSL_ESTATE, "cdsl_commit_soft needs a cdsl_verify_soft");
  return commit_impl(c, px, look, beam, n_accept, rtk_ids, rtk_lp, res_ids, res_lp, k, d, kk, emitted_host,
                     n_emit_host, next_beams, next_head_lp, false);
}

int cdsl_commit_prefix(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* n_accept, int32_t d,
                       int32_t kk, const int32_t* rtk_ids, const float* rtk_lp, int32_t* emitted_host,
                       int32_t* n_emit_host, int32_t* next_beams, float* next_head_lp) {
  CTX_CHECK(c);
  PX_CHECK(c, px);
  return commit_impl(c, px, look, nullptr, n_accept, rtk_ids, rtk_lp, nullptr, nullptr, 1, d, kk, emitted_host,
                     n_emit_host, next_beams, next_head_lp, true);
}

namespace {
// Beam commit (pfx false: emit [c_i*, x_i*,1..n], suffix slots 0..n hold
// their KV) or Alg. 1 commit (pfx: emit x_1..x_n, slots 1..n hold their KV;
// slot 0 re-fed the last prefix token).  The kernel only stages the
// decisions; they are carried out once every prompt's record has passed the
// host checks.  When the emitted tokens run past the rows the passes fed,
// the last one is fed through both models as a catch-up row that yields the
// next heads.
int commit_impl(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, const int32_t* n_accept,
                const int32_t* rtk_ids, const float* rtk_lp, const int32_t* res_ids, const float* res_lp, int32_t k,
                int32_t d, int32_t kk, int32_t* emitted_host, int32_t* n_emit_host, int32_t* next_beams,
                float* next_head_lp, bool pfx) {
  Range range_("cdsl_commit");
  if (!px || !look || (!beam && !pfx) || !n_accept || !rtk_ids || !rtk_lp || !emitted_host || !n_emit_host ||
      !next_beams || !next_head_lp)
    return fail(c, CDSL_EINVAL, "null argument");
  if (px->rolled_k != k || px->rolled_d != d || px->verified_k != k || px->verified_d != d)
    return fail(c, CDSL_ESTATE, "commit needs a rollout and a verify with the same k and d");
  if (px->rolled_pfx != (pfx ? 1 : 0) || px->verified_pfx != (pfx ? 1 : 0))
    return fail(c, CDSL_ESTATE,
                pfx ? "cdsl_commit_prefix needs cdsl_draft_prefix and a prefix verification"
                    : "a beam commit needs a beam rollout and verification");
  if (px->verified_kk != kk) return fail(c, CDSL_ESTATE, "commit needs a verify with the same top-k width");
  return guarded(c, [&]() {
    const int B = px->B;
    {
      Span sp(c, CDSL_K_STEP, 0.0, (double)B * (d + 1 + 2 * kk) * 4.0);
      if (pfx)
        CK(commit_prefix_launch(B, d, kk, look, n_accept, rtk_ids, rtk_lp, c->stage, c->stage_stride, c->stage_tcap,
                                c->st));
      else
        CK(commit_launch(B, k, d, kk, look, beam, n_accept, rtk_ids, rtk_lp, res_ids, res_lp, c->stage,
                         c->stage_stride, c->stage_tcap, c->st));
    }
    CK(hipMemcpyAsync(c->stage_host, c->stage, (size_t)B * c->stage_stride * sizeof(int), hipMemcpyDeviceToHost,
                      c->st));
    queue_bad(c);
    CK(hipStreamSynchronize(c->st));
    if (c->prof) harvest(c);
    check_bad(c);
    const int dlim = pfx ? d - 1 : d;      // emitted tokens whose KV the passes wrote
    for (int b = 0; b < B; ++b) {
      const int ne = c->stage_host[(size_t)b * c->stage_stride];
      if (ne < 0) {
        g_err = pfx ? "n_accept out of [0, d] for prompt " + std::to_string(b)
                    : "invalid beam index (NaN score or reward?) for prompt " + std::to_string(b);
        throw Fail{CDSL_EINVAL};
      }
      if (px->len[b] + ne > c->lim.max_ctx) {
        g_err = "prompt " + std::to_string(b) + " exceeds max_ctx";
        throw Fail{CDSL_ERANGE};
      }
    }
    int ncatch = 0;
    for (int b = 0; b < B; ++b) {
      const int* stg = c->stage_host + (size_t)b * c->stage_stride;
      ensure_blocks(c, px, b, px->len[b] + stg[0]);
      if (stg[1]) c->ids_host[ncatch++] = b;
    }
    upload_table(c, px);
    {
      Span sp(c, CDSL_K_STEP, 0.0, (double)B * (d + 1 + 2 * kk) * 8.0);
      CK(commit_apply_launch(B, c->stage, c->stage_stride, c->stage_tcap, kk, px->gen, c->lim.max_ctx, px->gen_len,
                             next_beams, next_head_lp, c->catch_tok, c->st));
    }
    if (dlim > 0)
      for (int mi = 0; mi < 2; ++mi) {
        Model& md = c->m[mi];
        Span sp(c, CDSL_K_STEP, 0.0, 0.0);
        CK(promote_launch(B, k, md.pool, md.c.n_layers, c->stage, c->stage_stride, dlim, pfx ? 1 : 0, px->Lp,
                          px->table_dev, c->pstride, c->stable, c->lim.max_k * c->sblocks, c->sblocks, md.c.dtype,
                          c->st));
      }
    CK(advance_launch(B, c->stage, c->stage_stride, dlim, px->Lp, c->st));
    for (int b = 0; b < B; ++b) px->len[b] += std::min(c->stage_host[(size_t)b * c->stage_stride], dlim);
    if (ncatch > 0) {
      CK(hipMemcpyAsync(c->ids_dev, c->ids_host, ncatch * sizeof(int), hipMemcpyHostToDevice, c->st));
      PassDesc p = base_pass(c, px);
      p.mode = kAppend;
      p.nb = ncatch;
      p.kp = 1;
      p.R = 1;
      p.j0 = 0;
      p.prompt_ids = c->ids_dev;
      p.tok = c->catch_tok;
      p.tok_stride = 1;
      p.tok_off = 0;
      const int Lmax = max_len(px);
      long long sl = 0;
      for (int u = 0; u < ncatch; ++u) sl += px->len[c->ids_host[u]];
      LogitArgs la{};
      la.bad = c->bad;
      la.V = c->m[1].c.vocab;
      la.want_lse = 1;
      la.kk = kk;
      la.topk_ids = next_beams;
      la.topk_lp = next_head_lp;
      la.topk_rows = c->ids_dev;
      run_pass(c, c->m[0], p, Lmax, sl, false, false, nullptr);
      run_pass(c, c->m[1], p, Lmax, sl, true, false, nullptr, false, nullptr, 0, &la);
      CK(add_launch(ncatch, c->ids_dev, px->Lp, 1, c->st));
      for (int u = 0; u < ncatch; ++u) px->len[c->ids_host[u]] += 1;
    }
    const int width = pfx ? d : d + 1;
    for (int b = 0; b < B; ++b) {
      const int* stg = c->stage_host + (size_t)b * c->stage_stride;
      n_emit_host[b] = stg[0];
      for (int t = 0; t < width; ++t) emitted_host[(size_t)b * width + t] = t < stg[0] ? stg[kStageHdr + t] : -1;
    }
    px->rolled_k = px->rolled_d = px->verified_k = px->verified_d = 0;
    px->rolled_pfx = px->verified_pfx = 0;
    px->verified_soft = 0;
    px->kept_logits = nullptr;
    return CDSL_OK;
  });
}
}  // namespace

}  // extern "C"

namespace {
// One emitted token per selected prompt (the head-only commit of the
// lookahead-heuristic step, or a token given directly): stage_launch
// writes the records, then each emitting prompt's token is appended to its
// generated tokens and fed through both models as one row, whose target
// row gives the next heads.
template <typename StageFn>
int append_impl(cdsl_ctx* c, cdsl_prefix* px, int32_t kk, const int32_t* mask_host, int32_t* emitted_host,
                int32_t* next_beams, float* next_head_lp, const char* bad_msg_c, StageFn&& stage_launch) {
  Range range_("cdsl_append");
  const std::string bad_msg = bad_msg_c;
  return guarded(c, [&]() {
    const int B = px->B;
    for (int b = 0; b < B; ++b) c->mask_host[b] = mask_host ? (mask_host[b] != 0) : 1;
    CK(hipMemcpyAsync(c->mask_dev, c->mask_host, (size_t)B * sizeof(int), hipMemcpyHostToDevice, c->st));
    {
      Span sp(c, CDSL_K_STEP, 0.0, (double)B * 16.0);
      stage_launch();
    }
    CK(hipMemcpyAsync(c->stage_host, c->stage, (size_t)B * c->stage_stride * sizeof(int), hipMemcpyDeviceToHost,
                      c->st));
    queue_bad(c);
    CK(hipStreamSynchronize(c->st));
    if (c->prof) harvest(c);
    check_bad(c);
    for (int b = 0; b < B; ++b) {
      const int* stg = c->stage_host + (size_t)b * c->stage_stride;
      if (stg[0] < 0) {
        g_err = bad_msg + std::to_string(b);
        throw Fail{CDSL_EINVAL};
      }
      if (stg[0] > 0 && px->len[b] + 1 > c->lim.max_ctx) {
        g_err = "prompt " + std::to_string(b) + " exceeds max_ctx";
        throw Fail{CDSL_ERANGE};
      }
    }
    int n = 0;
    for (int b = 0; b < B; ++b) {
      if (c->stage_host[(size_t)b * c->stage_stride] == 0) continue;
      ensure_blocks(c, px, b, px->len[b] + 1);
      c->ids_host[n++] = b;
    }
    if (n > 0) {
      // the chosen heads go through both models as one appended row each
      // (the rolled suffixes are dropped), and the target row gives the
      // next heads
      upload_table(c, px);
      CK(commit_apply_launch(B, c->stage, c->stage_stride, c->stage_tcap, kk, px->gen, c->lim.max_ctx, px->gen_len,
                             next_beams, next_head_lp, c->catch_tok, c->st));
      CK(hipMemcpyAsync(c->ids_dev, c->ids_host, n * sizeof(int), hipMemcpyHostToDevice, c->st));
      PassDesc p = base_pass(c, px);
      p.mode = kAppend;
      p.nb = n;
      p.kp = 1;
      p.R = 1;
      p.j0 = 0;
      p.prompt_ids = c->ids_dev;
      p.tok = c->catch_tok;
      p.tok_stride = 1;
      p.tok_off = 0;
      const int Lmax = max_len(px);
      long long sl = 0;
      for (int u = 0; u < n; ++u) sl += px->len[c->ids_host[u]];
      LogitArgs la{};
      la.bad = c->bad;
      la.V = c->m[1].c.vocab;
      la.want_lse = 1;
      la.kk = kk;
      la.topk_ids = next_beams;
      la.topk_lp = next_head_lp;
      la.topk_rows = c->ids_dev;
      run_pass(c, c->m[0], p, Lmax, sl, false, false, nullptr);
      run_pass(c, c->m[1], p, Lmax, sl, true, false, nullptr, false, nullptr, 0, &la);
      CK(add_launch(n, c->ids_dev, px->Lp, 1, c->st));
      for (int u = 0; u < n; ++u) px->len[c->ids_host[u]] += 1;
    }
    for (int b = 0; b < B; ++b) {
      const int* stg = c->stage_host + (size_t)b * c->stage_stride;
      emitted_host[b] = stg[0] > 0 ? stg[kStageHdr] : -1;
    }
    px->rolled_k = px->rolled_d = px->verified_k = px->verified_d = 0;
    px->rolled_pfx = px->verified_pfx = 0;
    px->verified_soft = 0;
    px->kept_logits = nullptr;
    return CDSL_OK;
  });
}

}  // namespace

extern "C" {

int cdsl_commit_heads(cdsl_ctx* c, cdsl_prefix* px, const int32_t* look, const int32_t* beam, int32_t k, int32_t d,
                      int32_t kk, const int32_t* mask_host, int32_t* emitted_host, int32_t* next_beams,
                      float* next_head_lp) {
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (kk <= 0 || kk > c->lim.max_k) return fail(c, CDSL_ERANGE, "top-k width beyond the limits");
  if (!px || !look || !beam || !emitted_host || !next_beams || !next_head_lp)
    return fail(c, CDSL_EINVAL, "null argument");
  if (px->rolled_k != k || px->rolled_d != d || px->rolled_pfx)
    return fail(c, CDSL_ESTATE, "commit_heads needs a beam rollout with the same k and d");
  return append_impl(c, px, kk, mask_host, emitted_host, next_beams, next_head_lp,
                     "invalid beam index (NaN reward?) for prompt ", [&]() {
                       CK(commit_heads_launch(px->B, k, d, look, beam, c->mask_dev, c->stage, c->stage_stride, c->st));
                     });
}

int cdsl_append(cdsl_ctx* c, cdsl_prefix* px, const int32_t* tokens, const int32_t* mask_host, int32_t kk,
                int32_t* emitted_host, int32_t* next_beams, float* next_head_lp) {
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (kk <= 0 || kk > c->lim.max_k) return fail(c, CDSL_ERANGE, "top-k width beyond the limits");
  if (!px || !tokens || !emitted_host || !next_beams || !next_head_lp) return fail(c, CDSL_EINVAL, "null argument");
  return append_impl(c, px, kk, mask_host, emitted_host, next_beams, next_head_lp,
                     "token id outside [0, vocab) for prompt ", [&]() {
                       CK(commit_tokens_launch(px->B, tokens, c->mask_dev, c->m[1].c.vocab, c->stage, c->stage_stride,
                                               c->st));
                     });
}

int cdsl_withdraw(cdsl_ctx* c, cdsl_prefix* px, const int32_t* count_host) {
  Range range_("cdsl_withdraw");
  CTX_CHECK(c);
  PX_CHECK(c, px);
  if (!px || !count_host) return fail(c, CDSL_EINVAL, "null argument");
  for (int b = 0; b < px->B; ++b)
    if (count_host[b] < 0 || count_host[b] > px->len[b] - px->L0)
      return fail(c, CDSL_EINVAL, "prompt " + std::to_string(b) + ": can only withdraw generated tokens");
  return guarded(c, [&]() {
    const int B = px->B;
    int any = 0;
    for (int b = 0; b < B; ++b) {
      c->cnt_host[b] = count_host[b];
      any |= count_host[b];
    }
    if (!any) return CDSL_OK;
    CK(hipMemcpyAsync(c->cnt_dev, c->cnt_host, (size_t)B * sizeof(int), hipMemcpyHostToDevice, c->st));
    {
      Span sp(c, CDSL_K_STEP, 0.0, (double)B * 12.0);
      CK(withdraw_launch(B, c->cnt_dev, px->Lp, px->gen_len, c->st));
    }
    for (int b = 0; b < B; ++b) px->len[b] -= count_host[b];
    // the counts are staged in pinned host memory: let the copy finish
    // before the next call refills it
    CK(hipStreamSynchronize(c->st));
    px->rolled_k = px->rolled_d = px->verified_k = px->verified_d = 0;
    px->rolled_pfx = px->verified_pfx = 0;
    px->verified_soft = 0;
    px->kept_logits = nullptr;
    return CDSL_OK;
  });
}

int cdsl_prefix_lengths(cdsl_ctx* c, const cdsl_prefix* px, int32_t* lengths_host) {
  CTX_CHECK(c);
  if (!px || !lengths_host) return fail(c, CDSL_EINVAL, "null argument");
  PX_CHECK(c, const_cast<cdsl_prefix*>(px));
  for (int b = 0; b < px->B; ++b) lengths_host[b] = px->len[b];
  return CDSL_OK;
}

int cdsl_profile_enable(cdsl_ctx* c, int32_t enable) {
  CTX_CHECK(c);
  return guarded(c, [&]() {
    CK(hipStreamSynchronize(c->st));
    harvest(c);
    c->acc = cdsl_kernel_stats{};
    c->prof = enable != 0;
    return CDSL_OK;
  });
}

int cdsl_profile_read(cdsl_ctx* c, cdsl_kernel_stats* out) {
  CTX_CHECK(c);
  if (!out) return fail(c, CDSL_EINVAL, "null argument");
  return guarded(c, [&]() {
    CK(hipStreamSynchronize(c->st));
    harvest(c);
    *out = c->acc;
    return CDSL_OK;
  });
}

int cdsl_free_prefix(cdsl_ctx* c, cdsl_prefix* px) {
  Range range_("cdsl_free_prefix");
  CTX_CHECK(c);
  if (!px) return CDSL_OK;
  PX_CHECK(c, px);
  return guarded(c, [&]() {
    CK(hipStreamSynchronize(c->st));
    c->pool_blocks.release(px->owned);
    free_px_buffers(c, px);
    c->prefixes.erase(px);
    delete px;
    c->live_prefixes--;
    return CDSL_OK;
  });
}

// ---------------------------------------------------------------------------
// kernel-level entry points (include/cdsl_ops.h)
// ---------------------------------------------------------------------------
// bf16 weights: the fp32 activation operand is split into its hi / lo planes
// at the start of the workspace, followed by the split-K planes
static size_t op_planes_bytes(int M, int K, int dtype) {
  return dtype == CDSL_BF16 ? ((size_t)2 * M * K * sizeof(bf16) + 255) & ~(size_t)255 : 0;
}

size_t cdsl_op_gemm_workspace(int32_t M, int32_t N, int32_t K, int32_t dtype) {
  if (M <= 0 || N <= 0 || K <= 0) return 0;
  return op_planes_bytes(M, K, dtype) + gemm_workspace_bytes(M, N, K, dtype);
}

int cdsl_op_gemm(const void* A, const void* B, float* C, int32_t M, int32_t N, int32_t K, int32_t dtype,
                 int32_t epilogue, void* workspace, size_t workspace_bytes, void* stream) {
  if (!A || !B || !C) return fail(nullptr, CDSL_EINVAL, "null argument");
  if (dtype != CDSL_F32 && dtype != CDSL_BF16) return fail(nullptr, CDSL_EINVAL, "bad dtype");
  if (epilogue != CDSL_EPI_STORE && epilogue != CDSL_EPI_RESIDUAL) return fail(nullptr, CDSL_EINVAL, "bad epilogue");
  if (gemm_check(M, N, K, dtype) != 0) return fail(nullptr, CDSL_EINVAL, "unsupported shape");
  if (cdsl_op_gemm_workspace(M, N, K, dtype) > workspace_bytes)
    return fail(nullptr, CDSL_EINVAL, "workspace too small");
  if (M == 0) return CDSL_OK;
  hipStream_t st = (hipStream_t)stream;
  GemmOperand op{nullptr, nullptr, (const float*)A};
  const size_t pb = op_planes_bytes(M, K, dtype);
  if (dtype == CDSL_BF16) {
    bf16* hi = (bf16*)workspace;
    bf16* lo = hi + (size_t)M * K;
    hipError_t e = split_planes_launch((const float*)A, hi, lo, (long long)M * K, st);
    if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
    op = GemmOperand{hi, lo, nullptr};
  }
  hipError_t e = gemm_launch(op, B, GemmOut{C, nullptr, nullptr, N}, M, N, K, dtype, epilogue,
                             (char*)workspace + pb, workspace_bytes - pb, st);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  return CDSL_OK;
}

}  // extern "C"

// The workspace of cdsl_op_gemm_static.  In host code `scratch` names a
// host-side stand-in, not the device memory: its device address (one per
// GPU) comes from hipGetSymbolAddress and only that address is passed on.
namespace {
static __device__ __align__(256) unsigned char scratch[CDSL_OP_GEMM_STATIC_BYTES];
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kScratchDevices] = {};
}  // namespace

extern "C" {

int cdsl_op_gemm_static(const void* A, const void* B, float* C, int32_t M, int32_t N, int32_t K, int32_t dtype,
                        int32_t epilogue, void* stream) {
  if (!A || !B || !C) return fail(nullptr, CDSL_EINVAL, "null argument");
  if (dtype != CDSL_F32 && dtype != CDSL_BF16) return fail(nullptr, CDSL_EINVAL, "bad dtype");
  if (gemm_check(M, N, K, dtype) != 0) return fail(nullptr, CDSL_EINVAL, "unsupported shape");
  const size_t need = cdsl_op_gemm_workspace(M, N, K, dtype);
  if (need > CDSL_OP_GEMM_STATIC_BYTES)
    return fail(nullptr, CDSL_ERANGE,
                "shape needs " + std::to_string(need) + " bytes of workspace; the static scratch holds " +
                    std::to_string((size_t)CDSL_OP_GEMM_STATIC_BYTES));
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  if (dev < 0 || dev >= kScratchDevices) return fail(nullptr, CDSL_EDEVICE, "device index beyond the scratch table");
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p) return fail(nullptr, CDSL_EDEVICE, "hipGetSymbolAddress of the scratch array failed");
      g_scratch_dev[dev] = p;
    }
    ws = g_scratch_dev[dev];
  }
  return cdsl_op_gemm(A, B, C, M, N, K, dtype, epilogue, ws, CDSL_OP_GEMM_STATIC_BYTES, stream);
}

int cdsl_op_logit_rows(const float* logits, int32_t M, int32_t V, const int32_t* gather, int32_t kk, float* lp,
                       int32_t* amax, int32_t* topk_ids, float* topk_lp, void* stream) {
  if (!logits || M < 0 || V <= 0 || kk < 0 || kk > 16 || kk > V) return fail(nullptr, CDSL_EINVAL, "bad argument");
  if ((gather && !lp) || (kk > 0 && (!topk_ids || !topk_lp))) return fail(nullptr, CDSL_EINVAL, "missing output");
  LogitArgs la{};
  la.logits = logits;
  la.V = V;
  la.want_lse = (gather || kk > 0) ? 1 : 0;
  la.kk = kk;
  la.amax = amax;
  la.lp = gather ? lp : nullptr;
  la.gather_tok = gather;
  la.topk_ids = topk_ids;
  la.topk_lp = topk_lp;
  hipError_t e = logit_rows_launch(la, M, (hipStream_t)stream);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  return CDSL_OK;
}

}  // extern "C"

int cdsl_op_soft_rows(const float* target_logits, const float* draft_logits, int32_t M, int32_t V, int32_t d,
                      const int32_t* lookaheads, const float* v, float* draft_lp, int32_t* res_ids, float* res_lp,
                      void* stream) {
  if (!target_logits || !draft_logits || !lookaheads || !v || !draft_lp || !res_ids || !res_lp || M < 0 || V <= 0 ||
      d <= 0 || M % d != 0)
    return fail(nullptr, CDSL_EINVAL, "bad argument");
  hipError_t e = soft_rows_launch(target_logits, draft_logits, M, V, d, lookaheads, v, draft_lp, res_ids, res_lp,
                                  (hipStream_t)stream);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  return CDSL_OK;
}

namespace {
struct LmHeadWs {
  size_t planes, mx, se, am, tv, tc, zx, total;
};
LmHeadWs lm_head_ws(int M, int V, int K, int dtype, int kk, int tiles) {
  auto al = [](size_t b) { return (b + 255) & ~(size_t)255; };
  LmHeadWs w{};
  const size_t mt = (size_t)M * tiles;
  w.planes = 0;
  w.mx = al(op_planes_bytes(M, K, dtype));
  w.se = w.mx + al(mt * 4);
  w.am = w.se + al(mt * 4);
  w.tv = w.am + al(mt * 4);
  w.tc = w.tv + al(mt * kk * 4);
  w.zx = w.tc + al(mt * kk * 4);
  w.total = w.zx + al((size_t)M * 4);
  (void)V;
  return w;
}
}  // namespace

size_t cdsl_op_lm_head_rows_workspace(int32_t M, int32_t V, int32_t K, int32_t dtype, int32_t kk) {
  if (M <= 0 || V <= 0 || K <= 0 || kk < 0 || kk > 16) return 0;
  const int tiles = gemm_rowstats_tiles(M, V, K, dtype);
  return tiles > 0 ? lm_head_ws(M, V, K, dtype, kk, tiles).total : 0;
}

int cdsl_op_lm_head_rows(const float* A, const void* B, int32_t M, int32_t V, int32_t K, int32_t dtype,
                         const int32_t* gather, int32_t kk, float* lp, int32_t* amax, int32_t* topk_ids,
                         float* topk_lp, void* workspace, size_t workspace_bytes, void* stream) {
  if (!A || !B || !workspace || M < 0 || V <= 0 || kk < 0 || kk > 16 || kk > V)
    return fail(nullptr, CDSL_EINVAL, "bad argument");
  if ((gather && !lp) || (kk > 0 && (!topk_ids || !topk_lp))) return fail(nullptr, CDSL_EINVAL, "missing output");
  if (dtype != CDSL_F32 && dtype != CDSL_BF16) return fail(nullptr, CDSL_EINVAL, "bad dtype");
  if (gemm_check(M, V, K, dtype) != 0) return fail(nullptr, CDSL_EINVAL, "unsupported shape");
  if (M == 0) return CDSL_OK;
  const int tiles = gemm_rowstats_tiles(M, V, K, dtype);
  if (tiles <= 0) return fail(nullptr, CDSL_EINVAL, "shape not covered by the fused epilogue");
  const LmHeadWs w = lm_head_ws(M, V, K, dtype, kk, tiles);
  if (workspace_bytes < w.total) return fail(nullptr, CDSL_EINVAL, "workspace too small");
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  GemmOperand op{nullptr, nullptr, A};
  if (dtype == CDSL_BF16) {
    bf16* hi = (bf16*)ws;
    bf16* lo = hi + (size_t)M * K;
    hipError_t e = split_planes_launch(A, hi, lo, (long long)M * K, st);
    if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
    op = GemmOperand{hi, lo, nullptr};
  }
  RowStats rs{};
  rs.mx = (float*)(ws + w.mx);
  rs.se = (float*)(ws + w.se);
  rs.am = (int*)(ws + w.am);
  rs.tv = (float*)(ws + w.tv);
  rs.tc = (int*)(ws + w.tc);
  rs.kk = kk;
  rs.zx = (float*)(ws + w.zx);
  rs.gather_tok = gather;
  hipError_t e = gemm_launch(op, B, GemmOut{nullptr, nullptr, nullptr, V}, M, V, K, dtype, kEpiRowStats, nullptr, 0,
                             st, false, nullptr, nullptr, &rs);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  LogitArgs la{};
  la.V = V;
  la.want_lse = (gather || kk > 0) ? 1 : 0;
  la.kk = kk;
  la.amax = amax;
  la.lp = gather ? lp : nullptr;
  la.gather_tok = gather;
  la.topk_ids = topk_ids;
  la.topk_lp = topk_lp;
  e = rowstats_merge_launch(rs, la, M, st);
  if (e != hipSuccess) return fail(nullptr, CDSL_EDEVICE, hipGetErrorString(e));
  return CDSL_OK;
}

