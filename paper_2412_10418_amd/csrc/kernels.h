// Internal interface of the row-wise kernels (kernels.hip).
#pragma once
#include "common.h"

namespace cdsl {

struct LogitArgs {
  const float* logits;     // [M][ld] (ld = V when 0)
  int V;
  long long ld;
  int want_lse;            // 0: argmax only
  int kk;                  // top-k per row (0..16)
  int* amax;               // argmax destination (RowMap or [M])
  RowMap amax_map;
  float* lp;               // [M] gathered log-prob, or null
  const int* gather_tok;   // token array read through gather_map
  RowMap gather_map;
  int* topk_ids;           // [rows][kk]
  float* topk_lp;
  const int* topk_rows;    // destination row of row m (null: m)
  int* bad;                // set to 1 when a gathered token id lies outside [0, V) (may be null)
};

// Commit records, one per prompt, stage_stride ints each:
//   [0] tokens emitted (-1: invalid beam or count)  [1] catch-up: the last
//   emitted token is fed as one appended row that yields the next heads
//   [2] selected beam  [3] the record holds the next heads
//   [kStageHdr, kStageHdr + tcap)               emitted tokens
//   [kStageHdr + tcap, + kk)                     next head ids
//   [kStageHdr + tcap + kk, + kk)                next head log-probs (float bits)
constexpr int kStageHdr = 4;

// rowinfo (may be null): [M] (block * 16 + slot, position) of each row.
hipError_t embed_launch(const PassDesc& p, const void* emb, float* h, int D, int V, int dtype, hipStream_t st,
                        int2* rowinfo = nullptr);
// S > 0: fold S split planes part[S][rows][D] into x first (written back);
// g == null then only folds.
hipError_t rmsnorm_launch(float* x, const float* g, float* out32, bf16* ohi, bf16* olo, int rows, int D,
                          float eps, int last_only, int R, float* hid, hipStream_t st, const float* part = nullptr,
                          int S = 0);
// S > 1: qkv holds S split planes of the projection (bf16-weight models)
hipError_t rope_kv_launch(const PassDesc& p, const float* qkv, void* qout, const KVPool& pool, int layer,
                          const float* cos_t, const float* sin_t, int H, int Hkv, int hd, int dtype, hipStream_t st,
                          int S = 0);
hipError_t logit_rows_launch(const LogitArgs& a, int M, hipStream_t st);
// logit_rows_launch's outputs (a.logits unused) from the per-tile row
// statistics of the LM-head GEMM (kEpiRowStats); s.kk must equal a.kk.
hipError_t rowstats_merge_launch(const RowStats& s, const LogitArgs& a, int M, hipStream_t st);
// lq, u non-null: soft rejection (speculative sampling) instead of the argmax match
hipError_t beam_scores_launch(int BK, int d, const int* look, const int* y, const float* lp, const float* head_lp,
                              const float* lq, const float* u, int* n_accept, float* scores, hipStream_t st);
// speculative sampling rows: draft log-prob of each row's token and the
// residual draw; see kernels.hip
hipError_t soft_rows_launch(const float* zp, const float* zq, int M, int V, int d, const int* look, const float* v,
                            float* draft_lp, int* res_ids, float* res_lp, hipStream_t st);
hipError_t select_launch(int B, int k, const float* scores, const float* reward, float alpha, int reward_only,
                         const float* first_at, int* beam, hipStream_t st);
hipError_t controller_states_launch(int B, int d, const int* n_accept, const float* reward, double a_t, double r_t,
                                    int b1, int* state, float* first_at, hipStream_t st);
hipError_t reward_keywords_launch(int B, int k, int d, const int* gen, int gen_stride, const int* gen_len,
                                  const int* look, const int* upto, int head, const int* kws, int n_kw, int normalize,
                                  float* reward, hipStream_t st);
hipError_t reward_linear_launch(int BK, const float* hidden, const float* w, int D, float* reward, hipStream_t st);
// the commit kernels write records only; commit_apply_launch carries them out
hipError_t commit_heads_launch(int B, int k, int d, const int* look, const int* beam, const int* mask, int* stage,
                               int stage_stride, hipStream_t st);
hipError_t commit_tokens_launch(int B, const int* tokens, const int* mask, int V, int* stage, int stage_stride,
                                hipStream_t st);
hipError_t withdraw_launch(int B, const int* cnt, int* Lp, int* gen_len, hipStream_t st);
hipError_t commit_launch(int B, int k, int d, int kk, const int* look, const int* beam, const int* n_accept,
                         const int* rtk_ids, const float* rtk_lp, const int* res_ids, const float* res_lp, int* stage,
                         int stage_stride, int tcap, hipStream_t st);
hipError_t commit_prefix_launch(int B, int d, int kk, const int* look, const int* n_accept, const int* rtk_ids,
                                const float* rtk_lp, int* stage, int stage_stride, int tcap, hipStream_t st);
hipError_t commit_apply_launch(int B, const int* stage, int stage_stride, int tcap, int kk, int* gen, int gen_stride,
                               int* gen_len, int* next_beams, float* next_head_lp, int* catch_tok, hipStream_t st);
hipError_t prefix_tail_launch(int B, const int* gen, int gen_stride, const int* gen_len, const int* ptail,
                              const int* Lp, int* Lm1, int* look, int look_stride, hipStream_t st);
hipError_t last_tokens_launch(int B, const int* tokens, int L, int* out, hipStream_t st);
hipError_t promote_launch(int B, int k, const KVPool& pool, int n_layers, const int* stage, int stage_stride, int dlim,
                          int soff, const int* Lp, const int* ptable, int ptable_stride, const int* stable,
                          int s_stride_b, int s_stride_i, int dtype, hipStream_t st);
hipError_t advance_launch(int B, const int* stage, int stage_stride, int dlim, int* Lp, hipStream_t st);
hipError_t add_launch(int n, const int* ids, int* v, int delta, hipStream_t st);
hipError_t fill_int_launch(int* p, int v, long long n, hipStream_t st);
hipError_t heads_to_lookaheads_launch(int BK, int d, const int* beams, int* look, hipStream_t st);

}  // namespace cdsl
