/*
 * cdsl_ops.h -- kernel-level entry points of the CDSL library, exported so
 * that single kernels can be checked in isolation.  They run exactly the
 * kernels that cdsl_rollout / cdsl_verify launch, on caller buffers.
 * All pointers are device pointers owned by the caller; calls are
 * asynchronous on `stream` (a hipStream_t, NULL = default stream) and return
 * CDSL_OK or a negative CDSL_E* code (see cdsl.h).  No call allocates.
 */
#ifndef CDSL_OPS_H
#define CDSL_OPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  CDSL_EPI_STORE = 0,     /* C[M,N] (fp32)  = A * B^T                 */
  CDSL_EPI_RESIDUAL = 1   /* C[M,N] (fp32) += A * B^T  (residual add)   */
};

/* Bytes of workspace cdsl_op_gemm needs for this shape: for bf16 weights
 * the hi / lo planes of A, then the fp32 partial planes of a split K; 0 if
 * none. */
size_t cdsl_op_gemm_workspace(int32_t M, int32_t N, int32_t K, int32_t dtype);

/* Dense projection C = A[M,K] * B[N,K]^T with fp32 accumulation: the
 * contraction of every linear layer of the decoders (q/k/v/o, gate/up/down,
 * LM head).  A (activations) is fp32; B (weights) is bf16 (dtype
 * CDSL_BF16: A is split into bf16 hi + lo halves, two MFMA products, so the
 * result keeps fp32-level accuracy) or fp32 (CDSL_F32); C is fp32.  K must
 * be a multiple of 32 for bf16 (16 for fp32).  The workspace must hold
 * cdsl_op_gemm_workspace(M, N, K, dtype) bytes; every call writes what it
 * reads there, so it needs no initial contents.  Errors: EINVAL. */
int cdsl_op_gemm(const void* A, const void* B, float* C, int32_t M, int32_t N,
                 int32_t K, int32_t dtype, int32_t epilogue, void* workspace,
                 size_t workspace_bytes, void* stream);

/* cdsl_op_gemm for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid allocation): the
 * same kernels, with the workspace taken from a scratch array the library
 * holds in device memory, CDSL_OP_GEMM_STATIC_BYTES (64 MiB) on each GPU it
 * runs on, until the process ends.  No allocation happens in the call.
 * Shapes whose cdsl_op_gemm_workspace exceeds that size are refused with
 * ERANGE (for bf16 weights: 4 M K bytes of planes plus 4 S M N bytes of S
 * K-split planes; e.g. M = 800 at N = K = 4096 needs 52 MB).  Every call on
 * one GPU shares that GPU's array: calls that overlap on one GPU (two
 * streams, two threads) race and must be serialised by the caller.  The
 * first call on a device looks up that device's copy of the array.  Errors:
 * EINVAL, ERANGE, EDEVICE. */
#define CDSL_OP_GEMM_STATIC_BYTES (64u << 20)
int cdsl_op_gemm_static(const void* A, const void* B, float* C, int32_t M,
                        int32_t N, int32_t K, int32_t dtype, int32_t epilogue,
                        void* stream);

/* Row statistics of logits[M, V] (fp32), one pass per row, never writing
 * probabilities: for row m,
 *   lp[m]        = logits[m, gather[m]] - logsumexp(logits[m, :])
 *                  (skipped, lp untouched, if gather is NULL)
 *   amax[m]      = argmax (lowest id on ties)
 *   topk_ids[m, 0..kk), topk_lp[m, 0..kk): the kk largest entries, value
 *                  descending then id ascending, as log-probs
 *                  (skipped if kk == 0; kk <= 16)
 * This is the log-softmax + gather + argmax + top-k step of verification.
 * Errors: EINVAL. */
int cdsl_op_logit_rows(const float* logits, int32_t M, int32_t V,
                       const int32_t* gather, int32_t kk, float* lp,
                       int32_t* amax, int32_t* topk_ids, float* topk_lp,
                       void* stream);

/* The LM head with its row statistics fused into the GEMM epilogue: the
 * same outputs as cdsl_op_logit_rows on logits = A[M,K] * B[V,K]^T
 * (cdsl_op_gemm's operands and dtypes; argmax and top-k ids identical, the
 * log-probs equal up to the summation order of the logsumexp), without the
 * logits ever reaching memory.  Each column tile of the GEMM reduces its
 * rows to (max, sum of exp, argmax, its kk best, the gathered value); one
 * workgroup per row folds the tiles.  amax may be NULL.  The workspace must
 * hold cdsl_op_lm_head_rows_workspace(M, V, K, dtype, kk) bytes (0 means
 * the shape is not covered).  Errors: EINVAL. */
size_t cdsl_op_lm_head_rows_workspace(int32_t M, int32_t V, int32_t K,
                                      int32_t dtype, int32_t kk);
int cdsl_op_lm_head_rows(const float* A, const void* B, int32_t M, int32_t V,
                         int32_t K, int32_t dtype, const int32_t* gather,
                         int32_t kk, float* lp, int32_t* amax,
                         int32_t* topk_ids, float* topk_lp, void* workspace,
                         size_t workspace_bytes, void* stream);

/* Speculative sampling rows (Sec. 3.2.2) over target_logits[M, V] (p) and
 * draft_logits[M, V] (q), fp32, rows ordered (row group g, position j) with
 * M = G * d; the row's draft token is x = lookaheads[g, j + 1] (an int32
 * [G, d + 1] array, as cdsl_rollout writes it).  For row m = g * d + j:
 *   draft_lp[m] = log q(x)
 *   res_ids[m]  = the draw at v[m] in [0, 1) from w = max(0, p - q) / Z:
 *                 the smallest token t with w_0 + ... + w_t > v[m] * Z
 *                 (argmax p, lowest id, when Z = 0)
 *   res_lp[m]   = log p(res_ids[m]).
 * This is the kernel cdsl_verify_soft runs after the verification pass.
 * Errors: EINVAL (null pointers, M not a multiple of d). */
int cdsl_op_soft_rows(const float* target_logits, const float* draft_logits,
                      int32_t M, int32_t V, int32_t d, const int32_t* lookaheads,
                      const float* v, float* draft_lp, int32_t* res_ids,
                      float* res_lp, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* CDSL_OPS_H */
