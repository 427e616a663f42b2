// Internal interface of the projection kernels (gemm.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

namespace cdsl {

enum GemmEpilogue { kEpiStore = 0, kEpiResidual = 1, kEpiSwiGLU = 2 };

// C = A[M,K] * B[N,K]^T with A fp32 (activations).  dtype 1: B bf16
// (weights; A is split into bf16 hi + lo so the product keeps fp32-level
// accuracy); dtype 0: B fp32.
//   kEpiStore:    C fp32 [M, ldc]  = product
//   kEpiResidual: C fp32 [M, ldc] += product
//   kEpiSwiGLU:   (bf16 only) B packs, per group of 32 rows, 16 gate rows
//                 then the 16 matching up rows; C fp32 [M, ldc = N/2]
//                 receives silu(gate) * up.
size_t gemm_workspace_bytes(int M, int N, int K, int dtype);
int gemm_check(int M, int N, int K, int dtype);
// 0: dense bf16 kernel, 1: skinny bf16 kernel, 2: fp32 kernel
int gemm_kind(int M, int N, int K, int dtype);
hipError_t gemm_launch(const void* A, const void* B, void* C, int M, int N, int K, int ldc, int dtype, int epi,
                       void* ws, size_t ws_bytes, hipStream_t st);
hipError_t swiglu_f32_launch(const float* gu, float* act, int M, int F, hipStream_t st);

}  // namespace cdsl
