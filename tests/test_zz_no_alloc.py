"""cdsl_op_gemm_static (the projection for callers that cannot allocate)
through the C ABI: two calls in a row, the second smaller, each equal to
cdsl_op_gemm with a caller workspace (the same kernels, so bitwise) and
within fp32 accuracy of float64; a shape whose workspace exceeds the static
scratch is refused."""
import ctypes

import numpy as np
import pytest
import torch

import cdsl_inputs as ci

pytestmark = pytest.mark.gpu


def _operands(M, N, K, seed):
    rng = np.random.default_rng([seed, M, N, K])
    a = rng.uniform(-1, 1, (M, K)).astype(np.float32)
    b = ci.round_to_bf16(rng.uniform(-1, 1, (N, K)).astype(np.float32))
    tb = torch.from_numpy(ci.f32_to_bf16_bits(b).view(np.int16)).cuda().view(torch.bfloat16)
    return a, b, torch.from_numpy(a).cuda(), tb


def _static(ta, tb, M, N, K):
    from paper_2412_10418_amd import binding as bd
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    rc = bd.lib().cdsl_op_gemm_static(ta.data_ptr(), tb.data_ptr(), C.data_ptr(), M, N, K, bd.CDSL_BF16,
                                      bd.CDSL_EPI_STORE, torch.cuda.current_stream().cuda_stream)
    return rc, C


def test_static_scratch_gemm_matches_the_workspace_entry_point():
    from paper_2412_10418_amd import binding as bd
    # the verification's o-projection (K split over 3 planes: 52 MB of
    # workspace), then a smaller rollout-sized call on the same scratch
    for M, N, K in [(800, 4096, 4096), (80, 3072, 2048)]:
        print(f"static-scratch gemm {M}x{N}x{K}", flush=True)
        assert bd.lib().cdsl_op_gemm_workspace(M, N, K, bd.CDSL_BF16) <= (64 << 20)
        a, b, ta, tb = _operands(M, N, K, 31)
        ref = bd.cdsl_op_gemm(ta, tb)
        rc, got = _static(ta, tb, M, N, K)
        assert rc == bd.CDSL_OK, bd.lib().cdsl_last_error(None)
        torch.cuda.synchronize()
        assert torch.equal(got, ref)
        exact = a.astype(np.float64) @ b.astype(np.float64).T
        err = np.max(np.abs(got.cpu().numpy() - exact)) / max(1.0, np.max(np.abs(exact)))
        assert err < 5e-6, err


def test_static_scratch_refuses_a_shape_beyond_its_size():
    from paper_2412_10418_amd import binding as bd
    M, N, K = 4160, 4096, 4096        # 65 MiB of hi / lo planes alone
    assert bd.lib().cdsl_op_gemm_workspace(M, N, K, bd.CDSL_BF16) > (64 << 20)
    a, b, ta, tb = _operands(M, N, K, 32)
    rc, got = _static(ta, tb, M, N, K)
    assert rc == bd.CDSL_ERANGE
    assert b"static scratch" in bd.lib().cdsl_last_error(None)
    assert torch.isnan(got).all()
