"""CPU checks of the C-ABI library: it loads, and it exports every entry
point the public headers declare (no compute calls: there may be no GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2412_10418_amd", "_lib", "libcdsl.so")


def declared():
    names = []
    for h in ("cdsl.h", "cdsl_ops.h"):
        src = open(os.path.join(ROOT, "include", h)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names += re.findall(r"\b(cdsl_[a-z_]+)\s*\(", src)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2412_10418_amd import build
        build.build(verbose=False)
    return ctypes.CDLL(LIB)


def test_headers_declare_the_step_calls():
    d = declared()
    for name in ("cdsl_init", "cdsl_prefill", "cdsl_rollout", "cdsl_verify", "cdsl_select",
                 "cdsl_commit", "cdsl_reward_keywords", "cdsl_reward_linear", "cdsl_destroy",
                 "cdsl_last_error", "cdsl_op_gemm", "cdsl_op_logit_rows"):
        assert name in d


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    from paper_2412_10418_amd import binding
    assert sorted(binding.EXPORTS) == declared()


def test_exports_are_c_linkage(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    syms = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for n in declared():
        assert n in syms, n          # unmangled


def test_error_paths_without_device(lib):
    """Argument checks happen on the host before any device work."""
    from paper_2412_10418_amd import binding
    L = binding.lib()
    assert L.cdsl_init(None, None, None, None, None) == binding.CDSL_EINVAL
    assert b"null" in L.cdsl_last_error(None)
    assert L.cdsl_destroy(None) == binding.CDSL_OK
    assert L.cdsl_rollout(None, None, None, 1, 1, None) == binding.CDSL_EINVAL
    assert L.cdsl_rollout_with(None, None, None, 1, 1, 0, None) == binding.CDSL_EINVAL
    assert L.cdsl_verify_kk(None, None, None, 1, 1, 1, None, None, None, None, None, None, None,
                            None) == binding.CDSL_EINVAL
    assert L.cdsl_commit_kk(None, None, None, None, None, None, None, 1, 1, 1, None, None, None,
                            None) == binding.CDSL_EINVAL
    assert L.cdsl_commit_heads(None, None, None, None, 1, 1, 1, None, None, None, None) == binding.CDSL_EINVAL
    assert L.cdsl_reward_keywords_upto(None, None, None, 1, 1, None, None, 1, 0, None) == binding.CDSL_EINVAL
    assert L.cdsl_select_first(None, None, None, 1, 1, None) == binding.CDSL_EINVAL
    assert L.cdsl_rollout_keep(None, None, None, 1, 1, None, None) == binding.CDSL_EINVAL
    assert L.cdsl_verify_soft(None, None, None, 1, 1, 1, *([None] * 14)) == binding.CDSL_EINVAL
    assert L.cdsl_commit_soft(None, None, None, None, None, None, None, None, None, 1, 1, 1, None, None, None,
                              None) == binding.CDSL_EINVAL
    assert L.cdsl_op_soft_rows(None, None, 1, 1, 1, None, None, None, None, None, None) == binding.CDSL_EINVAL
    assert L.cdsl_op_lm_head_rows(None, None, 1, 1, 1, 1, None, 0, None, None, None, None, None, 0,
                                  None) == binding.CDSL_EINVAL
    assert L.cdsl_op_lm_head_rows_workspace(80, 32000, 2048, binding.CDSL_BF16, 5) > 0
    assert L.cdsl_op_lm_head_rows_workspace(0, 32000, 2048, binding.CDSL_BF16, 5) == 0
    assert L.cdsl_controller_states(None, None, None, 1, 1, 0.5, 0.5, 1, None, None) == binding.CDSL_EINVAL
    assert L.cdsl_op_logit_rows(None, 1, 1, None, 0, None, None, None, None, None) == binding.CDSL_EINVAL
    assert L.cdsl_op_gemm_workspace(80, 3072, 2048, binding.CDSL_BF16) > 0
    assert L.cdsl_op_gemm_workspace(0, 3072, 2048, binding.CDSL_BF16) == 0
