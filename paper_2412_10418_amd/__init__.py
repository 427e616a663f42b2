"""MI355X-native CDSL lookahead step: HIP kernels behind a C ABI
(``include/cdsl.h``) with a thin ctypes binding.

    from paper_2412_10418_amd.binding import Context   # the C calls
    from paper_2412_10418_amd.engine import Engine     # a full step
"""
__all__ = ["binding", "engine", "build"]
