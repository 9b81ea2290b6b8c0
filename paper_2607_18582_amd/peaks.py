"""Thin ctypes binding of libmure_peaks.so (``include/mure_peaks.h``): the
HBM copy rate and the MFMA rates that this GPU sustains, the ceilings that
kernel times are reported against next to the vendor's figures.

torch supplies the device buffers and the stream; the copy and the MFMA loops
run in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict

HERE = os.path.dirname(os.path.abspath(__file__))
PEAKS_LIB_PATH = os.path.join(HERE, "libmure_peaks.so")
PEAKS_EXPORTED = ["mure_peak_copy", "mure_peak_mfma"]

_lib = None


def load_peaks_library(path: str = PEAKS_LIB_PATH) -> C.CDLL:
    """Load libmure_peaks.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it first (python -m paper_2607_18582_amd.build)")
    try:
        import torch  # noqa: F401  (one HIP runtime per process: torch's)
    except ImportError:
        pass
    lib = C.CDLL(path)
    P, D = C.c_void_p, C.POINTER(C.c_double)
    lib.mure_peak_copy.restype = C.c_int
    lib.mure_peak_copy.argtypes = [P, P, C.c_int64, C.c_int, P, D]
    lib.mure_peak_mfma.restype = C.c_int
    lib.mure_peak_mfma.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, P, P, D]
    _lib = lib
    return lib


def _check(st: int, what: str) -> None:
    if st != 0:
        raise RuntimeError(f"{what} failed with status {st}")


def peak_copy_gbs(copy_mib: int = 1024, reps: int = 10, device: int = 0) -> float:
    """Best STREAM-copy rate over two device buffers of ``copy_mib`` MiB each,
    counting read and written bytes (GB/s)."""
    import torch
    lib = load_peaks_library()
    n = int(copy_mib) << 20
    src = torch.randint(0, 256, (n,), dtype=torch.uint8, device=f"cuda:{device}")
    dst = torch.zeros_like(src)
    s = torch.cuda.current_stream(device).cuda_stream
    out = C.c_double()
    _check(lib.mure_peak_copy(C.c_void_p(src.data_ptr()), C.c_void_p(dst.data_ptr()), n, reps,
                              C.c_void_p(s), C.byref(out)), "mure_peak_copy")
    if not torch.equal(src[:4096], dst[:4096]) or not torch.equal(src[-4096:], dst[-4096:]):
        raise RuntimeError("mure_peak_copy: destination differs from the source")
    return out.value


def peak_mfma_tflops(dtype: str, waves_per_simd: int = 3, rounds: int = 4, iters: int = 20000,
                     reps: int = 5, device: int = 0) -> float:
    """Best rate of the register-only MFMA loop (``dtype`` 'bf16' or 'f32'),
    with ``waves_per_simd`` x ``rounds`` blocks of four wavefronts per CU."""
    import torch
    lib = load_peaks_library()
    cus = torch.cuda.get_device_properties(device).multi_processor_count
    blocks = cus * waves_per_simd * rounds
    sink = torch.empty(blocks * 256, dtype=torch.float32, device=f"cuda:{device}")
    s = torch.cuda.current_stream(device).cuda_stream
    out = C.c_double()
    _check(lib.mure_peak_mfma(1 if dtype == "bf16" else 0, blocks, iters, reps,
                              C.c_void_p(sink.data_ptr()), C.c_void_p(s), C.byref(out)),
           "mure_peak_mfma")
    if not bool(torch.isfinite(sink).all()):
        raise RuntimeError("mure_peak_mfma: non-finite sums")
    return out.value


def measure_peaks(device: int = 0) -> Dict[str, float]:
    """The three ceilings: HBM copy (GB/s), bf16 and fp32 MFMA (TFLOP/s)."""
    return {"hbm_copy_gbs": peak_copy_gbs(device=device),
            "mfma_bf16_tflops": peak_mfma_tflops("bf16", device=device),
            "mfma_f32_tflops": peak_mfma_tflops("f32", waves_per_simd=4, device=device)}
