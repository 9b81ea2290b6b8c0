"""The measured-ceiling library (include/mure_peaks.h) on the host: it loads,
exports what its header declares, and refuses invalid arguments before any
device work."""
import ctypes as C
import os
import re

import pytest

from paper_2607_18582_amd import peaks as PK

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_peaks_library_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "mure_peaks.h")) as f:
        declared = sorted(set(re.findall(r"\b(mure_[a-z_]+)\s*\(", f.read())))
    assert declared == sorted(PK.PEAKS_EXPORTED)
    lib = PK.load_peaks_library()
    for name in declared:
        assert hasattr(lib, name), name


@pytest.mark.parametrize("src,dst,nbytes,reps", [
    (16, 4096, 0, 1),            # empty
    (16, 4096, 24, 1),           # not a multiple of 16
    (8, 4096, 32, 1),            # misaligned source
    (16, 4096, 32, 0),           # no repetitions
    (16, 4096, 32, 1001),        # too many repetitions
    (16, 32, 32, 1),             # overlapping buffers
    (0, 4096, 32, 1),            # null source
])
def test_peak_copy_rejects_invalid_arguments(src, dst, nbytes, reps):
    lib = PK.load_peaks_library()
    out = C.c_double(-1.0)
    st = lib.mure_peak_copy(C.c_void_p(src), C.c_void_p(dst), nbytes, reps, None, C.byref(out))
    assert st == -1 and out.value == -1.0


@pytest.mark.parametrize("dtype,blocks,iters,reps,sink", [
    (2, 1, 1, 1, 4096),          # no such dtype
    (1, 0, 1, 1, 4096),          # no blocks
    (1, 65537, 1, 1, 4096),      # too many blocks
    (0, 1, 0, 1, 4096),          # no rounds
    (0, 1, 1, 101, 4096),        # too many repetitions
    (1, 1, 1, 1, 0),             # null sink
])
def test_peak_mfma_rejects_invalid_arguments(dtype, blocks, iters, reps, sink):
    lib = PK.load_peaks_library()
    out = C.c_double(-1.0)
    st = lib.mure_peak_mfma(dtype, blocks, iters, reps, C.c_void_p(sink), None, C.byref(out))
    assert st == -1 and out.value == -1.0
