"""The measured ceilings (include/mure_peaks.h) on the GPU.

The copy must move every byte of ragged sizes and nothing past them.  The
MFMA loops are pinned to closed forms of their lane sums.  Every operand of a
loop is a power of two, so each MFMA adds a fixed amount to each accumulator
element.  The accumulators stay small (below 1/4, multiples of 2^-25 or
2^-20), where every such addition is exact.  Larger ones lost addends: the
fp32 MFMA dropped 2^-19 added onto 8, and bf16 lane sums started near 1/4
came out up to 0.04 short after 100 steps.  The lane sum therefore fixes how
many MFMAs ran, which is the count the reported rate divides by."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2607_18582_amd import peaks as PK

pytestmark = pytest.mark.gpu

VENDOR = {"bf16": 2500.0, "f32": 157.3}   # MI355X dense MFMA, TFLOP/s


def _stream():
    return C.c_void_p(torch.cuda.current_stream(0).cuda_stream)


@pytest.mark.parametrize("nvec", [1, 1023, 1025, 12345, 65536])
def test_peak_copy_moves_exactly_the_requested_bytes(nvec):
    lib = PK.load_peaks_library()
    nbytes = 16 * nvec
    print(f"peak_copy {nbytes} bytes", flush=True)
    src = torch.randint(0, 256, (nbytes + 256,), dtype=torch.uint8, device="cuda:0")
    dst = torch.zeros_like(src)
    out = C.c_double()
    st = lib.mure_peak_copy(C.c_void_p(src.data_ptr()), C.c_void_p(dst.data_ptr()), nbytes, 2,
                            _stream(), C.byref(out))
    torch.cuda.synchronize()
    assert st == 0 and out.value > 0
    assert torch.equal(dst[:nbytes], src[:nbytes])
    assert int(dst[nbytes:].count_nonzero()) == 0


def test_peak_mfma_f32_lane_sums():
    # 8 chains of v4f; element 0 starts at (tid + j) / 1024, elements 1-3 at
    # 0; each 16x16x4 MFMA adds 4 * 2^-10 * 2^-11 = 2^-19 to every element
    lib = PK.load_peaks_library()
    blocks, iters = 256, 1000
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda:0")
    out = C.c_double()
    print("peak_mfma f32", flush=True)
    st = lib.mure_peak_mfma(0, blocks, iters, 1, C.c_void_p(sink.data_ptr()), _stream(), C.byref(out))
    torch.cuda.synchronize()
    assert st == 0 and out.value > 0
    s = sink.cpu().numpy().reshape(blocks, 256).astype(np.float64)
    tid = np.arange(256, dtype=np.float64)
    exact = (8 * tid + 28) * 2.0 ** -10 + 32 * iters * 2.0 ** -19
    # one MFMA more or less per chain moves a lane's sum by 32 * 2^-19 = 6e-5
    assert np.abs(s - exact).max() < 1e-5


def test_peak_mfma_bf16_lane_sums():
    # 4 chains of v16f starting at 0; each 32x32x16 MFMA of chain q adds
    # 2^-q * 2 * sum_e a_e b_e = 2^-q * 17 * 2^-17 to every element
    # (a, b in {2^-8, 2^-9})
    lib = PK.load_peaks_library()
    blocks, iters = 256, 100
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device="cuda:0")
    out = C.c_double()
    print("peak_mfma bf16", flush=True)
    st = lib.mure_peak_mfma(1, blocks, iters, 1, C.c_void_p(sink.data_ptr()), _stream(), C.byref(out))
    torch.cuda.synchronize()
    assert st == 0 and out.value > 0
    s = sink.cpu().numpy().reshape(blocks, 256).astype(np.float64)
    exact = 16 * iters * 17 * 2.0 ** -17 * (1 + 1 / 2 + 1 / 4 + 1 / 8)
    # one MFMA more or less in chain 3 moves a lane's sum by 16 * 17 * 2^-20 = 2.6e-4
    assert np.abs(s - exact).max() < 1e-5


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_peak_mfma_rate_within_the_vendor_peak(dtype):
    print(f"peak_mfma rate {dtype}", flush=True)
    r = PK.peak_mfma_tflops(dtype, waves_per_simd=3, rounds=2, iters=2000, reps=2)
    assert 0.2 * VENDOR[dtype] < r <= 1.02 * VENDOR[dtype], r


def test_peak_copy_rate_within_the_vendor_peak():
    print("peak_copy rate 1 GiB", flush=True)
    r = PK.peak_copy_gbs(copy_mib=1024, reps=3)
    assert 1000.0 < r <= 8000.0 * 1.02, r
