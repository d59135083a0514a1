"""The benchmark-support library (measured MFMA and HBM-read ceilings quoted by bench.py)."""
import ctypes
import os

import pytest

LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2605_07325_amd",
                   "libcsr_bench.so")


def _fn():
    lib = ctypes.CDLL(LIB)
    fn = lib.csr_bench_mfma_peak
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_int, ctypes.c_int] + [ctypes.POINTER(ctypes.c_double)] * 3
    return fn


def test_loads_and_rejects_bad_arguments_before_any_device_call():
    fn = _fn()
    d = [ctypes.c_double() for _ in range(3)]
    assert fn(0, 100, *map(ctypes.byref, d)) != 0
    assert fn(4, 0, *map(ctypes.byref, d)) != 0


@pytest.mark.gpu
def test_measured_ceiling_is_plausible():
    import torch

    torch.cuda.init()
    fn = _fn()
    ms, fl, ghz = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    wgs = torch.cuda.get_device_properties(0).multi_processor_count
    assert fn(wgs, 4000, ctypes.byref(ms), ctypes.byref(fl), ctypes.byref(ghz)) == 0
    tflops = fl.value / 1e12
    print(f"measured MFMA ceiling {tflops:.0f} TFLOP/s at {ghz.value:.2f} GHz ({ms.value:.3f} ms)", flush=True)
    # dense bf16: at most the published 2.5 PFLOP/s (2.4 GHz); the clock is a shader clock in GHz
    assert 500 < tflops < 2600
    assert 0.5 < ghz.value < 2.6
    # the loop issues one 32x32x16 MFMA per 32 clocks per SIMD at most
    assert tflops <= wgs * 4 * 32768 / 32 * ghz.value * 1e9 / 1e12 * 1.02


def _hbm():
    lib = ctypes.CDLL(LIB)
    fn = lib.csr_bench_hbm_read
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_size_t, ctypes.c_int, ctypes.c_int, ctypes.c_int] + [ctypes.POINTER(ctypes.c_double)] * 2
    return fn


def test_hbm_read_rejects_bad_arguments_before_any_device_call():
    fn = _hbm()
    d = [ctypes.c_double() for _ in range(2)]
    assert fn(0, 3, 10, 256, *map(ctypes.byref, d)) != 0      # no bytes
    assert fn(1000, 3, 10, 256, *map(ctypes.byref, d)) != 0   # not a multiple of 16
    assert fn(1 << 20, 0, 10, 256, *map(ctypes.byref, d)) != 0
    assert fn(1 << 20, 3, 0, 256, *map(ctypes.byref, d)) != 0
    assert fn(1 << 20, 3, 10, 0, *map(ctypes.byref, d)) != 0


@pytest.mark.gpu
def test_measured_hbm_read_is_plausible():
    import torch

    torch.cuda.init()
    fn = _hbm()
    ms, gbs = ctypes.c_double(), ctypes.c_double()
    wgs = torch.cuda.get_device_properties(0).multi_processor_count
    assert fn(251658240, 3, 20, wgs, ctypes.byref(ms), ctypes.byref(gbs)) == 0
    print(f"measured HBM read: {gbs.value:.0f} GB/s ({ms.value * 1e3:.1f} us per 252 MB)", flush=True)
    assert 1000 < gbs.value < 8000   # below the published 8 TB/s


def test_clock_detail_groups_a_decoded_table():
    # bench.py's breakdown of one clock-hooked launch, on a hand-made table: two kv heads on two
    # XCDs, two splits each; head 1 streams its tiles at twice the time per tile
    import sys

    import numpy as np

    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench

    t = {"start_us": np.array([0.0, 0.0, 1.0, 1.0]), "end_us": np.array([10.0, 12.0, 21.0, 25.0]),
         "tb": np.array([0, 10, 0, 10]), "te": np.array([10, 20, 10, 22]),
         "kv_head": np.array([0, 0, 1, 1]), "split": np.array([0, 1, 0, 1]), "xcd": np.array([0, 0, 1, 1])}
    d = bench.clock_detail(t)
    assert d["by_kv_head"]["0"] == {"n": 2, "end_median_us": 11.0, "us_per_tile_median": 1.1}
    assert d["by_kv_head"]["1"] == {"n": 2, "end_median_us": 23.0, "us_per_tile_median": 2.0}
    assert d["by_split"]["1"]["end_median_us"] == 18.5
    assert d["by_xcd"]["1"]["us_per_tile_median"] == 2.0
    many = dict(t, split=np.arange(4) * 9)
    assert bench.clock_detail(many)["by_split"] is not None
    many["split"] = np.arange(4) + 20
    t20 = {k: np.concatenate([v] * 5) for k, v in many.items()}
    t20["split"] = np.arange(20)
    assert bench.clock_detail(t20)["by_split"] is None  # more than 16 splits: left out
