"""The LDS plan checked on the GPU: the debug build of the library
(libvd_debug.so, VD_DEBUG=1) checks every index into a dynamically planned
LDS region against the extent the host planned for it and records a failing
site in a device error word instead of touching memory past the region (see
include/vd_debug.h).  The cases below run the pass, the standalone selection
and compaction, the geometry and both fused decode steps through that build,
over every score form, both dtypes and head_dims 64/128/256, with and without
a running sum, at partial staging, the slot limit, decode argmin and crossing
fill; after each, the error word must be 0.  Results are checked against the
oracle as in the other parity tests (the debug build must compute exactly
what the release build computes)."""
import ctypes
import os

import numpy as np
import pytest
import torch

from paper_2609_23314_amd import build as lib_build
from paper_2609_23314_amd import vd

pytestmark = pytest.mark.gpu

SITES = ["keys", "histograms", "evicted list", "mover list", "staged rows", "fp64 scratch",
         "FastCAOTE rows", "compaction lists"]


@pytest.fixture(scope="module", autouse=True)
def debug_library():
    """The binding pointed at libvd_debug.so for this module, then back."""
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    assert os.path.exists(lib_build.DEBUG_LIB), "build the debug library first"
    saved = (vd._lib, vd.LIB_PATH)
    vd._lib, vd.LIB_PATH = None, lib_build.DEBUG_LIB
    lib = vd.load()
    lib.vd_debug_take_error_word.argtypes = [ctypes.c_void_p]
    lib.vd_debug_take_error_word.restype = ctypes.c_int
    take_error_word()   # start clean
    yield lib
    vd._lib, vd.LIB_PATH = saved


def take_error_word():
    w = ctypes.c_uint32(0)
    st = vd.load().vd_debug_take_error_word(ctypes.byref(w))
    assert st == vd.VD_OK, st
    return w.value


def assert_clean(what):
    w = take_error_word()
    bad = [SITES[b] for b in range(len(SITES)) if w >> b & 1]
    assert w == 0, f"{what}: LDS index outside its planned region at {bad} (word {w:#x})"


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("D", [64, 128, 256])
@pytest.mark.parametrize("variant", ["l2", "dir", "norm", "key_l2", "key_dir", "key_norm"])
def test_pass_plans_hold(orc, dt, D, variant):
    import test_gpu_parity as tp
    dtype = tp.DTYPES[dt]
    # prefill boundary, decode argmin and a no-op unit in one launch
    rep = tp.run_step_case(orc, 3, 2, 2, 1300, D, dtype, n=[1300, 801, 300], N=[1000, 800, 400],
                           variant=variant, seed=40 + D)
    assert_clean(f"pass {dt} d={D} {variant}")
    # running sum with a crossing fill
    tp.run_step_case(orc, 4, 2, 2, 1300, D, dtype, [1300, 801, 300, 650], [1000, 800, 400, 640],
                     variant, seed=60, state="incremental", count=[1000, 800, 200, 600])
    assert_clean(f"pass with state {dt} d={D} {variant}")
    # partial staging (the appended rows do not all fit in LDS at d = 256)
    tp.run_step_case(orc, 2, 1, 2, 600, D, dtype, [600, 450], [400, 300], variant, seed=140,
                     state="incremental", count=[300, 100])
    tp.run_step_case(orc, 2, 1, 2, 600, D, dtype, [600, 450], [400, 300], variant, seed=141)
    assert_clean(f"partial staging {dt} d={D} {variant}")
    assert rep.units > 0


@pytest.mark.parametrize("dt,D,variant", [("bf16", 128, "l2"), ("f32", 256, "dir"),
                                         ("bf16", 64, "norm"), ("bf16", 256, "dir"),
                                         ("f32", 64, "key_norm")])
def test_pass_plans_hold_at_the_slot_limit(orc, dt, D, variant):
    import test_gpu_parity as tp
    C = vd.MAX_CAPACITY
    tp.run_step_case(orc, 3, 1, 1, C, D, tp.DTYPES[dt], [C, C, C], [12288, C - 1, 16000], variant,
                     seed=130 + D, state="incremental", count=[12288, C - 1, 9000])
    assert_clean(f"slot limit {dt} d={D} {variant}")


def test_select_compact_geometry_plans_hold(orc):
    import test_gpu_geometry as tg
    import test_gpu_parity as tp
    tp.test_select_matches_oracle_exactly(orc, ties=True)
    tp.test_select_negative_scores_and_signed_zeros(orc)
    assert_clean("standalone selection")
    for dt in ("bf16", "f32"):
        for D in (64, 128, 256):
            tp.test_compact_matches_oracle_exactly(orc, dt, D)
            tg.test_geometry_matches_oracle(orc, dt, D)
            tg.test_geometry_with_column_sums(orc, dt, D)
    tp.test_compact_with_unbalanced_masks(orc)
    assert_clean("standalone compaction and geometry")


@pytest.mark.parametrize("variant", ["l2", "fastcaote"])
def test_decode_step_plans_hold(orc, variant):
    import test_gpu_attention as ta
    for dt in ("bf16", "f32"):
        for D in (64, 128, 256):
            for G in (1, 2, 4):
                ta.run_case(orc, 3, 2, 2, G, 320, D, ta.DTYPES[dt], [300, 201, 150],
                            [299, 200, 200], seed=500 + D + G, variant=variant)
                assert_clean(f"decode step {variant} {dt} d={D} G={G}")
    # the decode workload's layer shape: 6 splits of 704 rows per unit
    rng = np.random.default_rng(9)
    ta.run_case(orc, 16, 1, 8, 4, 4097, 128, torch.bfloat16, [4097] * 16, [4096] * 16, seed=9,
                sample=np.sort(rng.choice(128, size=4, replace=False)), variant=variant)
    assert_clean(f"decode step {variant}, decode workload layer")
