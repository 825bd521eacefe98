"""CPU checks of the C-ABI library: it loads, exports every entry point that
include/gsc.h declares, and its host-side validation rejects bad arguments
before any HIP call (so these run without a GPU).  Also checks the product's
region lists against the oracle's, since the two are written independently."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle.gsc_oracle as O
from paper_1904_08755_amd import gsc, regions

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gsc.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gsc_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(gsc.LIB_PATH):
        pytest.skip("libgsc.so not built")
    return gsc.lib()


def test_header_symbols_exported(L):
    syms = declared_symbols()
    assert len(syms) >= 12
    for s in syms:
        assert hasattr(L, s), s
    assert sorted(gsc.exported_symbols()) == syms


def test_abi_version(L):
    assert L.gsc_abi_version() == 1


def test_size_queries(L):
    assert L.gsc_table_bytes(0) == 256 + 64 * 16
    assert L.gsc_table_bytes(16) == 256 + 64 * 16
    assert L.gsc_table_bytes(17) == 256 + 128 * 16
    assert L.gsc_table_bytes(300_000) == 256 + (1 << 21) * 16
    assert L.gsc_table_bytes(-1) == 0
    assert L.gsc_kmap_groups(0) == 0
    assert L.gsc_kmap_groups(1) == 1
    assert L.gsc_kmap_groups(64) == 1
    assert L.gsc_kmap_groups(65) == 2
    assert L.gsc_kmap_ws_bytes(1000, 27, 3) > 27 * 16 * 4
    assert L.gsc_kmap_ws_bytes(1000, 0, 3) == 0
    assert L.gsc_stride_ws_bytes(1000) >= 8000
    assert L.gsc_conv_bwd_ws_bytes(100000, 32, 32, 27) >= 27 * 32 * 32 * 4
    assert L.gsc_conv_bwd_ws_bytes(10, 0, 32, 27) == 0


def _err(L):
    return L.gsc_last_error().decode()


def test_coords_build_validation(L):
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    assert L.gsc_coords_build(fake, 10, 0, fake, 1 << 20, None) == gsc.GSC_EINVAL
    assert "D=0" in _err(L)
    assert L.gsc_coords_build(fake, 10, 8, fake, 1 << 20, None) == gsc.GSC_EINVAL
    assert L.gsc_coords_build(fake, -1, 3, fake, 1 << 20, None) == gsc.GSC_EINVAL
    assert L.gsc_coords_build(None, 10, 3, fake, 1 << 20, None) == gsc.GSC_EINVAL
    assert L.gsc_coords_build(fake, 10, 3, None, 1 << 20, None) == gsc.GSC_EINVAL
    need = L.gsc_table_bytes(1000)
    assert L.gsc_coords_build(fake, 1000, 3, fake, need - 1, None) == gsc.GSC_ESHORT
    assert str(need) in _err(L)


def test_coords_stride_validation(L):
    fake = ctypes.c_void_p(0x1000)
    n_out = ctypes.c_int64(0)
    st = (ctypes.c_int32 * 3)(2, 2, 0)
    assert L.gsc_coords_stride(fake, 100, 3, st, fake, ctypes.byref(n_out), fake, 1 << 20, fake, 1 << 20,
                               None) == gsc.GSC_EINVAL
    st = (ctypes.c_int32 * 3)(2, 2, 2)
    assert L.gsc_coords_stride(fake, 100, 3, st, fake, ctypes.byref(n_out), fake, 10, fake, 1 << 20,
                               None) == gsc.GSC_ESHORT
    assert L.gsc_coords_stride(fake, 100, 3, st, fake, ctypes.byref(n_out), fake, 1 << 20, fake, 8,
                               None) == gsc.GSC_ESHORT
    assert L.gsc_coords_stride(fake, 100, 3, None, fake, ctypes.byref(n_out), fake, 1 << 20, fake, 1 << 20,
                               None) == gsc.GSC_EINVAL


def test_kernel_map_validation(L):
    fake = ctypes.c_void_p(0x1000)
    n = ctypes.c_int64(0)
    offs = (ctypes.c_int32 * 3)(0, 0, 0)
    ts_bad = (ctypes.c_int32 * 3)(1, 0, 1)
    ws = L.gsc_kmap_ws_bytes(100, 1, 3)
    args = lambda K, ts, wsb, cap=10: (fake, fake, 100, 3, offs, K, ts, fake, fake, cap, fake, fake, None,
                                       ctypes.byref(n), fake, wsb, None)
    assert L.gsc_kernel_map(*args(0, None, ws)) == gsc.GSC_EINVAL
    assert L.gsc_kernel_map(*args(1, ts_bad, ws)) == gsc.GSC_EINVAL
    assert L.gsc_kernel_map(*args(1, None, ws - 1)) == gsc.GSC_ESHORT
    assert L.gsc_kernel_map(*args(1, None, ws, cap=-1)) == gsc.GSC_EINVAL
    # asynchronous mode (n_pairs NULL) needs cap_pairs >= K * n_out and K * D <= 768
    a = list(args(1, None, ws, cap=99))
    a[13] = None
    assert L.gsc_kernel_map(*a) == gsc.GSC_ESHORT and "asynchronous" in _err(L)
    K = 300
    offs300 = (ctypes.c_int32 * (3 * K))()
    ws300 = L.gsc_kmap_ws_bytes(100, K, 3)
    a = [fake, fake, 100, 3, offs300, K, None, fake, fake, K * 100, fake, fake, None, None, fake, ws300, None]
    assert L.gsc_kernel_map(*a) == gsc.GSC_EINVAL and "768" in _err(L)
    assert L.gsc_table_status(None, None) == gsc.GSC_EINVAL
    assert L.gsc_coords_build_async(fake, 10, 0, fake, 1 << 20, None) == gsc.GSC_EINVAL
    big = (ctypes.c_int32 * 3)(1 << 29, 0, 0)
    ts4 = (ctypes.c_int32 * 3)(4, 1, 1)
    a = list(args(1, ts4, ws))
    a[4] = big
    assert L.gsc_kernel_map(*a) == gsc.GSC_ERANGE


def test_conv_validation(L):
    fake = ctypes.c_void_p(0x1000)
    fwd = lambda dt, ci, K, npairs=10, co=4, ws=None, wsb=0: L.gsc_sparse_conv_fwd(
        dt, fake, 10, ci, fake, co, K, fake, fake, fake, fake, npairs, None, None, None, None, fake, 10, ws, wsb,
        None)
    assert fwd(7, 4, 27) == gsc.GSC_EINVAL
    assert fwd(0, 0, 27) == gsc.GSC_EINVAL
    assert fwd(0, 4, 0) == gsc.GSC_EINVAL
    assert fwd(0, 4, 5000) == gsc.GSC_EINVAL
    assert fwd(0, 4, 27, -1) == gsc.GSC_EINVAL
    # the bf16 engine for wide layers needs a workspace for the transposed weights
    need = L.gsc_conv_fwd_ws_bytes(gsc.GSC_BF16, 256, 256, 27)
    assert need == 27 * 256 * 256 * 2 + 256   # transposed weights, then the tile counter
    assert L.gsc_conv_fwd_ws_bytes(gsc.GSC_F32, 256, 256, 27) == 0
    assert fwd(gsc.GSC_BF16, 256, 27, co=256) == gsc.GSC_ESHORT
    assert fwd(gsc.GSC_BF16, 256, 27, co=256, ws=fake, wsb=need - 1) == gsc.GSC_ESHORT
    sel = (ctypes.c_int32 * 2)(0, 2)   # 2 is out of range for K = 2
    rc = L.gsc_sparse_conv_bwd(0, fake, fake, fake, 10, 4, 4, 2, fake, fake, fake, 10, fake, fake, fake, fake,
                               10, sel, None, None, None, None, fake, None, 10, None, 0, None)
    assert rc == gsc.GSC_EINVAL and "t_wsel" in _err(L)
    sel = (ctypes.c_int32 * 3)(2, 0, 2)   # in range, but offset 2's weights twice and offset 1's never
    rc = L.gsc_sparse_conv_bwd(0, fake, fake, fake, 10, 4, 4, 3, fake, fake, fake, 10, fake, fake, fake, fake,
                               10, sel, None, None, None, None, fake, None, 10, None, 0, None)
    assert rc == gsc.GSC_EINVAL and "permutation" in _err(L)
    sel = (ctypes.c_int32 * 2)(0, 1)
    rc = L.gsc_sparse_conv_bwd(0, fake, fake, fake, 10, 4, 4, 2, fake, fake, fake, 10, fake, fake, fake, fake,
                               10, sel, None, None, None, None, None,
                               ctypes.cast(fake, ctypes.POINTER(ctypes.c_float)), 10, fake, 8, None)
    assert rc == gsc.GSC_ESHORT


def test_map_transpose_and_fwdmap_validation(L):
    fake = ctypes.c_void_p(0x1000)
    need = L.gsc_kernel_map_transpose_ws_bytes(100, 27)
    assert need > 0 and L.gsc_kernel_map_transpose_ws_bytes(-1, 27) == 0
    tr = lambda K=27, cap=50, n=100, ws=fake, wsb=need, seg=fake: L.gsc_kernel_map_transpose(
        fake, fake, seg, K, cap, n, fake, fake, fake, fake, fake, ws, wsb, None)
    assert tr(K=0) == gsc.GSC_EINVAL
    assert tr(seg=None) == gsc.GSC_EINVAL
    assert tr(ws=None) == gsc.GSC_EINVAL
    assert tr(wsb=need - 1) == gsc.GSC_ESHORT
    assert L.gsc_kernel_map_transpose_status(None, None) == gsc.GSC_EINVAL
    wb = L.gsc_conv_bwd_fwdmap_ws_bytes(gsc.GSC_F32, 100, 500, 32, 32, 27)
    assert wb > L.gsc_conv_bwd_ws_bytes(500, 32, 32, 27) and L.gsc_conv_bwd_fwdmap_ws_bytes(7, 100, 500, 32, 32, 27) == 0
    bwd = lambda dt=0, K=27, wsb=wb: L.gsc_sparse_conv_bwd_fwdmap(
        dt, fake, fake, fake, 100, 32, 32, K, fake, fake, fake, 500, 0, fake, None, 100, fake, wsb, None)
    assert bwd(dt=7) == gsc.GSC_EINVAL
    assert bwd(K=0) == gsc.GSC_EINVAL
    assert bwd(wsb=wb - 1) == gsc.GSC_ESHORT


def test_affine_backward_validation(L):
    fake = ctypes.c_void_p(0x1000)
    need = L.gsc_affine_act_bwd_ws_bytes(1000, 32)
    assert need > 0 and L.gsc_affine_act_bwd_ws_bytes(-1, 32) == 0
    ab = lambda dt=0, act=1, ws=fake, wsb=need, dsc=fake: L.gsc_affine_act_bwd(
        dt, fake, fake, 1000, 32, None, None, act, fake, dsc, None, ws, wsb, None)
    assert ab(dt=7) == gsc.GSC_EINVAL
    assert ab(act=5) == gsc.GSC_EINVAL
    assert ab(wsb=need - 1) == gsc.GSC_ESHORT
    assert ab(ws=None) == gsc.GSC_ESHORT


def test_plan_validation(L):
    fake = ctypes.c_void_p(0x1000)
    ws = L.gsc_conv_plan_ws_bytes(100, 27)
    assert ws > 0 and L.gsc_conv_plan_ws_bytes(100, 129) == 0 and L.gsc_conv_plan_ws_bytes(100, 81) > 0
    # maps with more than 32 offsets: plans over ranges of consecutive offsets
    assert [L.gsc_plan_ranges(K) for K in (1, 32, 33, 64, 81, 125, 128, 129, 0)] == [1, 1, 2, 2, 3, 4, 4, 0, 0]
    assert L.gsc_plan_blocks(0) == 0 and L.gsc_plan_blocks(16) == 1 and L.gsc_plan_blocks(17) == 2
    cap = 27 * 7
    plan = lambda K, wsb=ws, cap=cap, ib=fake: L.gsc_conv_plan(fake, 100, K, fake, fake, ib, fake, cap, fake, wsb,
                                                               None)
    assert plan(129) == gsc.GSC_EINVAL and "K=129" in _err(L)
    assert plan(0) == gsc.GSC_EINVAL
    assert plan(27, wsb=ws - 1) == gsc.GSC_ESHORT
    assert plan(27, cap=cap - 1) == gsc.GSC_ESHORT and str(cap) in _err(L)
    assert plan(27, ib=None) == gsc.GSC_EINVAL
    assert L.gsc_conv_plan_status(None, ws, 100, 27, None) == gsc.GSC_EINVAL
    assert L.gsc_conv_plan_status(fake, ws - 1, 100, 27, None) == gsc.GSC_ESHORT
    # the block engines and the shapes they take
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 32, 32, 27) == 1
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 64, 64, 9) == 1
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 64, 64, 10) == 0
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 32, 32, 33) == 1    # two ranges of 17 offsets
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 32, 32, 81) == 1    # three of 27
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 64, 64, 81) == 0    # 27 weight matrices of 16 KiB do not fit
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 16, 16, 129) == 0
    assert L.gsc_conv_block_engine(gsc.GSC_BF16, 256, 256, 33) == 0
    assert L.gsc_conv_block_engine(gsc.GSC_F32, 3, 16, 27) == 0
    assert L.gsc_conv_block_engine(gsc.GSC_BF16, 256, 256, 27) == 1
    assert L.gsc_conv_block_engine(gsc.GSC_BF16, 32, 32, 27) == 0
    # a plan is all four pointers or none
    rc = L.gsc_sparse_conv_fwd(0, fake, 10, 16, fake, 16, 27, fake, fake, fake, fake, 10, fake, None, fake, fake,
                               fake, 10, None, 0, None)
    assert rc == gsc.GSC_EINVAL and "plan" in _err(L)
    # the affine forward validates its activation and then as the plain forward
    aff = lambda act, K=27: L.gsc_sparse_conv_fwd_affine(0, fake, 10, 16, fake, 16, K, fake, fake, fake, fake, 10,
                                                         None, None, None, None, fake, fake, act, fake, 10, None, 0,
                                                         None)
    assert aff(2) == gsc.GSC_EINVAL and "act" in _err(L)
    assert aff(1, K=0) == gsc.GSC_EINVAL and "K=0" in _err(L)


@pytest.mark.parametrize("name,K,D", [("cube", 3, 3), ("cube", 2, 3), ("cube", 5, 4), ("cross", 5, 3),
                                      ("hybrid", 3, 4), ("spatial", 3, 4), ("cube", 3, 7)])
def test_regions_match_oracle(name, K, D):
    assert np.array_equal(regions.region(name, K, D), O.region(name, K, D))


def test_negation_permutation():
    offs = regions.hypercube(3, 3)
    p = gsc.negation_permutation(offs)
    assert np.array_equal(offs[p], -offs)
    assert regions.is_symmetric(regions.hybrid(3, 4))
    assert not regions.is_symmetric(regions.hypercube(2, 3))
