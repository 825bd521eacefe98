"""The allocation-free kernel map (gsc_kernel_map_noalloc) against the kernel
map with a caller workspace (gsc_kernel_map), through the C ABI: two calls in
a row on one GPU, the second on a smaller input, every output bit-exact."""
import numpy as np
import pytest
import torch

from paper_1904_08755_amd import gsc, regions
from paper_1904_08755_amd import workloads as WL

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(msg):
    print(msg, flush=True)


def _pair(coords_np, offs, table_coords_np=None):
    """Both entry points on the same table and output coordinates; returns
    their maps (async mode, dense form)."""
    out = torch.from_numpy(coords_np).to(DEV)
    tc = out if table_coords_np is None else torch.from_numpy(table_coords_np).to(DEV)
    table = gsc.gsc_coords_build(tc)
    K, D = offs.shape
    n = out.shape[0]
    b_ref = gsc.MapBuffers(n, K, D, DEV, dense=True)
    b_new = gsc.MapBuffers(n, K, D, DEV, dense=True)
    # fill the outputs of the allocation-free call with garbage first
    for t in (b_new.in_idx, b_new.out_idx, b_new.seg, b_new.gidx, b_new.nbr):
        t.fill_(-7)
    ref = gsc.gsc_kernel_map(table, out, offs, sync=False, bufs=b_ref, dense=True)
    new = gsc.gsc_kernel_map_noalloc(table, out, offs, b_new)
    torch.cuda.synchronize()
    return ref, new


def _same(ref, new):
    K = ref.K
    seg = ref.seg.cpu().numpy()
    assert np.array_equal(seg, new.seg.cpu().numpy())
    assert np.array_equal(ref.gidx.cpu().numpy(), new.gidx.cpu().numpy())
    m = int(seg[K])
    assert np.array_equal(ref.in_idx[:m].cpu().numpy(), new.in_idx[:m].cpu().numpy())
    assert np.array_equal(ref.out_idx[:m].cpu().numpy(), new.out_idx[:m].cpu().numpy())
    assert np.array_equal(ref.nbr.cpu().numpy(), new.nbr.cpu().numpy())
    return m


def test_kernel_map_noalloc_matches_workspace_form():
    # first call: a scene-like tensor over a symmetric region (the self-map path)
    wl = WL.make_workload(1, scale=0.4)
    _say(f"[gpu] noalloc call 1: n={wl.n} cube3")
    ref, new = _pair(wl.coords, regions.hypercube(3, 3))
    m1 = _same(ref, new)
    assert m1 > wl.n
    # second call, smaller: random coordinates, a non-symmetric region, onto
    # other output coordinates (a strided layer's map)
    c = WL.random_coords(301, 3000, 3, -9, 9, batch=2)
    out = np.unique(np.concatenate([c[:, :1], (c[:, 1:] // 2) * 2], 1), axis=0).astype(np.int32)
    _say(f"[gpu] noalloc call 2: n_in={len(c)} n_out={len(out)} cube2")
    offs = regions.hypercube(2, 3)
    outt = torch.from_numpy(out).to(DEV)
    table = gsc.gsc_coords_build(torch.from_numpy(c).to(DEV))
    K, D = offs.shape
    b_ref = gsc.MapBuffers(len(out), K, D, DEV, dense=True)
    b_new = gsc.MapBuffers(len(out), K, D, DEV, dense=True)
    ref2 = gsc.gsc_kernel_map(table, outt, offs, sync=False, bufs=b_ref, dense=True)
    new2 = gsc.gsc_kernel_map_noalloc(table, outt, offs, b_new)
    torch.cuda.synchronize()
    m2 = _same(ref2, new2)
    assert 0 < m2 < m1 and m2 == len(c)   # the stride-2 map of {0,1}^3 pairs every input once


def test_kernel_map_noalloc_limits():
    # more scratch than the library holds: rejected on the host, before any GPU work
    n = 6_000_000
    assert gsc.lib().gsc_kernel_map_noalloc_bytes(n, 27) > 8 << 20
    c = torch.zeros((1, 4), dtype=torch.int32, device=DEV)
    table = torch.zeros(gsc.gsc_table_bytes(1), dtype=torch.uint8, device=DEV)
    offs = gsc._host_i32(regions.hypercube(3, 3))
    rc = gsc.lib().gsc_kernel_map_noalloc(gsc._ptr(table), gsc._ptr(c), n, 3, offs, 27, None, gsc._ptr(c),
                                          gsc._ptr(c), 27 * n, gsc._ptr(c), gsc._ptr(c), gsc._ptr(c), None)
    assert rc == gsc.GSC_ERANGE
    assert b"scratch" in gsc.lib().gsc_last_error()
