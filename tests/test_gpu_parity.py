"""Parity of the HIP path (through the C-ABI) with the CPU oracle.

Kernel maps and output coordinates must match bit-exactly (after canonical
alignment of strided output rows); features and gradients within the max
relative error 1e-5 (fp32) or 2e-2 (bf16 inputs, fp32 accumulation).

* all five workloads at full size, through the same pipeline the benchmark
  times;
* the same workloads shrunk (scale 0.3: several tiles and ragged tails, the
  oracle finishes in seconds);
* edge cases: empty input, one voxel, duplicates, key range, short buffers,
  negative coordinates over several batches, non-symmetric and large regions,
  tensor stride, odd channel counts, the centre-only identity kernel.
"""
import os
import sys

import numpy as np
import pytest
import torch

import oracle.gsc_oracle as O
from paper_1904_08755_amd import gsc, pipeline, regions
from paper_1904_08755_amd import workloads as WL
from parity import TOL, check_gidx, compare_step, gpu_pairs, maps_equal_exact, oracle_step, rel_err, to_np

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gsc.lib()


def _run(wl):
    _say(f"[gpu] {wl.name} n={wl.n}")
    dw = pipeline.to_device(wl, DEV)
    step = pipeline.run_step(dw)
    torch.cuda.synchronize()
    return step


@pytest.mark.parametrize("cid", [0, 1, 2, 3, 4])
def test_workload_small(cid):
    wl = WL.make_workload(cid, scale=0.3)
    step = _run(wl)
    errs = compare_step(wl, step, oracle_step(wl))
    _say(f"  errors {errs}")


@pytest.mark.parametrize("cid", [0, 1, 2, 3, 4])
def test_workload_full(cid):
    wl = WL.make_workload(cid)
    step = _run(wl)
    ref = oracle_step(wl)
    errs = compare_step(wl, step, ref)
    npairs = [km.count() for km in step.kmaps]
    _say(f"  pairs {npairs} errors {errs}")


def test_map_symmetry_on_gpu():
    wl = WL.make_workload(1, scale=0.3)
    dw = pipeline.to_device(wl, DEV)
    table = gsc.gsc_coords_build(dw.coords)
    offs = regions.hypercube(3, 3)
    pairs = gpu_pairs(gsc.gsc_kernel_map(table, dw.coords, offs))
    neg = gsc.negation_permutation(offs)
    for k in range(len(offs)):
        a = set(zip(pairs[k][0].tolist(), pairs[k][1].tolist()))
        b = set(zip(pairs[neg[k]][1].tolist(), pairs[neg[k]][0].tolist()))
        assert a == b
    centre = int(np.where((offs == 0).all(1))[0][0])
    assert np.array_equal(pairs[centre][0], np.arange(wl.n))


# --------------------------------------------------------------------------- #
# edge cases
# --------------------------------------------------------------------------- #
def _t(a, dtype=torch.int32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV).to(dtype)


def _conv_case(coords, ci, co, offs, seed, dtype="f32", ts=1):
    """Submanifold conv fwd + bwd on explicit coordinates vs the oracle.  Uses
    the explicitly built role-reversed map for dX (works for any region)."""
    c = _t(coords)
    X, Xb = WL.random_features(seed, len(coords), ci, dtype)
    W, Wb = WL.random_weights(seed, len(offs), ci, co, dtype)
    G, Gb = WL.random_features(seed + 1, len(coords), co, dtype)
    if dtype == "bf16":
        tX = torch.from_numpy(Xb.view(np.int16)).to(DEV).view(torch.bfloat16)
        tW = torch.from_numpy(Wb.view(np.int16)).to(DEV).view(torch.bfloat16)
        tG = torch.from_numpy(Gb.view(np.int16)).to(DEV).view(torch.bfloat16)
    else:
        tX, tW, tG = _t(X, torch.float32), _t(W, torch.float32), _t(G, torch.float32)
    table = gsc.gsc_coords_build(c)
    km = gsc.gsc_kernel_map(table, c, offs, tensor_stride=ts)
    tm = gsc.transposed_kernel_map(table, c, offs, tensor_stride=ts)
    Y = gsc.gsc_sparse_conv_fwd(tX, tW, km)
    dX, dW = gsc.gsc_sparse_conv_bwd(tX, tW, tG, km, tm, np.arange(len(offs)))
    torch.cuda.synchronize()
    m = O.kernel_map(coords, coords, np.asarray(offs), ts)
    maps_equal_exact(gpu_pairs(km), m)
    check_gidx(km)
    maps_equal_exact(gpu_pairs(tm), O.transposed_map(m))
    Yr = O.conv_forward(X, W, m, len(coords))
    dXr, dWr = O.conv_backward(X, W, G, m)
    tol = TOL[dtype]
    assert rel_err(to_np(Y), Yr) <= tol
    assert rel_err(to_np(dX), dXr) <= tol
    assert rel_err(to_np(dW), dWr) <= tol
    return km


@pytest.mark.parametrize("case", ["cube3", "cube5", "cross3", "hybrid4d", "cube3_ts2", "sync_async"])
def test_self_map_matches_copy(case):
    """A map of the table's own coordinate set onto itself over a symmetric
    listing probes half the offsets and mirrors the rest; it must equal the
    map over the same offsets listed in another (non-symmetric) order, which
    probes every offset, bit for bit once the order is undone, and the
    oracle's map."""
    if case == "hybrid4d":
        wl = WL.make_workload(3, scale=0.3)
        offs = regions.hybrid(3, 4)
    else:
        wl = WL.make_workload(1, scale=0.15)
        offs = {"cube3": regions.hypercube(3, 3), "cube5": regions.hypercube(5, 3),
                "cross3": regions.hypercross(3, 3), "cube3_ts2": regions.hypercube(3, 3),
                "sync_async": regions.hypercube(3, 3)}[case]
    ts = 2 if case == "cube3_ts2" else None
    coords = torch.from_numpy(wl.coords).to(DEV)
    if ts:
        coords = coords.clone()
        coords[:, 1:] *= 2
    table = gsc.gsc_coords_build(coords)
    self_map = gsc.gsc_kernel_map(table, coords, offs, tensor_stride=ts, dense=True,
                                  sync=case != "sync_async")
    rolled = np.roll(np.asarray(offs), 1, axis=0)                   # not a symmetric listing: full probe
    full_map = gsc.gsc_kernel_map(table, coords, rolled, tensor_stride=ts, dense=True)
    torch.cuda.synchronize()
    K = len(offs)
    a, b = gpu_pairs(self_map), gpu_pairs(full_map)
    for k in range(K):
        assert np.array_equal(a[k][0], b[(k + 1) % K][0]) and np.array_equal(a[k][1], b[(k + 1) % K][1])
    n = wl.n
    assert np.array_equal(to_np(self_map.nbr), np.roll(to_np(full_map.nbr).reshape(K, n), -1, axis=0))
    c_np = to_np(coords)
    ref = O.kernel_map(c_np, c_np, np.asarray(offs), ts or 1)
    for k in range(K):
        assert np.array_equal(a[k][0], np.asarray(ref[k][0])) and np.array_equal(a[k][1], np.asarray(ref[k][1]))
    check_gidx(self_map)
    _say(f"  {case}: K={K} pairs={self_map.count()}")


@pytest.mark.parametrize("change", ["shift_in_place", "permuted_copy", "two_rows_swapped", "one_row_moved"])
def test_self_map_premise_checked(change):
    """Output coordinates that are not the table's rows in the table's order,
    though as many: rows rewritten in place after the build (the same
    pointer), the rows in another order, two rows swapped, one row moved to a
    free coordinate.  The map must still be the full probe's, i.e. the
    oracle's map from the coordinates the table was built from to the output
    coordinates."""
    wl = WL.make_workload(1, scale=0.15)
    offs = regions.hypercube(3, 3)
    coords = torch.from_numpy(wl.coords.copy()).to(DEV)
    table = gsc.gsc_coords_build(coords)
    base = wl.coords.copy()
    if change == "shift_in_place":
        coords[:, 1] += 1                                             # same array, new values
    elif change == "permuted_copy":
        perm = np.random.default_rng(5).permutation(wl.n)
        coords = torch.from_numpy(base[perm]).to(DEV)
    elif change == "two_rows_swapped":
        c2 = base.copy()
        c2[[10, 500]] = c2[[500, 10]]
        coords.copy_(torch.from_numpy(c2))
    else:
        c2 = base.copy()
        c2[77, 1:] = base[:, 1:].max(0) + 5                          # outside every neighbourhood
        coords.copy_(torch.from_numpy(c2))
    for sync in (True, False):
        km = gsc.gsc_kernel_map(table, coords, offs, dense=True, sync=sync)
        torch.cuda.synchronize()
        ref = O.kernel_map(base, to_np(coords).astype(np.int64), offs)
        maps_equal_exact(gpu_pairs(km), ref)
        check_gidx(km)
        nb = to_np(km.nbr).astype(np.int64)
        for k, (ri, ro) in enumerate(ref):
            row = np.full(wl.n, -1)
            row[np.asarray(ro, np.int64)] = ri
            assert np.array_equal(nb[k], row)


def test_empty_input():
    c = torch.empty((0, 4), dtype=torch.int32, device=DEV)
    table = gsc.gsc_coords_build(c)
    km = gsc.gsc_kernel_map(table, c, regions.hypercube(3, 3))
    assert km.n_pairs == 0
    out, _ = gsc.gsc_coords_stride(c, 2)
    assert out.shape[0] == 0
    X = torch.empty((0, 8), device=DEV)
    W = torch.randn((27, 8, 4), device=DEV)
    Y = gsc.gsc_sparse_conv_fwd(X, W, km)
    assert Y.shape == (0, 4)
    dX, dW = gsc.gsc_sparse_conv_bwd(X, W, torch.empty((0, 4), device=DEV), km, km, np.arange(27))
    torch.cuda.synchronize()
    assert dX.shape == (0, 8)
    assert torch.count_nonzero(dW).item() == 0


def test_empty_output_rows_are_zero():
    # outputs that no input reaches: query a table of far-away inputs
    cin = np.array([[0, 100, 100, 100], [0, 101, 100, 100]], np.int32)
    cout = np.array([[0, 0, 0, 0], [0, 1, 1, 1], [0, 100, 100, 99]], np.int32)
    table = gsc.gsc_coords_build(_t(cin))
    km = gsc.gsc_kernel_map(table, _t(cout), regions.hypercube(3, 3))
    X = torch.randn((2, 5), device=DEV)
    W = torch.randn((27, 5, 3), device=DEV)
    Y = gsc.gsc_sparse_conv_fwd(X, W, km)
    torch.cuda.synchronize()
    ref = O.conv_forward(X.cpu().numpy(), W.cpu().numpy(), O.kernel_map(cin, cout, O.hypercube(3, 3)), 3)
    assert np.all(to_np(Y)[:2] == 0)
    assert rel_err(to_np(Y), ref) <= 1e-5


def test_single_voxel():
    _conv_case(np.array([[0, -7, 3, 11]], np.int32), 4, 6, regions.hypercube(3, 3), 51)


def test_duplicate_rejected():
    c = _t(np.array([[0, 1, 2, 3], [0, 4, 5, 6], [0, 1, 2, 3]], np.int32))
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_coords_build(c)
    assert e.value.code == gsc.GSC_EDUP


def test_table_full_reported(monkeypatch):
    """A table too small for its rows (its capacity capped from the host
    through the GSC_TABLE_CAP_LIMIT hook: 64 slots for 200 rows) reports
    EFULL; every insert's probe ends after one pass over the slots, and a
    kernel map queried from the failed table comes out empty (asynchronous)
    or reports it (synchronous)."""
    coords = _t(WL.random_coords(177, 200, 3, -20, 20, batch=1))
    monkeypatch.setenv("GSC_TABLE_CAP_LIMIT", "64")
    assert gsc.gsc_table_bytes(200) == gsc.gsc_table_bytes(1)   # 64 slots: the cap is in force
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_coords_build(coords)
    assert e.value.code == gsc.GSC_EFULL
    table = gsc.gsc_coords_build(coords, sync=False)
    km = gsc.gsc_kernel_map(table, coords, regions.hypercube(3, 3), sync=False)
    assert km.count() == 0
    with pytest.raises(gsc.GscError) as e:   # the synchronous map reports the invalid table
        gsc.gsc_kernel_map(table, coords, regions.hypercube(3, 3))
    assert e.value.code == gsc.GSC_EINVAL
    monkeypatch.delenv("GSC_TABLE_CAP_LIMIT")
    gsc.gsc_table_status(gsc.gsc_coords_build(coords))   # the normal capacity holds them


def test_key_range_rejected():
    # 8 columns each spanning 2^12 values need 96 key bits, past the 92 the
    # wide key holds; spanning 2^9 values (72 bits) they build
    rows = np.zeros((2, 8), np.int32)
    rows[1, :] = 4095
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_coords_build(_t(rows))
    assert e.value.code == gsc.GSC_ERANGE
    rows[1, :] = 511
    c = _t(rows)
    km = gsc.gsc_kernel_map(gsc.gsc_coords_build(c), c, np.zeros((1, 7), np.int32))
    assert np.array_equal(gpu_pairs(km)[0][0], np.arange(2))


def test_kernel_map_short_then_retry():
    coords = WL.random_coords(61, 3000, 3, -20, 20, batch=2)
    c = _t(coords)
    table = gsc.gsc_coords_build(c)
    offs = regions.hypercube(3, 3)
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_kernel_map(table, c, offs, cap_pairs=10)
    assert e.value.code == gsc.GSC_ESHORT
    ref = O.kernel_map(coords, coords, O.hypercube(3, 3))
    km = gsc.gsc_kernel_map(table, c, offs, cap_pairs=O.map_pair_count(ref))
    maps_equal_exact(gpu_pairs(km), ref)


def test_negative_coords_many_batches_cube():
    coords = WL.random_coords(71, 5000, 3, -30, 10, batch=5)
    _conv_case(coords, 16, 32, regions.hypercube(3, 3), 71)


def test_nonsymmetric_region_and_ragged_channels():
    coords = WL.random_coords(72, 4000, 3, -12, 12, batch=2)
    _conv_case(coords, 3, 70, regions.hypercube(2, 3), 72)   # 70 > 64: two column slices


def test_large_region_cube5_and_cross():
    coords = WL.random_coords(73, 2500, 3, -10, 10, batch=2)
    _conv_case(coords, 8, 8, regions.hypercube(5, 3), 73)
    _conv_case(coords, 5, 12, regions.hypercross(5, 3), 74)


def test_tensor_stride_two():
    coords = WL.random_coords(75, 3000, 3, -10, 10, batch=2)
    coords[:, 1:] *= 2
    _conv_case(coords, 8, 16, regions.hypercube(3, 3), 75, ts=2)


def test_bf16_odd_channels():
    coords = WL.random_coords(76, 3000, 3, -15, 15, batch=2)
    _conv_case(coords, 24, 40, regions.hypercube(3, 3), 76, dtype="bf16")


def test_bf16_forward_misaligned_weights():
    """Weights that start 2 bytes past a 16-byte boundary: the forward's
    transposed copy of W takes the element-wise path (the 16-byte one needs
    aligned matrices), and the result is still the oracle's."""
    coords = WL.random_coords(97, 1500, 3, -10, 10, batch=2)
    offs = regions.hypercube(3, 3)
    ci, co = 32, 64
    X, Xb = WL.random_features(98, len(coords), ci, "bf16")
    W, Wb = WL.random_weights(99, len(offs), ci, co, "bf16")
    dev = lambda b: torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
    flat = torch.zeros(Wb.size + 8, dtype=torch.bfloat16, device=DEV)
    base = (16 - flat.data_ptr() % 16) % 16 // 2 + 1      # one element past an aligned start
    tW = flat[base:base + Wb.size].view(len(offs), ci, co)
    tW.copy_(dev(Wb))
    assert tW.data_ptr() % 16 == 2
    table = gsc.gsc_coords_build(_t(coords))
    km = gsc.gsc_kernel_map(table, _t(coords), offs)
    _say("[gpu] bf16 forward, weights 2 bytes off alignment")
    Y = gsc.gsc_sparse_conv_fwd(dev(Xb), tW, km)
    torch.cuda.synchronize()
    m = O.kernel_map(coords, coords, np.asarray(offs))
    assert rel_err(to_np(Y), O.conv_forward(X, W, m, len(coords))) <= TOL["bf16"]


@pytest.mark.parametrize("ci,co,region", [(256, 256, "cube2"), (128, 256, "cube3"), (256, 128, "cube2"),
                                           (64, 128, "cube3"), (128, 64, "cube2"), (32, 256, "cube3")])
def test_bf16_wide_channel_engine(ci, co, region):
    # the MFMA engine for wide bf16 layers: forward, input gradient on the
    # role-reversed map (non-symmetric regions included) and weight gradient
    coords = WL.random_coords(90 + ci // 32 + co // 16, 2500, 3, -12, 12, batch=2)
    offs = regions.hypercube(int(region[-1]), 3)
    _say(f"[gpu] bf16 engine {ci}->{co} {region}")
    _conv_case(coords, ci, co, offs, 91, dtype="bf16")


def _check_plan(km):
    """The block plan of a map: rows stably sorted by neighbour count (capped
    to the spare bits of the sort's last 10-bit digit), then mask, 16-row
    blocks with their union masks and item bases, and each item holding the
    input rows of its block's positions at its offset (-1 where none).  A map
    with more than 32 offsets has one such plan per range of consecutive
    offsets (ceil(K / 32) ranges of equal size but the last)."""
    pl = km.plan
    n, K = km.n_out, km.K
    nb = (n + 15) // 16
    pairs = gpu_pairs(km)
    nbr = np.full((max(n, 1), K), -1, np.int64)
    for k, (i, o) in enumerate(pairs):
        nbr[o, k] = i
    assert np.array_equal(km.nbr.cpu().numpy().T.astype(np.int64), nbr[:n])   # the dense form lists the same pairs
    R = -(-K // 32)
    S = -(-K // R)
    assert gsc.gsc_plan_ranges(K) == R
    perm_all = pl.perm.cpu().numpy().astype(np.int64)
    bm_all = pl.bmask.cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    ib_all = pl.ibase.cpu().numpy()
    items_all = pl.items.cpu().numpy()
    for r in range(R):
        k0, k1 = r * S, min(K, r * S + S)
        _check_plan_range(n, nbr[:, k0:k1], perm_all[r * n:(r + 1) * n], bm_all[r * nb:(r + 1) * nb],
                          ib_all[r * (nb + 1):(r + 1) * (nb + 1)], items_all[k0 * nb:])


def _check_plan_range(n, nbr, perm, bm, ib, items):
    nb = (n + 15) // 16
    K = nbr.shape[1]
    assert np.array_equal(np.sort(perm), np.arange(n))
    mask = np.zeros(max(n, 1), np.int64)
    for k in range(K):
        mask |= (nbr[:, k] >= 0).astype(np.int64) << np.int64(k)
    pbits = min(-(-K // 10) * 10 - K, 32 - K, 6)                      # popcount field of the key
    cnt_rows = np.array([bin(int(x)).count("1") for x in mask], np.int64)
    key = (np.minimum(cnt_rows, (1 << pbits) - 1) << np.int64(K)) | mask
    ks = key[perm]
    assert np.all(ks[1:] >= ks[:-1])                                   # sorted by key
    same = ks[1:] == ks[:-1]
    assert np.all(perm[1:][same] > perm[:-1][same])                    # stable: row order within a key
    ms = mask[perm]
    msp = np.zeros(nb * 16, np.int64)
    msp[:n] = ms
    assert np.array_equal(bm, np.bitwise_or.reduce(msp.reshape(nb, 16), axis=1) if nb else bm)
    cnt = np.array([bin(int(x)).count("1") for x in bm], np.int64)
    assert ib[0] == 0 and np.array_equal(np.diff(ib), cnt)
    items = items[: ib[-1]]
    below = np.zeros(nb, np.int64)                                     # set bits of bmask below offset k
    pos = np.arange(nb)[:, None] * 16 + np.arange(16)[None, :]
    rows = perm[np.minimum(pos, max(n - 1, 0))] if n else pos
    for k in range(K):
        blocks = np.nonzero((bm >> k) & 1)[0]
        if len(blocks):
            exp = np.where(pos[blocks] < n, nbr[rows[blocks], k], -1)
            assert np.array_equal(items[ib[blocks] + below[blocks]], exp), k
        below += (bm >> k) & 1


@pytest.mark.parametrize("D", [3, 4])
def test_plan_lookback_give_up_is_reported(monkeypatch, D):
    """A sort pass whose look-back gives up (forced from the host: the
    environment's spin limit makes every poll give up at once) finishes
    normally and the plan call's status reports ETIMEOUT; with the normal
    bound the same buffers give a valid plan and status OK.  D = 4: the 81
    offsets of the tesseract, three plan ranges sorted in the same launches."""
    coords = WL.random_coords(175, 24000, D, -25 if D == 3 else -10, 25 if D == 3 else 10, batch=2)
    c = _t(coords)
    offs = regions.hypercube(3, D)
    km = gsc.gsc_kernel_map(gsc.gsc_coords_build(c), c, offs, dense=True)
    bufs = gsc.PlanBuffers(km.n_out, km.K, DEV)
    _say(f"[gpu] look-back give-up forced on n={km.n_out}")
    monkeypatch.setenv("GSC_PLAN_SPIN_LIMIT", "-1")
    gsc.gsc_conv_plan(km, bufs)
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_conv_plan_status(km, bufs)
    assert e.value.code == gsc.GSC_ETIMEOUT
    monkeypatch.delenv("GSC_PLAN_SPIN_LIMIT")
    pm = gsc.gsc_conv_plan(km, bufs)
    gsc.gsc_conv_plan_status(km, bufs)
    _check_plan(pm)


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_conv_plan_block_engine(cid):
    # the block engines on the plan against the oracle, the row-form kernels
    # and themselves (deterministic)
    wl = WL.make_workload(cid, scale=0.3)
    _say(f"[gpu] plan {wl.name} n={wl.n}")
    dw = pipeline.to_device(wl, DEV)
    base = pipeline.StepPlan(dw, use_plan=False).run()
    planned = pipeline.StepPlan(dw, use_plan=True)
    res = planned.run()
    torch.cuda.synchronize()
    assert planned.plans
    for km in planned.plans:
        _check_plan(km)
    compare_step(wl, res, oracle_step(wl))
    for a, b in zip(base.Ys + [base.dX], res.Ys + [res.dX]):
        assert rel_err(to_np(b), to_np(a)) <= TOL["f32"]
    for a, b in zip(base.dWs, res.dWs):   # same map; inner layers' inputs differ by rounding only
        assert rel_err(to_np(b), to_np(a)) <= TOL["f32"]
    again = planned.run()
    torch.cuda.synchronize()
    for a, b in zip(res.Ys + [res.dX], again.Ys + [again.dX]):
        assert torch.equal(a, b)


def test_conv_plan_structure_bf16_wide():
    # the plan depends only on the map: build it for the wide workload's map
    wl = WL.make_workload(4, scale=0.3)
    dw = pipeline.to_device(wl, DEV)
    table = gsc.gsc_coords_build(dw.coords)
    km = gsc.gsc_kernel_map(table, dw.coords, dw.offsets[0], dense=True)
    _check_plan(gsc.gsc_conv_plan(km))


def test_conv_plan_structure_full_size():
    """The block plan of the full 2 cm scene pair (300,577 rows: 18,787
    blocks, whose item counts take the two-kernel scan), entry by entry
    against the map."""
    wl = WL.make_workload(1)
    dw = pipeline.to_device(wl, DEV)
    table = gsc.gsc_coords_build(dw.coords)
    km = gsc.gsc_kernel_map(table, dw.coords, dw.offsets[0], dense=True)
    _say(f"[gpu] full-size plan n={wl.n}")
    _check_plan(gsc.gsc_conv_plan(km))


def _plan_case(coords, ci, co, offs, seed, ts=1, dtype="f32"):
    """_conv_case through the block engines: plans of the forward and the
    role-reversed map."""
    c = _t(coords)
    X, Xb = WL.random_features(seed, len(coords), ci, dtype)
    W, Wb = WL.random_weights(seed, len(offs), ci, co, dtype)
    G, Gb = WL.random_features(seed + 1, len(coords), co, dtype)
    if dtype == "bf16":
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
        tX, tW, tG = dev(Xb), dev(Wb), dev(Gb)
    else:
        tX, tW, tG = _t(X, torch.float32), _t(W, torch.float32), _t(G, torch.float32)
    table = gsc.gsc_coords_build(c)
    km = gsc.gsc_conv_plan(gsc.gsc_kernel_map(table, c, offs, tensor_stride=ts, dense=True))
    tm = gsc.gsc_conv_plan(gsc.transposed_kernel_map(table, c, offs, tensor_stride=ts, dense=True))
    Y = gsc.gsc_sparse_conv_fwd(tX, tW, km)
    dX, _ = gsc.gsc_sparse_conv_bwd(tX, tW, tG, km, tm, np.arange(len(offs)), need_dw=False)
    torch.cuda.synchronize()
    _check_plan(km)
    _check_plan(tm)
    m = O.kernel_map(coords, coords, np.asarray(offs), ts)
    assert rel_err(to_np(Y), O.conv_forward(X, W, m, len(coords))) <= TOL[dtype]
    assert rel_err(to_np(dX), O.conv_backward(X, W, G, m)[0]) <= TOL[dtype]


@pytest.mark.parametrize("ci,co,region", [(16, 16, "cube3"), (16, 64, "cube3"), (64, 16, "cube2"), (32, 64, "cube2"),
                                           (64, 32, "cube2"), (64, 64, "cube2"), (32, 32, "cube2")])
def test_block_engine_shapes(ci, co, region):
    coords = WL.random_coords(120 + ci + co, 3000, 3, -12, 12, batch=2)
    assert gsc.gsc_conv_block_engine(gsc.GSC_F32, ci, co, 27 if region == "cube3" else 8)
    _say(f"[gpu] block engine {ci}->{co} {region}")
    _plan_case(coords, ci, co, regions.hypercube(int(region[-1]), 3), 121)


@pytest.mark.parametrize("ci,co,region", [(256, 256, "cube3"), (128, 256, "cube2"), (256, 128, "cube3"),
                                           (64, 128, "cube3"), (128, 64, "cube2"), (64, 64, "cube3"),
                                           (256, 64, "cube2"), (64, 256, "cube2"), (128, 128, "cube3")])
def test_block_engine_bf16(ci, co, region):
    coords = WL.random_coords(140 + ci // 32 + co // 16, 2500, 3, -12, 12, batch=2)
    K = 27 if region == "cube3" else 8
    assert gsc.gsc_conv_block_engine(gsc.GSC_BF16, ci, co, K) and gsc.gsc_conv_block_engine(gsc.GSC_BF16, co, ci, K)
    _say(f"[gpu] bf16 block engine {ci}->{co} {region}")
    _plan_case(coords, ci, co, regions.hypercube(int(region[-1]), 3), 141, dtype="bf16")


@pytest.mark.parametrize("K", [29, 30, 32])
def test_block_engine_bf16_offset_limit(K):
    # the tile engine at its largest region (29 offsets: its item table fills
    # the LDS left by the stages) and the regions past it (30 and 32 offsets,
    # on the 16-block bf16 engine)
    extra = np.array([[2, 0, 0], [-2, 0, 0], [0, 2, 0], [0, -2, 0], [0, 0, 2]], np.int32)
    offs = np.concatenate([regions.hypercube(3, 3), extra[:K - 27]]).astype(np.int32)
    assert len(offs) == K and gsc.gsc_conv_block_engine(gsc.GSC_BF16, 256, 256, K)
    coords = WL.random_coords(150 + K, 1500, 3, -9, 9, batch=2)
    _say(f"[gpu] bf16 block engines 256->256, {K} offsets")
    _plan_case(coords, 256, 256, offs, 151, dtype="bf16")


def test_block_engine_edges():
    # one voxel, a ragged last block, no input rows, 4D hybrid region
    _plan_case(np.array([[0, -7, 3, 11]], np.int32), 16, 32, regions.hypercube(3, 3), 131)
    _plan_case(WL.random_coords(132, 37, 3, -3, 3, batch=2), 32, 32, regions.hypercube(3, 3), 132)
    _plan_case(WL.random_coords(133, 2000, 4, -5, 5, batch=1), 32, 32, regions.hybrid(3, 4), 133)
    _plan_case(WL.random_coords(135, 37, 3, -3, 3, batch=2), 128, 256, regions.hypercube(3, 3), 135, dtype="bf16")
    _plan_case(np.array([[0, -7, 3, 11]], np.int32), 64, 64, regions.hypercube(3, 3), 136, dtype="bf16")
    c = torch.empty((0, 4), dtype=torch.int32, device=DEV)
    km = gsc.gsc_conv_plan(gsc.gsc_kernel_map(gsc.gsc_coords_build(c), c, regions.hypercube(3, 3), dense=True))
    Y = gsc.gsc_sparse_conv_fwd(torch.empty((0, 16), device=DEV), torch.randn((27, 16, 16), device=DEV), km)
    assert Y.shape == (0, 16)
    # outputs no input reaches (a plan with empty blocks) and an input with no rows
    cin = np.array([[0, 100, 100, 100], [0, 101, 100, 100]], np.int32)
    cout = WL.random_coords(134, 40, 3, -3, 3, batch=1)
    cout = np.concatenate([cout, np.array([[0, 100, 100, 99]], np.int32)])
    km = gsc.gsc_conv_plan(gsc.gsc_kernel_map(gsc.gsc_coords_build(_t(cin)), _t(cout), regions.hypercube(3, 3),
                                              dense=True))
    X = torch.randn((2, 16), device=DEV)
    W = torch.randn((27, 16, 32), device=DEV)
    Y = gsc.gsc_sparse_conv_fwd(X, W, km)
    torch.cuda.synchronize()
    ref = O.conv_forward(X.cpu().numpy(), W.cpu().numpy(), O.kernel_map(cin, cout, O.hypercube(3, 3)), len(cout))
    assert rel_err(to_np(Y), ref) <= TOL["f32"] and np.all(to_np(Y)[:-1] == 0)
    _check_plan(km)
    empty_in = torch.empty((0, 16), device=DEV)
    km0 = gsc.gsc_conv_plan(gsc.gsc_kernel_map(gsc.gsc_coords_build(torch.empty((0, 4), dtype=torch.int32,
                                                                                device=DEV)),
                                               _t(cout), regions.hypercube(3, 3), dense=True))
    Y0 = gsc.gsc_sparse_conv_fwd(empty_in, W, km0)
    torch.cuda.synchronize()
    assert torch.count_nonzero(Y0).item() == 0 and Y0.shape == (len(cout), 32)


def test_4d_hybrid_and_tesseract():
    coords = WL.random_coords(77, 3000, 4, -5, 5, batch=1)
    _conv_case(coords, 8, 8, regions.hybrid(3, 4), 77)
    _conv_case(coords, 8, 8, regions.hypercube(3, 4), 78)
    _conv_case(coords, 8, 8, regions.spatial(3, 4), 79)


@pytest.mark.parametrize("region", ["tesseract", "cube5", "cube3+axes2"])
def test_block_engine_offset_ranges(region):
    """Maps with more than 32 offsets on the fp32 block engine (Sec. 5.1:
    the 3^4 tesseract's 81 offsets, the 5^3 cube's 125, and 33 offsets): one plan per
    range of consecutive offsets, the ranges' sums added in range order, in
    the forward pass and the input gradient."""
    if region == "tesseract":
        coords, offs, ci, co = WL.random_coords(171, 3000, 4, -5, 5, batch=1), regions.hypercube(3, 4), 32, 32
    elif region == "cube5":
        coords, offs, ci, co = WL.random_coords(172, 2500, 3, -9, 9, batch=2), regions.hypercube(5, 3), 16, 32
    else:
        two = np.concatenate([2 * np.eye(3, dtype=np.int32), -2 * np.eye(3, dtype=np.int32)])
        offs = np.concatenate([regions.hypercube(3, 3), two])   # the cube and six axis steps of 2: 33
        coords, ci, co = WL.random_coords(173, 3000, 3, -10, 10, batch=2), 32, 16
    K = len(offs)
    assert K > 32 and gsc.gsc_plan_ranges(K) == -(-K // 32)
    assert gsc.gsc_conv_block_engine(gsc.GSC_F32, ci, co, K) and gsc.gsc_conv_block_engine(gsc.GSC_F32, co, ci, K)
    _say(f"[gpu] block engine over offset ranges: {region} K={K} {ci}->{co}")
    _plan_case(coords, ci, co, offs, 174 + K)


def test_dilated_kernel():
    """Dilation (Sec. 3.1: the offset set is arbitrary): the 3^3 cube with
    offsets scaled by 2 and by 3."""
    coords = WL.random_coords(85, 3000, 3, -12, 12, batch=2)
    _conv_case(coords, 8, 16, regions.hypercube(3, 3) * 2, 85)
    _conv_case(coords, 16, 8, regions.hypercube(3, 3) * 3, 86)


def test_arbitrary_output_coordinates():
    """Generalized convolution onto a caller-given output set (Sec. 4.2: the
    output coordinates may be arbitrary): half of them input sites, half new
    sites (some with no input in reach); backward through the role-reversed
    map built from the output table."""
    cin = WL.random_coords(87, 2500, 3, -10, 10, batch=2)
    cnew = WL.random_coords(88, 2000, 3, -14, 14, batch=2)
    seen = {tuple(r) for r in cin[:1200].tolist()}
    cout = np.concatenate([cin[:1200], np.array([r for r in cnew.tolist() if tuple(r) not in seen], np.int32)])
    offs = regions.hypercube(3, 3)
    X, _ = WL.random_features(87, len(cin), 8)
    W, _ = WL.random_weights(87, len(offs), 8, 12)
    G, _ = WL.random_features(88, len(cout), 12)
    tin, tout = _t(cin), _t(cout)
    table_in = gsc.gsc_coords_build(tin)
    table_out = gsc.gsc_coords_build(tout)
    km = gsc.gsc_kernel_map(table_in, tout, offs)
    tm = gsc.gsc_kernel_map(table_out, tin, -offs)
    Y = gsc.gsc_sparse_conv_fwd(_t(X, torch.float32), _t(W, torch.float32), km)
    dX, dW = gsc.gsc_sparse_conv_bwd(_t(X, torch.float32), _t(W, torch.float32), _t(G, torch.float32), km, tm,
                                     np.arange(len(offs)))
    torch.cuda.synchronize()
    m = O.kernel_map(cin, cout, offs)
    maps_equal_exact(gpu_pairs(km), m)
    maps_equal_exact(gpu_pairs(tm), O.transposed_map(m))
    assert rel_err(to_np(Y), O.conv_forward(X, W, m, len(cout))) <= TOL["f32"]
    dXr, dWr = O.conv_backward(X, W, G, m)
    assert rel_err(to_np(dX), dXr) <= TOL["f32"]
    assert rel_err(to_np(dW), dWr) <= TOL["f32"]


def test_centre_only_identity_exact():
    coords = WL.random_coords(79, 1000, 3, -20, 20, batch=2)
    c = _t(coords)
    table = gsc.gsc_coords_build(c)
    km = gsc.gsc_kernel_map(table, c, np.zeros((1, 3), np.int32))
    X = torch.randn((len(coords), 32), device=DEV)
    Y = gsc.gsc_sparse_conv_fwd(X, torch.eye(32, device=DEV)[None].contiguous(), km)
    torch.cuda.synchronize()
    assert torch.equal(Y, X)


def test_stride_coords_floor_and_order():
    coords = WL.random_coords(81, 4000, 3, -9, 9, batch=3)
    out, out_table = gsc.gsc_coords_stride(_t(coords), 2)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = O.output_coordinates(coords, 2)
    assert {tuple(r) for r in got.tolist()} == {tuple(r) for r in ref.tolist()}
    assert len(got) == len(ref)
    # deterministic order: first input row producing each output
    first = {}
    for r, row in enumerate(coords.tolist()):
        key = (row[0],) + tuple((v // 2) * 2 for v in row[1:])
        first.setdefault(key, r)
    assert [first[tuple(r)] for r in got.tolist()] == sorted(first.values())
    # the output table answers queries for the output coordinates
    km = gsc.gsc_kernel_map(out_table, out, np.zeros((1, 3), np.int32))
    assert np.array_equal(gpu_pairs(km)[0][0], np.arange(len(got)))


@pytest.mark.parametrize("lead", [0, 3, 61, 250])
def test_stride_order_with_runs_across_lanes(lead):
    """Strided output coordinates from rows whose equal strided keys come in
    runs (the 8 fine voxels of each coarse cell consecutively, as sorted
    scene rows give them), shifted by ``lead`` singleton rows so that runs
    cross the 64-lane and 256-thread boundaries: the output keeps the order of
    each key's first input row exactly, and every input row's stride-2 map
    pair points at its own cell."""
    rng = np.random.default_rng(186 + lead)
    cells = np.unique(rng.integers(-20, 20, size=(700, 3)), axis=0) * 2   # coarse cells
    rng.shuffle(cells)
    fine = (cells[:, None, :] + regions.hypercube(2, 3)[None, :, :]).reshape(-1, 3)
    singles = np.stack([np.full(lead, 101), np.arange(lead) * 2, np.zeros(lead)], axis=1) if lead else np.zeros((0, 3))
    xyz = np.concatenate([singles, fine]).astype(np.int32)
    coords = np.concatenate([np.zeros((len(xyz), 1), np.int32), xyz], axis=1)
    out, out_table = gsc.gsc_coords_stride(_t(coords), 2)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    first = {}
    for r, row in enumerate(coords.tolist()):
        key = (row[0],) + tuple((v // 2) * 2 for v in row[1:])
        first.setdefault(key, r)
    order = sorted(first, key=first.get)
    assert got.tolist() == [list(k) for k in order]
    # every fine row pairs with the cell it lies in
    km = gsc.gsc_kernel_map(gsc.gsc_coords_build(_t(coords)), out, regions.hypercube(2, 3))
    ref = O.kernel_map(coords, got, O.hypercube(2, 3))
    maps_equal_exact(gpu_pairs(km), ref)


def test_stride_deferred_matches_sync(monkeypatch):
    """The deferred strided output coordinates (gsc_coords_stride_async, its
    count read after a map over its table was enqueued) equal the
    synchronous call's rows and table; a failed deferred build reports EFULL
    from its result."""
    coords = WL.random_coords(84, 5000, 3, -16, 16, batch=2)
    c = _t(coords)
    offs = -regions.hypercube(2, 3)
    ref_out, ref_table = gsc.gsc_coords_stride(c, 2)
    ref_pairs = gpu_pairs(gsc.gsc_kernel_map(ref_table, c, offs))
    pending = gsc.gsc_coords_stride(c, 2, defer=True)
    km = gsc.gsc_kernel_map(pending.out_table, c, offs, sync=False)   # needs only the output table
    out, table = pending.finish()
    assert torch.equal(out, ref_out)
    for (i1, o1), (i2, o2) in zip(gpu_pairs(km), ref_pairs):
        assert np.array_equal(i1, i2) and np.array_equal(o1, o2)
    monkeypatch.setenv("GSC_TABLE_CAP_LIMIT", "64")   # 64 slots for the ~2,500 output rows
    pending = gsc.gsc_coords_stride(c, 2, defer=True)
    with pytest.raises(gsc.GscError) as e:
        pending.finish()
    assert e.value.code == gsc.GSC_EFULL


def test_stride_then_second_level():
    coords = WL.random_coords(82, 6000, 3, -17, 17, batch=2)
    c = _t(coords)
    o1, t1 = gsc.gsc_coords_stride(c, 2)
    o2, t2 = gsc.gsc_coords_stride(o1, 4)
    torch.cuda.synchronize()
    r1 = O.output_coordinates(coords, 2)
    r2 = O.output_coordinates(r1, 4)
    assert {tuple(r) for r in o2.cpu().numpy().tolist()} == {tuple(r) for r in r2.tolist()}
    # stride-4 level map from the stride-2 level: tensor stride 2, size-2 kernel
    km = gsc.gsc_kernel_map(t1, o2, regions.hypercube(2, 3), tensor_stride=2)
    g1, g2 = o1.cpu().numpy(), o2.cpu().numpy()
    from parity import row_perm
    p1, p2 = row_perm(g1, r1), row_perm(g2, r2)
    ref = O.kernel_map(r1, r2, O.hypercube(2, 3), 2)
    maps_equal_exact(gpu_pairs(km), ref, out_perm=p2, in_perm=p1)


def test_async_map_matches_sync():
    coords = WL.random_coords(83, 6000, 3, -15, 15, batch=3)
    c = _t(coords)
    table = gsc.gsc_coords_build(c, sync=False)
    gsc.gsc_table_status(table)
    offs = regions.hypercube(3, 3)
    ks = gsc.gsc_kernel_map(table, c, offs)
    ka = gsc.gsc_kernel_map(table, c, offs, sync=False, dense=True)
    assert ka.n_pairs is None and ka.count() == ks.n_pairs
    for (a, b), (x, y) in zip(gpu_pairs(ka), gpu_pairs(ks)):
        assert np.array_equal(a, x) and np.array_equal(b, y)
    check_gidx(ka)
    dense = ka.nbr.cpu().numpy()
    for k, (i, o) in enumerate(gpu_pairs(ks)):
        col = np.full(len(coords), -1, np.int64)
        col[o] = i
        assert np.array_equal(dense[k], col)


def test_async_build_reports_duplicate_later():
    c = _t(np.array([[0, 1, 2, 3], [0, 4, 5, 6], [0, 1, 2, 3]], np.int32))
    table = gsc.gsc_coords_build(c, sync=False)        # enqueued only: no error yet
    km = gsc.gsc_kernel_map(table, c, regions.hypercube(3, 3), sync=False)
    assert km.count() == 0                             # a failed table yields an empty map
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_table_status(table)
    assert e.value.code == gsc.GSC_EDUP


# --------------------------------------------------------------------------- #
# pooling (Sec. 4.3, Alg. 3; Sec. 4.4, Alg. 4)
# --------------------------------------------------------------------------- #
def _pool_case(seed, scale, window, extra_outputs=0, C=32):
    """A scene, its stride-2 output coordinates (plus ``extra_outputs`` far
    away rows that no input reaches), the pooling maps on the GPU (forward
    and role-reversed, dense forms) and the oracle's map."""
    wl = WL.make_workload(1, scale=scale)
    coords = torch.from_numpy(wl.coords).to(DEV)
    table = gsc.gsc_coords_build(coords)
    out, out_table = gsc.gsc_coords_stride(coords, 2)
    if extra_outputs:
        far = out[:extra_outputs].clone()
        far[:, 1] += 10_000
        out = torch.cat([out, far]).contiguous()
        out_table = gsc.gsc_coords_build(out)
    offs = regions.hypercube(window, 3)
    fmap = gsc.gsc_kernel_map(table, out, offs, dense=True)
    tmap = gsc.transposed_kernel_map(out_table, coords, offs, dense=True)
    X, _ = WL.random_features(seed, wl.n, C)
    G, _ = WL.random_features(seed + 1, out.shape[0], C)
    ref_maps = O.kernel_map(wl.coords, to_np(out), np.asarray(offs))
    return wl, coords, out, fmap, tmap, X, G, ref_maps


@pytest.mark.parametrize("window,C", [(2, 32), (3, 32), (3, 6)])
@pytest.mark.parametrize("mode", ["max", "avg", "sum"])
def test_pool_parity(mode, window, C):
    """Four channels per lane (C = 32) and one (C = 6)."""
    wl, coords, out, fmap, tmap, X, G, ref_maps = _pool_case(81 + window, 0.3, window, extra_outputs=5, C=C)
    n_out = out.shape[0]
    _say(f"[gpu] pool {mode} window {window} C {C}: n_in={wl.n} n_out={n_out}")
    Xd = torch.from_numpy(X).to(DEV)
    p = gsc.gsc_sparse_pool_fwd(Xd, fmap, mode)
    dX = gsc.gsc_sparse_pool_bwd(torch.from_numpy(G).to(DEV), tmap, mode, p)
    torch.cuda.synchronize()
    Y, arg, N = O.pool_forward(X, ref_maps, n_out, mode)
    assert np.array_equal(to_np(p.cnt), N)
    assert N[-5:].max() == 0 and np.all(to_np(p.Y)[-5:] == 0)      # outputs no input reaches
    assert rel_err(to_np(p.Y), Y) <= TOL["f32"]
    if mode == "max":
        assert np.array_equal(to_np(p.arg), arg)                   # the same input wins, bit for bit
        assert np.all(to_np(p.Y) == X[np.maximum(arg, 0), np.arange(C)[None, :]] * (arg >= 0))
    ref_dX = O.pool_backward(G, ref_maps, wl.n, mode, arg, N)
    assert rel_err(to_np(dX), ref_dX) <= TOL["f32"]


@pytest.mark.parametrize("window", [2, 3])
@pytest.mark.parametrize("mode", ["avg", "sum"])
def test_unpool_parity(mode, window):
    """Unpooling (Sec. 4.4, transposed pooling): gsc_sparse_pool_fwd on the
    role-reversed map takes coarse features back to the fine rows, and
    gsc_sparse_pool_bwd on the forward map gives its gradient."""
    wl, coords, out, fmap, tmap, _, _, ref_maps = _pool_case(95 + window, 0.3, window, extra_outputs=5)
    n_out = out.shape[0]
    _say(f"[gpu] unpool {mode} window {window}: n_coarse={n_out} n_fine={wl.n}")
    Xc, _ = WL.random_features(97, n_out, 32)
    Gf, _ = WL.random_features(98, wl.n, 32)
    u = gsc.gsc_sparse_pool_fwd(torch.from_numpy(Xc).to(DEV), tmap, mode)
    dXc = gsc.gsc_sparse_pool_bwd(torch.from_numpy(Gf).to(DEV), fmap, mode, u)
    torch.cuda.synchronize()
    U, _, N = O.unpool_forward(Xc, ref_maps, wl.n, mode)
    assert np.array_equal(to_np(u.cnt), N) and N.min() >= 1
    assert rel_err(to_np(u.Y), U) <= TOL["f32"]
    ref = O.unpool_backward(Gf, ref_maps, n_out, mode, N)
    assert np.all(to_np(dXc)[-5:] == 0)                               # coarse rows no fine row reaches
    assert rel_err(to_np(dXc), ref) <= TOL["f32"]


@pytest.mark.parametrize("mode", ["max", "avg", "sum"])
def test_global_pool_parity(mode):
    c = WL.random_coords(91, 3000, 3, -20, 21, batch=3)
    X, _ = WL.random_features(91, len(c), 40)
    G, _ = WL.random_features(92, 3, 40)
    cd = torch.from_numpy(c).to(DEV)
    p = gsc.gsc_global_pool_fwd(torch.from_numpy(X).to(DEV), cd, 3, mode)
    dX = gsc.gsc_global_pool_bwd(torch.from_numpy(G).to(DEV), cd, mode, p)
    torch.cuda.synchronize()
    Y, arg, N = O.global_pool_forward(X, c[:, 0], 3, mode)
    assert np.array_equal(to_np(p.cnt), N)
    assert rel_err(to_np(p.Y), Y) <= TOL["f32"]
    if mode == "max":
        assert np.array_equal(to_np(p.arg), arg)
    assert rel_err(to_np(dX), O.global_pool_backward(G, c[:, 0], mode, arg, N)) <= TOL["f32"]


# --------------------------------------------------------------------------- #
# sparse tensor quantization (Sec. 4.1, Alg. 1)
# --------------------------------------------------------------------------- #
def _quant_compare(P, b, voxel, L):
    q = gsc.gsc_quantize(_t(P, torch.float32), voxel, batch=_t(b), labels=None if L is None else _t(L))
    torch.cuda.synchronize()
    C, rep, lab, inv = O.quantize(P, b, voxel, L)
    gc = q.coords.cpu().numpy().astype(np.int64)
    grep, ginv = q.rep.cpu().numpy().astype(np.int64), q.inverse.cpu().numpy().astype(np.int64)
    assert len(gc) == len(C)
    # rows come in the order of their first points; the oracle's in key order
    order = np.argsort(grep)
    oc = np.argsort(rep)
    assert np.array_equal(gc[order], C[oc]) and np.array_equal(grep[order], rep[oc])
    assert np.array_equal(grep, np.sort(grep))                      # first-point order
    if L is not None:
        assert np.array_equal(q.labels.cpu().numpy()[order], lab[oc])
    # every point lands in the voxel of its own coordinate
    assert np.array_equal(gc[ginv], C[inv])
    return q


def test_quantize_golden_on_gpu():
    pts, b, L = [], [], []
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "quantize_small.txt")):
        f = line.split("#")[0].split()
        if f and f[0] == "P":
            b.append(int(f[2]))
            pts.append([float(x) for x in f[3:6]])
            L.append(int(f[6]))
    _quant_compare(np.array(pts, np.float32), np.array(b, np.int32), 0.5, np.array(L, np.int32))


def test_quantize_exact_floor_on_gpu():
    """Voxel indices at voxel sizes that are not powers of two: the floor of the
    exact quotient (hand-worked golden file; 0.7 / 0.1 -> 6)."""
    rows = []
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "quantize_exact_floor.txt")):
        f = line.split("#")[0].split()
        if f:
            rows.append((np.float32(f[0]), np.float32(f[1]), int(f[4])))
    for v in sorted({r[1] for r in rows}):
        sel = [(p, want) for p, vv, want in rows if vv == v]
        P = np.array([[p, p] for p, _ in sel], np.float32)
        q = gsc.gsc_quantize(_t(P, torch.float32), (float(v), float(v)), batch=_t(np.arange(len(sel), dtype=np.int32)))
        torch.cuda.synchronize()
        got = q.coords.cpu().numpy()[q.inverse.cpu().numpy()]
        assert got[:, 1].tolist() == [w for _, w in sel] and got[:, 2].tolist() == [w for _, w in sel], v
        _quant_compare(P, np.arange(len(sel), dtype=np.int32), (float(v), float(v)), None)


def test_quantize_matches_workload_voxels():
    """The GPU quantization of the indoor-scene workload's own points (two
    scenes of 161,000 points at 2 cm) gives exactly the workload's voxel set:
    the generator and the kernel floor the same exact quotient."""
    pts, bs = [], []
    n = WL.SCENE_POINTS_2CM
    for bi in range(2):
        geom = WL.draw_scene(WL.rng_for(1, WL.S_GEOM, bi))
        p = WL.sample_points(geom, WL.rng_for(1, WL.S_GEOM, bi, 1), n)
        pts.append(np.asarray(p, np.float32))
        bs.append(np.full(len(p), bi, np.int32))
    q = gsc.gsc_quantize(_t(np.concatenate(pts), torch.float32), 0.02, batch=_t(np.concatenate(bs)))
    torch.cuda.synchronize()
    got = q.coords.cpu().numpy()
    ref = WL.make_workload(1).coords
    _say(f"  scene points {2 * n} -> voxels {len(got)} (workload {len(ref)})")
    assert len(got) == len(ref)
    assert np.array_equal(np.unique(got, axis=0), ref)


def test_quantize_random_and_scene():
    rng = np.random.default_rng(95)
    P = rng.uniform(-4, 4, size=(60000, 3)).astype(np.float32)
    b = rng.integers(0, 3, size=60000).astype(np.int32)
    L = rng.integers(0, 4, size=60000).astype(np.int32)
    _quant_compare(P, b, 0.1, L)
    _quant_compare(P, b, (0.05, 0.1, 0.2), None)                    # anisotropic voxels, no labels
    # the synthetic indoor scene's points (two scenes) at 2 cm
    pts, bs = [], []
    for bi in range(2):
        geom = WL.draw_scene(WL.rng_for(1, WL.S_GEOM, bi), scale=0.5)
        p = WL.sample_points(geom, WL.rng_for(1, WL.S_GEOM, bi, 1), 40000)
        pts.append(np.asarray(p, np.float32))
        bs.append(np.full(len(p), bi, np.int32))
    q = _quant_compare(np.concatenate(pts), np.concatenate(bs), 0.02, None)
    _say(f"  scene points {sum(len(p) for p in pts)} -> voxels {q.coords.shape[0]}")


def test_quantize_wide_keys():
    """Quantization of points whose voxel box needs more than 62 key bits
    (clusters of points spread over +-2e5 m at 1 mm voxels: 29 bits per axis)
    goes through the wide key form and still matches the oracle."""
    rng = np.random.default_rng(97)
    centres = rng.uniform(-2e5, 2e5, size=(1500, 3))
    P = (np.repeat(centres, 4, axis=0) + rng.uniform(-2e-3, 2e-3, size=(6000, 3))).astype(np.float32)
    b = rng.integers(0, 3, size=6000).astype(np.int32)
    L = rng.integers(0, 3, size=6000).astype(np.int32)
    v = np.floor(P.astype(np.float64) / np.float64(np.float32(1e-3)))
    bits = sum(int(s).bit_length() for s in (v.max(0) - v.min(0)).astype(np.int64)) + int(b.max()).bit_length()
    assert 62 < bits <= 92
    _say(f"[gpu] quantize with wide keys: {bits} key bits")
    q = _quant_compare(P, b, 1e-3, L)
    assert q.coords.shape[0] < len(P)   # clustered points share voxels


# --------------------------------------------------------------------------- #
# forward with the per-channel affine map and ReLU fused (Sec. 4.5)
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("dtype,ci,co,region,planned", [
    ("f32", 32, 32, "cube3", True), ("f32", 16, 64, "cube2", True), ("f32", 32, 32, "cube3", False),
    ("f32", 3, 16, "cube3", False), ("bf16", 256, 256, "cube3", True), ("bf16", 64, 128, "cube2", True),
    ("bf16", 256, 256, "cube3", False), ("bf16", 48, 80, "cube3", False), ("f32", 16, 16, "cube5", True)])
@pytest.mark.parametrize("mode", ["bn_relu", "scale_only", "shift_relu", "none"])
def test_conv_affine_epilogue(dtype, ci, co, region, planned, mode):
    """gsc_sparse_conv_fwd_affine against the oracle's convolution followed by
    batch normalisation (coefficients from the oracle's batch statistics) and
    ReLU; with no coefficients and no activation it is the plain forward."""
    _say(f"[gpu] affine epilogue {dtype} {ci}->{co} {region} planned={planned} {mode}")
    coords = WL.random_coords(160 + ci + co, 2600, 3, -12, 12, batch=2)
    offs = regions.hypercube(int(region[-1]), 3)
    X, Xb = WL.random_features(161, len(coords), ci, dtype)
    W, Wb = WL.random_weights(162, len(offs), ci, co, dtype)
    if dtype == "bf16":
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
        tX, tW = dev(Xb), dev(Wb)
    else:
        tX, tW = _t(X, torch.float32), _t(W, torch.float32)
    table = gsc.gsc_coords_build(_t(coords))
    km = gsc.gsc_kernel_map(table, _t(coords), offs, dense=planned)
    if planned:
        km = gsc.gsc_conv_plan(km)
        assert gsc.gsc_conv_block_engine(gsc.GSC_BF16 if dtype == "bf16" else gsc.GSC_F32, ci, co, len(offs))
    m = O.kernel_map(coords, coords, np.asarray(offs))
    S = O.conv_forward(X, W, m, len(coords))
    rng = np.random.default_rng(163)
    scale, shift = O.batchnorm_coefficients(S, rng.uniform(0.5, 2.0, co), rng.uniform(-0.5, 0.5, co))
    scale, shift = scale.astype(np.float32), shift.astype(np.float32)
    relu = mode in ("bn_relu", "shift_relu")
    sc = scale if mode in ("bn_relu", "scale_only") else None
    sh = shift if mode in ("bn_relu", "shift_relu") else None
    Y = gsc.gsc_sparse_conv_fwd_affine(tX, tW, km, None if sc is None else _t(sc, torch.float32),
                                       None if sh is None else _t(sh, torch.float32), relu=relu)
    torch.cuda.synchronize()
    ref = O.affine_act(S, sc, sh, relu)
    got = to_np(Y)
    assert rel_err(got, ref) <= TOL[dtype]
    if relu:
        assert np.all(got >= 0)
    if mode == "none":
        # the block engines add in a fixed order; the general row-form kernel
        # does not, so there only the tolerance holds between two calls
        plain = gsc.gsc_sparse_conv_fwd(tX, tW, km)
        torch.cuda.synchronize()
        if planned:
            assert torch.equal(plain, Y)
        else:
            assert rel_err(got, to_np(plain)) <= TOL[dtype]


def test_conv_affine_no_input_rows():
    """Outputs that no input reaches hold act(shift); an input with no rows
    gives the same through the engines' zero fill."""
    cin = np.array([[0, 100, 100, 100], [0, 101, 100, 100]], np.int32)
    cout = np.array([[0, 0, 0, 0], [0, 1, 1, 1], [0, 100, 100, 99]], np.int32)
    shift = np.linspace(-1, 1, 32).astype(np.float32)
    for planned in (False, True):
        km = gsc.gsc_kernel_map(gsc.gsc_coords_build(_t(cin)), _t(cout), regions.hypercube(3, 3), dense=planned)
        km = gsc.gsc_conv_plan(km) if planned else km
        X = _t(WL.random_features(171, 2, 16)[0], torch.float32)
        W = _t(WL.random_weights(172, 27, 16, 32)[0], torch.float32)
        Y = gsc.gsc_sparse_conv_fwd_affine(X, W, km, None, _t(shift, torch.float32), relu=True)
        torch.cuda.synchronize()
        ref = O.affine_act(O.conv_forward(to_np(X), to_np(W), O.kernel_map(cin, cout, O.hypercube(3, 3)), 3),
                           None, shift, True)
        assert rel_err(to_np(Y), ref) <= TOL["f32"]
        assert np.array_equal(to_np(Y)[:2], np.broadcast_to(np.maximum(shift, 0), (2, 32)))
    km0 = gsc.gsc_conv_plan(gsc.gsc_kernel_map(gsc.gsc_coords_build(torch.empty((0, 4), dtype=torch.int32,
                                                                                device=DEV)),
                                               _t(cout), regions.hypercube(3, 3), dense=True))
    Y0 = gsc.gsc_sparse_conv_fwd_affine(torch.empty((0, 16), device=DEV), W, km0, None, _t(shift, torch.float32),
                                        relu=True)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(Y0), np.broadcast_to(np.maximum(shift, 0), (3, 32)))


def test_block_engines_at_32_offsets():
    """K = 32, the widest region one block plan takes (masks use all 32 bits;
    the last offset is bit 31), on both engines, and K = 33, which the fp32
    engine takes in two plan ranges and the bf16 path on the row form."""
    extra = np.array([[2, 0, 0], [-2, 0, 0], [0, 2, 0], [0, -2, 0], [0, 0, 2], [0, 0, -2]], np.int32)
    offs32 = np.concatenate([regions.hypercube(3, 3), extra[:5]]).astype(np.int32)
    offs33 = np.concatenate([regions.hypercube(3, 3), extra]).astype(np.int32)
    coords = WL.random_coords(181, 3000, 3, -9, 9, batch=2)
    assert gsc.gsc_conv_block_engine(gsc.GSC_F32, 32, 32, 32) and gsc.gsc_conv_block_engine(gsc.GSC_BF16, 64, 64, 32)
    assert gsc.gsc_conv_block_engine(gsc.GSC_F32, 32, 32, 33) and gsc.gsc_plan_ranges(33) == 2
    assert not gsc.gsc_conv_block_engine(gsc.GSC_BF16, 64, 64, 33)
    _say("[gpu] block engines at K = 32 (fp32 32->32, bf16 64->64); K = 33 in two ranges and on the row form")
    _plan_case(coords, 32, 32, offs32, 182)
    _plan_case(coords, 64, 64, offs32, 183, dtype="bf16")
    _conv_case(coords, 16, 16, offs33, 184)
    _conv_case(coords, 64, 64, offs33, 185, dtype="bf16")


def _trilateral_7d():
    """A trilateral region of the 7D space-time-chroma space (Sec. 6): the
    spatial 3^3 cube plus the temporal and the three colour crosses (35)."""
    tri = {tuple(o) + (0,) * 4 for o in regions.hypercube(3, 3).tolist()}
    for ax in range(3, 7):
        for s in (-1, 1):
            o = [0] * 7
            o[ax] = s
            tri.add(tuple(o))
    return np.array(sorted(tri), np.int32)


def _key_bits(coords):
    span = coords.astype(np.int64).max(0) - coords.astype(np.int64).min(0)
    return sum(int(s).bit_length() for s in span)


def test_7d_space_time_chroma():
    """7D coordinates (b, x, y, z, t, r, g, b) as the space-time-chroma
    convolution of Sec. 6 uses them, with keys inside the 62-bit packing: the
    7D cross (15 offsets) and a trilateral region (35 offsets, two plan
    ranges) on the block engine and on the row form."""
    coords = WL.random_coords(191, 4000, 7, -2, 2, batch=2)
    cross = regions.hypercross(3, 7)
    tri = _trilateral_7d()
    assert len(cross) == 15 and len(tri) == 35 and regions.is_symmetric(tri)
    _say("[gpu] 7D space-time-chroma (small box): cross (15) and trilateral (35), block engine and row form")
    _plan_case(coords, 16, 32, cross, 192)
    _plan_case(coords, 16, 16, tri, 195)
    _conv_case(coords, 16, 16, cross, 193)
    _conv_case(coords, 8, 16, tri, 194)


def test_7d_space_time_chroma_real_extents():
    """7D rows at a real scene's extents (Sec. 6): the 2 cm voxels of an
    indoor scene over three frames with RGB channels of 0..255 (52 key bits),
    through the 7D cross and the trilateral region on the block engine and
    the row form."""
    coords = WL.space_time_chroma_coords(1)
    bits = _key_bits(coords)
    span = coords.max(0) - coords.min(0)
    assert bits >= 50 and np.all(span[5:] >= 250) and span[4] == 2 and np.all(span[1:4] >= 150)
    cross, tri = regions.hypercross(3, 7), _trilateral_7d()
    _say(f"[gpu] 7D space-time-chroma, real extents: {len(coords)} rows, {bits} key bits")
    _plan_case(coords, 16, 32, cross, 196)
    _plan_case(coords, 16, 16, tri, 197)
    _conv_case(coords, 16, 16, cross, 198)
    _conv_case(coords, 8, 16, tri, 199)


def test_7d_key_width_limit():
    """The packed key's limits on 7D rows: the space-time-chroma rows with
    their spatial axes scaled until the box needs exactly 62 bits (the widest
    key held in one 64-bit word), 63 bits (the wide form: 62 bits in the
    slot's key word, the rest in its second word) and 92 bits (the widest key)
    still map exactly; one bit more is rejected with ERANGE (the table is not
    built)."""
    base = WL.space_time_chroma_coords(1).astype(np.int64)
    at = base.copy()
    at[:, 1] *= 16
    at[:, 2:4] *= 8
    over = at.copy()
    over[:, 3] *= 2
    top = at.copy()
    top[:, 1:4] *= 1024
    past = top.copy()
    past[:, 3] *= 2
    assert [_key_bits(a) for a in (at, over, top, past)] == [62, 63, 92, 93]
    _say("[gpu] 7D key width: 62, 63 and 92 bits map, 93 is rejected")
    offs = _trilateral_7d()
    for a in (at, over, top):
        a = a.astype(np.int32)
        c = _t(a)
        km = gsc.gsc_kernel_map(gsc.gsc_coords_build(c), c, offs)
        maps_equal_exact(gpu_pairs(km), O.kernel_map(a, a, offs))
    with pytest.raises(gsc.GscError) as e:
        gsc.gsc_coords_build(_t(past.astype(np.int32)))
    assert e.value.code == gsc.GSC_ERANGE


def _wide_7d_rows():
    """The space-time-chroma rows of one building seen twice: the scene's
    crops and the same crops 2^13 voxels (164 m) further along x, y and z, a
    box of 68 key bits."""
    base = WL.space_time_chroma_coords(1).astype(np.int64)
    far = base.copy()
    far[:, 1:4] += 1 << 13
    rows = np.concatenate([base, far]).astype(np.int32)
    assert 62 < _key_bits(rows) <= 92
    return rows


def test_7d_wide_keys():
    """Rows whose box needs more than 62 key bits take the wide key form:
    exact maps over the 7D cross and the trilateral region, and convolutions
    on the block engine and the row form."""
    coords = _wide_7d_rows()
    cross, tri = regions.hypercross(3, 7), _trilateral_7d()
    _say(f"[gpu] 7D wide keys: {len(coords)} rows, {_key_bits(coords)} key bits")
    c = _t(coords)
    table = gsc.gsc_coords_build(c)
    for offs in (cross, tri):
        maps_equal_exact(gpu_pairs(gsc.gsc_kernel_map(table, c, offs)), O.kernel_map(coords, coords, offs))
    _plan_case(coords, 16, 32, cross, 203)
    _conv_case(coords, 8, 16, tri, 204)


def test_7d_wide_keys_strided():
    """Strided output coordinates of wide-key rows: the oracle's set, in
    first-input-row order, and an output table that answers for them."""
    coords = _wide_7d_rows()
    _say(f"[gpu] 7D wide keys, stride 2: {len(coords)} rows")
    out, out_table = gsc.gsc_coords_stride(_t(coords), 2)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = O.output_coordinates(coords, 2)
    assert len(got) == len(ref) and {tuple(r) for r in got.tolist()} == {tuple(r) for r in ref.tolist()}
    first = {}
    for r, row in enumerate(coords.tolist()):
        first.setdefault((row[0],) + tuple((v // 2) * 2 for v in row[1:]), r)
    assert [first[tuple(r)] for r in got.tolist()] == sorted(first.values())
    km = gsc.gsc_kernel_map(out_table, out, np.zeros((1, 7), np.int32))
    assert np.array_equal(gpu_pairs(km)[0][0], np.arange(len(got)))


# --------------------------------------------------------------------------- #
# the dX map from the pairs alone, and the backward from the forward map
# --------------------------------------------------------------------------- #
def _strided_case(seed):
    """A stride-2 downsampling map (size-2 kernel): fine coordinates in, the
    oracle's coarse coordinates out; returns the GPU map and the oracle's."""
    fine = WL.random_coords(seed, 5000, 3, -16, 16, batch=2)
    coarse = O.output_coordinates(fine, 2).astype(np.int32)
    offs = regions.hypercube(2, 3)
    km = gsc.gsc_kernel_map(gsc.gsc_coords_build(_t(fine)), _t(coarse), offs)
    return fine, coarse, km, O.kernel_map(fine, coarse, np.asarray(offs))


@pytest.mark.parametrize("case", ["cube3", "asymmetric", "stride2"])
def test_kernel_map_transpose_matches_table_query(case):
    """The role-reversed map built from a map's pairs (Sec. 4.2) equals the one
    the table query with negated offsets gives: pairs, segments, group index
    and dense form, bit for bit."""
    if case == "stride2":
        fine, coarse, km, m = _strided_case(176)
        n_rev = len(fine)
        ref = gsc.transposed_kernel_map(gsc.gsc_coords_build(_t(coarse)), _t(fine), km.offsets, tensor_stride=1,
                                        dense=True)
    else:
        coords = WL.random_coords(177, 4000, 3, -12, 12, batch=2)
        c = _t(coords)
        offs = regions.hypercube(3, 3) if case == "cube3" else np.array(
            [[0, 0, 0], [1, 0, 0], [0, 2, 0], [1, 1, -1], [-2, 0, 1]], np.int32)
        table = gsc.gsc_coords_build(c)
        km = gsc.gsc_kernel_map(table, c, offs)
        ref = gsc.transposed_kernel_map(table, c, offs, dense=True)
        n_rev = len(coords)
        m = O.kernel_map(coords, coords, np.asarray(offs))
    _say(f"[gpu] map transpose {case}: {km.n_pairs} pairs")
    tm = gsc.gsc_kernel_map_transpose(km, n_rev)
    torch.cuda.synchronize()
    maps_equal_exact(gpu_pairs(tm), O.transposed_map(m))
    for (a, b), (x, y) in zip(gpu_pairs(tm), gpu_pairs(ref)):
        assert np.array_equal(a, x) and np.array_equal(b, y)
    assert torch.equal(tm.seg.cpu(), ref.seg.cpu())
    assert torch.equal(tm.gidx.cpu(), ref.gidx.cpu())
    assert torch.equal(tm.nbr.cpu(), ref.nbr.cpu())


@pytest.mark.parametrize("dtype,ci,co,case,transpose", [
    ("f32", 32, 32, "cube3", False), ("f32", 16, 8, "stride2", False), ("f32", 8, 16, "stride2", True),
    ("bf16", 64, 64, "cube3", False), ("bf16", 48, 24, "stride2", True), ("f32", 3, 5, "cube3", False)])
def test_conv_bwd_from_forward_map(dtype, ci, co, case, transpose):
    """gsc_sparse_conv_bwd_fwdmap (the forward map plus a transpose flag; the
    library builds the dX map and its plan) against the oracle's gradients of
    the forward (transpose = 0) or the transposed convolution on the map."""
    if case == "stride2":
        fine, coarse, km, m = _strided_case(178)
        n_fine, n_coarse = len(fine), len(coarse)
    else:
        coords = WL.random_coords(179, 3000, 3, -10, 10, batch=2)
        c = _t(coords)
        offs = regions.hypercube(3, 3)
        km = gsc.gsc_kernel_map(gsc.gsc_coords_build(c), c, offs)
        m = O.kernel_map(coords, coords, np.asarray(offs))
        n_fine = n_coarse = len(coords)
    maps_equal_exact(gpu_pairs(km), m)
    n_x, n_y = (n_coarse, n_fine) if transpose else (n_fine, n_coarse)
    maps = O.transposed_map(m) if transpose else m
    X, Xb = WL.random_features(180, n_x, ci, dtype)
    W, Wb = WL.random_weights(181, km.K, ci, co, dtype)
    G, Gb = WL.random_features(182, n_y, co, dtype)
    if dtype == "bf16":
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
        tX, tW, tG = dev(Xb), dev(Wb), dev(Gb)
    else:
        tX, tW, tG = _t(X, torch.float32), _t(W, torch.float32), _t(G, torch.float32)
    _say(f"[gpu] bwd from the forward map: {dtype} {ci}->{co} {case} transpose={transpose}")
    dX, dW = gsc.gsc_sparse_conv_bwd_fwdmap(tX, tW, tG, km, transpose=transpose)
    torch.cuda.synchronize()
    dXr, dWr = O.conv_backward(X, W, G, maps)
    assert rel_err(to_np(dX), dXr) <= TOL[dtype]
    assert rel_err(to_np(dW), dWr) <= TOL[dtype]


# --------------------------------------------------------------------------- #
# training through the fused epilogue (Sec. 4.5): its backward, then the conv's
# --------------------------------------------------------------------------- #
@pytest.mark.parametrize("dtype,ci,co,planned,relu", [
    ("f32", 32, 32, True, True), ("f32", 16, 24, False, True), ("f32", 32, 32, True, False),
    ("bf16", 256, 256, True, True), ("bf16", 64, 128, True, True), ("bf16", 48, 80, False, True)])
def test_conv_bn_relu_backward(dtype, ci, co, planned, relu):
    """conv -> batch normalisation -> ReLU in training: the fused forward,
    gsc_affine_act_bwd (dZ, dscale, dshift), then gsc_sparse_conv_bwd on dZ,
    against the oracle's chain rule.  The gradient is zero where the ReLU's
    input lies within the kernels' rounding of 0 (float32 sums: 1e-3; a bf16
    output, which the row form rounds before the affine map and again after
    it: 0.1), so the oracle (float64) and the kernels need not take that
    decision alike."""
    coords = WL.random_coords(190 + ci + co, 2600, 3, -12, 12, batch=2)
    offs = regions.hypercube(3, 3)
    X, Xb = WL.random_features(191, len(coords), ci, dtype)
    W, Wb = WL.random_weights(192, len(offs), ci, co, dtype)
    m = O.kernel_map(coords, coords, np.asarray(offs))
    S = O.conv_forward(X, W, m, len(coords))
    rng = np.random.default_rng(193)
    scale, shift = O.batchnorm_coefficients(S, rng.uniform(0.5, 2.0, co), rng.uniform(-0.5, 0.5, co))
    scale, shift = scale.astype(np.float32), shift.astype(np.float32)
    dY, dYb = WL.random_features(194, len(coords), co, dtype)
    near = np.abs(S * scale.astype(np.float64) + shift.astype(np.float64)) < (1e-3 if dtype == "f32" else 0.1)
    dY = np.where(near, 0.0, dY).astype(np.float32)
    if dYb is not None:   # bf16 bits (f32 has none)
        dYb = np.where(near, 0, dYb).astype(dYb.dtype)
    if dtype == "bf16":
        dev = lambda b: torch.from_numpy(b.view(np.int16)).to(DEV).view(torch.bfloat16)
        tX, tW, tdY = dev(Xb), dev(Wb), dev(dYb)
    else:
        tX, tW, tdY = _t(X, torch.float32), _t(W, torch.float32), _t(dY, torch.float32)
    c = _t(coords)
    table = gsc.gsc_coords_build(c)
    km = gsc.gsc_kernel_map(table, c, offs, dense=planned)
    tm = gsc.transposed_kernel_map(table, c, offs, dense=planned)
    if planned:
        km, tm = gsc.gsc_conv_plan(km), gsc.gsc_conv_plan(tm)
    _say(f"[gpu] conv-BN-ReLU backward {dtype} {ci}->{co} planned={planned} relu={relu}")
    tsc, tsh = _t(scale, torch.float32), _t(shift, torch.float32)
    Y = gsc.gsc_sparse_conv_fwd_affine(tX, tW, km, tsc, tsh, relu=relu)
    dZ, dsc, dsh = gsc.gsc_affine_act_bwd(Y, tdY, tsc, tsh, relu=relu)
    dX, dW = gsc.gsc_sparse_conv_bwd(tX, tW, dZ, km, tm, np.arange(len(offs)))
    torch.cuda.synchronize()
    dZr, dscr, dshr = O.affine_act_backward(S, dY, scale, shift, relu)
    dXr, dWr = O.conv_backward(X, W, dZr, m)
    tol = TOL[dtype]
    assert rel_err(to_np(dZ), dZr) <= tol
    assert rel_err(to_np(dsh), dshr) <= tol
    assert rel_err(to_np(dsc), dscr) <= (tol if dtype == "f32" else 2 * tol)
    assert rel_err(to_np(dX), dXr) <= tol
    assert rel_err(to_np(dW), dWr) <= tol
    # deterministic sums
    _, dsc2, dsh2 = gsc.gsc_affine_act_bwd(Y, tdY, tsc, tsh, relu=relu)
    assert torch.equal(dsc, dsc2) and torch.equal(dsh, dsh2)


def test_block_plan_choice_is_measured():
    """The pipeline's plan-or-row-form choice (both timed on the device): the
    256-channel bf16 layer's block plans are several times faster than its row
    form, so they are chosen; a layer with no block engine is never planned;
    either choice gives the oracle's result (the pass itself is checked by the
    pipeline tests)."""
    wl = WL.make_workload(4, scale=0.3)
    dw = pipeline.to_device(wl, DEV)
    _say(f"[gpu] measured plan choice on {wl.name} n={wl.n}")
    assert pipeline.choose_block_plans(dw) is True
    wl0 = WL.make_workload(0)
    dw0 = pipeline.to_device(wl0, DEV)
    assert pipeline.choose_block_plans(dw0) in (True, False)
