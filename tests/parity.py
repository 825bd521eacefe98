"""Helpers for the GPU parity tests: run the oracle on a workload and compare
the HIP path's results with it (maps bit-exact after canonical alignment,
features within tolerance)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.gsc_oracle as O

TOL = {"f32": 1e-5, "bf16": 2e-2}


def to_np(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy().astype(np.float64)


def rel_err(got, ref) -> float:
    ref = np.asarray(ref, np.float64)
    got = np.asarray(got, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = np.abs(ref).max() if ref.size else 0.0
    num = np.abs(got - ref).max() if ref.size else 0.0
    return float(num / den) if den > 0 else float(num)


def gpu_pairs(km):
    seg = km.seg.cpu().numpy()
    I = km.in_idx.cpu().numpy().astype(np.int64)
    Oo = km.out_idx.cpu().numpy().astype(np.int64)
    return [(I[seg[k]:seg[k + 1]], Oo[seg[k]:seg[k + 1]]) for k in range(len(seg) - 1)]


def check_gidx(km):
    """The group index agrees with the pair list: group g of offset k holds
    exactly the pairs of k whose output row is in [64 g, 64 g + 64)."""
    G = (km.n_out + 63) // 64
    n_pairs = km.count()
    gidx = km.gidx.cpu().numpy()[: km.K * G + 1]
    seg = km.seg.cpu().numpy()
    Oo = km.out_idx.cpu().numpy()[:n_pairs].astype(np.int64)
    assert gidx[-1] == n_pairs == seg[-1]
    for k in range(km.K):
        if G:
            assert gidx[k * G] == seg[k]
        for g in range(G):
            a, b = gidx[k * G + g], gidx[k * G + g + 1]
            if b > a:
                assert np.all(Oo[a:b] // 64 == g)


def maps_equal_exact(gpu, ref, out_perm=None, in_perm=None):
    """Per offset, the GPU pairs (rows mapped to the oracle's numbering where
    the orders differ, then sorted by output row) equal the oracle's."""
    assert len(gpu) == len(ref)
    for k, ((gi, go), (ri, ro)) in enumerate(zip(gpu, ref)):
        if in_perm is not None:
            gi = in_perm[gi]
        if out_perm is not None:
            go = out_perm[go]
            order = np.lexsort((gi, go))
            gi, go = gi[order], go[order]
        if not (np.array_equal(gi, ri) and np.array_equal(go, ro)):
            raise AssertionError(f"offset {k}: map differs ({len(gi)} vs {len(ri)} pairs)")


def row_perm(gpu_coords: np.ndarray, ref_coords: np.ndarray) -> np.ndarray:
    """perm[g] = oracle row of GPU row g; asserts the row sets are identical."""
    assert gpu_coords.shape == ref_coords.shape, (gpu_coords.shape, ref_coords.shape)
    ref = O.coordinate_map(ref_coords)
    perm = np.array([ref[tuple(r)] for r in gpu_coords.tolist()], dtype=np.int64)
    assert len(np.unique(perm)) == len(perm)
    return perm


def oracle_step(wl):
    """The oracle's results for a workload: the same pass as the HIP pipeline."""
    kinds = [L.kind for L in wl.layers]
    X = wl.X.astype(np.float64)
    dY = wl.dY.astype(np.float64)
    res = {}
    if kinds == ["subm"]:
        L = wl.layers[0]
        offs = O.region(L.region, L.ksize, wl.D)
        m = O.kernel_map(wl.coords, wl.coords, offs)
        res["maps"] = [m]
        res["Ys"] = [O.conv_forward(X, L.W, m, wl.n)]
        dX, dW = O.conv_backward(X, L.W, dY, m)
        res.update(dX=dX, dWs=[dW], out_coords=None, inner=[])
    elif kinds == ["down", "up"]:
        L0, L1 = wl.layers
        offs = O.region(L0.region, L0.ksize, wl.D)
        out = O.output_coordinates(wl.coords, L0.stride)
        kd = O.kernel_map(wl.coords, out, offs)
        td = O.transposed_map(kd)
        Y1 = O.conv_forward(X, L0.W, kd, len(out))
        Y2 = O.conv_forward(Y1, L1.W, td, wl.n)
        dY1, dW2 = O.conv_backward(Y1, L1.W, dY, td)
        dX, dW1 = O.conv_backward(X, L0.W, dY1, kd)
        res.update(maps=[kd, td], Ys=[Y1, Y2], dX=dX, dWs=[dW1, dW2], out_coords=out, inner=[dY1])
    else:
        raise ValueError(kinds)
    return res


def compare_step(wl, step, ref):
    """Assert parity of a pipeline StepResult with oracle_step's result.
    Returns a dict of the measured errors."""
    tol = TOL[wl.dtype]
    errs = {}
    if ref["out_coords"] is None:
        maps_equal_exact(gpu_pairs(step.kmaps[0]), ref["maps"][0])
        check_gidx(step.kmaps[0])
        errs["Y"] = rel_err(to_np(step.Ys[0]), ref["Ys"][0])
    else:
        gcoords = step.out_coords.cpu().numpy()
        perm = row_perm(gcoords, ref["out_coords"])
        maps_equal_exact(gpu_pairs(step.kmaps[0]), ref["maps"][0], out_perm=perm)
        maps_equal_exact(gpu_pairs(step.kmaps[1]), ref["maps"][1], in_perm=perm)
        check_gidx(step.kmaps[0])
        check_gidx(step.kmaps[1])
        Y1 = to_np(step.Ys[0])
        Y1r = np.empty_like(Y1)
        Y1r[perm] = Y1
        errs["Y1"] = rel_err(Y1r, ref["Ys"][0])
        errs["Y2"] = rel_err(to_np(step.Ys[1]), ref["Ys"][1])
        dY1 = to_np(step.dYs_inner[0])
        dY1r = np.empty_like(dY1)
        dY1r[perm] = dY1
        errs["dY1"] = rel_err(dY1r, ref["inner"][0])
    errs["dX"] = rel_err(to_np(step.dX), ref["dX"])
    for i, (g, r) in enumerate(zip(step.dWs, ref["dWs"])):
        errs[f"dW{i}"] = rel_err(to_np(g), r)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"tolerance {tol} exceeded: {bad} (all: {errs})"
    return errs
