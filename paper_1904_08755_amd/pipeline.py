"""One pass of the hot path over a workload, through the C-ABI entry points.

A pass is: hash table of the input coordinates, output coordinates (strided
layers), kernel maps, convolution forward, then both backward passes.  It is
host orchestration only: every stage is one call of libgsc.so.

Map reuse (Sec. 4.2 builds the kernel map once per coordinate pair):
  * submanifold layer with a symmetric region: the input-gradient map is the
    forward map itself with offset s using the weight of -o_s (no rebuild);
  * otherwise the role-reversed map is built once and serves both the
    transposed convolution and the input gradient of the strided one.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Optional

import numpy as np
import torch

from . import gsc, regions
from .workloads import Workload


@dataclasses.dataclass
class DeviceWorkload:
    wl: Workload
    coords: torch.Tensor
    X: torch.Tensor
    Ws: List[torch.Tensor]
    dY: torch.Tensor
    offsets: List[np.ndarray]

    @property
    def dtype(self):
        return self.X.dtype


def _dev_feat(vals: np.ndarray, bits: Optional[np.ndarray], device) -> torch.Tensor:
    if bits is not None:
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(vals, np.float32)).to(device)


def to_device(wl: Workload, device="cuda") -> DeviceWorkload:
    coords = torch.from_numpy(np.ascontiguousarray(wl.coords, np.int32)).to(device)
    X = _dev_feat(wl.X, wl.X_bits, device)
    Ws = [_dev_feat(L.W, L.W_bits, device) for L in wl.layers]
    dY = _dev_feat(wl.dY, wl.dY_bits, device)
    offs = [regions.region(L.region, L.ksize, wl.D) for L in wl.layers]
    return DeviceWorkload(wl, coords, X, Ws, dY, offs)


@dataclasses.dataclass
class StepResult:
    out_coords: Optional[torch.Tensor]       # strided output coordinates (down layer), else None
    kmaps: List[gsc.KernelMap]               # forward map of every layer
    Ys: List[torch.Tensor]                   # output of every layer
    dX: torch.Tensor                         # gradient w.r.t. the workload input X
    dWs: List[torch.Tensor]                  # weight gradient of every layer (fp32)
    dYs_inner: List[torch.Tensor]            # gradients flowing between layers (down/up only)


def _identity(K: int) -> np.ndarray:
    return np.arange(K, dtype=np.int32)


def run_step(dw: DeviceWorkload, mark: Optional[Callable[[str], None]] = None, stream=None) -> StepResult:
    """Run one pass.  ``mark(name)`` (optional) is called after each stage is
    enqueued: "map" (coordinates + kernel maps), "fwd", "bwd"."""
    mark = mark or (lambda name: None)
    kinds = [L.kind for L in dw.wl.layers]
    if kinds == ["subm"]:
        offs = dw.offsets[0]
        table = gsc.gsc_coords_build(dw.coords, stream=stream)
        kmap = gsc.gsc_kernel_map(table, dw.coords, offs, stream=stream)
        if regions.is_symmetric(offs):
            tmap, wsel = kmap, gsc.negation_permutation(offs)
        else:
            tmap, wsel = gsc.transposed_kernel_map(table, dw.coords, offs, stream=stream), _identity(len(offs))
        mark("map")
        Y = gsc.gsc_sparse_conv_fwd(dw.X, dw.Ws[0], kmap, stream=stream)
        mark("fwd")
        dX, dW = gsc.gsc_sparse_conv_bwd(dw.X, dw.Ws[0], dw.dY, kmap, tmap, wsel, stream=stream)
        mark("bwd")
        return StepResult(None, [kmap], [Y], dX, [dW], [])
    if kinds == ["down", "up"]:
        L0 = dw.wl.layers[0]
        offs = dw.offsets[0]
        ident = _identity(len(offs))
        table = gsc.gsc_coords_build(dw.coords, stream=stream)
        out_coords, out_table = gsc.gsc_coords_stride(dw.coords, L0.stride, stream=stream)
        kd = gsc.gsc_kernel_map(table, out_coords, offs, stream=stream)
        td = gsc.transposed_kernel_map(out_table, dw.coords, offs, stream=stream)
        mark("map")
        Y1 = gsc.gsc_sparse_conv_fwd(dw.X, dw.Ws[0], kd, stream=stream)
        Y2 = gsc.gsc_sparse_conv_fwd(Y1, dw.Ws[1], td, stream=stream)
        mark("fwd")
        dY1, dW2 = gsc.gsc_sparse_conv_bwd(Y1, dw.Ws[1], dw.dY, td, kd, ident, stream=stream)
        dX, dW1 = gsc.gsc_sparse_conv_bwd(dw.X, dw.Ws[0], dY1, kd, td, ident, stream=stream)
        mark("bwd")
        return StepResult(out_coords, [kd, td], [Y1, Y2], dX, [dW1, dW2], [dY1])
    raise ValueError(f"unsupported layer sequence {kinds}")
