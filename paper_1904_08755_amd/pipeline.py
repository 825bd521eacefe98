"""One pass of the hot path over a workload, through the C-ABI entry points.

A pass is: hash table of the input coordinates, output coordinates (strided
layers), kernel maps, convolution forward, then both backward passes.  It is
host orchestration only: every stage is one call of libgsc.so.

``StepPlan`` allocates every buffer and converts every host array once, so a
pass only enqueues library calls.  The table build and the kernel maps run in
their asynchronous modes (the pair count stays on the device), so a pass of a
submanifold layer has no host round trip at all; a strided layer needs one,
to learn how many output coordinates it has, and takes it from the deferred
stride call once the transposed map (which needs only the output table) is
enqueued, so the GPU does not idle while the host waits.

Block plans: with ``use_plan`` (the default) every map that a block engine
can use (gsc_conv_block_engine) gets its block plan (gsc_conv_plan): output
rows ordered by neighbour count and mask, 16-row blocks with their per-offset items.
The forward and input-gradient passes then run on the plan; the weight
gradients always use the maps in row form.

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


class StepPlan:
    """Buffers for repeated passes over one device workload."""

    def __init__(self, dw: DeviceWorkload, use_plan: bool = True, epilogue=None):
        """``epilogue``: optional (scale, shift) float32 device tensors of c_out
        values; the forward pass of a single-layer workload then applies
        relu(Y * scale + shift) as it writes Y (gsc_sparse_conv_fwd_affine)."""
        self.dw = dw
        self.use_plan = use_plan
        self.epilogue = epilogue
        self.plans: List[gsc.KernelMap] = []
        wl = dw.wl
        self.kinds = [L.kind for L in wl.layers]
        n, D, dev = wl.n, wl.D, dw.X.device
        feat = dw.X.dtype
        self.table = torch.empty(gsc.gsc_table_bytes(n), dtype=torch.uint8, device=dev)
        if self.kinds == ["subm"]:
            L = wl.layers[0]
            offs = dw.offsets[0]
            K = len(offs)
            dt = gsc._dt(dw.X)
            self.plan_maps = use_plan and (gsc.gsc_conv_block_engine(dt, L.c_in, L.c_out, K)
                                           or gsc.gsc_conv_block_engine(dt, L.c_out, L.c_in, K))
            self.mb = gsc.MapBuffers(n, K, D, dev, dense=self.plan_maps)
            self.host_offs = gsc._host_i32(offs)
            self.symmetric = regions.is_symmetric(offs)
            if self.symmetric:
                wsel = gsc.negation_permutation(offs)
            else:
                self.tb = gsc.MapBuffers(n, K, D, dev, dense=self.plan_maps)
                self.host_offs_neg = gsc._host_i32(-offs)
                wsel = np.arange(K, dtype=np.int32)
            self.host_wsel = gsc._host_i32(wsel)
            if self.plan_maps:
                self.pb = gsc.PlanBuffers(n, K, dev)
                if not self.symmetric:
                    self.tpb = gsc.PlanBuffers(n, K, dev)
            self.ws_fwd = gsc._ws(gsc.gsc_conv_fwd_ws_bytes(gsc._dt(dw.X), L.c_in, L.c_out, K), dev)
            self.Y = torch.empty((n, L.c_out), dtype=feat, device=dev)
            self.dX = torch.empty((n, L.c_in), dtype=feat, device=dev)
            self.dW = torch.empty((K, L.c_in, L.c_out), dtype=torch.float32, device=dev)
            self.ws_bwd = gsc._ws(gsc.gsc_conv_bwd_ws_bytes(self.mb.cap, L.c_in, L.c_out, K), dev)
        elif self.kinds == ["down", "up"]:
            L0, L1 = wl.layers
            offs = dw.offsets[0]
            K = len(offs)
            self.out_table = torch.empty(gsc.gsc_table_bytes(n), dtype=torch.uint8, device=dev)
            self.stride_result = torch.empty(2, dtype=torch.int64, pin_memory=True)
            dt = gsc._dt(dw.X)
            eng = lambda a, b: gsc.gsc_conv_block_engine(dt, a, b, K)
            # kd feeds layer 0's forward and layer 1's dX; td layer 1's forward and layer 0's dX
            self.plan_kd = use_plan and (eng(L0.c_in, L0.c_out) or eng(L1.c_out, L1.c_in))
            self.plan_td = use_plan and (eng(L1.c_in, L1.c_out) or eng(L0.c_out, L0.c_in))
            # n_out <= n: size every coarse-side buffer for n rows
            self.kd = gsc.MapBuffers(n, K, D, dev, dense=self.plan_kd)
            self.td = gsc.MapBuffers(n, K, D, dev, dense=self.plan_td)
            self.host_offs = gsc._host_i32(offs)
            self.host_offs_neg = gsc._host_i32(-offs)
            self.host_ident = gsc._host_i32(np.arange(K, dtype=np.int32))
            if self.plan_kd:
                self.pkd = gsc.PlanBuffers(n, K, dev)
            if self.plan_td:
                self.ptd = gsc.PlanBuffers(n, K, dev)
            self.ws_fwd1 = gsc._ws(gsc.gsc_conv_fwd_ws_bytes(dt, L0.c_in, L0.c_out, K), dev)
            self.ws_fwd2 = gsc._ws(gsc.gsc_conv_fwd_ws_bytes(dt, L1.c_in, L1.c_out, K), dev)
            self.Y1 = torch.empty((n, L0.c_out), dtype=feat, device=dev)
            self.Y2 = torch.empty((n, L1.c_out), dtype=feat, device=dev)
            self.dY1 = torch.empty((n, L0.c_out), dtype=feat, device=dev)
            self.dX = torch.empty((n, L0.c_in), dtype=feat, device=dev)
            self.dW1 = torch.empty((K, L0.c_in, L0.c_out), dtype=torch.float32, device=dev)
            self.dW2 = torch.empty((K, L1.c_in, L1.c_out), dtype=torch.float32, device=dev)
            self.ws_bwd1 = gsc._ws(gsc.gsc_conv_bwd_ws_bytes(self.kd.cap, L0.c_in, L0.c_out, K), dev)
            self.ws_bwd2 = gsc._ws(gsc.gsc_conv_bwd_ws_bytes(self.kd.cap, L1.c_in, L1.c_out, K), dev)
        else:
            raise ValueError(f"unsupported layer sequence {self.kinds}")

    def planned(self) -> bool:
        """Whether the passes build block plans (some block engine applies)."""
        return bool(self.plan_maps if self.kinds == ["subm"] else (self.plan_kd or self.plan_td))

    def run(self, mark: Optional[Callable[[str], None]] = None, stream=None) -> StepResult:
        """Enqueue one pass.  ``mark(name)`` (optional) is called after each
        stage is enqueued: "map" (coordinates + kernel maps), "plan" (tile
        plans), "fwd", "bwd"; a two-layer pass also marks "fwd0" after the
        first layer's forward."""
        mark = mark or (lambda name: None)
        dw = self.dw
        if self.kinds == ["subm"]:
            offs = dw.offsets[0]
            gsc.gsc_coords_build(dw.coords, self.table, stream=stream, sync=False)
            kmap = gsc.gsc_kernel_map(self.table, dw.coords, offs, stream=stream, sync=False, bufs=self.mb,
                                      host_offsets=self.host_offs, dense=self.plan_maps)
            if self.symmetric:
                tmap = kmap
            else:
                tmap = gsc.gsc_kernel_map(self.table, dw.coords, -offs, stream=stream, sync=False, bufs=self.tb,
                                          host_offsets=self.host_offs_neg, dense=self.plan_maps)
            mark("map")
            fmap, dxmap = kmap, tmap
            if self.plan_maps:
                fmap = gsc.gsc_conv_plan(kmap, self.pb, stream=stream)
                dxmap = fmap if self.symmetric else gsc.gsc_conv_plan(tmap, self.tpb, stream=stream)
                self.plans = [fmap]
            mark("plan")
            if self.epilogue is None:
                Y = gsc.gsc_sparse_conv_fwd(dw.X, dw.Ws[0], fmap, Y=self.Y, stream=stream, ws=self.ws_fwd)
            else:
                Y = gsc.gsc_sparse_conv_fwd_affine(dw.X, dw.Ws[0], fmap, *self.epilogue, relu=True, Y=self.Y,
                                                   stream=stream, ws=self.ws_fwd)
            mark("fwd")
            dX, dW = gsc.gsc_sparse_conv_bwd(dw.X, dw.Ws[0], dw.dY, fmap, dxmap, None, dX=self.dX, dW=self.dW,
                                             ws=self.ws_bwd, stream=stream, host_wsel=self.host_wsel)
            mark("bwd")
            return StepResult(None, [kmap], [Y], dX, [dW], [])
        if self.epilogue is not None:
            raise ValueError("the epilogue option covers single-layer workloads")
        L0 = dw.wl.layers[0]
        offs = dw.offsets[0]
        gsc.gsc_coords_build(dw.coords, self.table, stream=stream, sync=False)
        # the output rows' count comes back while the transposed map (which
        # needs only their table) is already enqueued behind them
        pending = gsc.gsc_coords_stride(dw.coords, L0.stride, out_table=self.out_table, stream=stream, defer=True,
                                        result=self.stride_result)
        td = gsc.gsc_kernel_map(self.out_table, dw.coords, -offs, stream=stream, sync=False, bufs=self.td,
                                host_offsets=self.host_offs_neg, dense=self.plan_td)
        out_coords, _ = pending.finish()
        n_out = out_coords.shape[0]
        kd = gsc.gsc_kernel_map(self.table, out_coords, offs, stream=stream, sync=False, bufs=self.kd,
                                host_offsets=self.host_offs, dense=self.plan_kd)
        mark("map")
        pkd = gsc.gsc_conv_plan(kd, self.pkd, stream=stream) if self.plan_kd else kd
        ptd = gsc.gsc_conv_plan(td, self.ptd, stream=stream) if self.plan_td else td
        self.plans = [m for m in (pkd, ptd) if m.plan is not None]
        mark("plan")
        Y1 = gsc.gsc_sparse_conv_fwd(dw.X, dw.Ws[0], pkd, Y=self.Y1[:n_out], stream=stream, ws=self.ws_fwd1)
        mark("fwd0")   # the first layer's forward alone
        Y2 = gsc.gsc_sparse_conv_fwd(Y1, dw.Ws[1], ptd, Y=self.Y2, stream=stream, ws=self.ws_fwd2)
        mark("fwd")
        dY1, dW2 = gsc.gsc_sparse_conv_bwd(Y1, dw.Ws[1], dw.dY, ptd, pkd, None, dX=self.dY1[:n_out], dW=self.dW2,
                                           ws=self.ws_bwd2, stream=stream, host_wsel=self.host_ident)
        dX, dW1 = gsc.gsc_sparse_conv_bwd(dw.X, dw.Ws[0], dY1, pkd, ptd, None, dX=self.dX, dW=self.dW1,
                                          ws=self.ws_bwd1, stream=stream, host_wsel=self.host_ident)
        mark("bwd")
        return StepResult(out_coords, [kd, td], [Y1, Y2], dX, [dW1, dW2], [dY1])


def choose_block_plans(dw: DeviceWorkload, epilogue=None, reps: int = 3, margin: float = 0.9) -> bool:
    """Whether the passes over ``dw`` should build block plans: both ways are
    run and timed on the device (``reps`` passes each after a warm-up pass),
    and the row form is chosen only when its pass takes under ``margin`` times
    the planned one (the block engines add in a fixed order, so they are
    preferred when the two are close).  False without a block engine."""
    sp = StepPlan(dw, True, epilogue)
    if not sp.planned():
        return False
    times = {}
    for mode, plan in ((True, sp), (False, StepPlan(dw, False, epilogue))):
        plan.run()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            plan.run()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        times[mode] = sorted(ts)[len(ts) // 2]
    return not times[False] < margin * times[True]


def run_step(dw: DeviceWorkload, mark: Optional[Callable[[str], None]] = None, stream=None,
             use_plan: bool = True) -> StepResult:
    """One pass with freshly allocated buffers; the table build is then checked."""
    plan = StepPlan(dw, use_plan)
    res = plan.run(mark, stream)
    gsc.gsc_table_status(plan.table, stream)
    return res
