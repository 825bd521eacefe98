"""Python binding of libgsc.so (include/gsc.h): argument marshalling only.

Every function here checks tensor shapes, devices and dtypes, allocates the
caller-owned output and workspace buffers with torch (device memory and
streams are all torch provides), and calls the C entry point of the same
name.  All computation runs in the HIP kernels of the library; if the
library is missing, loading fails with an error (there is no fallback).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgsc.so")

GSC_OK, GSC_EINVAL, GSC_ESHORT, GSC_ERANGE, GSC_EDUP, GSC_EFULL, GSC_EHIP, GSC_ETIMEOUT = 0, -1, -2, -3, -4, -5, -6, -7
GSC_F32, GSC_BF16 = 0, 1
GROUP_ROWS = 64

_STATUS = {GSC_EINVAL: "EINVAL", GSC_ESHORT: "ESHORT", GSC_ERANGE: "ERANGE", GSC_EDUP: "EDUP",
           GSC_EFULL: "EFULL", GSC_EHIP: "EHIP", GSC_ETIMEOUT: "ETIMEOUT"}


class GscError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_STATUS.get(code, code)}: {msg}")
        self.code = code


_c_i32p = ctypes.POINTER(ctypes.c_int32)
_c_i64p = ctypes.POINTER(ctypes.c_int64)
_vp = ctypes.c_void_p
_i32, _i64, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t

_SIGS = {
    "gsc_last_error": (ctypes.c_char_p, []),
    "gsc_abi_version": (ctypes.c_int, []),
    "gsc_table_bytes": (_sz, [_i64]),
    "gsc_coords_build": (ctypes.c_int, [_vp, _i64, _i32, _vp, _sz, _vp]),
    "gsc_coords_build_async": (ctypes.c_int, [_vp, _i64, _i32, _vp, _sz, _vp]),
    "gsc_table_status": (ctypes.c_int, [_vp, _vp]),
    "gsc_stride_ws_bytes": (_sz, [_i64]),
    "gsc_coords_stride": (ctypes.c_int, [_vp, _i64, _i32, _c_i32p, _vp, _c_i64p, _vp, _sz, _vp, _sz, _vp]),
    "gsc_coords_stride_async": (ctypes.c_int, [_vp, _i64, _i32, _c_i32p, _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "gsc_coords_stride_result": (ctypes.c_int, [_vp, _c_i64p]),
    "gsc_quantize_ws_bytes": (_sz, [_i64, _i32]),
    "gsc_quantize": (ctypes.c_int, [_vp, _vp, _i64, _i32, ctypes.POINTER(ctypes.c_float), _vp, _i32, _vp, _c_i64p,
                                    _vp, _vp, _vp, _vp, _sz, _vp, _sz, _vp]),
    "gsc_kmap_groups": (_i64, [_i64]),
    "gsc_kmap_ws_bytes": (_sz, [_i64, _i32, _i32]),
    "gsc_kernel_map": (ctypes.c_int, [_vp, _vp, _i64, _i32, _c_i32p, _i32, _c_i32p, _vp, _vp, _i64, _vp, _vp,
                                      _vp, _c_i64p, _vp, _sz, _vp]),
    "gsc_kernel_map_noalloc_bytes": (_sz, [_i64, _i32]),
    "gsc_kernel_map_noalloc": (ctypes.c_int, [_vp, _vp, _i64, _i32, _c_i32p, _i32, _c_i32p, _vp, _vp, _i64, _vp,
                                              _vp, _vp, _vp]),
    "gsc_plan_blocks": (_i64, [_i64]),
    "gsc_plan_ranges": (_i32, [_i32]),
    "gsc_affine_act_bwd_ws_bytes": (_sz, [_i64, _i32]),
    "gsc_affine_act_bwd": (ctypes.c_int, [_i32, _vp, _vp, _i64, _i32, _vp, _vp, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gsc_kernel_map_transpose_ws_bytes": (_sz, [_i64, _i32]),
    "gsc_kernel_map_transpose": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _sz,
                                                _vp]),
    "gsc_kernel_map_transpose_status": (ctypes.c_int, [_vp, _vp]),
    "gsc_conv_bwd_fwdmap_ws_bytes": (_sz, [_i32, _i64, _i64, _i32, _i32, _i32]),
    "gsc_sparse_conv_bwd_fwdmap": (ctypes.c_int, [_i32, _vp, _vp, _vp, _i64, _i32, _i32, _i32, _vp, _vp, _vp, _i64,
                                                  _i32, _vp, _vp, _i64, _vp, _sz, _vp]),
    "gsc_conv_plan_status": (ctypes.c_int, [_vp, _sz, _i64, _i32, _vp]),
    "gsc_conv_plan_ws_bytes": (_sz, [_i64, _i32]),
    "gsc_conv_plan": (ctypes.c_int, [_vp, _i64, _i32, _vp, _vp, _vp, _vp, _i64, _vp, _sz, _vp]),
    "gsc_conv_block_engine": (_i32, [_i32, _i32, _i32, _i32]),
    "gsc_conv_fwd_ws_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "gsc_sparse_conv_fwd": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64,
                                           _vp, _vp, _vp, _vp, _vp, _i64, _vp, _sz, _vp]),
    "gsc_sparse_conv_fwd_affine": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _i64,
                                                  _vp, _vp, _vp, _vp, _vp, _vp, _i32, _vp, _i64, _vp, _sz, _vp]),
    "gsc_conv_bwd_ws_bytes": (_sz, [_i64, _i32, _i32, _i32]),
    "gsc_sparse_conv_bwd": (ctypes.c_int, [_i32, _vp, _vp, _vp, _i64, _i32, _i32, _i32, _vp, _vp, _vp, _i64, _vp,
                                           _vp, _vp, _vp, _i64, _c_i32p, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp,
                                           _sz, _vp]),
    "gsc_sparse_pool_fwd": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _i32, _i64, _vp, _vp, _vp, _vp]),
    "gsc_sparse_pool_bwd": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _i32, _i64, _vp, _vp, _vp, _vp]),
    "gsc_global_pool_ws_bytes": (_sz, [_i64, _i32, _i32]),
    "gsc_global_pool_fwd": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gsc_global_pool_bwd": (ctypes.c_int, [_i32, _vp, _i32, _i32, _vp, _i32, _i64, _vp, _vp, _vp, _vp]),
}

GSC_POOL_MAX, GSC_POOL_AVG, GSC_POOL_SUM = 0, 1, 2
POOL_MODES = {"max": GSC_POOL_MAX, "avg": GSC_POOL_AVG, "sum": GSC_POOL_SUM}

_lib = None


def lib() -> ctypes.CDLL:
    """Load libgsc.so (built in-tree by ``python -m paper_1904_08755_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise GscError(GSC_EHIP, f"{LIB_PATH} is not built; run python -m paper_1904_08755_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def exported_symbols():
    return list(_SIGS)


def _check(rc: int):
    if rc != GSC_OK:
        raise GscError(rc, lib().gsc_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _host_i32(a) -> ctypes.Array:
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32)).ravel()
    return (ctypes.c_int32 * max(len(a), 1))(*a.tolist())


def _need(t: torch.Tensor, dtype, name, dims=None):
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dims is not None and t.dim() != dims:
        raise ValueError(f"{name} must have {dims} dims")


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# --------------------------------------------------------------------------- #
# a1: coordinate hash table
# --------------------------------------------------------------------------- #
def gsc_table_bytes(n: int) -> int:
    return int(lib().gsc_table_bytes(n))


def gsc_coords_build(coords: torch.Tensor, table: Optional[torch.Tensor] = None, stream=None,
                     sync: bool = True) -> torch.Tensor:
    """Hash table of ``coords``.  ``sync=False`` calls gsc_coords_build_async
    (errors found on the device are then reported by gsc_table_status)."""
    _need(coords, torch.int32, "coords", 2)
    n, ncol = coords.shape
    if table is None:
        table = torch.empty(gsc_table_bytes(n), dtype=torch.uint8, device=coords.device)
    _need(table, torch.uint8, "table", 1)
    f = lib().gsc_coords_build if sync else lib().gsc_coords_build_async
    _check(f(_ptr(coords), n, ncol - 1, _ptr(table), table.numel(), _stream(stream)))
    return table


def gsc_table_status(table: torch.Tensor, stream=None) -> None:
    """Raise GscError if the build of ``table`` failed on the device."""
    _check(lib().gsc_table_status(_ptr(table), _stream(stream)))


# --------------------------------------------------------------------------- #
# a2: output coordinates of a strided convolution
# --------------------------------------------------------------------------- #
def gsc_coords_stride(coords: torch.Tensor, stride: Sequence[int], out_table: Optional[torch.Tensor] = None,
                      stream=None, defer: bool = False, result: Optional[torch.Tensor] = None):
    """Returns (out_coords [n_out, 1+D] int32, out_table).  With ``defer``
    the call returns a StridePending at once (gsc_coords_stride_async): work
    that needs only ``out_table`` can be enqueued before its ``finish()``
    reads the row count.  ``result`` (2 int64 in pinned host memory) may be
    given to reuse it across calls."""
    _need(coords, torch.int32, "coords", 2)
    n, ncol = coords.shape
    D = ncol - 1
    st = [int(stride)] * D if np.isscalar(stride) else [int(v) for v in stride]
    if len(st) != D:
        raise ValueError("stride needs D entries")
    dev = coords.device
    out = torch.empty((max(n, 1), ncol), dtype=torch.int32, device=dev)
    if out_table is None:
        out_table = torch.empty(gsc_table_bytes(n), dtype=torch.uint8, device=dev)
    ws = _ws(lib().gsc_stride_ws_bytes(n), dev)
    if defer:
        if result is None:
            result = torch.empty(2, dtype=torch.int64, pin_memory=True)
        _check(lib().gsc_coords_stride_async(_ptr(coords), n, D, _host_i32(st), _ptr(out), result.data_ptr(),
                                             _ptr(out_table), out_table.numel(), _ptr(ws), ws.numel(),
                                             _stream(stream)))
        ev = torch.cuda.Event()
        ev.record(torch.cuda.current_stream(dev) if stream is None else stream)
        return StridePending(out, out_table, result, ev, ws)
    n_out = ctypes.c_int64(0)
    _check(lib().gsc_coords_stride(_ptr(coords), n, D, _host_i32(st), _ptr(out), ctypes.byref(n_out),
                                   _ptr(out_table), out_table.numel(), _ptr(ws), ws.numel(), _stream(stream)))
    return out[: n_out.value], out_table


@dataclasses.dataclass
class StridePending:
    """An enqueued gsc_coords_stride_async: finish() waits for its result copy
    (not for work enqueued after it) and returns (out_coords, out_table)."""
    out: torch.Tensor
    out_table: torch.Tensor
    result: torch.Tensor
    done: "torch.cuda.Event"
    ws: torch.Tensor   # kept alive until the kernels that use it have run

    def finish(self):
        self.done.synchronize()
        n_out = ctypes.c_int64(0)
        _check(lib().gsc_coords_stride_result(self.result.data_ptr(), ctypes.byref(n_out)))
        return self.out[: n_out.value], self.out_table


# --------------------------------------------------------------------------- #
# a3: kernel map
# --------------------------------------------------------------------------- #
@dataclasses.dataclass
class KernelMap:
    in_idx: torch.Tensor       # int32 [>= n_pairs]
    out_idx: torch.Tensor      # int32 [>= n_pairs]
    seg: torch.Tensor          # int64 [K + 1]
    gidx: torch.Tensor         # int64 [K * G + 1]
    n_pairs: Optional[int]     # None when built asynchronously (the count stays on the device)
    n_out: int
    offsets: np.ndarray        # K x D
    n_bound: int = 0           # n_pairs, or an upper bound of it
    nbr: Optional[torch.Tensor] = None    # dense form [K, n_out]: input row or -1 (if requested)
    plan: Optional["BlockPlan"] = None    # block plan of the map (gsc_conv_plan), if built

    @property
    def K(self) -> int:
        return int(self.offsets.shape[0])

    def count(self) -> int:
        """Number of pairs (reads seg[K] from the device when unknown)."""
        return self.n_pairs if self.n_pairs is not None else int(self.seg[-1].item())


def gsc_kmap_groups(n_out: int) -> int:
    return int(lib().gsc_kmap_groups(n_out))


class MapBuffers:
    """Caller-owned buffers of one kernel map (reusable across calls)."""

    def __init__(self, n_out: int, K: int, D: int, device, cap_pairs: Optional[int] = None, dense: bool = False):
        G = gsc_kmap_groups(n_out)
        self.cap = K * n_out if cap_pairs is None else int(cap_pairs)
        # flat: a map over fewer rows than the buffers were sized for keeps row stride n_out
        self.nbr = torch.empty(max(K * n_out, 1), dtype=torch.int32, device=device) if dense else None
        self.in_idx = torch.empty(max(self.cap, 1), dtype=torch.int32, device=device)
        self.out_idx = torch.empty(max(self.cap, 1), dtype=torch.int32, device=device)
        self.seg = torch.empty(K + 1, dtype=torch.int64, device=device)
        self.gidx = torch.empty(K * G + 1, dtype=torch.int64, device=device)
        self.ws = _ws(lib().gsc_kmap_ws_bytes(n_out, K, D), device)


def gsc_kernel_map(in_table: torch.Tensor, out_coords: torch.Tensor, offsets, tensor_stride=None,
                   cap_pairs: Optional[int] = None, stream=None, sync: bool = True,
                   bufs: Optional[MapBuffers] = None, host_offsets=None, host_ts=None,
                   dense: bool = False) -> KernelMap:
    """Kernel map of ``offsets`` from the table ``in_table`` to ``out_coords``.
    ``sync=False`` builds it without a host round trip (n_pairs stays on the
    device).  ``dense`` also keeps the map's dense form (the input of
    gsc_conv_plan).  ``bufs``/``host_offsets``/``host_ts`` let a caller reuse
    buffers and converted host arrays across calls."""
    _need(in_table, torch.uint8, "in_table", 1)
    _need(out_coords, torch.int32, "out_coords", 2)
    offs = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    K, D = offs.shape
    n_out = out_coords.shape[0]
    if out_coords.shape[1] != D + 1:
        raise ValueError("offsets must be K x D with D = out_coords columns - 1")
    if bufs is None:
        bufs = MapBuffers(n_out, K, D, out_coords.device, cap_pairs, dense)
    if dense and bufs.nbr is None:
        raise ValueError("dense=True needs MapBuffers(..., dense=True)")
    nbr = bufs.nbr if dense else None
    if host_offsets is None:
        host_offsets = _host_i32(offs)
    if host_ts is None and tensor_stride is not None:
        host_ts = _host_i32([tensor_stride] * D if np.isscalar(tensor_stride) else tensor_stride)
    n_pairs = ctypes.c_int64(0)
    rc = lib().gsc_kernel_map(_ptr(in_table), _ptr(out_coords), n_out, D, host_offsets, K, host_ts,
                              _ptr(bufs.in_idx), _ptr(bufs.out_idx), bufs.cap, _ptr(bufs.seg), _ptr(bufs.gidx),
                              _ptr(nbr), ctypes.byref(n_pairs) if sync else None, _ptr(bufs.ws), bufs.ws.numel(),
                              _stream(stream))
    _check(rc)
    nbr = None if nbr is None else nbr[: K * n_out].view(K, n_out)
    if sync:
        m = n_pairs.value
        return KernelMap(bufs.in_idx[:m], bufs.out_idx[:m], bufs.seg, bufs.gidx, m, n_out, offs, m, nbr)
    return KernelMap(bufs.in_idx, bufs.out_idx, bufs.seg, bufs.gidx, None, n_out, offs, bufs.cap, nbr)


def gsc_kernel_map_noalloc(in_table: torch.Tensor, out_coords: torch.Tensor, offsets, bufs: MapBuffers,
                           tensor_stride=None, stream=None, host_offsets=None, host_ts=None) -> KernelMap:
    """gsc_kernel_map in its asynchronous mode without a workspace: the
    library's own per-GPU scratch array serves instead (for callers that
    cannot allocate).  ``bufs`` must hold the dense form (MapBuffers(...,
    dense=True)); its ``ws`` is not used."""
    _need(in_table, torch.uint8, "in_table", 1)
    _need(out_coords, torch.int32, "out_coords", 2)
    offs = np.ascontiguousarray(np.asarray(offsets, dtype=np.int32))
    K, D = offs.shape
    n_out = out_coords.shape[0]
    if out_coords.shape[1] != D + 1:
        raise ValueError("offsets must be K x D with D = out_coords columns - 1")
    if bufs.nbr is None or bufs.nbr.numel() < K * n_out:
        raise ValueError("gsc_kernel_map_noalloc needs MapBuffers(..., dense=True) for n_out rows")
    if host_offsets is None:
        host_offsets = _host_i32(offs)
    if host_ts is None and tensor_stride is not None:
        host_ts = _host_i32([tensor_stride] * D if np.isscalar(tensor_stride) else tensor_stride)
    rc = lib().gsc_kernel_map_noalloc(_ptr(in_table), _ptr(out_coords), n_out, D, host_offsets, K, host_ts,
                                      _ptr(bufs.in_idx), _ptr(bufs.out_idx), bufs.cap, _ptr(bufs.seg),
                                      _ptr(bufs.gidx), _ptr(bufs.nbr), _stream(stream))
    _check(rc)
    return KernelMap(bufs.in_idx, bufs.out_idx, bufs.seg, bufs.gidx, None, n_out, offs, bufs.cap,
                     bufs.nbr[: K * n_out].view(K, n_out))


def transposed_kernel_map(out_table: torch.Tensor, in_coords: torch.Tensor, offsets, tensor_stride=None,
                          stream=None, sync: bool = True, bufs: Optional[MapBuffers] = None,
                          dense: bool = False) -> KernelMap:
    """The role-reversed map (Sec. 4.2): same pairs, listed by original input row."""
    return gsc_kernel_map(out_table, in_coords, -np.asarray(offsets, dtype=np.int32), tensor_stride, stream=stream,
                          sync=sync, bufs=bufs, dense=dense)


@dataclasses.dataclass
class BlockPlan:
    """Block plan of a kernel map (see gsc_conv_plan in include/gsc.h)."""
    perm: torch.Tensor         # int32 [R * n_out]: output row at each position (R = offset ranges)
    bmask: torch.Tensor        # uint32 bits as int32 [R * nb]: union mask of each 16-position block
    ibase: torch.Tensor        # int64 [R * (nb + 1)]: first item of each block
    items: torch.Tensor        # int32 [cap_items, 16]: input rows of each item (-1: none)

    def ptrs(self):
        return _ptr(self.perm), _ptr(self.bmask), _ptr(self.ibase), _ptr(self.items)


def gsc_plan_blocks(n_out: int) -> int:
    return int(lib().gsc_plan_blocks(n_out))


def gsc_conv_block_engine(dtype: int, c_red: int, c_out: int, K: int) -> bool:
    return bool(lib().gsc_conv_block_engine(dtype, c_red, c_out, K))


def gsc_plan_ranges(K: int) -> int:
    return int(lib().gsc_plan_ranges(K))


class PlanBuffers:
    """Caller-owned buffers of one block plan (reusable across calls); a map
    with more than 32 offsets has gsc_plan_ranges(K) plans, one per range of
    offsets, stored one after another."""

    def __init__(self, n_out: int, K: int, device):
        nb = gsc_plan_blocks(n_out)
        R = gsc_plan_ranges(K)
        if R < 1:
            raise ValueError(f"no block plan for K={K} offsets")
        self.cap_items = K * nb
        self.perm = torch.empty(max(R * n_out, 1), dtype=torch.int32, device=device)
        self.bmask = torch.empty(max(R * nb, 1), dtype=torch.int32, device=device)
        self.ibase = torch.empty(R * (nb + 1), dtype=torch.int64, device=device)
        self.items = torch.empty((max(self.cap_items, 1), 16), dtype=torch.int32, device=device)
        self.ws = _ws(lib().gsc_conv_plan_ws_bytes(n_out, K), device)


def gsc_conv_plan(kmap: KernelMap, bufs: Optional[PlanBuffers] = None, stream=None) -> KernelMap:
    """The map with its block plan attached (rows ordered by neighbour count and mask,
    16-row blocks, per-block items of 16 input rows)."""
    n_out, K = kmap.n_out, kmap.K
    if kmap.nbr is None:
        raise ValueError("gsc_conv_plan needs the map's dense form: build it with dense=True")
    if bufs is None:
        bufs = PlanBuffers(n_out, K, kmap.seg.device)
    _check(lib().gsc_conv_plan(_ptr(kmap.nbr), n_out, K, _ptr(bufs.perm), _ptr(bufs.bmask), _ptr(bufs.ibase),
                               _ptr(bufs.items), bufs.cap_items, _ptr(bufs.ws), bufs.ws.numel(), _stream(stream)))
    plan = BlockPlan(bufs.perm[: gsc_plan_ranges(K) * n_out], bufs.bmask, bufs.ibase, bufs.items)
    return dataclasses.replace(kmap, plan=plan)


def gsc_conv_plan_status(kmap: KernelMap, bufs: PlanBuffers, stream=None) -> None:
    """Synchronise and raise GscError (ETIMEOUT) if the plan built into
    ``bufs`` for ``kmap`` came from a sort pass that gave up."""
    _check(lib().gsc_conv_plan_status(_ptr(bufs.ws), bufs.ws.numel(), kmap.n_out, kmap.K, _stream(stream)))


def gsc_kernel_map_transpose(kmap: KernelMap, n_rev: int, stream=None, check: bool = True) -> KernelMap:
    """The role-reversed map of ``kmap`` (pairs listed by the former input
    row, over ``n_rev`` rows) built from its pairs alone, with its dense form;
    segment k holds offset k's pairs, so its t_wsel is the identity.  With
    ``check`` the call synchronises and raises if a pair's input row lies
    outside [0, n_rev)."""
    K, dev = kmap.K, kmap.seg.device
    cap = kmap.n_bound
    G = gsc_kmap_groups(n_rev)
    t_in = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    t_out = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    t_seg = torch.empty(K + 1, dtype=torch.int64, device=dev)
    t_gidx = torch.empty(K * G + 1, dtype=torch.int64, device=dev)
    t_nbr = torch.empty((K, max(n_rev, 1)), dtype=torch.int32, device=dev)
    ws = _ws(lib().gsc_kernel_map_transpose_ws_bytes(n_rev, K), dev)
    _check(lib().gsc_kernel_map_transpose(_ptr(kmap.in_idx), _ptr(kmap.out_idx), _ptr(kmap.seg), K, cap, n_rev,
                                          _ptr(t_in), _ptr(t_out), _ptr(t_seg), _ptr(t_gidx), _ptr(t_nbr), _ptr(ws),
                                          ws.numel(), _stream(stream)))
    if check:
        _check(lib().gsc_kernel_map_transpose_status(_ptr(ws), _stream(stream)))
    return KernelMap(t_in, t_out, t_seg, t_gidx, kmap.n_pairs, n_rev, -np.asarray(kmap.offsets), cap,
                     nbr=t_nbr[:, :n_rev])


def negation_permutation(offsets) -> np.ndarray:
    """s -> index of -o_s (for symmetric offset sets)."""
    offs = np.asarray(offsets)
    index = {tuple(o): k for k, o in enumerate(offs.tolist())}
    return np.array([index[tuple(-v for v in o)] for o in offs.tolist()], dtype=np.int32)


# --------------------------------------------------------------------------- #
# a4-a7: convolution
# --------------------------------------------------------------------------- #
def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GSC_F32
    if t.dtype == torch.bfloat16:
        return GSC_BF16
    raise ValueError(f"unsupported feature dtype {t.dtype}")


def _plan_ptrs(kmap: KernelMap):
    return kmap.plan.ptrs() if kmap.plan is not None else (None, None, None, None)


def gsc_conv_fwd_ws_bytes(dtype: int, c_in: int, c_out: int, K: int) -> int:
    return int(lib().gsc_conv_fwd_ws_bytes(dtype, c_in, c_out, K))


def _fwd_args(X, W, kmap, n_out, Y, ws):
    dt = _dt(X)
    _need(X, X.dtype, "X", 2)
    _need(W, X.dtype, "W", 3)
    K, ci, co = W.shape
    if X.shape[1] != ci or K != kmap.K:
        raise ValueError("shape mismatch between X, W and the kernel map")
    n_out = kmap.n_out if n_out is None else n_out
    if n_out != kmap.n_out:
        raise ValueError("n_out differs from the kernel map's output rows")
    if Y is None:
        Y = torch.empty((n_out, co), dtype=X.dtype, device=X.device)
    _need(Y, X.dtype, "Y", 2)
    need = gsc_conv_fwd_ws_bytes(dt, ci, co, K)
    if ws is None and need > 0:
        ws = _ws(need, X.device)
    head = (dt, _ptr(X), X.shape[0], ci, _ptr(W), co, K, _ptr(kmap.in_idx), _ptr(kmap.out_idx), _ptr(kmap.seg),
            _ptr(kmap.gidx), kmap.n_bound, *_plan_ptrs(kmap))
    return head, Y, n_out, ws


def gsc_sparse_conv_fwd(X: torch.Tensor, W: torch.Tensor, kmap: KernelMap, n_out: Optional[int] = None,
                        Y: Optional[torch.Tensor] = None, stream=None, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    head, Y, n_out, ws = _fwd_args(X, W, kmap, n_out, Y, ws)
    _check(lib().gsc_sparse_conv_fwd(*head, _ptr(Y), n_out, _ptr(ws), 0 if ws is None else ws.numel(),
                                     _stream(stream)))
    return Y


GSC_ACT_NONE, GSC_ACT_RELU = 0, 1


def gsc_sparse_conv_fwd_affine(X: torch.Tensor, W: torch.Tensor, kmap: KernelMap,
                               scale: Optional[torch.Tensor] = None, shift: Optional[torch.Tensor] = None,
                               relu: bool = False, n_out: Optional[int] = None, Y: Optional[torch.Tensor] = None,
                               stream=None, ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Y = act(conv(X) * scale + shift), per output channel (float32 scale and
    shift of c_out values on X's device, each optional)."""
    co = W.shape[2]
    for name, v in (("scale", scale), ("shift", shift)):
        if v is not None:
            _need(v, torch.float32, name, 1)
            if v.shape[0] != co:
                raise ValueError(f"{name} needs {co} values")
    head, Y, n_out, ws = _fwd_args(X, W, kmap, n_out, Y, ws)
    _check(lib().gsc_sparse_conv_fwd_affine(*head, _ptr(scale), _ptr(shift), GSC_ACT_RELU if relu else GSC_ACT_NONE,
                                            _ptr(Y), n_out, _ptr(ws), 0 if ws is None else ws.numel(),
                                            _stream(stream)))
    return Y


def gsc_conv_bwd_ws_bytes(n_pairs: int, c_in: int, c_out: int, K: int) -> int:
    return int(lib().gsc_conv_bwd_ws_bytes(n_pairs, c_in, c_out, K))


def gsc_sparse_conv_bwd(X: torch.Tensor, W: torch.Tensor, dY: torch.Tensor, kmap: KernelMap,
                        tmap: KernelMap, wsel, need_dx: bool = True, need_dw: bool = True,
                        dX: Optional[torch.Tensor] = None, dW: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, stream=None, host_wsel=None):
    """Returns (dX or None, dW or None).  ``tmap`` is the dX map (role-reversed
    pairs, sorted by input row) and ``wsel`` its per-segment weight index."""
    dt = _dt(X)
    _need(X, X.dtype, "X", 2)
    _need(W, X.dtype, "W", 3)
    _need(dY, X.dtype, "dY", 2)
    K, ci, co = W.shape
    n_in, n_out = X.shape[0], dY.shape[0]
    if X.shape[1] != ci or dY.shape[1] != co or kmap.K != K or tmap.K != K:
        raise ValueError("shape mismatch")
    if kmap.n_out != n_out or tmap.n_out != n_in:
        raise ValueError("kernel maps do not match the row counts")
    dev = X.device
    if need_dx and dX is None:
        dX = torch.empty((n_in, ci), dtype=X.dtype, device=dev)
    if need_dw and dW is None:
        dW = torch.empty((K, ci, co), dtype=torch.float32, device=dev)
    if need_dw and ws is None:
        ws = _ws(gsc_conv_bwd_ws_bytes(kmap.n_bound, ci, co, K), dev)
    sel = _host_i32(wsel) if host_wsel is None else host_wsel
    _check(lib().gsc_sparse_conv_bwd(
        dt, _ptr(X), _ptr(W), _ptr(dY), n_in, ci, co, K,
        _ptr(kmap.in_idx), _ptr(kmap.out_idx), _ptr(kmap.seg), kmap.n_bound,
        _ptr(tmap.in_idx), _ptr(tmap.out_idx), _ptr(tmap.seg), _ptr(tmap.gidx), tmap.n_bound, sel, *_plan_ptrs(tmap),
        _ptr(dX) if need_dx else None, _ptr(dW) if need_dw else None, n_out,
        _ptr(ws) if need_dw else None, ws.numel() if need_dw else 0, _stream(stream)))
    return (dX if need_dx else None), (dW if need_dw else None)


def gsc_sparse_conv_bwd_fwdmap(X: torch.Tensor, W: torch.Tensor, dY: torch.Tensor, kmap: KernelMap,
                               transpose: bool = False, need_dx: bool = True, need_dw: bool = True,
                               ws: Optional[torch.Tensor] = None, stream=None):
    """(dX or None, dW or None) from the forward map alone: the library builds
    the dX map (and its plan) itself.  ``transpose``: the forward pass was the
    transposed convolution on ``kmap`` (out_idx rows of X, in_idx rows of Y)."""
    dt = _dt(X)
    _need(X, X.dtype, "X", 2)
    _need(W, X.dtype, "W", 3)
    _need(dY, X.dtype, "dY", 2)
    K, ci, co = W.shape
    n_in, n_out = X.shape[0], dY.shape[0]
    if X.shape[1] != ci or dY.shape[1] != co or kmap.K != K:
        raise ValueError("shape mismatch")
    dev = X.device
    dX = torch.empty((n_in, ci), dtype=X.dtype, device=dev) if need_dx else None
    dW = torch.empty((K, ci, co), dtype=torch.float32, device=dev) if need_dw else None
    if ws is None:
        ws = _ws(lib().gsc_conv_bwd_fwdmap_ws_bytes(dt, n_in, kmap.n_bound, ci, co, K), dev)
    _check(lib().gsc_sparse_conv_bwd_fwdmap(
        dt, _ptr(X), _ptr(W), _ptr(dY), n_in, ci, co, K, _ptr(kmap.in_idx), _ptr(kmap.out_idx), _ptr(kmap.seg),
        kmap.n_bound, 1 if transpose else 0, _ptr(dX) if need_dx else None, _ptr(dW) if need_dw else None, n_out,
        _ptr(ws), ws.numel(), _stream(stream)))
    return dX, dW


def gsc_affine_act_bwd(Y: torch.Tensor, dY: torch.Tensor, scale: Optional[torch.Tensor] = None,
                       shift: Optional[torch.Tensor] = None, relu: bool = False, need_sums: bool = True,
                       stream=None):
    """Backward of gsc_sparse_conv_fwd_affine's epilogue: (dZ, dscale, dshift),
    dZ the gradient of the convolution's sums (Y's dtype), dscale and dshift
    float32 per channel (None without ``need_sums``)."""
    _need(Y, Y.dtype, "Y", 2)
    _need(dY, Y.dtype, "dY", 2)
    n, c = Y.shape
    if dY.shape != Y.shape:
        raise ValueError("dY must have Y's shape")
    dev = Y.device
    dZ = torch.empty_like(Y)
    dsc = torch.empty(c, dtype=torch.float32, device=dev) if need_sums else None
    dsh = torch.empty(c, dtype=torch.float32, device=dev) if need_sums else None
    ws = _ws(lib().gsc_affine_act_bwd_ws_bytes(n, c), dev) if need_sums else None
    _check(lib().gsc_affine_act_bwd(_dt(Y), _ptr(Y), _ptr(dY), n, c, None if scale is None else _ptr(scale),
                                    None if shift is None else _ptr(shift), GSC_ACT_RELU if relu else GSC_ACT_NONE,
                                    _ptr(dZ), None if dsc is None else _ptr(dsc), None if dsh is None else _ptr(dsh),
                                    None if ws is None else _ptr(ws), 0 if ws is None else ws.numel(),
                                    _stream(stream)))
    return dZ, dsc, dsh


# --------------------------------------------------------------------------- #
# pooling (Sec. 4.3, 4.4)
# --------------------------------------------------------------------------- #
@dataclasses.dataclass
class Pooled:
    Y: torch.Tensor                  # float32 [n_out, C]
    arg: Optional[torch.Tensor]      # int32 [n_out, C]: input row of the maximum (max pooling)
    cnt: torch.Tensor                # int32 [n_out]: inputs per output


def gsc_sparse_pool_fwd(X: torch.Tensor, kmap: KernelMap, mode: str, stream=None,
                        out: Optional[Pooled] = None) -> Pooled:
    """Pooling of ``X`` over a kernel map built with ``dense=True``; ``out``
    (optional) holds preallocated output buffers."""
    _need(X, torch.float32, "X", 2)
    if kmap.nbr is None:
        raise ValueError("pooling needs the map's dense form (gsc_kernel_map(..., dense=True))")
    m = POOL_MODES[mode]
    n_out, C = kmap.n_out, X.shape[1]
    if out is None:
        out = Pooled(torch.empty((n_out, C), dtype=torch.float32, device=X.device),
                     torch.empty((n_out, C), dtype=torch.int32, device=X.device) if m == GSC_POOL_MAX else None,
                     torch.empty((n_out,), dtype=torch.int32, device=X.device))
    Y, arg, cnt = out.Y[:n_out], (out.arg[:n_out] if out.arg is not None else None), out.cnt[:n_out]
    if m == GSC_POOL_MAX and arg is None:
        raise ValueError("max pooling needs an arg buffer")
    _check(lib().gsc_sparse_pool_fwd(m, _ptr(X), X.shape[0], C, _ptr(kmap.nbr), kmap.K, n_out, _ptr(Y), _ptr(arg),
                                     _ptr(cnt), _stream(stream)))
    return Pooled(Y, arg, cnt)


def gsc_sparse_pool_bwd(dY: torch.Tensor, tmap: KernelMap, mode: str, pooled: Pooled, stream=None,
                        dX: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Input gradient of gsc_sparse_pool_fwd; ``tmap`` is the role-reversed map
    (dense form over the input rows)."""
    _need(dY, torch.float32, "dY", 2)
    if tmap.nbr is None:
        raise ValueError("the pooling gradient needs the role-reversed map's dense form")
    m = POOL_MODES[mode]
    n_in, C = tmap.n_out, dY.shape[1]
    if dX is None:
        dX = torch.empty((n_in, C), dtype=torch.float32, device=dY.device)
    _check(lib().gsc_sparse_pool_bwd(m, _ptr(dY), dY.shape[0], C, _ptr(tmap.nbr), tmap.K, n_in, _ptr(pooled.arg),
                                     _ptr(pooled.cnt), _ptr(dX), _stream(stream)))
    return dX


def gsc_global_pool_fwd(X: torch.Tensor, coords: torch.Tensor, n_batch: int, mode: str, stream=None) -> Pooled:
    """Global pooling: one output row per batch index (column 0 of ``coords``)."""
    _need(X, torch.float32, "X", 2)
    _need(coords, torch.int32, "coords", 2)
    m = POOL_MODES[mode]
    n, C = X.shape
    D = coords.shape[1] - 1
    Y = torch.empty((n_batch, C), dtype=torch.float32, device=X.device)
    arg = torch.empty((n_batch, C), dtype=torch.int32, device=X.device) if m == GSC_POOL_MAX else None
    cnt = torch.empty((n_batch,), dtype=torch.int32, device=X.device)
    ws = _ws(lib().gsc_global_pool_ws_bytes(n, C, n_batch), X.device)
    _check(lib().gsc_global_pool_fwd(m, _ptr(X), n, C, _ptr(coords), D, n_batch, _ptr(Y), _ptr(arg), _ptr(cnt),
                                     _ptr(ws), ws.numel(), _stream(stream)))
    return Pooled(Y, arg, cnt)


def gsc_global_pool_bwd(dY: torch.Tensor, coords: torch.Tensor, mode: str, pooled: Pooled, stream=None) -> torch.Tensor:
    _need(dY, torch.float32, "dY", 2)
    m = POOL_MODES[mode]
    n, C = coords.shape[0], dY.shape[1]
    dX = torch.empty((n, C), dtype=torch.float32, device=dY.device)
    _check(lib().gsc_global_pool_bwd(m, _ptr(dY), dY.shape[0], C, _ptr(coords), coords.shape[1] - 1, n,
                                     _ptr(pooled.arg), _ptr(pooled.cnt), _ptr(dX), _stream(stream)))
    return dX


# --------------------------------------------------------------------------- #
# sparse tensor quantization (Sec. 4.1, Alg. 1)
# --------------------------------------------------------------------------- #
@dataclasses.dataclass
class Quantized:
    coords: torch.Tensor             # int32 [n_out, 1 + D]
    rep: torch.Tensor                # int32 [n_out]: first point of each voxel
    labels: Optional[torch.Tensor]   # int32 [n_out] (when labels were given)
    inverse: torch.Tensor            # int32 [n]: voxel row of every point
    table: torch.Tensor              # hash table of the voxel coordinates


def gsc_quantize(points: torch.Tensor, voxel, batch: Optional[torch.Tensor] = None,
                 labels: Optional[torch.Tensor] = None, ignore_label: int = -100, stream=None) -> Quantized:
    _need(points, torch.float32, "points", 2)
    n, D = points.shape
    dev = points.device
    if batch is not None:
        _need(batch, torch.int32, "batch", 1)
    if labels is not None:
        _need(labels, torch.int32, "labels", 1)
    v = [float(voxel)] * D if np.isscalar(voxel) else [float(x) for x in voxel]
    hv = (ctypes.c_float * D)(*v)
    out = torch.empty((max(n, 1), D + 1), dtype=torch.int32, device=dev)
    rep = torch.empty((max(n, 1),), dtype=torch.int32, device=dev)
    out_labels = torch.empty((max(n, 1),), dtype=torch.int32, device=dev) if labels is not None else None
    inverse = torch.empty((max(n, 1),), dtype=torch.int32, device=dev)
    table = torch.empty(gsc_table_bytes(n), dtype=torch.uint8, device=dev)
    ws = _ws(lib().gsc_quantize_ws_bytes(n, D), dev)
    n_out = ctypes.c_int64(0)
    _check(lib().gsc_quantize(_ptr(points), _ptr(batch), n, D, hv, _ptr(labels), ignore_label, _ptr(out),
                              ctypes.byref(n_out), _ptr(rep), _ptr(out_labels), _ptr(inverse), _ptr(table),
                              table.numel(), _ptr(ws), ws.numel(), _stream(stream)))
    m = n_out.value
    return Quantized(out[:m], rep[:m], None if out_labels is None else out_labels[:m], inverse[:n], table)
