"""CPU oracle for the generalized sparse convolution.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this module.  The HIP library never calls it, and it imports nothing from the
HIP path: the two share no code.  It is deliberately plain and slow: a Python
dict maps coordinates to rows, the kernel map is built by one dict lookup per
(output, offset), and the convolution is a loop over offsets of float64
matmuls.  Every function below cites the passage of the paper it writes out.

Conventions (readings of the paper, listed with the others in the design notes):
  * a coordinate row is (b, x1..xD): batch index first (Sec. 3, Eq. 1 puts it
    last; only the column order differs);
  * ``W[k]`` is C_in x C_out, the transpose of the paper's W_i of Sec. 3.1, so a
    row-major feature row f contributes ``f @ W[k]``;
  * offsets are applied as in Eq. 3: output u reads input u + i (no flip);
  * the batch component of a coordinate is never offset or strided.

Parity status: every function is pinned by the CPU tests (brute-force maps,
closed-form counts, dense-convolution special cases, adjoint identities, finite
differences, dense max/average pooling and their gradients, per-batch
reductions, hand-written quantization examples (exact floors at voxel sizes
that are not powers of two among them), np.unique and the floor's bracketing
inequality in integer arithmetic, batch
statistics after normalisation); the row order
of ``output_coordinates`` is an implementation choice and is compared
canonically, not pinned.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction
from typing import Dict, List, Sequence, Tuple

import numpy as np

Pairs = Tuple[np.ndarray, np.ndarray]     # (I_k, O_k) int64 arrays


class DuplicateCoordinate(ValueError):
    pass


# --------------------------------------------------------------------------- #
# Kernel regions  (Sec. 3.1: hypercube V^D(K) and arbitrary offset sets N^D;
# Sec. 5.1 / Fig. 3: cross, hypercross, hybrid)
# --------------------------------------------------------------------------- #
def axis_offsets(K: int) -> List[int]:
    """V^1(K): K consecutive integers around the origin.

    Sec. 3.1 gives V^1(3) = {-1, 0, 1}.  For even K a centred set does not
    exist; the reading used here is {-floor((K-1)/2), ..., ceil((K-1)/2)}, i.e.
    {0, 1} for K = 2 (the kernel of a stride-2 down-sampling convolution)."""
    lo = -((K - 1) // 2)
    return list(range(lo, lo + K))


def hypercube(K: int, D: int) -> np.ndarray:
    """V^D(K) = (V^1(K))^D, in lexicographic order (last axis fastest)."""
    return np.array(list(itertools.product(axis_offsets(K), repeat=D)), dtype=np.int64).reshape(-1, D)


def hypercross(K: int, D: int) -> np.ndarray:
    """The origin plus the offsets along each single axis within V^1(K)
    (the "cross"/"hypercross" of Fig. 3), sorted lexicographically."""
    pts = {tuple([0] * D)}
    for d in range(D):
        for j in axis_offsets(K):
            o = [0] * D
            o[d] = j
            pts.add(tuple(o))
    return np.array(sorted(pts), dtype=np.int64).reshape(-1, D)


def hybrid(K: int, D: int) -> np.ndarray:
    """Hybrid kernel of Sec. 5.1: a cube over the D-1 spatial axes at zero time
    offset, plus a cross along the last (time) axis through the origin."""
    pts = {tuple(o) + (0,) for o in itertools.product(axis_offsets(K), repeat=D - 1)}
    for j in axis_offsets(K):
        pts.add(tuple([0] * (D - 1)) + (j,))
    return np.array(sorted(pts), dtype=np.int64).reshape(-1, D)


def spatial(K: int, D: int) -> np.ndarray:
    """The cube over the D-1 spatial axes at zero time offset: a 3D convolution
    of every frame of a 3D video on its own (the 3D counterpart of Sec. 7)."""
    pts = [tuple(o) + (0,) for o in itertools.product(axis_offsets(K), repeat=D - 1)]
    return np.array(sorted(pts), dtype=np.int64).reshape(-1, D)


def region(name: str, K: int, D: int) -> np.ndarray:
    return {"cube": hypercube, "cross": hypercross, "hybrid": hybrid, "spatial": spatial}[name](K, D)


# --------------------------------------------------------------------------- #
# Coordinate map (Sec. 3: COO coordinates with batch index; Sec. 2 / Sec. 4:
# a hash table answers neighbour queries -- a Python dict here)
# --------------------------------------------------------------------------- #
def coordinate_map(coords: np.ndarray) -> Dict[tuple, int]:
    """Map each coordinate row to its row index.  Coordinates of a sparse tensor
    are unique; a repeated row is an error (it would make Eq. 3 ambiguous)."""
    m: Dict[tuple, int] = {}
    for r, row in enumerate(np.asarray(coords).tolist()):
        key = tuple(row)
        if key in m:
            raise DuplicateCoordinate(f"row {r} repeats row {m[key]}: {key}")
        m[key] = r
    return m


# --------------------------------------------------------------------------- #
# Output coordinates (Sec. 4.2): from the convolution stride, the input
# coordinates and the input tensor stride.
# --------------------------------------------------------------------------- #
def output_coordinates(coords: np.ndarray, stride: Sequence[int] | int) -> np.ndarray:
    """C^out of a strided convolution: every spatial component c is replaced by
    floor(c / s) * s (floor, so -1 -> -2 for s = 2), the batch index is kept, and
    repeated rows are merged.  Stride 1 leaves C^in unchanged (the submanifold
    case of Sec. 3.1, same rows, same order).  Otherwise rows are returned in
    lexicographic order."""
    coords = np.asarray(coords)
    D = coords.shape[1] - 1
    s = [stride] * D if np.isscalar(stride) else list(stride)
    if all(v == 1 for v in s):
        return coords.astype(np.int64).copy()
    out = set()
    for row in coords.tolist():
        out.add((row[0],) + tuple((c // sd) * sd for c, sd in zip(row[1:], s)))
    return np.array(sorted(out), dtype=np.int64).reshape(-1, D + 1)


# --------------------------------------------------------------------------- #
# Kernel map (Sec. 4.2): M = {(I_i, O_i)}_i, for every offset i the input rows
# and output rows it connects; Eq. 3 defines which: u in C^out reads u + i
# when u + i is in C^in.
# --------------------------------------------------------------------------- #
def kernel_map(in_coords: np.ndarray, out_coords: np.ndarray, offsets: np.ndarray,
               tensor_stride: Sequence[int] | int = 1) -> List[Pairs]:
    """For each offset o_k (row of ``offsets``) the pairs (row of u + ts*o_k in
    C^in, row of u in C^out), listed in increasing output row."""
    in_map = coordinate_map(in_coords)
    out_rows = np.asarray(out_coords).tolist()
    D = np.asarray(offsets).shape[1]
    ts = [tensor_stride] * D if np.isscalar(tensor_stride) else list(tensor_stride)
    maps = []
    for o in np.asarray(offsets).tolist():
        step = [t * v for t, v in zip(ts, o)]
        I, O = [], []
        for j, u in enumerate(out_rows):
            q = (u[0],) + tuple(a + b for a, b in zip(u[1:], step))
            r = in_map.get(q)
            if r is not None:
                I.append(r)
                O.append(j)
        maps.append((np.array(I, dtype=np.int64), np.array(O, dtype=np.int64)))
    return maps


def transposed_map(maps: List[Pairs]) -> List[Pairs]:
    """Sec. 4.2, last sentence: the transposed convolution exchanges the roles
    of input and output coordinates, so each (I_k, O_k) becomes (O_k, I_k);
    pairs are re-listed in increasing (new) output row."""
    out = []
    for I, O in maps:
        order = np.argsort(I, kind="stable")
        out.append((O[order].copy(), I[order].copy()))
    return out


# --------------------------------------------------------------------------- #
# Convolution (Alg. 2 for the forward pass; backward by the chain rule of Eq. 3)
# --------------------------------------------------------------------------- #
def conv_forward(X: np.ndarray, W: np.ndarray, maps: List[Pairs], n_out: int) -> np.ndarray:
    """Alg. 2: F^o <- 0, then for every offset k gather the input rows I_k,
    multiply by the offset's weight and add the result into rows O_k."""
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    Y = np.zeros((n_out, W.shape[2]), dtype=np.float64)
    for k, (I, O) in enumerate(maps):
        if len(I) == 0:
            continue
        assert len(np.unique(O)) == len(O), "an offset maps two inputs to one output"
        Y[O] += X[I] @ W[k]
    return Y


def conv_backward(X: np.ndarray, W: np.ndarray, dY: np.ndarray, maps: List[Pairs]):
    """Gradients of Alg. 2.  Y[O_k] += X[I_k] W_k for every k, so
    dX[I_k] += dY[O_k] W_k^T and dW_k = X[I_k]^T dY[O_k] (zero for an empty k)."""
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    dY = np.asarray(dY, dtype=np.float64)
    dX = np.zeros_like(X)
    dW = np.zeros_like(W)
    for k, (I, O) in enumerate(maps):
        if len(I) == 0:
            continue
        assert len(np.unique(I)) == len(I), "an offset maps one input to two outputs"
        dX[I] += dY[O] @ W[k].T
        dW[k] = X[I].T @ dY[O]
    return dX, dW


# --------------------------------------------------------------------------- #
# Non-spatial functions (Sec. 4.5) on the output features of a convolution:
# batch normalisation (in the per-channel affine form it takes once its
# statistics are known) and ReLU act on each row on its own
# --------------------------------------------------------------------------- #
def batchnorm_coefficients(Y: np.ndarray, gamma=None, beta=None, eps: float = 1e-5):
    """scale, shift with scale * y + shift = gamma (y - mean) / sqrt(var + eps) + beta,
    mean and (biased) variance taken per channel over the rows of Y."""
    Y = np.asarray(Y, dtype=np.float64)
    C = Y.shape[1]
    gamma = np.ones(C) if gamma is None else np.asarray(gamma, dtype=np.float64)
    beta = np.zeros(C) if beta is None else np.asarray(beta, dtype=np.float64)
    mean = Y.mean(axis=0)
    var = Y.var(axis=0)
    scale = gamma / np.sqrt(var + eps)
    return scale, beta - mean * scale


def affine_act(Y: np.ndarray, scale=None, shift=None, relu: bool = False) -> np.ndarray:
    """Y * scale + shift per channel (column), then max(., 0) if relu."""
    Z = np.array(Y, dtype=np.float64)
    if scale is not None:
        Z = Z * np.asarray(scale, dtype=np.float64)[None, :]
    if shift is not None:
        Z = Z + np.asarray(shift, dtype=np.float64)[None, :]
    return np.maximum(Z, 0.0) if relu else Z


def affine_act_backward(S: np.ndarray, dY: np.ndarray, scale=None, shift=None, relu: bool = False):
    """Gradients of Y = affine_act(S, scale, shift, relu) (Sec. 4.5's
    non-spatial functions, by the chain rule per element): with G = dY where
    S * scale + shift > 0 (everywhere without the ReLU), returns dS = G * scale
    and, per channel, dscale = sum over rows of G * S and dshift = sum of G."""
    S = np.asarray(S, dtype=np.float64)
    G = np.array(dY, dtype=np.float64)
    C = S.shape[1]
    sc = np.ones(C) if scale is None else np.asarray(scale, dtype=np.float64)
    sh = np.zeros(C) if shift is None else np.asarray(shift, dtype=np.float64)
    if relu:
        G[S * sc[None, :] + sh[None, :] <= 0.0] = 0.0
    return G * sc[None, :], (G * S).sum(axis=0), G.sum(axis=0)


# --------------------------------------------------------------------------- #
# Eq. 3 evaluated one output (or one input) row at a time, for sampled checks
# at sizes where the full map is too slow in Python.
# --------------------------------------------------------------------------- #
def conv_forward_rows(X: np.ndarray, W: np.ndarray, in_map: Dict[tuple, int], out_coords: np.ndarray,
                      rows: Sequence[int], offsets: np.ndarray,
                      tensor_stride: Sequence[int] | int = 1) -> np.ndarray:
    """Eq. 3 for the listed outputs u: sum over offsets i with u + i in C^in of
    x^in_{u+i} W_i."""
    W = np.asarray(W, dtype=np.float64)
    offs = np.asarray(offsets).tolist()
    D = len(offs[0])
    ts = [tensor_stride] * D if np.isscalar(tensor_stride) else list(tensor_stride)
    Y = np.zeros((len(rows), W.shape[2]))
    for n, j in enumerate(rows):
        u = [int(v) for v in out_coords[j]]
        for k, o in enumerate(offs):
            q = (u[0],) + tuple(a + t * b for a, t, b in zip(u[1:], ts, o))
            r = in_map.get(q)
            if r is not None:
                Y[n] += np.asarray(X[r], dtype=np.float64) @ W[k]
    return Y


def conv_dx_rows(dY: np.ndarray, W: np.ndarray, out_map: Dict[tuple, int], in_coords: np.ndarray,
                 rows: Sequence[int], offsets: np.ndarray,
                 tensor_stride: Sequence[int] | int = 1) -> np.ndarray:
    """dX for the listed input rows r: input c_r feeds output u = c_r - i
    through offset i whenever that u is in C^out, so
    dX[r] = sum_i dY[u] W_i^T over those i."""
    W = np.asarray(W, dtype=np.float64)
    offs = np.asarray(offsets).tolist()
    D = len(offs[0])
    ts = [tensor_stride] * D if np.isscalar(tensor_stride) else list(tensor_stride)
    dX = np.zeros((len(rows), W.shape[1]))
    for n, r in enumerate(rows):
        c = [int(v) for v in in_coords[r]]
        for k, o in enumerate(offs):
            q = (c[0],) + tuple(a - t * b for a, t, b in zip(c[1:], ts, o))
            j = out_map.get(q)
            if j is not None:
                dX[n] += np.asarray(dY[j], dtype=np.float64) @ W[k].T
    return dX


def map_pair_count(maps: List[Pairs]) -> int:
    return int(sum(len(I) for I, _ in maps))


# --------------------------------------------------------------------------- #
# Sparse tensor quantization (Sec. 4.1, Alg. 1)
# --------------------------------------------------------------------------- #
def floor_quotient(p, v) -> int:
    """floor(p / v) for two stored float32 values, taken on the exact real
    quotient (Sec. 4.1, Alg. 1 floors C_p / v_l with C_p real-valued).
    ``Fraction(float(x))`` is the exact binary value of x, so no rounded
    quotient decides on which side of a voxel boundary a point falls."""
    return math.floor(Fraction(float(p)) / Fraction(float(v)))


def quantize(points: np.ndarray, batch: np.ndarray, voxel, labels=None, ignore_label: int = -100):
    """Alg. 1 in the paper's order.  C' = floor(C / v) per spatial axis, the
    floor of the exact quotient of the stored float32 point and voxel size
    (``floor_quotient``); the keys are the coordinate rows (batch index first); the pairs
    (i, l) are sorted by key, stably, so within a key the points keep their
    order; UniqueByKey keeps the first point of every run of equal (key,
    label); ReduceByKey merges the runs of one key with f, which turns any
    second run into IGNORE_LABEL and keeps the first point.  Returns the
    voxel coordinates (n_out x (1+D) int64, in key order), the representative
    point of each voxel, its label (None without labels) and, for every
    point, the row of its voxel."""
    P = np.asarray(points, dtype=np.float32)
    N, D = P.shape
    v = np.broadcast_to(np.asarray(voxel, dtype=np.float32), (D,))
    Cq = [[floor_quotient(x, v[d]) for d, x in enumerate(row)] for row in P.tolist()]   # C'_p
    keys = [(int(b),) + tuple(int(x) for x in row) for b, row in zip(np.asarray(batch).tolist(), Cq)]
    lab = [0] * N if labels is None else [int(x) for x in np.asarray(labels).tolist()]
    order = sorted(range(N), key=lambda i: keys[i])                   # SortByKey (stable)
    runs = []                                                         # UniqueByKey on (key, label)
    for i in order:
        if not runs or runs[-1][0] != keys[i] or runs[-1][1] != lab[i]:
            runs.append((keys[i], lab[i], i))
    vox, rep, out_lab = [], [], []                                    # ReduceByKey with f
    for key, l, i in runs:
        if vox and vox[-1] == key:
            out_lab[-1] = ignore_label
        else:
            vox.append(key)
            rep.append(i)
            out_lab.append(l)
    row_of = {k: r for r, k in enumerate(vox)}
    inverse = np.array([row_of[k] for k in keys], dtype=np.int64)
    return (np.array(vox, dtype=np.int64).reshape(-1, D + 1), np.array(rep, dtype=np.int64),
            None if labels is None else np.array(out_lab, dtype=np.int64), inverse)


# --------------------------------------------------------------------------- #
# Pooling over a kernel map (Sec. 4.3, Alg. 3; Sec. 4.4, Alg. 4)
# --------------------------------------------------------------------------- #
POOL_MODES = ("max", "avg", "sum")


def pool_pairs(maps: List[Pairs]) -> Pairs:
    """The concatenated lists I and O of Sec. 4.3 (all offsets' pairs, in
    offset order), stably sorted by output row as in the first step of Alg. 3
    (SortByKey(I, key=O)), so each output's inputs keep their offset order."""
    I = np.concatenate([np.asarray(a, dtype=np.int64) for a, _ in maps]) if maps else np.zeros(0, np.int64)
    O = np.concatenate([np.asarray(b, dtype=np.int64) for _, b in maps]) if maps else np.zeros(0, np.int64)
    order = np.argsort(O, kind="stable")
    return I[order], O[order]


def pool_forward(X: np.ndarray, maps: List[Pairs], n_out: int, mode: str):
    """Pooling of the input features over the kernel map M = (I, O).

    max (Sec. 4.3, Alg. 3): for every output coordinate, the channel-wise
    maximum over the inputs mapped to it; ``arg`` holds, per output and
    channel, the input row attaining it (the first such input in the sorted
    pair list), for the backward pass.
    avg / sum (Sec. 4.4, Alg. 4): F' = S_M F with S_M the 0/1 matrix of the
    map (row = O, column = I), N = S_M 1, and avg returns F' / N; sum pooling
    (the variant without the division) returns F'.
    An output with no input is 0 (arg -1, N 0).  Returns (Y, arg, N)."""
    assert mode in POOL_MODES
    X = np.asarray(X, dtype=np.float64)
    C = X.shape[1]
    I, O = pool_pairs(maps)
    Y = np.zeros((n_out, C))
    arg = np.full((n_out, C), -1, dtype=np.int64)
    N = np.zeros(n_out, dtype=np.int64)
    for i, j in zip(I.tolist(), O.tolist()):
        N[j] += 1
        if mode == "max":
            for c in range(C):
                if arg[j, c] < 0 or X[i, c] > Y[j, c]:
                    Y[j, c] = X[i, c]
                    arg[j, c] = i
        else:
            Y[j] += X[i]
    if mode == "avg":
        nz = N > 0
        Y[nz] /= N[nz][:, None]
    return Y, arg, N


def pool_backward(dY: np.ndarray, maps: List[Pairs], n_in: int, mode: str, arg: np.ndarray, N: np.ndarray):
    """Gradient of pool_forward with respect to the input features: sum
    pooling sends dY[j] to every input of j, avg pooling dY[j] / N[j], and max
    pooling dY[j, c] to the input that attained the maximum of channel c."""
    assert mode in POOL_MODES
    dY = np.asarray(dY, dtype=np.float64)
    C = dY.shape[1]
    dX = np.zeros((n_in, C))
    if mode == "max":
        for j in range(dY.shape[0]):
            for c in range(C):
                if arg[j, c] >= 0:
                    dX[arg[j, c], c] += dY[j, c]
        return dX
    I, O = pool_pairs(maps)
    for i, j in zip(I.tolist(), O.tolist()):
        dX[i] += dY[j] / (N[j] if mode == "avg" else 1)
    return dX


def unpool_forward(X: np.ndarray, maps: List[Pairs], n_fine: int, mode: str):
    """Transposed pooling (unpooling, Sec. 4.4): Alg. 4 on the pooling map with
    the roles of I and O reversed, so fine row i receives the sum (sum) or the
    mean (avg) of the coarse rows it is pooled into.  ``maps`` is the pooling
    map (fine inputs I, coarse outputs O); X holds the coarse features.
    Returns (Y, arg, N) as pool_forward, N counting each fine row's coarse rows."""
    assert mode in ("avg", "sum")
    return pool_forward(X, transposed_map(maps), n_fine, mode)


def unpool_backward(dY: np.ndarray, maps: List[Pairs], n_coarse: int, mode: str, N: np.ndarray):
    """Gradient of unpool_forward with respect to the coarse features: coarse
    row j receives dY[i] (sum) or dY[i] / N[i] (avg) of every fine row i
    pooled into it."""
    assert mode in ("avg", "sum")
    return pool_backward(dY, transposed_map(maps), n_coarse, mode, None, N)


def global_pool_forward(X: np.ndarray, batch: np.ndarray, n_batch: int, mode: str):
    """Global pooling (Sec. 4.4): the kernel map sends every input of batch
    index b to one output (the origin of b), then pool_forward; output b is the
    max / mean / sum of the features of batch b's rows."""
    batch = np.asarray(batch, dtype=np.int64)
    maps = [(np.arange(len(batch), dtype=np.int64), batch)]
    return pool_forward(X, maps, n_batch, mode)


def global_pool_backward(dY: np.ndarray, batch: np.ndarray, mode: str, arg: np.ndarray, N: np.ndarray):
    batch = np.asarray(batch, dtype=np.int64)
    maps = [(np.arange(len(batch), dtype=np.int64), batch)]
    return pool_backward(dY, maps, len(batch), mode, arg, N)
