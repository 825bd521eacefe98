"""Kernel regions N^D as explicit offset lists (host configuration).

Sec. 3.1 defines the generalized sparse convolution over an arbitrary offset
set N^D; the hypercube V^D(K) is the usual one (V^1(3) = {-1, 0, 1}).  Sec. 5.1
and Fig. 3 name the cross / hypercross and the hybrid kernel (a spatial cube
at zero time offset plus a temporal cross).  The spatial region (the cube of
the first D - 1 axes at zero offset on the last) is the 3D convolution applied
to every frame of a 3D video on its own, the 3D counterpart of Sec. 7.  The library takes the offsets
as a K x D array, so every region is just a different list; the order of the
list fixes which weight matrix W[k] belongs to which offset.  Lists here are
in lexicographic order of the offset tuples (last axis fastest).  For even
K the axis set is {-floor((K-1)/2), ..., ceil((K-1)/2)}, i.e. {0, 1} for K = 2.
"""
from __future__ import annotations

import itertools

import numpy as np


def _axis(K: int):
    lo = -((K - 1) // 2)
    return range(lo, lo + K)


def hypercube(K: int, D: int) -> np.ndarray:
    return np.array(list(itertools.product(_axis(K), repeat=D)), dtype=np.int32).reshape(-1, D)


def hypercross(K: int, D: int) -> np.ndarray:
    s = set()
    for d in range(D):
        for j in _axis(K):
            o = [0] * D
            o[d] = j
            s.add(tuple(o))
    return np.array(sorted(s), dtype=np.int32).reshape(-1, D)


def hybrid(K: int, D: int) -> np.ndarray:
    s = {tuple(o) + (0,) for o in itertools.product(_axis(K), repeat=D - 1)}
    s |= {(0,) * (D - 1) + (j,) for j in _axis(K)}
    return np.array(sorted(s), dtype=np.int32).reshape(-1, D)


def spatial(K: int, D: int) -> np.ndarray:
    return np.array([tuple(o) + (0,) for o in itertools.product(_axis(K), repeat=D - 1)],
                    dtype=np.int32).reshape(-1, D)


def region(name: str, K: int, D: int) -> np.ndarray:
    return {"cube": hypercube, "cross": hypercross, "hybrid": hybrid, "spatial": spatial}[name](K, D)


def is_symmetric(offsets: np.ndarray) -> bool:
    s = {tuple(o) for o in np.asarray(offsets).tolist()}
    return all(tuple(-v for v in o) in s for o in s)
