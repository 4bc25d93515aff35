"""CPU oracle for the sparse-binary BMU search -- TEST INFRASTRUCTURE ONLY.

Only the test suite, ``__graft_entry__.smoke()`` and the benchmark's
CPU-baseline leg import this package. The product library neither links nor
calls it, and it shares no code with the HIP path.

``oracle.c`` evaluates the definition of the best-matching unit (Method,
problem statement, Eq. (1)): D_i = sum_v (x_v - w_{v,i})^2 in fp64 over all
V features, then the lowest index attaining the minimum. This module wraps
it with ctypes and adds a block-streaming driver: the neuron axis is cut into
contiguous blocks, each block is evaluated by the single-threaded oracle
(several blocks may run on separate threads), and the per-block results are
merged with the same rule (smallest distance, then lowest index), so the
merged answer equals one oracle call over the whole map.

``bmu_sf`` ranks the same way for sparse real-valued rows (a value with each
feature id; the Discussion's gather-multiply variant).

``update`` performs one batch update of the codebook for binary rows (the
factorised box-blur update: scatter, three running-sum box passes per
lattice axis, quotient, zero-denominator units unchanged) in fp32 as the paper
fixes it.

``bmu2`` returns the two best units per sample in the order (distance,
index) -- the pair the paper's fused sweep produces (Figure 2 caption), which
defines the topographic error -- plus the third distance, for margin checks.

Parity status: pinned (see tests/test_oracle_pins.py) by exact integer
arithmetic on quantised codebooks (ranks 1-3 by a pure-Python sort for the
two-best oracle, and the same for real-valued rows), all-ones values
reducing to the binary oracle, exact scaling, scipy's cdist on both layouts, the expanded form of Eq. (1),
planted, tied and constant codebooks, and a mutation check that each
plausible slip in oracle.c fails a pin.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor
from typing import Callable

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

CFLAGS = ["-O2", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off", "-fno-fast-math"]

OK, BAD_ARG, BAD_CSR, NO_MEM = 0, 1, 2, 3


def build(src: str = _SRC, out: str = _LIB) -> str:
    """Compile the oracle with gcc (host code only)."""
    subprocess.run(["gcc", *CFLAGS, src, "-o", out, "-lm"], check=True)
    return out


def load(path: str | None = None):
    """Load an oracle library (the built one by default; tests may pass a variant)."""
    if path is None:
        path = _LIB
        if not os.path.exists(path):
            build()
    lib = ctypes.CDLL(path)
    i64, vp = ctypes.c_int64, ctypes.c_void_p
    lib.som_bmu_oracle_host.argtypes = [vp, i64, i64, i64, i64, vp, vp, i64, vp, vp, vp]
    lib.som_bmu_oracle_host.restype = ctypes.c_int
    lib.som_bmu2_oracle_host.argtypes = [vp, i64, i64, i64, i64, vp, vp, i64, vp, vp, vp, vp, vp]
    lib.som_bmu2_oracle_host.restype = ctypes.c_int
    lib.som_bmu_sf_oracle_host.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, i64, vp, vp, vp, vp, vp]
    lib.som_bmu_sf_oracle_host.restype = ctypes.c_int
    lib.som_update_oracle_host.argtypes = [vp, i64, i64, vp, vp, i64, vp, i64, vp]
    lib.som_update_oracle_host.restype = ctypes.c_int
    lib.som_norms_oracle_host.argtypes = [vp, i64, i64, i64, i64, vp]
    lib.som_norms_oracle_host.restype = ctypes.c_int
    return lib


_default = None


def _lib(lib=None):
    global _default
    if lib is not None:
        return lib
    if _default is None:
        _default = load()
    return _default


def _block_view(W: np.ndarray):
    if W.dtype != np.float32 or W.ndim != 2 or W.strides[1] != 4 or W.strides[0] % 4:
        raise ValueError("W must be a 2-D float32 array (features x neurons) with unit column stride")
    return W.strides[0] // 4


def bmu(W: np.ndarray, row_ptr: np.ndarray, col_idx: np.ndarray, i0: int = 0, lib=None):
    """Dense BMU of every CSR row over the neuron block W (V x B, feature-major).

    Returns (bmu int32[N] with global indices i0 + k, dist fp64[N], dist2 fp64[N]).
    """
    ldw = _block_view(W)
    V, B = W.shape
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    N = row_ptr.shape[0] - 1
    out_b = np.empty(N, dtype=np.int32)
    out_d = np.empty(N, dtype=np.float64)
    out_d2 = np.empty(N, dtype=np.float64)
    rc = _lib(lib).som_bmu_oracle_host(W.ctypes.data, ldw, V, i0, i0 + B, row_ptr.ctypes.data,
                                       col_idx.ctypes.data if col_idx.size else None, N,
                                       out_b.ctypes.data, out_d.ctypes.data, out_d2.ctypes.data)
    if rc != OK:
        raise ValueError(f"som_bmu_oracle_host returned {rc}")
    return out_b, out_d, out_d2


def bmu2(W: np.ndarray, row_ptr: np.ndarray, col_idx: np.ndarray, i0: int = 0, lib=None):
    """The two best units of every CSR row over the neuron block W, ranked by (distance, index).

    Returns (bmu, dist, bmu2, dist2, dist3): ranks 1 and 2 with global indices
    (bmu2 = -1, dist2 = +inf for a one-neuron block) and the rank-3 distance.
    """
    ldw = _block_view(W)
    V, B = W.shape
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    N = row_ptr.shape[0] - 1
    b1 = np.empty(N, dtype=np.int32)
    d1 = np.empty(N, dtype=np.float64)
    b2 = np.empty(N, dtype=np.int32)
    d2 = np.empty(N, dtype=np.float64)
    d3 = np.empty(N, dtype=np.float64)
    rc = _lib(lib).som_bmu2_oracle_host(W.ctypes.data, ldw, V, i0, i0 + B, row_ptr.ctypes.data,
                                        col_idx.ctypes.data if col_idx.size else None, N, b1.ctypes.data,
                                        d1.ctypes.data, b2.ctypes.data, d2.ctypes.data, d3.ctypes.data)
    if rc != OK:
        raise ValueError(f"som_bmu2_oracle_host returned {rc}")
    return b1, d1, b2, d2, d3


def bmu_sf(W: np.ndarray, row_ptr: np.ndarray, col_idx: np.ndarray, values: np.ndarray, i0: int = 0, lib=None):
    """bmu2() for sparse real-valued rows: values[p] is the value of feature col_idx[p].

    Returns (bmu, dist, bmu2, dist2, dist3) as bmu2().
    """
    ldw = _block_view(W)
    V, B = W.shape
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    values = np.ascontiguousarray(values, dtype=np.float32)
    if values.shape != col_idx.shape:
        raise ValueError("values must match col_idx")
    N = row_ptr.shape[0] - 1
    b1 = np.empty(N, dtype=np.int32)
    d1 = np.empty(N, dtype=np.float64)
    b2 = np.empty(N, dtype=np.int32)
    d2 = np.empty(N, dtype=np.float64)
    d3 = np.empty(N, dtype=np.float64)
    rc = _lib(lib).som_bmu_sf_oracle_host(W.ctypes.data, ldw, V, i0, i0 + B, row_ptr.ctypes.data,
                                          col_idx.ctypes.data if col_idx.size else None,
                                          values.ctypes.data if values.size else None, N, b1.ctypes.data,
                                          d1.ctypes.data, b2.ctypes.data, d2.ctypes.data, d3.ctypes.data)
    if rc != OK:
        raise ValueError(f"som_bmu_sf_oracle_host returned {rc}")
    return b1, d1, b2, d2, d3


def bmu_sf_streamed(block_fn: Callable[[int, int], np.ndarray], M: int, row_ptr: np.ndarray, col_idx: np.ndarray,
                    values: np.ndarray, block: int = 4096, nthreads: int = 1, lib=None):
    """bmu_sf() over a whole map whose codebook is produced block by block (see bmu_streamed)."""
    starts = list(range(0, M, block))

    def run(i0):
        i1 = min(M, i0 + block)
        return bmu_sf(block_fn(i0, i1), row_ptr, col_idx, values, i0=i0, lib=lib)

    if nthreads <= 1:
        parts = [run(i0) for i0 in starts]
    else:
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            parts = list(ex.map(run, starts))
    return merge_blocks2(parts)


def distance_sf_at(column: np.ndarray, ids: np.ndarray, vals: np.ndarray) -> float:
    """D for one neuron and one real-valued row."""
    col = np.ascontiguousarray(column, dtype=np.float32).reshape(-1, 1)
    rp = np.array([0, len(ids)], dtype=np.int32)
    return float(bmu_sf(col, rp, np.asarray(ids, dtype=np.int32), np.asarray(vals, dtype=np.float32))[1][0])


def update(W: np.ndarray, E: int, row_ptr: np.ndarray, col_idx: np.ndarray, bmu: np.ndarray, radius: int, lib=None):
    """One batch update of the V x (E*E) feature-major codebook W (binary rows, their best units); returns the new W."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    V, M = W.shape
    if M != E * E:
        raise ValueError("W must have E*E columns")
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    bmu = np.ascontiguousarray(bmu, dtype=np.int32)
    N = row_ptr.shape[0] - 1
    out = np.empty_like(W)
    rc = _lib(lib).som_update_oracle_host(W.ctypes.data, V, E, row_ptr.ctypes.data if N >= 0 else None,
                                          col_idx.ctypes.data if col_idx.size else None, N,
                                          bmu.ctypes.data if N else None, radius, out.ctypes.data)
    if rc != OK:
        raise ValueError(f"som_update_oracle_host returned {rc}")
    return out


def norms(W: np.ndarray, lib=None) -> np.ndarray:
    """n_i = sum_v w_{v,i}^2 (fp64, v ascending) for every column of W."""
    ldw = _block_view(W)
    V, B = W.shape
    out = np.empty(B, dtype=np.float64)
    rc = _lib(lib).som_norms_oracle_host(W.ctypes.data, ldw, V, 0, B, out.ctypes.data)
    if rc != OK:
        raise ValueError(f"som_norms_oracle_host returned {rc}")
    return out


def merge_blocks(parts):
    """Merge per-block (bmu, dist, dist2) results, given in ascending block order.

    The best is the smallest distance, the earliest block winning a tie (its
    index is the lower one); the second best is the smaller of the winning
    block's own second best and every other block's best.
    """
    b = parts[0][0].copy()
    d = parts[0][1].copy()
    d2 = parts[0][2].copy()
    for pb, pd, pd2 in parts[1:]:
        better = pd < d
        # the loser's best becomes a second-best candidate
        new_d2 = np.where(better, np.minimum(pd2, d), np.minimum(d2, pd))
        b = np.where(better, pb, b)
        d = np.where(better, pd, d)
        d2 = new_d2
    return b, d, d2


def merge_blocks2(parts):
    """Merge per-block bmu2() results (any block order).

    A unit in the global first two is among its own block's first two, so
    ranks 1 and 2 are the first two of all blocks' first-two lists in the
    order (distance, index); the k-th smallest distance of the whole map is
    the k-th smallest of all blocks' first three distances.
    """
    cd = np.stack([p[1] for p in parts] + [p[3] for p in parts], axis=1)
    cb = np.stack([p[0] for p in parts] + [p[2] for p in parts], axis=1).astype(np.int64)
    cb = np.where(cb < 0, np.iinfo(np.int64).max, cb)  # an absent rank 2 sorts last
    order = np.lexsort((cb, cd), axis=-1)
    rows = np.arange(cd.shape[0])
    b1 = cb[rows, order[:, 0]]
    b2 = cb[rows, order[:, 1]]
    dist_all = np.sort(np.stack([p[k] for p in parts for k in (1, 3, 4)], axis=1), axis=1)
    d1, d2, d3 = dist_all[:, 0], dist_all[:, 1], dist_all[:, 2]
    b2 = np.where(np.isinf(d2), -1, b2)
    return b1.astype(np.int32), d1, b2.astype(np.int32), d2, d3


def bmu2_streamed(block_fn: Callable[[int, int], np.ndarray], M: int, row_ptr: np.ndarray, col_idx: np.ndarray,
                  block: int = 4096, nthreads: int = 1, lib=None):
    """bmu2() over a whole map whose codebook is produced block by block (see bmu_streamed)."""
    starts = list(range(0, M, block))

    def run(i0):
        i1 = min(M, i0 + block)
        return bmu2(block_fn(i0, i1), row_ptr, col_idx, i0=i0, lib=lib)

    if nthreads <= 1:
        parts = [run(i0) for i0 in starts]
    else:
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            parts = list(ex.map(run, starts))
    return merge_blocks2(parts)


def bmu_streamed(block_fn: Callable[[int, int], np.ndarray], M: int, row_ptr: np.ndarray, col_idx: np.ndarray,
                 block: int = 4096, nthreads: int = 1, lib=None):
    """Oracle over a whole map whose codebook is produced block by block.

    block_fn(i0, i1) must return the V x (i1-i0) feature-major float32 block
    of neurons [i0, i1). Blocks are evaluated independently (on up to
    nthreads threads, each running the single-threaded oracle) and merged.
    """
    starts = list(range(0, M, block))

    def run(i0):
        i1 = min(M, i0 + block)
        return bmu(block_fn(i0, i1), row_ptr, col_idx, i0=i0, lib=lib)

    if nthreads <= 1:
        parts = [run(i0) for i0 in starts]
    else:
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            parts = list(ex.map(run, starts))
    return merge_blocks(parts)


def distance_at(column: np.ndarray, ids: np.ndarray) -> float:
    """D for one neuron: column is its V weights (float32), ids the active features."""
    col = np.ascontiguousarray(column, dtype=np.float32).reshape(-1, 1)
    rp = np.array([0, len(ids)], dtype=np.int32)
    _, d, _ = bmu(col, rp, np.asarray(ids, dtype=np.int32))
    return float(d[0])
