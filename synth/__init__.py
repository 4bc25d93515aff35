"""Seeded synthetic workloads for the sparse-binary BMU search.

Test and benchmark infrastructure: both the HIP path and the CPU oracle take
their inputs from here, and nothing here computes any part of the search.

The inputs stand in for the MEDLINE/MeSH corpus the paper trains on (corpus
section and Table 1: sparse-binary CSR rows of sorted descriptor ids, about
30k descriptors, about 11 per article), which is not available. Row lengths
are 1 + Poisson(11); feature ids are Zipf(1.1) draws over ranks 1..V taken
without replacement (id = rank - 1, so frequent features have low ids);
codebook values come from a counter-based SplitMix64 hash of the element's
feature-major position. Every row and every codebook block is a pure function
of (seed, position).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "synth.c")
_LIB = os.path.join(_HERE, "libsynth.so")

UNIFORM = 0
QUANTISED = 1
UNIFORM_BLUR3 = 2

KIND_NAMES = {UNIFORM: "uniform", QUANTISED: "quantised k/256", UNIFORM_BLUR3: "uniform + 3x3 lattice mean"}


def build() -> str:
    """Compile libsynth.so with gcc (host code only)."""
    cmd = ["gcc", "-O2", "-fPIC", "-shared", "-std=c11", "-Wall", "-Wextra", "-pthread", _SRC, "-o", _LIB, "-lm"]
    subprocess.run(cmd, check=True)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        i64, u64, i32p, f32p = ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p
        lib.synth_codebook.argtypes = [u64, ctypes.c_int, i64, i64, i64, i64, i64, i64, f32p, i64, ctypes.c_int]
        lib.synth_codebook.restype = ctypes.c_int
        lib.synth_csr_row_ptr.argtypes = [u64, i64, i64, ctypes.c_double, i32p, ctypes.c_int]
        lib.synth_csr_row_ptr.restype = ctypes.c_int64
        lib.synth_csr_col_idx.argtypes = [u64, i64, i64, ctypes.c_double, ctypes.c_double, i32p, i32p, ctypes.c_int]
        lib.synth_csr_col_idx.restype = ctypes.c_int
        lib.synth_values.argtypes = [u64, ctypes.c_int, i64, f32p, ctypes.c_int]
        lib.synth_values.restype = ctypes.c_int
        lib.synth_tile_distinct.argtypes = [i32p, i32p, i64, i64, i32p, ctypes.c_int]
        lib.synth_tile_distinct.restype = ctypes.c_int
        _lib = lib
    return _lib


def default_threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


@dataclass(frozen=True)
class Config:
    name: str
    edge: int          # lattice edge E, M = E*E
    V: int             # features
    N: int             # samples in one batch
    kind: int          # codebook value kind
    seed: int
    lam: float = 11.0  # row length = 1 + Poisson(lam)
    zipf_s: float = 1.1

    @property
    def M(self) -> int:
        return self.edge * self.edge

    def describe(self) -> str:
        return (f"{self.edge}x{self.edge} map (M={self.M}), V={self.V}, N={self.N}, "
                f"nnz=1+Poisson({self.lam:g}), Zipf({self.zipf_s:g}) ids, "
                f"codebook {KIND_NAMES[self.kind]} fp32 feature-major, seed {self.seed}")


CONFIGS = {
    "tiny": Config("tiny", 16, 2000, 10_000, QUANTISED, 0),
    "64": Config("64", 64, 30_000, 29_900_000, UNIFORM, 1),
    "256": Config("256", 256, 30_000, 4_000_000, UNIFORM, 2),
    "512": Config("512", 512, 30_000, 2_000_000, UNIFORM_BLUR3, 3),
    "1024": Config("1024", 1024, 30_000, 500_000, UNIFORM, 4),
}


def make_csr(seed: int, N: int, V: int, lam: float = 11.0, zipf_s: float = 1.1, nthreads: int | None = None):
    """Sparse-binary CSR batch: (row_ptr int32[N+1], col_idx int32[nnz]); rows sorted, distinct ids."""
    lib = _load()
    nt = nthreads or default_threads()
    row_ptr = np.empty(N + 1, dtype=np.int32)
    total = lib.synth_csr_row_ptr(seed, N, V, lam, _ptr(row_ptr), nt)
    if total < 0:
        raise ValueError(f"synth_csr_row_ptr failed ({total})")
    col_idx = np.empty(max(total, 1), dtype=np.int32)[:total]
    rc = lib.synth_csr_col_idx(seed, N, V, lam, zipf_s, _ptr(row_ptr), _ptr(col_idx) if total else None, nt)
    if rc != 0:
        raise ValueError(f"synth_csr_col_idx failed ({rc})")
    return row_ptr, col_idx


def codebook(seed: int, kind: int, V: int, M: int, v0: int = 0, v1: int | None = None, i0: int = 0,
             i1: int | None = None, out: np.ndarray | None = None, nthreads: int | None = None) -> np.ndarray:
    """Feature-major codebook block W[v0:v1, i0:i1] as float32 (rows = features)."""
    lib = _load()
    v1 = V if v1 is None else v1
    i1 = M if i1 is None else i1
    shape = (v1 - v0, i1 - i0)
    if out is None:
        out = np.empty(shape, dtype=np.float32)
    if not (out.dtype == np.float32 and out.ndim == 2 and out.shape == shape and out.strides[1] == 4
            and out.strides[0] % 4 == 0 and out.strides[0] >= 4 * shape[1]):
        raise ValueError("out must be a float32 array of the block's shape with unit column stride")
    ld = out.strides[0] // 4
    rc = lib.synth_codebook(seed, kind, V, M, v0, v1, i0, i1, _ptr(out), ld, nthreads or default_threads())
    if rc != 0:
        raise ValueError(f"synth_codebook failed ({rc})")
    return out


VAL_UNIFORM = 0    # (h+1) * 2^-24, in (0, 1]
VAL_QUANTISED = 1  # (k+1) / 256, in [1/256, 1]


def values(seed: int, n: int, kind: int = VAL_UNIFORM, nthreads: int | None = None) -> np.ndarray:
    """Values for the first n CSR positions of a sparse real-valued batch (float32, all positive)."""
    out = np.empty(max(n, 1), dtype=np.float32)[:n]
    rc = _load().synth_values(seed, kind, n, _ptr(out) if n else None, nthreads or default_threads())
    if rc != 0:
        raise ValueError("synth_values failed")
    return out


def tile_distinct(row_ptr: np.ndarray, col_idx: np.ndarray, TA: int = 16, nthreads: int | None = None) -> np.ndarray:
    """Distinct feature ids in each group of TA consecutive rows (the row_ptr must start at 0)."""
    lib = _load()
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int32)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    if row_ptr[0] != 0:
        raise ValueError("row_ptr must start at 0")
    N = row_ptr.shape[0] - 1
    out = np.empty((N + TA - 1) // TA, dtype=np.int32)
    rc = lib.synth_tile_distinct(_ptr(row_ptr), _ptr(col_idx) if col_idx.size else None, N, TA, _ptr(out),
                                 nthreads or default_threads())
    if rc != 0 or (out < 0).any():
        raise ValueError("synth_tile_distinct failed")
    return out


def codebook_to_device(seed: int, kind: int, V: int, M: int, device, chunk_bytes: int = 1 << 28,
                       nthreads: int | None = None, dtype=None):
    """The whole V x M codebook as a device tensor, drawn on the host in row chunks.

    Two pinned staging buffers alternate, so drawing the next chunk overlaps
    the copy of the previous one; host memory stays at two chunks. With
    dtype=torch.float16 each chunk is rounded to binary16 on the device
    (round to nearest even, as numpy's astype(np.float16)).
    """
    import torch

    dtype = dtype or torch.float32
    W = torch.empty((V, M), dtype=dtype, device=device)
    rows = max(1, min(V, chunk_bytes // (4 * M)))
    bufs = [torch.empty((rows, M), dtype=torch.float32, pin_memory=True) for _ in range(2)]
    events = [None, None]
    stream = torch.cuda.current_stream(device)
    for n, v0 in enumerate(range(0, V, rows)):
        v1 = min(V, v0 + rows)
        k = n & 1
        if events[k] is not None:
            events[k].synchronize()
        host = bufs[k][: v1 - v0]
        codebook(seed, kind, V, M, v0, v1, 0, M, out=host.numpy(), nthreads=nthreads)
        if dtype == torch.float32:
            W[v0:v1].copy_(host, non_blocking=True)
        else:
            W[v0:v1].copy_(host.to(device, non_blocking=True))
        ev = torch.cuda.Event()
        ev.record(stream)
        events[k] = ev
    torch.cuda.synchronize(device)
    return W
