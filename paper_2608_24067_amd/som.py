"""ctypes binding of libsom.so (include/som.h). Argument marshalling only.

Every function takes torch tensors, checks dtype, device, size and
contiguity, and passes raw pointers plus the current torch stream's handle
to the C entry point of the same name; all work runs in the library's HIP
kernels on that stream. If libsom.so is missing, loading fails loudly: there
is no fallback of any kind.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsom.so")

SOM_OK, SOM_ERR_INVALID_ARG, SOM_ERR_BAD_CSR, SOM_ERR_WORKSPACE, SOM_ERR_HIP = range(5)
MAX_NEURONS = 1 << 20
DEFAULT_TILE_SAMPLES = 8
FLAG_ID_RANGE, FLAG_UNSORTED, FLAG_ROW_PTR = 0x1, 0x2, 0x4

EXPORTS = (
    "som_bmu_workspace_bytes", "som_codebook_norms", "som_bmu_search", "som_bmu_search_noalloc", "som_bmu_plan",
    "som_bmu_sweep",
    "som_bmu_finalize", "som_bmu2_workspace_bytes", "som_bmu2_search", "som_bmu2_sweep", "som_bmu2_finalize",
    "som_codebook_norms_f16", "som_bmu_search_f16", "som_bmu_sweep_f16", "som_bmu2_search_f16", "som_bmu2_sweep_f16",
    "som_bmu_sf_workspace_bytes", "som_bmu_sf_search", "som_bmu_sf_search_f16", "som_bmu_sf_plan", "som_bmu_sf_sweep",
    "som_bmu_sf_sweep_f16", "som_bmu_sf_finalize", "som_update_workspace_bytes", "som_update", "som_update_f16",
    "som_sigma", "som_radius", "som_bmu_input_flags",
    "som_validate_csr_host", "som_last_error",
)


class SomError(RuntimeError):
    def __init__(self, status: int, where: str, text: str):
        super().__init__(f"{where}: status {status}: {text}")
        self.status = status


class _Config(ctypes.Structure):
    _fields_ = [("tile_samples", ctypes.c_int32), ("keep_order", ctypes.c_int32), ("reserved", ctypes.c_int32 * 6)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load():
    """Load libsom.so (built by __graft_entry__.build()); raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"libsom.so not found at {_LIB_PATH}: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(_LIB_PATH)
    i64, vp, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_size_t
    cfgp = ctypes.POINTER(_Config)
    lib.som_bmu_workspace_bytes.argtypes = [i64, i64, i64, i64, cfgp]
    lib.som_bmu_workspace_bytes.restype = sz
    lib.som_codebook_norms.argtypes = [vp, i64, i64, vp, vp]
    lib.som_bmu_search.argtypes = [vp, vp, i64, i64, vp, vp, i64, i64, vp, vp, vp, sz, cfgp, vp]
    lib.som_bmu_search_noalloc.argtypes = [vp, vp, i64, i64, vp, vp, i64, i64, vp, vp, cfgp, vp]
    lib.som_bmu_plan.argtypes = [vp, vp, i64, i64, i64, i64, vp, sz, cfgp, vp]
    lib.som_bmu_sweep.argtypes = [vp, vp, i64, i64, i64, i64, vp, sz, cfgp, vp]
    lib.som_bmu_finalize.argtypes = [vp, i64, i64, vp, i64, i64, vp, vp, vp, sz, cfgp, vp]
    lib.som_bmu2_workspace_bytes.argtypes = [i64, i64, i64, i64, cfgp]
    lib.som_bmu2_workspace_bytes.restype = sz
    lib.som_bmu2_search.argtypes = [vp, vp, i64, i64, vp, vp, i64, i64, vp, vp, vp, vp, vp, sz, cfgp, vp]
    lib.som_bmu2_sweep.argtypes = [vp, vp, i64, i64, i64, i64, vp, sz, cfgp, vp]
    lib.som_bmu2_finalize.argtypes = [vp, i64, i64, vp, i64, i64, vp, vp, vp, vp, vp, sz, cfgp, vp]
    # fp16 codebooks: the same arguments with W holding binary16 values
    for name in ("som_codebook_norms", "som_bmu_search", "som_bmu_sweep", "som_bmu2_search", "som_bmu2_sweep"):
        getattr(lib, name + "_f16").argtypes = getattr(lib, name).argtypes
        getattr(lib, name + "_f16").restype = ctypes.c_int
    i32 = ctypes.c_int32
    lib.som_bmu_sf_workspace_bytes.argtypes = [i64, i64, i64, i64, cfgp]
    lib.som_bmu_sf_workspace_bytes.restype = sz
    lib.som_bmu_sf_search.argtypes = [vp, vp, i64, i64, vp, vp, vp, i64, i64, vp, vp, vp, vp, vp, sz, cfgp, vp]
    lib.som_bmu_sf_search_f16.argtypes = lib.som_bmu_sf_search.argtypes
    lib.som_bmu_sf_plan.argtypes = [vp, vp, vp, i64, i64, i64, i64, vp, sz, cfgp, vp]
    lib.som_bmu_sf_sweep.argtypes = [vp, vp, i64, i64, i64, i64, i32, vp, sz, cfgp, vp]
    lib.som_bmu_sf_sweep_f16.argtypes = lib.som_bmu_sf_sweep.argtypes
    lib.som_bmu_sf_finalize.argtypes = [vp, i64, i64, vp, i64, i64, vp, vp, vp, vp, vp, sz, cfgp, vp]
    for name in ("som_bmu_sf_search", "som_bmu_sf_search_f16", "som_bmu_sf_plan", "som_bmu_sf_sweep",
                 "som_bmu_sf_sweep_f16", "som_bmu_sf_finalize"):
        getattr(lib, name).restype = ctypes.c_int
    lib.som_update_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.som_update_workspace_bytes.restype = sz
    lib.som_update.argtypes = [vp, i64, i64, vp, vp, i64, i64, vp, i32, i64, vp, sz, vp]
    lib.som_update.restype = ctypes.c_int
    lib.som_update_f16.argtypes = lib.som_update.argtypes
    lib.som_update_f16.restype = ctypes.c_int
    lib.som_sigma.argtypes = [i32, ctypes.c_double, ctypes.c_double, ctypes.c_double]
    lib.som_sigma.restype = ctypes.c_double
    lib.som_radius.argtypes = [ctypes.c_double]
    lib.som_radius.restype = ctypes.c_int32
    lib.som_bmu_input_flags.argtypes = [vp, sz, i64, i64, i64, i64, cfgp, ctypes.POINTER(ctypes.c_uint32), vp]
    lib.som_validate_csr_host.argtypes = [vp, vp, i64, i64]
    for name in ("som_codebook_norms", "som_bmu_search", "som_bmu_search_noalloc", "som_bmu_plan", "som_bmu_sweep",
                 "som_bmu_finalize",
                 "som_bmu2_search", "som_bmu2_sweep", "som_bmu2_finalize", "som_bmu_input_flags",
                 "som_validate_csr_host"):
        getattr(lib, name).restype = ctypes.c_int
    lib.som_last_error.argtypes = []
    lib.som_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return load().som_last_error().decode()


def _check(status: int, where: str):
    if status != SOM_OK:
        raise SomError(status, where, last_error())


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype, min_numel: int = 0) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {min_numel}")
    return t.data_ptr()


def _cfg(tile_samples: int = 0, keep_order: bool = False):
    c = _Config()
    c.tile_samples = int(tile_samples)
    c.keep_order = 1 if keep_order else 0
    return ctypes.byref(c)


def workspace_bytes(N: int, M: int, V: int, nnz: int, tile_samples: int = 0, keep_order: bool = False) -> int:
    n = load().som_bmu_workspace_bytes(N, M, V, nnz, _cfg(tile_samples, keep_order))
    if n == 0:
        raise ValueError("som_bmu_workspace_bytes: invalid sizes or config")
    return n


def alloc_workspace(N: int, M: int, V: int, nnz: int, device, tile_samples: int = 0,
                    keep_order: bool = False) -> torch.Tensor:
    return torch.empty(workspace_bytes(N, M, V, nnz, tile_samples, keep_order), dtype=torch.uint8, device=device)


def workspace2_bytes(N: int, M: int, V: int, nnz: int, tile_samples: int = 0, keep_order: bool = False) -> int:
    n = load().som_bmu2_workspace_bytes(N, M, V, nnz, _cfg(tile_samples, keep_order))
    if n == 0:
        raise ValueError("som_bmu2_workspace_bytes: invalid sizes or config")
    return n


def alloc_workspace2(N: int, M: int, V: int, nnz: int, device, tile_samples: int = 0,
                     keep_order: bool = False) -> torch.Tensor:
    return torch.empty(workspace2_bytes(N, M, V, nnz, tile_samples, keep_order), dtype=torch.uint8, device=device)


def _book(W: torch.Tensor, V: int, M: int, entry: str):
    """The entry point for W's element type (fp32, or fp16 storage: the name + "_f16") and W's pointer."""
    if not isinstance(W, torch.Tensor):
        raise TypeError("W must be a torch.Tensor")
    if W.numel() != V * M:
        raise ValueError("W must hold V*M elements")
    if W.dtype == torch.float16:
        return getattr(load(), entry + "_f16"), _dev(W, "W", torch.float16), entry + "_f16"
    return getattr(load(), entry), _dev(W, "W", torch.float32), entry


def codebook_norms(W: torch.Tensor, V: int, M: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """fp64 per-neuron squared norms of the feature-major V x M codebook W (float32 or float16)."""
    fn, wp, name = _book(W, V, M, "som_codebook_norms")
    if out is None:
        out = torch.empty(M, dtype=torch.float64, device=W.device)
    op = _dev(out, "norms", torch.float64, M)
    _check(fn(wp, V, M, op, _stream(W)), name)
    return out


def _csr(row_ptr, col_idx, N, nnz=None):
    rp = _dev(row_ptr, "row_ptr", torch.int32, N + 1)
    ci = _dev(col_idx, "col_idx", torch.int32) if col_idx.numel() else None
    if nnz is not None and col_idx.numel() < nnz:
        raise ValueError(f"col_idx holds {col_idx.numel()} ids, nnz is {nnz}")
    return rp, ci


def _nnz(row_ptr: torch.Tensor, N: int, nnz: int | None) -> int:
    if nnz is None:  # one device read; pass nnz to avoid it
        nnz = int(row_ptr[N].item()) - int(row_ptr[0].item())
    return int(nnz)


def bmu_search(W, norms, row_ptr, col_idx, V: int, M: int, nnz: int | None = None, bmu=None, dist=None,
               workspace=None, tile_samples: int = 0, keep_order: bool = False):
    """BMU index (int32) and squared distance (fp64) of every CSR row. Returns (bmu, dist)."""
    N = row_ptr.numel() - 1
    nnz = _nnz(row_ptr, N, nnz)
    dev = W.device
    if bmu is None:
        bmu = torch.empty(N, dtype=torch.int32, device=dev)
    if dist is None:
        dist = torch.empty(N, dtype=torch.float64, device=dev)
    if workspace is None:
        workspace = alloc_workspace(N, M, V, nnz, dev, tile_samples, keep_order)
    fn, wp, name = _book(W, V, M, "som_bmu_search")
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, rp, ci, N, nnz,
            _dev(bmu, "bmu", torch.int32, N), _dev(dist, "dist", torch.float64, N),
            _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)
    return bmu, dist


NOALLOC_SCRATCH_BYTES = 64 << 20


def bmu_search_noalloc(W, norms, row_ptr, col_idx, V: int, M: int, nnz: int, bmu, dist, tile_samples: int = 0,
                       keep_order: bool = False):
    """bmu_search through som_bmu_search_noalloc: no workspace, the library's own scratch array (fp32 codebook).

    bmu and dist must be passed (the call itself allocates nothing); returns them.
    """
    N = row_ptr.numel() - 1
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    if W.dtype != torch.float32:
        raise TypeError("som_bmu_search_noalloc takes an fp32 codebook")
    st = load().som_bmu_search_noalloc(_dev(W, "W", torch.float32, V * M), _dev(norms, "norms", torch.float64, M), V,
                                       M, rp, ci, N, int(nnz), _dev(bmu, "bmu", torch.int32, N),
                                       _dev(dist, "dist", torch.float64, N), _cfg(tile_samples, keep_order),
                                       _stream(W))
    _check(st, "som_bmu_search_noalloc")
    return bmu, dist


def bmu2_search(W, norms, row_ptr, col_idx, V: int, M: int, nnz: int | None = None, out=None, workspace=None,
                tile_samples: int = 0, keep_order: bool = False):
    """The two best units of every CSR row, ranked by (distance, index).

    Returns (bmu, dist, bmu2, dist2); bmu2 = -1 and dist2 = +inf when M == 1.
    ``out`` may pass the four output tensors.
    """
    N = row_ptr.numel() - 1
    nnz = _nnz(row_ptr, N, nnz)
    dev = W.device
    if out is None:
        out = (torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev),
               torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev))
    bmu, dist, bmu2, dist2 = out
    if workspace is None:
        workspace = alloc_workspace2(N, M, V, nnz, dev, tile_samples, keep_order)
    fn, wp, name = _book(W, V, M, "som_bmu2_search")
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, rp, ci, N, nnz,
            _dev(bmu, "bmu", torch.int32, N), _dev(dist, "dist", torch.float64, N),
            _dev(bmu2, "bmu2", torch.int32, N), _dev(dist2, "dist2", torch.float64, N),
            _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)
    return bmu, dist, bmu2, dist2


def bmu_plan(row_ptr, col_idx, V: int, M: int, nnz: int, workspace, tile_samples: int = 0, keep_order: bool = False):
    N = row_ptr.numel() - 1
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    st = load().som_bmu_plan(rp, ci, N, nnz, V, M, _dev(workspace, "workspace", torch.uint8), workspace.numel(),
                             _cfg(tile_samples, keep_order), _stream(row_ptr))
    _check(st, "som_bmu_plan")


def bmu_sweep(W, norms, V: int, M: int, N: int, nnz: int, workspace, tile_samples: int = 0, keep_order: bool = False):
    fn, wp, name = _book(W, V, M, "som_bmu_sweep")
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, N, nnz, _dev(workspace, "workspace", torch.uint8),
            workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)


def bmu_finalize(norms, row_ptr, V: int, M: int, nnz: int, bmu, dist, workspace, tile_samples: int = 0,
                 keep_order: bool = False):
    N = row_ptr.numel() - 1
    st = load().som_bmu_finalize(
        _dev(norms, "norms", torch.float64, M), V, M, _dev(row_ptr, "row_ptr", torch.int32, N + 1), N, nnz,
        _dev(bmu, "bmu", torch.int32, N), _dev(dist, "dist", torch.float64, N),
        _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(norms))
    _check(st, "som_bmu_finalize")



def bmu2_sweep(W, norms, V: int, M: int, N: int, nnz: int, workspace, tile_samples: int = 0, keep_order: bool = False):
    fn, wp, name = _book(W, V, M, "som_bmu2_sweep")
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, N, nnz, _dev(workspace, "workspace", torch.uint8),
            workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)


def bmu2_finalize(norms, row_ptr, V: int, M: int, nnz: int, out, workspace, tile_samples: int = 0,
                  keep_order: bool = False):
    """out = (bmu, dist, bmu2, dist2) tensors, written."""
    N = row_ptr.numel() - 1
    bmu, dist, bmu2, dist2 = out
    st = load().som_bmu2_finalize(
        _dev(norms, "norms", torch.float64, M), V, M, _dev(row_ptr, "row_ptr", torch.int32, N + 1), N, nnz,
        _dev(bmu, "bmu", torch.int32, N), _dev(dist, "dist", torch.float64, N),
        _dev(bmu2, "bmu2", torch.int32, N), _dev(dist2, "dist2", torch.float64, N),
        _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(norms))
    _check(st, "som_bmu2_finalize")

def input_flags(workspace, N: int, M: int, V: int, nnz: int, tile_samples: int = 0, keep_order: bool = False) -> int:
    """SOM_FLAG_* bits the last plan recorded (waits for the current stream)."""
    out = ctypes.c_uint32(0)
    st = load().som_bmu_input_flags(_dev(workspace, "workspace", torch.uint8), workspace.numel(), N, M, V, nnz,
                                    _cfg(tile_samples, keep_order), ctypes.byref(out), _stream(workspace))
    _check(st, "som_bmu_input_flags")
    return int(out.value)


def validate_csr_host(row_ptr, col_idx, V: int) -> None:
    """Raises SomError(SOM_ERR_BAD_CSR) if a host CSR breaks the sorted, distinct, in-range rules."""
    rp = np.ascontiguousarray(np.asarray(row_ptr), dtype=np.int32)
    ci = np.ascontiguousarray(np.asarray(col_idx), dtype=np.int32)
    N = rp.shape[0] - 1
    st = load().som_validate_csr_host(rp.ctypes.data, ci.ctypes.data if ci.size else None, N, V)
    _check(st, "som_validate_csr_host")


# ------------------------------------------------------------ sparse real-valued rows

def workspace_sf_bytes(N: int, M: int, V: int, nnz: int, tile_samples: int = 0, keep_order: bool = False) -> int:
    n = load().som_bmu_sf_workspace_bytes(N, M, V, nnz, _cfg(tile_samples, keep_order))
    if n == 0:
        raise ValueError("som_bmu_sf_workspace_bytes: invalid sizes or config")
    return n


def alloc_workspace_sf(N: int, M: int, V: int, nnz: int, device, tile_samples: int = 0,
                       keep_order: bool = False) -> torch.Tensor:
    return torch.empty(workspace_sf_bytes(N, M, V, nnz, tile_samples, keep_order), dtype=torch.uint8, device=device)


def bmu_sf_search(W, norms, row_ptr, col_idx, values, V: int, M: int, nnz: int | None = None, two_best: bool = False,
                  out=None, workspace=None, tile_samples: int = 0, keep_order: bool = False):
    """BMU search over sparse real-valued rows (values[p] belongs to col_idx[p]).

    Returns (bmu, dist), or (bmu, dist, bmu2, dist2) with two_best. W float32 or float16.
    """
    N = row_ptr.numel() - 1
    nnz = _nnz(row_ptr, N, nnz)
    dev = W.device
    if out is None:
        out = (torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev))
        if two_best:
            out = out + (torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev))
    if workspace is None:
        workspace = alloc_workspace_sf(N, M, V, nnz, dev, tile_samples, keep_order)
    if values.numel() < nnz:
        raise ValueError(f"values holds {values.numel()} entries, nnz is {nnz}")
    fn, wp, name = _book(W, V, M, "som_bmu_sf_search")
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    vp = _dev(values, "values", torch.float32) if values.numel() else None
    b2 = _dev(out[2], "bmu2", torch.int32, N) if two_best else None
    d2 = _dev(out[3], "dist2", torch.float64, N) if two_best else None
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, rp, ci, vp, N, nnz,
            _dev(out[0], "bmu", torch.int32, N), _dev(out[1], "dist", torch.float64, N), b2, d2,
            _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)
    return out


def bmu_sf_plan(row_ptr, col_idx, values, V: int, M: int, nnz: int, workspace, tile_samples: int = 0,
                keep_order: bool = False):
    N = row_ptr.numel() - 1
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    vp = _dev(values, "values", torch.float32) if values.numel() else None
    st = load().som_bmu_sf_plan(rp, ci, vp, N, nnz, V, M, _dev(workspace, "workspace", torch.uint8), workspace.numel(),
                                _cfg(tile_samples, keep_order), _stream(row_ptr))
    _check(st, "som_bmu_sf_plan")


def bmu_sf_sweep(W, norms, V: int, M: int, N: int, nnz: int, workspace, two_best: bool = False,
                 tile_samples: int = 0, keep_order: bool = False):
    fn, wp, name = _book(W, V, M, "som_bmu_sf_sweep")
    st = fn(wp, _dev(norms, "norms", torch.float64, M), V, M, N, nnz, 1 if two_best else 0,
            _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(W))
    _check(st, name)


def bmu_sf_finalize(norms, row_ptr, V: int, M: int, nnz: int, out, workspace, tile_samples: int = 0,
                    keep_order: bool = False):
    """out = (bmu, dist) or (bmu, dist, bmu2, dist2) tensors, written."""
    N = row_ptr.numel() - 1
    b2 = _dev(out[2], "bmu2", torch.int32, N) if len(out) == 4 else None
    d2 = _dev(out[3], "dist2", torch.float64, N) if len(out) == 4 else None
    st = load().som_bmu_sf_finalize(
        _dev(norms, "norms", torch.float64, M), V, M, _dev(row_ptr, "row_ptr", torch.int32, N + 1), N, nnz,
        _dev(out[0], "bmu", torch.int32, N), _dev(out[1], "dist", torch.float64, N), b2, d2,
        _dev(workspace, "workspace", torch.uint8), workspace.numel(), _cfg(tile_samples, keep_order), _stream(norms))
    _check(st, "som_bmu_sf_finalize")


# ------------------------------------------------------------------- batch update

def update_workspace_bytes(V: int, E: int, N: int, chunk_features: int = 0) -> int:
    n = load().som_update_workspace_bytes(V, E, N, chunk_features)
    if n == 0:
        raise ValueError("som_update_workspace_bytes: invalid sizes")
    return n


def update(W, row_ptr, col_idx, bmu, V: int, E: int, radius: int, nnz: int | None = None, chunk_features: int = 0,
           workspace=None):
    """One batch update of the feature-major V x E*E codebook W in place (float32 or float16); returns W."""
    N = row_ptr.numel() - 1
    nnz = _nnz(row_ptr, N, nnz)
    if not isinstance(W, torch.Tensor) or W.numel() != V * E * E:
        raise ValueError("W must be a tensor of V*E*E elements")
    if workspace is None:
        workspace = torch.empty(update_workspace_bytes(V, E, N, chunk_features), dtype=torch.uint8, device=W.device)
    f16 = W.dtype == torch.float16
    wp = _dev(W, "W", torch.float16 if f16 else torch.float32)
    rp, ci = _csr(row_ptr, col_idx, N, nnz)
    fn = load().som_update_f16 if f16 else load().som_update
    st = fn(wp, V, E, rp, ci, N, nnz, _dev(bmu, "bmu", torch.int32, N), int(radius), chunk_features,
            _dev(workspace, "workspace", torch.uint8), workspace.numel(), _stream(W))
    _check(st, "som_update_f16" if f16 else "som_update")
    return W


def sigma(epoch: int, sigma0: float, sigma_min: float, rate: float = 0.3) -> float:
    return float(load().som_sigma(epoch, sigma0, sigma_min, rate))


def radius(sigma_value: float) -> int:
    return int(load().som_radius(sigma_value))
