"""CPU tests of the C ABI: the library loads and exports every declared entry
point, the workspace query, the host CSR validator, and every argument check
that returns before anything reaches the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2608_24067_amd.som as som

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_entry_points():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            names += re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(som_[a-z_0-9]+)\s*\(", text, re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    lib = som.load()
    names = declared_entry_points()
    assert set(names) == set(som.EXPORTS), names
    for n in names:
        assert hasattr(lib, n), n


def test_read_probe_library_loads():
    # the benchmark's read-stream probe: its own library, one entry point, argument checks on the host
    from paper_2608_24067_amd import build as pkg_build

    lib = ctypes.CDLL(pkg_build.PROBE_LIB)
    lib.somprobe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    assert lib.somprobe_read(None, 1024, None, 8, None) != 0
    assert lib.somprobe_read(ctypes.c_void_p(4096 + 8), 1024, ctypes.c_void_p(4096), 8, None) != 0  # misaligned
    assert lib.somprobe_read(ctypes.c_void_p(4096), 1024, ctypes.c_void_p(4096), 0, None) != 0  # no workgroups


def test_header_constants_match_binding():
    text = open(os.path.join(ROOT, "include", "som.h")).read()
    assert re.search(r"^#define SOM_DEFAULT_TILE_SAMPLES (\d+)$", text, re.M).group(1) == str(som.DEFAULT_TILE_SAMPLES)
    assert re.search(r"^#define SOM_MAX_NEURONS \(1 << (\d+)\)$", text, re.M).group(1) == "20"
    assert som.MAX_NEURONS == 1 << 20


def test_workspace_bytes():
    n = som.workspace_bytes(10_000, 256, 2000, 120_000)
    assert n > 0 and n % 256 == 0
    # grows with every size it depends on
    assert som.workspace_bytes(20_000, 256, 2000, 120_000) > n
    assert som.workspace_bytes(10_000, 4096, 2000, 120_000) > n
    assert som.workspace_bytes(10_000, 256, 2000, 240_000) > n
    lib = som.load()
    assert lib.som_bmu_workspace_bytes(-1, 256, 2000, 0, None) == 0
    assert lib.som_bmu_workspace_bytes(10, 0, 2000, 0, None) == 0
    assert lib.som_bmu_workspace_bytes(10, (1 << 20) + 1, 2000, 0, None) == 0
    assert lib.som_bmu_workspace_bytes(10, 1 << 20, 2000, 0, None) > 0
    assert lib.som_bmu_workspace_bytes(10, 256, 2000, 0, _cfg(7)) == 0
    # larger tiles use narrower strips, hence more partial keys
    assert som.workspace_bytes(10_000, 4096, 2000, 0, 16) > som.workspace_bytes(10_000, 4096, 2000, 0, 8)
    # the regrouped copy of the batch is only held when the order is not kept
    assert som.workspace_bytes(10_000, 4096, 2000, 120_000, keep_order=True) < som.workspace_bytes(10_000, 4096, 2000,
                                                                                                    120_000)



def test_f16_entry_points_check_alignment():
    lib = som.load()
    odd = ctypes.c_void_p((1 << 20) + 1)
    assert lib.som_codebook_norms_f16(None, 10, 10, FAKE, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_codebook_norms_f16(odd, 10, 10, FAKE, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu_search_f16(odd, FAKE, 100, 64, FAKE, FAKE, 10, 50, FAKE, FAKE, FAKE, 1 << 30, None,
                                  None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu_sweep_f16(odd, FAKE, 100, 64, 10, 50, FAKE, 1 << 30, None, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu2_sweep_f16(FAKE, FAKE, 100, 64, 10, 50, FAKE, 100, None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu2_search_f16(FAKE, FAKE, 100, 64, FAKE, FAKE, 10, 50, FAKE, FAKE, None, FAKE, FAKE, 1 << 30,
                                   None, None) == som.SOM_ERR_INVALID_ARG
    # a 2-byte aligned fp16 codebook is fine where fp32 needs 4 bytes
    two = ctypes.c_void_p((1 << 20) + 2)
    assert lib.som_bmu_sweep_f16(two, FAKE, 100, 64, 10, 50, FAKE, 100, None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_sweep(two, FAKE, 100, 64, 10, 50, FAKE, 100, None, None) == som.SOM_ERR_INVALID_ARG


def test_real_valued_workspace_and_checks():
    lib = som.load()
    n2 = som.workspace2_bytes(10_000, 4096, 2000, 120_000)
    nsf = som.workspace_sf_bytes(10_000, 4096, 2000, 120_000)
    # per-entry values (8 per id) and ||x||^2 per sample on top of the two-best layout
    assert nsf >= n2 + 32 * 120_000 + 8 * 10_000
    assert lib.som_bmu_sf_workspace_bytes(10, 64, 100, 50, _cfg(16)) == 0  # tiles of 8 only
    assert lib.som_bmu_sf_search(FAKE, FAKE, 100, 64, FAKE, FAKE, None, 10, 50, FAKE, FAKE, None, None, FAKE,
                                 1 << 30, None, None) == som.SOM_ERR_INVALID_ARG  # no values
    small2 = som.workspace2_bytes(10, 64, 100, 50)  # two-best room, but not the values
    assert lib.som_bmu_sf_search(FAKE, FAKE, 100, 64, FAKE, FAKE, FAKE, 10, 50, FAKE, FAKE, None, None, FAKE, small2,
                                 None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_sf_plan(FAKE, FAKE, FAKE, 10, 50, 100, 64, FAKE, 1 << 30, _cfg(32),
                               None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu_sf_sweep(FAKE, FAKE, 100, 64, 10, 50, 1, FAKE, 100, None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_sf_search(None, None, 100, 64, None, None, None, 0, 0, None, None, None, None, None, 0, None,
                                 None) == som.SOM_OK


def test_schedule_and_radius():
    assert som.sigma(1, 512.0, 0.5) == 512.0
    vals = [som.sigma(e, 512.0, 0.5) for e in range(1, 60)]
    assert all(a > b for a, b in zip(vals, vals[1:])) and abs(vals[-1] - 0.5) < 1e-3
    assert abs(som.sigma(3, 32.0, 0.5, 0.3) - (0.5 + 31.5 * np.exp(-0.6))) < 1e-12
    assert som.sigma(0, 10.0, 1.0) == 10.0  # epochs below 1 count as the first
    assert [som.radius(x) for x in (0.0, 0.4, 1.0, 1.49, 1.5, 2.5, 512.3, float("nan"))] == [1, 1, 1, 1, 2, 3, 512, 1]


def test_update_workspace_and_checks():
    lib = som.load()
    full = som.update_workspace_bytes(300, 16, 10)
    part = som.update_workspace_bytes(300, 16, 10, 10)
    assert full > part > 0 and full >= 3 * 300 * 256 * 4
    # the sort of crowded units' samples holds one int32 per sample
    assert som.update_workspace_bytes(300, 16, 10 + 10**6) >= full + 4 * 10**6
    assert lib.som_update_workspace_bytes(0, 16, 10, 0) == 0
    assert lib.som_update_workspace_bytes(10, 1025, 10, 0) == 0  # E*E beyond 2^20
    assert lib.som_update_workspace_bytes(10, 16, -1, 0) == 0
    assert lib.som_update(FAKE, 300, 16, FAKE, FAKE, 10, 50, FAKE, 0, 0, FAKE, 1 << 30, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_update(FAKE, 300, 16, FAKE, FAKE, 10, 50, None, 1, 0, FAKE, 1 << 30, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_update(FAKE, 300, 16, FAKE, FAKE, 10, 50, FAKE, 1, 0, FAKE, part, None) == som.SOM_ERR_WORKSPACE
    odd = ctypes.c_void_p((1 << 20) + 1)
    assert lib.som_update_f16(odd, 300, 16, FAKE, FAKE, 10, 50, FAKE, 1, 0, FAKE, 1 << 30, None) == som.SOM_ERR_INVALID_ARG


def test_two_best_workspace_and_checks():
    lib = som.load()
    for tile, keep in ((0, False), (16, False), (32, True)):
        n1 = som.workspace_bytes(10_000, 4096, 2000, 120_000, tile, keep)
        n2 = som.workspace2_bytes(10_000, 4096, 2000, 120_000, tile, keep)
        # a second 8-byte key and 4-byte dot product per sample and strip, appended
        strips = -(-4096 // (512 if tile in (0, 8) else 256))
        assert n2 >= n1 + 12 * 10_000 * strips and n2 % 256 == 0
    assert lib.som_bmu2_workspace_bytes(-1, 256, 2000, 0, None) == 0
    assert lib.som_bmu2_workspace_bytes(10, 256, 2000, 0, _cfg(12)) == 0
    n1 = som.workspace_bytes(10, 64, 100, 50)
    # null outputs, then a workspace that only fits the single-best search
    assert lib.som_bmu2_search(FAKE, FAKE, 100, 64, FAKE, FAKE, 10, 50, FAKE, FAKE, None, FAKE, FAKE, 1 << 30, None,
                               None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu2_search(FAKE, FAKE, 100, 64, FAKE, FAKE, 10, 50, FAKE, FAKE, FAKE, FAKE, FAKE, n1, None,
                               None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu2_search(FAKE, FAKE, 100, 0, FAKE, FAKE, 10, 50, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None,
                               None) == som.SOM_ERR_INVALID_ARG
    # N == 0 is a no-op that touches nothing
    assert lib.som_bmu2_search(None, None, 100, 64, None, None, 0, 0, None, None, None, None, None, 0, None,
                               None) == som.SOM_OK

def _status(rp, ci, V):
    lib = som.load()
    rp = np.ascontiguousarray(rp, dtype=np.int32)
    ci = np.ascontiguousarray(ci, dtype=np.int32)
    return lib.som_validate_csr_host(rp.ctypes.data, ci.ctypes.data if ci.size else None, rp.size - 1, V)


def test_validate_csr_host():
    assert _status([0, 2, 3], [1, 4, 0], 5) == som.SOM_OK
    assert _status([0, 0, 0], [], 5) == som.SOM_OK           # empty rows are allowed
    assert _status([0], [], 5) == som.SOM_OK                 # N = 0
    assert _status([3, 5], [9, 9, 9, 1, 2], 5) == som.SOM_OK  # a slice: row_ptr need not start at 0
    assert _status([0, 2, 1], [1, 2], 5) == som.SOM_ERR_BAD_CSR      # row_ptr decreases
    assert _status([0, 2], [1, 5], 5) == som.SOM_ERR_BAD_CSR         # id == V
    assert _status([0, 2], [-1, 2], 5) == som.SOM_ERR_BAD_CSR        # negative id
    assert _status([0, 2], [3, 1], 5) == som.SOM_ERR_BAD_CSR         # unsorted
    assert _status([0, 2], [3, 3], 5) == som.SOM_ERR_BAD_CSR         # repeated id
    assert "ascending" in som.last_error()
    assert _status([0, 1], [0], 0) == som.SOM_ERR_INVALID_ARG         # V < 1
    with pytest.raises(som.SomError):
        som.validate_csr_host([0, 2], [3, 3], 5)
    som.validate_csr_host([0, 2], [1, 3], 5)


def test_generated_workloads_are_valid_csr():
    import synth
    for seed, N, V in [(0, 5000, 2000), (1, 5000, 30000)]:
        rp, ci = synth.make_csr(seed, N, V)
        som.validate_csr_host(rp, ci, V)


# Argument checks that fail before any HIP call (no GPU here). Pointers are fake
# but never dereferenced: every call below must return an error status first.
FAKE = ctypes.c_void_p(1 << 20)


def _search(W=FAKE, norms=FAKE, V=100, M=64, rp=FAKE, ci=FAKE, N=10, nnz=50, bmu=FAKE, dist=FAKE, ws=FAKE,
            ws_bytes=1 << 30, cfg=None):
    lib = som.load()
    return lib.som_bmu_search(W, norms, V, M, rp, ci, N, nnz, bmu, dist, ws, ws_bytes, cfg, None)


def _cfg(ta, reserved0=0, keep_order=0):
    c = som._Config()
    c.tile_samples = ta
    c.keep_order = keep_order
    c.reserved[0] = reserved0
    return ctypes.pointer(c)


@pytest.mark.parametrize("kwargs,status", [
    (dict(M=0), som.SOM_ERR_INVALID_ARG),
    (dict(M=(1 << 20) + 1), som.SOM_ERR_INVALID_ARG),
    (dict(V=0), som.SOM_ERR_INVALID_ARG),
    (dict(N=-1), som.SOM_ERR_INVALID_ARG),
    (dict(nnz=-1), som.SOM_ERR_INVALID_ARG),
    (dict(W=None), som.SOM_ERR_INVALID_ARG),
    (dict(norms=None), som.SOM_ERR_INVALID_ARG),
    (dict(rp=None), som.SOM_ERR_INVALID_ARG),
    (dict(ci=None), som.SOM_ERR_INVALID_ARG),
    (dict(bmu=None), som.SOM_ERR_INVALID_ARG),
    (dict(dist=None), som.SOM_ERR_INVALID_ARG),
    (dict(W=ctypes.c_void_p((1 << 20) + 2)), som.SOM_ERR_INVALID_ARG),  # W not 4-byte aligned
    (dict(cfg=_cfg(7)), som.SOM_ERR_INVALID_ARG),
    (dict(cfg=_cfg(16, reserved0=1)), som.SOM_ERR_INVALID_ARG),
    (dict(cfg=_cfg(8, keep_order=2)), som.SOM_ERR_INVALID_ARG),
    (dict(ws=None), som.SOM_ERR_WORKSPACE),
    (dict(ws=ctypes.c_void_p((1 << 20) + 64)), som.SOM_ERR_WORKSPACE),  # not 256-byte aligned
    (dict(ws_bytes=1024), som.SOM_ERR_WORKSPACE),
])
def test_search_argument_checks(kwargs, status):
    assert _search(**kwargs) == status
    assert som.last_error() != ""


def test_zero_samples_is_a_no_op():
    # N == 0 succeeds without touching any pointer
    assert _search(N=0, nnz=0, W=None, norms=None, rp=None, ci=None, bmu=None, dist=None, ws=None) == som.SOM_OK


def test_phase_and_norms_argument_checks():
    lib = som.load()
    assert lib.som_codebook_norms(None, 10, 10, FAKE, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_codebook_norms(FAKE, 10, 0, FAKE, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_codebook_norms(FAKE, 0, 10, FAKE, None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu_plan(FAKE, FAKE, 10, 50, 100, 64, FAKE, 100, None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_sweep(FAKE, FAKE, 100, 64, 10, 50, FAKE, 100, None, None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_finalize(FAKE, 100, 64, FAKE, 10, 50, FAKE, FAKE, FAKE, 100, None,
                                None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_finalize(None, 100, 64, FAKE, 10, 50, FAKE, FAKE, FAKE, 100, None,
                                None) == som.SOM_ERR_INVALID_ARG
    out = ctypes.c_uint32(7)
    assert lib.som_bmu_input_flags(FAKE, 100, 10, 64, 100, 50, None, ctypes.byref(out), None) == som.SOM_ERR_WORKSPACE
    assert lib.som_bmu_input_flags(FAKE, 100, 10, 64, 100, 50, None, None, None) == som.SOM_ERR_INVALID_ARG


def test_noalloc_rejects_searches_beyond_its_array():
    # checked on the host before anything touches a device: fake pointers are never dereferenced
    lib = som.load()
    V, M = 30_000, 1 << 20
    N, nnz = 4_000, 48_000
    assert som.workspace_bytes(N, M, V, nnz) > som.NOALLOC_SCRATCH_BYTES
    assert lib.som_bmu_search_noalloc(FAKE, FAKE, V, M, FAKE, FAKE, N, nnz, FAKE, FAKE, None,
                                      None) == som.SOM_ERR_WORKSPACE
    assert b"scratch" in lib.som_last_error()
    assert lib.som_bmu_search_noalloc(FAKE, FAKE, V, M + 1, FAKE, FAKE, N, nnz, FAKE, FAKE, None,
                                      None) == som.SOM_ERR_INVALID_ARG
    assert lib.som_bmu_search_noalloc(FAKE, FAKE, V, M, FAKE, FAKE, N, nnz, FAKE, FAKE, _cfg(7),
                                      None) == som.SOM_ERR_INVALID_ARG
    text = open(os.path.join(ROOT, "include", "som.h")).read()
    assert re.search(r"^#define SOM_NOALLOC_SCRATCH_BYTES \(64u << 20\)$", text, re.M)
    assert som.NOALLOC_SCRATCH_BYTES == 64 << 20
