"""GPU parity of the search over sparse real-valued rows (som_bmu_sf_*) against the real-valued oracle.

Quantised codebooks with quantised values ((k+1)/256) make every product,
sum and distance exact, so both ranks are compared bit for bit; continuous
ones use the margin rule of parity.check_top2. With every value 1 the
real-valued search must reproduce the binary search exactly.
"""
import os

import numpy as np
import pytest
import torch

import paper_2608_24067_amd.som as som
import synth
from parity import compare_sf, gpu_run, gpu_run2, gpu_run_sf, to_dev

pytestmark = pytest.mark.gpu

HOST_THREADS = max(1, min(16, os.cpu_count() or 1))


def case(seed, N, V, M, kind, vkind):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, M)
    vals = synth.values(seed, len(ci), vkind)
    return rp, ci, vals, W


def test_tiny_workload_bit_exact(dev):
    cfg = synth.CONFIGS["tiny"]
    rp, ci, vals, W = case(cfg.seed, cfg.N, cfg.V, cfg.M, cfg.kind, synth.VAL_QUANTISED)
    g = gpu_run_sf(W, rp, ci, vals, dev)
    compare_sf(W, rp, ci, vals, g, exact=True, what="tiny sf")
    # the single-best form returns the same rank 1
    g1 = gpu_run_sf(W, rp, ci, vals, dev, two_best=False)
    assert np.array_equal(g1[0], g[0]) and np.array_equal(g1[1], g[1])


SHAPES = [
    (81, 1, 50, 1, synth.QUANTISED, synth.VAL_QUANTISED),
    (82, 19, 300, 5, synth.QUANTISED, synth.VAL_QUANTISED),
    (83, 700, 2000, 300, synth.QUANTISED, synth.VAL_QUANTISED),
    (84, 333, 500, 1544, synth.QUANTISED, synth.VAL_QUANTISED),
    (85, 1025, 1000, 1024, synth.UNIFORM, synth.VAL_UNIFORM),
    (86, 200, 30000, 4099, synth.UNIFORM, synth.VAL_UNIFORM),
    (87, 300, 4000, 3, synth.UNIFORM, synth.VAL_UNIFORM),
    (88, 400, 3000, 729, synth.UNIFORM_BLUR3, synth.VAL_UNIFORM),
]


@pytest.mark.parametrize("keep", [False, True])
@pytest.mark.parametrize("seed,N,V,M,kind,vkind", SHAPES)
def test_shapes(dev, seed, N, V, M, kind, vkind, keep):
    rp, ci, vals, W = case(seed, N, V, M, kind, vkind)
    g = gpu_run_sf(W, rp, ci, vals, dev, keep_order=keep)
    compare_sf(W, rp, ci, vals, g, exact=kind == synth.QUANTISED, what=f"sf seed {seed} keep {keep}")


@pytest.mark.parametrize("seed,N,V,M,kind,vkind", SHAPES[2:])
def test_unit_values_equal_binary_search(dev, seed, N, V, M, kind, vkind):
    rp, ci, _, W = case(seed, N, V, M, kind, vkind)
    ones = np.ones(len(ci), dtype=np.float32)
    g = gpu_run_sf(W, rp, ci, ones, dev)
    b2 = gpu_run2(W, rp, ci, dev)
    for a, b in zip(g, b2):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("seed,N,V,M,kind,vkind", SHAPES[2:])
def test_f16_codebook_equals_fp32(dev, seed, N, V, M, kind, vkind):
    rp, ci, vals, W = case(seed, N, V, M, kind, vkind)
    W16 = W.astype(np.float16)
    g16 = gpu_run_sf(W16, rp, ci, vals, dev)
    g32 = gpu_run_sf(W16.astype(np.float32), rp, ci, vals, dev)
    for a, b in zip(g16, g32):
        assert np.array_equal(a, b)


def test_planted_and_empty_rows(dev):
    rp, ci, vals, W = case(89, 200, 900, 700, synth.UNIFORM, synth.VAL_UNIFORM)
    s = 11
    ids, xv = ci[rp[s]:rp[s + 1]], vals[rp[s]:rp[s + 1]]
    for j in (650, 40):  # two exact copies of sample 11 in different strips
        W[:, j] = 0.0
        W[ids, j] = xv
    lens = np.diff(rp)
    keep = np.arange(200) % 9 != 4  # every ninth row emptied
    keep[s] = True
    rp2 = np.zeros(201, dtype=np.int32)
    rp2[1:] = np.cumsum(np.where(keep, lens, 0))
    sel = np.concatenate([np.arange(rp[r], rp[r + 1]) for r in range(200) if keep[r]])
    g = gpu_run_sf(W, rp2, ci[sel], vals[sel], dev)
    # distance 0 up to the fp32 rounding of the dot product (the squares of 24-bit values do not fit fp32)
    assert (g[0][s], g[2][s]) == (40, 650) and abs(g[1][s]) < 1e-5 and abs(g[3][s]) < 1e-5
    compare_sf(W, rp2, ci[sel], vals[sel], g, exact=False, what="planted/empty sf")


def test_phases_equal_search_and_tile_rule(dev):
    rp, ci, vals, W = case(90, 999, 3000, 1111, synth.UNIFORM, synth.VAL_UNIFORM)
    V, M, N, nnz = 3000, 1111, 999, int(rp[-1])
    Wd, rpd, cid, vd = to_dev(W, dev), to_dev(rp, dev), to_dev(ci, dev), to_dev(vals, dev)
    norms = som.codebook_norms(Wd, V, M)
    whole = som.bmu_sf_search(Wd, norms, rpd, cid, vd, V, M, nnz=nnz, two_best=True)
    ws = som.alloc_workspace_sf(N, M, V, nnz, dev)
    out = tuple(torch.empty_like(t) for t in whole)
    som.bmu_sf_plan(rpd, cid, vd, V, M, nnz, ws)
    som.bmu_sf_sweep(Wd, norms, V, M, N, nnz, ws, two_best=True)
    som.bmu_sf_finalize(norms, rpd, V, M, nnz, out, ws)
    assert som.input_flags(ws, N, M, V, nnz) == 0
    for a, b in zip(whole, out):
        assert torch.equal(a, b)
    # tiles of 8 only: the library rejects 16 before launching anything
    with pytest.raises(som.SomError):
        som.bmu_sf_search(Wd, norms, rpd, cid, vd, V, M, nnz=nnz, workspace=ws, tile_samples=16)
    with pytest.raises(ValueError):
        som.workspace_sf_bytes(N, M, V, nnz, tile_samples=16)


@pytest.mark.parametrize("name,rows", [("64", 1024), ("256", 256)])
def test_workload_prefix(dev, name, rows):
    cfg = synth.CONFIGS[name]
    rp, ci = synth.make_csr(cfg.seed, rows, cfg.V)
    vals = synth.values(cfg.seed, len(ci))
    W = synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M)
    g = gpu_run_sf(W, rp, ci, vals, dev)
    print(compare_sf(W, rp, ci, vals, g, exact=False, what=f"{name} prefix sf", nthreads=HOST_THREADS))
