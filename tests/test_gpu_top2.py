"""GPU parity of the two-best search (som_bmu2_search) against the two-best oracle.

The pair is what the fused sweep returns per sample (Figure 2 caption); the
second unit defines the topographic error. Quantised (k/256) codebooks are
compared bit for bit, continuous ones by the margin rule of parity.check_top2.
"""
import os

import numpy as np
import pytest
import torch

import paper_2608_24067_amd.som as som
import synth
from parity import compare2, gpu_run, gpu_run2, to_dev

pytestmark = pytest.mark.gpu

HOST_THREADS = max(1, min(16, os.cpu_count() or 1))


def case(seed, N, V, M, kind):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, M)
    return rp, ci, W


def test_tiny_workload_bit_exact(dev):
    cfg = synth.CONFIGS["tiny"]
    rp, ci, W = case(cfg.seed, cfg.N, cfg.V, cfg.M, cfg.kind)
    g = gpu_run2(W, rp, ci, dev)
    compare2(W, rp, ci, g, exact=True, what="tiny top-2")


SHAPES = [
    (41, 1, 50, 1, synth.QUANTISED),
    (42, 19, 300, 2, synth.QUANTISED),
    (43, 700, 2000, 300, synth.QUANTISED),
    (44, 333, 500, 1537, synth.QUANTISED),
    (45, 1025, 1000, 1024, synth.UNIFORM),
    (46, 200, 30000, 4099, synth.UNIFORM),
    (47, 300, 4000, 3, synth.UNIFORM),
    (48, 400, 3000, 729, synth.UNIFORM_BLUR3),
]


@pytest.mark.parametrize("tile,keep", [(8, False), (16, False), (32, False), (8, True)])
@pytest.mark.parametrize("seed,N,V,M,kind", SHAPES)
def test_shapes(dev, seed, N, V, M, kind, tile, keep):
    rp, ci, W = case(seed, N, V, M, kind)
    g = gpu_run2(W, rp, ci, dev, tile_samples=tile, keep_order=keep)
    compare2(W, rp, ci, g, exact=kind == synth.QUANTISED, what=f"seed {seed} tile {tile} keep {keep}")


def test_rank1_equals_single_best_search(dev):
    # the two-best search returns exactly the single-best search's unit and distance
    for seed, N, V, M, kind in SHAPES[2:]:
        rp, ci, W = case(seed, N, V, M, kind)
        b, d, _ = gpu_run(W, rp, ci, dev)
        g = gpu_run2(W, rp, ci, dev)
        assert np.array_equal(g[0], b) and np.array_equal(g[1], d), f"seed {seed}"


def test_tile_and_order_invariance(dev):
    rp, ci, W = case(49, 900, 2500, 1300, synth.UNIFORM)
    runs = [gpu_run2(W, rp, ci, dev, tile_samples=t, keep_order=k) for t in (8, 16, 32) for k in (False, True)]
    for r in runs[1:]:
        for a, b in zip(runs[0], r):
            assert np.array_equal(a, b)


def test_ties_constant_and_planted(dev):
    V, M, N = 400, 600, 64
    rp, ci = synth.make_csr(50, N, V)
    Wc = np.full((V, M), 0.375, dtype=np.float32)
    g = gpu_run2(Wc, rp, ci, dev)
    assert (g[0] == 0).all() and (g[2] == 1).all() and np.array_equal(g[1], g[3])
    # three exact copies of sample 5 at 530, 17, 300 (different strips): ranks 17, 300
    W = synth.codebook(50, synth.UNIFORM, V, M)
    s = 5
    for j in (530, 17, 300):
        W[:, j] = 0.0
        W[ci[rp[s]:rp[s + 1]], j] = 1.0
    g = gpu_run2(W, rp, ci, dev)
    assert (g[0][s], g[1][s], g[2][s], g[3][s]) == (17, 0.0, 300, 0.0)
    compare2(W, rp, ci, g, exact=False, what="planted copies")


def test_empty_rows_and_batch_slice(dev):
    # empty rows rank by the norms alone; a slice with row_ptr[0] != 0 gives the same answers
    rp, ci, W = case(51, 300, 800, 513, synth.QUANTISED)
    lens = np.diff(rp)
    keep = np.arange(300) % 7 != 3
    rp2 = np.zeros(301, dtype=np.int32)
    rp2[1:] = np.cumsum(np.where(keep, lens, 0))
    ci2 = np.concatenate([ci[rp[r]:rp[r + 1]] for r in range(300) if keep[r]])
    g = gpu_run2(W, rp2, ci2, dev)
    compare2(W, rp2, ci2, g, exact=True, what="empty rows")
    Wd = to_dev(W, dev)
    rpd, cid = to_dev(rp2, dev), to_dev(ci2, dev)
    norms = som.codebook_norms(Wd, 800, 513)
    lo, hi = 40, 250
    nnz = int(rp2[hi] - rp2[lo])
    sl = som.bmu2_search(Wd, norms, rpd[lo:hi + 1], cid, 800, 513, nnz=nnz)
    torch.cuda.synchronize()
    for a, b in zip(sl, g):
        assert np.array_equal(a.cpu().numpy(), b[lo:hi])


@pytest.mark.parametrize("name,rows", [("64", 1024), ("256", 256)])
def test_workload_prefix(dev, name, rows):
    # the first rows of a full-size workload over its full map; the oracle runs on several threads
    cfg = synth.CONFIGS[name]
    rp, ci = synth.make_csr(cfg.seed, rows, cfg.V)
    W = synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M)
    g = gpu_run2(W, rp, ci, dev)
    print(compare2(W, rp, ci, g, exact=False, what=f"{name} prefix top-2", nthreads=HOST_THREADS))


def test_phases_equal_search(dev):
    rp, ci, W = case(52, 999, 3000, 1111, synth.UNIFORM)
    V, M, N, nnz = 3000, 1111, 999, int(rp[-1])
    Wd, rpd, cid = to_dev(W, dev), to_dev(rp, dev), to_dev(ci, dev)
    norms = som.codebook_norms(Wd, V, M)
    whole = som.bmu2_search(Wd, norms, rpd, cid, V, M, nnz=nnz)
    ws = som.alloc_workspace2(N, M, V, nnz, dev)
    out = (torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev),
           torch.empty(N, dtype=torch.int32, device=dev), torch.empty(N, dtype=torch.float64, device=dev))
    som.bmu_plan(rpd, cid, V, M, nnz, ws)
    som.bmu2_sweep(Wd, norms, V, M, N, nnz, ws)
    som.bmu2_finalize(norms, rpd, V, M, nnz, out, ws)
    assert som.input_flags(ws, N, M, V, nnz) == 0
    for a, b in zip(whole, out):
        assert torch.equal(a, b)
    # the two-best workspace serves the single-best finalize: rank 1, the same bits
    b1 = torch.full((N,), -7, dtype=torch.int32, device=dev)
    d1 = torch.full((N,), -7.0, dtype=torch.float64, device=dev)
    som.bmu_finalize(norms, rpd, V, M, nnz, b1, d1, ws)
    assert torch.equal(b1, whole[0]) and torch.equal(d1, whole[1])
