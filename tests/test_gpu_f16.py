"""GPU parity of the fp16-storage search (som_*_f16) against the oracle.

An fp16 codebook holds values that are exact in fp32, so the oracle runs on
the same values widened to fp32 and every bar is the fp32 one. Stronger
still: the fp16 path must return exactly what the fp32 path returns on the
widened codebook (same fp32 sums in the same order, same fp64 norms), which
is checked bit for bit.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24067_amd.som as som
import synth
from parity import compare, compare2, gpu_run, gpu_run2, to_dev

pytestmark = pytest.mark.gpu

HOST_THREADS = max(1, min(16, os.cpu_count() or 1))


def half_case(seed, N, V, M, kind):
    rp, ci = synth.make_csr(seed, N, V)
    W16 = synth.codebook(seed, kind, V, M).astype(np.float16)  # round to nearest even
    return rp, ci, W16, W16.astype(np.float32)                 # exact widening


@pytest.mark.parametrize("V,M", [(2000, 256), (300, 1), (37, 5), (1000, 1029), (30000, 300)])
def test_norms_f16_bitwise(dev, V, M):
    W16 = synth.codebook(8, synth.UNIFORM, V, M).astype(np.float16)
    n = som.codebook_norms(to_dev(W16, dev), V, M).cpu().numpy()
    assert np.array_equal(n, oracle.norms(W16.astype(np.float32)))


def test_tiny_workload_bit_exact(dev):
    # k/256 values are exact in fp16: the whole 16x16 workload, every index and distance exact
    cfg = synth.CONFIGS["tiny"]
    rp, ci, W16, W32 = half_case(cfg.seed, cfg.N, cfg.V, cfg.M, cfg.kind)
    assert np.array_equal(W32, synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M))
    b, d, _ = gpu_run(W16, rp, ci, dev)
    compare(W32, rp, ci, b, d, exact=True, what="tiny f16")


SHAPES = [
    # M off multiples of 8 takes the scalar load path
    (61, 1, 50, 1, synth.QUANTISED),
    (62, 17, 300, 5, synth.QUANTISED),
    (63, 1000, 2000, 300, synth.QUANTISED),
    (64, 333, 500, 1544, synth.QUANTISED),
    (65, 2049, 1000, 1024, synth.UNIFORM),
    (66, 300, 30000, 4099, synth.UNIFORM),
    (67, 520, 4000, 3, synth.UNIFORM),
    (68, 400, 3000, 729, synth.UNIFORM_BLUR3),
]


@pytest.mark.parametrize("tile,keep", [(8, False), (16, False), (32, False), (8, True)])
@pytest.mark.parametrize("seed,N,V,M,kind", SHAPES)
def test_shapes_equal_fp32_and_oracle(dev, seed, N, V, M, kind, tile, keep):
    rp, ci, W16, W32 = half_case(seed, N, V, M, kind)
    b16, d16, _ = gpu_run(W16, rp, ci, dev, tile_samples=tile, keep_order=keep)
    b32, d32, _ = gpu_run(W32, rp, ci, dev, tile_samples=tile, keep_order=keep)
    assert np.array_equal(b16, b32) and np.array_equal(d16, d32), "fp16 storage differs from fp32 on the same values"
    compare(W32, rp, ci, b16, d16, exact=kind == synth.QUANTISED, what=f"f16 seed {seed} tile {tile}")


@pytest.mark.parametrize("seed,N,V,M,kind", SHAPES[2:])
def test_two_best_equal_fp32(dev, seed, N, V, M, kind):
    rp, ci, W16, W32 = half_case(seed, N, V, M, kind)
    g16 = gpu_run2(W16, rp, ci, dev)
    g32 = gpu_run2(W32, rp, ci, dev)
    for a, b in zip(g16, g32):
        assert np.array_equal(a, b)
    compare2(W32, rp, ci, g16, exact=kind == synth.QUANTISED, what=f"f16 top-2 seed {seed}")


def test_unaligned_codebook_takes_scalar_loads(dev):
    # a view starting one element in: 2-byte aligned only, so the vector loads are off
    rp, ci, W16, W32 = half_case(69, 700, 900, 1032, synth.UNIFORM)
    V, M = W16.shape
    flat = torch.empty(V * M + 8, dtype=torch.float16, device=dev)
    flat[1:1 + V * M].copy_(torch.from_numpy(W16.reshape(-1)).to(dev))
    view = flat[1:1 + V * M].view(V, M)
    assert view.data_ptr() % 16 != 0
    b_view, d_view, _ = gpu_run(view, rp, ci, dev)
    b, d, _ = gpu_run(W16, rp, ci, dev)
    assert np.array_equal(b_view, b) and np.array_equal(d_view, d)


def test_phases_equal_search(dev):
    rp, ci, W16, _ = half_case(70, 999, 3000, 1111, synth.UNIFORM)
    V, M, N, nnz = 3000, 1111, 999, int(rp[-1])
    Wd, rpd, cid = to_dev(W16, dev), to_dev(rp, dev), to_dev(ci, dev)
    norms = som.codebook_norms(Wd, V, M)
    b1, d1 = som.bmu_search(Wd, norms, rpd, cid, V, M, nnz=nnz)
    ws = som.alloc_workspace2(N, M, V, nnz, dev)
    b2 = torch.empty(N, dtype=torch.int32, device=dev)
    d2 = torch.empty(N, dtype=torch.float64, device=dev)
    som.bmu_plan(rpd, cid, V, M, nnz, ws)
    som.bmu_sweep(Wd, norms, V, M, N, nnz, ws)
    som.bmu_finalize(norms, rpd, V, M, nnz, b2, d2, ws)
    assert torch.equal(b1, b2) and torch.equal(d1, d2)
    whole = som.bmu2_search(Wd, norms, rpd, cid, V, M, nnz=nnz)
    out = tuple(torch.empty_like(t) for t in whole)
    som.bmu_plan(rpd, cid, V, M, nnz, ws)
    som.bmu2_sweep(Wd, norms, V, M, N, nnz, ws)
    som.bmu2_finalize(norms, rpd, V, M, nnz, out, ws)
    for a, b in zip(whole, out):
        assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["256", "1024"])
def test_full_workload_f16(name):
    # the full batch on the full map with an fp16 codebook; sampled rows against the streamed oracle
    cfg = synth.CONFIGS[name]
    dev = torch.device("cuda:0")
    row_ptr, col_idx = synth.make_csr(cfg.seed, cfg.N, cfg.V, cfg.lam, cfg.zipf_s)
    nnz = int(row_ptr[-1])
    W = synth.codebook_to_device(cfg.seed, cfg.kind, cfg.V, cfg.M, dev, dtype=torch.float16)
    # the device rounding equals numpy's on a few rows
    for v in (0, cfg.V // 2, cfg.V - 1):
        host = synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M, v, v + 1).astype(np.float16)
        assert np.array_equal(W[v].cpu().numpy(), host[0])
    rp = torch.from_numpy(row_ptr).to(dev)
    ci = torch.from_numpy(col_idx).to(dev)
    norms = som.codebook_norms(W, cfg.V, cfg.M)
    ws = som.alloc_workspace2(cfg.N, cfg.M, cfg.V, nnz, dev)
    g = tuple(t.cpu().numpy() for t in som.bmu2_search(W, norms, rp, ci, cfg.V, cfg.M, nnz=nnz, workspace=ws))
    assert som.input_flags(ws, cfg.N, cfg.M, cfg.V, nnz) == 0
    del W, ws, rp, ci, norms
    torch.cuda.empty_cache()
    assert g[0].min() >= 0 and g[0].max() < cfg.M and np.isfinite(g[1]).all() and (g[2] != g[0]).all()

    rows = np.array(sorted(set(np.linspace(0, cfg.N - 1, 24).astype(int).tolist()) | {0, 1, cfg.N - 2, cfg.N - 1}))
    sub_rp = np.zeros(len(rows) + 1, dtype=np.int32)
    sub_rp[1:] = np.cumsum(row_ptr[rows + 1] - row_ptr[rows])
    sub_ci = np.concatenate([col_idx[row_ptr[r]:row_ptr[r + 1]] for r in rows])

    def block(i0, i1):
        return synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M, i0=i0, i1=i1, nthreads=1).astype(
            np.float16).astype(np.float32)

    ref = oracle.bmu2_streamed(block, cfg.M, sub_rp, sub_ci, block=4096, nthreads=HOST_THREADS)

    def dist_at(k, i):
        return oracle.distance_at(block(i, i + 1)[:, 0], sub_ci[sub_rp[k]:sub_rp[k + 1]])

    from parity import check_top2
    print(check_top2(tuple(x[rows] for x in g), ref, dist_at, exact=False, what=f"{name} full f16"))
