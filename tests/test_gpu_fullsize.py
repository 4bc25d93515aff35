"""GPU parity at the full workload sizes, in the launch configuration bench.py times.

The whole batch runs on the GPU (default tile size, the full map), through the
single-best and the two-best searches; the two-best oracle then evaluates a
sample of rows -- the first and last rows (the last tile is ragged) and rows
spread over the batch: 1,000 on the 64x64 map, about 28 on the larger ones --
over the whole map, streamed in neuron blocks on several host threads, and
both GPU results are checked against it.
Properties that hold at any size are checked on every row.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2608_24067_amd.som as som
import synth
from parity import check_margin_rule, check_top2

pytestmark = pytest.mark.gpu

HOST_THREADS = max(1, min(16, os.cpu_count() or 1))
SAMPLED_ROWS = {"64": 1000}


def sampled_rows(N, k=24):
    rows = set(np.linspace(0, N - 1, k).astype(int).tolist())
    rows |= {0, 1, N - 2, N - 1}
    return np.array(sorted(r for r in rows if 0 <= r < N))


def run_full(name):
    cfg = synth.CONFIGS[name]
    dev = torch.device("cuda:0")
    row_ptr, col_idx = synth.make_csr(cfg.seed, cfg.N, cfg.V, cfg.lam, cfg.zipf_s)
    nnz = int(row_ptr[-1])
    W = synth.codebook_to_device(cfg.seed, cfg.kind, cfg.V, cfg.M, dev)
    rp = torch.from_numpy(row_ptr).to(dev)
    ci = torch.from_numpy(col_idx).to(dev)
    norms = som.codebook_norms(W, cfg.V, cfg.M)
    # one two-best workspace serves both searches (the single-best layout is its prefix)
    ws = som.alloc_workspace2(cfg.N, cfg.M, cfg.V, nnz, dev)
    b, d = som.bmu_search(W, norms, rp, ci, cfg.V, cfg.M, nnz=nnz, workspace=ws)
    torch.cuda.synchronize()
    flags = som.input_flags(ws, cfg.N, cfg.M, cfg.V, nnz)
    out = b.cpu().numpy(), d.cpu().numpy()
    del b, d
    top2 = tuple(t.cpu().numpy() for t in som.bmu2_search(W, norms, rp, ci, cfg.V, cfg.M, nnz=nnz, workspace=ws))
    flags2 = som.input_flags(ws, cfg.N, cfg.M, cfg.V, nnz)
    del W, ws, rp, ci, norms
    torch.cuda.empty_cache()
    return cfg, row_ptr, col_idx, out, top2, flags | flags2


@pytest.mark.parametrize("name", ["64", "256", "512", "1024"])
def test_full_workload(name):
    cfg, row_ptr, col_idx, (b, d), top2, flags = run_full(name)
    assert flags == 0
    # every row: a valid unit and a finite, non-negative (up to rounding) squared distance
    assert b.min() >= 0 and b.max() < cfg.M
    assert np.isfinite(d).all() and d.min() > -1e-6
    # the two-best search repeats the single-best answer and adds a different, no-closer unit
    assert np.array_equal(top2[0], b) and np.array_equal(top2[1], d)
    assert (top2[2] != b).all() and top2[2].min() >= 0 and top2[2].max() < cfg.M and (top2[3] >= d).all()

    rows = sampled_rows(cfg.N, k=SAMPLED_ROWS.get(name, 24))
    sub_rp = np.zeros(len(rows) + 1, dtype=np.int32)
    sub_rp[1:] = np.cumsum(row_ptr[rows + 1] - row_ptr[rows])
    sub_ci = np.concatenate([col_idx[row_ptr[r]:row_ptr[r + 1]] for r in rows])

    def block(i0, i1):
        return synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M, i0=i0, i1=i1, nthreads=1)

    ref = oracle.bmu2_streamed(block, cfg.M, sub_rp, sub_ci, block=4096, nthreads=HOST_THREADS)
    b_ref, d_ref, d2_ref = ref[0], ref[1], ref[3]

    def dist_at(k, i):
        return oracle.distance_at(block(i, i + 1)[:, 0], sub_ci[sub_rp[k]:sub_rp[k + 1]])

    stats = check_margin_rule(b[rows], d[rows], b_ref, d_ref, d2_ref, dist_at, what=f"{name} full")
    stats2 = check_top2(tuple(x[rows] for x in top2), ref, dist_at, exact=False, what=f"{name} full top-2")
    print(f"{cfg.describe()}: {stats} top-2 {stats2}")
