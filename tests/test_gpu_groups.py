"""GPU parity when the sweep's workgroups take long groups of consecutive tiles.

A batch of 1.1 M rows gives 137,500 tiles of 8, enough for groups of 8 tiles per
workgroup (two per wave) -- the smaller parity tests run with groups of 4, and the
full-size workloads check samples only. A k/256 codebook with 1,100 neurons (two
strips, the second ragged) and k/256 values make every distance exact, so each
form of the search is compared bit for bit with the oracle on 1,500 rows spread
over the whole batch, and the forms are compared with each other on every row:
fp16 storage of a k/256 codebook is exact, and unit values reproduce the binary
search.
"""
import os

import numpy as np
import pytest

import synth
from parity import compare, compare2, compare_sf, gpu_run, gpu_run2, gpu_run_sf, to_dev

pytestmark = pytest.mark.gpu

HOST_THREADS = max(1, min(16, os.cpu_count() or 1))
N, V, M, SEED = 1_100_000, 2000, 1100, 121


@pytest.fixture(scope="module")
def batch():
    rp, ci = synth.make_csr(SEED, N, V)
    W = synth.codebook(SEED, synth.QUANTISED, V, M)
    vals = synth.values(SEED, len(ci), synth.VAL_QUANTISED)
    rows = np.sort(np.random.default_rng(SEED).choice(N, 1500, replace=False))
    return rp, ci, W, vals, rows


def test_best_unit_fp32_and_fp16(dev, batch):
    import torch

    rp, ci, W, _, rows = batch
    b, d, _ = gpu_run(W, rp, ci, dev)
    compare(W, rp, ci, b, d, exact=True, what="grouped tiles fp32", rows=rows, nthreads=HOST_THREADS)
    b16, d16, _ = gpu_run(to_dev(W, dev).to(torch.float16), rp, ci, dev)
    assert np.array_equal(b16, b) and np.array_equal(d16, d)


def test_two_best(dev, batch):
    rp, ci, W, _, rows = batch
    g = gpu_run2(W, rp, ci, dev)
    compare2(W, rp, ci, g, exact=True, what="grouped tiles two-best", rows=rows,
             nthreads=HOST_THREADS)
    b, d, _ = gpu_run(W, rp, ci, dev)
    assert np.array_equal(g[0], b) and np.array_equal(g[1], d)


def test_real_valued_rows(dev, batch):
    rp, ci, W, vals, rows = batch
    g = gpu_run_sf(W, rp, ci, vals, dev)
    compare_sf(W, rp, ci, vals, g, exact=True, what="grouped tiles real values", rows=rows,
               nthreads=HOST_THREADS)
    ones = gpu_run_sf(W, rp, ci, np.ones(len(ci), dtype=np.float32), dev)
    g2 = gpu_run2(W, rp, ci, dev)
    for a, b in zip(ones, g2):
        assert np.array_equal(a, b)
