"""som_bmu_search_noalloc (no workspace argument; the library's own scratch array) against som_bmu_search.

Two calls in a row on one GPU, the second with a smaller batch on a smaller map (the
array keeps the first call's contents), each bit-identical to the workspace entry
point on the same inputs, and held to the oracle's bar (k/256 codebooks bit-exact,
continuous ones the margin rule). Runs alone in a fresh process or after the other
GPU tests. (The host check that rejects a search larger than the array is a CPU
test in test_abi.py.)
"""
import numpy as np
import pytest
import torch

import paper_2608_24067_amd.som as som
import synth
from parity import compare, to_dev

pytestmark = pytest.mark.gpu


def run_both(seed, N, V, M, kind, tile, keep, dev):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, M)
    Wd = to_dev(W, dev)
    norms = som.codebook_norms(Wd, V, M)
    rpd, cid = to_dev(rp, dev), to_dev(ci, dev)
    nnz = int(rp[-1])
    assert som.workspace_bytes(N, M, V, nnz, tile, keep) <= som.NOALLOC_SCRATCH_BYTES
    b_ref, d_ref = som.bmu_search(Wd, norms, rpd, cid, V, M, nnz=nnz, tile_samples=tile, keep_order=keep)
    b = torch.full((N,), -7, dtype=torch.int32, device=dev)
    d = torch.full((N,), -7.0, dtype=torch.float64, device=dev)
    som.bmu_search_noalloc(Wd, norms, rpd, cid, V, M, nnz, b, d, tile_samples=tile, keep_order=keep)
    torch.cuda.synchronize()
    b, d = b.cpu().numpy(), d.cpu().numpy()
    assert np.array_equal(b, b_ref.cpu().numpy()) and np.array_equal(d, d_ref.cpu().numpy())
    compare(W, rp, ci, b, d, exact=(kind == synth.QUANTISED), what=f"noalloc N={N} M={M}",
            rows=None if N <= 2000 else np.linspace(0, N - 1, 400).astype(int), nthreads=8)


@pytest.mark.parametrize("tile,keep", [(8, False), (16, True)])
def test_noalloc_equals_workspace_search_twice(dev, tile, keep):
    run_both(61, 20_000, 30_000, 4099, synth.UNIFORM, tile, keep, dev)   # first call: 20,000 rows, M = 4,099
    run_both(62, 1_500, 2_000, 1_300, synth.QUANTISED, tile, keep, dev)  # second call: smaller batch and map
