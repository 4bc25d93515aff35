"""GPU parity of the batch update (som_update, som_update_f16) against the update oracle.

The oracle runs the paper's steps in their order and precision (integer
counts, fp32 running-sum box passes along rows then columns, fp32 quotient),
and the kernels run the same operations in the same order, so the new
codebook must agree bit for bit -- also where the blurred sums exceed 2^24
and fp32 rounds. An fp16 codebook gets the fp32 quotient rounded once.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_24067_amd.som as som
import synth
from parity import to_dev

pytestmark = pytest.mark.gpu


def update_case(seed, N, V, E, kind=synth.UNIFORM, spread=1.0):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, E * E)
    rng = np.random.default_rng(seed)
    bmu = rng.integers(0, max(1, int(E * E * spread)), N).astype(np.int32)
    return rp, ci, W, bmu


def gpu_update(W, rp, ci, bmu, E, r, dev, chunk=0):
    V = W.shape[0]
    Wd = to_dev(W, dev)
    som.update(Wd, to_dev(rp, dev), to_dev(ci, dev), to_dev(bmu, dev), V, E, r, nnz=int(rp[-1] - rp[0]),
               chunk_features=chunk)
    torch.cuda.synchronize()
    return Wd.cpu().numpy()


@pytest.mark.parametrize("seed,N,V,E,r,chunk,spread", [
    (91, 300, 40, 9, 1, 0, 1.0),
    (92, 2000, 300, 16, 2, 0, 1.0),
    (93, 2000, 300, 16, 5, 7, 0.3),    # a third of the lattice holds every sample: zero-den units stay
    (94, 500, 120, 12, 1, 1, 0.1),
    (95, 30000, 500, 64, 32, 64, 1.0),  # sums far beyond 2^24: fp32 rounding, same order on both sides
    (96, 5000, 2000, 32, 16, 0, 1.0),
    (97, 1, 30, 5, 3, 0, 1.0),         # one sample
    (98, 400, 64, 1, 1, 0, 1.0),       # a one-unit map
    (109, 800, 50, 6, 9, 0, 1.0),      # radius beyond the lattice: every window is the whole line
    (110, 600, 40, 8, 7, 3, 1.0),      # radius E - 1
    (111, 3000, 60, 7, 2, 0, 1.0),     # odd lattice, short lines
])
def test_update_bit_exact(dev, seed, N, V, E, r, chunk, spread):
    rp, ci, W, bmu = update_case(seed, N, V, E, spread=spread)
    got = gpu_update(W, rp, ci, bmu, E, r, dev, chunk)
    ref = oracle.update(W, E, rp, ci, bmu, r)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} weights differ, first {bad[:5]}: {got.reshape(-1)[bad[:5]]} vs {ref.reshape(-1)[bad[:5]]}"


def crowded_bmu(seed, N, M, shares):
    """Best units where unit u takes the fraction shares[u] (or the exact count, if an int)
    of the batch and the rest spread uniformly: crowded units take the LDS-counting path
    (1024 samples or more), runs of 16384 sorted samples split one unit across workgroups."""
    rng = np.random.default_rng(seed)
    rest = np.setdiff1d(np.arange(M), list(shares))
    bmu = rest[rng.integers(0, rest.size, N)].astype(np.int32) if rest.size else np.zeros(N, np.int32)
    at = 0
    for u, share in shares.items():
        n = share if isinstance(share, int) else int(share * N)
        bmu[at:at + n] = u
        at += n
    return bmu[rng.permutation(N)]


@pytest.mark.parametrize("seed,N,V,E,r,chunk,shares", [
    (101, 20000, 17000, 8, 2, 0, {0: 1.0}),            # one unit takes all: two runs, two LDS passes
    (102, 30000, 600, 16, 3, 250, {7: 0.55, 200: 0.25}),  # two crowded units, the rest spread; 3 chunks
    (103, 3400, 90, 12, 1, 1, {3: 1023, 4: 1024, 5: 1025}),  # either side of the threshold
    (104, 40000, 300, 32, 5, 0, {1023: 0.5}),          # the last unit, runs ending at the batch end
])
def test_update_crowded_units(dev, seed, N, V, E, r, chunk, shares):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, synth.UNIFORM, V, E * E)
    bmu = crowded_bmu(seed, N, E * E, shares)
    got = gpu_update(W, rp, ci, bmu, E, r, dev, chunk)
    ref = oracle.update(W, E, rp, ci, bmu, r)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} weights differ, first {bad[:5]}"


@pytest.mark.parametrize("seed,N,V,E,shares", [
    (105, 6000, 200, 16, {9: 0.4}),     # a crowded unit among the skipped samples
    (106, 3000, 150, 12, {}),           # uncrowded units only
])
def test_update_skips_invalid_units(dev, seed, N, V, E, shares):
    # best units outside [0, M) are skipped: the result equals the update of the batch without those samples
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, synth.UNIFORM, V, E * E)
    bmu = crowded_bmu(seed, N, E * E, shares)
    rng = np.random.default_rng(seed + 1)
    bad = rng.random(N) < 0.15
    bmu[bad] = np.where(rng.random(int(bad.sum())) < 0.5, -1, E * E + rng.integers(0, 5, int(bad.sum())))
    got = gpu_update(W, rp, ci, bmu, E, 2, dev)
    keep = np.flatnonzero(~bad)
    lens = np.diff(rp)[keep]
    rp_k = np.zeros(keep.size + 1, np.int32)
    np.cumsum(lens, out=rp_k[1:])
    ci_k = np.concatenate([ci[rp[k]:rp[k + 1]] for k in keep]).astype(np.int32)
    ref = oracle.update(W, E, rp_k, ci_k, bmu[keep], 2)
    assert np.array_equal(got, ref)


def test_update_empty_batch_keeps_codebook(dev):
    # no samples: every blurred den is zero, so every prototype stays as it was
    W = synth.codebook(107, synth.UNIFORM, 50, 64)
    rp = np.zeros(1, np.int32)
    got = gpu_update(W, rp, np.zeros(0, np.int32), np.zeros(0, np.int32), 8, 2, dev)
    assert np.array_equal(got, W)


@pytest.mark.parametrize("how", ["decreasing", "negative_first"])
def test_update_invalid_row_ptr_keeps_codebook(dev, how):
    """Row pointers that decrease (overlapping rows), or a negative first offset (which would name ids before
    col_idx), are caught on the device before any row is read, and the update then leaves the codebook as it is."""
    rp, ci, W, bmu = update_case(108, 600, 80, 10)
    nnz = int(rp[-1])
    if how == "decreasing":
        bad = rp.copy()
        bad[1::2] = nnz
    else:
        bad = (rp - 3).astype(np.int32)
    with pytest.raises(som.SomError):
        som.validate_csr_host(bad, ci, 80)
    Wd = to_dev(W, dev)
    som.update(Wd, to_dev(bad, dev), to_dev(ci, dev), to_dev(bmu, dev), 80, 10, 2, nnz=nnz)
    torch.cuda.synchronize()
    assert np.array_equal(Wd.cpu().numpy(), W)


def test_update_f16(dev):
    rp, ci, W, bmu = update_case(99, 3000, 400, 24, spread=0.5)
    W16 = W.astype(np.float16)
    got = gpu_update(W16, rp, ci, bmu, 24, 3, dev, chunk=50)
    ref = oracle.update(W16.astype(np.float32), 24, rp, ci, bmu, 3)
    assert np.array_equal(got, ref.astype(np.float16))


def test_update_repeatable_and_chunk_invariant(dev):
    rp, ci, W, bmu = update_case(100, 8000, 700, 32, spread=1.0)
    a = gpu_update(W, rp, ci, bmu, 32, 9, dev, chunk=0)
    b = gpu_update(W, rp, ci, bmu, 32, 9, dev, chunk=33)
    c = gpu_update(W, rp, ci, bmu, 32, 9, dev, chunk=0)
    assert np.array_equal(a, b) and np.array_equal(a, c)


def test_one_epoch_on_the_tiny_workload(dev):
    # search -> update -> norms -> search, against the oracle chain
    cfg = synth.CONFIGS["tiny"]
    rp, ci = synth.make_csr(cfg.seed, cfg.N, cfg.V)
    W = synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M)
    r = som.radius(som.sigma(1, 0.5 * cfg.edge, 0.5))
    Wd, rpd, cid = to_dev(W, dev), to_dev(rp, dev), to_dev(ci, dev)
    norms = som.codebook_norms(Wd, cfg.V, cfg.M)
    b, _ = som.bmu_search(Wd, norms, rpd, cid, cfg.V, cfg.M)
    som.update(Wd, rpd, cid, b, cfg.V, cfg.edge, r)
    norms = som.codebook_norms(Wd, cfg.V, cfg.M)
    b2, d2 = som.bmu_search(Wd, norms, rpd, cid, cfg.V, cfg.M)
    torch.cuda.synchronize()
    b_ref, _, _ = oracle.bmu(W, rp, ci)
    assert np.array_equal(b.cpu().numpy(), b_ref)
    W1 = oracle.update(W, cfg.edge, rp, ci, b_ref, r)
    assert np.array_equal(Wd.cpu().numpy(), W1)
    b2_ref, d2_ref, dd2_ref = oracle.bmu(W1, rp, ci)
    from parity import check_margin_rule

    def dist_at(k, i):
        return oracle.distance_at(W1[:, i], ci[rp[k]:rp[k + 1]])

    check_margin_rule(b2.cpu().numpy(), d2.cpu().numpy(), b2_ref, d2_ref, dd2_ref, dist_at, what="epoch 2")


@pytest.mark.parametrize("f16", [False, True])
def test_update_residual_den_keeps_unreached_units(dev, f16):
    """fp32 running sums past 2^24 leave den = 2 at four units no sample reaches (the oracle pins' residual case,
    369,767 samples on a 10 x 10 lattice): the kernels take the keep-the-prototype rule on the exact support, as the
    oracle does, so the codebook matches it bit for bit and those units keep their prototype."""
    import oracle_pins

    E, r, W, rp, ci, bmu = oracle_pins.residual_case()
    if f16:
        W = W.astype(np.float16)
    got = gpu_update(W, rp, ci, bmu, E, r, dev)
    ref = oracle.update(W.astype(np.float32), E, rp, ci, bmu, r).astype(W.dtype)
    assert np.array_equal(got, ref)
    unreached = np.zeros((E, E), dtype=bool)
    unreached[6:, 5] = True
    assert np.array_equal(got[:, unreached.ravel()], W[:, unreached.ravel()])
