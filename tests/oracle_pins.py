"""Pins that tie the CPU oracle to facts fixed outside it.

Each check takes an oracle library handle (the built oracle, or a mutated
build in the mutation test) and raises AssertionError on a mismatch. None of
them re-calls the oracle's own formula: they use exact integer arithmetic,
scipy's cdist, the expanded form of Eq. (1) through a matrix product, a
pure-Python node-major loop, and closed forms for planted and constant
codebooks.
"""
from __future__ import annotations

import os

import numpy as np
from scipy.spatial.distance import cdist

import oracle
import synth


def dense_x(row_ptr, col_idx, V):
    N = row_ptr.shape[0] - 1
    X = np.zeros((N, V), dtype=np.int64)
    for s in range(N):
        X[s, col_idx[row_ptr[s]:row_ptr[s + 1]]] = 1
    return X


def small_case(seed=5, N=48, V=300, M=40, kind=synth.QUANTISED):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, M)
    return rp, ci, W


def first_min_and_second(D):
    """Lowest-index argmin per row and the smallest value over the other columns."""
    b = np.argmin(D, axis=1)  # numpy returns the first occurrence
    masked = D.astype(np.float64).copy()
    masked[np.arange(D.shape[0]), b] = np.inf
    return b, masked.min(axis=1)


# ---------------------------------------------------------------- the checks

def check_exact_integer_direct(lib):
    """Quantised k/256 codebook: 65536*D_i = sum_v (256 x_v - k_{v,i})^2 exactly, in int64."""
    rp, ci, W = small_case()
    K = np.rint(W * 256).astype(np.int64)
    X = dense_x(rp, ci, W.shape[0])
    Dint = ((256 * X[:, :, None] - K[None, :, :]) ** 2).sum(axis=1)  # N x M, exact
    b_ref, d2_ref = first_min_and_second(Dint)
    b, d, d2 = oracle.bmu(W, rp, ci, lib=lib)
    assert np.array_equal(b, b_ref), "argmin differs from the exact integer argmin"
    assert np.array_equal(d * 65536.0, Dint[np.arange(len(b)), b_ref].astype(np.float64)), "distance not exact"
    assert np.array_equal(d2 * 65536.0, d2_ref), "second-best distance not exact"


def check_exact_integer_tiny(lib, n_samples=None):
    """The full tiny workload (16x16 map, V=2000, k/256): indices and distances exact.

    The integer reference uses the expanded identity in int64, which is exact
    (no rounding), so it is an independent evaluation of the same integers.
    """
    cfg = synth.CONFIGS["tiny"]
    rp, ci = synth.make_csr(cfg.seed, cfg.N, cfg.V)
    if n_samples is not None:
        rp = rp[: n_samples + 1]
    W = synth.codebook(cfg.seed, cfg.kind, cfg.V, cfg.M)
    K = np.rint(W * 256).astype(np.int64)
    N = rp.shape[0] - 1
    nnz = np.diff(rp).astype(np.int64)
    XK = np.zeros((N, cfg.M), dtype=np.int64)
    for s in range(N):
        XK[s] = K[ci[rp[s]:rp[s + 1]]].sum(axis=0)
    Dint = 65536 * nnz[:, None] - 512 * XK + (K * K).sum(axis=0)[None, :]
    b_ref, d2_ref = first_min_and_second(Dint)
    b, d, d2 = oracle.bmu(W, rp, ci, lib=lib)
    assert np.array_equal(b, b_ref)
    assert np.array_equal(d * 65536.0, Dint[np.arange(N), b_ref].astype(np.float64))
    assert np.array_equal(d2 * 65536.0, d2_ref)


def check_cdist_node_major(lib):
    """scipy's sqeuclidean distance on the node-major transpose agrees (continuous codebook)."""
    rp, ci, W = small_case(seed=11, kind=synth.UNIFORM, M=57)
    X = dense_x(rp, ci, W.shape[0]).astype(np.float64)
    Wnm = np.ascontiguousarray(W.T).astype(np.float64)  # node-major: row i = prototype w_i
    D = cdist(X, Wnm, "sqeuclidean")
    b, d, d2 = oracle.bmu(W, rp, ci, lib=lib)
    assert np.allclose(d, D[np.arange(len(b)), b], rtol=1e-12, atol=0)
    srt = np.sort(D, axis=1)
    assert np.allclose(d, srt[:, 0], rtol=1e-12, atol=0), "not the minimum distance"
    assert np.allclose(d2, srt[:, 1], rtol=1e-12, atol=0), "not the second-smallest distance"


def check_expanded_form(lib):
    """Eq. (1): ||x - w||^2 = ||w||^2 - 2<x,w> + ||x||^2, evaluated by a matrix product."""
    rp, ci, W = small_case(seed=12, kind=synth.UNIFORM, N=40, V=500, M=33)
    X = dense_x(rp, ci, W.shape[0]).astype(np.float64)
    W64 = W.astype(np.float64)
    D = (W64 * W64).sum(axis=0)[None, :] - 2.0 * (X @ W64) + X.sum(axis=1)[:, None]
    b, d, _ = oracle.bmu(W, rp, ci, lib=lib)
    assert np.allclose(d, D.min(axis=1), rtol=1e-11, atol=1e-9)
    assert np.allclose(d, D[np.arange(len(b)), b], rtol=1e-11, atol=1e-9)


def check_node_major_python_loop(lib):
    """A pure-Python node-major loop in ascending v gives bit-identical fp64 distances."""
    rp, ci, W = small_case(seed=13, kind=synth.UNIFORM, N=6, V=37, M=9)
    V, M = W.shape
    Wnm = [[float(W[v, i]) for v in range(V)] for i in range(M)]
    for s in range(rp.shape[0] - 1):
        active = set(int(v) for v in ci[rp[s]:rp[s + 1]])
        Ds = []
        for i in range(M):
            acc = 0.0
            for v in range(V):
                diff = (1.0 if v in active else 0.0) - Wnm[i][v]
                acc += diff * diff
            Ds.append(acc)
        best = min(range(M), key=lambda i: (Ds[i], i))
        b, d, _ = oracle.bmu(W, rp[s:s + 2], ci, lib=lib)
        assert int(b[0]) == best and float(d[0]) == Ds[best]


def check_planted_neuron(lib):
    """A prototype equal to the input has distance 0 and wins."""
    rp, ci, W = small_case(seed=14, kind=synth.UNIFORM, N=20, V=200, M=31)
    W = W.copy()
    for s, j in [(3, 17), (7, 0), (19, 30)]:
        Wp = W.copy()
        Wp[:, j] = 0.0
        Wp[ci[rp[s]:rp[s + 1]], j] = 1.0
        b, d, d2 = oracle.bmu(Wp, rp[s:s + 2], ci, lib=lib)
        assert int(b[0]) == j and float(d[0]) == 0.0 and d2[0] > 0


def check_constant_codebook(lib):
    """All prototypes equal: every distance ties, the lowest index (0) wins, closed-form distance."""
    rp, ci, W = small_case(seed=15, N=30, V=120, M=13)
    c = 0.25
    Wc = np.full_like(W, c)
    b, d, d2 = oracle.bmu(Wc, rp, ci, lib=lib)
    nnz = np.diff(rp).astype(np.float64)
    closed = nnz * (1 - c) ** 2 + (W.shape[0] - nnz) * c ** 2
    assert (b == 0).all()
    assert np.array_equal(d, closed) and np.array_equal(d2, closed)


def check_tie_lowest_index(lib):
    """Two identical best prototypes far apart: the lower index wins."""
    rp, ci, W = small_case(seed=16, kind=synth.UNIFORM, N=10, V=150, M=64)
    s = 4
    Wp = W.copy()
    for j in (5, 61):
        Wp[:, j] = 0.0
        Wp[ci[rp[s]:rp[s + 1]], j] = 0.9
    b, d, d2 = oracle.bmu(Wp, rp[s:s + 2], ci, lib=lib)
    assert int(b[0]) == 5 and d2[0] == d[0]
    # the same pair seen from a block that starts past the first copy
    b2, _, _ = oracle.bmu(np.ascontiguousarray(Wp[:, 6:]), rp[s:s + 2], ci, i0=6, lib=lib)
    assert int(b2[0]) == 61


def check_single_neuron_and_empty_row(lib):
    """M = 1 gives index 0 and an infinite second best; an empty row ranks by ||w||^2."""
    rp, ci, W = small_case(seed=17, kind=synth.UNIFORM, N=8, V=90, M=21)
    b, d, d2 = oracle.bmu(np.ascontiguousarray(W[:, 4:5]), rp, ci, i0=4, lib=lib)
    assert (b == 4).all() and np.isinf(d2).all()
    X = dense_x(rp, ci, W.shape[0]).astype(np.float64)
    assert np.allclose(d, ((X - W[:, 4].astype(np.float64)[None, :]) ** 2).sum(axis=1), rtol=1e-13)
    empty_rp = np.array([0, 0], dtype=np.int32)
    b, d, _ = oracle.bmu(W, empty_rp, ci, lib=lib)
    n = (W.astype(np.float64) ** 2).sum(axis=0)
    assert int(b[0]) == int(np.argmin(n)) and np.isclose(d[0], n.min(), rtol=1e-13)


def check_quantisation_error(lib):
    """QE, the mean input-to-BMU distance (Background, quality measures), recomputed at the returned units."""
    rp, ci, W = small_case(seed=18, kind=synth.UNIFORM, N=50, V=250, M=36)
    X = dense_x(rp, ci, W.shape[0]).astype(np.float64)
    b, d, _ = oracle.bmu(W, rp, ci, lib=lib)
    D = cdist(X, W.T.astype(np.float64), "sqeuclidean")
    qe_ref = D.min(axis=1).mean()
    assert np.isclose(d.mean(), qe_ref, rtol=1e-12)
    assert np.isclose(np.mean(D[np.arange(len(b)), b]), qe_ref, rtol=1e-12)


def check_offset_rows_and_blocks(lib):
    """A batch slice (row_ptr not starting at 0) and a streamed, merged run equal one whole call."""
    rp, ci, W = small_case(seed=19, kind=synth.UNIFORM, N=30, V=160, M=50)
    whole = oracle.bmu(W, rp, ci, lib=lib)
    sl = oracle.bmu(W, rp[10:21], ci, lib=lib)
    for a, bb in zip(sl, whole):
        assert np.array_equal(a, bb[10:20])
    streamed = oracle.bmu_streamed(lambda i0, i1: np.ascontiguousarray(W[:, i0:i1]), W.shape[1], rp, ci,
                                   block=7, nthreads=3, lib=lib)
    for a, bb in zip(streamed, whole):
        assert np.array_equal(a, bb)


def check_norms(lib):
    """Per-neuron squared norms: exact for k/256 weights, fp64-close otherwise."""
    _, _, Wq = small_case(seed=20, V=700, M=29)
    n = oracle.norms(Wq, lib=lib)
    K = np.rint(Wq * 256).astype(np.int64)
    assert np.array_equal(n * 65536.0, (K * K).sum(axis=0).astype(np.float64))
    _, _, Wu = small_case(seed=21, kind=synth.UNIFORM, V=700, M=29)
    assert np.allclose(oracle.norms(Wu, lib=lib), (Wu.astype(np.float64) ** 2).sum(axis=0), rtol=1e-14)


def check_error_codes(lib):
    """Invalid CSR and bad shapes are rejected with the documented codes."""
    W = np.zeros((5, 3), dtype=np.float32)
    out = np.zeros(4, dtype=np.float64)
    ob = np.zeros(4, dtype=np.int32)
    f = lib.som_bmu_oracle_host
    rp = np.array([0, 2], dtype=np.int32)
    bad_id = np.array([1, 5], dtype=np.int32)
    assert f(W.ctypes.data, 3, 5, 0, 3, rp.ctypes.data, bad_id.ctypes.data, 1, ob.ctypes.data, out.ctypes.data,
             None) == oracle.BAD_CSR
    dec = np.array([2, 0], dtype=np.int32)
    ok_ids = np.array([1, 2], dtype=np.int32)
    assert f(W.ctypes.data, 3, 5, 0, 3, dec.ctypes.data, ok_ids.ctypes.data, 1, ob.ctypes.data, out.ctypes.data,
             None) == oracle.BAD_CSR
    assert f(W.ctypes.data, 2, 5, 0, 3, rp.ctypes.data, ok_ids.ctypes.data, 1, ob.ctypes.data, out.ctypes.data,
             None) == oracle.BAD_ARG
    assert f(None, 3, 5, 0, 3, rp.ctypes.data, ok_ids.ctypes.data, 1, ob.ctypes.data, out.ctypes.data,
             None) == oracle.BAD_ARG


# ------------------------------------------------- the two best units (top-2)

def exact_ranks(Dint_row):
    """Units in the order (distance, index) from exact integer distances: pure Python sort."""
    return sorted(range(len(Dint_row)), key=lambda i: (int(Dint_row[i]), i))


def check_top2_exact_integer(lib):
    """Quantised codebook: ranks 1-3 from an exact int64 brute force and a Python sort on (D, i)."""
    rp, ci, W = small_case(seed=22, N=60, V=200, M=37)
    K = np.rint(W * 256).astype(np.int64)
    X = dense_x(rp, ci, W.shape[0])
    Dint = ((256 * X[:, :, None] - K[None, :, :]) ** 2).sum(axis=1)
    b1, d1, b2, d2, d3 = oracle.bmu2(W, rp, ci, lib=lib)
    for s in range(len(b1)):
        r = exact_ranks(Dint[s])
        assert (int(b1[s]), int(b2[s])) == (r[0], r[1]), f"sample {s}: ranks differ"
        assert (d1[s] * 65536.0, d2[s] * 65536.0, d3[s] * 65536.0) == tuple(float(Dint[s, i]) for i in r[:3])


def check_top2_ties_and_small_maps(lib):
    """Three identical best prototypes at indices 9, 2, 5 rank 2 then 5 (d3 = 0 too); a planted
    near-copy one feature away is the runner-up at distance 1; one and two neurons give -1 / +inf."""
    rp, ci, W = small_case(seed=23, kind=synth.UNIFORM, N=8, V=120, M=20)
    s = 3
    ids = ci[rp[s]:rp[s + 1]]
    Wt = W.copy()
    for j in (9, 2, 5):
        Wt[:, j] = 0.0
        Wt[ids, j] = 1.0
    b1, d1, b2, d2, d3 = oracle.bmu2(Wt, rp[s:s + 2], ci, lib=lib)
    assert (int(b1[0]), int(b2[0])) == (2, 5) and d1[0] == d2[0] == d3[0] == 0.0
    Wp = W.copy()
    Wp[:, 11] = 0.0
    Wp[ids, 11] = 1.0                   # exact copy of the input: distance 0
    Wp[:, 4] = Wp[:, 11]
    Wp[ids[0], 4] = 0.0                 # one active feature dropped: distance 1
    b1, d1, b2, d2, d3 = oracle.bmu2(Wp, rp[s:s + 2], ci, lib=lib)
    assert (int(b1[0]), float(d1[0]), int(b2[0]), float(d2[0])) == (11, 0.0, 4, 1.0) and d3[0] > 1.0
    one = oracle.bmu2(np.ascontiguousarray(W[:, 7:8]), rp, ci, i0=7, lib=lib)
    assert (one[0] == 7).all() and (one[2] == -1).all() and np.isinf(one[3]).all() and np.isinf(one[4]).all()
    two = oracle.bmu2(np.ascontiguousarray(W[:, 7:9]), rp, ci, i0=7, lib=lib)
    assert set(zip(two[0].tolist(), two[2].tolist())) <= {(7, 8), (8, 7)} and np.isinf(two[4]).all()


def check_top2_cdist_and_top1(lib):
    """Continuous codebook: scipy's distances sorted agree; rank 1 and the second distance equal
    what the single-best oracle returns for the same rows."""
    rp, ci, W = small_case(seed=24, kind=synth.UNIFORM, N=45, V=260, M=48)
    X = dense_x(rp, ci, W.shape[0]).astype(np.float64)
    D = cdist(X, np.ascontiguousarray(W.T).astype(np.float64), "sqeuclidean")
    b1, d1, b2, d2, d3 = oracle.bmu2(W, rp, ci, lib=lib)
    order = np.argsort(D, axis=1, kind="stable")
    assert np.array_equal(b1, order[:, 0]) and np.array_equal(b2, order[:, 1])
    srt = np.sort(D, axis=1)
    for got, k in ((d1, 0), (d2, 1), (d3, 2)):
        assert np.allclose(got, srt[:, k], rtol=1e-12, atol=0)
    t1 = oracle.bmu(W, rp, ci, lib=lib)
    assert np.array_equal(t1[0], b1) and np.array_equal(t1[1], d1) and np.array_equal(t1[2], d2)


def check_top2_blocks(lib):
    """Streamed over small neuron blocks and merged, ranks 1-3 equal one whole call."""
    rp, ci, W = small_case(seed=25, N=40, V=150, M=45)
    Wd = W.copy()
    Wd[:, 30] = Wd[:, 3]  # an exact duplicate across blocks: the tie must still go to 3
    whole = oracle.bmu2(Wd, rp, ci, lib=lib)
    streamed = oracle.bmu2_streamed(lambda i0, i1: np.ascontiguousarray(Wd[:, i0:i1]), 45, rp, ci, block=6,
                                    nthreads=2, lib=lib)
    for a, b in zip(whole, streamed):
        assert np.array_equal(a, b)


# ----------------------------------------------- sparse real-valued inputs

def sf_case(seed, N, V, M, kind=synth.QUANTISED, vkind=synth.VAL_QUANTISED):
    rp, ci = synth.make_csr(seed, N, V)
    W = synth.codebook(seed, kind, V, M)
    vals = synth.values(seed, len(ci), vkind)
    return rp, ci, vals, W


def dense_values(row_ptr, col_idx, vals, V):
    N = row_ptr.shape[0] - 1
    X = np.zeros((N, V), dtype=np.float64)
    for s in range(N):
        X[s, col_idx[row_ptr[s]:row_ptr[s + 1]]] = vals[row_ptr[s]:row_ptr[s + 1]]
    return X


def check_sf_exact_integer(lib):
    """k/256 codebook and (j+1)/256 values: 65536*D_i = sum_v (256 x_v - k_{v,i})^2 in int64; ranks by a Python sort."""
    rp, ci, vals, W = sf_case(26, 50, 220, 31)
    K = np.rint(W * 256).astype(np.int64)
    X256 = np.rint(dense_values(rp, ci, vals, W.shape[0]) * 256).astype(np.int64)
    Dint = ((X256[:, :, None] - K[None, :, :]) ** 2).sum(axis=1)
    b1, d1, b2, d2, d3 = oracle.bmu_sf(W, rp, ci, vals, lib=lib)
    for s in range(len(b1)):
        r = exact_ranks(Dint[s])
        assert (int(b1[s]), int(b2[s])) == (r[0], r[1]), f"sample {s}: ranks differ"
        assert (d1[s] * 65536.0, d2[s] * 65536.0, d3[s] * 65536.0) == tuple(float(Dint[s, i]) for i in r[:3])


def check_sf_binary_values_reduce(lib):
    """All values 1: the real-valued oracle returns exactly the binary two-best oracle's answer."""
    rp, ci, _, W = sf_case(27, 40, 300, 45, kind=synth.UNIFORM)
    ones = np.ones(len(ci), dtype=np.float32)
    for a, b in zip(oracle.bmu_sf(W, rp, ci, ones, lib=lib), oracle.bmu2(W, rp, ci, lib=lib)):
        assert np.array_equal(a, b)


def check_sf_cdist_and_planted(lib):
    """Continuous values: scipy cdist sorted agrees; a prototype equal to the input has distance 0, one
    whose value for the first feature is halved has distance (x/2)^2 exactly; three tied copies rank by
    index; doubling x and W scales every distance by exactly 4."""
    rp, ci, vals, W = sf_case(28, 36, 240, 40, kind=synth.UNIFORM, vkind=synth.VAL_UNIFORM)
    X = dense_values(rp, ci, vals, W.shape[0])
    D = cdist(X, np.ascontiguousarray(W.T).astype(np.float64), "sqeuclidean")
    b1, d1, b2, d2, d3 = oracle.bmu_sf(W, rp, ci, vals, lib=lib)
    order = np.argsort(D, axis=1, kind="stable")
    assert np.array_equal(b1, order[:, 0]) and np.array_equal(b2, order[:, 1])
    srt = np.sort(D, axis=1)
    for got, k in ((d1, 0), (d2, 1), (d3, 2)):
        assert np.allclose(got, srt[:, k], rtol=1e-12, atol=0)
    s = 7
    ids, xv = ci[rp[s]:rp[s + 1]], vals[rp[s]:rp[s + 1]]
    Wp = W.copy()
    Wp[:, 13] = 0.0
    Wp[ids, 13] = xv
    Wp[:, 2] = Wp[:, 13]
    Wp[ids[0], 2] = xv[0] / 2
    r = oracle.bmu_sf(Wp, rp[s:s + 2], ci, vals, lib=lib)
    assert (int(r[0][0]), float(r[1][0]), int(r[2][0])) == (13, 0.0, 2)
    assert float(r[3][0]) == (float(xv[0]) / 2) ** 2
    Wt = W.copy()
    for j in (9, 2, 5):  # three exact copies of the input: ranks 2 then 5, all at distance 0
        Wt[:, j] = 0.0
        Wt[ids, j] = xv
    r = oracle.bmu_sf(Wt, rp[s:s + 2], ci, vals, lib=lib)
    assert (int(r[0][0]), int(r[2][0]), float(r[1][0]), float(r[3][0]), float(r[4][0])) == (2, 5, 0.0, 0.0, 0.0)
    r2 = oracle.bmu_sf(np.ascontiguousarray(2 * W), rp, ci, 2 * vals, lib=lib)
    assert np.array_equal(r2[0], b1) and np.array_equal(r2[2], b2)
    assert np.array_equal(r2[1], 4 * d1) and np.array_equal(r2[3], 4 * d2)


# ----------------------------------------------------------- batch update

def box3_direct(field, r, axis):
    """Three clamped, unnormalised box passes of half-width r along one axis, by direct window sums in int64."""
    f = np.asarray(field, dtype=np.int64)
    n = f.shape[axis]
    for _ in range(3):
        c = np.cumsum(f, axis=axis)
        c = np.concatenate([np.zeros_like(np.take(c, [0], axis=axis)), c], axis=axis)  # c[k] = sum of the first k
        hi = np.minimum(np.arange(n) + r + 1, n)
        lo = np.maximum(np.arange(n) - r, 0)
        f = np.take(c, hi, axis=axis) - np.take(c, lo, axis=axis)
    return f


def update_direct(W, E, rp, ci, bmu, r):
    """The update by its definition, in exact integers: counts, direct window sums (rows, then columns), fp32 quotient."""
    V, M = W.shape
    den = np.bincount(bmu, minlength=M).reshape(E, E)
    num = np.zeros((V, E, E), dtype=np.int64)
    for s in range(len(bmu)):
        for v in ci[rp[s]:rp[s + 1]]:
            num[v, bmu[s] // E, bmu[s] % E] += 1
    den_b = box3_direct(box3_direct(den, r, 1), r, 0)
    num_b = box3_direct(box3_direct(num, r, 2), r, 1)
    assert den_b.max() < 2 ** 24 and num_b.max() < 2 ** 24  # every partial sum exact in fp32 too
    q = num_b.astype(np.float32) / np.maximum(den_b, 1).astype(np.float32)[None]
    return np.where(den_b[None] > 0, q, W.reshape(V, E, E)).reshape(V, M)


def check_update_direct_windows(lib):
    """Integer counts small enough for exact fp32: the running-sum blur equals direct window sums, for several radii;
    units without a sample in reach keep their prototype."""
    E, V, N = 9, 24, 40
    rp, ci = synth.make_csr(29, N, V)
    W = synth.codebook(29, synth.UNIFORM, V, E * E)
    rng = np.random.default_rng(29)
    bmu = rng.integers(0, E * E // 3, N).astype(np.int32)  # the lower third of the lattice only
    for r in (1, 2, 4):
        got = oracle.update(W, E, rp, ci, bmu, r, lib=lib)
        ref = update_direct(W, E, rp, ci, bmu, r)
        assert np.array_equal(got, ref), f"radius {r}"
    got = oracle.update(W, E, rp, ci, bmu, 1, lib=lib)
    assert np.array_equal(got[:, -E:], W[:, -E:]), "units out of reach must keep their prototype"


def check_update_impulse_and_pair(lib):
    """One sample: its unit's neighbourhood becomes exactly its input (1 on its features, 0 elsewhere), the clamped
    support (3r cells per axis, no wrap) ends at the lattice edge. Two samples with disjoint features: the new
    prototype is each one's kernel weight over the sum."""
    E, V = 12, 10
    W = synth.codebook(30, synth.UNIFORM, V, E * E)
    rp = np.array([0, 3], dtype=np.int32)
    ci = np.array([1, 4, 7], dtype=np.int32)
    r = 1
    got = oracle.update(W, E, rp, ci, np.array([0], dtype=np.int32), r, lib=lib).reshape(V, E, E)
    reach = np.zeros((E, E), dtype=bool)
    reach[:3 * r + 1, :3 * r + 1] = True  # corner unit: support [0, 3r] on both axes
    for v in range(V):
        want = 1.0 if v in (1, 4, 7) else 0.0
        assert (got[v][reach] == want).all()
        assert np.array_equal(got[v][~reach], W.reshape(V, E, E)[v][~reach])
    rp2 = np.array([0, 2, 4], dtype=np.int32)
    ci2 = np.array([0, 2, 5, 9], dtype=np.int32)
    bmu2 = np.array([E + 1, 3 * E + 5], dtype=np.int32)  # units (1,1) and (3,5)
    got2 = oracle.update(W, E, rp2, ci2, bmu2, 2, lib=lib)
    ref2 = update_direct(W, E, rp2, ci2, bmu2, 2)
    assert np.array_equal(got2, ref2)
    k1 = update_direct(W, E, rp2[:2], ci2[:2], bmu2[:1], 2)[0]  # sample 1 alone: weight-1 field on feature 0
    assert np.allclose(got2[0][k1 == 1.0] + got2[5][k1 == 1.0], 1.0, rtol=0, atol=1e-6)


def residual_case():
    """A batch whose blurred den, summed in fp32 with running windows, keeps a residual outside the exact support:
    352,197 samples at unit (2, 5) of a 10 x 10 lattice (all holding feature 0) and 17,570 at unit (0, 7) (feature
    1), radius 1. The window sums pass 2^24, and the running sums leave den = 2 at four units of column 5 that no
    sample reaches (rows 6-9: more than 3 cells from row 2)."""
    E, r = 10, 1
    n_a, n_b = 352_197, 17_570
    bmu = np.concatenate([np.full(n_a, 2 * E + 5), np.full(n_b, 7)]).astype(np.int32)
    rp = np.arange(n_a + n_b + 1, dtype=np.int32)
    ci = np.concatenate([np.zeros(n_a), np.ones(n_b)]).astype(np.int32)
    W = (0.125 + np.arange(2 * E * E, dtype=np.float32) / 1024).astype(np.float32).reshape(2, E * E)
    return E, r, W, rp, ci, bmu


def check_update_residual_support(lib):
    """Units that no sample reaches (beyond 3r cells along either axis; exact integer arithmetic gives den = 0 there)
    keep their prototype bit for bit even where the fp32 running sums leave a residual, and every prototype stays
    in [0, 1], the range of a mean of 0/1 inputs."""
    E, r, W, rp, ci, bmu = residual_case()
    got = oracle.update(W, E, rp, ci, bmu, r, lib=lib)
    occ = np.zeros((E, E), dtype=bool)
    occ.flat[np.unique(bmu)] = True
    near = np.zeros((E, E), dtype=bool)
    for i, j in np.argwhere(occ):
        near[max(0, i - 3 * r):i + 3 * r + 1, max(0, j - 3 * r):j + 3 * r + 1] = True
    assert not near[6:, 5].any(), "the case's residual units must lie outside the support"
    assert np.array_equal(got[:, ~near.ravel()], W[:, ~near.ravel()]), "units out of reach must keep their prototype"
    assert ((got >= 0) & (got <= 1)).all()
    # every unit in reach changed: the batch moves them all away from these prototypes
    assert (got[:, near.ravel()] != W[:, near.ravel()]).all()


GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def check_update_kernel_width(lib):
    """The kernel of the update, read out of the oracle: one sample with feature 0 at the centre unit c of a
    (12r+1)^2 lattice, one sample with feature 1 at every unit. Where c's kernel reaches, every unit's all-ones
    blur is (2r+1)^6 (its whole support lies inside), so the new feature-0 weight is k/(k + (2r+1)^6) and gives back
    the integer kernel k. It must be separable, symmetric, of mass (2r+1)^6, of variance exactly r(r+1) per axis
    (three convolved uniforms on [-r, r]) -- and of the standard deviation the paper gives for three passes of
    half-width r (Section 3.4), the values in golden/box_blur_width.txt."""
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "box_blur_width.txt")) if ln.strip() and ln[0] != "#"]
    assert rows, "golden file is empty"
    for r_txt, width_txt in rows:
        r, width = int(r_txt), float(width_txt)
        E = 12 * r + 1
        M, c = E * E, 6 * r
        rp = np.arange(M + 2, dtype=np.int32)
        ci = np.array([0] + [1] * M, dtype=np.int32)
        bmu = np.array([c * E + c] + list(range(M)), dtype=np.int32)
        W = synth.codebook(31, synth.UNIFORM, 2, M)
        q = oracle.update(W, E, rp, ci, bmu, r, lib=lib)[0].reshape(E, E).astype(np.float64)
        C = float((2 * r + 1) ** 6)
        with np.errstate(divide="ignore", invalid="ignore"):  # a broken oracle may return q = 1
            k = q * C / (1.0 - q)
        kr = np.rint(k)
        assert np.isfinite(k).all() and np.abs(k - kr).max() < 1e-3, f"r={r}: feature-0 weights are not k/(k+C) of an integer kernel"
        kr = kr.astype(np.int64)
        assert (kr[np.abs(np.arange(E) - c) > 3 * r, :] == 0).all() and (kr[:, np.abs(np.arange(E) - c) > 3 * r] == 0).all()
        assert kr.sum() == (2 * r + 1) ** 6, f"r={r}: kernel mass"
        assert np.array_equal(kr, kr.T) and np.array_equal(kr, kr[::-1, ::-1]), f"r={r}: kernel symmetry"
        a = kr.sum(axis=0)
        assert np.array_equal(kr * a.sum(), np.outer(a, a)), f"r={r}: kernel not separable"
        d = np.arange(E) - c
        var2 = int((a * d * d).sum())  # var * mass, exact
        assert var2 == r * (r + 1) * int(a.sum()), f"r={r}: variance {var2 / a.sum()} != r(r+1)"
        assert abs(np.sqrt(var2 / a.sum()) - width) <= 0.1, f"r={r}: width {np.sqrt(var2 / a.sum())} vs {width}"


ALL_CHECKS = [
    check_exact_integer_direct,
    check_cdist_node_major,
    check_expanded_form,
    check_node_major_python_loop,
    check_planted_neuron,
    check_constant_codebook,
    check_tie_lowest_index,
    check_single_neuron_and_empty_row,
    check_quantisation_error,
    check_offset_rows_and_blocks,
    check_norms,
    check_error_codes,
    check_top2_exact_integer,
    check_top2_ties_and_small_maps,
    check_top2_cdist_and_top1,
    check_top2_blocks,
    check_sf_exact_integer,
    check_sf_binary_values_reduce,
    check_sf_cdist_and_planted,
    check_update_direct_windows,
    check_update_impulse_and_pair,
    check_update_kernel_width,
    check_update_residual_support,
]
