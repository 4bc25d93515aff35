"""CPU tests of the host-side measurement logic: the algorithmic-byte count the
roofline divides by, and bench.py's one-GPU contract."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("N,TA", [(1, 16), (37, 16), (1000, 16), (1003, 8), (250, 1), (64, 32)])
def test_tile_distinct_matches_brute_force(N, TA):
    """Distinct ids per group of TA consecutive rows, the unit of the algorithmic bytes (4*M per distinct id),
    against numpy's unique on each group; the last group is ragged."""
    rp, ci = synth.make_csr(17 + N, N, 3000)
    got = synth.tile_distinct(rp, ci, TA)
    want = [np.unique(ci[rp[t]:rp[min(N, t + TA)]]).size for t in range(0, N, TA)]
    assert np.array_equal(got, np.array(want, dtype=np.int32))
    if TA == 1:
        assert np.array_equal(got, np.diff(rp))  # ids are distinct within a row


def test_tile_distinct_rows_per_sample_at_full_vocabulary():
    """The 64x64 workload's statistics on a 200,000-row prefix: about 8.1 distinct ids per sample in 16-row tiles
    (of 12.0 ids per row), so the algorithmic bytes are ~68% of a per-sample gather's."""
    cfg = synth.CONFIGS["64"]
    N = 200_000
    rp, ci = synth.make_csr(cfg.seed, N, cfg.V, cfg.lam, cfg.zipf_s)
    per_sample = synth.tile_distinct(rp, ci, 16).astype(np.int64).sum() / N
    assert 11.8 < rp[-1] / N < 12.2
    assert 7.9 < per_sample < 8.4, per_sample


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus"] == 2 and "one GPU" in msg["error"]
