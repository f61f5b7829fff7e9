"""The row kernels (frontiers of single-device candidates, uniform beta, no
variant) against the oracle on shapes that reach their edge cases: k_rows,
one row per lane, in every device-count class (4, 8 and 16 lanes, including
D = 1, 2, 3, 5 and 9), no prefix slots and the most prefix slots, more
completed parents than lanes in a group, instances whose frontier spans
several 128-stage chunks, a parameter set's horizon below the packed one, and
top-k above the one-lane ranking (the group ranks then); k_rows4, one row per
four lanes, for 17 to 64 devices (quads whose upper lanes hold no device,
the largest tables, several chunks, dense parents, top-k up to 64)."""

import numpy as np
import pytest

from gpu_util import check_against_oracle, run_gpu
from paper_2605_07238_amd import synth

pytestmark = pytest.mark.gpu


def _rows_workload(seed, **kw):
    args = dict(B=3, n=40, H=3, max_shard=1, shard_frac=0.0, uniform_beta=True, p_edge=0.25)
    args.update(kw)
    return synth.make_random_small(seed, **args)


@pytest.mark.parametrize("seed,kw", [
    (1, dict(D=1, M=2, K=2)),
    (2, dict(D=2, M=3, K=0)),
    (3, dict(D=3, M=3, K=1)),
    (4, dict(D=4, M=3, K=4)),
    (5, dict(D=5, M=4, K=8)),
    (6, dict(D=8, M=6, K=32)),
    (7, dict(D=9, M=5, K=3)),
    (8, dict(D=16, M=12, K=16)),
    (9, dict(D=16, M=32, K=32)),
], ids=["d1", "d2-k0", "d3", "d4", "d5", "d8-k32", "d9", "d16", "d16-m32"])
def test_rows_random(seed, kw):
    w = _rows_workload(seed, **kw)
    print("[rows] random", seed, kw, flush=True)
    check_against_oracle(w, run_gpu(w, k=4), k=4)


def test_rows_dense_parents():
    """Up to five completed parents per stage on 4-lane groups."""
    w = _rows_workload(11, D=4, M=3, K=4, n=30, p_edge=0.7)
    print("[rows] dense parents", flush=True)
    check_against_oracle(w, run_gpu(w, k=4), k=4)


def test_rows_several_chunks():
    """Instances whose frontier holds more than 128 stages."""
    w = _rows_workload(12, B=2, n=700, D=16, M=6, K=4, p_edge=0.003)
    g = run_gpu(w, k=4)
    per_inst = np.bincount(np.searchsorted(w.stage_off, g["flat_v"], side="right") - 1, minlength=w.B)
    print("[rows] several chunks, frontier per instance", per_inst.tolist(), flush=True)
    assert per_inst.max() > 128
    check_against_oracle(w, g, k=4)


@pytest.mark.parametrize("H", [0, 1, 2])
def test_rows_horizon_below_packed(H):
    """The descendant lists are packed for H = 3; a parameter set with a
    smaller H takes the prefix of each list within its horizon."""
    w = _rows_workload(13, D=8, M=5, K=4, n=60, p_edge=0.2)
    print("[rows] H", H, "packed 3", flush=True)
    check_against_oracle(w, run_gpu(w, H=H, pack_H=3, k=4), H=H, k=4)


@pytest.mark.parametrize("k", [5, 16, 64])
def test_rows_topk_above_lane_ranking(k):
    w = _rows_workload(14, D=16, M=6, K=4, n=50)
    print("[rows] k", k, flush=True)
    check_against_oracle(w, run_gpu(w, k=k), k=k)


@pytest.mark.parametrize("seed,kw", [
    (21, dict(D=17, M=5, K=4)),
    (22, dict(D=24, M=8, K=2)),
    (23, dict(D=33, M=12, K=8)),
    (24, dict(D=48, M=20, K=16)),
    (25, dict(D=64, M=32, K=16)),
    (26, dict(D=64, M=40, K=0)),
    (27, dict(D=50, M=64, K=4)),
], ids=["d17", "d24", "d33", "d48", "d64", "d64-k0", "d50-m64"])
def test_rows4_random(seed, kw):
    w = _rows_workload(seed, **kw)
    print("[rows4] random", seed, kw, flush=True)
    check_against_oracle(w, run_gpu(w, k=4), k=4)


def test_rows4_dense_parents_and_chunks():
    """Up to five completed parents per stage, and instances of more than 128
    frontier stages, on 64 devices."""
    w = _rows_workload(31, B=2, n=600, D=64, M=16, K=8, p_edge=0.004)
    g = run_gpu(w, k=4)
    per_inst = np.bincount(np.searchsorted(w.stage_off, g["flat_v"], side="right") - 1, minlength=w.B)
    print("[rows4] several chunks, frontier per instance", per_inst.tolist(), flush=True)
    assert per_inst.max() > 128
    check_against_oracle(w, g, k=4)
    w = _rows_workload(32, D=40, M=6, K=4, n=30, p_edge=0.7)
    print("[rows4] dense parents", flush=True)
    check_against_oracle(w, run_gpu(w, k=4), k=4)


@pytest.mark.parametrize("H", [0, 2])
def test_rows4_horizon_below_packed(H):
    w = _rows_workload(33, D=36, M=5, K=4, n=60, p_edge=0.2)
    print("[rows4] H", H, "packed 3", flush=True)
    check_against_oracle(w, run_gpu(w, H=H, pack_H=3, k=4), H=H, k=4)


@pytest.mark.parametrize("k", [1, 16, 64])
def test_rows4_topk(k):
    w = _rows_workload(34, D=64, M=6, K=4, n=50)
    print("[rows4] k", k, flush=True)
    check_against_oracle(w, run_gpu(w, k=k), k=k)
