"""The native plan execution and baseline placements (fate_simulate,
fate_place_baseline, host code in libfate) against the plan-execution oracle
on the same inputs (no GPU): placements identical, integer metrics equal,
times within 1e-12 relative."""

import dataclasses

import numpy as np
import pytest

import sim_pins
from oracle import simulate as S
from paper_2605_07238_amd import fate, synth


def _pending_completed(w):
    """The execution model knows pending and completed stages only: running
    and committed ones become pending."""
    return dataclasses.replace(w, status=np.where(w.status == 1, 1, 0).astype(np.uint8))


def _compare(got, want):
    for k in ("tasks", "xdev_edges", "cache_hits", "model_cont"):
        assert np.array_equal(got[k], want[k]), k
    for k in ("makespan", "p95"):
        assert np.allclose(got[k], want[k], rtol=1e-12, atol=0), (k, np.abs(got[k] - want[k]).max())


MAKERS = [
    ("hand", lambda: sim_pins._w()),
    ("d4", lambda: synth.make_random_small(3, B=3, n=24, D=4, M=3, K=2, max_shard=3, shard_frac=0.5)),
    ("d8-tight", lambda: synth.make_random_small(4, B=3, n=30, D=8, M=5, K=3, tight_caps=True)),
    ("d16", lambda: synth.make_random_small(5, B=2, n=30, D=16, M=6, K=4, p_edge=0.4)),
    ("layered", lambda: synth.make_workload("layered-1024x200-d8", B=3)),
    ("forkjoin", lambda: synth.make_workload("forkjoin-4096x1000-d16", B=2)),
    ("shards", lambda: synth.make_workload("shards-1024x500-d16", B=2)),
]


@pytest.mark.parametrize("policy", [fate.FATE_PLACE_ROUND_ROBIN, fate.FATE_PLACE_HEFT], ids=["rr", "heft"])
@pytest.mark.parametrize("name,make", MAKERS, ids=[m[0] for m in MAKERS])
def test_baseline_placement_and_execution(name, make, policy):
    w = _pending_completed(make())
    dev, order = fate.fate_place_baseline(w, policy)
    wdev, word = (S.place_round_robin(w) if policy == fate.FATE_PLACE_ROUND_ROBIN else S.place_heft(w))
    assert np.array_equal(dev, wdev) and np.array_equal(order, word)
    _compare(fate.fate_simulate(w, dev, order), S.simulate(w, wdev, word))


@pytest.mark.parametrize("seed", range(4))
def test_random_plans_with_windows(seed):
    """Random placements with windows and a random topological order key."""
    w = _pending_completed(synth.make_random_small(20 + seed, B=3, n=24, D=6, M=4, K=2, max_shard=3,
                                                   shard_frac=0.6))
    rng = np.random.default_rng(seed)
    dev = np.zeros(w.N, np.uint64)
    for g in range(w.N):
        if w.status[g] == 1:
            continue
        feas = [d for d in range(w.D) if (int(w.elig[g]) >> d) & 1 and w.weight_bytes[w.model[g]] <= w.cap_bytes[d]]
        k = int(rng.integers(1, 4))
        starts = [i for i in range(w.D - k + 1) if all(d in feas for d in range(i, i + k))]
        if k > 1 and starts:
            i = int(rng.choice(starts))
            dev[g] = np.uint64(((1 << k) - 1) << i)
        else:
            dev[g] = np.uint64(1 << int(rng.choice(feas)))
    # a key that respects the DAG: depth from the sources plus noise below 1
    order = np.zeros(w.N, np.int64)
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        depth = np.zeros(hi - lo, np.int64)
        for v in range(hi - lo):
            ps = w.par_idx[w.par_off[lo + v]:w.par_off[lo + v + 1]]
            depth[v] = 1 + max((depth[int(p)] for p in ps), default=-1)
        order[lo:hi] = depth * 1000 + rng.integers(0, 1000, size=hi - lo)
    _compare(fate.fate_simulate(w, dev, order), S.simulate(w, dev, order))


def test_simulate_errors():
    w = sim_pins._w()
    dev = np.array([0, 2, 1, 1], np.uint64)
    with pytest.raises(fate.FateError) as e:  # v2 before its parent v1
        fate.fate_simulate(w, dev, np.array([0, 5, 1, 0], np.int64))
    assert e.value.status == fate.FATE_ESTATE
    with pytest.raises(fate.FateError) as e:  # a device past D
        fate.fate_simulate(w, np.array([0, 4, 1, 1], np.uint64), np.zeros(4, np.int64))
    assert e.value.status == fate.FATE_EINVAL
    with pytest.raises(fate.FateError) as e:  # running stages are not part of the execution model
        fate.fate_simulate(dataclasses.replace(w, status=np.array([1, 2, 0, 0], np.uint8)), dev, np.zeros(4, np.int64))
    assert e.value.status == fate.FATE_ESTATE
    with pytest.raises(fate.FateError) as e:
        fate.fate_place_baseline(w, 7)
    assert e.value.status == fate.FATE_EINVAL


def _oracle_fate_plan(w, k=4, max_waves=200):
    """A FATE plan built by the oracle alone: score, top-k, one planning wave,
    commit, until the frontier is empty.  Returns (devices, order) with the
    wave number as the order key (commit order within a wave is by stage id)."""
    from oracle import oracle
    devices = np.zeros(w.N, np.uint64)
    order = np.zeros(w.N, np.int64)
    cur = w
    fin = None
    for wave in range(max_waves):
        ref = oracle.score(cur)
        if len(ref["front_v"]) == 0:
            return devices, order, wave
        idx, val = oracle.topk(ref, k)
        _, _, f_off = oracle.frontier(cur)
        sel, n = oracle.plan_wave(cur.D, f_off, np.diff(ref["cand_off"]), idx, val.astype(np.float32))
        assert n > 0
        nxt, _, rej, fin = oracle.commit(cur, sel, fin=fin)
        assert rej == 0
        for f in np.nonzero(sel >= 0)[0]:
            g = int(cur.stage_off[ref["front_b"][f]]) + int(ref["front_v"][f])
            devices[g] = nxt.holders[g]
            order[g] = wave
        cur = nxt
    raise AssertionError("the plan did not finish")


@pytest.mark.parametrize("seed", range(3))
def test_fate_plan_executes_alike(seed):
    """A FATE plan from the oracle's own planning loop runs through both
    executions alike, and every pending stage is placed."""
    w = _pending_completed(synth.make_random_small(40 + seed, B=3, n=24, D=5, M=4, K=2, max_shard=3,
                                                   shard_frac=0.4, p_edge=0.3))
    dev, order, waves = _oracle_fate_plan(w)
    assert waves > 1
    assert np.all((dev != 0) == (w.status == 0))
    got = fate.fate_simulate(w, dev, order)
    _compare(got, S.simulate(w, dev, order))
    assert np.array_equal(got["tasks"], np.array([np.count_nonzero(w.status[int(w.stage_off[b]):int(w.stage_off[b + 1])] == 0)
                                                  for b in range(w.B)]))
