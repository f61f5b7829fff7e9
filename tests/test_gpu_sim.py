"""Plan execution and baseline placements on the GPU (fate_simulate_device,
fate_place_baseline_device) against the plan-execution oracle on the same
inputs: placements identical, integer metrics equal, times within 1e-12
relative of the oracle and bit for bit equal to the host executor (the same
fp64 operations in the same order).  The plans are the oracle's baselines,
random plans with windows, and the plan that the device planning loop builds
(score, top-k, planning wave, commit, until the frontier is empty)."""

import dataclasses

import numpy as np
import pytest

import sim_pins
from oracle import simulate as S
from paper_2605_07238_amd import fate, synth

pytestmark = pytest.mark.gpu


def _pending_completed(w):
    """The execution model knows pending and completed stages only: running
    and committed ones become pending."""
    return dataclasses.replace(w, status=np.where(w.status == 1, 1, 0).astype(np.uint8))


def _compare(got, want, host=None):
    for k in ("tasks", "xdev_edges", "cache_hits", "model_cont"):
        assert np.array_equal(got[k], want[k]), (k, got[k], want[k])
    for k in ("makespan", "p95"):
        assert np.allclose(got[k], want[k], rtol=1e-12, atol=0), (k, np.abs(got[k] - want[k]).max())
        if host is not None:
            assert np.array_equal(got[k].view(np.uint64), host[k].view(np.uint64)), (k, got[k] - host[k])


def _packed(w):
    pk = fate.fate_pack_dags(w)
    return pk, fate.fate_pack_state(pk, w)


def _run_device(w, pk, st, dev, order):
    import torch
    d = torch.from_numpy(np.ascontiguousarray(dev, np.uint64).view(np.int64)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(order, np.int64)).cuda()
    return fate.fate_simulate_device(pk, st, d, o, w.params["kappa_prefix"])


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
def test_device_baselines(name, make, policy):
    w = _pending_completed(make())
    pk, st = _packed(w)
    print("[sim] baseline", name, policy, flush=True)
    dt, ot = fate.fate_place_baseline_device(pk, st, policy, w.params["kappa_prefix"])
    dev = dt.cpu().numpy().view(np.uint64)
    order = ot.cpu().numpy()
    wdev, word = (S.place_round_robin(w) if policy == fate.FATE_PLACE_ROUND_ROBIN else S.place_heft(w))
    assert np.array_equal(dev, wdev), "placement differs"
    assert np.array_equal(order, word), "order differs"
    got = fate.fate_simulate_device(pk, st, dt, ot, w.params["kappa_prefix"])
    _compare(got, S.simulate(w, wdev, word), fate.fate_simulate(w, wdev, word))


@pytest.mark.parametrize("seed", range(4))
def test_device_random_plans_with_windows(seed):
    """Random placements with windows and a random key that respects the DAG."""
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
            dev[g] = np.uint64(((1 << k) - 1) << int(rng.choice(starts)))
        else:
            dev[g] = np.uint64(1 << int(rng.choice(feas)))
    order = np.zeros(w.N, np.int64)
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        depth = np.zeros(hi - lo, np.int64)
        for v in range(hi - lo):
            ps = w.par_idx[w.par_off[lo + v]:w.par_off[lo + v + 1]]
            depth[v] = 1 + max((depth[int(p)] for p in ps), default=-1)
        # negative keys too: the order key is a signed integer
        order[lo:hi] = depth * 1000 + rng.integers(0, 1000, size=hi - lo) - 5000
    pk, st = _packed(w)
    print("[sim] random plan", seed, flush=True)
    _compare(_run_device(w, pk, st, dev, order), S.simulate(w, dev, order), fate.fate_simulate(w, dev, order))


def device_fate_plan(w, k=4, max_waves=2000):
    """The FATE plan the device planning loop builds: each placed stage's
    devices (its holders in the planning state) and the wave it was placed
    in (commit order within a wave is by stage id)."""
    import torch
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    params = fate.make_params(w)
    cap = max(1, st.n_frontier)
    scores = torch.empty(max(1, st.n_cand), dtype=torch.float32, device="cuda")
    idx = torch.empty((cap, k), dtype=torch.int32, device="cuda")
    val = torch.empty((cap, k), dtype=torch.float32, device="cuda")
    sel = torch.empty(cap, dtype=torch.int32, device="cuda")
    wave_of = np.full(w.N, -1, np.int64)
    waves = 0
    while waves < max_waves:
        nF = st.counts()[0]
        if nF == 0:
            break
        fate.fate_score_frontier(pk, st, params, out=scores)
        fate.fate_topk(st, scores, k, idx=idx, val=val)
        fate.fate_plan_wave(st, idx, val, sel=sel)
        fv, _, _ = fate.frontier_table(st)
        s_host = sel[:nF].cpu().numpy()
        assert (s_host >= 0).any(), "a planning wave placed nothing"
        wave_of[fv[s_host >= 0]] = waves
        fate.fate_commit_advance(pk, st, sel)
        waves += 1
    assert waves < max_waves
    holders = fate.state_arrays(st)["holders"]
    return np.where(wave_of >= 0, holders, 0).astype(np.uint64), np.maximum(wave_of, 0), waves


@pytest.mark.parametrize("name,make", MAKERS[1:], ids=[m[0] for m in MAKERS[1:]])
def test_device_fate_plan(name, make):
    """The plan built by the device planning loop runs alike on the device,
    on the host and in the oracle, and places every pending stage."""
    w = _pending_completed(make())
    print("[sim] device FATE plan", name, flush=True)
    dev, order, waves = device_fate_plan(w)
    assert np.all((dev != 0) == (w.status == 0))
    pk, st = _packed(w)
    got = _run_device(w, pk, st, dev, order)
    _compare(got, S.simulate(w, dev, order), fate.fate_simulate(w, dev, order))
    tasks = [np.count_nonzero(w.status[int(w.stage_off[b]):int(w.stage_off[b + 1])] == 0) for b in range(w.B)]
    assert np.array_equal(got["tasks"], np.array(tasks))


def test_device_simulate_errors():
    """Errors in the device arrays come back per instance."""
    w = sim_pins._w()
    pk, st = _packed(w)
    with pytest.raises(fate.FateError) as e:  # v2 before its parent v1
        _run_device(w, pk, st, np.array([0, 2, 1, 1], np.uint64), np.array([0, 5, 1, 0], np.int64))
    assert e.value.status == fate.FATE_ESTATE
    with pytest.raises(fate.FateError) as e:  # a device past D
        _run_device(w, pk, st, np.array([0, 4, 1, 1], np.uint64), np.zeros(4, np.int64))
    assert e.value.status == fate.FATE_EINVAL
    with pytest.raises(fate.FateError) as e:
        fate.fate_place_baseline_device(pk, st, 7, 1e-4)
    assert e.value.status == fate.FATE_EINVAL
    # a stage left unplaced is not run, and the rest still runs
    got = _run_device(w, pk, st, np.array([0, 2, 1, 0], np.uint64), np.array([0, 0, 1, 0], np.int64))
    want = S.simulate(w, np.array([0, 2, 1, 0], np.uint64), np.array([0, 0, 1, 0], np.int64))
    _compare(got, want)


def test_device_full_batch_forkjoin():
    """Every instance of the 16-device fork-join batch: the HEFT-style
    placement and its execution against the host executor (the oracle's
    Python loops would take minutes at this size)."""
    w = _pending_completed(synth.make_workload("forkjoin-4096x1000-d16", B=512))
    pk, st = _packed(w)
    print("[sim] fork-join B=512 HEFT", flush=True)
    dt, ot = fate.fate_place_baseline_device(pk, st, fate.FATE_PLACE_HEFT, w.params["kappa_prefix"])
    hdev, hord = fate.fate_place_baseline(w, fate.FATE_PLACE_HEFT)
    assert np.array_equal(dt.cpu().numpy().view(np.uint64), hdev)
    assert np.array_equal(ot.cpu().numpy(), hord)
    got = fate.fate_simulate_device(pk, st, dt, ot, w.params["kappa_prefix"])
    host = fate.fate_simulate(w, hdev, hord)
    for k in got:
        assert np.array_equal(got[k], host[k]), k
