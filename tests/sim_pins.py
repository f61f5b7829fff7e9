"""Pins of the plan-execution oracle (oracle/simulate.py) against values
worked out by hand and against closed forms and invariants."""

from __future__ import annotations

import dataclasses

import numpy as np

import builders
from oracle import simulate as S
from paper_2605_07238_amd import synth

# D = 2, both models fit everywhere (10 GB each, 25 GB capacity).
# exec m0 = [1, 2], m1 = [0.5, 0.5]; switch m0 0.25, m1 0.5; beta 2^-30 off the
# diagonal; kappa_prefix 2^-10.  Stage 0 (m0) completed on d0 with 2^30
# bytes; 1 (m0, grp 7, L 1024, 2^31 bytes) after 0; 2 (m1, grp 7, L 512)
# after 1; 3 (m1) alone.  t0 = 1, tau = [1, 1.5], d0 holds m0, d1 nothing;
# d1 caches grp 7.
SIM_SPEC = dict(D=2, M=2, K=1, exec=[[1.0, 2.0], [0.5, 0.5]], switch_s=[[0.25, 0.25], [0.5, 0.5]],
                weight_gb=[10, 10], cap_gb=[25, 25], beta=[[0.0, 2.0 ** -30], [2.0 ** -30, 0.0]],
                instances=[dict(parents=[[], [0], [1], []], model=[0, 0, 1, 1], elig=[3, 3, 3, 3],
                                prefix_hash=[0, 7, 7, 0], prefix_tokens=[0.0, 1024.0, 512.0, 0.0],
                                out_bytes=[2.0 ** 30, 2.0 ** 31, 1.0, 1.0], status=[1, 0, 0, 0],
                                holders=[1, 0, 0, 0], resident=[1, 0], prefix_cache=[[0], [7]],
                                tau_free=[1.0, 1.5], t_now=1.0)])
KPF = 2.0 ** -10


def _w():
    return builders.from_spec(SIM_SPEC, H=1, params=dict(kappa_prefix=KPF))


def check_sim_hand():
    """v1 on d1 (order 0), v3 on d0 (1), v2 on d0 (2):
    v1: parent output 2^30 * 2^-30 = 1 -> ready 2; start max(1.5, 2) = 2;
        switch 0.25; grp 7 cached on d1: run 2 - 1 = 1 -> 3.25 (hit, 1 x-dev edge)
    v3: start 1; switch 0.5 (m1 absent); run 0.5 -> 2.0
    v2: v1's 2^31 bytes * 2^-30 -> ready 5.25; m1 resident (no switch); d0 had
        no grp 7: run 0.5 -> 5.75; d0 ran m1 just before (continuation); x-dev
    makespan 4.75; sinks v2, v3 at 4.75, 1.0 -> p95 4.75."""
    w = _w()
    dev = np.array([0, 2, 1, 1], np.uint64)
    order = np.array([0, 0, 2, 1], np.int64)
    r = S.simulate(w, dev, order)
    assert r["tasks"].tolist() == [3]
    assert r["makespan"].tolist() == [4.75]
    assert r["p95"].tolist() == [4.75]
    assert r["xdev_edges"].tolist() == [2]
    assert r["cache_hits"].tolist() == [1]
    assert r["model_cont"].tolist() == [1]


def check_round_robin_hand():
    """Pending stages 1, 2, 3 in id order go to d0, d1, d0."""
    dev, order = S.place_round_robin(_w())
    assert dev.tolist() == [0, 1, 2, 1] and order.tolist() == [0, 1, 2, 3]


def check_heft_hand():
    """Upward ranks: v1 = 1.5 + (2^31 * 2^-30 + 0.5) = 4, v2 = v3 = 0.5 (v2 first
    by id).  v1: EFT d0 = 2.0 (d1 3.25) -> d0.  v2: d0: ready 2, switch 0.5,
    grp 7 now cached on d0, run 0.5 - 0.5 = 0 -> 2.5; d1: ready 4 -> 4.5 -> d0.
    v3: d0 3.0, d1 1.5 + 0.5 + 0.5 = 2.5 -> d1.  Executed: makespan 1.5."""
    w = _w()
    dev, order = S.place_heft(w)
    assert dev.tolist() == [0, 1, 1, 2] and order.tolist() == [0, 0, 1, 2]
    r = S.simulate(w, dev, order)
    assert r["makespan"].tolist() == [1.5]


def check_single_device_sum(seed: int):
    """One device, no transfer cost, no prefix benefit: the device runs every
    pending stage back to back, so makespan = (tau - t0)^+ + sum of switch and
    runtime, with switches exactly where the Load rule says."""
    w = synth.make_random_small(seed, B=2, n=12, D=1, M=3, K=2, max_shard=1, tight_caps=False)
    w = dataclasses.replace(w, beta=np.zeros_like(w.beta), status=np.where(w.status == 1, 1, 0).astype(np.uint8))
    dev = np.where(w.status == 1, 0, 1).astype(np.uint64)
    order = np.arange(w.N, dtype=np.int64)
    r = S.simulate(w, dev, order, kappa_prefix=0.0)
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        t0 = float(np.float32(w.t_now[b]))
        t = max(float(np.float32(w.tau_free[b, 0])), t0)
        res = int(w.resident[b, 0])
        for g in range(lo, hi):
            if w.status[g] == 1:
                continue
            m = int(w.model[g])
            if not (res >> m) & 1:
                t += float(w.switch_s[m, 0])
                res |= 1 << m
                tot = sum(int(w.weight_bytes[i]) for i in range(w.M) if (res >> i) & 1)
                for i in range(w.M):
                    if tot <= int(w.cap_bytes[0]):
                        break
                    if i != m and (res >> i) & 1:
                        res &= ~(1 << i)
                        tot -= int(w.weight_bytes[i])
            t += float(w.exec[m, 0])
        assert abs(r["makespan"][b] - (t - t0)) <= 1e-12 * max(1.0, t), (b, r["makespan"][b], t - t0)


def check_lower_bounds(seed: int):
    """Every plan's makespan is at least the longest pending chain of minimal
    runtimes (switches, transfers and waits only add; the prefix benefit is
    off), and round robin uses each device in turn."""
    w = synth.make_random_small(seed, B=3, n=16, D=4, M=3, K=2, max_shard=1)
    w = dataclasses.replace(w, status=np.where(w.status == 1, 1, 0).astype(np.uint8))
    for dev, order in (S.place_round_robin(w), S.place_heft(w, kappa_prefix=0.0)):
        r = S.simulate(w, dev, order, kappa_prefix=0.0)
        for b in range(w.B):
            lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
            best = {}
            for v in range(hi - lo):
                g = lo + v
                if w.status[g] == 1:
                    best[v] = 0.0
                    continue
                cmin = min(float(w.exec[w.model[g], d]) for d in range(w.D)
                           if (int(w.elig[g]) >> d) & 1 and w.weight_bytes[w.model[g]] <= w.cap_bytes[d])
                ps = w.par_idx[w.par_off[g]:w.par_off[g + 1]]
                best[v] = cmin + max((best[int(p)] for p in ps), default=0.0)
            assert r["makespan"][b] >= max(best.values()) - 1e-12, b
            assert r["tasks"][b] == int(np.count_nonzero(w.status[lo:hi] != 1))


def check_window_hand():
    """v1 on the window {d0, d1} (k = 2), then v3 on d1 and v2 on d0:
    v1: d0: parent local, start 1, no switch, no hit (d0 has no grp 7),
            run 1/2 -> 1.5;
        d1: transfer 2^30 * 2^-30 / 2 = 0.5 -> ready 1.5, start max(1.5, 1.5),
            switch 0.25, grp 7 cached: run max(0, 2/2 - 1/2) = 0.5 -> 2.25
        finish 2.25 on {d0, d1}; first device d0: no hit, no continuation
    v3 (order 1) on d1: start 2.25, switch 0.5, run 0.5 -> 3.25
    v2 (order 2) on d0: v1's output is local; start max(1.5, 2.25) = 2.25;
        switch 0.5; grp 7 now cached on d0 (pushed by v1): run
        max(0, 0.5 - 0.5) = 0 -> 2.75; d0 ran m0 before: no continuation
    makespan 3.25 - 1 = 2.25; sinks v2, v3 -> p95 2.25; no cross-device edge
    (v1 runs on d0, which holds stage 0's output); one hit (v2)."""
    w = _w()
    dev = np.array([0, 3, 1, 2], np.uint64)
    order = np.array([0, 0, 2, 1], np.int64)
    r = S.simulate(w, dev, order)
    assert r["makespan"].tolist() == [2.25], r["makespan"]
    assert r["p95"].tolist() == [2.25]
    assert r["xdev_edges"].tolist() == [0]
    assert r["cache_hits"].tolist() == [1]
    assert r["model_cont"].tolist() == [0]


def check_ring_drops_oldest():
    """One device, K = 2 slots holding [5, 6].  a (grp 7) makes them [6, 7]
    (5, the oldest, is dropped); b (grp 5) misses and makes them [7, 5]; c
    (grp 6) misses too.  Runtimes 1 each -> makespan 3, no hit.  (Dropping
    the newest instead would give [5, 7], a hit for b and makespan 2.5.)"""
    spec = dict(D=1, M=1, K=2, exec=[[1.0]], switch_s=[[0.0]], weight_gb=[10], cap_gb=[20], beta=[[0.0]],
                instances=[dict(parents=[[], [0], [1]], model=[0, 0, 0], elig=[1, 1, 1],
                                prefix_hash=[7, 5, 6], prefix_tokens=[512.0] * 3, out_bytes=[1.0] * 3,
                                status=[0, 0, 0], holders=[0, 0, 0], resident=[1], prefix_cache=[[5, 6]],
                                tau_free=[0.0], t_now=0.0)])
    w = builders.from_spec(spec, H=1, params=dict(kappa_prefix=KPF))
    r = S.simulate(w, np.ones(3, np.uint64), np.arange(3, dtype=np.int64))
    assert r["cache_hits"].tolist() == [0] and r["makespan"].tolist() == [3.0], r


def check_p95_chain_and_antichain():
    """A chain has one sink, so p95 = makespan; stages without edges are all
    sinks, so p95 is the nearest-rank 95th percentile of all finishes."""
    n = 25
    for parents, want in (([[]] + [[v - 1] for v in range(1, n)], "chain"), ([[]] * n, "flat")):
        spec = dict(D=1, M=1, K=1, exec=[[1.0]], switch_s=[[0.0]], weight_gb=[10], cap_gb=[20], beta=[[0.0]],
                    instances=[dict(parents=parents, model=[0] * n, elig=[1] * n, out_bytes=[1.0] * n,
                                    status=[0] * n, holders=[0] * n, resident=[1], tau_free=[0.0], t_now=0.0)])
        w = builders.from_spec(spec, H=1)
        r = S.simulate(w, np.ones(n, np.uint64), np.arange(n, dtype=np.int64))
        # one device runs them back to back: finishes 1, 2, ..., 25
        assert r["makespan"].tolist() == [25.0]
        assert r["p95"].tolist() == ([25.0] if want == "chain" else [24.0]), (want, r["p95"])


def check_order_must_respect_dag():
    w = _w()
    dev = np.array([0, 2, 1, 1], np.uint64)
    try:
        S.simulate(w, dev, np.array([0, 5, 1, 0], np.int64))  # v2 before its parent v1
    except ValueError:
        return
    raise AssertionError("an order that runs a stage before its parent must be rejected")


ALL = ([("sim_hand", check_sim_hand), ("window_hand", check_window_hand), ("round_robin_hand", check_round_robin_hand), ("heft_hand", check_heft_hand),
        ("order_rejected", check_order_must_respect_dag), ("ring_drops_oldest", check_ring_drops_oldest),
        ("p95_chain", check_p95_chain_and_antichain)]
       + [("single_device_sum:%d" % s, (lambda s: lambda: check_single_device_sum(s))(s)) for s in range(3)]
       + [("lower_bounds:%d" % s, (lambda s: lambda: check_lower_bounds(s))(s)) for s in range(3)])
