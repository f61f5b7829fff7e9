"""Checks that pin the fp64 oracle to the paper and to mathematics.

Each ``check_*`` function raises AssertionError on a mismatch and takes an
optional oracle library handle, so the same checks run against the real
oracle (tests/test_oracle_pins.py) and against copies of it with a planted
mistake (tests/test_oracle_mutants.py), which they must reject.

Kinds of pins used here:
* hand-derived values for small scenarios (tests/scenarios.py) and for the
  worked example in tests/golden/worked_example.json;
* closed-form reductions computed with numpy and scipy's breadth-first
  shortest paths (only base runtimes, or only waiting costs, switched on);
* invariants: device relabelling, H = 0 equals gamma = 0, stages outside the
  horizon do not matter, an added isolated stage changes nothing else;
* the magnitude A that every parity tolerance divides by: hand-derived values,
  A >= |Psi|, and A = |Psi| exactly when no benefit term enters;
* an independent brute-force evaluation (tests/brute.py): materialised
  post-states, costs from scratch, joint enumeration of the horizon stages'
  placements, and the GPU kernel's outside / inside rearrangement.
"""

from __future__ import annotations

import dataclasses
import json
import os

import numpy as np
import scipy.sparse as sp
from scipy.sparse.csgraph import shortest_path

import brute
import builders
import scenarios
from oracle import oracle
from paper_2605_07238_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _close(a, b, rtol=1e-12, atol=1e-12):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    inf_a, inf_b = np.isinf(a), np.isinf(b)
    assert np.array_equal(inf_a, inf_b) and np.array_equal(a[inf_a], b[inf_b]), (a, b)
    fa, fb = a[~inf_a], b[~inf_b]
    assert np.allclose(fa, fb, rtol=rtol, atol=atol), (fa, fb, np.abs(fa - fb).max() if fa.size else 0)


def check_scenario(name: str, lib=None):
    sc = scenarios.ALL[name]
    w = builders.from_spec(sc["spec"], H=sc["H"], params=sc["params"])
    r = oracle.score(w, lib=lib)
    assert list(r["front_v"]) == sc["front_v"], (list(r["front_v"]), sc["front_v"])
    _close(r["psi"], sc["psi"], rtol=1e-12)
    if "mag" in sc:
        _close(r["mag"], sc["mag"], rtol=1e-12)
    if "topk3" in sc:
        idx, _ = oracle.topk(r, 3, lib=lib)
        assert idx[0].tolist() == sc["topk3"], idx
    if "topk4" in sc:
        idx, val = oracle.topk(r, 4, lib=lib)
        assert idx.tolist() == sc["topk4"], idx


def check_worked_example(lib=None):
    spec = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    for key, H in (("H1", 1), ("H0", 0)):
        exp = spec["expected"][key]
        w = builders.from_spec(spec, H=H)
        r = oracle.score(w, lib=lib)
        assert list(r["front_v"]) == exp["front_v"]
        # inputs such as 1.1 s are float32-rounded, hence 1e-6
        _close(r["psi"], exp["psi"], rtol=1e-6, atol=0)
        _close(r["mag"], exp["mag"], rtol=1e-6, atol=0)
        idx, _ = oracle.topk(r, 3, lib=lib)
        assert idx[0].tolist() == exp["topk3"], idx


# ---------------------------------------------------------------------------
# closed-form reductions
# ---------------------------------------------------------------------------

def _frontier(w, b):
    lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
    out = []
    for v in range(hi - lo):
        g = lo + v
        ps = w.par_idx[w.par_off[g]:w.par_off[g + 1]]
        if w.status[g] == 0 and all(w.status[lo + p] == 1 for p in ps):
            out.append(v)
    return out


def _windows(D, r):
    c = [(i, 1) for i in range(D)]
    for k in range(2, r + 1):
        c += [(i, k) for i in range(D - k + 1)]
    return c


def _feasible(w, g, d):
    m = int(w.model[g])
    return bool((int(w.elig[g]) >> d) & 1) and w.weight_bytes[m] <= w.cap_bytes[d]


def check_exec_only_reduction(seed: int, lib=None, H: int = 3):
    """With every weight but the base runtime at zero, the score is
    -(max_{d in S} c(v,d)/|S| + sum_h gamma^h sum_{dist(v,w)=h} min_feasible c(w,.)).
    Hop distances come from scipy's unweighted shortest paths."""
    w = synth.make_random_small(seed, B=2, n=14, D=4, M=3, K=2, H=H, max_shard=3)
    zero = dict(lam_q=0.0, lam_s=0.0, lam_tr=0.0, lam_c=0.0, lam_p=0.0, gamma=0.5)
    r = oracle.score(w, params=zero, lib=lib)
    gam = oracle.f32(0.5)
    exp, fronts = [], []
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        n = hi - lo
        rows, cols = [], []
        for x in range(n):
            g = lo + x
            for p in w.par_idx[w.par_off[g]:w.par_off[g + 1]]:
                rows.append(int(p))
                cols.append(x)
        adj = sp.csr_matrix((np.ones(len(rows)), (rows, cols)), shape=(n, n))
        dist = shortest_path(adj, directed=True, unweighted=True)
        for v in _frontier(w, b):
            fronts.append(v)
            g = lo + v
            tail = 0.0
            for x in range(n):
                h = dist[v, x]
                if 1 <= h <= H:
                    gx = lo + x
                    best = min(float(w.exec[w.model[gx], d]) for d in range(w.D) if _feasible(w, gx, d))
                    tail += gam ** int(h) * best
            r_v = min(int(w.shard_max[g]), w.max_shard, w.D)
            for (i, k) in _windows(w.D, r_v):
                S = range(i, i + k)
                if not all(_feasible(w, g, d) for d in S):
                    exp.append(-np.inf)
                    continue
                j0 = max(float(w.exec[w.model[g], d]) / k for d in S)
                exp.append(-(j0 + tail))
    assert list(r["front_v"]) == fronts
    _close(r["psi"], exp, rtol=1e-12)


def check_wait_only_reduction(seed: int, lib=None):
    """Only the waiting cost switched on and H = 0: Psi = -max_{d in S} max(0, tau_d - t)."""
    w = synth.make_random_small(seed, B=3, n=10, D=5, M=2, K=2, H=0, max_shard=4)
    w.exec[:] = 0.0
    only = dict(lam_q=1.0, lam_s=0.0, lam_tr=0.0, lam_c=0.0, lam_p=0.0)
    r = oracle.score(w, params=only, lib=lib)
    exp = []
    for b in range(w.B):
        lo = int(w.stage_off[b])
        for v in _frontier(w, b):
            g = lo + v
            r_v = min(int(w.shard_max[g]), w.max_shard, w.D)
            for (i, k) in _windows(w.D, r_v):
                S = range(i, i + k)
                if not all(_feasible(w, g, d) for d in S):
                    exp.append(-np.inf)
                    continue
                exp.append(-max(max(0.0, float(w.tau_free[b, d]) - float(w.t_now[b])) for d in S))
    _close(r["psi"], exp, rtol=1e-12)


# ---------------------------------------------------------------------------
# invariants
# ---------------------------------------------------------------------------

def _permute_bits(x: int, perm) -> int:
    out = 0
    for d, pd in enumerate(perm):
        if (x >> d) & 1:
            out |= 1 << int(pd)
    return out


def relabel(w, perm):
    """Apply device relabelling d -> perm[d] to every device-indexed input."""
    perm = np.asarray(perm)
    D = w.D
    inv = np.argsort(perm)  # new index -> old index
    beta = w.beta[np.ix_(inv, inv)]
    return dataclasses.replace(
        w,
        exec=w.exec[:, inv].copy(), switch_s=w.switch_s[:, inv].copy(), beta=beta.copy(),
        cap_bytes=w.cap_bytes[inv].copy(),
        elig=np.array([_permute_bits(int(e), perm) for e in w.elig], np.uint64),
        holders=np.array([_permute_bits(int(e), perm) for e in w.holders], np.uint64),
        resident=w.resident[:, inv].copy(), prefix_cache=w.prefix_cache[:, inv, :].copy(),
        tau_free=w.tau_free[:, inv].copy(), params=dict(w.params),
    )


def check_relabel_singletons(seed: int, lib=None):
    w = synth.make_random_small(seed, B=2, n=12, D=5, M=3, K=3, H=2, max_shard=1)
    perm = np.random.default_rng(seed).permutation(w.D)
    r0 = oracle.score(w, lib=lib)
    r1 = oracle.score(relabel(w, perm), lib=lib)
    assert np.array_equal(r0["front_v"], r1["front_v"])
    co = r0["cand_off"]
    for f in range(len(r0["front_v"])):
        a = r0["psi"][co[f]:co[f] + w.D]
        b = r1["psi"][co[f]:co[f] + w.D]
        _close(b[perm], a, rtol=1e-13, atol=0)


def check_reversal_windows(seed: int, lib=None):
    w = synth.make_random_small(seed, B=2, n=12, D=5, M=3, K=3, H=2, max_shard=4, shard_frac=0.8)
    D = w.D
    perm = np.arange(D)[::-1]
    r0 = oracle.score(w, lib=lib)
    r1 = oracle.score(relabel(w, perm), lib=lib)
    co = r0["cand_off"]
    for f in range(len(r0["front_v"])):
        nc = int(co[f + 1] - co[f])
        r_v = 1
        while D + sum(D - k + 1 for k in range(2, r_v + 1)) < nc:
            r_v += 1
        cands = _windows(D, r_v)
        pos = {c: j for j, c in enumerate(cands)}
        a = r0["psi"][co[f]:co[f + 1]]
        b = r1["psi"][co[f]:co[f + 1]]
        mapped = np.array([b[pos[(D - i - k, k)]] for (i, k) in cands])
        _close(mapped, a, rtol=1e-12, atol=0)


def check_h0_equals_gamma0(seed: int, lib=None):
    w = synth.make_random_small(seed, B=2, n=12, D=4, M=3, K=2, H=3)
    a = oracle.score(w, H=0, lib=lib)["psi"]
    b = oracle.score(w, params=dict(gamma=0.0), lib=lib)["psi"]
    assert np.array_equal(a, b)


def _reach(w, b, v, H):
    """Stages whose attributes may enter v's scores: v, its parents, the
    stages within H hops below v and their parents."""
    lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
    n = hi - lo
    ch = [[] for _ in range(n)]
    for x in range(n):
        for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]]:
            ch[int(p)].append(x)
    seen = {v: 0}
    fr = [v]
    for h in range(1, H + 1):
        nxt = []
        for x in fr:
            for c in ch[x]:
                if c not in seen:
                    seen[c] = h
                    nxt.append(c)
        fr = nxt
    keep = set(seen)
    for x in list(seen):
        keep.update(int(p) for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]])
    return keep


def check_truncation(seed: int, lib=None):
    """Changing stages outside every frontier stage's horizon (and their
    parents) leaves every score unchanged."""
    w = synth.make_random_small(seed, B=1, n=16, D=4, M=3, K=2, H=1, p_edge=0.25, tight_caps=False)
    r0 = oracle.score(w, lib=lib)
    keep = set()
    for v in _frontier(w, 0):
        keep |= _reach(w, 0, v, w.H)
    w2 = dataclasses.replace(w, model=w.model.copy(), out_bytes=w.out_bytes.copy(),
                             prefix_hash=w.prefix_hash.copy(), prefix_tokens=w.prefix_tokens.copy())
    rng = np.random.default_rng(seed)
    far = [x for x in range(w.N) if x not in keep]
    for x in far:
        w2.model[x] = (w2.model[x] + 1) % w.M
        w2.out_bytes[x] *= 3.0
        w2.prefix_hash[x] = np.uint64(int(rng.integers(1, 1 << 60)))
        w2.prefix_tokens[x] += 100.0
    r1 = oracle.score(w2, lib=lib)
    assert np.array_equal(r0["psi"], r1["psi"])


def check_isolated_stage(seed: int, lib=None):
    """Appending an isolated pending root adds one frontier stage and changes
    no other score."""
    w = synth.make_random_small(seed, B=1, n=12, D=4, M=3, K=2, H=2)
    r0 = oracle.score(w, lib=lib)
    n = w.N
    par_off = np.append(w.par_off, w.par_off[-1])
    w2 = dataclasses.replace(
        w, stage_off=np.array([0, n + 1], np.int64), par_off=par_off,
        model=np.append(w.model, 0).astype(np.int32),
        elig=np.append(w.elig, np.uint64((1 << w.D) - 1)).astype(np.uint64),
        shard_max=np.append(w.shard_max, 1).astype(np.int32),
        prefix_hash=np.append(w.prefix_hash, np.uint64(5)).astype(np.uint64),
        prefix_tokens=np.append(w.prefix_tokens, 10.0).astype(np.float32),
        out_bytes=np.append(w.out_bytes, 1e6).astype(np.float32),
        holders=np.append(w.holders, np.uint64(0)).astype(np.uint64),
        status=np.append(w.status, 0).astype(np.uint8))
    r1 = oracle.score(w2, lib=lib)
    F = len(r0["front_v"])
    assert list(r1["front_v"][:F]) == list(r0["front_v"]) and r1["front_v"][F] == n
    assert np.array_equal(r1["psi"][:len(r0["psi"])], r0["psi"])


def check_mag_bounds(seed: int, lib=None):
    """A >= |Psi| for every finite score (triangle inequality over the terms
    that were added).  With the benefit weights (colocation, prefix) at zero
    every term is a cost, so A = |Psi| up to rounding: a slip that adds a term
    to A twice, weights a horizon stage without gamma^depth, or takes the
    terms of more than one device breaks the equality."""
    w = synth.make_random_small(seed, B=3, n=14, D=5, M=3, K=2, H=3, max_shard=3, shard_frac=0.6)
    r = oracle.score(w, lib=lib)
    fin = np.isfinite(r["psi"])
    assert fin.sum() > 10
    assert np.all(r["mag"][fin] >= np.abs(r["psi"][fin]) * (1 - 1e-14)), "A below |Psi|"
    assert np.all(r["mag"][~fin] == 0.0)
    costs = oracle.score(w, params=dict(lam_c=0.0, lam_p=0.0), lib=lib)
    fin = np.isfinite(costs["psi"])
    _close(costs["mag"][fin], np.abs(costs["psi"][fin]), rtol=1e-14, atol=0)
    # and some candidate's A exceeds |Psi| once the benefits are back
    assert np.any(r["mag"][fin] > np.abs(r["psi"][fin]) * (1 + 1e-9))


def check_brute_force(group: int, lib=None, per_group: int = 10):
    """Scores and magnitudes of the oracle equal tests/brute.py's on tiny
    seeded DAGs (windows, multi-device holders, running and committed stages,
    asymmetric and uniform beta) at 1e-12: the post-state materialised by an
    independent state update and priced from scratch, the horizon enumerated
    jointly over every placement of its stages, and the GPU kernel's
    outside / inside rearrangement (brute.py asserts the three agree)."""
    cases = list(brute.tiny_cases(5 * per_group))[group * per_group:(group + 1) * per_group]
    n_fin = 0
    for seed, w, H, ms in cases:
        psi, mag, front = brute.score(w, H=H, max_shard=ms)
        r = oracle.score(w, H=H, max_shard=ms, lib=lib)
        assert [(b, v) for b, v, _ in front] == list(zip(r["front_b"].tolist(), r["front_v"].tolist())), seed
        _close(r["psi"], psi, rtol=1e-12, atol=1e-12)
        fin = np.isfinite(psi)
        _close(r["mag"][fin], mag[fin], rtol=1e-12, atol=1e-12)
        n_fin += int(fin.sum())
    assert n_fin > 0


def check_commit_scenario(name: str, lib=None):
    """Commit-and-advance against the hand-derived state of a scenario."""
    sc = scenarios.COMMITS[name]
    w = builders.from_spec(sc["spec"], H=1)
    _, fv, _ = oracle.frontier(w, lib=lib)
    assert fv.tolist() == sc["front_v"], fv
    new, tau, rejected, fin = oracle.commit(w, sc["sel"], lib=lib)
    assert rejected == sc["rejected"], rejected
    assert new.resident.reshape(-1).tolist() == sc["resident"], new.resident
    assert new.prefix_cache.reshape(w.D, w.K).tolist() == sc["prefix_cache"], new.prefix_cache
    assert new.holders.tolist() == sc["holders"], new.holders
    assert new.status.tolist() == sc["status"], new.status
    _close(tau.reshape(-1), sc["tau"], rtol=0, atol=0)
    _, fv2, _ = oracle.frontier(new, lib=lib)
    assert fv2.tolist() == sc["next_front_v"], fv2


def check_commit_ready(lib=None):
    """Two commits in a row where shards wait for their parents' outputs."""
    sc = scenarios.COMMIT_READY
    w = builders.from_spec(sc["spec"], H=1)
    fin = None
    for step in sc["steps"]:
        _, fv, _ = oracle.frontier(w, lib=lib)
        assert fv.tolist() == step["front_v"], fv
        w, tau, rejected, fin = oracle.commit(w, step["sel"], lib=lib, fin=fin)
        assert rejected == 0
        _close(tau.reshape(-1), step["tau"], rtol=0, atol=0)
        assert fin.tolist() == step["fin"], fin


def check_commit_invariants(seed: int, lib=None):
    """Committing each frontier stage's best candidate: every such stage is
    completed on exactly its candidate's devices, each touched device then
    holds the stage's model within its capacity after dropping the
    smallest-id other models, caches the stage's prefix group, and never
    frees up earlier than before; the next frontier is the set of pending
    stages whose parents are all completed (recomputed here with numpy).
    Committing nothing changes nothing."""
    w = synth.make_random_small(seed, B=3, n=24, D=6, M=5, K=3, max_shard=3, shard_frac=0.6, tight_caps=True)
    r = oracle.score(w, lib=lib)
    idx, _ = oracle.topk(r, 1, lib=lib)
    none, _, rej0, fin0 = oracle.commit(w, np.full(len(r["front_v"]), -1, np.int32), lib=lib)
    assert rej0 == 0
    for f in ("resident", "prefix_cache", "holders", "status", "tau_free"):
        assert np.array_equal(getattr(none, f), getattr(w, f)), f
    assert np.array_equal(fin0, oracle.initial_finish(w))
    new, tau, rej, fin = oracle.commit(w, idx[:, 0], lib=lib)
    assert rej == 0
    D, K = w.D, w.K

    def devices(j):
        k, i = 1, int(j)
        if j >= D:  # windows by size, then start
            t = int(j) - D
            k = 2
            while t >= D - k + 1:
                t -= D - k + 1
                k += 1
            i = t
        return list(range(i, i + k))

    # a device that takes several stages in one commit sees them in turn; the
    # per-device checks below are for devices that take exactly one
    uses = np.zeros((w.B, D), np.int64)
    for f, j in enumerate(idx[:, 0]):
        if j >= 0:
            for d in devices(j):
                uses[int(r["front_b"][f]), d] += 1
    for f, j in enumerate(idx[:, 0]):
        b, v = int(r["front_b"][f]), int(r["front_v"][f])
        g = int(w.stage_off[b]) + v
        if j < 0:
            assert new.status[g] == w.status[g]
            continue
        S = devices(j)
        assert new.status[g] == 1 and int(new.holders[g]) == sum(1 << d for d in S)
        m = int(w.model[g])
        k = len(S)
        # the stage finishes with its latest shard
        assert any(uses[b, d] != 1 for d in S) or fin[g] == np.float32(max(tau[b, d] for d in S))
        for d in S:
            assert tau[b, d] >= float(w.tau_free[b, d])
            if uses[b, d] != 1:
                continue
            # a shard starts no earlier than the device is free, than t, and
            # than each parent's output is there, and at one of those times
            run = float(w.exec[m, d]) / k + (0.0 if (int(w.resident[b, d]) >> m) & 1 else float(w.switch_s[m, d]))
            start = tau[b, d] - run
            lo = int(w.stage_off[b])
            arrivals = [max(float(w.tau_free[b, d]), float(np.float32(w.t_now[b])))]
            for p in w.par_idx[w.par_off[g]:w.par_off[g + 1]]:
                u = lo + int(p)
                hu = int(w.holders[u])
                t_u = float(np.float32(w.t_now[b]))  # completed before planning
                if not (hu >> d) & 1:
                    t_u += float(w.out_bytes[u]) * min(float(w.beta[i, d]) for i in range(D) if (hu >> i) & 1) / k
                arrivals.append(t_u)
            assert start >= max(arrivals) - 1e-9 * max(1.0, start), (g, d, start, arrivals)
            assert min(abs(start - a) for a in arrivals) <= 1e-9 * max(1.0, start), (g, d, start, arrivals)
            old = int(w.resident[b, d])
            res = int(new.resident[b, d])
            assert (res >> m) & 1
            used = sum(int(w.weight_bytes[x]) for x in range(w.M) if (res >> x) & 1)
            assert used <= int(w.cap_bytes[d])
            if not (old >> m) & 1:
                # models dropped from d are the smallest ids other than m
                dropped = [x for x in range(w.M) if (old >> x) & 1 and not (res >> x) & 1]
                kept = [x for x in range(w.M) if (old >> x) & 1 and (res >> x) & 1 and x != m]
                assert not dropped or not kept or max(dropped) < min(kept), (old, res, m)
            h = int(w.prefix_hash[g])
            if h and K:
                assert h in [int(x) for x in new.prefix_cache[b, d]]
    # next frontier, recomputed from the parent lists
    npar = np.diff(w.par_off)
    inst = np.repeat(np.arange(w.B), np.diff(w.stage_off))
    pg = w.par_idx.astype(np.int64) + w.stage_off[np.repeat(inst, npar)]
    done = np.zeros(len(npar), np.int64)
    np.add.at(done, np.repeat(np.arange(len(npar)), npar), (new.status[pg] == 1).astype(np.int64))
    ready = np.nonzero((new.status == 0) & (done == npar))[0]
    fb2, fv2, _ = oracle.frontier(new, lib=lib)
    got = (w.stage_off[fb2] + fv2).astype(np.int64)
    assert np.array_equal(got, ready), (got, ready)


# ---------------------------------------------------------------------------
# scoring variants (oracle V1-V4)
# ---------------------------------------------------------------------------

def check_variant_scenario(name: str, lib=None):
    sc = scenarios.VARIANTS[name]
    w = builders.from_spec(sc["spec"], H=sc["H"], params=sc["params"])
    r = oracle.score(w, lib=lib)
    assert list(r["front_v"]) == sc["front_v"], (list(r["front_v"]), sc["front_v"])
    _close(r["psi"], sc["psi"], rtol=1e-12)
    if "topk3" in sc:
        idx, _ = oracle.topk(r, 3, lib=lib)
        assert idx[0].tolist() == sc["topk3"], idx


def _levels_scipy(adj):
    """Topological level of every stage: the length of the longest path that
    ends there, from Bellman-Ford shortest paths with every edge weighted -1."""
    n = adj.shape[0]
    neg = sp.csr_matrix((-np.ones(adj.nnz), adj.indices, adj.indptr), shape=(n, n))
    dist = shortest_path(neg, method="BF", directed=True)
    lv = np.where(np.isfinite(dist), -dist, 0.0).max(axis=0)
    return np.maximum(lv, 0.0).astype(np.int64)


def check_variant_reduction(seed: int, lib=None, H: int = 3, topo: bool = False, mean: bool = False):
    """Base runtimes only, under the horizon variants: the tail is
    sum_h gamma^h agg_{w at depth h} min_feasible c(w,.), agg = sum or mean,
    depth = hop distance (scipy, unweighted) or the difference of longest-path
    levels (scipy Bellman-Ford on -1 weights) among stages reachable from v."""
    w = synth.make_random_small(seed, B=2, n=16, D=4, M=3, K=2, H=H, max_shard=3, p_edge=0.35)
    zero = dict(lam_q=0.0, lam_s=0.0, lam_tr=0.0, lam_c=0.0, lam_p=0.0, gamma=0.5,
                topo_levels=int(topo), mean_levels=int(mean))
    r = oracle.score(w, params=zero, lib=lib)
    gam = oracle.f32(0.5)
    exp, fronts = [], []
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        n = hi - lo
        rows, cols = [], []
        for x in range(n):
            g = lo + x
            for p in w.par_idx[w.par_off[g]:w.par_off[g + 1]]:
                rows.append(int(p))
                cols.append(x)
        adj = sp.csr_matrix((np.ones(len(rows)), (rows, cols)), shape=(n, n))
        dist = shortest_path(adj, directed=True, unweighted=True)
        lv = _levels_scipy(adj)
        for v in _frontier(w, b):
            fronts.append(v)
            g = lo + v
            by_depth = {}
            for x in range(n):
                if not np.isfinite(dist[v, x]) or x == v:
                    continue
                h = int(lv[x] - lv[v]) if topo else int(dist[v, x])
                if 1 <= h <= H:
                    gx = lo + x
                    best = min(float(w.exec[w.model[gx], d]) for d in range(w.D) if _feasible(w, gx, d))
                    by_depth.setdefault(h, []).append(best)
            tail = sum(gam ** h * (np.mean(vals) if mean else np.sum(vals)) for h, vals in by_depth.items())
            r_v = min(int(w.shard_max[g]), w.max_shard, w.D)
            for (i, k) in _windows(w.D, r_v):
                S = range(i, i + k)
                if not all(_feasible(w, g, d) for d in S):
                    exp.append(-np.inf)
                    continue
                j0 = max(float(w.exec[w.model[g], d]) / k for d in S)
                exp.append(-(j0 + tail))
    assert list(r["front_v"]) == fronts
    _close(r["psi"], exp, rtol=1e-12)


def check_topo_equals_hop_on_layers(seed: int, lib=None):
    """Where every edge joins consecutive layers (the layered and fork-join
    recipes) the topological-level horizon is the breadth-first one."""
    name = ("tiny-layered-1x24-d4", "layered-1024x200-d8", "forkjoin-4096x1000-d16")[seed]
    w = synth.make_workload(name, B=2 if seed else 1)
    a = oracle.score(w, lib=lib)
    b = oracle.score(w, params=dict(topo_levels=1), lib=lib)
    assert np.array_equal(a["psi"], b["psi"])


def check_mean_equals_sum_on_chains(seed: int, lib=None):
    """On chains every horizon level holds one stage, so mean = sum."""
    w = synth.make_random_small(seed, B=2, n=12, D=4, M=3, K=2, H=4, max_shard=3, p_edge=0.0)
    # relink every stage to its predecessor only: a chain per instance
    par_off = [0]
    par_idx = []
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        for x in range(hi - lo):
            if x > 0:
                par_idx.append(x - 1)
            par_off.append(len(par_idx))
    import dataclasses
    st = w.status.copy()
    hold = w.holders.copy()
    for b in range(w.B):  # completed stages must stay down-closed on the chain
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        done = True
        for g in range(lo, hi):
            done = done and st[g] == 1
            if not done and st[g] in (1, 2):
                st[g], hold[g] = 0, 0
    w = dataclasses.replace(w, par_off=np.array(par_off, np.int64), par_idx=np.array(par_idx, np.int32),
                            status=st, holders=hold)
    a = oracle.score(w, lib=lib)
    b = oracle.score(w, params=dict(mean_levels=1), lib=lib)
    assert len(a["psi"]) > 0
    _close(b["psi"], a["psi"], rtol=1e-15)


def check_no_windows_keeps_singletons(seed: int, lib=None):
    """Without windows the singletons score as under max_shard = 1, and every
    window slot is -inf."""
    w = synth.make_random_small(seed, B=3, n=16, D=5, M=3, K=2, max_shard=3, shard_frac=0.6)
    a = oracle.score(w, params=dict(no_windows=1), lib=lib)
    b = oracle.score(w, max_shard=1, lib=lib)
    nf = len(a["front_v"])
    assert nf == len(b["front_v"]) and nf > 0
    for f in range(nf):
        seg = a["psi"][a["cand_off"][f]:a["cand_off"][f + 1]]
        assert np.array_equal(seg[:w.D], b["psi"][b["cand_off"][f]:b["cand_off"][f + 1]])
        assert np.all(np.isneginf(seg[w.D:]))
    assert any(a["cand_off"][f + 1] - a["cand_off"][f] > w.D for f in range(nf))


def check_same_model_weight_linear(seed: int, lib=None):
    """Psi is affine in lam_m with slope -(number of same-model events the
    maximising shard and the minimising descendant devices see): checked by
    Psi(2x) - Psi(x) = Psi(x) - Psi(0) on candidates whose choices do not flip,
    which holds for every candidate when all devices share one speed class
    and every model is resident everywhere (the bonus is then uniform)."""
    w = synth.make_random_small(seed, B=2, n=16, D=4, M=3, K=2, max_shard=3, tight_caps=False)
    import dataclasses
    full = np.uint64((1 << w.M) - 1)
    w = dataclasses.replace(w, resident=np.full_like(w.resident, full))
    if any(int(w.weight_bytes.sum()) > int(c) for c in w.cap_bytes):
        return  # all models cannot be resident together: not this check's case
    r0 = oracle.score(w, params=dict(lam_m=0.0), lib=lib)
    r1 = oracle.score(w, params=dict(lam_m=0.125), lib=lib)
    H = int(w.H)
    fin = np.isfinite(r0["psi"])
    # every shard device and every descendant device holds its model: the
    # immediate cost drops by lam_m and each horizon stage's value by lam_m
    for f in range(len(r0["front_v"])):
        lo, hi = r0["cand_off"][f], r0["cand_off"][f + 1]
        b, v = int(r0["front_b"][f]), int(r0["front_v"][f])
        n_at = _horizon_counts(w, b, v, H)
        drop = 0.125 * (1.0 + sum(oracle.f32(w.params["gamma"]) ** h * c for h, c in n_at.items()))
        _close(r1["psi"][lo:hi][fin[lo:hi]], r0["psi"][lo:hi][fin[lo:hi]] + drop, rtol=1e-12)


def _horizon_counts(w, b, v, H):
    lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
    n = hi - lo
    rows, cols = [], []
    for x in range(n):
        for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]]:
            rows.append(int(p))
            cols.append(x)
    adj = sp.csr_matrix((np.ones(len(rows)), (rows, cols)), shape=(n, n))
    dist = shortest_path(adj, directed=True, unweighted=True, indices=[v])[0]
    out = {}
    for x in range(n):
        h = dist[x]
        if np.isfinite(h) and 1 <= h <= H:
            out[int(h)] = out.get(int(h), 0) + 1
    return out


# ---------------------------------------------------------------------------
# frontier planning wave (oracle step 12)
# ---------------------------------------------------------------------------

def check_plan_scenario(name: str, lib=None):
    sc = scenarios.PLANS[name]
    sel, n = oracle.plan_wave(sc["D"], sc["f_off"], sc["n_cand"], np.array(sc["idx"], np.int32),
                              np.array(sc["val"], np.float32), lib=lib)
    assert sel.tolist() == sc["sel"], (sel.tolist(), sc["sel"])
    assert n == sum(1 for x in sc["sel"] if x >= 0)


def _window_mask(D, j):
    k, i = 1, int(j)
    if j >= D:
        t, k = int(j) - D, 2
        while t >= D - k + 1:
            t -= D - k + 1
            k += 1
        i = t
    return ((1 << k) - 1) << i


def random_plan_input(seed: int, B=5, D=6, k=4, max_shard=3, p_inf=0.15, ties=False):
    """Seeded top-k-like choices: per slot k distinct candidate indices of a
    stage with windows up to max_shard (or singletons only), a few past the
    stage's candidates, scores descending per slot (as a top-k reports them),
    some -inf / padded."""
    rng = np.random.default_rng(seed)
    nC = D + sum(D - w + 1 for w in range(2, max_shard + 1))
    nf = rng.integers(0, 9, size=B)
    f_off = np.concatenate([[0], np.cumsum(nf)]).astype(np.int64)
    F = int(f_off[-1])
    n_cand = np.where(rng.random(F) < 0.3, D, nC).astype(np.int64)
    idx = np.full((F, k), -1, np.int32)
    val = np.full((F, k), -np.inf, np.float32)
    for f in range(F):
        m = int(rng.integers(0, k + 1))
        js = rng.choice(nC + 3, size=min(m, nC), replace=False)  # indices up to nC + 2 < D (D + 1) / 2
        vs = (np.round(rng.normal(-3.0, 1.0, size=len(js)) * 4) / 4) if ties else rng.normal(-3.0, 1.0, size=len(js))
        order = np.argsort(-vs, kind="stable")
        for r, o in enumerate(order):
            if rng.random() < p_inf:
                break  # the rest of this slot is padding
            idx[f, r] = js[o]
            val[f, r] = vs[o]
    return D, f_off, n_cand, idx, val


def check_plan_certificate(seed: int, lib=None, ties=False):
    """The greedy wave is feasible (one choice per stage, devices disjoint per
    instance), maximal (no untaken valid choice has a free stage and free
    devices), and every untaken valid choice is blocked by a taken choice
    that scores at least as high (the greedy exchange certificate)."""
    D, f_off, n_cand, idx, val = random_plan_input(seed, ties=ties)
    sel, n = oracle.plan_wave(D, f_off, n_cand, idx, val, lib=lib)
    assert n == int(np.count_nonzero(sel >= 0))
    for b in range(len(f_off) - 1):
        lo, hi = int(f_off[b]), int(f_off[b + 1])
        taken = {}
        used = 0
        for f in range(lo, hi):
            if sel[f] < 0:
                continue
            rs = [r for r in range(idx.shape[1]) if idx[f, r] == sel[f] and np.isfinite(val[f, r])]
            assert sel[f] < n_cand[f], (f, sel[f])
            assert rs, (f, sel[f])
            m = _window_mask(D, sel[f])
            assert used & m == 0, "devices used twice"
            used |= m
            taken[f] = (float(val[f, rs[0]]), m)
        for f in range(lo, hi):
            for r in range(idx.shape[1]):
                if idx[f, r] < 0 or idx[f, r] >= n_cand[f] or not np.isfinite(val[f, r]) or sel[f] == idx[f, r]:
                    continue
                m, v = _window_mask(D, idx[f, r]), float(val[f, r])
                if f not in taken:
                    assert used & m, "maximality: slot %d choice %d fits" % (f, r)
                # blocked by its own stage or by a device: some blocker scores >= v
                blockers = [tv for g, (tv, tm) in taken.items() if g == f or tm & m]
                assert blockers and max(blockers) >= v, (f, r, v, blockers)


def check_plan_no_conflicts(seed: int, lib=None):
    """With one instance per slot (nothing shared), the wave takes every
    stage's best valid choice."""
    D, f_off, n_cand, idx, val = random_plan_input(seed)
    F = int(f_off[-1])
    sel, _ = oracle.plan_wave(D, np.arange(F + 1), n_cand, idx, val, lib=lib)
    for f in range(F):
        ok = [r for r in range(idx.shape[1]) if 0 <= idx[f, r] < n_cand[f] and np.isfinite(val[f, r])]
        want = idx[f, max(ok, key=lambda r: (val[f, r], -r))] if ok else -1
        assert sel[f] == want, (f, sel[f], want)


ALL_CHECKS = (
    [("scenario:" + k, (lambda k: lambda lib: check_scenario(k, lib))(k)) for k in scenarios.ALL]
    + [("worked_example", check_worked_example)]
    + [("exec_only:%d" % s, (lambda s: lambda lib: check_exec_only_reduction(s, lib))(s)) for s in range(3)]
    + [("wait_only:%d" % s, (lambda s: lambda lib: check_wait_only_reduction(s, lib))(s)) for s in range(2)]
    + [("relabel:%d" % s, (lambda s: lambda lib: check_relabel_singletons(s, lib))(s)) for s in range(2)]
    + [("reversal:%d" % s, (lambda s: lambda lib: check_reversal_windows(s, lib))(s)) for s in range(2)]
    + [("h0_gamma0:%d" % s, (lambda s: lambda lib: check_h0_equals_gamma0(s, lib))(s)) for s in range(2)]
    + [("mag_bounds:%d" % s, (lambda s: lambda lib: check_mag_bounds(s, lib))(s)) for s in range(3)]
    + [("brute_force:%d" % g, (lambda g: lambda lib: check_brute_force(g, lib))(g)) for g in range(5)]
    + [("truncation:%d" % s, (lambda s: lambda lib: check_truncation(s, lib))(s)) for s in range(3)]
    + [("isolated:%d" % s, (lambda s: lambda lib: check_isolated_stage(s, lib))(s)) for s in range(2)]
    + [("commit:" + k, (lambda k: lambda lib: check_commit_scenario(k, lib))(k)) for k in scenarios.COMMITS]
    + [("commit_invariants:%d" % s, (lambda s: lambda lib: check_commit_invariants(s, lib))(s)) for s in range(3)]
    + [("commit_ready", check_commit_ready)]
    + [("variant:" + k, (lambda k: lambda lib: check_variant_scenario(k, lib))(k)) for k in scenarios.VARIANTS]
    + [("variant_reduction:%s:%d" % (m, s),
        (lambda s, t, mn: lambda lib: check_variant_reduction(s, lib, topo=t, mean=mn))(s, t, mn))
       for m, t, mn in (("topo", True, False), ("mean", False, True), ("topo_mean", True, True))
       for s in range(3)]
    + [("topo_equals_hop:%d" % s, (lambda s: lambda lib: check_topo_equals_hop_on_layers(s, lib))(s))
       for s in range(2)]
    + [("mean_equals_sum_chain:%d" % s, (lambda s: lambda lib: check_mean_equals_sum_on_chains(s, lib))(s))
       for s in range(2)]
    + [("no_windows:%d" % s, (lambda s: lambda lib: check_no_windows_keeps_singletons(s, lib))(s)) for s in range(2)]
    + [("same_model_uniform:%d" % s, (lambda s: lambda lib: check_same_model_weight_linear(s, lib))(s))
       for s in range(3)]
    + [("plan:" + k, (lambda k: lambda lib: check_plan_scenario(k, lib))(k)) for k in scenarios.PLANS]
    + [("plan_certificate:%d" % s, (lambda s: lambda lib: check_plan_certificate(s, lib, ties=s % 2 == 1))(s))
       for s in range(6)]
    + [("plan_no_conflicts:%d" % s, (lambda s: lambda lib: check_plan_no_conflicts(s, lib))(s)) for s in range(2)]
)
