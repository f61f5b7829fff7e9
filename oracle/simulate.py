"""Plain Python reference of the discrete-event execution of a plan and of
the two baseline placements (test infrastructure only: only the test suite,
``__graft_entry__.smoke()`` and the benchmark's CPU-baseline leg may use it).

What it computes, per workflow instance, from the instance's state at t0 =
t_now and a placement (the devices S(v) of every pending stage, 0 = not
placed) with an execution order key per stage.  Readings of passages the paper
leaves open are marked [reading]; each is listed in the design notes.

Execution (Sec. 2 stage tuple and state; App. A.3 / A.4 cost terms as
execution times) [reading: each device runs its stages in order-key order;
processing all placed stages of the instance in (key, id) order computes
that schedule exactly when the keys respect the DAG, which is checked]:
  for v in (key, id) order, k = |S(v)|, for each d in S(v) ascending:
    ready  = max(t0, max over parents u of finish(u) + transfer(u, d) / k),
             transfer(u, d) = 0 if d holds u's output, else
             sigma(u) * min over holders i of beta[i][d]
    start  = max(free(d), ready)
    switch = kappa_switch(m(v), d) if m(v) is not resident on d, else 0;
             then Load (add m(v); evict the smallest-id other models while
             the resident weights exceed the capacity)
    hit    = grp(v) != 0 and grp(v) is in d's prefix slots
    run    = max(0, c(v, d) / k - (kappa_prefix * L(v) / k if hit else 0))
    free(d) = start + switch + run; grp(v) joins d's slots (first empty
             slot, else drop slot 0 and append)
  finish(v) = max over d of free(d); v's output is then held by S(v).
Metrics (App. C.2):
  tasks        stages executed
  makespan     max finish - t0 (0 without tasks)
  p95          nearest-rank 95th percentile of finish - t0 over the executed
               stages without children [reading: a query completes with its
               workflow's final outputs]
  xdev_edges   edges u -> v whose v runs on no device holding u's output
  cache_hits   executed v with a hit on the first device of S(v)
  model_cont   executed v whose first device ran a stage of the same model
               just before (within this execution)
Baselines (App. B): round robin places each pending stage, in id order, on
the next feasible device after the previous placement; the HEFT-style list
scheduler orders pending stages by upward rank (mean runtime over feasible
devices plus the largest mean transfer + rank over children; ties to the
lower id) and gives each the feasible device with the earliest finish under
the execution rule above (ties to the lower device).
"""

from __future__ import annotations

import math

import numpy as np

COMPLETED = 1


def _bits(m):
    d = 0
    while m:
        if m & 1:
            yield d
        m >>= 1
        d += 1


class _Inst:
    """One instance's tables and state, as plain Python values."""

    def __init__(self, w, b, kappa_prefix):
        self.D, self.M, self.K = int(w.D), int(w.M), int(w.K)
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        self.lo, self.n = lo, hi - lo
        self.parents = [[int(p) for p in w.par_idx[w.par_off[lo + v]:w.par_off[lo + v + 1]]] for v in range(self.n)]
        self.children = [[] for _ in range(self.n)]
        for v in range(self.n):
            for u in self.parents[v]:
                self.children[u].append(v)
        self.model = [int(x) for x in w.model[lo:hi]]
        self.elig = [int(x) for x in w.elig[lo:hi]]
        self.grp = [int(x) for x in w.prefix_hash[lo:hi]]
        self.tokens = [float(np.float32(x)) for x in w.prefix_tokens[lo:hi]]
        self.sigma = [float(np.float32(x)) for x in w.out_bytes[lo:hi]]
        self.status = [int(x) for x in w.status[lo:hi]]
        self.holders = [int(x) for x in w.holders[lo:hi]]
        self.exec = np.asarray(w.exec, np.float64)
        self.ksw = np.asarray(w.switch_s, np.float64)
        self.beta = np.asarray(w.beta, np.float64)
        self.weight = [int(x) for x in w.weight_bytes]
        self.cap = [int(x) for x in w.cap_bytes]
        self.t0 = float(np.float32(w.t_now[b]))
        self.kpf = float(np.float32(kappa_prefix))
        self.free = [max(float(np.float32(w.tau_free[b, d])), self.t0) for d in range(self.D)]
        self.res = [int(w.resident[b, d]) for d in range(self.D)]
        self.ring = [[int(x) for x in w.prefix_cache[b, d]] for d in range(self.D)]
        self.last_model = [-1] * self.D
        self.finish = [self.t0 if s == COMPLETED else None for s in self.status]

    def feasible(self, v, d):
        m = self.model[v]
        return (self.elig[v] >> d) & 1 and self.weight[m] <= self.cap[d]

    def load(self, res, m, d):
        if (res >> m) & 1:
            return res
        res |= 1 << m
        total = sum(self.weight[i] for i in range(self.M) if (res >> i) & 1)
        for i in range(self.M):
            if total <= self.cap[d]:
                break
            if i != m and (res >> i) & 1:
                res &= ~(1 << i)
                total -= self.weight[i]
        return res

    def shard(self, v, d, k, free, res, ring):
        """Start, finish and side effects of v's shard on d: (finish, res', hit)."""
        ready = self.t0
        for u in self.parents[v]:
            hu = self.holders[u]
            if (hu >> d) & 1:
                arr = self.finish[u]
            else:
                bmin = min(self.beta[i, d] for i in _bits(hu))
                arr = self.finish[u] + self.sigma[u] * bmin / k
            ready = max(ready, arr)
        start = max(free, ready)
        m = self.model[v]
        sw = 0.0 if (res >> m) & 1 else self.ksw[m, d]
        hit = self.grp[v] != 0 and self.grp[v] in ring
        run = self.exec[m, d] / k
        if hit:
            run = max(0.0, run - self.kpf * self.tokens[v] / k)
        return start + sw + run, self.load(res, m, d), hit

    def ring_push(self, d, h):
        if h == 0 or self.K == 0:
            return
        r = self.ring[d]
        if h in r:
            return
        if 0 in r:
            r[r.index(0)] = h
        else:
            del r[0]
            r.append(h)

    def run(self, v, S):
        """Execute v on device set S; returns (hit on first device, continuation)."""
        devs = list(_bits(S))
        k = len(devs)
        fin, hit0, cont0 = self.t0, False, False
        for q, d in enumerate(devs):
            f, res, hit = self.shard(v, d, k, self.free[d], self.res[d], self.ring[d])
            if q == 0:
                hit0 = hit
                cont0 = self.last_model[d] == self.model[v]
            self.free[d] = f
            self.res[d] = res
            self.ring_push(d, self.grp[v])
            self.last_model[d] = self.model[v]
            fin = max(fin, f)
        self.finish[v] = fin
        self.holders[v] = S
        return hit0, cont0


def simulate(w, devices, order, kappa_prefix=None):
    """Execute the placement ``devices`` [N] (uint64 device masks, 0 = not
    placed) in ``order`` [N] (int64 keys) on every instance of ``w``.
    Returns a dict of per-instance arrays: tasks, makespan, p95, xdev_edges,
    cache_hits, model_cont."""
    kpf = w.params["kappa_prefix"] if kappa_prefix is None else kappa_prefix
    out = {k: [] for k in ("tasks", "makespan", "p95", "xdev_edges", "cache_hits", "model_cont")}
    for b in range(w.B):
        I = _Inst(w, b, kpf)
        todo = [v for v in range(I.n) if I.status[v] != COMPLETED and int(devices[I.lo + v]) != 0]
        todo.sort(key=lambda v: (int(order[I.lo + v]), v))
        tasks = xdev = hits = cont = 0
        for v in todo:
            S = int(devices[I.lo + v])
            for u in I.parents[v]:
                if I.finish[u] is None:
                    raise ValueError("instance %d: stage %d runs before its parent %d" % (b, v, u))
                if I.holders[u] & S == 0:
                    xdev += 1
            h, c = I.run(v, S)
            tasks += 1
            hits += int(h)
            cont += int(c)
        done = [v for v in todo]
        mk = max((I.finish[v] for v in done), default=I.t0) - I.t0
        sinks = sorted(I.finish[v] - I.t0 for v in done if not I.children[v])
        p95 = sinks[max(0, math.ceil(0.95 * len(sinks)) - 1)] if sinks else 0.0
        for key, val in (("tasks", tasks), ("makespan", mk), ("p95", p95), ("xdev_edges", xdev),
                         ("cache_hits", hits), ("model_cont", cont)):
            out[key].append(val)
    return {k: np.asarray(v, np.float64 if k in ("makespan", "p95") else np.int64) for k, v in out.items()}


def place_round_robin(w):
    """Round-robin placement: (devices [N] uint64, order [N] int64)."""
    devices = np.zeros(w.N, np.uint64)
    order = np.zeros(w.N, np.int64)
    for b in range(w.B):
        I = _Inst(w, b, 0.0)
        nxt = 0
        for v in range(I.n):
            if I.status[v] == COMPLETED:
                continue
            for q in range(I.D):
                d = (nxt + q) % I.D
                if I.feasible(v, d):
                    devices[I.lo + v] = np.uint64(1 << d)
                    nxt = d + 1
                    break
            order[I.lo + v] = v
    return devices, order


def place_heft(w, kappa_prefix=None):
    """HEFT-style list scheduling: (devices [N] uint64, order [N] int64)."""
    kpf = w.params["kappa_prefix"] if kappa_prefix is None else kappa_prefix
    devices = np.zeros(w.N, np.uint64)
    order = np.zeros(w.N, np.int64)
    D = int(w.D)
    offd = [float(w.beta[i, j]) for i in range(D) for j in range(D) if i != j]
    bmean = sum(offd) / len(offd) if offd else 0.0
    for b in range(w.B):
        I = _Inst(w, b, kpf)
        rank = [0.0] * I.n
        for v in range(I.n - 1, -1, -1):  # children have larger ids
            feas = [d for d in range(D) if I.feasible(v, d)]
            wbar = sum(I.exec[I.model[v], d] for d in feas) / len(feas)
            tail = max((I.sigma[v] * bmean + rank[c] for c in I.children[v]), default=0.0)
            rank[v] = wbar + tail
        todo = [v for v in range(I.n) if I.status[v] != COMPLETED]
        todo.sort(key=lambda v: (-rank[v], v))
        for pos, v in enumerate(todo):
            best_d, best_f = -1, math.inf
            for d in range(D):
                if not I.feasible(v, d):
                    continue
                f, _, _ = I.shard(v, d, 1, I.free[d], I.res[d], I.ring[d])
                if f < best_f:
                    best_d, best_f = d, f
            I.run(v, 1 << best_d)
            devices[I.lo + v] = np.uint64(1 << best_d)
            order[I.lo + v] = pos
    return devices, order
