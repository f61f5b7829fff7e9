"""Brute-force and materialised-state checkers for the fp64 oracle (CPU,
test infrastructure only).

Written from the paper's definitions and the readings recorded in the design
notes, independently of ``oracle/``: nothing here imports or calls it, and the
code is organised differently (whole-state copies instead of a state view,
child sets instead of a queue, joint enumeration instead of a running
minimum).  The tests compare the oracle's scores and magnitudes with the
values computed here.

For a candidate placement S of a frontier stage v (Sec. 3.3 shard slots,
App. A.2 bounded shard execution):

* ``materialise`` copies the instance's state and applies the placement the
  way Sec. 3.2 describes the future state: on every device of S the model of
  v is loaded (added, then the smallest-id other models are dropped while
  the resident weights exceed the capacity), the prefix group of v joins the
  device's cached groups (a hypothetical insert that drops nothing), and v's
  output is held by exactly the devices of S.
* ``c_hat`` evaluates the state-corrected cost of App. A.1 / A.4 with the
  terms of App. A.3 from the materialised arrays alone.
* The horizon (Sec. 3.3; H counts levels beyond v, App. D.4) is grown level
  by level as sets of children; a stage belongs to the first level that
  reaches it.
* ``joint_minimum`` enumerates every joint placement of the horizon stages
  (D^|U| of them) and keeps the smallest gamma-weighted total.  Because each
  horizon stage is priced in the same post-state, that minimum must equal the
  sum of the per-stage minima.
* ``decomposed_value`` prices a horizon stage the way the GPU kernel does: a
  row B(d') in the current state, where uncompleted parents contribute
  nothing, then the minimum over devices outside S (a child of v also pays
  for v's output there) and over devices inside S (the row corrected by what
  the placement changes on that device).  It must agree with the
  from-scratch value.

Magnitudes A follow the same definition as the oracle's: the absolute values
of the weighted terms of the device that sets the immediate cost (the first
maximising shard device), plus the gather term, plus gamma^depth times the
absolute terms of the first minimising device of each horizon stage.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Tuple

import numpy as np

PENDING, COMPLETED = 0, 1


def _f32(x) -> float:
    return float(np.float32(x))


def _devs(mask: int) -> List[int]:
    return [d for d in range(64) if (mask >> d) & 1]


@dataclass
class State:
    """One instance's state, as plain Python values (a full copy)."""
    resident: List[int]          # per device: bitmask of resident models
    cached: List[set]            # per device: prefix groups cached
    holders: Dict[int, int]      # stage -> device bitmask holding its output
    wait: List[float]            # per device: max(0, tau_d - t)


class Instance:
    """The static data of instance b of a workload, instance-local ids."""

    def __init__(self, w, b: int, params: dict):
        self.w, self.b = w, b
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        self.lo, self.n, self.D, self.M = lo, hi - lo, int(w.D), int(w.M)
        self.parents = [[int(p) for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]]] for x in range(self.n)]
        self.children: List[List[int]] = [[] for _ in range(self.n)]
        for x, ps in enumerate(self.parents):
            for p in ps:
                self.children[p].append(x)
        self.model = [int(w.model[lo + x]) for x in range(self.n)]
        self.elig = [int(w.elig[lo + x]) for x in range(self.n)]
        self.group = [int(w.prefix_hash[lo + x]) for x in range(self.n)]
        self.tokens = [_f32(w.prefix_tokens[lo + x]) for x in range(self.n)]
        self.sigma = [_f32(w.out_bytes[lo + x]) for x in range(self.n)]
        self.status = [int(w.status[lo + x]) for x in range(self.n)]
        self.rmax = [int(w.shard_max[lo + x]) for x in range(self.n)]
        self.exec = [[_f32(w.exec[m, d]) for d in range(self.D)] for m in range(self.M)]
        self.ksw = [[_f32(w.switch_s[m, d]) for d in range(self.D)] for m in range(self.M)]
        self.beta = [[_f32(w.beta[i, j]) for j in range(self.D)] for i in range(self.D)]
        self.W = [int(x) for x in w.weight_bytes]
        self.cap = [int(x) for x in w.cap_bytes]
        p = dict(w.params)
        p.update(params or {})
        for key in ("lam_m", "topo_levels", "mean_levels", "no_windows"):
            if p.get(key, 0):
                raise ValueError("the brute-force checker covers the default method only (%s set)" % key)
        self.lq, self.ls, self.ltr = _f32(p["lam_q"]), _f32(p["lam_s"]), _f32(p["lam_tr"])
        self.lc, self.lp = _f32(p["lam_c"]), _f32(p["lam_p"])
        self.kpf, self.gamma = _f32(p["kappa_prefix"]), _f32(p["gamma"])
        t = _f32(w.t_now[b])
        self.state = State(
            resident=[int(w.resident[b, d]) for d in range(self.D)],
            cached=[set(int(h) for h in w.prefix_cache[b, d] if int(h) != 0) for d in range(self.D)],
            holders={x: int(w.holders[lo + x]) for x in range(self.n) if int(w.holders[lo + x]) != 0},
            wait=[max(0.0, _f32(w.tau_free[b, d]) - t) for d in range(self.D)],
        )

    # -- feasibility (Sec. 2 feasible set: eligible and the model fits) ------
    def feasible(self, x: int, d: int) -> bool:
        return bool((self.elig[x] >> d) & 1) and self.W[self.model[x]] <= self.cap[d]

    # -- ready frontier (Sec. 2 ready set; App. A.1 excludes running/committed)
    def frontier(self) -> List[int]:
        return [x for x in range(self.n)
                if self.status[x] == PENDING and all(self.status[p] == COMPLETED for p in self.parents[x])]

    # -- candidate device sets, in the output order --------------------------
    def candidates(self, v: int, max_shard: int) -> List[Tuple[int, ...]]:
        r = max(1, min(self.rmax[v], max_shard, self.D))
        out = [(d,) for d in range(self.D)]
        for k in range(2, r + 1):
            out += [tuple(range(i, i + k)) for i in range(self.D - k + 1)]
        return out

    # -- Load under capacity (reading of the eviction rule) ------------------
    def load(self, res: int, m: int, d: int) -> int:
        models = sorted(x for x in range(self.M) if (res >> x) & 1)
        if m in models:
            return res
        models.append(m)
        while sum(self.W[x] for x in models) > self.cap[d]:
            others = [x for x in models if x != m]
            if not others:
                break
            models.remove(min(others))
        out = 0
        for x in models:
            out |= 1 << x
        return out

    # -- the future state after placing v on S (Sec. 3.2) --------------------
    def materialise(self, v: int, S) -> State:
        s = self.state
        res = list(s.resident)
        cached = [set(c) for c in s.cached]
        holders = dict(s.holders)
        mask = 0
        for d in S:
            res[d] = self.load(res[d], self.model[v], d)
            if self.group[v] != 0:
                cached[d].add(self.group[v])
            mask |= 1 << d
        holders[v] = mask
        return State(resident=res, cached=cached, holders=holders, wait=list(s.wait))

    # -- App. A.3 terms and the App. A.1 / A.4 estimator ---------------------
    def terms(self, s: State, x: int, d: int) -> Tuple[float, float, float, float, float]:
        """(c, switch, transfer, colocation, prefix) of stage x on device d in
        state s, each already weighted, benefits as positive amounts."""
        m = self.model[x]
        c = self.exec[m][d]
        sw = 0.0 if (s.resident[d] >> m) & 1 else self.ksw[m][d]
        tr, held = 0.0, 0
        for u in self.parents[x]:
            hu = s.holders.get(u, 0)
            if hu == 0:
                continue  # no output anywhere yet: no transfer, no colocation
            if (hu >> d) & 1:
                held += 1
            else:
                tr += self.sigma[u] * min(self.beta[i][d] for i in _devs(hu))
        colo = held / len(self.parents[x]) if self.parents[x] else 0.0
        pf = self.kpf * self.tokens[x] if self.group[x] != 0 and self.group[x] in s.cached[d] else 0.0
        return c, self.ls * sw, self.ltr * tr, self.lc * colo, self.lp * pf

    def c_hat(self, s: State, x: int, d: int) -> Tuple[float, float]:
        c, sw, tr, co, pf = self.terms(s, x, d)
        return c + sw + tr - co - pf, abs(c) + abs(sw) + abs(tr) + abs(co) + abs(pf)

    # -- horizon levels (Sec. 3.3) -------------------------------------------
    def horizon(self, v: int, H: int) -> List[Tuple[int, int]]:
        seen = {v}
        level = {v}
        out = []
        for h in range(1, H + 1):
            nxt = set()
            for x in level:
                nxt.update(c for c in self.children[x] if c not in seen)
            seen |= nxt
            out += [(x, h) for x in sorted(nxt)]
            level = nxt
        return out

    # -- immediate cost of S (App. A.3 terms; window reading of B_parallel) --
    def immediate(self, v: int, S) -> Tuple[float, float]:
        k = len(S)
        s = self.state
        best, best_mag = -np.inf, 0.0
        for d in S:
            c, sw, tr, co, pf = self.terms(s, v, d)
            q = self.lq * s.wait[d]
            t = q + c / k + sw + tr / k - pf / k - co
            if t > best:
                best, best_mag = t, abs(q) + abs(c / k) + abs(sw) + abs(tr / k) + abs(pf / k) + abs(co)
        gather = 0.0
        if k > 1:
            gather = min(sum(self.beta[d][p] * self.sigma[v] / k for d in S if d != p) for p in S)
        return best + self.ltr * gather, best_mag + abs(self.ltr * gather)

    def value_rows(self, s: State, U) -> List[Tuple[List[float], List[float]]]:
        """Per horizon stage: (c_hat over all devices, +inf where infeasible;
        magnitudes)."""
        rows = []
        for x, _ in U:
            vals, mags = [], []
            for d in range(self.D):
                if self.feasible(x, d):
                    a, m = self.c_hat(s, x, d)
                else:
                    a, m = np.inf, 0.0
                vals.append(a)
                mags.append(m)
            rows.append((vals, mags))
        return rows


def joint_minimum(weights: List[float], rows) -> float:
    """Smallest sum of weights[i] * rows[i][d_i] over every joint choice of
    devices (D^len(rows) of them), enumerated in full."""
    total = np.zeros(1)
    for g, (vals, _) in zip(weights, rows):
        total = (total[:, None] + g * np.asarray(vals, np.float64)[None, :]).ravel()
    return float(total.min())


def decomposed_value(inst: Instance, v: int, S, x: int, depth_child: bool) -> float:
    """The GPU kernel's rearrangement of one horizon stage's value under the
    placement S, from the current state only."""
    s = inst.state
    # row B(d') in s: v has no output yet, so it enters neither transfer nor colocation
    B = [inst.c_hat(s, x, d)[0] if inst.feasible(x, d) else np.inf for d in range(inst.D)]
    outside = np.inf
    for d in range(inst.D):
        if d in S:
            continue
        extra = 0.0
        if depth_child:  # v's output has to reach d from its cheapest shard device
            extra = inst.ltr * inst.sigma[v] * min(inst.beta[i][d] for i in S)
        outside = min(outside, B[d] + extra)
    inside = np.inf
    m, mv = inst.model[x], inst.model[v]
    for d in S:
        if not inst.feasible(x, d):
            continue
        delta = 0.0
        was = (s.resident[d] >> m) & 1
        now = (inst.load(s.resident[d], mv, d) >> m) & 1
        if was and not now:
            delta += inst.ls * inst.ksw[m][d]
        if now and not was:
            delta -= inst.ls * inst.ksw[m][d]
        g = inst.group[x]
        if g != 0 and g == inst.group[v] and g not in s.cached[d]:
            delta -= inst.lp * inst.kpf * inst.tokens[x]
        if depth_child:
            delta -= inst.lc / len(inst.parents[x])
        inside = min(inside, B[d] + delta)
    return min(outside, inside)


def score(w, params=None, H=None, max_shard=None, max_enum=1 << 16):
    """Score every candidate of every frontier stage of ``w`` from scratch.

    Returns (psi, mag, front) with ``front`` a list of (b, v, first candidate
    index), in the oracle's output order.  The horizon of a frontier stage is
    enumerated jointly when D^|U| <= max_enum; every stage's horizon value is
    also evaluated through ``decomposed_value``.  Raises AssertionError if the
    three evaluations disagree beyond 1e-12 relative."""
    H = int(w.H if H is None else H)
    ms = int(w.max_shard if max_shard is None else max_shard)
    psi, mag, front = [], [], []
    for b in range(w.B):
        inst = Instance(w, b, params or {})
        for v in inst.frontier():
            front.append((b, v, len(psi)))
            U = inst.horizon(v, H)
            weights = [inst.gamma ** h for _, h in U]
            for S in inst.candidates(v, ms):
                if not all(inst.feasible(v, d) for d in S):
                    psi.append(-np.inf)
                    mag.append(0.0)
                    continue
                j0, a0 = inst.immediate(v, S)
                post = inst.materialise(v, S)
                rows = inst.value_rows(post, U)
                tail, tail_mag = 0.0, 0.0
                for (x, h), g, (vals, mags) in zip(U, weights, rows):
                    best = min(vals)
                    first = vals.index(best)
                    tail += g * best
                    tail_mag += g * mags[first]
                    dec = decomposed_value(inst, v, S, x, h == 1)
                    assert abs(dec - best) <= 1e-12 * max(1.0, abs(best)), (b, v, S, x, dec, best)
                if U and inst.D ** len(U) <= max_enum:
                    joint = joint_minimum(weights, rows)
                    assert abs(joint - tail) <= 1e-12 * max(1.0, abs(tail)), (b, v, S, joint, tail)
                psi.append(-(j0 + tail))
                mag.append(a0 + tail_mag)
    return np.array(psi, np.float64), np.array(mag, np.float64), front


def tiny_cases(n_cases: int = 50):
    """Seeded tiny workloads for the brute-force checks: D <= 4, at most a
    dozen stages, windows, multi-device holders, running and committed
    stages, asymmetric beta.  Yields (seed, workload, H, max_shard)."""
    from paper_2605_07238_amd import synth
    for seed in range(n_cases):
        D = 2 + seed % 3
        H = 1 + seed % 3
        ms = 1 + seed % 4
        n = 7 + seed % 5
        w = synth.make_random_small(1000 + seed, B=2, n=n, D=D, M=3, K=2, H=H, max_shard=ms,
                                    p_edge=0.3 + 0.05 * (seed % 4), shard_frac=0.5,
                                    uniform_beta=(seed % 5 == 0), tight_caps=(seed % 2 == 0))
        yield seed, w, H, ms

