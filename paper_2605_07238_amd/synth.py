"""Seeded synthetic workloads for horizon-aware candidate scoring.

This module only builds inputs: workflow DAG batches, the cluster tables, and
an execution state reached by a random partial execution.  It holds none of
the scoring arithmetic.  Both the HIP path and the fp64 oracle consume what it
returns, and neither is imported here.

Every recipe mirrors the shape of the paper's setting (Sec. 2 stage tuple and
state s_t; App. C.1 proxies for runtime, switch, transfer and prefix reuse):

* Stage v carries a model id m(v), an eligible-device bitmask A(v), a shard cap
  R(v), a shared-prefix group hash grp(v) (0 = none) with its token length,
  and an output size sigma(v) in bytes.
* The cluster carries the base runtime table exec[m][d] (seconds), the switch
  cost table kappa_switch[m][d] (seconds), model weights W(m) and device
  capacities (integer bytes), and the transfer coefficient beta[i][j] (s/byte).
* The state is what a random partial execution of 30% of the stages leaves
  behind: resident-model bitmasks per device, a K-slot prefix ring per device,
  device bitmasks holding each completed stage's output, device free times and
  the current time t = min_d tau_d.  Every stage that is ready afterwards is
  pending, so the frontier is the whole ready set.  On request
  (``mark_statuses``) a share of the ready stages is marked running or
  committed instead, which exercises the frontier rule of App. A.1 at scale.

Randomness: instance b of a recipe draws from
``Generator(PCG64(SeedSequence([seed, b])))`` so its data does not depend on
the batch size; the cluster tables draw from ``SeedSequence([seed, 2**31])``.

The partial execution evicts resident models uniformly at random when a load
overflows a device; this is a property of the synthetic history only.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Sequence

import numpy as np

GB = 1_000_000_000
MIB = float(1 << 20)
LINK_BYTES_PER_S = 25e9

# Stage status codes (App. A.1: completed, running, committed are tracked).
PENDING, COMPLETED, RUNNING, COMMITTED = 0, 1, 2, 3

DEFAULT_PARAMS = dict(
    lam_q=1.0, lam_s=1.0, lam_tr=1.0, lam_c=0.1, lam_p=1.0,
    kappa_prefix=1e-4, gamma=0.5,
)


@dataclasses.dataclass
class Workload:
    """A batch of B DAG instances plus cluster tables and an execution state."""

    name: str
    D: int
    M: int
    K: int
    H: int
    max_shard: int
    # cluster
    exec: np.ndarray          # float32 [M, D]
    switch_s: np.ndarray      # float32 [M, D]
    weight_bytes: np.ndarray  # int64 [M]
    cap_bytes: np.ndarray     # int64 [D]
    beta: np.ndarray          # float32 [D, D]
    # DAG batch (flat; stage ids inside an instance are topological)
    stage_off: np.ndarray     # int64 [B+1]
    par_off: np.ndarray       # int64 [N+1]
    par_idx: np.ndarray       # int32 [E] instance-local parent ids
    model: np.ndarray         # int32 [N]
    elig: np.ndarray          # uint64 [N]
    shard_max: np.ndarray     # int32 [N]
    prefix_hash: np.ndarray   # uint64 [N]
    prefix_tokens: np.ndarray  # float32 [N]
    out_bytes: np.ndarray     # float32 [N]
    # state
    resident: np.ndarray      # uint64 [B, D]
    prefix_cache: np.ndarray  # uint64 [B, D, K]
    holders: np.ndarray       # uint64 [N]
    status: np.ndarray        # uint8 [N]
    tau_free: np.ndarray      # float32 [B, D]
    t_now: np.ndarray         # float32 [B]
    params: Dict[str, float] = dataclasses.field(default_factory=lambda: dict(DEFAULT_PARAMS))

    @property
    def B(self) -> int:
        return int(self.stage_off.shape[0] - 1)

    @property
    def N(self) -> int:
        return int(self.stage_off[-1])

    def instance(self, b: int) -> "Workload":
        """Return instance b alone as a batch of one (copies)."""
        return self.subset([b])

    def subset(self, idx: Sequence[int]) -> "Workload":
        """Return the instances listed in idx, in that order, as a new batch."""
        idx = [int(i) for i in idx]
        so = self.stage_off
        lens = [int(so[i + 1] - so[i]) for i in idx]
        stage_off = np.zeros(len(idx) + 1, np.int64)
        stage_off[1:] = np.cumsum(lens)
        sel = np.concatenate([np.arange(so[i], so[i + 1]) for i in idx]) if idx else np.zeros(0, np.int64)
        sel = sel.astype(np.int64)
        npar = (self.par_off[1:] - self.par_off[:-1])[sel]
        par_off = np.zeros(len(sel) + 1, np.int64)
        par_off[1:] = np.cumsum(npar)
        par_idx = np.concatenate(
            [self.par_idx[self.par_off[g]:self.par_off[g + 1]] for g in sel]
        ).astype(np.int32) if len(sel) else np.zeros(0, np.int32)
        return dataclasses.replace(
            self,
            stage_off=stage_off, par_off=par_off, par_idx=par_idx,
            model=self.model[sel].copy(), elig=self.elig[sel].copy(),
            shard_max=self.shard_max[sel].copy(), prefix_hash=self.prefix_hash[sel].copy(),
            prefix_tokens=self.prefix_tokens[sel].copy(), out_bytes=self.out_bytes[sel].copy(),
            resident=self.resident[idx].copy(), prefix_cache=self.prefix_cache[idx].copy(),
            holders=self.holders[sel].copy(), status=self.status[sel].copy(),
            tau_free=self.tau_free[idx].copy(), t_now=self.t_now[idx].copy(),
            params=dict(self.params),
        )

    def parents(self, b: int, v: int) -> np.ndarray:
        g = int(self.stage_off[b]) + v
        return self.par_idx[self.par_off[g]:self.par_off[g + 1]]


# ---------------------------------------------------------------------------
# Recipes.  Names describe the workload; sizes follow the benchmark settings.
# ---------------------------------------------------------------------------

RECIPES: Dict[str, dict] = {
    # B=1 layered DAG, 6 layers x 4, fan-in 1..3 from the previous layer.
    "tiny-layered-1x24-d4": dict(
        B=1, topology="layered_fixed", layers=6, width=4, fanin=(1, 3),
        D=4, speeds=(1.0,), M=3, wgb=(2.0, 16.0), capgb=40.0,
        sigma_mu=math.log(MIB), sigma_s=1.0, p_inherit=0.5, L_fresh=None,
        shard_frac=0.0, H=2, seed=0),
    # B=1024 layered DAGs, 200 stages, widths 10..20, fan-in 1..4.
    "layered-1024x200-d8": dict(
        B=1024, topology="layered", n=200, widths=(10, 20), fanin=(1, 4),
        D=8, speeds=(1.0, 1.5), M=6, wgb=(4.0, 70.0), capgb=192.0,
        sigma_mu=math.log(MIB), sigma_s=1.0, p_inherit=0.5, L_fresh=None,
        shard_frac=0.0, H=3, seed=1),
    # B=4096 fork-join DAGs, 1000 stages: fan-out <=32, join fan-in <=8.
    "forkjoin-4096x1000-d16": dict(
        B=4096, topology="forkjoin", n=1000, fanout=32, group=8, rounds=5,
        D=16, speeds=(1.0,), M=12, wgb=(4.0, 140.0), capgb=288.0,
        sigma_mu=math.log(MIB), sigma_s=1.0, p_inherit=0.7, L_fresh=(128, 4096),
        shard_frac=0.0, H=3, seed=2),
    # B=1024 layered DAGs, 500 stages, 30% shardable over 2..4 devices.
    "shards-1024x500-d16": dict(
        B=1024, topology="layered", n=500, widths=(10, 20), fanin=(1, 4),
        D=16, speeds=(1.0,), M=12, wgb=(4.0, 140.0), capgb=288.0,
        sigma_mu=math.log(MIB), sigma_s=1.0, p_inherit=0.5, L_fresh=None,
        shard_frac=0.3, H=3, seed=3),
    # B=256 power-law DAGs, 10000 stages, out-degree ~ k^-2.1 on [1, 64].
    "powerlaw-256x10000-d64": dict(
        B=256, topology="powerlaw", n=10000, alpha=2.1, kmax=64, window=256, incap=16,
        D=64, speeds=(1.0, 1.5, 2.25, 3.375), M=32, wgb=(4.0, 140.0), capgb=288.0,
        sigma_mu=math.log(4 * MIB), sigma_s=1.5, p_inherit=0.6, L_fresh=None,
        shard_frac=0.0, H=4, seed=4),
}

# Short aliases in benchmark order.
RECIPE_ORDER = list(RECIPES.keys())

COMMON = dict(K=16, max_shard=4, exec_frac=0.3, p_running=0.10, p_committed=0.05,
              p_all_eligible=0.85, p_dev_eligible=0.6, L_default=1024.0)


# ---------------------------------------------------------------------------
# Topologies: each returns a list of parent lists with parent id < child id.
# ---------------------------------------------------------------------------

def _layered_fixed(rng, layers: int, width: int, fanin) -> List[List[int]]:
    parents: List[List[int]] = []
    for layer in range(layers):
        for _ in range(width):
            if layer == 0:
                parents.append([])
                continue
            prev0 = (layer - 1) * width
            k = int(rng.integers(fanin[0], fanin[1] + 1))
            k = min(k, width)
            ps = rng.choice(width, size=k, replace=False) + prev0
            parents.append(sorted(int(p) for p in ps))
    return parents


def _layered(rng, n: int, widths, fanin) -> List[List[int]]:
    parents: List[List[int]] = []
    prev_lo, prev_hi = 0, 0  # previous layer [lo, hi)
    while len(parents) < n:
        w = int(rng.integers(widths[0], widths[1] + 1))
        w = min(w, n - len(parents))
        lo = len(parents)
        for _ in range(w):
            if lo == 0:
                parents.append([])
                continue
            pw = prev_hi - prev_lo
            k = min(int(rng.integers(fanin[0], fanin[1] + 1)), pw)
            ps = rng.choice(pw, size=k, replace=False) + prev_lo
            parents.append(sorted(int(p) for p in ps))
        prev_lo, prev_hi = lo, lo + w
    return parents


def _forkjoin(rng, n: int, fanout: int, group: int, rounds: int) -> List[List[int]]:
    """One source; each round every join stage forks 1..fanout workers, then
    consecutive worker groups of 1..group stages join into one aggregator.
    Rounds repeat (at least ``rounds`` of them, more only if n is not yet
    reached) and generation stops at exactly n stages."""
    parents: List[List[int]] = [[]]
    joins = [0]
    r = 0
    while len(parents) < n:
        r += 1
        workers: List[int] = []
        for a in joins:
            c = int(rng.integers(1, fanout + 1))
            for _ in range(c):
                if len(parents) >= n:
                    break
                parents.append([a])
                workers.append(len(parents) - 1)
        if len(parents) >= n:
            break
        new_joins: List[int] = []
        i = 0
        while i < len(workers) and len(parents) < n:
            g = int(rng.integers(1, group + 1))
            grp = workers[i:i + g]
            i += g
            parents.append(list(grp))
            new_joins.append(len(parents) - 1)
        joins = new_joins if new_joins else joins
    return parents


def _powerlaw(rng, n: int, alpha: float, kmax: int, window: int, incap: int) -> List[List[int]]:
    ks = np.arange(1, kmax + 1, dtype=np.float64)
    p = ks ** (-alpha)
    p /= p.sum()
    outdeg = rng.choice(np.arange(1, kmax + 1), size=n, p=p)
    indeg = [0] * n
    parents: List[List[int]] = [[] for _ in range(n)]
    draws = rng.integers(0, 1 << 30, size=int(outdeg.sum()) * 3 + 64).tolist()
    di = 0
    nd = len(draws)
    for v in range(n - 1):
        wsz = min(window, n - 1 - v)
        k = min(int(outdeg[v]), wsz)
        chosen = set()
        tries = 0
        while len(chosen) < k and tries < 4 * k + 16:
            if di >= nd:
                draws = rng.integers(0, 1 << 30, size=1024).tolist()
                di, nd = 0, len(draws)
            t = v + 1 + draws[di] % wsz
            di += 1
            tries += 1
            if t in chosen or indeg[t] >= incap:
                continue
            chosen.add(t)
            indeg[t] += 1
        for t in chosen:
            parents[t].append(v)
    for lst in parents:
        lst.sort()
    return parents


# ---------------------------------------------------------------------------
# Cluster tables
# ---------------------------------------------------------------------------

def make_cluster(rc: dict, seed: int):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 2 ** 31])))
    D, M = rc["D"], rc["M"]
    ncls = len(rc["speeds"])
    speed = np.array([rc["speeds"][d * ncls // D] for d in range(D)], np.float64)
    exec_ = rng.lognormal(0.0, 0.5, size=(M, D)) / speed[None, :]
    wlo, whi = rc["wgb"]
    weight = np.rint(rng.uniform(wlo, whi, size=M) * GB).astype(np.int64)
    cap = np.full(D, int(round(rc["capgb"] * GB)), np.int64)
    switch = np.repeat((weight.astype(np.float64) / LINK_BYTES_PER_S)[:, None], D, axis=1)
    beta = np.full((D, D), 1.0 / LINK_BYTES_PER_S, np.float64)
    np.fill_diagonal(beta, 0.0)
    return (exec_.astype(np.float32), switch.astype(np.float32), weight, cap,
            beta.astype(np.float32))


# ---------------------------------------------------------------------------
# One instance
# ---------------------------------------------------------------------------

def _fresh_hash(rng) -> int:
    return int(rng.integers(1, np.iinfo(np.uint64).max, dtype=np.uint64, endpoint=True))


def _bits(mask: int) -> List[int]:
    out = []
    while mask:
        low = mask & -mask
        out.append(low.bit_length() - 1)
        mask ^= low
    return out


def _gen_instance(rc: dict, cluster, seed: int, b: int, K: int, max_shard: int, mark_statuses: bool = False):
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b])))
    D, M = rc["D"], rc["M"]
    exec_, switch, weight, cap, _beta = cluster
    topo = rc["topology"]
    if topo == "layered_fixed":
        parents = _layered_fixed(rng, rc["layers"], rc["width"], rc["fanin"])
    elif topo == "layered":
        parents = _layered(rng, rc["n"], rc["widths"], rc["fanin"])
    elif topo == "forkjoin":
        parents = _forkjoin(rng, rc["n"], rc["fanout"], rc["group"], rc["rounds"])
    elif topo == "powerlaw":
        parents = _powerlaw(rng, rc["n"], rc["alpha"], rc["kmax"], rc["window"], rc["incap"])
    else:
        raise ValueError(topo)
    n = len(parents)

    fits = [sum(1 << d for d in range(D) if weight[m] <= cap[d]) for m in range(M)]
    model = rng.integers(0, M, size=n).astype(np.int32)
    full = (1 << D) - 1
    elig = np.zeros(n, np.uint64)
    u_all = rng.random(n)
    for v in range(n):
        if u_all[v] < COMMON["p_all_eligible"]:
            e = full
        else:
            e = 0
            while (e & fits[model[v]]) == 0:
                e = int(sum(1 << d for d in range(D) if rng.random() < COMMON["p_dev_eligible"]))
        elig[v] = np.uint64(e)
    shard = np.ones(n, np.int32)
    if rc["shard_frac"] > 0:
        sel = rng.random(n) < rc["shard_frac"]
        shard[sel] = rng.integers(2, 5, size=int(sel.sum()))
    sigma = rng.lognormal(rc["sigma_mu"], rc["sigma_s"], size=n).astype(np.float32)

    hashes = [0] * n
    toks = np.zeros(n, np.float32)
    for v in range(n):
        if parents[v] and rng.random() < rc["p_inherit"]:
            p0 = parents[v][0]
            hashes[v] = hashes[p0]
            toks[v] = toks[p0]
        else:
            hashes[v] = _fresh_hash(rng)
            if rc["L_fresh"] is None:
                toks[v] = COMMON["L_default"]
            else:
                lo, hi = rc["L_fresh"]
                toks[v] = float(rng.integers(lo, hi + 1))

    # initial residency: each model on each device w.p. 0.5, then random trim
    resident = [0] * D
    used = [0] * D
    for d in range(D):
        for m in range(M):
            if rng.random() < 0.5:
                resident[d] |= 1 << m
                used[d] += int(weight[m])
        while used[d] > cap[d]:
            ms = _bits(resident[d])
            m = ms[int(rng.integers(len(ms)))]
            resident[d] &= ~(1 << m)
            used[d] -= int(weight[m])

    ring = [[0] * K for _ in range(D)]
    ring_pos = [0] * D
    tau = [0.0] * D
    status = np.zeros(n, np.uint8)
    holders = np.zeros(n, np.uint64)
    children: List[List[int]] = [[] for _ in range(n)]
    remaining = [len(p) for p in parents]
    for v in range(n):
        for p in parents[v]:
            children[p].append(v)
    ready = [v for v in range(n) if remaining[v] == 0]

    n_exec = int(math.ceil(COMMON["exec_frac"] * n))
    for _ in range(n_exec):
        if not ready:
            break
        i = int(rng.integers(len(ready)))
        v = ready[i]
        ready[i] = ready[-1]
        ready.pop()
        m = int(model[v])
        feas = int(elig[v]) & fits[m]
        devs = _bits(feas)
        k = 1
        r = min(int(shard[v]), max_shard)
        S: List[int]
        if r > 1:
            k = int(rng.integers(1, r + 1))
        if k > 1:
            starts = [s for s in range(D - k + 1)
                      if all((feas >> (s + j)) & 1 for j in range(k))]
            if starts:
                s0 = starts[int(rng.integers(len(starts)))]
                S = list(range(s0, s0 + k))
            else:
                k = 1
        if k == 1:
            S = [devs[int(rng.integers(len(devs)))]]
        hm = 0
        for d in S:
            hm |= 1 << d
            loaded = 0.0
            if not (resident[d] >> m) & 1:
                resident[d] |= 1 << m
                used[d] += int(weight[m])
                loaded = float(switch[m, d])
                while used[d] > cap[d]:
                    ms = [x for x in _bits(resident[d]) if x != m]
                    x = ms[int(rng.integers(len(ms)))]
                    resident[d] &= ~(1 << x)
                    used[d] -= int(weight[x])
            h = hashes[v]
            if h != 0 and h not in ring[d]:
                ring[d][ring_pos[d]] = h
                ring_pos[d] = (ring_pos[d] + 1) % K if K > 0 else 0
            tau[d] += float(exec_[m, d]) / k + loaded
        holders[v] = np.uint64(hm)
        status[v] = COMPLETED
        for c in children[v]:
            remaining[c] -= 1
            if remaining[c] == 0:
                ready.append(c)
    # on request, some ready stages are already running or committed
    # (App. A.1); these draws come last, so nothing else depends on them
    if mark_statuses:
        for v in ready:
            u = rng.random()
            if u < COMMON["p_running"]:
                status[v] = RUNNING
            elif u < COMMON["p_running"] + COMMON["p_committed"]:
                status[v] = COMMITTED

    tau_a = np.array(tau, np.float32)
    t_now = np.float32(tau_a.min()) if D else np.float32(0)
    res_a = np.array(resident, dtype=np.uint64)
    cache_a = np.array(ring, dtype=np.uint64).reshape(D, K)
    par_lens = np.array([len(p) for p in parents], np.int64)
    par_flat = np.array([p for ps in parents for p in ps], np.int32)
    return dict(
        n=n, par_lens=par_lens, par_flat=par_flat, model=model, elig=elig, shard=shard,
        hash=np.array(hashes, dtype=np.uint64), toks=toks, sigma=sigma,
        resident=res_a, cache=cache_a, holders=holders, status=status,
        tau=tau_a, t_now=t_now,
    )


def _assemble(name: str, rc: dict, cluster, insts: List[dict], K: int, max_shard: int) -> Workload:
    exec_, switch, weight, cap, beta = cluster
    B = len(insts)
    ns = np.array([it["n"] for it in insts], np.int64)
    stage_off = np.zeros(B + 1, np.int64)
    stage_off[1:] = np.cumsum(ns)
    par_lens = np.concatenate([it["par_lens"] for it in insts]) if B else np.zeros(0, np.int64)
    par_off = np.zeros(len(par_lens) + 1, np.int64)
    par_off[1:] = np.cumsum(par_lens)
    cat = lambda key, dt: (np.concatenate([it[key] for it in insts]).astype(dt)
                           if B else np.zeros(0, dt))
    D = rc["D"]
    return Workload(
        name=name, D=D, M=rc["M"], K=K, H=rc["H"], max_shard=max_shard,
        exec=exec_, switch_s=switch, weight_bytes=weight, cap_bytes=cap, beta=beta,
        stage_off=stage_off, par_off=par_off, par_idx=cat("par_flat", np.int32),
        model=cat("model", np.int32), elig=cat("elig", np.uint64), shard_max=cat("shard", np.int32),
        prefix_hash=cat("hash", np.uint64), prefix_tokens=cat("toks", np.float32),
        out_bytes=cat("sigma", np.float32),
        resident=(np.stack([it["resident"] for it in insts]) if B else np.zeros((0, D), np.uint64)),
        prefix_cache=(np.stack([it["cache"] for it in insts]) if B else np.zeros((0, D, K), np.uint64)),
        holders=cat("holders", np.uint64), status=cat("status", np.uint8),
        tau_free=(np.stack([it["tau"] for it in insts]) if B else np.zeros((0, D), np.float32)),
        t_now=np.array([it["t_now"] for it in insts], np.float32),
    )


def _gen_range(args):
    name, rc, seed, lo, hi, K, max_shard, mark = args
    cluster = make_cluster(rc, seed)
    return [_gen_instance(rc, cluster, seed, b, K, max_shard, mark) for b in range(lo, hi)]


def make_workload(name: str, B: Optional[int] = None, instances: Optional[Sequence[int]] = None,
                  seed: Optional[int] = None, workers: int = 1, mark_statuses: bool = False) -> Workload:
    """Build a recipe's workload.

    ``B`` truncates the batch to its first B instances; ``instances`` picks
    explicit instance ids (their data equals that of the full batch).
    ``workers`` > 1 spreads instance generation over forked processes.
    ``mark_statuses`` marks 10% of the ready stages running and 5% committed
    (off for the recipes themselves: their frontier is every ready stage).
    """
    rc = dict(RECIPES[name])
    seed = rc["seed"] if seed is None else seed
    K, max_shard = COMMON["K"], COMMON["max_shard"]
    ids = list(instances) if instances is not None else list(range(rc["B"] if B is None else B))
    cluster = make_cluster(rc, seed)
    if workers > 1 and len(ids) > 64 and instances is None:
        import multiprocessing as mp
        chunks = []
        step = max(1, (len(ids) + workers * 4 - 1) // (workers * 4))
        for lo in range(0, len(ids), step):
            chunks.append((name, rc, seed, lo, min(len(ids), lo + step), K, max_shard, mark_statuses))
        ctx = mp.get_context("fork")
        with ctx.Pool(workers) as pool:
            parts = pool.map(_gen_range, chunks)
        insts = [it for part in parts for it in part]
    else:
        insts = [_gen_instance(rc, cluster, seed, b, K, max_shard, mark_statuses) for b in ids]
    return _assemble(name + ("+statuses" if mark_statuses else ""), rc, cluster, insts, K, max_shard)


# ---------------------------------------------------------------------------
# Small random workloads for property and edge-case tests
# ---------------------------------------------------------------------------

def make_random_small(seed: int, B: int = 2, n: int = 12, D: int = 4, M: int = 3, K: int = 4,
                      H: int = 2, max_shard: int = 3, p_edge: float = 0.3,
                      shard_frac: float = 0.4, uniform_beta: bool = False,
                      tight_caps: bool = True, p_no_prefix: float = 0.2) -> Workload:
    """Random tiny DAGs with eligibility holes, capacity-blocked models,
    non-uniform (asymmetric) beta, shardable stages, multi-device holders,
    zero prefix groups, and running/committed stages."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 7919])))
    exec_ = rng.uniform(0.2, 3.0, size=(M, D)).astype(np.float32)
    switch = rng.uniform(0.0, 2.0, size=(M, D)).astype(np.float32)
    weight = rng.integers(2, 20, size=M).astype(np.int64) * GB
    if tight_caps:
        cap = rng.integers(15, 40, size=D).astype(np.int64) * GB
        # keep every model placeable on at least one device
        for m in range(M):
            if not (weight[m] <= cap).any():
                cap[int(rng.integers(D))] = int(weight[m])
    else:
        cap = np.full(D, 40 * GB, np.int64)
    if uniform_beta:
        beta = np.full((D, D), 3e-10, np.float32)
    else:
        beta = rng.uniform(1e-10, 9e-10, size=(D, D)).astype(np.float32)
    np.fill_diagonal(beta, 0.0)
    fits = [sum(1 << d for d in range(D) if weight[m] <= cap[d]) for m in range(M)]
    insts = []
    for b in range(B):
        parents = []
        for v in range(n):
            ps = [u for u in range(v) if rng.random() < p_edge]
            if len(ps) > 5:
                ps = sorted(rng.choice(ps, size=5, replace=False).tolist())
            parents.append(ps)
        model = rng.integers(0, M, size=n).astype(np.int32)
        elig = np.zeros(n, np.uint64)
        for v in range(n):
            e = 0
            while (e & fits[model[v]]) == 0:
                e = int(sum(1 << d for d in range(D) if rng.random() < 0.7))
            elig[v] = np.uint64(e)
        shard = np.where(rng.random(n) < shard_frac, rng.integers(2, 5, size=n), 1).astype(np.int32)
        sigma = rng.lognormal(math.log(5e8), 1.0, size=n).astype(np.float32)
        hashes = [0] * n
        toks = rng.integers(100, 3000, size=n).astype(np.float32)
        pool = [int(x) for x in rng.integers(1, 1 << 62, size=3)]
        for v in range(n):
            u = rng.random()
            hashes[v] = 0 if u < p_no_prefix else pool[int(rng.integers(3))]
        resident = np.zeros(D, np.uint64)
        for d in range(D):
            used = 0
            r = 0
            for m in rng.permutation(M):
                if rng.random() < 0.6 and used + weight[m] <= cap[d]:
                    r |= 1 << int(m)
                    used += int(weight[m])
            resident[d] = np.uint64(r)
        cache = np.zeros((D, K), np.uint64)
        for d in range(D):
            for s in range(K):
                u = rng.random()
                if u < 0.4:
                    cache[d, s] = np.uint64(pool[int(rng.integers(3))])
                elif u < 0.6:
                    cache[d, s] = np.uint64(int(rng.integers(1, 1 << 62)))
        # completed set: a random down-closed prefix in topological order
        status = np.zeros(n, np.uint8)
        holders = np.zeros(n, np.uint64)
        for v in range(n):
            if all(status[p] == COMPLETED for p in parents[v]) and rng.random() < 0.45:
                status[v] = COMPLETED
                hm = 0
                while hm == 0:
                    hm = int(sum(1 << d for d in range(D) if rng.random() < 0.35))
                holders[v] = np.uint64(hm)
        for v in range(n):
            if status[v] == PENDING and all(status[p] == COMPLETED for p in parents[v]):
                u = rng.random()
                if u < 0.15:
                    status[v] = RUNNING
                elif u < 0.25:
                    status[v] = COMMITTED
        tau = rng.uniform(0.0, 3.0, size=D).astype(np.float32)
        t_now = np.float32(rng.uniform(0.0, 2.0))
        insts.append(dict(
            n=n, par_lens=np.array([len(p) for p in parents], np.int64),
            par_flat=np.array([p for ps in parents for p in ps], np.int32),
            model=model, elig=elig, shard=shard, hash=np.array(hashes, np.uint64), toks=toks,
            sigma=sigma, resident=resident, cache=cache, holders=holders, status=status,
            tau=tau, t_now=t_now))
    rc = dict(D=D, M=M, H=H)
    w = _assemble(f"random-small-{seed}", rc, (exec_, switch, weight, cap, beta), insts, K, max_shard)
    return w


# ---------------------------------------------------------------------------
# Saving a generated batch (so a process that must not fork can reuse one)
# ---------------------------------------------------------------------------

_ARRAY_FIELDS = [f.name for f in dataclasses.fields(Workload)
                 if f.name not in ("name", "D", "M", "K", "H", "max_shard", "params")]


def save_workload(w: Workload, path: str) -> None:
    """Write ``w`` as an uncompressed .npz (plain arrays plus a JSON header)."""
    import json
    meta = dict(name=w.name, D=w.D, M=w.M, K=w.K, H=w.H, max_shard=w.max_shard, params=w.params)
    np.savez(path, _meta=np.array(json.dumps(meta)), **{k: getattr(w, k) for k in _ARRAY_FIELDS})


def load_workload(path: str) -> Workload:
    """Read a batch written by :func:`save_workload` (no pickled objects)."""
    import json
    with np.load(path, allow_pickle=False) as z:
        meta = json.loads(str(z["_meta"]))
        arrays = {k: z[k] for k in _ARRAY_FIELDS}
    return Workload(name=meta["name"], D=int(meta["D"]), M=int(meta["M"]), K=int(meta["K"]), H=int(meta["H"]),
                    max_shard=int(meta["max_shard"]), params=dict(meta["params"]), **arrays)


def fingerprint(w: Workload) -> str:
    """SHA-256 over a batch's arrays and header (identifies the generated input)."""
    import hashlib
    import json
    h = hashlib.sha256()
    h.update(json.dumps(dict(name=w.name, D=w.D, M=w.M, K=w.K, H=w.H, max_shard=w.max_shard,
                             params=w.params), sort_keys=True).encode())
    for k in _ARRAY_FIELDS:
        a = np.ascontiguousarray(getattr(w, k))
        h.update(k.encode())
        h.update(str(a.dtype).encode())
        h.update(memoryview(a).cast("B"))
    return h.hexdigest()
