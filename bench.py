#!/usr/bin/env python3
"""Benchmark of horizon-aware candidate scoring on one MI355X.

One step = one pass of the scoring path over the whole batch with the packed
DAGs and state already resident in HBM: fate_score_topk, one launch that
scores every candidate of every frontier stage (immediate cost plus the
depth-H horizon) and ranks each stage's top-k; --two-calls times
fate_score_frontier then fate_topk instead.  Packing (host validation, layout and the
host-to-device copy) is done once before timing and reported separately.

The timed steps rotate through --copies independently packed copies of the
DAGs and the state (default 3, about 3 x 170 MB touched per launch on the
fork-join batch), so that no launch finds its inputs in the 256 MB Infinity
Cache that the previous launch filled; the same launches repeated on one copy
are timed as well and reported as the warm figure.

Prints one JSON line (rank 0, N=1):
  value          candidate-horizon evaluations per second over the timed steps;
                 one evaluation per feasible candidate and per (feasible
                 candidate, horizon descendant) pair
  roofline       the score kernel's algorithmic bytes per launch / its average
                 launch time over rotated copies (HIP events on the launch
                 stream) vs 8 TB/s HBM
  roofline_valu  VALU wave-instructions per launch (rocprofv3 SQ_INSTS_VALU in
                 the committed profile of the same kernel source) / the same
                 launch time vs 256 CUs x 4 SIMDs x 2.4 GHz / 4 cycles
  cpu_baseline   the fp64 oracle timed on this host's cores over the same batch
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

DEFAULT_WORKLOAD = "forkjoin-4096x1000-d16"
HBM_PEAK_GBS = 8000.0
# VALU issue: 256 CUs x 4 SIMDs x 2.4 GHz, one wave64 instruction per SIMD every
# 4 cycles (16 lanes wide), in G wave-instructions per second
VALU_PEAK_GIPS = 256 * 4 * 2.4 / 4.0
METRIC = "candidate-horizon evaluations/sec and achieved HBM GB/s (fraction of peak)"
# the score kernel and the header that fixes its launch geometry (slice length)
KERNEL_SRC = [os.path.join(ROOT, "paper_2605_07238_amd", "csrc", f) for f in ("fate_kernels.hip", "fate_internal.h")]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_sha() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SRC:
        h.update(open(path, "rb").read())
    return h.hexdigest()


def counted_work(w, pk, st, scores_host, H):
    """Exact evaluation count and algorithmic bytes of one score launch,
    counted from the packed structures (each needed byte once)."""
    import torch
    from paper_2605_07238_amd import fate

    fv, fb, co = fate.frontier_table(st)
    F = len(fv)
    h = pk.handle
    base = pk.buf.data_ptr()
    N = int(h.N)
    doff = pk.buf[h.desc_off - base:h.desc_off - base + 4 * (N + 1)].view(torch.int32).cpu().numpy().astype(np.int64)
    desc = pk.buf[h.desc - base:h.desc - base + 4 * int(h.n_desc)].view(torch.int32).cpu().numpy().astype(np.int64)
    desc &= 0xFFFFFFFF
    depth = desc >> 28
    wid = desc & ((1 << 28) - 1)
    # per frontier stage: entries with depth <= H
    lens = doff[fv + 1] - doff[fv]
    starts = doff[fv]
    idx = np.repeat(starts - np.concatenate([[0], np.cumsum(lens)[:-1]]), lens) + np.arange(int(lens.sum()))
    ent_depth = depth[idx]
    keep = ent_depth <= H
    seg = np.repeat(np.arange(F), lens)
    ndesc = np.bincount(seg[keep], minlength=F)
    feas = np.add.reduceat(np.isfinite(scores_host).astype(np.int64), co[:-1]) if F else np.zeros(0, np.int64)
    per_stage = feas * (1 + ndesc)
    n_eval = int(per_stage.sum())
    touched = np.unique(np.concatenate([fv, wid[idx][keep]]))
    npar = np.diff(w.par_off)
    inst = np.repeat(np.arange(w.B), np.diff(w.stage_off))
    par_global = w.par_idx.astype(np.int64) + w.stage_off[np.repeat(inst, npar)]
    pstart = w.par_off[touched]
    plen = npar[touched]
    pidx = np.repeat(pstart - np.concatenate([[0], np.cumsum(plen)[:-1]]), plen) + np.arange(int(plen.sum()))
    parents = np.unique(par_global[pidx])
    completed = int(np.count_nonzero(w.holders[parents] != 0))
    D, M, K = w.D, w.M, w.K
    active = len(np.unique(fb))
    nbytes = dict(
        frontier=8 * F + 4 * (F + 1),
        desc=8 * F + 4 * int(keep.sum()),
        records=32 * len(touched),
        parents=4 * int(plen.sum()) + 8 * len(parents) + 4 * completed,
        state=active * (8 * D + 8 * D * K + 4 * D + 4),
        cluster=8 * M * D + 4 * D * D + 8 * (2 * M + D),
        scores=4 * int(co[-1]),
    )
    return n_eval, int(sum(nbytes.values())), nbytes, dict(F=F, C=int(co[-1]), touched=len(touched),
                                                            desc_entries=int(keep.sum()),
                                                            per_stage=per_stage, stage_inst=fb)


def score_kernel(w, params) -> str:
    """Which scoring kernel the library launches for this batch (a label for
    the report): k_rows for frontiers of single-device candidates with a
    uniform off-diagonal beta, D <= 16, at most 32 models and no scoring
    variant; k_score otherwise."""
    off = w.beta[~np.eye(w.D, dtype=bool)]
    uniform = off.size == 0 or bool(np.all(off == off[0]))
    singles = min(int(np.max(w.shard_max)) if w.N else 1, int(w.max_shard), int(w.D)) <= 1
    variant = bool(w.params.get("topo_levels")) or params.lam_m != 0.0 or params.flags != 0
    return "k_rows" if uniform and singles and w.D <= 16 and w.M <= 32 and not variant else "k_score"


def read_counters(workload: str):
    """HBM traffic and VALU instructions per launch of the score kernel from
    the committed rocprofv3 counter runs, if they were taken on the current
    kernel source: (hbm bytes or None, SQ_INSTS_VALU or None)."""
    for kern in ("k_rows", "k_score"):
        hbm, valu = read_counter_file(os.path.join(ROOT, "profiles", "%s_%s_counters.txt" % (kern, workload)))
        if hbm is not None or valu is not None:
            return hbm, valu
    return None, None


def read_counter_file(path: str):
    if not os.path.exists(path):
        return None, None
    vals = {}
    valu = None
    for line in open(path):
        if line.startswith("counter SQ_INSTS_VALU"):
            try:
                valu = float(line.rsplit(":", 1)[1])
            except ValueError:
                valu = None
        elif ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256") != kernel_sha():
        return None, None
    try:
        hbm = float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        hbm = None
    return hbm, valu


def host_info():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return dict(cpu_model=model, nproc=os.cpu_count(), omp_num_threads=os.environ.get("OMP_NUM_THREADS"))


def cpu_per_core(w, H, counts, n_inst=64):
    """One oracle thread on the first ``n_inst`` instances (evaluations/s)."""
    from oracle import oracle
    n_inst = min(n_inst, w.B)
    sub = w.subset(list(range(n_inst)))
    evals = int(counts["per_stage"][counts["stage_inst"] < n_inst].sum())
    t = time.perf_counter()
    oracle.score(sub, H=H, threads=1)
    return evals / (time.perf_counter() - t), n_inst


def host_threads() -> int:
    """Host cores the oracle may use: OMP_NUM_THREADS when the environment
    sets it (the share of the host given to this process), else every core
    this process may run on."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        return int(env)
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:
        return max(1, os.cpu_count() or 1)


def cpu_baseline(w, H, min_seconds=10.0, max_passes=50):
    """Time the fp64 oracle over the whole batch, repeating passes until at
    least ``min_seconds`` of host work; returns (seconds per pass, passes, threads)."""
    from oracle import oracle
    threads = host_threads()
    passes, total = 0, 0.0
    while passes < max_passes and (total < min_seconds or passes == 0):
        t = time.perf_counter()
        oracle.score(w, H=H, threads=threads)
        total += time.perf_counter() - t
        passes += 1
    return total / passes, passes, threads


def edge_table(w):
    """Flat parent and child id of every edge of the batch."""
    npar = np.diff(w.par_off)
    child = np.repeat(np.arange(w.N, dtype=np.int64), npar)
    inst = np.repeat(np.arange(w.B, dtype=np.int64), np.diff(w.stage_off))
    parent = w.stage_off[inst[child]] + w.par_idx.astype(np.int64)
    return parent, child, npar


def commit_bytes(w, edges, front_v, sel, status, nF1, nS1, K, max_shard):
    """Algorithmic bytes of one commit-and-advance on the device, from the
    frontier it started from (front_v, its selections sel) and the statuses
    it left: each frontier slot's id, selection, record and children range
    are read; a completed stage's holders, status and finish are written and
    its parents' ids, holders, finish times and sizes read; for each child of
    a completed stage its id and record, its parents' ids, statuses, holders
    and sizes are read and its completed-parent entries and count written;
    each (instance, device) state word, free time and prefix slots are read
    and written; the new frontier goes through the workspace list (written,
    read) into its slots and candidate offsets, the slices are written, and
    the per-instance totals and offsets are written and read."""
    parent, child, npar = edges
    B, D = w.B, w.D
    done = np.zeros(w.N, bool)
    done[front_v[(sel >= 0) & (status[front_v] == 1)]] = True
    from_done = done[parent]
    kids = child[from_done]
    ndone = np.bincount(child[status[parent] == 1], minlength=w.N)
    nb = (len(front_v) * (8 + 4 + 32 + 8)
          + int(done.sum()) * (8 + 1 + 4) + int(npar[done].sum()) * (4 + 8 + 4 + 4)
          + len(kids) * (4 + 32 + 4) + int(npar[kids].sum()) * (4 + 1 + 8 + 4) + int(ndone[kids].sum()) * 16
          + 2 * B * D * (8 + 4 + 8 * K)
          + nF1 * (8 + 4 + 8 + 8 + (32 if max_shard > 1 and D > 1 else 0)) + 12 * nS1
          + B * (16 + 16 + 8 + 8 + 4 + 4) + 16)
    return nb


def sweep_grid(w, H_max=4):
    """The sensitivity grid of App. D.4 (Tab. 6: H = 0..4, then the state,
    locality and prefix weight groups at x0.5 and x1.5 with H = 4) and the
    scoring-side ablations of App. C.3 (locality off, prefix off, no windows)."""
    from paper_2605_07238_amd import fate
    b = dict(w.params)
    lm = float(b.get("lam_m", 0.0))
    sets, names = [], []
    for H in range(H_max + 1):
        sets.append(fate.make_params(w, H=H))
        names.append("H=%d" % H)
    for f in (0.5, 1.5):
        sets.append(fate.make_params(w, H=H_max, lam_s=b["lam_s"] * f, lam_m=lm * f))
        names.append("state x%g" % f)
        sets.append(fate.make_params(w, H=H_max, lam_tr=b["lam_tr"] * f, lam_c=b["lam_c"] * f))
        names.append("locality x%g" % f)
        sets.append(fate.make_params(w, H=H_max, lam_p=b["lam_p"] * f))
        names.append("prefix x%g" % f)
    sets.append(fate.make_params(w, H=H_max, lam_tr=0.0, lam_c=0.0))
    names.append("w/o locality")
    sets.append(fate.make_params(w, H=H_max, lam_p=0.0))
    names.append("w/o prefix")
    sets.append(fate.make_params(w, H=H_max, no_windows=1))
    names.append("w/o shard")
    return sets, names


def sweep_bench(w, k, reps, log):
    """One fate_score_sweep + fate_topk_sweep launch over the grid of
    sweep_grid, against the same sets scored and ranked one call at a time;
    every set's scores must match the single call bit for bit."""
    import torch
    from paper_2605_07238_amd import fate
    H_max = 4
    pk = fate.fate_pack_dags(w, H=H_max)
    st = fate.fate_pack_state(pk, w)
    sets, names = sweep_grid(w, H_max)
    P, nc = len(sets), st.n_cand
    out = torch.empty((P, max(1, nc)), dtype=torch.float32, device="cuda")
    idx = torch.empty((P, max(1, st.n_frontier), k), dtype=torch.int32, device="cuda")
    val = torch.empty_like(idx, dtype=torch.float32)
    one = torch.empty(max(1, nc), dtype=torch.float32, device="cuda")
    i1 = torch.empty((max(1, st.n_frontier), k), dtype=torch.int32, device="cuda")
    v1 = torch.empty_like(i1, dtype=torch.float32)
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def sweep():
        fate.fate_score_sweep(pk, st, sets, out=out)
        fate.fate_topk_sweep(st, out, k, idx=idx, val=val)

    def singles():
        for prm in sets:
            fate.fate_score_frontier(pk, st, prm, out=one)
            fate.fate_topk(st, one, k, idx=i1, val=v1)

    t = {}
    for name, fn in (("sweep", sweep), ("single_calls", singles)):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = mk(), mk()
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        t[name] = float(np.median(ts))
    sweep()
    torch.cuda.synchronize()
    same = True
    host = out.cpu().numpy()
    for p_, prm in enumerate(sets):
        fate.fate_score_frontier(pk, st, prm, out=one)
        torch.cuda.synchronize()
        same = same and np.array_equal(host[p_, :nc].view(np.uint32), one[:nc].cpu().numpy().view(np.uint32))
    evals, seen = 0, {}
    for p_, prm in enumerate(sets):  # the count depends on H and on which candidates are feasible
        key = (int(prm.H), int(prm.flags) & fate.FATE_NO_WINDOWS)
        if key not in seen:
            seen[key] = counted_work(w, pk, st, host[p_, :nc], int(prm.H))[0]
        evals += seen[key]
    log("sweep: %d sets in %.3f ms (one launch each for scores and top-k), %.3f ms as single calls"
        % (P, t["sweep"], t["single_calls"]))
    return dict(sets=names, H_packed=H_max, ms=t["sweep"], single_calls_ms=t["single_calls"],
                evals=evals, evals_per_s=evals / (t["sweep"] * 1e-3), bitwise_equal_to_single_calls=bool(same),
                kernels="k_rows for the sets without a variant and k_score for the others (grid rows = "
                        "parameter sets), then k_topk")


def planning_loop(w, pk, params, k, steps, log, full_plan=True, max_waves=2000):
    """Repeated planning steps on the device (Alg. 1): score the frontier and
    take each stage's top-k (one launch), build one planning wave (fate_plan_wave: each
    device at most once per instance), then commit it and advance the
    frontier (fate_commit_advance).  The first ``steps`` steps are timed one
    launch at a time with HIP events; with ``full_plan`` the loop then
    continues until every instance's frontier is empty and reports the whole
    plan's time and rate."""
    import torch
    from paper_2605_07238_amd import fate
    st = fate.fate_pack_state(pk, w, advance=True)
    cap = max(1, st.n_frontier)
    scores = torch.empty(max(1, st.n_cand), dtype=torch.float32, device="cuda")
    idx = torch.empty((cap, k), dtype=torch.int32, device="cuda")
    val = torch.empty((cap, k), dtype=torch.float32, device="cuda")
    sel = torch.empty(cap, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, fate.fate_commit_ws_size(pk, st)), dtype=torch.uint8, device="cuda")
    mk = lambda: torch.cuda.Event(enable_timing=True)
    edges = edge_table(w)

    def step():
        fate.fate_score_topk(pk, st, params, k, out=scores, idx=idx, val=val)
        fate.fate_plan_wave(st, idx, val, sel=sel)
        fate.fate_commit_advance(pk, st, sel, ws=ws)

    rows = []
    for i in range(steps):
        nF0 = st.counts()[0]
        if nF0 == 0:
            break
        front_v = fate.frontier_table(st)[0]  # the frontier the step starts from
        e = [mk() for _ in range(4)]
        # keep the device busy while the host enqueues the step, so that the
        # first event does not also time the host's call overhead
        torch.cuda._sleep(1000000)
        e[0].record()
        fate.fate_score_topk(pk, st, params, k, out=scores, idx=idx, val=val)
        e[1].record()
        fate.fate_plan_wave(st, idx, val, sel=sel)
        e[2].record()
        fate.fate_commit_advance(pk, st, sel, ws=ws)
        e[3].record()
        torch.cuda.synchronize()
        nF1, _, nS1, _ = st.counts()
        sel_h = sel[:nF0].cpu().numpy()
        cb = commit_bytes(w, edges, front_v, sel_h, fate.state_arrays(st)["status"], nF1, nS1, int(st.handle.K),
                          int(st.handle.max_shard))
        placed = int(np.count_nonzero(sel_h >= 0))
        row = dict(frontier=nF0, placed=placed, next_frontier=nF1, score_topk_ms=e[0].elapsed_time(e[1]),
                   plan_ms=e[1].elapsed_time(e[2]), commit_ms=e[2].elapsed_time(e[3]), commit_bytes=cb)
        if i == 0:
            row["warmup"] = True  # first launch of the plan and commit kernels (code loading); not in the means
        rows.append(row)
        log("planning step %d: frontier %d, placed %d -> %d; score + top-k %.4f, plan %.4f, commit %.4f ms%s"
            % (i, nF0, placed, nF1, row["score_topk_ms"], row["plan_ms"], row["commit_ms"],
               " (first launches: warm-up, not in the means)" if i == 0 else ""))
    out = dict(steps=rows, planner="fate_plan_wave (greedy wave, top-%d choices)" % k)
    timed = rows[1:] or rows  # the first launch of each kernel warms up
    if timed:
        cms = [r["commit_ms"] for r in timed]
        cbs = [r["commit_bytes"] for r in timed]
        achieved = float(np.mean(cbs)) / (float(np.mean(cms)) * 1e-3) / 1e9
        out.update(commit_ms_mean=float(np.mean(cms)), plan_ms_mean=float(np.mean([r["plan_ms"] for r in timed])),
                   step_ms_mean=float(np.mean([r["score_topk_ms"] + r["plan_ms"] + r["commit_ms"] for r in timed])),
                   commit_roofline={"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                    "frac": achieved / HBM_PEAK_GBS, "kernels": "fate_commit_advance (3 launches)"})
    if full_plan:
        # the rest of the plan, untimed per launch: one event pair around the whole loop
        n = len(rows)
        e0, e1 = mk(), mk()
        e0.record()
        while st.counts()[0] > 0 and n < max_waves:
            step()
            n += 1
        e1.record()
        torch.cuda.synchronize()
        rest_ms = e0.elapsed_time(e1)
        total_ms = rest_ms + sum(r["score_topk_ms"] + r["plan_ms"] + r["commit_ms"] for r in rows)
        arr = fate.state_arrays(st)
        planned = int(np.count_nonzero(arr["status"] == 1) - np.count_nonzero(w.status == 1))
        out["full_plan"] = dict(waves=n, ms=total_ms, stages_planned=planned,
                                stages_per_s=planned / (total_ms * 1e-3) if total_ms > 0 else None,
                                frontier_left=st.counts()[0],
                                note="time includes one host read of the frontier count per wave")
        log("full plan: %d waves, %d stages in %.2f ms (%.3g stages/s)"
            % (n, planned, total_ms, out["full_plan"]["stages_per_s"] or 0))
    return out


def record_fate_plan(w, params, k, log, max_waves=2000):
    """Run the device planning loop to the end and record the plan: each
    placed stage's devices (its holders in the planning state) and the wave it
    was placed in (the execution order key; commit order within a wave is by
    stage id).  Reads the frontier and the wave's selection each wave."""
    import torch
    from paper_2605_07238_amd import fate
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    cap = max(1, st.n_frontier)
    scores = torch.empty(max(1, st.n_cand), dtype=torch.float32, device="cuda")
    idx = torch.empty((cap, k), dtype=torch.int32, device="cuda")
    val = torch.empty((cap, k), dtype=torch.float32, device="cuda")
    sel = torch.empty(cap, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(1, fate.fate_commit_ws_size(pk, st)), dtype=torch.uint8, device="cuda")
    wave_of = np.full(w.N, -1, np.int64)
    t0 = time.perf_counter()
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
        wave_of[fv[s_host >= 0]] = waves
        fate.fate_commit_advance(pk, st, sel, ws=ws)
        waves += 1
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    holders = fate.state_arrays(st)["holders"]
    devices = np.where(wave_of >= 0, holders, 0).astype(np.uint64)
    log("recorded FATE plan: %d waves in %.2f s (with a host read of each wave's selection)" % (waves, dt))
    return devices, np.maximum(wave_of, 0), waves, dt


def sim_compare(w, params, k, log):
    """Execute the FATE plan and the round-robin and HEFT-style placements of
    the same batch (running / committed stages made pending) on the device
    and report the App. C.2 metrics, normalised by round robin as the paper
    does.  The baselines are built on the device too."""
    import dataclasses
    import torch
    from paper_2605_07238_amd import fate
    ws = dataclasses.replace(w, status=np.where(w.status == 1, 1, 0).astype(np.uint8))
    kpf = float(ws.params["kappa_prefix"])
    plans = {}
    fdev, ford = record_fate_plan(ws, params, k, log)[:2]
    pk = fate.fate_pack_dags(ws)
    st = fate.fate_pack_state(pk, ws)
    work = torch.empty(max(1, fate.fate_sim_ws_size(pk)), dtype=torch.uint8, device="cuda")
    plans["FATE"] = (torch.from_numpy(np.ascontiguousarray(fdev, np.uint64).view(np.int64)).cuda(),
                     torch.from_numpy(np.ascontiguousarray(ford, np.int64)).cuda())
    t = {}
    for name, pol in (("RoundRobin", fate.FATE_PLACE_ROUND_ROBIN), ("HEFT", fate.FATE_PLACE_HEFT)):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        plans[name] = fate.fate_place_baseline_device(pk, st, pol, kpf, ws=work)
        torch.cuda.synchronize()
        t[name] = time.perf_counter() - t0
    res, sim_s = {}, {}
    for name, (dev, order) in plans.items():
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res[name] = fate.fate_simulate_device(pk, st, dev, order, kpf, ws=work)
        sim_s[name] = time.perf_counter() - t0
    rr = res["RoundRobin"]
    ok = rr["makespan"] > 0
    out = {}
    for name, r in res.items():
        tasks = max(1, int(r["tasks"].sum()))
        out[name] = dict(
            NormMS=float(np.exp(np.mean(np.log(r["makespan"][ok] / rr["makespan"][ok])))),
            NormP95=float(np.exp(np.mean(np.log(r["p95"][ok] / rr["p95"][ok])))),
            XDevEdge=float(r["xdev_edges"].sum() / tasks), CacheScore=float(r["cache_hits"].sum() / tasks),
            ModelCont=float(r["model_cont"].sum() / tasks), tasks=int(r["tasks"].sum()),
            mean_makespan_s=float(r["makespan"].mean()), simulate_s=sim_s[name],
            simulated_tasks_per_s=float(r["tasks"].sum() / sim_s[name]))
        if name in t:
            out[name]["place_s"] = t[name]
        log("%-10s NormMS %.3f NormP95 %.3f XDevEdge %.3f CacheScore %.3f ModelCont %.3f (%d tasks)"
            % (name, out[name]["NormMS"], out[name]["NormP95"], out[name]["XDevEdge"], out[name]["CacheScore"],
               out[name]["ModelCont"], out[name]["tasks"]))
    out["note"] = ("synthetic execution model (fate_simulate_device, placements by fate_place_baseline_device); "
                   "running / committed stages made pending; "
                   "FATE = device planning loop with top-%d choices per stage" % k)
    return out


def describe(k):
    """Per-recipe sizes of one planning step (one JSON line each)."""
    import torch
    from paper_2605_07238_amd import fate, synth
    assert torch.cuda.is_available(), "--describe needs a GPU (evaluations count feasible candidates)"
    torch.cuda.set_device(0)
    fate.load()
    for name in synth.RECIPE_ORDER:
        w = synth.make_workload(name, workers=min(16, os.cpu_count() or 1))
        pk = fate.fate_pack_dags(w, H=w.H)
        st = fate.fate_pack_state(pk, w)
        params = fate.make_params(w, H=w.H)
        scores, idx, val = fate.fate_score_topk(pk, st, params, k)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
        for e0, e1 in evs:
            e0.record()
            fate.fate_score_topk(pk, st, params, k, out=scores, idx=idx, val=val)
            e1.record()
        torch.cuda.synchronize()
        ms = float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))
        n_eval, alg, parts, counts = counted_work(w, pk, st, scores[:st.n_cand].cpu().numpy(), w.H)
        alg += 8 * k * counts["F"]
        print(json.dumps(dict(workload=name, B=w.B, N=w.N, D=w.D, H=w.H, frontier_stages=counts["F"],
                              candidates=counts["C"], horizon_entries=counts["desc_entries"], evals=n_eval,
                              algorithmic_bytes=alg, fused_median_ms=ms, evals_per_s=n_eval / (ms * 1e-3),
                              achieved_gbs=alg / (ms * 1e-3) / 1e9, input_sha256=synth.fingerprint(w))), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--topk", type=int, default=4)
    ap.add_argument("--two-calls", action="store_true",
                    help="time fate_score_frontier then fate_topk instead of the one-launch fate_score_topk")
    ap.add_argument("--fused", action="store_true", help="the default: time fate_score_topk (one launch)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--planning-steps", type=int, default=6,
                    help="after the timed steps, run this many score / top-k / commit-and-advance planning steps "
                         "on a planning state and report them (0 = skip)")
    ap.add_argument("--no-sim", action="store_true",
                    help="skip the plan execution comparison (FATE plan vs round robin vs HEFT-style)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the parameter-sweep measurement (fate_score_sweep over the sensitivity grid)")
    ap.add_argument("--no-medians", action="store_true",
                    help="skip the extra median timings of the three launch variants (profiling runs)")
    ap.add_argument("--describe", action="store_true",
                    help="print |F|, candidates, horizon entries, evaluations, algorithmic bytes and the fused "
                         "kernel's median time for every recipe, then exit")
    ap.add_argument("--workload-file", default=None,
                    help="load the batch from this .npz if it exists, else generate it and save it there "
                         "(lets profiled runs skip the forked generator)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after timing, run one plain device copy of 512 MiB (counter calibration)")
    ap.add_argument("--copies", type=int, default=3,
                    help="independently packed copies of the DAGs and state the timed steps rotate through")
    ap.add_argument("--no-warm", action="store_true",
                    help="skip timing repeated launches on one copy (profiling runs: every launch rotates)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the scoring path has no cross-GPU step "
              "(instances shard across GPUs with no exchange); --gpus %d is not supported." % args.gpus,
              file=sys.stderr)
        sys.exit(2)

    from paper_2605_07238_amd import synth
    if args.describe:
        describe(args.topk)
        return
    t0 = time.perf_counter()
    if args.workload_file and os.path.exists(args.workload_file):
        w = synth.load_workload(args.workload_file)
        if w.name != args.workload:
            raise SystemExit("%s holds %s, not %s" % (args.workload_file, w.name, args.workload))
        log("loaded %s from %s: B=%d N=%d in %.1fs" % (w.name, args.workload_file, w.B, w.N, time.perf_counter() - t0))
    else:
        w = synth.make_workload(args.workload, workers=min(16, os.cpu_count() or 1))
        log("generated %s: B=%d N=%d in %.1fs" % (args.workload, w.B, w.N, time.perf_counter() - t0))
        if args.workload_file:
            synth.save_workload(w, args.workload_file)
            log("saved to %s" % args.workload_file)

    import torch
    from paper_2605_07238_amd import fate
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    fate.load()
    H = w.H
    R = max(1, args.copies)
    copies = []
    t_pack_dags = t_pack_state = 0.0
    for c in range(R):  # independently packed copies: separate device buffers, same contents
        t0 = time.perf_counter()
        pk_c = fate.fate_pack_dags(w, H=H)
        t_pack_dags = time.perf_counter() - t0
        t0 = time.perf_counter()
        st_c = fate.fate_pack_state(pk_c, w)
        t_pack_state = time.perf_counter() - t0
        copies.append(dict(
            pk=pk_c, st=st_c, scores=torch.empty(max(1, st_c.n_cand), dtype=torch.float32, device="cuda"),
            idx=torch.empty((max(1, st_c.n_frontier), args.topk), dtype=torch.int32, device="cuda"),
            val=torch.empty((max(1, st_c.n_frontier), args.topk), dtype=torch.float32, device="cuda")))
    pk, st = copies[0]["pk"], copies[0]["st"]
    scores, idx, val = copies[0]["scores"], copies[0]["idx"], copies[0]["val"]
    log("packed %d copies: dags %.2fs (%.1f MB), state %.2fs (%.1f MB) each; %d frontier stages, %d candidates"
        % (R, t_pack_dags, pk.handle.bytes / 1e6, t_pack_state, st.handle.bytes / 1e6, st.n_frontier, st.n_cand))
    params = fate.make_params(w, H=H)

    args.fused = not args.two_calls

    def score_call(c):
        x = copies[c]
        if args.fused:
            fate.fate_score_topk(x["pk"], x["st"], params, args.topk, out=x["scores"], idx=x["idx"], val=x["val"])
        else:
            fate.fate_score_frontier(x["pk"], x["st"], params, out=x["scores"])

    def topk_call(c):
        x = copies[c]
        if not args.fused:
            fate.fate_topk(x["st"], x["scores"], args.topk, idx=x["idx"], val=x["val"])

    for i in range(args.warmup):
        score_call(i % R)
        topk_call(i % R)
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)

    # Timed region: K steps, step i on copy i mod R.  Events on the launch
    # stream bracket the score kernel (the dominant one) and the whole step.
    K = args.steps
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def timed(n, rotate):
        ev = [(mk(), mk(), mk()) for _ in range(n)]
        torch.cuda.synchronize()
        t_a = time.perf_counter()
        for i in range(n):
            c = i % R if rotate else 0
            ev[i][0].record()
            score_call(c)
            ev[i][1].record()
            topk_call(c)
            ev[i][2].record()
        torch.cuda.synchronize()
        wall = (time.perf_counter() - t_a) * 1e3 / n
        return (wall, float(np.mean([a.elapsed_time(b) for a, b, _ in ev])),
                float(np.mean([a.elapsed_time(c) for a, _, c in ev])))

    ms_step, kern_ms, step_kern_ms = timed(K, rotate=True)
    log("timed %d steps over %d copies: %.4f ms/step; %s kernel %.4f ms, all kernels %.4f ms"
        % (K, R, ms_step, "fused score + top-k" if args.fused else "score", kern_ms, step_kern_ms))
    warm_kern_ms = None
    if not args.no_warm:
        warm_kern_ms = timed(K, rotate=False)[1]
        log("the same launches repeated on one copy (warm): kernel %.4f ms" % warm_kern_ms)

    def median_ms(fn, n=20):
        for i in range(3):
            fn(i % R)
        evs = [(mk(), mk()) for _ in range(n)]
        for i, (e0, e1) in enumerate(evs):
            e0.record()
            fn(i % R)
            e1.record()
        torch.cuda.synchronize()
        return float(np.median([e0.elapsed_time(e1) for e0, e1 in evs]))

    def fused_c(c):
        x = copies[c]
        fate.fate_score_topk(x["pk"], x["st"], params, args.topk, out=x["scores"], idx=x["idx"], val=x["val"])

    def score_c(c):
        x = copies[c]
        fate.fate_score_frontier(x["pk"], x["st"], params, out=x["scores"])

    def two_c(c):
        score_c(c)
        x = copies[c]
        fate.fate_topk(x["st"], x["scores"], args.topk, idx=x["idx"], val=x["val"])

    medians = None
    if not args.no_medians:
        medians = {"fused_score_topk": median_ms(fused_c), "score_only": median_ms(score_c),
                   "score_then_topk_two_calls": median_ms(two_c), "copies_rotated": R}
        score_call(0)  # leave this step's results in place for the counts below
        topk_call(0)
        torch.cuda.synchronize()
        log("medians (ms, rotated copies): %s" % json.dumps(medians))

    if args.copy_calibration:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 536870912 bytes read + written")

    scores_host = scores[:st.n_cand].cpu().numpy()
    n_eval, alg_bytes, parts, counts = counted_work(w, pk, st, scores_host, H)
    if args.fused:  # the top-k output belongs to the timed kernel
        parts["topk"] = 8 * args.topk * counts["F"]
        alg_bytes += parts["topk"]
    achieved = alg_bytes / (kern_ms * 1e-3) / 1e9
    traffic, valu_insts = read_counters(args.workload) if args.fused else (None, None)
    out = {
        "metric": METRIC,
        "value": n_eval / (ms_step * 1e-3),
        "unit": "evals/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": args.workload, "B": w.B, "stages_per_dag": int(np.diff(w.stage_off).max()),
            "D": w.D, "M": w.M, "K": w.K, "H": H, "max_shard": w.max_shard, "topk": args.topk,
            "frontier_stages": counts["F"], "candidates": counts["C"], "horizon_entries": counts["desc_entries"],
            "evals_per_step": n_eval, "step": "fused score + top-k" if args.fused else "score, then top-k",
            "kernel_ms": kern_ms, "step_kernels_ms": step_kern_ms, "copies_rotated": R,
            "kernel_ms_warm_one_copy": warm_kern_ms,
            "median_ms": medians,
            "input_sha256": synth.fingerprint(w),
            "pack_dags_s": t_pack_dags, "pack_state_s": t_pack_state,
            "algorithmic_bytes_per_launch": alg_bytes, "algorithmic_bytes_parts": parts,
        },
        "roofline": {
            "bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
            "kernel": score_kernel(w, params) + (" with the fused top-k" if args.fused else ""),
            "kernel_ms": kern_ms, "copies_rotated": R,
        },
    }
    # the roof the kernel meets first: VALU issue (SQ_INSTS_VALU of the profiled
    # kernel source over the same rotated launch time)
    valu_g = valu_insts / (kern_ms * 1e-3) / 1e9 if valu_insts else None
    out["roofline_valu"] = {
        "bound": "alu", "achieved": valu_g, "peak": VALU_PEAK_GIPS, "unit": "G VALU wave-instructions/s",
        "frac": valu_g / VALU_PEAK_GIPS if valu_g else None,
        "valu_insts_per_launch": valu_insts,
        "note": "peak = 256 CUs x 4 SIMDs x 2.4 GHz / 4 cycles per wave64 VALU instruction; instructions from "
                "profiles/%s_%s_counters.txt when its kernel source hash matches, else null"
                % (score_kernel(w, params), args.workload),
    }
    if args.planning_steps > 0:
        out["planning_loop"] = planning_loop(w, pk, params, args.topk, args.planning_steps, log)
    if not args.no_sweep:
        out["sweep"] = sweep_bench(w, args.topk, 5, log)
    if not args.no_sim:
        out["execution"] = sim_compare(w, params, args.topk, log)
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the host ...")
        dt, passes, threads = cpu_baseline(w, H)
        # the oracle evaluates the same frontier, candidates and horizon sets
        # (checked by the parity tests), so the evaluation count is shared
        out["cpu_baseline"] = {"value": n_eval / dt, "unit": "evals/s", "cores": threads, "kind": "oracle",
                               "sample": "all %d instances of %s, %d passes of %.2f s" % (w.B, args.workload, passes, dt)}
        per_core, n_inst = cpu_per_core(w, H, counts)
        out["cpu_baseline"].update(host_info())
        out["cpu_baseline"]["per_core_value"] = per_core
        out["cpu_baseline"]["per_core_sample"] = "1 thread, first %d instances" % n_inst
        log("oracle: %d passes, %.2f s each, %d threads; %.3g evals/s on one thread" % (passes, dt, threads, per_core))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
