"""Commit-and-advance on the GPU against the oracle (step 11), step by step.

Each step selects, for every frontier stage, the oracle's best candidate (so
no input of the oracle comes from the HIP path), commits it on the GPU with
fate_commit_advance and in the oracle with oracle.commit, and compares:
the state arrays (bit-exact, free times included: both sides sum them in
fp64 and round once to fp32), the rebuilt frontier, candidate offsets, slices and
completed-parent lists (against the host packer run on the oracle's new
state), and the next step's scores (within the scoring tolerance).
"""

import numpy as np
import pytest

import builders
from gpu_util import RTOL
from oracle import oracle
from paper_2605_07238_amd import fate, parity, synth

pytestmark = pytest.mark.gpu


def _sections(st):
    """Device planning-state sections as host arrays, cut to the current counts."""
    import torch
    h = st.handle
    nF, nC, nS, rej = st.counts()
    base = st.buf.data_ptr()

    def take(ptr, n, dt=np.uint32):
        off = ptr - base
        nb = n * np.dtype(dt).itemsize
        return st.buf[off:off + nb].cpu().numpy().view(dt).copy() if n else np.zeros(0, dt)

    N, B, E = int(h.N), int(h.B), int(h.n_done_edges)
    return dict(frontier=take(h.frontier, 2 * nF).reshape(nF, 2), cand_off=take(h.cand_off, nF + 1),
                slices=take(h.slices, 3 * nS).reshape(nS, 3), done_n=take(h.done_n, N),
                done=take(h.done, 4 * E).reshape(-1, 4), fr_off=take(h.fr_off, B + 1), order=take(h.order, B),
                slice=int(h.slice), counts=(nF, nC, nS, rej))


def _host_sections(pk, w):
    """The same sections from the host packer (fate_layout_state) for state w."""
    buf, h, hi = fate.fate_layout_state(pk.handle, w)
    base = buf.ctypes.data
    nF, nS, N = int(h.n_frontier), int(h.n_slices), int(h.N)

    def take(ptr, n, dt=np.uint32):
        return np.frombuffer(buf, dt, n, ptr - base).copy() if n else np.zeros(0, dt)

    B, E = int(h.B), int(h.n_done_edges)
    return dict(frontier=take(h.frontier, 2 * nF).reshape(nF, 2), cand_off=take(h.cand_off, nF + 1),
                slices=take(h.slices, 3 * nS).reshape(nS, 3), done_n=take(h.done_n, N),
                done=take(h.done, 4 * E).reshape(-1, 4), fr_off=take(h.fr_off, B + 1), order=take(h.order, B),
                slice=int(h.slice), n_cand=int(h.n_cand))


def check_order(order, fr_off):
    """The dispatch order: instances by size class of their frontier (eight
    classes in proportion to the largest frontier, largest first), each class
    in instance order."""
    n = np.diff(np.asarray(fr_off, np.int64))
    mx = int(n.max()) if len(n) else 0
    cls = 7 - np.minimum(7, n * 8 // (mx + 1))
    assert np.array_equal(order, np.argsort(cls, kind="stable")), "dispatch order"


def rows_candidate(pk, st):
    """Whether variant-free scoring of this batch may take a row kernel, which
    does not use the slices (single-device candidates, uniform beta, hop
    levels); whether its tables fit is the library's call."""
    h = pk.handle
    r = min(int(h.max_r), int(st.handle.max_shard), int(h.D))
    return bool(h.beta_uniform) and r <= 1 and h.levels != fate.FATE_LEVELS_TOPO


def check_slices(sec, may_keep_order):
    """Each instance's frontier range cut into pieces of the state's slice
    length, the instances in the dispatch order, or by id where a row kernel
    scores the batch."""
    fr, L = sec["fr_off"], sec["slice"]

    def cut(insts):
        want = [(b, f, min(int(fr[b + 1]), f + L)) for b in insts for f in range(int(fr[b]), int(fr[b + 1]), L)]
        return np.array(want, np.uint32).reshape(-1, 3)

    ok = np.array_equal(sec["slices"], cut(sec["order"]))
    if may_keep_order:
        ok = ok or np.array_equal(sec["slices"], cut(range(len(sec["order"]))))
    assert ok, "slices"


def pending_lists(sec, par_off, status):
    """Completed-parent counts of the pending stages, and their entries
    (holders, size) concatenated in stage order: each pending stage's list
    is the first done_n of its parent slots."""
    pend = np.flatnonzero(status == 0)
    cnt = sec["done_n"][pend].astype(np.int64)
    first = np.repeat(np.asarray(par_off, np.int64)[pend], cnt)
    within = np.arange(int(cnt.sum())) - np.repeat(np.cumsum(cnt) - cnt, cnt)
    return cnt, sec["done"][first + within, :3]


def _compare_state(st, w_ref, tau_ref, fin_ref=None):
    got = fate.state_arrays(st)
    if fin_ref is not None:  # planned finish of the completed stages, rounded once to fp32 on both sides
        done = w_ref.status == 1
        assert np.array_equal(got["finish"][done].view(np.uint32), np.asarray(fin_ref, np.float32)[done].view(np.uint32)), \
            "planned finish times"
    assert np.array_equal(got["resident"], w_ref.resident.reshape(got["resident"].shape)), "resident models"
    assert np.array_equal(got["prefix_cache"], w_ref.prefix_cache.reshape(got["prefix_cache"].shape)), "prefix slots"
    assert np.array_equal(got["holders"], w_ref.holders), "holders"
    assert np.array_equal(got["status"], w_ref.status), "status"
    # both sides sum a step's free times in fp64 and round once to the
    # state's fp32, so they agree bit for bit
    ref = np.asarray(tau_ref, np.float64).astype(np.float32).reshape(got["tau_free"].shape)
    assert np.array_equal(got["tau_free"].view(np.uint32), ref.view(np.uint32)), \
        "free times: max err %.3g" % np.abs(got["tau_free"].astype(np.float64) - ref).max()


def _compare_sections(pk, st, w_ref):
    dev = _sections(st)
    host = _host_sections(pk, w_ref)
    nF, nC, nS, _ = dev["counts"]
    assert np.array_equal(dev["frontier"], host["frontier"]), "frontier"
    assert np.array_equal(dev["cand_off"], host["cand_off"]), "candidate offsets"
    assert nC == host["n_cand"]
    assert np.array_equal(dev["fr_off"], host["fr_off"]), "frontier offsets per instance"
    for sec in (dev, host):
        check_order(sec["order"], sec["fr_off"])
        check_slices(sec, rows_candidate(pk, st))
    assert np.array_equal(dev["order"], host["order"]), "dispatch order"
    assert np.array_equal(dev["slices"], host["slices"]), "slices"
    dn, de = pending_lists(dev, w_ref.par_off, w_ref.status)
    hn, he = pending_lists(host, w_ref.par_off, w_ref.status)
    assert np.array_equal(dn, hn), "completed-parent counts"
    assert np.array_equal(de, he), "completed-parent entries"


def _score_and_check(pk, st, w, params=None):
    """GPU scores of the planning state against the oracle on state w."""
    import torch
    p = fate.make_params(w, **(params or {}))
    scores = fate.fate_score_frontier(pk, st, p)
    torch.cuda.synchronize()
    nF, nC = st.counts()[:2]
    ref = oracle.score(w, params=params)
    fv, fb, co = fate.frontier_table(st)
    flat = w.stage_off[ref["front_b"]] + ref["front_v"]
    assert np.array_equal(fv, flat), "frontier differs from the oracle's"
    assert np.array_equal(co, ref["cand_off"]), "candidate offsets differ from the oracle's"
    err, nbad, ninf = parity.compare(scores[:nC].cpu().numpy(), ref["psi"], ref["mag"], RTOL)
    assert ninf == 0 and nbad == 0, "scores after commit: %d bad (max rel err %.3g), %d -inf mismatches" % (
        nbad, err, ninf)
    return ref


def _run_steps(w, steps, params=None, sel_fn=None):
    import torch
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    cur = w
    fin = None
    ws = None
    for step in range(steps):
        print("[gpu] commit step", step, "frontier", st.counts()[0], flush=True)
        ref = _score_and_check(pk, st, cur, params)
        if len(ref["front_v"]) == 0:
            break
        idx, _ = oracle.topk(ref, 1)
        sel = idx[:, 0] if sel_fn is None else sel_fn(ref, idx[:, 0])
        nxt, tau, rej, fin = oracle.commit(cur, sel, fin=fin)
        d_sel = torch.from_numpy(np.ascontiguousarray(sel, np.int32)).cuda()
        ws = fate.fate_commit_advance(pk, st, d_sel, ws=ws)
        torch.cuda.synchronize()
        assert st.counts()[3] == rej, (st.counts(), rej)
        _compare_state(st, nxt, tau, fin)
        _compare_sections(pk, st, nxt)
        cur = nxt
    return pk, st, cur


CASES = [
    ("d4-windows", dict(seed=3, D=4, n=24, M=3, max_shard=3, shard_frac=0.6), 5),
    ("d6-nonuniform", dict(seed=5, D=6, n=24, M=5, K=3, max_shard=3, shard_frac=0.5), 6),
    ("d16-uniform", dict(seed=7, D=16, n=30, M=8, K=4, max_shard=4, shard_frac=0.5, uniform_beta=True), 6),
    ("d13-dense", dict(seed=11, D=13, n=30, M=6, p_edge=0.5, uniform_beta=True), 6),
    ("d40", dict(seed=13, D=40, n=20, M=6, K=2), 4),
    ("d2-chains", dict(seed=17, D=2, n=30, p_edge=0.2), 8),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_commit_steps_match_oracle(case):
    _, spec, steps = case
    spec = dict(spec)
    w = synth.make_random_small(spec.pop("seed"), B=3, H=2, **spec)
    _run_steps(w, steps)


def test_commit_until_done():
    """Commit best candidates until the frontier is empty: every pending stage
    completes and the planning state agrees with the oracle at every step."""
    w = synth.make_random_small(23, B=2, n=16, D=5, M=4, max_shard=2, shard_frac=0.4)
    pk, st, cur = _run_steps(w, 40)
    assert st.counts()[0] == 0
    # what stays pending waits on a running or committed stage, which the
    # planning state never completes
    npar = np.diff(w.par_off)
    inst = np.repeat(np.arange(w.B), np.diff(w.stage_off))
    for g in np.nonzero(cur.status == 0)[0]:
        pars = w.par_idx[w.par_off[g]:w.par_off[g + 1]].astype(np.int64) + w.stage_off[inst[g]]
        assert npar[g] > 0 and np.any(cur.status[pars] != 1), g
    assert np.count_nonzero(cur.status == 1) > np.count_nonzero(w.status == 1)


@pytest.mark.parametrize("name", ["shards-1024x500-d16", "forkjoin-4096x1000-d16", "layered-1024x200-d8"])
def test_commit_recipes(name):
    w = synth.make_workload(name, B=12)
    _run_steps(w, 3)


def test_commit_several_chunks_per_instance():
    """80 fork-join instances of 1,000 stages: frontiers of more than 64
    slots (several apply chunks per instance) and instance starts at every
    alignment of the bitmap words."""
    w = synth.make_workload("forkjoin-4096x1000-d16", B=80)
    fb, _, _ = oracle.frontier(w)
    assert np.bincount(fb, minlength=w.B).max() > 64
    _run_steps(w, 2)


def _sized_workload(name, sizes, seed=5):
    """Instances of the recipe with the given stage counts."""
    rc = synth.RECIPES[name]
    cluster = synth.make_cluster(rc, seed)
    K, ms = synth.COMMON["K"], synth.COMMON["max_shard"]
    insts = [synth._gen_instance(dict(rc, n=n), cluster, seed, b, K, ms) for b, n in enumerate(sizes)]
    return synth._assemble(name + "+sizes", rc, cluster, insts, K, ms)


def test_commit_large_instance_bitmap_in_workspace():
    """An instance of more than 32,768 stages moves every instance's frontier
    bitmap from LDS to the workspace; the next instances start at offsets
    that are not multiples of 32."""
    w = _sized_workload("forkjoin-4096x1000-d16", [33005, 997, 1003])
    pk = fate.fate_pack_dags(w)
    assert pk.handle.max_stages == 33005 and w.stage_off[1] % 32 != 0
    _run_steps(w, 3)


def _join_spec():
    """100 roots (two apply chunks), joins whose parents sit in both chunks,
    a stage with 20 parents (three batches of parent loads), a child of a
    root and a join, and an empty instance in between."""
    D, M = 4, 2
    parents = [[] for _ in range(100)]
    parents += [[3, 70, 99], list(range(20, 40)), [5, 100], [64], [0, 63, 64, 65]]
    n = len(parents)
    big = dict(parents=parents, model=[v % M for v in range(n)], elig=[(1 << D) - 1] * n,
               prefix_hash=[0 if v % 3 else 17 + v % 2 for v in range(n)], prefix_tokens=[200.0] * n,
               out_bytes=[1e6 * (1 + v % 7) for v in range(n)], status=[0] * n, holders=[0] * n,
               resident=[1, 2, 0, 3], tau_free=[0.0, 0.5, 1.0, 0.25], t_now=0.0)
    empty = dict(parents=[], model=[], elig=[], out_bytes=[], status=[], holders=[],
                 resident=[0] * D, tau_free=[0.0] * D, t_now=0.0)
    small = dict(parents=[[], [0], [0, 1]], model=[0, 1, 0], elig=[15, 15, 15], out_bytes=[1e6, 2e6, 3e6],
                 status=[1, 0, 0], holders=[2, 0, 0], resident=[1, 0, 0, 2], tau_free=[0.0] * D, t_now=0.0)
    return dict(D=D, M=M, K=2, exec=[[1.0, 1.5, 2.0, 0.5]] * M, switch_s=[[0.3] * D] * M, weight_gb=[10, 20],
                cap_gb=[40, 40, 25, 40], beta=[[0.0 if i == j else 2e-10 for j in range(D)] for i in range(D)],
                max_shard=1, instances=[big, empty, small])


def test_commit_joins_across_chunks():
    w = builders.from_spec(_join_spec(), H=2)
    pk, st, cur = _run_steps(w, 4)
    # the joins joined the frontier once all their parents completed
    assert (cur.status[100:105] == 1).sum() > 0


def test_commit_more_instances_than_one_scan_batch():
    """4,100 instances: the one-workgroup scan takes two batches of 4,096."""
    w = synth.make_random_small(31, B=4100, n=6, D=4, M=3, max_shard=2, shard_frac=0.3, p_edge=0.4)
    _run_steps(w, 2)


def test_commit_partial_and_rejected_selections():
    """Stages left at -1 stay pending; out-of-range and infeasible selections
    are rejected, counted and change nothing."""
    w = synth.make_random_small(29, B=3, n=24, D=6, M=4, max_shard=3, shard_frac=0.6)

    def mixed(ref, best):
        sel = best.copy()
        co = ref["cand_off"]
        for f in range(len(sel)):
            if f % 3 == 1:
                sel[f] = -1
            elif f % 3 == 2:
                sel[f] = int(co[f + 1] - co[f]) + 5  # past the last candidate
        return sel

    _run_steps(w, 3, sel_fn=mixed)


def test_commit_top_k_array_as_selection():
    """A [F, k] selection array is read through its first column."""
    import torch
    w = synth.make_random_small(31, B=2, n=20, D=8, M=4, max_shard=2, shard_frac=0.5)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    ref = oracle.score(w)
    idx, _ = oracle.topk(ref, 1)
    sel2 = np.full((len(idx), 3), 12345, np.int32)  # columns 1, 2 would be rejected if read
    sel2[:, 0] = idx[:, 0]
    nxt, tau, rej, fin = oracle.commit(w, idx[:, 0])
    fate.fate_commit_advance(pk, st, torch.from_numpy(sel2).cuda())
    torch.cuda.synchronize()
    assert st.counts()[3] == 0
    _compare_state(st, nxt, tau, fin)


def test_commit_nothing_keeps_everything():
    import torch
    w = synth.make_random_small(37, B=2, n=20, D=6, M=4, max_shard=3, shard_frac=0.5)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    before = _sections(st)
    arrays = fate.state_arrays(st)
    sel = torch.full((max(1, st.counts()[0]),), -1, dtype=torch.int32, device="cuda")
    fate.fate_commit_advance(pk, st, sel)
    torch.cuda.synchronize()
    after = _sections(st)
    for k in ("frontier", "cand_off", "slices", "done_n", "done", "fr_off"):
        assert np.array_equal(before[k], after[k]), k
    now = fate.state_arrays(st)
    for k, v in arrays.items():
        assert np.array_equal(v, now[k]), k


def test_planning_state_scores_and_topk_match_plain_state():
    """Scoring, top-k and the fused call on a planning state write the same
    bits as on the plainly packed state."""
    import torch
    w = synth.make_random_small(41, B=3, n=24, D=8, M=4, max_shard=3, shard_frac=0.5)
    pk = fate.fate_pack_dags(w)
    st0 = fate.fate_pack_state(pk, w)
    st1 = fate.fate_pack_state(pk, w, advance=True)
    p = fate.make_params(w)
    nF, nC = st0.n_frontier, st0.n_cand
    assert st1.counts()[:2] == (nF, nC)
    s0 = fate.fate_score_frontier(pk, st0, p)
    s1 = fate.fate_score_frontier(pk, st1, p)
    i0, v0 = fate.fate_topk(st0, s0, 3)
    i1, v1 = fate.fate_topk(st1, s1, 3)
    f1, fi1, fv1 = fate.fate_score_topk(pk, st1, p, 3)
    torch.cuda.synchronize()
    assert np.array_equal(s0[:nC].cpu().numpy().view(np.uint32), s1[:nC].cpu().numpy().view(np.uint32))
    assert np.array_equal(i0.cpu().numpy(), i1[:nF].cpu().numpy())
    assert np.array_equal(v0.cpu().numpy().view(np.uint32), v1[:nF].cpu().numpy().view(np.uint32))
    assert np.array_equal(i0.cpu().numpy(), fi1[:nF].cpu().numpy())
    assert np.array_equal(s0[:nC].cpu().numpy().view(np.uint32), f1[:nC].cpu().numpy().view(np.uint32))


def _lowest_feasible(ref, best):
    """Each stage's lowest-numbered candidate with a finite score."""
    co, psi = ref["cand_off"], ref["psi"]
    sel = best.copy()
    for f in range(len(sel)):
        fin = np.nonzero(np.isfinite(psi[co[f]:co[f + 1]]))[0]
        sel[f] = fin[0] if len(fin) else -1
    return sel


def test_commit_long_device_chains_wrap_prefix_rows():
    """Every stage takes its lowest feasible candidate, so the low devices get
    long chains of placements in one step; with more prefix groups than
    slots the rows wrap many times, and they start with holes."""
    import dataclasses
    w = synth.make_random_small(43, B=2, n=120, D=4, M=5, K=3, max_shard=2, p_edge=0.03, shard_frac=0.3)
    rng = np.random.default_rng(43)
    pool = rng.integers(1, 1 << 62, size=7).astype(np.uint64)
    ph = pool[rng.integers(0, 7, size=w.N)]
    ph[rng.random(w.N) < 0.1] = 0
    pc = w.prefix_cache.copy().reshape(-1)
    pc[::4] = 0  # holes before filled slots
    w = dataclasses.replace(w, prefix_hash=ph, prefix_cache=pc.reshape(w.prefix_cache.shape))
    assert np.count_nonzero(np.isfinite(oracle.score(w)["psi"])) > 40
    _run_steps(w, 4, sel_fn=_lowest_feasible)


def test_commit_inputs_ready_scenario():
    """The two-step hand scenario where shards wait for their parents' outputs
    (window shards waiting for half a transfer, a busy device, a remote parent
    in the next step), on the GPU."""
    import builders
    import scenarios
    sc = scenarios.COMMIT_READY
    w = builders.from_spec(sc["spec"], H=1)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    import torch
    for step in sc["steps"]:
        assert st.counts()[0] == len(step["sel"])
        fate.fate_commit_advance(pk, st, torch.tensor(step["sel"], dtype=torch.int32, device="cuda"))
        torch.cuda.synchronize()
        got = fate.state_arrays(st)
        assert got["tau_free"].reshape(-1).tolist() == step["tau"], got["tau_free"]
        done = got["status"] == 1
        assert got["finish"][done].tolist() == [x for x, dn in zip(step["fin"], done) if dn], got["finish"]
