"""Property-based checks of the host packer on random tiny DAGs (hypothesis,
no GPU): the frontier, candidate counts, breadth-first horizon lists and
completed-parent lists that fate_layout_dags / fate_layout_state build must
equal what the oracle and the independent checker in tests/brute.py derive
from the same inputs (Sec. 2 ready set; App. A.1 implementation frontier;
Sec. 3.3 horizon levels; App. A.2 shard windows)."""

import numpy as np
from hypothesis import HealthCheck, given, settings, strategies as st

import brute
import builders
from oracle import oracle
from paper_2605_07238_amd import fate


@st.composite
def dag_specs(draw):
    D = draw(st.integers(1, 6))
    M = draw(st.integers(1, 4))
    K = draw(st.integers(0, 3))
    n = draw(st.integers(1, 14))
    weight = [draw(st.integers(2, 12)) for _ in range(M)]
    cap = [draw(st.integers(8, 30)) for _ in range(D)]
    for m in range(M):  # every model fits some device
        if not any(weight[m] <= c for c in cap):
            cap[draw(st.integers(0, D - 1))] = weight[m]
    full = (1 << D) - 1
    parents, model, elig, shard, status, holders, groups = [], [], [], [], [], [], []
    for v in range(n):
        ps = sorted(draw(st.sets(st.integers(0, v - 1), max_size=min(4, v)))) if v else []
        m = draw(st.integers(0, M - 1))
        fits = sum(1 << d for d in range(D) if weight[m] <= cap[d])
        e = draw(st.integers(1, full)) | (1 << draw(st.sampled_from([d for d in range(D) if (fits >> d) & 1])))
        done_ok = all(status[p] == 1 for p in ps)
        # completed and running stages need completed parents (else FATE_ESTATE)
        s = draw(st.sampled_from([0, 1, 2, 3] if done_ok else [0, 3]))
        parents.append(ps)
        model.append(m)
        elig.append(e & full)
        shard.append(draw(st.integers(1, 4)))
        status.append(s)
        holders.append(draw(st.integers(1, full)) if s == 1 else 0)
        groups.append(draw(st.sampled_from([0, 11, 12, 13])))
    inst = dict(parents=parents, model=model, elig=elig, shard_max=shard, prefix_hash=groups,
                prefix_tokens=[100.0] * n, out_bytes=[1e6 * (1 + v) for v in range(n)], status=status, holders=holders,
                resident=[draw(st.integers(0, (1 << M) - 1)) for _ in range(D)],
                prefix_cache=[[draw(st.sampled_from([0, 11, 12, 99])) for _ in range(max(K, 1))][:K] or [] for _ in range(D)],
                tau_free=[1.0] * D, t_now=0.5)
    if K == 0:
        inst["prefix_cache"] = [[] for _ in range(D)]
    spec = dict(D=D, M=M, K=K, exec=[[1.0] * D for _ in range(M)], switch_s=[[0.5] * D for _ in range(M)],
                weight_gb=weight, cap_gb=cap, beta=[[0.0 if i == j else 1e-10 for j in range(D)] for i in range(D)],
                max_shard=draw(st.integers(1, 4)), instances=[inst])
    H = draw(st.integers(0, 4))
    return spec, H


@settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(dag_specs())
def test_host_layouts_match_independent_derivations(case):
    spec, H = case
    w = builders.from_spec(spec, H=H)
    buf, hd, _ = fate.fate_layout_dags(w)
    sbuf, hs, _ = fate.fate_layout_state(hd, w)
    base, sbase = buf.ctypes.data, sbuf.ctypes.data
    N, nF = int(hd.N), int(hs.n_frontier)

    def take(b, ptr, n, dt=np.uint32):
        return np.frombuffer(b, dt, n, ptr - (base if b is buf else sbase)).astype(np.int64) if n else np.zeros(0, np.int64)

    # frontier and candidate offsets against the oracle
    fb, fv, _ = oracle.frontier(w)
    front = take(sbuf, hs.frontier, 2 * nF).reshape(nF, 2)
    assert front[:, 0].tolist() == (w.stage_off[fb] + fv).tolist()
    assert front[:, 1].tolist() == fb.tolist()
    inst = brute.Instance(w, 0, {})
    co = take(sbuf, hs.cand_off, nF + 1)
    assert [len(inst.candidates(int(v), w.max_shard)) for v in fv] == np.diff(co).tolist()
    # horizon lists: breadth-first levels 1..H, each stage once at its minimum distance, by (depth, id)
    doff = take(buf, hd.desc_off, N + 1)
    desc = take(buf, hd.desc, int(hd.n_desc))
    for v in range(N):
        ent = desc[doff[v]:doff[v + 1]]
        got = [(int(e >> 28), int(e & ((1 << 28) - 1))) for e in ent]
        want = sorted((h, x) for x, h in inst.horizon(v, H))
        assert got == want, (v, got, want)
    # children lists: every stage that names v as a parent, ascending
    E = int(hd.E)
    ch_off = take(buf, hd.ch_off, N + 1)
    ch_idx = take(buf, hd.ch_idx, E)
    for v in range(N):
        assert ch_idx[ch_off[v]:ch_off[v + 1]].tolist() == [c for c in range(N) if v in inst.parents[c]], v
    # frontier offsets per instance, and the dispatch order
    assert take(sbuf, hs.fr_off, w.B + 1).tolist() == [0, nF]
    assert take(sbuf, hs.order, w.B).tolist() == [0]
    # completed-parent lists of pending stages, in parent order, in the
    # first of each stage's parent slots
    done_n = take(sbuf, hs.done_n, N)
    done = np.frombuffer(sbuf, np.uint32, 4 * E, hs.done - sbase).reshape(-1, 4)
    for v in range(N):
        rows = done[w.par_off[v]:w.par_off[v] + done_n[v]]
        assert done_n[v] <= w.par_off[v + 1] - w.par_off[v]
        want = [u for u in inst.parents[v] if inst.status[u] == 1] if inst.status[v] == 0 else []
        hold = [int(r[0]) | (int(r[1]) << 32) for r in rows]
        assert hold == [int(w.holders[u]) for u in want], (v, hold, want)
        assert np.array_equal(rows[:, 2].view(np.float32), np.asarray([w.out_bytes[u] for u in want], np.float32))


@settings(max_examples=60, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(dag_specs(), st.data())
def test_running_or_completed_stage_under_a_pending_parent_is_rejected(case, data):
    spec, H = case
    inst = spec["instances"][0]
    kids = [v for v, ps in enumerate(inst["parents"]) if ps]
    if not kids:
        return
    v = data.draw(st.sampled_from(kids))
    p = data.draw(st.sampled_from(inst["parents"][v]))
    inst["status"][p], inst["holders"][p] = 0, 0
    s = data.draw(st.sampled_from([1, 2]))
    inst["status"][v], inst["holders"][v] = s, (1 if s == 1 else 0)
    w = builders.from_spec(spec, H=H)
    _, hd, _ = fate.fate_layout_dags(w)
    try:
        fate.fate_layout_state(hd, w)
    except fate.FateError as e:
        assert e.status == -6
    else:
        raise AssertionError("inconsistent state accepted")
