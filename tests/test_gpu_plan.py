"""Frontier planning wave on the GPU (fate_plan_wave) against the oracle's
step 12, on the same choice arrays: seeded synthetic choices over real
frontiers, and the oracle's own top-k rounded to float32 (so no input of the
oracle comes from the HIP path).  Selections must match exactly; chained with
fate_commit_advance they must drive the planning state as the oracle's
plan-and-commit does."""

import numpy as np
import pytest

import scenarios
from oracle import oracle
from paper_2605_07238_amd import fate, synth

pytestmark = pytest.mark.gpu


def _n_cands(w, g):
    r = max(1, min(int(w.shard_max[g]), int(w.max_shard), int(w.D)))
    return int(w.D) + sum(int(w.D) - k + 1 for k in range(2, r + 1))


def synthetic_choices(w, k, seed, ties=True, p_pad=0.2, p_bad=0.05):
    """Seeded choices per frontier slot: distinct candidate indices of the
    stage, scores on a coarse grid (ties) or continuous, descending per slot,
    with padding (-1, -inf) and a few out-of-range indices."""
    rng = np.random.default_rng(seed)
    front_b, front_v, f_off = oracle.frontier(w)
    F = len(front_v)
    idx = np.full((F, k), -1, np.int32)
    val = np.full((F, k), -np.inf, np.float32)
    n_cand = np.zeros(F, np.int64)
    for f in range(F):
        g = int(w.stage_off[front_b[f]]) + int(front_v[f])
        nc = _n_cands(w, g)
        n_cand[f] = nc
        m = min(k, nc)
        js = rng.choice(nc, size=m, replace=False)
        vs = rng.normal(-3.0, 1.0, size=m)
        if ties:
            vs = np.round(vs * 2) / 2
        vs = np.sort(vs)[::-1]
        for r in range(m):
            if rng.random() < p_pad:
                break
            idx[f, r] = js[r] if rng.random() >= p_bad else nc + 1000  # past every candidate
            val[f, r] = vs[r]
    return f_off, n_cand, idx, val


def _gpu_plan(w, idx, val, advance=False):
    import torch
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=advance)
    d_idx = torch.from_numpy(np.ascontiguousarray(idx)).cuda()
    d_val = torch.from_numpy(np.ascontiguousarray(val)).cuda()
    sel = fate.fate_plan_wave(st, d_idx, d_val)
    torch.cuda.synchronize()
    return sel.cpu().numpy()


CASES = [
    ("d4", lambda: synth.make_random_small(71, B=4, n=30, D=4, M=3, max_shard=3, shard_frac=0.6, p_edge=0.1), 4),
    ("d7-k1", lambda: synth.make_random_small(72, B=3, n=30, D=7, M=4, max_shard=4, shard_frac=0.5, p_edge=0.1), 1),
    ("d16", lambda: synth.make_random_small(73, B=3, n=40, D=16, M=6, max_shard=4, shard_frac=0.5, p_edge=0.05), 8),
    ("d64", lambda: synth.make_random_small(74, B=2, n=40, D=64, M=6, max_shard=2, p_edge=0.05), 4),
    ("d16-k64-overflow", lambda: synth.make_random_small(75, B=2, n=80, D=16, M=6, max_shard=4, shard_frac=0.7,
                                                         p_edge=0.0), 64),
    ("forkjoin", lambda: synth.make_workload("forkjoin-4096x1000-d16", B=16), 4),
    ("shards", lambda: synth.make_workload("shards-1024x500-d16", B=16), 4),
]


@pytest.mark.parametrize("ties", [True, False])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_plan_synthetic_choices(case, ties):
    name, make, k = case
    w = make()
    for seed in range(3):
        f_off, n_cand, idx, val = synthetic_choices(w, k, 100 + seed, ties=ties)
        print("[gpu] plan", name, "k", k, "seed", seed, "frontier", len(idx), flush=True)
        want, n = oracle.plan_wave(w.D, f_off, n_cand, idx, val)
        got = _gpu_plan(w, idx, val)
        assert np.array_equal(got, want), np.nonzero(got != want)[0][:10]
        assert n == int(np.count_nonzero(got >= 0))
    if name == "d16-k64-overflow":  # one instance holds more choices than the LDS stages
        assert int(np.max(np.diff(f_off))) * k > 1024


@pytest.mark.parametrize("case", CASES[:4], ids=[c[0] for c in CASES[:4]])
def test_plan_from_oracle_topk(case):
    name, make, k = case
    w = make()
    ref = oracle.score(w)
    idx, val = oracle.topk(ref, k)
    val32 = val.astype(np.float32)
    _, _, f_off = oracle.frontier(w)
    want, _ = oracle.plan_wave(w.D, f_off, np.diff(ref["cand_off"]), idx, val32)
    got = _gpu_plan(w, idx, val32)
    assert np.array_equal(got, want)


def test_plan_then_commit_loop():
    """Plan and commit, step after step, on the GPU's planning state; the
    choices come from the oracle's top-k of the oracle's state at each step."""
    import torch
    from test_gpu_commit import _compare_state, _compare_sections
    w = synth.make_random_small(81, B=3, n=30, D=6, M=4, K=3, max_shard=3, shard_frac=0.5, p_edge=0.2)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    cur = w
    fin = None
    k = 4
    ws = None
    for step in range(12):
        ref = oracle.score(cur)
        if len(ref["front_v"]) == 0:
            break
        idx, val = oracle.topk(ref, k)
        val32 = val.astype(np.float32)
        _, _, f_off = oracle.frontier(cur)
        want, n = oracle.plan_wave(cur.D, f_off, np.diff(ref["cand_off"]), idx, val32)
        assert n > 0
        # the planning state holds its frontier at capacity: pad the choices
        cap = st.n_frontier
        pidx = np.full((cap, k), -1, np.int32)
        pval = np.full((cap, k), -np.inf, np.float32)
        pidx[:len(idx)] = idx
        pval[:len(idx)] = val32
        sel = fate.fate_plan_wave(st, torch.from_numpy(pidx).cuda(), torch.from_numpy(pval).cuda())
        torch.cuda.synchronize()
        got = sel.cpu().numpy()[:len(idx)]
        assert np.array_equal(got, want), step
        ws = fate.fate_commit_advance(pk, st, sel, ws=ws)
        torch.cuda.synchronize()
        nxt, tau, rej, fin = oracle.commit(cur, want, fin=fin)
        assert rej == 0 and st.counts()[3] == 0
        _compare_state(st, nxt, tau, fin)
        _compare_sections(pk, st, nxt)
        cur = nxt
    assert step >= 3


@pytest.mark.parametrize("name", sorted(scenarios.PLANS))
def test_plan_scenarios(name):
    """The hand scenarios of step 12 on the GPU: one stage per instance and
    frontier slot, built to the scenario's instance layout."""
    sc = scenarios.PLANS[name]
    D, f_off = sc["D"], sc["f_off"]
    nf = np.diff(f_off)
    w = synth.make_random_small(90, B=len(nf), n=int(max(nf.max(), 1)), D=D, M=2, max_shard=min(3, D),
                                shard_frac=1.0, p_edge=0.0)
    # every stage pending with no parents: the frontier is each instance's first nf[b] stages
    import dataclasses
    st_ = np.zeros(w.N, np.uint8)
    for b in range(w.B):
        st_[int(w.stage_off[b]) + int(nf[b]):int(w.stage_off[b + 1])] = 3  # committed: not in the frontier
    w = dataclasses.replace(w, status=st_, holders=np.zeros(w.N, np.uint64))
    _, _, fo = oracle.frontier(w)
    assert np.array_equal(fo, f_off)
    ref = oracle.score(w)
    n_cand = np.diff(ref["cand_off"])  # this state's candidate counts bound the choices
    idx = np.array(sc["idx"], np.int32)
    val = np.array(sc["val"], np.float32)
    want, _ = oracle.plan_wave(D, f_off, n_cand, idx, val)
    if np.array_equal(n_cand, sc["n_cand"]):
        assert want.tolist() == sc["sel"]
    assert np.array_equal(_gpu_plan(w, idx, val), want)


def test_plan_errors():
    import torch
    w = synth.make_random_small(82, B=2, n=12, D=4, M=3)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w)
    F = st.n_frontier
    idx = torch.full((max(1, F), 65), -1, dtype=torch.int32, device="cuda")
    val = torch.full((max(1, F), 65), -float("inf"), dtype=torch.float32, device="cuda")
    with pytest.raises(fate.FateError) as e:
        fate.fate_plan_wave(st, idx, val)
    assert e.value.status == fate.FATE_ERANGE
    sel = fate.fate_plan_wave(st, idx[:, :4].contiguous(), val[:, :4].contiguous())
    torch.cuda.synchronize()
    assert np.all(sel.cpu().numpy() == -1)  # nothing valid to take
