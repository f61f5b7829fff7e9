"""Host half of packing, run without a GPU: the packed image round-trips the
inputs, the descendant lists equal breadth-first distances computed with
scipy, the frontier and candidate offsets follow the definitions, and every
validation error code fires on the input that should trigger it."""

import dataclasses

import numpy as np
import pytest
import scipy.sparse as sp
from scipy.sparse.csgraph import shortest_path

from paper_2605_07238_amd import fate, synth

REC = np.dtype([("elig", "<u8"), ("hash", "<u8"), ("tokens", "<f4"), ("sigma", "<f4"),
                ("par_begin", "<u4"), ("model", "u1"), ("shard", "u1"), ("npar", "<u2")])
ROWREC = np.dtype([("hash", "<u8"), ("tokens", "<f4"), ("meta", "<u4")])


def _view(buf, base, ptr, dtype, count):
    off = ptr - base
    return np.frombuffer(buf, dtype=dtype, count=count, offset=off)


def unpack_dags(buf, h):
    base = buf.ctypes.data
    N, E = int(h.N), int(h.E)
    return dict(
        rec=_view(buf, base, h.records, REC, N),
        par=_view(buf, base, h.par_idx, np.uint32, E),
        desc_off=_view(buf, base, h.desc_off, np.uint32, N + 1),
        desc=_view(buf, base, h.desc, np.uint32, int(h.n_desc)),
        fits=_view(buf, base, h.fits, np.uint64, int(h.M)),
    )


@pytest.mark.parametrize("maker", [
    lambda: synth.make_workload("tiny-layered-1x24-d4"),
    lambda: synth.make_workload("layered-1024x200-d8", B=3),
    lambda: synth.make_workload("forkjoin-4096x1000-d16", B=2),
    lambda: synth.make_workload("shards-1024x500-d16", B=2),
    lambda: synth.make_random_small(3, B=3, n=15),
])
def test_dags_image_roundtrip(maker):
    w = maker()
    buf, h, _ = fate.fate_layout_dags(w)
    u = unpack_dags(buf, h)
    rec = u["rec"]
    assert np.array_equal(rec["elig"], w.elig)
    assert np.array_equal(rec["hash"], w.prefix_hash)
    assert np.array_equal(rec["model"], w.model.astype(np.uint8))
    assert np.array_equal(rec["shard"], w.shard_max.astype(np.uint8))
    assert np.array_equal(rec["tokens"], w.prefix_tokens)
    assert np.array_equal(rec["sigma"], w.out_bytes)
    assert np.array_equal(rec["npar"], np.diff(w.par_off).astype(np.uint16))
    assert np.array_equal(rec["par_begin"], w.par_off[:-1].astype(np.uint32))
    inst = np.repeat(np.arange(w.B), np.diff(w.stage_off))
    exp_par = (w.par_idx.astype(np.int64) + w.stage_off[inst[np.repeat(np.arange(w.N), np.diff(w.par_off))]])
    assert np.array_equal(u["par"], exp_par.astype(np.uint32))
    fits = [sum(1 << d for d in range(w.D) if w.weight_bytes[m] <= w.cap_bytes[d]) for m in range(w.M)]
    assert u["fits"].tolist() == fits
    # 16-byte row records (the row kernel for D <= 16, M <= 32): present exactly then
    npar = np.diff(w.par_off)
    expect_rows = w.D <= 16 and w.M <= 32 and (len(npar) == 0 or npar.max() <= 2047)
    assert bool(h.row_records) == expect_rows
    if expect_rows:
        rr = _view(buf, buf.ctypes.data, h.row_records, ROWREC, int(h.N))
        assert np.array_equal(rr["hash"], w.prefix_hash)
        assert np.array_equal(rr["tokens"], w.prefix_tokens)
        meta = rr["meta"].astype(np.uint64)
        assert np.array_equal(meta & 0xFFFF, w.elig & np.uint64(0xFFFF))
        assert np.array_equal((meta >> 16) & 31, w.model.astype(np.uint64))
        assert np.array_equal(meta >> 21, npar.astype(np.uint64))
    # descendant lists = breadth-first distances 1..H, ordered by (distance, id)
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        n = hi - lo
        rows = []
        cols = []
        for x in range(n):
            for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]]:
                rows.append(int(p))
                cols.append(x)
        dist = shortest_path(sp.csr_matrix((np.ones(len(rows)), (rows, cols)), shape=(n, n)),
                             directed=True, unweighted=True)
        for v in range(n):
            ents = u["desc"][u["desc_off"][lo + v]:u["desc_off"][lo + v + 1]]
            got = [(int(e >> 28), int(e & ((1 << 28) - 1)) - lo) for e in ents]
            exp = sorted((int(dist[v, x]), x) for x in range(n) if 1 <= dist[v, x] <= w.H)
            assert got == exp, (b, v)


def _cands(D, r):
    return D + sum(D - k + 1 for k in range(2, r + 1))


@pytest.mark.parametrize("seed", range(4))
def test_state_image_frontier(seed):
    w = synth.make_random_small(seed, B=3, n=14, D=5, max_shard=3)
    buf, h, _ = fate.fate_layout_dags(w)
    sbuf, sh, _ = fate.fate_layout_state(h, w)
    base = sbuf.ctypes.data
    F = int(sh.n_frontier)
    fr = _view(sbuf, base, sh.frontier, np.uint32, 2 * F).reshape(F, 2)
    co = _view(sbuf, base, sh.cand_off, np.uint32, F + 1)
    exp_f, exp_c = [], [0]
    for b in range(w.B):
        lo = int(w.stage_off[b])
        for v in range(int(w.stage_off[b + 1]) - lo):
            g = lo + v
            ps = w.par_idx[w.par_off[g]:w.par_off[g + 1]]
            if w.status[g] == 0 and all(w.status[lo + p] == 1 for p in ps):
                exp_f.append((g, b))
                exp_c.append(exp_c[-1] + _cands(w.D, min(int(w.shard_max[g]), w.max_shard, w.D)))
    assert [tuple(x) for x in fr.tolist()] == exp_f
    assert co.tolist() == exp_c
    assert int(sh.n_cand) == exp_c[-1]
    res = _view(sbuf, base, sh.resident, np.uint64, w.B * w.D)
    assert np.array_equal(res, w.resident.reshape(-1))
    assert np.array_equal(_view(sbuf, base, sh.holders, np.uint64, w.N), w.holders)


@pytest.mark.parametrize("seed,uniform", [(0, False), (1, True), (2, False), (3, True)])
def test_state_offsets_order_and_slices(seed, uniform):
    """Per-instance frontier offsets; the dispatch order (eight size classes
    in proportion to the largest frontier, largest first, each class in
    instance order); the slices cut each instance's range into pieces of the
    slice length, in the dispatch order unless the row kernel scores the
    batch (single-device candidates, uniform beta, D <= 16, M <= 32), which
    does not use them and keeps instance order."""
    w = synth.make_random_small(seed, B=23, n=12 + seed, D=6, max_shard=1 if uniform else 3,
                                shard_frac=0.0 if uniform else 0.4, uniform_beta=uniform)
    buf, h, _ = fate.fate_layout_dags(w)
    sbuf, sh, _ = fate.fate_layout_state(h, w)
    base = sbuf.ctypes.data
    F, S = int(sh.n_frontier), int(sh.n_slices)
    fr = _view(sbuf, base, sh.frontier, np.uint32, 2 * F).reshape(F, 2)
    fr_off = _view(sbuf, base, sh.fr_off, np.uint32, w.B + 1).astype(np.int64)
    assert fr_off.tolist() == np.searchsorted(fr[:, 1], np.arange(w.B + 1), side="left").tolist()
    n = np.diff(fr_off)
    cls = 7 - np.minimum(7, n * 8 // (n.max() + 1))
    order = _view(sbuf, base, sh.order, np.uint32, w.B)
    assert order.tolist() == sorted(range(w.B), key=lambda b: (cls[b], b))
    rows_batch = bool(h.beta_uniform) and min(int(h.max_r), w.max_shard, w.D) <= 1 and w.D <= 16 and w.M <= 32
    assert rows_batch == uniform
    L = int(sh.slice)
    insts = range(w.B) if rows_batch else order
    want = [(b, f, min(int(fr_off[b + 1]), f + L)) for b in insts for f in range(int(fr_off[b]), int(fr_off[b + 1]), L)]
    assert _view(sbuf, base, sh.slices, np.uint32, 3 * S).reshape(S, 3).tolist() == [list(x) for x in want]


def _status(fn, w, H=None):
    try:
        fn(w, H)
    except fate.FateError as e:
        return e.status
    return 0


def _pack_dags(w, H=None):
    fate.fate_layout_dags(w, H)


def _pack_state(w, H=None):
    _, h, _ = fate.fate_layout_dags(w, H)
    fate.fate_layout_state(h, w)


def test_error_codes():
    base = synth.make_random_small(1, B=1, n=8, D=4)
    assert _status(_pack_dags, base) == 0
    assert _status(_pack_state, base) == 0
    # parent id not below the child's id
    w = dataclasses.replace(base, par_idx=base.par_idx.copy())
    g = int(np.argmax(np.diff(w.par_off) > 0))
    w.par_idx[w.par_off[g]] = g
    assert _status(_pack_dags, w) == -3
    # eligibility outside the device range
    w = dataclasses.replace(base, elig=base.elig.copy())
    w.elig[0] = np.uint64(1 << 5)
    assert _status(_pack_dags, w) == -1
    # no eligible device can hold the model
    w = dataclasses.replace(base, elig=base.elig.copy(), cap_bytes=base.cap_bytes.copy())
    m0 = int(w.model[0])
    w.cap_bytes[:] = int(w.weight_bytes[m0]) - 1
    assert _status(_pack_dags, w) == -4
    # horizon out of range
    assert _status(_pack_dags, base, 16) == -2
    # negative runtime
    w = dataclasses.replace(base, exec=base.exec.copy())
    w.exec[0, 0] = -1.0
    assert _status(_pack_dags, w) == -1
    # NaN inputs are rejected (host validation is compiled with NaN semantics)
    w = dataclasses.replace(base, exec=base.exec.copy())
    w.exec[0, 1] = np.nan
    assert _status(_pack_dags, w) == -1
    w = dataclasses.replace(base, out_bytes=base.out_bytes.copy())
    w.out_bytes[2] = np.nan
    assert _status(_pack_dags, w) == -1
    w = dataclasses.replace(base, tau_free=base.tau_free.copy())
    w.tau_free[0, 0] = np.inf
    assert _status(_pack_state, w) == -1
    # too many devices
    w = dataclasses.replace(base, D=65)
    assert _status(_pack_dags, w) == -2
    # completed stage without holders
    w = dataclasses.replace(base, holders=base.holders.copy(), status=base.status.copy())
    done = np.nonzero(w.status == 1)[0]
    w.holders[done[0]] = np.uint64(0)
    assert _status(_pack_state, w) == -6
    # holder bit outside the device range
    w = dataclasses.replace(base, holders=base.holders.copy())
    w.holders[done[0]] = np.uint64(1 << 7)
    assert _status(_pack_state, w) == -6
    # bad status code
    w = dataclasses.replace(base, status=base.status.copy())
    w.status[0] = 9
    assert _status(_pack_state, w) == -1
    # resident model id >= M
    w = dataclasses.replace(base, resident=base.resident.copy())
    w.resident[0, 0] = np.uint64(1 << 20)
    assert _status(_pack_state, w) == -1


def test_too_small_buffer_is_rejected():
    w = synth.make_random_small(2, B=1, n=8)
    lib = fate.load()
    hi = fate.HostInputs(w)
    import ctypes as C
    need = C.c_size_t(0)
    assert lib.fate_pack_dags_size(C.byref(hi.cluster), C.byref(hi.batch), 2, C.byref(need)) == 0
    buf = np.zeros(need.value, np.uint8)
    h = fate.Dags()
    assert lib.fate_layout_dags(C.byref(hi.cluster), C.byref(hi.batch), 2, buf.ctypes.data, need.value - 1,
                                C.byref(h)) == -5
    assert lib.fate_layout_dags(C.byref(hi.cluster), C.byref(hi.batch), 2, buf.ctypes.data, need.value,
                                C.byref(h)) == 0


def test_every_scenario_packs_on_the_host():
    """Includes batches without any edge (no parent array at all)."""
    import builders
    import scenarios
    for name, sc in scenarios.ALL.items():
        w = builders.from_spec(sc["spec"], H=max(sc["H"], 1), params=sc["params"])
        _, h, _ = fate.fate_layout_dags(w)
        _, sh, _ = fate.fate_layout_state(h, w)
        assert int(sh.n_frontier) == len(sc["front_v"]), name


def test_all_committed_gives_empty_frontier():
    w = synth.make_random_small(5, B=2, n=8)
    w = dataclasses.replace(w, status=np.where(w.status == 0, 3, w.status).astype(np.uint8))
    _, h, _ = fate.fate_layout_dags(w)
    _, sh, _ = fate.fate_layout_state(h, w)
    assert int(sh.n_frontier) == 0 and int(sh.n_cand) == 0


def test_topk_of_scores_rule():
    """Host top-k rule used to check the kernels: score descending, ties to
    the lower index, -inf skipped, -1 padding."""
    from paper_2605_07238_amd import parity
    inf = np.inf
    psi = np.array([1.0, 3.0, 3.0, -inf, 2.0,   -inf, -inf,   0.0, -0.0], np.float32)
    co = np.array([0, 5, 7, 9])
    got = parity.topk_of_scores(psi, co, 4)
    assert got.tolist() == [[1, 2, 4, 0], [-1, -1, -1, -1], [0, 1, -1, -1]]
    assert parity.topk_of_scores(psi, np.array([0]), 3).shape == (0, 3)


def test_workload_save_load_roundtrip(tmp_path):
    w = synth.make_random_small(3, B=3, n=20, D=8)
    p = str(tmp_path / "w.npz")
    synth.save_workload(w, p)
    v = synth.load_workload(p)
    for f in synth._ARRAY_FIELDS:
        a, b = getattr(w, f), getattr(v, f)
        assert a.dtype == b.dtype and np.array_equal(a, b), f
    assert (w.name, w.D, w.M, w.K, w.H, w.max_shard, w.params) == (v.name, v.D, v.M, v.K, v.H, v.max_shard, v.params)


def test_planning_state_size_and_commit_errors():
    """Host side of the planning state: its capacity sizing, and the commit
    entry points refusing a plainly packed state (no HIP call is made)."""
    import ctypes as C
    w = synth.make_random_small(3, B=3, n=20, D=6)
    lib = fate.load()
    buf, h, hi = fate.fate_layout_dags(w)
    sbuf, sh, shi = fate.fate_layout_state(h, w)
    plain = C.c_size_t(0)
    nf, nc = C.c_int64(0), C.c_int64(0)
    assert lib.fate_pack_state_size(C.byref(h), C.byref(shi.batch), C.byref(shi.state), w.max_shard,
                                    C.byref(plain), C.byref(nf), C.byref(nc)) == 0
    adv = C.c_size_t(0)
    assert lib.fate_pack_state_advance_size(C.byref(h), C.byref(shi.batch), C.byref(shi.state), w.max_shard,
                                            C.byref(adv)) == 0
    assert adv.value > plain.value
    assert lib.fate_pack_state_advance_size(C.byref(h), C.byref(shi.batch), C.byref(shi.state), w.max_shard,
                                            None) == fate.FATE_EINVAL
    ws = C.c_size_t(0)
    assert sh.advance == 0
    assert lib.fate_commit_ws_size(C.byref(h), C.byref(sh), C.byref(ws)) == fate.FATE_EINVAL
    assert lib.fate_commit_advance(C.byref(h), C.byref(sh), None, 1, None, 0, None) == fate.FATE_EINVAL


def _levels_bf(adj):
    """Longest-path levels from Bellman-Ford shortest paths on -1 weights."""
    n = adj.shape[0]
    neg = sp.csr_matrix((-np.ones(adj.nnz), adj.indices, adj.indptr), shape=(n, n))
    d = shortest_path(neg, method="BF", directed=True)
    return np.maximum(np.where(np.isfinite(d), -d, 0.0).max(axis=0), 0.0).astype(np.int64)


@pytest.mark.parametrize("maker", [
    lambda: synth.make_workload("layered-1024x200-d8", B=2),
    lambda: synth.make_random_small(4, B=3, n=20, p_edge=0.35, H=3),
    lambda: synth.make_random_small(5, B=2, n=25, p_edge=0.5, H=5),
])
def test_topological_level_lists_and_weights(maker):
    """With topological levels the lists hold every stage reachable from v whose
    longest-path level exceeds v's by 1..H, at that difference, ordered by
    (depth, id); level weights are 1 / (entries at that depth)."""
    w = maker()
    H = min(int(w.H), 4)
    buf, h, _ = fate.fate_layout_dags(w, H=H, levels=fate.FATE_LEVELS_TOPO, level_weights=True)
    assert int(h.levels) == fate.FATE_LEVELS_TOPO and h.desc_w
    u = unpack_dags(buf, h)
    wts = _view(buf, buf.ctypes.data, h.desc_w, np.float32, int(h.n_desc))
    for b in range(w.B):
        lo, hi = int(w.stage_off[b]), int(w.stage_off[b + 1])
        n = hi - lo
        rows, cols = [], []
        for x in range(n):
            for p in w.par_idx[w.par_off[lo + x]:w.par_off[lo + x + 1]]:
                rows.append(int(p))
                cols.append(x)
        adj = sp.csr_matrix((np.ones(len(rows)), (rows, cols)), shape=(n, n))
        reach = np.isfinite(shortest_path(adj, directed=True, unweighted=True))
        lv = _levels_bf(adj)
        for v in range(n):
            e0, e1 = u["desc_off"][lo + v], u["desc_off"][lo + v + 1]
            ents = u["desc"][e0:e1]
            got = [(int(e >> 28), int(e & ((1 << 28) - 1)) - lo) for e in ents]
            exp = sorted((int(lv[x] - lv[v]), x) for x in range(n)
                         if x != v and reach[v, x] and 1 <= lv[x] - lv[v] <= H)
            assert got == exp, (b, v)
            depths = np.array([d for d, _ in got], np.int64)
            if len(depths):
                cnt = np.bincount(depths)[depths]
                assert np.array_equal(wts[e0:e1], (1.0 / cnt).astype(np.float32)), (b, v)


def test_hop_options_give_the_plain_image():
    w = synth.make_random_small(6, B=3, n=20, p_edge=0.35, H=3)
    a, ha, _ = fate.fate_layout_dags(w)
    b, hb, _ = fate.fate_layout_dags(w, levels=fate.FATE_LEVELS_HOP, level_weights=False)
    assert int(ha.n_desc) == int(hb.n_desc) and not hb.desc_w
    assert np.array_equal(a[:int(ha.bytes) if ha.bytes else len(a)], b[:len(a)])
    c, hc, _ = fate.fate_layout_dags(w, level_weights=True)  # weights appended after the lists
    uc, ua = unpack_dags(c, hc), unpack_dags(a, ha)
    assert np.array_equal(uc["desc"], ua["desc"]) and np.array_equal(uc["desc_off"], ua["desc_off"])


def test_pack_option_and_flag_errors():
    import ctypes as C
    w = synth.make_random_small(7, B=1, n=10, D=4)
    lib = fate.load()
    hi = fate.HostInputs(w)
    for lv, lw in ((2, 0), (-1, 0), (0, 2)):
        o = fate.PackOpts(int(w.H), lv, lw)
        n = C.c_size_t(0)
        assert lib.fate_pack_dags_opt_size(C.byref(hi.cluster), C.byref(hi.batch), C.byref(o), C.byref(n)) \
            == fate.FATE_EINVAL, (lv, lw)
    assert lib.fate_pack_dags_opt_size(C.byref(hi.cluster), C.byref(hi.batch), None, C.byref(n)) == fate.FATE_EINVAL
    # scoring validates parameters before touching any device memory
    _, dh, _ = fate.fate_layout_dags(w)
    _, sh, _ = fate.fate_layout_state(dh, w)
    for over in (dict(flags=4), dict(lam_m=-1.0), dict(lam_m=float("nan")), dict(flags=fate.FATE_MEAN_PER_LEVEL)):
        p = fate.make_params(w)
        for k, v in over.items():
            setattr(p, k, v)
        st = lib.fate_score_frontier(C.byref(dh), C.byref(sh), C.byref(p), None, 1 << 20, None, 0, None)
        assert st == fate.FATE_EINVAL, over
    p = fate.make_params(w)
    arr = (fate.Params * 17)(*([p] * 17))
    st = lib.fate_score_sweep(C.byref(dh), C.byref(sh), arr, 17, None, 1 << 20, int(sh.n_cand), None, 0, None)
    assert st == fate.FATE_ERANGE
    st = lib.fate_score_sweep(C.byref(dh), C.byref(sh), arr, 0, None, 1 << 20, int(sh.n_cand), None, 0, None)
    assert st == fate.FATE_ERANGE
    st = lib.fate_score_sweep(C.byref(dh), C.byref(sh), arr, 2, None, 1 << 20, int(sh.n_cand) - 1, None, 0, None)
    assert st == fate.FATE_ESIZE
    st = lib.fate_topk_sweep(C.byref(sh), None, 1 << 20, int(sh.n_cand), 17, 4, None, None, None)
    assert st == fate.FATE_ERANGE
