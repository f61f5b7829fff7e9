"""fate_commit_advance_noalloc (the library-held workspace) against
fate_commit_advance (a caller workspace) through the C ABI.

Two planning states of the same batch are advanced side by side, one by each
entry point, with the same selections (the oracle's top-1 per frontier
stage, so nothing the GPU computed chooses them); after every step every
array and section of the two states must be bit-identical.  A first batch
takes two steps, then a second, smaller batch takes one, so the library's
array serves a call after a larger one.  A planning state that needs more
workspace than the array holds is rejected before anything is enqueued."""

import numpy as np
import pytest

from oracle import oracle
from paper_2605_07238_amd import fate, synth

pytestmark = pytest.mark.gpu


def _snapshot(st):
    """Every array and current section of a planning state, as host bytes."""
    h = st.handle
    nF, nC, nS, rej = st.counts()
    base = st.buf.data_ptr()
    N = int(h.N)

    def take(ptr, n, dt=np.uint32):
        off = ptr - base
        nb = n * np.dtype(dt).itemsize
        return st.buf[off:off + nb].cpu().numpy().view(dt).copy() if n else np.zeros(0, dt)

    out = {k: np.asarray(v).view(np.uint8) for k, v in fate.state_arrays(st).items()}
    out.update(frontier=take(h.frontier, 2 * nF), cand_off=take(h.cand_off, nF + 1), slices=take(h.slices, 3 * nS),
               done_n=take(h.done_n, N), done=take(h.done, 4 * int(h.n_done_edges)),
               fr_off=take(h.fr_off, int(h.B) + 1), order=take(h.order, int(h.B)),
               counts=np.array([nF, nC, nS, rej], np.int64))
    return out


def _advance_side_by_side(w, steps):
    import torch
    pk = fate.fate_pack_dags(w)
    with_ws = fate.fate_pack_state(pk, w, advance=True)
    no_ws = fate.fate_pack_state(pk, w, advance=True)
    cur, fin, ws = w, None, None
    assert fate.fate_commit_ws_size(pk, no_ws) <= fate.FATE_NOALLOC_WS_BYTES
    for step in range(steps):
        ref = oracle.score(cur)
        print("[gpu] no-alloc commit: B", w.B, "step", step, "frontier", len(ref["front_v"]), flush=True)
        assert len(ref["front_v"]) > 0
        idx, _ = oracle.topk(ref, 1)
        sel = np.ascontiguousarray(idx[:, 0], np.int32)
        sel[::7] = -1  # some stages stay pending
        cur, _, _, fin = oracle.commit(cur, sel, fin=fin)
        d_sel = torch.from_numpy(sel).cuda()
        ws = fate.fate_commit_advance(pk, with_ws, d_sel, ws=ws)
        fate.fate_commit_advance_noalloc(pk, no_ws, d_sel)
        torch.cuda.synchronize()
        a, b = _snapshot(with_ws), _snapshot(no_ws)
        assert a.keys() == b.keys()
        for key in a:
            assert np.array_equal(a[key], b[key]), "%s differs after step %d" % (key, step)
        # and the state is the oracle's
        assert np.array_equal(fate.state_arrays(no_ws)["status"], cur.status)


def test_noalloc_commit_matches_workspace_commit():
    import torch
    assert torch.cuda.is_available(), "needs a GPU"
    torch.cuda.set_device(0)
    _advance_side_by_side(synth.make_workload("forkjoin-4096x1000-d16", B=48), steps=2)
    _advance_side_by_side(synth.make_workload("shards-1024x500-d16", B=8), steps=1)


def test_noalloc_commit_rejects_a_state_beyond_its_workspace():
    import torch
    torch.cuda.set_device(0)
    w = synth.make_workload("forkjoin-4096x1000-d16", B=4400, workers=16)  # 4.4 M stages: about 36 MB
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w, advance=True)
    need = fate.fate_commit_ws_size(pk, st)
    assert need > fate.FATE_NOALLOC_WS_BYTES
    sel = torch.full((st.n_frontier,), -1, dtype=torch.int32, device="cuda")
    before = _snapshot(st)
    with pytest.raises(fate.FateError) as err:
        fate.fate_commit_advance_noalloc(pk, st, sel)
    assert err.value.status == -2  # FATE_ERANGE
    torch.cuda.synchronize()
    after = _snapshot(st)
    for key in before:
        assert np.array_equal(before[key], after[key]), key
