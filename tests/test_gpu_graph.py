"""The one-launch score and top-k captured in a HIP graph: every replay,
with eager calls of the same entry point in between, writes the same bits
as the eager call (the kernels record no memset and allocate nothing)."""

import numpy as np
import pytest

from paper_2605_07238_amd import fate, synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["forkjoin-4096x1000-d16", "shards-1024x500-d16"])
def test_graph_replays_match_eager(name):
    import torch
    w = synth.make_workload(name, B=24)
    print("[gpu] graph replay", name, flush=True)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w)
    p = fate.make_params(w)
    k = 4
    F, nC = st.n_frontier, st.n_cand
    s_e = torch.empty(nC, dtype=torch.float32, device="cuda")
    i_e = torch.empty((F, k), dtype=torch.int32, device="cuda")
    v_e = torch.empty((F, k), dtype=torch.float32, device="cuda")
    fate.fate_score_topk(pk, st, p, k, out=s_e, idx=i_e, val=v_e)
    torch.cuda.synchronize()
    ref = (s_e.cpu().numpy().view(np.uint32).copy(), i_e.cpu().numpy().copy(), v_e.cpu().numpy().view(np.uint32).copy())

    s_g = torch.full((nC,), -1.0, dtype=torch.float32, device="cuda")
    i_g = torch.full((F, k), -7, dtype=torch.int32, device="cuda")
    v_g = torch.full((F, k), -1.0, dtype=torch.float32, device="cuda")
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm the call on the capture stream first
        fate.fate_score_topk(pk, st, p, k, out=s_g, idx=i_g, val=v_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fate.fate_score_topk(pk, st, p, k, out=s_g, idx=i_g, val=v_g)
    for r in range(3):
        s_g.fill_(-1.0)
        i_g.fill_(-7)
        v_g.fill_(-1.0)
        g.replay()
        fate.fate_score_topk(pk, st, p, k, out=s_e, idx=i_e, val=v_e)  # eager work between replays
        torch.cuda.synchronize()
        assert np.array_equal(s_g.cpu().numpy().view(np.uint32), ref[0]), "replay %d scores" % r
        assert np.array_equal(i_g.cpu().numpy(), ref[1]), "replay %d top-k indices" % r
        assert np.array_equal(v_g.cpu().numpy().view(np.uint32), ref[2]), "replay %d top-k values" % r
        assert np.array_equal(s_e.cpu().numpy().view(np.uint32), ref[0]), "eager call %d" % r
