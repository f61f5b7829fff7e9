"""Helpers for GPU tests: run the HIP path through the C ABI and the oracle
on the same seeded inputs and compare them."""

from __future__ import annotations

import numpy as np

from oracle import oracle
from paper_2605_07238_amd import fate, parity

RTOL = 1e-5  # relative to the sum of absolute weighted terms


def run_gpu(w, H=None, params=None, max_shard=None, k=4, pack_H=None):
    import torch
    pp = dict(w.params, **(params or {}))
    pk = fate.fate_pack_dags(w, H=pack_H if pack_H is not None else (w.H if H is None else H),
                             levels=fate.FATE_LEVELS_TOPO if pp.get("topo_levels") else fate.FATE_LEVELS_HOP,
                             level_weights=bool(pp.get("mean_levels")))
    st = fate.fate_pack_state(pk, w, max_shard=max_shard)
    p = fate.make_params(w, H=(w.H if H is None else H), **(params or {}))
    scores = fate.fate_score_frontier(pk, st, p)
    idx, val = fate.fate_topk(st, scores, k)
    # the fused entry point must write the same bits
    s2, i2, v2 = fate.fate_score_topk(pk, st, p, k)
    torch.cuda.synchronize()
    fv, fb, co = fate.frontier_table(st)
    out = dict(flat_v=fv, front_b=fb, cand_off=co, psi=scores[:st.n_cand].cpu().numpy(),
               idx=idx.cpu().numpy(), val=val.cpu().numpy(), nF=st.n_frontier)
    assert np.array_equal(out["psi"].view(np.uint32), s2[:st.n_cand].cpu().numpy().view(np.uint32)), \
        "fused scores differ"
    assert np.array_equal(out["idx"], i2.cpu().numpy()), "fused top-k indices differ"
    assert np.array_equal(out["val"].view(np.uint32), v2.cpu().numpy().view(np.uint32)), "fused top-k values differ"
    return out


def check_against_oracle(w, gpu, H=None, params=None, max_shard=None, k=4, rtol=RTOL):
    ref = oracle.score(w, params=params, H=H, max_shard=max_shard)
    flat = w.stage_off[ref["front_b"]] + ref["front_v"]
    assert np.array_equal(gpu["flat_v"], flat), "frontier differs"
    assert np.array_equal(gpu["cand_off"], ref["cand_off"]), "candidate offsets differ"
    err, nbad, ninf = parity.compare(gpu["psi"], ref["psi"], ref["mag"], rtol)
    assert ninf == 0, "-inf pattern differs (%d)" % ninf
    assert nbad == 0, "max rel err %.3g over %d candidates" % (err, nbad)
    bad = parity.topk_mismatches(gpu["idx"], ref["psi"], ref["mag"], ref["cand_off"], k, rtol)
    assert bad == 0, "%d top-k ranks differ" % bad
    # the kernel's selection over its own scores is exact: (score desc, index asc)
    want_idx = parity.topk_of_scores(gpu["psi"], gpu["cand_off"], k)
    assert np.array_equal(gpu["idx"][:gpu["nF"]], want_idx), "top-k selection differs from the rule"
    # each reported value is the score at the reported index; padding is (-1, -inf)
    idx, val = gpu["idx"], gpu["val"]
    if idx.size and gpu["nF"]:
        pos = np.asarray(gpu["cand_off"][:-1], np.int64)[:, None] + np.maximum(idx, 0)
        want = np.where(idx >= 0, gpu["psi"][np.minimum(pos, max(len(gpu["psi"]) - 1, 0))], -np.inf)
        assert np.array_equal(val[:gpu["nF"]].view(np.uint32),
                              want[:gpu["nF"]].astype(np.float32).view(np.uint32)), "top-k values differ from scores"
    return err
