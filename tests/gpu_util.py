"""Helpers for GPU tests: run the HIP path through the C ABI and the oracle
on the same seeded inputs and compare them."""

from __future__ import annotations

import numpy as np

from oracle import oracle
from paper_2605_07238_amd import fate, parity

RTOL = 1e-5  # relative to the sum of absolute weighted terms


def run_gpu(w, H=None, params=None, max_shard=None, k=4, pack_H=None):
    import torch
    pk = fate.fate_pack_dags(w, H=pack_H if pack_H is not None else (w.H if H is None else H))
    st = fate.fate_pack_state(pk, w, max_shard=max_shard)
    p = fate.make_params(w, H=(w.H if H is None else H), **(params or {}))
    scores = fate.fate_score_frontier(pk, st, p)
    idx, val = fate.fate_topk(st, scores, k)
    torch.cuda.synchronize()
    fv, fb, co = fate.frontier_table(st)
    return dict(flat_v=fv, front_b=fb, cand_off=co, psi=scores[:st.n_cand].cpu().numpy(),
                idx=idx.cpu().numpy(), val=val.cpu().numpy(), nF=st.n_frontier)


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
    return err
