"""Every workload recipe at its full batch size, scored in one launch exactly
as the benchmark does (the fused score and top-4), against the oracle on
every instance of the batch: scores element by element within the tolerance,
the -inf pattern exactly, the top-4 tie-aware against the oracle and
bit-exact against the selection rule applied to the GPU's own scores."""

import json
import os
import time

import numpy as np
import pytest

from gpu_util import RTOL
from oracle import oracle
from paper_2605_07238_amd import parity, synth

pytestmark = pytest.mark.gpu

K = 4


@pytest.mark.parametrize("name", synth.RECIPE_ORDER)
def test_full_batch_every_instance(name):
    import torch
    from paper_2605_07238_amd import fate
    w = synth.make_workload(name, workers=16)
    print("[gpu] full-size", name, "B", w.B, "N", w.N, flush=True)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w)
    scores, idx, val = fate.fate_score_topk(pk, st, fate.make_params(w), K)
    torch.cuda.synchronize()
    psi = scores[:st.n_cand].cpu().numpy()
    idx = idx.cpu().numpy()
    val = val.cpu().numpy()
    fv, fb, co = fate.frontier_table(st)
    print("[gpu] scored", st.n_frontier, "stages", st.n_cand, "candidates; oracle next", flush=True)
    t0 = time.perf_counter()
    ref = oracle.score(w)
    oracle_s = time.perf_counter() - t0
    assert np.array_equal(fv, w.stage_off[ref["front_b"]] + ref["front_v"]), "frontier differs"
    assert np.array_equal(co, ref["cand_off"]), "candidate offsets differ"
    err, nbad, ninf = parity.compare(psi, ref["psi"], ref["mag"], RTOL)
    print("[gpu] %s: max err %.3g A over %d candidates" % (name, err, len(psi)), flush=True)
    assert ninf == 0, "-inf pattern differs at %d candidates" % ninf
    assert nbad == 0, "%d candidates beyond the tolerance (max %.3g)" % (nbad, err)
    bad = parity.topk_mismatches(idx, ref["psi"], ref["mag"], ref["cand_off"], K, RTOL)
    assert bad == 0, "%d top-k ranks differ from the oracle's beyond ties" % bad
    assert np.array_equal(idx, parity.topk_of_scores(psi, co, K)), "top-k differs from the rule on the GPU's scores"
    pos = co[:-1, None] + np.maximum(idx, 0)
    want = np.where(idx >= 0, psi[np.minimum(pos, max(len(psi) - 1, 0))], -np.inf).astype(np.float32)
    assert np.array_equal(val.view(np.uint32), want.view(np.uint32)), "top-k values differ from the scores"
    # one summary line per recipe: the parity figures and the oracle's whole-batch rate
    stage = fv[np.repeat(np.arange(len(fv)), np.diff(co))] if len(fv) else np.zeros(0, np.int64)
    n_eval = int((1 + fate.desc_counts(pk)[stage])[np.isfinite(psi)].sum())
    print("[parity] " + json.dumps(dict(workload=name, instances=w.B, candidates=len(psi), max_err_over_A=err,
                                        topk_rank_mismatches=bad, evals=n_eval, oracle_s=oracle_s,
                                        oracle_threads=os.environ.get("OMP_NUM_THREADS", str(os.cpu_count())),
                                        oracle_evals_per_s=n_eval / oracle_s)), flush=True)
