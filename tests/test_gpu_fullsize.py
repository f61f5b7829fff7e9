"""Every workload recipe at its full batch size, scored in one launch exactly
as the benchmark does; the oracle recomputes a sample of instances (instance
data does not depend on the batch size) and those slices must match."""

import numpy as np
import pytest

from gpu_util import RTOL, run_gpu
from oracle import oracle
from paper_2605_07238_amd import parity, synth

pytestmark = pytest.mark.gpu

SAMPLES = 6


@pytest.mark.parametrize("name", synth.RECIPE_ORDER)
def test_full_batch_sampled_parity(name):
    w = synth.make_workload(name, workers=16)
    print("[gpu] full-size", name, "B", w.B, "N", w.N, flush=True)
    g = run_gpu(w)
    rng = np.random.default_rng(2024)
    pick = sorted(set([0, w.B - 1] + rng.choice(w.B, size=min(SAMPLES, w.B), replace=False).tolist()))
    for b in pick:
        sub = w.subset([b])
        ref = oracle.score(sub)
        slots = np.nonzero(g["front_b"] == b)[0]
        assert np.array_equal(g["flat_v"][slots] - w.stage_off[b], ref["front_v"]), b
        if len(slots) == 0:
            continue
        lo, hi = g["cand_off"][slots[0]], g["cand_off"][slots[-1] + 1]
        err, nbad, ninf = parity.compare(g["psi"][lo:hi], ref["psi"], ref["mag"], RTOL)
        assert ninf == 0 and nbad == 0, (b, err, nbad, ninf)
        bad = parity.topk_mismatches(g["idx"][slots], ref["psi"], ref["mag"], ref["cand_off"], 4, RTOL)
        assert bad == 0, (b, bad)
    print("[gpu] sampled instances", pick, "ok", flush=True)
