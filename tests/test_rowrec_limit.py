"""The 16-byte row records and the row kernel's limit on |Pa(v)|: a batch
whose join stage has 2,048 completed parents gets no row records (their
packed word holds |Pa(v)| in 11 bits), so its frontier is scored by the
general kernel; with 2,047 parents the records exist and the row kernel
scores it.  Both against the oracle."""

import numpy as np
import pytest

import builders
from paper_2605_07238_amd import fate


def _join_batch(npar: int):
    """One instance: npar completed roots, a pending join of all of them (in
    the frontier) with a pending child (its horizon row), and a pending root
    with a child; D = 4, uniform beta, single-device candidates."""
    D, M = 4, 2
    parents = [[] for _ in range(npar)] + [list(range(npar)), [npar], [], [npar + 2]]
    n = len(parents)
    inst = dict(parents=parents, model=[v % M for v in range(n)], elig=[(1 << D) - 1] * n,
                prefix_hash=[0 if v % 3 else 17 + v % 2 for v in range(n)], prefix_tokens=[200.0] * n,
                out_bytes=[1e6 * (1 + v % 5) for v in range(n)],
                status=[1] * npar + [0] * 4, holders=[1 << (v % D) for v in range(npar)] + [0] * 4,
                resident=[1, 2, 0, 3], tau_free=[0.0, 0.5, 1.0, 0.25], t_now=0.0)
    spec = dict(D=D, M=M, K=2, exec=[[1.0, 1.5, 2.0, 0.5]] * M, switch_s=[[0.3] * D] * M, weight_gb=[10, 20],
                cap_gb=[40, 40, 25, 40], beta=[[0.0 if i == j else 2e-10 for j in range(D)] for i in range(D)],
                max_shard=1, instances=[inst])
    return builders.from_spec(spec, H=2)


@pytest.mark.parametrize("npar,records", [(2047, True), (2048, False)])
def test_row_records_present_up_to_2047_parents(npar, records):
    w = _join_batch(npar)
    _, h, _ = fate.fate_layout_dags(w)
    assert bool(h.row_records) == records


@pytest.mark.gpu
@pytest.mark.parametrize("npar", [2047, 2048])
def test_join_of_many_parents_against_oracle(npar):
    from gpu_util import check_against_oracle, run_gpu
    w = _join_batch(npar)
    print("[gpu] join of %d completed parents" % npar, flush=True)
    check_against_oracle(w, run_gpu(w))
