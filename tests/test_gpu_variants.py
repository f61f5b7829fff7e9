"""Scoring variants and parameter sweeps on the GPU against the oracle.

Variants: the same-model weight lam_m, topological-level horizons, the
mean-per-level tail and scoring without windows (oracle V1-V4).  Sweeps:
fate_score_sweep / fate_topk_sweep over several parameter sets in one launch
must write, set by set, the same bits as one fate_score_frontier /
fate_topk call per set.
"""

import numpy as np
import pytest

import builders
import scenarios
from gpu_util import RTOL, check_against_oracle, run_gpu
from oracle import oracle
from paper_2605_07238_amd import fate, parity, synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", sorted(scenarios.VARIANTS))
def test_variant_scenario(name):
    sc = scenarios.VARIANTS[name]
    w = builders.from_spec(sc["spec"], H=sc["H"], params=sc["params"])
    print("[gpu] variant scenario", name, flush=True)
    gpu = run_gpu(w, k=3)
    check_against_oracle(w, gpu, k=3)
    psi = np.asarray(sc["psi"], np.float64)
    fin = np.isfinite(psi)
    assert np.array_equal(np.isneginf(gpu["psi"]), ~fin)
    assert np.allclose(gpu["psi"][fin], psi[fin], rtol=1e-6, atol=0)


VARIANTS = {
    "same_model": dict(lam_m=0.3),
    "same_model_strong": dict(lam_m=2.0, lam_s=0.5),
    "topo": dict(topo_levels=1),
    "mean": dict(mean_levels=1),
    "topo_mean": dict(topo_levels=1, mean_levels=1),
    "no_windows": dict(no_windows=1),
    "all": dict(lam_m=0.25, topo_levels=1, mean_levels=1, no_windows=1),
}

RANDOM = [
    dict(seed=51, D=4, n=24, M=3, max_shard=3, shard_frac=0.6, p_edge=0.35),
    dict(seed=52, D=7, n=30, M=5, K=3, max_shard=4, shard_frac=0.5, p_edge=0.3),
    dict(seed=53, D=16, n=30, M=8, K=4, max_shard=4, shard_frac=0.5, uniform_beta=True, p_edge=0.3),
    dict(seed=54, D=16, n=30, M=40, K=4, max_shard=3, uniform_beta=True),
    dict(seed=55, D=33, n=24, M=6, K=2, p_edge=0.4),
    dict(seed=56, D=64, n=20, M=6, K=2, max_shard=2),
]


@pytest.mark.parametrize("variant", sorted(VARIANTS))
@pytest.mark.parametrize("case", range(len(RANDOM)))
def test_variant_random(variant, case):
    spec = dict(RANDOM[case])
    seed = spec.pop("seed")
    w = synth.make_random_small(seed, B=3, H=4, **spec)
    params = VARIANTS[variant]
    print("[gpu] variant", variant, "case", case, flush=True)
    gpu = run_gpu(w, params=params)
    check_against_oracle(w, gpu, params=params)


@pytest.mark.parametrize("variant", ["same_model", "topo_mean", "no_windows"])
@pytest.mark.parametrize("name", ["forkjoin-4096x1000-d16", "shards-1024x500-d16", "powerlaw-256x10000-d64"])
def test_variant_recipes(variant, name):
    w = synth.make_workload(name, B=6)
    params = VARIANTS[variant]
    print("[gpu] variant", variant, "recipe", name, flush=True)
    gpu = run_gpu(w, params=params)
    check_against_oracle(w, gpu, params=params)


def _grid(w, H_max):
    """A Tab. 6-style grid: every H up to H_max, then the state, locality and
    prefix weight groups at x0.5 and x1.5, plus variants."""
    base = dict(w.params)
    sets = []
    for H in range(H_max + 1):
        sets.append(fate.make_params(w, H=H))
    for f in (0.5, 1.5):
        sets.append(fate.make_params(w, lam_s=base["lam_s"] * f, lam_m=0.2 * f))
        sets.append(fate.make_params(w, lam_tr=base["lam_tr"] * f, lam_c=base["lam_c"] * f))
        sets.append(fate.make_params(w, lam_p=base["lam_p"] * f))
    sets.append(fate.make_params(w, mean_levels=1))
    sets.append(fate.make_params(w, no_windows=1))
    return sets


@pytest.mark.parametrize("name,advance", [("forkjoin-4096x1000-d16", False), ("shards-1024x500-d16", False),
                                          ("layered-1024x200-d8", True), ("powerlaw-256x10000-d64", False)])
def test_sweep_matches_single_calls(name, advance):
    import torch
    w = synth.make_workload(name, B=8)
    pk = fate.fate_pack_dags(w, level_weights=True)
    st = fate.fate_pack_state(pk, w, advance=advance)
    sets = _grid(w, int(w.H))
    assert len(sets) <= fate.FATE_MAX_SWEEP
    print("[gpu] sweep", name, len(sets), "sets", flush=True)
    k = 4
    sweep = fate.fate_score_sweep(pk, st, sets)
    sidx, sval = fate.fate_topk_sweep(st, sweep, k)
    torch.cuda.synchronize()
    nC = st.counts()[1] if advance else st.n_cand
    nF = st.counts()[0] if advance else st.n_frontier
    got = sweep.cpu().numpy()
    gi, gv = sidx.cpu().numpy(), sval.cpu().numpy()
    for p, prm in enumerate(sets):
        one = fate.fate_score_frontier(pk, st, prm)
        i1, v1 = fate.fate_topk(st, one, k)
        torch.cuda.synchronize()
        assert np.array_equal(got[p, :nC].view(np.uint32), one[:nC].cpu().numpy().view(np.uint32)), p
        assert np.array_equal(gi[p, :nF], i1[:nF].cpu().numpy()), p
        assert np.array_equal(gv[p, :nF].view(np.uint32), v1[:nF].cpu().numpy().view(np.uint32)), p


def test_sweep_sets_against_oracle():
    """Each set of a sweep against the oracle run with that set's parameters."""
    import torch
    w = synth.make_random_small(61, B=3, n=30, D=8, M=5, K=3, H=4, max_shard=3, shard_frac=0.5, p_edge=0.3)
    pk = fate.fate_pack_dags(w, level_weights=True)
    st = fate.fate_pack_state(pk, w)
    over = [dict(), dict(lam_m=0.5), dict(mean_levels=1), dict(no_windows=1), dict(gamma=0.9, lam_q=2.0),
            dict(lam_tr=0.0, lam_c=0.0), dict(lam_p=3.0, lam_m=0.1, mean_levels=1)]
    Hs = [4, 3, 2, 4, 1, 0, 4]
    sets = [fate.make_params(w, H=H, **o) for o, H in zip(over, Hs)]
    sweep = fate.fate_score_sweep(pk, st, sets)
    torch.cuda.synchronize()
    got = sweep.cpu().numpy()
    for p, (o, H) in enumerate(zip(over, Hs)):
        ref = oracle.score(w, params=o, H=H)
        err, nbad, ninf = parity.compare(got[p, :st.n_cand], ref["psi"], ref["mag"], RTOL)
        assert ninf == 0 and nbad == 0, (p, err, nbad, ninf)


def test_sweep_limits():
    import torch
    w = synth.make_random_small(62, B=2, n=16, D=4, M=3)
    pk = fate.fate_pack_dags(w)
    st = fate.fate_pack_state(pk, w)
    sets = [fate.make_params(w)] * 16
    out = fate.fate_score_sweep(pk, st, sets)
    torch.cuda.synchronize()
    assert out.shape[0] == 16
    with pytest.raises(fate.FateError) as e:
        fate.fate_score_sweep(pk, st, sets + [fate.make_params(w)])
    assert e.value.status == fate.FATE_ERANGE
    with pytest.raises(fate.FateError) as e:  # mean per level needs packed level weights
        fate.fate_score_sweep(pk, st, [fate.make_params(w, mean_levels=1)])
    assert e.value.status == fate.FATE_EINVAL
    with pytest.raises(fate.FateError) as e:  # stride below the candidate count
        fate.fate_score_sweep(pk, st, sets[:2], stride=max(1, st.n_cand - 1))
    assert e.value.status == fate.FATE_ESIZE
