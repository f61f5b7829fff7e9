"""Plant plausible mistakes in copies of the plan-execution oracle and check
that its pins reject each of them (no GPU)."""

import importlib.util
import os

import pytest

import sim_pins
from oracle import simulate as S

MUTANTS = {
    "transfer_not_split": [("arr = self.finish[u] + self.sigma[u] * bmin / k",
                            "arr = self.finish[u] + self.sigma[u] * bmin")],
    "switch_always": [("sw = 0.0 if (res >> m) & 1 else self.ksw[m, d]", "sw = self.ksw[m, d]")],
    "hit_on_group_zero": [("hit = self.grp[v] != 0 and self.grp[v] in ring", "hit = self.grp[v] in ring")],
    "no_prefix_benefit": [("run = max(0.0, run - self.kpf * self.tokens[v] / k)", "run = run")],
    "ring_overwrites_newest": [("            del r[0]\n            r.append(h)", "            r[-1] = h")],
    "p95_over_all_stages": [("for v in done if not I.children[v])", "for v in done)")],
    "xdev_counts_local": [("if I.holders[u] & S == 0:", "if I.holders[u] & S != 0:")],
    "continuation_last_device": [("            if q == 0:\n                hit0 = hit\n                cont0",
                                  "            if q == len(devs) - 1:\n                hit0 = hit\n                cont0")],
    "round_robin_restarts": [("nxt = d + 1", "nxt = 0")],
    "heft_latest_finish": [("if f < best_f:", "if best_d < 0 or f > best_f:")],
    "heft_rank_no_tail": [("rank[v] = wbar + tail", "rank[v] = wbar")],
    "holders_not_updated": [("        self.holders[v] = S\n", "")],
}


def _load_mutant(name, tmp_path):
    src = open(S.__file__).read()
    for old, new in MUTANTS[name]:
        assert src.count(old) == 1, (name, old)
        src = src.replace(old, new)
    path = os.path.join(tmp_path, "sim_%s.py" % name)
    with open(path, "w") as fh:
        fh.write(src)
    spec = importlib.util.spec_from_file_location("sim_" + name, path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_sim_pins_reject_mutant(name, tmp_path, monkeypatch):
    monkeypatch.setattr(sim_pins, "S", _load_mutant(name, str(tmp_path)))
    caught = False
    for _, check in sim_pins.ALL:
        try:
            check()
        except (AssertionError, ValueError, TypeError):
            caught = True
            break
    assert caught, "no simulator pin rejects the planted mistake '%s'" % name
