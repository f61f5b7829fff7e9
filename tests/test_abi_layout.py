"""The binding's ctypes mirrors of the public structs against the header:
a small C program built with the host compiler prints every field's offset
and each struct's size, and the mirrors must agree field by field (a field
added to the header but not to the binding, or in another place, shifts
every later offset)."""

import ctypes as C
import os
import subprocess

import pytest

from paper_2605_07238_amd import fate

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

STRUCTS = [
    ("fate_cluster_t", fate.Cluster),
    ("fate_dag_batch_t", fate.DagBatch),
    ("fate_state_t", fate.State),
    ("fate_params_t", fate.Params),
    ("fate_sim_metrics_t", fate.SimMetrics),
    ("fate_pack_opts_t", fate.PackOpts),
    ("fate_dags_t", fate.Dags),
    ("fate_state_h", fate.StateH),
]


@pytest.fixture(scope="module")
def c_layout(tmp_path_factory):
    d = tmp_path_factory.mktemp("abi")
    src = ['#include <stddef.h>', '#include <stdio.h>', '#include "fate.h"', "int main(void) {"]
    for cname, py in STRUCTS:
        src.append('printf("%s size %%zu\\n", sizeof(%s));' % (cname, cname))
        for fname, _ in py._fields_:
            src.append('printf("%s %s %%zu\\n", offsetof(%s, %s));' % (cname, fname, cname, fname))
    src.append("return 0; }")
    (d / "layout.c").write_text("\n".join(src) + "\n")
    exe = d / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(d / "layout.c"), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    table = {}
    for line in out.splitlines():
        s, f, v = line.split()
        table[(s, f)] = int(v)
    return table


@pytest.mark.parametrize("cname,py", STRUCTS, ids=[s[0] for s in STRUCTS])
def test_mirror_matches_header(c_layout, cname, py):
    assert C.sizeof(py) == c_layout[(cname, "size")], "size"
    for fname, _ in py._fields_:
        assert getattr(py, fname).offset == c_layout[(cname, fname)], fname
