"""Build small hand-specified workloads for the pinned oracle tests.

Input construction only: a JSON-like dict lists the cluster tables and, per
instance, the parent lists, stage attributes and state arrays.  Nothing here
computes a score.
"""

from __future__ import annotations

import numpy as np

from paper_2605_07238_amd import synth


def from_spec(spec: dict, H: int = 1, params: dict | None = None) -> synth.Workload:
    D, M, K = int(spec["D"]), int(spec["M"]), int(spec.get("K", 1))
    insts = []
    for it in spec["instances"]:
        parents = it["parents"]
        n = len(parents)
        cache = np.array(it.get("prefix_cache", [[0] * K for _ in range(D)]), dtype=np.uint64).reshape(D, K)
        insts.append(dict(
            n=n,
            par_lens=np.array([len(p) for p in parents], np.int64),
            par_flat=np.array([p for ps in parents for p in ps], np.int32),
            model=np.array(it["model"], np.int32),
            elig=np.array([int(e) for e in it["elig"]], np.uint64),
            shard=np.array(it.get("shard_max", [1] * n), np.int32),
            hash=np.array([int(h) for h in it.get("prefix_hash", [0] * n)], np.uint64),
            toks=np.array(it.get("prefix_tokens", [0.0] * n), np.float32),
            sigma=np.array(it["out_bytes"], np.float32),
            resident=np.array([int(r) for r in it["resident"]], np.uint64),
            cache=cache,
            holders=np.array([int(h) for h in it["holders"]], np.uint64),
            status=np.array(it["status"], np.uint8),
            tau=np.array(it["tau_free"], np.float32),
            t_now=np.float32(it["t_now"]),
        ))
    cluster = (
        np.array(spec["exec"], np.float32).reshape(M, D),
        np.array(spec["switch_s"], np.float32).reshape(M, D),
        np.array([int(round(x * synth.GB)) for x in spec["weight_gb"]], np.int64),
        np.array([int(round(x * synth.GB)) for x in spec["cap_gb"]], np.int64),
        np.array(spec["beta"], np.float32).reshape(D, D),
    )
    rc = dict(D=D, M=M, H=H)
    w = synth._assemble(spec.get("title", "spec"), rc, cluster, insts, K, int(spec.get("max_shard", 4)))
    if params:
        w.params.update(params)
    return w
