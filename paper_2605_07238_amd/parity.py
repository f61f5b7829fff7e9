"""Parity comparison between the HIP path's outputs and reference scores.

Pure numpy on host arrays: given the GPU's frontier table, scores and top-k,
and reference scores with their magnitudes (the sum of absolute values of
the weighted terms that went into each score), report the largest error
relative to that magnitude and every top-k rank whose pick differs from the
reference by more than the tolerance.  Used by the tests, the smoke check and
the benchmark; it computes nothing about the method itself.
"""

from __future__ import annotations

import numpy as np


def compare(psi_gpu, psi_ref, mag_ref, rtol=1e-5):
    """Return (max_rel_err, n_bad, n_inf_mismatch) with err relative to mag."""
    g = np.asarray(psi_gpu, np.float64)
    r = np.asarray(psi_ref, np.float64)
    m = np.asarray(mag_ref, np.float64)
    gi, ri = np.isneginf(g), np.isneginf(r)
    inf_bad = int(np.count_nonzero(gi != ri)) + int(np.count_nonzero(~np.isfinite(g) & ~gi))
    fin = ~gi & ~ri & np.isfinite(g)
    if not fin.any():
        return 0.0, 0, inf_bad
    err = np.abs(g[fin] - r[fin]) / np.maximum(m[fin], np.finfo(np.float64).tiny)
    return float(err.max()), int(np.count_nonzero(err > rtol)), inf_bad


def topk_mismatches(idx_gpu, psi_ref, mag_ref, cand_off, k, rtol=1e-5):
    """Ranks where the GPU's pick is not tied (within tolerance) with the
    reference's pick at that rank, plus padding mismatches."""
    bad = 0
    idx_gpu = np.asarray(idx_gpu)
    for f in range(len(cand_off) - 1):
        seg = np.asarray(psi_ref[cand_off[f]:cand_off[f + 1]], np.float64)
        mag = np.asarray(mag_ref[cand_off[f]:cand_off[f + 1]], np.float64)
        order = sorted((j for j in range(len(seg)) if np.isfinite(seg[j])), key=lambda j: (-seg[j], j))
        tol = rtol * (mag.max() if len(mag) else 0.0)
        picks = idx_gpu[f]
        seen = set()
        for rnk in range(k):
            p = int(picks[rnk])
            if rnk >= len(order):
                bad += p != -1
                continue
            if p < 0 or p >= len(seg) or p in seen or not np.isfinite(seg[p]):
                bad += 1
                continue
            seen.add(p)
            if abs(seg[p] - seg[order[rnk]]) > 2 * tol:
                bad += 1
    return bad


def topk_of_scores(psi, cand_off, k):
    """Per-stage top-k of given scores by (score descending, index ascending),
    -inf excluded, padded with -1: the selection rule the top-k kernels
    implement, applied on the host to the same float32 scores."""
    psi = np.asarray(psi, np.float32)
    co = np.asarray(cand_off, np.int64)
    nF = len(co) - 1
    out = np.full((nF, k), -1, np.int32)
    if nF == 0 or k == 0 or co[-1] == 0:
        return out
    C = np.diff(co)
    stage = np.repeat(np.arange(nF), C)
    j = np.arange(co[-1]) - np.repeat(co[:-1], C)
    order = np.lexsort((j, -psi.astype(np.float64), stage))
    order = order[np.isfinite(psi[order])]
    st = stage[order]
    first = np.searchsorted(st, st, side="left")
    rank = np.arange(len(order)) - first
    keep = rank < k
    out[st[keep], rank[keep]] = j[order[keep]]
    return out
