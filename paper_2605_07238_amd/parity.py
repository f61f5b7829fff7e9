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
    reference's pick at that rank, plus padding mismatches.  Two candidates
    count as tied when their reference scores differ by at most the sum of
    their own tolerances, rtol * (A_p + A_q): each GPU score may sit rtol * A
    away from its reference.  A pick must be a finite-scored candidate of its
    stage, listed once."""
    idx_gpu = np.asarray(idx_gpu, np.int64)
    psi = np.asarray(psi_ref, np.float64)
    mag = np.asarray(mag_ref, np.float64)
    co = np.asarray(cand_off, np.int64)
    nF = len(co) - 1
    if nF == 0 or k == 0:
        return 0
    ref = _topk_order(psi, co, k).astype(np.int64)
    got = idx_gpu[:nF, :k]
    C = np.diff(co)[:, None]
    c0 = co[:-1, None]
    q_ok = ref >= 0
    p_in = (got >= 0) & (got < C)
    pos_p = c0 + np.where(p_in, got, 0)
    pos_q = c0 + np.where(q_ok, ref, 0)
    last = max(len(psi) - 1, 0)
    sp = psi[np.minimum(pos_p, last)] if len(psi) else np.zeros_like(pos_p, np.float64)
    sq = psi[np.minimum(pos_q, last)] if len(psi) else np.zeros_like(pos_q, np.float64)
    mp = mag[np.minimum(pos_p, last)] if len(mag) else np.zeros_like(pos_p, np.float64)
    mq = mag[np.minimum(pos_q, last)] if len(mag) else np.zeros_like(pos_q, np.float64)
    srt = np.sort(got, axis=1)
    dup = np.zeros_like(got, bool)
    dup[:, 1:] = (srt[:, 1:] == srt[:, :-1]) & (srt[:, 1:] >= 0)
    n_dup = int(dup.sum())
    pad_bad = ~q_ok & (got != -1)
    pick_bad = q_ok & (~p_in | ~np.isfinite(sp))
    with np.errstate(invalid="ignore"):  # -inf - -inf where the pick is already counted
        far = q_ok & ~pick_bad & (np.abs(sp - sq) > rtol * (mp + mq))
    return int(pad_bad.sum() + pick_bad.sum() + far.sum()) + n_dup


def _topk_order(psi, cand_off, k):
    """Per-stage top-k indices of ``psi`` by (score descending, index
    ascending), -inf excluded, padded with -1."""
    co = np.asarray(cand_off, np.int64)
    nF = len(co) - 1
    out = np.full((nF, k), -1, np.int32)
    if nF == 0 or k == 0 or co[-1] == 0:
        return out
    C = np.diff(co)
    stage = np.repeat(np.arange(nF), C)
    j = np.arange(co[-1]) - np.repeat(co[:-1], C)
    order = np.lexsort((j, -np.asarray(psi, np.float64)[:co[-1]], stage))
    order = order[np.isfinite(np.asarray(psi)[order])]
    st = stage[order]
    first = np.searchsorted(st, st, side="left")
    rank = np.arange(len(order)) - first
    keep = rank < k
    out[st[keep], rank[keep]] = j[order[keep]]
    return out


def topk_of_scores(psi, cand_off, k):
    """Per-stage top-k of given scores by (score descending, index ascending),
    -inf excluded, padded with -1: the selection rule the top-k kernels
    implement, applied on the host to the same float32 scores."""
    return _topk_order(np.asarray(psi, np.float32), cand_off, k)
