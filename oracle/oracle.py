"""Python front end of the fp64 CPU oracle (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this module.  It compiles ``fate_oracle.c`` with gcc
on first use (or when the source is newer than the library), marshals a
:class:`~paper_2605_07238_amd.synth.Workload`'s flat arrays into the C input
record and returns plain numpy arrays.  It never touches the HIP library.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading
from typing import Dict, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "fate_oracle.c")
# FATE_ORACLE_LIBRARY names another build of the same source (the sanitizer build).
LIB = os.environ.get("FATE_ORACLE_LIBRARY") or os.path.join(HERE, "libfate_oracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False, src: str = SRC, out: str = LIB) -> str:
    """Compile the oracle (plain C, fp64, OpenMP over instances)."""
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-shared", "-fPIC", "-Wall", "-Wextra",
               "-Wno-unused-parameter", src, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


SAN_LIB = os.path.join(HERE, "_build_san", "libfate_oracle_san.so")


def build_sanitized(out: str = SAN_LIB) -> str:
    """The oracle built with clang's AddressSanitizer and
    UndefinedBehaviorSanitizer (load it with the matching runtime preloaded;
    OpenMP off, so the build needs no sanitized OpenMP runtime)."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    clang = "/opt/rocm/llvm/bin/clang"
    cmd = [clang, "-O1", "-g", "-std=c11", "-shared", "-fPIC", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libasan",
           "-Wno-unknown-pragmas", SRC, "-o", out, "-lm"]
    subprocess.run(cmd, check=True)
    return out


class _In(C.Structure):
    _fields_ = [
        ("D", C.c_int), ("M", C.c_int), ("K", C.c_int), ("H", C.c_int), ("max_shard", C.c_int),
        ("exec", C.c_void_p), ("switch_s", C.c_void_p), ("beta", C.c_void_p),
        ("weight", C.c_void_p), ("cap", C.c_void_p),
        ("stage_off", C.c_void_p), ("par_off", C.c_void_p),
        ("par_idx", C.c_void_p), ("model", C.c_void_p), ("shard", C.c_void_p),
        ("elig", C.c_void_p), ("hash", C.c_void_p),
        ("tokens", C.c_void_p), ("sigma", C.c_void_p),
        ("resident", C.c_void_p), ("cache", C.c_void_p),
        ("holders", C.c_void_p), ("status", C.c_void_p),
        ("tau", C.c_void_p), ("t_now", C.c_void_p),
        ("lam_q", C.c_double), ("lam_s", C.c_double), ("lam_tr", C.c_double),
        ("lam_c", C.c_double), ("lam_p", C.c_double), ("kappa_prefix", C.c_double),
        ("gamma", C.c_double),
        ("lam_m", C.c_double), ("topo_levels", C.c_int), ("mean_levels", C.c_int), ("no_windows", C.c_int),
    ]


def load(path: Optional[str] = None):
    """Load (building if needed) the oracle library; ``path`` loads another
    build of the same source (used by tests that plant mistakes)."""
    global _lib
    if path is not None:
        lib = C.CDLL(path)
        _bind(lib)
        return lib
    with _lock:
        if _lib is None:
            build()
            _lib = C.CDLL(LIB)
            _bind(_lib)
    return _lib


def _bind(lib):
    lib.oracle_count.argtypes = [C.POINTER(_In), C.c_int, C.c_void_p, C.c_void_p]
    lib.oracle_count.restype = C.c_int
    lib.oracle_score.argtypes = [C.POINTER(_In), C.c_int, C.c_void_p, C.c_void_p, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_void_p, C.c_int]
    lib.oracle_score.restype = C.c_int
    lib.oracle_topk.argtypes = [C.c_void_p, C.c_int64, C.c_int, C.c_void_p, C.c_void_p]
    lib.oracle_topk.restype = C.c_int
    lib.oracle_frontier.argtypes = [C.POINTER(_In), C.c_int, C.c_void_p, C.c_void_p]
    lib.oracle_frontier.restype = C.c_int
    lib.oracle_commit.argtypes = [C.POINTER(_In), C.c_int, C.c_void_p, C.c_void_p, C.c_void_p,
                                  C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.oracle_commit.restype = C.c_int
    lib.oracle_plan_wave.argtypes = [C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int,
                                     C.c_void_p]
    lib.oracle_plan_wave.restype = C.c_int


def f32(x: float) -> float:
    """Round a parameter to float32, the precision the GPU receives it in."""
    return float(np.float32(x))


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def _record(w, params=None, H=None, max_shard=None):
    """The C input record for workload ``w`` (and the arrays it points into)."""
    p = dict(w.params)
    if params:
        p.update(params)
    keep = dict(
        exec=_c(w.exec, np.float32), switch_s=_c(w.switch_s, np.float32), beta=_c(w.beta, np.float32),
        weight=_c(w.weight_bytes, np.int64), cap=_c(w.cap_bytes, np.int64),
        stage_off=_c(w.stage_off, np.int64), par_off=_c(w.par_off, np.int64),
        par_idx=_c(w.par_idx, np.int32), model=_c(w.model, np.int32), shard=_c(w.shard_max, np.int32),
        elig=_c(w.elig, np.uint64), hash=_c(w.prefix_hash, np.uint64),
        tokens=_c(w.prefix_tokens, np.float32), sigma=_c(w.out_bytes, np.float32),
        resident=_c(w.resident, np.uint64), cache=_c(w.prefix_cache, np.uint64),
        holders=_c(w.holders, np.uint64), status=_c(w.status, np.uint8),
        tau=_c(w.tau_free, np.float32), t_now=_c(w.t_now, np.float32),
    )
    rec = _In()
    rec.D, rec.M, rec.K = int(w.D), int(w.M), int(w.K)
    rec.H = int(w.H if H is None else H)
    rec.max_shard = int(w.max_shard if max_shard is None else max_shard)
    for k, a in keep.items():
        setattr(rec, k, a.ctypes.data)
    for k in ("lam_q", "lam_s", "lam_tr", "lam_c", "lam_p", "kappa_prefix", "gamma"):
        setattr(rec, k, f32(p[k]))
    # scoring variants, off unless asked for: same-model weight, topological
    # levels, mean per level, no windows
    rec.lam_m = f32(p.get("lam_m", 0.0))
    rec.topo_levels = int(bool(p.get("topo_levels", 0)))
    rec.mean_levels = int(bool(p.get("mean_levels", 0)))
    rec.no_windows = int(bool(p.get("no_windows", 0)))
    return rec, keep


def score(w, params: Optional[Dict[str, float]] = None, H: Optional[int] = None,
          max_shard: Optional[int] = None, threads: Optional[int] = None, lib=None) -> dict:
    """Score every candidate of every frontier stage of workload ``w``.

    Returns a dict with ``front_b``, ``front_v`` (instance-local ids),
    ``cand_off`` ([n_frontier+1], global candidate offsets), ``psi`` and
    ``mag`` (fp64, per candidate) and ``nf`` (frontier size per instance).
    Parameters are rounded to float32 first, as the GPU path sees them.
    """
    lib = lib or load()
    rec, keep = _record(w, params, H, max_shard)
    B = w.B
    nf = np.zeros(B, np.int64)
    nc = np.zeros(B, np.int64)
    lib.oracle_count(C.byref(rec), B, nf.ctypes.data, nc.ctypes.data)
    f_off = np.zeros(B + 1, np.int64)
    c_off = np.zeros(B + 1, np.int64)
    f_off[1:] = np.cumsum(nf)
    c_off[1:] = np.cumsum(nc)
    F, NC = int(f_off[-1]), int(c_off[-1])
    front_v = np.zeros(F, np.int32)
    cand_off = np.zeros(F + 1, np.int64)
    psi = np.zeros(NC, np.float64)
    mag = np.zeros(NC, np.float64)
    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    rc = lib.oracle_score(C.byref(rec), B, f_off.ctypes.data, c_off.ctypes.data, front_v.ctypes.data,
                          cand_off.ctypes.data, psi.ctypes.data, mag.ctypes.data, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the input (code %d)" % rc)
    cand_off[F] = NC
    front_b = np.repeat(np.arange(B, dtype=np.int32), nf)
    return dict(front_b=front_b, front_v=front_v, cand_off=cand_off, psi=psi, mag=mag, nf=nf)


def topk(res: dict, k: int, lib=None):
    """Per-frontier-stage top-k of an oracle result: (idx [F,k], val [F,k])."""
    lib = lib or load()
    F = len(res["front_v"])
    idx = np.full((F, k), -1, np.int32)
    val = np.full((F, k), -np.inf, np.float64)
    psi = res["psi"]
    co = res["cand_off"]
    for f in range(F):
        seg = np.ascontiguousarray(psi[co[f]:co[f + 1]])
        lib.oracle_topk(seg.ctypes.data, int(co[f + 1] - co[f]), int(k),
                        idx[f].ctypes.data, val[f].ctypes.data)
    return idx, val


def frontier(w, max_shard: Optional[int] = None, lib=None):
    """Frontier of ``w``: (front_b, front_v instance-local, f_off [B+1], cand_off [F+1])."""
    lib = lib or load()
    rec, keep = _record(w, None, None, max_shard)
    B = w.B
    nf = np.zeros(B, np.int64)
    nc = np.zeros(B, np.int64)
    lib.oracle_count(C.byref(rec), B, nf.ctypes.data, nc.ctypes.data)
    f_off = np.zeros(B + 1, np.int64)
    f_off[1:] = np.cumsum(nf)
    front_v = np.zeros(int(f_off[-1]), np.int32)
    lib.oracle_frontier(C.byref(rec), B, f_off.ctypes.data, front_v.ctypes.data)
    front_b = np.repeat(np.arange(B, dtype=np.int32), nf)
    return front_b, front_v, f_off


def initial_finish(w):
    """Planned finish times at the start of planning: t for completed stages
    (their outputs are available when planning begins), 0 for the others
    (never read before they are committed).  float32, the planning state's
    format."""
    inst = np.repeat(np.arange(w.B), np.diff(w.stage_off))
    return np.where(w.status == 1, np.asarray(w.t_now, np.float32)[inst], 0.0).astype(np.float32)


def commit(w, sel, max_shard: Optional[int] = None, lib=None, fin=None):
    """Commit-and-advance (oracle step 11): apply the candidate ``sel[f]``
    chosen for each frontier slot f of ``w`` (-1 = leave pending).  ``fin``
    [N] holds the planned finish times of completed stages (default:
    initial_finish(w), the start of planning).

    Returns (new workload, tau in fp64 [B, D], number of rejected
    selections, fin [N] float32).  The new workload is a copy of ``w`` whose
    resident models, prefix slots, holders, statuses and free times (rounded
    to float32, the state's format) are the committed state; fin gains the
    committed stages' planned finish, rounded to float32 the same way."""
    import dataclasses
    lib = lib or load()
    front_b, front_v, f_off = frontier(w, max_shard, lib)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    if sel.shape != (len(front_v),):
        raise ValueError("one selection per frontier slot expected (%d), got %s" % (len(front_v), sel.shape))
    rec, keep = _record(w, None, None, max_shard)
    res = np.array(w.resident, dtype=np.uint64, copy=True)
    cache = np.array(w.prefix_cache, dtype=np.uint64, copy=True)
    holders = np.array(w.holders, dtype=np.uint64, copy=True)
    status = np.array(w.status, dtype=np.uint8, copy=True)
    tau = np.array(w.tau_free, dtype=np.float64, copy=True)
    fin64 = np.array(initial_finish(w) if fin is None else fin, dtype=np.float32).astype(np.float64)
    rejected = lib.oracle_commit(C.byref(rec), w.B, f_off.ctypes.data, front_v.ctypes.data, sel.ctypes.data,
                                 res.ctypes.data, cache.ctypes.data, holders.ctypes.data, status.ctypes.data,
                                 tau.ctypes.data, fin64.ctypes.data)
    new = dataclasses.replace(w, resident=res, prefix_cache=cache, holders=holders, status=status,
                              tau_free=tau.astype(np.float32))
    return new, tau, int(rejected), fin64.astype(np.float32)


def plan_wave(D: int, f_off, n_cand, idx, val, lib=None):
    """One frontier planning wave (oracle step 12).  ``f_off`` [B+1] gives
    each instance's frontier slots, ``n_cand`` [F] each slot's number of
    candidates; ``idx`` / ``val`` [F, k] are each slot's choices (local
    candidate indices, -1 = none) and their float32 scores.  Returns
    (sel [F] int32, -1 = not assigned in this wave; stages assigned)."""
    lib = lib or load()
    f_off = np.ascontiguousarray(f_off, np.int64)
    n_cand = np.ascontiguousarray(n_cand, np.int64)
    idx = np.ascontiguousarray(idx, np.int32)
    val = np.ascontiguousarray(val, np.float32)
    F = int(f_off[-1])
    if idx.ndim != 2 or idx.shape[0] != F or val.shape != idx.shape or n_cand.shape != (F,):
        raise ValueError("idx / val must be [F, k] and n_cand [F] with F = f_off[-1]")
    sel = np.full(F, -1, np.int32)
    n = lib.oracle_plan_wave(len(f_off) - 1, int(D), f_off.ctypes.data, n_cand.ctypes.data, idx.ctypes.data,
                             val.ctypes.data, int(idx.shape[1]), sel.ctypes.data)
    return sel, int(n)
