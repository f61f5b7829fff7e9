"""Thin ctypes binding of libfate (include/fate.h).

Argument marshalling only: numpy host arrays are passed by pointer, device
buffers are torch tensors (torch is used for device memory and streams), and
every step of the scoring path runs in libfate's HIP kernels.  There is no
fallback: if the library is missing or a call fails, an exception is raised.

Entry points mirror the C names: :func:`fate_pack_dags`,
:func:`fate_pack_state`, :func:`fate_score_frontier`, :func:`fate_topk`, plus
the host-only :func:`fate_layout_dags` / :func:`fate_layout_state`.
"""

from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# FATE_LIBRARY names another build of the same sources (the sanitizer build).
LIB_PATH = os.environ.get("FATE_LIBRARY") or os.path.join(HERE, "libfate.so")

FATE_OK = 0
FATE_EINVAL, FATE_ERANGE, FATE_ECYCLE, FATE_ENOFEAS, FATE_ESIZE, FATE_ESTATE, FATE_EHIP = -1, -2, -3, -4, -5, -6, -7
STATUS_NAMES = {0: "FATE_OK", -1: "FATE_EINVAL", -2: "FATE_ERANGE", -3: "FATE_ECYCLE", -4: "FATE_ENOFEAS",
                -5: "FATE_ESIZE", -6: "FATE_ESTATE", -7: "FATE_EHIP"}

# Every symbol declared in include/fate.h.
EXPORTS = ["fate_version", "fate_strerror", "fate_pack_dags_size", "fate_pack_dags", "fate_layout_dags",
           "fate_pack_state_size", "fate_pack_state", "fate_layout_state", "fate_score_ws_size",
           "fate_score_frontier", "fate_score_topk", "fate_topk", "fate_pack_state_advance_size",
           "fate_pack_state_advance", "fate_commit_ws_size", "fate_commit_advance", "fate_commit_advance_noalloc",
           "fate_pack_dags_opt_size",
           "fate_pack_dags_opt", "fate_layout_dags_opt", "fate_score_sweep", "fate_topk_sweep", "fate_plan_wave",
           "fate_simulate", "fate_place_baseline", "fate_sim_ws_size", "fate_simulate_device",
           "fate_place_baseline_device"]

# Scoring variants and packing options (fate_params_t.flags, fate_pack_opts_t.levels).
FATE_MEAN_PER_LEVEL, FATE_NO_WINDOWS = 1, 2
FATE_LEVELS_HOP, FATE_LEVELS_TOPO = 0, 1
FATE_MAX_SWEEP = 16
FATE_PLACE_ROUND_ROBIN, FATE_PLACE_HEFT = 0, 1
FATE_NOALLOC_WS_BYTES = 32 << 20  # workspace the library holds per GPU for fate_commit_advance_noalloc


class FateError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (what, STATUS_NAMES.get(status, status), _strerror(status)))


class Cluster(C.Structure):
    _fields_ = [("D", C.c_int32), ("M", C.c_int32), ("exec", C.c_void_p), ("switch_s", C.c_void_p),
                ("weight_bytes", C.c_void_p), ("cap_bytes", C.c_void_p), ("beta", C.c_void_p)]


class DagBatch(C.Structure):
    _fields_ = [("B", C.c_int32), ("stage_off", C.c_void_p), ("par_off", C.c_void_p), ("par_idx", C.c_void_p),
                ("model", C.c_void_p), ("elig", C.c_void_p), ("shard_max", C.c_void_p),
                ("prefix_hash", C.c_void_p), ("prefix_tokens", C.c_void_p), ("out_bytes", C.c_void_p)]


class State(C.Structure):
    _fields_ = [("K", C.c_int32), ("resident", C.c_void_p), ("prefix_cache", C.c_void_p),
                ("holders", C.c_void_p), ("status", C.c_void_p), ("tau_free", C.c_void_p),
                ("t_now", C.c_void_p)]


class Params(C.Structure):
    _fields_ = [("lam_q", C.c_float), ("lam_s", C.c_float), ("lam_tr", C.c_float), ("lam_c", C.c_float),
                ("lam_p", C.c_float), ("kappa_prefix", C.c_float), ("gamma", C.c_float), ("H", C.c_int32),
                ("lam_m", C.c_float), ("flags", C.c_int32)]


class SimMetrics(C.Structure):
    _fields_ = [("tasks", C.c_int64), ("makespan", C.c_double), ("p95", C.c_double), ("xdev_edges", C.c_int64),
                ("cache_hits", C.c_int64), ("model_cont", C.c_int64)]


class PackOpts(C.Structure):
    _fields_ = [("H", C.c_int32), ("levels", C.c_int32), ("level_weights", C.c_int32)]


class Dags(C.Structure):
    _fields_ = [("B", C.c_int32), ("D", C.c_int32), ("M", C.c_int32), ("H", C.c_int32),
                ("N", C.c_int64), ("E", C.c_int64), ("n_desc", C.c_int64),
                ("beta_uniform", C.c_int32), ("beta0", C.c_float),
                ("base", C.c_void_p), ("bytes", C.c_size_t),
                ("exec", C.c_void_p), ("switch_s", C.c_void_p), ("beta", C.c_void_p),
                ("weight", C.c_void_p), ("cap", C.c_void_p), ("fits", C.c_void_p),
                ("records", C.c_void_p), ("par_idx", C.c_void_p), ("desc_off", C.c_void_p),
                ("desc", C.c_void_p), ("stage_off", C.c_void_p), ("levels", C.c_int32), ("desc_w", C.c_void_p),
                ("max_r", C.c_int32), ("ch_off", C.c_void_p), ("ch_idx", C.c_void_p),
                ("max_stages", C.c_int64), ("row_records", C.c_void_p)]


class StateH(C.Structure):
    _fields_ = [("B", C.c_int32), ("D", C.c_int32), ("K", C.c_int32), ("max_shard", C.c_int32),
                ("N", C.c_int64), ("n_frontier", C.c_int64), ("n_cand", C.c_int64),
                ("base", C.c_void_p), ("bytes", C.c_size_t),
                ("resident", C.c_void_p), ("prefix_cache", C.c_void_p), ("holders", C.c_void_p),
                ("tau_free", C.c_void_p), ("t_now", C.c_void_p),
                ("frontier", C.c_void_p), ("cand_off", C.c_void_p),
                ("n_slices", C.c_int64), ("slices", C.c_void_p),
                ("n_done_edges", C.c_int64), ("done_n", C.c_void_p), ("done", C.c_void_p),
                ("advance", C.c_int32), ("status", C.c_void_p), ("counts", C.c_void_p), ("finish", C.c_void_p),
                ("slice", C.c_int32), ("fr_off", C.c_void_p), ("order", C.c_void_p)]


_lib = None


def load(path: Optional[str] = None):
    """Load libfate.so; raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError("libfate.so not found at %s; build it with `python -m paper_2605_07238_amd.build`" % p)
    lib = C.CDLL(p)
    P = C.POINTER
    st = C.c_int
    lib.fate_version.restype = C.c_char_p
    lib.fate_strerror.restype = C.c_char_p
    lib.fate_strerror.argtypes = [st]
    lib.fate_pack_dags_size.argtypes = [P(Cluster), P(DagBatch), C.c_int32, P(C.c_size_t)]
    lib.fate_pack_dags.argtypes = [P(Cluster), P(DagBatch), C.c_int32, C.c_void_p, C.c_size_t, C.c_void_p, P(Dags)]
    lib.fate_layout_dags.argtypes = [P(Cluster), P(DagBatch), C.c_int32, C.c_void_p, C.c_size_t, P(Dags)]
    lib.fate_pack_state_size.argtypes = [P(Dags), P(DagBatch), P(State), C.c_int32, P(C.c_size_t),
                                         P(C.c_int64), P(C.c_int64)]
    lib.fate_pack_state.argtypes = [P(Dags), P(DagBatch), P(State), C.c_int32, C.c_void_p, C.c_size_t,
                                    C.c_void_p, P(StateH)]
    lib.fate_layout_state.argtypes = [P(Dags), P(DagBatch), P(State), C.c_int32, C.c_void_p, C.c_size_t, P(StateH)]
    lib.fate_score_ws_size.argtypes = [P(Dags), P(StateH), P(C.c_size_t)]
    lib.fate_score_frontier.argtypes = [P(Dags), P(StateH), P(Params), C.c_void_p, C.c_int64, C.c_void_p,
                                        C.c_size_t, C.c_void_p]
    lib.fate_score_topk.argtypes = [P(Dags), P(StateH), P(Params), C.c_void_p, C.c_int64, C.c_int32, C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.fate_topk.argtypes = [P(StateH), C.c_void_p, C.c_int64, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.fate_pack_state_advance_size.argtypes = [P(Dags), P(DagBatch), P(State), C.c_int32, P(C.c_size_t)]
    lib.fate_pack_state_advance.argtypes = [P(Dags), P(DagBatch), P(State), C.c_int32, C.c_void_p, C.c_size_t,
                                            C.c_void_p, P(StateH)]
    lib.fate_commit_ws_size.argtypes = [P(Dags), P(StateH), P(C.c_size_t)]
    lib.fate_commit_advance.argtypes = [P(Dags), P(StateH), C.c_void_p, C.c_int32, C.c_void_p, C.c_size_t,
                                        C.c_void_p]
    lib.fate_commit_advance_noalloc.argtypes = [P(Dags), P(StateH), C.c_void_p, C.c_int32, C.c_void_p]
    lib.fate_pack_dags_opt_size.argtypes = [P(Cluster), P(DagBatch), P(PackOpts), P(C.c_size_t)]
    lib.fate_pack_dags_opt.argtypes = [P(Cluster), P(DagBatch), P(PackOpts), C.c_void_p, C.c_size_t, C.c_void_p,
                                       P(Dags)]
    lib.fate_layout_dags_opt.argtypes = [P(Cluster), P(DagBatch), P(PackOpts), C.c_void_p, C.c_size_t, P(Dags)]
    lib.fate_score_sweep.argtypes = [P(Dags), P(StateH), P(Params), C.c_int32, C.c_void_p, C.c_int64, C.c_int64,
                                     C.c_void_p, C.c_size_t, C.c_void_p]
    lib.fate_topk_sweep.argtypes = [P(StateH), C.c_void_p, C.c_int64, C.c_int64, C.c_int32, C.c_int32, C.c_void_p,
                                    C.c_void_p, C.c_void_p]
    lib.fate_plan_wave.argtypes = [P(StateH), C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p]
    lib.fate_simulate.argtypes = [P(Cluster), P(DagBatch), P(State), C.c_void_p, C.c_void_p, C.c_float,
                                  P(SimMetrics)]
    lib.fate_place_baseline.argtypes = [P(Cluster), P(DagBatch), P(State), C.c_int32, C.c_float, C.c_void_p,
                                        C.c_void_p]
    lib.fate_sim_ws_size.argtypes = [P(Dags), P(C.c_size_t)]
    lib.fate_simulate_device.argtypes = [P(Dags), P(StateH), C.c_void_p, C.c_void_p, C.c_float, C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    lib.fate_place_baseline_device.argtypes = [P(Dags), P(StateH), C.c_int32, C.c_float, C.c_void_p, C.c_void_p,
                                               C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
    for name in EXPORTS[2:]:
        getattr(lib, name).restype = st
    if path is None:
        _lib = lib
    return lib


def _strerror(status: int) -> str:
    try:
        return load().fate_strerror(status).decode()
    except Exception:  # noqa: BLE001 - best effort in an error path
        return "?"


def _check(status: int, what: str):
    if status != FATE_OK:
        raise FateError(status, what)


def version() -> str:
    return load().fate_version().decode()


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


class HostInputs:
    """C views of a workload's host arrays (kept alive by this object)."""

    def __init__(self, w):
        self.keep = dict(
            exec=_c(w.exec, np.float32), switch_s=_c(w.switch_s, np.float32),
            weight=_c(w.weight_bytes, np.int64), cap=_c(w.cap_bytes, np.int64), beta=_c(w.beta, np.float32),
            stage_off=_c(w.stage_off, np.int64), par_off=_c(w.par_off, np.int64), par_idx=_c(w.par_idx, np.int32),
            model=_c(w.model, np.int32), elig=_c(w.elig, np.uint64), shard=_c(w.shard_max, np.int32),
            hash=_c(w.prefix_hash, np.uint64), tokens=_c(w.prefix_tokens, np.float32),
            sigma=_c(w.out_bytes, np.float32),
            resident=_c(w.resident, np.uint64), cache=_c(w.prefix_cache, np.uint64),
            holders=_c(w.holders, np.uint64), status=_c(w.status, np.uint8),
            tau=_c(w.tau_free, np.float32), t_now=_c(w.t_now, np.float32),
        )
        k = self.keep
        ptr = lambda a: a.ctypes.data if a.size else None
        self.cluster = Cluster(int(w.D), int(w.M), ptr(k["exec"]), ptr(k["switch_s"]), ptr(k["weight"]),
                               ptr(k["cap"]), ptr(k["beta"]))
        self.batch = DagBatch(int(w.B), k["stage_off"].ctypes.data, ptr(k["par_off"]), ptr(k["par_idx"]),
                              ptr(k["model"]), ptr(k["elig"]), ptr(k["shard"]), ptr(k["hash"]), ptr(k["tokens"]),
                              ptr(k["sigma"]))
        self.state = State(int(w.K), ptr(k["resident"]), ptr(k["cache"]), ptr(k["holders"]), ptr(k["status"]),
                           ptr(k["tau"]), ptr(k["t_now"]))


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class PackedDags:
    def __init__(self, buf, handle: Dags, host: HostInputs):
        self.buf = buf          # torch uint8 device tensor owning the memory
        self.handle = handle
        self.host = host


class PackedState:
    def __init__(self, buf, handle: StateH, host: HostInputs):
        self.buf = buf
        self.handle = handle
        self.host = host

    @property
    def n_frontier(self) -> int:
        return int(self.handle.n_frontier)

    @property
    def n_cand(self) -> int:
        return int(self.handle.n_cand)

    @property
    def advance(self) -> bool:
        return bool(self.handle.advance)

    def counts(self):
        """Current (frontier stages, candidates, slices, rejected selections):
        read from the device for a planning state (synchronises)."""
        import torch
        h = self.handle
        if not h.advance:
            return int(h.n_frontier), int(h.n_cand), int(h.n_slices), 0
        off = h.counts - self.buf.data_ptr()
        c = self.buf[off:off + 16].view(torch.int32).cpu().numpy().astype(np.int64)
        return int(c[0]), int(c[1]), int(c[2]), int(c[3])


def fate_pack_dags_size(w, H: int) -> int:
    hi = HostInputs(w)
    nbytes = C.c_size_t(0)
    _check(load().fate_pack_dags_size(C.byref(hi.cluster), C.byref(hi.batch), int(H), C.byref(nbytes)),
           "fate_pack_dags_size")
    return int(nbytes.value)


def _pack_opts(w, H, levels, level_weights) -> PackOpts:
    p = dict(w.params) if w is not None else {}
    lv = int(levels if levels is not None else (FATE_LEVELS_TOPO if p.get("topo_levels") else FATE_LEVELS_HOP))
    lw = int(bool(level_weights if level_weights is not None else p.get("mean_levels", 0)))
    return PackOpts(int(w.H if H is None else H), lv, lw)


def fate_pack_dags(w, H: Optional[int] = None, device="cuda", stream=None, levels: Optional[int] = None,
                   level_weights: Optional[bool] = None) -> PackedDags:
    """Validate and pack workload ``w``'s DAG batch into a device buffer.
    ``levels`` (FATE_LEVELS_HOP / _TOPO) and ``level_weights`` default to the
    workload's ``topo_levels`` / ``mean_levels`` parameters."""
    import torch
    o = _pack_opts(w, H, levels, level_weights)
    lib = load()
    hi = HostInputs(w)
    nbytes = C.c_size_t(0)
    _check(lib.fate_pack_dags_opt_size(C.byref(hi.cluster), C.byref(hi.batch), C.byref(o), C.byref(nbytes)),
           "fate_pack_dags_opt_size")
    buf = torch.empty(max(1, nbytes.value), dtype=torch.uint8, device=device)
    h = Dags()
    _check(lib.fate_pack_dags_opt(C.byref(hi.cluster), C.byref(hi.batch), C.byref(o), C.c_void_p(buf.data_ptr()),
                                  nbytes.value, C.c_void_p(_stream_ptr(stream)), C.byref(h)), "fate_pack_dags_opt")
    return PackedDags(buf, h, hi)


def fate_layout_dags(w, H: Optional[int] = None, levels: Optional[int] = None,
                     level_weights: Optional[bool] = None):
    """Host-only packed image of the DAG batch: (numpy uint8 buffer, Dags handle)."""
    o = _pack_opts(w, H, levels, level_weights)
    lib = load()
    hi = HostInputs(w)
    nbytes = C.c_size_t(0)
    _check(lib.fate_pack_dags_opt_size(C.byref(hi.cluster), C.byref(hi.batch), C.byref(o), C.byref(nbytes)),
           "fate_pack_dags_opt_size")
    buf = np.zeros(max(1, nbytes.value), np.uint8)
    h = Dags()
    _check(lib.fate_layout_dags_opt(C.byref(hi.cluster), C.byref(hi.batch), C.byref(o), buf.ctypes.data,
                                    nbytes.value, C.byref(h)), "fate_layout_dags_opt")
    return buf, h, hi


def fate_pack_state(packed: PackedDags, w, max_shard: Optional[int] = None, device="cuda",
                    stream=None, advance: bool = False) -> PackedState:
    """Validate the state of ``w`` against ``packed`` and pack state + frontier.
    ``advance`` packs a planning state for fate_commit_advance."""
    import torch
    ms = int(w.max_shard if max_shard is None else max_shard)
    lib = load()
    hi = HostInputs(w)
    nbytes = C.c_size_t(0)
    if advance:
        _check(lib.fate_pack_state_advance_size(C.byref(packed.handle), C.byref(hi.batch), C.byref(hi.state), ms,
                                                C.byref(nbytes)), "fate_pack_state_advance_size")
        buf = torch.empty(max(1, nbytes.value), dtype=torch.uint8, device=device)
        h = StateH()
        _check(lib.fate_pack_state_advance(C.byref(packed.handle), C.byref(hi.batch), C.byref(hi.state), ms,
                                           C.c_void_p(buf.data_ptr()), nbytes.value,
                                           C.c_void_p(_stream_ptr(stream)), C.byref(h)), "fate_pack_state_advance")
        return PackedState(buf, h, hi)
    nf, nc = C.c_int64(0), C.c_int64(0)
    _check(lib.fate_pack_state_size(C.byref(packed.handle), C.byref(hi.batch), C.byref(hi.state), ms,
                                    C.byref(nbytes), C.byref(nf), C.byref(nc)), "fate_pack_state_size")
    buf = torch.empty(max(1, nbytes.value), dtype=torch.uint8, device=device)
    h = StateH()
    _check(lib.fate_pack_state(C.byref(packed.handle), C.byref(hi.batch), C.byref(hi.state), ms,
                               C.c_void_p(buf.data_ptr()), nbytes.value, C.c_void_p(_stream_ptr(stream)),
                               C.byref(h)), "fate_pack_state")
    return PackedState(buf, h, hi)


def fate_layout_state(dags_handle: Dags, w, max_shard: Optional[int] = None):
    """Host-only packed state image: (numpy uint8 buffer, StateH handle)."""
    ms = int(w.max_shard if max_shard is None else max_shard)
    lib = load()
    hi = HostInputs(w)
    nbytes = C.c_size_t(0)
    nf, nc = C.c_int64(0), C.c_int64(0)
    _check(lib.fate_pack_state_size(C.byref(dags_handle), C.byref(hi.batch), C.byref(hi.state), ms,
                                    C.byref(nbytes), C.byref(nf), C.byref(nc)), "fate_pack_state_size")
    buf = np.zeros(max(1, nbytes.value), np.uint8)
    h = StateH()
    _check(lib.fate_layout_state(C.byref(dags_handle), C.byref(hi.batch), C.byref(hi.state), ms, buf.ctypes.data,
                                 nbytes.value, C.byref(h)), "fate_layout_state")
    return buf, h, hi


def make_params(w=None, H: Optional[int] = None, **over) -> Params:
    from . import synth
    p = dict(synth.DEFAULT_PARAMS)
    if w is not None:
        p.update(w.params)
    p.update({k: v for k, v in over.items() if k != "H"})
    Hv = int(H if H is not None else (w.H if w is not None else 0))
    flags = (FATE_MEAN_PER_LEVEL if p.get("mean_levels") else 0) | (FATE_NO_WINDOWS if p.get("no_windows") else 0)
    return Params(p["lam_q"], p["lam_s"], p["lam_tr"], p["lam_c"], p["lam_p"], p["kappa_prefix"], p["gamma"], Hv,
                  float(p.get("lam_m", 0.0)), flags)


def fate_score_frontier(packed: PackedDags, state: PackedState, params: Params, out=None, stream=None):
    """Score every candidate; returns a float32 device tensor [n_cand]."""
    import torch
    lib = load()
    nc = state.n_cand
    if out is None:
        out = torch.empty(max(1, nc), dtype=torch.float32, device=packed.buf.device)
    ws = C.c_size_t(0)
    _check(lib.fate_score_ws_size(C.byref(packed.handle), C.byref(state.handle), C.byref(ws)), "fate_score_ws_size")
    wsbuf = torch.empty(max(1, ws.value), dtype=torch.uint8, device=packed.buf.device) if ws.value else None
    _check(lib.fate_score_frontier(C.byref(packed.handle), C.byref(state.handle), C.byref(params),
                                   C.c_void_p(out.data_ptr()), int(out.numel()),
                                   C.c_void_p(wsbuf.data_ptr()) if wsbuf is not None else None, ws.value,
                                   C.c_void_p(_stream_ptr(stream))), "fate_score_frontier")
    return out


def fate_score_topk(packed: PackedDags, state: PackedState, params: Params, k: int, out=None, idx=None, val=None,
                    stream=None):
    """Scores and per-stage top-k in one launch; returns (scores, idx [F,k], val [F,k])."""
    import torch
    lib = load()
    nc, F = state.n_cand, state.n_frontier
    dev = packed.buf.device
    if out is None:
        out = torch.empty(max(1, nc), dtype=torch.float32, device=dev)
    if idx is None:
        idx = torch.empty((max(1, F), k), dtype=torch.int32, device=dev)
    if val is None:
        val = torch.empty((max(1, F), k), dtype=torch.float32, device=dev)
    ws = C.c_size_t(0)
    _check(lib.fate_score_ws_size(C.byref(packed.handle), C.byref(state.handle), C.byref(ws)), "fate_score_ws_size")
    wsbuf = torch.empty(max(1, ws.value), dtype=torch.uint8, device=dev) if ws.value else None
    _check(lib.fate_score_topk(C.byref(packed.handle), C.byref(state.handle), C.byref(params),
                               C.c_void_p(out.data_ptr()), int(out.numel()), int(k), C.c_void_p(idx.data_ptr()),
                               C.c_void_p(val.data_ptr()),
                               C.c_void_p(wsbuf.data_ptr()) if wsbuf is not None else None, ws.value,
                               C.c_void_p(_stream_ptr(stream))), "fate_score_topk")
    return out, idx[:F], val[:F]


def fate_topk(state: PackedState, scores, k: int, idx=None, val=None, stream=None):
    """Per-frontier-stage top-k; returns (int32 [F, k], float32 [F, k]) device tensors."""
    import torch
    lib = load()
    F = state.n_frontier
    dev = scores.device
    if idx is None:
        idx = torch.empty((max(1, F), k), dtype=torch.int32, device=dev)
    if val is None:
        val = torch.empty((max(1, F), k), dtype=torch.float32, device=dev)
    _check(lib.fate_topk(C.byref(state.handle), C.c_void_p(scores.data_ptr()), int(scores.numel()), int(k),
                         C.c_void_p(idx.data_ptr()), C.c_void_p(val.data_ptr()),
                         C.c_void_p(_stream_ptr(stream))), "fate_topk")
    return idx[:F], val[:F]


def fate_score_sweep(packed: PackedDags, state: PackedState, params, out=None, stride: Optional[int] = None,
                     stream=None):
    """Score every candidate under each of ``params`` (a list of Params, at
    most FATE_MAX_SWEEP) in one launch; returns a float32 device tensor
    [len(params), stride] (set p in row p)."""
    import torch
    lib = load()
    P = len(params)
    stride = int(stride if stride is not None else max(1, state.n_cand))
    if out is None:
        out = torch.empty((max(1, P), stride), dtype=torch.float32, device=packed.buf.device)
    arr = (Params * max(1, P))(*params)
    _check(lib.fate_score_sweep(C.byref(packed.handle), C.byref(state.handle), arr, int(P),
                                C.c_void_p(out.data_ptr()), int(out.numel()), stride, None, 0,
                                C.c_void_p(_stream_ptr(stream))), "fate_score_sweep")
    return out


def fate_topk_sweep(state: PackedState, scores, k: int, idx=None, val=None, stream=None):
    """Top-k of every row of a [P, stride] score tensor (the fate_score_sweep
    layout); returns (int32 [P, F, k], float32 [P, F, k]) device tensors, F the
    handle's frontier size (its capacity for a planning state)."""
    import torch
    lib = load()
    P, stride = int(scores.shape[0]), int(scores.shape[1])
    F = state.n_frontier
    dev = scores.device
    if idx is None:
        idx = torch.empty((P, max(1, F), k), dtype=torch.int32, device=dev)
    if val is None:
        val = torch.empty((P, max(1, F), k), dtype=torch.float32, device=dev)
    _check(lib.fate_topk_sweep(C.byref(state.handle), C.c_void_p(scores.data_ptr()), int(scores.numel()), stride,
                               P, int(k), C.c_void_p(idx.data_ptr()), C.c_void_p(val.data_ptr()),
                               C.c_void_p(_stream_ptr(stream))), "fate_topk_sweep")
    return idx[:, :F], val[:, :F]


def fate_plan_wave(state: PackedState, idx, val, sel=None, stream=None):
    """One frontier planning wave from per-stage choices ``idx`` / ``val``
    ([F, k] device tensors, the fate_topk layout); returns the int32 device
    tensor sel [F] (-1 = not placed in this wave)."""
    import torch
    lib = load()
    F = state.n_frontier
    k = int(idx.shape[1]) if idx.dim() == 2 else 1
    if sel is None:
        sel = torch.empty(max(1, F), dtype=torch.int32, device=idx.device)
    _check(lib.fate_plan_wave(C.byref(state.handle), C.c_void_p(idx.data_ptr()), C.c_void_p(val.data_ptr()), k,
                              C.c_void_p(sel.data_ptr()), C.c_void_p(_stream_ptr(stream))), "fate_plan_wave")
    return sel[:F]


def fate_simulate(w, devices, order, kappa_prefix: Optional[float] = None) -> dict:
    """Execute a placement (host arrays: devices [N] uint64 masks, order [N]
    int64 keys) on every instance of ``w``; returns per-instance numpy arrays
    tasks, makespan, p95, xdev_edges, cache_hits, model_cont."""
    lib = load()
    hi = HostInputs(w)
    kpf = float(w.params["kappa_prefix"] if kappa_prefix is None else kappa_prefix)
    dev = np.ascontiguousarray(devices, np.uint64)
    odr = np.ascontiguousarray(order, np.int64)
    out = (SimMetrics * max(1, w.B))()
    _check(lib.fate_simulate(C.byref(hi.cluster), C.byref(hi.batch), C.byref(hi.state), dev.ctypes.data,
                             odr.ctypes.data, kpf, out), "fate_simulate")
    res = {}
    for name, _ in SimMetrics._fields_:
        res[name] = np.array([getattr(out[b], name) for b in range(w.B)],
                             np.float64 if name in ("makespan", "p95") else np.int64)
    return res


def fate_place_baseline(w, policy: int, kappa_prefix: Optional[float] = None):
    """Round-robin or HEFT-style placement of ``w``'s pending stages:
    (devices [N] uint64, order [N] int64) host arrays."""
    lib = load()
    hi = HostInputs(w)
    kpf = float(w.params["kappa_prefix"] if kappa_prefix is None else kappa_prefix)
    dev = np.zeros(w.N, np.uint64)
    odr = np.zeros(w.N, np.int64)
    _check(lib.fate_place_baseline(C.byref(hi.cluster), C.byref(hi.batch), C.byref(hi.state), int(policy), kpf,
                                   dev.ctypes.data, odr.ctypes.data), "fate_place_baseline")
    return dev, odr


def fate_commit_ws_size(packed: PackedDags, state: PackedState) -> int:
    ws = C.c_size_t(0)
    _check(load().fate_commit_ws_size(C.byref(packed.handle), C.byref(state.handle), C.byref(ws)),
           "fate_commit_ws_size")
    return int(ws.value)


def fate_commit_advance(packed: PackedDags, state: PackedState, sel, ws=None, stream=None):
    """Commit the candidate chosen per frontier slot and advance the planning
    state on the device.  ``sel``: int32 device tensor [F] or [F, k] (a top-k
    array: its first column is used), -1 = leave pending.  Returns ``ws``."""
    import torch
    lib = load()
    if sel.dtype != torch.int32 or not sel.is_contiguous():
        raise ValueError("sel must be a contiguous int32 tensor")
    stride = int(sel.shape[1]) if sel.dim() == 2 else 1
    nbytes = fate_commit_ws_size(packed, state)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=packed.buf.device)
    _check(lib.fate_commit_advance(C.byref(packed.handle), C.byref(state.handle), C.c_void_p(sel.data_ptr()),
                                   stride, C.c_void_p(ws.data_ptr()), nbytes, C.c_void_p(_stream_ptr(stream))),
           "fate_commit_advance")
    return ws


def fate_commit_advance_noalloc(packed: PackedDags, state: PackedState, sel, stream=None):
    """fate_commit_advance with the library-held workspace (no device
    allocation by the library or here).  ``sel`` as for fate_commit_advance."""
    import torch
    if sel.dtype != torch.int32 or not sel.is_contiguous():
        raise ValueError("sel must be a contiguous int32 tensor")
    stride = int(sel.shape[1]) if sel.dim() == 2 else 1
    _check(load().fate_commit_advance_noalloc(C.byref(packed.handle), C.byref(state.handle),
                                              C.c_void_p(sel.data_ptr()), stride, C.c_void_p(_stream_ptr(stream))),
           "fate_commit_advance_noalloc")


def fate_sim_ws_size(packed: PackedDags) -> int:
    n = C.c_size_t(0)
    _check(load().fate_sim_ws_size(C.byref(packed.handle), C.byref(n)), "fate_sim_ws_size")
    return int(n.value)


def _sim_status(status, what: str):
    bad = status.cpu().numpy()
    nz = np.nonzero(bad != FATE_OK)[0]
    if len(nz):
        raise FateError(int(bad[nz[0]]), "%s (instance %d)" % (what, int(nz[0])))


def fate_simulate_device(packed: PackedDags, state: PackedState, devices, order, kappa_prefix: float,
                         ws=None, stream=None) -> dict:
    """Execute a placement on the device: ``devices`` uint64 (as int64) and
    ``order`` int64 device tensors [N] over flat stage ids.  Returns the
    per-instance metrics as numpy arrays (tasks, makespan, p95, xdev_edges,
    cache_hits, model_cont); raises on a per-instance error status."""
    import torch
    lib = load()
    dev = packed.buf.device
    for t, nm in ((devices, "devices"), (order, "order")):
        if t.dtype != torch.int64 or not t.is_contiguous() or t.numel() < packed.handle.N:
            raise ValueError("%s must be a contiguous int64 tensor of N elements" % nm)
    nbytes = fate_sim_ws_size(packed)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=dev)
    B = int(packed.handle.B)
    out = torch.empty((max(1, B), C.sizeof(SimMetrics)), dtype=torch.uint8, device=dev)
    status = torch.empty(max(1, B), dtype=torch.int32, device=dev)
    _check(lib.fate_simulate_device(C.byref(packed.handle), C.byref(state.handle), C.c_void_p(devices.data_ptr()),
                                    C.c_void_p(order.data_ptr()), float(kappa_prefix), C.c_void_p(out.data_ptr()),
                                    C.c_void_p(status.data_ptr()), C.c_void_p(ws.data_ptr()), nbytes,
                                    C.c_void_p(_stream_ptr(stream))), "fate_simulate_device")
    _sim_status(status[:B], "fate_simulate_device")
    raw = out[:B].cpu().numpy()
    rec = np.frombuffer(raw.tobytes(), dtype=np.dtype([(name, np.float64 if name in ("makespan", "p95") else np.int64)
                                                       for name, _ in SimMetrics._fields_]), count=B)
    return {name: np.array(rec[name]) for name, _ in SimMetrics._fields_}


def fate_place_baseline_device(packed: PackedDags, state: PackedState, policy: int, kappa_prefix: float,
                               ws=None, stream=None):
    """Round-robin or HEFT-style placement built on the device: (devices,
    order) int64 device tensors [N] (devices holds the uint64 masks)."""
    import torch
    lib = load()
    dev = packed.buf.device
    N, B = int(packed.handle.N), int(packed.handle.B)
    nbytes = fate_sim_ws_size(packed)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(1, nbytes), dtype=torch.uint8, device=dev)
    devices = torch.empty(max(1, N), dtype=torch.int64, device=dev)
    order = torch.empty(max(1, N), dtype=torch.int64, device=dev)
    status = torch.empty(max(1, B), dtype=torch.int32, device=dev)
    _check(lib.fate_place_baseline_device(C.byref(packed.handle), C.byref(state.handle), int(policy),
                                          float(kappa_prefix), C.c_void_p(devices.data_ptr()),
                                          C.c_void_p(order.data_ptr()), C.c_void_p(status.data_ptr()),
                                          C.c_void_p(ws.data_ptr()), nbytes, C.c_void_p(_stream_ptr(stream))),
           "fate_place_baseline_device")
    _sim_status(status[:B], "fate_place_baseline_device")
    return devices[:N], order[:N]


def state_arrays(state: PackedState):
    """Host copies of the packed state arrays: resident [B, D], prefix slots
    [B, D, K], holders [N], free times [B, D], and (planning state) status [N]
    and planned finish [N]."""
    import torch
    h = state.handle
    base = state.buf.data_ptr()
    B, D, K, N = int(h.B), int(h.D), int(h.K), int(h.N)

    def take(ptr, n, dt):
        off = ptr - base
        nb = n * np.dtype(dt).itemsize
        if n == 0:
            return np.zeros(0, dt)
        return state.buf[off:off + nb].cpu().numpy().view(dt).copy()

    out = dict(resident=take(h.resident, B * D, np.uint64).reshape(B, D),
               prefix_cache=take(h.prefix_cache, B * D * K, np.uint64).reshape(B, D, K),
               holders=take(h.holders, N, np.uint64), tau_free=take(h.tau_free, B * D, np.float32).reshape(B, D))
    if h.advance:
        out["status"] = take(h.status, N, np.uint8)
        out["finish"] = take(h.finish, N, np.float32)
    return out


def frontier_table(state: PackedState):
    """Host copies of the packed frontier: (flat stage ids, instances, cand_off)."""
    import torch
    h = state.handle
    F = state.counts()[0]
    base = state.buf.data_ptr()
    off_f = h.frontier - base
    off_c = h.cand_off - base
    fr = state.buf[off_f:off_f + 8 * F].view(torch.int32).cpu().numpy().reshape(F, 2) if F else np.zeros((0, 2), np.int32)
    co = state.buf[off_c:off_c + 4 * (F + 1)].view(torch.int32).cpu().numpy()
    return fr[:, 0].astype(np.int64), fr[:, 1].astype(np.int64), co.astype(np.int64)


def desc_counts(packed: PackedDags):
    """Host copy of every stage's horizon-descendant count (from desc_off)."""
    import torch
    h = packed.handle
    N = int(h.N)
    off = h.desc_off - packed.buf.data_ptr()
    do = packed.buf[off:off + 4 * (N + 1)].view(torch.int32).cpu().numpy().astype(np.int64)
    return np.diff(do)
