"""CPU oracle for NetKV decode-instance selection -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports, links or calls it, and this package never imports
the product.  The arithmetic lives in ``netkv_oracle.c`` (plain C, fp64);
this module only builds it with gcc and marshals numpy arrays through ctypes.

Sources of every computed quantity are cited in ``netkv_oracle.c``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "netkv_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_netkv.so")
# a checking build (build_sanitized) loaded instead of the default one
_LIB_OVERRIDE = os.environ.get("NETKV_ORACLE_LIB")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no intrinsics)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def build_sanitized(path: str) -> str:
    """Compile the oracle with AddressSanitizer and UndefinedBehaviorSanitizer
    (every report fatal) into `path`.  A process loads it by setting
    NETKV_ORACLE_LIB=path and preloading gcc's libasan (the ASan runtime must
    come first)."""
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-o", path, _SRC, "-lm"])
    return path


class _Snap(C.Structure):
    _fields_ = [
        ("n_prefill", C.c_uint32), ("n_decode", C.c_uint32),
        ("tier_map", C.c_void_p), ("util", C.c_void_p), ("n_inflight", C.c_void_p),
        ("tier_bw", C.c_double * 4), ("tier_lat", C.c_double * 4),
        ("free_mem", C.c_void_p), ("queue_depth", C.c_void_p), ("batch_size", C.c_void_p),
        ("t_iter_a", C.c_double), ("t_iter_b", C.c_double), ("beta_max", C.c_uint32),
        ("alpha", C.c_double), ("m_min", C.c_uint64), ("kv_bytes_per_token", C.c_uint64),
        ("block_tokens", C.c_uint32),
        ("route_tier1", C.c_void_p), ("route_util1", C.c_void_p),
        ("route_tier2", C.c_void_p), ("route_util2", C.c_void_p),
    ]


class _Flows(C.Structure):
    _fields_ = [("n_links", C.c_uint32), ("cap", C.c_void_p), ("n_flows", C.c_uint32),
                ("path_off", C.c_void_p), ("path", C.c_void_p), ("bytes", C.c_void_p), ("start", C.c_void_p)]


class _Req(C.Structure):
    _fields_ = [("n_req", C.c_uint32), ("prefill", C.c_void_p), ("len_tokens", C.c_void_p),
                ("hash_off", C.c_void_p), ("hashes", C.c_void_p)]


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = C.CDLL(_LIB_OVERRIDE)
        else:
            build(force=False)
            lib = C.CDLL(_LIB)
        lib.orc_cache_build.restype = C.c_void_p
        lib.orc_cache_build.argtypes = [C.c_uint32, C.c_void_p, C.c_void_p, C.c_int]
        lib.orc_cache_free.argtypes = [C.c_void_p]
        lib.orc_select.restype = C.c_uint64
        lib.orc_select.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint32,
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_int]
        lib.orc_rank_sweep.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint32,
                                       C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_int]
        lib.orc_tier_inversions.argtypes = [C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p, C.c_int]
        lib.orc_commit.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_uint32, C.c_uint32, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p]
        lib.orc_select_sequential.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint32,
                                              C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        lib.orc_tier_counts.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        lib.orc_prefix_len.restype = C.c_uint32
        lib.orc_prefix_len.argtypes = [C.c_void_p, C.c_uint32, C.c_void_p, C.c_uint32]
        lib.orc_route_of.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p]
        lib.orc_smooth.restype = C.c_uint64
        lib.orc_smooth.argtypes = [C.c_void_p, C.c_void_p, C.c_uint64, C.c_double]
        lib.orc_max_threads.restype = C.c_int
        lib.orc_selection_bytes.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint32, C.c_void_p,
                                            C.c_void_p]
        lib.orc_pair_congestion.argtypes = [C.c_uint32, C.c_uint32] + [C.c_void_p] * 12
        lib.orc_ar1_step.argtypes = [C.c_uint64, C.c_void_p, C.c_void_p, C.c_void_p, C.c_double, C.c_double,
                                     C.c_void_p]
        lib.orc_link_noise.argtypes = [C.c_uint64, C.c_void_p, C.c_void_p, C.c_double, C.c_void_p]
        lib.orc_maxmin.restype = C.c_uint32
        lib.orc_maxmin.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        lib.orc_flow_sim.restype = C.c_uint64
        lib.orc_flow_sim.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _arr(a, dt):
    return np.ascontiguousarray(np.asarray(a, dtype=dt))


class Snapshot:
    """Keeps the numpy arrays alive behind the C struct."""

    def __init__(self, snap: Dict[str, object]):
        self.keep = dict(
            tier_map=_arr(snap["tier_map"], np.uint8), util=_arr(snap["util"], np.float32),
            n_inflight=_arr(snap["n_inflight"], np.uint16),
            free_mem=_arr(snap["free_mem"], np.uint64),
            queue_depth=_arr(snap["queue_depth"], np.uint32),
            batch_size=_arr(snap["batch_size"], np.uint32))
        s = _Snap()
        s.n_prefill = int(snap["n_prefill"])
        s.n_decode = int(snap["n_decode"])
        for f in ("tier_map", "util", "n_inflight", "free_mem", "queue_depth", "batch_size"):
            setattr(s, f, self.keep[f].ctypes.data)
        for i in range(4):
            s.tier_bw[i] = float(snap["tier_bw"][i])
            s.tier_lat[i] = float(snap["tier_lat"][i])
        s.t_iter_a = float(snap["t_iter_a"])
        s.t_iter_b = float(snap["t_iter_b"])
        s.beta_max = int(snap["beta_max"])
        s.alpha = float(snap["alpha"])
        s.m_min = int(snap["m_min"])
        s.kv_bytes_per_token = int(snap["kv_bytes_per_token"])
        s.block_tokens = int(snap["block_tokens"])
        if snap.get("route_tier1") is not None:   # two-hop routing (Sec. VIII)
            for f, dt in (("route_tier1", np.uint8), ("route_util1", np.float32),
                          ("route_tier2", np.uint8), ("route_util2", np.float32)):
                self.keep[f] = _arr(np.asarray(snap[f]).reshape(-1), dt)
                setattr(s, f, self.keep[f].ctypes.data)
        self.s = s
        self.n_prefill, self.n_decode = s.n_prefill, s.n_decode


class Requests:
    def __init__(self, req: Dict[str, np.ndarray]):
        self.keep = dict(prefill=_arr(req["prefill"], np.uint32),
                         len_tokens=_arr(req["len_tokens"], np.uint32),
                         hash_off=_arr(req["hash_off"], np.uint64),
                         hashes=_arr(req["hashes"], np.uint64))
        r = _Req()
        r.n_req = len(self.keep["prefill"])
        for f in ("prefill", "len_tokens", "hash_off", "hashes"):
            setattr(r, f, self.keep[f].ctypes.data)
        self.r = r
        self.n_req = r.n_req


class Cache:
    """Sorted copies of every decode's resident hash list."""

    def __init__(self, cache: Dict[str, np.ndarray], n_threads: int = 1):
        lib = _load()
        off = _arr(cache["hash_off"], np.uint64)
        h = _arr(cache["hashes"], np.uint64)
        self.n_decode = len(off) - 1
        self.h = lib.orc_cache_build(self.n_decode, off.ctypes.data, h.ctypes.data, int(n_threads))

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.orc_cache_free(self.h)
            self.h = None

    def prefix_len(self, d: int, hashes: np.ndarray) -> int:
        hashes = _arr(hashes, np.uint64)
        return int(_load().orc_prefix_len(self.h, d, hashes.ctypes.data, len(hashes)))


def max_threads() -> int:
    return int(_load().orc_max_threads())


def select(snap, cache, req, k: int = 1, pairs: bool = False, n_threads: int = 1):
    """Top-k selection for every request.

    Returns dict(idx [R,k] int32, score [R,k] float64, tests (sum of
    membership tests), and if ``pairs``: j [R,D] uint32, feasible [R,D]
    uint8, cost [R,D] float64)."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    c = cache if isinstance(cache, Cache) else Cache(cache)
    q = req if isinstance(req, Requests) else Requests(req)
    R, D = q.n_req, s.n_decode
    idx = np.empty((R, k), dtype=np.int32)
    score = np.empty((R, k), dtype=np.float64)
    out = dict(idx=idx, score=score)
    pj = pf = pc = None
    if pairs:
        pj = np.empty((R, D), dtype=np.uint32)
        pf = np.empty((R, D), dtype=np.uint8)
        pc = np.empty((R, D), dtype=np.float64)
        out.update(j=pj, feasible=pf, cost=pc)
    out["tests"] = int(lib.orc_select(C.byref(s.s), c.h, C.byref(q.r), k, idx.ctypes.data,
                                      score.ctypes.data, _ptr(pj), _ptr(pf), _ptr(pc),
                                      int(n_threads)))
    return out


def rank_sweep(snap, cache, req, util_scen: np.ndarray, k: int = 3, n_threads: int = 1):
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    c = cache if isinstance(cache, Cache) else Cache(cache)
    q = req if isinstance(req, Requests) else Requests(req)
    u = _arr(util_scen, np.float32)
    S = u.shape[0]
    R = q.n_req
    idx = np.empty((S, R, k), dtype=np.int32)
    score = np.empty((S, R, k), dtype=np.float64)
    flips = np.empty((S, 2), dtype=np.uint64)
    lib.orc_rank_sweep(C.byref(s.s), c.h, C.byref(q.r), S, u.ctypes.data, k, idx.ctypes.data,
                       score.ctypes.data, flips.ctypes.data, int(n_threads))
    return dict(idx=idx, score=score, flips=flips)


def tier_inversions(snap, util_scen: np.ndarray, n_threads: int = 1) -> np.ndarray:
    """Proposition 2's quantity per congestion scenario (netkv_oracle.c):
    [S, 3] = (pairs the sufficient condition covers, inverted pairs among
    them, all inverted pairs), over pairs of decodes on different tiers."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    u = _arr(util_scen, np.float32)
    S = u.shape[0]
    assert u.size == S * s.n_prefill * s.n_decode
    out = np.empty((S, 3), dtype=np.uint64)
    lib.orc_tier_inversions(C.byref(s.s), S, u.ctypes.data, out.ctypes.data, int(n_threads))
    return out


def commit(snap, cache, req, sel: np.ndarray, cap: int, mu: int, state: Dict[str, np.ndarray]):
    """Between-batch state update (in place on copies); returns the new state
    dict with n_inflight, queue_depth, free_mem, admitted_prev."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    c = cache if isinstance(cache, Cache) else Cache(cache)
    q = req if isinstance(req, Requests) else Requests(req)
    st = dict(n_inflight=_arr(state["n_inflight"], np.uint16).copy(),
              queue_depth=_arr(state["queue_depth"], np.uint32).copy(),
              free_mem=_arr(state["free_mem"], np.uint64).copy(),
              admitted_prev=_arr(state["admitted_prev"], np.uint64).copy())
    sel = _arr(sel, np.int32)
    lib.orc_commit(C.byref(s.s), c.h, C.byref(q.r), sel.ctypes.data, int(cap), int(mu),
                   st["n_inflight"].ctypes.data, st["queue_depth"].ctypes.data,
                   st["free_mem"].ctypes.data, st["admitted_prev"].ctypes.data)
    return st


def select_sequential(snap, cache, req, cap: int = 16, follow: Optional[np.ndarray] = None):
    """Algorithm 1 request by request in batch order (in-flight counters
    incremented after each selection).  Returns dict(idx [R], score [R],
    and with `follow`: follow_cost [R])."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    c = cache if isinstance(cache, Cache) else Cache(cache)
    q = req if isinstance(req, Requests) else Requests(req)
    R = q.n_req
    idx = np.empty(R, dtype=np.int32)
    score = np.empty(R, dtype=np.float64)
    fc = None
    f = None
    if follow is not None:
        f = _arr(follow, np.int32)
        fc = np.empty(R, dtype=np.float64)
    lib.orc_select_sequential(C.byref(s.s), c.h, C.byref(q.r), int(cap), _ptr(f), idx.ctypes.data,
                              score.ctypes.data, _ptr(fc))
    out = dict(idx=idx, score=score)
    if fc is not None:
        out["follow_cost"] = fc
    return out


def tier_counts(snap, req, sel: np.ndarray) -> np.ndarray:
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    q = req if isinstance(req, Requests) else Requests(req)
    sel = _arr(sel, np.int32)
    out = np.empty(5, dtype=np.uint64)
    lib.orc_tier_counts(C.byref(s.s), C.byref(q.r), sel.ctypes.data, out.ctypes.data)
    return out


def smooth(c: np.ndarray, obs: np.ndarray, beta: float):
    """One step of the predictive-congestion smoothing (Sec. VIII): returns
    (the new fp64 congestion, the number of observations outside [0, 1))."""
    lib = _load()
    out = np.array(c, dtype=np.float64, copy=True).reshape(-1)
    o = _arr(np.asarray(obs, np.float32).reshape(-1), np.float32)
    assert o.size == out.size
    bad = lib.orc_smooth(out.ctypes.data, o.ctypes.data, C.c_uint64(out.size), C.c_double(beta))
    return out, int(bad)


def route_of(snap, cache, req, idx: np.ndarray, k: int) -> np.ndarray:
    """Two-hop routing (Sec. VIII): 1 where a selection's staged route is
    strictly faster, 0 direct, -1 no selection."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    q = req if isinstance(req, Requests) else Requests(req)
    cc = cache if isinstance(cache, Cache) else Cache(cache)
    idx = _arr(np.asarray(idx).reshape(-1), np.int32)
    out = np.empty(idx.size, dtype=np.int8)
    lib.orc_route_of(C.byref(s.s), cc.h, C.byref(q.r), int(k), idx.ctypes.data, out.ctypes.data)
    return out


def selection_bytes(snap, cache, req, idx: np.ndarray, k: int) -> np.ndarray:
    """Eq. (2)'s non-cached bytes of each selection idx [R*k] (0 for none)."""
    lib = _load()
    s = snap if isinstance(snap, Snapshot) else Snapshot(snap)
    q = req if isinstance(req, Requests) else Requests(req)
    cc = cache if isinstance(cache, Cache) else Cache(cache)
    idx = _arr(np.asarray(idx).reshape(-1), np.int32)
    out = np.empty(idx.size, dtype=np.uint64)
    lib.orc_selection_bytes(C.byref(s.s), cc.h, C.byref(q.r), int(k), idx.ctypes.data, out.ctypes.data)
    return out


class Flows:
    """A flow set for the transfer simulation: link capacities cap [L]
    (bytes/s), per flow a path (CSR path_off [N+1], path: link ids), bytes
    [N] and start [N] (s)."""

    def __init__(self, f):
        self.keep = dict(cap=_arr(f["cap"], np.float64), path_off=_arr(f["path_off"], np.uint64),
                         path=_arr(f["path"], np.uint32), bytes=_arr(f["bytes"], np.float64),
                         start=_arr(f["start"], np.float64))
        k = self.keep
        self.n = len(k["bytes"])
        assert len(k["path_off"]) == self.n + 1 and len(k["start"]) == self.n
        assert (k["cap"] > 0).all() and (np.diff(k["path_off"].astype(np.int64)) > 0).all()
        if len(k["path"]):
            assert int(k["path"].max()) < len(k["cap"])
        self.s = _Flows(len(k["cap"]), k["cap"].ctypes.data, self.n, k["path_off"].ctypes.data,
                        k["path"].ctypes.data if len(k["path"]) else None, k["bytes"].ctypes.data,
                        k["start"].ctypes.data)


def maxmin(flows, active=None):
    """Max-min fair rates (progressive filling) of the active flows
    (default: all).  Returns (rates [N] float64, filling rounds)."""
    lib = _load()
    fl = flows if isinstance(flows, Flows) else Flows(flows)
    act = np.ones(fl.n, np.uint8) if active is None else _arr(np.asarray(active, np.uint8), np.uint8)
    rate = np.empty(fl.n, np.float64)
    rounds = lib.orc_maxmin(C.byref(fl.s), act.ctypes.data, rate.ctypes.data)
    return rate, int(rounds)


def flow_sim(flows, stats: bool = False):
    """Event-driven transfer simulation under max-min fair link sharing.
    Returns (finish times [N] float64, number of allocations computed), and
    with stats also (allocations, filling rounds, flows in progress summed
    over the allocations)."""
    lib = _load()
    fl = flows if isinstance(flows, Flows) else Flows(flows)
    fin = np.empty(fl.n, np.float64)
    st = np.zeros(3, np.uint64)
    ev = lib.orc_flow_sim(C.byref(fl.s), fin.ctypes.data, st.ctypes.data)
    if stats:
        return fin, int(ev), tuple(int(x) for x in st)
    return fin, int(ev)


# ---------------------------------------------------------------- telemetry derivations

def pair_congestion(p_coords, d_coords, links):
    """Per-pair tier and congestion from per-link utilisation (netkv_oracle.c,
    orc_pair_congestion).  p_coords / d_coords: (node, leaf, pod) index
    arrays of each prefill / decode instance's GPU; links: dict u0..u3.
    Returns (tier [P, D] uint8, util [P, D] float32)."""
    lib = _load()
    pn, pl, pp = (_arr(x, np.uint32) for x in p_coords)
    dn, dl, dp = (_arr(x, np.uint32) for x in d_coords)
    u = [_arr(links[f"u{t}"], np.float64) for t in range(4)]
    P, D = len(pn), len(dn)
    tier = np.empty((P, D), np.uint8)
    util = np.empty((P, D), np.float32)
    lib.orc_pair_congestion(P, D, pn.ctypes.data, pl.ctypes.data, pp.ctypes.data, dn.ctypes.data,
                            dl.ctypes.data, dp.ctypes.data, *[x.ctypes.data for x in u], tier.ctypes.data,
                            util.ctypes.data)
    return tier, util


def ar1_step(cur, mean, eps, rho: float, sigma: float) -> np.ndarray:
    """One AR(1) step of link utilisations (orc_ar1_step)."""
    lib = _load()
    c, m, e = (_arr(x, np.float64) for x in (cur, mean, eps))
    out = np.empty(len(c), np.float64)
    lib.orc_ar1_step(len(c), c.ctypes.data, m.ctypes.data, e.ctypes.data, float(rho), float(sigma),
                     out.ctypes.data)
    return out


def link_noise(u, z, sigma: float) -> np.ndarray:
    """Lognormal telemetry noise on link utilisations (orc_link_noise)."""
    lib = _load()
    a, b = _arr(u, np.float64), _arr(z, np.float64)
    out = np.empty(len(a), np.float64)
    lib.orc_link_noise(len(a), a.ctypes.data, b.ctypes.data, float(sigma), out.ctypes.data)
    return out
