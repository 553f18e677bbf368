"""ctypes binding of libnetkv (include/netkv.h) -- argument marshalling only.

Every function named ``netkv_*`` here calls the C function of the same name;
it checks tensor dtypes, shapes, devices and contiguity, passes raw device
pointers and the current HIP stream, and raises :class:`NetKVError` on a
non-zero status.  All scoring, matching, selection and state updates run in
the library's HIP kernels; PyTorch only provides device memory and streams.

The library must have been built (``python -m paper_2606_03910_amd.build``
or ``__graft_entry__.build()``); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libnetkv.so")

NETKV_OK = 0
STATUS = {0: "OK", -1: "EINVAL", -2: "ENOTREADY", -3: "ENOMEM", -4: "EDEVICE", -5: "ECAPACITY"}

_lib = None


class NetKVError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"netkv {STATUS.get(status, status)}: {msg}")
        self.status = status


class netkv_oracle_t(C.Structure):
    _fields_ = [
        ("n_prefill", C.c_uint32), ("n_decode", C.c_uint32),
        ("tier_map", C.c_void_p), ("util", C.c_void_p),
        ("tier_bw", C.c_double * 4), ("tier_lat", C.c_double * 4),
        ("n_inflight", C.c_void_p), ("free_mem", C.c_void_p),
        ("queue_depth", C.c_void_p), ("batch_size", C.c_void_p),
        ("t_iter_a", C.c_double), ("t_iter_b", C.c_double), ("beta_max", C.c_uint32),
        ("alpha", C.c_double), ("m_min", C.c_uint64), ("kv_bytes_per_token", C.c_uint64),
        ("block_tokens", C.c_uint32),
    ]


class netkv_requests_t(C.Structure):
    _fields_ = [("n_req", C.c_uint32), ("prefill", C.c_void_p), ("len_tokens", C.c_void_p),
                ("hash_off", C.c_void_p), ("hashes", C.c_void_p), ("n_hashes", C.c_uint64)]


class netkv_pairs_t(C.Structure):
    _fields_ = [("prefix_blocks", C.c_void_p), ("feasible", C.c_void_p), ("score", C.c_void_p)]


_SIGS = {
    "netkv_create": (C.c_int32, [C.POINTER(C.c_void_p), C.c_int]),
    "netkv_destroy": (None, [C.c_void_p]),
    "netkv_last_error": (C.c_char_p, [C.c_void_p]),
    "netkv_oracle_load": (C.c_int32, [C.c_void_p, C.POINTER(netkv_oracle_t), C.c_void_p]),
    "netkv_oracle_set_util": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "netkv_congestion_smooth": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_float, C.c_void_p]),
    "netkv_congestion_get": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p]),
    "netkv_route2_load": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                      C.c_void_p]),
    "netkv_route2_clear": (C.c_int32, [C.c_void_p]),
    "netkv_route2_of": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32, C.c_void_p,
                                    C.c_void_p, C.c_void_p]),
    "netkv_cache_load": (C.c_int32, [C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p, C.c_uint64,
                                     C.c_float, C.c_void_p]),
    "netkv_select_batch": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32,
                                       C.c_void_p, C.c_void_p, C.POINTER(netkv_pairs_t),
                                       C.c_void_p]),
    "netkv_select_batch_noalloc": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32,
                                               C.c_void_p, C.c_void_p, C.c_void_p]),
    "netkv_reserve": (C.c_int32, [C.c_void_p, C.c_uint32, C.c_uint64, C.c_uint32, C.c_void_p]),
    "netkv_rank_sweep": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32,
                                     C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p, C.c_void_p,
                                     C.c_void_p, C.c_void_p]),
    "netkv_commit_batch": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_void_p,
                                       C.c_uint32, C.c_uint32, C.c_void_p]),
    "netkv_state_get": (C.c_int32, [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                    C.c_void_p]),
    "netkv_sync_errors": (C.c_int32, [C.c_void_p, C.c_void_p]),
    "netkv_set_timing": (C.c_int32, [C.c_void_p, C.c_int]),
    "netkv_kernel_ms": (C.c_int32, [C.c_void_p, C.POINTER(C.c_float)]),
    "netkv_cache_info": (C.c_int32, [C.c_void_p, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                     C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]),
    "netkv_set_option": (C.c_int32, [C.c_void_p, C.c_int, C.c_uint32]),
    "netkv_tier_counts": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_void_p, C.c_void_p,
                                      C.c_void_p]),
    "netkv_select_sequential": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32,
                                            C.c_void_p, C.c_void_p, C.c_void_p]),
    "netkv_selection_bytes": (C.c_int32, [C.c_void_p, C.POINTER(netkv_requests_t), C.c_uint32, C.c_void_p,
                                          C.c_void_p, C.c_void_p]),
    "netkv_flow_sim": (C.c_int32, [C.c_void_p, C.c_uint32, C.c_uint32, C.c_void_p, C.c_void_p, C.c_uint64,
                                   C.c_void_p, C.c_void_p, C.c_uint64, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p]),
}

NETKV_OPT_RUN_LEN = 1
NETKV_OPT_REUSE = 2
NETKV_OPT_COLS = 3
NETKV_OPT_POLICY = 4
NETKV_OPT_LEAD_CAP = 5


def load_library(path: str = LIB_PATH):
    """Load libnetkv.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"libnetkv.so not built at {path}: run __graft_entry__.build()")
        torch.cuda.is_available  # torch's HIP runtime is mapped before ours binds to it
        lib = C.CDLL(path)
        _one_hip_runtime()
        for name, (res, args) in _SIGS.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def _one_hip_runtime():
    """libnetkv binds to the HIP runtime torch has already mapped (same
    SONAME).  Two different runtimes in one process would make torch's
    streams and allocations foreign to the library: refuse that."""
    try:
        with open("/proc/self/maps") as f:
            maps = f.read()
    except OSError:
        return
    paths = {ln.split()[-1] for ln in maps.splitlines()
             if ln.rstrip().endswith(".so") or "libamdhip64" in ln}
    hip = {os.path.realpath(p) for p in paths if "libamdhip64" in os.path.basename(p)}
    if len(hip) > 1:
        raise RuntimeError(f"two HIP runtimes are mapped ({sorted(hip)}); import torch before "
                           "loading libnetkv")


def _check(h, st: int):
    if st != NETKV_OK:
        msg = load_library().netkv_last_error(h)
        raise NetKVError(st, msg.decode() if msg else "")


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _dptr(t: Optional[torch.Tensor], dtype, n: Optional[int] = None, name: str = "tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} CUDA tensor")
    if n is not None and t.numel() < n:
        raise ValueError(f"{name} has {t.numel()} elements, needs {n}")
    return t.data_ptr()


# ---------------------------------------------------------------- C functions

def netkv_create(device: int = 0) -> int:
    h = C.c_void_p()
    st = load_library().netkv_create(C.byref(h), int(device))
    if st != NETKV_OK:
        raise NetKVError(st, f"netkv_create(device={device}) failed")
    return h.value


def netkv_destroy(h: int) -> None:
    load_library().netkv_destroy(h)


def netkv_last_error(h: int) -> str:
    m = load_library().netkv_last_error(h)
    return m.decode() if m else ""


def netkv_oracle_load(h: int, snap: Dict[str, object], device) -> None:
    """snap: dict with the fields of netkv_oracle_t; arrays as CUDA tensors."""
    P, D = int(snap["n_prefill"]), int(snap["n_decode"])
    o = netkv_oracle_t()
    o.n_prefill, o.n_decode = P, D
    o.tier_map = _dptr(snap["tier_map"], torch.uint8, P * D, "tier_map")
    o.util = _dptr(snap["util"], torch.float32, P * D, "util")
    o.n_inflight = _dptr(snap["n_inflight"], torch.uint16, 4 * P, "n_inflight")
    o.free_mem = _dptr(snap["free_mem"], torch.uint64, D, "free_mem")
    o.queue_depth = _dptr(snap["queue_depth"], torch.uint32, D, "queue_depth")
    o.batch_size = _dptr(snap["batch_size"], torch.uint32, D, "batch_size")
    for i in range(4):
        o.tier_bw[i] = float(snap["tier_bw"][i])
        o.tier_lat[i] = float(snap["tier_lat"][i])
    o.t_iter_a, o.t_iter_b = float(snap["t_iter_a"]), float(snap["t_iter_b"])
    o.beta_max, o.alpha = int(snap["beta_max"]), float(snap["alpha"])
    o.m_min, o.kv_bytes_per_token = int(snap["m_min"]), int(snap["kv_bytes_per_token"])
    o.block_tokens = int(snap["block_tokens"])
    _check(h, load_library().netkv_oracle_load(h, C.byref(o), _stream(device)))


def netkv_oracle_set_util(h: int, util: torch.Tensor, device) -> None:
    _check(h, load_library().netkv_oracle_set_util(h, _dptr(util, torch.float32, name="util"),
                                                   _stream(device)))


def netkv_congestion_smooth(h: int, obs: torch.Tensor, beta: float, device) -> None:
    _check(h, load_library().netkv_congestion_smooth(h, _dptr(obs, torch.float32, name="obs"), float(beta),
                                                     _stream(device)))


def netkv_congestion_get(h: int, out: torch.Tensor, device) -> None:
    _check(h, load_library().netkv_congestion_get(h, _dptr(out, torch.float32, name="out"), _stream(device)))


def netkv_route2_load(h: int, tier1: torch.Tensor, util1: torch.Tensor, tier2: torch.Tensor,
                      util2: torch.Tensor, device) -> None:
    _check(h, load_library().netkv_route2_load(
        h, _dptr(tier1, torch.uint8, name="tier1"), _dptr(util1, torch.float32, name="util1"),
        _dptr(tier2, torch.uint8, name="tier2"), _dptr(util2, torch.float32, name="util2"), _stream(device)))


def netkv_route2_clear(h: int) -> None:
    _check(h, load_library().netkv_route2_clear(h))


def netkv_route2_of(h: int, req: Dict[str, torch.Tensor], k: int, idx: torch.Tensor, out_route: torch.Tensor,
                    device) -> None:
    r = _requests(req)
    _check(h, load_library().netkv_route2_of(h, C.byref(r), int(k),
                                             _dptr(idx, torch.int32, r.n_req * k, "idx"),
                                             _dptr(out_route, torch.int8, r.n_req * k, "out_route"),
                                             _stream(device)))


def netkv_selection_bytes(h: int, req: Dict[str, torch.Tensor], k: int, idx: torch.Tensor,
                          out_bytes: torch.Tensor, device) -> None:
    r = _requests(req)
    _check(h, load_library().netkv_selection_bytes(h, C.byref(r), int(k),
                                                   _dptr(idx, torch.int32, r.n_req * k, "idx"),
                                                   _dptr(out_bytes, torch.uint64, r.n_req * k, "out_bytes"),
                                                   _stream(device)))


def netkv_flow_sim(h: int, n_inst: int, n_links: int, cap: torch.Tensor, flow_off: torch.Tensor,
                   path_off: torch.Tensor, path: torch.Tensor, nbytes: torch.Tensor, start: torch.Tensor,
                   finish: torch.Tensor, stats: Optional[torch.Tensor], device) -> None:
    n_flows = int(nbytes.numel())
    n_path = int(path.numel())
    _check(h, load_library().netkv_flow_sim(
        h, int(n_inst), int(n_links), _dptr(cap, torch.float64, n_inst * n_links, "cap"),
        _dptr(flow_off, torch.uint64, n_inst + 1, "flow_off"), n_flows,
        _dptr(path_off, torch.uint64, n_flows + 1, "path_off"), _dptr(path, torch.uint32, name="path"), n_path,
        _dptr(nbytes, torch.float64, n_flows, "bytes"), _dptr(start, torch.float64, n_flows, "start"),
        _dptr(finish, torch.float64, n_flows, "finish"),
        _dptr(stats, torch.uint64, 3 * n_inst, "stats") if stats is not None else None, _stream(device)))


def netkv_cache_load(h: int, n_decode: int, hash_off: torch.Tensor, hashes: torch.Tensor,
                     max_load_factor: float, device) -> None:
    _check(h, load_library().netkv_cache_load(
        h, int(n_decode), _dptr(hash_off, torch.uint64, n_decode + 1, "hash_off"),
        _dptr(hashes, torch.uint64, name="hashes"), int(hashes.numel()),
        float(max_load_factor), _stream(device)))


def _requests(req: Dict[str, torch.Tensor]) -> netkv_requests_t:
    n = int(req["prefill"].numel())
    r = netkv_requests_t()
    r.n_req = n
    r.prefill = _dptr(req["prefill"], torch.uint32, n, "prefill")
    r.len_tokens = _dptr(req["len_tokens"], torch.uint32, n, "len_tokens")
    r.hash_off = _dptr(req["hash_off"], torch.uint64, n + 1, "hash_off")
    r.hashes = _dptr(req["hashes"], torch.uint64, name="hashes")
    r.n_hashes = int(req["hashes"].numel())
    return r


def netkv_select_batch(h: int, req: Dict[str, torch.Tensor], k: int, out_idx: torch.Tensor,
                       out_score: torch.Tensor, pairs: Optional[Dict[str, torch.Tensor]],
                       device) -> None:
    r = _requests(req)
    n = r.n_req
    pp = None
    if pairs is not None:
        D = pairs["n_decode"]
        pp = netkv_pairs_t()
        pp.prefix_blocks = _dptr(pairs.get("prefix_blocks"), torch.uint16, n * D, "prefix_blocks")
        pp.feasible = _dptr(pairs.get("feasible"), torch.uint8, n * D, "feasible")
        pp.score = _dptr(pairs.get("score"), torch.float32, n * D, "score")
    _check(h, load_library().netkv_select_batch(
        h, C.byref(r), int(k), _dptr(out_idx, torch.int32, n * k, "out_idx"),
        _dptr(out_score, torch.float32, n * k, "out_score"),
        C.byref(pp) if pp is not None else None, _stream(device)))


def netkv_select_batch_noalloc(h: int, req: Dict[str, torch.Tensor], k: int, out_idx: torch.Tensor,
                               out_score: torch.Tensor, device) -> None:
    r = _requests(req)
    n = r.n_req
    _check(h, load_library().netkv_select_batch_noalloc(
        h, C.byref(r), int(k), _dptr(out_idx, torch.int32, n * k, "out_idx"),
        _dptr(out_score, torch.float32, n * k, "out_score"), _stream(device)))


def netkv_reserve(h: int, max_req: int, max_hashes: int, max_k: int, device) -> None:
    _check(h, load_library().netkv_reserve(h, int(max_req), int(max_hashes), int(max_k), _stream(device)))


def netkv_rank_sweep(h: int, req: Dict[str, torch.Tensor], n_scen: int, util_scen: torch.Tensor,
                     k: int, out_idx: torch.Tensor, out_score: torch.Tensor,
                     out_flips: Optional[torch.Tensor], device, n_cells: int,
                     out_inversions: Optional[torch.Tensor] = None) -> None:
    r = _requests(req)
    n = r.n_req
    _check(h, load_library().netkv_rank_sweep(
        h, C.byref(r), int(n_scen), _dptr(util_scen, torch.float32, n_scen * n_cells, "util_scen"),
        int(k), _dptr(out_idx, torch.int32, n_scen * n * k, "out_idx"),
        _dptr(out_score, torch.float32, n_scen * n * k, "out_score"),
        _dptr(out_flips, torch.uint64, 2 * n_scen, "out_flips"),
        _dptr(out_inversions, torch.uint64, 3 * n_scen, "out_inversions"), _stream(device)))


def netkv_commit_batch(h: int, req: Dict[str, torch.Tensor], sel: torch.Tensor, cap: int, mu: int,
                       device) -> None:
    r = _requests(req)
    _check(h, load_library().netkv_commit_batch(h, C.byref(r), _dptr(sel, torch.int32, r.n_req, "sel"),
                                                int(cap), int(mu), _stream(device)))


def netkv_state_get(h: int, P: int, D: int, device) -> Dict[str, np.ndarray]:
    out = dict(n_inflight=np.empty(4 * P, np.uint16), queue_depth=np.empty(D, np.uint32),
               free_mem=np.empty(D, np.uint64), admitted_prev=np.empty(D, np.uint64))
    _check(h, load_library().netkv_state_get(h, out["n_inflight"].ctypes.data,
                                             out["queue_depth"].ctypes.data,
                                             out["free_mem"].ctypes.data,
                                             out["admitted_prev"].ctypes.data, _stream(device)))
    return out


def netkv_sync_errors(h: int, device) -> None:
    _check(h, load_library().netkv_sync_errors(h, _stream(device)))


def netkv_set_timing(h: int, enable: bool) -> None:
    _check(h, load_library().netkv_set_timing(h, int(bool(enable))))


def netkv_kernel_ms(h: int) -> float:
    ms = C.c_float()
    _check(h, load_library().netkv_kernel_ms(h, C.byref(ms)))
    return float(ms.value)


def netkv_tier_counts(h: int, req: Dict[str, torch.Tensor], sel: torch.Tensor, counts: torch.Tensor,
                      device) -> None:
    r = _requests(req)
    _check(h, load_library().netkv_tier_counts(h, C.byref(r), _dptr(sel, torch.int32, r.n_req, "sel"),
                                               _dptr(counts, torch.uint64, 5, "counts"), _stream(device)))


def netkv_select_sequential(h: int, req: Dict[str, torch.Tensor], cap: int, out_idx: torch.Tensor,
                            out_score: torch.Tensor, device) -> None:
    r = _requests(req)
    _check(h, load_library().netkv_select_sequential(
        h, C.byref(r), int(cap), _dptr(out_idx, torch.int32, r.n_req, "out_idx"),
        _dptr(out_score, torch.float32, r.n_req, "out_score"), _stream(device)))


def netkv_set_option(h: int, option: int, value: int) -> None:
    _check(h, load_library().netkv_set_option(h, int(option), int(value)))


def netkv_cache_info(h: int) -> Dict[str, int]:
    v = [C.c_uint64() for _ in range(4)]
    _check(h, load_library().netkv_cache_info(h, *[C.byref(x) for x in v]))
    return dict(index_slots=int(v[0].value), distinct_hashes=int(v[1].value),
                shared_hashes=int(v[2].value), index_bytes=int(v[3].value))


# ---------------------------------------------------------------- convenience

_SIGNED_TWIN = {np.dtype(np.uint16): (np.int16, torch.uint16),
                np.dtype(np.uint32): (np.int32, torch.uint32),
                np.dtype(np.uint64): (np.int64, torch.uint64)}


def to_device(a: np.ndarray, device) -> torch.Tensor:
    """Copy a numpy array to the device; unsigned types travel as their
    signed twins and are re-viewed on the device (bit-identical)."""
    a = np.ascontiguousarray(a)
    if a.dtype in _SIGNED_TWIN:
        st, ut = _SIGNED_TWIN[a.dtype]
        return torch.from_numpy(a.view(st)).to(device).view(ut)
    return torch.from_numpy(a).to(device)


def to_numpy(t: torch.Tensor) -> np.ndarray:
    """Device tensor to numpy, unsigned types bit-identical."""
    tw = {torch.uint16: (torch.int16, np.uint16), torch.uint32: (torch.int32, np.uint32),
          torch.uint64: (torch.int64, np.uint64)}
    if t.dtype in tw:
        st, un = tw[t.dtype]
        return t.view(st).cpu().numpy().view(un)
    return t.cpu().numpy()


def requests_to_device(req: Dict[str, np.ndarray], device) -> Dict[str, torch.Tensor]:
    return {k: to_device(np.asarray(req[k], dt), device) for k, dt in
            (("prefill", np.uint32), ("len_tokens", np.uint32), ("hash_off", np.uint64),
             ("hashes", np.uint64))}


class Selector:
    """A handle on one device with its snapshot and resident-set tables."""

    def __init__(self, device: int = 0):
        self.device = torch.device("cuda", device)
        self.h = netkv_create(device)
        self.P = self.D = 0

    def close(self):
        if self.h:
            netkv_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def load_snapshot(self, snap: Dict[str, object]) -> None:
        dev = self.device
        d = dict(snap)
        for k, dt in (("tier_map", np.uint8), ("util", np.float32), ("n_inflight", np.uint16),
                      ("free_mem", np.uint64), ("queue_depth", np.uint32),
                      ("batch_size", np.uint32)):
            d[k] = to_device(np.asarray(snap[k], dt), dev)
        netkv_oracle_load(self.h, d, dev)
        self.P, self.D = int(snap["n_prefill"]), int(snap["n_decode"])

    def set_util(self, util: np.ndarray) -> None:
        netkv_oracle_set_util(self.h, to_device(np.asarray(util, np.float32), self.device),
                              self.device)

    def smooth_congestion(self, obs, beta: float) -> None:
        """Fold one congestion observation [P*D] (numpy or device tensor)
        into the forecast the selections use."""
        if not isinstance(obs, torch.Tensor):
            obs = to_device(np.asarray(obs, np.float32), self.device)
        netkv_congestion_smooth(self.h, obs, beta, self.device)

    def congestion(self) -> np.ndarray:
        """The congestion matrix the selections currently use [P*D]."""
        out = torch.empty(self.P * self.D, dtype=torch.float32, device=self.device)
        netkv_congestion_get(self.h, out, self.device)
        return to_numpy(out)

    def load_cache(self, cache: Dict[str, np.ndarray], max_load_factor: float = 0.5) -> None:
        dev = self.device
        off = to_device(np.asarray(cache["hash_off"], np.uint64), dev)
        hs = to_device(np.asarray(cache["hashes"], np.uint64), dev)
        netkv_cache_load(self.h, len(off) - 1, off, hs, max_load_factor, dev)
        del off, hs

    def select(self, req_dev: Dict[str, torch.Tensor], k: int = 1, pairs: bool = False,
               out=None):
        n = int(req_dev["prefill"].numel())
        dev = self.device
        if out is None:
            out = dict(idx=torch.empty(n * k, dtype=torch.int32, device=dev),
                       score=torch.empty(n * k, dtype=torch.float32, device=dev))
        pp = None
        if pairs:
            pp = dict(n_decode=self.D,
                      prefix_blocks=torch.empty(n * self.D, dtype=torch.uint16, device=dev),
                      feasible=torch.empty(n * self.D, dtype=torch.uint8, device=dev),
                      score=torch.empty(n * self.D, dtype=torch.float32, device=dev))
            out.update(pairs=pp)
        netkv_select_batch(self.h, req_dev, k, out["idx"], out["score"], pp, dev)
        return out

    def load_routes(self, tier1, util1, tier2, util2) -> None:
        """Staged (two-hop) routes per (p, d): hop tiers and congestion [P*D]."""
        dev = self.device
        netkv_route2_load(self.h, to_device(np.asarray(tier1, np.uint8).reshape(-1), dev),
                          to_device(np.asarray(util1, np.float32).reshape(-1), dev),
                          to_device(np.asarray(tier2, np.uint8).reshape(-1), dev),
                          to_device(np.asarray(util2, np.float32).reshape(-1), dev), dev)

    def clear_routes(self) -> None:
        netkv_route2_clear(self.h)

    def routes_of(self, req_dev, idx: torch.Tensor, k: int) -> np.ndarray:
        """1 where a selection takes its staged route, 0 direct, -1 none."""
        n = int(req_dev["prefill"].numel())
        out = torch.empty(n * k, dtype=torch.int8, device=self.device)
        netkv_route2_of(self.h, req_dev, k, idx, out, self.device)
        return to_numpy(out)

    def selection_bytes(self, req_dev, idx: torch.Tensor, k: int) -> torch.Tensor:
        """Non-cached bytes (Eq. (2)) of each selection; 0 for none."""
        n = int(req_dev["prefill"].numel())
        out = torch.empty(n * k, dtype=torch.uint64, device=self.device)
        netkv_selection_bytes(self.h, req_dev, k, idx, out, self.device)
        return out

    def flow_sim(self, fl: Dict[str, torch.Tensor], n_inst: int, n_links: int):
        """Flow-level transfer simulation of n_inst instances (device
        tensors cap [n_inst * n_links] f64, flow_off [n_inst + 1] u64,
        path_off u64, path u32, bytes f64, start f64): finish times [n_flows]
        and per instance (allocations, filling rounds, moving flows summed
        over the allocations) [n_inst, 3]."""
        fin = torch.empty(int(fl["bytes"].numel()), dtype=torch.float64, device=self.device)
        st = torch.empty(3 * n_inst, dtype=torch.uint64, device=self.device)
        netkv_flow_sim(self.h, n_inst, n_links, fl["cap"], fl["flow_off"], fl["path_off"], fl["path"],
                       fl["bytes"], fl["start"], fin, st, self.device)
        return fin, st

    def rank_sweep(self, req_dev, util_scen: torch.Tensor, k: int = 3):
        n = int(req_dev["prefill"].numel())
        cells = self.P * self.D
        if util_scen.numel() % cells:
            raise ValueError(f"util_scen has {util_scen.numel()} values, not a multiple of P*D={cells}")
        S = int(util_scen.numel() // cells)
        dev = self.device
        out = dict(idx=torch.empty(S * n * k, dtype=torch.int32, device=dev),
                   score=torch.empty(S * n * k, dtype=torch.float32, device=dev),
                   flips=torch.empty(2 * S, dtype=torch.uint64, device=dev),
                   inversions=torch.empty(3 * S, dtype=torch.uint64, device=dev))
        netkv_rank_sweep(self.h, req_dev, S, util_scen, k, out["idx"], out["score"],
                         out["flips"], dev, self.P * self.D, out["inversions"])
        return out

    def commit(self, req_dev, sel: torch.Tensor, cap: int, mu: int) -> None:
        netkv_commit_batch(self.h, req_dev, sel, cap, mu, self.device)

    def select_sequential(self, req_dev, cap: int = 16):
        n = int(req_dev["prefill"].numel())
        out = dict(idx=torch.empty(n, dtype=torch.int32, device=self.device),
                   score=torch.empty(n, dtype=torch.float32, device=self.device))
        netkv_select_sequential(self.h, req_dev, cap, out["idx"], out["score"], self.device)
        return out

    def tier_counts(self, req_dev, sel: torch.Tensor) -> np.ndarray:
        c = torch.empty(5, dtype=torch.uint64, device=self.device)
        netkv_tier_counts(self.h, req_dev, sel, c, self.device)
        return to_numpy(c)

    def set_policy(self, policy: int) -> None:
        netkv_set_option(self.h, NETKV_OPT_POLICY, policy)

    def state(self) -> Dict[str, np.ndarray]:
        return netkv_state_get(self.h, self.P, self.D, self.device)

    def sync_errors(self) -> None:
        netkv_sync_errors(self.h, self.device)


