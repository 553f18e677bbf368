"""The oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(every report fatal), run over every entry point on a small workload in a
child process, must finish cleanly and give the same results as the default
build.  CPU only."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Every oracle entry point on a scaled 64-GPU workload (two prefill
# instances' worth of requests, random in-flight counters, staged routes);
# prints a digest of every output.
_SCRIPT = r"""
import hashlib, json, sys
import numpy as np
sys.path.insert(0, sys.argv[1])
import oracle
from paper_2606_03910_amd import workload as W

def dig(*arrs):
    h = hashlib.sha256()
    for a in arrs:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()

cfg = W.scaled(W.CONFIGS["c0"], n_requests=300)
snap = W.make_snapshot(cfg, 5, inflight="random")
ch = W.prefix_chains(cfg, 5)
req = W.make_requests(cfg, 5, chains=ch)
cache = W.make_caches(cfg, 5, chains=ch)
c = oracle.Cache(cache, n_threads=2)
out = {}
o = oracle.select(snap, c, req, k=3, pairs=True, n_threads=2)
out["select"] = dig(o["idx"], o["score"], o["j"], o["feasible"], o["cost"])
links = W.draw_links(cfg, 5)
us, _ = W.scenario_utils(cfg, 5, links, n_scen=8, sigmas=(0.05, 0.4))
sw = oracle.rank_sweep(snap, c, req, us, k=2, n_threads=2)
out["sweep"] = dig(sw["idx"], sw["score"], sw["flips"])
out["inversions"] = dig(oracle.tier_inversions(snap, us, n_threads=2))
state = dict(n_inflight=snap["n_inflight"], queue_depth=snap["queue_depth"], free_mem=snap["free_mem"],
             admitted_prev=np.zeros(cfg.n_decode, np.uint64))
st = oracle.commit(snap, c, req, o["idx"][:, 0], 16, 2, state)
out["commit"] = dig(*[st[k] for k in sorted(st)])
sq = oracle.select_sequential(snap, c, req, cap=4)
fq = oracle.select_sequential(snap, c, req, cap=4, follow=sq["idx"])
out["sequential"] = dig(sq["idx"], sq["score"], fq["follow_cost"])
out["tier_counts"] = dig(oracle.tier_counts(snap, req, o["idx"][:, 0]))
sm, bad = oracle.smooth(np.asarray(snap["util"], np.float64), us[0], 0.3)
out["smooth"] = dig(sm) + str(bad)
rs = dict(snap)
rs.update(W.make_routes(cfg, 5))
r2 = oracle.select(rs, c, req, k=2, n_threads=2)
out["route_of"] = dig(r2["idx"], oracle.route_of(rs, c, req, r2["idx"], 2))
off = np.asarray(req["hash_off"], np.int64)
out["prefix_len"] = [c.prefix_len(d, req["hashes"][off[0]:off[1]]) for d in range(4)]
rng = np.random.default_rng(9)
L, N = 40, 200
plen = rng.integers(1, 5, N)
poff = np.concatenate([[0], np.cumsum(plen)]).astype(np.uint64)
path = np.concatenate([rng.choice(L, k, replace=False) for k in plen]).astype(np.uint32)
fl = dict(cap=rng.uniform(1.0, 9.0, L), path_off=poff, path=path, bytes=rng.uniform(0.0, 4.0, N),
          start=rng.uniform(0.0, 1.0, N))
rt, nr = oracle.maxmin(fl)
fin, ev = oracle.flow_sim(fl)
out["flows"] = dig(rt, fin) + str(nr) + str(ev)
nd, lf, pd = cfg.cluster.coords()
pg, dg = cfg.cluster.prefill_gpus(), cfg.cluster.decode_gpus()
tr, pu = oracle.pair_congestion((nd[pg], lf[pg], pd[pg]), (nd[dg], lf[dg], pd[dg]), links)
ar = oracle.ar1_step(links["u1"], links["u1"], rng.standard_normal(len(links["u1"])), 0.9, 0.05)
nz = oracle.link_noise(links["u2"], rng.standard_normal(len(links["u2"])), 0.4)
out["telemetry"] = dig(tr, pu, ar, nz)
import os
if os.environ.get("NETKV_ORACLE_LIB"):   # the checking build and the ASan runtime are the ones mapped
    maps = open("/proc/self/maps").read()
    assert os.environ["NETKV_ORACLE_LIB"] in maps and "libasan" in maps
print(json.dumps(out))
"""


def _run(env_extra):
    env = dict(os.environ)
    env.update(env_extra)
    env["OMP_NUM_THREADS"] = "2"
    r = subprocess.run([sys.executable, "-c", _SCRIPT, ROOT], env=env, capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, f"exit {r.returncode}\n{r.stderr[-4000:]}"
    return json.loads(r.stdout.strip().splitlines()[-1])


def test_oracle_under_asan_and_ubsan(tmp_path):
    import oracle
    libasan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("gcc has no AddressSanitizer runtime here")
    lib = oracle.build_sanitized(str(tmp_path / "liboracle_asan.so"))
    checked = _run({"NETKV_ORACLE_LIB": lib, "LD_PRELOAD": libasan,
                    "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:exitcode=23",
                    "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1:exitcode=24"})
    plain = _run({})
    assert checked == plain
