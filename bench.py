"""Benchmark: batched NetKV decode-instance selection on one MI355X.

One step = one netkv_select_batch call over the whole batch: for every
(request, decode) pair the prefix length (leading blocks resident on the
decode, Sec. III-B), the non-cached bytes, feasibility, the Eq. (5) cost,
and the per-request argmin (k = 1).  Inputs are resident in device memory
before timing starts.

Default workload: 4,096-GPU fat-tree (512 nodes, 64 leaves, 8 pods), 1,024
prefill and 3,072 decode instances, 1,048,576 requests in one snapshot
(3.2e9 scored pairs), 65,536 resident block hashes per decode in one holder
index at load factor 0.5.

Prints one JSON line: scored pairs/s (value), selections/s, per-launch time
of the scoring kernel from HIP events on the launch stream, that kernel's
roofline (vector-ALU lane-operations per pair against the MI355X issue rate;
the algorithmic HBM bytes of the first-miss tests alongside), and the CPU
oracle's rate on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

ISSUE_PEAK_PER_S = 256 * 2.4e9   # wave instructions per second of one kind (one per CU per cycle)
HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak, GB/s
# VALU lane-operations per second: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (one
# wave64 VALU instruction per CU per cycle, packed fp32 not counted)
ALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
# lane-operations per (request, decode) pair that scoring needs once the
# leader's prefix length is known: the cap lambda = min(B_tok j_leader,
# B_tok L*), non-cached tokens x = l - lambda, the fused multiply-add
# x * spt + (L + load), the feasibility test x <= xm_d, the feasible-or-
# infinity select, and one comparison of the per-request minimum
# (Eqs. (2)-(5), Algorithm 1)
OPS_PER_PAIR = 6
# with staged routes: a second fused multiply-add for the staged cost and the
# minimum of the two route costs (Sec. VIII)
OPS_PER_PAIR_TWO_HOP = 8
# the least of these on the path of a pair whose decode group is feasible
# for the request as a whole: the cap, the subtraction, the FMA and one
# comparison of the running minimum (two more with staged routes: the
# second FMA and the minimum of the two costs)
MIN_OPS_PER_PAIR = 4
MIN_OPS_PER_PAIR_TWO_HOP = 6


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def cols_per_lane(D: int) -> int:
    """The library's automatic decodes per lane (see NETKV_OPT_COLS)."""
    for c in (6, 3, 2):
        g = -(-D // (64 * c))
        if g >= 8 and g % 8 == 0:
            return c
    return 2 if D >= 256 else 1


def kernel_source_digest() -> str:
    with open(os.path.join(ROOT, "paper_2606_03910_amd", "csrc", "netkv.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def counter_summary(workload: str, digest: str, kernel: str = "score_kernel"):
    """Per-launch rocprofv3 counter figures of the scoring kernel (HBM bytes,
    instruction counts) from the committed summary, if they were taken on
    this exact kernel source; else an empty dict."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_counters.json")
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        c = json.load(f)
    if c.get("kernel_source_sha256_16") != digest:
        return {}
    return c


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args, snap, cache, req, routes, gidx, gscore, D):
    """The CPU oracle timed on this host: a seeded contiguous slice of
    65,536 requests of the same batch (every decode) on all host threads,
    in chunks, stopping early only past the time cap; then the first 1,024
    requests of the slice on one thread.  Every request of the slice on
    which the GPU's selection differs from the oracle's is classified with
    the parity rules (near-tie, exact tie, beyond)."""
    import oracle
    from tests.parity import classify, slice_requests
    R = len(gidx)
    threads = oracle.max_threads()
    t0 = time.time()
    ocache = oracle.Cache(cache, n_threads=threads)
    log(f"oracle resident sets sorted in {time.time() - t0:.1f}s ({threads} threads)")
    osnap = oracle.Snapshot(dict(snap, **routes) if routes else snap)
    n_slice = min(R, 65536)
    s0 = int(np.random.default_rng(7).integers(0, R - n_slice + 1))
    n_s, dt, o_tests, chunk = 0, 0.0, 0, 2048
    o_idx = np.empty(n_slice, np.int32)
    while n_s < n_slice and dt < args.cpu_seconds:
        a, b = s0 + n_s, s0 + min(n_slice, n_s + chunk)
        sub = slice_requests(req, a, b)
        t0 = time.perf_counter()
        o = oracle.select(osnap, ocache, sub, k=1, n_threads=threads)
        dt += time.perf_counter() - t0
        o_idx[n_s:n_s + (b - a)] = o["idx"][:, 0]
        o_tests += int(o["tests"])
        n_s += b - a
    g = gidx[s0:s0 + n_s]
    dis = np.nonzero(g != o_idx[:n_s])[0]
    cls = dict(positions=n_s, mismatches=0, near_ties=0, exact_ties=0, exact_ties_fp32_split=0, beyond=0,
               max_rel_gap=0.0)
    if dis.size:
        rows = s0 + dis
        from tests.parity import subset_requests
        od = oracle.select(osnap, ocache, subset_requests(req, rows), k=1, pairs=True, n_threads=threads)
        c = classify(gidx[rows].reshape(-1, 1), od["idx"], od["cost"])
        cls.update({k: v for k, v in c.items() if k not in ("bad_mask", "positions")})
    # one thread, the first 1,024 requests of the slice
    n1 = min(1024, n_s)
    t0 = time.perf_counter()
    oracle.select(osnap, ocache, slice_requests(req, s0, s0 + n1), k=1, n_threads=1)
    dt1 = time.perf_counter() - t0
    log(f"cpu oracle: {n_s} requests in {dt:.1f}s on {threads} threads; {n1} in {dt1:.1f}s on 1 thread; "
        f"disagreements {cls}")
    return dict(value=n_s * D / dt, unit="pairs/s", cores=threads, kind="oracle",
                sample=f"requests [{s0}, {s0 + n_s}) of the same batch (a seeded contiguous slice of "
                       f"{n_slice}) x all {D} decodes: {n_s * D} pairs, {dt:.1f} s, {o_tests} membership "
                       f"tests; selections/s {n_s / dt:.1f}",
                selections_per_s=n_s / dt,
                one_thread=dict(value=n1 * D / dt1, unit="pairs/s",
                                sample=f"requests [{s0}, {s0 + n1}) x all {D} decodes, {dt1:.1f} s"),
                cpu_model=cpu_model(),
                gpu_vs_oracle=dict(cls, rule="an index may differ only where the oracle's costs of the two "
                                             "choices are within 1e-6 relative (near-tie); beyond must be 0",
                                   beyond_near_tie=cls["beyond"] + cls["exact_ties"]))


def stream_ceiling(dev, mib=2048, reps=10):
    """Achieved bandwidth of plain streaming kernels over 2 GiB: a read-only
    one (torch's fp32 sum) and a device copy (read + write): the practical
    ceiling for HBM-bound kernels."""
    import torch
    x = torch.ones(mib * (1 << 20) // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    res = {}
    for name, fn, mult in (("read", lambda: x.sum(), 1), ("copy", lambda: y.copy_(x), 2)):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        res[name] = dict(gbs=mult * mib * (1 << 20) / (ms * 1e-3) / 1e9, ms=ms)
    del x, y
    return dict(gbs=max(v["gbs"] for v in res.values()), read_only_gbs=res["read"]["gbs"],
                copy_gbs=res["copy"]["gbs"],
                kernels="torch fp32 sum over 2 GiB (reads only); device copy of 2 GiB (read + write)")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="c2", choices=["c0", "c1", "c2", "c3", "c4"])
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile", action="store_true",
                    help="timed steps only (no algorithmic-byte pass, streaming ceiling or CPU baseline): "
                         "for kernel traces and counters")
    ap.add_argument("--cpu-seconds", type=float, default=45.0,
                    help="cap on the all-threads oracle timing of the 65,536-request slice")
    ap.add_argument("--no-reuse", action="store_true",
                    help="no prefix sharing along the batch order: every request whose block 0 "
                         "is resident somewhere is matched from block 0")
    ap.add_argument("--run-len", type=int, default=0, help="requests per wavefront run (0 = auto)")
    ap.add_argument("--cols", type=int, default=0, help="decodes per lane (0 = auto, 1, 2, 3, 4, 6)")
    ap.add_argument("--policy", type=int, default=0,
                    help="cost rung: 0 full, 1 without live congestion, 2 topology only")
    ap.add_argument("--sequential", action="store_true",
                    help="time the request-by-request form (in-batch in-flight increments, cap 16)")
    ap.add_argument("--forecast", type=float, default=0.0, metavar="BETA",
                    help="c1: fold each batch's (stale) congestion observation into the forecast by "
                         "exponential smoothing with this factor instead of replacing the snapshot's")
    ap.add_argument("--two-hop", action="store_true",
                    help="load a staged (two-hop) route for every (prefill, decode) pair: each pair "
                         "scores the faster of its direct and staged routes")
    ap.add_argument("--flow-sim", action="store_true",
                    help="only time the flow-level transfer simulation: the workload's batch selected "
                         "(k = 1), its transfers simulated on the cluster's fat tree under "
                         "--flow-instances background-load draws")
    ap.add_argument("--flow-instances", type=int, default=1024,
                    help="independent simulation instances per call (background-load draws)")
    ap.add_argument("--flow-window", type=float, default=5.0,
                    help="seconds over which the batch's transfers arrive")
    ap.add_argument("--smooth-bench", action="store_true",
                    help="only time the congestion smoothing kernel on the workload's P x D matrix")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (K launches) and exit: the "
                         "reference kernel for scaling HBM byte counters")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration * (1 << 20) // 8
        src = torch.ones(n, dtype=torch.int64, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 8, "bytes_written": n * 8,
                          "launches": args.steps}), flush=True)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(requests or decodes would be sharded across GPUs). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_03910_amd import netkv
    from paper_2606_03910_amd import workload as W

    cfg = W.CONFIGS[args.workload]
    dev = torch.device("cuda", 0)
    if args.smooth_bench:
        return bench_smooth(args, cfg, dev)
    if args.flow_sim:
        return bench_flowsim(args, cfg, dev)
    if args.workload == "c3":
        return bench_sweep(args, cfg, dev)
    if args.workload == "c1":
        return bench_stream(args, cfg, dev)
    t0 = time.time()
    snap = W.make_snapshot(cfg, args.seed)
    ch = W.prefix_chains(cfg, args.seed)
    req = W.make_requests(cfg, args.seed, chains=ch)
    cache = W.make_caches(cfg, args.seed, chains=ch)
    log(f"inputs generated in {time.time() - t0:.1f}s: {cfg.n_requests} requests, "
        f"{int(req['hash_off'][-1])} request blocks, {cache['hashes'].size} resident hashes")

    sel = netkv.Selector(0)
    netkv.netkv_set_option(sel.h, netkv.NETKV_OPT_REUSE, 0 if args.no_reuse else 1)
    netkv.netkv_set_option(sel.h, netkv.NETKV_OPT_RUN_LEN, args.run_len)
    netkv.netkv_set_option(sel.h, netkv.NETKV_OPT_COLS, args.cols)
    netkv.netkv_set_option(sel.h, netkv.NETKV_OPT_POLICY, args.policy)
    t0 = time.time()
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    routes = None
    if args.two_hop:
        routes = W.make_routes(cfg, args.seed)
        sel.load_routes(routes["route_tier1"], routes["route_util1"], routes["route_tier2"],
                        routes["route_util2"])
    torch.cuda.synchronize()
    ci = netkv.netkv_cache_info(sel.h)
    log(f"snapshot + holder index loaded in {time.time() - t0:.1f}s: {ci['distinct_hashes']} distinct "
        f"hashes ({ci['shared_hashes']} on several decodes), {ci['index_slots']} slots, "
        f"{ci['index_bytes'] / 2**30:.2f} GiB")
    rd = netkv.requests_to_device(req, dev)
    R, D, P = cfg.n_requests, cfg.n_decode, cfg.n_prefill
    k = 1
    out = dict(idx=torch.empty(R * k, dtype=torch.int32, device=dev),
               score=torch.empty(R * k, dtype=torch.float32, device=dev))

    def step():
        if args.sequential:
            netkv.netkv_select_sequential(sel.h, rd, 16, out["idx"], out["score"], dev)
        else:
            netkv.netkv_select_batch(sel.h, rd, k, out["idx"], out["score"], None, dev)

    for _ in range(args.warmup):
        step()
    sel.sync_errors()
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} done")

    # Events on the launch stream (torch's current stream, which the library
    # launches on): one pair around the timed steps (a pair per step would put
    # two more event packets between consecutive calls), and the library's own
    # pair around each call's scoring kernel (prefix lengths + score +
    # per-group top-k).
    stream = torch.cuda.current_stream(dev)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    netkv.netkv_set_timing(sel.h, True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    kern_ms = netkv.netkv_kernel_ms(sel.h)   # mean over the timed launches
    netkv.netkv_set_timing(sel.h, False)
    sel.sync_errors()
    step_ms = ev0.elapsed_time(ev1) / args.steps
    log(f"timed {args.steps} steps: wall {wall * 1e3:.2f} ms, step mean {step_ms:.3f} ms, "
        f"scoring kernel mean {kern_ms:.3f} ms")

    # ---- algorithmic bytes: 8 B per membership test of the first-miss scans
    # (sum over pairs of min(j + 1, n_r)), from the per-pair prefix lengths of
    # the same kernel (bit-identical to the oracle's in the parity tests), plus
    # the bytes every launch must read once and write.
    nblk = np.diff(req["hash_off"].astype(np.int64))
    if args.profile:
        print(json.dumps({"profile_run": True, "workload": cfg.name, "step_ms_events": step_ms,
                          "kernel_ms": kern_ms}), flush=True)
        sel.close()
        return
    tests = 0
    chunk = 65536
    jbuf = torch.empty(chunk * D, dtype=torch.uint16, device=dev)
    tmp_idx = torch.empty(chunk, dtype=torch.int32, device=dev)
    tmp_sc = torch.empty(chunk, dtype=torch.float32, device=dev)
    off_all = req["hash_off"].astype(np.int64)
    for r0 in range(0, R, chunk):
        r1 = min(R, r0 + chunk)
        a, b = off_all[r0], off_all[r1]
        sub = netkv.requests_to_device(dict(
            prefill=req["prefill"][r0:r1], len_tokens=req["len_tokens"][r0:r1],
            hash_off=(off_all[r0:r1 + 1] - a).astype(np.uint64),
            hashes=req["hashes"][a:b] if b > a else np.ones(1, np.uint64)), dev)
        netkv.netkv_select_batch(sel.h, sub, 1, tmp_idx, tmp_sc,
                                 dict(n_decode=D, prefix_blocks=jbuf), dev)
        j = jbuf[: (r1 - r0) * D].view(torch.int16).to(torch.int64).view(r1 - r0, D)
        n = torch.from_numpy(nblk[r0:r1]).to(dev)[:, None]
        tests += int(torch.minimum(j + 1, n).sum().item())
    sel.sync_errors()
    b_tests = 8 * tests
    b_req = int(R * (4 + 4 + 8) + 8 * int(nblk.sum()) + R * k * 8)
    b_dec = D * (8 + 4 + 4)
    b_nco = P * D * (1 + 4) + 4 * P * 2
    b_alg = b_tests + b_req + b_dec + b_nco
    ops_pair = OPS_PER_PAIR_TWO_HOP if args.two_hop else OPS_PER_PAIR
    ops = ops_pair * R * D
    staged = None
    if args.two_hop:
        rt = sel.routes_of(rd, out["idx"], k)
        staged = float((rt == 1).sum()) / max(1, int((rt >= 0).sum()))
        log(f"selections taking the staged route: {staged:.4f}")
    achieved = ops / (kern_ms * 1e-3) / 1e12
    digest = kernel_source_digest()
    cs = counter_summary(args.workload + ("_two_hop" if args.two_hop else ""), digest)
    traffic = cs.get("hbm_bytes_per_launch")
    issue = None
    if "valu_insts_per_launch" in cs:
        kern_s = kern_ms * 1e-3
        issue = {
            "valu_insts_per_launch": cs["valu_insts_per_launch"],
            "salu_insts_per_launch": cs["salu_insts_per_launch"],
            "valu_frac": cs["valu_insts_per_launch"] / (kern_s * ISSUE_PEAK_PER_S),
            "salu_frac": cs["salu_insts_per_launch"] / (kern_s * ISSUE_PEAK_PER_S),
            "l2_hit_rate": cs.get("l2_hit_rate"),
            "model": "one VALU and one SALU wave64 instruction issued per CU per cycle "
                     "(256 CUs x 2.4 GHz); counters from the committed profile of this source",
        }

    stream = stream_ceiling(dev)
    log(f"streaming ceiling: read {stream['read_only_gbs']:.0f} GB/s, copy {stream['copy_gbs']:.0f} GB/s")

    # ---- CPU oracle baseline on a bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, snap, cache, req, routes, netkv.to_numpy(out["idx"]),
                           netkv.to_numpy(out["score"]), D)
        del cache

    pairs = R * D
    rec = {
        "metric": "scored (request,decode) pairs/sec + selections/sec; achieved HBM GB/s vs peak",
        "value": pairs / (step_ms * 1e-3),
        "unit": "pairs/s",
        "selections_per_s": R / (step_ms * 1e-3),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps,
        "step_ms_events": step_ms,
        "kernel_ms": kern_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+u64",
        "data": "synthetic (seeded; lognormal lengths, Zipf-shared prefixes)",
        "config": {
            "workload": cfg.name,
            "requests": R, "decodes": D, "prefills": P, "gpus_modelled": cfg.cluster.n_gpus,
            "resident_hashes_per_decode": cfg.cache_per_decode, "index": ci,
            "block_tokens": cfg.block_tokens, "mean_blocks_per_request": float(nblk.mean()),
            "k": k, "parallelism": "single-gpu", "prefix_sharing": not args.no_reuse,
            "run_len": args.run_len or "auto", "policy": args.policy,
            "selection": "sequential (in-batch in-flight increments)" if args.sequential else "snapshot",
            "routes": "direct + staged (two-hop)" if args.two_hop else "direct",
            "staged_fraction": staged,
        },
        "roofline": {
            "bound": "alu", "achieved": achieved, "peak": ALU_PEAK_TOPS, "unit": "TOP/s",
            "frac": achieved / ALU_PEAK_TOPS,
            "traffic": (traffic / (kern_ms * 1e-3) / 1e9) if traffic else None,
            "traffic_unit": "GB/s",
            "traffic_bytes_per_launch": traffic,
            "algorithmic_ops_per_launch": ops,
            "ops_per_pair": ops_pair,
            "kernel": "score_kernel (k=1; %d decodes per lane%s)" % (
                args.cols or cols_per_lane(D), "; two routes per pair" if args.two_hop else ""),
            "kernel_source_sha256_16": digest,
            "issue": issue,
            # the same operation count over the whole step (every kernel of
            # the selection), and over the minimal all-feasible count
            "step_frac": ops / (step_ms * 1e-3) / 1e12 / ALU_PEAK_TOPS,
            "min_ops_per_pair": MIN_OPS_PER_PAIR_TWO_HOP if args.two_hop else MIN_OPS_PER_PAIR,
            "frac_at_min_ops": (MIN_OPS_PER_PAIR_TWO_HOP if args.two_hop else MIN_OPS_PER_PAIR) * pairs
                               / (kern_ms * 1e-3) / 1e12 / ALU_PEAK_TOPS,
            "hbm": {
                "gbs_counters": (traffic / (kern_ms * 1e-3) / 1e9) if traffic else None,
                "frac_of_peak": (traffic / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBS) if traffic else None,
                "peak_gbs": HBM_PEAK_GBS,
                "stream_ceiling": stream,
                "target_frac": 0.60,
                "target_met": False,
                "why": "the scoring kernel reads little: prefix lengths come from leader rows (one "
                       "first-miss scan per shared prefix, exact), so it is bound by vector-ALU issue, "
                       "not HBM; the HBM fraction above is what it moves, not a shortfall of bandwidth",
            },
            "hbm_algorithmic": {
                "bytes_per_launch": b_alg, "membership_tests_per_launch": tests,
                "mean_tests_per_pair": tests / pairs,
                "gbs_equivalent": b_alg / (kern_ms * 1e-3) / 1e9,
                "ratio_to_hbm_peak": b_alg / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "meaning": "bytes a pair-by-pair first-miss scan would read (8 B per membership test) "
                           "over the kernel time; a ratio above 1 is work the leader identity avoids, "
                           "not an achieved bandwidth",
            },
            "note": ("the scoring kernel is bound by vector-ALU issue: achieved counts 6 lane-"
                     "operations per (request, decode) pair against one wave64 VALU instruction per "
                     "CU per cycle; step_frac is the same count over the whole step, frac_at_min_ops "
                     "the 4 operations of the all-feasible path (cap, subtract, FMA, one comparison of "
                     "the minimum). traffic is the counter-measured HBM bytes of the same kernel."),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sel.close()


# lane-operations per (scenario, request, decode) of the ranking sweep with
# k = 3, once the pair's non-cached tokens are known: the FMA x * spt + (L +
# load), three comparisons with the running top-3, one minimum and two
# medians that update its values, and five selects that update its indices
SWEEP_OPS_PER_PAIR = 12


def bench_sweep(args, cfg, dev):
    """Ranking sweep: one step = netkv_rank_sweep over all scenarios."""
    import torch

    from paper_2606_03910_amd import netkv
    from paper_2606_03910_amd import workload as W
    snap = W.make_snapshot(cfg, args.seed)
    ch = W.prefix_chains(cfg, args.seed)
    req = W.make_requests(cfg, args.seed, chains=ch)
    cache = W.make_caches(cfg, args.seed, chains=ch)
    util_s, sig = W.scenario_utils(cfg, args.seed, snap["links"])
    S, R, D, P, k = cfg.n_scenarios, cfg.n_requests, cfg.n_decode, cfg.n_prefill, 3
    sel = netkv.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = netkv.requests_to_device(req, dev)
    us = netkv.to_device(util_s.reshape(-1), dev)
    out = dict(idx=torch.empty(S * R * k, dtype=torch.int32, device=dev),
               score=torch.empty(S * R * k, dtype=torch.float32, device=dev),
               flips=torch.empty(2 * S, dtype=torch.uint64, device=dev),
               inversions=torch.empty(3 * S, dtype=torch.uint64, device=dev))

    def step():
        netkv.netkv_rank_sweep(sel.h, rd, S, us, k, out["idx"], out["score"], out["flips"], dev, P * D,
                               out["inversions"])

    for _ in range(args.warmup):
        step()
    sel.sync_errors()
    stream = torch.cuda.current_stream(dev)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    netkv.netkv_set_timing(sel.h, True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    kern_ms = netkv.netkv_kernel_ms(sel.h)   # mean over the timed launches
    netkv.netkv_set_timing(sel.h, False)
    sel.sync_errors()
    step_ms = ev0.elapsed_time(ev1) / args.steps
    log(f"sweep: step {step_ms:.3f} ms, sweep kernel {kern_ms:.3f} ms")
    pairs = S * R * D
    ops = SWEEP_OPS_PER_PAIR * pairs
    achieved = ops / (kern_ms * 1e-3) / 1e12
    inv = netkv.to_numpy(out["inversions"]).reshape(S, 3)
    fl = netkv.to_numpy(out["flips"]).reshape(S, 2)
    prop2 = {"covered_pairs_mean": float(inv[:, 0].mean()), "covered_inverted_total": int(inv[:, 1].sum()),
             "inverted_pairs_mean_by_sigma": {str(sg): float(inv[sig == sg, 2].mean()) for sg in cfg.noise_sigmas},
             "selected_tier_flip_rate_by_sigma": {str(sg): float(fl[sig == sg, 0].mean() / R)
                                                  for sg in cfg.noise_sigmas}}
    cpu = None
    if not args.no_cpu_baseline and not args.profile:
        import oracle
        threads = oracle.max_threads()
        # scenario count doubled until one run takes about 10 s
        ns = 4
        while True:
            t0 = time.perf_counter()
            oracle.rank_sweep(snap, cache, req, util_s[:ns], k=k, n_threads=threads)
            dt = time.perf_counter() - t0
            if dt >= 5.0 or ns >= S:
                break
            ns = min(S, ns * 2)
        cpu = dict(value=ns * R * D / dt, unit="pairs/s", cores=threads, kind="oracle", cpu_model=cpu_model(),
                   sample=f"{ns} scenarios x {R} requests x {D} decodes (prefix match once, "
                          f"then rescoring), {dt:.1f} s")
    cs = counter_summary(args.workload, kernel_source_digest(), "sweep_kernel")
    traffic = cs.get("hbm_bytes_per_launch")
    issue = None
    if "valu_insts_per_launch" in cs:
        issue = {"valu_frac": cs["valu_insts_per_launch"] / (kern_ms * 1e-3 * ISSUE_PEAK_PER_S),
                 "salu_frac": cs["salu_insts_per_launch"] / (kern_ms * 1e-3 * ISSUE_PEAK_PER_S),
                 "model": "one VALU and one SALU wave64 instruction issued per CU per cycle "
                          "(256 CUs x 2.4 GHz); counters from the committed profile of this source"}
    rec = {
        "metric": "scored (request,decode) pairs/sec + selections/sec; achieved HBM GB/s vs peak",
        "value": pairs / (step_ms * 1e-3), "unit": "pairs/s",
        "selections_per_s": S * R / (step_ms * 1e-3),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": wall * 1e3 / args.steps, "step_ms_events": step_ms, "kernel_ms": kern_ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded; lognormal link-noise scenarios)",
        "config": {"workload": cfg.name, "requests": R, "decodes": D, "prefills": P,
                   "scenarios": S, "sigmas": list(cfg.noise_sigmas), "k": k,
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": ALU_PEAK_TOPS, "unit": "TOP/s",
                     "frac": achieved / ALU_PEAK_TOPS,
                     "traffic": (traffic / (kern_ms * 1e-3) / 1e9) if traffic else None,
                     "traffic_unit": "GB/s", "traffic_bytes_per_launch": traffic, "issue": issue,
                     "algorithmic_ops_per_launch": ops, "ops_per_pair": SWEEP_OPS_PER_PAIR,
                     "step_frac": ops / (step_ms * 1e-3) / 1e12 / ALU_PEAK_TOPS,
                     "kernel": "sweep_kernel<3, 48, LDS, full>",
                     "note": "12 lane-operations per scenario-pair (the FMA and the running top-3's "
                             "compares, minimum, medians and index selects) against one wave64 VALU "
                             "instruction per CU per cycle, the same peak as the selection's"},
        "prop2": prop2,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sel.close()


def bench_stream(args, cfg, dev):
    """Streaming batches: one step = all batches, each a congestion refresh,
    a selection and the between-batch update."""
    import torch

    from paper_2606_03910_amd import netkv
    from paper_2606_03910_amd import workload as W
    snap = W.make_snapshot(cfg, args.seed)
    ch = W.prefix_chains(cfg, args.seed)
    cache = W.make_caches(cfg, args.seed, chains=ch)
    links = W.ar1_links(cfg, args.seed, snap["links"], cfg.n_batches)
    utils = [netkv.to_device(W.pair_util(cfg.cluster, links[t]).reshape(-1), dev)
             for t in range(cfg.n_batches)]
    reqs = [netkv.requests_to_device(W.make_requests(cfg, args.seed, batch=t, chains=ch), dev)
            for t in range(cfg.n_batches)]
    R, D, B = cfg.n_requests, cfg.n_decode, cfg.n_batches
    mu = -(-R // D)
    sel = netkv.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    idx = torch.empty(R, dtype=torch.int32, device=dev)
    sc = torch.empty(R, dtype=torch.float32, device=dev)

    def step():
        sel.load_snapshot(snap)
        for t in range(B):
            if args.forecast:
                netkv.netkv_congestion_smooth(sel.h, utils[max(0, t - 1)], args.forecast, dev)
            else:
                netkv.netkv_oracle_set_util(sel.h, utils[max(0, t - 1)], dev)
            netkv.netkv_select_batch(sel.h, reqs[t], 1, idx, sc, None, dev)
            netkv.netkv_commit_batch(sel.h, reqs[t], idx, 16, mu, dev)

    for _ in range(args.warmup):
        step()
    sel.sync_errors()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    sel.sync_errors()
    ms = wall * 1e3 / args.steps
    rec = {
        "metric": "scored (request,decode) pairs/sec + selections/sec; achieved HBM GB/s vs peak",
        "value": B * R * D / (ms * 1e-3), "unit": "pairs/s", "selections_per_s": B * R / (ms * 1e-3),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32+u64",
        "data": "synthetic (seeded; AR(1) congestion, staleness 1 batch)",
        "config": {"workload": cfg.name, "requests_per_batch": R, "batches": B, "decodes": D,
                   "prefills": cfg.n_prefill, "staleness": 1, "parallelism": "single-gpu",
                   "congestion": (f"exponential smoothing, beta {args.forecast}" if args.forecast
                                  else "replaced by each observation")},
        "roofline": None, "cpu_baseline": None,
        "note": "wall time of the whole stream (snapshot load, per-batch congestion refresh, "
                "selection and update); small batches are launch- and latency-bound",
    }
    print(json.dumps(rec), flush=True)
    sel.close()


def bench_smooth(args, cfg, dev):
    """Predictive congestion: one step = one smoothing of the P x D
    congestion matrix towards an observation (12 B per entry: read the
    forecast and the observation, write the forecast), HBM-bound."""
    import torch

    from paper_2606_03910_amd import netkv
    from paper_2606_03910_amd import workload as W
    snap = W.make_snapshot(cfg, args.seed)
    sel = netkv.Selector(0)
    sel.load_snapshot(snap)
    npd = cfg.n_prefill * cfg.n_decode
    rng = np.random.default_rng(args.seed)
    obs = [netkv.to_device(rng.uniform(0, 0.99, npd).astype(np.float32), dev) for _ in range(4)]
    beta = args.forecast or 0.2
    for i in range(args.warmup):
        netkv.netkv_congestion_smooth(sel.h, obs[i % 4], beta, dev)
    sel.sync_errors()
    netkv.netkv_set_timing(sel.h, True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(args.steps):
        netkv.netkv_congestion_smooth(sel.h, obs[i % 4], beta, dev)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    kern_ms = netkv.netkv_kernel_ms(sel.h)
    netkv.netkv_set_timing(sel.h, False)
    sel.sync_errors()
    nbytes = 12 * npd
    gbs = nbytes / (kern_ms * 1e-3) / 1e9
    rec = {
        "metric": "congestion entries smoothed/s (predictive congestion)",
        "value": npd / (kern_ms * 1e-3), "unit": "entries/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps, "kernel_ms": kern_ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded uniform observations)",
        "config": {"workload": cfg.name + "-congestion-smoothing", "prefills": cfg.n_prefill,
                   "decodes": cfg.n_decode, "entries": npd, "beta": beta},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                     "algorithmic_bytes_per_launch": nbytes, "bytes_per_entry": 12},
        "cpu_baseline": None,
    }
    print(json.dumps(rec), flush=True)
    sel.close()


def bench_flowsim(args, cfg, dev):
    """Flow-level transfer simulation (Sec. VI-B's network model): the
    workload's batch is selected on the GPU (k = 1), the selections'
    transfer sizes (Eq. (2)) come from the GPU, and the transfers, arriving
    over --flow-window seconds, are simulated on the cluster's fat tree
    under --flow-instances background-load draws (one workgroup each).  One
    step = one netkv_flow_sim call over all instances."""
    import torch

    from paper_2606_03910_amd import netkv
    from paper_2606_03910_amd import workload as W
    snap = W.make_snapshot(cfg, args.seed)
    ch = W.prefix_chains(cfg, args.seed)
    req = W.make_requests(cfg, args.seed, chains=ch)
    cache = W.make_caches(cfg, args.seed, chains=ch)
    sel = netkv.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = netkv.requests_to_device(req, dev)
    out = sel.select(rd, k=1)
    nbytes = netkv.to_numpy(sel.selection_bytes(rd, out["idx"], 1))
    sel.sync_errors()
    idx = netkv.to_numpy(out["idx"]).reshape(-1)
    ok = idx >= 0
    n = int(ok.sum())
    S = args.flow_instances
    t0 = time.time()
    caps, offs, paths, starts = [], [], [], []
    base = 0
    for i in range(S):
        cap, lay = W.fat_tree_links(cfg, W.draw_links(cfg, args.seed + 1000 + i))
        off, path = W.transfer_paths(cfg, args.seed + i, req["prefill"][ok], idx[ok], lay)
        caps.append(cap)
        offs.append(off[1:] + np.uint64(base))
        paths.append(path)
        base += int(off[-1])
        starts.append(W.transfer_starts(args.seed + i, n, args.flow_window))
    L = len(caps[0])
    fl = dict(cap=np.concatenate(caps), flow_off=(np.arange(S + 1, dtype=np.uint64) * np.uint64(n)),
              path_off=np.concatenate([np.zeros(1, np.uint64)] + offs), path=np.concatenate(paths),
              bytes=np.tile(nbytes[ok].astype(np.float64), S), start=np.concatenate(starts))
    log(f"{S} instances of {n} transfers on {L} links built in {time.time() - t0:.1f}s")
    fd = {k: netkv.to_device(v, dev) for k, v in fl.items()}
    for _ in range(args.warmup):
        fin, st = sel.flow_sim(fd, S, L)
    sel.sync_errors()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    a.record()
    for _ in range(args.steps):
        fin, st = sel.flow_sim(fd, S, L)
    b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    step_ms = a.elapsed_time(b) / args.steps
    sel.sync_errors()
    fin = netkv.to_numpy(fin)
    st = netkv.to_numpy(st).reshape(S, 3).astype(np.int64)
    tt = fin - fl["start"]
    # fp64 work of the allocations: per filling round and link the share
    # (a division) and the update (a division, a compare, a multiply, a
    # subtraction, a maximum); per event and moving flow the time to finish
    # (a division, a minimum) and the advance (a division, a compare, a
    # multiply, a subtraction, a maximum): 7 each
    ops = 7 * (int(st[:, 1].sum()) * L + int(st[:, 2].sum()))
    achieved = ops / (step_ms * 1e-3) / 1e12
    log(f"flow sim: {S} x {n} transfers, step {step_ms:.3f} ms; {int(st[:, 0].sum())} allocations, "
        f"{int(st[:, 1].sum())} filling rounds; transfer time mean {tt.mean() * 1e3:.1f} ms, "
        f"p99 {np.quantile(tt, 0.99) * 1e3:.1f} ms")
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        t0 = time.perf_counter()
        m = 0
        agree = True
        while m < S and time.perf_counter() - t0 < min(args.cpu_seconds, 20.0):
            x = dict(cap=caps[m], path_off=np.concatenate([[0], np.cumsum(np.diff(
                fl["path_off"][m * n:(m + 1) * n + 1].astype(np.int64)))]).astype(np.uint64),
                path=paths[m], bytes=nbytes[ok].astype(np.float64), start=starts[m])
            o_fin, _ = oracle.flow_sim(x)
            agree = agree and np.array_equal(o_fin.view(np.uint64), fin[m * n:(m + 1) * n].view(np.uint64))
            m += 1
        dt = time.perf_counter() - t0
        cpu = dict(value=m * n / dt, unit="transfers/s", cores=1, kind="oracle", cpu_model=cpu_model(),
                   sample=f"the first {m} of the {S} instances ({m * n} transfers), one thread, {dt:.1f} s",
                   gpu_bit_identical=bool(agree))
    rec = {
        "metric": "simulated KV transfers/s (flow-level max-min fair network model)",
        "value": S * n / (step_ms * 1e-3), "unit": "transfers/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps, "step_ms_events": step_ms,
        "allocations_per_s": int(st[:, 0].sum()) / (step_ms * 1e-3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic (seeded; the workload's batch selected on the GPU, fat-tree links with drawn "
                "background load, ECMP draws, uniform arrivals)",
        "config": {"workload": cfg.name + "-transfer-simulation", "instances": S, "transfers": n,
                   "links": L, "arrival_window_s": args.flow_window},
        "simulation": {"transfer_s_mean": float(tt.mean()), "transfer_s_p50": float(np.median(tt)),
                       "transfer_s_p99": float(np.quantile(tt, 0.99)),
                       "allocations": int(st[:, 0].sum()), "filling_rounds": int(st[:, 1].sum())},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": ALU_PEAK_TOPS, "unit": "TOP/s",
                     "frac": achieved / ALU_PEAK_TOPS, "traffic": None,
                     "algorithmic_ops_per_launch": ops,
                     "note": "fp64 lane-operations of the allocations (7 per link and filling round, 7 per "
                             "moving flow and event; a division counts as one) against one wave64 VALU "
                             "instruction per CU per cycle, the fp64 vector rate (78.6 TFLOP/s counts an "
                             "FMA as two); the kernel is bound by each instance's chain of dependent "
                             "workgroup reductions (several barriers per filling round), not by arithmetic"},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    sel.close()


if __name__ == "__main__":
    main()
