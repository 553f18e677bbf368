"""HIP path against the CPU oracle on the same seeded inputs (64-GPU sizes,
edge cases, the C-ABI contract).  Needs an MI355X and the built library."""
import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import check_pairs, check_self_topk, check_topk, subset_requests

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _say(*a):
    print("[gpu-case]", *a, flush=True)


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03910_amd import netkv
    netkv.load_library()
    return netkv


def _inputs(cfg, seed, inflight="zero", **snap_over):
    snap = W.make_snapshot(cfg, seed, inflight=inflight)
    snap.update(snap_over)
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    return snap, req, cache


def _gpu(nk, snap, cache, lf=0.5):
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, lf)
    return sel


def _run(nk, sel, req, k, pairs=True):
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=k, pairs=pairs)
    sel.sync_errors()
    res = dict(idx=nk.to_numpy(out["idx"]).reshape(-1, k), score=nk.to_numpy(out["score"]).reshape(-1, k))
    if pairs:
        p = out["pairs"]
        res.update(j=nk.to_numpy(p["prefix_blocks"]), feas=nk.to_numpy(p["feasible"]),
                   cost=nk.to_numpy(p["score"]))
    return res


def _check_all(g, o):
    """Per-pair outputs against the oracle, the selections against the
    oracle (near-tie rule, exact ties to the lowest index), and the
    selections against the exact top-k of the GPU's own per-pair scores."""
    err = check_pairs(g["j"], g["feas"], g["cost"], o)
    R, k = g["idx"].shape
    D = o["j"].shape[1]
    res = check_topk(g["idx"], g["score"], o["idx"], o["cost"], o["feasible"],
                     g_cost=g["cost"].reshape(R, D))
    check_self_topk(g["idx"], g["score"], g["cost"].reshape(R, D), g["feas"].reshape(R, D))
    return res, err


@pytest.mark.parametrize("inflight", ["zero", "random"])
@pytest.mark.parametrize("k", [1, 3, 8])
def test_c0_full_parity(nk, inflight, k):
    _say("c0 full", inflight, "k", k)
    cfg = W.CONFIGS["c0"]
    snap, req, cache = _inputs(cfg, 0, inflight)
    sel = _gpu(nk, snap, cache)
    g = _run(nk, sel, req, k)
    o = oracle.select(snap, cache, req, k=k, pairs=True, n_threads=8)
    (n, near), _ = _check_all(g, o)
    assert n > 0.99 * cfg.n_requests * k
    g2 = _run(nk, sel, req, k, pairs=False)
    assert np.array_equal(g2["idx"], g["idx"])
    assert np.array_equal(g2["score"].view(np.uint32), g["score"].view(np.uint32))
    sel.close()


def test_c0_load_terms_and_memory_pressure(nk):
    """Non-zero slope of t_iter, alpha != 1, wide batch sizes and a reserve
    that makes a third of the pairs infeasible."""
    _say("c0 variant load terms")
    cfg = W.scaled(W.CONFIGS["c0"], beta_range=(0, 64), t_iter_a=0.02, t_iter_b=0.0006,
                   alpha=0.5, queue_mean=30.0)
    snap, req, cache = _inputs(cfg, 3, "random")
    snap["m_min"] = 60 * 10 ** 9
    sel = _gpu(nk, snap, cache)
    g = _run(nk, sel, req, 4)
    o = oracle.select(snap, cache, req, k=4, pairs=True, n_threads=8)
    assert 0.05 < 1 - o["feasible"].mean() < 0.9
    _check_all(g, o)
    sel.close()


def test_ragged_decodes_long_runs_and_empty_runs(nk):
    """90 decodes (a full and a partial wavefront of decodes), 16-token
    blocks so that runs exceed 256 blocks (several 64-block steps of the
    leader kernel), and requests shorter than one block (empty runs)."""
    _say("ragged decodes / long runs")
    cl = W.Cluster(8, 5, 1, 3)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=cl, block_tokens=16, n_requests=700,
                   cache_per_decode=6000, len_median=3000.0)
    snap, req, cache = _inputs(cfg, 5, "random")
    assert cfg.n_decode == 90
    # a few requests with fewer tokens than one block
    req["len_tokens"][:5] = np.array([1, 5, 15, 3, 9], np.uint32)
    n = (req["len_tokens"] // 16).astype(np.int64)
    old = req["hash_off"].astype(np.int64)
    keep = np.concatenate([np.arange(old[r], old[r] + n[r]) for r in range(len(n))])
    req["hashes"] = req["hashes"][keep]
    req["hash_off"] = np.concatenate([[0], np.cumsum(n)]).astype(np.uint64)
    assert n.max() > 256
    sel = _gpu(nk, snap, cache)
    g = _run(nk, sel, req, 3)
    o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=8)
    _check_all(g, o)
    assert o["j"].max() > 256
    sel.close()


def test_tuning_options_leave_results_unchanged(nk):
    """Decodes per lane (1, 2, 3, 4, 6), run lengths (1, 7, automatic, longer
    than the batch), prefix sharing on/off and the leader table's size are
    layout choices only:
    every pair and every top-k entry is bit-identical across them, and the
    first matches the oracle.  270 decodes leave a partial last group of
    decodes at every width."""
    _say("tuning options")
    cl = W.Cluster(8, 5, 3, 3)
    cfg = W.scaled(W.CONFIGS["c2"], cluster=cl, n_requests=3000, cache_per_decode=4096)
    assert cfg.n_decode == 270
    snap, req, cache = _inputs(cfg, 8, "random")
    sel = _gpu(nk, snap, cache)
    base = None
    for cols in (1, 2, 3, 4, 6):
        for rl in (1, 7, 0, 5000):
            for reuse in (1, 0):
                if reuse == 0 and rl not in (0, 7):
                    continue
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, cols)
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_RUN_LEN, rl)
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_REUSE, reuse)
                g = _run(nk, sel, req, 3)
                if base is None:
                    base = g
                    o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=8)
                    _check_all(g, o)
                    continue
                for key in base:
                    assert np.array_equal(g[key], base[key]), (cols, rl, reuse, key)
    # a leader table that takes 1, 13 or 200 leaders (and as many blocks'
    # holder values): leaders past it, and the requests that follow them,
    # are matched on their own; leaders without holder room look up their
    # blocks themselves
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, 0)
    for cap in (1, 13, 200):
        for reuse in (1, 0):
            nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, cap)
            nk.netkv_set_option(sel.h, nk.NETKV_OPT_REUSE, reuse)
            nk.netkv_set_option(sel.h, nk.NETKV_OPT_RUN_LEN, 7 if reuse else 0)
            g = _run(nk, sel, req, 3)
            for key in base:
                assert np.array_equal(g[key], base[key]), (cap, reuse, key)
            g2 = _run(nk, sel, req, 3, pairs=False)
            assert np.array_equal(g2["idx"], base["idx"]), (cap, reuse)
            assert np.array_equal(g2["score"].view(np.uint32), base["score"].view(np.uint32)), (cap, reuse)
    sel.close()


def test_six_columns_with_a_partial_second_group(nk):
    """420 decodes at 6 decodes per lane: one whole group of 384 and one of
    36, whose other columns read past the last decode (the next row, or the
    padding after the last row for the last prefill) and must never be
    selected.  Per-pair outputs and top-3 against the oracle; the top-1
    kernel (three requests reduced together) bit-identical to the per-pair
    kernel's top-1, with and without requests that skip the feasibility
    test."""
    cl = W.Cluster(8, 7, 5, 2)
    cfg = W.scaled(W.CONFIGS["c2"], cluster=cl, n_requests=3000, cache_per_decode=4096)
    assert cfg.n_decode == 420
    for m_min in (None, 15 * 10 ** 9):
        _say("six columns, partial second group, m_min", m_min)
        snap, req, cache = _inputs(cfg, 21, "random")
        if m_min is not None:
            snap["m_min"] = m_min
        assert (np.asarray(req["prefill"]) == cfg.n_prefill - 1).any()
        sel = _gpu(nk, snap, cache)
        nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, 6)
        o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=8)
        g = _run(nk, sel, req, 3)
        _check_all(g, o)
        assert (g["idx"] < cfg.n_decode).all()
        g1 = _run(nk, sel, req, 1)
        g2 = _run(nk, sel, req, 1, pairs=False)
        assert np.array_equal(g2["idx"], g1["idx"])
        assert np.array_equal(g2["score"].view(np.uint32), g1["score"].view(np.uint32))
        sel.close()


def test_all_feasible_path_matches_general_path(nk):
    """A pool of whole wavefronts of decodes (384), where a request no
    longer than every feasibility limit of a decode group is scored without
    per-pair feasibility tests: the top-k-only kernel must match the
    per-pair kernel bit for bit, and the oracle, under every decodes-per-lane
    choice, with requests on both sides of the limits."""
    _say("all-feasible path")
    cl = W.Cluster(8, 8, 4, 2)
    cfg = W.scaled(W.CONFIGS["c2"], cluster=cl, n_requests=4000, cache_per_decode=4096)
    assert cfg.n_decode == 384
    snap, req, cache = _inputs(cfg, 11, "random")
    snap["m_min"] = 15 * 10 ** 9
    sel = _gpu(nk, snap, cache)
    o = oracle.select(snap, cache, req, k=2, pairs=True, n_threads=8)
    allf = o["feasible"].all(axis=1)
    assert 0.05 < allf.mean() < 0.95, allf.mean()
    for cols in (0, 1, 2, 3, 6):
        nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, cols)
        g = _run(nk, sel, req, 2)
        _check_all(g, o)
        g2 = _run(nk, sel, req, 2, pairs=False)
        assert np.array_equal(g2["idx"], g["idx"]), cols
        assert np.array_equal(g2["score"].view(np.uint32), g["score"].view(np.uint32)), cols
    sel.close()


@pytest.mark.parametrize("lf", [0.9, 0.99])
def test_dense_tables(nk, lf):
    """A dense holder index (load factor capped at 0.85, buckets rounded to a
    power of two): many displacements while building; membership must be
    unaffected.  The index holds exactly the distinct resident hashes, and
    a bitmap row for exactly those resident on two or more decodes."""
    _say("dense tables lf", lf)
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=1500, cache_per_decode=3000)
    snap, req, cache = _inputs(cfg, 7)
    sel = _gpu(nk, snap, cache, lf=lf)
    ci = nk.netkv_cache_info(sel.h)
    off = cache["hash_off"].astype(np.int64)
    owner = np.repeat(np.arange(cfg.n_decode), np.diff(off))
    pairs = np.unique(np.stack([cache["hashes"].astype(np.uint64), owner.astype(np.uint64)]), axis=1)
    hs, holders = np.unique(pairs[0], return_counts=True)
    assert ci["distinct_hashes"] == hs.size
    assert ci["shared_hashes"] == int((holders >= 2).sum()) > 0
    buckets = 8
    while 2 * buckets * min(lf, 0.85) < hs.size:
        buckets *= 2
    assert ci["index_slots"] in (2 * buckets, 4 * buckets, 8 * buckets)
    g = _run(nk, sel, req, 2)
    o = oracle.select(snap, cache, req, k=2, pairs=True, n_threads=8)
    _check_all(g, o)
    sel.close()


def test_all_infeasible_and_full_hits(nk):
    _say("all infeasible / full hits")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=300)
    snap, req, cache = _inputs(cfg, 9)
    # every decode caches the whole run of request 0..9: full hits, s_eff = bpt * (l mod B_tok)
    off = req["hash_off"].astype(np.int64)
    extra = np.concatenate([req["hashes"][off[r]:off[r + 1]] for r in range(10)])
    extra = np.unique(extra)
    per = []
    coff = cache["hash_off"].astype(np.int64)
    for d in range(cfg.n_decode):
        h = cache["hashes"][coff[d]:coff[d + 1]]
        per.append(np.union1d(h, extra))
    cache2 = dict(hash_off=np.concatenate([[0], np.cumsum([len(x) for x in per])]).astype(np.uint64),
                  hashes=np.concatenate(per).astype(np.uint64))
    sel = _gpu(nk, snap, cache2)
    g = _run(nk, sel, req, 2)
    o = oracle.select(snap, cache2, req, k=2, pairs=True, n_threads=8)
    n10 = (np.diff(off)[:10])
    assert (o["j"][:10] == n10[:, None]).all()
    _check_all(g, o)
    # a reserve larger than any free memory rejects every request
    snap2 = dict(snap)
    snap2["m_min"] = 2 ** 63
    sel.load_snapshot(snap2)
    g2 = _run(nk, sel, req, 3, pairs=False)
    assert (g2["idx"] == -1).all() and np.isinf(g2["score"]).all()
    sel.close()


def test_determinism_and_insertion_order(nk):
    _say("determinism / insertion order")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=2000)
    snap, req, cache = _inputs(cfg, 11)
    sel = _gpu(nk, snap, cache)
    a = _run(nk, sel, req, 3)
    b = _run(nk, sel, req, 3)
    for key in a:
        np.testing.assert_array_equal(a[key], b[key])
    # permute each decode's hash list: slots move, membership does not
    rng = np.random.default_rng(0)
    off = cache["hash_off"].astype(np.int64)
    perm = np.concatenate([off[d] + rng.permutation(off[d + 1] - off[d]) for d in range(cfg.n_decode)])
    cache_p = dict(hash_off=cache["hash_off"], hashes=cache["hashes"][perm])
    sel.load_cache(cache_p, 0.5)
    c = _run(nk, sel, req, 3)
    for key in a:
        np.testing.assert_array_equal(a[key], c[key])
    sel.close()


def test_subset_batches_match_full_batch(nk):
    """Scoring is per request: any subset, in any order, gives the same rows."""
    _say("subset batches")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=3000)
    snap, req, cache = _inputs(cfg, 13)
    sel = _gpu(nk, snap, cache)
    full = _run(nk, sel, req, 2, pairs=False)
    rows = np.random.default_rng(1).permutation(3000)[:777]
    sub = _run(nk, sel, subset_requests(req, rows), 2, pairs=False)
    np.testing.assert_array_equal(sub["idx"], full["idx"][rows])
    np.testing.assert_array_equal(sub["score"], full["score"][rows])
    sel.close()


def test_invalid_requests_are_flagged(nk):
    """Requests with no such prefill instance or a run length inconsistent
    with l_r are answered with -1 / NaN and reported; a block hash 0 (which
    no resident set can hold) is an ordinary miss."""
    _say("invalid requests")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=64)
    snap, req, cache = _inputs(cfg, 15)
    sel = _gpu(nk, snap, cache)
    bad = {k: v.copy() for k, v in req.items() if k in ("prefill", "len_tokens", "hash_off", "hashes")}
    bad["prefill"][3] = 999            # no such prefill instance
    bad["len_tokens"][7] += 512 * 3    # run length inconsistent with l_r
    # a hash 0 inside the longest run that some decode matches past it
    o0 = oracle.select(snap, cache, req, k=1, pairs=True)
    r0 = int(np.argmax(o0["j"].max(axis=1)))
    assert r0 not in (3, 7) and o0["j"][r0].max() >= 2
    bad["hashes"][int(bad["hash_off"][r0]) + 1] = 0
    rd = nk.requests_to_device(bad, sel.device)
    out = sel.select(rd, k=2)
    with pytest.raises(nk.NetKVError) as e:
        sel.sync_errors()
    assert e.value.status == -1
    idx = nk.to_numpy(out["idx"]).reshape(-1, 2)
    sc = nk.to_numpy(out["score"]).reshape(-1, 2)
    for r in (3, 7):
        assert (idx[r] == -1).all() and np.isnan(sc[r]).all()
    good = [r for r in range(64) if r not in (3, 7)]
    o = oracle.select(snap, cache, subset_requests(bad, good), k=2, pairs=True)
    assert o["j"][good.index(r0)].max() == 1
    check_topk(idx[good], sc[good], o["idx"], o["cost"], o["feasible"])
    sel.sync_errors()  # cleared
    sel.close()


def test_contract_errors_write_nothing(nk):
    _say("contract errors")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=32)
    snap, req, cache = _inputs(cfg, 17)
    sel = nk.Selector(0)
    rd = nk.requests_to_device(req, sel.device)
    idx = torch.full((32 * 9,), 7, dtype=torch.int32, device=sel.device)
    sc = torch.full((32 * 9,), 7.0, dtype=torch.float32, device=sel.device)
    with pytest.raises(nk.NetKVError) as e:
        nk.netkv_select_batch(sel.h, rd, 2, idx, sc, None, sel.device)
    assert e.value.status == -2  # ENOTREADY
    sel.load_snapshot(snap)
    with pytest.raises(nk.NetKVError) as e:
        nk.netkv_select_batch(sel.h, rd, 2, idx, sc, None, sel.device)
    assert e.value.status == -2
    sel.load_cache(cache)
    for kk in (0, 9):
        with pytest.raises(nk.NetKVError) as e:
            nk.netkv_select_batch(sel.h, rd, kk, idx, sc, None, sel.device)
        assert e.value.status == -1
    torch.cuda.synchronize()
    assert (idx == 7).all() and (sc == 7.0).all()
    # invalid snapshot values are rejected and the old snapshot is kept
    s2 = dict(snap)
    s2["util"] = snap["util"].copy()
    s2["util"][5] = 1.0
    with pytest.raises(nk.NetKVError) as e:
        sel.load_snapshot(s2)
    assert e.value.status == -1
    s3 = dict(snap)
    s3["tier_map"] = snap["tier_map"].copy()
    s3["tier_map"][0] = 4
    with pytest.raises(nk.NetKVError):
        sel.load_snapshot(s3)
    s4 = dict(snap)
    s4["batch_size"] = snap["batch_size"].copy()
    s4["batch_size"][0] = 65
    with pytest.raises(nk.NetKVError):
        sel.load_snapshot(s4)
    s5 = dict(snap)
    s5["tier_bw"] = np.array([1.0, 0.0, 1.0, 1.0])
    with pytest.raises(nk.NetKVError):
        sel.load_snapshot(s5)
    # a cache with the reserved value or a mismatched decode count
    c2 = dict(hash_off=cache["hash_off"], hashes=cache["hashes"].copy())
    c2["hashes"][17] = 0
    with pytest.raises(nk.NetKVError) as e:
        sel.load_cache(c2)
    assert e.value.status == -1
    c3 = dict(hash_off=cache["hash_off"][:-1], hashes=cache["hashes"])
    with pytest.raises(nk.NetKVError):
        sel.load_cache(c3)
    with pytest.raises(nk.NetKVError):
        sel.load_cache(cache, 1.0)
    # the previously loaded state still answers like the oracle
    g = _run(nk, sel, req, 2)
    o = oracle.select(snap, cache, req, k=2, pairs=True)
    check_pairs(g["j"], g["feas"], g["cost"], o)
    # empty batch is a no-op
    empty = dict(prefill=np.zeros(0, np.uint32), len_tokens=np.zeros(0, np.uint32),
                 hash_off=np.zeros(1, np.uint64), hashes=np.zeros(1, np.uint64))
    sel.select(nk.requests_to_device(empty, sel.device), k=1)
    sel.sync_errors()
    sel.close()


def test_kernel_timing_mean_over_launches(nk):
    """Timing records one scan per select without synchronising; the mean
    covers the launches since timing was enabled, and enabling restarts it."""
    _say("kernel timing")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=512)
    snap, req, cache = _inputs(cfg, 21)
    sel = _gpu(nk, snap, cache)
    rd = nk.requests_to_device(req, sel.device)
    idx = torch.empty(512, dtype=torch.int32, device=sel.device)
    sc = torch.empty(512, dtype=torch.float32, device=sel.device)
    nk.netkv_set_timing(sel.h, True)
    with pytest.raises(nk.NetKVError) as e:
        nk.netkv_kernel_ms(sel.h)
    assert e.value.status == -2
    for _ in range(300):          # more than the ring holds
        nk.netkv_select_batch(sel.h, rd, 1, idx, sc, None, sel.device)
    ms = nk.netkv_kernel_ms(sel.h)
    assert 0.0 < ms < 100.0
    nk.netkv_set_timing(sel.h, True)
    with pytest.raises(nk.NetKVError):
        nk.netkv_kernel_ms(sel.h)
    nk.netkv_set_timing(sel.h, False)
    nk.netkv_select_batch(sel.h, rd, 1, idx, sc, None, sel.device)
    with pytest.raises(nk.NetKVError):
        nk.netkv_kernel_ms(sel.h)
    sel.close()


def test_requests_across_2_pow_24_tokens(nk):
    """Token counts below 2^24 are scored in fp32, longer requests are
    matched on their own and scored in integers; a request of 2^25 tokens
    leads the shorter ones that share its chain, so those read its prefix
    lengths capped by their own.  Both kernels (per-pair outputs and
    top-k only) must equal the oracle across the boundary."""
    _say("requests across 2^24 tokens")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=8)
    bt = cfg.block_tokens
    snap = W.make_snapshot(cfg, 23)
    D = cfg.n_decode
    rng = np.random.default_rng(23)
    lens = np.array([2**25 - 1000, 2**24 - 1, 2**24, 2**24 + 300, 2**24 + 5 * bt + 7, 1000, 2**24 - bt, 70000],
                    dtype=np.uint32)
    nb = (lens // bt).astype(np.int64)
    chain = (np.arange(1, nb.max() + 1, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15)) | np.uint64(1)
    # decode 0 holds the whole chain, decodes 1 and 2 its first 20000 and 100 blocks
    sets = [chain, chain[:20000], chain[:100]] + [rng.integers(1, 2**63, 500, dtype=np.uint64)
                                                  for _ in range(D - 3)]
    cache = dict(n_decode=D, hash_off=np.concatenate([[0], np.cumsum([len(x) for x in sets])]).astype(np.uint64),
                 hashes=np.concatenate(sets).astype(np.uint64))
    runs = [chain[:n] for n in nb]
    runs[3] = np.concatenate([chain[:nb[3] - 10], rng.integers(1, 2**63, 10, dtype=np.uint64)])
    runs[7] = rng.integers(1, 2**63, nb[7], dtype=np.uint64)
    req = dict(n_req=len(lens), prefill=rng.integers(0, cfg.n_prefill, len(lens)).astype(np.uint32),
               len_tokens=lens, hash_off=np.concatenate([[0], np.cumsum(nb)]).astype(np.uint64),
               hashes=np.concatenate(runs).astype(np.uint64))
    assert nb.max() < 65535
    sel = _gpu(nk, snap, cache)
    o = oracle.select(snap, cache, req, k=2, pairs=True)
    # the long requests fit only where their whole run is resident
    long = [0, 1, 2, 3, 4, 6]
    assert o["feasible"][long, 0].all() and not o["feasible"][long, 1:].any()
    g = _run(nk, sel, req, 2)
    _check_all(g, o)
    g2 = _run(nk, sel, req, 2, pairs=False)
    assert np.array_equal(g2["idx"], g["idx"])
    assert np.array_equal(g2["score"].view(np.uint32), g["score"].view(np.uint32))
    sel.close()


def test_long_runs_and_invalid_requests_in_every_mode(nk):
    """Runs longer than 65535 blocks (B_tok = 1): the batch selection scores
    them exactly and writes prefix lengths saturated at 65535; the ranking
    sweep under the snapshot's own congestion and the sequential form with
    no counter growth (cap 0) reproduce the selection for them, from leader
    rows and from each request's own scan; a request whose run length
    contradicts l_r is answered with -1 / NaN in every mode and reported.
    A block hash 0 ends a match."""
    _say("long runs, B_tok 1")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=6, block_tokens=1)
    snap = W.make_snapshot(cfg, 21)
    D = cfg.n_decode
    rng = np.random.default_rng(21)
    chain = np.arange(1, 70001, dtype=np.uint64) * np.uint64(0x9E3779B97F4A7C15) | np.uint64(1)
    # decode 0 holds the whole chain, decode 1 its first 100 blocks, the rest random filler
    sets = [chain, chain[:100]] + [rng.integers(1, 2**63, 500, dtype=np.uint64) for _ in range(D - 2)]
    cache = dict(n_decode=D, hash_off=np.concatenate([[0], np.cumsum([len(x) for x in sets])]).astype(np.uint64),
                 hashes=np.concatenate(sets).astype(np.uint64))
    lens = np.array([70000, 70500, 1000, 900, 40, 66000], dtype=np.uint32)
    runs = [chain, np.concatenate([chain, rng.integers(1, 2**63, 500, dtype=np.uint64)]),
            chain[:1000], rng.integers(1, 2**63, 900, dtype=np.uint64), chain[:40],
            np.concatenate([chain[:50], rng.integers(1, 2**63, 65950, dtype=np.uint64)])]
    lens[3] += 1        # run length != l_r / B_tok: request 3 is invalid everywhere
    runs[2] = runs[2].copy()
    runs[2][500] = 0    # resident nowhere: request 2 matches 500 blocks on decode 0
    req = dict(n_req=6, prefill=rng.integers(0, cfg.n_prefill, 6).astype(np.uint32), len_tokens=lens,
               hash_off=np.concatenate([[0], np.cumsum([len(x) for x in runs])]).astype(np.uint64),
               hashes=np.concatenate(runs).astype(np.uint64))
    sel = _gpu(nk, snap, cache)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=2, pairs=True)
    with pytest.raises(nk.NetKVError):
        sel.sync_errors()
    idx = nk.to_numpy(out["idx"]).reshape(-1, 2)
    sc = nk.to_numpy(out["score"]).reshape(-1, 2)
    good = [0, 1, 2, 4, 5]
    o = oracle.select(snap, cache, subset_requests(req, good), k=2, pairs=True)
    assert int(o["j"][0, 0]) == 70000 and int(o["j"][1, 0]) == 70000 and int(o["j"][2, 0]) == 500
    check_topk(idx[good], sc[good], o["idx"], o["cost"], o["feasible"])
    j = nk.to_numpy(out["pairs"]["prefix_blocks"]).reshape(6, D)[good].astype(np.int64)
    assert np.array_equal(j, np.minimum(o["j"], 65535))
    assert (idx[3] == -1).all() and np.isnan(sc[3]).all()
    # ranking sweep under the snapshot's own congestion, and the sequential form
    us = nk.to_device(np.asarray(snap["util"], np.float32).reshape(-1), sel.device)
    sw = sel.rank_sweep(rd, us, k=2)
    with pytest.raises(nk.NetKVError):
        sel.sync_errors()
    sq = sel.select_sequential(rd, cap=0)
    with pytest.raises(nk.NetKVError):
        sel.sync_errors()
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, 1)   # one leader row: the rest match on their own
    sq1 = sel.select_sequential(rd, cap=0)
    with pytest.raises(nk.NetKVError):
        sel.sync_errors()
    si = nk.to_numpy(sw["idx"]).reshape(-1, 2)
    ss = nk.to_numpy(sw["score"]).reshape(-1, 2)
    # the sweep and the sequential form take prefix lengths from leader rows
    # (or own scans): every valid request, long runs included, reproduces
    # the selection; the invalid one is -1/NaN
    assert (si[3] == -1).all() and np.isnan(ss[3]).all()
    for r in (0, 1, 2, 4, 5):
        assert np.array_equal(si[r], idx[r]) and np.array_equal(ss[r].view(np.uint32), sc[r].view(np.uint32))
    for q in (sq, sq1):
        qi, qs = nk.to_numpy(q["idx"]), nk.to_numpy(q["score"])
        assert qi[3] == -1 and np.isnan(qs[3])
        for r in (0, 1, 2, 4, 5):
            assert qi[r] == idx[r, 0] and qs[r].view(np.uint32) == sc[r, 0].view(np.uint32)
    sel.close()


def _uniform_snapshot(cfg, queue=6, tier=2, util=0.3):
    """A snapshot on which every decode is identical from every prefill: one
    tier, one congestion value, one queue depth, batch size and free memory."""
    P, D = cfg.n_prefill, cfg.n_decode
    snap = dict(W.params_of(cfg))
    snap.update(n_prefill=P, n_decode=D, tier_map=np.full(P * D, tier, np.uint8),
                util=np.full(P * D, util, np.float32), n_inflight=np.zeros(4 * P, np.uint16),
                free_mem=np.full(D, 100 * 10 ** 9, np.uint64), queue_depth=np.full(D, queue, np.uint32),
                batch_size=np.full(D, 60, np.uint32))
    return snap


def test_exact_ties_go_to_the_lowest_index(nk):
    """Algorithm 1's argmin with ties to the lowest decode index, on exact
    ties spread over lanes, decode columns and decode groups (3,072 decodes,
    every decodes-per-lane choice, k = 1, 3, 8):
      * every decode identical: the top-k is decodes 0..k-1;
      * the decodes of S one queue slot shorter (identical among
        themselves): S in ascending order, then 0, 1, ...;
      * S plus decodes of S2 that also hold a request's whole run: the
        oracle's order, which the GPU must reproduce exactly.
    The expected lists of the first two cases are written out here; every
    case is also checked against the oracle and against the exact top-k of
    the GPU's own per-pair scores."""
    cfg = W.scaled(W.CONFIGS["c2"], n_requests=200, cache_per_decode=64)
    D = cfg.n_decode
    assert D == 3072
    S = np.array([5, 64 + 5, 3 * 64 + 7, 384 + 2, 2 * 384 + 3 * 64 + 1, 1000, 2047, 3071])
    S2 = np.array([7, 64 + 9, 700, 3000])
    ch = W.prefix_chains(cfg, 31)
    req = W.make_requests(cfg, 31, chains=ch)
    n_r = np.diff(req["hash_off"].astype(np.int64))
    rng = np.random.default_rng(31)
    base_sets = [rng.integers(1, 2 ** 63, 64, dtype=np.uint64) for _ in range(D)]
    runs = np.unique(np.concatenate([req["hashes"][int(req["hash_off"][r]):int(req["hash_off"][r + 1])]
                                     for r in range(20)]))
    rows = np.arange(cfg.n_requests)

    def cache_of(extra):
        sets = [np.union1d(base_sets[d], runs) if d in extra else base_sets[d] for d in range(D)]
        return dict(n_decode=D, hash_off=np.concatenate([[0], np.cumsum([len(x) for x in sets])]).astype(np.uint64),
                    hashes=np.concatenate(sets).astype(np.uint64))

    cases = []
    snap_a = _uniform_snapshot(cfg)
    exp_a = np.tile(np.arange(8), (cfg.n_requests, 1))
    cases.append(("all identical", snap_a, cache_of(set()), exp_a))
    snap_b = _uniform_snapshot(cfg)
    snap_b["queue_depth"] = snap_b["queue_depth"].copy()
    snap_b["queue_depth"][S] = 5   # one blocked request fewer (4 free batch slots)
    exp_b = np.tile(np.concatenate([np.sort(S), [0, 1, 2, 3]])[:8], (cfg.n_requests, 1))
    cases.append(("S shorter queues", snap_b, cache_of(set()), exp_b))
    cases.append(("S and S2 with cached runs", snap_b, cache_of(set(S2.tolist())), None))
    for name, snap, cache, exp in cases:
        o = oracle.select(snap, cache, req, k=8, pairs=True, n_threads=8)
        if exp is not None:
            assert np.array_equal(o["idx"], exp), name
        else:
            # requests 0..19 hold their whole run on S2 (when they have blocks)
            assert (o["j"][:20][:, S2] == n_r[:20, None]).all()
        sel = _gpu(nk, snap, cache)
        for cols in (0, 1, 2, 3, 4, 6):
            nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, cols)
            for k in (1, 3, 8):
                _say("exact ties:", name, "cols", cols, "k", k)
                g = _run(nk, sel, req, k)
                ok = o["idx"][:, :k]
                assert np.array_equal(g["idx"], ok), (name, cols, k)
                oo = dict(o, idx=ok)
                _check_all(g, oo)
                g2 = _run(nk, sel, req, k, pairs=False)
                assert np.array_equal(g2["idx"], g["idx"]), (name, cols, k)
        sel.close()
    del rows


def _holed_cache(cfg, ch, wl_seed, seed):
    """Resident sets that are not prefix-closed: for each decode, segments of
    the shared chains with holes -- blocks a+1..a+5 without block a, a
    chain without its block 0, every other block, Bernoulli(0.6) scatter --
    next to ordinary leading segments, plus private filler."""
    rng = np.random.default_rng(seed)
    D = cfg.n_decode
    S = ch["blocks"]
    top = np.argsort(-ch["weights"])[:60]
    sets = []
    for d in range(D):
        parts = [rng.integers(1, 2 ** 63, 300, dtype=np.uint64)]
        for k in top:
            n = int(S[k])
            if n == 0 or rng.random() < 0.3:
                continue
            kind = rng.integers(0, 5)
            if kind == 0:      # blocks [0, a) and a+1 .. a+5, hole at a
                a = int(rng.integers(0, n))
                blk = np.concatenate([np.arange(0, a), np.arange(a + 1, min(n, a + 6))])
            elif kind == 1:    # everything but block 0
                blk = np.arange(1, n)
            elif kind == 2:    # every other block
                blk = np.arange(int(rng.integers(0, 2)), n, 2)
            elif kind == 3:    # scattered
                blk = np.nonzero(rng.random(n) < 0.6)[0]
            else:              # an ordinary leading segment
                blk = np.arange(0, int(rng.integers(1, n + 1)))
            if blk.size:
                parts.append(W.block_hash(wl_seed, int(ch["domain"]), np.full(blk.size, k), blk))
        sets.append(np.unique(np.concatenate(parts)))
    return dict(n_decode=D, hash_off=np.concatenate([[0], np.cumsum([len(x) for x in sets])]).astype(np.uint64),
                hashes=np.concatenate(sets).astype(np.uint64))


def test_holed_resident_sets(nk):
    """Resident sets with holes (Sec. III-B: the block LCP is the leading run
    up to the first miss, and K_d need not be prefix-closed).  Prefix
    lengths, feasibility and scores bit-exact against the oracle on 270
    decodes, with and without the batch order's sharing, under every
    decodes-per-lane choice and a leader table of 3."""
    cl = W.Cluster(8, 5, 3, 3)
    cfg = W.scaled(W.CONFIGS["c2"], cluster=cl, n_requests=3000, cache_per_decode=4096, n_prefixes=80)
    assert cfg.n_decode == 270
    seed = 3
    snap = W.make_snapshot(cfg, seed, inflight="random")
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = _holed_cache(cfg, ch, seed, 77)
    o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=8)
    # holes matter: some decode holds block j (and beyond) of a request
    # without holding all blocks before it
    assert o["j"].max() > 3
    sel = _gpu(nk, snap, cache)
    for cols in (0, 1, 3, 6):
        for reuse in (1, 0):
            for cap in (0, 3):
                _say("holed sets cols", cols, "reuse", reuse, "lead cap", cap)
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_COLS, cols)
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_REUSE, reuse)
                nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, cap)
                g = _run(nk, sel, req, 3)
                _check_all(g, o)
    sel.close()


_GOLDEN = 0x9E3779B97F4A7C15
_GOLDEN_INV = pow(_GOLDEN, -1, 1 << 64)


def _colliding_hashes(rng, n, bucket_bits=19):
    """n distinct nonzero 64-bit hashes whose Fibonacci products agree in the
    top bucket_bits bits -- the bits of the first block that the batch
    order groups requests by -- so that different chains share one group."""
    y0 = int(rng.integers(0, 1 << 63)) << 1
    top = (y0 >> (64 - bucket_bits)) << (64 - bucket_bits)
    out = set()
    while len(out) < n:
        y = top | int(rng.integers(0, 1 << (64 - bucket_bits)))
        h = (y * _GOLDEN_INV) % (1 << 64)
        if h:
            out.add(h)
    hs = np.array(sorted(out), dtype=np.uint64)
    prods = (hs.astype(object) * _GOLDEN) % (1 << 64)
    assert len({int(p) >> (64 - bucket_bits) for p in prods}) == 1
    return hs


def test_first_block_key_collisions(nk):
    """Chains whose first blocks differ but fall in the same group of the
    batch order (their sort keys agree in the first-block bits): the
    requests of the chains interleave by length in the hash order, so
    neighbours share no leading run and every switch starts a leader.  A
    batch of 70,000 requests (the library's own batch sorts) on 48 decodes:
    every pair bit-exact against the oracle, every top-3 within the rules."""
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=70000, block_tokens=64)
    rng = np.random.default_rng(41)
    snap = W.make_snapshot(cfg, 41, inflight="random")
    ch = W.prefix_chains(cfg, 41)
    req = W.make_requests(cfg, 41, chains=ch)
    D = cfg.n_decode
    nch, clen = 6, 300
    firsts = _colliding_hashes(rng, nch)
    chains = [np.concatenate([[firsts[c]], rng.integers(1, 2 ** 63, clen - 1, dtype=np.uint64)])
              for c in range(nch)]
    # 40 % of the requests switch to one of the colliding chains
    off = req["hash_off"].astype(np.int64)
    n_r = np.diff(off)
    pick = np.nonzero((rng.random(cfg.n_requests) < 0.4) & (n_r > 0))[0]
    hs = req["hashes"].copy()
    for r in pick:
        c = chains[int(rng.integers(0, nch))]
        m = min(int(n_r[r]), clen)
        hs[off[r]:off[r] + m] = c[:m]
    req = dict(req, hashes=hs)
    # decodes hold leading segments of the colliding chains (and some holes)
    base = W.make_caches(cfg, 41, chains=ch)
    coff = base["hash_off"].astype(np.int64)
    sets = []
    for d in range(D):
        parts = [base["hashes"][coff[d]:coff[d + 1]]]
        for c in range(nch):
            if rng.random() < 0.5:
                a = int(rng.integers(1, clen + 1))
                blk = np.arange(a)
                if rng.random() < 0.3 and a > 3:
                    blk = np.delete(blk, int(rng.integers(1, a)))
                parts.append(chains[c][blk])
        sets.append(np.unique(np.concatenate(parts)))
    cache = dict(n_decode=D, hash_off=np.concatenate([[0], np.cumsum([len(x) for x in sets])]).astype(np.uint64),
                 hashes=np.concatenate(sets).astype(np.uint64))
    o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=8)
    assert o["j"][pick].max() > 100
    sel = _gpu(nk, snap, cache)
    for reuse in (1, 0):
        _say("first-block key collisions, 70,000 x 48, reuse", reuse)
        nk.netkv_set_option(sel.h, nk.NETKV_OPT_REUSE, reuse)
        g = _run(nk, sel, req, 3)
        _check_all(g, o)
        g2 = _run(nk, sel, req, 3, pairs=False)
        assert np.array_equal(g2["idx"], g["idx"])
        assert np.array_equal(g2["score"].view(np.uint32), g["score"].view(np.uint32))
    sel.close()
