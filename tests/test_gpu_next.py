"""Ablation rungs of the cost, per-tier selection counts and the sequential
(request-by-request) form of Algorithm 1 on the GPU, against the CPU
oracle.  Needs an MI355X and the built library."""
import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import NEAR_TIE, SCORE_RTOL, check_pairs, check_topk, subset_requests

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


def _inputs(cfg, seed, inflight="random"):
    snap = W.make_snapshot(cfg, seed, inflight=inflight)
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    return snap, req, cache


@pytest.mark.parametrize("policy", [1, 2])
def test_policy_rungs_match_zeroed_snapshots(nk, policy):
    """Rung 1 (static tier map + self-contention) is the full cost with zero
    congestion; rung 2 (static tier map only) also zeroes the in-flight
    counters (Sec. VI, Experiment 6)."""
    _say("policy", policy)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=2000)
    snap, req, cache = _inputs(cfg, 41)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    sel.set_policy(policy)
    out = sel.select(nk.requests_to_device(req, sel.device), k=3, pairs=True)
    sel.sync_errors()
    osnap = dict(snap)
    osnap["util"] = np.zeros_like(snap["util"])
    if policy == 2:
        osnap["n_inflight"] = np.zeros_like(snap["n_inflight"])
    o = oracle.select(osnap, cache, req, k=3, pairs=True, n_threads=8)
    p = out["pairs"]
    check_pairs(nk.to_numpy(p["prefix_blocks"]), nk.to_numpy(p["feasible"]), nk.to_numpy(p["score"]), o)
    check_topk(nk.to_numpy(out["idx"]).reshape(-1, 3), nk.to_numpy(out["score"]).reshape(-1, 3),
               o["idx"], o["cost"], o["feasible"])
    sel.close()


def test_tier_counts(nk):
    _say("tier counts")
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=3000)
    snap, req, cache = _inputs(cfg, 43)
    # a reserve only the three freest decodes can meet (by 5 GB): requests
    # with more non-cached bytes than that are rejected
    snap["m_min"] = int(np.sort(snap["free_mem"])[-3]) - 5 * 10 ** 9
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=1)
    g_idx = nk.to_numpy(out["idx"])
    counts = sel.tier_counts(rd, out["idx"])
    sel.sync_errors()
    want = oracle.tier_counts(snap, req, g_idx)
    np.testing.assert_array_equal(counts, want)
    assert counts.sum() == cfg.n_requests and 0 < counts[4] < cfg.n_requests
    assert (counts[:4] > 0).sum() >= 2
    o = oracle.select(snap, cache, req, k=1, n_threads=8)
    ocounts = oracle.tier_counts(snap, req, o["idx"][:, 0])
    assert np.abs(counts.astype(np.int64) - ocounts.astype(np.int64)).sum() <= 2 * int(
        (g_idx != o["idx"][:, 0]).sum())
    sel.close()


def _check_sequential(g_idx, g_score, ref):
    """GPU choices against the oracle run in follow mode (counters advanced
    with the GPU's own choices): each choice must be the oracle's argmin or
    a near-tie of it, with its score within the fp32 tolerance."""
    o_idx, o_sc, f_cost = ref["idx"], ref["score"], ref["follow_cost"]
    rej = o_idx < 0
    assert (g_idx[rej] == -1).all()
    ok = ~rej
    assert (g_idx[ok] >= 0).all()
    assert np.isfinite(f_cost[ok]).all(), "GPU picked an infeasible decode"
    diff = ok & (g_idx != o_idx)
    assert (np.abs(f_cost[diff] - o_sc[diff]) <= NEAR_TIE * o_sc[diff]).all()
    rel = np.abs(g_score[ok].astype(np.float64) - f_cost[ok]) / f_cost[ok]
    assert rel.max() <= SCORE_RTOL
    return int(diff.sum())


@pytest.mark.parametrize("cap", [16, 2])
def test_sequential_stream_batch(nk, cap):
    """A 65,536-request batch at TP=4 sizing on the 64-GPU cluster, with
    in-flight counters starting from random values."""
    _say("sequential c1 batch cap", cap)
    cfg = W.CONFIGS["c1"]
    snap, req, cache = _inputs(cfg, 45)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select_sequential(rd, cap=cap)
    sel.sync_errors()
    g_idx, g_sc = nk.to_numpy(out["idx"]), nk.to_numpy(out["score"])
    ref = oracle.select_sequential(snap, oracle.Cache(cache, n_threads=8), req, cap=cap, follow=g_idx)
    near = _check_sequential(g_idx, g_sc, ref)
    assert near < 0.001 * cfg.n_requests
    # the sequential counters change selections relative to the snapshot semantics
    snap_sel = nk.to_numpy(sel.select(rd, k=1)["idx"])
    assert (snap_sel != g_idx).sum() > 0
    sel.close()


def test_sequential_cap_zero_is_snapshot_selection(nk):
    _say("sequential cap 0")
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=3000)
    snap, req, cache = _inputs(cfg, 47)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    a = sel.select_sequential(rd, cap=0)
    b = sel.select(rd, k=1)
    sel.sync_errors()
    np.testing.assert_array_equal(nk.to_numpy(a["idx"]), nk.to_numpy(b["idx"]))
    np.testing.assert_array_equal(nk.to_numpy(a["score"]), nk.to_numpy(b["score"]))
    sel.close()


@pytest.mark.timeout(900)
def test_sequential_full_size_two_prefill_instances(nk):
    """The full 4,096-GPU batch, sequential; every request of two prefill
    instances (in batch order, which is all that couples them) is checked
    against the oracle."""
    _say("sequential c2 full")
    cfg = W.CONFIGS["c2"]
    snap, req, cache = _inputs(cfg, 49)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select_sequential(rd, cap=16)
    sel.sync_errors()
    g_idx, g_sc = nk.to_numpy(out["idx"]), nk.to_numpy(out["score"])
    ocache = oracle.Cache(cache, n_threads=16)
    del cache
    for p in (5, 777):
        rows = np.flatnonzero(req["prefill"] == p)
        _say("oracle prefill", p, len(rows), "requests")
        ref = oracle.select_sequential(snap, ocache, subset_requests(req, rows), cap=16, follow=g_idx[rows])
        _check_sequential(g_idx[rows], g_sc[rows], ref)
    sel.close()


@pytest.mark.parametrize("shape", [(8, 8, 4, 4), (8, 8, 8, 4), (8, 8, 8, 5), (8, 8, 8, 6), (8, 8, 10, 8),
                                   (8, 8, 12, 8)])
def test_sequential_pool_sizes(nk, shape):
    """Pools of 768 / 1,536 / 1,920 / 2,304 / 3,840 / 4,608 decodes (4, 6,
    8, 12 and 16 decodes per thread of the register-held chain, and the
    general form beyond them), with 6,000
    requests from three prefill instances so that the counters of every
    tier grow and saturate within the batch; then the same batch with the
    prefix lengths taken by each request's own scan."""
    cl = W.Cluster(*shape)
    cfg = W.scaled(W.CONFIGS["c2"], cluster=cl, n_requests=6000, cache_per_decode=512)
    _say("sequential pool", cfg.n_decode)
    snap, req, cache = _inputs(cfg, 51)
    req["prefill"] = (np.arange(cfg.n_requests) % 3 * 7).astype(np.uint32)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select_sequential(rd, cap=16)
    sel.sync_errors()
    g_idx, g_sc = nk.to_numpy(out["idx"]), nk.to_numpy(out["score"])
    ref = oracle.select_sequential(snap, oracle.Cache(cache, n_threads=8), req, cap=16, follow=g_idx)
    near = _check_sequential(g_idx, g_sc, ref)
    assert near < 0.01 * cfg.n_requests
    # a leader table of two rows: nearly every request is matched on its own
    # (first-miss scan of its run) instead of from a leader row; the chain's
    # prefix lengths, and so its selections, are the same bits
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, 2)
    own = sel.select_sequential(rd, cap=16)
    sel.sync_errors()
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, 0)
    np.testing.assert_array_equal(nk.to_numpy(own["idx"]), g_idx)
    np.testing.assert_array_equal(nk.to_numpy(own["score"]).view(np.uint32), g_sc.view(np.uint32))
    sel.close()


def test_congestion_smoothing_matches_oracle(nk):
    """Predictive congestion (Sec. VIII; reading: simple exponential
    smoothing): a series of observations folded in with beta 1, 0.5 and
    0.1 gives the oracle's fp64 forecast within the fp32 rounding of the
    steps (at most ~1.2e-7 per step), an invalid observation leaves its entry
    unchanged and is reported, and a selection under the forecast matches
    the oracle's under the same forecast."""
    _say("congestion smoothing")
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=1500)
    snap, req, cache = _inputs(cfg, 43)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    npd = cfg.n_prefill * cfg.n_decode
    rng = np.random.default_rng(43)
    c = np.asarray(snap["util"], np.float32).astype(np.float64).reshape(-1)
    assert np.array_equal(sel.congestion(), np.asarray(snap["util"], np.float32).reshape(-1))
    steps = [1.0, 0.5, 0.5, 0.1, 0.1, 0.1]
    for s, beta in enumerate(steps):
        obs = rng.uniform(0, 0.99, npd).astype(np.float32)
        if s == 2:
            obs[[0, 7, npd - 1]] = [np.nan, 1.0, -0.5]
        sel.smooth_congestion(obs, beta)
        c, bad = oracle.smooth(c, obs, beta)
        if s == 2:
            assert bad == 3
            with pytest.raises(nk.NetKVError):
                sel.sync_errors()
        else:
            sel.sync_errors()
        g = sel.congestion().astype(np.float64)
        assert ((g >= 0) & (g < 1)).all()
        np.testing.assert_allclose(g, c, rtol=0, atol=1.2e-7 * (s + 1) + 1e-9)
    # selection under the forecast
    fsnap = dict(snap)
    fsnap["util"] = sel.congestion().reshape(np.asarray(snap["util"]).shape)
    out = sel.select(nk.requests_to_device(req, sel.device), k=2, pairs=True)
    sel.sync_errors()
    o = oracle.select(fsnap, cache, req, k=2, pairs=True, n_threads=8)
    check_pairs(nk.to_numpy(out["pairs"]["prefix_blocks"]), nk.to_numpy(out["pairs"]["feasible"]),
                nk.to_numpy(out["pairs"]["score"]), o)
    check_topk(nk.to_numpy(out["idx"]).reshape(-1, 2), nk.to_numpy(out["score"]).reshape(-1, 2),
               o["idx"], o["cost"], o["feasible"])
    # contract: beta outside (0, 1] is rejected and changes nothing
    before = sel.congestion()
    for beta in (0.0, 1.5, float("nan")):
        with pytest.raises(nk.NetKVError):
            sel.smooth_congestion(np.zeros(npd, np.float32), beta)
    assert np.array_equal(sel.congestion(), before)
    sel.close()


def test_congestion_smoothing_odd_sizes_and_unaligned_observations(nk):
    """The vectorised smoothing path's tail (P * D = 21, not a multiple of 4)
    and the scalar path (an observation that is not 16-byte aligned)."""
    _say("congestion smoothing, odd sizes")
    from tests.test_oracle_pins import tiny_snapshot
    rng = np.random.default_rng(44)
    P, D = 3, 7
    util = rng.uniform(0, 0.99, P * D).astype(np.float32)
    snap = tiny_snapshot(P, D, rng.integers(0, 4, P * D), util)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    c = util.astype(np.float64)
    for beta, offset in ((0.25, 0), (0.6, 1), (1.0, 3)):
        obs = rng.uniform(0, 0.99, P * D).astype(np.float32)
        buf = torch.zeros(P * D + 4, dtype=torch.float32, device=sel.device)
        buf[offset:offset + P * D] = torch.from_numpy(obs).to(sel.device)
        view = buf[offset:offset + P * D]
        assert (view.data_ptr() % 16 == 0) == (offset == 0)
        sel.smooth_congestion(view, beta)
        sel.sync_errors()
        c, _ = oracle.smooth(c, obs, beta)
        np.testing.assert_allclose(sel.congestion().astype(np.float64), c, rtol=0, atol=4e-7)
    sel.close()
