"""Streaming batches with between-batch updates and stale congestion
(64 GPUs, TP=4 sizing), and the stale-telemetry ranking sweep, against the
CPU oracle.  Needs an MI355X and the built library."""
import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import check_topk

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

COUNTER_CAP = 16     # self-contention counter cap (Sec. V-C default)


def _say(*a):
    print("[gpu-case]", *a, flush=True)


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03910_amd import netkv
    netkv.load_library()
    return netkv


@pytest.mark.parametrize("staleness", [0, 1, 4])
def test_c1_stream_with_updates(nk, staleness):
    """16 batches of 65,536 requests; congestion drifts as AR(1) and the
    selector sees it `staleness` batches late; decode state and in-flight
    counters are updated after every batch from the GPU's selections (both
    sides apply the update; the states must stay bit-identical)."""
    cfg = W.CONFIGS["c1"]
    seed = 21
    snap = W.make_snapshot(cfg, seed)
    ch = W.prefix_chains(cfg, seed)
    cache = W.make_caches(cfg, seed, chains=ch)
    links = W.ar1_links(cfg, seed, snap["links"], cfg.n_batches)
    mu = -(-cfg.n_requests // cfg.n_decode)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    ocache = oracle.Cache(cache, n_threads=8)
    state = dict(n_inflight=snap["n_inflight"].copy(), queue_depth=snap["queue_depth"].copy(),
                 free_mem=snap["free_mem"].copy(), admitted_prev=np.zeros(cfg.n_decode, np.uint64))
    near_total = 0
    for t in range(cfg.n_batches):
        _say("c1 staleness", staleness, "batch", t)
        util = W.pair_util(cfg.cluster, links[max(0, t - staleness)]).reshape(-1)
        sel.set_util(util)
        req = W.make_requests(cfg, seed, batch=t, chains=ch)
        rd = nk.requests_to_device(req, sel.device)
        out = sel.select(rd, k=1)
        sel.sync_errors()
        g_idx = nk.to_numpy(out["idx"]).reshape(-1, 1)
        g_sc = nk.to_numpy(out["score"]).reshape(-1, 1)
        osnap = dict(snap)
        osnap.update(util=util, n_inflight=state["n_inflight"], queue_depth=state["queue_depth"],
                     free_mem=state["free_mem"])
        o = oracle.select(osnap, ocache, req, k=1, pairs=True, n_threads=8)
        _, near = check_topk(g_idx, g_sc, o["idx"], o["cost"], o["feasible"])
        near_total += near
        # both sides apply the between-batch update from the GPU's selections
        sel.commit(rd, out["idx"], COUNTER_CAP, mu)
        sel.sync_errors()
        state = oracle.commit(osnap, ocache, req, g_idx[:, 0], COUNTER_CAP, mu, state)
        gs = sel.state()
        for key in ("n_inflight", "queue_depth", "free_mem", "admitted_prev"):
            np.testing.assert_array_equal(gs[key], state[key], err_msg=f"{key} batch {t}")
        assert state["n_inflight"].max() <= COUNTER_CAP
    assert near_total < 0.001 * cfg.n_requests * cfg.n_batches
    sel.close()


def test_c3_rank_sweep(nk):
    """16,384 requests x 48 decodes under 1,024 noisy congestion scenarios
    (sigma 0.05 / 0.1 / 0.2 / 0.4): top-3 per scenario and the flip counts
    against the noise-free ranking.  The oracle checks a spread of 64
    scenarios element by element; the flip counts of all 1,024 are checked
    against the GPU's own selections."""
    cfg = W.CONFIGS["c3"]
    seed = 31
    snap = W.make_snapshot(cfg, seed)
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    util_s, sig = W.scenario_utils(cfg, seed, snap["links"])
    S, R, K = cfg.n_scenarios, cfg.n_requests, 3
    _say("c3 sweep GPU", S, "scenarios")
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    us = nk.to_device(util_s.reshape(-1), sel.device)
    out = sel.rank_sweep(rd, us, k=K)
    sel.sync_errors()
    g_idx = nk.to_numpy(out["idx"]).reshape(S, R, K)
    g_sc = nk.to_numpy(out["score"]).reshape(S, R, K)
    g_fl = nk.to_numpy(out["flips"]).reshape(S, 2)
    # flips are consistent with the GPU's own top-1 and its noise-free selection
    base = sel.select(rd, k=1)
    b_idx = nk.to_numpy(base["idx"])
    tm = snap["tier_map"].reshape(cfg.n_prefill, cfg.n_decode)
    p = req["prefill"].astype(np.int64)

    def tiers(ix):
        return np.where(ix >= 0, tm[p, np.maximum(ix, 0)], -1)

    bt = tiers(b_idx)
    for s in range(S):
        top = g_idx[s, :, 0]
        assert int(g_fl[s, 1]) == int((top != b_idx).sum())
        assert int(g_fl[s, 0]) == int((tiers(top) != bt).sum())
    # element-wise parity on a spread of scenarios
    pick = np.linspace(0, S - 1, 64).astype(int)
    _say("c3 sweep oracle on", len(pick), "scenarios")
    o = oracle.rank_sweep(snap, cache, req, util_s[pick], k=K, n_threads=8)
    ocache = oracle.Cache(cache, n_threads=8)
    o_base = oracle.select(snap, ocache, req, k=1)["idx"][:, 0]
    for i, s in enumerate(pick):
        osnap = dict(snap)
        osnap["util"] = util_s[s]
        op = oracle.select(osnap, ocache, req, k=K, pairs=True, n_threads=8)
        np.testing.assert_array_equal(op["idx"], o["idx"][i])
        check_topk(g_idx[s], g_sc[s], o["idx"][i], op["cost"], op["feasible"])
        # flip counts may differ from the oracle's only by near-tie choices
        near = int((g_idx[s, :, 0] != o["idx"][i][:, 0]).sum())
        near += int((b_idx != o_base).sum())
        assert abs(int(g_fl[s, 1]) - int(o["flips"][i, 1])) <= near
    # more noise, more flips (monotone in sigma on average)
    per_sigma = [g_fl[sig == sg, 0].mean() for sg in cfg.noise_sigmas]
    assert per_sigma[0] <= per_sigma[-1]
    sel.close()
