"""Two-hop KV routing (Sec. VIII) on the GPU against the CPU oracle: every
pair scores the faster of its direct route and its staged route through a
staging store, and a separate call reports which route each selection
takes.  Needs an MI355X and the built library."""
import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import NEAR_TIE, check_pairs, check_topk, subset_requests

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
    return snap, req, cache, W.make_routes(cfg, seed)


def _selector(nk, snap, cache, routes):
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    sel.load_routes(routes["route_tier1"], routes["route_util1"], routes["route_tier2"],
                    routes["route_util2"])
    return sel


def _select(nk, sel, req, k, pairs):
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=k, pairs=pairs)
    sel.sync_errors()
    res = dict(rd=rd, idx_dev=out["idx"], idx=nk.to_numpy(out["idx"]).reshape(-1, k),
               score=nk.to_numpy(out["score"]).reshape(-1, k))
    if pairs:
        p = out["pairs"]
        res.update(j=nk.to_numpy(p["prefix_blocks"]), feas=nk.to_numpy(p["feasible"]),
                   cost=nk.to_numpy(p["score"]))
    return res


def _check_routes(g_route, idx, snap, routes, cache, req, k):
    """The GPU's route of each selection against the oracle's; a different
    answer is allowed only where the two routes' costs are a near-tie (the
    staged cost alone is the oracle's cost with the direct routes made
    ten million times slower)."""
    both = dict(snap, **routes)
    o_route = oracle.route_of(both, cache, req, idx, k)
    g_route = np.asarray(g_route).reshape(-1)
    flat = idx.reshape(-1)
    np.testing.assert_array_equal(g_route < 0, flat < 0)
    diff = np.nonzero(g_route != o_route)[0]
    if diff.size:
        r, q = np.divmod(diff, k)
        d = flat[diff]
        sub = subset_requests(req, r)
        direct = oracle.select(snap, cache, sub, k=1, pairs=True)["cost"]
        slow = dict(both, util=np.full_like(snap["util"], np.float32(1 - 1e-7)))
        staged = oracle.select(slow, cache, sub, k=1, pairs=True)["cost"]
        rows = np.arange(len(diff))
        a, b = direct[rows, d], staged[rows, d]
        assert (np.abs(a - b) <= NEAR_TIE * np.minimum(a, b)).all(), "route differs off a near-tie"
    assert diff.size <= max(2, flat.size // 1000)
    return o_route


@pytest.mark.parametrize("k", [1, 3])
def test_two_hop_pairs_topk_and_routes(nk, k):
    _say("two-hop c0 scaled k", k)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=3000)
    snap, req, cache, routes = _inputs(cfg, 51)
    sel = _selector(nk, snap, cache, routes)
    g = _select(nk, sel, req, k, pairs=True)
    o = oracle.select(dict(snap, **routes), cache, req, k=k, pairs=True, n_threads=8)
    check_pairs(g["j"], g["feas"], g["cost"], o)
    check_topk(g["idx"], g["score"], o["idx"], o["cost"], o["feasible"])
    g_route = sel.routes_of(g["rd"], g["idx_dev"], k)
    sel.sync_errors()
    o_route = _check_routes(g_route, g["idx"], snap, routes, cache, req, k)
    # both routes are taken by some selections, and staged ones really are cheaper
    assert (o_route == 1).sum() > 0.02 * o_route.size and (o_route == 0).sum() > 0.02 * o_route.size
    base = oracle.select(snap, cache, req, k=k, pairs=True, n_threads=8)
    assert (o["cost"] <= base["cost"]).all() and (o["cost"] < base["cost"]).any()
    # the top-k only path agrees with the per-pair path bit for bit
    g2 = _select(nk, sel, req, k, pairs=False)
    np.testing.assert_array_equal(g2["idx"], g["idx"])
    np.testing.assert_array_equal(g2["score"].view(np.uint32), g["score"].view(np.uint32))
    sel.close()


@pytest.mark.parametrize("policy", [1, 2])
def test_two_hop_policy_rungs_apply_to_both_hops(nk, policy):
    _say("two-hop policy", policy)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=2000)
    snap, req, cache, routes = _inputs(cfg, 53)
    sel = _selector(nk, snap, cache, routes)
    sel.set_policy(policy)
    g = _select(nk, sel, req, 2, pairs=True)
    osnap = dict(snap, **routes)
    for key in ("util", "route_util1", "route_util2"):
        osnap[key] = np.zeros_like(osnap[key])
    if policy == 2:
        osnap["n_inflight"] = np.zeros_like(snap["n_inflight"])
    o = oracle.select(osnap, cache, req, k=2, pairs=True, n_threads=8)
    check_pairs(g["j"], g["feas"], g["cost"], o)
    check_topk(g["idx"], g["score"], o["idx"], o["cost"], o["feasible"])
    sel.close()


def test_two_hop_clear_and_reshape_restore_direct_routes(nk):
    _say("two-hop clear")
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=1500)
    snap, req, cache, routes = _inputs(cfg, 55)
    plain = nk.Selector(0)
    plain.load_snapshot(snap)
    plain.load_cache(cache, 0.5)
    ref = _select(nk, plain, req, 3, pairs=True)
    sel = _selector(nk, snap, cache, routes)
    two = _select(nk, sel, req, 3, pairs=True)
    assert (two["cost"] != ref["cost"]).any()
    sel.clear_routes()
    back = _select(nk, sel, req, 3, pairs=True)
    for key in ("idx", "score", "j", "feas", "cost"):
        np.testing.assert_array_equal(back[key].view(np.uint8), ref[key].view(np.uint8))
    with pytest.raises(nk.NetKVError) as e:
        sel.routes_of(back["rd"], back["idx_dev"], 3)
    assert e.value.status == -2   # no route maps
    # a snapshot of the same shape keeps the maps; one of another shape drops them
    sel.load_routes(routes["route_tier1"], routes["route_util1"], routes["route_tier2"],
                    routes["route_util2"])
    sel.load_snapshot(snap)
    again = _select(nk, sel, req, 3, pairs=True)
    np.testing.assert_array_equal(again["cost"].view(np.uint32), two["cost"].view(np.uint32))
    P, D = snap["n_prefill"], snap["n_decode"]
    s2 = dict(snap, n_prefill=P - 1,
              tier_map=snap["tier_map"].reshape(P, D)[:-1].reshape(-1).copy(),
              util=snap["util"].reshape(P, D)[:-1].reshape(-1).copy(),
              n_inflight=snap["n_inflight"].reshape(4, P)[:, :-1].reshape(-1).copy())
    sel.load_snapshot(s2)   # one prefill instance fewer: the route maps no longer fit
    sel.load_snapshot(snap)
    back2 = _select(nk, sel, req, 3, pairs=True)
    np.testing.assert_array_equal(back2["cost"].view(np.uint32), ref["cost"].view(np.uint32))
    sel.close()
    plain.close()


def test_two_hop_contract_errors(nk):
    _say("two-hop contract errors")
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=500)
    snap, req, cache, routes = _inputs(cfg, 57)
    sel = nk.Selector(0)
    t1, u1, t2, u2 = (routes[k] for k in ("route_tier1", "route_util1", "route_tier2", "route_util2"))
    with pytest.raises(nk.NetKVError) as e:
        sel.load_routes(t1, u1, t2, u2)
    assert e.value.status == -2   # no snapshot
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    ref = _select(nk, sel, req, 2, pairs=True)
    for bad in ("tier1", "tier2", "util1", "util1_nan", "util2", "util2_neg"):
        a, b, c, d = t1.copy(), u1.copy(), t2.copy(), u2.copy()
        if bad == "tier1":
            a[7] = 4
        elif bad == "tier2":
            c[-1] = 9
        elif bad == "util1":
            b[3] = 1.0
        elif bad == "util1_nan":
            b[0] = np.nan
        elif bad == "util2":
            d[11] = 1.5
        else:
            d[2] = -0.5
        with pytest.raises(nk.NetKVError) as e:
            sel.load_routes(a, b, c, d)
        assert e.value.status == -1, bad
    # nothing was loaded: still the direct routes
    g = _select(nk, sel, req, 2, pairs=True)
    np.testing.assert_array_equal(g["cost"].view(np.uint32), ref["cost"].view(np.uint32))
    sel.load_routes(t1, u1, t2, u2)
    g = _select(nk, sel, req, 2, pairs=False)
    n = len(req["prefill"])
    idx9 = torch.full((n * 9,), -1, dtype=torch.int32, device=sel.device)
    out9 = torch.full((n * 9,), 5, dtype=torch.int8, device=sel.device)
    for kk in (0, 9):
        with pytest.raises(nk.NetKVError) as e:
            nk.netkv_route2_of(sel.h, g["rd"], kk, idx9, out9, sel.device)
        assert e.value.status == -1
    torch.cuda.synchronize()
    assert (out9 == 5).all()
    sel.close()


@pytest.mark.timeout(900)
def test_two_hop_full_size_sampled(nk):
    """The 3,072-decode workload in the launch configuration the benchmark
    times (k = 1, no per-pair outputs), with staged routes loaded, checked
    on a seeded sample of requests against the oracle."""
    cfg = W.CONFIGS["c2"]
    seed = 0
    snap, req, cache, routes = _inputs(cfg, seed, inflight="zero")
    _say("two-hop c2 full: inputs ready")
    sel = _selector(nk, snap, cache, routes)
    g = _select(nk, sel, req, 1, pairs=False)
    g_route = sel.routes_of(g["rd"], g["idx_dev"], 1)
    sel.sync_errors()
    _say("two-hop c2 full: selected")
    rows = np.sort(np.random.default_rng(101).choice(cfg.n_requests, 384, replace=False))
    sub = subset_requests(req, rows)
    ocache = oracle.Cache(cache, n_threads=16)
    del cache
    o = oracle.select(dict(snap, **routes), ocache, sub, k=1, pairs=True, n_threads=16)
    _say("two-hop c2 full: oracle sample done")
    n, near = check_topk(g["idx"][rows], g["score"][rows], o["idx"], o["cost"], o["feasible"])
    assert near <= max(2, n // 100)
    o_route = _check_routes(g_route.reshape(-1, 1)[rows], g["idx"][rows], snap, routes, ocache, sub, 1)
    assert 0 < (o_route == 1).sum() < o_route.size
    sel.close()


def test_two_hop_leaves_sweep_and_sequential_direct(nk):
    """Only the batch selection takes staged routes: the ranking sweep and
    the sequential form give the same bits with and without route maps."""
    _say("two-hop: sweep and sequential unchanged")
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 2, 2), n_requests=1000)
    snap, req, cache, routes = _inputs(cfg, 59)
    plain = nk.Selector(0)
    plain.load_snapshot(snap)
    plain.load_cache(cache, 0.5)
    sel = _selector(nk, snap, cache, routes)
    scen = torch.from_numpy(np.random.default_rng(5).uniform(0, 0.9, (4, cfg.n_prefill * cfg.n_decode))
                            .astype(np.float32)).to(sel.device)
    outs = []
    for s_ in (plain, sel):
        rd = nk.requests_to_device(req, s_.device)
        sw = s_.rank_sweep(rd, scen, k=2)
        sq = s_.select_sequential(rd, cap=4)
        s_.sync_errors()
        outs.append([nk.to_numpy(sw["idx"]), nk.to_numpy(sw["score"]).view(np.uint32), nk.to_numpy(sw["flips"]),
                     nk.to_numpy(sq["idx"]), nk.to_numpy(sq["score"]).view(np.uint32)])
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
    # the batch selection itself does change
    g0 = _select(nk, plain, req, 1, pairs=True)
    g1 = _select(nk, sel, req, 1, pairs=True)
    assert (g1["cost"] < g0["cost"]).any()
    sel.close()
    plain.close()
