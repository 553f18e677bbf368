"""Generator checks: topology, telemetry collapse, request and cache structure.

The tier rule is re-derived here from GPU ids with plain loops, independently
of the generator's vectorised code.
"""
import numpy as np
import pytest

from paper_2606_03910_amd import workload as W


def _tier_loop(cl, g1, g2):
    n1, n2 = g1 // cl.gpus_per_node, g2 // cl.gpus_per_node
    if n1 == n2:
        return 0
    l1, l2 = n1 // cl.nodes_per_leaf, n2 // cl.nodes_per_leaf
    if l1 == l2:
        return 1
    if l1 // cl.leaves_per_pod == l2 // cl.leaves_per_pod:
        return 2
    return 3


@pytest.mark.parametrize("name", ["c0", "c2"])
def test_tier_map_matches_topology(name):
    cfg = W.CONFIGS[name]
    cl = cfg.cluster
    t = W.pair_tiers(cl)
    pg, dg = cl.prefill_gpus(), cl.decode_gpus()
    rng = np.random.default_rng(0)
    for _ in range(2000):
        p, d = rng.integers(len(pg)), rng.integers(len(dg))
        assert t[p, d] == _tier_loop(cl, pg[p], dg[d])
    assert (cfg.n_prefill, cfg.n_decode) == ((16, 48) if name == "c0" else (1024, 3072))


def test_cluster_shapes():
    c2 = W.CONFIGS["c2"].cluster
    assert (c2.n_gpus, c2.n_nodes, c2.n_leaves, c2.pods) == (4096, 512, 64, 8)
    c0 = W.CONFIGS["c0"].cluster
    assert (c0.n_gpus, c0.n_nodes, c0.n_leaves, c0.pods) == (64, 8, 2, 1)


def test_constant_link_util_gives_per_tier_congestion():
    cl = W.CONFIGS["c0"].cluster
    cl2 = W.Cluster(8, 2, 2, 2)
    for c in (cl, cl2):
        links = dict(u0=np.full(c.n_nodes, 0.1), u1=np.full(c.n_nodes, 0.2),
                     u2=np.full(c.n_leaves, 0.3), u3=np.full(c.pods, 0.4))
        u = W.pair_util(c, links)
        t = W.pair_tiers(c)
        np.testing.assert_array_equal(u, np.array([0.1, 0.2, 0.3, 0.4], np.float32)[t])


def test_requests_structure_and_determinism():
    cfg = W.CONFIGS["c0"]
    a = W.make_requests(cfg, 0)
    b = W.make_requests(cfg, 0)
    for k in ("prefill", "len_tokens", "hash_off", "hashes"):
        np.testing.assert_array_equal(a[k], b[k])
    n = np.diff(a["hash_off"].astype(np.int64))
    np.testing.assert_array_equal(n, a["len_tokens"] // cfg.block_tokens)
    assert (a["hashes"] != 0).all()
    assert a["len_tokens"].min() >= 128 and a["len_tokens"].max() <= 131072
    assert (a["prefill"] < cfg.n_prefill).all()
    c = W.make_requests(cfg, 1)
    assert not np.array_equal(a["hashes"][:100], c["hashes"][:100])


def test_caches_unique_per_decode_and_sized():
    cfg = W.scaled(W.CONFIGS["c0"], cache_per_decode=1000)
    c = W.make_caches(cfg, 0)
    off = c["hash_off"].astype(np.int64)
    assert (np.diff(off) == 1000).all()
    for d in range(cfg.n_decode):
        h = c["hashes"][off[d]:off[d + 1]]
        assert len(np.unique(h)) == len(h)
        assert (h != 0).all()


def test_long_context_shape():
    cfg = W.scaled(W.CONFIGS["c4"], n_requests=2000, cache_per_decode=4096,
                   cluster=W.CONFIGS["c0"].cluster)
    r = W.make_requests(cfg, 0)
    n = np.diff(r["hash_off"].astype(np.int64))
    assert n.min() >= 128 and n.max() <= 256
    share = (r["shared_blocks"] > 0).mean()
    assert 0.75 < share < 0.85


def test_scenarios_noise_free_limit_and_cap():
    cfg = W.scaled(W.CONFIGS["c3"], n_scenarios=8)
    links = W.draw_links(cfg, 0)
    u, sig = W.scenario_utils(cfg, 0, links, n_scen=8, sigmas=(0.0, 5.0))
    base = W.pair_util(cfg.cluster, links).reshape(-1)
    np.testing.assert_array_equal(u[0], base)
    assert u.max() <= np.float32(0.99)
    assert list(sig) == [0.0] * 4 + [5.0] * 4


def test_ar1_stays_in_range_and_starts_at_draw():
    cfg = W.CONFIGS["c1"]
    links = W.draw_links(cfg, 0)
    seq = W.ar1_links(cfg, 0, links, 16)
    assert len(seq) == 16
    np.testing.assert_array_equal(seq[0]["u2"], links["u2"])
    for s in seq:
        for v in s.values():
            assert v.min() >= 0 and v.max() <= 0.99


def _coords(cfg):
    node, leaf, pod = cfg.cluster.coords()
    pg, dg = cfg.cluster.prefill_gpus(), cfg.cluster.decode_gpus()
    return (node[pg], leaf[pg], pod[pg]), (node[dg], leaf[dg], pod[dg])


@pytest.mark.parametrize("name", ["c0", "c2"])
def test_generator_congestion_matches_the_oracles_derivation(name):
    """The snapshots' tier and congestion maps are what the oracle derives
    from the same link draws (one congestion value per pair from the
    tier-level links at both ends), bit for bit."""
    import oracle
    cfg = W.CONFIGS[name]
    links = W.draw_links(cfg, 7)
    tier, util = oracle.pair_congestion(*_coords(cfg), links)
    np.testing.assert_array_equal(tier, W.pair_tiers(cfg.cluster))
    np.testing.assert_array_equal(util, W.pair_util(cfg.cluster, links))
    snap = W.make_snapshot(cfg, 7)
    np.testing.assert_array_equal(snap["tier_map"].reshape(tier.shape), tier)


def test_generator_ar1_matches_the_oracles_step():
    """The streaming workload's per-batch link utilisations are the oracle's
    AR(1) steps from the initial draw, with the generator's normal draws
    (the same seeded stream, links in key order, batch after batch)."""
    import oracle
    cfg = W.CONFIGS["c1"]
    links0 = W.draw_links(cfg, 5)
    seq = W.ar1_links(cfg, 5, links0, 6)
    rng = W._rng(5, 51)
    cur = {k: np.asarray(v, np.float64) for k, v in links0.items()}
    for t in range(1, 6):
        nxt = {}
        for key in sorted(cur):
            eps = rng.standard_normal(len(cur[key]))
            nxt[key] = oracle.ar1_step(cur[key], links0[key], eps, cfg.ar1_rho, cfg.ar1_sigma)
            np.testing.assert_array_equal(nxt[key], seq[t][key])
        cur = nxt


def test_generator_scenarios_match_the_oracles_noise():
    """The ranking sweep's scenarios are the oracle's lognormal noise on every
    link (the generator's normal draws), collapsed to pairs as in the
    snapshot; equal to within one fp32 ulp (the two sides' exp may round
    differently in the last bit)."""
    import oracle
    cfg = W.CONFIGS["c3"]
    links = W.draw_links(cfg, 9)
    S = 16
    util, sig = W.scenario_utils(cfg, 9, links, n_scen=S)
    rng = W._rng(9, 61)
    pc, dc = _coords(cfg)
    for s in range(S):
        noisy = {}
        for key in sorted(links):
            z = rng.standard_normal(len(links[key]))
            noisy[key] = oracle.link_noise(links[key], z, sig[s])
        _, u = oracle.pair_congestion(pc, dc, noisy)
        a = u.reshape(-1).view(np.int32).astype(np.int64)
        b = util[s].view(np.int32).astype(np.int64)
        assert np.abs(a - b).max() <= 1
