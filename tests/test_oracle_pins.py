"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle (``oracle/``) against something other than
itself: values the paper prints (``tests/golden/``), the two propositions,
closed forms of the component equations computed by hand, exact rational
brute force and set-membership brute force on tiny inputs, and invariants.
The choice is such that a dropped term, a wrong sign, a wrong index or a
transposed operand in the oracle fails at least one of them.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- helpers

def tiny_snapshot(P, D, tier_map, util, *, bw=(900e9, 50e9, 25e9, 12.5e9),
                  lat=(0.0, 0.0, 0.0, 0.0), n_inflight=None, free_mem=None, queue=None,
                  batch=None, a=0.05, b=0.0, beta_max=64, alpha=1.0, m_min=0, bpt=1,
                  block_tokens=1):
    return dict(
        n_prefill=P, n_decode=D,
        tier_map=np.asarray(tier_map, dtype=np.uint8).reshape(-1),
        util=np.asarray(util, dtype=np.float32).reshape(-1),
        n_inflight=(np.zeros(4 * P, np.uint16) if n_inflight is None
                    else np.asarray(n_inflight, np.uint16).reshape(-1)),
        tier_bw=np.asarray(bw, dtype=np.float64), tier_lat=np.asarray(lat, dtype=np.float64),
        free_mem=(np.full(D, 1 << 62, np.uint64) if free_mem is None
                  else np.asarray(free_mem, np.uint64)),
        queue_depth=np.zeros(D, np.uint32) if queue is None else np.asarray(queue, np.uint32),
        batch_size=(np.full(D, beta_max, np.uint32) if batch is None
                    else np.asarray(batch, np.uint32)),
        t_iter_a=a, t_iter_b=b, beta_max=beta_max, alpha=alpha, m_min=m_min,
        kv_bytes_per_token=bpt, block_tokens=block_tokens)


def requests(rows):
    """rows: list of (prefill, len_tokens, [hashes])"""
    off = np.zeros(len(rows) + 1, np.uint64)
    off[1:] = np.cumsum([len(h) for _, _, h in rows])
    hs = np.array([x for _, _, h in rows for x in h], dtype=np.uint64)
    return dict(prefill=np.array([p for p, _, _ in rows], np.uint32),
                len_tokens=np.array([l for _, l, _ in rows], np.uint32),
                hash_off=off, hashes=hs)


def caches(sets):
    off = np.zeros(len(sets) + 1, np.uint64)
    off[1:] = np.cumsum([len(s) for s in sets])
    hs = np.array([x for s in sets for x in s], dtype=np.uint64)
    return dict(hash_off=off, hashes=hs)


# ---------------------------------------------------------------- paper values

def _worked_example(c3):
    g = _gold("worked_example.json")
    bw = (1e12, 1e12, g["tier_bw_bytes_per_s"]["2"], g["tier_bw_bytes_per_s"]["3"])
    n_inf = np.zeros(4, np.uint16)
    n_inf[2] = g["n_inflight"]["2"]
    n_inf[3] = g["n_inflight"]["3"]
    # bpt = 1e9 bytes/token with 1-token blocks: a 10-token request is 10 GB;
    # d1 holds the first 5 blocks (50 % hit), d2 the first 9 (90 % hit).
    h = list(range(101, 111))
    snap = tiny_snapshot(1, 2, [2, 3], [g["congestion"]["2"], c3], bw=bw, n_inflight=n_inf,
                         alpha=0.0, bpt=10 ** 9)
    out = oracle.select(snap, caches([h[:5], h[:9]]), requests([(0, 10, h)]), k=2, pairs=True)
    return g, snap, out


def test_worked_example_transfer_times():
    g, _, out = _worked_example(0.2)
    e = g["expected"]
    assert out["j"][0].tolist() == [5, 9]
    s_eff = np.array([10 - 5, 10 - 9]) * 1e9
    assert s_eff.tolist() == [g["s_eff_bytes"]["d1"], g["s_eff_bytes"]["d2"]]
    np.testing.assert_allclose(out["cost"][0], [e["t_transfer_d1"], e["t_transfer_d2"]], rtol=1e-7)
    np.testing.assert_allclose(s_eff / out["cost"][0], [e["b_eff_d1"], e["b_eff_d2"]], rtol=1e-7)
    assert out["idx"][0, 0] == 1  # d2 wins
    assert out["cost"][0, 0] / out["cost"][0, 1] == pytest.approx(e["ratio"], rel=1e-7)


def test_worked_example_perturbed_congestion():
    g, _, out = _worked_example(g_c3 := _gold("worked_example.json")["perturbed"]["congestion_tier3"])
    pert = g["perturbed"]
    b_eff_d2 = 1e9 / out["cost"][0, 1]
    assert round(b_eff_d2 / 1e9, pert["b_eff_d2_printed_decimals"]) == pert["b_eff_d2_printed"]
    assert out["cost"][0, 1] == pytest.approx(pert["t_transfer_d2"], rel=1e-7)
    ratio = out["cost"][0, 0] / out["cost"][0, 1]
    assert round(ratio) == pert["ratio_printed"]
    assert out["idx"][0, 0] == 1
    assert g_c3 == 0.5


def test_worked_example_with_latencies():
    g = _gold("worked_example.json")
    lat = g["latencies_s_for_full_formula"]
    h = list(range(101, 111))
    snap = tiny_snapshot(1, 2, [2, 3], [0.2, 0.2],
                         bw=(1e12, 1e12, 6.25e9, 3.125e9), lat=(0, 0, lat["2"], lat["3"]),
                         n_inflight=[0, 0, 1, 0], alpha=0.0, bpt=10 ** 9)
    out = oracle.select(snap, caches([h[:5], h[:9]]), requests([(0, 10, h)]), k=2, pairs=True)
    np.testing.assert_allclose(out["cost"][0], [2.0 + lat["2"], 0.4 + lat["3"]], rtol=1e-7)


def test_intro_transfer_time():
    g = _gold("paper_constants.json")["intro_transfer"]
    snap = tiny_snapshot(1, 1, [3], [0.0], bw=(1, 1, 1, g["link_gbps"] * 1e9 / 8), alpha=0.0,
                         bpt=10 ** 9)
    out = oracle.select(snap, caches([[7]]), requests([(0, 10, [1] * 0 + list(range(11, 21)))]),
                        k=1, pairs=True)
    assert out["cost"][0, 0] == pytest.approx(g["seconds"], rel=1e-12)


def test_kv_bytes_per_token_eq1():
    from paper_2606_03910_amd import workload as W
    g = _gold("paper_constants.json")["kv_bytes"]
    assert W.KV_LLAMA3_70B == g["aggregate_kib_per_token"] * 1024
    assert W.CONFIGS["c1"].kv_bytes_per_token == g["tp4_shard_kib_per_token"] * 1024


# ---------------------------------------------------------------- Proposition 1

def _two_candidate(rho1, rho2, c1, c3, k, q1=0, q2=0, n_blocks=20, a=0.05, bpt=1000, scale=1):
    """d0 same-rack (tier 1), d1 cross-pod (tier 3); B1 = k B3."""
    B3 = 1e6
    h = list(range(1, n_blocks + 1))
    j1, j2 = int(round(rho1 * n_blocks)), int(round(rho2 * n_blocks))
    snap = tiny_snapshot(1, 2, [1, 3], [c1, c3], bw=(1e12, k * B3, 1e12, B3),
                         queue=[64 + q1, 64 + q2], batch=[64, 64], a=a, b=0.0,
                         bpt=bpt * scale)
    out = oracle.select(snap, caches([h[:j1], h[:j2]]), requests([(0, n_blocks, h)]), k=2,
                        pairs=True)
    return snap, out


def test_prop1_numerical_example():
    g = _gold("paper_constants.json")["prop1_example"]
    snap, out = _two_candidate(g["rho1"], g["rho2"], 0.3, 0.3, g["k"], a=0.0)
    t1, t2 = out["cost"][0]
    # the cache-only choice (larger hit) is d1 = cross-pod; the oracle picks d0
    assert out["j"][0, 1] > out["j"][0, 0]
    assert out["idx"][0, 0] == 0
    assert t2 / t1 == pytest.approx(g["transfer_time_ratio"], rel=1e-6)
    lhs = 1 - g["rho1"]
    rhs = g["k"] * (1 - g["rho2"])
    assert (lhs, rhs) == (g["lhs"], g["rhs"])


@pytest.mark.parametrize("seed", range(5))
def test_prop1_inequality_decides_the_oracle(seed):
    """Proposition 1: d_same-rack beats d_cross-pod iff
    (1-rho1) < k (1-c1)/(1-c3) (1-rho2) + B1 (1-c1)/s (Tq2 - Tq1)."""
    rng = np.random.default_rng(seed)
    n = 40
    checked = 0
    for _ in range(200):
        j1, j2 = sorted(rng.integers(0, n + 1, 2))
        rho1, rho2 = j1 / n, j2 / n
        c1, c3 = np.float32(rng.uniform(0, 0.9)), np.float32(rng.uniform(0, 0.9))
        k = float(rng.choice([1, 2, 4, 8]))
        q1, q2 = (int(x) for x in rng.integers(0, 6, 2))
        a = 0.01
        snap, out = _two_candidate(rho1, rho2, c1, c3, k, q1=q1, q2=q2, n_blocks=n, a=a)
        B1 = k * 1e6
        s = snap["kv_bytes_per_token"] * n
        lhs = 1 - rho1
        rhs = k * (1 - float(c1)) / (1 - float(c3)) * (1 - rho2) + B1 * (1 - float(c1)) / s * (
            q2 * a - q1 * a)
        if abs(lhs - rhs) < 1e-9:
            continue
        assert (out["idx"][0, 0] == 0) == (lhs < rhs)
        checked += 1
    assert checked > 150


def test_prop1_regret_grows_linearly_with_context():
    """Cache-only choice regret is affine and increasing in the context length."""
    reg = []
    for scale in (1, 2, 4, 8):
        _, out = _two_candidate(0.0, 0.5, 0.2, 0.2, 4.0, n_blocks=16, scale=scale)
        c = out["cost"][0]
        reg.append(c[1] - c[0])
    reg = np.array(reg)
    assert np.all(np.diff(reg) > 0)
    np.testing.assert_allclose(reg / reg[0], [1, 2, 4, 8], rtol=1e-9)


# ---------------------------------------------------------------- Proposition 2

def test_prop2_numerical_bound():
    g = _gold("paper_constants.json")["prop2_example"]
    Bf, Bs = float(g["bw_ratio"]), 1.0
    eps = (Bf * (1 - g["c_fast"]) - Bs * (1 - g["c_slow"])) / (Bf + Bs)
    assert eps == pytest.approx(g["epsilon_bound"], abs=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_prop2_no_inversion_below_bound(seed):
    """Equal non-cached bytes, no in-flight transfers, no load term: the
    oracle's choice between a faster and a slower tier is unchanged by any
    congestion error below the bound, and the worst-case error just above it
    inverts the choice."""
    rng = np.random.default_rng(100 + seed)
    h = [5, 6, 7, 8]
    inverted = 0
    for _ in range(100):
        Bf, Bs = 1e9 * rng.uniform(1, 8), 1e9
        cf, cs = rng.uniform(0, 0.9, 2)
        if Bf * (1 - cf) <= Bs * (1 - cs):
            continue
        bound = (Bf * (1 - cf) - Bs * (1 - cs)) / (Bf + Bs)
        mk = lambda uf, us: tiny_snapshot(1, 2, [1, 3], [uf, us], bw=(1, Bf, 1, Bs),
                                          alpha=0.0, bpt=10 ** 6)
        cs_, rq = caches([[], []]), requests([(0, 4, h)])
        truth = oracle.select(mk(cf, cs), cs_, rq)["idx"][0, 0]
        assert truth == 0
        for _ in range(10):
            e = rng.uniform(0, 0.98) * bound
            uf = np.clip(cf + rng.uniform(-e, e), 0, 0.99)
            us = np.clip(cs + rng.uniform(-e, e), 0, 0.99)
            assert oracle.select(mk(uf, us), cs_, rq)["idx"][0, 0] == truth
        e = bound * 1.05
        if cf + e < 0.99 and cs - e > 0:
            inverted += oracle.select(mk(cf + e, cs - e), cs_, rq)["idx"][0, 0] == 1
    assert inverted > 10


def _two_tier_snapshot(c_fast, c_slow, ratio=4.0, n=(0, 0)):
    """One prefill, a decode on a fast tier (1) and one on a slow tier (3)
    with B_1 = ratio * B_3 (the 4:1 oversubscription of Proposition 2's
    example)."""
    nf = np.zeros(4, np.uint16)
    nf[1], nf[3] = n
    return tiny_snapshot(1, 2, [1, 3], [c_fast, c_slow], bw=(1, ratio * 1e9, 1, 1e9), n_inflight=nf)


def test_prop2_count_on_the_papers_example():
    """Sec. V-D's example: B_1 / B_3 = 4 and c* = 0.3 on both tiers give the
    bound 0.42.  An error of 0.41 on the fast tier is covered and keeps the
    order; 0.43 is beyond the bound (not covered) but, one-sided, still
    keeps it; 0.53 inverts it (4 * 0.17 < 0.7)."""
    g = _gold("paper_constants.json")["prop2_example"]
    snap = _two_tier_snapshot(g["c_fast"], g["c_slow"], ratio=g["bw_ratio"])
    c = g["c_fast"]
    scen = np.array([[c + 0.41, c], [c + 0.43, c], [c + 0.53, c], [c, c]], np.float32)
    out = oracle.tier_inversions(snap, scen)
    assert out.tolist() == [[1, 0, 0], [0, 0, 0], [0, 0, 1], [1, 0, 0]]


def test_prop2_count_worst_case_around_the_bound():
    """The proof's worst case -- the faster tier's congestion raised and the
    slower one's lowered by the same error -- on c_fast = 0.3, c_slow = 0.5
    (bound (4 * 0.7 - 0.5) / 5 = 0.46): 0.45 is covered and keeps the order,
    0.47 inverts it; with 3 transfers in flight on the fast tier (B_1 / 4 vs
    B_3: 0.7 < 0.5 fails, so the slow tier leads) the roles swap."""
    snap = _two_tier_snapshot(0.3, 0.5)
    scen = np.array([[0.3 + 0.45, 0.5 - 0.45], [0.3 + 0.47, 0.5 - 0.47]], np.float32)
    assert oracle.tier_inversions(snap, scen).tolist() == [[1, 0, 0], [0, 0, 1]]
    # B'_1 = B_1 / 4 = B_3: X_fast = 0.7 B_3 > X_slow = 0.5 B_3 still, bound (0.7 - 0.5) / 2 = 0.1
    snap_n = _two_tier_snapshot(0.3, 0.5, n=(3, 0))
    scen_n = np.array([[0.3 + 0.09, 0.5 - 0.09], [0.3 + 0.11, 0.5 - 0.11]], np.float32)
    assert oracle.tier_inversions(snap_n, scen_n).tolist() == [[1, 0, 0], [0, 0, 1]]


@pytest.mark.parametrize("seed", range(3))
def test_prop2_no_covered_pair_ever_inverts(seed):
    """Proposition 2 on random clusters: whatever the scenario, no pair the
    sufficient condition covers is inverted; noisier scenarios invert more
    pairs; a noise-free scenario inverts none and covers every ordered pair
    across tiers; pairs on one tier are never counted."""
    rng = np.random.default_rng(200 + seed)
    P, D = 3, 12
    tm = rng.integers(0, 4, (P, D))
    snap = tiny_snapshot(P, D, tm, rng.uniform(0, 0.9, (P, D)), bw=(900e9, 50e9, 25e9, 12.5e9),
                         n_inflight=rng.integers(0, 5, 4 * P))
    u = snap["util"].reshape(P, D).astype(np.float64)
    scen = [u]
    for sg in (0.05, 0.2, 0.8, 2.0):
        for _ in range(25):
            scen.append(np.minimum(u * np.exp(sg * rng.standard_normal((P, D))), 0.99))
    out = oracle.tier_inversions(snap, np.array(scen, np.float32).reshape(len(scen), -1))
    assert (out[:, 1] == 0).all()
    across = sum(int(tm[p, a] != tm[p, b]) for p in range(P) for a in range(D) for b in range(a + 1, D))
    assert out[0].tolist() == [across, 0, 0]
    by_sigma = out[1:, 2].reshape(4, 25).mean(axis=1)
    assert by_sigma[0] <= by_sigma[-1] and by_sigma[-1] > 0
    one = tiny_snapshot(1, D, np.full(D, 2), rng.uniform(0, 0.9, D))
    assert oracle.tier_inversions(one, np.array(scen, np.float32)[:, 0, :]).sum() == 0


def test_prop2_count_is_invariant_to_decode_order():
    """Counts are over unordered pairs: permuting the decodes (with their
    tiers and congestion) leaves them unchanged."""
    rng = np.random.default_rng(7)
    P, D = 2, 10
    tm = rng.integers(0, 4, (P, D))
    u = rng.uniform(0, 0.9, (P, D))
    scen = np.minimum(u[None] * np.exp(0.5 * rng.standard_normal((6, P, D))), 0.99)
    a = oracle.tier_inversions(tiny_snapshot(P, D, tm, u), scen.reshape(6, -1).astype(np.float32))
    perm = rng.permutation(D)
    b = oracle.tier_inversions(tiny_snapshot(P, D, tm[:, perm], u[:, perm]),
                               scen[:, :, perm].reshape(6, -1).astype(np.float32))
    assert np.array_equal(a, b) and a[:, 2].sum() > 0


# ---------------------------------------------------------------- tiers

def test_tier_ordering_at_equal_load():
    """Same hit, congestion, in-flight count and load: cost strictly grows
    with the tier (same node < same leaf < same pod < cross pod), whatever
    position each tier's decode has in the pool."""
    from paper_2606_03910_amd import workload as W
    cfg = W.CONFIGS["c0"]
    h = list(range(1, 9))
    for perm in itertools.permutations(range(4)):
        snap = tiny_snapshot(1, 4, list(perm), [0.3] * 4, bw=cfg.tier_bw, lat=cfg.tier_lat,
                             bpt=cfg.kv_bytes_per_token, block_tokens=512)
        out = oracle.select(snap, caches([h[:3]] * 4), requests([(0, 8 * 512 + 17, h)]), k=4,
                            pairs=True)
        cost_by_tier = [out["cost"][0, perm.index(t)] for t in range(4)]
        assert all(x < y for x, y in zip(cost_by_tier, cost_by_tier[1:]))
        assert out["idx"][0].tolist() == [perm.index(t) for t in range(4)]


def test_inflight_counter_is_tier_major_per_prefill():
    """n_inflight is indexed [tier][prefill]: only (p=1, tier 2) is derated."""
    P, D = 2, 4
    tmap = np.array([[0, 1, 2, 3], [0, 1, 2, 3]], np.uint8)
    n = np.zeros((4, P), np.uint16)
    n[2, 1] = 3
    bw = (8e9, 4e9, 2e9, 1e9)
    snap = tiny_snapshot(P, D, tmap, np.full(P * D, 0.5), bw=bw, n_inflight=n, alpha=0.0,
                         bpt=10 ** 6)
    rq = requests([(0, 4, [1, 2, 3, 4]), (1, 4, [1, 2, 3, 4])])
    out = oracle.select(snap, caches([[]] * 4), rq, k=1, pairs=True)
    s = 4e6
    want0 = [s / (b * 0.5) for b in bw]
    want1 = list(want0)
    want1[2] = s / (bw[2] * 0.5 / 4)
    np.testing.assert_allclose(out["cost"][0], want0, rtol=1e-12)
    np.testing.assert_allclose(out["cost"][1], want1, rtol=1e-12)


# ---------------------------------------------------------------- load terms

def test_queue_and_decode_terms_closed_form():
    """t_iter(beta) = a + b beta with a = 0.03, b = 0.001, beta_max = 64:
    q = 10, beta = 60 -> 6 blocked, T_queue = 6 * 0.09 = 0.54,
    T_decode = t_iter(61) = 0.091; q = 3, beta = 60 -> nothing blocked."""
    h = [1, 2]
    snap = tiny_snapshot(1, 3, [0, 0, 0], [0, 0, 0], queue=[10, 3, 0], batch=[60, 60, 64],
                         a=0.03, b=0.001, beta_max=64, bpt=1)
    rq = requests([(0, 2, h)])  # fully cached below: no transfer bytes
    out = oracle.select(snap, caches([h, h, h]), rq, k=3, pairs=True)
    np.testing.assert_allclose(out["cost"][0], [0.631, 0.091, 0.095], rtol=1e-12, atol=1e-15)
    snap["alpha"] = 2.0
    out = oracle.select(snap, caches([h, h, h]), rq, k=3, pairs=True)
    np.testing.assert_allclose(out["cost"][0], [1.262, 0.182, 0.19], rtol=1e-12)


def test_alpha_zero_is_pure_network_cost():
    h = list(range(1, 11))
    snap = tiny_snapshot(1, 2, [2, 2], [0.1, 0.1], queue=[1000, 0], alpha=0.0, bpt=10 ** 6)
    out = oracle.select(snap, caches([h[:8], h[:2]]), requests([(0, 10, h)]), k=1, pairs=True)
    assert out["idx"][0, 0] == 0
    snap["alpha"] = 1.0
    out = oracle.select(snap, caches([h[:8], h[:2]]), requests([(0, 10, h)]), k=1)
    assert out["idx"][0, 0] == 1


def test_equal_tiers_rank_by_cache_then_load():
    """Equal bandwidth and latency on every tier and no congestion: the
    network term only sees the non-cached bytes, so the largest hit wins and
    equal hits fall back to the load term (the cache+load ordering)."""
    h = list(range(1, 11))
    snap = tiny_snapshot(1, 4, [0, 1, 2, 3], [0, 0, 0, 0], bw=(1e9,) * 4, lat=(1e-6,) * 4,
                         queue=[66, 65, 66, 64], batch=[64] * 4, bpt=10 ** 9)
    sets = [h[:3], h[:7], h[:7], h[:1]]
    out = oracle.select(snap, caches(sets), requests([(0, 10, h)]), k=4, pairs=True)
    assert out["idx"][0].tolist() == [1, 2, 0, 3]


# ---------------------------------------------------------------- feasibility

def test_feasibility_boundary_and_rejection():
    """m_d >= s_eff + m_min, exactly at the boundary; no feasible -> -1, +inf."""
    h = [1, 2, 3, 4]
    bpt, m_min = 1000, 500
    s_eff = bpt * (4 - 1)  # one cached block
    snap = tiny_snapshot(1, 3, [0, 0, 0], [0, 0, 0],
                         free_mem=[s_eff + m_min, s_eff + m_min - 1, 2 ** 64 - 1],
                         m_min=m_min, bpt=bpt)
    out = oracle.select(snap, caches([h[:1]] * 3), requests([(0, 4, h)]), k=3, pairs=True)
    assert out["feasible"][0].tolist() == [1, 0, 1]
    assert out["idx"][0].tolist() == [0, 2, -1]
    assert np.isinf(out["score"][0, 2])
    snap["m_min"] = 2 ** 63
    out = oracle.select(snap, caches([h[:1]] * 3), requests([(0, 4, h)]), k=2, pairs=True)
    assert out["feasible"][0].tolist() == [0, 0, 1]
    snap["free_mem"] = np.array([5, 6, 7], np.uint64)
    out = oracle.select(snap, caches([h[:1]] * 3), requests([(0, 4, h)]), k=2, pairs=True)
    assert out["idx"][0].tolist() == [-1, -1] and np.all(np.isinf(out["score"][0]))


def test_full_hit_has_no_transfer_bytes_but_a_partial_block_does():
    """n_r = floor(l_r / B_tok): the trailing partial block is never cached."""
    h = [9, 8]
    snap = tiny_snapshot(1, 1, [0], [0], bw=(1e3,) * 4, alpha=0.0, bpt=1, block_tokens=16)
    out = oracle.select(snap, caches([h]), requests([(0, 32, h), (0, 40, h)]), k=1, pairs=True)
    assert out["j"][:, 0].tolist() == [2, 2]
    np.testing.assert_allclose(out["cost"][:, 0], [0.0, 8 / 1e3])


def test_runs_longer_than_16_bits():
    """Sec. III-B bounds no run: with one-token blocks a 70,000-block request
    fully resident on decode 0 has j = 70,000 and no transfer bytes there,
    and 70,000 - 100 non-cached tokens on decode 1, which holds its first 100
    blocks; the sweep, which reuses j, agrees with the selection."""
    h = list(range(1, 70001))
    snap = tiny_snapshot(1, 2, [0, 0], [0, 0], bw=(1e3,) * 4, alpha=0.0, bpt=1, block_tokens=1)
    cache = caches([h, h[:100]])
    out = oracle.select(snap, cache, requests([(0, 70000, h)]), k=2, pairs=True)
    assert out["j"][0].tolist() == [70000, 100]
    np.testing.assert_allclose(out["cost"][0], [0.0, 69900 / 1e3])
    assert out["idx"][0].tolist() == [0, 1]
    sw = oracle.rank_sweep(snap, cache, requests([(0, 70000, h)]), np.zeros((1, 2), np.float32), k=2)
    assert sw["idx"][0, 0].tolist() == [0, 1]
    np.testing.assert_allclose(sw["score"][0, 0], [0.0, 69900 / 1e3])


# ---------------------------------------------------------------- prefix match

def _brute_lcp(hs, kset):
    j = 0
    while j < len(hs) and hs[j] in kset:
        j += 1
    return j


@pytest.mark.parametrize("seed", range(4))
def test_prefix_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    universe = rng.integers(1, 2 ** 63, 60).astype(np.uint64)
    D = 7
    sets = []
    for d in range(D):
        if d % 2 == 0:   # prefix-closed sets: leading segment of the run
            sets.append(list(universe[: rng.integers(0, 30)]))
        else:            # arbitrary subsets: holes stop the scan
            sets.append(list(universe[rng.random(60) < 0.7]))
    rows = []
    for _ in range(25):
        n = int(rng.integers(0, 20))
        start = 0 if rng.random() < 0.7 else int(rng.integers(0, 5))
        hs = list(universe[start:start + n])
        rows.append((0, n * 3 + int(rng.integers(0, 3)), hs))
    snap = tiny_snapshot(1, D, [0] * D, [0] * D, block_tokens=3)
    out = oracle.select(snap, caches(sets), requests(rows), k=1, pairs=True)
    tests = 0
    for r, (_, _, hs) in enumerate(rows):
        for d in range(D):
            j = _brute_lcp(hs, set(sets[d]))
            assert out["j"][r, d] == j
            if d % 2 == 0 and hs and hs[0] == universe[0]:
                # a prefix-closed set covering the run's start: j = overlap depth
                assert j == min(len(hs), len(sets[d]))
            tests += min(j + 1, len(hs))
    assert out["tests"] == tests


def test_prefix_match_first_miss_not_longest_run():
    h = [11, 12, 13, 14, 15]
    c = oracle.Cache(caches([[12, 13, 14, 15], [11, 13, 14, 15], [11, 12, 13, 14, 15]]))
    assert [c.prefix_len(d, h) for d in range(3)] == [0, 1, 5]


def test_prefix_match_monotone_in_resident_set():
    rng = np.random.default_rng(7)
    h = list(range(1, 30))
    base = set(rng.choice(h, 15, replace=False).tolist())
    grown = base | set(rng.choice(h, 10, replace=False).tolist())
    c = oracle.Cache(caches([sorted(base), sorted(grown)]))
    for start in range(10):
        run = h[start:]
        assert c.prefix_len(0, run) <= c.prefix_len(1, run)


# ---------------------------------------------------------------- exact brute force

def _exact_costs(snap, sets, rows):
    """Eq. (5) over every decode in exact rational arithmetic."""
    D, P = snap["n_decode"], snap["n_prefill"]
    res = []
    for p, l, hs in rows:
        costs = []
        for d in range(D):
            j = _brute_lcp(hs, set(sets[d]))
            s_eff = snap["kv_bytes_per_token"] * (l - snap["block_tokens"] * j)
            feas = int(snap["free_mem"][d]) >= s_eff + snap["m_min"]
            tau = int(snap["tier_map"][p * D + d])
            c = Fraction(float(snap["util"][p * D + d]))
            n = int(snap["n_inflight"][tau * P + p])
            beff = Fraction(float(snap["tier_bw"][tau])) * (1 - c) / (1 + n)
            tx = s_eff / beff + Fraction(float(snap["tier_lat"][tau]))
            q, beta = int(snap["queue_depth"][d]), int(snap["batch_size"][d])
            A, B = Fraction(snap["t_iter_a"]), Fraction(snap["t_iter_b"])
            tq = max(0, q - (snap["beta_max"] - beta)) * (A + B * beta)
            td = A + B * (beta + 1)
            costs.append((tx + Fraction(snap["alpha"]) * (tq + td), feas))
        res.append(costs)
    return res


@pytest.mark.parametrize("seed", range(3))
def test_exact_rational_brute_force_small_cluster(seed):
    """16-GPU two-pod cluster with four prefill and twelve decode instances."""
    from paper_2606_03910_amd import workload as W
    cl = W.Cluster(4, 2, 1, 2, prefill_every=4)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=cl, n_requests=30, cache_per_decode=64,
                   n_prefixes=12, len_median=3000.0)
    snap = W.make_snapshot(cfg, seed, inflight="random")
    snap["t_iter_b"] = 0.0007
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    D = cfg.n_decode
    assert (cfg.n_prefill, D) == (4, 12)
    sets = [cache["hashes"][cache["hash_off"][d]:cache["hash_off"][d + 1]].tolist()
            for d in range(D)]
    rows = [(int(req["prefill"][r]), int(req["len_tokens"][r]),
             req["hashes"][req["hash_off"][r]:req["hash_off"][r + 1]].tolist())
            for r in range(cfg.n_requests)]
    out = oracle.select(snap, cache, req, k=3, pairs=True)
    exact = _exact_costs(snap, sets, rows)
    for r in range(cfg.n_requests):
        feas = [d for d in range(D) if exact[r][d][1]]
        assert out["feasible"][r].tolist() == [int(exact[r][d][1]) for d in range(D)]
        for d in range(D):
            assert float(exact[r][d][0]) == pytest.approx(out["cost"][r, d], rel=1e-13)
        order = sorted(feas, key=lambda d: (exact[r][d][0], d))[:3]
        order += [-1] * (3 - len(order))
        assert out["idx"][r].tolist() == order


# ---------------------------------------------------------------- ranking sweep

def test_rank_sweep_noise_free_scenario_has_no_flips():
    from paper_2606_03910_amd import workload as W
    cfg = W.scaled(W.CONFIGS["c3"], n_requests=200, n_scenarios=4)
    snap = W.make_snapshot(cfg, 1)
    ch = W.prefix_chains(cfg, 1)
    req = W.make_requests(cfg, 1, chains=ch)
    cache = W.make_caches(cfg, 1, chains=ch)
    util = np.stack([snap["util"]] * 2)
    sw = oracle.rank_sweep(snap, cache, req, util, k=3)
    base = oracle.select(snap, cache, req, k=3)
    assert sw["flips"].tolist() == [[0, 0], [0, 0]]
    for s in range(2):
        assert (sw["idx"][s] == base["idx"]).all()
        np.testing.assert_array_equal(sw["score"][s], base["score"])


def test_rank_sweep_congested_fast_tiers_flip_to_slow_ones():
    """Saturating every tier below cross-pod moves selections across tiers."""
    from paper_2606_03910_amd import workload as W
    cfg = W.scaled(W.CONFIGS["c0"], cluster=W.Cluster(8, 2, 1, 2), n_requests=300)
    snap = W.make_snapshot(cfg, 2)
    ch = W.prefix_chains(cfg, 2)
    req = W.make_requests(cfg, 2, chains=ch)
    cache = W.make_caches(cfg, 2, chains=ch)
    u = snap["util"].copy()
    tm = snap["tier_map"]
    u2 = np.where(tm < 3, 0.99, 0.0).astype(np.float32)
    sw = oracle.rank_sweep(snap, cache, req, np.stack([u, u2]), k=1)
    base = oracle.select(snap, cache, req, k=1)
    assert sw["flips"][0].tolist() == [0, 0]
    sel_tiers = tm.reshape(cfg.n_prefill, -1)[req["prefill"], sw["idx"][1, :, 0]]
    base_tiers = tm.reshape(cfg.n_prefill, -1)[req["prefill"], base["idx"][:, 0]]
    assert int(sw["flips"][1, 0]) == int((sel_tiers != base_tiers).sum()) > 0
    assert int(sw["flips"][1, 1]) == int((sw["idx"][1, :, 0] != base["idx"][:, 0]).sum())


# ---------------------------------------------------------------- between-batch update

def test_commit_closed_form():
    """Hand-worked between-batch update (counter cap 16, service mu = 2)."""
    cap = _gold("paper_constants.json")["counter_cap"]["value"]
    P, D = 2, 3
    tmap = np.array([[0, 1, 3], [2, 0, 1]], np.uint8)
    snap = tiny_snapshot(P, D, tmap, np.zeros(6), bpt=100, block_tokens=1)
    h = [1, 2, 3]
    cache = caches([[1], [1, 2, 3], []])
    rows = [(0, 3, h)] * 18 + [(1, 3, h), (1, 5, h), (0, 3, h)]
    sel = [2] * 18 + [0, 0, -1]
    state = dict(n_inflight=np.full(4 * P, 7, np.uint16), queue_depth=np.array([1, 5, 0], np.uint32),
                 free_mem=np.array([10 ** 6, 10 ** 6, 1000], np.uint64),
                 admitted_prev=np.array([0, 7, 11], np.uint64))
    st = oracle.commit(snap, cache, requests(rows), np.array(sel, np.int32), cap, 2, state)
    # p=0 -> d2 is tier 3 (18 selections, capped); p=1 -> d0 is tier 2 (2)
    want_n = np.zeros((4, P), np.uint16)
    want_n[3, 0] = cap
    want_n[2, 1] = 2
    assert st["n_inflight"].tolist() == want_n.reshape(-1).tolist()
    assert st["queue_depth"].tolist() == [1 + 2 - 2, max(0, 5 - 2), 18 - 2]
    # d0: two requests with j = 1: s_eff = 100*(3-1) + 100*(5-1) = 600
    # d2: 18 requests with j = 0: 18 * 300 = 5400 > 1000 -> clamps to 0
    assert st["free_mem"].tolist() == [10 ** 6 - 600 + 0, 10 ** 6 + 7, 0 + 11]
    assert st["admitted_prev"].tolist() == [600, 0, 5400]


# ---------------------------------------------------------------- sequential Algorithm 1

def test_sequential_increment_moves_the_second_request():
    """Two identical requests from one prefill instance: the first takes the
    faster same-leaf decode; its in-flight increment halves that tier's
    effective bandwidth (Eq. (4): 1 + n), so the second takes the same-pod
    decode.  Numbers: s = 1e9 B, B1 = 4e9, B2 = 3e9 B/s, no congestion:
    first 0.25 s vs 0.333 s; then 0.5 s vs 0.333 s."""
    h = [1, 2]
    snap = tiny_snapshot(1, 2, [1, 2], [0, 0], bw=(1, 4e9, 3e9, 1), alpha=0.0, bpt=5 * 10 ** 8)
    rq = requests([(0, 2, h), (0, 2, h)])
    seq = oracle.select_sequential(snap, caches([[], []]), rq, cap=16)
    assert seq["idx"].tolist() == [0, 1]
    np.testing.assert_allclose(seq["score"], [0.25, 1e9 / 3e9], rtol=1e-12)
    snapshot_sel = oracle.select(snap, caches([[], []]), rq, k=1)["idx"][:, 0]
    assert snapshot_sel.tolist() == [0, 0]
    # a cap of 0 freezes the counters: the batch reduces to snapshot semantics
    seq0 = oracle.select_sequential(snap, caches([[], []]), rq, cap=0)
    assert seq0["idx"].tolist() == [0, 0]


def test_sequential_counter_saturates_at_cap():
    """Five requests, one decode per tier 1 and 2 with B1 = 10 B2: tier 1
    stays best while 1 + n <= 10; with cap 3 the counter stops at 3, so
    every request keeps tier 1."""
    h = [1]
    snap = tiny_snapshot(1, 2, [1, 2], [0, 0], bw=(1, 10e9, 1e9, 1), alpha=0.0, bpt=10 ** 9)
    rq = requests([(0, 1, h)] * 5)
    assert oracle.select_sequential(snap, caches([[], []]), rq, cap=3)["idx"].tolist() == [0] * 5
    # without a binding cap: costs 0.1 n' for tier 1 (n' = 1 + n) vs 1.0 for tier 2
    out = oracle.select_sequential(snap, caches([[], []]), rq, cap=100)
    np.testing.assert_allclose(out["score"], [0.1, 0.2, 0.3, 0.4, 0.5], rtol=1e-12)


def test_sequential_prefill_instances_do_not_interact():
    """Interleaving the requests of two prefill instances does not change any
    selection (counters are per prefill instance)."""
    from paper_2606_03910_amd import workload as W
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=400)
    snap = W.make_snapshot(cfg, 4)
    ch = W.prefix_chains(cfg, 4)
    req = W.make_requests(cfg, 4, chains=ch)
    cache = W.make_caches(cfg, 4, chains=ch)
    from tests.parity import subset_requests
    base = oracle.select_sequential(snap, cache, req, cap=16)
    rng = np.random.default_rng(0)
    # a random interleaving that keeps each prefill instance's order
    groups = {}
    for r in range(cfg.n_requests):
        groups.setdefault(int(req["prefill"][r]), []).append(r)
    keys = list(groups)
    perm = []
    ptr = {k: 0 for k in keys}
    while len(perm) < cfg.n_requests:
        k = keys[rng.integers(len(keys))]
        if ptr[k] < len(groups[k]):
            perm.append(groups[k][ptr[k]])
            ptr[k] += 1
    perm = np.array(perm)
    inter = oracle.select_sequential(snap, cache, subset_requests(req, perm), cap=16)
    np.testing.assert_array_equal(inter["idx"], base["idx"][perm])
    np.testing.assert_array_equal(inter["score"], base["score"][perm])


def test_sequential_follow_mode_reports_costs_of_given_choices():
    h = [1, 2]
    snap = tiny_snapshot(1, 2, [1, 2], [0, 0], bw=(1, 4e9, 3e9, 1), alpha=0.0, bpt=5 * 10 ** 8)
    rq = requests([(0, 2, h), (0, 2, h)])
    # follow the other choice first: then decode 0 keeps its bandwidth
    out = oracle.select_sequential(snap, caches([[], []]), rq, cap=16, follow=np.array([1, 0], np.int32))
    np.testing.assert_allclose(out["follow_cost"], [1e9 / 3e9, 0.25], rtol=1e-12)
    assert out["idx"].tolist() == [0, 0]


def test_tier_counts_closed_form():
    tmap = np.array([[0, 1, 2, 3], [3, 2, 1, 0]], np.uint8)
    snap = tiny_snapshot(2, 4, tmap, np.zeros(8))
    rq = requests([(0, 1, [5]), (1, 1, [5]), (1, 1, [5]), (0, 1, [5]), (1, 1, [5])])
    cnt = oracle.tier_counts(snap, rq, np.array([2, 2, 3, -1, 0], np.int32))
    # p0->d2 tier 2, p1->d2 tier 1, p1->d3 tier 0, rejected, p1->d0 tier 3
    assert cnt.tolist() == [1, 1, 1, 1, 1]


# ---- predictive congestion (Sec. VIII; reading: simple exponential smoothing)

def test_smoothing_with_beta_one_takes_the_observation():
    rng = np.random.default_rng(5)
    c0 = rng.uniform(0, 0.99, 50)
    obs = rng.uniform(0, 0.99, 50).astype(np.float32)
    c1, bad = oracle.smooth(c0, obs, 1.0)
    assert bad == 0
    np.testing.assert_array_equal(c1, obs.astype(np.float64))


def test_smoothing_constant_observation_closed_form():
    """A constant observation o, k times from c0: c_k = o + (1 - beta)^k (c0 - o)."""
    rng = np.random.default_rng(6)
    c0 = rng.uniform(0, 0.99, 40)
    o = rng.uniform(0, 0.99, 40).astype(np.float32)
    for beta in (0.05, 0.3, 0.7):
        c = c0.copy()
        for k in range(1, 25):
            c, _ = oracle.smooth(c, o, beta)
            expect = o.astype(np.float64) + (1 - beta) ** k * (c0 - o.astype(np.float64))
            np.testing.assert_allclose(c, expect, rtol=0, atol=1e-14)


def test_smoothing_stays_between_forecast_and_observation_and_skips_invalid():
    rng = np.random.default_rng(7)
    c0 = rng.uniform(0, 0.99, 64)
    obs = rng.uniform(0, 0.99, 64).astype(np.float32)
    obs[[3, 9, 20, 41]] = [np.nan, 1.0, -0.25, np.inf]
    c1, bad = oracle.smooth(c0, obs, 0.4)
    assert bad == 4
    keep = np.isin(np.arange(64), [3, 9, 20, 41])
    np.testing.assert_array_equal(c1[keep], c0[keep])
    o = obs.astype(np.float64)
    lo, hi = np.minimum(c0, o), np.maximum(c0, o)
    assert ((c1[~keep] >= lo[~keep]) & (c1[~keep] <= hi[~keep])).all()
    # the step moves 40 % of the way: c1 - c0 = 0.4 (obs - c0)
    np.testing.assert_allclose((c1 - c0)[~keep], 0.4 * (o - c0)[~keep], rtol=1e-12, atol=1e-15)


# ---- two-hop routing (Sec. VIII; reading: the staged route's transfer time
# is the sum of its hops' Eq. (3) times, the pair takes the faster route)

def _routes(t1, u1, t2, u2):
    return dict(route_tier1=np.asarray(t1, np.uint8), route_util1=np.asarray(u1, np.float32),
                route_tier2=np.asarray(t2, np.uint8), route_util2=np.asarray(u2, np.float32))


def test_two_hop_hand_worked_example():
    """10 GB to move (10 tokens of 1 GB, nothing cached).  d0: direct on the
    1 GB/s tier, 10 s + 0.03 s; staged over a 10 GB/s hop at half load with
    one transfer in flight (2.5 GB/s: 4 s + 0.01 s) and a 5 GB/s hop at 20 %
    load (4 GB/s: 2.5 s + 0.02 s) = 6.53 s, so it goes staged.  d1: direct
    on the 5 GB/s tier, 2 s + 0.02 s; its staged route is d0's, slower."""
    snap = tiny_snapshot(1, 2, [3, 2], [0.0, 0.0], bw=(1e12, 1e10, 5e9, 1e9),
                         lat=(0.0, 0.01, 0.02, 0.03), n_inflight=[0, 1, 0, 0], alpha=0.0,
                         bpt=10 ** 9)
    snap.update(_routes([1, 1], [0.5, 0.5], [2, 2], [0.2, 0.2]))
    rq = requests([(0, 10, list(range(31, 41)))])
    out = oracle.select(snap, caches([[], []]), rq, k=2, pairs=True)
    assert out["idx"][0].tolist() == [1, 0]
    np.testing.assert_allclose(out["cost"][0], [6.53, 2.02], rtol=1e-7)
    np.testing.assert_allclose(out["score"][0], [2.02, 6.53], rtol=1e-7)
    assert oracle.route_of(snap, caches([[], []]), rq, out["idx"], 2).tolist() == [0, 1]


def test_two_hop_exact_tie_goes_direct():
    """Direct at 5 GB/s (2 s) against two 10 GB/s hops (1 s + 1 s): equal in
    binary floating point, so the direct route is kept."""
    snap = tiny_snapshot(1, 1, [2], [0.0], bw=(1e10, 1e10, 5e9, 1e9), alpha=0.0, bpt=10 ** 9)
    snap.update(_routes([0], [0.0], [1], [0.0]))
    rq = requests([(0, 10, list(range(31, 41)))])
    out = oracle.select(snap, caches([[]]), rq, k=1, pairs=True)
    assert out["cost"][0, 0] == 2.0
    assert oracle.route_of(snap, caches([[]]), rq, out["idx"], 1).tolist() == [0]
    # one byte per second faster on the second hop: staged, strictly cheaper
    snap["tier_bw"] = np.array([1e10, 1e10 + 1, 5e9, 1e9])
    out = oracle.select(snap, caches([[]]), rq, k=1, pairs=True)
    assert out["cost"][0, 0] < 2.0
    assert oracle.route_of(snap, caches([[]]), rq, out["idx"], 1).tolist() == [1]


def _random_cluster(seed, P=3, D=7, n_req=40):
    rng = np.random.default_rng(seed)
    snap = tiny_snapshot(P, D, rng.integers(0, 4, P * D), rng.uniform(0, 0.9, P * D),
                         lat=(2e-6, 5e-6, 1e-5, 2e-5), n_inflight=rng.integers(0, 5, 4 * P),
                         free_mem=rng.integers(0, 40, D) * 10 ** 6, alpha=0.3, bpt=10 ** 5,
                         block_tokens=4)
    pool = list(range(1000, 1040))
    sets = [sorted(rng.choice(pool, rng.integers(0, 30), replace=False).tolist()) for _ in range(D)]
    rows = []
    for _ in range(n_req):
        nb = int(rng.integers(1, 12))
        rows.append((int(rng.integers(0, P)), 4 * nb - int(rng.integers(0, 4)), pool[:nb]))
    return snap, caches(sets), requests(rows)


@pytest.mark.parametrize("seed", range(4))
def test_two_hop_never_raises_a_cost_and_keeps_feasibility(seed):
    snap, cache, rq = _random_cluster(seed)
    base = oracle.select(snap, cache, rq, k=3, pairs=True)
    rng = np.random.default_rng(100 + seed)
    n = snap["n_prefill"] * snap["n_decode"]
    snap2 = dict(snap)
    snap2.update(_routes(rng.integers(0, 4, n), rng.uniform(0, 0.9, n),
                         rng.integers(0, 4, n), rng.uniform(0, 0.9, n)))
    two = oracle.select(snap2, cache, rq, k=3, pairs=True)
    np.testing.assert_array_equal(two["j"], base["j"])
    np.testing.assert_array_equal(two["feasible"], base["feasible"])
    assert (two["cost"] <= base["cost"]).all()
    # the pair cost is the direct one wherever the chosen route is direct
    full = np.tile(np.arange(snap["n_decode"], dtype=np.int32), (rq["prefill"].size, 1))
    route = oracle.route_of(snap2, cache, rq, full, snap["n_decode"]).reshape(full.shape)
    assert set(np.unique(route).tolist()) == {0, 1}
    np.testing.assert_array_equal(two["cost"][route == 0], base["cost"][route == 0])
    assert (two["cost"][route == 1] < base["cost"][route == 1]).all()
    # rejections and the empty top-k slots have no route
    r = oracle.route_of(snap2, cache, rq, two["idx"], 3)
    np.testing.assert_array_equal(r < 0, two["idx"].reshape(-1) < 0)


def test_two_hop_staged_cost_is_additive_over_hops():
    """Doubling the bytes to move doubles both hops' serialisation terms:
    staged(2s) - staged(s) = s (1/b1 + 1/b2) while the latencies cancel; a
    staging store that replicates the direct route on both hops costs the
    direct time twice over, so it never wins."""
    P, D = 1, 4
    tmap = [0, 1, 2, 3]
    util = [0.1, 0.3, 0.5, 0.7]
    lat = (1e-3, 2e-3, 3e-3, 4e-3)
    snap = tiny_snapshot(P, D, tmap, util, lat=lat, n_inflight=[2, 0, 1, 3], alpha=0.0, bpt=10 ** 6)
    snap.update(_routes(tmap, util, tmap, util))
    sizes = [(0, 8, list(range(1, 9))), (0, 16, list(range(1, 17)))]
    out = oracle.select(snap, caches([[]] * D), requests(sizes), k=4, pairs=True)
    full = np.tile(np.arange(D, dtype=np.int32), (2, 1))
    assert (oracle.route_of(snap, caches([[]] * D), requests(sizes), full, D) == 0).all()
    # staged over two hops, the second without the prefill's in-flight count
    snap.update(_routes([1, 1, 1, 1], [0.5] * 4, [0, 0, 0, 0], [0.0] * 4))
    two = oracle.select(snap, caches([[]] * D), requests(sizes), k=4, pairs=True)
    b1 = 50e9 * 0.5 / (1 + 0)
    b2 = 900e9
    hop = lambda s: s / b1 + lat[1] + s / b2 + lat[0]
    staged = np.array([hop(8e6), hop(16e6)])
    direct = out["cost"]
    expect = np.minimum(direct, staged[:, None])
    np.testing.assert_allclose(two["cost"], expect, rtol=1e-12)
    assert two["cost"][1, 3] - two["cost"][0, 3] == pytest.approx(8e6 * (1 / b1 + 1 / b2), rel=1e-12)


def test_two_hop_leaves_sweep_and_sequential_direct():
    snap, cache, rq = _random_cluster(9)
    n = snap["n_prefill"] * snap["n_decode"]
    snap2 = dict(snap)
    snap2.update(_routes(np.ones(n), np.zeros(n), np.zeros(n), np.zeros(n)))
    scen = np.random.default_rng(3).uniform(0, 0.9, (3, n)).astype(np.float32)
    a = oracle.rank_sweep(snap, cache, rq, scen, k=2)
    b = oracle.rank_sweep(snap2, cache, rq, scen, k=2)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    s1 = oracle.select_sequential(snap, oracle.Cache(cache), rq, cap=4)
    s2 = oracle.select_sequential(snap2, oracle.Cache(cache), rq, cap=4)
    for key in s1:
        np.testing.assert_array_equal(s1[key], s2[key])


# ---------------------------------------------------------------- flow-level transfer simulation (Sec. VI-B)

def _flows(cap, paths, nbytes, start):
    off = np.zeros(len(paths) + 1, np.uint64)
    off[1:] = np.cumsum([len(p) for p in paths])
    return dict(cap=np.asarray(cap, np.float64), path_off=off,
                path=np.asarray([l for p in paths for l in p], np.uint32),
                bytes=np.asarray(nbytes, np.float64), start=np.asarray(start, np.float64))


def test_flowsim_single_flow_moves_at_its_bottleneck():
    """Sec. VI-B's first validation: one flow on an uncontested path runs at
    the bandwidth of its slowest link (here a 25 GB/s link between two of
    50 GB/s; 10 GB arriving at t = 1 s)."""
    f = _flows([50e9, 25e9, 50e9, 900e9], [[0, 1, 2]], [10e9], [1.0])
    rate, rounds = oracle.maxmin(f)
    assert rate[0] == 25e9 and rounds == 1
    fin, ev = oracle.flow_sim(f)
    assert fin[0] == 1.0 + 10e9 / 25e9 and ev == 1


def test_flowsim_n_flows_share_a_bottleneck_equally():
    """Sec. VI-B's second validation: N flows through one bottleneck each get
    1/N of it (private access links are faster); equal flows starting
    together finish together at N * bytes / capacity."""
    for n in (1, 2, 5, 16):
        cap = [10.0] + [100.0] * n
        f = _flows(cap, [[0, 1 + i] for i in range(n)], [4.0] * n, [0.0] * n)
        rate, _ = oracle.maxmin(f)
        assert np.all(rate == 10.0 / n)
        fin, ev = oracle.flow_sim(f)
        np.testing.assert_allclose(fin, n * 4.0 / 10.0, rtol=1e-15)
        assert ev == 1


def test_flowsim_reallocation_after_completion_and_arrival():
    """Sec. VI-B's third validation: when a flow completes (or arrives) the
    others' shares are re-evaluated at once.  On one link of capacity C,
    flows sharing it form a processor-sharing queue: with sizes b1 <= ... <=
    bN starting together, flow k finishes at (b1 + ... + bk + (N - k) bk) / C.
    A late arrival: flow a (2 bytes) alone at rate 2 until t = 0.5, then
    both at 1 until a finishes at 1.5, then b alone at 2 until 2.0."""
    b = np.array([1.0, 2.0, 2.0, 5.0, 9.0])
    n = len(b)
    f = _flows([3.0] + [50.0] * n, [[0, 1 + i] for i in range(n)], b, np.zeros(n))
    fin, ev = oracle.flow_sim(f)
    want = np.array([(b[:k + 1].sum() + (n - k - 1) * b[k]) / 3.0 for k in range(n)])
    np.testing.assert_allclose(fin, want, rtol=1e-14)
    assert ev == 4   # the two flows of 2 bytes finish at the same event
    f = _flows([2.0, 10.0, 10.0], [[0, 1], [0, 2]], [2.0, 2.0], [0.0, 0.5])
    fin, ev = oracle.flow_sim(f)
    np.testing.assert_allclose(fin, [1.5, 2.0], rtol=1e-15)
    assert ev == 3


def test_maxmin_parking_lot():
    """The textbook case: flow 0 crosses links 0 (capacity 1) and 1
    (capacity 2), flow 1 only link 0, flow 2 only link 1.  Link 0 fills
    first at 1/2 each; flow 2 then takes the rest of link 1: 3/2."""
    f = _flows([1.0, 2.0], [[0, 1], [0], [1]], [1.0] * 3, [0.0] * 3)
    rate, rounds = oracle.maxmin(f)
    assert rate.tolist() == [0.5, 0.5, 1.5] and rounds == 2
    fin, _ = oracle.flow_sim(f)
    # flow 2 ends at 2/3; flows 0 and 1 then share link 0 until 2
    np.testing.assert_allclose(fin, [2.0, 2.0, 2.0 / 3.0], rtol=1e-15)


@pytest.mark.parametrize("seed", range(12))
def test_maxmin_allocation_has_a_bottleneck_for_every_flow(seed):
    """Max-min fairness by its characterisation (Bertsekas & Gallager,
    Prop. 6.5.1): a feasible allocation is max-min fair iff every flow
    crosses a saturated link on which no other flow has a larger rate.
    Checked directly on random paths and capacities, with a random subset
    of flows active."""
    rng = np.random.default_rng(seed)
    L, N = int(rng.integers(3, 12)), int(rng.integers(1, 30))
    cap = rng.uniform(1.0, 10.0, L)
    paths = [sorted(rng.choice(L, int(rng.integers(1, min(L, 4) + 1)), replace=False).tolist()) for _ in range(N)]
    active = (rng.uniform(size=N) < 0.8).astype(np.uint8)
    f = _flows(cap, paths, np.ones(N), np.zeros(N))
    rate, _ = oracle.maxmin(f, active)
    assert (rate[active == 0] == 0).all()
    load = np.zeros(L)
    for i, p in enumerate(paths):
        load[p] += rate[i]
    assert (load <= cap * (1 + 1e-12)).all()
    for i, p in enumerate(paths):
        if not active[i]:
            continue
        ok = False
        for l in p:
            others = [rate[j] for j, q in enumerate(paths) if l in q and active[j]]
            if load[l] >= cap[l] * (1 - 1e-12) and rate[i] >= max(others) * (1 - 1e-12):
                ok = True
        assert ok, f"flow {i} has no bottleneck link"


@pytest.mark.parametrize("seed", range(6))
def test_flowsim_never_beats_the_path_alone_and_matches_it_without_sharing(seed):
    """A flow can never finish earlier than alone on its path; flows whose
    paths share no link with any other finish exactly as alone; and the
    link carrying every flow (a common bottleneck) is never idle while
    flows are in progress, so with all flows starting together the last
    one finishes at sum(bytes) / capacity."""
    rng = np.random.default_rng(100 + seed)
    N = 20
    L = 2 * N + 1
    cap = rng.uniform(1.0, 10.0, L)
    nbytes = rng.uniform(0.5, 5.0, N)
    start = rng.uniform(0.0, 2.0, N)
    # disjoint paths: flow i on links 2i, 2i+1
    f = _flows(cap, [[2 * i, 2 * i + 1] for i in range(N)], nbytes, start)
    fin, _ = oracle.flow_sim(f)
    alone = start + nbytes / np.minimum(cap[0:2 * N:2], cap[1:2 * N:2])
    np.testing.assert_allclose(fin, alone, rtol=1e-14)
    # one common link (index L-1), slower than every private link
    cap2 = cap.copy()
    cap2[-1] = 0.5
    f = _flows(cap2, [[2 * i, L - 1] for i in range(N)], nbytes, np.zeros(N))
    fin, _ = oracle.flow_sim(f)
    assert (fin >= nbytes / np.minimum(cap2[0:2 * N:2], 0.5) * (1 - 1e-14)).all()
    np.testing.assert_allclose(fin.max(), nbytes.sum() / 0.5, rtol=1e-12)


def test_selection_bytes_is_eq2_on_a_hand_built_case():
    """Eq. (2) for the flows the transfer simulation takes: a request of
    1,000 tokens in blocks of 100 (10 hashed blocks), whose first three
    blocks are resident on decode 0 and whose first block is missing on
    decode 1 (a later block resident there does not count: Sec. III-B's
    leading run).  With Eq. (1)'s 327,680 bytes per token: decode 0 moves
    700 tokens, decode 1 all 1,000; no selection moves nothing."""
    bpt = 327680
    snap = tiny_snapshot(1, 2, [1, 1], [0.0, 0.0], bpt=bpt, block_tokens=100)
    h = [11, 12, 13, 14, 15, 16, 17, 18, 19, 20]
    cache = caches([[11, 12, 13, 15], [12, 13]])
    req = requests([(0, 1000, h), (0, 1000, h), (0, 1000, h)])
    out = oracle.selection_bytes(snap, cache, req, np.array([0, 1, -1], np.int32), 1)
    assert out.tolist() == [700 * bpt, 1000 * bpt, 0]


# ---------------------------------------------------------------- telemetry derivations

def _two_pod_coords():
    """8 GPUs: 2 per node, 2 nodes per leaf, 1 leaf per pod, 2 pods.  Prefill
    on GPU 0; decodes on GPUs 1 (same node), 2 (same leaf), 4 and 6 (other
    pod)."""
    node = np.array([0, 0, 1, 1, 2, 2, 3, 3])
    leaf = node // 2
    pod = leaf
    pg, dg = [0], [1, 2, 4, 6]
    return (node[pg], leaf[pg], pod[pg]), (node[dg], leaf[dg], pod[dg])


def test_pair_congestion_constant_per_tier_is_the_papers_c_tau():
    """Sec. III-E gives one congestion value c_tau per tier.  With every link
    of tier tau at the same utilisation, each pair of tier tau gets exactly
    c_tau, and the tiers follow the topology (same node 0, same leaf 1,
    other pod 3)."""
    pc, dc = _two_pod_coords()
    c = [0.125, 0.25, 0.5, 0.75]
    links = {f"u{t}": np.full(4, c[t]) for t in range(4)}
    tier, util = oracle.pair_congestion(pc, dc, links)
    assert tier.tolist() == [[0, 1, 3, 3]]
    assert util.tolist() == [[0.125, 0.25, 0.75, 0.75]]


def test_pair_congestion_takes_the_busier_end():
    """With per-link values, a pair reads the tier-level links at both of its
    ends and takes the larger: node 0's fabric (0.1) against itself; NIC
    uplinks of nodes 0 and 1 (0.2, 0.6); the pod uplinks of pods 0 and 1
    (0.3, 0.05) for the cross-pod pairs."""
    pc, dc = _two_pod_coords()
    links = dict(u0=np.array([0.1, 0.9, 0.9, 0.9]), u1=np.array([0.2, 0.6, 0.0, 0.0]),
                 u2=np.array([0.7, 0.7]), u3=np.array([0.3, 0.05]))
    _, util = oracle.pair_congestion(pc, dc, links)
    np.testing.assert_array_equal(util, np.float32([[0.1, 0.6, 0.3, 0.3]]))


def test_ar1_step_closed_forms():
    """The AR(1) telemetry step: rho = 1 and sigma = 0 keep the value; sigma
    = 0 contracts the deviation from the mean by rho per step (k steps:
    mean + rho^k (u0 - mean)); rho = 0 gives mean + sigma eps; the result is
    clamped to [0, 0.99]."""
    rng = np.random.default_rng(3)
    mean = rng.uniform(0.1, 0.8, 50)
    u = rng.uniform(0.0, 0.9, 50)
    eps = rng.standard_normal(50)
    np.testing.assert_allclose(oracle.ar1_step(u, mean, eps, 1.0, 0.0), u, rtol=0, atol=2e-16)
    x = u.copy()
    for _ in range(5):
        x = oracle.ar1_step(x, mean, eps, 0.5, 0.0)
    np.testing.assert_allclose(x, mean + 0.5 ** 5 * (u - mean), rtol=0, atol=1e-15)
    np.testing.assert_allclose(oracle.ar1_step(u, mean, eps, 0.0, 0.05),
                               np.clip(mean + 0.05 * eps, 0.0, 0.99), rtol=0, atol=1e-16)
    hi = oracle.ar1_step(np.full(3, 0.98), np.full(3, 0.98), np.array([10.0, -100.0, 0.0]), 0.9, 0.05)
    assert hi.tolist() == [0.99, 0.0, 0.98]


def test_link_noise_closed_forms():
    """Lognormal telemetry noise: sigma = 0 or z = 0 leaves the utilisation
    unchanged; z = 1 multiplies by e^sigma; the result is capped at 0.99;
    the multiplier's median over many draws is 1."""
    u = np.array([0.1, 0.3, 0.5, 0.9])
    z = np.array([1.0, -2.0, 0.5, 3.0])
    np.testing.assert_array_equal(oracle.link_noise(u, z, 0.0), u)
    np.testing.assert_array_equal(oracle.link_noise(u, np.zeros(4), 0.4), u)
    np.testing.assert_allclose(oracle.link_noise(u, np.ones(4), 0.2), np.minimum(u * np.e ** 0.2, 0.99),
                               rtol=1e-15)
    assert oracle.link_noise(np.array([0.9]), np.array([3.0]), 0.4)[0] == 0.99
    zz = np.random.default_rng(4).standard_normal(20001)
    m = oracle.link_noise(np.full(zz.size, 0.001), zz, 0.4) / 0.001
    assert abs(np.median(m) - 1.0) < 0.02
