"""Full-size workloads on the GPU (4,096-GPU cluster: 3,072 decodes), in the
launch configuration the benchmark times, checked against the CPU oracle on a
seeded sample of requests (every decode of each sampled request), plus
per-pair outputs of the sample.  Needs an MI355X and the built library."""
import time

import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import check_pairs, check_topk, subset_requests

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


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,n_sample", [("c2", 768), ("c4", 192)])
def test_full_size_sampled(nk, name, n_sample):
    cfg = W.CONFIGS[name]
    seed = 0
    t0 = time.time()
    snap = W.make_snapshot(cfg, seed)
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    _say(name, "inputs generated in %.1fs" % (time.time() - t0))
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    ci = nk.netkv_cache_info(sel.h)
    n_res = int(cache["hashes"].size)
    assert 0 < ci["shared_hashes"] < ci["distinct_hashes"] <= n_res
    assert ci["distinct_hashes"] <= 0.85 * ci["index_slots"]
    _say(name, "holder index built: %d distinct hashes, %d shared, %d slots, %.2f GiB"
         % (ci["distinct_hashes"], ci["shared_hashes"], ci["index_slots"], ci["index_bytes"] / 2 ** 30))
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=1)
    sel.sync_errors()
    g_idx = nk.to_numpy(out["idx"]).reshape(-1, 1)
    g_sc = nk.to_numpy(out["score"]).reshape(-1, 1)
    _say(name, "full batch selected:", len(g_idx), "requests")
    # properties of every row
    assert ((g_idx >= -1) & (g_idx < cfg.n_decode)).all()
    ok = g_idx >= 0
    assert np.isfinite(g_sc[ok]).all() and (g_sc[ok] > 0).all()
    assert np.isinf(g_sc[~ok]).all()
    # sampled rows against the oracle
    rows = np.sort(np.random.default_rng(100).choice(cfg.n_requests, n_sample, replace=False))
    sub = subset_requests(req, rows)
    ocache = oracle.Cache(cache, n_threads=16)
    del cache
    o = oracle.select(snap, ocache, sub, k=1, pairs=True, n_threads=16)
    _say(name, "oracle sample done")
    n, near = check_topk(g_idx[rows], g_sc[rows], o["idx"], o["cost"], o["feasible"])
    assert near <= max(2, n // 100)
    # per-pair outputs of the sampled rows
    g = sel.select(nk.requests_to_device(sub, sel.device), k=1, pairs=True)
    sel.sync_errors()
    p = g["pairs"]
    check_pairs(nk.to_numpy(p["prefix_blocks"]), nk.to_numpy(p["feasible"]),
                nk.to_numpy(p["score"]), o)
    assert o["j"].max() > 0
    sel.close()
