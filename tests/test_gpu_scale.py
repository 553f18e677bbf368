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


def _sentinel_select(nk, sel, req, k):
    """Top-k of every request into outputs pre-filled with a sentinel: a
    request that the batch orders lost or duplicated would keep it."""
    n = len(req["prefill"])
    out = dict(idx=torch.full((n * k,), -7, dtype=torch.int32, device=sel.device),
               score=torch.full((n * k,), -7.0, dtype=torch.float32, device=sel.device))
    sel.select(nk.requests_to_device(req, sel.device), k=k, out=out)
    sel.sync_errors()
    idx = nk.to_numpy(out["idx"]).reshape(-1, k)
    sc = nk.to_numpy(out["score"]).reshape(-1, k)
    assert not (idx == -7).any() and not (sc == -7.0).any(), "a request's result was never written"
    return idx, sc


def test_batch_sort_path_every_request(nk):
    """150,000 requests (above the 65,536 where the library's own batch
    sorts take over, 37 tiles with a ragged last one) on 48 decodes: every
    request against the oracle."""
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=150000)
    snap = W.make_snapshot(cfg, 21, inflight="random")
    ch = W.prefix_chains(cfg, 21)
    req = W.make_requests(cfg, 21, chains=ch)
    cache = W.make_caches(cfg, 21, chains=ch)
    _say("own-sort batch: 150,000 x 48")
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    idx, sc = _sentinel_select(nk, sel, req, 3)
    o = oracle.select(snap, cache, req, k=3, pairs=True, n_threads=16)
    n, near = check_topk(idx, sc, o["idx"], o["cost"], o["feasible"])
    assert n > 0.99 * 3 * cfg.n_requests and near <= max(2, n // 1000)
    sel.close()


@pytest.mark.timeout(900)
def test_two_pass_prefill_order(nk):
    """2,048 prefill instances (8,192 GPUs): the prefill key takes 12 bits,
    so the prefill order takes two sort passes; 70,000 requests over 6,144
    decodes, every result written, a seeded sample against the oracle."""
    cl = W.Cluster(8, 16, 16, 4)
    cfg = W.scaled(W.CONFIGS["c0"], cluster=cl, n_requests=70000, cache_per_decode=1024)
    assert cfg.n_prefill == 2048 and cfg.n_decode == 6144
    snap = W.make_snapshot(cfg, 23)
    ch = W.prefix_chains(cfg, 23)
    req = W.make_requests(cfg, 23, chains=ch)
    cache = W.make_caches(cfg, 23, chains=ch)
    _say("two-pass prefill order: 70,000 x 6,144")
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    idx, sc = _sentinel_select(nk, sel, req, 1)
    ok = idx[:, 0] >= 0
    assert ((idx[:, 0] >= -1) & (idx[:, 0] < cfg.n_decode)).all() and ok.mean() > 0.9
    assert np.isfinite(sc[ok]).all() and np.isinf(sc[~ok]).all()
    rows = np.sort(np.random.default_rng(102).choice(cfg.n_requests, 256, replace=False))
    o = oracle.select(snap, cache, subset_requests(req, rows), k=1, pairs=True, n_threads=16)
    n, near = check_topk(idx[rows], sc[rows], o["idx"], o["cost"], o["feasible"])
    assert near <= 2
    sel.close()
