"""Full-size workloads on the GPU (4,096-GPU cluster: 3,072 decodes), in the
launch configuration the benchmark times: every request against the exact
argmin of the GPU's own per-pair scores, a seeded slice of requests against
the CPU oracle (selections and per-pair outputs), leader-table overflow, and
the library's own batch sorts.  Needs an MI355X and the built library."""
import time

import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W
from tests.parity import check_pairs, check_topk, classify, slice_requests, subset_requests

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


def _self_argmin_torch(score, feas, D):
    """Exact top-1 by (fp32 score bits, index) over the feasible pairs of
    per-pair outputs [n*D] on the device: (idx int64 [n], score bits [n]);
    -1 / +inf bits where nothing is feasible."""
    n = score.numel() // D
    bits = score.view(torch.int32).to(torch.int64).view(n, D)
    key = (bits << 32) | torch.arange(D, device=score.device, dtype=torch.int64)[None, :]
    big = torch.iinfo(torch.int64).max
    key = torch.where(feas.view(n, D) != 0, key, torch.full_like(key, big))
    m = key.min(dim=1).values
    idx = torch.where(m == big, torch.full_like(m, -1), m & 0xFFFFFFFF)
    sb = torch.where(m == big, torch.full_like(m, 0x7F800000), m >> 32)
    return idx, sb


@pytest.mark.timeout(1500)
@pytest.mark.parametrize("name,n_slice", [("c2", 65536), ("c4", 4096)])
def test_full_size(nk, name, n_slice):
    """The whole batch in the benchmark's launch configuration (k = 1,
    throughput mode), then:
      * every request: its selection equals the exact lowest-index argmin of
        the GPU's own per-pair scores over its feasible decodes (per-pair
        outputs taken in chunks of 65,536 requests), score bits included;
      * a seeded contiguous slice of n_slice requests x every decode against
        the CPU oracle: the selections (near-tie rule, no exact tie broken
        away from the lowest index) and the per-pair prefix lengths,
        feasibility and scores;
      * a leader table far smaller than the batch's leaders (the requests
        after the leaders that do not fit are matched on their own): every
        selection and score bit-identical."""
    cfg = W.CONFIGS[name]
    seed = 0
    D = cfg.n_decode
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
    ok = g_idx >= 0
    assert ((g_idx >= -1) & (g_idx < D)).all()
    assert np.isfinite(g_sc[ok]).all() and (g_sc[ok] > 0).all()
    assert np.isinf(g_sc[~ok]).all()
    # the oracle slice: a seeded contiguous range inside a seeded chunk
    chunk = 65536
    R = cfg.n_requests
    rng = np.random.default_rng(100)
    c_star = int(rng.integers(0, R // chunk))
    s0 = c_star * chunk + int(rng.integers(0, chunk - n_slice + 1))
    s1 = s0 + n_slice
    g_full_idx = out["idx"].to(torch.int64)
    g_full_bits = out["score"].view(torch.int32).to(torch.int64)
    slice_pairs = None
    for r0 in range(0, R, chunk):
        r1 = min(R, r0 + chunk)
        sub = slice_requests(req, r0, r1)
        g = sel.select(nk.requests_to_device(sub, sel.device), k=1, pairs=True)
        sel.sync_errors()
        p = g["pairs"]
        ei, eb = _self_argmin_torch(p["score"], p["feasible"], D)
        bad_i = int((ei != g_full_idx[r0:r1]).sum().item())
        bad_b = int((eb != g_full_bits[r0:r1]).sum().item())
        assert bad_i == 0 and bad_b == 0, (
            f"requests {r0}..{r1}: {bad_i} selections / {bad_b} scores differ from the lowest-index "
            f"argmin of the per-pair scores")
        assert torch.equal(g["idx"], out["idx"][r0:r1]), "chunked selection differs from the full batch"
        if r0 <= s0 < r1:
            a, b = s0 - r0, s1 - r0
            slice_pairs = dict(j=nk.to_numpy(p["prefix_blocks"][a * D:b * D]),
                               feas=nk.to_numpy(p["feasible"][a * D:b * D]),
                               cost=nk.to_numpy(p["score"][a * D:b * D]))
        del g, p, ei, eb
    _say(name, "every request equals the lowest-index argmin of its per-pair scores")
    # the oracle on the slice
    t0 = time.time()
    ocache = oracle.Cache(cache, n_threads=16)
    del cache
    o = oracle.select(snap, ocache, slice_requests(req, s0, s1), k=1, pairs=True, n_threads=16)
    _say(name, "oracle slice [%d, %d) x %d decodes in %.1fs" % (s0, s1, D, time.time() - t0))
    c = classify(g_idx[s0:s1], o["idx"], o["cost"], g_cost=slice_pairs["cost"].reshape(n_slice, D))
    _say(name, "slice selections:", {k: v for k, v in c.items() if k != "bad_mask"})
    check_topk(g_idx[s0:s1], g_sc[s0:s1], o["idx"], o["cost"], o["feasible"],
               g_cost=slice_pairs["cost"].reshape(n_slice, D))
    err = check_pairs(slice_pairs["j"], slice_pairs["feas"], slice_pairs["cost"], o)
    assert o["j"].max() > 0
    _say(name, "slice pairs bit-exact (j, mask), max score rel err %.2e" % err)
    del o, slice_pairs
    # leader-table overflow on the whole batch
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, 256)
    cap = sel.select(rd, k=1)
    sel.sync_errors()
    nk.netkv_set_option(sel.h, nk.NETKV_OPT_LEAD_CAP, 0)
    assert torch.equal(cap["idx"], out["idx"])
    assert torch.equal(cap["score"].view(torch.int32), out["score"].view(torch.int32))
    _say(name, "leader table of 256: every selection and score bit-identical")
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


@pytest.mark.parametrize("n_req", [150000, 530000])
def test_batch_sort_path_every_request(nk, n_req):
    """Batches above the 65,536 where the library's own batch sorts take
    over, on 48 decodes, every request against the oracle: 150,000 requests
    (147 tiles of 1,024, the last ragged) and 530,000 (just above the 2^19
    where the sorts switch to tiles of 4,096: 130 tiles, the last ragged)."""
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=n_req)
    snap = W.make_snapshot(cfg, 21, inflight="random")
    ch = W.prefix_chains(cfg, 21)
    req = W.make_requests(cfg, 21, chains=ch)
    cache = W.make_caches(cfg, 21, chains=ch)
    _say(f"own-sort batch: {n_req:,} x 48")
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
