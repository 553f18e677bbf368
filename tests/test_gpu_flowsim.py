"""The flow-level transfer simulation (Sec. VI-B's network model) and the
selections' transfer sizes (Eq. (2)) on the GPU, against the CPU oracle.
Finish times and allocation counts must be bit-identical: both sides run
the same fp64 operations in the same order.  Needs an MI355X and the built
library."""
import numpy as np
import pytest

import oracle
from paper_2606_03910_amd import workload as W

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


def _instances(insts):
    """Concatenate instances (each dict(cap, path_off, path, bytes, start)
    on the same number of links) into the call's arrays."""
    L = len(insts[0]["cap"])
    assert all(len(x["cap"]) == L for x in insts)
    flow_off = np.zeros(len(insts) + 1, np.uint64)
    flow_off[1:] = np.cumsum([len(x["bytes"]) for x in insts])
    path_off, paths, base = [np.zeros(1, np.uint64)], [], 0
    for x in insts:
        po = np.asarray(x["path_off"], np.uint64)
        path_off.append(po[1:] + np.uint64(base))
        paths.append(np.asarray(x["path"], np.uint32))
        base += int(po[-1])
    return dict(cap=np.concatenate([np.asarray(x["cap"], np.float64) for x in insts]), flow_off=flow_off,
                path_off=np.concatenate(path_off), path=np.concatenate(paths) if paths else np.zeros(0, np.uint32),
                bytes=np.concatenate([np.asarray(x["bytes"], np.float64) for x in insts]),
                start=np.concatenate([np.asarray(x["start"], np.float64) for x in insts])), L


def _run(nk, sel, insts):
    arr, L = _instances(insts)
    dev = {k: nk.to_device(v, sel.device) for k, v in arr.items()}
    fin, st = sel.flow_sim(dev, len(insts), L)
    st = nk.to_numpy(st).reshape(-1, 3).astype(np.int64)
    return nk.to_numpy(fin), st, arr


def _check_against_oracle(insts, fin, st, arr):
    """Finish times bit for bit; allocations, filling rounds and moving-flow
    sums equal."""
    for i, x in enumerate(insts):
        a, b = int(arr["flow_off"][i]), int(arr["flow_off"][i + 1])
        o_fin, _, o_st = oracle.flow_sim(x, stats=True)
        assert np.array_equal(fin[a:b].view(np.uint64), o_fin.view(np.uint64)), \
            f"instance {i}: finish times differ (max abs {np.max(np.abs(fin[a:b] - o_fin))})"
        assert tuple(st[i]) == o_st, f"instance {i}: counts {tuple(st[i])}, oracle {o_st}"


def _flows(cap, paths, nbytes, start):
    off = np.zeros(len(paths) + 1, np.uint64)
    off[1:] = np.cumsum([len(p) for p in paths])
    return dict(cap=np.asarray(cap, np.float64), path_off=off,
                path=np.asarray([l for p in paths for l in p], np.uint32),
                bytes=np.asarray(nbytes, np.float64), start=np.asarray(start, np.float64))


def _selection_flows(nk, cfg, seed, n_inst):
    """A batch selected on the GPU (k = 1), its transfers' sizes from the GPU
    and from the oracle, and n_inst instances of those transfers on the
    cluster's fat tree under different background-load draws."""
    snap = W.make_snapshot(cfg, seed, inflight="random")
    ch = W.prefix_chains(cfg, seed)
    req = W.make_requests(cfg, seed, chains=ch)
    cache = W.make_caches(cfg, seed, chains=ch)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    out = sel.select(rd, k=1)
    by = nk.to_numpy(sel.selection_bytes(rd, out["idx"], 1))
    sel.sync_errors()
    idx = nk.to_numpy(out["idx"]).reshape(-1)
    o_by = oracle.selection_bytes(snap, cache, req, idx, 1)
    assert np.array_equal(by, o_by), "selection bytes differ from the oracle's"
    ok = idx >= 0
    p_inst = req["prefill"][ok]
    d_inst = idx[ok]
    insts = []
    for i in range(n_inst):
        cap, lay = W.fat_tree_links(cfg, W.draw_links(cfg, seed + 1000 + i))
        off, path = W.transfer_paths(cfg, seed + i, p_inst, d_inst, lay)
        insts.append(dict(cap=cap, path_off=off, path=path, bytes=by[ok].astype(np.float64),
                          start=W.transfer_starts(seed + i, int(ok.sum()))))
    return sel, insts


def test_paper_validation_cases_on_the_gpu(nk):
    """Sec. VI-B's three validation claims, each an instance of one call: a
    lone flow at its bottleneck bandwidth, N flows with 1/N of a common
    bottleneck, reallocation after a completion and after an arrival; plus
    the parking-lot case, zero-byte flows, simultaneous arrivals and an
    instance with no flows.  Closed forms, and the oracle bit for bit."""
    _say("flow sim validation cases")
    n = 5
    b = np.array([1.0, 2.0, 2.0, 5.0, 9.0])
    insts = [
        _flows([50e9, 25e9, 50e9, 900e9, 1.0, 1.0], [[0, 1, 2]], [10e9], [1.0]),
        _flows([10.0] + [100.0] * n, [[0, 1 + i] for i in range(n)], [4.0] * n, [0.0] * n),
        _flows([3.0] + [50.0] * n, [[0, 1 + i] for i in range(n)], b, np.zeros(n)),
        _flows([2.0, 10.0, 10.0, 1.0, 1.0, 1.0], [[0, 1], [0, 2]], [2.0, 2.0], [0.0, 0.5]),
        _flows([1.0, 2.0, 1.0, 1.0, 1.0, 1.0], [[0, 1], [0], [1]], [1.0] * 3, [0.0] * 3),
        _flows([1.0] * 6, [[0], [1, 2], [0, 3]], [0.0, 3.0, 0.0], [0.2, 0.2, 0.7]),
        _flows([1.0] * 6, [], [], []),
    ]
    # one link count for the call: pad every instance's capacities to 6 links
    for x in insts:
        x["cap"] = np.concatenate([x["cap"], np.ones(6 - len(x["cap"]))])
    sel = nk.Selector(0)
    fin, ev, arr = _run(nk, sel, insts)
    sel.sync_errors()
    off = arr["flow_off"].astype(np.int64)
    assert fin[off[0]] == 1.0 + 10e9 / 25e9
    np.testing.assert_allclose(fin[off[1]:off[2]], n * 4.0 / 10.0, rtol=1e-15)
    want = np.array([(b[:k + 1].sum() + (n - k - 1) * b[k]) / 3.0 for k in range(n)])
    np.testing.assert_allclose(fin[off[2]:off[3]], want, rtol=1e-14)
    np.testing.assert_allclose(fin[off[3]:off[4]], [1.5, 2.0], rtol=1e-15)
    np.testing.assert_allclose(fin[off[4]:off[5]], [2.0, 2.0, 2.0 / 3.0], rtol=1e-15)
    assert fin[off[5]] == 0.2 and fin[off[5] + 2] == 0.7
    assert tuple(ev[6]) == (0, 0, 0)
    _check_against_oracle(insts, fin, ev, arr)
    sel.close()


def test_selected_transfers_on_the_64_gpu_fat_tree(nk):
    """The c0 batch (4,096 requests on the 64-GPU cluster) selected on the
    GPU; its transfer sizes bit-exact against the oracle's Eq. (2); the
    transfers (arrivals over 50 ms) simulated on the fat tree under four
    background-load draws: every finish time and allocation count bit for
    bit against the oracle."""
    _say("flow sim c0 transfers")
    sel, insts = _selection_flows(nk, W.CONFIGS["c0"], 3, 4)
    fin, ev, arr = _run(nk, sel, insts)
    sel.sync_errors()
    assert (ev[:, 0] > len(insts[0]["bytes"]) // 2).all()
    _check_against_oracle(insts, fin, ev, arr)
    # no flow beats its path alone
    for i, x in enumerate(insts):
        a = int(arr["flow_off"][i])
        po = x["path_off"].astype(np.int64)
        best = np.array([x["cap"][x["path"][po[f]:po[f + 1]]].min() for f in range(len(x["bytes"]))])
        assert (fin[a:a + len(best)] - x["start"] >= x["bytes"] / best * (1 - 1e-12)).all()
    sel.close()


def test_links_beyond_the_lds_limit(nk):
    """The 4,096-GPU fat tree (16,960 links: the link state lives in device
    memory instead of LDS): 600 random transfers between prefill and decode
    instances, arrivals over 10 ms, three background-load draws, against
    the oracle bit for bit."""
    _say("flow sim 4096-gpu links")
    cfg = W.CONFIGS["c2"]
    rng = np.random.default_rng(5)
    n = 600
    p_inst = rng.integers(0, cfg.n_prefill, n)
    d_inst = rng.integers(0, cfg.n_decode, n)
    insts = []
    for i in range(3):
        cap, lay = W.fat_tree_links(cfg, W.draw_links(cfg, 50 + i))
        off, path = W.transfer_paths(cfg, 60 + i, p_inst, d_inst, lay)
        insts.append(dict(cap=cap, path_off=off, path=path, bytes=rng.uniform(1e8, 4e9, n),
                          start=np.sort(rng.uniform(0.0, 0.01, n))))
    assert len(insts[0]["cap"]) == 16960
    sel = nk.Selector(0)
    fin, ev, arr = _run(nk, sel, insts)
    sel.sync_errors()
    _check_against_oracle(insts, fin, ev, arr)
    sel.close()


def test_invalid_instances_are_reported_and_others_unaffected(nk):
    """A link id past the link count, a capacity of 0, a negative size and
    a NaN arrival each poison their own instance only (all its finish times
    NaN, reported by netkv_sync_errors); the valid instances of the same
    call match the oracle."""
    _say("flow sim invalid instances")
    good = _flows([1.0, 2.0, 3.0], [[0, 1], [1, 2], [2]], [1.0, 2.0, 3.0], [0.0, 0.1, 0.2])
    bad_link = _flows([1.0, 2.0, 3.0], [[0, 1], [1, 3]], [1.0, 1.0], [0.0, 0.0])
    bad_cap = _flows([1.0, 0.0, 3.0], [[0, 1]], [1.0], [0.0])
    bad_bytes = _flows([1.0, 2.0, 3.0], [[0]], [-1.0], [0.0])
    bad_start = _flows([1.0, 2.0, 3.0], [[0]], [1.0], [np.nan])
    insts = [good, bad_link, bad_cap, good, bad_bytes, bad_start]
    sel = nk.Selector(0)
    fin, ev, arr = _run(nk, sel, insts)
    with pytest.raises(nk.NetKVError):
        sel.sync_errors()
    off = arr["flow_off"].astype(np.int64)
    for i in (1, 2, 4, 5):
        assert np.isnan(fin[off[i]:off[i + 1]]).all() and tuple(ev[i]) == (0, 0, 0)
    for i in (0, 3):
        o_fin, _, o_st = oracle.flow_sim(good, stats=True)
        assert np.array_equal(fin[off[i]:off[i + 1]], o_fin) and tuple(ev[i]) == o_st
    sel.sync_errors()   # cleared by the previous report
    sel.close()


def test_offsets_that_are_not_a_partition_invalidate_the_call(nk):
    """Flow offsets that decrease, or end past the call's flows, make every
    instance of the call invalid (finish times NaN on every instance whose
    own range lies inside the flows, all counts 0, reported by
    netkv_sync_errors); the same flows with valid offsets then match the
    oracle."""
    _say("flow sim offsets not a partition")
    good = _flows([1.0, 2.0, 3.0], [[0, 1], [1, 2], [2]], [1.0, 2.0, 3.0], [0.0, 0.1, 0.2])
    arr, L = _instances([good, good, good])
    sel = nk.Selector(0)
    # (offsets, flows covered by an instance whose range is inside the 9 flows)
    for off, covered in (([0, 3, 1, 9], 9), ([0, 3, 6, 10], 6)):
        bad = dict(arr, flow_off=np.asarray(off, np.uint64))
        dev = {k: nk.to_device(v, sel.device) for k, v in bad.items()}
        fin, st = sel.flow_sim(dev, 3, L)
        with pytest.raises(nk.NetKVError):
            sel.sync_errors()
        assert np.isnan(nk.to_numpy(fin)[:covered]).all(), off
        assert (nk.to_numpy(st) == 0).all(), off
    fin, st, arr2 = _run(nk, sel, [good, good, good])
    sel.sync_errors()
    _check_against_oracle([good, good, good], fin, st, arr2)
    sel.close()


def test_bursts_cross_the_wavefront_and_workgroup_sizes(nk):
    """Arrivals in bursts of 10, 70, 300 and 40 flows, apart and
    overlapping, on the 64-GPU fat tree: the flows in progress cross 64
    (one wavefront's lanes) and 256 (one flow per thread) upward and
    downward many times, so every hand-over between the wavefront run, the
    per-thread workgroup passes and the general workgroup passes is taken;
    four load draws, every finish time and count against the oracle bit for
    bit."""
    _say("flow sim bursts")
    cfg = W.CONFIGS["c0"]
    rng = np.random.default_rng(17)
    bursts = [(0.0, 10), (0.002, 70), (0.004, 300), (0.0041, 40), (0.05, 300), (0.3, 70), (0.31, 10)]
    start = np.concatenate([np.full(n, t0) + rng.uniform(0.0, 1e-4, n) for t0, n in bursts])
    n = len(start)
    p_inst = rng.integers(0, cfg.n_prefill, n)
    d_inst = rng.integers(0, cfg.n_decode, n)
    insts = []
    for i in range(4):
        cap, lay = W.fat_tree_links(cfg, W.draw_links(cfg, 70 + i))
        off, path = W.transfer_paths(cfg, 80 + i, p_inst, d_inst, lay)
        insts.append(dict(cap=cap, path_off=off, path=path, bytes=rng.uniform(1e6, 2e9, n), start=start.copy()))
    sel = nk.Selector(0)
    fin, ev, arr = _run(nk, sel, insts)
    sel.sync_errors()
    # many flows in progress at once on average, so the larger passes ran
    assert (ev[:, 2] / ev[:, 0] > 64).all(), ev
    _check_against_oracle(insts, fin, ev, arr)
    sel.close()
