"""The allocation-free selection captured into a HIP graph and replayed:
every replay bit-identical to the allocating call.  A batch of 100,000
requests: a first sub-batch of 65,536 (which forks the handle's second
stream; the capture takes both branches) and a second of 34,464."""
import numpy as np
import pytest

from paper_2606_03910_amd import workload as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def nk():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_03910_amd import netkv
    netkv.load_library()
    return netkv


def test_noalloc_selection_replays_from_a_graph(nk):
    print("[gpu-case] graph capture of the allocation-free selection", flush=True)
    cfg = W.scaled(W.CONFIGS["c0"], n_requests=100000)
    snap = W.make_snapshot(cfg, 17, inflight="random")
    ch = W.prefix_chains(cfg, 17)
    req = W.make_requests(cfg, 17, chains=ch)
    cache = W.make_caches(cfg, 17, chains=ch)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    rd = nk.requests_to_device(req, sel.device)
    k = 2
    n = cfg.n_requests
    ref = sel.select(rd, k=k)
    sel.sync_errors()
    ri, rs = nk.to_numpy(ref["idx"]), nk.to_numpy(ref["score"])
    bi = torch.empty(n * k, dtype=torch.int32, device=sel.device)
    bs = torch.empty(n * k, dtype=torch.float32, device=sel.device)
    nk.netkv_select_batch_noalloc(sel.h, rd, k, bi, bs, sel.device)   # eager once
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        nk.netkv_select_batch_noalloc(sel.h, rd, k, bi, bs, sel.device)
    torch.cuda.synchronize()
    for rep in range(3):
        bi.fill_(-7)
        bs.fill_(-7.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        gi, gs = nk.to_numpy(bi), nk.to_numpy(bs)
        assert np.array_equal(gi, ri), f"replay {rep}: {int((gi != ri).sum())} selections differ"
        assert np.array_equal(gs.view(np.uint32), rs.view(np.uint32)), f"replay {rep}: scores differ"
        # eager work between replays
        sel.select(rd, k=1)
        torch.cuda.synchronize()
    sel.sync_errors()
    del g
    sel.close()
