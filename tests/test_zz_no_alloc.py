"""The no-allocation selection (netkv_select_batch_noalloc) against the
allocating one (netkv_select_batch) through the C ABI: selections and
scores bit-identical, on consecutive calls with a smaller second input,
across the sub-batches a large batch is split into, and the clear error
for a decode pool too large for its static scratch.  Needs an MI355X and
the built library."""
import numpy as np
import pytest

from paper_2606_03910_amd import workload as W
from tests.parity import slice_requests

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


def _both(nk, sel, req, k, sentinel=-7):
    """(idx, score) of the allocating and of the no-allocation call; the
    latter's outputs start as a sentinel that no result may keep."""
    rd = nk.requests_to_device(req, sel.device)
    n = int(rd["prefill"].numel())
    a = sel.select(rd, k=k)
    bi = torch.full((n * k,), sentinel, dtype=torch.int32, device=sel.device)
    bs = torch.full((n * k,), float(sentinel), dtype=torch.float32, device=sel.device)
    nk.netkv_select_batch_noalloc(sel.h, rd, k, bi, bs, sel.device)
    sel.sync_errors()
    ai, asc = nk.to_numpy(a["idx"]), nk.to_numpy(a["score"])
    bi, bsc = nk.to_numpy(bi), nk.to_numpy(bs)
    assert not (bi == sentinel).any(), "a request's result was never written"
    return ai, asc, bi, bsc


def _same(ai, asc, bi, bsc, what):
    assert np.array_equal(ai, bi), f"{what}: {int((ai != bi).sum())} selections differ"
    assert np.array_equal(asc.view(np.uint32), bsc.view(np.uint32)), f"{what}: scores differ"


def test_noalloc_full_batch_then_smaller(nk):
    """The whole 4,096-GPU-scale batch (1,048,576 requests: sixteen
    sub-batches of the static scratch), then a smaller batch of 50,000
    requests and a small one with k = 8, each against the allocating call on
    the same handle."""
    cfg = W.CONFIGS["c2"]
    snap = W.make_snapshot(cfg, 0)
    ch = W.prefix_chains(cfg, 0)
    req = W.make_requests(cfg, 0, chains=ch)
    cache = W.make_caches(cfg, 0, chains=ch)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    del cache
    _say("no-alloc: c2 full batch, k = 1")
    ai, asc, bi, bsc = _both(nk, sel, req, 1)
    _same(ai, asc, bi, bsc, "c2 full batch")
    assert (ai >= 0).mean() > 0.99
    _say("no-alloc: 50,000 requests, k = 3")
    sub = slice_requests(req, 123456, 173456)
    _same(*_both(nk, sel, sub, 3), "50,000 requests k=3")
    _say("no-alloc: 700 requests, k = 8")
    sub = slice_requests(req, 5000, 5700)
    _same(*_both(nk, sel, sub, 8), "700 requests k=8")
    sel.close()


def test_noalloc_small_pool_in_flight_and_repeat(nk):
    """64-GPU pool with random in-flight counters: a 4,096-request batch,
    then 1,000 of its requests, k = 1, 2 and 5, each twice in a row."""
    cfg = W.CONFIGS["c0"]
    snap = W.make_snapshot(cfg, 3, inflight="random")
    ch = W.prefix_chains(cfg, 3)
    req = W.make_requests(cfg, 3, chains=ch)
    cache = W.make_caches(cfg, 3, chains=ch)
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    sel.load_cache(cache, 0.5)
    for k in (1, 2, 5):
        for rows in ((0, 4096), (1000, 2000)):
            for rep in range(2):
                _say("no-alloc: c0", rows, "k", k, "call", rep)
                _same(*_both(nk, sel, slice_requests(req, *rows), k), f"c0 {rows} k={k} call {rep}")
    sel.close()


def test_noalloc_rejects_a_pool_beyond_its_scratch(nk):
    """2^23 decodes: one leader row and the all-zero row alone exceed the
    64 MiB static scratch, so the call fails with ECAPACITY before any
    launch and writes nothing; the allocating call still answers."""
    D = 1 << 23
    snap = dict(W.params_of(W.CONFIGS["c0"]))
    snap.update(n_prefill=1, n_decode=D, tier_map=np.zeros(D, np.uint8), util=np.zeros(D, np.float32),
                n_inflight=np.zeros(4, np.uint16), free_mem=np.full(D, 100 * 10 ** 9, np.uint64),
                queue_depth=np.zeros(D, np.uint32), batch_size=np.zeros(D, np.uint32))
    sel = nk.Selector(0)
    sel.load_snapshot(snap)
    cache = dict(hash_off=np.zeros(D + 1, np.uint64), hashes=np.ones(1, np.uint64))
    sel.load_cache(cache, 0.5)
    req = dict(prefill=np.zeros(2, np.uint32), len_tokens=np.array([1000, 20], np.uint32),
               hash_off=np.array([0, 1, 1], np.uint64), hashes=np.array([12345], np.uint64))
    rd = nk.requests_to_device(req, sel.device)
    bi = torch.full((2,), -7, dtype=torch.int32, device=sel.device)
    bs = torch.full((2,), -7.0, dtype=torch.float32, device=sel.device)
    with pytest.raises(nk.NetKVError) as e:
        nk.netkv_select_batch_noalloc(sel.h, rd, 1, bi, bs, sel.device)
    assert e.value.status == -5 and "no-allocation scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (bi == -7).all() and (bs == -7.0).all()
    out = sel.select(rd, k=1)
    sel.sync_errors()
    assert (nk.to_numpy(out["idx"]) == 0).all()
    sel.close()
