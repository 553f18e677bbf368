"""Parity helpers shared by the GPU tests and the benchmark's CPU leg (no
test functions here).

Tolerances:
  * prefix lengths j and the feasibility mask: bit-exact;
  * scores: the HIP path computes in fp32, the oracle in fp64; relative
    difference at most SCORE_RTOL;
  * selected indices: exact, ties to the lowest index.  The one exception is
    a near-tie: where the oracle's costs of the GPU's choice and of the
    oracle's choice differ, but by at most NEAR_TIE relative, fp32 rounding
    may order the two either way.  An exact fp64 tie is not a near-tie: the
    oracle's choice is then the lower index, and the GPU must make the same
    choice unless its own fp32 scores of the two decodes differ (checked
    when the GPU's per-pair scores are passed in).
"""
import numpy as np

SCORE_RTOL = 1e-5
NEAR_TIE = 1e-6


def _bits(x):
    return np.ascontiguousarray(np.asarray(x, dtype=np.float32)).view(np.uint32)


def classify(g_idx, o_idx, o_cost, near=NEAR_TIE, g_cost=None):
    """Classify the positions where the GPU's selection differs from the
    oracle's.  g_idx / o_idx [R, k]; o_cost [R, D] (fp64) and optionally
    g_cost [R, D] (the GPU's fp32 per-pair scores).

    Returns dict(positions, mismatches, near_ties, exact_ties_fp32_split,
    exact_ties, beyond, max_rel_gap), where exact_ties counts rows whose
    first difference is at an exact fp64 tie that the GPU's fp32 scores do
    not separate (a tie-break error: the oracle's choice is the lowest index
    among the tied), exact_ties_fp32_split those that they do, and beyond
    the mismatches further apart than the near-tie rule allows."""
    g_idx = np.asarray(g_idx).reshape(np.asarray(o_idx).shape)
    R = g_idx.shape[0]
    rows = np.arange(R)[:, None]
    ok = (o_idx >= 0) & (g_idx >= 0)
    gi = np.where(g_idx >= 0, g_idx, 0)
    oi = np.where(o_idx >= 0, o_idx, 0)
    cg = o_cost[rows, gi]
    co = o_cost[rows, oi]
    mism = ok & (g_idx != o_idx)
    # the exact-tie rule applies at a row's first difference: after it, a
    # near-tie substitution shifts the rest of a top-k list, so later
    # positions may pair up equal costs of different decodes
    first = mism & (np.cumsum(mism, axis=1) == 1)
    tie = first & (cg == co)
    split = np.zeros_like(tie)
    if g_cost is not None and tie.any():
        gc = np.asarray(g_cost, dtype=np.float32).reshape(R, -1)
        gb = _bits(gc[rows, gi])
        ob = _bits(gc[rows, oi])
        split = tie & (gb < ob)
    near_m = mism & ~tie & (np.abs(cg - co) <= near * np.abs(co))   # includes later equal costs
    beyond = mism & ~tie & ~near_m
    gap = np.abs(cg - co)[mism] / np.abs(co[mism]) if mism.any() else np.zeros(0)
    return dict(positions=int(ok.sum()), mismatches=int(mism.sum()), near_ties=int(near_m.sum()),
                exact_ties_fp32_split=int(split.sum()), exact_ties=int((tie & ~split).sum()),
                beyond=int(beyond.sum()), max_rel_gap=float(gap.max()) if gap.size else 0.0,
                bad_mask=beyond | (tie & ~split))


def check_topk(g_idx, g_score, o_idx, o_cost, o_feas, near=NEAR_TIE, rtol=SCORE_RTOL, g_cost=None):
    """g_*: GPU [R, k]; o_idx [R, k] oracle; o_cost / o_feas [R, D] oracle;
    g_cost: optional GPU per-pair fp32 scores [R, D] of the same call.
    Returns (number of positions, number accepted as near-ties)."""
    g_idx = np.asarray(g_idx).reshape(o_idx.shape)
    g_score = np.asarray(g_score, dtype=np.float64).reshape(o_idx.shape)
    R, k = o_idx.shape
    rows = np.arange(R)[:, None]
    pad = o_idx < 0
    assert (g_idx[pad] == -1).all(), "GPU selected where the oracle rejects"
    assert np.isinf(g_score[pad]).all() and (g_score[pad] > 0).all()
    ok = ~pad
    assert (g_idx[ok] >= 0).all(), "GPU rejects where the oracle selects"
    gi = np.where(g_idx >= 0, g_idx, 0)
    oi = np.where(o_idx >= 0, o_idx, 0)
    assert o_feas[rows, gi][ok].all(), "GPU selected an infeasible decode"
    cg = o_cost[rows, gi]
    co = o_cost[rows, oi]
    c = classify(g_idx, o_idx, o_cost, near, g_cost)
    if c["beyond"] or c["exact_ties"]:
        at = np.argwhere(c["bad_mask"])[0].tolist()
        raise AssertionError(
            f"{c['beyond']} selections differ beyond the near-tie rule and {c['exact_ties']} break an "
            f"exact tie away from the lowest index; first at {at}: gpu {g_idx[tuple(at)]} "
            f"({cg[tuple(at)]!r}) oracle {o_idx[tuple(at)]} ({co[tuple(at)]!r})")
    err = np.abs(g_score - cg)
    sbad = ok & ~(err <= rtol * np.abs(cg))
    assert not sbad.any(), f"score error {np.max(err[ok] / np.abs(cg[ok]))} > {rtol}"
    if k > 1:
        s = np.sort(np.where(g_idx >= 0, g_idx, -1 - np.arange(k)[None, :]), axis=1)
        assert (np.diff(s, axis=1) != 0).all(), "repeated decode in a top-k list"
        # ascending (score, index)
        gs = np.where(ok, g_score, np.inf)
        assert (np.diff(gs, axis=1) >= 0).all(), "top-k not ascending"
    return c["positions"], c["mismatches"]


def self_topk(g_cost, g_feas, k):
    """The exact top-k by (fp32 score bits, index) over the feasible pairs of
    the GPU's own per-pair outputs [R, D]: (idx [R, k] int32, score bits
    [R, k] uint32); -1 / +inf bits where fewer than k are feasible."""
    gc = np.asarray(g_cost, dtype=np.float32)
    R, D = gc.shape
    key = (_bits(gc).astype(np.uint64) << np.uint64(32)) | np.arange(D, dtype=np.uint64)[None, :]
    key = np.where(np.asarray(g_feas).reshape(R, D) != 0, key, np.uint64(0xFFFFFFFFFFFFFFFF))
    kk = min(k, D)
    part = np.sort(np.partition(key, kk - 1, axis=1)[:, :kk], axis=1)
    idx = np.full((R, k), -1, dtype=np.int32)
    bits = np.full((R, k), 0x7F800000, dtype=np.uint32)
    full = part != np.uint64(0xFFFFFFFFFFFFFFFF)
    idx[:, :kk] = np.where(full, (part & np.uint64(0xFFFFFFFF)).astype(np.int64), -1)
    bits[:, :kk] = np.where(full, (part >> np.uint64(32)).astype(np.uint32), np.uint32(0x7F800000))
    return idx, bits


def check_self_topk(g_idx, g_score, g_cost, g_feas):
    """The GPU's top-k list must be exactly the lexicographic (score, index)
    top-k of its own per-pair scores over the feasible pairs: ties of equal
    fp32 scores go to the lowest index, with no tolerance."""
    g_idx = np.asarray(g_idx)
    R, k = g_idx.shape
    D = np.asarray(g_cost).size // R
    ei, eb = self_topk(np.asarray(g_cost).reshape(R, D), np.asarray(g_feas).reshape(R, D), k)
    bad = ei != g_idx
    assert not bad.any(), (f"{int(bad.sum())} top-k entries are not the lowest-index top-k of the GPU's own "
                           f"scores; first at {np.argwhere(bad)[0].tolist()}")
    assert np.array_equal(eb, _bits(g_score).reshape(R, k)), "top-k scores differ from the per-pair scores"


def check_pairs(g_j, g_feas, g_cost, o, rtol=SCORE_RTOL):
    """Per-pair outputs [R*D] of the GPU against the oracle's [R, D]."""
    R, D = o["j"].shape
    np.testing.assert_array_equal(np.asarray(g_j).reshape(R, D), o["j"])
    np.testing.assert_array_equal(np.asarray(g_feas).reshape(R, D), o["feasible"])
    gc = np.asarray(g_cost, dtype=np.float64).reshape(R, D)
    rel = np.abs(gc - o["cost"]) / np.abs(o["cost"])
    assert np.nanmax(rel) <= rtol, f"max relative score error {np.nanmax(rel)}"
    return float(np.max(rel))


def subset_requests(req, rows):
    """CSR of a subset of requests (in the given order)."""
    rows = np.asarray(rows, dtype=np.int64)
    off = req["hash_off"].astype(np.int64)
    n = off[rows + 1] - off[rows]
    new_off = np.zeros(len(rows) + 1, dtype=np.uint64)
    new_off[1:] = np.cumsum(n)
    idx = np.concatenate([np.arange(off[r], off[r + 1]) for r in rows]) if len(rows) else \
        np.zeros(0, np.int64)
    return dict(prefill=req["prefill"][rows].copy(), len_tokens=req["len_tokens"][rows].copy(),
                hash_off=new_off, hashes=req["hashes"][idx].copy())


def slice_requests(req, r0, r1):
    """CSR of the contiguous requests [r0, r1) (offsets rebased to 0)."""
    off = req["hash_off"].astype(np.int64)
    a, b = off[r0], off[r1]
    return dict(prefill=req["prefill"][r0:r1].copy(), len_tokens=req["len_tokens"][r0:r1].copy(),
                hash_off=(off[r0:r1 + 1] - a).astype(np.uint64),
                hashes=req["hashes"][a:b].copy() if b > a else np.ones(1, np.uint64))
