"""Parity helpers shared by the GPU tests (no test functions here).

Tolerances:
  * prefix lengths j and the feasibility mask: bit-exact;
  * scores: the HIP path computes in fp32, the oracle in fp64; relative
    difference at most SCORE_RTOL;
  * selected indices: exact (ties to the lowest index), except where the
    oracle's costs of the GPU's choice and of the oracle's choice are within
    NEAR_TIE relative -- fp32 rounding may order such near-ties either way.
"""
import numpy as np

SCORE_RTOL = 1e-5
NEAR_TIE = 1e-6


def check_topk(g_idx, g_score, o_idx, o_cost, o_feas, near=NEAR_TIE, rtol=SCORE_RTOL):
    """g_*: GPU [R, k]; o_idx [R, k] oracle; o_cost / o_feas [R, D] oracle.
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
    mism = ok & (g_idx != o_idx)
    bad = mism & ~(np.abs(cg - co) <= near * np.abs(co))
    assert not bad.any(), (
        f"{int(bad.sum())} selections differ beyond the near-tie rule; first at "
        f"{np.argwhere(bad)[0].tolist()}: gpu {g_idx[bad][0]} ({cg[bad][0]!r}) "
        f"oracle {o_idx[bad][0]} ({co[bad][0]!r})")
    err = np.abs(g_score - cg)
    sbad = ok & ~(err <= rtol * np.abs(cg))
    assert not sbad.any(), f"score error {np.max(err[ok] / np.abs(cg[ok]))} > {rtol}"
    if k > 1:
        s = np.sort(np.where(g_idx >= 0, g_idx, -1 - np.arange(k)[None, :]), axis=1)
        assert (np.diff(s, axis=1) != 0).all(), "repeated decode in a top-k list"
        # ascending (score, index)
        gs = np.where(ok, g_score, np.inf)
        assert (np.diff(gs, axis=1) >= 0).all(), "top-k not ascending"
    return int(ok.sum()), int(mism.sum())


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
