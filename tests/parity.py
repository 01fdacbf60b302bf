"""Comparison rules between the GPU path and the CPU oracle.

Two bars:
* exact: the selected index set and every selected score must match bit for
  bit (select-only entries, and fused runs on inputs whose arithmetic is
  exact in float32);
* tolerance (fused runs on real-valued inputs): every returned score is
  within rtol of the oracle's score of the same key, relative to
  max(|I_ref(key)|, |I_ref,(k)|) where I_ref,(k) is the row's oracle k-th
  score; and the returned set may differ from the oracle's only by swapping
  keys whose oracle scores lie within rtol * |I_ref,(k)| of that k-th score.
  rtol is 1e-3 for float32 / bf16 inputs and 2e-2 for fp8.
"""
from __future__ import annotations

import numpy as np

RTOL = {"f32": 1e-3, "bf16": 1e-3, "fp8": 2e-2}


def _valid(idx_row):
    return idx_row[idx_row >= 0]


def check_padding(gi, gs, e, k):
    m = min(k, e)
    assert np.all(gi[:m] >= 0), "fewer than min(k, e) entries"
    assert np.all(gi[m:] == -1), "padding index must be -1"
    assert np.all(np.isneginf(gs[m:])), "padding score must be -inf"


def check_row_exact(gi, gs, ri, rs, e, k, sorted_output=False):
    """Bit-exact comparison of one row (index set and per-key score bits)."""
    check_padding(gi, gs, e, k)
    m = min(k, e)
    if sorted_output:
        np.testing.assert_array_equal(gi, ri)
        np.testing.assert_array_equal(gs[:m].view(np.uint32), rs[:m].view(np.uint32))
        return
    og = np.argsort(gi[:m], kind="stable")
    orr = np.argsort(ri[:m], kind="stable")
    np.testing.assert_array_equal(gi[:m][og], ri[:m][orr])
    np.testing.assert_array_equal(gs[:m][og].view(np.uint32), rs[:m][orr].view(np.uint32))


def check_row_tol(gi, gs, ri, rs, full, e, k, rtol):
    """Tolerance comparison of one row against the oracle. `full` holds the
    oracle's float32 score of every visible key of the row."""
    check_padding(gi, gs, e, k)
    m = min(k, e)
    g = gi[:m].astype(np.int64)
    assert len(set(g.tolist())) == m, "duplicate indices"
    assert np.all((g >= 0) & (g < e)), "index outside the visible range"
    if m == 0:
        return
    kth = float(rs[m - 1])
    ref_g = full[g].astype(np.float64)
    bound = rtol * np.maximum(np.abs(ref_g), abs(kth))
    err = np.abs(gs[:m].astype(np.float64) - ref_g)
    bad = np.nonzero(err > bound)[0]
    assert bad.size == 0, "score error beyond tolerance at keys %s (got %s, want %s)" % (
        g[bad[:5]], gs[:m][bad[:5]], ref_g[bad[:5]])
    diff = set(g.tolist()) ^ set(ri[:m].astype(np.int64).tolist())
    if diff:
        d = np.array(sorted(diff))
        far = np.abs(full[d].astype(np.float64) - kth) > rtol * abs(kth)
        assert not np.any(far), "set differs beyond the swap rule at keys %s (scores %s, k-th %r)" % (
            d[far][:5], full[d][far][:5], kth)


def visible(offsets, nq, nk):
    if offsets is None:
        return np.full(nq, nk, dtype=np.int64)
    return np.clip(np.asarray(offsets, dtype=np.int64), 0, nk)
