"""CPU oracle for the fused Indexer-TopK operation.

TEST INFRASTRUCTURE ONLY. The library never imports, links or calls this
module; only the test suite, the smoke check and the benchmark's CPU-baseline
leg do. It shares no code with the GPU path.

What it computes is the plain definition of the operation, with none of the
method's performance devices (sampling, binning, thresholds, candidate
buffers): those cannot change an exact top-k, so the oracle leaves them out.

* Index score -- Eq. (1), sec. 2.1 (DSA indexer):
      I[t, s] = sum_j w[t, j] * ReLU(q[t, j] . k[s])
  evaluated in float64 from exactly dequantised inputs, then rounded once to
  float32 (round to nearest even).
* Inner-product score -- the k-NN case of sec. 3.1 (Eq. 2 with f an inner
  product, sec. 3.2 "inner-product-based" scorers): the same sum without the
  ReLU; with one head and unit weights it is q . k.
* Exact top-k -- Eq. (2), sec. 3.1: for every query the k visible keys with the
  highest score. The paper requires exactness (sec. 3.1 "exactly identify",
  sec. 3.2 "preserving exact Top-k correctness") but does not say how ties are
  broken; this oracle makes the answer unique with one total order:
      higher score first; -0.0 equals +0.0; NaN ranks below -inf;
      equal scores -> lower key index first.
  Rows with fewer than k visible keys return all of them, then padding
  (index -1, score -inf).
* Visibility -- the query chunk attends to the preceding context (sec. 1, the
  DSA prefill description): row t sees keys [0, e_t) with
  e_t = clamp(causal_offsets[t], 0, Nk), or all Nk keys when no offsets are
  given. Optional per-row starts narrow this to [s_t, e_t),
  s_t = clamp(visible_start[t], 0, e_t): several sequences packed into one
  key array, each query seeing its own sequence's keys.
* fp8 inputs are OCP E4M3FN bytes (decoded here from the format definition:
  1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits, no infinities,
  S.1111.111 is NaN) times a positive float32 per-token scale; the product is
  exact in float64.
* bf16 inputs are the upper 16 bits of a float32.
* Previous-chunk sample -- sec. 3.2 "Sampling": for a prefill chunk the
  sample is the k' keys that occur most often in the previous chunk's top-k
  results. The paper does not say how equal counts are ordered or what
  happens when fewer than k' distinct keys occur; the oracle takes equal
  counts in ascending key order and returns only keys that occur at least
  once (then padding -1), listed in ascending key order.
* LiteDSA union and membership masks -- sec. 3.3: a group of consecutive
  queries attends over the union of their top-k keys, one shared list, and
  each query keeps a bitmask over that list marking its own keys. The oracle
  takes the union as a set, lists it ascending (the order the paper's bitmap
  sweep produces), and sets bit j of a query's mask iff the union's j-th key
  is in that query's list.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np

PAD_INDEX = -1
PAD_SCORE = np.float32(-np.inf)


# ----------------------------------------------------------------------------
# Decoding of the storage formats
# ----------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64 (exact)."""
    b = np.asarray(bits).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def e4m3fn_to_f64(bits: np.ndarray) -> np.ndarray:
    """OCP FP8 E4M3FN bit patterns (uint8) -> float64 (exact)."""
    b = np.asarray(bits).astype(np.int64)
    sign = np.where((b >> 7) & 1, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = (b & 0x7).astype(np.float64)
    normal = (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0)
    subnormal = (m / 8.0) * np.exp2(-6.0)
    mag = np.where(e == 0, subnormal, normal)
    mag = np.where((e == 15) & ((b & 0x7) == 7), np.nan, mag)
    return sign * mag


def dequantize(x: np.ndarray, dtype: str, scale: Optional[np.ndarray] = None) -> np.ndarray:
    """Storage array -> float64 values.

    dtype "f32": x is float32; "bf16": x is uint16 bit patterns; "fp8": x is
    uint8 E4M3FN bit patterns and ``scale`` (float32, broadcast over the last
    axis) multiplies every value."""
    if dtype == "f32":
        v = np.asarray(x, dtype=np.float32).astype(np.float64)
    elif dtype == "bf16":
        v = bf16_to_f64(x)
    elif dtype == "fp8":
        v = e4m3fn_to_f64(x)
    else:
        raise ValueError(dtype)
    if scale is not None:
        v = v * np.asarray(scale, dtype=np.float32).astype(np.float64)[..., None]
    return v


def visible_counts(causal_offsets: Optional[np.ndarray], nq: int, nk: int) -> np.ndarray:
    """e_t for every row (see the module docstring)."""
    if causal_offsets is None:
        return np.full(nq, nk, dtype=np.int64)
    return np.clip(np.asarray(causal_offsets, dtype=np.int64), 0, nk)


def visible_ranges(causal_offsets: Optional[np.ndarray], visible_start: Optional[np.ndarray], nq: int,
                   nk: int) -> Tuple[np.ndarray, np.ndarray]:
    """(s_t, e_t) for every row: row t sees keys [s_t, e_t), e_t as in
    visible_counts and s_t = clamp(visible_start[t], 0, e_t) (0 without
    starts). Several sequences packed into one key array give each query its
    own sequence's span this way."""
    e = visible_counts(causal_offsets, nq, nk)
    if visible_start is None:
        return np.zeros(nq, dtype=np.int64), e
    s = np.minimum(np.maximum(np.asarray(visible_start, dtype=np.int64), 0), e)
    return s, e


# ----------------------------------------------------------------------------
# Scores -- Eq. (1)
# ----------------------------------------------------------------------------

def row_scores(q_row: np.ndarray, w_row: Optional[np.ndarray], keys: np.ndarray, mode: str) -> np.ndarray:
    """Scores of one query against every row of ``keys``.

    q_row [H, d] float64, w_row [H] float64 or None (unit weights), keys [n, d]
    float64. Returns float32 [n]: the float64 value of Eq. (1) (mode "dsa") or
    of the weighted inner product (mode "ip"), rounded once to float32."""
    x = q_row @ keys.T                      # [H, n]: per-head q_{t,j} . k_s
    if mode == "dsa":
        x = np.maximum(x, 0.0)              # ReLU of each head's dot product
    elif mode != "ip":
        raise ValueError(mode)
    w = np.ones(q_row.shape[0]) if w_row is None else w_row
    return (w @ x).astype(np.float32)       # weighted sum over heads, one rounding


def index_scores(q: np.ndarray, w: Optional[np.ndarray], keys: np.ndarray, mode: str,
                 rows: Optional[Sequence[int]] = None, ncols: Optional[int] = None) -> np.ndarray:
    """Dense float32 score matrix [len(rows), ncols] for dequantised float64
    inputs q [Nq, H, d], w [Nq, H] (or None), keys [Nk, d]. Every column is
    scored, visible or not."""
    rows = range(q.shape[0]) if rows is None else rows
    ncols = keys.shape[0] if ncols is None else ncols
    out = np.empty((len(rows), ncols), dtype=np.float32)
    for i, t in enumerate(rows):
        out[i] = row_scores(q[t], None if w is None else w[t], keys[:ncols], mode)
    return out


# ----------------------------------------------------------------------------
# Exact selection -- Eq. (2)
# ----------------------------------------------------------------------------

def order(scores: np.ndarray) -> np.ndarray:
    """Indices of ``scores`` (float32, 1-D) sorted by the oracle's total order:
    score descending, NaN last, -0.0 == +0.0, ties by ascending index."""
    s = np.asarray(scores, dtype=np.float32).astype(np.float64)
    nan = np.isnan(s)
    neg = np.where(nan, 0.0, -s)            # -(-0.0) == 0.0 == -(+0.0) compare equal
    idx = np.arange(s.size)
    # lexsort: last key is primary; stable, so equal keys keep index order.
    return np.lexsort((idx, neg, nan))


def select_row(scores: np.ndarray, e: int, k: int, s: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Exact top-k of the visible keys [s, e) of one row, scores[s:e].

    Returns (idx int32 [k], score float32 [k]) sorted by the total order, with
    min(k, e - s) real entries (key indices) followed by padding (-1, -inf)."""
    vis = np.asarray(scores[s:e], dtype=np.float32)
    o = order(vis)[:k]
    idx = np.full(k, PAD_INDEX, dtype=np.int32)
    sc = np.full(k, PAD_SCORE, dtype=np.float32)
    idx[:o.size] = o + s
    sc[:o.size] = vis[o]
    return idx, sc


def topk_select(scores: np.ndarray, nk: int, k: int, causal_offsets: Optional[np.ndarray] = None,
                rows: Optional[Sequence[int]] = None,
                visible_start: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Scores-in selection: exact top-k of every requested row of a float32
    score matrix whose first ``nk`` columns are keys."""
    nq = scores.shape[0]
    rows = list(range(nq)) if rows is None else list(rows)
    s0, e = visible_ranges(causal_offsets, visible_start, nq, nk)
    out_i = np.empty((len(rows), k), dtype=np.int32)
    out_s = np.empty((len(rows), k), dtype=np.float32)
    for i, t in enumerate(rows):
        out_i[i], out_s[i] = select_row(scores[t, :nk], int(e[t]), k, int(s0[t]))
    return out_i, out_s


def indexer_topk(q: np.ndarray, q_dtype: str, q_scale: Optional[np.ndarray], w: Optional[np.ndarray],
                 keys: np.ndarray, k_scale: Optional[np.ndarray], k: int, mode: str = "dsa",
                 causal_offsets: Optional[np.ndarray] = None, rows: Optional[Sequence[int]] = None,
                 return_scores: bool = False, visible_start: Optional[np.ndarray] = None):
    """Fused operation, defined plainly: Eq. (1) scores for the visible keys of
    each requested row, then the exact top-k of Eq. (2).

    q [Nq, H, d] and keys [Nk, d] in storage form (float32 / uint16 bf16 bits /
    uint8 E4M3FN bits, all with the same ``q_dtype``); q_scale [Nq, H] and
    k_scale [Nk] for fp8; w [Nq, H] float32 or None. Returns (idx, scores)
    [len(rows), k], plus the full per-row float32 score rows when
    ``return_scores``."""
    nq, nk = q.shape[0], keys.shape[0]
    rows = list(range(nq)) if rows is None else list(rows)
    s0, e = visible_ranges(causal_offsets, visible_start, nq, nk)
    kd = dequantize(keys, q_dtype, k_scale)
    wd = None if w is None else np.asarray(w, dtype=np.float32).astype(np.float64)
    out_i = np.empty((len(rows), k), dtype=np.int32)
    out_s = np.empty((len(rows), k), dtype=np.float32)
    full = []
    for i, t in enumerate(rows):
        qd = dequantize(q[t], q_dtype, None if q_scale is None else q_scale[t])
        # scores of the visible keys [s_t, e_t) only; full rows keep zeros
        # before s_t so that row[j] is key j's score
        vis = row_scores(qd, None if wd is None else wd[t], kd[s0[t]: e[t]], mode)
        sr = np.zeros(int(e[t]), dtype=np.float32)
        sr[s0[t]:] = vis
        out_i[i], out_s[i] = select_row(sr, int(e[t]), k, int(s0[t]))
        if return_scores:
            full.append(sr)
    if return_scores:
        return out_i, out_s, full
    return out_i, out_s


def sample_from_topk(prev_idx: np.ndarray, num_keys: int, sample_size: int) -> np.ndarray:
    """Previous-chunk sample, sec. 3.2 "Sampling": count how often every key
    in [0, num_keys) occurs in the previous chunk's top-k lists (entries
    outside that range, such as the -1 padding, are not keys), rank keys by
    (count desc, key asc), keep the first ``sample_size`` of them that occur
    at least once, and return them ascending, padded with -1 to
    ``sample_size`` (int32)."""
    v = np.asarray(prev_idx, dtype=np.int64).ravel()
    v = v[(v >= 0) & (v < num_keys)]
    counts = np.bincount(v, minlength=num_keys)
    rank = np.lexsort((np.arange(num_keys), -counts))
    chosen = rank[:sample_size]
    chosen = np.sort(chosen[counts[chosen] >= 1])
    out = np.full(sample_size, -1, dtype=np.int32)
    out[: chosen.size] = chosen
    return out


def dsa_union(topk_idx: np.ndarray, group: int):
    """LiteDSA union, sec. 3.3. topk_idx [Nq, k] (negative entries are
    padding). For each group of ``group`` consecutive rows (the last may be
    shorter): the ascending list of distinct keys in any of its rows, and per
    row the slots of that list holding the row's keys. Returns (union_idx
    [G, group * k] int32 padded with -1, union_count [G] int32, member_mask
    [Nq, W] uint32 with W = ceil(group * k / 32), bit j % 32 of word j // 32
    for slot j)."""
    idx = np.asarray(topk_idx, dtype=np.int64)
    nq, k = idx.shape
    n = group * k
    ngroups = -(-nq // group)
    words = -(-n // 32)
    union_idx = np.full((ngroups, n), -1, dtype=np.int32)
    union_count = np.zeros(ngroups, dtype=np.int32)
    mask = np.zeros((nq, words), dtype=np.uint32)
    for g in range(ngroups):
        rows = range(g * group, min(nq, (g + 1) * group))
        keys = sorted({int(v) for t in rows for v in idx[t] if v >= 0})
        union_idx[g, : len(keys)] = keys
        union_count[g] = len(keys)
        slot = {key: j for j, key in enumerate(keys)}
        for t in rows:
            for v in {int(v) for v in idx[t] if v >= 0}:
                j = slot[v]
                mask[t, j // 32] |= np.uint32(1 << (j % 32))
    return union_idx, union_count, mask
