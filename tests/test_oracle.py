"""Pins for the CPU oracle, against facts fixed by the paper's definitions and
by mathematics rather than by the oracle itself:

* brute force over all k-subsets on tiny rows (Eq. 2 plus the tie order);
* an independent repeated-argmax selector on many random rows with ties,
  NaN, +-0 and +-inf;
* exact rational evaluation of Eq. (1) by pure-Python loops on small inputs;
* closed forms (a ramp whose top-k is the last k visible keys; one-hot head
  weights that reduce Eq. (1) to one head's ReLU'd dot product);
* the storage formats decoded by torch, and the E4M3FN table of the OCP spec;
* a hand-worked example stored under tests/golden/.

The last test plants plausible mistakes in copies of the oracle's score
function and checks that the pins above catch every one of them.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# independent helpers (pure Python)
# --------------------------------------------------------------------------

def rank_key(v, i):
    """Larger is better: real values above NaN, higher value first, lower index
    first on ties. Python's float comparison already has -0.0 == 0.0."""
    v = float(v)
    if math.isnan(v):
        return (0, 0.0, -i)
    return (1, v, -i)


def brute_topk(row, k):
    n = len(row)
    kk = min(k, n)
    winners = []
    for sub in itertools.combinations(range(n), kk):
        s = set(sub)
        rest = [u for u in range(n) if u not in s]
        if all(rank_key(row[a], a) > rank_key(row[b], b) for a in s for b in rest):
            winners.append(sub)
    assert len(winners) == 1, "the total order must make the top-k unique"
    chosen = sorted(winners[0], key=lambda i: rank_key(row[i], i), reverse=True)
    return chosen


def argmax_topk(row, k):
    remaining = list(range(len(row)))
    out = []
    for _ in range(min(k, len(row))):
        best = remaining[0]
        for i in remaining[1:]:
            if rank_key(row[i], i) > rank_key(row[best], best):
                best = i
        out.append(best)
        remaining.remove(best)
    return out


def exact_score(qrow, wrow, keys_rows, mode):
    """Eq. (1) in exact rational arithmetic, pure-Python loops."""
    H, d = len(qrow), len(qrow[0])
    res = []
    for krow in keys_rows:
        tot = Fraction(0)
        for j in range(H):
            dot = Fraction(0)
            for i in range(d):
                dot += Fraction(float(qrow[j][i])) * Fraction(float(krow[i]))
            if mode == "dsa" and dot < 0:
                dot = Fraction(0)
            wj = Fraction(1) if wrow is None else Fraction(float(wrow[j]))
            tot += wj * dot
        res.append(tot)
    return res


def special_row(rng, n):
    pool = [np.nan, np.inf, -np.inf, 0.0, -0.0, 1.0, -1.0, 0.5, 2.0]
    row = rng.standard_normal(n).astype(np.float32)
    for i in range(n):
        u = rng.random()
        if u < 0.35:
            row[i] = pool[rng.integers(len(pool))]
        elif u < 0.55:
            row[i] = np.float32(np.round(row[i] * 2) / 2)
    return row


# --------------------------------------------------------------------------
# selection (Eq. 2)
# --------------------------------------------------------------------------

def test_select_matches_brute_force_on_tiny_rows():
    rng = np.random.default_rng(7)
    for trial in range(300):
        n = int(rng.integers(1, 9))
        k = int(rng.integers(1, n + 3))
        row = special_row(rng, n)
        e = n
        idx, sc = orc.select_row(row, e, k)
        want = brute_topk(row, k)
        assert list(idx[: len(want)]) == want
        assert np.all(idx[len(want):] == -1)
        assert np.all(np.isneginf(sc[len(want):]))
        np.testing.assert_array_equal(sc[: len(want)].view(np.uint32), row[want].view(np.uint32))


def test_select_matches_repeated_argmax():
    rng = np.random.default_rng(11)
    for trial in range(400):
        n = int(rng.integers(1, 60))
        e = int(rng.integers(0, n + 1))
        k = int(rng.integers(1, 70))
        row = special_row(rng, n)
        idx, _ = orc.select_row(row, e, k)
        want = argmax_topk(row[:e], k)
        assert list(idx[: len(want)]) == want
        assert np.all(idx[len(want):] == -1)


def test_select_invariants_random_rows():
    rng = np.random.default_rng(3)
    for trial in range(50):
        n = int(rng.integers(1, 5000))
        e = int(rng.integers(0, n + 1))
        k = int(rng.integers(1, 600))
        row = np.round(rng.standard_normal(n) * 4).astype(np.float32) / np.float32(4)
        idx, sc = orc.select_row(row, e, k)
        m = min(k, e)
        sel = idx[:m]
        assert len(set(sel.tolist())) == m                  # unique
        assert np.all((sel >= 0) & (sel < e))               # visible
        assert np.all(idx[m:] == -1) and np.all(np.isneginf(sc[m:]))
        np.testing.assert_array_equal(sc[:m], row[sel])
        if 0 < m < e:
            mask = np.ones(e, bool)
            mask[sel] = False
            assert sc[:m].min() >= row[:e][mask].max()       # dominance
            # ties at the boundary go to the lower index
            kth = sc[m - 1]
            left = np.nonzero(mask & (row[:e] == kth))[0]
            chosen = sel[sc[:m] == kth]
            if left.size:
                assert chosen.max() < left.min()


def test_select_zero_and_nan_semantics():
    row = np.array([-0.0, 0.0, np.nan, -np.inf, np.inf, np.nan], dtype=np.float32)
    idx, sc = orc.select_row(row, 6, 6)
    assert idx.tolist() == [4, 0, 1, 3, 2, 5]   # -0 == +0 (index order), NaN last
    idx, _ = orc.select_row(row, 6, 1)
    assert idx.tolist() == [4]


def test_topk_select_rows_and_offsets():
    s = workloads.score_rows(5, 300, seed=1, kind="ties", ld=320).numpy()
    s[4] = s[3]
    offs = np.array([0, 1, 299, 300, 1000], dtype=np.int32)
    idx, sc = orc.topk_select(s, 300, 16, offs)
    assert np.all(idx[0] == -1)
    assert idx[1, 0] == 0 and np.all(idx[1, 1:] == -1)
    for t in (2, 3, 4):
        e = min(300, offs[t])
        assert idx[t].max() < e
    np.testing.assert_array_equal(idx[3], idx[4])   # offsets beyond Nk clamp to Nk


# --------------------------------------------------------------------------
# scores (Eq. 1)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("mode", ["dsa", "ip"])
def test_scores_exact_rational_small(mode):
    rng = np.random.default_rng(5 if mode == "dsa" else 6)
    for trial in range(20):
        H, d, n = int(rng.integers(1, 5)), int(rng.integers(1, 7)), int(rng.integers(1, 9))
        q = rng.integers(-4, 5, size=(H, d)).astype(np.float64)
        keys = rng.integers(-4, 5, size=(n, d)).astype(np.float64)
        w = (2.0 ** rng.integers(-3, 3, size=H)) * rng.choice([1.0, -1.0], size=H)
        got = orc.row_scores(q, w, keys, mode)
        want = exact_score(q, w, keys, mode)
        assert got.dtype == np.float32
        for g, x in zip(got, want):
            assert Fraction(float(g)) == x   # every value here is exact in float32


def test_scores_real_inputs_within_one_rounding():
    rng = np.random.default_rng(9)
    H, d, n = 3, 5, 11
    q = rng.standard_normal((H, d)).astype(np.float32).astype(np.float64)
    keys = rng.standard_normal((n, d)).astype(np.float32).astype(np.float64)
    w = rng.random(H).astype(np.float32).astype(np.float64)
    got = orc.row_scores(q, w, keys, "dsa")
    want = exact_score(q, w, keys, "dsa")
    for g, x in zip(got, want):
        # float64 evaluation then one rounding: within one float32 ulp of exact
        ulp = np.spacing(np.float32(abs(float(x)))) if x != 0 else np.float32(1e-45)
        assert abs(Fraction(float(g)) - x) <= Fraction(float(ulp))


def test_ramp_closed_form_top_k_is_last_visible_keys():
    # q_{t,j} = u and k_s = (s+1) u with w >= 0 give
    # I[t,s] = (sum_j w_j) (s+1) |u|^2, increasing in s.
    rng = np.random.default_rng(2)
    H, d, nk, nq, k = 4, 8, 300, 6, 37
    u = rng.integers(1, 3, size=d).astype(np.float32)
    q = np.broadcast_to(u, (nq, H, d)).astype(np.float32).copy()
    keys = (np.arange(1, nk + 1, dtype=np.float32)[:, None] * u[None, :]).astype(np.float32)
    w = rng.random((nq, H)).astype(np.float32)
    offs = np.array([300, 299, 150, 37, 10, 0], dtype=np.int32)
    idx, sc = orc.indexer_topk(q, "f32", None, w, keys, None, k, "dsa", offs)
    for t in range(nq):
        e = offs[t]
        m = min(k, e)
        assert idx[t, :m].tolist() == list(range(e - 1, e - 1 - m, -1))
        want = np.float64(w[t].astype(np.float64).sum()) * np.arange(e, e - m, -1) * float(u @ u)
        np.testing.assert_allclose(sc[t, :m], want, rtol=1e-6)


def test_ramp_closed_form_with_visible_starts():
    # the ramp above with per-row starts: the top-k is the last min(k, e - s)
    # keys of [s, e), i.e. e-1 down to max(s, e-k)
    rng = np.random.default_rng(12)
    H, d, nk, nq, k = 4, 8, 300, 7, 37
    u = rng.integers(1, 3, size=d).astype(np.float32)
    q = np.broadcast_to(u, (nq, H, d)).astype(np.float32).copy()
    keys = (np.arange(1, nk + 1, dtype=np.float32)[:, None] * u[None, :]).astype(np.float32)
    w = rng.random((nq, H)).astype(np.float32)
    offs = np.array([300, 299, 150, 37, 10, 0, 200], dtype=np.int32)
    starts = np.array([0, 280, 100, 30, 20, -5, 199], dtype=np.int32)
    idx, sc = orc.indexer_topk(q, "f32", None, w, keys, None, k, "dsa", offs, visible_start=starts)
    for t in range(nq):
        e = int(offs[t])
        s = min(max(int(starts[t]), 0), e)
        m = min(k, e - s)
        assert idx[t, :m].tolist() == list(range(e - 1, e - 1 - m, -1)), t
        assert np.all(idx[t, m:] == -1)


def test_select_with_starts_matches_brute_force():
    rng = np.random.default_rng(17)
    for trial in range(200):
        n = int(rng.integers(1, 10))
        row = special_row(rng, n)
        e = int(rng.integers(0, n + 1))
        s = int(rng.integers(0, e + 1))
        k = int(rng.integers(1, n + 2))
        idx, sc = orc.select_row(row, e, k, s)
        want = [j + s for j in brute_topk(row[s:e], k)] if e > s else []
        assert list(idx[: len(want)]) == want
        assert np.all(idx[len(want):] == -1)


def test_packed_sequences_equal_separate_sequences():
    # keys of three sequences packed into one array, each query seeing only
    # its own sequence (start = the sequence's base): the result is each
    # sequence computed alone, with indices shifted by the base
    rng = np.random.default_rng(21)
    H, d, k = 4, 16, 20
    lens = [50, 120, 33]
    nqs = [5, 7, 4]
    bases = np.cumsum([0] + lens[:-1])
    keys = rng.standard_normal((sum(lens), d)).astype(np.float32)
    qs = [rng.standard_normal((n, H, d)).astype(np.float32) for n in nqs]
    ws = [rng.random((n, H)).astype(np.float32) for n in nqs]
    q = np.concatenate(qs)
    w = np.concatenate(ws)
    ends, starts = [], []
    for b, (L, n) in enumerate(zip(lens, nqs)):
        e_local = L - n + np.arange(n) + 1
        ends.append(bases[b] + e_local)
        starts.append(np.full(n, bases[b]))
    ends = np.concatenate(ends).astype(np.int32)
    starts = np.concatenate(starts).astype(np.int32)
    pi, ps = orc.indexer_topk(q, "f32", None, w, keys, None, k, "dsa", ends, visible_start=starts)
    r = 0
    for b, (L, n) in enumerate(zip(lens, nqs)):
        kb = keys[bases[b]: bases[b] + L]
        si, ss = orc.indexer_topk(qs[b], "f32", None, ws[b], kb, None, k, "dsa", L - n + np.arange(n) + 1)
        want = np.where(si >= 0, si + bases[b], -1)
        np.testing.assert_array_equal(pi[r: r + n], want)
        np.testing.assert_array_equal(ps[r: r + n].view(np.uint32), ss.view(np.uint32))
        r += n


def test_one_hot_weights_reduce_to_one_head():
    rng = np.random.default_rng(4)
    H, d, n = 5, 16, 40
    q = rng.standard_normal((H, d)).astype(np.float32).astype(np.float64)
    keys = rng.standard_normal((n, d)).astype(np.float32).astype(np.float64)
    for j in range(H):
        w = np.zeros(H)
        w[j] = 1.0
        got = orc.row_scores(q, w, keys, "dsa")
        x = np.array([sum(q[j, i] * keys[s, i] for i in range(d)) for s in range(n)])
        np.testing.assert_array_equal(got, np.maximum(x, 0).astype(np.float32))
        assert np.all(got >= 0)


def test_ip_mode_single_head_is_plain_dot_product():
    rng = np.random.default_rng(8)
    q = rng.standard_normal((1, 7)).astype(np.float32).astype(np.float64)
    keys = rng.standard_normal((9, 7)).astype(np.float32).astype(np.float64)
    got = orc.row_scores(q, None, keys, "ip")
    assert np.any(got < 0)   # no ReLU in inner-product mode
    want = exact_score(q, None, keys, "ip")
    for g, x in zip(got, want):
        assert abs(Fraction(float(g)) - x) <= Fraction(float(np.spacing(np.float32(abs(float(x))))))


# --------------------------------------------------------------------------
# storage formats
# --------------------------------------------------------------------------

def test_e4m3fn_spec_table():
    table = {0x00: 0.0, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9, 0x08: 2.0 ** -6, 0x38: 1.0,
             0x3C: 1.5, 0x40: 2.0, 0x7E: 448.0, 0xFE: -448.0, 0xB8: -1.0, 0x77: 240.0}
    for b, v in table.items():
        assert orc.e4m3fn_to_f64(np.array([b], np.uint8))[0] == v
    assert np.isnan(orc.e4m3fn_to_f64(np.array([0x7F, 0xFF], np.uint8))).all()
    neg0 = orc.e4m3fn_to_f64(np.array([0x80], np.uint8))[0]
    assert neg0 == 0.0 and math.copysign(1.0, neg0) < 0


def test_e4m3fn_all_codes_match_torch():
    b = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = b.view(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)
    got = orc.e4m3fn_to_f64(b.numpy())
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(got[ok], ref[ok])


def test_bf16_all_codes_match_torch():
    b = torch.arange(65536, dtype=torch.int32).to(torch.int16).view(torch.bfloat16)
    ref = b.to(torch.float32).numpy().astype(np.float64)
    got = orc.bf16_to_f64(b.view(torch.int16).numpy().view(np.uint16))
    np.testing.assert_array_equal(np.isnan(got), np.isnan(ref))
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(got[ok], ref[ok])


def test_fp8_scaled_scores_exact():
    # fp8 payloads decoded by torch, scales applied in exact rationals.
    rng = np.random.default_rng(12)
    H, d, n = 3, 6, 8
    qb = rng.integers(0, 256, size=(H, d)).astype(np.uint8)
    kb = rng.integers(0, 256, size=(n, d)).astype(np.uint8)
    qb[(qb & 0x7F) == 0x7F] = 0x38
    kb[(kb & 0x7F) == 0x7F] = 0x38
    qs = (2.0 ** rng.integers(-4, 4, size=H)).astype(np.float32) * np.float32(1.25)
    ks = (2.0 ** rng.integers(-4, 4, size=n)).astype(np.float32) * np.float32(0.75)
    w = rng.random(H).astype(np.float32)
    tq = torch.from_numpy(qb).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    tk = torch.from_numpy(kb).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    qv = [[Fraction(float(tq[j, i])) * Fraction(float(qs[j])) for i in range(d)] for j in range(H)]
    kv = [[Fraction(float(tk[s, i])) * Fraction(float(ks[s])) for i in range(d)] for s in range(n)]
    idx, sc, full = orc.indexer_topk(qb[None], "fp8", qs[None], w[None], kb, ks, n, "dsa", None,
                                     return_scores=True)
    for s in range(n):
        tot = Fraction(0)
        for j in range(H):
            dot = sum((qv[j][i] * kv[s][i] for i in range(d)), Fraction(0))
            tot += Fraction(float(w[j])) * max(dot, Fraction(0))
        g = Fraction(float(full[0][s]))
        ulp = Fraction(float(np.spacing(np.float32(abs(float(tot)))))) if tot else Fraction(0)
        assert abs(g - tot) <= ulp


def test_visible_counts_clamp():
    e = orc.visible_counts(np.array([-5, 0, 3, 10, 11], np.int32), 5, 10)
    assert e.tolist() == [0, 0, 3, 10, 10]
    assert orc.visible_counts(None, 3, 7).tolist() == [7, 7, 7]


# --------------------------------------------------------------------------
# hand-worked example (tests/golden)
# --------------------------------------------------------------------------

def test_golden_hand_worked_example():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        g = json.load(f)
    q = np.array(g["q"], dtype=np.float32)
    w = np.array(g["w"], dtype=np.float32)
    keys = np.array(g["keys"], dtype=np.float32)
    offs = np.array(g["causal_offsets"], dtype=np.int32)
    s = orc.index_scores(q.astype(np.float64), w.astype(np.float64), keys.astype(np.float64), "dsa")
    np.testing.assert_array_equal(s, np.array(g["scores"], dtype=np.float32))
    idx, sc = orc.indexer_topk(q, "f32", None, w, keys, None, g["k"], "dsa", offs)
    assert idx.tolist() == g["topk_idx"]
    np.testing.assert_array_equal(sc, np.array(g["topk_scores"], dtype=np.float32))


# --------------------------------------------------------------------------
# the pins catch planted mistakes
# --------------------------------------------------------------------------

def _planted_variants():
    def dropped_relu(q, w, keys, mode):
        x = q @ keys.T
        return ((np.ones(q.shape[0]) if w is None else w) @ x).astype(np.float32)

    def relu_on_query(q, w, keys, mode):     # the misplaced ReLU of Eq. (3)
        x = np.maximum(q, 0) @ keys.T
        return ((np.ones(q.shape[0]) if w is None else w) @ x).astype(np.float32)

    def dropped_last_head(q, w, keys, mode):
        x = np.maximum(q[:-1] @ keys.T, 0)
        return ((np.ones(q.shape[0]) if w is None else w)[:-1] @ x).astype(np.float32)

    def unweighted(q, w, keys, mode):
        return np.maximum(q @ keys.T, 0).sum(0).astype(np.float32)

    def wrong_sign(q, w, keys, mode):
        x = np.maximum(-(q @ keys.T), 0)
        return ((np.ones(q.shape[0]) if w is None else w) @ x).astype(np.float32)

    def dropped_last_dim(q, w, keys, mode):
        x = np.maximum(q[:, :-1] @ keys[:, :-1].T, 0)
        return ((np.ones(q.shape[0]) if w is None else w) @ x).astype(np.float32)

    return [dropped_relu, relu_on_query, dropped_last_head, unweighted, wrong_sign, dropped_last_dim]


@pytest.mark.parametrize("variant", _planted_variants(), ids=lambda f: f.__name__)
def test_pins_catch_planted_score_mistakes(variant, monkeypatch):
    monkeypatch.setattr(orc, "row_scores", variant)
    with pytest.raises(AssertionError):
        test_scores_exact_rational_small("dsa")
        test_one_hot_weights_reduce_to_one_head()
        test_golden_hand_worked_example()


def test_pins_catch_planted_selection_mistakes(monkeypatch):
    def ascending(scores):
        s = np.asarray(scores, dtype=np.float32).astype(np.float64)
        return np.lexsort((np.arange(s.size), np.where(np.isnan(s), 0.0, s), np.isnan(s)))

    def ties_high_index(scores):
        s = np.asarray(scores, dtype=np.float32).astype(np.float64)
        return np.lexsort((-np.arange(s.size), np.where(np.isnan(s), 0.0, -s), np.isnan(s)))

    def nan_first(scores):
        s = np.asarray(scores, dtype=np.float32).astype(np.float64)
        return np.lexsort((np.arange(s.size), np.where(np.isnan(s), 0.0, -s), ~np.isnan(s)))

    for bad in (ascending, ties_high_index, nan_first):
        monkeypatch.setattr(orc, "order", bad)
        with pytest.raises(AssertionError):
            test_select_matches_brute_force_on_tiny_rows()


# --------------------------------------------------------------------------
# previous-chunk sample (sec. 3.2 "Sampling")
# --------------------------------------------------------------------------

def test_golden_previous_chunk_sample():
    with open(os.path.join(GOLDEN, "sample_from_topk.json")) as f:
        g = json.load(f)
    prev = np.array(g["prev_idx"], dtype=np.int32)
    for case in g["cases"]:
        got = orc.sample_from_topk(prev, g["num_keys"], case["sample_size"])
        assert got.dtype == np.int32
        assert got.tolist() == case["sample"]


def _occurrences(prev, nk):
    c = {}
    for v in np.asarray(prev).ravel().tolist():
        if 0 <= v < nk:
            c[v] = c.get(v, 0) + 1
    return c


def check_sample_invariants(out, prev, nk, ns):
    """What fixes the previous-chunk sample uniquely: its size, ascending
    distinct keys that occur, and dominance -- every sampled key ranks above
    every key left out under (count desc, key asc)."""
    c = _occurrences(prev, nk)
    assert out.dtype == np.int32 and out.shape == (ns,)
    n = min(ns, len(c))
    sel = out[:n].tolist()
    assert np.all(out[n:] == -1)
    assert sel == sorted(set(sel)) and all(s >= 0 for s in sel)
    assert all(c.get(s, 0) >= 1 for s in sel)
    left = set(c) - set(sel)
    if sel and left:
        worst_in = min((c[s], -s) for s in sel)
        best_out = max((c[u], -u) for u in left)
        assert worst_in > best_out


SAMPLE_CASES = [
    # rows, k, num_keys, sample_size, law
    (8, 16, 50, 20, "zipf"),
    (8, 16, 50, 200, "zipf"),
    (32, 64, 5000, 300, "zipf"),
    (16, 32, 400, 64, "uniform"),
    (5, 7, 30, 3, "dirty"),
    (0, 4, 30, 5, "zipf"),
    (3, 5, 4, 10, "dirty"),
]


def sample_case_input(rows, k, nk, law, seed):
    rng = np.random.default_rng(seed)
    if law == "uniform":
        p = rng.integers(0, nk, size=(rows, k))
    else:
        p = np.minimum(rng.zipf(1.3, size=(rows, k)) - 1, nk - 1)
    p = p.astype(np.int32)
    if law == "dirty" and p.size:
        m = rng.random(p.shape)
        p[m < 0.15] = -1
        p[(m >= 0.15) & (m < 0.25)] = nk + 3
    return p


@pytest.mark.parametrize("case", SAMPLE_CASES, ids=[f"{c[0]}x{c[1]}-nk{c[2]}-ns{c[3]}-{c[4]}" for c in SAMPLE_CASES])
def test_previous_chunk_sample_invariants(case):
    rows, k, nk, ns, law = case
    prev = sample_case_input(rows, k, nk, law, seed=rows * 31 + nk)
    check_sample_invariants(orc.sample_from_topk(prev, nk, ns), prev, nk, ns)


def test_pins_catch_planted_sample_mistakes(monkeypatch):
    good = orc.sample_from_topk

    def ties_high_key(prev, nk, ns):
        v = np.asarray(prev, dtype=np.int64).ravel()
        v = v[(v >= 0) & (v < nk)]
        c = np.bincount(v, minlength=nk)
        r = np.lexsort((-np.arange(nk), -c))[:ns]
        r = np.sort(r[c[r] >= 1])
        out = np.full(ns, -1, np.int32)
        out[: r.size] = r
        return out

    def zero_counts_kept(prev, nk, ns):
        v = np.asarray(prev, dtype=np.int64).ravel()
        v = v[(v >= 0) & (v < nk)]
        c = np.bincount(v, minlength=nk)
        r = np.sort(np.lexsort((np.arange(nk), -c))[:ns])
        out = np.full(ns, -1, np.int32)
        out[: r.size] = r
        return out

    def padding_counted(prev, nk, ns):
        p = np.where(np.asarray(prev) < 0, 0, prev)
        return good(p, nk, ns)

    def unsorted(prev, nk, ns):
        out = good(prev, nk, ns)
        n = int((out >= 0).sum())
        out[:n] = out[:n][::-1].copy()
        return out

    for bad in (ties_high_key, zero_counts_kept, padding_counted, unsorted):
        monkeypatch.setattr(orc, "sample_from_topk", bad)
        with pytest.raises(AssertionError):
            test_golden_previous_chunk_sample()
            for case in SAMPLE_CASES:
                test_previous_chunk_sample_invariants(case)


# --------------------------------------------------------------------------
# LiteDSA union and membership masks (sec. 3.3)
# --------------------------------------------------------------------------

def test_golden_dsa_union():
    with open(os.path.join(GOLDEN, "dsa_union.json")) as f:
        g = json.load(f)
    u, c, m = orc.dsa_union(np.array(g["topk_idx"], dtype=np.int32), g["group"])
    assert u.tolist() == g["union_idx"]
    assert c.tolist() == g["union_count"]
    assert m.astype(np.int64).tolist() == g["member_mask"]


def check_union_invariants(u, c, m, idx, group):
    """What fixes the union uniquely: per group, the listed keys are exactly
    the set of keys of its rows, ascending and distinct, then -1; and each
    row's mask decodes (through that list) to exactly its own key set."""
    idx = np.asarray(idx)
    nq, k = idx.shape
    ng = -(-nq // group)
    assert u.shape == (ng, group * k) and c.shape == (ng,) and m.shape == (nq, -(-group * k // 32))
    for g in range(ng):
        rows = list(range(g * group, min(nq, (g + 1) * group)))
        want = set()
        for t in rows:
            want |= {int(v) for v in idx[t] if v >= 0}
        n = int(c[g])
        lst = [int(v) for v in u[g, :n]]
        assert lst == sorted(want) and len(lst) == len(set(lst))
        assert np.all(u[g, n:] == -1)
        for t in rows:
            bits = [j for j in range(group * k) if (int(m[t, j // 32]) >> (j % 32)) & 1]
            assert all(j < n for j in bits)
            assert {lst[j] for j in bits} == {int(v) for v in idx[t] if v >= 0}


UNION_CASES = [
    # nq, k, group, key range, padding fraction
    (10, 8, 3, 40, 0.2),
    (16, 16, 4, 1000, 0.0),
    (7, 5, 1, 20, 0.3),
    (9, 32, 16, 100, 0.1),
]


def union_case_input(nq, k, keys, pad, seed):
    rng = np.random.default_rng(seed)
    base = rng.integers(0, keys, size=k)
    idx = np.empty((nq, k), dtype=np.int32)
    for t in range(nq):  # neighbours share part of their keys, as in sparse attention
        own = rng.integers(0, keys, size=k)
        idx[t] = np.where(rng.random(k) < 0.5, base, own)
    idx[rng.random((nq, k)) < pad] = -1
    return idx


@pytest.mark.parametrize("case", UNION_CASES, ids=[f"{c[0]}x{c[1]}-g{c[2]}" for c in UNION_CASES])
def test_dsa_union_invariants(case):
    nq, k, group, keys, pad = case
    idx = union_case_input(nq, k, keys, pad, seed=nq * k + group)
    u, c, m = orc.dsa_union(idx, group)
    check_union_invariants(u, c, m, idx, group)


def test_pins_catch_planted_union_mistakes(monkeypatch):
    good = orc.dsa_union

    def descending(idx, group):
        u, c, m = good(idx, group)
        for g in range(len(c)):
            u[g, : c[g]] = u[g, : c[g]][::-1].copy()
        return u, c, m

    def slot_off_by_one(idx, group):
        u, c, m = good(idx, group)
        return u, c, (m.astype(np.uint64) << 1).astype(np.uint32)

    def padding_is_a_key(idx, group):
        return good(np.where(np.asarray(idx) < 0, 0, idx), group)

    def groups_shifted(idx, group):
        return good(np.asarray(idx)[1:], group)

    for bad in (descending, slot_off_by_one, padding_is_a_key, groups_shifted):
        monkeypatch.setattr(orc, "dsa_union", bad)
        with pytest.raises(Exception):
            test_golden_dsa_union()
            for case in UNION_CASES:
                test_dsa_union_invariants(case)
