"""GPU parity of the fused Indexer-TopK (lt_indexer_topk) against the oracle.

* real-valued inputs of every workload law, at sizes the oracle finishes in
  seconds (several query and key tiles, ragged tails): tolerance + swap rule;
* exact-arithmetic inputs: bit-exact sets and scores;
* internal consistency: the fused result equals lt_topk_select over the dense
  score matrix, bit for bit (same score arithmetic);
* forced fallback, tiny capacity, one bin, no sample: unchanged results;
* edge shapes: k = 1, rows shorter than k, empty rows, no mask.
"""
import numpy as np
import pytest
import torch

from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_topk, to_dev
from parity import RTOL, check_row_exact, check_row_tol, visible

pytestmark = pytest.mark.gpu


def _fused(x, k, mode="dsa", **opt):
    d = to_dev(x)
    nq = d["q"].shape[0]
    stats = torch.full((nq, lt.LT_ROW_STATS), -7, dtype=torch.int32, device="cuda")
    opts = lt.make_options(row_stats=stats, **opt)
    gi, gs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"], mode=mode,
                             options=opts)
    torch.cuda.synchronize()
    return gi.cpu().numpy(), gs.cpu().numpy(), stats.cpu().numpy()


def _check_tol(x, dtype, k, mode, gi, gs, rows=None):
    ri, rs, full = oracle_topk(x, dtype, k, mode, rows=rows)
    nq, nk = x["q"].shape[0], x["keys"].shape[0]
    e = visible(None if x["offsets"] is None else x["offsets"].numpy(), nq, nk)
    rows = range(nq) if rows is None else rows
    for i, t in enumerate(rows):
        check_row_tol(gi[t], gs[t], ri[i], rs[i], full[i], int(e[t]), k, RTOL[dtype])


LAWS = [
    # name, base config, nq, nk, k
    ("tiny_fp32_full", "tiny_fp32", None, None, None),
    ("dsa_bf16", "dsa_bf16_128k", 21, 20011, 2048),
    ("dsa_bf16_smallk", "dsa_bf16_128k", 19, 7000, 64),
    ("dsa_fp8", "dsa_fp8_1m", 17, 30001, 2048),
    ("adversarial_bf16", "adversarial_bf16_256k", 16, 40000, 2048),
    ("retrieval_bf16", "retrieval_bf16_4m", 70, 50000, 100),
    ("dsa_bf16_kmax", "dsa_bf16_128k", 10, 30000, 8192),     # the largest k (LT_K_MAX)
    ("dsa_fp8_kmax", "dsa_fp8_1m", 9, 25000, 8192),
]


@pytest.mark.parametrize("law", LAWS, ids=[l[0] for l in LAWS])
def test_fused_parity_real_inputs(lib, law):
    name, base, nq, nk, k = law
    cfg = workloads.CONFIGS[base]
    cfg = workloads.scaled(cfg, nq=nq, nk=nk) if nq else cfg
    k = cfg.k if k is None else k
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[base])
    gi, gs, stats = _fused(x, k, cfg.mode)
    _check_tol(x, cfg.dtype, k, cfg.mode, gi, gs)
    assert not np.any(stats[:, 2] == 4)


@pytest.mark.parametrize("dtype,h,d", [("f32", 4, 64), ("bf16", 64, 128), ("bf16", 4, 128), ("bf16", 1, 128),
                                       ("fp8", 64, 128)])
@pytest.mark.parametrize("sorted_out", [True, False])
def test_fused_exact_inputs_bit_exact(lib, dtype, h, d, sorted_out):
    nq, nk, k = 23, 3001, 200
    x = workloads.exact_inputs(nq, nk, h, d, dtype, seed=11)
    gi, gs, _ = _fused(x, k, "dsa", sorted_output=sorted_out)
    ri, rs, _ = oracle_topk(x, dtype, k, "dsa")
    e = visible(x["offsets"].numpy(), nq, nk)
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e[t]), k, sorted_out)


@pytest.mark.parametrize("base", ["dsa_bf16_128k", "dsa_fp8_1m", "tiny_fp32", "adversarial_bf16_256k"])
def test_fused_equals_select_over_dense_scores(lib, base):
    cfg = workloads.CONFIGS[base]
    cfg = workloads.scaled(cfg, nq=min(cfg.nq, 24), nk=min(cfg.nk, 25000))
    k = min(cfg.k, 1024)
    x = workloads.generate(cfg, seed=5)
    d = to_dev(x)
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=cfg.mode)
    si, ss = lt.topk_select(dense, k, causal_offsets=d["offsets"], options=lt.make_options(sorted_output=True))
    fi, fs, _ = _fused(x, k, cfg.mode, sorted_output=True)
    np.testing.assert_array_equal(fi, si.cpu().numpy())
    np.testing.assert_array_equal(fs.view(np.uint32), ss.cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("ns", [16384, 32768])
def test_long_sample_same_results(lib, ns):
    # samples of 16384 to 32768 keys (the range stage's wide blocks): results
    # equal the default sample's
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=10, nk=40000)
    k = 256
    x = workloads.generate(cfg, seed=21)
    ref = _fused(x, k, "dsa", sorted_output=True)
    got = _fused(x, k, "dsa", sorted_output=True, sample_size=ns)
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))
    _check_tol(x, "bf16", k, "dsa", got[0], got[1])
    assert np.all(got[2][:, 2] == 0)


@pytest.mark.parametrize("opt", [
    dict(force_fallback=True),
    dict(capacity=64),
    dict(num_bins=1),
    dict(sample_size=0),
    dict(key_splits=4),
    dict(num_bins=16, capacity=3000),
], ids=lambda o: ",".join(f"{a}={b}" for a, b in o.items()))
def test_fused_forced_paths_are_exact(lib, opt):
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=10, nk=9000)
    k = 256
    x = workloads.generate(cfg, seed=8)
    ref = _fused(x, k, "dsa", sorted_output=True)
    got = _fused(x, k, "dsa", sorted_output=True, **opt)
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))
    _check_tol(x, "bf16", k, "dsa", got[0], got[1])
    if opt.get("force_fallback"):
        assert np.all(got[2][:, 2] == 3)
    if opt.get("capacity") == 64:
        assert np.all(got[2][:, 2] == 1)


def test_fused_edge_shapes(lib):
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=13, nk=700)
    x = workloads.generate(cfg, seed=4)
    offs = np.array([0, 1, 2, 5, 63, 64, 65, 300, 699, 700, 800, -4, 511], dtype=np.int32)
    x["offsets"] = torch.from_numpy(offs)
    for k in (1, 3, 64, 512, 1000):
        gi, gs, _ = _fused(x, k, "dsa")
        _check_tol(x, "bf16", k, "dsa", gi, gs)
    x["offsets"] = None
    gi, gs, _ = _fused(x, 50, "dsa")
    _check_tol(x, "bf16", 50, "dsa", gi, gs)


def test_fused_deterministic(lib):
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=16, nk=20000)
    x = workloads.generate(cfg, seed=6)
    a = _fused(x, 512, "dsa")
    b = _fused(x, 512, "dsa")
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1].view(np.uint32), b[1].view(np.uint32))
    np.testing.assert_array_equal(a[2], b[2])


# The grouped filter (H <= 4: many queries per wave): key splits that share a
# threshold (up to 8) and splits that do not, bins past what a published byte
# holds, rows without a gate (every score passes: the in-place path), tiny
# lists (overflow and fallback), and the forced fallback -- every result the
# same, bit for bit, and within tolerance of the oracle.
GROUPED = [
    # id, base config, nq, nk, k, mode
    ("ip_bf16_h1", "retrieval_bf16_4m", 300, 50001, 100, "ip"),
    ("dsa_f32_h4", "tiny_fp32", 40, 9001, 256, "dsa"),
]


@pytest.mark.parametrize("opt", [
    dict(key_splits=2),
    dict(key_splits=5),
    dict(key_splits=8),
    dict(key_splits=12),
    dict(key_splits=6, num_bins=300),
    dict(sample_size=0),
    dict(key_splits=3, sample_size=0),
    dict(capacity=48),
    dict(force_fallback=True),
], ids=lambda o: ",".join(f"{a}={b}" for a, b in o.items()))
@pytest.mark.parametrize("law", GROUPED, ids=[g[0] for g in GROUPED])
def test_grouped_forced_paths_are_exact(lib, law, opt):
    name, base, nq, nk, k, mode = law
    cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
    x = workloads.generate(cfg, seed=12)
    ref = _fused(x, k, mode, sorted_output=True)
    got = _fused(x, k, mode, sorted_output=True, **opt)
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))
    _check_tol(x, cfg.dtype, k, mode, got[0], got[1])
    if opt.get("force_fallback"):
        assert np.all(got[2][:, 2] == 3)


@pytest.mark.parametrize("law", [
    # id, base config, nq, nk, k, mode
    ("dsa_bf16_h64", "dsa_bf16_128k", 10, 9000, 256, "dsa"),
    ("dsa_fp8_h64", "dsa_fp8_1m", 9, 30001, 2048, "dsa"),
    ("ip_bf16_h1", "retrieval_bf16_4m", 300, 50001, 100, "ip"),
    ("dsa_f32_h4", "tiny_fp32", 40, 9001, 256, "dsa"),
], ids=lambda l: l[0])
def test_overflow_second_filter_pass(lib, law):
    """Rows whose candidate buffer overflows but whose keys at or above the
    exact final bin fit in one list are finished by a second filter pass
    gated at that bin (row_stats reason 6): results bit-identical to the
    default launch, and within tolerance of the oracle. One key split. The
    capacity comes from a first launch: fewer than k keys lie above a row's
    final bin, so a row with k - 1 + (its threshold-bin count) <= capacity
    < (its candidate count) must take the second pass; the capacity is the
    value that makes the most rows do so. Other overflowed rows may take the
    second pass or the dense fallback; rows that fit take neither."""
    name, base, nq, nk, k, mode = law
    cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
    x = workloads.generate(cfg, seed=14)
    ref = _fused(x, k, mode, sorted_output=True, key_splits=1)
    need, cand = k - 1 + ref[2][:, 3].astype(np.int64), ref[2][:, 0].astype(np.int64)
    caps = np.unique(need)
    hits = [int(((need <= c) & (cand > c)).sum()) for c in caps]
    cap = int(caps[int(np.argmax(hits))])
    must = (need <= cap) & (cand > cap)
    assert must.sum() >= nq // 4, "too few rows would take the second pass (cap %d, candidates %s, need %s)" % (
        cap, cand, need)
    got = _fused(x, k, mode, sorted_output=True, key_splits=1, capacity=cap)
    np.testing.assert_array_equal(got[0], ref[0])
    np.testing.assert_array_equal(got[1].view(np.uint32), ref[1].view(np.uint32))
    reasons = got[2][:, 2]
    np.testing.assert_array_equal(reasons[cand <= cap], 0)
    np.testing.assert_array_equal(reasons[must], 6)
    assert np.all(np.isin(reasons[(cand > cap) & ~must], (1, 2, 6)))
    _check_tol(x, cfg.dtype, k, mode, got[0], got[1])


@pytest.mark.parametrize("law", [
    # id, base config, nq, boundary row b, k, capacity, mode
    ("dsa_bf16_h64", "dsa_bf16_128k", 600, 195, 400, 300, "dsa"),
    ("dsa_fp8_h64", "dsa_fp8_1m", 520, 99, 256, 200, "dsa"),
    ("ip_bf16_h1", "retrieval_bf16_4m", 700, 77, 300, 250, "ip"),
], ids=lambda l: l[0])
def test_dense_fallback_batches_rows_of_a_tile(lib, law):
    """More than 256 queued rows make the dense fallback take several queued
    rows of one query tile per pass (ceil(Nq / 256) of them). Causal rows see
    Nk - Nq + 1 + t keys, with Nk chosen so that rows t > b see more than the
    capacity: with k above the capacity those rows overflow and go to the
    dense fallback (reason 1), the others return every visible key, so the
    query tile around row b holds queued and unqueued rows together. Every
    row equals radix selection over the dense scores bit for bit (sorted),
    and evenly spaced rows meet the oracle."""
    name, base, nq, b, k, cap, mode = law
    nk = cap + nq - 1 - b
    assert nk % 4 == 0, "the dense score rows must stay 16-byte aligned"
    cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
    x = workloads.generate(cfg, seed=23)
    if x["offsets"] is None:
        x["offsets"] = torch.from_numpy(workloads.causal_offsets(nq, nk))
    gi, gs, st = _fused(x, k, mode, sorted_output=True, key_splits=1, capacity=cap)
    reasons = st[:, 2]
    np.testing.assert_array_equal(reasons, np.where(np.arange(nq) > b, 1, 0))
    d = to_dev(x)
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=mode)
    ri, rs = lt.topk_radix(dense, k, causal_offsets=d["offsets"], sorted_output=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gi, ri.cpu().numpy())
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32))
    rows = sorted(set(np.linspace(0, nq - 1, 24).round().astype(int).tolist()) | {b, b + 1})
    _check_tol(x, cfg.dtype, k, mode, gi, gs, rows=rows)


@pytest.mark.parametrize("sorted_out", [True, False], ids=["sorted", "unsorted"])
@pytest.mark.parametrize("law", [
    # id, base config, nq, nk, k, mode
    ("dsa_bf16_h64", "dsa_bf16_128k", 3, 262144, 2048, "dsa"),
    ("dsa_fp8_h64", "dsa_fp8_1m", 2, 1048576, 2048, "dsa"),
    ("ip_bf16_h1", "retrieval_bf16_4m", 5, 1000004, 100, "ip"),
    ("dsa_bf16_kmax", "dsa_bf16_128k", 3, 200000, 8192, "dsa"),     # k = LT_K_MAX, chunks shorter than k
], ids=lambda l: l[0])
def test_dense_fallback_splits_few_rows_over_blocks(lib, law, sorted_out):
    """A few queued rows at a large Nk: the dense fallback cuts each row's
    visible keys into chunks re-scored by different blocks, and the block that
    scores a row's last chunk selects the row. Forced fallback on rows of
    different lengths (the whole context, about half of it, none, fewer keys
    than k, all but 77): every row equals radix selection over the dense
    scores bit for bit (sorted output; unsorted: the same set and scores), and
    the non-empty rows meet the oracle."""
    name, base, nq, nk, k, mode = law
    assert nk % 4 == 0, "the dense score rows must stay 16-byte aligned"
    cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
    x = workloads.generate(cfg, seed=29)
    offs = np.array([nk, nk // 2 + 3, 0, k - 5, nk - 77], dtype=np.int32)[:nq]
    x["offsets"] = torch.from_numpy(offs)
    gi, gs, st = _fused(x, k, mode, sorted_output=sorted_out, force_fallback=True)
    np.testing.assert_array_equal(st[:, 2], 3)
    d = to_dev(x)
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=mode)
    ri, rs = lt.topk_radix(dense, k, causal_offsets=d["offsets"], sorted_output=True)
    torch.cuda.synchronize()
    ri, rs = ri.cpu().numpy(), rs.cpu().numpy()
    e = visible(offs, nq, nk)
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e[t]), k, sorted_out)
    rows = [t for t in range(nq) if e[t] > 0][:2]
    _check_tol(x, cfg.dtype, k, mode, gi, gs, rows=rows)


@pytest.mark.parametrize("base,nq,nk", [("dsa_bf16_128k", 128, 16384), ("dsa_bf16_128k", 129, 16384),
                                        ("dsa_bf16_128k", 2304, 8192), ("dsa_fp8_1m", 300, 20000),
                                        ("tiny_fp32", 200, 9000)],
                         ids=["split_128_rows", "dense_129_rows", "whole_rows_2304", "dense_fp8_300_rows",
                              "dense_f32_h4_200_rows"])
def test_dense_fallback_mode_boundary(lib, base, nq, nk):
    """The fallback splits rows over blocks for up to 128 queued rows (two
    chunks each here); above that, while every row of the call has a scratch
    row of its own (here up to 2048 rows), it re-scores the queued rows'
    query tiles in (tile, key slice) items and selects each row in a block
    of its own; beyond, blocks take whole rows from the shared cursor. Each
    mode with every row forced, causal rows of different lengths, equal to
    radix selection over the dense scores bit for bit."""
    k = 300
    cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
    x = workloads.generate(cfg, seed=37)
    gi, gs, st = _fused(x, k, "dsa", sorted_output=True, force_fallback=True)
    np.testing.assert_array_equal(st[:, 2], 3)
    d = to_dev(x)
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode="dsa")
    ri, rs = lt.topk_radix(dense, k, causal_offsets=d["offsets"], sorted_output=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(gi, ri.cpu().numpy())
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32))
    _check_tol(x, cfg.dtype, k, "dsa", gi, gs, rows=[0, nq // 2, nq - 1])
