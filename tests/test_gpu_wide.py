"""The wide-vector scan: one head of 768-dimensional bf16 embeddings, the
paper's retrieval shapes (sec. 4.1 "Large-Scale Retrieval Benchmark"), where
all key splits of a row share one histogram and threshold bin (each split
keeps its own candidate list).

* real-valued inputs of that law (queries are corpus passages), several query
  tiles and ragged key tails, k from 1 to 8192: tolerance + swap rule against
  the oracle, and no row left to the fallback;
* exact-arithmetic inputs (integer entries, power-of-two weights, many equal
  scores): bit-exact sets and scores, sorted and unsorted output, inner
  product and ReLU scorers;
* internal consistency: the fused result equals plain radix selection over
  the dense score matrix of the same arithmetic, bit for bit;
* forced fallback, a capacity too small for the candidates, one bin, no
  sample, a caller's sample list, causal ends and packed starts;
* full size (slow): 64 queries x 5M passages at k = 128 and 8192, every row
  against radix selection over the dense scores and sampled rows against the
  oracle, in the benchmark's launch configuration.
"""
import numpy as np
import pytest
import torch

from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_topk, to_dev
from parity import RTOL, check_row_exact, check_row_tol, visible

pytestmark = pytest.mark.gpu

E7 = workloads.CONFIGS["retrieval_e7_bf16_5m"]


def _fused(x, k, mode="ip", **opt):
    d = to_dev(x)
    nq = d["q"].shape[0]
    stats = torch.full((nq, lt.LT_ROW_STATS), -7, dtype=torch.int32, device="cuda")
    gi, gs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], None, None, mode=mode,
                             options=lt.make_options(row_stats=stats, **opt))
    torch.cuda.synchronize()
    return gi.cpu().numpy(), gs.cpu().numpy(), stats.cpu().numpy()


def _sorted_pairs(idx, sc):
    """Rows sorted by the total order (score desc, -0 == +0, NaN last, index
    asc; padding last)."""
    nq, k = idx.shape
    row = np.repeat(np.arange(nq), k)
    i = idx.ravel().astype(np.int64)
    s = sc.ravel().astype(np.float64)
    nan = np.isnan(s) | (i < 0)
    key = np.where(nan, 0.0, -s) + 0.0
    o = np.lexsort((np.where(i < 0, 1 << 40, i), key, nan, row))
    return idx.ravel()[o].reshape(nq, k), sc.ravel()[o].reshape(nq, k)


CASES = [
    # nq, nk, k
    (64, 20000, 128),
    (64, 20011, 1024),
    (70, 33001, 4096),     # two query tiles, the second with 6 rows
    (3, 9000, 8192),       # most keys selected
    (1, 777, 1),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "nq%d-nk%d-k%d" % c)
def test_wide_parity_real_inputs(lib, case):
    nq, nk, k = case
    x = workloads.generate(workloads.scaled(E7, nq=nq, nk=nk), seed=nk + k)
    gi, gs, st = _fused(x, k)
    ri, rs, full = oracle_topk(x, "bf16", k, "ip")
    for t in range(nq):
        check_row_tol(gi[t], gs[t], ri[t], rs[t], full[t], nk, k, RTOL["bf16"])
    assert np.all(st[:, 2] == 0), "rows fell back: %s" % st[st[:, 2] != 0][:4]


@pytest.mark.parametrize("mode", ["ip", "dsa"])
@pytest.mark.parametrize("sorted_output", [False, True])
def test_wide_exact_inputs_bit_exact(lib, mode, sorted_output):
    nq, nk, k = 70, 3001, 700
    x = workloads.exact_inputs(nq, nk, 1, 768, "bf16", seed=5 + sorted_output, causal=True)
    gi, gs, _ = _fused(x, k, mode=mode, sorted_output=sorted_output)
    ri, rs, _ = oracle_topk(x, "bf16", k, mode)
    e = visible(x["offsets"].numpy(), nq, nk)
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e[t]), k, sorted_output)


@pytest.mark.parametrize("k", [64, 2048])
def test_wide_equals_radix_over_dense(lib, k):
    x = workloads.generate(workloads.scaled(E7, nq=100, nk=40000), seed=9)
    d = to_dev(x)
    fi, fs = lt.indexer_topk(d["q"], None, d["keys"], k, None, mode="ip")
    dense = lt.indexer_scores(d["q"], None, d["keys"], mode="ip")
    ri, rs = lt.topk_radix(dense, k, sorted_output=True)
    torch.cuda.synchronize()
    gi, gs = _sorted_pairs(fi.cpu().numpy(), fs.cpu().numpy())
    np.testing.assert_array_equal(gi, ri.cpu().numpy())
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32))


OPTION_CASES = [
    dict(flags_force=True),
    dict(capacity=8),            # overflows: exact fallback
    dict(num_bins=1),
    dict(sample_size=0),         # no gate at all
    dict(sample_size=50),        # loose initial gate
    dict(key_splits=3),
]


@pytest.mark.parametrize("opt", OPTION_CASES, ids=lambda o: "-".join("%s%s" % kv for kv in o.items()))
def test_wide_options_do_not_change_results(lib, opt):
    x = workloads.generate(workloads.scaled(E7, nq=66, nk=25000, causal=True), seed=12)
    k = 512
    base_i, base_s, _ = _fused(x, k, sorted_output=True)
    opt = dict(opt)
    if opt.pop("flags_force", False):
        opt["force_fallback"] = True
    gi, gs, st = _fused(x, k, sorted_output=True, **opt)
    np.testing.assert_array_equal(gi, base_i)
    np.testing.assert_array_equal(gs.view(np.uint32), base_s.view(np.uint32))
    if "capacity" in opt:
        assert np.all(st[:, 2] == 1), "an 8-slot list per split must overflow"
    ri, rs, full = oracle_topk(x, "bf16", k, "ip")
    e = visible(x["offsets"].numpy(), 66, 25000)
    for t in range(66):
        check_row_tol(gi[t], gs[t], ri[t], rs[t], full[t], int(e[t]), k, RTOL["bf16"])


def test_wide_sample_list_and_packed_rows(lib):
    lens, nqs, k = [12000, 30000, 7000], [20, 50, 9], 300
    x = workloads.packed_batch(workloads.scaled(E7, causal=True), lens, nqs, seed=4)
    d = to_dev(x)
    nk = sum(lens)
    # a caller's sample: every 7th key, some repeats and out-of-range entries
    lst = np.concatenate([np.arange(0, nk, 7), [5, 5, -3, nk + 10]]).astype(np.int32)
    gi, gs = lt.indexer_topk(d["q"], None, d["keys"], k, d["offsets"], mode="ip",
                             options=lt.make_options(sorted_output=True, visible_start=d["starts"],
                                                     sample_keys=torch.from_numpy(lst).cuda()))
    torch.cuda.synchronize()
    gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
    oi, os_, full = oracle_topk(x, "bf16", k, "ip")
    s0, e0 = orc.visible_ranges(x["offsets"].numpy(), x["starts"].numpy(), gi.shape[0], nk)
    for t in range(gi.shape[0]):
        v = gi[t][gi[t] >= 0]
        assert np.all((v >= s0[t]) & (v < e0[t])), "row %d: index outside its sequence" % t
        loc = lambda a: np.where(a >= 0, a - s0[t], -1)  # noqa: E731
        check_row_tol(loc(gi[t]), gs[t], loc(oi[t]), os_[t], full[t][s0[t]:], int(e0[t] - s0[t]), k,
                      RTOL["bf16"])


def test_wide_rows_shorter_than_k_and_empty(lib):
    nq, nk, k = 65, 2000, 1500
    x = workloads.generate(workloads.scaled(E7, nq=nq, nk=nk), seed=2)
    offs = np.linspace(-5, nk + 5, nq).round().astype(np.int32)   # empty rows, short rows, full rows
    x["offsets"] = torch.from_numpy(offs)
    gi, gs, _ = _fused(x, k)
    ri, rs, full = oracle_topk(x, "bf16", k, "ip")
    e = visible(offs, nq, nk)
    for t in range(nq):
        check_row_tol(gi[t], gs[t], ri[t], rs[t], full[t], int(e[t]), k, RTOL["bf16"])


@pytest.mark.parametrize("nk", [0, 5, 31, 33])
def test_wide_tiny_key_counts(lib, nk):
    """Fewer keys than one wave tile (or none): every visible key, sorted."""
    nq, k = 3, 40
    x = workloads.generate(workloads.scaled(E7, nq=nq, nk=max(nk, 1)), seed=7 + nk)
    if nk == 0:
        x["keys"] = x["keys"][:0].contiguous()
    gi, gs, st = _fused(x, k)
    if nk == 0:
        assert np.all(gi == -1) and np.all(np.isneginf(gs))
        return
    ri, rs, full = oracle_topk(x, "bf16", k, "ip")
    for t in range(nq):
        check_row_tol(gi[t], gs[t], ri[t], rs[t], full[t], nk, k, RTOL["bf16"])


def test_wide_all_scores_equal_goes_to_fallback(lib):
    """Every key identical: every key passes every gate and the threshold bin
    holds all of them, so every row takes the exact fallback (list overflow or
    threshold-bin overflow), and equal scores go to the lowest key indices."""
    nq, nk, k = 66, 20000, 100
    x = workloads.generate(workloads.scaled(E7, nq=nq, nk=nk), seed=21)
    x["keys"] = x["keys"][:1].repeat(nk, 1).contiguous()
    gi, gs, st = _fused(x, k, sorted_output=True)
    assert np.all((st[:, 2] == 1) | (st[:, 2] == 2)), "expected an overflow: %s" % st[:4]
    ri, rs, _ = oracle_topk(x, "bf16", k, "ip")
    np.testing.assert_array_equal(gi, ri)
    np.testing.assert_array_equal(gi, np.tile(np.arange(k, dtype=np.int32), (nq, 1)))
    for t in range(nq):
        assert np.all(np.abs(gs[t].astype(np.float64) - rs[t]) <= 1e-3 * np.abs(rs[t]).max())


def _oracle_rows_chunked(q_bits, keys_dev, rows, k, chunk=1 << 19):
    """The oracle's scores and top-k of a few rows over a corpus too large to
    dequantise at once: row_scores over key chunks (each score is one key's
    own float64 dot product, so chunking changes nothing), then select_row."""
    qd = orc.dequantize(q_bits, "bf16")
    nk = keys_dev.shape[0]
    full = np.empty((len(rows), nk), dtype=np.float32)
    for s0 in range(0, nk, chunk):
        kb = keys_dev[s0:s0 + chunk].cpu().view(torch.int16).numpy().view(np.uint16)
        kd = orc.dequantize(kb, "bf16")
        for i, t in enumerate(rows):
            full[i, s0:s0 + kd.shape[0]] = orc.row_scores(qd[t], None, kd, "ip")
    out = [orc.select_row(full[i], nk, k) for i in range(len(rows))]
    return np.stack([o[0] for o in out]), np.stack([o[1] for o in out]), full


@pytest.mark.slow
@pytest.mark.parametrize("k", [128, 8192])
def test_wide_full_size(lib, k):
    x = workloads.unit_corpus_gpu(E7, seed=workloads.CONFIG_SEEDS[E7.name], device="cuda")
    nq, nk = E7.nq, E7.nk
    stats = torch.zeros((nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    fi, fs = lt.indexer_topk(x["q"], None, x["keys"], k, None, mode="ip", options=lt.make_options(row_stats=stats))
    dense = lt.indexer_scores(x["q"], None, x["keys"], mode="ip")
    ri, rs = lt.topk_radix(dense, k, sorted_output=True)
    del dense
    torch.cuda.synchronize()
    gi, gs = _sorted_pairs(fi.cpu().numpy(), fs.cpu().numpy())
    np.testing.assert_array_equal(gi, ri.cpu().numpy(), err_msg="fused sets differ from radix over dense scores")
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32))
    st = stats.cpu().numpy()
    assert np.all(st[:, 2] == 0), "rows fell back: %s" % st[st[:, 2] != 0][:4]
    # each query is a corpus passage: it finds itself with a score near 1
    assert np.all(np.isin(x["pick"], gi[:, :1].ravel()) | (gs[:, 0] > 0.99))
    rows = [0, nq - 1]
    q_bits = x["q"].cpu().view(torch.int16).numpy().view(np.uint16)
    oi, os_, full = _oracle_rows_chunked(q_bits, x["keys"], rows, k)
    fi_h, fs_h = fi.cpu().numpy(), fs.cpu().numpy()
    for j, t in enumerate(rows):
        check_row_tol(fi_h[t], fs_h[t], oi[j], os_[j], full[j], nk, k, RTOL["bf16"])


def test_wide_fallback_splits_few_rows_over_blocks(lib):
    """Three queued rows over 300000 passages: the fallback cuts each row's
    visible passages into chunks re-scored by different blocks, and the block
    that scores a row's last chunk selects the row. Forced fallback, rows of
    different lengths, sorted and unsorted output: every row equals radix
    selection over the dense scores bit for bit (unsorted: the same set and
    scores), and the shorter rows meet the oracle."""
    nq, nk, k = 3, 300000, 1024
    x = workloads.generate(workloads.scaled(E7, nq=nq, nk=nk), seed=31)
    offs = np.array([nk, nk // 3 + 1, 700], dtype=np.int32)
    x["offsets"] = torch.from_numpy(offs)
    d = to_dev(x)
    dense = lt.indexer_scores(d["q"], None, d["keys"], mode="ip")
    ri, rs = lt.topk_radix(dense, k, causal_offsets=d["offsets"], sorted_output=True)
    torch.cuda.synchronize()
    ri, rs = ri.cpu().numpy(), rs.cpu().numpy()
    e = visible(offs, nq, nk)
    for sorted_out in (True, False):
        gi, gs, st = _fused(x, k, sorted_output=sorted_out, force_fallback=True)
        np.testing.assert_array_equal(st[:, 2], 3)
        for t in range(nq):
            check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e[t]), k, sorted_out)
    oi, os_, full = oracle_topk(x, "bf16", k, "ip", rows=[1, 2])
    for j, t in enumerate([1, 2]):
        check_row_tol(gi[t], gs[t], oi[j], os_[j], full[j], int(e[t]), k, RTOL["bf16"])
