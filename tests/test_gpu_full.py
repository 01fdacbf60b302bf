"""Parity at the full workload sizes, in the launch configuration the
benchmark times (default options):

* every row: the fused result equals plain radix selection (lt_topk_radix,
  no sampling or filtering) over the dense score matrix (lt_indexer_scores,
  the same score arithmetic), bit for bit after sorting both by the total
  order; every row holds exactly min(k, e_t) distinct visible indices; no row
  needed the fallback for an internal inconsistency;
* an evenly spaced sample of rows (first and last included): the fused result
  against the CPU oracle, within the fp32/bf16 (1e-3) or fp8 (2e-2) tolerance
  and the swap rule.
"""
import numpy as np
import pytest
import torch

from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_topk, to_dev
from parity import RTOL, check_row_tol, visible

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

FULL = ["tiny_fp32", "dsa_bf16_128k", "dsa_fp8_1m", "adversarial_bf16_256k"]


def _sorted_pairs(idx, sc):
    """Sort every row by the total order (score desc, NaN last, -0 == +0,
    index asc; padding last), on the host."""
    idx, sc = idx.cpu().numpy(), sc.cpu().numpy()
    nq, k = idx.shape
    row = np.repeat(np.arange(nq), k)
    i = idx.ravel().astype(np.int64)
    s = sc.ravel().astype(np.float64)
    nan = np.isnan(s) | (i < 0)
    key = np.where(nan, 0.0, -s) + 0.0
    o = np.lexsort((np.where(i < 0, 1 << 40, i), key, nan, row))
    return idx.ravel()[o].reshape(nq, k), sc.ravel()[o].reshape(nq, k)


@pytest.mark.parametrize("name", FULL)
def test_full_size_parity(lib, name):
    cfg = workloads.CONFIGS[name]
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[name])
    d = to_dev(x)
    nq, nk, k = cfg.nq, cfg.nk, cfg.k
    stats = torch.zeros((nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    fi, fs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"],
                             mode=cfg.mode, options=lt.make_options(row_stats=stats))
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=cfg.mode)
    ri, rs = lt.topk_radix(dense, k, causal_offsets=d["offsets"], sorted_output=True)
    del dense
    torch.cuda.synchronize()
    gi, gs = _sorted_pairs(fi, fs)
    np.testing.assert_array_equal(gi, ri.cpu().numpy(), err_msg="fused sets differ from radix over dense scores")
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32),
                                  err_msg="fused scores differ from dense scores")
    e = visible(None if x["offsets"] is None else x["offsets"].numpy(), nq, nk)
    valid = gi >= 0
    np.testing.assert_array_equal(valid.sum(1), np.minimum(e, k), err_msg="wrong number of entries")
    assert np.all((gi < e[:, None]) | ~valid), "index outside the visible range"
    for t in range(nq):
        v = gi[t][valid[t]]
        assert np.unique(v).size == v.size, "duplicate index in row %d" % t
    st = stats.cpu().numpy()
    assert not np.any(st[:, 2] == 4)
    # sampled rows against the CPU oracle
    rows = sorted(set(np.linspace(0, nq - 1, 8).round().astype(int).tolist()))
    oi, os_, full = oracle_topk(x, cfg.dtype, k, cfg.mode, rows=rows)
    fi_h, fs_h = fi.cpu().numpy(), fs.cpu().numpy()
    ev = visible(None if x["offsets"] is None else x["offsets"].numpy(), nq, nk)
    for j, t in enumerate(rows):
        check_row_tol(fi_h[t], fs_h[t], oi[j], os_[j], full[j], int(ev[t]), k, RTOL[cfg.dtype])


def test_full_size_retrieval(lib):
    """10000 queries x 4M items, inner product, k = 100. The dense check runs
    on three 512-row blocks (first, middle, last query tiles): the full dense
    matrix would take 160 GB."""
    name = "retrieval_bf16_4m"
    cfg = workloads.CONFIGS[name]
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[name])
    d = to_dev(x)
    nq, nk, k = cfg.nq, cfg.nk, cfg.k
    stats = torch.zeros((nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    fi, fs = lt.indexer_topk(d["q"], None, d["keys"], k, None, mode="ip", options=lt.make_options(row_stats=stats))
    torch.cuda.synchronize()
    gi, gs = _sorted_pairs(fi, fs)
    assert np.all(gi >= 0) and np.all(gi < nk)
    for t in range(nq):
        assert np.unique(gi[t]).size == k, "duplicate index in row %d" % t
    assert not np.any(stats.cpu().numpy()[:, 2] == 4)
    for r0 in (0, nq // 2 - 256, nq - 512):
        qb = d["q"][r0:r0 + 512].contiguous()
        dense = lt.indexer_scores(qb, None, d["keys"], mode="ip")
        ri, rs = lt.topk_radix(dense, k, sorted_output=True)
        del dense
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gi[r0:r0 + 512], ri.cpu().numpy())
        np.testing.assert_array_equal(gs[r0:r0 + 512].view(np.uint32), rs.cpu().numpy().view(np.uint32))
    rows = sorted(set(np.linspace(0, nq - 1, 8).round().astype(int).tolist()))
    oi, os_, full = oracle_topk(x, cfg.dtype, k, cfg.mode, rows=rows)
    fi_h, fs_h = fi.cpu().numpy(), fs.cpu().numpy()
    for j, t in enumerate(rows):
        check_row_tol(fi_h[t], fs_h[t], oi[j], os_[j], full[j], nk, k, RTOL[cfg.dtype])


@pytest.mark.parametrize("over", [False, True])
@pytest.mark.parametrize("dtype,h,mode", [("bf16", 64, "dsa"), ("bf16", 1, "ip"), ("fp8", 64, "dsa")])
def test_sample_scan_around_4gib_of_keys(lib, dtype, h, mode, over):
    """Key arrays just under and just over 4 GiB: the sample scorer gathers
    its rows through one buffer descriptor (byte offsets up to 4 GiB) below
    that size, through per-lane global addresses above it. The fused result
    must equal radix selection over the dense scores, with no row taking the
    fallback (a wrong sample threshold would send rows there)."""
    d, nq, k = 128, 8, 64
    row_bytes = d * (2 if dtype == "bf16" else 1)
    nk = (1 << 32) // row_bytes + (4096 if over else -64)
    g = torch.Generator(device="cuda").manual_seed(7)
    if dtype == "bf16":
        keys = (torch.randn((nk, d), device="cuda", generator=g) * 0.1).to(torch.bfloat16)
        q = (torch.randn((nq, h, d), device="cuda", generator=g) * 0.1).to(torch.bfloat16)
        qs = ks = None
    else:
        # E4M3FN bytes without the two NaN encodings (0x7F, 0xFF)
        keys = torch.randint(0, 0x7F, (nk, d), device="cuda", generator=g, dtype=torch.int32)
        keys = (keys | (torch.randint(0, 2, (nk, d), device="cuda", generator=g, dtype=torch.int32) << 7)).to(torch.uint8)
        q = torch.randint(0, 0x7F, (nq, h, d), device="cuda", generator=g, dtype=torch.int32).to(torch.uint8)
        qs = torch.rand((nq, h), device="cuda", generator=g) * 1e-2 + 1e-3
        ks = torch.rand((nk,), device="cuda", generator=g) * 1e-2 + 1e-3
    w = torch.rand((nq, h), device="cuda", generator=g) if mode == "dsa" else None
    stats = torch.zeros((nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    # a sample large enough for the range estimate to hold the top-k of 2^25
    # keys (the default 3k keys would put every top-k key in the clamped top
    # bin and send the rows to the fallback by design)
    opts = lt.make_options(row_stats=stats, sample_size=65536)
    fi, fs = lt.indexer_topk(q, w, keys, k, None, qs, ks, mode=mode, options=opts)
    dense = lt.indexer_scores(q, w, keys, qs, ks, mode=mode)
    ri, rs = lt.topk_radix(dense, k, sorted_output=True)
    torch.cuda.synchronize()
    del dense, keys
    gi, gs = _sorted_pairs(fi, fs)
    np.testing.assert_array_equal(gi, ri.cpu().numpy())
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32))
    assert int((stats[:, 2] != 0).sum()) == 0, "rows took the fallback"


def _dense_radix_check(d, mode, k, fi, fs, rows=None):
    """Every row of the fused result equals radix selection over the dense
    scores (same arithmetic), bit for bit after sorting both."""
    q = d["q"] if rows is None else d["q"][rows].contiguous()
    w = d["w"] if (rows is None or d["w"] is None) else d["w"][rows].contiguous()
    qs = d["q_scale"] if (rows is None or d["q_scale"] is None) else d["q_scale"][rows].contiguous()
    offs = d["offsets"] if (rows is None or d["offsets"] is None) else d["offsets"][rows].contiguous()
    dense = lt.indexer_scores(q, w, d["keys"], qs, d["k_scale"], mode=mode)
    ri, rs = lt.topk_radix(dense, k, causal_offsets=offs, sorted_output=True)
    del dense
    torch.cuda.synchronize()
    gi, gs = _sorted_pairs(fi, fs)
    np.testing.assert_array_equal(gi, ri.cpu().numpy(), err_msg="fused sets differ from radix over dense scores")
    np.testing.assert_array_equal(gs.view(np.uint32), rs.cpu().numpy().view(np.uint32),
                                  err_msg="fused scores differ from dense scores")


def _oracle_rows(x, cfg, k, fi, fs, rows, xrows=None):
    """Rows `rows` of the fused result against the CPU oracle (tolerance and
    swap rule); xrows are the same rows' indices into x (default: rows)."""
    xrows = rows if xrows is None else xrows
    oi, os_, full = oracle_topk(x, cfg.dtype, k, cfg.mode, rows=xrows)
    ev = visible(None if x["offsets"] is None else x["offsets"].numpy(), x["q"].shape[0], cfg.nk)
    for j, (t, tx) in enumerate(zip(rows, xrows)):
        check_row_tol(fi[t], fs[t], oi[j], os_[j], full[j], int(ev[tx]), k, RTOL[cfg.dtype])


@pytest.mark.parametrize("opt,reason", [(dict(capacity=8192), 6), (dict(capacity=1024), 1),
                                        (dict(capacity=262144, num_bins=2), 2)],
                         ids=["overflow-refilter", "overflow-dense", "tie-bin"])
def test_fallback_at_full_size_adversarial(lib, opt, reason):
    """The adversarial 1024 x 256K workload at full size, in three forms that
    send rows past the first select for real. Candidate buffers below its
    ~21K survivors per row (the capacity is per key split; the launch splits
    the keys in two, ~10.6K survivors each) overflow: with 8192 slots the
    keys at or above each row's exact final bin fit in one list, so a second
    filter pass gated at that bin finishes the row (reason 6); with 1024
    slots (below k) they cannot, and the dense fallback does (reason 1).
    Two bins with room for every key leave a threshold bin too large to sort
    (reason 2: dense fallback). Every row equals radix selection over the
    dense scores bit for bit; evenly spaced rows meet the oracle."""
    name = "adversarial_bf16_256k"
    cfg = workloads.CONFIGS[name]
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[name])
    d = to_dev(x)
    k = cfg.k
    stats = torch.zeros((cfg.nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    fi, fs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], mode=cfg.mode,
                             options=lt.make_options(row_stats=stats, **opt))
    torch.cuda.synchronize()
    st = stats.cpu().numpy()
    n_fb = int((st[:, 2] == reason).sum())
    print("%s: %d of %d rows took the fallback with reason %d" % (name, n_fb, cfg.nq, reason), flush=True)
    assert n_fb >= cfg.nq // 4, "too few rows reached the fallback"
    assert set(np.unique(st[:, 2]).tolist()) <= {0, reason}
    _dense_radix_check(d, cfg.mode, k, fi, fs)
    rows = sorted(set(np.linspace(0, cfg.nq - 1, 8).round().astype(int).tolist()))
    _oracle_rows(x, cfg, k, fi.cpu().numpy(), fs.cpu().numpy(), rows)


@pytest.fixture(scope="module")
def fp8_1m_rows():
    """64 evenly spaced rows of the 2048 x 1M fp8 workload (all 1M keys)."""
    name = "dsa_fp8_1m"
    cfg = workloads.CONFIGS[name]
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[name])
    rows = np.linspace(0, cfg.nq - 1, 64).round().astype(np.int64)
    xs = dict(x)
    for key in ("q", "q_scale", "w", "offsets"):
        xs[key] = x[key][torch.from_numpy(rows)].contiguous()
    return cfg, x, xs, rows


@pytest.mark.parametrize("opt,reason", [(dict(force_fallback=True), 3), (dict(num_bins=1), 1)],
                         ids=["forced", "one-bin"])
def test_fallback_at_full_size_fp8_1m(lib, fp8_1m_rows, opt, reason):
    """64 rows of the 1M-context fp8 workload through the exact fallback at
    full context: forced (reason 3), and one bin, where every key passes the
    gate and the 24576-entry buffers overflow (reason 1). The fallback
    re-scores each row's 1M keys into its scratch row and radix-selects it."""
    cfg, x, xs, rows = fp8_1m_rows
    d = to_dev(xs)
    k = cfg.k
    nq = len(rows)
    stats = torch.zeros((nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
    fi, fs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"],
                             mode=cfg.mode, options=lt.make_options(row_stats=stats, **opt))
    torch.cuda.synchronize()
    st = stats.cpu().numpy()
    assert np.all(st[:, 2] == reason), np.unique(st[:, 2])
    _dense_radix_check(d, cfg.mode, k, fi, fs)
    sel = list(range(0, nq, 8)) + [nq - 1]
    _oracle_rows(x, cfg, k, fi.cpu().numpy(), fs.cpu().numpy(), sel, xrows=[int(rows[i]) for i in sel])


# Every row of the 128K and 256K workloads against the oracle, in blocks of
# rows (the fused call runs once per workload and is kept for its blocks).
ALL_ROWS = {"dsa_bf16_128k": 256, "adversarial_bf16_256k": 128}


@pytest.fixture(scope="module")
def full_fused():
    cache = {}

    def get(name):
        if name not in cache:
            cache.clear()
            cfg = workloads.CONFIGS[name]
            x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS[name])
            d = to_dev(x)
            fi, fs = lt.indexer_topk(d["q"], d["w"], d["keys"], cfg.k, d["offsets"], d["q_scale"], d["k_scale"],
                                     mode=cfg.mode)
            torch.cuda.synchronize()
            cache[name] = (cfg, x, fi.cpu().numpy(), fs.cpu().numpy())
            del d
        return cache[name]
    return get


@pytest.mark.parametrize("name,block", [(n, b) for n, rows in ALL_ROWS.items()
                                        for b in range(workloads.CONFIGS[n].nq // rows)])
def test_every_row_against_oracle(lib, full_fused, name, block):
    cfg, x, fi, fs = full_fused(name)
    per = ALL_ROWS[name]
    rows = list(range(block * per, (block + 1) * per))
    _oracle_rows(x, cfg, cfg.k, fi, fs, rows)


def test_chunked_prefill_1m_equals_one_launch(lib):
    """The paper's chunked-prefill setting at 1M context (sec. 4.1, 4.2): the
    last 8192 tokens as queries in chunks of 1024, every chunk after the first
    sampling the previous chunk's most frequent top-k keys, and the first 2048
    tokens again in chunks of 128; each chunk's rows equal one launch over all
    8192 rows, bit for bit."""
    cfg = workloads.scaled(workloads.CONFIGS["dsa_fp8_1m"], nq=8192)
    x = workloads.generate(cfg, seed=workloads.CONFIG_SEEDS["dsa_fp8_1m"])
    d = to_dev(x)
    k, nk = cfg.k, cfg.nk
    sopt = lt.make_options(sorted_output=True)
    ri, rs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"], options=sopt)
    torch.cuda.synchronize()
    ri, rs = ri.cpu().numpy(), rs.cpu().numpy()
    for chunk, upto in ((1024, cfg.nq), (128, 2048)):
        prev = None
        for c0 in range(0, upto, chunk):
            sl = slice(c0, c0 + chunk)
            part = {n: d[n][sl].contiguous() for n in ("q", "w", "q_scale", "offsets")}
            hint = None if prev is None else lt.sample_from_topk(prev, nk, 3 * k)
            stats = torch.zeros((chunk, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
            gi, gs = lt.indexer_topk(part["q"], part["w"], d["keys"], k, part["offsets"], part["q_scale"],
                                     d["k_scale"], options=lt.make_options(sorted_output=True, sample_keys=hint,
                                                                           row_stats=stats))
            torch.cuda.synchronize()
            np.testing.assert_array_equal(gi.cpu().numpy(), ri[sl], err_msg="chunk %d at %d" % (chunk, c0))
            np.testing.assert_array_equal(gs.cpu().numpy().view(np.uint32), rs[sl].view(np.uint32))
            assert not np.any(stats.cpu().numpy()[:, 2] == 5)
            prev = gi
