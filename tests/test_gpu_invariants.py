"""Internal invariants of the fused pipeline, checked on device output
(sec. 3.2), and the tie rule of the scans whose candidate lists fill in
arrival order.

Per row, from lt_options.row_stats and the dense score matrix of the same
arithmetic (lt_indexer_scores):
* no row needed the fallback, and the final threshold bin tau_f is at or
  above the sample's initial bin tau0 (sec. 3.2 "Sampling": the sample is a
  subset of the row's keys, so its k-th score is a lower bound);
* the sample's k-th score ranks at or below the row's k-th score;
* count(bin > tau_f) < k <= count(bin >= tau_f) over the row's visible keys,
  with the bins taken from the row's own bin map (sec. 3.2 "Top-k Selection":
  only bin tau_f needs sorting);
* every visible key in a bin >= tau_f was written to the candidate buffer.

Ties: in the one-head scan passing scores are queued per wave and written
when the queues drain, so a row's list is not in key order; equal scores at
the k-th place must still go to the lower key index (the total order). Keys
are duplicated so that many scores tie, and the fused result is compared bit
for bit with the scores-in selection over the dense scores, and with the
oracle's rule.
"""
import numpy as np
import pytest
import torch

from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import to_dev
from parity import visible

pytestmark = pytest.mark.gpu


def ord_key(s: np.ndarray) -> np.ndarray:
    """Order keys of float32 scores under the total order (larger = ranks
    higher; -0 == +0; NaN lowest)."""
    s = np.asarray(s, dtype=np.float32)
    b = s.view(np.uint32).astype(np.uint64)
    b = np.where(b == 0x80000000, 0, b)
    o = np.where(b & 0x80000000, (~b) & 0xFFFFFFFF, b | 0x80000000)
    return np.where(np.isnan(s), 0, o).astype(np.uint64)


def bins_of(scores: np.ndarray, delta: np.float32, c: np.float32, m: int) -> np.ndarray:
    """floor(fmaf(I, delta, c)) clamped to m - 1, -1 below 0 or NaN. The
    product of two float32 values is exact in extended precision and the sum
    rounds once there before the one rounding to float32, as fmaf does."""
    x = (scores.astype(np.longdouble) * np.longdouble(delta) + np.longdouble(c)).astype(np.float32)
    with np.errstate(invalid="ignore"):
        b = np.where(x >= 0, np.floor(np.where(np.isfinite(x), x, 0)), -1)
        b = np.where(np.isinf(x) & (x > 0), m - 1, b)
    return np.minimum(b, m - 1).astype(np.int64)


CASES = [
    # id, base config, nq, nk, k, num_bins requested (the one-head shapes
    # have LDS for fewer: the test reads the bins in use from the stats)
    ("dsa_bf16", "dsa_bf16_128k", 21, 20011, 2048, 256),
    ("dsa_fp8", "dsa_fp8_1m", 17, 30001, 2048, 256),
    ("adversarial_bf16", "adversarial_bf16_256k", 16, 40000, 2048, 256),
    ("tiny_fp32", "tiny_fp32", None, None, None, 256),
    ("ip_bf16_h1", "retrieval_bf16_4m", 300, 50001, 100, 64),
    ("ip_bf16_d768", "retrieval_e7_bf16_5m", 64, 20000, 128, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fused_row_invariants(lib, case):
    name, base, nq, nk, k, m = case
    cfg = workloads.CONFIGS[base]
    cfg = workloads.scaled(cfg, nq=nq, nk=nk) if nq else cfg
    k = cfg.k if k is None else k
    x = workloads.generate(cfg, seed=21)
    d = to_dev(x)
    stats = torch.full((cfg.nq, lt.LT_ROW_STATS), -7, dtype=torch.int32, device="cuda")
    gi, gs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"], mode=cfg.mode,
                             options=lt.make_options(row_stats=stats, num_bins=m, sorted_output=True))
    dense = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=cfg.mode)
    torch.cuda.synchronize()
    gi, gs, st, dense = gi.cpu().numpy(), gs.cpu().numpy(), stats.cpu().numpy(), dense.cpu().numpy()
    e = visible(None if x["offsets"] is None else x["offsets"].numpy(), cfg.nq, cfg.nk)
    gated = 0
    for t in range(cfg.nq):
        written, tau_f, reason, _, tau0 = (int(v) for v in st[t, :5])
        assert reason == 0, "row %d took the fallback (reason %d)" % (t, reason)
        assert tau_f >= tau0, "row %d: final bin %d below the sample's %d" % (t, tau_f, tau0)
        delta, c = st[t, 6:8].view(np.float32)
        m_used = int(st[t, 8])
        assert 1 <= m_used <= m
        b = bins_of(dense[t, :e[t]], delta, c, m_used)
        if tau_f >= 0:
            above, at_or_above = int((b > tau_f).sum()), int((b >= tau_f).sum())
            assert above < k <= at_or_above, "row %d: %d above, %d at or above bin %d" % (t, above, at_or_above,
                                                                                          tau_f)
            assert written >= at_or_above, "row %d: %d written < %d at or above tau_f" % (t, written, at_or_above)
        samp_kth = st[t, 5:6].view(np.float32)
        if tau0 >= 0:
            gated += 1
            assert not np.isneginf(samp_kth[0]), "row %d: gated without a sample k-th score" % t
            m_t = min(k, int(e[t]))
            row_kth = gs[t, m_t - 1:m_t]
            assert ord_key(samp_kth)[0] <= ord_key(row_kth)[0], \
                "row %d: sample k-th %r above the row's k-th %r" % (t, samp_kth[0], row_kth[0])
    assert gated > 0, "no row was gated: the invariants were not exercised"


@pytest.mark.parametrize("layout", ["strided", "adjacent"])
@pytest.mark.parametrize("opt", [dict(), dict(key_splits=4), dict(key_splits=1)],
                         ids=["auto", "splits4", "splits1"])
def test_grouped_ties_go_to_the_lower_key(lib, layout, opt):
    """One-head inner-product scan (lists fill in arrival order): each key
    appears four times, so most scores tie with three others."""
    cfg = workloads.scaled(workloads.CONFIGS["retrieval_bf16_4m"], nq=300, nk=50000)
    x = workloads.generate(cfg, seed=31)
    base = x["keys"][: cfg.nk // 4]
    nb = base.shape[0]
    if layout == "strided":      # copies a quarter of the keys apart (other tiles and splits)
        keys = base.repeat(4, 1)
    else:                        # copies next to each other (one tile, one drain record)
        keys = base.repeat_interleave(4, dim=0)
    x["keys"] = keys.contiguous()
    q = x["keys"][torch.from_numpy(np.arange(cfg.nq) * 7 % nb)].unsqueeze(1).contiguous()
    x["q"] = q
    d = to_dev(x)
    k = 102                      # cuts through a group of four equal scores
    for sorted_out in (True, False):
        fi, fs = lt.indexer_topk(d["q"], None, d["keys"], k, None, mode="ip",
                                 options=lt.make_options(sorted_output=sorted_out, **opt))
        dense = lt.indexer_scores(d["q"], None, d["keys"], mode="ip")
        si, ss = lt.topk_select(dense, k, options=lt.make_options(sorted_output=True))
        torch.cuda.synchronize()
        fi, fs, si, ss = fi.cpu().numpy(), fs.cpu().numpy(), si.cpu().numpy(), ss.cpu().numpy()
        # rows of this shape are always returned sorted
        np.testing.assert_array_equal(fi, si)
        np.testing.assert_array_equal(fs.view(np.uint32), ss.view(np.uint32))
        dn = dense.cpu().numpy()
        # the oracle's rule, on the dense scores of the same arithmetic:
        # every tie at the k-th score keeps the lowest keys
        for t in range(0, cfg.nq, 7):
            kth = fs[t, k - 1]
            tied = np.nonzero(dn[t] == kth)[0]
            kept = np.sort(fi[t][fs[t] == kth])
            np.testing.assert_array_equal(kept, tied[: kept.size])
        assert np.mean([np.sum(dn[t] == fs[t, k - 1]) > 1 for t in range(cfg.nq)]) > 0.5, "too few ties"
