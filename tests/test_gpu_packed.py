"""Packed multi-sequence batches: per-row visible ranges [s_t, e_t)
(lt_options.visible_start). Several sequences' keys are concatenated and
each query sees only its own sequence's causal prefix.

* fused results equal the oracle's (tolerance + near-tie rule) and equal,
  bit for bit, each sequence computed in its own launch with its indices
  shifted by the sequence's base (bf16 64 heads, fp8, fp32 4 heads, bf16
  one-head inner product);
* scores-in selection with arbitrary starts (negative, past the end, equal to
  the end) is bit-exact against the oracle;
* the exact fallback honours the starts (forced fallback, both entries)."""
import numpy as np
import pytest
import torch

from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_topk, to_dev
from parity import RTOL, check_row_exact, check_row_tol

pytestmark = pytest.mark.gpu

BATCHES = [
    # base workload, sequence key counts, queries per sequence, k
    ("dsa_bf16_128k", [9000, 20000, 5000], [8, 11, 6], 512),
    ("dsa_fp8_1m", [12000, 7000], [9, 5], 1024),
    ("tiny_fp32", [4096, 1500, 3000], [20, 7, 9], 256),
    ("retrieval_bf16_4m", [30000, 12000], [40, 25], 100),
]


def _fused(d, k, mode, **opt):
    gi, gs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"], mode=mode,
                             options=lt.make_options(sorted_output=True, **opt))
    torch.cuda.synchronize()
    return gi.cpu().numpy(), gs.cpu().numpy()


@pytest.mark.parametrize("batch", BATCHES, ids=[b[0] for b in BATCHES])
def test_packed_matches_oracle_and_separate_launches(lib, batch):
    base, lens, nqs, k = batch
    cfg = workloads.CONFIGS[base]
    x = workloads.packed_batch(cfg, lens, nqs, seed=31)
    d = to_dev(x)
    gi, gs = _fused(d, k, cfg.mode, visible_start=d["starts"])
    # oracle, every row
    oi, os_, full = oracle_topk(x, cfg.dtype, k, cfg.mode)
    s0, e0 = orc.visible_ranges(x["offsets"].numpy(), x["starts"].numpy(), gi.shape[0], x["keys"].shape[0])
    for t in range(gi.shape[0]):
        v = gi[t][gi[t] >= 0]
        assert np.all((v >= s0[t]) & (v < e0[t])), "row %d: index outside its sequence" % t
        m = min(k, int(e0[t] - s0[t]))
        assert v.size == m
        # shift the row into its own range for the tolerance check
        loc = lambda a: np.where(a >= 0, a - s0[t], -1)  # noqa: E731
        check_row_tol(loc(gi[t]), gs[t], loc(oi[t]), os_[t], full[t][s0[t]:], int(e0[t] - s0[t]), k,
                      RTOL[cfg.dtype])
    # each sequence alone
    r = 0
    for b, (L, n) in enumerate(zip(lens, nqs)):
        kb = int(x["bases"][b])
        sub = {"q": x["q"][r:r + n].contiguous(), "keys": x["keys"][kb:kb + L].contiguous(),
               "w": None if x["w"] is None else x["w"][r:r + n].contiguous(),
               "q_scale": None if x["q_scale"] is None else x["q_scale"][r:r + n].contiguous(),
               "k_scale": None if x["k_scale"] is None else x["k_scale"][kb:kb + L].contiguous(),
               "offsets": (x["offsets"][r:r + n] - kb).contiguous()}
        si, ss = _fused(to_dev(sub), k, cfg.mode)
        np.testing.assert_array_equal(gi[r:r + n], np.where(si >= 0, si + kb, -1), err_msg="sequence %d" % b)
        np.testing.assert_array_equal(gs[r:r + n].view(np.uint32), ss.view(np.uint32), err_msg="sequence %d" % b)
        r += n


def test_packed_forced_fallback_and_exact_inputs(lib):
    nq, nk, k = 14, 3001, 150
    x = workloads.exact_inputs(nq, nk, 64, 128, "bf16", seed=5)
    rng = np.random.default_rng(2)
    starts = rng.integers(-10, 2500, size=nq).astype(np.int32)
    starts[0], starts[1] = nk + 5, int(x["offsets"][2])  # past the end; equal to the row's end
    x["starts"] = torch.from_numpy(starts)
    d = to_dev(x)
    ri, rs, _ = oracle_topk(x, "bf16", k, "dsa")
    s0, e0 = orc.visible_ranges(x["offsets"].numpy(), starts, nq, nk)
    for opt in (dict(), dict(force_fallback=True), dict(key_splits=3)):
        gi, gs = _fused(d, k, "dsa", visible_start=d["starts"], **opt)
        for t in range(nq):
            check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e0[t] - s0[t]), k, True)


@pytest.mark.parametrize("opt", [dict(), dict(force_fallback=True), dict(key_splits=3), dict(sample_size=0)],
                         ids=["default", "fallback", "splits", "nosample"])
def test_scores_in_select_with_starts(lib, opt):
    nq, nk, k = 24, 9000, 300
    scores = workloads.score_rows(nq, nk, seed=13, kind="ties")
    offs = workloads.causal_offsets(nq, nk)
    rng = np.random.default_rng(4)
    starts = rng.integers(-50, 8000, size=nq).astype(np.int32)
    starts[3] = offs[3]
    starts[4] = nk + 1
    ri, rs = orc.topk_select(scores.numpy(), nk, k, offs, visible_start=starts)
    gi, gs = lt.topk_select(scores.cuda(), k, causal_offsets=torch.from_numpy(offs).cuda(),
                            options=lt.make_options(sorted_output=True, visible_start=torch.from_numpy(starts).cuda(),
                                                    **opt))
    torch.cuda.synchronize()
    s0, e0 = orc.visible_ranges(offs, starts, nq, nk)
    gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e0[t] - s0[t]), k, True)


def test_packed_rows_split_over_fallback_blocks(lib):
    """A few forced rows over 40000 keys take the fallback's split mode (each
    row's visible keys in chunks over many blocks); with packed starts the
    chunks cover [s_t, e_t) only: exact inputs, sorted output, bit-exact
    against the oracle, including a row whose start is past its end and one
    that sees fewer keys than k."""
    nq, nk, k = 6, 40000, 256
    x = workloads.exact_inputs(nq, nk, 64, 128, "bf16", seed=9, causal=False)
    ends = np.array([nk, 31000, 25000, 40000, 9000, 20000], dtype=np.int32)
    starts = np.array([0, 7003, 26000, 39900, 1, 12345], dtype=np.int32)
    x["offsets"] = torch.from_numpy(ends)
    x["starts"] = torch.from_numpy(starts)
    d = to_dev(x)
    ri, rs, _ = oracle_topk(x, "bf16", k, "dsa")
    s0, e0 = orc.visible_ranges(ends, starts, nq, nk)
    gi, gs = _fused(d, k, "dsa", visible_start=d["starts"], force_fallback=True)
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e0[t] - s0[t]), k, True)
