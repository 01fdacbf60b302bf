"""GPU parity of the sample lists (sec. 3.2 "Sampling").

* lt_sample_from_topk against the oracle's previous-chunk sample, bit-exact,
  from small hand-sized cases to counts that need every digit of the radix
  selection (>= 2^10 and >= 2^21 occurrences of one key);
* a caller's sample list never changes a result: fused and scores-in
  selection stay bit-exact (and within tolerance of the oracle) for the
  previous chunk's sample, the row's true top-k, lists with repeats,
  negative and out-of-range entries, keys beyond some rows' visible range,
  an all-invalid list and a one-entry list;
* chunked prefill: chunks that take their sample from the previous chunk's
  output give the same result as one launch over all queries.
"""
import numpy as np
import pytest
import torch

from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_topk, to_dev
from parity import RTOL, check_row_tol, visible
from test_oracle import SAMPLE_CASES, check_sample_invariants, sample_case_input

pytestmark = pytest.mark.gpu


def _gpu_sample(prev, nk, ns):
    p = torch.from_numpy(np.ascontiguousarray(prev, dtype=np.int32)).cuda()
    if p.dim() == 1:
        p = p.view(1, -1)
    out = lt.sample_from_topk(p, nk, ns)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("case", SAMPLE_CASES, ids=[f"{c[0]}x{c[1]}-nk{c[2]}-ns{c[3]}-{c[4]}" for c in SAMPLE_CASES])
def test_sample_from_topk_matches_oracle(lib, case):
    rows, k, nk, ns, law = case
    prev = sample_case_input(rows, k, nk, law, seed=rows * 31 + nk)
    if rows == 0:
        prev = np.zeros((0, k), dtype=np.int32)
    got = _gpu_sample(prev, nk, ns)
    np.testing.assert_array_equal(got, orc.sample_from_topk(prev, nk, ns))
    check_sample_invariants(got, prev, nk, ns)


def test_sample_from_topk_golden_example(lib):
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sample_from_topk.json")))
    prev = np.array(g["prev_idx"], dtype=np.int32)
    for case in g["cases"]:
        assert _gpu_sample(prev, g["num_keys"], case["sample_size"]).tolist() == case["sample"]


def test_sample_from_topk_dsa_shaped(lib):
    """A previous chunk of 512 rows x k = 2048 over 131072 keys (the 128K DSA
    workload's context), sample k' = 3k = 6144; taken from real fused output."""
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=512)
    x = workloads.generate(cfg, seed=3)
    d = to_dev(x)
    gi, _ = lt.indexer_topk(d["q"], d["w"], d["keys"], cfg.k, d["offsets"])
    got = lt.sample_from_topk(gi, cfg.nk, 3 * cfg.k)
    torch.cuda.synchronize()
    prev = gi.cpu().numpy()
    np.testing.assert_array_equal(got.cpu().numpy(), orc.sample_from_topk(prev, cfg.nk, 3 * cfg.k))


@pytest.mark.parametrize("nk", [70000, 300000])
@pytest.mark.parametrize("big", [1500, 2_200_000])
def test_sample_from_topk_large_counts(lib, big, nk):
    """Counts above 2^10 and 2^21 exercise the upper digits of the radix pick;
    ties between keys with equal large counts must still go to the lower key.
    70000 keys are counted in LDS, 300000 with global atomics."""
    rng = np.random.default_rng(big)
    heavy = np.array([5, 60000, 123, 777, 69999, 40000], dtype=np.int32)
    reps = np.array([big, big, big - 1, big + 3, 2, big], dtype=np.int64)
    body = np.repeat(heavy, reps)
    noise = rng.integers(-2, nk + 2, size=300000).astype(np.int32)
    flat = np.concatenate([body, noise])
    rng.shuffle(flat)
    cols = 1000
    flat = np.concatenate([flat, np.full((-flat.size) % cols, -1, np.int32)])
    prev = flat.reshape(-1, cols)
    for ns in (1, 2, 4, 5, 300):
        np.testing.assert_array_equal(_gpu_sample(prev, nk, ns), orc.sample_from_topk(prev, nk, ns))


@pytest.mark.parametrize("nk", [262144, 262145, 500000])
def test_sample_from_topk_around_the_lds_count_limit(lib, nk):
    """Key arrays at, just past and well past the largest one counted in LDS,
    with the clamped single histogram pass (few entries) and the digit passes
    (a sample larger than entries / 2047 allows)."""
    rng = np.random.default_rng(nk)
    prev = np.minimum(rng.zipf(1.3, size=(96, 2048)) * 7 + rng.integers(0, 7, size=(96, 2048)), nk + 3) - 2
    prev = prev.astype(np.int32)
    for ns in (1, 97, 6144):
        np.testing.assert_array_equal(_gpu_sample(prev, nk, ns), orc.sample_from_topk(prev, nk, ns))


def test_sample_from_topk_strided_rows_and_limits(lib):
    """prev_idx with a row stride larger than k (a column slice), nk < ns, and
    the longest list."""
    rng = np.random.default_rng(1)
    full = rng.integers(-1, 3000, size=(40, 300)).astype(np.int32)
    t = torch.from_numpy(full).cuda()[:, :128]
    got = lt.sample_from_topk(t, 3000, 500)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), orc.sample_from_topk(full[:, :128], 3000, 500))
    np.testing.assert_array_equal(_gpu_sample(full[:3, :5], 7, 100), orc.sample_from_topk(full[:3, :5], 7, 100))
    prev = rng.integers(0, 200000, size=(64, 2048)).astype(np.int32)
    ns = lt.LT_SAMPLE_LIST_MAX
    np.testing.assert_array_equal(_gpu_sample(prev, 200000, ns), orc.sample_from_topk(prev, 200000, ns))


# --------------------------------------------------------------------------
# sample lists never change a result
# --------------------------------------------------------------------------

def _lists(rng, x, k, nk, truth):
    prev = truth[: max(1, truth.shape[0] // 2)]
    lists = {
        "prev_chunk": orc.sample_from_topk(prev, nk, 3 * k),
        "true_topk_row0": truth[0][truth[0] >= 0],
        "dirty": np.concatenate([rng.integers(-50, nk + 50, 2000), np.repeat(truth[0][:40], 3),
                                 np.full(30, nk - 1)]).astype(np.int32),
        "all_invalid": np.array([-1, -7, nk, nk + 100], dtype=np.int32),
        "one": np.array([truth[-1][0]], dtype=np.int32),
        "beyond_early_rows": np.arange(nk - 3 * k, nk, dtype=np.int32),
        # ascending in-range entries with holes and out-of-range entries between them
        "ascending_with_holes": np.where(np.arange(3 * k) % 5 == 1, -3,
                                         np.where(np.arange(3 * k) % 7 == 2, nk + 11,
                                                  np.arange(3 * k) * (nk // (3 * k)))).astype(np.int32),
        # ascending except one repeated key
        "ascending_one_repeat": np.concatenate([np.arange(0, nk, 97)[:200], [97 * 199],
                                                np.arange(97 * 200, nk, 97)[:100]]).astype(np.int32),
    }
    return lists


@pytest.mark.parametrize("base", ["dsa_bf16_128k", "dsa_fp8_1m", "tiny_fp32"])
def test_sample_list_keeps_fused_exact(lib, base):
    cfg = workloads.CONFIGS[base]
    cfg = workloads.scaled(cfg, nq=min(cfg.nq, 20), nk=min(cfg.nk, 24000))
    k = min(cfg.k, 512)
    x = workloads.generate(cfg, seed=21)
    d = to_dev(x)
    ref_i, ref_s = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"],
                                   mode=cfg.mode, options=lt.make_options(sorted_output=True))
    torch.cuda.synchronize()
    ref_i, ref_s = ref_i.cpu().numpy(), ref_s.cpu().numpy()
    rng = np.random.default_rng(2)
    oi, os_, full = oracle_topk(x, cfg.dtype, k, cfg.mode)
    e = visible(None if x["offsets"] is None else x["offsets"].numpy(), cfg.nq, cfg.nk)
    for name, lst in _lists(rng, x, k, cfg.nk, ref_i).items():
        keys = torch.from_numpy(np.ascontiguousarray(lst, dtype=np.int32)).cuda()
        stats = torch.zeros((cfg.nq, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
        gi, gs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"],
                                 mode=cfg.mode,
                                 options=lt.make_options(sorted_output=True, sample_keys=keys, row_stats=stats))
        torch.cuda.synchronize()
        gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
        np.testing.assert_array_equal(gi, ref_i, err_msg=name)
        np.testing.assert_array_equal(gs.view(np.uint32), ref_s.view(np.uint32), err_msg=name)
        assert not np.any(stats.cpu().numpy()[:, 2] == 4), name
        for t in range(cfg.nq):
            check_row_tol(gi[t], gs[t], oi[t], os_[t], full[t], int(e[t]), k, RTOL[cfg.dtype])


def test_sample_list_keeps_scores_in_select_exact(lib):
    nq, nk, k = 16, 9000, 300
    scores = workloads.score_rows(nq, nk, seed=5, kind="ties")
    offs = workloads.causal_offsets(nq, nk)
    ri, rs = orc.topk_select(scores.numpy(), nk, k, offs)
    s = scores.cuda()
    o = torch.from_numpy(offs).cuda()
    rng = np.random.default_rng(3)
    for name, lst in _lists(rng, None, k, nk, ri).items():
        keys = torch.from_numpy(np.ascontiguousarray(lst, dtype=np.int32)).cuda()
        gi, gs = lt.topk_select(s, k, causal_offsets=o,
                                options=lt.make_options(sorted_output=True, sample_keys=keys))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gi.cpu().numpy(), ri, err_msg=name)
        np.testing.assert_array_equal(gs.cpu().numpy().view(np.uint32), rs.view(np.uint32), err_msg=name)


def test_chunked_prefill_with_previous_chunk_sample(lib):
    """Queries of one sequence processed in chunks, each chunk sampling from
    the previous chunk's top-k: same result as one launch over all rows, and
    the reused sample starts the gate at least as tight on this workload."""
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=256, nk=40000)
    k, chunk = 512, 64
    x = workloads.generate(cfg, seed=12)
    d = to_dev(x)
    ref_i, ref_s = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"],
                                   options=lt.make_options(sorted_output=True))
    cand_rand, cand_hint = [], []
    prev = None
    for c0 in range(0, cfg.nq, chunk):
        sl = slice(c0, c0 + chunk)
        q, w, offs = d["q"][sl].contiguous(), d["w"][sl].contiguous(), d["offsets"][sl].contiguous()
        st_r = torch.zeros((chunk, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
        ri, rs = lt.indexer_topk(q, w, d["keys"], k, offs, options=lt.make_options(sorted_output=True, row_stats=st_r))
        np.testing.assert_array_equal(ri.cpu().numpy(), ref_i[sl].cpu().numpy())
        if prev is not None:
            hint = lt.sample_from_topk(prev, cfg.nk, 3 * k)
            st_h = torch.zeros((chunk, lt.LT_ROW_STATS), dtype=torch.int32, device="cuda")
            hi, hs = lt.indexer_topk(q, w, d["keys"], k, offs,
                                     options=lt.make_options(sorted_output=True, sample_keys=hint, row_stats=st_h))
            torch.cuda.synchronize()
            np.testing.assert_array_equal(hi.cpu().numpy(), ref_i[sl].cpu().numpy())
            np.testing.assert_array_equal(hs.cpu().numpy().view(np.uint32), ref_s[sl].cpu().numpy().view(np.uint32))
            cand_rand.append(st_r.cpu().numpy()[:, 0].mean())
            cand_hint.append(st_h.cpu().numpy()[:, 0].mean())
        prev = ri
    assert np.mean(cand_hint) <= 1.05 * np.mean(cand_rand), (cand_hint, cand_rand)
