"""GPU parity of the scores-in selection entries (lt_topk_select through the
sample / filter / select pipeline, and lt_topk_radix) against the oracle.
The bar is bit-exact: same index set, same score bits, and with sorted
output the same arrays."""
import numpy as np
import pytest
import torch

from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from parity import check_row_exact, visible

pytestmark = pytest.mark.gpu


def _offsets(rng, nq, nk, kind):
    if kind == "none":
        return None
    if kind == "causal":
        return workloads.causal_offsets(nq, nk)
    o = rng.integers(-3, nk + 5, size=nq).astype(np.int32)
    o[0] = 0
    if nq > 2:
        o[1] = nk + 100
        o[2] = 1
    return o


def _run(scores, nk, k, offs, entry, **opt):
    dev = torch.device("cuda")
    s = scores.to(dev)
    o = None if offs is None else torch.from_numpy(offs).to(dev)
    sorted_out = opt.pop("sorted_output", False)
    if entry == "select":
        stats = torch.full((scores.shape[0], lt.LT_ROW_STATS), -7, dtype=torch.int32, device=dev)
        opts = lt.make_options(sorted_output=sorted_out, row_stats=stats, **opt)
        gi, gs = lt.topk_select(s, k, num_keys=nk, causal_offsets=o, options=opts)
    else:
        stats = None
        gi, gs = lt.topk_radix(s, k, num_keys=nk, causal_offsets=o, sorted_output=sorted_out)
    torch.cuda.synchronize()
    return gi.cpu().numpy(), gs.cpu().numpy(), None if stats is None else stats.cpu().numpy()


def _check_all(scores, nk, k, offs, gi, gs, sorted_out):
    s = scores.numpy()
    ri, rs = orc.topk_select(s, nk, k, offs)
    e = visible(offs, s.shape[0], nk)
    for t in range(s.shape[0]):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e[t]), k, sorted_out)


CASES = [
    # nq, nk, ld, k, kind, offsets
    (7, 1000, 1000, 10, "normal", "none"),
    (33, 5000, 5004, 256, "ties", "causal"),
    (16, 4097, 4100, 100, "special", "random"),
    (9, 3000, 3000, 64, "const", "causal"),
    (64, 20000, 20000, 2048, "normal", "causal"),
    (5, 300, 300, 1, "ties", "random"),
    (5, 300, 300, 300, "normal", "none"),
    (4, 257, 260, 512, "special", "random"),
    (6, 40000, 40000, 8192, "ties", "causal"),     # the largest k (LT_K_MAX)
]


@pytest.mark.parametrize("entry", ["select", "radix"])
@pytest.mark.parametrize("sorted_out", [False, True])
@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}x{c[1]}k{c[3]}-{c[4]}-{c[5]}" for c in CASES])
def test_select_parity(lib, entry, sorted_out, case):
    nq, nk, ld, k, kind, okind = case
    rng = np.random.default_rng(nq * 7 + nk)
    scores = workloads.score_rows(nq, nk, seed=nq + k, kind=kind, ld=ld)
    offs = _offsets(rng, nq, nk, okind)
    gi, gs, stats = _run(scores, nk, k, offs, entry, sorted_output=sorted_out)
    _check_all(scores, nk, k, offs, gi, gs, sorted_out)
    if stats is not None:
        assert not np.any(stats[:, 2] == 4), "candidate count disagrees with the histogram"


@pytest.mark.parametrize("opt", [
    dict(force_fallback=True),
    dict(capacity=1),
    dict(num_bins=1),
    dict(sample_size=0),
    dict(num_bins=3, capacity=50),
    dict(key_splits=3),
    dict(num_bins=7),
], ids=lambda d: ",".join(f"{k}={v}" for k, v in d.items()))
def test_select_forced_paths_are_still_exact(lib, opt):
    nq, nk, k = 12, 9000, 300
    scores = workloads.score_rows(nq, nk, seed=5, kind="ties")
    offs = workloads.causal_offsets(nq, nk)
    gi, gs, stats = _run(scores, nk, k, offs, "select", sorted_output=True, **opt)
    _check_all(scores, nk, k, offs, gi, gs, True)
    if opt.get("force_fallback"):
        assert np.all(stats[:, 2] == 3)
    if opt.get("capacity") == 1:
        assert np.all(stats[:, 2] == 1)


@pytest.mark.parametrize("ns", [16384, 32768])
def test_select_long_sample(lib, ns):
    # samples of 16384 to 32768 keys (the range stage's wide blocks)
    nq, nk, k = 12, 40000, 300
    scores = workloads.score_rows(nq, nk, seed=9, kind="ties")
    offs = workloads.causal_offsets(nq, nk)
    gi, gs, stats = _run(scores, nk, k, offs, "select", sorted_output=True, sample_size=ns)
    _check_all(scores, nk, k, offs, gi, gs, True)


def test_select_row_stats_invariants(lib):
    """Invariants of the filter (sec. 3.2): the final threshold bin leaves
    fewer than k candidates above it, survivors stay below capacity, and the
    scan wrote far fewer candidates than keys."""
    nq, nk, k = 32, 131072, 2048
    scores = workloads.score_rows(nq, nk, seed=9, kind="normal")
    offs = workloads.causal_offsets(nq, nk)
    gi, gs, stats = _run(scores, nk, k, offs, "select", sorted_output=False)
    _check_all(scores, nk, k, offs, gi, gs, False)
    assert np.all(stats[:, 2] == 0)
    assert np.all(stats[:, 1] >= 0)
    assert np.all(stats[:, 0] < 12 * k)
    assert stats[:, 0].mean() < 0.25 * nk


def test_select_deterministic(lib):
    nq, nk, k = 20, 30000, 500
    scores = workloads.score_rows(nq, nk, seed=2, kind="ties")
    a = _run(scores, nk, k, None, "select")
    b = _run(scores, nk, k, None, "select")
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1].view(np.uint32), b[1].view(np.uint32))


def test_select_c1_shaped_rows(lib):
    """Rows of the 4096 x 131072 DSA workload's size (128K keys, k = 2048)."""
    nq, nk, k = 48, 131072, 2048
    scores = workloads.score_rows(nq, nk, seed=1, kind="normal")
    offs = workloads.causal_offsets(nq, nk)
    gi, gs, _ = _run(scores, nk, k, offs, "select", sorted_output=True)
    _check_all(scores, nk, k, offs, gi, gs, True)


def _order_key_edge_rows(n, seed):
    """Rows whose k-th score (k = 300) sits where the order-key digits of the
    radix passes meet the float encoding: among negative denormals (just
    below -0), at -inf, at NaN, at +inf, among positive denormals, at the
    largest finite float, and in rows of arbitrary bit patterns (NaN codes of
    either sign included)."""
    rng = np.random.default_rng(seed)

    def f32(b):
        return np.asarray(b, dtype=np.uint32).view(np.float32)

    rows = []
    r = f32(rng.integers(0x80000001, 0x80800000, n, dtype=np.uint64))  # negative denormals
    r[:60] = 1.0
    r[60:110] = 0.0
    r[110:160] = -0.0
    rows.append(r)
    r = np.full(n, -np.inf, np.float32)
    r[:50] = np.nan
    r[50:150] = np.inf
    r[150:250] = rng.standard_normal(100)
    rows.append(r)
    r = np.full(n, np.nan, np.float32)
    r[:100] = rng.standard_normal(100)
    rows.append(r)
    r = rng.standard_normal(n).astype(np.float32)
    r[:500] = np.inf
    rows.append(r)
    r = f32(rng.integers(1, 0x00800000, n, dtype=np.uint64))  # positive denormals
    r[:40] = 0.0
    r[40:80] = -0.0
    r[80:100] = -1.0
    rows.append(r)
    r = f32(rng.integers(0x7F7FF000, 0x7F800000, n, dtype=np.uint64))  # the largest finite floats
    r[:30] = np.inf
    r[30:60] = np.nan
    rows.append(r)
    for _ in range(2):
        rows.append(f32(rng.integers(0, 1 << 32, n, dtype=np.uint64)))
    for r in rows:
        rng.shuffle(r)
    # rows padded to a multiple of 4 floats with a large score the selection
    # must not see
    ld = (n + 3) // 4 * 4
    out = np.full((len(rows), ld), np.float32(3e38), np.float32)
    out[:, :n] = np.stack(rows)
    return torch.from_numpy(out)


@pytest.mark.parametrize("entry", ["radix", "select"])
@pytest.mark.parametrize("sorted_out", [False, True])
@pytest.mark.parametrize("n", [5000, 40001])
def test_radix_order_key_edges(lib, entry, sorted_out, n):
    """Exact selection where the k-th score is a special or boundary float
    (the scores-in entry with every row sent to the fallback's radix
    selection, and the plain radix entry)."""
    k = 300
    scores = _order_key_edge_rows(n, seed=n)
    opt = dict(force_fallback=True) if entry == "select" else {}
    gi, gs, _ = _run(scores, n, k, None, entry, sorted_output=sorted_out, **opt)
    _check_all(scores, n, k, None, gi, gs, sorted_out)


@pytest.mark.parametrize("sorted_out", [False, True])
def test_select_fallback_splits_few_long_rows(lib, sorted_out):
    """A few forced rows of a million scores take the scores-in fallback's
    split mode (each row's visible keys in chunks over many blocks, the last
    chunk's block merging the chunks' top k): rows of different lengths and
    starts, one shorter than k, one with special values, against the oracle."""
    nq, nk, k = 5, 1_000_001, 2048
    ld = (nk + 3) // 4 * 4
    rows = workloads.score_rows(nq, nk, seed=21, kind="ties", ld=ld).numpy()
    rows[4, : nk // 2] = workloads.score_rows(1, nk // 2, seed=22, kind="special").numpy()[0]
    scores = torch.from_numpy(rows)
    offs = np.array([nk, 700_001, 1000, nk, 999_999], dtype=np.int32)
    starts = np.array([0, 3, 0, 400_000, 1], dtype=np.int32)
    ri, rs = orc.topk_select(rows, nk, k, offs, visible_start=starts)
    gi, gs = lt.topk_select(scores.cuda(), k, num_keys=nk, causal_offsets=torch.from_numpy(offs).cuda(),
                            options=lt.make_options(sorted_output=sorted_out, force_fallback=True,
                                                    visible_start=torch.from_numpy(starts).cuda()))
    torch.cuda.synchronize()
    s0, e0 = orc.visible_ranges(offs, starts, nq, nk)
    gi, gs = gi.cpu().numpy(), gs.cpu().numpy()
    for t in range(nq):
        check_row_exact(gi[t], gs[t], ri[t], rs[t], int(e0[t] - s0[t]), k, sorted_out)
