"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every symbol the header declares, and its argument checks and workspace
sizing behave as documented (no device work is enqueued by these calls)."""
import ctypes
import os
import re

import pytest

from paper_2607_11976_amd import litetopk as lt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "litetopk.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(lt_[a-z_0-9]+)\s*\(", src)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lt.LIB_PATH):
        pytest.fail("liblitetopk.so is not built; run python -m paper_2607_11976_amd.build")
    return lt.load()


def test_library_exports_every_header_symbol(lib):
    names = header_functions()
    assert len(names) >= 12
    assert set(names) == set(lt.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_options_struct_layout_and_defaults(lib):
    assert ctypes.sizeof(lt.LtOptions) == 64  # 5 x int32/uint32, pad, seed, 4 pointers
    o = lt.lt_options_default()
    assert o.num_bins == 256 and o.sample_size < 0 and o.capacity == 0 and o.key_splits == 0
    assert o.flags == 0 and not o.stage_events and not o.row_stats and not o.sample_keys
    assert not o.visible_start


def test_strerror(lib):
    assert lt.lt_strerror(0) == "ok"
    assert "workspace" in lt.lt_strerror(lt.LT_EWORKSPACE)
    assert "unknown" in lt.lt_strerror(-99)


def test_workspace_sizes(lib):
    n1 = lt.lt_indexer_topk_workspace_size(4096, 131072, 64, 128, lt.LT_BF16, lt.LT_SCORE_DSA, 2048)
    # candidate buffer alone: 4096 rows * 12k slots * 8 bytes
    assert n1 >= 4096 * 12 * 2048 * 8
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256) > 0
    # unsupported shapes and k report 0
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 3, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256) == 0
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 0) == 0
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 8193) == 0
    o = lt.lt_options_default()
    o.capacity = 100
    small = lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256, o)
    assert 0 < small < lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256)
    assert lt.lt_topk_select_workspace_size(128, 1000, 10) > 0
    assert lt.lt_topk_select_workspace_size(128, 1000, 0) == 0
    # a sample list needs a length in [1, LT_SAMPLE_LIST_MAX]
    o = lt.lt_options_default()
    o.sample_keys = 256
    o.sample_size = 0
    assert lt.lt_topk_select_workspace_size(128, 1000, 10, o) == 0
    o.sample_size = lt.LT_SAMPLE_LIST_MAX + 1
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256, o) == 0
    o.sample_size = 1000
    assert lt.lt_indexer_topk_workspace_size(64, 4096, 4, 64, lt.LT_F32, lt.LT_SCORE_DSA, 256, o) > 0
    # the 768-d one-head shapes (the wide scan): per-(row, split) lists of
    # k + max(1024, k/2) slots over 256 splits for a 64-query batch, plus one
    # shared histogram per row; other long dims are not built
    for mode in (lt.LT_SCORE_IP, lt.LT_SCORE_DSA):
        w = lt.lt_indexer_topk_workspace_size(64, 5000000, 1, 768, lt.LT_BF16, mode, 1024)
        assert w >= 64 * 256 * (1024 + 1024) * 8
    assert lt.lt_indexer_topk_workspace_size(64, 5000000, 1, 768, lt.LT_F32, lt.LT_SCORE_IP, 1024) == 0
    assert lt.lt_indexer_topk_workspace_size(64, 5000000, 1, 512, lt.LT_BF16, lt.LT_SCORE_IP, 1024) == 0
    assert lt.lt_indexer_topk_workspace_size(64, 5000000, 2, 768, lt.LT_BF16, lt.LT_SCORE_IP, 1024) == 0
    # previous-chunk sampler: the per-key counts dominate
    assert lt.lt_sample_from_topk_workspace_size(1 << 20) >= 4 << 20
    assert lt.lt_sample_from_topk_workspace_size(-1) == 0


def test_argument_checks_reject_before_any_device_work(lib):
    P = 256  # a fake, aligned, never dereferenced address
    # null q
    assert lt.lt_indexer_topk(None, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                              P, P, P, 1 << 20, None, None) == lt.LT_EINVAL
    # misaligned keys
    assert lt.lt_indexer_topk(P, None, None, P + 4, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                              P, P, P, 1 << 20, None, None) == lt.LT_EINVAL
    # unsupported head count
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 3, 64, 2, None,
                              P, P, P, 1 << 20, None, None) == lt.LT_EUNSUPPORTED
    # k out of range
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 0, None,
                              P, P, P, 1 << 20, None, None) == lt.LT_EINVAL
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 9000, None,
                              P, P, P, 1 << 20, None, None) == lt.LT_EUNSUPPORTED
    # fp8 without scales
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_FP8_E4M3FN, lt.LT_SCORE_DSA, 4, 8, 64, 128, 2,
                              None, P, P, P, 1 << 30, None, None) == lt.LT_EINVAL
    # workspace too small
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                              P, P, P, 16, None, None) == lt.LT_EWORKSPACE
    # workspace misaligned
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                              P, P, P + 8, 1 << 20, None, None) == lt.LT_EINVAL
    # select: stride smaller than num_keys, stride not a multiple of 4, k too large
    assert lt.lt_topk_select(P, 7, 2, 8, 2, None, P, P, P, 1 << 20, None, None) == lt.LT_EINVAL
    assert lt.lt_topk_select(P, 10, 2, 8, 2, None, P, P, P, 1 << 20, None, None) == lt.LT_EINVAL
    assert lt.lt_topk_select(P, 8, 2, 8, 9000, None, P, P, P, 1 << 20, None, None) == lt.LT_EUNSUPPORTED
    assert lt.lt_topk_select(P, 8, 2, 8, 2, None, P, P, P, 16, None, None) == lt.LT_EWORKSPACE
    assert lt.lt_topk_radix(P, 8, 2, 8, 0, None, P, P, 0, None) == lt.LT_EINVAL
    assert lt.lt_indexer_scores(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 2, 8, 4, 64, P, 4,
                                None) == lt.LT_EINVAL
    # sample list with a bad length
    o = lt.lt_options_default()
    o.sample_keys = P
    o.sample_size = 0
    assert lt.lt_indexer_topk(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                              P, P, P, 1 << 20, o, None) == lt.LT_EINVAL
    assert lt.lt_topk_select(P, 8, 2, 8, 2, None, P, P, P, 1 << 20, o, None) == lt.LT_EINVAL
    # previous-chunk sampler: sample size, ld < k, workspace
    ws = lt.lt_sample_from_topk_workspace_size(100)
    assert lt.lt_sample_from_topk(P, 4, 2, 4, 100, 0, P, P, ws, None) == lt.LT_EINVAL
    assert lt.lt_sample_from_topk(P, 4, 2, 4, 100, lt.LT_SAMPLE_LIST_MAX + 1, P, P, ws, None) == lt.LT_EINVAL
    assert lt.lt_sample_from_topk(P, 3, 2, 4, 100, 10, P, P, ws, None) == lt.LT_EINVAL
    assert lt.lt_sample_from_topk(None, 4, 2, 4, 100, 10, P, P, ws, None) == lt.LT_EINVAL
    assert lt.lt_sample_from_topk(P, 4, 2, 4, 100, 10, P, P, ws - 1, None) == lt.LT_EWORKSPACE
    assert lt.lt_sample_from_topk(P, 4, 2, 4, 100, 10, P, P + 8, ws, None) == lt.LT_EINVAL
    # union builder: group * k over the limit, ld < k, null outputs
    assert lt.lt_dsa_union(P, 8, 4, 8, lt.LT_UNION_MAX // 8 + 1, P, P, P, None) == lt.LT_EINVAL
    assert lt.lt_dsa_union(P, 7, 4, 8, 2, P, P, P, None) == lt.LT_EINVAL
    assert lt.lt_dsa_union(P, 8, 4, 8, 0, P, P, P, None) == lt.LT_EINVAL
    assert lt.lt_dsa_union(P, 8, 4, 8, 2, P, None, P, None) == lt.LT_EINVAL
    assert lt.lt_dsa_union(None, 8, 0, 8, 2, None, None, None, None) == lt.LT_OK
    # the static-scratch variant: argument errors as lt_indexer_topk, and a
    # shape whose workspace exceeds the static array is refused on the host
    assert lt.lt_indexer_topk_static(None, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 4, 64, 2, None,
                                     P, P, None, None) == lt.LT_EINVAL
    assert lt.lt_indexer_topk_static(P, None, None, P, None, lt.LT_F32, lt.LT_SCORE_DSA, 4, 8, 3, 64, 2, None,
                                     P, P, None, None) == lt.LT_EUNSUPPORTED
    need = lt.lt_indexer_topk_workspace_size(4096, 131072, 64, 128, lt.LT_BF16, lt.LT_SCORE_DSA, 2048)
    assert need > lt.LT_STATIC_SCRATCH_BYTES
    assert lt.lt_indexer_topk_static(P, None, P, P, None, lt.LT_BF16, lt.LT_SCORE_DSA, 4096, 131072, 64, 128, 2048,
                                     None, P, P, None, None) == lt.LT_ESCRATCH
    assert "static scratch" in lt.lt_strerror(lt.LT_ESCRATCH)
    assert lt.lt_indexer_topk_static(None, None, None, None, None, lt.LT_F32, lt.LT_SCORE_DSA, 0, 0, 4, 64, 2, None,
                                     None, None, None, None) == lt.LT_OK
    # empty problems are valid and do nothing
    assert lt.lt_indexer_topk(None, None, None, None, None, lt.LT_F32, lt.LT_SCORE_DSA, 0, 0, 4, 64, 2, None,
                              None, None, None, 0, None, None) == lt.LT_OK
    assert lt.lt_topk_radix(None, 0, 0, 0, 5, None, None, None, 0, None) == lt.LT_OK
