"""GPU parity of the LiteDSA union builder (lt_dsa_union, sec. 3.3) against
the oracle: bit-exact union lists, sizes and membership masks, for groups of
1 to 16 rows, short last groups, padding and repeated keys within a row, the
largest group * k, and real fused top-k output of the 128K DSA law."""
import numpy as np
import pytest
import torch

from oracle import litetopk_oracle as orc
from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import to_dev
from test_oracle import UNION_CASES, check_union_invariants, union_case_input

pytestmark = pytest.mark.gpu


def _gpu_union(idx, group):
    t = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
    u, c, m = lt.dsa_union(t, group)
    torch.cuda.synchronize()
    return u.cpu().numpy(), c.cpu().numpy(), m.cpu().numpy().view(np.uint32)


def _check(idx, group):
    u, c, m = _gpu_union(idx, group)
    ru, rc, rm = orc.dsa_union(idx, group)
    np.testing.assert_array_equal(c, rc)
    np.testing.assert_array_equal(u, ru)
    np.testing.assert_array_equal(m, rm)
    check_union_invariants(u, c, m, idx, group)


@pytest.mark.parametrize("case", UNION_CASES, ids=[f"{c[0]}x{c[1]}-g{c[2]}" for c in UNION_CASES])
def test_union_matches_oracle(lib, case):
    nq, k, group, keys, pad = case
    _check(union_case_input(nq, k, keys, pad, seed=nq * k + group), group)


@pytest.mark.parametrize("nq,k,group", [(33, 64, 4), (5, 1, 2), (100, 300, 16), (17, 2048, 16), (8, 4096, 8),
                                        (3, 8192, 4), (1, 32768, 1)])
def test_union_shapes(lib, nq, k, group):
    """Ragged last groups, k = 1, and group * k up to LT_UNION_MAX."""
    idx = union_case_input(nq, k, keys=max(4 * k, 50), pad=0.05, seed=nq + k + group)
    _check(idx, group)


def test_union_all_padding_and_strided_rows(lib):
    idx = np.full((6, 10), -1, dtype=np.int32)
    _check(idx, 4)
    full = union_case_input(12, 40, 500, 0.1, seed=3)
    t = torch.from_numpy(full).cuda()[:, :16]
    u, c, m = lt.dsa_union(t, 5)
    torch.cuda.synchronize()
    ru, rc, rm = orc.dsa_union(full[:, :16], 5)
    np.testing.assert_array_equal(u.cpu().numpy(), ru)
    np.testing.assert_array_equal(c.cpu().numpy(), rc)
    np.testing.assert_array_equal(m.cpu().numpy().view(np.uint32), rm)


def test_union_of_fused_topk(lib):
    """Top-2048 lists of 64 rows of the 128K DSA law (neighbouring rows share
    most of their keys), groups of 4 and 16."""
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=64)
    x = workloads.generate(cfg, seed=9)
    d = to_dev(x)
    gi, _ = lt.indexer_topk(d["q"], d["w"], d["keys"], cfg.k, d["offsets"])
    torch.cuda.synchronize()
    idx = gi.cpu().numpy()
    for group in (4, 16):
        _check(idx, group)
