"""GPU parity of the MFMA score stage (lt_indexer_scores, the dense score
matrix) against the oracle's Eq. (1): within the float32-accumulation
tolerance on real-valued inputs, bit-exact on inputs whose arithmetic is exact."""
import numpy as np
import pytest
import torch

from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import oracle_dense, to_dev

pytestmark = pytest.mark.gpu

# (dtype, mode, H, d) variants the library builds
VARIANTS = [
    ("f32", "dsa", 4, 64),
    ("f32", "dsa", 1, 64),
    ("f32", "ip", 1, 64),
    ("bf16", "dsa", 64, 128),
    ("bf16", "dsa", 4, 128),
    ("bf16", "dsa", 1, 128),
    ("bf16", "ip", 1, 128),
    ("fp8", "dsa", 64, 128),
    ("bf16", "ip", 1, 768),
    ("bf16", "dsa", 1, 768),
]


def _dense(x, mode):
    d = to_dev(x)
    out = lt.indexer_scores(d["q"], d["w"], d["keys"], d["q_scale"], d["k_scale"], mode=mode)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("var", VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_dense_scores_exact_inputs_bit_exact(lib, var):
    dtype, mode, h, d = var
    nq, nk = 37, 1000          # ragged against every query tile and key tile
    x = workloads.exact_inputs(nq, nk, h, d, dtype, seed=h + d, causal=False)
    if mode == "ip":
        x["w"] = None
    got = _dense(x, mode)
    want = oracle_dense(x, dtype, mode)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.parametrize("var", VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_dense_scores_real_inputs(lib, var):
    dtype, mode, h, d = var
    nq, nk = 21, 777
    base = workloads.CONFIGS["dsa_bf16_128k"] if h > 1 else workloads.CONFIGS["retrieval_bf16_4m"]
    cfg = workloads.scaled(base, nq=nq, nk=nk, h=h, d=d, dtype=dtype, mode=mode, causal=False)
    x = workloads.generate(cfg, seed=3)
    got = _dense(x, mode)
    want = oracle_dense(x, dtype, mode)
    rtol = 2e-2 if dtype == "fp8" else 1e-3
    # relative to the row's largest magnitude (the k-th score of any useful k
    # is of that order for these laws); fp32 accumulation of 64 x 128 terms
    scale = np.abs(want).max(axis=1, keepdims=True)
    err = np.abs(got.astype(np.float64) - want) / scale
    assert err.max() < rtol * 1e-1, err.max()


def test_dense_fp8_unit_scale_matches_decoded_values(lib):
    """Every E4M3FN code against one-hot keys: the score is the decoded value."""
    h, d = 64, 128
    codes = np.arange(256, dtype=np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x38           # NaN codes -> 1.0
    q = np.zeros((4, h, d), dtype=np.uint8)
    q[:, 0, :] = codes[: 4 * d].reshape(4, d) if 4 * d <= 256 else np.resize(codes, (4, d))
    keys = np.zeros((d, d), dtype=np.uint8)
    keys[np.arange(d), np.arange(d)] = 0x38        # identity (1.0)
    x = dict(q=torch.from_numpy(q), keys=torch.from_numpy(keys),
             q_scale=torch.ones((4, h), dtype=torch.float32), k_scale=torch.ones(d, dtype=torch.float32),
             w=torch.zeros((4, h), dtype=torch.float32), offsets=None)
    x["w"][:, 0] = 1.0
    got = _dense(x, "ip" if False else "dsa")
    want = oracle_dense(x, "fp8", "dsa")
    np.testing.assert_array_equal(got, want)
