"""The allocation-free entry point (lt_indexer_topk_static) against
lt_indexer_topk with a caller workspace, called through the C ABI: the same
results bit for bit, on two calls in a row where the second is smaller (the
static scratch keeps the first call's contents), on each compiled score
layout; no device memory is allocated by the static calls (torch's
allocator is not touched; the library allocates nothing itself); and a shape
too large for the static scratch is refused without device work."""
import numpy as np
import pytest
import torch

from paper_2607_11976_amd import litetopk as lt
from paper_2607_11976_amd import workloads
from helpers import to_dev

pytestmark = pytest.mark.gpu

# (id, base config, [(nq, nk, k), (smaller nq, nk, k)])
CASES = [
    ("dsa_bf16_h64", "dsa_bf16_128k", [(40, 20011, 512), (17, 9001, 256)]),
    ("dsa_fp8_h64", "dsa_fp8_1m", [(16, 30001, 2048), (9, 12000, 1000)]),
    ("dsa_f32_h4", "tiny_fp32", [(64, 4096, 256), (30, 2000, 100)]),
    ("ip_bf16_h1", "retrieval_bf16_4m", [(70, 50000, 100), (33, 20001, 64)]),
    ("ip_bf16_d768", "retrieval_e7_bf16_5m", [(64, 20000, 128), (20, 9000, 50)]),
]


def _raw_static(d, cfg, k, out_i, out_s, opts):
    dt = lt._dtype_code(d["q"])
    nq, h, dd = d["q"].shape
    p = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    return lt.lt_indexer_topk_static(p(d["q"]), p(d["q_scale"]), p(d["w"]), p(d["keys"]), p(d["k_scale"]), dt,
                                     lt._mode_code(cfg.mode), nq, d["keys"].shape[0], h, dd, k, p(d["offsets"]),
                                     out_i.data_ptr(), out_s.data_ptr(), opts,
                                     torch.cuda.current_stream().cuda_stream)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_static_scratch_matches_workspace_entry(lib, case):
    name, base, shapes = case
    for call, (nq, nk, k) in enumerate(shapes):
        cfg = workloads.scaled(workloads.CONFIGS[base], nq=nq, nk=nk)
        x = workloads.generate(cfg, seed=40 + call)
        d = to_dev(x)
        print("static scratch: %s call %d nq=%d nk=%d k=%d" % (name, call, nq, nk, k), flush=True)
        need = lt.lt_indexer_topk_workspace_size(nq, nk, cfg.h, cfg.d, lt._dtype_code(d["q"]),
                                                 lt._mode_code(cfg.mode), k)
        assert 0 < need <= lt.LT_STATIC_SCRATCH_BYTES
        # the caller-workspace entry point
        st_ref = torch.full((nq, lt.LT_ROW_STATS), -7, dtype=torch.int32, device="cuda")
        ri, rs = lt.indexer_topk(d["q"], d["w"], d["keys"], k, d["offsets"], d["q_scale"], d["k_scale"],
                                 mode=cfg.mode, options=lt.make_options(row_stats=st_ref))
        # the static-scratch entry point, outputs allocated beforehand
        gi = torch.full((nq, k), -9, dtype=torch.int32, device="cuda")
        gs = torch.full((nq, k), 7.0, dtype=torch.float32, device="cuda")
        st = torch.full((nq, lt.LT_ROW_STATS), -7, dtype=torch.int32, device="cuda")
        opts = lt.make_options(row_stats=st)
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        rc = _raw_static(d, cfg, k, gi, gs, opts)
        assert rc == lt.LT_OK, lt.lt_strerror(rc)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        np.testing.assert_array_equal(gi.cpu().numpy(), ri.cpu().numpy())
        np.testing.assert_array_equal(gs.cpu().numpy().view(np.uint32), rs.cpu().numpy().view(np.uint32))
        # every row statistic but the count of candidates written: where key
        # splits share thresholds that count depends on when each split sees
        # the others' published bins, in any two calls
        np.testing.assert_array_equal(st.cpu().numpy()[:, 1:], st_ref.cpu().numpy()[:, 1:])


def test_static_scratch_refuses_large_shapes(lib):
    cfg = workloads.scaled(workloads.CONFIGS["dsa_bf16_128k"], nq=512, nk=131072)
    need = lt.lt_indexer_topk_workspace_size(cfg.nq, cfg.nk, cfg.h, cfg.d, lt.LT_BF16, lt.LT_SCORE_DSA, cfg.k)
    assert need > lt.LT_STATIC_SCRATCH_BYTES
    q = torch.zeros((cfg.nq, cfg.h, cfg.d), dtype=torch.bfloat16, device="cuda")
    keys = torch.zeros((cfg.nk, cfg.d), dtype=torch.bfloat16, device="cuda")
    out = (torch.empty((cfg.nq, cfg.k), dtype=torch.int32, device="cuda"),
           torch.empty((cfg.nq, cfg.k), dtype=torch.float32, device="cuda"))
    with pytest.raises(lt.LiteTopKError, match="static scratch"):
        lt.indexer_topk_static(q, None, keys, cfg.k, out=out)
