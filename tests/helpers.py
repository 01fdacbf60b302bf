"""Glue between the seeded workloads, the GPU binding and the CPU oracle."""
from __future__ import annotations

import numpy as np
import torch

from oracle import litetopk_oracle as orc


def storage_np(t: torch.Tensor, dtype: str) -> np.ndarray:
    """Storage tensor -> the numpy form the oracle decodes itself."""
    t = t.cpu()
    if dtype == "f32":
        return t.numpy()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16)
    if dtype == "fp8":
        return t.view(torch.uint8).numpy()
    raise ValueError(dtype)


def oracle_topk(x: dict, dtype: str, k: int, mode: str, rows=None):
    """Oracle (idx, scores, full score rows) for a generated workload."""
    return orc.indexer_topk(
        storage_np(x["q"], dtype), dtype, None if x.get("q_scale") is None else x["q_scale"].numpy(),
        None if x.get("w") is None else x["w"].numpy(), storage_np(x["keys"], dtype),
        None if x.get("k_scale") is None else x["k_scale"].numpy(), k, mode,
        None if x.get("offsets") is None else x["offsets"].numpy(), rows=rows, return_scores=True,
        visible_start=None if x.get("starts") is None else x["starts"].numpy())


def oracle_dense(x: dict, dtype: str, mode: str, rows=None):
    qd = orc.dequantize(storage_np(x["q"], dtype), dtype, None if x.get("q_scale") is None else x["q_scale"].numpy())
    kd = orc.dequantize(storage_np(x["keys"], dtype), dtype,
                        None if x.get("k_scale") is None else x["k_scale"].numpy())
    wd = None if x.get("w") is None else x["w"].numpy().astype(np.float64)
    return orc.index_scores(qd, wd, kd, mode, rows=rows)


def to_dev(x: dict, dev="cuda"):
    keys = ("q", "q_scale", "w", "keys", "k_scale", "offsets", "starts")
    return {n: (None if x.get(n) is None else x[n].to(dev)) for n in keys}
