"""Seeded synthetic inputs for the fused Indexer-TopK operation.

This module only draws random inputs and casts them to the storage formats the
library accepts. It holds none of the method's arithmetic (no scores, no
selection), so both the CPU oracle's tests and the GPU path can be fed from it.

Workload shapes follow the paper's kernel benchmarks (sec. 4.1, "Sparse-Attention
Kernel Benchmark" and "Large-Scale Retrieval Benchmark"): a DSA indexer with 64
heads of dimension 128, k = 2048 (sec. 2.1), a query chunk placed at the end of
a long context, and a single-head inner-product retrieval case. The paper's own
inputs (GLM-5.2 layer-1 activations on Wikipedia text; MSMARCO-v2.1 passage
embeddings) are not available, so every tensor here is drawn from a seeded
numpy PCG64 generator with the distributions listed in ``CONFIGS``.

Storage formats handed to the library:
  * "f32"  : float32 values.
  * "bf16" : bfloat16 (round-to-nearest-even from float32).
  * "fp8"  : OCP FP8 E4M3FN bytes with per-token float32 scales (keys: one scale
             per key; queries: one per (query, head)); scale = amax/448 and the
             payload is round-to-nearest-even of value/scale.

Every function returns CPU tensors; callers move them to the device.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

FP8_MAX = 448.0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    nq: int          # queries in the chunk
    nk: int          # keys in the context
    h: int           # indexer heads
    d: int           # head dimension
    dtype: str       # "f32" | "bf16" | "fp8"
    k: int
    mode: str        # "dsa" (ReLU, weighted head sum) | "ip" (inner product)
    causal: bool     # chunk at the end of the context, self-inclusive
    dist: str        # "iid" | "dsa_mean" | "unit" | "adversarial"


CONFIGS = {
    "tiny_fp32": Workload("tiny_fp32", 64, 4096, 4, 64, "f32", 256, "dsa", True, "iid"),
    "dsa_bf16_128k": Workload("dsa_bf16_128k", 4096, 131072, 64, 128, "bf16", 2048, "dsa", True, "dsa_mean"),
    "dsa_fp8_1m": Workload("dsa_fp8_1m", 2048, 1048576, 64, 128, "fp8", 2048, "dsa", True, "dsa_mean"),
    "retrieval_bf16_4m": Workload("retrieval_bf16_4m", 10000, 4000000, 1, 128, "bf16", 100, "ip", False, "unit"),
    "adversarial_bf16_256k": Workload("adversarial_bf16_256k", 1024, 262144, 64, 128, "bf16", 2048, "dsa", True, "adversarial"),
    # sec. 4.1 "Large-Scale Retrieval Benchmark": 768-dimensional passage
    # embeddings, a batch of 64 queries that are themselves corpus passages,
    # corpora of 1M-5M (the sweep takes prefixes), k from 128 to 8192
    "retrieval_e7_bf16_5m": Workload("retrieval_e7_bf16_5m", 64, 5000000, 1, 768, "bf16", 1024, "ip", False,
                                     "unit_self"),
}

# Queries of the "unit_self" law are drawn from the first QUERY_POOL corpus
# rows, so that every corpus prefix of at least that size contains them.
QUERY_POOL = 1000000

CONFIG_SEEDS = {name: i for i, name in enumerate(CONFIGS)}


def scaled(cfg: Workload, nq: Optional[int] = None, nk: Optional[int] = None, **kw) -> Workload:
    """The same workload law at a smaller (or different) shape."""
    return dataclasses.replace(cfg, nq=cfg.nq if nq is None else nq, nk=cfg.nk if nk is None else nk, **kw)


def causal_offsets(nq: int, nk: int) -> np.ndarray:
    """Visible-key counts for a chunk of nq queries that ends a context of nk
    tokens: query t sees keys [0, nk - nq + t + 1) (itself included)."""
    t = np.arange(nq, dtype=np.int64)
    return np.clip(nk - nq + t + 1, 0, nk).astype(np.int32)


def _normal(rng: np.random.Generator, shape, chunk=1 << 24) -> np.ndarray:
    out = np.empty(int(np.prod(shape)), dtype=np.float32)
    for s in range(0, out.size, chunk):
        e = min(out.size, s + chunk)
        rng.standard_normal(e - s, dtype=np.float32, out=out[s:e])
    return out.reshape(shape)


def _quantize_fp8(x: torch.Tensor, groups_dims: int):
    """Per-token E4M3FN quantisation. x is float32; the scale is taken over the
    trailing (head-dim) axis. Returns (uint8 payload, float32 scales)."""
    amax = x.abs().amax(dim=-1)
    scale = torch.where(amax > 0, amax / FP8_MAX, torch.ones_like(amax)).to(torch.float32)
    payload = (x / scale.unsqueeze(-1)).clamp_(-FP8_MAX, FP8_MAX).to(torch.float8_e4m3fn)
    return payload.view(torch.uint8), scale


def _cast(x: np.ndarray, dtype: str):
    t = torch.from_numpy(x)
    if dtype == "f32":
        return t.contiguous(), None
    if dtype == "bf16":
        return t.to(torch.bfloat16).contiguous(), None
    if dtype == "fp8":
        p, s = _quantize_fp8(t, 1)
        return p.contiguous(), s.contiguous()
    raise ValueError(dtype)


def generate(cfg: Workload, seed: int) -> dict:
    """Draw one workload. Keys of the returned dict:

    q        [nq, h, d]  storage dtype (float32, bfloat16, or uint8 E4M3FN bytes)
    q_scale  [nq, h]     float32 (fp8 only, else None)
    w        [nq, h]     float32 head weights (None in inner-product mode)
    keys     [nk, d]     storage dtype
    k_scale  [nk]        float32 (fp8 only, else None)
    offsets  [nq]        int32 visible-key counts (None when not causal)
    q_f32, keys_f32      the float32 values before the storage cast
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    nq, nk, h, d = cfg.nq, cfg.nk, cfg.h, cfg.d
    if cfg.dist == "iid":
        q = _normal(rng, (nq, h, d))
        keys = _normal(rng, (nk, d))
    elif cfg.dist == "dsa_mean":
        # A shared per-sequence mean vector added to every key and every query
        # head concentrates the scores in a narrow band (the paper's sec. 1
        # observation on DSA scores).
        mu = _normal(rng, (d,)) / np.float32(np.sqrt(d))
        inv = np.float32(1.0 / np.sqrt(d))
        q = _normal(rng, (nq, h, d))
        q *= inv
        q += mu
        keys = _normal(rng, (nk, d))
        keys *= inv
        keys += mu
    elif cfg.dist == "unit":
        q = _normal(rng, (nq, h, d))
        q /= np.linalg.norm(q, axis=-1, keepdims=True)
        keys = _normal(rng, (nk, d))
        keys /= np.linalg.norm(keys, axis=-1, keepdims=True)
    elif cfg.dist == "unit_self":
        # unit-normalised Gaussian passages; the queries are copies of
        # distinct passages (the paper samples its queries from the corpus)
        keys = _normal(rng, (nk, d))
        for s0 in range(0, nk, 1 << 16):
            blk = keys[s0:s0 + (1 << 16)]
            blk /= np.linalg.norm(blk, axis=-1, keepdims=True)
        pick = rng.choice(min(nk, QUERY_POOL), size=nq, replace=nq > min(nk, QUERY_POOL))
        q = np.ascontiguousarray(keys[pick][:, None, :].repeat(h, axis=1))
    elif cfg.dist == "adversarial":
        # 99.9% N(0, 1) keys, 0.1% outliers scaled by 20, and 1% of keys
        # replaced by exact copies of other random keys (duplicate-score ties).
        q = _normal(rng, (nq, h, d))
        q *= np.float32(1.0 / np.sqrt(d))
        keys = _normal(rng, (nk, d))
        outlier = rng.random(nk) < 0.001
        keys[outlier] *= np.float32(20.0)
        ndup = max(1, nk // 100)
        dst = rng.choice(nk, size=ndup, replace=False)
        src = rng.integers(0, nk, size=ndup)
        keys[dst] = keys[src]
    else:
        raise ValueError(cfg.dist)

    qs, q_scale = _cast(q, cfg.dtype)
    ks, k_scale = _cast(keys, cfg.dtype)
    w = None
    if cfg.mode == "dsa":
        w = torch.from_numpy(rng.random((nq, h), dtype=np.float32))
    offsets = torch.from_numpy(causal_offsets(nq, nk)) if cfg.causal else None
    return dict(q=qs, q_scale=q_scale, w=w, keys=ks, k_scale=k_scale, offsets=offsets,
                q_f32=torch.from_numpy(q), keys_f32=torch.from_numpy(keys))


def unit_corpus_gpu(cfg: Workload, seed: int, device, nk: Optional[int] = None) -> dict:
    """The "unit_self" law at corpus sizes numpy would take minutes to draw:
    keys drawn on ``device`` by torch's seeded generator (Philox), in chunks of
    2**20 rows, normalised in float32 and rounded to bfloat16; the nq queries
    are copies of distinct rows among the first QUERY_POOL (picked by a seeded
    CPU generator). It draws the same law as generate() but from a different
    random stream, so its corpus is not generate()'s. Returns the generate()
    keys q, w (None), keys, offsets (None) on ``device``, plus "pick" (the
    query rows)."""
    import torch as _t
    nk = cfg.nk if nk is None else nk
    g = _t.Generator(device=device)
    g.manual_seed(seed)
    keys = _t.empty((nk, cfg.d), dtype=_t.bfloat16, device=device)
    for s0 in range(0, nk, 1 << 20):
        n = min(1 << 20, nk - s0)
        x = _t.randn((n, cfg.d), generator=g, device=device, dtype=_t.float32)
        x /= x.norm(dim=1, keepdim=True)
        keys[s0:s0 + n] = x.to(_t.bfloat16)
        del x
    rng = np.random.Generator(np.random.PCG64(seed))
    pool = min(nk, QUERY_POOL)
    pick = rng.choice(pool, size=cfg.nq, replace=cfg.nq > pool)
    q = keys[_t.from_numpy(pick).to(device)].unsqueeze(1).repeat(1, cfg.h, 1).contiguous()
    return dict(q=q, q_scale=None, w=None, keys=keys, k_scale=None, offsets=None, pick=pick)


def exact_inputs(nq: int, nk: int, h: int, d: int, dtype: str, seed: int, causal: bool = True):
    """Inputs on which every product and partial sum of the score is exactly
    representable in float32, so any summation order gives the same bits:
    small integers for q and keys, power-of-two head weights (and scales for
    fp8), with |sums| far below 2**24."""
    rng = np.random.Generator(np.random.PCG64(seed))
    qv = rng.integers(-3, 4, size=(nq, h, d)).astype(np.float32)
    kv = rng.integers(-3, 4, size=(nk, d)).astype(np.float32)
    w = (2.0 ** rng.integers(-3, 2, size=(nq, h))).astype(np.float32)
    out = dict(w=torch.from_numpy(w), q_f32=torch.from_numpy(qv), keys_f32=torch.from_numpy(kv),
               offsets=torch.from_numpy(causal_offsets(nq, nk)) if causal else None)
    if dtype == "fp8":
        # Small integers are exact in E4M3FN; scales are powers of two.
        out["q"] = torch.from_numpy(qv).to(torch.float8_e4m3fn).view(torch.uint8).contiguous()
        out["keys"] = torch.from_numpy(kv).to(torch.float8_e4m3fn).view(torch.uint8).contiguous()
        out["q_scale"] = torch.from_numpy((2.0 ** rng.integers(-2, 3, size=(nq, h))).astype(np.float32))
        out["k_scale"] = torch.from_numpy((2.0 ** rng.integers(-2, 3, size=(nk,))).astype(np.float32))
    else:
        out["q"], _ = _cast(qv, dtype)
        out["keys"], _ = _cast(kv, dtype)
        out["q_scale"] = None
        out["k_scale"] = None
    return out


def score_rows(nq: int, nk: int, seed: int, kind: str = "normal", ld: Optional[int] = None) -> torch.Tensor:
    """fp32 score matrices for the scores-in selection entry. ``kind``:
    normal     N(0, 1);
    ties       N(0, 1) rounded to multiples of 1/8 (many exact duplicates);
    special    normal values with NaN, +-inf and +-0 sprinkled in;
    const      every score equal (a single value).
    ``ld`` >= nk pads each row (the padding holds garbage that must be ignored)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ld = nk if ld is None else ld
    s = _normal(rng, (nq, ld))
    if kind == "ties":
        s = np.round(s * 8.0) / np.float32(8.0)
    elif kind == "special":
        u = rng.random((nq, ld))
        s[u < 0.01] = np.nan
        s[(u >= 0.01) & (u < 0.02)] = np.inf
        s[(u >= 0.02) & (u < 0.03)] = -np.inf
        s[(u >= 0.03) & (u < 0.04)] = 0.0
        s[(u >= 0.04) & (u < 0.05)] = -0.0
    elif kind == "const":
        s[:] = np.float32(1.5)
    elif kind != "normal":
        raise ValueError(kind)
    if ld > nk:
        s[:, nk:] = np.float32(1e30)
    return torch.from_numpy(s.astype(np.float32))


def packed_batch(cfg: Workload, lens, nqs, seed: int):
    """Several sequences of the ``cfg`` law packed into one batch: sequence b
    has lens[b] keys and its last nqs[b] positions as queries. Keys are
    concatenated ([sum(lens), d]), queries too; row t of sequence b sees its
    own sequence's causal prefix [base_b, base_b + e_local) through
    offsets (ends) and starts. Returns the generate() dict plus "starts"
    (int32 [Nq]) and "bases"."""
    parts = [generate(scaled(cfg, nq=n, nk=L), seed=seed + 7 * b) for b, (L, n) in enumerate(zip(lens, nqs))]
    bases = np.cumsum([0] + list(lens[:-1])).astype(np.int64)
    out = {}
    for key in ("q", "w", "keys", "q_scale", "k_scale"):
        vals = [p_[key] for p_ in parts]
        out[key] = None if vals[0] is None else torch.cat(vals, 0).contiguous()
    ends, starts = [], []
    for b, (p_, L, n) in enumerate(zip(parts, lens, nqs)):
        e_local = p_["offsets"].numpy().astype(np.int64) if p_["offsets"] is not None else np.full(n, L)
        ends.append(bases[b] + e_local)
        starts.append(np.full(n, bases[b]))
    out["offsets"] = torch.from_numpy(np.concatenate(ends).astype(np.int32))
    out["starts"] = torch.from_numpy(np.concatenate(starts).astype(np.int32))
    out["bases"] = bases
    return out
