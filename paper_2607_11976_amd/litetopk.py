"""Python binding of the C ABI in include/litetopk.h (argument marshalling only).

Every computation runs in the HIP library liblitetopk.so built next to this
file (``python -m paper_2607_11976_amd.build``). torch is used for device
memory and streams: tensors hand over their device pointers and the current
HIP stream. There is no CPU fallback: if the library is missing or no GPU is
visible, the calls raise.

Two layers:
  * the raw entry points with the C names (``lt_indexer_topk`` ...), taking
    integers for pointers, exactly as declared in the header;
  * convenience wrappers (``indexer_topk``, ``topk_select``, ...) that check
    tensor shapes, allocate outputs and workspace with torch and call them.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# LT_LIBRARY names another build of the same library (the host-sanitizer
# build that tests/test_abi_sanitized.py makes); default: the in-tree build
LIB_PATH = os.environ.get("LT_LIBRARY") or os.path.join(_HERE, "liblitetopk.so")

LT_OK, LT_EINVAL, LT_EUNSUPPORTED, LT_EWORKSPACE, LT_EHIP, LT_ESCRATCH = 0, -1, -2, -3, -4, -5
LT_F32, LT_BF16, LT_FP8_E4M3FN = 0, 1, 2
LT_SCORE_DSA, LT_SCORE_IP = 0, 1
LT_SORTED_OUTPUT, LT_FORCE_FALLBACK = 1, 2
LT_K_MAX = 8192
LT_SAMPLE_LIST_MAX = 32768
LT_UNION_MAX = 32768
LT_ROW_STATS = 12
LT_STATIC_SCRATCH_BYTES = 256 << 20
LT_NUM_STAGE_EVENTS = 6
STAGES = ("sample", "range", "filter", "select", "fallback")

EXPORTED = (
    "lt_options_default", "lt_indexer_topk_workspace_size", "lt_indexer_topk", "lt_indexer_topk_static",
    "lt_indexer_scores",
    "lt_topk_select_workspace_size", "lt_topk_select", "lt_topk_radix",
    "lt_sample_from_topk_workspace_size", "lt_sample_from_topk", "lt_dsa_union", "lt_event_create",
    "lt_event_destroy", "lt_event_record", "lt_event_elapsed_ms", "lt_strerror",
)


class LtOptions(ctypes.Structure):
    _fields_ = [
        ("num_bins", ctypes.c_int32),
        ("sample_size", ctypes.c_int32),
        ("capacity", ctypes.c_int32),
        ("key_splits", ctypes.c_int32),
        ("flags", ctypes.c_uint32),
        ("seed", ctypes.c_uint64),
        ("stage_events", ctypes.c_void_p),
        ("row_stats", ctypes.c_void_p),
        ("sample_keys", ctypes.c_void_p),
        ("visible_start", ctypes.c_void_p),
    ]


class LiteTopKError(RuntimeError):
    pass


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t


def load(path: str = LIB_PATH):
    """Load the shared library (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise LiteTopKError("HIP library not built: %s (run python -m paper_2607_11976_amd.build)" % path)
    lib = ctypes.CDLL(path)
    lib.lt_options_default.argtypes = [ctypes.POINTER(LtOptions)]
    lib.lt_options_default.restype = None
    lib.lt_indexer_topk_workspace_size.argtypes = [_I32, _I32, _I32, _I32, ctypes.c_int, ctypes.c_int, _I32,
                                                   ctypes.POINTER(LtOptions)]
    lib.lt_indexer_topk_workspace_size.restype = _SZ
    lib.lt_indexer_topk.argtypes = [_P, _P, _P, _P, _P, ctypes.c_int, ctypes.c_int, _I32, _I32, _I32, _I32, _I32,
                                    _P, _P, _P, _P, _SZ, ctypes.POINTER(LtOptions), _P]
    lib.lt_indexer_topk.restype = ctypes.c_int
    lib.lt_indexer_topk_static.argtypes = [_P, _P, _P, _P, _P, ctypes.c_int, ctypes.c_int, _I32, _I32, _I32, _I32,
                                           _I32, _P, _P, _P, ctypes.POINTER(LtOptions), _P]
    lib.lt_indexer_topk_static.restype = ctypes.c_int
    lib.lt_indexer_scores.argtypes = [_P, _P, _P, _P, _P, ctypes.c_int, ctypes.c_int, _I32, _I32, _I32, _I32,
                                      _P, _I64, _P]
    lib.lt_indexer_scores.restype = ctypes.c_int
    lib.lt_topk_select_workspace_size.argtypes = [_I32, _I32, _I32, ctypes.POINTER(LtOptions)]
    lib.lt_topk_select_workspace_size.restype = _SZ
    lib.lt_topk_select.argtypes = [_P, _I64, _I32, _I32, _I32, _P, _P, _P, _P, _SZ, ctypes.POINTER(LtOptions), _P]
    lib.lt_topk_select.restype = ctypes.c_int
    lib.lt_topk_radix.argtypes = [_P, _I64, _I32, _I32, _I32, _P, _P, _P, ctypes.c_uint32, _P]
    lib.lt_topk_radix.restype = ctypes.c_int
    lib.lt_sample_from_topk_workspace_size.argtypes = [_I32]
    lib.lt_sample_from_topk_workspace_size.restype = _SZ
    lib.lt_sample_from_topk.argtypes = [_P, _I64, _I32, _I32, _I32, _I32, _P, _P, _SZ, _P]
    lib.lt_sample_from_topk.restype = ctypes.c_int
    lib.lt_dsa_union.argtypes = [_P, _I64, _I32, _I32, _I32, _P, _P, _P, _P]
    lib.lt_dsa_union.restype = ctypes.c_int
    lib.lt_event_create.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.lt_event_create.restype = ctypes.c_int
    lib.lt_event_destroy.argtypes = [_P]
    lib.lt_event_destroy.restype = ctypes.c_int
    lib.lt_event_record.argtypes = [_P, _P]
    lib.lt_event_record.restype = ctypes.c_int
    lib.lt_event_elapsed_ms.argtypes = [_P, _P, ctypes.POINTER(ctypes.c_float)]
    lib.lt_event_elapsed_ms.restype = ctypes.c_int
    lib.lt_strerror.argtypes = [ctypes.c_int]
    lib.lt_strerror.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int, what: str):
    if status != LT_OK:
        msg = load().lt_strerror(status).decode()
        raise LiteTopKError("%s failed: %s (%d)" % (what, msg, status))


# ---------------------------------------------------------------------------
# raw entry points (same names and argument order as the header)
# ---------------------------------------------------------------------------

def lt_options_default() -> LtOptions:
    o = LtOptions()
    load().lt_options_default(ctypes.byref(o))
    return o


def lt_indexer_topk_workspace_size(nq, nk, h, d, dtype, mode, k, opts: Optional[LtOptions] = None) -> int:
    return load().lt_indexer_topk_workspace_size(nq, nk, h, d, dtype, mode, k,
                                                 ctypes.byref(opts) if opts is not None else None)


def lt_indexer_topk(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, k, causal_offsets, out_idx,
                    out_scores, workspace, workspace_bytes, opts, stream) -> int:
    return load().lt_indexer_topk(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, k, causal_offsets,
                                  out_idx, out_scores, workspace, workspace_bytes,
                                  ctypes.byref(opts) if opts is not None else None, stream)


def lt_indexer_topk_static(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, k, causal_offsets, out_idx,
                           out_scores, opts, stream) -> int:
    return load().lt_indexer_topk_static(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, k,
                                         causal_offsets, out_idx, out_scores,
                                         ctypes.byref(opts) if opts is not None else None, stream)


def lt_indexer_scores(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, scores, ld, stream) -> int:
    return load().lt_indexer_scores(q, q_scale, w, keys, k_scale, dtype, mode, nq, nk, h, d, scores, ld, stream)


def lt_topk_select_workspace_size(nq, nk, k, opts: Optional[LtOptions] = None) -> int:
    return load().lt_topk_select_workspace_size(nq, nk, k, ctypes.byref(opts) if opts is not None else None)


def lt_topk_select(scores, row_stride, nq, nk, k, causal_offsets, out_idx, out_scores, workspace,
                   workspace_bytes, opts, stream) -> int:
    return load().lt_topk_select(scores, row_stride, nq, nk, k, causal_offsets, out_idx, out_scores, workspace,
                                 workspace_bytes, ctypes.byref(opts) if opts is not None else None, stream)


def lt_topk_radix(scores, row_stride, nq, nk, k, causal_offsets, out_idx, out_scores, flags, stream) -> int:
    return load().lt_topk_radix(scores, row_stride, nq, nk, k, causal_offsets, out_idx, out_scores, flags, stream)


def lt_sample_from_topk_workspace_size(nk) -> int:
    return load().lt_sample_from_topk_workspace_size(nk)


def lt_sample_from_topk(prev_idx, ld, prev_rows, prev_k, nk, sample_size, sample_keys, workspace, workspace_bytes,
                        stream) -> int:
    return load().lt_sample_from_topk(prev_idx, ld, prev_rows, prev_k, nk, sample_size, sample_keys, workspace,
                                      workspace_bytes, stream)


def lt_dsa_union(topk_idx, ld, nq, k, group, union_idx, union_count, member_mask, stream) -> int:
    return load().lt_dsa_union(topk_idx, ld, nq, k, group, union_idx, union_count, member_mask, stream)


def lt_strerror(status: int) -> str:
    return load().lt_strerror(status).decode()


# ---------------------------------------------------------------------------
# tensor helpers
# ---------------------------------------------------------------------------

def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return LT_F32
    if t.dtype == torch.bfloat16:
        return LT_BF16
    if t.dtype in (torch.uint8, torch.float8_e4m3fn):
        return LT_FP8_E4M3FN
    raise LiteTopKError("unsupported storage dtype %s" % t.dtype)


def _need(cond: bool, msg: str):
    if not cond:
        raise LiteTopKError(msg)


def _on_gpu(*ts):
    for t in ts:
        if t is not None:
            _need(t.is_cuda, "tensors must be on the GPU")
            _need(t.is_contiguous(), "tensors must be contiguous")


def make_options(num_bins=None, sample_size=None, capacity=None, key_splits=None,
                 sorted_output=False, force_fallback=False, seed=None, stage_events=None,
                 row_stats: Optional[torch.Tensor] = None,
                 sample_keys: Optional[torch.Tensor] = None,
                 visible_start: Optional[torch.Tensor] = None) -> LtOptions:
    """lt_options from keyword arguments. sample_keys: a GPU int32 list used
    as the sample (its length becomes sample_size); the tensor must stay
    alive until the call that uses these options has run."""
    o = lt_options_default()
    if num_bins is not None:
        o.num_bins = num_bins
    if sample_size is not None:
        o.sample_size = sample_size
    if capacity is not None:
        o.capacity = capacity
    if key_splits is not None:
        o.key_splits = key_splits
    o.flags = (LT_SORTED_OUTPUT if sorted_output else 0) | (LT_FORCE_FALLBACK if force_fallback else 0)
    if seed is not None:
        o.seed = seed
    if stage_events is not None:
        o.stage_events = ctypes.cast(stage_events.array, ctypes.c_void_p)
    if row_stats is not None:
        _on_gpu(row_stats)
        _need(row_stats.dtype == torch.int32 and row_stats.dim() == 2 and row_stats.shape[1] == LT_ROW_STATS,
              "row_stats must be an int32 [Nq, LT_ROW_STATS] GPU tensor")
        o.row_stats = row_stats.data_ptr()
        o.row_stats_rows = row_stats.shape[0]
    if sample_keys is not None:
        _on_gpu(sample_keys)
        _need(sample_keys.dtype == torch.int32 and sample_keys.dim() == 1, "sample_keys must be int32 [n]")
        o.sample_keys = sample_keys.data_ptr()
        o.sample_size = sample_keys.numel()
    if visible_start is not None:
        _on_gpu(visible_start)
        _need(visible_start.dtype == torch.int32 and visible_start.dim() == 1, "visible_start must be int32 [Nq]")
        o.visible_start = visible_start.data_ptr()
    return o


class StageEvents:
    """LT_NUM_STAGE_EVENTS HIP events for lt_options.stage_events."""

    def __init__(self):
        lib = load()
        self.array = (ctypes.c_void_p * LT_NUM_STAGE_EVENTS)()
        for i in range(LT_NUM_STAGE_EVENTS):
            h = ctypes.c_void_p()
            _check(lib.lt_event_create(ctypes.byref(h)), "lt_event_create")
            self.array[i] = h.value

    def stage_ms(self):
        """Device milliseconds of each stage of the last call (synchronises)."""
        lib = load()
        out = {}
        for i, name in enumerate(STAGES):
            ms = ctypes.c_float()
            _check(lib.lt_event_elapsed_ms(self.array[i], self.array[i + 1], ctypes.byref(ms)), "elapsed")
            out[name] = ms.value
        return out

    def close(self):
        lib = load()
        for i in range(LT_NUM_STAGE_EVENTS):
            if self.array[i]:
                lib.lt_event_destroy(self.array[i])
                self.array[i] = None


def _check_rows(nq: int, causal_offsets: Optional[torch.Tensor], options: Optional[LtOptions]):
    """Per-row arguments: causal_offsets int32 [Nq] on the GPU; the options'
    row_stats (checked in make_options for its shape) must cover Nq rows."""
    if causal_offsets is not None:
        _on_gpu(causal_offsets)
        _need(causal_offsets.dtype == torch.int32 and causal_offsets.numel() == nq,
              "causal_offsets must be int32 [Nq]")
    if options is not None and options.row_stats:
        n = getattr(options, "row_stats_rows", None)
        _need(n is not None and n >= nq, "row_stats must hold LT_ROW_STATS fields for each of the Nq rows "
              "(pass it through make_options)")


def _check_score_inputs(q, w, keys, causal_offsets, q_scale, k_scale, options):
    nq, h, _ = q.shape
    nk = keys.shape[0]
    if w is not None:
        _need(w.dtype == torch.float32 and tuple(w.shape) == (nq, h), "w must be float32 [Nq, H]")
    if _dtype_code(q) == LT_FP8_E4M3FN:
        _need(q_scale is not None and q_scale.dtype == torch.float32 and tuple(q_scale.shape) == (nq, h),
              "fp8: q_scale must be float32 [Nq, H]")
        _need(k_scale is not None and k_scale.dtype == torch.float32 and tuple(k_scale.shape) == (nk,),
              "fp8: k_scale must be float32 [Nk]")
    _check_rows(nq, causal_offsets, options)


def _mode_code(mode: str) -> int:
    if mode == "dsa":
        return LT_SCORE_DSA
    if mode == "ip":
        return LT_SCORE_IP
    raise LiteTopKError("mode must be 'dsa' or 'ip'")


def indexer_topk_workspace(nq, nk, h, d, dtype: int, mode: str, k: int, options: Optional[LtOptions] = None,
                           device=None) -> torch.Tensor:
    n = lt_indexer_topk_workspace_size(nq, nk, h, d, dtype, _mode_code(mode), k, options)
    _need(n > 0, "unsupported shape for lt_indexer_topk")
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def indexer_topk(q: torch.Tensor, w: Optional[torch.Tensor], keys: torch.Tensor, k: int,
                 causal_offsets: Optional[torch.Tensor] = None, q_scale: Optional[torch.Tensor] = None,
                 k_scale: Optional[torch.Tensor] = None, mode: str = "dsa",
                 options: Optional[LtOptions] = None, out=None, workspace: Optional[torch.Tensor] = None,
                 stream=None):
    """Exact per-row top-k of the index score. q [Nq, H, d], keys [Nk, d] in
    float32 / bfloat16 / uint8 (E4M3FN bytes, with q_scale [Nq, H] and k_scale
    [Nk]); w [Nq, H] float32 or None. Returns (idx int32 [Nq, k], scores
    float32 [Nq, k])."""
    _on_gpu(q, w, keys, causal_offsets, q_scale, k_scale)
    _need(q.dim() == 3 and keys.dim() == 2 and q.shape[2] == keys.shape[1], "q [Nq,H,d] and keys [Nk,d] required")
    dt = _dtype_code(q)
    _need(_dtype_code(keys) == dt, "q and keys must share a dtype")
    nq, h, d = q.shape
    nk = keys.shape[0]
    _check_score_inputs(q, w, keys, causal_offsets, q_scale, k_scale, options)
    if out is None:
        out = (torch.empty((nq, k), dtype=torch.int32, device=q.device),
               torch.empty((nq, k), dtype=torch.float32, device=q.device))
    if workspace is None:
        workspace = indexer_topk_workspace(nq, nk, h, d, dt, mode, k, options, q.device)
    st = lt_indexer_topk(_ptr(q), _ptr(q_scale), _ptr(w), _ptr(keys), _ptr(k_scale), dt, _mode_code(mode), nq, nk,
                         h, d, k, _ptr(causal_offsets), _ptr(out[0]), _ptr(out[1]), _ptr(workspace),
                         workspace.numel(), options, _stream(stream))
    _check(st, "lt_indexer_topk")
    return out


def indexer_topk_static(q: torch.Tensor, w: Optional[torch.Tensor], keys: torch.Tensor, k: int,
                        causal_offsets: Optional[torch.Tensor] = None, q_scale: Optional[torch.Tensor] = None,
                        k_scale: Optional[torch.Tensor] = None, mode: str = "dsa",
                        options: Optional[LtOptions] = None, out=None, stream=None):
    """indexer_topk with the library's static per-GPU workspace
    (lt_indexer_topk_static): the call allocates no device memory when `out`
    is given. Calls whose work overlaps on one GPU race."""
    _on_gpu(q, w, keys, causal_offsets, q_scale, k_scale)
    _need(q.dim() == 3 and keys.dim() == 2 and q.shape[2] == keys.shape[1], "q [Nq,H,d] and keys [Nk,d] required")
    dt = _dtype_code(q)
    _need(_dtype_code(keys) == dt, "q and keys must share a dtype")
    nq, h, d = q.shape
    nk = keys.shape[0]
    _check_score_inputs(q, w, keys, causal_offsets, q_scale, k_scale, options)
    if out is None:
        out = (torch.empty((nq, k), dtype=torch.int32, device=q.device),
               torch.empty((nq, k), dtype=torch.float32, device=q.device))
    _on_gpu(*out)
    _need(tuple(out[0].shape) == (nq, k) and out[0].dtype == torch.int32 and tuple(out[1].shape) == (nq, k)
          and out[1].dtype == torch.float32, "out must be (int32 [Nq, k], float32 [Nq, k])")
    st = lt_indexer_topk_static(_ptr(q), _ptr(q_scale), _ptr(w), _ptr(keys), _ptr(k_scale), dt, _mode_code(mode), nq,
                                nk, h, d, k, _ptr(causal_offsets), _ptr(out[0]), _ptr(out[1]), options,
                                _stream(stream))
    _check(st, "lt_indexer_topk_static")
    return out


def indexer_scores(q: torch.Tensor, w: Optional[torch.Tensor], keys: torch.Tensor,
                   q_scale: Optional[torch.Tensor] = None, k_scale: Optional[torch.Tensor] = None,
                   mode: str = "dsa", out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Dense float32 index scores [Nq, Nk] (the materialising baseline)."""
    _on_gpu(q, w, keys, q_scale, k_scale)
    _need(q.dim() == 3 and keys.dim() == 2 and q.shape[2] == keys.shape[1], "q [Nq,H,d] and keys [Nk,d] required")
    dt = _dtype_code(q)
    _need(_dtype_code(keys) == dt, "q and keys must share a dtype")
    _check_score_inputs(q, w, keys, None, q_scale, k_scale, None)
    nq, h, d = q.shape
    nk = keys.shape[0]
    if out is None:
        out = torch.empty((nq, nk), dtype=torch.float32, device=q.device)
    _need(out.dim() == 2 and out.shape[0] == nq and out.shape[1] >= nk and out.stride(1) == 1, "bad out")
    st = lt_indexer_scores(_ptr(q), _ptr(q_scale), _ptr(w), _ptr(keys), _ptr(k_scale), dt, _mode_code(mode), nq, nk,
                           h, d, _ptr(out), out.stride(0), _stream(stream))
    _check(st, "lt_indexer_scores")
    return out


def topk_select(scores: torch.Tensor, k: int, num_keys: Optional[int] = None,
                causal_offsets: Optional[torch.Tensor] = None, options: Optional[LtOptions] = None, out=None,
                workspace: Optional[torch.Tensor] = None, stream=None):
    """Exact per-row top-k of a float32 score matrix [Nq, ld] (first num_keys
    columns are keys) through the sample / filter / select pipeline."""
    _need(scores.is_cuda and scores.dtype == torch.float32 and scores.dim() == 2 and scores.stride(1) == 1,
          "scores must be a float32 [Nq, ld] GPU matrix with unit column stride")
    nq = scores.shape[0]
    nk = scores.shape[1] if num_keys is None else num_keys
    _check_rows(nq, causal_offsets, options)
    if out is None:
        out = (torch.empty((nq, k), dtype=torch.int32, device=scores.device),
               torch.empty((nq, k), dtype=torch.float32, device=scores.device))
    if workspace is None:
        n = lt_topk_select_workspace_size(nq, nk, k, options)
        _need(n > 0, "unsupported shape for lt_topk_select")
        workspace = torch.empty(n, dtype=torch.uint8, device=scores.device)
    st = lt_topk_select(_ptr(scores), scores.stride(0), nq, nk, k, _ptr(causal_offsets), _ptr(out[0]),
                        _ptr(out[1]), _ptr(workspace), workspace.numel(), options, _stream(stream))
    _check(st, "lt_topk_select")
    return out


def topk_radix(scores: torch.Tensor, k: int, num_keys: Optional[int] = None,
               causal_offsets: Optional[torch.Tensor] = None, sorted_output: bool = False, out=None, stream=None):
    """Exact per-row top-k by plain radix selection (no filter)."""
    _need(scores.is_cuda and scores.dtype == torch.float32 and scores.dim() == 2 and scores.stride(1) == 1,
          "scores must be a float32 [Nq, ld] GPU matrix with unit column stride")
    nq = scores.shape[0]
    nk = scores.shape[1] if num_keys is None else num_keys
    _check_rows(nq, causal_offsets, None)
    if out is None:
        out = (torch.empty((nq, k), dtype=torch.int32, device=scores.device),
               torch.empty((nq, k), dtype=torch.float32, device=scores.device))
    st = lt_topk_radix(_ptr(scores), scores.stride(0), nq, nk, k, _ptr(causal_offsets), _ptr(out[0]), _ptr(out[1]),
                       LT_SORTED_OUTPUT if sorted_output else 0, _stream(stream))
    _check(st, "lt_topk_radix")
    return out


def sample_from_topk(prev_idx: torch.Tensor, num_keys: int, sample_size: int, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The previous chunk's sample (sec. 3.2 "Sampling"): the sample_size keys
    that occur most often in prev_idx [rows, k] (int32, -1 padding ignored),
    ascending, then -1. Returns int32 [sample_size]."""
    _need(prev_idx.is_cuda and prev_idx.dtype == torch.int32 and prev_idx.dim() == 2
          and (prev_idx.numel() == 0 or prev_idx.stride(1) == 1),
          "prev_idx must be an int32 [rows, k] GPU matrix with unit column stride")
    rows, pk = prev_idx.shape
    if out is None:
        out = torch.empty(sample_size, dtype=torch.int32, device=prev_idx.device)
    _need(out.dtype == torch.int32 and out.numel() == sample_size and out.is_contiguous(), "bad out")
    if workspace is None:
        workspace = torch.empty(lt_sample_from_topk_workspace_size(num_keys), dtype=torch.uint8,
                                device=prev_idx.device)
    st = lt_sample_from_topk(_ptr(prev_idx), prev_idx.stride(0) if prev_idx.numel() else pk, rows, pk, num_keys,
                             sample_size, _ptr(out), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "lt_sample_from_topk")
    return out


def dsa_union(topk_idx: torch.Tensor, group: int, stream=None):
    """LiteDSA union (sec. 3.3) of each group of `group` consecutive rows of
    topk_idx [Nq, k] (int32, -1 padding). Returns (union_idx int32
    [G, group * k], union_count int32 [G], member_mask int32 [Nq, W]; the
    mask words are uint32 bit patterns, W = ceil(group * k / 32))."""
    _need(topk_idx.is_cuda and topk_idx.dtype == torch.int32 and topk_idx.dim() == 2
          and (topk_idx.numel() == 0 or topk_idx.stride(1) == 1),
          "topk_idx must be an int32 [Nq, k] GPU matrix with unit column stride")
    nq, k = topk_idx.shape
    _need(group >= 1 and k >= 1 and group * k <= LT_UNION_MAX, "need 1 <= group, group * k <= LT_UNION_MAX")
    ngroups = (nq + group - 1) // group
    words = (group * k + 31) // 32
    dev = topk_idx.device
    uidx = torch.empty((ngroups, group * k), dtype=torch.int32, device=dev)
    ucnt = torch.empty((ngroups,), dtype=torch.int32, device=dev)
    mask = torch.empty((nq, words), dtype=torch.int32, device=dev)
    st = lt_dsa_union(_ptr(topk_idx), topk_idx.stride(0) if topk_idx.numel() else k, nq, k, group, _ptr(uidx),
                      _ptr(ucnt), _ptr(mask), _stream(stream))
    _check(st, "lt_dsa_union")
    return uidx, ucnt, mask
