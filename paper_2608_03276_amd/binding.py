"""ctypes binding of libtaskpress (include/taskpress.h): argument marshalling only.

Every step of the eviction path runs in the library's HIP kernels; PyTorch only
provides device memory and the current HIP stream.  Importing this module on a
machine without the built library raises ImportError (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libtaskpress.so")

TP_OK, TP_ERR_NULL, TP_ERR_SHAPE, TP_ERR_PARAM, TP_ERR_UNSUPPORTED, TP_ERR_WORKSPACE, TP_ERR_HIP = range(7)
TP_QFMT_INT, TP_QFMT_FP8_E4M3 = 0, 1
TP_COMBINE_MUL, TP_COMBINE_NORM_ADD, TP_COMBINE_HARMONIC, TP_COMBINE_KEY_ONLY = 0, 1, 2, 3
TP_FN_GUIDE_SCORES, TP_FN_COMBINE_SELECT_TOPK, TP_FN_EVICT, TP_FN_GUIDE_ATTENTION = 0, 1, 2, 3
TP_MAX_BATCH = 64
TP_EVICT_EVENTS = 8

EXPORTED = ("tp_version", "tp_status_string", "tp_last_error", "tp_keep_count", "tp_workspace_size",
            "tp_guide_scores", "tp_guide_scores_lse", "tp_guide_attention", "tp_guide_attention_quantize",
            "tp_quantize_v_scales",
            "tp_combine_select_topk",
            "tp_combine_select_topk_static", "tp_compact_kv", "tp_compact_quantize_kv", "tp_evict")
TP_STATIC_SCRATCH_BYTES = 64 << 20


class TaskPressError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_STATUS_NAMES = {0: "TP_OK", 1: "TP_ERR_NULL", 2: "TP_ERR_SHAPE", 3: "TP_ERR_PARAM", 4: "TP_ERR_UNSUPPORTED",
                 5: "TP_ERR_WORKSPACE", 6: "TP_ERR_HIP"}


class TpDims(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32)]


class TpBatch(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("ctx_offsets", ctypes.POINTER(ctypes.c_int64)),
                ("guide_offsets", ctypes.POINTER(ctypes.c_int64))]


class TpProfile(ctypes.Structure):
    _fields_ = [("num_events", ctypes.c_int32), ("events", ctypes.c_void_p * TP_EVICT_EVENTS)]


def _i64_array(vals):
    vals = [int(v) for v in vals]
    return (ctypes.c_int64 * len(vals))(*vals)


class Batch:
    """A tp_batch plus the host offset arrays it points to (kept alive here)."""

    def __init__(self, ctx_offsets, guide_offsets=None):
        self.ctx_offsets = [int(x) for x in ctx_offsets]
        self.guide_offsets = None if guide_offsets is None else [int(x) for x in guide_offsets]
        self._ctx = _i64_array(self.ctx_offsets)
        self._g = None if guide_offsets is None else _i64_array(self.guide_offsets)
        self.c = TpBatch(len(self.ctx_offsets) - 1, self._ctx,
                         self._g if self._g is not None else ctypes.POINTER(ctypes.c_int64)())

    @property
    def batch(self):
        return len(self.ctx_offsets) - 1

    @property
    def n_tot(self):
        return self.ctx_offsets[-1]

    @property
    def g_tot(self):
        return self.guide_offsets[-1]


def dims(L, Hq, Hkv, d) -> TpDims:
    return TpDims(L, Hq, Hkv, d)


_lib = None


def load():
    """Load libtaskpress.so (raises ImportError when it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    pd, pb = ctypes.POINTER(TpDims), ctypes.POINTER(TpBatch)
    pi64 = ctypes.POINTER(ctypes.c_int64)
    lib.tp_version.restype = ctypes.c_char_p
    lib.tp_version.argtypes = []
    lib.tp_status_string.restype = ctypes.c_char_p
    lib.tp_status_string.argtypes = [ctypes.c_int32]
    lib.tp_last_error.restype = ctypes.c_char_p
    lib.tp_last_error.argtypes = []
    lib.tp_keep_count.restype = ctypes.c_int64
    lib.tp_keep_count.argtypes = [ctypes.c_int64, ctypes.c_double, ctypes.c_int64]
    lib.tp_workspace_size.restype = ctypes.c_int32
    lib.tp_workspace_size.argtypes = [ctypes.c_int32, pd, pb, ctypes.POINTER(ctypes.c_size_t)]
    lib.tp_guide_scores.restype = ctypes.c_int32
    lib.tp_guide_scores.argtypes = [pd, pb, P, P, P, ctypes.c_float, ctypes.c_int32, P, P, ctypes.c_size_t, P]
    lib.tp_guide_scores_lse.restype = ctypes.c_int32
    lib.tp_guide_scores_lse.argtypes = [pd, pb, P, P, P, ctypes.c_float, ctypes.c_int32, P, P, ctypes.c_size_t, P]
    lib.tp_guide_attention.restype = ctypes.c_int32
    lib.tp_guide_attention.argtypes = [pd, pb, P, P, P, P, P, ctypes.c_float, P, P, P, ctypes.c_size_t, P]
    lib.tp_guide_attention_quantize.restype = ctypes.c_int32
    lib.tp_guide_attention_quantize.argtypes = [pd, pb, P, P, P, P, P, ctypes.c_float, ctypes.c_int32,
                                                ctypes.c_int32, P, P, P, P, P, ctypes.c_size_t, P]
    lib.tp_quantize_v_scales.restype = ctypes.c_int32
    lib.tp_quantize_v_scales.argtypes = [pd, pb, P, ctypes.c_int32, ctypes.c_int32, P, P, P]
    lib.tp_combine_select_topk.restype = ctypes.c_int32
    lib.tp_combine_select_topk.argtypes = [pd, pb, P, P, ctypes.c_int32, ctypes.c_double, ctypes.c_int64, pi64,
                                           P, P, P, ctypes.c_size_t, P]
    lib.tp_combine_select_topk_static.restype = ctypes.c_int32
    lib.tp_combine_select_topk_static.argtypes = [pd, pb, P, P, ctypes.c_int32, ctypes.c_double, ctypes.c_int64,
                                                  pi64, P, P]
    lib.tp_compact_kv.restype = ctypes.c_int32
    lib.tp_compact_kv.argtypes = [pd, pb, pi64, P, P, P, P, ctypes.c_int32, ctypes.c_int32, P, P, P, P]
    lib.tp_compact_quantize_kv.restype = ctypes.c_int32
    lib.tp_compact_quantize_kv.argtypes = [pd, pb, pi64, P, P, P, ctypes.c_int32, ctypes.c_int32, P, P, P, P]
    lib.tp_evict.restype = ctypes.c_int32
    lib.tp_evict.argtypes = [pd, pb, P, P, P, P, P, ctypes.c_float, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                             ctypes.c_int32, ctypes.c_double, ctypes.c_int64, pi64, P, P, P, P, P, P, P, P, P,
                             ctypes.c_size_t, ctypes.POINTER(TpProfile), P]
    _lib = lib
    return lib


def _check(status: int):
    if status != TP_OK:
        raise TaskPressError(status, load().tp_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _need(t, numel, name, device=True):
    if t is None:
        return
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device and not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.numel() * t.element_size() < numel:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, needs {numel}")


def _nbytes(t):
    return t.numel() * t.element_size() if t is not None else 0


# ----------------------------------------------------------------------------- entry points
def tp_version() -> str:
    return load().tp_version().decode()


def tp_keep_count(n: int, keep_ratio: float = 0.0, keep_budget: int = 0) -> int:
    return int(load().tp_keep_count(int(n), float(keep_ratio), int(keep_budget)))


def tp_workspace_size(fn: int, d: TpDims, batch: Batch) -> int:
    out = ctypes.c_size_t(0)
    _check(load().tp_workspace_size(fn, ctypes.byref(d), ctypes.byref(batch.c), ctypes.byref(out)))
    return int(out.value)


def tp_guide_scores(d: TpDims, batch: Batch, q_guide, k, softmax_scale: float, pool_k: int, s_key, workspace,
                    stream=None, k_guide=None):
    """k_guide: the guide tokens' keys bf16 [L][Hkv][G_tot][d] (paper-literal normaliser) or None."""
    L, Hq, Hkv, D = d.num_layers, d.num_q_heads, d.num_kv_heads, d.head_dim
    _need(q_guide, L * Hq * batch.g_tot * D * 2, "q_guide")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(k_guide, L * Hkv * batch.g_tot * D * 2, "k_guide")
    _need(s_key, L * Hkv * batch.n_tot * 4, "s_key")
    _check(load().tp_guide_scores(ctypes.byref(d), ctypes.byref(batch.c), _ptr(q_guide), _ptr(k), _ptr(k_guide),
                                  float(softmax_scale), int(pool_k), _ptr(s_key), _ptr(workspace),
                                  workspace.numel() * workspace.element_size() if workspace is not None else 0,
                                  _stream(stream)))


def tp_guide_scores_lse(d: TpDims, batch: Batch, q_guide, k, guide_lse, softmax_scale: float, pool_k: int, s_key,
                        workspace, stream=None):
    """Step 1 with the guide rows' log-normalisers supplied: guide_lse fp32 [L][Hq][G_tot]
    (natural log of each row's softmax normaliser over the scaled logits)."""
    L, Hq, Hkv, D = d.num_layers, d.num_q_heads, d.num_kv_heads, d.head_dim
    _need(q_guide, L * Hq * batch.g_tot * D * 2, "q_guide")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(guide_lse, L * Hq * batch.g_tot * 4, "guide_lse")
    _need(s_key, L * Hkv * batch.n_tot * 4, "s_key")
    _check(load().tp_guide_scores_lse(ctypes.byref(d), ctypes.byref(batch.c), _ptr(q_guide), _ptr(k),
                                      _ptr(guide_lse), float(softmax_scale), int(pool_k), _ptr(s_key),
                                      _ptr(workspace), _nbytes(workspace), _stream(stream)))


def tp_guide_attention(d: TpDims, batch: Batch, q_guide, k, v, softmax_scale: float, o_guide, guide_lse,
                       workspace=None, stream=None, k_guide=None, v_guide=None):
    """The prefill's attention for the appended guide rows: o_guide fp32 [L][Hq][G_tot][d] and
    guide_lse fp32 [L][Hq][G_tot] (natural log), over the context and, with k_guide / v_guide
    bf16 [L][Hkv][G_tot][d], the guide keys 0..j of each row j."""
    L, Hq, Hkv, D = d.num_layers, d.num_q_heads, d.num_kv_heads, d.head_dim
    _need(q_guide, L * Hq * batch.g_tot * D * 2, "q_guide")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(v, L * Hkv * batch.n_tot * D * 2, "v")
    _need(k_guide, L * Hkv * batch.g_tot * D * 2, "k_guide")
    _need(v_guide, L * Hkv * batch.g_tot * D * 2, "v_guide")
    _need(o_guide, L * Hq * batch.g_tot * D * 4, "o_guide")
    _need(guide_lse, L * Hq * batch.g_tot * 4, "guide_lse")
    if workspace is None:
        workspace = torch.empty(tp_workspace_size(TP_FN_GUIDE_ATTENTION, d, batch), dtype=torch.uint8,
                                device=q_guide.device)
    _check(load().tp_guide_attention(ctypes.byref(d), ctypes.byref(batch.c), _ptr(q_guide), _ptr(k), _ptr(v),
                                     _ptr(k_guide), _ptr(v_guide), float(softmax_scale), _ptr(o_guide),
                                     _ptr(guide_lse), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def tp_guide_attention_quantize(d: TpDims, batch: Batch, q_guide, k, v, softmax_scale: float, qfmt: int,
                                bits: int, o_guide, guide_lse, scales, v_q, workspace=None, stream=None,
                                k_guide=None, v_guide=None):
    """tp_guide_attention plus step 2 from the same sweep over V: scales fp32 [L][Hkv][N_tot]
    and the codes v_q [L][Hkv][N_tot][row_bytes], as tp_quantize_v_scales writes them."""
    L, Hq, Hkv, D = d.num_layers, d.num_q_heads, d.num_kv_heads, d.head_dim
    _need(q_guide, L * Hq * batch.g_tot * D * 2, "q_guide")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(v, L * Hkv * batch.n_tot * D * 2, "v")
    _need(k_guide, L * Hkv * batch.g_tot * D * 2, "k_guide")
    _need(v_guide, L * Hkv * batch.g_tot * D * 2, "v_guide")
    _need(o_guide, L * Hq * batch.g_tot * D * 4, "o_guide")
    _need(guide_lse, L * Hq * batch.g_tot * 4, "guide_lse")
    _need(scales, L * Hkv * batch.n_tot * 4, "scales")
    _need(v_q, L * Hkv * batch.n_tot * row_bytes(qfmt, bits, D), "v_q")
    if workspace is None:
        workspace = torch.empty(tp_workspace_size(TP_FN_GUIDE_ATTENTION, d, batch), dtype=torch.uint8,
                                device=q_guide.device)
    _check(load().tp_guide_attention_quantize(ctypes.byref(d), ctypes.byref(batch.c), _ptr(q_guide), _ptr(k),
                                              _ptr(v), _ptr(k_guide), _ptr(v_guide), float(softmax_scale),
                                              int(qfmt), int(bits), _ptr(o_guide), _ptr(guide_lse), _ptr(scales),
                                              _ptr(v_q), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def row_bytes(qfmt: int, bits: int, head_dim: int) -> int:
    return head_dim // 2 if (qfmt == TP_QFMT_INT and bits <= 4) else head_dim


def tp_quantize_v_scales(d: TpDims, batch: Batch, v, qfmt: int, bits: int, scales, v_q=None, stream=None):
    L, Hkv, D = d.num_layers, d.num_kv_heads, d.head_dim
    _need(v, L * Hkv * batch.n_tot * D * 2, "v")
    _need(scales, L * Hkv * batch.n_tot * 4, "scales")
    _need(v_q, L * Hkv * batch.n_tot * row_bytes(qfmt, bits, D), "v_q")
    _check(load().tp_quantize_v_scales(ctypes.byref(d), ctypes.byref(batch.c), _ptr(v), int(qfmt), int(bits),
                                       _ptr(scales), _ptr(v_q), _stream(stream)))


def kept_offsets_for(batch: Batch, keep_ratio: float = 0.0, keep_budget: int = 0):
    out = [0]
    for b in range(batch.batch):
        n = batch.ctx_offsets[b + 1] - batch.ctx_offsets[b]
        out.append(out[-1] + tp_keep_count(n, keep_ratio, keep_budget))
    return out


def tp_combine_select_topk(d: TpDims, batch: Batch, s_key, scales, rule: int, keep_ratio: float, keep_budget: int,
                           kept_offsets, kept_idx, s_out=None, workspace=None, stream=None):
    L, Hkv = d.num_layers, d.num_kv_heads
    _need(s_key, L * Hkv * batch.n_tot * 4, "s_key")
    _need(scales, L * Hkv * batch.n_tot * 4, "scales")
    _need(kept_idx, L * Hkv * int(kept_offsets[-1]) * 4, "kept_idx")
    _need(s_out, L * Hkv * batch.n_tot * 4, "s_out")
    ko = _i64_array(kept_offsets)
    if workspace is None:  # the caller passed none: one of the size the library asks for
        workspace = torch.empty(tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, d, batch), dtype=torch.uint8,
                                device=s_key.device)
    ws_bytes = workspace.numel() * workspace.element_size()
    _check(load().tp_combine_select_topk(ctypes.byref(d), ctypes.byref(batch.c), _ptr(s_key), _ptr(scales),
                                         int(rule), float(keep_ratio), int(keep_budget), ko, _ptr(kept_idx),
                                         _ptr(s_out), _ptr(workspace), ws_bytes, _stream(stream)))


def tp_combine_select_topk_static(d: TpDims, batch: Batch, s_key, scales, rule: int, keep_ratio: float,
                                  keep_budget: int, kept_offsets, kept_idx, stream=None):
    """Step 3 without a workspace: the combined scores are staged in the library's static
    device buffer (TP_STATIC_SCRATCH_BYTES per GPU); calls that overlap on one GPU race."""
    L, Hkv = d.num_layers, d.num_kv_heads
    _need(s_key, L * Hkv * batch.n_tot * 4, "s_key")
    _need(scales, L * Hkv * batch.n_tot * 4, "scales")
    _need(kept_idx, L * Hkv * int(kept_offsets[-1]) * 4, "kept_idx")
    ko = _i64_array(kept_offsets)
    _check(load().tp_combine_select_topk_static(ctypes.byref(d), ctypes.byref(batch.c), _ptr(s_key), _ptr(scales),
                                                int(rule), float(keep_ratio), int(keep_budget), ko, _ptr(kept_idx),
                                                _stream(stream)))


def tp_compact_kv(d: TpDims, batch: Batch, kept_offsets, kept_idx, k, v_q, scales, qfmt: int, bits: int, k_out,
                  v_q_out, scales_out, stream=None):
    L, Hkv, D = d.num_layers, d.num_kv_heads, d.head_dim
    kt = int(kept_offsets[-1])
    _need(kept_idx, L * Hkv * kt * 4, "kept_idx")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(k_out, L * Hkv * kt * D * 2, "k_out")
    _need(v_q, L * Hkv * batch.n_tot * row_bytes(qfmt, bits, D), "v_q")
    _need(v_q_out, L * Hkv * kt * row_bytes(qfmt, bits, D), "v_q_out")
    _need(scales, L * Hkv * batch.n_tot * 4, "scales")
    _need(scales_out, L * Hkv * kt * 4, "scales_out")
    ko = _i64_array(kept_offsets)
    _check(load().tp_compact_kv(ctypes.byref(d), ctypes.byref(batch.c), ko, _ptr(kept_idx), _ptr(k), _ptr(v_q),
                                _ptr(scales), int(qfmt), int(bits), _ptr(k_out), _ptr(v_q_out), _ptr(scales_out),
                                _stream(stream)))


# ----------------------------------------------------------------------------- whole path
class EvictBuffers:
    """Device buffers of one eviction: outputs and workspaces, allocated once and reused."""

    def __init__(self, d: TpDims, batch: Batch, qfmt: int, bits: int, kept_offsets, device="cuda"):
        L, Hkv, D = d.num_layers, d.num_kv_heads, d.head_dim
        n, kt = batch.n_tot, int(kept_offsets[-1])
        rb = row_bytes(qfmt, bits, D)
        self.kept_offsets = list(kept_offsets)
        self.s_key = torch.empty(L * Hkv * n, dtype=torch.float32, device=device)
        self.scales = torch.empty(L * Hkv * n, dtype=torch.float32, device=device)
        self.v_q = torch.empty(L * Hkv * n * rb, dtype=torch.uint8, device=device)
        self.s_comb = torch.empty(L * Hkv * n, dtype=torch.float32, device=device)
        self.kept_idx = torch.empty(L * Hkv * max(kt, 1), dtype=torch.int32, device=device)
        self.k_c = torch.empty(L * Hkv * max(kt, 1) * D, dtype=torch.bfloat16, device=device)
        self.v_q_c = torch.empty(L * Hkv * max(kt, 1) * rb, dtype=torch.uint8, device=device)
        self.scales_c = torch.empty(L * Hkv * max(kt, 1), dtype=torch.float32, device=device)
        # one workspace serves both paths: tp_evict's holds the score passes' workspace first
        # (at least TP_FN_GUIDE_SCORES bytes), so evict() hands the same buffer to tp_guide_scores
        self.ws_evict = torch.empty(tp_workspace_size(TP_FN_EVICT, d, batch), dtype=torch.uint8, device=device)


def evict(d: TpDims, batch: Batch, q_guide, k, v, *, softmax_scale: float, pool_k: int, qfmt: int, bits: int,
          rule: int = TP_COMBINE_MUL, keep_ratio: float = 0.0, keep_budget: int = 0, bufs: EvictBuffers = None,
          stream=None, k_guide=None) -> EvictBuffers:
    """Run the four steps on one stream; returns the buffers (kept_idx, k_c, v_q_c, scales_c, ...)."""
    ko = kept_offsets_for(batch, keep_ratio, keep_budget)
    if bufs is None:
        bufs = EvictBuffers(d, batch, qfmt, bits, ko, device=k.device)
    tp_guide_scores(d, batch, q_guide, k, softmax_scale, pool_k, bufs.s_key, bufs.ws_evict, stream, k_guide)
    tp_quantize_v_scales(d, batch, v, qfmt, bits, bufs.scales, bufs.v_q, stream)
    tp_combine_select_topk(d, batch, bufs.s_key, bufs.scales, rule, keep_ratio, keep_budget, ko, bufs.kept_idx,
                           bufs.s_comb, None, stream)
    tp_compact_kv(d, batch, ko, bufs.kept_idx, k, bufs.v_q, bufs.scales, qfmt, bits, bufs.k_c, bufs.v_q_c,
                  bufs.scales_c, stream)
    return bufs


def tp_compact_quantize_kv(d: TpDims, batch: Batch, kept_offsets, kept_idx, k, v, qfmt: int, bits: int, k_out,
                           v_q_out, scales_out, stream=None):
    L, Hkv, D = d.num_layers, d.num_kv_heads, d.head_dim
    kt = int(kept_offsets[-1])
    _need(kept_idx, L * Hkv * kt * 4, "kept_idx")
    _need(k, L * Hkv * batch.n_tot * D * 2, "k")
    _need(v, L * Hkv * batch.n_tot * D * 2, "v")
    _need(k_out, L * Hkv * kt * D * 2, "k_out")
    _need(v_q_out, L * Hkv * kt * row_bytes(qfmt, bits, D), "v_q_out")
    _need(scales_out, L * Hkv * kt * 4, "scales_out")
    ko = _i64_array(kept_offsets)
    _check(load().tp_compact_quantize_kv(ctypes.byref(d), ctypes.byref(batch.c), ko, _ptr(kept_idx), _ptr(k), _ptr(v),
                                         int(qfmt), int(bits), _ptr(k_out), _ptr(v_q_out), _ptr(scales_out),
                                         _stream(stream)))


def tp_evict(d: TpDims, batch: Batch, q_guide, k, v, softmax_scale: float, pool_k: int, qfmt: int, bits: int,
             rule: int, keep_ratio: float, keep_budget: int, kept_offsets, s_key, scales, v_q, s_out, kept_idx,
             k_out, v_q_out, scales_out, workspace, events=None, stream=None, k_guide=None, guide_lse=None):
    """The whole path in one call.  `events`: None, or TP_EVICT_EVENTS torch.cuda.Event objects
    (enable_timing=True) that the library records between its kernels."""
    L, Hq, Hkv, D = d.num_layers, d.num_q_heads, d.num_kv_heads, d.head_dim
    n = batch.n_tot
    _need(q_guide, L * Hq * batch.g_tot * D * 2, "q_guide")
    _need(k, L * Hkv * n * D * 2, "k")
    _need(v, L * Hkv * n * D * 2, "v")
    _need(k_guide, L * Hkv * batch.g_tot * D * 2, "k_guide")
    _need(guide_lse, L * Hq * batch.g_tot * 4, "guide_lse")
    for t, nbytes, name in ((s_key, L * Hkv * n * 4, "s_key"), (scales, L * Hkv * n * 4, "scales"),
                            (v_q, L * Hkv * n * row_bytes(qfmt, bits, D), "v_q")):
        _need(t, nbytes, name)
    ko = _i64_array(kept_offsets)
    prof = None
    if events is not None:
        if len(events) != TP_EVICT_EVENTS:
            raise ValueError(f"need {TP_EVICT_EVENTS} events")
        s = torch.cuda.current_stream() if stream is None else stream
        handles = []
        for e in events:
            if not e.cuda_event:
                e.record(s)  # creates the underlying event
            handles.append(e.cuda_event)
        prof = TpProfile(TP_EVICT_EVENTS, (ctypes.c_void_p * TP_EVICT_EVENTS)(*handles))
    ws = workspace
    _check(load().tp_evict(ctypes.byref(d), ctypes.byref(batch.c), _ptr(q_guide), _ptr(k), _ptr(k_guide),
                           _ptr(guide_lse), _ptr(v),
                           float(softmax_scale), int(pool_k), int(qfmt), int(bits), int(rule), float(keep_ratio),
                           int(keep_budget), ko, _ptr(s_key), _ptr(scales), _ptr(v_q), _ptr(s_out),
                           _ptr(kept_idx), _ptr(k_out), _ptr(v_q_out), _ptr(scales_out), _ptr(ws),
                           _nbytes(ws), ctypes.byref(prof) if prof is not None else None, _stream(stream)))


def evict_fused(d: TpDims, batch: Batch, q_guide, k, v, *, softmax_scale: float, pool_k: int, qfmt: int,
                bits: int, rule: int = TP_COMBINE_MUL, keep_ratio: float = 0.0, keep_budget: int = 0,
                bufs: EvictBuffers = None, events=None, stream=None, k_guide=None, guide_lse=None,
                full_codes: bool = True) -> EvictBuffers:
    """The whole path through tp_evict; returns the buffers (kept_idx, k_c, v_q_c, scales_c, ...).
    full_codes=False: no code tensor for every token (bufs.v_q untouched); the compaction
    quantises the kept rows."""
    ko = kept_offsets_for(batch, keep_ratio, keep_budget)
    if bufs is None:
        bufs = EvictBuffers(d, batch, qfmt, bits, ko, device=k.device)
    tp_evict(d, batch, q_guide, k, v, softmax_scale, pool_k, qfmt, bits, rule, keep_ratio, keep_budget, ko,
             bufs.s_key, bufs.scales, bufs.v_q if full_codes else None, bufs.s_comb, bufs.kept_idx, bufs.k_c,
             bufs.v_q_c, bufs.scales_c, bufs.ws_evict, events, stream, k_guide, guide_lse)
    return bufs
