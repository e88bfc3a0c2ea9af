"""Thin ctypes binding of libws.so (the C ABI of include/ws.h).

Functions carry the C names and only marshal arguments; every step of the
attention path runs in the HIP kernels of libws.so.  ``Cache`` is a small
convenience wrapper that takes torch tensors (device memory and the current
stream are torch's; nothing is computed with torch).

Importing this module loads libws.so and raises if it is missing: there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

# torch first: libws.so then binds to the HIP runtime torch has loaded, so
# both share one runtime (loaded ahead of torch, libws.so pulls in the system
# runtime, which found no device next to torch's ROCm build).
import torch  # noqa: F401

from . import _build

if not os.path.exists(_build.LIB_PATH):
    raise ImportError(
        f"libws.so not built ({_build.LIB_PATH}); run __graft_entry__.build() or "
        "`python -m paper_2607_04443_amd._build`")

_lib = ctypes.CDLL(_build.LIB_PATH)

# --------------------------------------------------------------------------- #
# types (mirror include/ws.h)
# --------------------------------------------------------------------------- #
WS_OK, WS_ERR_INVALID_ARG, WS_ERR_SHAPE, WS_ERR_OUT_OF_PAGES = 0, 1, 2, 3
WS_ERR_UNKNOWN_UNIT, WS_ERR_COMMITTED, WS_ERR_UNSUPPORTED, WS_ERR_HIP = 4, 5, 6, 7
STATUS_NAMES = {0: "WS_OK", 1: "WS_ERR_INVALID_ARG", 2: "WS_ERR_SHAPE", 3: "WS_ERR_OUT_OF_PAGES",
                4: "WS_ERR_UNKNOWN_UNIT", 5: "WS_ERR_COMMITTED", 6: "WS_ERR_UNSUPPORTED",
                7: "WS_ERR_HIP"}
WS_KIND_COND, WS_KIND_VIDEO, WS_KIND_AUDIO = 0, 1, 2
WS_APPEND_RAW, WS_APPEND_NORM_ROPE, WS_QUERY_PREPARED = 0, 1, 2
WS_OPT_VIDEO_KV_SPLITS, WS_OPT_AUDIO_KV_SPLITS, WS_OPT_VIDEO_RUNNING_MAX = 0, 1, 2
WS_OPT_VIDEO_CLASS_CUS = 3
WS_OPT_STEP_SEPARATE_AUDIO = 4
INT32_MIN = -(2 ** 31)


def WS_KIND_BIT(kind):
    return 1 << kind


class ws_cache_config(ctypes.Structure):
    _fields_ = [("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_tokens", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("max_q_tokens", ctypes.c_int32), ("rope_max_pos", ctypes.c_int32 * 3),
                ("rope_pairs", ctypes.c_int32 * 3), ("rope_theta", ctypes.c_double)]


class ws_append_desc(ctypes.Structure):
    _fields_ = [("unit", ctypes.c_int32), ("kind", ctypes.c_int32), ("n_tokens", ctypes.c_int32),
                ("mode", ctypes.c_int32), ("positions", ctypes.c_void_p),
                ("gamma", ctypes.c_void_p), ("eps", ctypes.c_float)]


class ws_append_item(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("tok_stride", ctypes.c_int64),
                ("head_stride", ctypes.c_int64), ("desc", ws_append_desc)]


WS_MAX_APPEND_ITEMS = 16


class ws_query_desc(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("positions", ctypes.c_void_p),
                ("gamma", ctypes.c_void_p), ("eps", ctypes.c_float),
                ("softmax_scale", ctypes.c_float)]


class ws_query_item(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("tok_stride", ctypes.c_int64),
                ("head_stride", ctypes.c_int64), ("n_q", ctypes.c_int32),
                ("desc", ws_query_desc), ("q_out", ctypes.c_void_p),
                ("out_tok_stride", ctypes.c_int64), ("out_head_stride", ctypes.c_int64)]


WS_MAX_QUERY_ITEMS = 4


class ws_mask_spec(ctypes.Structure):
    _fields_ = [("q_unit", ctypes.c_int32), ("min_visible_unit", ctypes.c_int32),
                ("kind_mask", ctypes.c_uint32)]


class ws_attn_call(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("q_tok_stride", ctypes.c_int64),
                ("q_head_stride", ctypes.c_int64), ("n_q", ctypes.c_int32),
                ("desc", ws_query_desc), ("mask", ws_mask_spec), ("out", ctypes.c_void_p),
                ("out_tok_stride", ctypes.c_int64), ("out_head_stride", ctypes.c_int64)]


class ws_query_group(ctypes.Structure):
    _fields_ = [("n_q", ctypes.c_int32), ("mask", ws_mask_spec)]


WS_MAX_QUERY_GROUPS = 8


class ws_block_step_args(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("n_video", ctypes.c_int32), ("n_audio", ctypes.c_int32),
                ("unit", ctypes.c_int32), ("video_positions", ctypes.c_void_p),
                ("audio_positions", ctypes.c_void_p), ("gamma_q", ctypes.c_void_p),
                ("gamma_k", ctypes.c_void_p), ("eps", ctypes.c_float),
                ("softmax_scale", ctypes.c_float), ("video_mask", ws_mask_spec),
                ("audio_mask", ws_mask_spec), ("attn_out", ctypes.c_void_p), ("y", ctypes.c_void_p)]


class ws_cache_stats(ctypes.Structure):
    _fields_ = [("pages_total", ctypes.c_int32), ("pages_free", ctypes.c_int32),
                ("n_segments", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class ws_call_timing(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("n_splits", ctypes.c_int32),
                ("attn_us", ctypes.c_float), ("merge_us", ctypes.c_float)]


_vp, _i32, _i64, _u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
_P = ctypes.POINTER
_SIGS = {
    "ws_cache_create": [_P(ws_cache_config), _P(_vp)],
    "ws_cache_destroy": [_vp],
    "ws_cache_reset": [_vp],
    "ws_kv_append": [_vp, _vp, _vp, _i64, _i64, _P(ws_append_desc), _vp],
    "ws_kv_append_many": [_vp, _i32, _P(ws_append_item), _vp],
    "ws_step_append": [_vp, _i32, _P(ws_append_item), _i32, _P(ws_query_item), _vp],
    "ws_unit_commit": [_vp, _i32],
    "ws_kv_evict_before": [_vp, _i32],
    "ws_kv_release": [_vp, _i32, _i32],
    "ws_unit_attention": [_vp, _i64, _i64, _i32, _P(ws_query_desc), _vp, _P(ws_mask_spec), _vp,
                          _i64, _i64, _vp],
    "ws_audio_attention": [_vp, _i64, _i64, _i32, _P(ws_query_desc), _vp, _P(ws_mask_spec), _vp,
                           _i64, _i64, _vp],
    "ws_unit_attention_groups": [_vp, _i64, _i64, _i32, _P(ws_query_group), _P(ws_query_desc), _vp,
                                 _vp, _i64, _i64, _vp],
    "ws_step_attention": [_vp, _P(ws_attn_call), _P(ws_attn_call), _vp],
    "ws_step_attention_noalloc": [_vp, _P(ws_attn_call), _P(ws_attn_call), _vp],
    "ws_cache_export": [_vp, _i32, _i32, _vp, _vp],
    "ws_block_create": [_vp, _vp, _vp, _i32, _P(_vp)],
    "ws_block_destroy": [_vp],
    "ws_block_step": [_vp, _P(ws_block_step_args), _vp],
    "ws_segment_tokens": [_vp, _i32, _i32, _P(_i32)],
    "ws_segment_pages": [_vp, _i32, _i32, _P(_i32), _i32, _P(_i32)],
    "ws_cache_info": [_vp, _P(ws_cache_stats)],
    "ws_cache_check": [_vp, _P(_u32)],
    "ws_cache_set_option": [_vp, _i32, _i32],
    "ws_cache_timing_enable": [_vp, _i32],
    "ws_cache_timing_read": [_vp, _P(ws_call_timing), _i32, _P(_i32)],
    "ws_probe_mfma": [_i32, _i32, _vp, _P(ctypes.c_double), _vp],
    "ws_probe_mfma_random": [_i32, _i32, _vp, _P(ctypes.c_double), _vp],
    "ws_probe_read": [_vp, _i64, _i32, _vp, _vp],
}
for _name, _args in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = ctypes.c_int
_lib.ws_last_error.argtypes = []
_lib.ws_last_error.restype = ctypes.c_char_p


class WsError(RuntimeError):
    def __init__(self, status, fn):
        self.status = status
        msg = _lib.ws_last_error().decode(errors="replace")
        super().__init__(f"{fn}: {STATUS_NAMES.get(status, status)}: {msg}")


def _check(status, fn):
    if status != WS_OK:
        raise WsError(status, fn)


# --------------------------------------------------------------------------- #
# same-named entry points (raw pointers / ints)
# --------------------------------------------------------------------------- #
def ws_cache_create(cfg: ws_cache_config) -> int:
    h = _vp()
    _check(_lib.ws_cache_create(ctypes.byref(cfg), ctypes.byref(h)), "ws_cache_create")
    return h.value


def ws_cache_destroy(cache):
    _check(_lib.ws_cache_destroy(cache), "ws_cache_destroy")


def ws_cache_reset(cache):
    _check(_lib.ws_cache_reset(cache), "ws_cache_reset")


def ws_kv_append(cache, k, v, tok_stride, head_stride, desc: ws_append_desc, stream):
    _check(_lib.ws_kv_append(cache, k, v, tok_stride, head_stride, ctypes.byref(desc), stream),
           "ws_kv_append")


def ws_kv_append_many(cache, items, stream):
    """items: a sequence of ws_append_item."""
    arr = (ws_append_item * len(items))(*items)
    _check(_lib.ws_kv_append_many(cache, len(items), arr, stream), "ws_kv_append_many")


def ws_step_append(cache, items, queries, stream):
    """items: a sequence of ws_append_item; queries: a sequence of ws_query_item."""
    arr = (ws_append_item * len(items))(*items) if items else None
    qarr = (ws_query_item * len(queries))(*queries) if queries else None
    _check(_lib.ws_step_append(cache, len(items), arr, len(queries), qarr, stream),
           "ws_step_append")


def ws_unit_commit(cache, unit):
    _check(_lib.ws_unit_commit(cache, unit), "ws_unit_commit")


def ws_kv_evict_before(cache, unit):
    _check(_lib.ws_kv_evict_before(cache, unit), "ws_kv_evict_before")


def ws_kv_release(cache, unit, kind):
    _check(_lib.ws_kv_release(cache, unit, kind), "ws_kv_release")


def ws_unit_attention(q, q_tok_stride, q_head_stride, n_q, qdesc, cache, mask, out,
                      out_tok_stride, out_head_stride, stream):
    _check(_lib.ws_unit_attention(q, q_tok_stride, q_head_stride, n_q, ctypes.byref(qdesc), cache,
                                  ctypes.byref(mask), out, out_tok_stride, out_head_stride,
                                  stream), "ws_unit_attention")


def ws_audio_attention(q, q_tok_stride, q_head_stride, n_q, qdesc, cache, mask, out,
                       out_tok_stride, out_head_stride, stream):
    _check(_lib.ws_audio_attention(q, q_tok_stride, q_head_stride, n_q, ctypes.byref(qdesc), cache,
                                   ctypes.byref(mask), out, out_tok_stride, out_head_stride,
                                   stream), "ws_audio_attention")


def ws_unit_attention_groups(q, q_tok_stride, q_head_stride, groups, qdesc, cache, out,
                             out_tok_stride, out_head_stride, stream):
    """groups: a sequence of ws_query_group."""
    arr = (ws_query_group * max(len(groups), 1))(*groups)
    _check(_lib.ws_unit_attention_groups(q, q_tok_stride, q_head_stride, len(groups), arr,
                                         ctypes.byref(qdesc), cache, out, out_tok_stride,
                                         out_head_stride, stream), "ws_unit_attention_groups")


def ws_step_attention(cache, video: ws_attn_call, audio: ws_attn_call, stream):
    _check(_lib.ws_step_attention(cache, ctypes.byref(video), ctypes.byref(audio), stream),
           "ws_step_attention")


def ws_step_attention_noalloc(cache, video: ws_attn_call, audio: ws_attn_call, stream):
    _check(_lib.ws_step_attention_noalloc(cache, ctypes.byref(video), ctypes.byref(audio), stream),
           "ws_step_attention_noalloc")


def ws_block_create(cache, w_qkv, w_out, max_rows) -> int:
    h = _vp()
    _check(_lib.ws_block_create(cache, w_qkv, w_out, max_rows, ctypes.byref(h)), "ws_block_create")
    return h.value


def ws_block_destroy(block):
    _check(_lib.ws_block_destroy(block), "ws_block_destroy")


def ws_block_step(block, args: ws_block_step_args, stream):
    _check(_lib.ws_block_step(block, ctypes.byref(args), stream), "ws_block_step")


def ws_cache_export(cache, unit, kind, k_host, v_host):
    _check(_lib.ws_cache_export(cache, unit, kind, k_host, v_host), "ws_cache_export")


def ws_segment_tokens(cache, unit, kind) -> int:
    n = _i32()
    _check(_lib.ws_segment_tokens(cache, unit, kind, ctypes.byref(n)), "ws_segment_tokens")
    return n.value


def ws_segment_pages(cache, unit, kind) -> list:
    n = _i32()
    _check(_lib.ws_segment_pages(cache, unit, kind, None, 0, ctypes.byref(n)), "ws_segment_pages")
    buf = (_i32 * max(n.value, 1))()
    _check(_lib.ws_segment_pages(cache, unit, kind, buf, n.value, ctypes.byref(n)), "ws_segment_pages")
    return [buf[i] for i in range(n.value)]


def ws_cache_info(cache) -> ws_cache_stats:
    st = ws_cache_stats()
    _check(_lib.ws_cache_info(cache, ctypes.byref(st)), "ws_cache_info")
    return st


def ws_cache_check(cache) -> int:
    f = _u32()
    _check(_lib.ws_cache_check(cache, ctypes.byref(f)), "ws_cache_check")
    return f.value


def ws_cache_set_option(cache, opt, value):
    _check(_lib.ws_cache_set_option(cache, opt, value), "ws_cache_set_option")


def ws_cache_timing_enable(cache, capacity):
    _check(_lib.ws_cache_timing_enable(cache, capacity), "ws_cache_timing_enable")


def ws_cache_timing_read(cache, max_calls):
    buf = (ws_call_timing * max(max_calls, 1))()
    n = _i32()
    _check(_lib.ws_cache_timing_read(cache, buf, max_calls, ctypes.byref(n)), "ws_cache_timing_read")
    return [buf[i] for i in range(n.value)]


def ws_probe_mfma(workgroups, iters, sink, stream):
    """Enqueues the bf16 MFMA calibration loop; returns its FLOP count.
    sink: device address of a float; stream: HIP stream handle."""
    flop = ctypes.c_double()
    _check(_lib.ws_probe_mfma(workgroups, iters, sink, ctypes.byref(flop), stream), "ws_probe_mfma")
    return flop.value


def ws_probe_mfma_random(workgroups, iters, sink, stream):
    """The same loop on hashed random operands; returns its FLOP count."""
    flop = ctypes.c_double()
    _check(_lib.ws_probe_mfma_random(workgroups, iters, sink, ctypes.byref(flop), stream),
           "ws_probe_mfma_random")
    return flop.value


def ws_probe_read(buf, nbytes, workgroups, sink, stream):
    """Enqueues one streaming read of nbytes at device address buf."""
    _check(_lib.ws_probe_read(buf, nbytes, workgroups, sink, stream), "ws_probe_read")


def ws_last_error() -> str:
    return _lib.ws_last_error().decode(errors="replace")


# --------------------------------------------------------------------------- #
# torch-facing convenience wrapper (marshalling only)
# --------------------------------------------------------------------------- #
def _stream_handle(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check_tensor(name, t, dtype):
    import torch
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}")
    if dtype == torch.bfloat16 and (t.dim() != 3 or t.stride(2) != 1):
        raise ValueError(f"{name} must be [tokens, heads, 128] with unit innermost stride")


class Cache:
    """Owns one ws_cache; methods mirror ws_kv_append / ws_unit_attention / ..."""

    def __init__(self, num_heads, max_pages, max_q_tokens=1024, rope_max_pos=(65536, 256, 256),
                 rope_pairs=(22, 21, 21), rope_theta=10000.0):
        cfg = ws_cache_config()
        cfg.num_heads, cfg.head_dim, cfg.page_tokens = num_heads, 128, 64
        cfg.max_pages, cfg.max_q_tokens = max_pages, max_q_tokens
        cfg.rope_max_pos[:] = list(rope_max_pos)
        cfg.rope_pairs[:] = list(rope_pairs)
        cfg.rope_theta = rope_theta
        self.num_heads = num_heads
        self.handle = ws_cache_create(cfg)

    def close(self):
        if self.handle:
            ws_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def _item(unit, kind, k, v, mode=WS_APPEND_RAW, positions=None, gamma=None, eps=1e-6):
        import torch
        _check_tensor("k", k, torch.bfloat16)
        _check_tensor("v", v, torch.bfloat16)
        if k.stride() != v.stride() or k.shape != v.shape:
            raise ValueError("k and v must share shape and strides")
        it = ws_append_item()
        it.k, it.v = k.data_ptr(), v.data_ptr()
        it.tok_stride, it.head_stride = k.stride(0), k.stride(1)
        d = it.desc
        d.unit, d.kind, d.n_tokens, d.mode = unit, kind, k.shape[0], mode
        d.positions = positions.data_ptr() if positions is not None else None
        d.gamma = gamma.data_ptr() if gamma is not None else None
        d.eps = eps
        return it

    def append(self, unit, kind, k, v, mode=WS_APPEND_RAW, positions=None, gamma=None, eps=1e-6,
               stream=None):
        it = self._item(unit, kind, k, v, mode, positions, gamma, eps)
        ws_kv_append(self.handle, it.k, it.v, it.tok_stride, it.head_stride, it.desc,
                     _stream_handle(stream))

    def append_many(self, items, stream=None):
        """items: dicts with the keyword arguments of append (stream aside)."""
        ws_kv_append_many(self.handle, [self._item(**x) for x in items], _stream_handle(stream))

    @staticmethod
    def _query_item(q, q_out, mode=WS_APPEND_NORM_ROPE, positions=None, gamma=None, eps=1e-6,
                    scale=0.0):
        import torch
        _check_tensor("q", q, torch.bfloat16)
        _check_tensor("q_out", q_out, torch.bfloat16)
        if q.shape != q_out.shape:
            raise ValueError("q and q_out must have the same shape")
        it = ws_query_item()
        it.q, it.tok_stride, it.head_stride, it.n_q = q.data_ptr(), q.stride(0), q.stride(1), q.shape[0]
        d = it.desc
        d.mode = mode
        d.positions = positions.data_ptr() if positions is not None else None
        d.gamma = gamma.data_ptr() if gamma is not None else None
        d.eps, d.softmax_scale = eps, scale
        it.q_out, it.out_tok_stride, it.out_head_stride = q_out.data_ptr(), q_out.stride(0), q_out.stride(1)
        return it

    def step_append(self, items=(), queries=(), stream=None):
        """One launch for a step's K/V appends (dicts with the keyword arguments
        of append) and query preparations (dicts with q, q_out, mode, positions,
        gamma, eps, scale); q_out then feeds the attention calls with mode
        WS_QUERY_PREPARED."""
        ws_step_append(self.handle, [self._item(**x) for x in items],
                       [self._query_item(**x) for x in queries], _stream_handle(stream))

    def _attn(self, fn, q, out, mask, mode, positions, gamma, eps, scale, stream):
        import torch
        _check_tensor("q", q, torch.bfloat16)
        _check_tensor("out", out, torch.bfloat16)
        qd = ws_query_desc()
        qd.mode = mode
        qd.positions = positions.data_ptr() if positions is not None else None
        qd.gamma = gamma.data_ptr() if gamma is not None else None
        qd.eps, qd.softmax_scale = eps, scale
        fn(q.data_ptr(), q.stride(0), q.stride(1), q.shape[0], qd, self.handle, mask,
           out.data_ptr(), out.stride(0), out.stride(1), _stream_handle(stream))
        return out

    @staticmethod
    def _call(q, out, mask, mode=WS_APPEND_NORM_ROPE, positions=None, gamma=None, eps=1e-6,
              scale=0.0):
        import torch
        _check_tensor("q", q, torch.bfloat16)
        _check_tensor("out", out, torch.bfloat16)
        c = ws_attn_call()
        c.q, c.q_tok_stride, c.q_head_stride, c.n_q = q.data_ptr(), q.stride(0), q.stride(1), q.shape[0]
        d = c.desc
        d.mode = mode
        d.positions = positions.data_ptr() if positions is not None else None
        d.gamma = gamma.data_ptr() if gamma is not None else None
        d.eps, d.softmax_scale = eps, scale
        c.mask = mask
        c.out, c.out_tok_stride, c.out_head_stride = out.data_ptr(), out.stride(0), out.stride(1)
        return c

    def step_attention(self, video, audio, stream=None):
        """video, audio: dicts with the arguments of unit_attention /
        audio_attention (q, out, mask, mode, positions, gamma, eps, scale)."""
        ws_step_attention(self.handle, self._call(**video), self._call(**audio),
                          _stream_handle(stream))

    def step_attention_noalloc(self, video, audio, stream=None):
        """step_attention with the split-KV partials in the library's static
        workspace (no device allocation by the call)."""
        ws_step_attention_noalloc(self.handle, self._call(**video), self._call(**audio),
                                  _stream_handle(stream))

    def unit_attention(self, q, out, mask, mode=WS_APPEND_NORM_ROPE, positions=None, gamma=None,
                       eps=1e-6, scale=0.0, stream=None):
        return self._attn(ws_unit_attention, q, out, mask, mode, positions, gamma, eps, scale,
                          stream)

    def unit_attention_groups(self, q, out, groups, mode=WS_APPEND_NORM_ROPE, positions=None,
                              gamma=None, eps=1e-6, scale=0.0, stream=None):
        """groups: (n_rows, ws_mask_spec) pairs; q's rows are the groups' rows in order."""
        import torch
        _check_tensor("q", q, torch.bfloat16)
        _check_tensor("out", out, torch.bfloat16)
        qd = ws_query_desc()
        qd.mode = mode
        qd.positions = positions.data_ptr() if positions is not None else None
        qd.gamma = gamma.data_ptr() if gamma is not None else None
        qd.eps, qd.softmax_scale = eps, scale
        gs = []
        for n, m in groups:
            g = ws_query_group()
            g.n_q, g.mask = n, m
            gs.append(g)
        ws_unit_attention_groups(q.data_ptr(), q.stride(0), q.stride(1), gs, qd, self.handle,
                                 out.data_ptr(), out.stride(0), out.stride(1), _stream_handle(stream))
        return out

    def audio_attention(self, q, out, mask, mode=WS_APPEND_NORM_ROPE, positions=None,
                        gamma=None, eps=1e-6, scale=0.0, stream=None):
        return self._attn(ws_audio_attention, q, out, mask, mode, positions, gamma, eps, scale,
                          stream)

    def commit(self, unit):
        ws_unit_commit(self.handle, unit)

    def evict_before(self, unit):
        ws_kv_evict_before(self.handle, unit)

    def release(self, unit, kind):
        ws_kv_release(self.handle, unit, kind)

    def export(self, unit, kind):
        """(K, V) of a segment as numpy uint16 bf16 bits [n, H, 128]."""
        import numpy as np
        n = ws_segment_tokens(self.handle, unit, kind)
        k = np.empty((n, self.num_heads, 128), dtype=np.uint16)
        v = np.empty_like(k)
        ws_cache_export(self.handle, unit, kind, k.ctypes.data, v.ctypes.data)
        return k, v

    def pages(self, unit, kind):
        """Pool page ids of a segment, in token order."""
        return ws_segment_pages(self.handle, unit, kind)

    def info(self):
        return ws_cache_info(self.handle)

    def check(self):
        return ws_cache_check(self.handle)

    def set_option(self, opt, value):
        ws_cache_set_option(self.handle, opt, value)

    def timing_enable(self, capacity):
        ws_cache_timing_enable(self.handle, capacity)
        self._timing_cap = capacity

    def timing_read(self):
        """Per-call launch timing recorded since the last read, oldest first:
        dicts with path ('video', 'audio', 'append', 'qkv_gemm', 'out_gemm', or
        'audio_riders': a step's audio call with its rows in the video kernel),
        n_splits, attn_us, merge_us."""
        out = ws_cache_timing_read(self.handle, getattr(self, "_timing_cap", 0))
        names = {0: "video", 1: "audio", 2: "append", 3: "qkv_gemm", 4: "out_gemm", 5: "audio_riders"}
        return [dict(path=names.get(t.path, str(t.path)), n_splits=t.n_splits, attn_us=t.attn_us,
                     merge_us=t.merge_us) for t in out]


class Block:
    """Owns one ws_block over a Cache: the attention sub-block of a performer
    layer (QKV projection, append, attention, output projection)."""

    def __init__(self, cache, w_qkv, w_out, max_rows):
        import torch
        for name, w in (("w_qkv", w_qkv), ("w_out", w_out)):
            if not w.is_cuda or w.dtype != torch.bfloat16 or not w.is_contiguous():
                raise ValueError(f"{name} must be a contiguous bf16 device tensor")
        self._keep = (cache, w_qkv, w_out)
        self.handle = ws_block_create(cache.handle, w_qkv.data_ptr(), w_out.data_ptr(), max_rows)

    def close(self):
        if self.handle:
            ws_block_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, x, n_video, unit, video_positions, audio_positions, gamma_q, gamma_k, y,
             video_mask, audio_mask, eps=1e-6, scale=0.0, attn_out=None, stream=None):
        """x, y (and attn_out): contiguous bf16 [n_video + n_audio, hidden] device tensors."""
        a = ws_block_step_args()
        a.x, a.n_video, a.n_audio, a.unit = x.data_ptr(), n_video, x.shape[0] - n_video, unit
        a.video_positions = video_positions.data_ptr()
        a.audio_positions = audio_positions.data_ptr() if audio_positions is not None else None
        a.gamma_q, a.gamma_k = gamma_q.data_ptr(), gamma_k.data_ptr()
        a.eps, a.softmax_scale = eps, scale
        a.video_mask, a.audio_mask = video_mask, audio_mask
        a.attn_out = attn_out.data_ptr() if attn_out is not None else None
        a.y = y.data_ptr()
        ws_block_step(self.handle, a, _stream_handle(stream))
        return y


def mask_spec(q_unit, min_visible_unit=INT32_MIN, kinds=(WS_KIND_COND, WS_KIND_VIDEO)):
    m = ws_mask_spec()
    m.q_unit, m.min_visible_unit = q_unit, min_visible_unit
    m.kind_mask = sum(1 << k for k in kinds)
    return m
