"""The C ABI boundary, checked without a GPU: every declared entry point is
exported by libws.so, and the ctypes mirrors of the header's structs have the
C layout (sizes and offsets measured by compiling the header with gcc)."""
import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ws.h")


def _ensure_built():
    from paper_2607_04443_amd import _build
    if not (os.path.exists(_build.LIB_PATH) and os.path.exists(_build.HOST_LIB_PATH)):
        _build.build()
    return _build


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"WS_API\s+[\w\s\*]+?\b(ws_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("ws_cache_create", "ws_kv_append", "ws_unit_attention",
                     "ws_audio_attention", "ws_cache_export", "ws_last_error"):
        assert required in names


def test_library_exports_every_declared_symbol():
    b = _ensure_built()
    lib = ctypes.CDLL(b.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    out = subprocess.run(["nm", "-D", "--defined-only", b.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(set(re.findall(r"\bT (ws_\w+)", out)))
    assert exported == declared_functions()


def test_probe_arguments_rejected_before_any_device_call():
    """The calibration probes validate on the host: bad sizes and alignments
    return WS_ERR_INVALID_ARG (1) without touching a device (the fake,
    non-null addresses below are never dereferenced)."""
    b = _ensure_built()
    lib = ctypes.CDLL(b.LIB_PATH)
    lib.ws_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                  ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    lib.ws_probe_mfma_random.argtypes = lib.ws_probe_mfma.argtypes
    lib.ws_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                  ctypes.c_void_p]
    lib.ws_last_error.restype = ctypes.c_char_p
    flop = ctypes.c_double()
    fake = ctypes.c_void_p(4096)
    for probe in (lib.ws_probe_mfma, lib.ws_probe_mfma_random):
        for wg, it in [(0, 1), (65537, 1), (1, 0), (1, (1 << 24) + 1)]:
            assert probe(wg, it, fake, ctypes.byref(flop), None) == 1, (wg, it)
        assert probe(1, 1, None, ctypes.byref(flop), None) == 1
    assert lib.ws_probe_read(fake, 0, 1, fake, None) == 1
    assert lib.ws_probe_read(fake, 24, 1, fake, None) == 1          # not a multiple of 16
    assert lib.ws_probe_read(ctypes.c_void_p(4104), 32, 1, fake, None) == 1  # misaligned
    assert lib.ws_probe_read(fake, 32, 0, fake, None) == 1
    assert b"workgroups" in lib.ws_last_error()


def test_last_error_callable_without_device():
    b = _ensure_built()
    lib = ctypes.CDLL(b.LIB_PATH)
    lib.ws_last_error.restype = ctypes.c_char_p
    assert isinstance(lib.ws_last_error(), bytes)


def test_binding_names_match_header():
    _ensure_built()
    from paper_2607_04443_amd import ws
    for n in declared_functions():
        assert callable(getattr(ws, n)), n


_PROBE = r"""
#include <stddef.h>
#include <stdio.h>
#include "ws.h"
#define P(T, F) printf(#T "." #F " %zu\n", offsetof(T, F));
#define S(T) printf(#T " %zu\n", sizeof(T));
int main(void) {
  S(ws_cache_config) P(ws_cache_config, max_q_tokens) P(ws_cache_config, rope_max_pos)
  P(ws_cache_config, rope_pairs) P(ws_cache_config, rope_theta)
  S(ws_append_desc) P(ws_append_desc, kind) P(ws_append_desc, mode) P(ws_append_desc, positions)
  P(ws_append_desc, gamma) P(ws_append_desc, eps)
  S(ws_query_desc) P(ws_query_desc, positions) P(ws_query_desc, gamma) P(ws_query_desc, eps)
  P(ws_query_desc, softmax_scale)
  S(ws_mask_spec) P(ws_mask_spec, kind_mask)
  S(ws_cache_stats)
  S(ws_call_timing) P(ws_call_timing, n_splits) P(ws_call_timing, attn_us) P(ws_call_timing, merge_us)
  S(ws_append_item) P(ws_append_item, v) P(ws_append_item, tok_stride) P(ws_append_item, head_stride)
  P(ws_append_item, desc)
  S(ws_query_item) P(ws_query_item, tok_stride) P(ws_query_item, head_stride) P(ws_query_item, n_q)
  P(ws_query_item, desc) P(ws_query_item, q_out) P(ws_query_item, out_tok_stride)
  P(ws_query_item, out_head_stride)
  S(ws_attn_call) P(ws_attn_call, q_tok_stride) P(ws_attn_call, n_q) P(ws_attn_call, desc)
  P(ws_attn_call, mask) P(ws_attn_call, out) P(ws_attn_call, out_tok_stride)
  P(ws_attn_call, out_head_stride)
  printf("max_items %d\n", WS_MAX_APPEND_ITEMS);
  printf("max_query_items %d\n", WS_MAX_QUERY_ITEMS);
  printf("prepared %d\n", (int)WS_QUERY_PREPARED);
  printf("enum %zu\n", sizeof(ws_kind));
  return 0;
}
"""


def test_struct_layouts_match_c(tmp_path):
    _ensure_built()
    from paper_2607_04443_amd import ws
    src = tmp_path / "probe.c"
    src.write_text(_PROBE)
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o",
                    str(exe)], check=True)
    c = dict(line.rsplit(" ", 1) for line in
             subprocess.run([str(exe)], capture_output=True, text=True, check=True)
             .stdout.splitlines())
    c = {k: int(v) for k, v in c.items()}
    assert c["enum"] == 4
    assert c["max_items"] == ws.WS_MAX_APPEND_ITEMS
    assert c["max_query_items"] == ws.WS_MAX_QUERY_ITEMS
    assert c["prepared"] == ws.WS_QUERY_PREPARED
    for name, typ in (("ws_cache_config", ws.ws_cache_config),
                      ("ws_append_desc", ws.ws_append_desc), ("ws_query_desc", ws.ws_query_desc),
                      ("ws_mask_spec", ws.ws_mask_spec), ("ws_cache_stats", ws.ws_cache_stats),
                      ("ws_call_timing", ws.ws_call_timing),
                      ("ws_append_item", ws.ws_append_item),
                      ("ws_query_item", ws.ws_query_item), ("ws_attn_call", ws.ws_attn_call)):
        assert ctypes.sizeof(typ) == c[name], name
        for key, off in c.items():
            if key.startswith(name + "."):
                assert getattr(typ, key.split(".")[1]).offset == off, key
