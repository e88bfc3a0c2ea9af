"""Parity of the HIP attention paths with the fp64 oracle.

The performer's per-step attention of a unit's video latent queries, and
separately of its few audio latent queries, over the K/V cache (Wan-Streamer
v0.2, Sec. 3), with block-causal visibility by unit (Fig. 1 caption).  Inputs
are the seeded bf16 workloads; every check goes through the C ABI.
"""
import numpy as np
import pytest

import oracle
from helpers import (Loaded, assert_gates, bf16_f64, dev_f32, dev_i32, errors, from_dev,
                     to_dev)
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu

VIDEO_KINDS = (synth.KIND_COND, synth.KIND_VIDEO)
ALL_KINDS = (synth.KIND_COND, synth.KIND_VIDEO, synth.KIND_AUDIO)


def _video(L, step=0, heads=None, **kw):
    st = L.wl.steps[step]
    got = L.run("video", st.q_video, st.q_video_pos, L.wl.current_unit, VIDEO_KINDS, **kw)
    ref = L.oracle(st.q_video, st.q_video_pos, L.wl.current_unit, VIDEO_KINDS, heads=heads, **kw)
    if heads is not None:
        got = got[:, heads]
    return got, ref


def _video_bound(L, step=0, heads=None, **kw):
    st = L.wl.steps[step]
    return L.bound(st.q_video, st.q_video_pos, L.wl.current_unit, VIDEO_KINDS, heads=heads, **kw)


@pytest.mark.parametrize("name,heads", [("v01", None), ("v02_single", None), ("v02_hist8", None)])
def test_video_parity(ws, name, heads):
    wl = synth.make_workload(name)
    L = Loaded(ws, wl)
    try:
        got, ref = _video(L, heads=heads)
        e = assert_gates(got, ref, label=name, bound=_video_bound(L, heads=heads))
        print(name, e)
    finally:
        L.close()


def test_long_history_back_to_back_steps(ws):
    """32 history units (30616 keys) and 4 denoising steps issued one after
    another on one stream, each rewriting the current unit's K/V in place
    (the appends and attentions of all steps are enqueued before the first
    read-back).  Heads 0, 13, 26, 39 of steps 0 and 3 against the oracle,
    which applies the same rewrites to its logical cache."""
    import torch
    wl = synth.make_workload("long32")
    heads = [0, 13, 26, 39]
    L = Loaded(ws, wl)
    try:
        outs = []
        for s, st in enumerate(wl.steps):
            if s > 0:
                for seg in st.segments:
                    L.append(seg)  # same (unit, kind): rewritten in place
            q, pos = to_dev(st.q_video), dev_i32(st.q_video_pos)
            out = torch.full_like(q, float("nan"))
            L._keep += [q, pos]
            L.cache.unit_attention(q, out, ws.mask_spec(wl.current_unit, -(2 ** 31), VIDEO_KINDS),
                                   ws.WS_APPEND_NORM_ROPE, pos, L.gq, wl.eps)
            outs.append(out)
        torch.cuda.synchronize()
        # the oracle cache holds the last step's K/V: check step 3 first
        st = wl.steps[3]
        ref = L.oracle(st.q_video, st.q_video_pos, wl.current_unit, VIDEO_KINDS, heads=heads)
        print("step 3", assert_gates(bf16_f64(from_dev(outs[3]))[:, heads], ref, label="long32 step 3"))
        st0 = wl.steps[0]
        for seg in st0.segments:
            L.ocache.append(seg.unit, seg.kind, seg.k, seg.v, oracle.MODE_NORM_ROPE, seg.positions,
                            wl.gamma_k.astype(np.float64), wl.eps)
        ref = L.oracle(st0.q_video, st0.q_video_pos, wl.current_unit, VIDEO_KINDS, heads=heads)
        print("step 0", assert_gates(bf16_f64(from_dev(outs[0]))[:, heads], ref, label="long32 step 0"))
    finally:
        L.close()


@pytest.mark.parametrize("variant", ["seeded", "sharp"])
def test_video_parity_gamma_variants(ws, variant):
    wl = synth.make_workload("v01", variant=variant)
    L = Loaded(ws, wl)
    try:
        got, ref = _video(L)
        if variant == "sharp":
            # gamma_q = 4 widens the logits 4x and with them the bf16 logit error; where
            # two keys compete the output error is ~ p1 p2 d(s1 - s2) |v1 - v2|, so only
            # the scale-free Frobenius gate and 4x-widened contract gates apply
            print(variant, assert_gates(got, ref, label=variant, scale=4.0, strict=False,
                                        bound=_video_bound(L)))
            assert np.linalg.norm(got - ref) <= 1e-2 * np.linalg.norm(ref)
        else:
            print(variant, assert_gates(got, ref, label=variant, bound=_video_bound(L)))
    finally:
        L.close()


@pytest.mark.parametrize("name", ["audio_c256", "audio"])
def test_audio_parity(ws, name):
    wl = synth.make_workload(name)
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        got = L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        ref = L.oracle(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        bound = L.bound(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        print(name, assert_gates(got, ref, label=name, bound=bound))
    finally:
        L.close()


def test_audio_kernel_agrees_with_video_kernel(ws):
    """Same 4 queries through both kernels over the same cache."""
    wl = synth.make_workload("audio_c256")
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        a = L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        v = L.run("video", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        assert_gates(a, v, label="audio vs video")
    finally:
        L.close()


TINY = synth.Config("tiny", 17, 3, (5, 7), 10, 2, audio=3)  # 35-token units: ragged pages


@pytest.mark.parametrize("n_q", [1, 2, 31, 33, 128, 129, 200])
def test_video_ragged_query_counts(ws, n_q):
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        rng = np.random.default_rng(n_q)
        q = synth.normal_bf16(rng, (n_q, TINY.heads, 128))
        pos = np.stack([np.full(n_q, wl.current_unit), rng.integers(0, 5, n_q),
                        rng.integers(0, 7, n_q)], axis=1).astype(np.int32)
        got = L.run("video", q, pos, wl.current_unit, ALL_KINDS)
        ref = L.oracle(q, pos, wl.current_unit, ALL_KINDS)
        assert_gates(got, ref, label=f"n_q={n_q}")
        if n_q <= 64:
            got = L.run("audio", q, pos, wl.current_unit, ALL_KINDS)
            assert_gates(got, ref, label=f"audio n_q={n_q}")
    finally:
        L.close()


@pytest.mark.parametrize("splits", [1, 2, 3, 8])
def test_video_split_counts(ws, splits):
    wl = synth.make_workload("v01")
    L = Loaded(ws, wl)
    try:
        L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, splits)
        got, ref = _video(L)
        assert_gates(got, ref, label=f"splits={splits}")
    finally:
        L.close()


@pytest.mark.parametrize("splits", [1, 7, 64])
def test_audio_split_counts(ws, splits):
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        L.cache.set_option(ws.WS_OPT_AUDIO_KV_SPLITS, splits)
        st = wl.steps[0]
        got = L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        ref = L.oracle(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        assert_gates(got, ref, label=f"audio splits={splits}")
    finally:
        L.close()


def test_window_and_causality(ws):
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        for q_unit, min_unit, kinds in ((2, 1, ALL_KINDS), (1, -(2 ** 31), VIDEO_KINDS),
                                        (2, 2, (synth.KIND_VIDEO,)), (0, 0, (synth.KIND_COND,))):
            got = L.run("video", st.q_video, st.q_video_pos, q_unit, kinds, min_unit=min_unit)
            ref = L.oracle(st.q_video, st.q_video_pos, q_unit, kinds, min_unit=min_unit)
            assert_gates(got, ref, label=f"mask {q_unit} {min_unit} {kinds}")
    finally:
        L.close()


def test_nothing_visible_gives_zero(ws):
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        for path in ("video", "audio"):
            got = L.run(path, st.q_audio, st.q_audio_pos, 7, (synth.KIND_VIDEO,), min_unit=5)
            assert (got == 0).all(), path
    finally:
        L.close()


def test_single_key_returns_value_exactly(ws):
    rng = np.random.default_rng(5)
    cfg = synth.Config("one", 18, 2, (1, 1), 1, 0)
    wl = synth.make_workload(cfg)
    L = Loaded(ws, wl)
    try:
        q = synth.normal_bf16(rng, (5, 2, 128))
        pos = np.zeros((5, 3), np.int32)
        for path in ("video", "audio"):
            got = L.run(path, q, pos, 0, (synth.KIND_COND,))
            want = bf16_f64(np.repeat(wl.cached[0].v, 5, axis=0))
            np.testing.assert_array_equal(got, want)
    finally:
        L.close()


def test_needle_per_page(ws):
    """Each query has one dominant RAW key (4x its own direction) in a
    different page and slot; the output must be exactly that key's value,
    which proves the page/slot indexing end to end."""
    rng = np.random.default_rng(6)
    H, n_keys, n_q = 2, 64 * 9 + 17, 150
    k = synth.normal_bf16(rng, (n_keys, H, 128))
    v = synth.normal_bf16(rng, (n_keys, H, 128))
    qf = rng.standard_normal((n_q, H, 128)).astype(np.float32)
    qf /= np.sqrt((qf * qf).mean(-1, keepdims=True))
    q = synth.bf16_bits(qf)
    needle = (np.arange(n_q) * 37 + 11) % n_keys
    for i, j in enumerate(needle):
        k[j] = synth.bf16_bits(4.0 * synth.bf16_to_f32(q[i]))
    cfg = synth.Config("needle", 19, H, (1, 1), n_keys, 0)
    wl = synth.make_workload(cfg)
    wl.cached[0].k, wl.cached[0].v = k, v
    L = Loaded(ws, wl)
    try:
        for path in ("video",):
            got = L.run(path, q, np.zeros((n_q, 3), np.int32), 0, (synth.KIND_COND,),
                        mode=ws.WS_APPEND_RAW)
            np.testing.assert_array_equal(got, bf16_f64(v[needle]))
        sub = slice(0, 40)
        got = L.run("audio", q[sub], np.zeros((40, 3), np.int32), 0, (synth.KIND_COND,),
                    mode=ws.WS_APPEND_RAW)
        np.testing.assert_array_equal(got, bf16_f64(v[needle[sub]]))
    finally:
        L.close()


def test_reruns_are_bit_identical(ws):
    wl = synth.make_workload("v02_single")
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        a = L.run("video", st.q_video, st.q_video_pos, wl.current_unit, VIDEO_KINDS)
        b = L.run("video", st.q_video, st.q_video_pos, wl.current_unit, VIDEO_KINDS)
        np.testing.assert_array_equal(a, b)
        a = L.run("audio", st.q_video[:4], st.q_video_pos[:4], wl.current_unit, VIDEO_KINDS)
        b = L.run("audio", st.q_video[:4], st.q_video_pos[:4], wl.current_unit, VIDEO_KINDS)
        np.testing.assert_array_equal(a, b)
    finally:
        L.close()


def test_masked_segment_equals_deleted_segment(ws):
    """Masking a history unit out (window) gives the same bits as never
    having appended it (one split, so the page order is the same)."""
    wl = synth.make_workload(TINY)
    A = Loaded(ws, wl)
    wl_b = synth.make_workload(TINY)
    wl_b.cached = [s for s in wl_b.cached if s.unit != 0 or s.kind == synth.KIND_COND]
    B = Loaded(ws, wl_b)
    try:
        for L in (A, B):
            L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, 1)
        st = wl.steps[0]
        a = A.run("video", st.q_video, st.q_video_pos, wl.current_unit, ALL_KINDS, min_unit=1)
        b = B.run("video", st.q_video, st.q_video_pos, wl.current_unit, ALL_KINDS)
        np.testing.assert_array_equal(a, b)
    finally:
        A.close()
        B.close()


@pytest.mark.parametrize("name", ["v01", "tiny"])
def test_video_running_max_path(ws, name):
    """The lazily raised running maximum (forced by option) against the
    oracle, and against the default key-norm-bound shift on the same cache:
    the two shifts give the same softmax."""
    wl = synth.make_workload(TINY if name == "tiny" else name)
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        kinds = ALL_KINDS if name == "tiny" else VIDEO_KINDS
        fixed = L.run("video", st.q_video, st.q_video_pos, wl.current_unit, kinds)
        L.cache.set_option(ws.WS_OPT_VIDEO_RUNNING_MAX, 1)
        for splits in (1, 3):
            L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, splits)
            lazy = L.run("video", st.q_video, st.q_video_pos, wl.current_unit, kinds)
            ref = L.oracle(st.q_video, st.q_video_pos, wl.current_unit, kinds)
            assert_gates(lazy, ref, label=f"running max, splits={splits}")
        assert_gates(fixed, lazy, label="bound shift vs running max")
        if st.q_audio is not None:  # the audio kernel follows the same option
            got = L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
            ref = L.oracle(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
            assert_gates(got, ref, label="audio, running max")
    finally:
        L.close()


def _unit_rows(rng, shape):
    """N(0,1) rows rescaled to an rms of 1 over the head dimension (fp32)."""
    x = rng.standard_normal(shape).astype(np.float32)
    return x / np.sqrt((x * x).mean(-1, keepdims=True))


def _logit_bound(q_bits, k_bits):
    """Per (query, head): the largest log2-domain logit over the keys and the
    Cauchy-Schwarz bound |Q''| max|k| the video kernel takes as its shift,
    from the bf16 inputs of a RAW call with the default scale (fp64)."""
    s = np.log2(np.e) / np.sqrt(128.0)
    q = bf16_f64(q_bits) * s
    k = bf16_f64(k_bits)
    logits = np.einsum("qhd,khd->qhk", q, k)
    bound = np.linalg.norm(q, axis=-1) * np.linalg.norm(k, axis=-1).max(axis=0)[None, :]
    return logits.max(axis=-1), bound


def test_video_single_anti_aligned_key_returns_value_exactly(ws):
    """One RAW key k = -2 q per head, RAW queries q: the logit bound
    |q''| |k| (about 32.6 in log2 units) selects the bound shift, and the only
    logit sits at minus the bound, so its weight is about 2^-65 while the 63
    empty slots of the page would weigh 2^-32.6 each.  Empty slots must not
    reach the row sum at all: the output must be V bit for bit, on the video
    path (bound shift and running maximum) and on the audio path."""
    rng = np.random.default_rng(31)
    H, n_q = 2, 5
    q1 = synth.bf16_bits(_unit_rows(rng, (1, H, 128)))
    k = synth.bf16_bits(-2.0 * synth.bf16_to_f32(q1))
    v = synth.normal_bf16(rng, (1, H, 128))
    q = np.repeat(q1, n_q, axis=0)
    mx, bound = _logit_bound(q, k)
    assert (bound <= 38.0).all() and (bound >= 28.0).all(), bound
    assert (mx <= -28.0).all(), mx
    wl = _raw_cond_workload("anti", H, k, v)
    L = Loaded(ws, wl)
    try:
        pos = np.zeros((n_q, 3), np.int32)
        want = bf16_f64(np.repeat(v, n_q, axis=0))
        for path in ("video", "audio"):
            got = L.run(path, q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
            np.testing.assert_array_equal(got, want, err_msg=path)
        L.cache.set_option(ws.WS_OPT_VIDEO_RUNNING_MAX, 1)
        got = L.run("video", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        np.testing.assert_array_equal(got, want, err_msg="video, running maximum")
    finally:
        L.close()


@pytest.mark.parametrize("n_keys", [24, 64 * 2 + 24])
def test_video_partial_page_far_below_shift(ws, n_keys):
    """A key set ending in a page with 24 valid slots whose every logit lies
    far below zero (all <= -12, about -24 in log2 units) while the logit bound
    stays under the bound-shift limit: the weights (about 2^-49) are far
    smaller than an empty slot's (about 2^-25), so any empty-slot mass left in
    the row sum would swamp them.  Against the oracle, with the gates, and
    against the running-maximum path."""
    rng = np.random.default_rng(32)
    H, n_q = 2, 40
    base = _unit_rows(rng, (1, H, 128))
    q = synth.bf16_bits(_unit_rows(rng, (n_q, H, 128)) * 0.1 + base)
    k = synth.bf16_bits(-1.5 * base + 0.3 * rng.standard_normal((n_keys, H, 128)).astype(np.float32))
    v = synth.normal_bf16(rng, (n_keys, H, 128))
    mx, bound = _logit_bound(q, k)
    assert (mx <= -12.0).all(), float(mx.max())
    assert (bound <= 38.0).all(), float(bound.max())
    wl = _raw_cond_workload("below", H, k, v)
    L = Loaded(ws, wl)
    try:
        pos = np.zeros((n_q, 3), np.int32)
        ref = L.oracle(q, pos, 0, (synth.KIND_COND,), mode=oracle.MODE_RAW)
        got = L.run("video", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        print("bound shift", assert_gates(got, ref, label=f"far below, {n_keys} keys"))
        got_a = L.run("audio", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        assert_gates(got_a, ref, label=f"audio, far below, {n_keys} keys")
        L.cache.set_option(ws.WS_OPT_VIDEO_RUNNING_MAX, 1)
        lazy = L.run("video", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        assert_gates(lazy, ref, label=f"running max, far below, {n_keys} keys")
    finally:
        L.close()


def _raw_cond_workload(name, H, k, v):
    cfg = synth.Config(name, 20, H, (1, 1), k.shape[0], 0)
    wl = synth.make_workload(cfg)
    wl.cached[0].k, wl.cached[0].v = k, v
    return wl


@pytest.mark.parametrize("splits", [1, 3])
def test_video_large_key_norm_falls_back(ws, splits):
    """A page with a few long keys (norm 40 along one axis) lifts that key
    range's logit bound above 40, so its waves fall back to the running
    maximum while the other ranges keep the bound shift; the merged result
    must match the oracle.  The queries are short along those axes, so the
    long keys' logits stay ordinary (about 1.3 sigma in log2 units) and the
    bf16 rounding of the queries does not dominate the comparison."""
    rng = np.random.default_rng(21)
    H, n_keys, n_q = 3, 64 * 9 + 5, 150
    k = synth.normal_bf16(rng, (n_keys, H, 128))
    v = synth.normal_bf16(rng, (n_keys, H, 128))
    axes = []
    for j in range(64 * 6 + 3, 64 * 6 + 9):
        row = np.zeros((H, 128), np.float32)
        row[:, (7 * j) % 128] = 40.0
        axes.append((7 * j) % 128)
        k[j] = synth.bf16_bits(row)
    wl = _raw_cond_workload("longkeys", H, k, v)
    L = Loaded(ws, wl)
    try:
        L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, splits)
        qf = rng.standard_normal((n_q, H, 128)).astype(np.float32)
        qf[:, :, axes] *= 0.25
        q = synth.bf16_bits(qf)
        pos = np.zeros((n_q, 3), np.int32)
        got = L.run("video", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        ref = L.oracle(q, pos, 0, (synth.KIND_COND,), mode=oracle.MODE_RAW)
        assert_gates(got, ref, label=f"long keys, splits={splits}")
        L.cache.set_option(ws.WS_OPT_AUDIO_KV_SPLITS, splits)
        got = L.run("audio", q[:40], pos[:40], 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        assert_gates(got, ref[:40], label=f"audio, long keys, splits={splits}")
    finally:
        L.close()


def test_video_tight_bound_shift(ws):
    """Each query's dominant RAW key is 2x its own direction, so the logit
    bound |q''| |k| is attained (about 33 in log2 units, under the fallback
    limit): the bound shift then works at its tightest."""
    rng = np.random.default_rng(22)
    H, n_keys, n_q = 2, 64 * 7 + 30, 140
    k = synth.normal_bf16(rng, (n_keys, H, 128))
    v = synth.normal_bf16(rng, (n_keys, H, 128))
    qf = rng.standard_normal((n_q, H, 128)).astype(np.float32)
    qf /= np.sqrt((qf * qf).mean(-1, keepdims=True))
    q = synth.bf16_bits(qf)
    needle = (np.arange(n_q) * 29 + 3) % n_keys
    for i, j in enumerate(needle):
        k[j] = synth.bf16_bits(2.0 * synth.bf16_to_f32(q[i]))
    wl = _raw_cond_workload("tight", H, k, v)
    L = Loaded(ws, wl)
    try:
        pos = np.zeros((n_q, 3), np.int32)
        got = L.run("video", q, pos, 0, (synth.KIND_COND,), mode=ws.WS_APPEND_RAW)
        ref = L.oracle(q, pos, 0, (synth.KIND_COND,), mode=oracle.MODE_RAW)
        assert_gates(got, ref, label="tight bound")
    finally:
        L.close()


@pytest.mark.parametrize("splits", [1, 7])
@pytest.mark.parametrize("n_q", [17, 64])
def test_audio_query_tiles(ws, splits, n_q):
    """The audio path with more than one 16-query tile: a ragged count (17:
    two tiles, the second holding one query) and the largest count a call
    takes (64: four full tiles), against the oracle."""
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        L.cache.set_option(ws.WS_OPT_AUDIO_KV_SPLITS, splits)
        st = wl.steps[0]
        reps = -(-n_q // st.q_video.shape[0])
        q = np.concatenate([st.q_video] * reps)[:n_q]
        pos = np.concatenate([st.q_video_pos] * reps)[:n_q]
        print(f"audio query tiles: splits={splits} n_q={n_q}", flush=True)
        got = L.run("audio", q, pos, wl.current_unit, ALL_KINDS)
        ref = L.oracle(q, pos, wl.current_unit, ALL_KINDS)
        assert_gates(got, ref, label=f"audio n_q={n_q} splits={splits}")
        if n_q == 64:  # one query more than a call takes: rejected before any launch
            q65 = np.concatenate([q, q[:1]])
            pos65 = np.concatenate([pos, pos[:1]])
            with pytest.raises(ws.WsError):
                L.run("audio", q65, pos65, wl.current_unit, ALL_KINDS)
    finally:
        L.close()


def test_launch_timing_ring(ws):
    """ws_cache_timing_*: one record per attention call, oldest first, with
    the attention kernel and the merge timed separately; disabled -> error."""
    wl = synth.make_workload(TINY)
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        with pytest.raises(ws.WsError):
            L.cache.timing_read()
        L.cache.timing_enable(4)
        L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, 3)
        L.run("video", st.q_video, st.q_video_pos, wl.current_unit, ALL_KINDS)
        L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, 1)
        L.run("video", st.q_video, st.q_video_pos, wl.current_unit, ALL_KINDS)
        L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        rec = L.cache.timing_read()
        assert [r["path"] for r in rec] == ["video", "video", "audio"]
        # video records carry the workgroup-group count: H * s for s forced splits
        H = wl.config.heads
        assert [r["n_splits"] for r in rec][:2] == [3 * H, H]
        assert all(r["attn_us"] > 0 for r in rec)
        assert rec[0]["merge_us"] > 0 and rec[2]["merge_us"] > 0
        assert L.cache.timing_read() == []
        for _ in range(6):  # ring of 4 keeps the last 4
            L.run("audio", st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        assert len(L.cache.timing_read()) == 4
        # append calls record their launches too (an in-place rewrite here)
        L.append(st.segments[0])
        rec = L.cache.timing_read()
        assert [r["path"] for r in rec] == ["append"] and rec[0]["attn_us"] > 0
        L.cache.timing_enable(0)
        with pytest.raises(ws.WsError):
            L.cache.timing_read()
    finally:
        L.close()


def _prepare(L, q_bits, pos, mode=None, scale=0.0, kv_segments=()):
    """One ws_step_append: the given K/V segments plus the preparation of
    q_bits; returns the prepared Q'' tensor on the device."""
    import torch
    ws = L.ws
    q = to_dev(q_bits)
    q_out = torch.full_like(q, float("nan"))
    L._keep += [q, q_out]
    mode = ws.WS_APPEND_NORM_ROPE if mode is None else mode
    items = []
    for seg in kv_segments:
        k, v = to_dev(seg.k), to_dev(seg.v)
        p = dev_i32(seg.positions) if seg.positions is not None else None
        L._keep += [k, v, p]
        if seg.mode == synth.MODE_RAW:
            items.append(dict(unit=seg.unit, kind=seg.kind, k=k, v=v, mode=ws.WS_APPEND_RAW))
        else:
            items.append(dict(unit=seg.unit, kind=seg.kind, k=k, v=v, mode=ws.WS_APPEND_NORM_ROPE,
                              positions=p, gamma=L.gk, eps=L.wl.eps))
        L.ocache.append(seg.unit, seg.kind, seg.k, seg.v,
                        oracle.MODE_RAW if seg.mode == synth.MODE_RAW else oracle.MODE_NORM_ROPE,
                        seg.positions, L.wl.gamma_k.astype(np.float64), L.wl.eps)
    qpos = dev_i32(pos)
    L._keep.append(qpos)
    L.cache.step_append(items, [dict(q=q, q_out=q_out, mode=mode, positions=qpos, gamma=L.gq,
                                     eps=L.wl.eps, scale=scale)])
    return q_out


def _run_prepared(L, path, q_out, q_unit, kinds):
    import torch
    ws = L.ws
    out = torch.full_like(q_out, float("nan"))
    fn = L.cache.unit_attention if path == "video" else L.cache.audio_attention
    fn(q_out, out, ws.mask_spec(q_unit, -(2 ** 31), kinds), ws.WS_QUERY_PREPARED)
    torch.cuda.synchronize()
    return bf16_f64(from_dev(out))


@pytest.mark.parametrize("mode", ["norm_rope", "raw"])
def test_prepared_queries_match_the_oracle_prologue(ws, mode):
    """Q'' written by ws_step_append: the oracle's Q' (RMS-norm, gamma,
    rotary, or Q as given) times softmax scale * log2(e), within one bf16 ulp
    (plus the fp32 error of a rotated pair that cancels to near zero); ragged
    query count (3 chunks of 64, the last holding 9 tokens)."""
    wl = synth.make_workload("v01", variant="seeded")
    L = Loaded(ws, wl)
    try:
        rng = np.random.default_rng(synth.SEED_BASE + 91)
        n_q = 137
        q = synth.normal_bf16(rng, (n_q, wl.config.heads, 128))
        pos = np.stack([np.full(n_q, 5), rng.integers(0, 12, n_q), rng.integers(0, 21, n_q)],
                       axis=1).astype(np.int32)
        scale = 0.07 if mode == "raw" else 0.0
        wmode = ws.WS_APPEND_RAW if mode == "raw" else ws.WS_APPEND_NORM_ROPE
        omode = oracle.MODE_RAW if mode == "raw" else oracle.MODE_NORM_ROPE
        q_out = _prepare(L, q, pos, mode=wmode, scale=scale)
        import torch
        torch.cuda.synchronize()
        got = bf16_f64(from_dev(q_out))
        s = (scale if scale > 0 else 1.0 / np.sqrt(128.0)) * np.log2(np.e)
        for h in range(wl.config.heads):
            ref = s * oracle.query_prologue(q[:, h, :], omode, pos, wl.gamma_q.astype(np.float64),
                                            wl.eps)
            err = np.abs(got[:, h] - ref)
            ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7)
            assert (err <= ulp + 2.0 ** -15).all(), (h, float(err.max()))
    finally:
        L.close()


@pytest.mark.parametrize("name", ["v02_single", "audio_c256"])
def test_prepared_step_parity(ws, name):
    """A step through ws_step_append (the current unit's K/V and the query
    preparation in one launch) and the attention on the prepared queries:
    within the gates of the oracle, and close to the NORM_ROPE path on the raw
    queries (the two differ only in the summation order of the RMS norm)."""
    wl = synth.make_workload(name)
    L = Loaded(ws, wl, step_segments=False)
    try:
        st = wl.steps[0]
        if name.startswith("audio"):
            path, qb, qp, kinds = "audio", st.q_audio, st.q_audio_pos, ALL_KINDS
        else:
            path, qb, qp, kinds = "video", st.q_video, st.q_video_pos, VIDEO_KINDS
        q_out = _prepare(L, qb, qp, kv_segments=st.segments)
        got = _run_prepared(L, path, q_out, wl.current_unit, kinds)
        ref = L.oracle(qb, qp, wl.current_unit, kinds)
        print(name, assert_gates(got, ref, label=f"{name} prepared"))
        direct = L.run(path, qb, qp, wl.current_unit, kinds)
        e = errors(got, direct)
        assert e["frob"] <= 2e-3, e
    finally:
        L.close()


@pytest.mark.parametrize("name,splits", [("audio_c256", 0), ("audio_c256", 3)])
def test_step_attention_equals_separate_calls(ws, name, splits):
    """ws_step_attention (video kernel, audio kernel, one launch merging both)
    writes exactly what ws_unit_attention and ws_audio_attention write, with
    and without video key ranges to merge; with timing on it records the two
    calls."""
    import torch
    wl = synth.make_workload(name)
    L = Loaded(ws, wl)
    try:
        if splits:
            L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, splits)
        st = wl.steps[0]
        qv, qa = to_dev(st.q_video), to_dev(st.q_audio)
        pv, pa = dev_i32(st.q_video_pos), dev_i32(st.q_audio_pos)
        vmask = ws.mask_spec(wl.current_unit, -(2 ** 31), VIDEO_KINDS)
        amask = ws.mask_spec(wl.current_unit, -(2 ** 31), ALL_KINDS)
        sep_v, sep_a = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
        L.cache.unit_attention(qv, sep_v, vmask, ws.WS_APPEND_NORM_ROPE, pv, L.gq, wl.eps)
        L.cache.audio_attention(qa, sep_a, amask, ws.WS_APPEND_NORM_ROPE, pa, L.gq, wl.eps)
        L.cache.timing_enable(4)
        step_v, step_a = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
        L.cache.step_attention(
            dict(q=qv, out=step_v, mask=vmask, mode=ws.WS_APPEND_NORM_ROPE, positions=pv,
                 gamma=L.gq, eps=wl.eps),
            dict(q=qa, out=step_a, mask=amask, mode=ws.WS_APPEND_NORM_ROPE, positions=pa,
                 gamma=L.gq, eps=wl.eps))
        torch.cuda.synchronize()
        np.testing.assert_array_equal(from_dev(step_v), from_dev(sep_v))
        np.testing.assert_array_equal(from_dev(step_a), from_dev(sep_a))
        rec = L.cache.timing_read()
        assert [r["path"] for r in rec] == ["video", "audio"]
        assert all(r["attn_us"] > 0 for r in rec) and rec[1]["merge_us"] > 0
        ref = L.oracle(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        assert_gates(bf16_f64(from_dev(step_a)), ref, label=f"{name} step audio")
    finally:
        L.close()


def test_bench_step_at_full_size(ws):
    """The step as the benchmark issues it, at full size (H = 40; video: 920
    queries over 8536 keys; audio: 4 queries over 8572 keys).  One
    ws_step_append holds the current unit's video and audio K/V and the
    preparation of both query sets, then one ws_step_attention runs on the
    prepared queries.  Every video and audio head is checked against the
    oracle.  A second step with the same inputs (an in-place rewrite) must be
    bit-identical."""
    import torch
    wl = synth.make_workload("audio_c256")
    L = Loaded(ws, wl, step_segments=False)
    try:
        st = wl.steps[0]
        items = []
        for seg in st.segments:
            k, v, p = to_dev(seg.k), to_dev(seg.v), dev_i32(seg.positions)
            L._keep += [k, v, p]
            items.append(dict(unit=seg.unit, kind=seg.kind, k=k, v=v, mode=ws.WS_APPEND_NORM_ROPE,
                              positions=p, gamma=L.gk, eps=wl.eps))
            L.ocache.append(seg.unit, seg.kind, seg.k, seg.v, oracle.MODE_NORM_ROPE, seg.positions,
                            wl.gamma_k.astype(np.float64), wl.eps)
        assert {seg.kind for seg in st.segments} == {synth.KIND_VIDEO, synth.KIND_AUDIO}
        qv, qa = to_dev(st.q_video), to_dev(st.q_audio)
        pv, pa = dev_i32(st.q_video_pos), dev_i32(st.q_audio_pos)
        L._keep += [qv, qa, pv, pa]
        vmask = ws.mask_spec(wl.current_unit, -(2 ** 31), VIDEO_KINDS)
        amask = ws.mask_spec(wl.current_unit, -(2 ** 31), ALL_KINDS)
        outs = []
        for rep in range(2):
            print(f"bench step at full size: repetition {rep}", flush=True)
            qv2, qa2 = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
            L.cache.step_append(items, [
                dict(q=qv, q_out=qv2, mode=ws.WS_APPEND_NORM_ROPE, positions=pv, gamma=L.gq,
                     eps=wl.eps, scale=0.0),
                dict(q=qa, q_out=qa2, mode=ws.WS_APPEND_NORM_ROPE, positions=pa, gamma=L.gq,
                     eps=wl.eps, scale=0.0)])
            ov, oa = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
            L.cache.step_attention(dict(q=qv2, out=ov, mask=vmask, mode=ws.WS_QUERY_PREPARED),
                                   dict(q=qa2, out=oa, mask=amask, mode=ws.WS_QUERY_PREPARED))
            torch.cuda.synchronize()
            outs.append((from_dev(ov), from_dev(oa)))
        np.testing.assert_array_equal(outs[0][0], outs[1][0])
        np.testing.assert_array_equal(outs[0][1], outs[1][1])
        refv = L.oracle(st.q_video, st.q_video_pos, wl.current_unit, VIDEO_KINDS)
        bv = L.bound(st.q_video, st.q_video_pos, wl.current_unit, VIDEO_KINDS)
        print("video", assert_gates(bf16_f64(outs[0][0]), refv, label="bench step video", bound=bv))
        refa = L.oracle(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        ba = L.bound(st.q_audio, st.q_audio_pos, wl.current_unit, ALL_KINDS)
        print("audio", assert_gates(bf16_f64(outs[0][1]), refa, label="bench step audio", bound=ba))
    finally:
        L.close()
