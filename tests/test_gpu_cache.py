"""Paged K/V cache on the GPU: ingest of the thinker's slice (stored as given),
per-step append of a generated unit (RMS-norm + rotary on K), in-place
rewrite, and read-back (Wan-Streamer v0.2, Sec. 3: ranks write incoming K/V
into their local cache; Sec. 2.1: units committed into history).  Cache
indexing must be bit-exact; normed/rotated keys within one bf16 ulp of the
fp64 oracle."""
import numpy as np
import pytest

import oracle
from helpers import Loaded, bf16_f64, dev_f32, dev_i32, from_dev, to_dev
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu


def _ulp_bf16(x):
    ax = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 7)


def test_raw_append_is_bit_exact(ws):
    wl = synth.make_workload("v01", steps=1)
    L = Loaded(ws, wl)
    try:
        cond = wl.cached[0]
        k, v = L.cache.export(0, synth.KIND_COND)
        np.testing.assert_array_equal(k, cond.k)
        np.testing.assert_array_equal(v, cond.v)
        # values of generated units are stored as given too
        for seg in wl.cached[1:] + wl.steps[0].segments:
            _, v = L.cache.export(seg.unit, seg.kind)
            np.testing.assert_array_equal(v, seg.v)
    finally:
        L.close()


@pytest.mark.parametrize("variant", ["plain", "seeded"])
def test_norm_rope_keys_within_one_ulp(ws, variant):
    wl = synth.make_workload("v01", variant=variant, steps=1)
    L = Loaded(ws, wl)
    try:
        for seg in wl.cached[1:] + wl.steps[0].segments:
            k, _ = L.cache.export(seg.unit, seg.kind)
            got = bf16_f64(k)
            for h in range(wl.config.heads):
                ref, _ = L.ocache.segment_kv(L.ocache.segments[
                    [(s.unit, s.kind) for s in L.ocache.segments].index((seg.unit, seg.kind))], h)
                # one bf16 ulp, plus the fp32 evaluation error of a rotated pair,
                # which dominates only where the rotation cancels to near zero
                err = np.abs(got[:, h] - ref)
                assert (err <= _ulp_bf16(ref) + 2.0 ** -16).all(), (seg.unit, h, float(err.max()))
    finally:
        L.close()


def test_rewrite_is_idempotent_and_isolated(ws):
    wl = synth.make_workload("v01", steps=2)
    L = Loaded(ws, wl, step=0)
    try:
        before = {(s.unit, s.kind): L.cache.export(s.unit, s.kind) for s in wl.cached}
        cur = wl.steps[0].segments[0]
        k0, v0 = L.cache.export(cur.unit, cur.kind)
        L.append(cur)  # same input again
        k1, v1 = L.cache.export(cur.unit, cur.kind)
        np.testing.assert_array_equal(k0, k1)
        np.testing.assert_array_equal(v0, v1)
        nxt = wl.steps[1].segments[0]  # the next denoising step rewrites the unit
        L.append(nxt)
        k2, v2 = L.cache.export(cur.unit, cur.kind)
        np.testing.assert_array_equal(v2, nxt.v)
        assert not np.array_equal(k2, k0)
        for key, (k, v) in before.items():
            kk, vv = L.cache.export(*key)
            np.testing.assert_array_equal(kk, k)
            np.testing.assert_array_equal(vv, v)
        assert L.cache.info().pages_free == L.cache.info().pages_total - (1 + 3 * 4)
    finally:
        L.close()


def test_errors_and_commit(ws):
    wl = synth.make_workload("v01", steps=1)
    L = Loaded(ws, wl)
    try:
        seg = wl.cached[1]
        with pytest.raises(ws.WsError) as e:
            L.append(synth.SegmentInput(seg.unit, seg.kind, seg.mode, seg.k[:10], seg.v[:10],
                                        seg.positions[:10]))
        assert e.value.status == ws.WS_ERR_SHAPE
        L.cache.commit(seg.unit)
        with pytest.raises(ws.WsError) as e:
            L.append(seg)
        assert e.value.status == ws.WS_ERR_COMMITTED
        big = synth.SegmentInput(99, synth.KIND_VIDEO, synth.MODE_RAW,
                                 np.zeros((64 * 100, wl.config.heads, 128), np.uint16),
                                 np.zeros((64 * 100, wl.config.heads, 128), np.uint16), None)
        with pytest.raises(ws.WsError) as e:
            L.append(big)
        assert e.value.status == ws.WS_ERR_OUT_OF_PAGES
        assert L.cache.check() == 0
    finally:
        L.close()


def test_position_clamp_is_flagged(ws):
    wl = synth.make_workload("v01", steps=1)
    L = Loaded(ws, wl)
    try:
        seg = wl.steps[0].segments[0]
        bad = seg.positions.copy()
        bad[3, 1] = 10 ** 6
        L.append(synth.SegmentInput(seg.unit, seg.kind, seg.mode, seg.k, seg.v, bad))
        assert L.cache.check() == 1
        assert L.cache.check() == 0
    finally:
        L.close()


# --------------------------------------------------------------------------- #
# batched append (one launch for several segments)
# --------------------------------------------------------------------------- #
def _seg_args(ws, seg, keep, gk, eps):
    k, v = to_dev(seg.k), to_dev(seg.v)
    keep += [k, v]
    if seg.mode == synth.MODE_RAW:
        return dict(unit=seg.unit, kind=seg.kind, k=k, v=v, mode=ws.WS_APPEND_RAW)
    pos = dev_i32(seg.positions)
    keep.append(pos)
    return dict(unit=seg.unit, kind=seg.kind, k=k, v=v, mode=ws.WS_APPEND_NORM_ROPE,
                positions=pos, gamma=gk, eps=eps)


def _random_segments(rng, heads, specs):
    """specs: (unit, kind, mode, n_tokens)."""
    out = []
    for unit, kind, mode, n in specs:
        k = synth.normal_bf16(rng, (n, heads, 128))
        v = synth.normal_bf16(rng, (n, heads, 128))
        pos = rng.integers(0, 200, size=(n, 3)).astype(np.int32) if mode == synth.MODE_NORM_ROPE \
            else None
        out.append(synth.SegmentInput(unit, kind, mode, k, v, pos))
    return out


def _same_caches(segs, a, b):
    for seg in segs:
        ka, va = a.export(seg.unit, seg.kind)
        kb, vb = b.export(seg.unit, seg.kind)
        np.testing.assert_array_equal(kb, ka)
        np.testing.assert_array_equal(vb, va)
    assert a.info().pages_free == b.info().pages_free


def test_append_many_matches_separate_appends(ws):
    """A step's cond + history + current segments written in batches of up to 7
    items (several launches, each with up to 4 segments) store exactly what one
    append per segment stores, and the attention over both caches agrees bit
    for bit (so the per-page key-norm table agrees too)."""
    import torch
    wl = synth.make_workload("audio_c256", steps=1)
    cfg = wl.config
    segs = list(wl.cached) + list(wl.steps[0].segments)
    max_pages = 8 + (cfg.hist + 2) * (cfg.unit_tokens // 64 + 3) + cfg.cond // 64
    keep = []
    gk = dev_f32(wl.gamma_k)
    a = ws.Cache(cfg.heads, max_pages)
    b = ws.Cache(cfg.heads, max_pages)
    try:
        for seg in segs:
            a.append(**_seg_args(ws, seg, keep, gk, wl.eps))
        for i in range(0, len(segs), 7):
            b.append_many([_seg_args(ws, s, keep, gk, wl.eps) for s in segs[i:i + 7]])
        torch.cuda.synchronize()
        _same_caches(segs, a, b)
        st = wl.steps[0]
        q, pos, gq = to_dev(st.q_video), dev_i32(st.q_video_pos), dev_f32(wl.gamma_q)
        mask = ws.mask_spec(wl.current_unit, -(2 ** 31), (synth.KIND_COND, synth.KIND_VIDEO))
        outs = []
        for c in (a, b):
            out = torch.full_like(q, float("nan"))
            c.unit_attention(q, out, mask, ws.WS_APPEND_NORM_ROPE, pos, gq, wl.eps)
            outs.append(from_dev(out))
        np.testing.assert_array_equal(outs[1], outs[0])
    finally:
        a.close()
        b.close()


@pytest.mark.parametrize("layout", ["long_segment", "many_segments"])
def test_append_many_launch_packing(ws, layout):
    """Segments split across launches: one longer than a launch's 192 pages,
    and ten one-page segments (more than a launch's eight)."""
    import torch
    rng = np.random.default_rng(synth.SEED_BASE + 77)
    R, N = synth.MODE_RAW, synth.MODE_NORM_ROPE
    V, A, C = synth.KIND_VIDEO, synth.KIND_AUDIO, synth.KIND_COND
    if layout == "long_segment":
        specs = [(1, V, N, 150), (2, C, R, 200 * 64 - 5), (3, V, N, 1), (4, A, R, 100),
                 (5, A, N, 64)]
    else:
        specs = [(u, V if u % 2 else A, N if u % 3 else R, 1 + 6 * u) for u in range(10)]
    heads = 2
    segs = _random_segments(rng, heads, specs)
    gamma = rng.uniform(0.5, 1.5, size=128).astype(np.float32)
    gk = dev_f32(gamma)
    keep = []
    a = ws.Cache(heads, 260)
    b = ws.Cache(heads, 260)
    try:
        for seg in segs:
            a.append(**_seg_args(ws, seg, keep, gk, 1e-6))
        b.append_many([_seg_args(ws, s, keep, gk, 1e-6) for s in segs])
        torch.cuda.synchronize()
        _same_caches(segs, a, b)
        # the second call rewrites every segment in place
        segs2 = _random_segments(rng, heads, specs)
        for seg in segs2:
            a.append(**_seg_args(ws, seg, keep, gk, 1e-6))
        b.append_many([_seg_args(ws, s, keep, gk, 1e-6) for s in segs2])
        torch.cuda.synchronize()
        _same_caches(segs2, a, b)
        assert a.check() == 0 and b.check() == 0
    finally:
        a.close()
        b.close()


def test_append_many_failures_take_nothing(ws):
    """A failing item leaves the cache as it was: no segment of the call is
    created, no page is taken."""
    import torch
    rng = np.random.default_rng(synth.SEED_BASE + 78)
    R, V, A = synth.MODE_RAW, synth.KIND_VIDEO, synth.KIND_AUDIO
    heads = 2
    c = ws.Cache(heads, 20)
    keep = []
    gk = dev_f32(np.ones(128, np.float32))

    def item(seg):
        return _seg_args(ws, seg, keep, gk, 1e-6)

    try:
        base = _random_segments(rng, heads, [(0, V, R, 64 * 3), (1, V, R, 64 * 2)])
        c.append_many([item(s) for s in base])
        c.commit(0)
        before = c.info()
        assert (before.pages_free, before.n_segments) == (15, 2)
        fresh, = _random_segments(rng, heads, [(2, A, R, 10)])
        big, = _random_segments(rng, heads, [(3, V, R, 64 * 16)])
        short1, = _random_segments(rng, heads, [(1, V, R, 64)])
        cases = [
            ([item(fresh), item(fresh)], ws.WS_ERR_INVALID_ARG),        # same (unit, kind)
            ([item(fresh), item(big)], ws.WS_ERR_OUT_OF_PAGES),
            ([item(fresh), item(base[0])], ws.WS_ERR_COMMITTED),
            ([item(fresh), item(short1)], ws.WS_ERR_SHAPE),
            ([], ws.WS_ERR_INVALID_ARG),
            ([item(fresh)] * 17, ws.WS_ERR_INVALID_ARG),
        ]
        for items, status in cases:
            with pytest.raises(ws.WsError) as e:
                c.append_many(items)
            assert e.value.status == status
            after = c.info()
            assert (after.pages_free, after.n_segments) == (before.pages_free, before.n_segments)
        # the cache still works: the fresh segment goes in, the uncommitted one is rewritten
        again, = _random_segments(rng, heads, [(1, V, R, 64 * 2)])
        c.append_many([item(fresh), item(again)])
        torch.cuda.synchronize()
        k, v = c.export(2, A)
        np.testing.assert_array_equal(k, fresh.k)
        np.testing.assert_array_equal(v, fresh.v)
        k, v = c.export(1, V)
        np.testing.assert_array_equal(v, again.v)
        assert c.info().pages_free == 14
        assert c.check() == 0
    finally:
        c.close()


def test_calibration_probes(ws):
    """ws_probe_mfma reports the FLOP count of its launch (workgroups x 4 waves
    x iters x 4 MFMAs x 32768) and finishes; ws_probe_read finishes on a small
    zero buffer; neither writes its sink for these inputs."""
    import torch
    sink = torch.full((4,), 7.0, dtype=torch.float32, device="cuda")
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
    h = torch.cuda.current_stream().cuda_stream
    flop = ws.ws_probe_mfma(8, 16, sink.data_ptr(), h)
    assert flop == 8 * 4 * 16 * 4 * 2.0 * 32 * 32 * 16
    assert ws.ws_probe_mfma_random(8, 16, sink.data_ptr(), h) == flop
    ws.ws_probe_read(buf.data_ptr(), buf.numel(), 64, sink.data_ptr() + 4, h)
    torch.cuda.synchronize()
    assert (sink.cpu() == 7.0).all()
    with pytest.raises(ws.WsError):
        ws.ws_probe_read(buf.data_ptr() + 8, 64, 1, sink.data_ptr(), h)
