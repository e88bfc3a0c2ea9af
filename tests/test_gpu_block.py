"""The attention sub-block of one performer layer (ws_block_step): QKV
projection (hipBLASLt), the unit's K/V append with the query preparation,
the video and audio attention, and the output projection (Wan-Streamer v0.2,
Sec. 3), against the oracle's block_step on the same bf16 inputs and random
weights.  The projections round Q, K, V to bf16 on both sides; the oracle
keeps O and Y in float64."""
import numpy as np
import pytest

import oracle
from helpers import assert_gates, bf16_f64, dev_f32, dev_i32, from_dev, to_dev
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu

H, GRID, COND, AUDIO, HIST = 4, (5, 7), 10, 3, 2
LU = GRID[0] * GRID[1]
HID = H * 128


def _setup(ws, seed):
    import torch
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + seed))
    cache = ws.Cache(H, 64, max_q_tokens=128)
    oc = oracle.OracleCache(num_heads=H)
    g = np.ones(128, np.float32)
    gd = dev_f32(g)
    keep = [gd]
    ck, cv = synth.normal_bf16(rng, (COND, H, 128)), synth.normal_bf16(rng, (COND, H, 128))
    keep += [to_dev(ck), to_dev(cv)]
    cache.append(0, ws.WS_KIND_COND, keep[-2], keep[-1], ws.WS_APPEND_RAW)
    oc.append(0, oracle.KIND_COND, ck, cv, oracle.MODE_RAW)
    for u in range(HIST):
        for kind, n, pos in ((ws.WS_KIND_VIDEO, LU, synth.video_positions(u, GRID)),
                             (ws.WS_KIND_AUDIO, AUDIO, synth.audio_positions(u, AUDIO))):
            k, v = synth.normal_bf16(rng, (n, H, 128)), synth.normal_bf16(rng, (n, H, 128))
            dk, dv, dp = to_dev(k), to_dev(v), dev_i32(pos)
            keep += [dk, dv, dp]
            cache.append(u, kind, dk, dv, ws.WS_APPEND_NORM_ROPE, dp, gd, 1e-6)
            oc.append(u, kind, k, v, oracle.MODE_NORM_ROPE, pos, g, 1e-6)
        cache.commit(u)
        oc.commit(u)
    w_qkv = synth.bf16_bits(rng.standard_normal((HID, 3 * HID)).astype(np.float32) / np.sqrt(HID))
    w_out = synth.bf16_bits(rng.standard_normal((HID, HID)).astype(np.float32) / np.sqrt(HID))
    dwq, dwo = to_dev(w_qkv), to_dev(w_out)
    keep += [dwq, dwo]
    block = ws.Block(cache, dwq, dwo, max_rows=128)
    torch.cuda.synchronize()
    return rng, cache, oc, block, w_qkv, w_out, gd, keep


def _step(ws, L, unit, x, n_video, window=None):
    import torch
    rng, cache, oc, block, w_qkv, w_out, gd, keep = L
    n_audio = x.shape[0] - n_video
    vpos, apos = synth.video_positions(unit, GRID)[:n_video], synth.audio_positions(unit, n_audio)
    dx = to_dev(x)
    dvp, dap = dev_i32(vpos), dev_i32(apos) if n_audio else None
    y = torch.full_like(dx, float("nan"))
    o = torch.full_like(dx, float("nan"))
    keep += [dx, dvp, dap, y, o]
    mn = -(2 ** 31) if window is None else unit - window
    block.step(dx, n_video, unit, dvp, dap, gd, gd, y,
               ws.mask_spec(unit, mn, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO)),
               ws.mask_spec(unit, mn, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO)),
               attn_out=o)
    torch.cuda.synchronize()
    g = np.ones(128)
    ry, ro = oracle.block_step(oc, x, n_video, w_qkv, w_out, unit, video_positions=vpos,
                               audio_positions=apos, gamma_q=g, gamma_k=g, eps=1e-6,
                               video_mask=(mn, 0b011), audio_mask=(mn, 0b111))
    return (bf16_f64(from_dev(y)), bf16_f64(from_dev(o)).reshape(-1, H, 128)), (ry, ro)


def test_block_step_matches_oracle_and_rewrites(ws):
    L = _setup(ws, 61)
    try:
        rng = L[0]
        # first step of unit 2 (fresh pages), then a second denoising step (rewrite)
        for step in range(2):
            x = synth.normal_bf16(rng, (LU + AUDIO, HID))
            (y, o), (ry, ro) = _step(ws, L, HIST, x, LU)
            print(f"step {step}: attention", assert_gates(o, ro, label=f"block attention {step}"))
            print(f"step {step}: output", assert_gates(y, ry, label=f"block output {step}"))
        # a video-only step of the next unit with a one-unit window
        L[1].commit(HIST)
        L[2].commit(HIST)
        x = synth.normal_bf16(rng, (LU, HID))
        (y, o), (ry, ro) = _step(ws, L, HIST + 1, x, LU, window=1)
        assert_gates(o, ro, label="video-only attention")
        assert_gates(y, ry, label="video-only output")
    finally:
        L[3].close()
        L[1].close()


def test_block_step_rejects_before_enqueue(ws):
    import torch
    L = _setup(ws, 62)
    rng, cache, oc, block, w_qkv, w_out, gd, keep = L
    try:
        x = to_dev(synth.normal_bf16(rng, (LU + AUDIO, HID)))
        y = torch.full_like(x, float("nan"))
        vp, ap = dev_i32(synth.video_positions(1, GRID)), dev_i32(synth.audio_positions(1, AUDIO))
        vm = ws.mask_spec(1, -(2 ** 31), (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))
        am = ws.mask_spec(1, -(2 ** 31), (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO))
        with pytest.raises(ws.WsError) as e:   # unit 1 is committed history
            block.step(x, LU, 1, vp, ap, gd, gd, y, vm, am)
        assert e.value.status == ws.WS_ERR_COMMITTED
        with pytest.raises(ws.WsError) as e:   # a rewrite must keep the token count
            block.step(x[:LU + 1], LU - 1, HIST, vp, ap, gd, gd, y, vm, am)
            block.step(x, LU, HIST, vp, ap, gd, gd, y, vm, am)
        assert e.value.status == ws.WS_ERR_SHAPE
        torch.cuda.synchronize()
        free = cache.info().pages_free
        with pytest.raises(ws.WsError) as e:   # more rows than the block takes
            block.step(torch.zeros((200, HID), dtype=torch.bfloat16, device="cuda"), 190, 7, vp, ap, gd,
                       gd, torch.zeros((200, HID), dtype=torch.bfloat16, device="cuda"), vm, am)
        assert e.value.status == ws.WS_ERR_SHAPE
        assert cache.info().pages_free == free
    finally:
        block.close()
        cache.close()


def test_block_step_at_bench_size(ws):
    """The sub-block the bench times: 40 heads (hidden 5120), a 924-row step
    (920 video + 4 audio tokens) over a 256-token slice and 8 history units,
    with the projections' algorithms picked by timing at this row count.
    Attention output and projected output, all heads, against the oracle."""
    import torch
    H_, grid, cond, audio, hist = 40, (23, 40), 256, 4, 8
    hid = H_ * 128
    lu = grid[0] * grid[1]
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 63))
    cache = ws.Cache(H_, 4 + (hist + 2) * 16 + 8, max_q_tokens=1024)
    oc = oracle.OracleCache(num_heads=H_)
    g = np.ones(128, np.float32)
    gd = dev_f32(g)
    keep = [gd]
    block = None
    try:
        ck, cv = synth.normal_bf16(rng, (cond, H_, 128)), synth.normal_bf16(rng, (cond, H_, 128))
        keep += [to_dev(ck), to_dev(cv)]
        cache.append(0, ws.WS_KIND_COND, keep[-2], keep[-1], ws.WS_APPEND_RAW)
        oc.append(0, oracle.KIND_COND, ck, cv, oracle.MODE_RAW)
        for u in range(hist):
            for kind, n, pos in ((ws.WS_KIND_VIDEO, lu, synth.video_positions(u, grid)),
                                 (ws.WS_KIND_AUDIO, audio, synth.audio_positions(u, audio))):
                k, v = synth.normal_bf16(rng, (n, H_, 128)), synth.normal_bf16(rng, (n, H_, 128))
                dk, dv, dp = to_dev(k), to_dev(v), dev_i32(pos)
                keep += [dk, dv, dp]
                cache.append(u, kind, dk, dv, ws.WS_APPEND_NORM_ROPE, dp, gd, 1e-6)
                oc.append(u, kind, k, v, oracle.MODE_NORM_ROPE, pos, g, 1e-6)
            cache.commit(u)
            oc.commit(u)
        # N(0, 1) / 64 (about 1 / sqrt(hidden); a power of two keeps the draw's bf16 rounding)
        w_qkv = synth.bf16_bits(rng.standard_normal((hid, 3 * hid), dtype=np.float32) * np.float32(2 ** -6))
        w_out = synth.bf16_bits(rng.standard_normal((hid, hid), dtype=np.float32) * np.float32(2 ** -6))
        dwq, dwo = to_dev(w_qkv), to_dev(w_out)
        keep += [dwq, dwo]
        block = ws.Block(cache, dwq, dwo, max_rows=lu + audio)
        x = synth.normal_bf16(rng, (lu + audio, hid))
        vpos, apos = synth.video_positions(hist, grid), synth.audio_positions(hist, audio)
        dx, dvp, dap = to_dev(x), dev_i32(vpos), dev_i32(apos)
        y = torch.full_like(dx, float("nan"))
        o = torch.full_like(dx, float("nan"))
        keep += [dx, dvp, dap, y, o]
        block.step(dx, lu, hist, dvp, dap, gd, gd, y,
                   ws.mask_spec(hist, -(2 ** 31), (ws.WS_KIND_COND, ws.WS_KIND_VIDEO)),
                   ws.mask_spec(hist, -(2 ** 31), (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO)),
                   attn_out=o)
        torch.cuda.synchronize()
        ry, ro = oracle.block_step(oc, x, lu, w_qkv, w_out, hist, video_positions=vpos, audio_positions=apos,
                                   gamma_q=np.ones(128), gamma_k=np.ones(128), eps=1e-6,
                                   video_mask=(-(2 ** 31), 0b011), audio_mask=(-(2 ** 31), 0b111))
        got_o = bf16_f64(from_dev(o)).reshape(-1, H_, 128)
        print("attention", assert_gates(got_o, ro, label="bench-size block attention"))
        print("output", assert_gates(bf16_f64(from_dev(y)), ry, label="bench-size block output"))
    finally:
        if block is not None:
            block.close()
        cache.close()
