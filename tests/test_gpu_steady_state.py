"""The streaming loop at steady state on the GPU: every unit brings a fresh
conditioning slice (rewritten in place of the previous one), the unit's video
and audio K/V (appended with RMS-norm and rotary) and its prepared queries,
one ws_step_attention, then the unit is committed to history and the unit
that left the window is evicted (Wan-Streamer v0.2, Sec. 2.1: latents
committed into history after each unit; Sec. 3: the performer updates its
cache every unit).  The pool is sized so that every new unit must take the
pages the last eviction freed.  The oracle's logical cache applies the same
appends, commits and evictions; outputs are compared at several units."""
import numpy as np
import pytest

import oracle
from helpers import assert_gates, bf16_f64, dev_f32, dev_i32, from_dev, to_dev
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu

H, GRID, COND, AUDIO = 40, (23, 40), 256, 4
LU = GRID[0] * GRID[1]
WINDOW = 2          # history units visible besides the current one
UNITS = 13          # 11 units past the window
CHECK_AT = (3, 8, UNITS - 1)
VIDEO_KINDS = (synth.KIND_COND, synth.KIND_VIDEO)
ALL_KINDS = (synth.KIND_COND, synth.KIND_VIDEO, synth.KIND_AUDIO)


def test_window_eviction_reuses_pages_and_matches_oracle(ws):
    import torch
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 41))
    pages_per_unit = -(-LU // 64) + -(-AUDIO // 64)   # 15 video + 1 audio
    max_pages = COND // 64 + (WINDOW + 1) * pages_per_unit
    cache = ws.Cache(H, max_pages, max_q_tokens=1024)
    oc = oracle.OracleCache(num_heads=H)
    gamma = np.ones(128, np.float32)
    g_dev = dev_f32(gamma)
    eps = 1e-6
    keep = []
    freed = set()   # pages of evicted units, not yet taken again
    pages_of = {}
    checked = 0
    try:
        for u in range(UNITS):
            ck, cv = synth.normal_bf16(rng, (COND, H, 128)), synth.normal_bf16(rng, (COND, H, 128))
            kv = synth.normal_bf16(rng, (LU, H, 128))
            vv = synth.normal_bf16(rng, (LU, H, 128))
            ka = synth.normal_bf16(rng, (AUDIO, H, 128))
            va = synth.normal_bf16(rng, (AUDIO, H, 128))
            qv = synth.normal_bf16(rng, (LU, H, 128))
            qa = synth.normal_bf16(rng, (AUDIO, H, 128))
            vpos, apos = synth.video_positions(u, GRID), synth.audio_positions(u, AUDIO)
            d = dict(ck=to_dev(ck), cv=to_dev(cv), kv=to_dev(kv), vv=to_dev(vv), ka=to_dev(ka),
                     va=to_dev(va), qv=to_dev(qv), qa=to_dev(qa), vpos=dev_i32(vpos),
                     apos=dev_i32(apos))
            q_v, q_a = torch.full_like(d["qv"], float("nan")), torch.full_like(d["qa"], float("nan"))
            out_v, out_a = torch.full_like(d["qv"], float("nan")), torch.full_like(d["qa"], float("nan"))
            keep.append((d, q_v, q_a, out_v, out_a))
            print(f"steady state: unit {u}", flush=True)
            cache.step_append([
                dict(unit=0, kind=ws.WS_KIND_COND, k=d["ck"], v=d["cv"], mode=ws.WS_APPEND_RAW),
                dict(unit=u, kind=ws.WS_KIND_VIDEO, k=d["kv"], v=d["vv"], mode=ws.WS_APPEND_NORM_ROPE,
                     positions=d["vpos"], gamma=g_dev, eps=eps),
                dict(unit=u, kind=ws.WS_KIND_AUDIO, k=d["ka"], v=d["va"], mode=ws.WS_APPEND_NORM_ROPE,
                     positions=d["apos"], gamma=g_dev, eps=eps)],
                [dict(q=d["qv"], q_out=q_v, positions=d["vpos"], gamma=g_dev, eps=eps),
                 dict(q=d["qa"], q_out=q_a, positions=d["apos"], gamma=g_dev, eps=eps)])
            oc.append(0, oracle.KIND_COND, ck, cv, oracle.MODE_RAW)
            oc.append(u, oracle.KIND_VIDEO, kv, vv, oracle.MODE_NORM_ROPE, vpos, gamma, eps)
            oc.append(u, oracle.KIND_AUDIO, ka, va, oracle.MODE_NORM_ROPE, apos, gamma, eps)

            # page bookkeeping: once the window is full, the unit lives exactly
            # in the pages the previous eviction freed
            mine = set(cache.pages(u, ws.WS_KIND_VIDEO)) | set(cache.pages(u, ws.WS_KIND_AUDIO))
            assert len(mine) == pages_per_unit
            pages_of[u] = mine
            if u > WINDOW:
                assert mine == freed, (u, sorted(mine), sorted(freed))
                assert cache.info().pages_free == 0
            freed -= mine

            vmask = ws.mask_spec(u, u - WINDOW, VIDEO_KINDS)
            amask = ws.mask_spec(u, u - WINDOW, ALL_KINDS)
            cache.step_attention(dict(q=q_v, out=out_v, mask=vmask, mode=ws.WS_QUERY_PREPARED),
                                 dict(q=q_a, out=out_a, mask=amask, mode=ws.WS_QUERY_PREPARED))
            if u in CHECK_AT:
                torch.cuda.synchronize()
                refv, _ = oracle.unit_attention(oc, qv, u, positions=vpos, gamma=gamma, eps=eps,
                                                min_visible_unit=u - WINDOW, kind_mask=0b011)
                refa, _ = oracle.unit_attention(oc, qa, u, positions=apos, gamma=gamma, eps=eps,
                                                min_visible_unit=u - WINDOW, kind_mask=0b111)
                print(f"unit {u} video", assert_gates(bf16_f64(from_dev(out_v)), refv,
                                                      label=f"steady state video, unit {u}"))
                print(f"unit {u} audio", assert_gates(bf16_f64(from_dev(out_a)), refa,
                                                      label=f"steady state audio, unit {u}"))
                checked += 1
            cache.commit(u)
            oc.commit(u)
            cache.evict_before(u - WINDOW + 1)
            oc.evict_before(u - WINDOW + 1)
            if u - WINDOW >= 0:
                freed |= pages_of.pop(u - WINDOW)
        assert checked == len(CHECK_AT)
        # what is left: the last slice and the window's units, stored as given
        torch.cuda.synchronize()
        present = sorted({(s.unit, s.kind) for s in oc.segments})
        assert present == [(0, 0)] + [(u, k) for u in range(UNITS - WINDOW, UNITS) for k in (1, 2)]
        for s in oc.segments:
            k_got, v_got = cache.export(s.unit, s.kind)
            np.testing.assert_array_equal(v_got, s.v_bits)
            if s.kind == oracle.KIND_COND:
                np.testing.assert_array_equal(k_got, s.k_bits)
        for u in range(UNITS - WINDOW):
            with pytest.raises(ws.WsError):
                cache.pages(u, ws.WS_KIND_VIDEO)
        assert cache.check() == 0
    finally:
        cache.close()
