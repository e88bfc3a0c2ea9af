"""ws_step_attention_noalloc (split-KV partials in the library's static
device workspace) against ws_step_attention (the cache's workspaces): the
same outputs bit for bit, on two calls in a row, the second with a smaller
input, and a step whose partials exceed the static workspace is rejected
before anything is enqueued."""
import numpy as np
import pytest

from helpers import Loaded, from_dev, to_dev, dev_i32
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu

VIDEO_KINDS = (synth.KIND_COND, synth.KIND_VIDEO)
ALL_KINDS = (synth.KIND_COND, synth.KIND_VIDEO, synth.KIND_AUDIO)


def _both(ws, L, qv, pv, qa, pa, vmask, amask):
    """(regular, noalloc) outputs of one step: ((video, audio), (video, audio))."""
    import torch
    outs = []
    for fn in (L.cache.step_attention, L.cache.step_attention_noalloc):
        ov, oa = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
        fn(dict(q=qv, out=ov, mask=vmask, mode=ws.WS_APPEND_NORM_ROPE, positions=pv, gamma=L.gq,
                eps=L.wl.eps),
           dict(q=qa, out=oa, mask=amask, mode=ws.WS_APPEND_NORM_ROPE, positions=pa, gamma=L.gq,
                eps=L.wl.eps))
        torch.cuda.synchronize()
        outs.append((from_dev(ov), from_dev(oa)))
    return outs


def test_noalloc_step_matches_step_attention(ws):
    wl = synth.make_workload("audio_c256")
    L = Loaded(ws, wl)
    try:
        st = wl.steps[0]
        u = wl.current_unit
        # call 1: the full step (920 video queries over 8536 keys, 4 audio
        # queries over 8572 keys; video key ranges merged)
        qv, qa = to_dev(st.q_video), to_dev(st.q_audio)
        pv, pa = dev_i32(st.q_video_pos), dev_i32(st.q_audio_pos)
        L._keep += [qv, qa, pv, pa]
        print("noalloc: full step", flush=True)
        (rv, ra), (nv, na) = _both(ws, L, qv, pv, qa, pa, ws.mask_spec(u, -(2 ** 31), VIDEO_KINDS),
                                   ws.mask_spec(u, -(2 ** 31), ALL_KINDS))
        assert np.isfinite(synth.bf16_to_f32(nv)).all() and np.isfinite(synth.bf16_to_f32(na)).all()
        np.testing.assert_array_equal(nv, rv)
        np.testing.assert_array_equal(na, ra)
        # call 2, smaller: 300 video and 2 audio queries over a 3-unit window
        # (the workspace still holds call 1's larger partials)
        qv2, qa2 = to_dev(st.q_video[:300]), to_dev(st.q_audio[:2])
        pv2, pa2 = dev_i32(st.q_video_pos[:300]), dev_i32(st.q_audio_pos[:2])
        L._keep += [qv2, qa2, pv2, pa2]
        print("noalloc: smaller step", flush=True)
        (rv2, ra2), (nv2, na2) = _both(ws, L, qv2, pv2, qa2, pa2, ws.mask_spec(u, u - 2, VIDEO_KINDS),
                                       ws.mask_spec(u, u - 2, ALL_KINDS))
        np.testing.assert_array_equal(nv2, rv2)
        np.testing.assert_array_equal(na2, ra2)
        assert not np.array_equal(rv2, rv[:300])  # the window did change the result
        # 8 forced key ranges per head at full size need 8 x 40 x 920 rows of
        # 260 bytes (76.5 MB): more than the 32 MiB workspace
        L.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, 8)
        import torch
        ov, oa = torch.full_like(qv, float("nan")), torch.full_like(qa, float("nan"))
        call_v = dict(q=qv, out=ov, mask=ws.mask_spec(u, -(2 ** 31), VIDEO_KINDS),
                      mode=ws.WS_APPEND_NORM_ROPE, positions=pv, gamma=L.gq, eps=wl.eps)
        call_a = dict(q=qa, out=oa, mask=ws.mask_spec(u, -(2 ** 31), ALL_KINDS),
                      mode=ws.WS_APPEND_NORM_ROPE, positions=pa, gamma=L.gq, eps=wl.eps)
        with pytest.raises(ws.WsError) as e:
            L.cache.step_attention_noalloc(call_v, call_a)
        assert e.value.status == ws.WS_ERR_SHAPE and "static workspace" in str(e.value)
        torch.cuda.synchronize()
        assert np.isnan(synth.bf16_to_f32(from_dev(ov))).all()  # nothing was enqueued
        L.cache.step_attention(call_v, call_a)  # the regular entry point still takes it
        torch.cuda.synchronize()
        assert np.isfinite(synth.bf16_to_f32(from_dev(ov))).all()
    finally:
        L.close()


def test_noalloc_step_with_riding_audio_rows(ws):
    """The bench's step shape with prepared queries, where the audio rows ride
    in the video kernel and their key ranges (the shared pages' and the
    audio-token pages') also live in the static workspace: bit for bit equal
    to ws_step_attention, on a full step and then a smaller one."""
    import torch
    from test_gpu_riders import Step
    S = Step(ws, 40, (23, 40), 256, 4, 8, 71)
    try:
        u = S.unit
        qv, qa = S.queries(920), S.queries(4)
        for n_v, n_a, mn in ((920, 4, -(2 ** 31)), (300, 2, u - 2)):
            dqv, dqa = to_dev(qv[:n_v]), to_dev(qa[:n_a])
            S.keep += [dqv, dqa]
            outs = []
            for fn in (S.cache.step_attention, S.cache.step_attention_noalloc):
                ov, oa = torch.full_like(dqv, float("nan")), torch.full_like(dqa, float("nan"))
                fn(dict(q=dqv, out=ov, mask=ws.mask_spec(u, mn, VIDEO_KINDS), mode=ws.WS_QUERY_PREPARED),
                   dict(q=dqa, out=oa, mask=ws.mask_spec(u, mn, ALL_KINDS), mode=ws.WS_QUERY_PREPARED))
                torch.cuda.synchronize()
                outs.append((from_dev(ov), from_dev(oa)))
            (rv, ra), (nv, na) = outs
            print(f"noalloc with riders: {n_v} + {n_a} rows", flush=True)
            assert np.isfinite(synth.bf16_to_f32(nv)).all() and np.isfinite(synth.bf16_to_f32(na)).all()
            np.testing.assert_array_equal(nv, rv)
            np.testing.assert_array_equal(na, ra)
    finally:
        S.close()
