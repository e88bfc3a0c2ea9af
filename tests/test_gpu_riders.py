"""ws_step_attention with the audio rows riding in the video kernel: the audio
queries of a step see the video queries' pages plus the units' audio tokens
(Sec. 3: both latent streams of a unit attend over the one cache), so the
video kernel computes the audio rows over the shared pages in the spare rows
of its last query tile, and the audio-token pages are walked by that tile's
waves without rows (or by the audio kernel).
Checked against the oracle, against the separate audio kernel
(WS_OPT_STEP_SEPARATE_AUDIO) and, for the video rows, bit for bit against
ws_unit_attention; steps that do not qualify take the separate kernel."""
import numpy as np
import pytest

import oracle
from helpers import assert_gates, bf16_f64, dev_f32, dev_i32, from_dev, rounding_bound, to_dev
from paper_2607_04443_amd import synth

pytestmark = pytest.mark.gpu

VIDEO = (synth.KIND_COND, synth.KIND_VIDEO)
ALL = (synth.KIND_COND, synth.KIND_VIDEO, synth.KIND_AUDIO)
LN2 = float(np.log(2.0))


def _km(kinds):
    return sum(1 << k for k in kinds)


class Step:
    """A cache with a cond slice, `units` committed units (video and audio
    K/V, NORM_ROPE keys) and the current unit's video and audio K/V, mirrored
    in an oracle cache; prepared queries (Q'' bits: the scale and log2(e)
    folded in, so the oracle takes them RAW with scale ln 2)."""

    def __init__(self, ws, H, grid, cond, audio_tokens, units, seed):
        import torch
        self.ws, self.H = ws, H
        rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + seed))
        self.rng = rng
        lu = grid[0] * grid[1]
        pages = cond // 64 + 2 + (units + 1) * (-(-lu // 64) + -(-audio_tokens // 64))
        self.cache = ws.Cache(H, pages, max_q_tokens=2048)
        self.oc = oracle.OracleCache(num_heads=H)
        g = np.ones(128, np.float32)
        dg = dev_f32(g)
        self.keep = [dg]
        ck, cv = synth.normal_bf16(rng, (cond, H, 128)), synth.normal_bf16(rng, (cond, H, 128))
        self._append(0, ws.WS_KIND_COND, oracle.KIND_COND, ck, cv, None, dg)
        for u in range(units + 1):
            for kind, okind, n, pos in ((ws.WS_KIND_VIDEO, oracle.KIND_VIDEO, lu, synth.video_positions(u, grid)),
                                        (ws.WS_KIND_AUDIO, oracle.KIND_AUDIO, audio_tokens,
                                         synth.audio_positions(u, audio_tokens))):
                k, v = synth.normal_bf16(rng, (n, H, 128)), synth.normal_bf16(rng, (n, H, 128))
                self._append(u, kind, okind, k, v, pos, dg)
            if u < units:
                self.cache.commit(u)
                self.oc.commit(u)
        self.unit = units
        self.grid = grid
        self.dg = dg
        torch.cuda.synchronize()

    def _append(self, unit, kind, okind, k, v, pos, dg):
        dk, dv = to_dev(k), to_dev(v)
        self.keep += [dk, dv]
        if pos is None:
            self.cache.append(unit, kind, dk, dv, self.ws.WS_APPEND_RAW)
            self.oc.append(unit, okind, k, v, oracle.MODE_RAW)
        else:
            dp = dev_i32(pos)
            self.keep.append(dp)
            self.cache.append(unit, kind, dk, dv, self.ws.WS_APPEND_NORM_ROPE, dp, dg, 1e-6)
            self.oc.append(unit, okind, k, v, oracle.MODE_NORM_ROPE, pos, np.ones(128), 1e-6)

    def queries(self, n):
        return synth.bf16_bits(self.rng.standard_normal((n, self.H, 128), dtype=np.float32) * 0.15)

    def video_call(self, qv, vmask, norm_rope):
        """The video call's dict: prepared rows, or raw rows with RMS-norm and
        rotary in the kernel's prologue (positions of the current unit)."""
        ws = self.ws
        dqv = to_dev(qv)
        call = dict(q=dqv, mask=ws.mask_spec(*vmask), mode=ws.WS_QUERY_PREPARED)
        if norm_rope:
            dp = dev_i32(synth.video_positions(self.unit, self.grid)[:len(qv)])
            self.keep.append(dp)
            call.update(mode=ws.WS_APPEND_NORM_ROPE, positions=dp, gamma=self.dg, eps=1e-6)
        return call

    def step(self, qv, qa, vmask, amask, separate=False, norm_rope=False):
        """ws_step_attention on the video rows (prepared, or NORM_ROPE) and
        prepared audio rows; returns the two outputs (bf16 bits) and the
        timing records."""
        import torch
        ws = self.ws
        self.cache.set_option(ws.WS_OPT_STEP_SEPARATE_AUDIO, 1 if separate else 0)
        vcall = self.video_call(qv, vmask, norm_rope)
        dqa = to_dev(qa)
        ov, oa = torch.full_like(vcall["q"], float("nan")), torch.full_like(dqa, float("nan"))
        vcall["out"] = ov
        self.cache.timing_enable(4)
        self.cache.step_attention(vcall, dict(q=dqa, out=oa, mask=ws.mask_spec(*amask), mode=ws.WS_QUERY_PREPARED))
        torch.cuda.synchronize()
        rec = self.cache.timing_read()
        self.cache.timing_enable(0)
        self.cache.set_option(ws.WS_OPT_STEP_SEPARATE_AUDIO, 0)
        return from_dev(ov), from_dev(oa), rec

    def separate_video(self, qv, vmask, norm_rope=False):
        import torch
        c = self.video_call(qv, vmask, norm_rope)
        ov = torch.full_like(c["q"], float("nan"))
        self.cache.unit_attention(c["q"], ov, c["mask"], c["mode"], c.get("positions"), c.get("gamma"),
                                  c.get("eps", 1e-6))
        torch.cuda.synchronize()
        return from_dev(ov)

    def oracle(self, q, mask, norm_rope=False):
        u, mn, kinds = mask
        if norm_rope:
            return oracle.unit_attention(self.oc, q, u, positions=synth.video_positions(u, self.grid)[:len(q)],
                                         gamma=np.ones(128), eps=1e-6, min_visible_unit=mn,
                                         kind_mask=_km(kinds))[0]
        return oracle.unit_attention(self.oc, q, u, mode=oracle.MODE_RAW, scale=LN2, min_visible_unit=mn,
                                     kind_mask=_km(kinds))[0]

    def bound(self, q, mask):
        """rounding_bound of the prepared rows' attention (oracle's RAW reading)."""
        u, mn, kinds = mask
        return rounding_bound(self.oc, q, u, mode=oracle.MODE_RAW, scale=LN2, min_visible_unit=mn,
                              kind_mask=_km(kinds))

    def close(self):
        self.cache.close()


# Where the audio-only pages are attended: by the video kernel's waves without
# rows ("video": the last query tile leaves at least two), by the audio kernel
# ("kernel": a fuller last tile, or forced by an audio split count), or
# nowhere ("none": no such pages).
@pytest.mark.parametrize("n_v,n_a,audio_tokens,splits,akinds,norm_rope,asplits,where", [
    (920, 4, 4, 0, ALL, False, 0, "video"),     # the v0.2 unit: riders in rows 920..923
    (920, 4, 4, 0, ALL, False, 2, "kernel"),    # the same, audio pages in the audio kernel
    (100, 33, 40, 0, ALL, False, 0, "video"),   # 33 riders over two waves, one shared; 40-token pages
    (920, 4, 4, 3, ALL, False, 0, "video"),     # three forced key ranges per head
    (920, 12, 40, 0, ALL, False, 0, "video"),   # 12 riders over 4 pages of 40 tokens
    (700, 64, 4, 0, ALL, False, 0, "kernel"),   # 64 riders (the audio maximum), to the tile's end
    (920, 4, 4, 0, VIDEO, False, 0, "none"),    # no audio-only pages: no audio kernel at all
    (910, 9, 4, 0, ALL, True, 0, "video"),      # NORM_ROPE video rows and prepared riders in one wave
])
def test_riders_match_oracle_and_separate_kernel(ws, n_v, n_a, audio_tokens, splits, akinds, norm_rope,
                                                 asplits, where):
    H = 8
    S = Step(ws, H, (23, 40), 256, audio_tokens, 4, 61)
    try:
        if splits:
            S.cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, splits)
        if asplits:
            S.cache.set_option(ws.WS_OPT_AUDIO_KV_SPLITS, asplits)
        u = S.unit
        vmask, amask = (u, u - 3, VIDEO), (u, u - 3, akinds)
        qv, qa = S.queries(n_v), S.queries(n_a)
        if norm_rope:
            qv = synth.normal_bf16(S.rng, (n_v, H, 128))
        print(f"riders: n_v={n_v} n_a={n_a} audio_tokens={audio_tokens} splits={splits} "
              f"norm_rope={norm_rope} asplits={asplits} where={where}", flush=True)
        fv, fa, rec = S.step(qv, qa, vmask, amask, norm_rope=norm_rope)
        assert [r["path"] for r in rec] == ["video", "audio_riders"], rec
        # the audio kernel's range count: 0 when it was not launched
        if where == "kernel":
            assert rec[1]["n_splits"] >= 1, rec
        else:
            assert rec[1]["n_splits"] == 0, rec
        sv, sa, rec2 = S.step(qv, qa, vmask, amask, separate=True, norm_rope=norm_rope)
        assert [r["path"] for r in rec2] == ["video", "audio"], rec2
        np.testing.assert_array_equal(fv, sv)
        np.testing.assert_array_equal(fv, S.separate_video(qv, vmask, norm_rope))
        refa = S.oracle(qa, amask)
        ba = S.bound(qa, amask)
        print("riders audio", assert_gates(bf16_f64(fa), refa, label="audio rows in the video kernel", bound=ba))
        print("separate audio", assert_gates(bf16_f64(sa), refa, label="separate audio kernel", bound=ba))
        print("video", assert_gates(bf16_f64(fv), S.oracle(qv, vmask, norm_rope), label="video rows"))
        # a repeat is bit-identical (every partial row the merge reads is rewritten)
        fv2, fa2, _ = S.step(qv, qa, vmask, amask, norm_rope=norm_rope)
        np.testing.assert_array_equal(fa, fa2)
        np.testing.assert_array_equal(fv, fv2)
    finally:
        S.close()


def test_steps_that_do_not_ride(ws):
    """No spare rows (256 video rows), an audio window that hides a page the
    video call sees, and audio rows that are not prepared: the separate audio
    kernel, with correct outputs."""
    H = 4
    S = Step(ws, H, (5, 7), 64, 4, 4, 62)
    try:
        u = S.unit
        qa = S.queries(4)
        cases = [(S.queries(256), (u, u - 3, VIDEO), (u, u - 3, ALL)),
                 (S.queries(35), (u, u - 3, VIDEO), (u, u - 1, ALL))]
        for qv, vmask, amask in cases:
            fv, fa, rec = S.step(qv, qa, vmask, amask)
            assert [r["path"] for r in rec] == ["video", "audio"], (len(qv), vmask, amask, rec)
            print(assert_gates(bf16_f64(fa), S.oracle(qa, amask), label=f"no riders {len(qv)} {amask}"))
            print(assert_gates(bf16_f64(fv), S.oracle(qv, vmask), label=f"no riders video {len(qv)}"))
        # RAW audio rows (the kernel folds the scale in) do not ride either
        import torch
        ws_ = S.ws
        qv = S.queries(35)
        dqv, dqa = to_dev(qv), to_dev(qa)
        ov, oa = torch.full_like(dqv, float("nan")), torch.full_like(dqa, float("nan"))
        S.cache.timing_enable(4)
        S.cache.step_attention(dict(q=dqv, out=ov, mask=ws_.mask_spec(u, u - 3, VIDEO), mode=ws_.WS_QUERY_PREPARED),
                               dict(q=dqa, out=oa, mask=ws_.mask_spec(u, u - 3, ALL), mode=ws_.WS_APPEND_RAW))
        torch.cuda.synchronize()
        rec = S.cache.timing_read()
        assert [r["path"] for r in rec] == ["video", "audio"], rec
        ref = oracle.unit_attention(S.oc, qa, u, mode=oracle.MODE_RAW, min_visible_unit=u - 3,
                                    kind_mask=_km(ALL))[0]
        print(assert_gates(bf16_f64(from_dev(oa)), ref, label="RAW audio rows"))
    finally:
        S.close()
