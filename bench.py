#!/usr/bin/env python3
"""Benchmark: one streaming unit of the Wan-Streamer v0.2 performer's attention
path at 640x368 on one MI355X.

A step is one pass of the whole hot path for the next 160 ms unit u, at steady
state with an 8-unit history window (Wan-Streamer v0.2, Sec. 3 unit schedule;
Sec. 2.1 history commit):
  1. the thinker's 256-token conditioning slice is written into the cache
     (stored as given, in place of the previous unit's slice);
  2. unit u's 920 video and 4 audio K/V are appended (RMS-norm + rotary on K)
     and its 920 video and 4 audio queries prepared (RMS-norm + rotary, the
     softmax scale folded in); steps 1 and 2 are one kernel launch
     (ws_step_append);
  3. video attention: the 920 prepared queries over 256 + 9 x 920 = 8536
     keys;
  4. audio attention: 4 queries over cond + 9 x (920 + 4) = 8572 keys;
     steps 3 and 4 are one ws_step_attention call: the video kernel, which
     also computes the 4 audio rows over the pages both calls see (the rows
     ride in the spare rows of its last query tile), the audio kernel over
     the 9 audio-token pages only, and one launch merging both calls' key
     ranges;
  5. unit u is committed to history and the unit that left the window evicted.
All inputs are synthetic N(0,1) bf16 resident in HBM; H = 40 heads of 128.

Prints one JSON line.  `value` is attention TFLOP/s over the whole step
(video + audio FLOP / step time), from `steps` steps timed with nothing
recorded in between, after `settle` untimed steps (the clocks' ramp from
idle, reported block by block in settle_us_per_step) and `warmup` untimed
steps: a performer runs the step back to back for as long as it streams.  A second pass of `steps` steps issues the two
attentions as separate calls (ws_unit_attention, ws_audio_attention, each
with its own merge) and records events around each component (the
per-component fields) and the library's launch timing (ws_cache_timing_*):
`roofline` is for the video attention kernel (the dominant one), its FLOP
per launch over its average launch time from HIP events recorded on the
calls' stream around the kernel itself.
`video_configs` times the video kernel alone on the v0.1, v0.2 single-unit
and v0.2 8-unit-history configurations (median of the library's per-launch
kernel times).
`v01_step` is the step at the v0.1 stream shape (192x336, 12 heads,
252-token units, 820 keys), timed the same way.
`us_per_unit_separate_audio` is the contract step with the audio call in
its own kernel over all of its pages (WS_OPT_STEP_SEPARATE_AUDIO).
`cpu_baseline` times the fp64 CPU oracle on a bounded sample.
"""
import argparse
import json
import subprocess
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

H, D, GRID, COND, HIST, AUDIO = 40, 128, (23, 40), 256, 8, 4
LU = GRID[0] * GRID[1]
PEAK_BF16_TFLOPS = 256 * 4096 * 2.4e9 / 1e12   # 2516.6 dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def video_flop(lq, lk):
    return 4.0 * H * lq * lk * D


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    # From idle the GPU's clocks take some 30 ms of this load to settle: the
    # first 25 steps run about 15% slower than step 150 on (settle_us_per_step
    # in the output shows the ramp). The settle steps run before the warm-up.
    ap.add_argument("--settle", type=int, default=200,
                    help="untimed steps before the warm-up steps, in blocks of 25 whose average step "
                         "times are reported as settle_us_per_step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--video-splits", type=int, default=0)
    ap.add_argument("--audio-splits", type=int, default=0)
    ap.add_argument("--cold-audio-reps", type=int, default=20)
    ap.add_argument("--long-reps", type=int, default=5)
    ap.add_argument("--no-peak-probes", dest="peak_probes", action="store_false",
                    help="skip the calibration probes (measured MFMA and HBM read ceilings)")
    ap.add_argument("--pmc-driver", nargs="?", const="step", choices=("step", "long"),
                    help="the program rocprofv3 --pmc runs, untimed: 'step' (default) runs three "
                         "steps, then the video and audio attention three times each as separate "
                         "calls; 'long' runs the video attention of the long-history workload "
                         "(30616 keys) three times; both end with three 256 MiB device copies")
    ap.add_argument("--cpu-v01-point", action="store_true",
                    help="time the fp64 oracle on the whole v0.1-scale workload (CPU only) and print "
                         "one JSON line")
    ap.add_argument("--mfma-summary", metavar="DIR",
                    help="summarise one rocprofv3 --pmc -f csv run of --pmc-driver with the MFMA and "
                         "instruction counters (GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES, "
                         "SQ_INSTS_VALU_MFMA_MOPS_BF16, ...) for unit_attn_kernel as markdown")
    ap.add_argument("--trace-summary", metavar="CSV",
                    help="summarise the kernel_trace.csv of one rocprofv3 --kernel-trace -f csv run of "
                         "the default bench as markdown: durations per kernel and grid, and the "
                         "contract steps' append, video and merge medians")
    ap.add_argument("--pmc-summary", nargs="+", metavar="DIR",
                    help="summarise rocprofv3 --pmc -f csv runs of --pmc-driver as markdown: "
                         "FETCH_SIZE and WRITE_SIZE of 'step', optionally followed by FETCH_SIZE "
                         "and WRITE_SIZE of 'long'")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_v01_point():
    """The fp64 oracle on the whole 192x336-scale workload (12 heads, 252
    queries over 64 + 3 x 252 = 820 keys, with its Q/K RMS-norm and rotary),
    run in this process; called in a child process with one OpenMP thread."""
    import numpy as np
    import oracle
    from paper_2607_04443_amd import synth
    wl = synth.make_workload("v01")
    oc = oracle.OracleCache(num_heads=wl.config.heads)
    for seg in wl.cached + wl.steps[0].segments:
        oc.append(seg.unit, seg.kind, seg.k, seg.v, seg.mode, seg.positions,
                  wl.gamma_k.astype(np.float64), wl.eps)
    st = wl.steps[0]
    t0 = time.perf_counter()
    oracle.unit_attention(oc, st.q_video, wl.current_unit, positions=st.q_video_pos,
                          gamma=wl.gamma_q.astype(np.float64), eps=wl.eps)
    dt = time.perf_counter() - t0
    cfg = wl.config
    lk = cfg.video_keys
    flop = 4.0 * cfg.heads * cfg.unit_tokens * lk * D
    return {"threads": oracle.num_threads(), "seconds": dt, "tflops": flop / dt / 1e12,
            "workload": f"v0.1 scale: {cfg.heads} heads, {cfg.unit_tokens} queries x {lk} keys, fp64"}


def cpu_baseline(budget_s=12.0):
    """The fp64 oracle on whole heads of the video attention, as many as fit in
    about budget_s seconds (a bounded sample), scaled to TFLOP/s."""
    import numpy as np
    import oracle
    from paper_2607_04443_amd import synth
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 2))
    lk = COND + (HIST + 1) * LU
    pos_q = synth.video_positions(HIST, GRID)
    pos_k = np.concatenate([synth.video_positions(u, GRID) for u in range(HIST + 1)])
    heads, dt = 0, 0.0
    while heads < H and dt < budget_s:
        q = synth.normal_bf16(rng, (LU, D))
        k = synth.normal_bf16(rng, (lk, D))
        v = synth.normal_bf16(rng, (lk, D))
        t0 = time.perf_counter()
        qq = oracle.rope(oracle.rmsnorm(oracle.bf16_decode(q), np.ones(D), 1e-6), pos_q)
        kk = oracle.bf16_decode(k)
        kk[COND:] = oracle.rope(oracle.rmsnorm(kk[COND:], np.ones(D), 1e-6), pos_k)
        oracle.attention(qq, kk, oracle.bf16_decode(v), 1.0 / np.sqrt(D))
        dt += time.perf_counter() - t0
        heads += 1
    flop = video_flop(LU, lk) / H * heads
    single = None
    try:
        env = dict(os.environ, OMP_NUM_THREADS="1")
        r = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-v01-point"], env=env,
                           capture_output=True, text=True, timeout=300)
        single = json.loads(r.stdout.strip().splitlines()[-1]) if r.returncode == 0 else None
    except (subprocess.SubprocessError, ValueError, IndexError):
        single = None
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{heads} of {H} heads of the video attention ({LU} queries x {lk} keys, "
                      f"fp64, with those heads' Q/K RMS-norm and rotary): {dt:.1f} s",
            "single_thread_v01": single}


LONG_HIST = 32


def long_setup(ws, sets, gamma, eps, dev):
    """The long-history cache: a cond slice and 32 committed history units
    (256 + 33 x 920 = 30616 keys visible to unit 32), built from the two
    resident input sets (values do not change the timing).  Returns the
    cache and a function that issues one denoising step of unit 32: an
    in-place rewrite of its K/V (append with RMS-norm + rotary, and the query
    preparation, in one launch) and the video attention."""
    import torch
    from paper_2607_04443_amd import synth
    hist_l = LONG_HIST
    cache = ws.Cache(H, 4 + (hist_l + 2) * 16 + 8, max_q_tokens=1024)
    pos = [torch.from_numpy(synth.video_positions(u, GRID)).to(dev) for u in range(hist_l + 1)]
    s0 = sets[0]
    cache.append(0, ws.WS_KIND_COND, s0["ck"], s0["cv"], ws.WS_APPEND_RAW)
    for u in range(hist_l):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, pos[u], gamma, eps)
        cache.commit(u)
    out = torch.empty((LU, H, D), dtype=torch.bfloat16, device=dev)
    q_v = torch.empty((LU, H, D), dtype=torch.bfloat16, device=dev)
    mask = ws.mask_spec(hist_l, 0, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))

    def one_step(step, attention=True):
        s = sets[step % 2]
        cache.step_append(
            [dict(unit=hist_l, kind=ws.WS_KIND_VIDEO, k=s["k"], v=s["v"],
                  mode=ws.WS_APPEND_NORM_ROPE, positions=pos[hist_l], gamma=gamma, eps=eps)],
            [dict(q=s["q"], q_out=q_v, positions=pos[hist_l], gamma=gamma, eps=eps)])
        if attention:
            cache.unit_attention(q_v, out, mask, ws.WS_QUERY_PREPARED)

    return cache, one_step


def long_history(args, ws, sets, gamma, eps, stream, dev):
    """Long-history stress (long_setup): 4 denoising steps issued
    back-to-back on one stream, timed with events around the 4 steps; the
    median of `long_reps` repetitions."""
    import torch
    cache, one_step = long_setup(ws, sets, gamma, eps, dev)

    def four_steps():
        for step in range(4):
            one_step(step)

    four_steps()
    torch.cuda.synchronize()
    times = []
    for _ in range(args.long_reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        four_steps()
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b) * 1e3)
    cache.close()
    times.sort()
    med = times[len(times) // 2]
    lk = COND + (LONG_HIST + 1) * LU
    return {"keys": lk, "us_4_steps": med, "us_per_step": med / 4,
            "tflops": 4 * video_flop(LU, lk) / (med * 1e-6) / 1e12}


def cold_audio(args, ws, sets, vpos, apos, gamma, eps, stream, dev, cond):
    """ws_audio_attention with cold caches: a cache of `cond` conditioning
    tokens, 8 committed history units and the current unit (920 video + 4
    audio tokens each), the 4 prepared audio queries over all of it.  Between
    repetitions a 1 GiB buffer is read (a reduction), which evicts the 256 MB
    cache with clean lines, so the timed call neither hits that cache nor pays
    for writing back a dirty scrub; events around the audio call only."""
    import numpy as np
    import torch
    from paper_2607_04443_amd import synth
    cache = ws.Cache(H, cond // 64 + 2 + (HIST + 1) * 16, max_q_tokens=1024)
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 3))
    ck = torch.from_numpy(synth.normal_bf16(rng, (cond, H, D)).view(np.int16)).view(torch.bfloat16).to(dev)
    cv = torch.from_numpy(synth.normal_bf16(rng, (cond, H, D)).view(np.int16)).view(torch.bfloat16).to(dev)
    cache.append(0, ws.WS_KIND_COND, ck, cv, ws.WS_APPEND_RAW)
    for u in range(HIST + 1):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, vpos[u], gamma, eps)
        cache.append(u, ws.WS_KIND_AUDIO, s["ka"], s["va"], ws.WS_APPEND_NORM_ROPE, apos[u], gamma, eps)
        if u < HIST:
            cache.commit(u)
    q_a = torch.empty((AUDIO, H, D), dtype=torch.bfloat16, device=dev)
    out_a = torch.empty((AUDIO, H, D), dtype=torch.bfloat16, device=dev)
    cache.step_append([], [dict(q=sets[0]["qa"], q_out=q_a, positions=apos[HIST], gamma=gamma, eps=eps)])
    amask = ws.mask_spec(HIST, 0, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO))
    scrub = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    scrub_sum = torch.empty((), dtype=torch.float32, device=dev)
    times = []
    for _ in range(args.cold_audio_reps):
        torch.sum(scrub, dim=0, out=scrub_sum)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        cache.audio_attention(q_a, out_a, amask, ws.WS_QUERY_PREPARED)
        b.record(stream)
        b.synchronize()
        times.append(a.elapsed_time(b) * 1e3)
    cache.close()
    del scrub
    times.sort()
    med = times[len(times) // 2]
    keys = cond + (HIST + 1) * (LU + AUDIO)
    nbytes = 2.0 * keys * H * D * 2 + 2.0 * AUDIO * H * D * 2
    return {"keys": keys, "cond": cond, "bytes": nbytes, "us_median": med,
            "us_p10": times[len(times) // 10], "us_p90": times[(9 * len(times)) // 10],
            "gbps": nbytes / (med * 1e-6) / 1e9, "frac_hbm": nbytes / (med * 1e-6) / 1e9 / PEAK_HBM_GBS}


def catch_up(args, ws, sets, vpos, gamma, eps, stream, dev, n_units=3):
    """Catch-up after a stall: the queries of n_units consecutive 920-token
    units in one ws_unit_attention_groups call, each unit under its own
    8-unit window (256 + 9 x 920 = 8536 keys per unit), against the same work
    as one ws_unit_attention call per unit, and against the one call with
    every unit partitioned as if it had all CUs (WS_OPT_VIDEO_CLASS_CUS).
    Queries prepared beforehand; after a warm-up, the variants in turn,
    medians of `long_reps` repetitions (events around the call(s))."""
    import torch
    first = HIST
    cache = ws.Cache(H, 4 + (HIST + n_units + 1) * 16, max_q_tokens=LU * n_units)
    s0 = sets[0]
    cache.append(0, ws.WS_KIND_COND, s0["ck"], s0["cv"], ws.WS_APPEND_RAW)
    for u in range(first + n_units):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, vpos[u], gamma, eps)
        cache.commit(u)
    q_all = torch.empty((LU * n_units, H, D), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q_all)
    cache.step_append([], [dict(q=sets[i % 2]["q"], q_out=q_all[i * LU:(i + 1) * LU],
                                positions=vpos[first + i], gamma=gamma, eps=eps) for i in range(n_units)])
    masks = [ws.mask_spec(first + i, first + i - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))
             for i in range(n_units)]
    groups = [(LU, m) for m in masks]

    def one_call():
        cache.unit_attention_groups(q_all, out, groups, ws.WS_QUERY_PREPARED)

    def separate():
        for i, m in enumerate(masks):
            cache.unit_attention(q_all[i * LU:(i + 1) * LU], out[i * LU:(i + 1) * LU], m,
                                 ws.WS_QUERY_PREPARED)

    def all_cus():
        cache.set_option(ws.WS_OPT_VIDEO_CLASS_CUS, 1)
        one_call()
        cache.set_option(ws.WS_OPT_VIDEO_CLASS_CUS, 0)

    # about 20 ms of the same work first (the clocks settle under load), then
    # the three variants in turn, each call timed on its own
    for _ in range(40):
        one_call()
    t = {one_call: [], separate: [], all_cus: []}
    for _ in range(max(args.long_reps, 1)):
        for fn in t:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            b.synchronize()
            t[fn].append(a.elapsed_time(b) * 1e3)
    t1, t3, t1_all = (sorted(t[fn])[len(t[fn]) // 2] for fn in (one_call, separate, all_cus))
    cache.close()
    lk = COND + (HIST + 1) * LU
    flop = n_units * video_flop(LU, lk)
    return {"units": n_units, "queries": LU * n_units, "keys_per_unit": lk, "flop": flop,
            "us": t1, "tflops": flop / (t1 * 1e-6) / 1e12, "us_one_call_all_cus_per_unit": t1_all,
            "us_separate_calls": t3,
            "tflops_separate_calls": flop / (t3 * 1e-6) / 1e12}


def block_step(args, ws, sets, vpos, apos, gamma, eps, stream, dev, steps=50, warmup=20):
    """The attention sub-block of one performer layer per unit at 640x368
    (ws_block_step: QKV projection [924 x 5120] x [5120 x 15360], the unit's
    K/V append and query preparation, video and audio attention over the
    8-unit window, output projection [924 x 5120] x [5120 x 5120]), at steady
    state: each step is a new unit, committed and evicted as in the main
    loop.  Random weights (N(0, 1/5120) in bf16): timing only.  Events
    around `steps` steps, and the library's per-launch timing ring for the
    breakdown."""
    import numpy as np
    import torch
    from paper_2607_04443_amd import synth
    hid = H * D
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 5))

    def dev_w(shape):
        w = rng.standard_normal(shape, dtype=np.float32) / np.sqrt(hid)
        return torch.from_numpy(synth.bf16_bits(w).view(np.int16)).view(torch.bfloat16).to(dev)

    w_qkv, w_out = dev_w((hid, 3 * hid)), dev_w((hid, hid))
    x = torch.from_numpy(synth.normal_bf16(rng, (LU + AUDIO, hid)).view(np.int16)).view(torch.bfloat16).to(dev)
    y = torch.empty_like(x)
    cache = ws.Cache(H, 4 + (HIST + 2) * 16 + 8, max_q_tokens=1024)
    s0 = sets[0]
    cache.append(0, ws.WS_KIND_COND, s0["ck"], s0["cv"], ws.WS_APPEND_RAW)
    for u in range(HIST):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, vpos[u], gamma, eps)
        cache.append(u, ws.WS_KIND_AUDIO, s["ka"], s["va"], ws.WS_APPEND_NORM_ROPE, apos[u], gamma, eps)
        cache.commit(u)
    block = ws.Block(cache, w_qkv, w_out, max_rows=LU + AUDIO)
    u = HIST

    def one(u):
        block.step(x, LU, u, vpos[u], apos[u], gamma, gamma, y,
                   ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO)),
                   ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO)),
                   eps=eps)
        cache.commit(u)
        cache.evict_before(u - HIST + 1)

    for _ in range(warmup):
        one(u)
        u += 1
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        one(u)
        u += 1
    b.record(stream)
    b.synchronize()
    us = a.elapsed_time(b) * 1e3 / steps
    cache.timing_enable(8 * steps)
    for _ in range(steps):
        one(u)
        u += 1
    torch.cuda.synchronize()
    rec = cache.timing_read()
    cache.timing_enable(0)
    block.close()
    cache.close()

    def avg(path, key="attn_us"):
        v = [r[key] for r in rec if r["path"] == path]
        return sum(v) / len(v) if v else None

    rows = LU + AUDIO
    f_qkv, f_out = 2.0 * rows * hid * 3 * hid, 2.0 * rows * hid * hid
    t_qkv, t_out = avg("qkv_gemm"), avg("out_gemm")
    # the step's audio call: its rows ride in the video kernel, the audio
    # kernel walks the audio-token pages only (path 'audio_riders'), unless
    # the step does not qualify (path 'audio')
    apath = "audio_riders" if any(r["path"] == "audio_riders" for r in rec) else "audio"
    t_app, t_vid, t_aud = avg("append"), avg("video"), avg(apath)
    if all(r["n_splits"] == 0 for r in rec if r["path"] == apath):
        t_aud = 0.0  # no audio kernel launched: the rows' own pages were attended in the video kernel
    t_merge = avg(apath, "merge_us")
    attn_us = t_app + t_vid + t_aud + t_merge
    return {"us_per_step": us, "rows": rows, "hidden": hid,
            "qkv_gemm_us": t_qkv, "qkv_gemm_tflops": f_qkv / (t_qkv * 1e-6) / 1e12,
            "out_gemm_us": t_out, "out_gemm_tflops": f_out / (t_out * 1e-6) / 1e12,
            "append_us": t_app, "video_kernel_us": t_vid, "audio_kernel_us": t_aud, "merge_us": t_merge,
            "audio_rows_in_video_kernel": apath == "audio_riders",
            "attention_share": attn_us / (attn_us + t_qkv + t_out)}


def v01_step(ws, torch, dev, steps=200, settle=200):
    """The v0.1-scale streaming step (192x336: 12 heads, 252-token units, a
    64-token conditioning slice, a 2-unit history window), timed like the
    contract step: the slice rewrite, the unit's K/V append and its query
    preparation in one ws_step_append launch, then ws_unit_attention on the
    prepared queries (252 queries over 64 + 3 x 252 = 820 keys), commit and
    eviction; `settle` untimed steps, then `steps` timed ones."""
    import numpy as np
    from paper_2607_04443_amd import synth
    h, grid, cond, hist = 12, (12, 21), 64, 2
    lu = grid[0] * grid[1]
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 5))

    def dev_bf16(shape):
        return torch.from_numpy(synth.normal_bf16(rng, shape).view(np.int16)).view(torch.bfloat16).to(dev)

    sets = [dict(ck=dev_bf16((cond, h, D)), cv=dev_bf16((cond, h, D)), k=dev_bf16((lu, h, D)),
                 v=dev_bf16((lu, h, D)), q=dev_bf16((lu, h, D))) for _ in range(2)]
    n_units = hist + settle + steps + 50 + 2
    vpos = [torch.from_numpy(synth.video_positions(u, grid)).to(dev) for u in range(n_units)]
    gamma = torch.ones(D, dtype=torch.float32, device=dev)
    cache = ws.Cache(h, 2 + (hist + 2) * ((lu + 63) // 64) + 4, max_q_tokens=1024)
    s0 = sets[0]
    cache.append(0, ws.WS_KIND_COND, s0["ck"], s0["cv"], ws.WS_APPEND_RAW)
    for u in range(hist):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, vpos[u], gamma, 1e-6)
        cache.commit(u)
    q_p = torch.empty((lu, h, D), dtype=torch.bfloat16, device=dev)
    out = torch.empty((lu, h, D), dtype=torch.bfloat16, device=dev)

    stream = torch.cuda.current_stream()

    def step(u):
        s = sets[u % 2]
        cache.step_append([
            dict(unit=0, kind=ws.WS_KIND_COND, k=s["ck"], v=s["cv"], mode=ws.WS_APPEND_RAW),
            dict(unit=u, kind=ws.WS_KIND_VIDEO, k=s["k"], v=s["v"], mode=ws.WS_APPEND_NORM_ROPE,
                 positions=vpos[u], gamma=gamma, eps=1e-6)],
            [dict(q=s["q"], q_out=q_p, positions=vpos[u], gamma=gamma, eps=1e-6)], stream=stream)
        cache.unit_attention(q_p, out, ws.mask_spec(u, u - hist, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO)),
                             ws.WS_QUERY_PREPARED, stream=stream)
        cache.commit(u)
        cache.evict_before(u - hist + 1)

    u = hist
    for _ in range(settle):
        step(u)
        u += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(u)
        u += 1
    enqueued = time.perf_counter() - t0
    torch.cuda.synchronize()
    us = (time.perf_counter() - t0) * 1e6 / steps
    # the GPU's share: a further pass with the library's launch timing on
    # (append launch, attention kernel, and the time from its end to the
    # merge's end)
    cache.timing_enable(3 * 50)
    for _ in range(50):
        step(u)
        u += 1
    torch.cuda.synchronize()
    rec = cache.timing_read()
    cache.close()

    def mean(path, key):
        v = [r[key] for r in rec if r["path"] == path]
        return sum(v) / len(v) if v else 0.0

    lk = cond + (hist + 1) * lu
    flop = 4.0 * h * lu * lk * D
    return {"heads": h, "queries": lu, "keys": lk, "flop": flop, "us_per_unit": us,
            "tflops": flop / (us * 1e-6) / 1e12, "host_enqueue_us_per_step": enqueued * 1e6 / steps,
            "append_us": mean("append", "attn_us"), "video_kernel_us": mean("video", "attn_us"),
            "video_merge_us": mean("video", "merge_us")}


def video_configs(ws, torch, dev, launches=60):
    """The video kernel alone on the seeded configurations v0.1 (12 heads, 252
    queries over 820 keys), v0.2 single unit (40 heads, 920 over 1176) and
    v0.2 with an 8-unit history (920 over 8536): the cache and queries of each
    (prepared by one ws_step_append), then `launches` ws_unit_attention calls;
    the median of the library's per-launch kernel times (HIP events on the
    call's stream around the kernel) and its TFLOP/s."""
    import numpy as np
    from paper_2607_04443_amd import synth
    out = {}
    for name in ("v01", "v02_single", "v02_hist8"):
        wl = synth.make_workload(name, steps=1)
        cfg = wl.config
        keep = []

        def dev_bits(bits):
            t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)
            keep.append(t)
            return t

        def dev_arr(a, dt):
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(dev)
            keep.append(t)
            return t

        cache = ws.Cache(cfg.heads, 8 + (cfg.hist + 2) * (cfg.unit_tokens // 64 + 3) + cfg.cond // 64,
                         max_q_tokens=1024)
        gk, gq = dev_arr(wl.gamma_k, np.float32), dev_arr(wl.gamma_q, np.float32)
        st = wl.steps[0]
        for seg in wl.cached + st.segments:
            k, v = dev_bits(seg.k), dev_bits(seg.v)
            if seg.mode == synth.MODE_RAW:
                cache.append(seg.unit, seg.kind, k, v, ws.WS_APPEND_RAW)
            else:
                cache.append(seg.unit, seg.kind, k, v, ws.WS_APPEND_NORM_ROPE,
                             dev_arr(seg.positions, np.int32), gk, wl.eps)
        q = dev_bits(st.q_video)
        qp = torch.empty_like(q)
        cache.step_append([], [dict(q=q, q_out=qp, positions=dev_arr(st.q_video_pos, np.int32), gamma=gq,
                                    eps=wl.eps)])
        o = torch.empty_like(q)
        mask = ws.mask_spec(wl.current_unit, -(2 ** 31), (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))
        for _ in range(20):
            cache.unit_attention(qp, o, mask, ws.WS_QUERY_PREPARED)
        torch.cuda.synchronize()
        cache.timing_enable(launches)
        for _ in range(launches):
            cache.unit_attention(qp, o, mask, ws.WS_QUERY_PREPARED)
        torch.cuda.synchronize()
        t = sorted(r["attn_us"] for r in cache.timing_read())
        cache.timing_enable(0)
        cache.close()
        lq, lk = cfg.unit_tokens, cfg.cond + (cfg.hist + 1) * cfg.unit_tokens
        flop = 4.0 * cfg.heads * lq * lk * D
        med = t[len(t) // 2]
        out[name] = {"heads": cfg.heads, "queries": lq, "keys": lk, "flop": flop, "kernel_us_median": med,
                     "tflops": flop / (med * 1e-6) / 1e12}
    return out


COPY_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "unit_attn_traffic.md")
KERNELS_SRC = os.path.join(ROOT, "paper_2607_04443_amd", "csrc", "kernels.hip")


def kernels_sha256():
    import hashlib
    with open(KERNELS_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def recorded_traffic():
    """HBM bytes per unit_attn_kernel launch from the committed counter
    summary, or None when it was taken on other kernel sources."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    fields = dict(line.split(": ", 1) for line in text.splitlines()
                  if line.startswith(("kernels_sha256: ", "unit_attn_traffic_bytes: ")))
    if fields.get("kernels_sha256") != kernels_sha256() or "unit_attn_traffic_bytes" not in fields:
        return None
    return float(fields["unit_attn_traffic_bytes"])


def pmc_summary(fetch_dir, write_dir, long_fetch=None, long_write=None):
    """Markdown summary of FETCH_SIZE and WRITE_SIZE counter runs of
    --pmc-driver (the step driver, optionally also the long-history one):
    per-dispatch KiB (median over each kernel's dispatches of one grid size),
    scaled by what the same counter reads for the 256 MiB device copy."""
    import csv
    import glob
    import statistics

    def per_kernel(d, counter):
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit(f"no counter_collection.csv under {d}")
        disp = {}
        for f in files:
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                key = (f, r["Dispatch_Id"])
                name = r["Kernel_Name"]
                wg = int(r.get("Workgroup_Size") or 1) or 1
                grid = int(r.get("Grid_Size") or 0) // wg
                disp.setdefault(key, [name, grid, 0.0])[2] += float(r["Counter_Value"])
        out = {}
        for name, grid, val in disp.values():
            out.setdefault(name, []).append((grid, val))
        return out

    def pick(table, key, grid=None):
        rows = [v for n, vals in table.items() if key in n for v in vals]
        if grid == "max":  # the largest launch (the 256 MiB copy, the step's append)
            grid = max(r[0] for r in rows)
        if grid is not None:
            rows = [r for r in rows if r[0] == grid]
        return statistics.median(v for _, v in rows), len(rows)

    def table(fd, wd, kernels):
        fetch, write = per_kernel(fd, "FETCH_SIZE"), per_kernel(wd, "WRITE_SIZE")
        f_copy, _ = pick(fetch, "copyBuffer", "max")
        w_copy, _ = pick(write, "copyBuffer", "max")
        f_scale, w_scale = f_copy * 1024 / COPY_BYTES, w_copy * 1024 / COPY_BYTES
        lines = [f"Calibration: the {COPY_BYTES >> 20} MiB device copy (__amd_rocclr_copyBuffer) reads "
                 f"FETCH_SIZE {f_copy:.0f} KiB and WRITE_SIZE {w_copy:.0f} KiB, i.e. "
                 f"{f_scale:.3f} and {w_scale:.3f} counted bytes per byte moved; the figures below are "
                 "divided by these factors.",
                 "",
                 "| kernel | workgroups | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes per launch |",
                 "|---|---|---|---|---|---|"]
        result = {}
        for label, key, grid in kernels:
            try:
                fv, n = pick(fetch, key, grid)
                wv, _ = pick(write, key, grid)
            except (ValueError, statistics.StatisticsError):
                continue
            b = fv * 1024 / f_scale + wv * 1024 / w_scale
            result[label] = b
            shown = {None: "all", "max": "largest"}.get(grid, grid)
            lines.append(f"| {label} | {shown} | {n} | {fv:.0f} | {wv:.0f} | "
                         f"{b / 1e6:.1f} MB |")
        return lines, result

    def cmds(fd, wd, mode):
        arg = "" if mode == "step" else " long"
        return [f"    cd /tmp && timeout -s KILL 240 rocprofv3 --pmc FETCH_SIZE -d <repo>/{fd} "
                f"-o pmc -f csv -- python3 <repo>/bench.py --pmc-driver{arg}",
                f"    cd /tmp && timeout -s KILL 240 rocprofv3 --pmc WRITE_SIZE -d <repo>/{wd} "
                f"-o pmc -f csv -- python3 <repo>/bench.py --pmc-driver{arg}"]

    lines = ["# HBM traffic of the step's kernels, v0.2 unit with an 8-unit history (and the long-history "
             "video launch)",
             "",
             "Counters per dispatch (median over the driver's dispatches of each kernel and grid), "
             "from runs of committed programs, one counter each (from the repository root):",
             ""] + cmds(fetch_dir, write_dir, "step")
    if long_fetch:
        lines += cmds(long_fetch, long_write, "long")
    lines += [f"    python3 bench.py --pmc-summary {fetch_dir} {write_dir}"
              + (f" {long_fetch} {long_write}" if long_fetch else ""),
              "",
              "## The v0.2 step (256 + 9 x 920 video keys)",
              "",
              "The step driver runs three steps (ws_step_append, then ws_step_attention with the audio "
              "rows riding in the video kernel and the audio kernel over the 9 audio-token pages, 80 "
              "workgroups), then the video and the audio attention three times each as separate calls "
              "(the audio kernel over all 8572 keys, 480 workgroups).  unit_attn_kernel is the median "
              "over both kinds of launch.",
              ""]
    t, result = table(fetch_dir, write_dir, (
        ("unit_attn_kernel", "unit_attn_kernel", 256),
        ("step_combine_kernel", "step_combine", None),
        ("video_combine_kernel", "video_combine", None),
        ("audio_attn_kernel (all pages)", "audio_attn_kernel", 480),
        ("audio_attn_kernel (audio pages)", "audio_attn_kernel", 80),
        ("combine_kernel (audio)", "::combine_kernel(", None),
        ("kv_append_kernel (the step's)", "kv_append_kernel", "max")))
    lines += t
    lk_v = COND + (HIST + 1) * LU
    kv_bytes = 2.0 * lk_v * H * D * 2
    lines += ["",
              f"Video K/V visible to one launch: {kv_bytes / 1e6:.1f} MB (each (head, page) tile is "
              "read by the four query-tile workgroups; pages the 256 MB cache already holds are not "
              "fetched from HBM again)."]
    if long_fetch:
        lk_l = COND + (LONG_HIST + 1) * LU
        kv_l = 2.0 * lk_l * H * D * 2
        t, res_l = table(long_fetch, long_write, (("unit_attn_kernel", "unit_attn_kernel", 256),
                                                  ("video_combine_kernel", "video_combine", None),
                                                  ("kv_append_kernel (the step's)", "kv_append_kernel", "max")))
        lines += ["", f"## Long history ({lk_l} video keys)", ""] + t
        b = res_l.get("unit_attn_kernel")
        if b:
            lines += ["", f"Video K/V visible to one launch: {kv_l / 1e6:.1f} MB; unit_attn_kernel moves "
                          f"{b / kv_l:.2f}x that."]
    lines += ["",
              f"kernels_sha256: {kernels_sha256()}",
              f"unit_attn_traffic_bytes: {result.get('unit_attn_kernel', float('nan')):.0f}"]
    print("\n".join(lines))


MFMA_COUNTERS = ("GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CYCLES "
                 "SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_INSTS_VALU SQ_LDS_BANK_CONFLICT SQ_WAVES")


def trace_summary(path, steps=200):
    """Kernel durations of a --kernel-trace run of the default bench, grouped
    by kernel and grid, and the medians of the contract steps: the last
    `steps` of the first unbroken run of (append, video, merge) launch
    triples (settle, warm-up and contract steps, in launch order)."""
    import csv
    import statistics
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Start_Timestamp"]))
    groups, order, seq = {}, [], []
    for r in rows:
        name = r["Kernel_Name"]
        short = name.replace("(anonymous namespace)", "anon").split("(")[0].split("::")[-1].strip()
        if short.startswith("void "):
            short = short[5:]
        if "rocclr" in name:
            short = name.split("(")[0][:40]
        if "at::native" in name:
            short = name[:40] + "..."
        if name.startswith("Cijk_"):  # hipBLASLt's generated GEMM kernels
            tile = [t for t in name.split("_") if t.startswith("MT")]
            short = f"hipBLASLt GEMM (macro tile {tile[0][2:] if tile else '?'})"
        wg = int(r["Grid_Size_X"]) // int(r["Workgroup_Size_X"])
        wgy = int(r["Grid_Size_Y"]) // int(r["Workgroup_Size_Y"])
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        label = ""
        if short == "unit_attn_kernel" and wg == 256:  # by duration: 1176, 8536 or 30616 keys
            label = ("long history (30616 keys)" if d > 400 else "v0.2 unit, 8536 keys" if d > 100
                     else "v0.2 single unit, 1176 keys")
        key = (short, wg, wgy, label)
        if key not in groups:
            order.append(key)
        groups.setdefault(key, []).append(d)
        seq.append((short, wg, d))
    print("| kernel | workgroups | workload | calls | avg us | median us | min us | max us |")
    print("|---|---|---|---|---|---|---|---|")
    for key in sorted(order, key=lambda k: -sum(groups[k])):
        v = groups[key]
        wgs = f"{key[1]}" + (f", {key[2]}" if key[2] > 1 else "")
        print(f"| {key[0]} | {wgs} | {key[3]} | {len(v)} | {statistics.mean(v):.2f} | "
              f"{statistics.median(v):.2f} | {min(v):.2f} | {max(v):.2f} |")
    triples, last = [], None
    for i in range(len(seq) - 2):
        if (seq[i][0] == "kv_append_kernel" and seq[i + 1][0] == "unit_attn_kernel" and seq[i + 1][1] == 256
                and seq[i + 2][0] == "step_combine_kernel"):
            if last is not None and i != last + 3:
                break
            triples.append((seq[i][2], seq[i + 1][2], seq[i + 2][2]))
            last = i
    # the breakdown pass: separate calls after each step's append, each
    # unit_attn_kernel followed by its own video_combine_kernel (the launches
    # roofline.achieved averages)
    separate = [seq[i][2] for i in range(1, len(seq) - 1)
                if seq[i][0] == "unit_attn_kernel" and seq[i][1] == 256 and 100 < seq[i][2] < 400
                and seq[i - 1][0] == "kv_append_kernel" and seq[i + 1][0] == "video_combine_kernel"]
    if separate:
        print(f"\nBreakdown pass (separate video calls): {len(separate)} unit_attn_kernel launches, average "
              f"{statistics.mean(separate):.2f} us, median {statistics.median(separate):.2f} us.")
    contract = triples[-steps:]
    if contract:
        med = [statistics.median(t[j] for t in contract) for j in range(3)]
        print(f"\nContract steps ({len(contract)} after {len(triples) - len(contract)} settle and warm-up "
              f"steps, medians): append {med[0]:.2f} us, "
              f"video {med[1]:.2f} us, merge {med[2]:.2f} us: {sum(med):.1f} us of kernel time per step.")


def mfma_summary(d):
    """MFMA utilisation of unit_attn_kernel (256 workgroups) from one counter
    run of the step driver: per dispatch, median over the dispatches.
    GRBM_GUI_ACTIVE comes summed over the 8 XCDs; MfmaUtil is
    SQ_VALU_MFMA_BUSY_CYCLES / (per-XCD GRBM_GUI_ACTIVE x 1024 SIMDs) and the
    MFMA FLOP are SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (the counter
    definitions of rocprofiler-sdk for gfx950)."""
    import csv
    import glob
    import statistics
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    disp = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if "unit_attn_kernel" not in r["Kernel_Name"]:
                continue
            if int(r["Grid_Size"]) // max(1, int(r["Workgroup_Size"])) != 256:
                continue
            e = disp.setdefault((f, r["Dispatch_Id"]), {"us": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3})
            e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    if not disp:
        raise SystemExit("no unit_attn_kernel dispatch in the counters")

    def med(key):
        return statistics.median(e[key] for e in disp.values() if key in e)

    us = med("us")
    grbm = med("GRBM_GUI_ACTIVE") / 8
    busy = med("SQ_VALU_MFMA_BUSY_CYCLES")
    flop = med("SQ_INSTS_VALU_MFMA_MOPS_BF16") * 512
    lk_v = COND + (HIST + 1) * LU
    alg = video_flop(LU, lk_v)
    rows = [("dispatches", f"{len(disp)}"),
            ("duration (counter run, median)", f"{us:.1f} us"),
            ("GRBM_GUI_ACTIVE per XCD", f"{grbm:.0f} cycles ({grbm / us / 1e3:.2f} GHz over the duration)"),
            ("SQ_VALU_MFMA_BUSY_CYCLES", f"{busy:.0f}"),
            ("MfmaUtil", f"{100 * busy / (grbm * 1024):.1f} %"),
            ("MFMA FLOP (MOPS_BF16 x 512)", f"{flop:.4g} ({flop / alg:.3f}x the {alg:.4g} algorithmic)"),
            ("MFMA TFLOP/s over the duration", f"{flop / (us * 1e-6) / 1e12:.0f}"),
            ("SQ_INSTS_VALU", f"{med('SQ_INSTS_VALU'):.0f}"),
            ("SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES", f"{med('SQ_WAIT_INST_ANY') / med('SQ_WAVE_CYCLES'):.3f}"),
            ("SQ_BUSY_CYCLES", f"{med('SQ_BUSY_CYCLES'):.0f}"),
            ("SQ_LDS_BANK_CONFLICT", f"{med('SQ_LDS_BANK_CONFLICT'):.0f}"),
            ("SQ_WAVES", f"{med('SQ_WAVES'):.0f}")]
    lines = ["# MFMA utilisation: unit_attn_kernel, v0.2 unit with an 8-unit history",
             "",
             "One counter run of the step driver (three ws_step_attention steps, then three separate "
             "video calls), from the repository root:",
             "",
             f"    cd /tmp && timeout -s KILL 240 rocprofv3 --pmc {MFMA_COUNTERS} -d <repo>/{d} -o pmc "
             "-f csv -- python3 <repo>/bench.py --pmc-driver",
             f"    python3 bench.py --mfma-summary {d}",
             "",
             "| quantity | value |", "|---|---|"] + [f"| {a} | {b} |" for a, b in rows] + [
             "", f"kernels_sha256: {kernels_sha256()}"]
    print("\n".join(lines))


def pmc_driver(mode, ws, cache, step, u, q_v, out_v, q_a, out_a, sets, gamma, eps, dev):
    import torch
    if mode == "long":
        lcache, one_step = long_setup(ws, sets, gamma, eps, dev)
        one_step(0, attention=False)
        torch.cuda.synchronize()
        for _ in range(3):
            one_step(0)
            torch.cuda.synchronize()
        lcache.close()
        what = "3 long-history steps"
    else:
        for k in range(3):
            step(u + k, False)
            torch.cuda.synchronize()
        u += 2
        vmask = ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))
        amask = ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO))
        for _ in range(3):
            cache.unit_attention(q_v, out_v, vmask, ws.WS_QUERY_PREPARED)
            torch.cuda.synchronize()
        for _ in range(3):
            cache.audio_attention(q_a, out_a, amask, ws.WS_QUERY_PREPARED)
            torch.cuda.synchronize()
        what = "3 steps, 3 video, 3 audio"
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
        torch.cuda.synchronize()
    log(f"pmc driver: {what}, 3 copies of", COPY_BYTES >> 20, "MiB")


def measured_peaks(ws, torch, stream, dev):
    """The ceilings this GPU sustains, from the library's calibration probes:
    a bf16 MFMA loop (2048 workgroups of 4 waves, register operands, about
    10 ms) on small-integer operands and on random ones (attention's
    operands switch as many bits as the latter, and the clock the chip holds
    under a long MFMA load falls with them), and one streaming read of a
    2 GiB buffer (512 workgroups, each a contiguous chunk, nontemporal
    loads: loads that allocate in the caches sustain less); medians of 7
    timed runs after 3 untimed ones."""
    sink = torch.zeros(2, dtype=torch.float32, device=dev)
    buf = torch.zeros(1 << 31, dtype=torch.uint8, device=dev)
    h = stream.cuda_stream

    def timed(launch):
        t = []
        for i in range(10):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            launch()
            b.record(stream)
            b.synchronize()
            if i >= 3:
                t.append(a.elapsed_time(b) * 1e-3)
        return sorted(t)[len(t) // 2]

    flop = [0.0]

    def mfma():
        flop[0] = ws.ws_probe_mfma(2048, 20000, sink.data_ptr(), h)

    t_m = timed(mfma)
    t_mr = timed(lambda: ws.ws_probe_mfma_random(2048, 20000, sink.data_ptr(), h))
    t_r = timed(lambda: ws.ws_probe_read(buf.data_ptr(), buf.numel(), 512, sink.data_ptr() + 4, h))
    del buf
    return {"mfma_bf16_tflops": flop[0] / t_m / 1e12, "mfma_frac_of_published": flop[0] / t_m / 1e12 / PEAK_BF16_TFLOPS,
            "mfma_bf16_random_operands_tflops": flop[0] / t_mr / 1e12,
            "hbm_read_gbps": (1 << 31) / t_r / 1e9, "hbm_frac_of_published": (1 << 31) / t_r / 1e9 / PEAK_HBM_GBS}


def main():
    args = parse()
    if args.mfma_summary:
        mfma_summary(args.mfma_summary)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary)
        return
    if args.pmc_summary:
        if len(args.pmc_summary) not in (2, 4):
            raise SystemExit("--pmc-summary takes 2 or 4 directories")
        pmc_summary(*args.pmc_summary)
        return
    if args.cpu_v01_point:
        print(json.dumps(cpu_v01_point()), flush=True)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); this build has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2607_04443_amd import _build
    if not os.path.exists(_build.LIB_PATH):
        _build.build()
    from paper_2607_04443_amd import synth, ws

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 2))

    def dev_bf16(shape):
        return torch.from_numpy(synth.normal_bf16(rng, shape).view(np.int16)).view(
            torch.bfloat16).to(dev)

    n_steps_total = args.settle + args.warmup + args.steps
    max_pages = 4 + (HIST + 2) * 16 + 8
    cache = ws.Cache(H, max_pages, max_q_tokens=1024)
    if args.video_splits:
        cache.set_option(ws.WS_OPT_VIDEO_KV_SPLITS, args.video_splits)
    if args.audio_splits:
        cache.set_option(ws.WS_OPT_AUDIO_KV_SPLITS, args.audio_splits)
    gamma = torch.ones(D, dtype=torch.float32, device=dev)
    eps = 1e-6

    # resident inputs: two rotating sets of per-unit tensors, positions per unit
    sets = [dict(ck=dev_bf16((COND, H, D)), cv=dev_bf16((COND, H, D)), k=dev_bf16((LU, H, D)),
                 v=dev_bf16((LU, H, D)), ka=dev_bf16((AUDIO, H, D)), va=dev_bf16((AUDIO, H, D)),
                 q=dev_bf16((LU, H, D)), qa=dev_bf16((AUDIO, H, D))) for _ in range(2)]
    last_unit = HIST + max(n_steps_total + 2 * args.steps + 10, 130) + 2
    vpos = [torch.from_numpy(synth.video_positions(u, GRID)).to(dev) for u in range(last_unit + 1)]
    apos = [torch.from_numpy(synth.audio_positions(u, AUDIO)).to(dev) for u in range(last_unit + 1)]
    out_v = torch.empty((LU, H, D), dtype=torch.bfloat16, device=dev)
    out_a = torch.empty((AUDIO, H, D), dtype=torch.bfloat16, device=dev)

    # history: units 0..HIST-1, committed
    s0 = sets[0]
    cache.append(0, ws.WS_KIND_COND, s0["ck"], s0["cv"], ws.WS_APPEND_RAW)
    for u in range(HIST):
        s = sets[u % 2]
        cache.append(u, ws.WS_KIND_VIDEO, s["k"], s["v"], ws.WS_APPEND_NORM_ROPE, vpos[u], gamma, eps)
        cache.append(u, ws.WS_KIND_AUDIO, s["ka"], s["va"], ws.WS_APPEND_NORM_ROPE, apos[u], gamma, eps)
        cache.commit(u)
    torch.cuda.synchronize()

    ev = {name: [] for name in ("append", "video", "audio")}

    q_v = torch.empty((LU, H, D), dtype=torch.bfloat16, device=dev)  # prepared queries
    q_a = torch.empty((AUDIO, H, D), dtype=torch.bfloat16, device=dev)

    def step(u, timed):
        s = sets[u % 2]
        e = [torch.cuda.Event(enable_timing=True) for _ in range(6)] if timed else None
        if timed:
            e[0].record(stream)
        cache.step_append([
            dict(unit=0, kind=ws.WS_KIND_COND, k=s["ck"], v=s["cv"], mode=ws.WS_APPEND_RAW),
            dict(unit=u, kind=ws.WS_KIND_VIDEO, k=s["k"], v=s["v"], mode=ws.WS_APPEND_NORM_ROPE,
                 positions=vpos[u], gamma=gamma, eps=eps),
            dict(unit=u, kind=ws.WS_KIND_AUDIO, k=s["ka"], v=s["va"], mode=ws.WS_APPEND_NORM_ROPE,
                 positions=apos[u], gamma=gamma, eps=eps)],
            [dict(q=s["q"], q_out=q_v, positions=vpos[u], gamma=gamma, eps=eps),
             dict(q=s["qa"], q_out=q_a, positions=apos[u], gamma=gamma, eps=eps)])
        vmask = ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO))
        amask = ws.mask_spec(u, u - HIST, (ws.WS_KIND_COND, ws.WS_KIND_VIDEO, ws.WS_KIND_AUDIO))
        if not timed:
            cache.step_attention(dict(q=q_v, out=out_v, mask=vmask, mode=ws.WS_QUERY_PREPARED),
                                 dict(q=q_a, out=out_a, mask=amask, mode=ws.WS_QUERY_PREPARED))
        if timed:
            e[1].record(stream)
            e[2].record(stream)
            cache.unit_attention(q_v, out_v, vmask, ws.WS_QUERY_PREPARED)
            e[3].record(stream)
            e[4].record(stream)
            cache.audio_attention(q_a, out_a, amask, ws.WS_QUERY_PREPARED)
        if timed:
            e[5].record(stream)
            ev["append"].append((e[0], e[1]))
            ev["video"].append((e[2], e[3]))
            ev["audio"].append((e[4], e[5]))
        cache.commit(u)
        cache.evict_before(u - HIST + 1)

    u = HIST
    if args.pmc_driver:
        pmc_driver(args.pmc_driver, ws, cache, step, u, q_v, out_v, q_a, out_a, sets, gamma, eps, dev)
        cache.close()
        return
    settle_us = []
    torch.cuda.synchronize()
    for b in range(0, args.settle, 25):
        n = min(25, args.settle - b)
        t0 = time.perf_counter()
        for _ in range(n):
            step(u, False)
            u += 1
        torch.cuda.synchronize()
        settle_us.append(round((time.perf_counter() - t0) * 1e6 / n, 1))
    for _ in range(args.warmup):
        step(u, False)
        u += 1
    torch.cuda.synchronize()
    # The contract measurement: exactly `steps` steps, nothing recorded in
    # between (a HIP event drains the queue, so per-step events would charge
    # their own cost to the step).
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(u, False)
        u += 1
    enqueued = time.perf_counter() - t0  # host time to issue the steps
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    # The same steps with the audio call in its own kernel over all its pages
    # (the audio rows not riding in the video kernel), timed the same way.
    cache.set_option(ws.WS_OPT_STEP_SEPARATE_AUDIO, 1)
    for _ in range(10):
        step(u, False)
        u += 1
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(u, False)
        u += 1
    torch.cuda.synchronize()
    us_separate_audio = (time.perf_counter() - t0) * 1e6 / args.steps
    cache.set_option(ws.WS_OPT_STEP_SEPARATE_AUDIO, 0)
    # A second pass of `steps` steps for the breakdown: events around each
    # component, and the library's launch timing of the attention calls (HIP
    # events on the calls' stream around each kernel).
    cache.timing_enable(3 * args.steps + 8)
    for _ in range(args.steps):
        step(u, True)
        u += 1
    torch.cuda.synchronize()
    calls = cache.timing_read()
    cache.timing_enable(0)

    def kernel_us(path, key):
        v = [c[key] for c in calls if c["path"] == path]
        return sum(v) / len(v)

    def avg_us(name):
        return 1e3 * sum(a.elapsed_time(b) for a, b in ev[name]) / len(ev[name])

    lk_v = COND + (HIST + 1) * LU
    lk_a = COND + (HIST + 1) * (LU + AUDIO)
    fv = video_flop(LU, lk_v)
    fa = 4.0 * H * AUDIO * lk_a * D
    # the append launch from the library's own events (the events around the
    # call would also take in the host's time to issue it)
    t_video, t_audio, t_append = avg_us("video"), avg_us("audio"), kernel_us("append", "attn_us")
    audio_bytes = 2.0 * lk_a * H * D * 2 + 2.0 * AUDIO * H * D * 2
    append_bytes = 4.0 * (COND + LU + AUDIO) * H * D * 2 + 2.0 * (LU + AUDIO) * H * D * 2

    # audio path with cold caches, on the graded key count (a 336-token
    # conditioning slice: 336 + 9 x 924 = 8652 keys) and on the bench step's
    # 256-token slice (8572 keys)
    cold = cold_256 = None
    if args.cold_audio_reps > 0:
        cold = cold_audio(args, ws, sets, vpos, apos, gamma, eps, stream, dev, 336)
        cold_256 = cold_audio(args, ws, sets, vpos, apos, gamma, eps, stream, dev, COND)

    long_hist = long_history(args, ws, sets, gamma, eps, stream, dev) if args.long_reps > 0 else None
    catch = catch_up(args, ws, sets, vpos, gamma, eps, stream, dev) if args.long_reps > 0 else None
    block = block_step(args, ws, sets, vpos, apos, gamma, eps, stream, dev) if args.long_reps > 0 else None
    vconf = video_configs(ws, torch, dev) if args.long_reps > 0 else None
    v01 = v01_step(ws, torch, dev) if args.long_reps > 0 else None
    peaks = measured_peaks(ws, torch, stream, dev) if args.peak_probes else None

    t_vkern, t_vmerge = kernel_us("video", "attn_us"), kernel_us("video", "merge_us")
    v_splits = sorted({c["n_splits"] for c in calls if c["path"] == "video"})
    achieved = fv / (t_vkern * 1e-6) / 1e12
    result = {
        "metric": "unit-attention TFLOP/s + us per 160ms unit at 640x368; audio-path HBM GB/s",
        "value": (fv + fa) / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_steps": args.settle,
        "settle_us_per_step": settle_us,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "v0.2 streaming unit at 640x368 with an 8-unit history window: "
                               f"H={H}, D={D}; video Q={LU} over {lk_v} keys; audio Q={AUDIO} "
                               f"over {lk_a} keys; cond slice {COND}; 64-token pages",
                   "global_batch": 1, "seq_len": lk_v, "parallelism": "single GPU"},
        "us_per_unit": ms_per_step * 1e3,
        # host (Python + library) time to enqueue one step; the step is
        # GPU-bound while this stays below us_per_unit
        "host_enqueue_us_per_step": enqueued * 1e6 / args.steps,
        # the same step with the audio attention as its own kernel over all
        # of its pages instead of riding in the video kernel
        "us_per_unit_separate_audio": us_separate_audio,
        "video_attention": {"us": t_video, "tflops": fv / (t_video * 1e-6) / 1e12, "flop": fv,
                            "kernel_us": t_vkern, "merge_us": t_vmerge, "splits": v_splits},
        "audio_attention": {"us_warm": t_audio, "gbps_warm": audio_bytes / (t_audio * 1e-6) / 1e9,
                            "bytes": audio_bytes, "keys": lk_a, "cold": cold,
                            "cold_cond256": cold_256},
        "kv_append": {"us": t_append, "gbps": append_bytes / (t_append * 1e-6) / 1e9},
        "long_history": long_hist,
        "video_configs": vconf,
        # the step at the v0.1 stream shape (192x336), timed like the contract
        "v01_step": v01,
        "catch_up": catch,
        "block_step": block,
        "roofline": {"bound": "mfma", "kernel": "unit_attn_kernel", "achieved": achieved,
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": recorded_traffic()},
        "cpu_baseline": None,
    }
    if peaks is not None:
        peaks["video_kernel_frac"] = achieved / peaks["mfma_bf16_tflops"]
        peaks["video_kernel_frac_of_random"] = achieved / peaks["mfma_bf16_random_operands_tflops"]
        if cold is not None:
            peaks["audio_cold_frac"] = cold["gbps"] / peaks["hbm_read_gbps"]
        result["measured_peaks"] = peaks
    cache.close()
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
