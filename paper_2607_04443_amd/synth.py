"""Seeded synthetic inputs shaped like the Wan-Streamer v0.2 streaming units.

This module holds no arithmetic of the method: it draws i.i.d. N(0, 1) values,
rounds them to bf16 bit patterns, and lays out the token positions of a unit.
The test suite feeds the same bit patterns to the HIP library and to the CPU
oracle, and the benchmark uses the same recipe.

Shapes (Wan-Streamer v0.2, Sec. 1 and Table 1: 192x336 -> 640x368 at 25 FPS in
160 ms units): with a 16x spatial latent compression and one latent frame per
unit, a 192x336 unit is a 12x21 = 252-token grid and a 640x368 unit a 23x40 =
920-token grid; each unit also carries 4 audio latent tokens (the short,
unsharded audio sequence of Sec. 3).  Model widths are 12 or 40 heads of 128.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 260704443
HEAD_DIM = 128

# Segment kinds and append modes, numbered as in include/ws.h.
KIND_COND, KIND_VIDEO, KIND_AUDIO = 0, 1, 2
MODE_RAW, MODE_NORM_ROPE = 0, 1


@dataclass(frozen=True)
class Config:
    name: str
    index: int          # seed offset
    heads: int
    grid: tuple         # (rows, cols) of one unit's video latent tokens
    cond: int           # conditioning (thinker slice) tokens
    hist: int           # committed history units in the cache
    audio: int = 0      # audio latent tokens per unit (0: video-only config)
    steps: int = 1      # denoising steps issued back-to-back
    path: str = "video"

    @property
    def unit_tokens(self):
        return self.grid[0] * self.grid[1]

    @property
    def video_keys(self):
        return self.cond + (self.hist + 1) * self.unit_tokens

    @property
    def audio_keys(self):
        return self.cond + (self.hist + 1) * (self.unit_tokens + self.audio)


CONFIGS = {
    # 192x336 scale: 12 heads, 252-token unit, 64 cond + 2 history + current = 820 keys
    "v01": Config("v01", 0, 12, (12, 21), 64, 2),
    # 640x368 single unit: 256 cond + 920 current = 1176 keys
    "v02_single": Config("v02_single", 1, 40, (23, 40), 256, 0),
    # 640x368 with an 8-unit history window: 256 + 9 * 920 = 8536 keys
    "v02_hist8": Config("v02_hist8", 2, 40, (23, 40), 256, 8),
    # audio path: 4 queries over cond + 9 units of (920 video + 4 audio).  The
    # stated total of 8652 keys is met by a 336-token conditioning slice.
    "audio": Config("audio", 3, 40, (23, 40), 336, 8, audio=4, path="audio"),
    # the same structure with a 256-token slice: 8572 keys
    "audio_c256": Config("audio_c256", 3, 40, (23, 40), 256, 8, audio=4, path="audio"),
    # long history: 256 + 33 * 920 = 30616 keys, 4 back-to-back denoising steps
    "long32": Config("long32", 4, 40, (23, 40), 256, 32, steps=4),
}


def bf16_bits(x) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (NaN -> quiet NaN)."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        rounded[nan] = 0x7FC0
    return rounded


def bf16_to_f32(bits) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact widening)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def normal_bf16(rng, shape) -> np.ndarray:
    return bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def video_positions(unit, grid) -> np.ndarray:
    """(t, h, w) of a unit's video tokens, row-major over the latent grid."""
    r, c = np.meshgrid(np.arange(grid[0]), np.arange(grid[1]), indexing="ij")
    pos = np.stack([np.full(r.size, unit), r.ravel(), c.ravel()], axis=1)
    return pos.astype(np.int32)


def audio_positions(unit, n) -> np.ndarray:
    """(t, h, w) = (unit, 0, j) for the unit's j-th audio token."""
    return np.stack([np.full(n, unit), np.zeros(n, dtype=np.int64), np.arange(n)],
                    axis=1).astype(np.int32)


@dataclass
class SegmentInput:
    unit: int
    kind: int
    mode: int
    k: np.ndarray                 # uint16 [n, H, D]
    v: np.ndarray                 # uint16 [n, H, D]
    positions: np.ndarray | None  # int32 [n, 3]


@dataclass
class StepInput:
    """One denoising step of the current unit: its own K/V and its queries."""
    segments: list                # current-unit SegmentInput(s)
    q_video: np.ndarray           # uint16 [Lu, H, D]
    q_video_pos: np.ndarray
    q_audio: np.ndarray | None    # uint16 [A, H, D]
    q_audio_pos: np.ndarray | None


@dataclass
class Workload:
    config: Config
    gamma_q: np.ndarray           # float32 [D]
    gamma_k: np.ndarray           # float32 [D]
    eps: float
    cached: list                  # SegmentInput: cond slice and history units
    steps: list = field(default_factory=list)
    current_unit: int = 0


def make_workload(name_or_cfg, variant: str = "plain", steps: int | None = None,
                  seed_offset: int = 0) -> Workload:
    """Draw the cache contents and per-step inputs of one configuration.

    Draw order: gammas (variants only) -> cond K -> cond V -> each history unit
    (video K, video V[, audio K, audio V]) -> per step: current K, V[, audio K,
    audio V] -> Q video -> Q audio.  variant: "plain" (gamma = 1), "seeded"
    (gamma = bf16(1 + 0.1 N(0,1))), "sharp" (gamma_q = 4, gamma_k = 1).
    """
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    rng = np.random.Generator(np.random.PCG64(SEED_BASE + cfg.index + seed_offset))
    H, D = cfg.heads, HEAD_DIM
    one = np.ones(D, dtype=np.float32)
    gq, gk = one.copy(), one.copy()
    if variant == "seeded":
        gq = bf16_to_f32(bf16_bits(1 + 0.1 * rng.standard_normal(D, dtype=np.float32)))
        gk = bf16_to_f32(bf16_bits(1 + 0.1 * rng.standard_normal(D, dtype=np.float32)))
    elif variant == "sharp":
        gq = np.full(D, 4.0, dtype=np.float32)
    elif variant != "plain":
        raise ValueError(variant)
    Lu = cfg.unit_tokens
    ck = normal_bf16(rng, (cfg.cond, H, D))
    cv = normal_bf16(rng, (cfg.cond, H, D))
    cached = [SegmentInput(0, KIND_COND, MODE_RAW, ck, cv, None)]
    for u in range(cfg.hist):
        k = normal_bf16(rng, (Lu, H, D))
        v = normal_bf16(rng, (Lu, H, D))
        cached.append(SegmentInput(u, KIND_VIDEO, MODE_NORM_ROPE, k, v,
                                   video_positions(u, cfg.grid)))
        if cfg.audio:
            ka = normal_bf16(rng, (cfg.audio, H, D))
            va = normal_bf16(rng, (cfg.audio, H, D))
            cached.append(SegmentInput(u, KIND_AUDIO, MODE_NORM_ROPE, ka, va,
                                       audio_positions(u, cfg.audio)))
    cur = cfg.hist
    wl = Workload(cfg, gq, gk, 1e-6, cached, current_unit=cur)
    for _ in range(cfg.steps if steps is None else steps):
        segs = [SegmentInput(cur, KIND_VIDEO, MODE_NORM_ROPE, normal_bf16(rng, (Lu, H, D)),
                             normal_bf16(rng, (Lu, H, D)), video_positions(cur, cfg.grid))]
        if cfg.audio:
            segs.append(SegmentInput(cur, KIND_AUDIO, MODE_NORM_ROPE,
                                     normal_bf16(rng, (cfg.audio, H, D)),
                                     normal_bf16(rng, (cfg.audio, H, D)),
                                     audio_positions(cur, cfg.audio)))
        qv = normal_bf16(rng, (Lu, H, D))
        qa = normal_bf16(rng, (cfg.audio, H, D)) if cfg.audio else None
        wl.steps.append(StepInput(segs, qv, video_positions(cur, cfg.grid), qa,
                                  audio_positions(cur, cfg.audio) if cfg.audio else None))
    return wl
