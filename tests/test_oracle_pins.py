"""Pins of the fp64 CPU oracle to facts outside itself.

The paper prints no worked example, so every pin is a closed form, an
invariant, a special case that reduces to a library routine, or brute force on
a tiny input.  Each pin is written as a function of an implementation object
so that ``test_planted_mistakes`` can show that a plausible mistake in the
oracle (a flipped sign, a swapped band, a dropped term, a transposed operand)
makes at least one pin fail.
"""
import math
import os
import types

import numpy as np
import pytest
import scipy.special
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _impl(**override):
    ns = types.SimpleNamespace(
        bf16_decode=oracle.bf16_decode, rmsnorm=oracle.rmsnorm, rope=oracle.rope,
        rope_angle=oracle.rope_angle, attention=oracle.attention, lse_merge=oracle.lse_merge)
    for k, v in override.items():
        setattr(ns, k, v)
    return ns


def _read_kv(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, v = line.split()
            out[k] = float(v)
    return out


def _read_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            rows.append([float(x) for x in line.split()])
    return rows


# --------------------------------------------------------------------------- #
# pins (each raises AssertionError when violated)
# --------------------------------------------------------------------------- #
def pin_bf16_decode(im):
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F80, 0x8000, 0x4049], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, math.inf, -0.0, 3.140625]
    got = im.bf16_decode(bits)
    assert list(got) == want
    assert math.copysign(1.0, got[5]) == -1.0


def pin_rmsnorm_hand(im):
    for x0, x1, g0, g1, eps, o0, o1 in _read_rows("rmsnorm_hand.txt"):
        got = im.rmsnorm(np.array([[x0, x1]]), np.array([g0, g1]), eps)[0]
        np.testing.assert_allclose(got, [o0, o1], rtol=1e-14, atol=0)


def pin_rmsnorm_mean_square(im):
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 128)) * rng.uniform(0.1, 10, (7, 1))
    eps = 1e-3
    y = im.rmsnorm(x, np.ones(128), eps)
    ms = np.mean(x * x, axis=1)
    np.testing.assert_allclose(np.mean(y * y, axis=1), ms / (ms + eps), rtol=1e-12)
    # scale invariance holds exactly when eps = 0
    y0 = im.rmsnorm(x, np.ones(128), 0.0)
    np.testing.assert_allclose(im.rmsnorm(3.7 * x, np.ones(128), 0.0), y0, rtol=1e-13)
    # gamma is an elementwise weight
    g = rng.uniform(0.5, 2, 128)
    np.testing.assert_allclose(im.rmsnorm(x, g, eps), im.rmsnorm(x, np.ones(128), eps) * g,
                               rtol=1e-13)


def pin_rope_golden(im):
    for pair, t, h, w, angle in _read_rows("rope_angles.txt"):
        pair = int(pair)
        pos = np.array([[int(t), int(h), int(w)]], dtype=np.int32)
        x = np.zeros((1, 128))
        x[0, 2 * pair] = 1.0
        y = im.rope(x, pos)
        want = np.zeros(128)
        want[2 * pair] = math.cos(angle)
        want[2 * pair + 1] = math.sin(angle)
        np.testing.assert_allclose(y[0], want, rtol=0, atol=1e-13)
        # the second element of the pair turns to (-sin, cos)
        x = np.zeros((1, 128))
        x[0, 2 * pair + 1] = 1.0
        y = im.rope(x, pos)
        want = np.zeros(128)
        want[2 * pair] = -math.sin(angle)
        want[2 * pair + 1] = math.cos(angle)
        np.testing.assert_allclose(y[0], want, rtol=0, atol=1e-13)


def pin_rope_isometry_and_identity(im):
    rng = np.random.default_rng(2)
    x = rng.standard_normal((9, 128))
    pos = rng.integers(0, 500, (9, 3)).astype(np.int32)
    y = im.rope(x, pos)
    np.testing.assert_allclose(np.hypot(y[:, 0::2], y[:, 1::2]), np.hypot(x[:, 0::2], x[:, 1::2]),
                               rtol=1e-13)
    np.testing.assert_array_equal(im.rope(x, np.zeros((9, 3), dtype=np.int32)), x)


def pin_rope_relativity(im):
    """<R(p) q, R(p') k> depends only on p - p' (per band)."""
    rng = np.random.default_rng(3)
    q = rng.standard_normal((5, 128))
    k = rng.standard_normal((6, 128))
    pq = rng.integers(0, 50, (5, 3)).astype(np.int32)
    pk = rng.integers(0, 50, (6, 3)).astype(np.int32)
    base = im.rope(q, pq) @ im.rope(k, pk).T
    for shift in ([7, 0, 0], [0, 11, 0], [0, 0, 13], [3, 5, 8]):
        s = np.array(shift, dtype=np.int32)
        np.testing.assert_allclose(im.rope(q, pq + s) @ im.rope(k, pk + s).T, base,
                                   rtol=1e-10, atol=1e-10)


def pin_rope_complex_form(im):
    """Same rotation written as complex multiplication by exp(i*angle)."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal((4, 128))
    pos = rng.integers(0, 300, (4, 3)).astype(np.int32)
    bands = np.repeat([0, 1, 2], [22, 21, 21])
    local = np.concatenate([np.arange(22) / 22, np.arange(21) / 21, np.arange(21) / 21])
    omega = 10000.0 ** (-local)
    ang = pos[:, bands] * omega[None, :]
    z = (x[:, 0::2] + 1j * x[:, 1::2]) * np.exp(1j * ang)
    want = np.empty_like(x)
    want[:, 0::2], want[:, 1::2] = z.real, z.imag
    np.testing.assert_allclose(im.rope(x, pos), want, rtol=1e-12, atol=1e-12)


def pin_attention_golden(im):
    g = _read_kv("attention_two_keys.txt")
    q = np.array([[g["q0"], g["q1"]]])
    k = np.array([[g["k1_0"], g["k1_1"]], [g["k2_0"], g["k2_1"]]])
    v = np.array([[g["v1_0"], g["v1_1"]], [g["v2_0"], g["v2_1"]]])
    o, lse = im.attention(q, k, v, g["scale"])
    np.testing.assert_allclose(o[0], [g["out0"], g["out1"]], rtol=1e-14)
    np.testing.assert_allclose(lse[0], g["lse"], rtol=1e-14)


def pin_attention_softmax_rows(im):
    """With V a permutation matrix the output is the softmax row, permuted
    (compared with scipy's softmax); rows sum to 1."""
    rng = np.random.default_rng(5)
    nk = 9
    q = rng.standard_normal((4, nk))
    k = rng.standard_normal((nk, nk))
    perm = rng.permutation(nk)
    vperm = np.eye(nk)[perm]          # row j is e_perm[j]
    o, lse = im.attention(q, k, vperm, 0.37)
    np.testing.assert_allclose(o.sum(axis=1), 1.0, rtol=1e-13)
    assert (o >= 0).all()
    ref = scipy.special.softmax(0.37 * q @ k.T, axis=1)
    np.testing.assert_allclose(o[:, perm], ref, rtol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(0.37 * q @ k.T, axis=1),
                               rtol=1e-13)


def pin_attention_vs_torch(im):
    """Special case that is a library routine: torch SDPA in float64 on the CPU."""
    rng = np.random.default_rng(6)
    for nq, nk, d in ((1, 1, 4), (3, 5, 8), (5, 9, 128), (2, 7, 16)):
        q, k, v = (rng.standard_normal(s) for s in ((nq, d), (nk, d), (nk, d)))
        mask = rng.random((nq, nk)) < 0.7
        mask[:, 0] = True
        scale = 1.0 / math.sqrt(d)
        for vis in (None, mask):
            o, _ = im.attention(q, k, v, scale, None if vis is None else vis.astype(np.uint8))
            ref = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q)[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None],
                attn_mask=None if vis is None else torch.from_numpy(vis)[None],
                scale=scale)[0].numpy()
            np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)


def pin_attention_single_key(im):
    rng = np.random.default_rng(7)
    v = rng.standard_normal((1, 128))
    o, lse = im.attention(rng.standard_normal((3, 128)), rng.standard_normal((1, 128)), v, 0.1)
    np.testing.assert_array_equal(o, np.repeat(v, 3, axis=0))


def pin_attention_identical_keys(im):
    rng = np.random.default_rng(8)
    k = np.repeat(rng.standard_normal((1, 32)), 6, axis=0)
    v = rng.standard_normal((6, 32))
    o, lse = im.attention(rng.standard_normal((2, 32)), k, v, 0.5)
    np.testing.assert_allclose(o, np.repeat(v.mean(axis=0, keepdims=True), 2, axis=0),
                               rtol=1e-13, atol=1e-15)


def pin_attention_two_keys_sigmoid(im):
    rng = np.random.default_rng(9)
    q = rng.standard_normal((1, 16))
    k = rng.standard_normal((2, 16))
    v = rng.standard_normal((2, 16))
    s = 0.25 * (q @ k.T)[0]
    p1 = 1.0 / (1.0 + math.exp(-(s[0] - s[1])))
    o, _ = im.attention(q, k, v, 0.25)
    np.testing.assert_allclose(o[0], p1 * v[0] + (1 - p1) * v[1], rtol=1e-13, atol=1e-15)


def pin_attention_permutation_and_mask(im):
    rng = np.random.default_rng(10)
    q = rng.standard_normal((4, 64))
    k = rng.standard_normal((20, 64))
    v = rng.standard_normal((20, 64))
    o, lse = im.attention(q, k, v, 0.125)
    perm = rng.permutation(20)
    o2, lse2 = im.attention(q, k[perm], v[perm], 0.125)
    np.testing.assert_allclose(o2, o, rtol=1e-13, atol=1e-15)
    # masking keys = deleting them
    keep = rng.random(20) < 0.5
    keep[3] = True
    vis = np.repeat(keep[None, :], 4, axis=0).astype(np.uint8)
    om, lm = im.attention(q, k, v, 0.125, vis)
    od, ld = im.attention(q, k[keep], v[keep], 0.125)
    np.testing.assert_allclose(om, od, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lm, ld, rtol=1e-13)
    # a fully masked row is zero with lse = -inf
    vis[1, :] = 0
    om, lm = im.attention(q, k, v, 0.125, vis)
    assert (om[1] == 0).all() and lm[1] == -math.inf


def pin_lse_merge(im):
    rng = np.random.default_rng(11)
    q = rng.standard_normal((3, 32))
    k = rng.standard_normal((40, 32))
    v = rng.standard_normal((40, 32))
    o, lse = im.attention(q, k, v, 0.3)
    cuts = [0, 5, 5, 17, 33, 40]  # includes an empty part
    parts_o, parts_l = [], []
    for a, b in zip(cuts[:-1], cuts[1:]):
        if a == b:
            parts_o.append(np.zeros((3, 32)))
            parts_l.append(np.full(3, -math.inf))
        else:
            po, pl = im.attention(q, k[a:b], v[a:b], 0.3)
            parts_o.append(po)
            parts_l.append(pl)
    mo, ml = im.lse_merge(np.stack(parts_o), np.stack(parts_l))
    np.testing.assert_allclose(mo, o, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ml, lse, rtol=1e-13)


ALL_PINS = [pin_bf16_decode, pin_rmsnorm_hand, pin_rmsnorm_mean_square, pin_rope_golden,
            pin_rope_isometry_and_identity, pin_rope_relativity, pin_rope_complex_form,
            pin_attention_golden, pin_attention_softmax_rows, pin_attention_vs_torch,
            pin_attention_single_key, pin_attention_identical_keys,
            pin_attention_two_keys_sigmoid, pin_attention_permutation_and_mask, pin_lse_merge]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(_impl())


# --------------------------------------------------------------------------- #
# planted mistakes: each wrong variant must fail at least one pin
# --------------------------------------------------------------------------- #
def _rope_generic(x, pos, band_pairs=(22, 21, 21), theta=10000.0, sign=1.0, bands=(0, 1, 2),
                  denom_shift=0):
    x = np.asarray(x, dtype=np.float64)
    pos = np.asarray(pos)
    out = np.empty_like(x)
    bp = list(band_pairs)
    starts = [0, bp[0], bp[0] + bp[1]]
    for p in range(x.shape[1] // 2):
        b = 0 if p < starts[1] else (1 if p < starts[2] else 2)
        pb = p - starts[b]
        ang = pos[:, bands[b]] * theta ** (-pb / (bp[b] + denom_shift))
        c, s = np.cos(ang), sign * np.sin(ang)
        a, bb = x[:, 2 * p], x[:, 2 * p + 1]
        out[:, 2 * p] = a * c - bb * s
        out[:, 2 * p + 1] = a * s + bb * c
    return out


def _attention_no_scale(q, k, v, scale, visible=None):
    return oracle.attention(q, k, v, 1.0, visible)


def _attention_transposed_v(q, k, v, scale, visible=None):
    v = np.asarray(v)
    if v.shape[0] == v.shape[1]:
        v = v.T
    return oracle.attention(q, k, v, scale, visible)


def _attention_ignores_mask(q, k, v, scale, visible=None):
    return oracle.attention(q, k, v, scale, None)


def _lse_merge_no_weights(o_parts, lse_parts):
    o = np.asarray(o_parts)
    l = np.asarray(lse_parts)
    alive = np.isfinite(l)[..., None]
    return (o * alive).sum(0) / np.maximum(alive.sum(0), 1), scipy.special.logsumexp(l, axis=0)


def _rmsnorm_no_eps(x, gamma, eps):
    return oracle.rmsnorm(x, gamma, 0.0)


def _rmsnorm_sum_not_mean(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt((x * x).sum(-1, keepdims=True) + eps) * np.asarray(gamma)


PLANTS = {
    "rope_sin_sign": dict(rope=lambda x, pos, bp=(22, 21, 21), th=10000.0:
                          _rope_generic(x, pos, bp, th, sign=-1.0)),
    "rope_bands_swapped": dict(rope=lambda x, pos, bp=(22, 21, 21), th=10000.0:
                               _rope_generic(x, pos, bp, th, bands=(0, 2, 1))),
    "rope_freq_denominator": dict(rope=lambda x, pos, bp=(22, 21, 21), th=10000.0:
                                  _rope_generic(x, pos, bp, th, denom_shift=1)),
    "attention_no_scale": dict(attention=_attention_no_scale),
    "attention_transposed_v": dict(attention=_attention_transposed_v),
    "attention_ignores_mask": dict(attention=_attention_ignores_mask),
    "lse_merge_unweighted": dict(lse_merge=_lse_merge_no_weights),
    "rmsnorm_no_eps": dict(rmsnorm=_rmsnorm_no_eps),
    "rmsnorm_sum_not_mean": dict(rmsnorm=_rmsnorm_sum_not_mean),
}


@pytest.mark.parametrize("plant", sorted(PLANTS))
def test_planted_mistakes(plant):
    im = _impl(**PLANTS[plant])
    failed = []
    for pin in ALL_PINS:
        try:
            pin(im)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"planted mistake {plant} passed every pin"


# --------------------------------------------------------------------------- #
# bf16 rounding of float64 values, and the attention sub-block
# --------------------------------------------------------------------------- #
def test_bf16_round_exact_values():
    """Ties to even and ordinary rounding at 8 significant bits, exact powers
    of two and signs, against hand-worked bit patterns; and agreement with
    the two-step float32 path where float32 holds the value exactly."""
    cases = [(1.0, 0x3F80), (1.0 + 2 ** -8, 0x3F80), (1.0 + 3 * 2 ** -8, 0x3F82),
             (1.0 + 2 ** -8 + 2 ** -30, 0x3F81), (-2.0, 0xC000), (0.0, 0x0000),
             (1.5 * 2 ** -100, 0x0DC0), (255.0, 0x437F), (255.5, 0x4380), (256.5, 0x4380),
             (257.0, 0x4380), (259.0, 0x4382)]
    got = oracle.bf16_round(np.array([c[0] for c in cases]))
    assert [int(g) for g in got] == [c[1] for c in cases], [hex(int(g)) for g in got]
    rng = np.random.default_rng(7)
    f = rng.standard_normal(4096).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    want = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    np.testing.assert_array_equal(oracle.bf16_round(f.astype(np.float64)), want)
