"""The oracle's logical cache and its unit attention, pinned on tiny inputs.

The unit attention is checked against an independent composition written
with torch float64 CPU ops: RMS-norm as x * rsqrt(mean(x^2) + eps) * gamma,
the rotation as complex multiplication by exp(i * angle), and torch's
scaled_dot_product_attention over the keys the block-causal mask leaves
visible (Wan-Streamer v0.2, Fig. 1 caption; Sec. 2.1; Sec. 3).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2607_04443_amd import synth

H, D = 2, 128


def _torch_prologue(bits, positions, gamma, eps):
    x = torch.from_numpy(synth.bf16_to_f32(bits).astype(np.float64))
    x = x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * torch.as_tensor(gamma,
                                                                               dtype=torch.float64)
    bands = np.repeat([0, 1, 2], [22, 21, 21])
    local = np.concatenate([np.arange(22) / 22, np.arange(21) / 21, np.arange(21) / 21])
    ang = torch.from_numpy(np.asarray(positions)[:, bands] * (10000.0 ** -local)[None, :])
    z = torch.complex(x[:, 0::2], x[:, 1::2]) * torch.polar(torch.ones_like(ang), ang)
    out = torch.empty_like(x)
    out[:, 0::2], out[:, 1::2] = z.real, z.imag
    return out


def _tiny_cache(rng):
    c = oracle.OracleCache(num_heads=H)
    segs = []
    k = synth.normal_bf16(rng, (3, H, D))
    v = synth.normal_bf16(rng, (3, H, D))
    c.append(0, oracle.KIND_COND, k, v, oracle.MODE_RAW)
    segs.append((0, oracle.KIND_COND, k, v, None))
    for u in range(3):
        for kind, n in ((oracle.KIND_VIDEO, 5), (oracle.KIND_AUDIO, 2)):
            k = synth.normal_bf16(rng, (n, H, D))
            v = synth.normal_bf16(rng, (n, H, D))
            pos = (synth.video_positions(u, (1, 5)) if kind == oracle.KIND_VIDEO
                   else synth.audio_positions(u, 2))
            c.append(u, kind, k, v, oracle.MODE_NORM_ROPE, pos, np.ones(D), 1e-6)
            segs.append((u, kind, k, v, pos))
    return c, segs


def _visible(segs, q_unit, min_unit, kind_mask):
    out = []
    for u, kind, k, v, pos in segs:
        if not (kind_mask >> kind) & 1 or u > q_unit:
            continue
        if kind != oracle.KIND_COND and u < min_unit:
            continue
        out.append((u, kind, k, v, pos))
    return out


@pytest.mark.parametrize("q_unit,min_unit,kind_mask", [
    (2, -(2 ** 31), 0b011), (2, -(2 ** 31), 0b111), (1, -(2 ** 31), 0b111), (2, 1, 0b011),
    (2, 2, 0b110), (0, -(2 ** 31), 0b001)])
def test_unit_attention_matches_torch_composition(q_unit, min_unit, kind_mask):
    rng = np.random.default_rng(100)
    cache, segs = _tiny_cache(rng)
    qb = synth.normal_bf16(rng, (4, H, D))
    qpos = synth.video_positions(q_unit, (1, 4))
    gq = synth.bf16_to_f32(synth.bf16_bits(1 + 0.1 * rng.standard_normal(D).astype(np.float32)))
    out, lse = oracle.unit_attention(cache, qb, q_unit, positions=qpos, gamma=gq, eps=1e-6,
                                     min_visible_unit=min_unit, kind_mask=kind_mask)
    vis = _visible(segs, q_unit, min_unit, kind_mask)
    for h in range(H):
        q = _torch_prologue(qb[:, h], qpos, gq, 1e-6)
        ks, vs = [], []
        for u, kind, k, v, pos in vis:
            if kind == oracle.KIND_COND:
                ks.append(torch.from_numpy(synth.bf16_to_f32(k[:, h]).astype(np.float64)))
            else:
                ks.append(_torch_prologue(k[:, h], pos, np.ones(D), 1e-6))
            vs.append(torch.from_numpy(synth.bf16_to_f32(v[:, h]).astype(np.float64)))
        ref = torch.nn.functional.scaled_dot_product_attention(
            q[None], torch.cat(ks)[None], torch.cat(vs)[None], scale=1 / math.sqrt(D))[0]
        np.testing.assert_allclose(out[:, h], ref.numpy(), rtol=1e-11, atol=1e-12)


def test_cache_rewrite_commit_evict():
    rng = np.random.default_rng(101)
    cache, segs = _tiny_cache(rng)
    order = [(s.unit, s.kind) for s in cache.segments]
    # rewriting an uncommitted unit keeps its place
    k = synth.normal_bf16(rng, (5, H, D))
    cache.append(1, oracle.KIND_VIDEO, k, k, oracle.MODE_NORM_ROPE,
                 synth.video_positions(1, (1, 5)), np.ones(D), 1e-6)
    assert [(s.unit, s.kind) for s in cache.segments] == order
    with pytest.raises(ValueError):
        cache.append(1, oracle.KIND_VIDEO, k[:4], k[:4], oracle.MODE_RAW)
    cache.commit(1)
    with pytest.raises(ValueError):
        cache.append(1, oracle.KIND_VIDEO, k, k, oracle.MODE_RAW)
    cache.evict_before(2)
    assert [(s.unit, s.kind) for s in cache.segments] == [(0, 0), (2, 1), (2, 2)]
    cache.release(0, oracle.KIND_COND)
    assert [(s.unit, s.kind) for s in cache.segments] == [(2, 1), (2, 2)]


def test_needle_per_page_selects_value():
    """A RAW key equal to c * Q'_i dominates: the output is that key's value."""
    rng = np.random.default_rng(102)
    cache = oracle.OracleCache(num_heads=1)
    q = synth.normal_bf16(rng, (1, 1, D))
    qp = oracle.query_prologue(q[:, 0], oracle.MODE_NORM_ROPE, np.zeros((1, 3), np.int32),
                               np.ones(D), 1e-6)
    k = synth.normal_bf16(rng, (64, 1, D))
    k[17, 0] = synth.bf16_bits(4.0 * qp[0])
    v = synth.normal_bf16(rng, (64, 1, D))
    cache.append(0, oracle.KIND_COND, k, v, oracle.MODE_RAW)
    out, _ = oracle.unit_attention(cache, q, 0, positions=np.zeros((1, 3), np.int32),
                                   kind_mask=0b001)
    np.testing.assert_allclose(out[0, 0], synth.bf16_to_f32(v[17, 0]), rtol=0, atol=1e-12)


def test_empty_visible_set_gives_zero():
    rng = np.random.default_rng(103)
    cache, _ = _tiny_cache(rng)
    qb = synth.normal_bf16(rng, (2, H, D))
    out, lse = oracle.unit_attention(cache, qb, 5, positions=synth.video_positions(5, (1, 2)),
                                     min_visible_unit=4, kind_mask=0b110)
    assert (out == 0).all() and np.isneginf(lse).all()


# --------------------------------------------------------------------------- #
# queries from several units in one call (block-causal across units)
# --------------------------------------------------------------------------- #
def test_groups_identical_keys_give_mean_of_visible_values():
    """Closed form: when every stored key is the same RAW vector, each query
    row's output is the plain mean of the values its group sees.  Three query
    groups (units 0, 1 and 2, the last with a window that hides units 0-1, and
    a fourth group that sees nothing) over a cache of one conditioning key and
    one key per unit."""
    rng = np.random.default_rng(301)
    key = synth.normal_bf16(rng, (1, H, D))
    c = oracle.OracleCache(num_heads=H)
    vals = {}
    for u, kind in ((0, oracle.KIND_COND), (0, oracle.KIND_VIDEO), (1, oracle.KIND_VIDEO),
                    (2, oracle.KIND_VIDEO)):
        v = synth.normal_bf16(rng, (1, H, D))
        vals[(u, kind)] = synth.bf16_to_f32(v[0]).astype(np.float64)
        c.append(u, kind, key, v, oracle.MODE_RAW)
    groups = [(0, -(2 ** 31), 0b011, 2), (1, -(2 ** 31), 0b011, 3), (2, 2, 0b011, 1),
              (1, 5, 0b010, 2)]
    q = synth.normal_bf16(rng, (8, H, D))
    out, lse = oracle.unit_attention_groups(c, q, groups, mode=oracle.MODE_RAW)
    want = [np.mean([vals[(0, 0)], vals[(0, 1)]], axis=0)] * 2 + \
        [np.mean([vals[(0, 0)], vals[(0, 1)], vals[(1, 1)]], axis=0)] * 3 + \
        [np.mean([vals[(0, 0)], vals[(2, 1)]], axis=0)] + [np.zeros((H, D))] * 2
    np.testing.assert_allclose(out, np.stack(want), rtol=0, atol=1e-12)
    assert np.isneginf(lse[:, 6:]).all() and np.isfinite(lse[:, :6]).all()


def test_groups_masked_equals_deleted():
    """I4 per group: a group's rows over the full cache equal the same rows
    over a cache from which the segments its mask hides were deleted."""
    rng = np.random.default_rng(302)
    cache, segs = _tiny_cache(rng)
    groups = [(0, -(2 ** 31), 0b011, 3), (2, 1, 0b111, 4), (1, -(2 ** 31), 0b101, 2)]
    qb = synth.normal_bf16(rng, (9, H, D))
    qpos = np.concatenate([synth.video_positions(g[0], (1, g[3])) for g in groups])
    out, lse = oracle.unit_attention_groups(cache, qb, groups, positions=qpos, gamma=np.ones(D))
    r0 = 0
    for q_unit, min_unit, kind_mask, n in groups:
        pruned = oracle.OracleCache(num_heads=H)
        for u, kind, k, v, pos in _visible(segs, q_unit, min_unit, kind_mask):
            pruned.append(u, kind, k, v, oracle.MODE_RAW if kind == oracle.KIND_COND
                          else oracle.MODE_NORM_ROPE, pos, np.ones(D), 1e-6)
        o, l = oracle.unit_attention(pruned, qb[r0:r0 + n], q_unit, positions=qpos[r0:r0 + n],
                                     gamma=np.ones(D), kind_mask=0b111)
        np.testing.assert_allclose(out[r0:r0 + n], o, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse[:, r0:r0 + n], l, rtol=0, atol=1e-12)
        r0 += n


def test_groups_match_per_row_visibility_matrix():
    """The groups' result against dense attention over every stored key with
    an explicit per-(row, key) visibility matrix (the C routine's mask path,
    not the segment selection), on the tiny cache: rows of units 0, 1 and 2
    with different windows and kinds."""
    rng = np.random.default_rng(303)
    cache, segs = _tiny_cache(rng)
    groups = [(2, 2, 0b111, 2), (0, -(2 ** 31), 0b011, 3), (1, 1, 0b110, 2)]
    qb = synth.normal_bf16(rng, (7, H, D))
    qpos = np.concatenate([synth.video_positions(g[0], (1, g[3])) for g in groups])
    out, _ = oracle.unit_attention_groups(cache, qb, groups, positions=qpos, gamma=np.ones(D))
    row_group = np.repeat(np.arange(len(groups)), [g[3] for g in groups])
    for h in range(H):
        ks, vs, labels = [], [], []
        for s in cache.segments:
            k, v = cache.segment_kv(s, h)
            ks.append(k)
            vs.append(v)
            labels += [(s.unit, s.kind)] * k.shape[0]
        k, v = np.concatenate(ks), np.concatenate(vs)
        vis = np.zeros((qb.shape[0], k.shape[0]), np.uint8)
        for i, g in enumerate(row_group):
            q_unit, min_unit, kind_mask, _ = groups[g]
            for j, (u, kind) in enumerate(labels):
                vis[i, j] = ((kind_mask >> kind) & 1) and u <= q_unit and \
                    (kind == oracle.KIND_COND or u >= min_unit)
        q = oracle.query_prologue(qb[:, h], oracle.MODE_NORM_ROPE, qpos, np.ones(D), 1e-6)
        o, _ = oracle.attention(q, k, v, 1.0 / math.sqrt(D), visible=vis)
        np.testing.assert_allclose(out[:, h], o, rtol=0, atol=1e-12)


# --------------------------------------------------------------------------- #
# the attention sub-block of one performer layer (projections around the attention)
# --------------------------------------------------------------------------- #
def test_block_step_with_selection_weights_reduces_to_attention():
    """With W_qkv = [I I I] (Q = K = V = X, head h in columns 128 h ..) and
    W_out = I, the sub-block's output is the unit attention of X's bits used
    as Q, K and V: the projection's column layout, the bf16 rounding of its
    output (exact here), the append and the two query sets are pinned by the
    already-pinned unit attention."""
    rng = np.random.default_rng(11)
    H, D, nv, na = 2, 128, 5, 2
    hid, n = H * D, nv + na
    x = synth.normal_bf16(rng, (n, hid))
    w3 = oracle.bf16_round(np.concatenate([np.eye(hid)] * 3, axis=1))
    w_out = oracle.bf16_round(np.eye(hid))
    kc, vc = synth.normal_bf16(rng, (3, H, D)), synth.normal_bf16(rng, (3, H, D))
    vpos, apos = synth.video_positions(1, (1, nv)), synth.audio_positions(1, na)
    g = np.ones(D)

    def fresh():
        c = oracle.OracleCache(num_heads=H)
        c.append(0, oracle.KIND_COND, kc, vc, oracle.MODE_RAW)
        return c

    y, o = oracle.block_step(fresh(), x, nv, w3, w_out, 1, video_positions=vpos,
                             audio_positions=apos, gamma_q=g, gamma_k=g, eps=1e-6,
                             video_mask=(-(2 ** 31), 0b011), audio_mask=(-(2 ** 31), 0b111))
    c2 = fresh()
    xb = x.reshape(n, H, D)
    c2.append(1, oracle.KIND_VIDEO, xb[:nv], xb[:nv], oracle.MODE_NORM_ROPE, vpos, g, 1e-6)
    c2.append(1, oracle.KIND_AUDIO, xb[nv:], xb[nv:], oracle.MODE_NORM_ROPE, apos, g, 1e-6)
    ov, _ = oracle.unit_attention(c2, xb[:nv], 1, positions=vpos, gamma=g, kind_mask=0b011)
    oa, _ = oracle.unit_attention(c2, xb[nv:], 1, positions=apos, gamma=g, kind_mask=0b111)
    np.testing.assert_allclose(o, np.concatenate([ov, oa]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(y, np.concatenate([ov, oa]).reshape(n, hid), rtol=0, atol=1e-12)


def test_block_step_projections_are_linear():
    """Y scales with W_out (Y(2 W_out) = 2 Y(W_out), exact in binary), and a
    zero W_qkv makes every logit zero: O is then the plain mean of the values
    each query set sees, i.e. of the conditioning values only (the unit's own
    values are zero) weighted by their count."""
    rng = np.random.default_rng(12)
    H, D, nv, na = 2, 128, 4, 1
    hid, n = H * D, 5
    x = synth.normal_bf16(rng, (n, hid))
    w_qkv = synth.bf16_bits(rng.standard_normal((hid, 3 * hid)).astype(np.float32) / 16)
    w_out = synth.bf16_bits(rng.standard_normal((hid, hid)).astype(np.float32) / 16)
    w_out2 = oracle.bf16_round(2.0 * oracle.bf16_decode(w_out))
    kc, vc = synth.normal_bf16(rng, (3, H, D)), synth.normal_bf16(rng, (3, H, D))
    vpos, apos = synth.video_positions(0, (1, nv)), synth.audio_positions(0, na)
    g = np.ones(D)
    kw = dict(video_positions=vpos, audio_positions=apos, gamma_q=g, gamma_k=g, eps=1e-6,
              video_mask=(-(2 ** 31), 0b011), audio_mask=(-(2 ** 31), 0b111))
    outs = []
    for w in (w_out, w_out2):
        c = oracle.OracleCache(num_heads=H)
        c.append(0, oracle.KIND_COND, kc, vc, oracle.MODE_RAW)
        outs.append(oracle.block_step(c, x, nv, w_qkv, w, 0, **kw)[0])
    np.testing.assert_allclose(outs[1], 2.0 * outs[0], rtol=1e-14, atol=1e-14)
    c = oracle.OracleCache(num_heads=H)
    c.append(0, oracle.KIND_COND, np.zeros_like(kc), vc, oracle.MODE_RAW)
    _, o = oracle.block_step(c, x, nv, np.zeros_like(w_qkv), w_out, 0, **kw)
    vcond = oracle.bf16_decode(vc)
    np.testing.assert_allclose(o[:nv], np.broadcast_to(vcond.sum(0) / (3 + nv), (nv, H, D)),
                               rtol=0, atol=1e-12)
    np.testing.assert_allclose(o[nv:], np.broadcast_to(vcond.sum(0) / (3 + nv + na), (na, H, D)),
                               rtol=0, atol=1e-12)


@pytest.mark.parametrize("gamma_q", [1.0, 4.0])
def test_rounding_bound_covers_the_bf16_rounding_model(gamma_q):
    """helpers.rounding_bound (the GPU parity tests' independent elementwise
    gate) covers an emulation of the GPU path's roundings written here from
    the model, on a cache of a RAW slice and three NORM_ROPE units: Q'' and
    K' rounded to bf16, softmax weights rounded to bf16 against each key
    range's maximum (the shift cancels in the weights' relative rounding),
    two key ranges written as bf16 partials and merged by log-sum-exp, the
    output rounded to bf16."""
    from helpers import rounding_bound
    rng = np.random.Generator(np.random.PCG64(synth.SEED_BASE + 71))
    grid = (6, 8)
    c = oracle.OracleCache(num_heads=H)
    ck, cv = synth.normal_bf16(rng, (40, H, D)), synth.normal_bf16(rng, (40, H, D))
    c.append(0, oracle.KIND_COND, ck, cv, oracle.MODE_RAW)
    ones = np.ones(D)
    for u in range(3):
        k, v = synth.normal_bf16(rng, (48, H, D)), synth.normal_bf16(rng, (48, H, D))
        c.append(u, oracle.KIND_VIDEO, k, v, oracle.MODE_NORM_ROPE, synth.video_positions(u, grid), ones, 1e-6)
    q = synth.normal_bf16(rng, (24, H, D))
    qpos = synth.video_positions(2, grid)[:24]
    gq = np.full(D, gamma_q)
    kw = dict(positions=qpos, gamma=gq, eps=1e-6, kind_mask=0b011)
    exact, _ = oracle.unit_attention(c, q, 2, **kw)
    bound = rounding_bound(c, q, 2, **kw)
    scale = 1.0 / np.sqrt(D)
    log2e = 1.0 / np.log(2.0)

    def rnd(x):
        return oracle.bf16_decode(oracle.bf16_round(x))

    worst = 0.0
    for h in range(H):
        qh = oracle.query_prologue(q[:, h, :], oracle.MODE_NORM_ROPE, qpos, gq, 1e-6)
        k, v = c.keys_values(h, 2, -(2 ** 31), 0b011)
        s = rnd(qh * scale * log2e) @ rnd(k).T  # log2 domain
        half = k.shape[0] // 2
        parts = []
        for lo, hi in ((0, half), (half, k.shape[0])):
            m = s[:, lo:hi].max(axis=1, keepdims=True)
            p = rnd(np.exp2(s[:, lo:hi] - m))
            l = p.sum(axis=1, keepdims=True)
            parts.append((rnd(p @ v[lo:hi] / l), m[:, 0] + np.log2(l[:, 0])))
        mx = np.maximum(parts[0][1], parts[1][1])
        w = [np.exp2(lse - mx)[:, None] for _, lse in parts]
        emu = rnd((w[0] * parts[0][0] + w[1] * parts[1][0]) / (w[0] + w[1]))
        err = np.abs(emu - exact[:, h, :])
        assert (err <= bound[:, h, :]).all(), float((err / bound[:, h, :]).max())
        worst = max(worst, float((err / bound[:, h, :]).max()))
    print(f"gamma_q={gamma_q}: worst error / bound = {worst:.3f}")
    assert 0.0 < worst < 1.0
    # and the bound is far below the outputs' spread: it can still tell a wrong row
    assert bound.max() < 0.25 * np.abs(exact).max()
