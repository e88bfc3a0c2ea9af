"""Shared helpers of the GPU parity tests: load a seeded workload into both
the HIP cache (through the C ABI binding) and the oracle's logical cache, and
compare outputs against the oracle with the parity gates."""
import numpy as np

import oracle
from paper_2607_04443_amd import synth

# Gates.  Contract: max |err| <= 2e-2 and mean |err| <= 2e-3 on bf16 outputs.
# Internal, stricter, and scale-free: relative Frobenius <= 1e-2 (one dropped
# 64-key page at 8.5k keys gives ~9%), and elementwise
#   |err| <= 2^-7 |ref| + 0.08 rms(ref)
# (one bf16 ulp of output rounding, plus a term sized to ~3x the largest
# logit/P rounding error seen at 124..30616 keys; a wrong row, tile or page
# errs by O(|ref|) and fails it).  A workload whose logits are k times wider
# (gamma_q = k) scales the contract's absolute gates by k.
CONTRACT_MAX, CONTRACT_MEAN = 2e-2, 2e-3
STRICT_FROB, STRICT_REL, STRICT_RMS = 1e-2, 2.0 ** -7, 0.08

# Independent of any kernel output: a first-order bound on |GPU - exact| per
# output element, from the roundings the GPU path makes (bf16 unit roundoff
# u = 2^-9) and the oracle's own fp64 data.  For query row q, key k, dim d,
# with p the exact softmax weights, O the exact output and s the logit scale:
#   output and key-range partials rounded to bf16     2u * A_qd,  A = sum_k p|v_kd|
#   P rounded to bf16 before P*V (and its row sum)     u  * sum_k p (|v_kd| + |O_qd|)
#   Q'' and K' rounded to bf16: a logit errs by at most
#     D_qk = 2u * s * sum_i |q'_i k'_i|, which moves O by sum_k p D_qk (|v_kd| + |O_qd|)
#   fp32 sums of n_k terms (row sum, P*V)              2 n_k 2^-24 * A_qd
# (to first order; 5% margin for the second-order terms).  Rigorous but
# loose: it assumes every rounding error aligned.  The Frobenius gate above
# follows the same model's rms (about 3e-3 at 8.5k keys, gate 1e-2).
ROUND_U = 2.0 ** -9


def to_dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def from_dev(t):
    return t.detach().cpu().view(__import__("torch").int16).numpy().view(np.uint16)


def bf16_f64(bits):
    return synth.bf16_to_f32(bits).astype(np.float64)


def dev_i32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()


def dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


class Loaded:
    """A workload written into a GPU cache and mirrored in an oracle cache."""

    def __init__(self, ws, wl, max_pages=None, step=0, max_q_tokens=1024, keep=None,
                 step_segments=True):
        cfg = wl.config
        if max_pages is None:
            max_pages = 8 + (cfg.hist + 2) * (cfg.unit_tokens // 64 + 3) + cfg.cond // 64
        self.ws, self.wl = ws, wl
        self.cache = ws.Cache(cfg.heads, max_pages, max_q_tokens=max_q_tokens)
        self.ocache = oracle.OracleCache(num_heads=cfg.heads)
        self.gk = dev_f32(wl.gamma_k)
        self.gq = dev_f32(wl.gamma_q)
        self._keep = [] if keep is None else keep
        for seg in wl.cached:
            self.append(seg)
        if wl.steps and step_segments:
            for seg in wl.steps[step].segments:
                self.append(seg)

    def append(self, seg):
        k, v = to_dev(seg.k), to_dev(seg.v)
        pos = dev_i32(seg.positions) if seg.positions is not None else None
        self._keep += [k, v, pos]
        if seg.mode == synth.MODE_RAW:
            self.cache.append(seg.unit, seg.kind, k, v, self.ws.WS_APPEND_RAW)
            self.ocache.append(seg.unit, seg.kind, seg.k, seg.v, oracle.MODE_RAW)
        else:
            self.cache.append(seg.unit, seg.kind, k, v, self.ws.WS_APPEND_NORM_ROPE, pos, self.gk,
                              self.wl.eps)
            self.ocache.append(seg.unit, seg.kind, seg.k, seg.v, oracle.MODE_NORM_ROPE,
                               seg.positions, self.wl.gamma_k.astype(np.float64), self.wl.eps)

    def run(self, path, q_bits, q_pos, q_unit, kinds, min_unit=-(2 ** 31), mode=None):
        import torch
        ws = self.ws
        q = to_dev(q_bits)
        out = torch.full_like(q, float("nan"))
        pos = dev_i32(q_pos)
        mask = ws.mask_spec(q_unit, min_unit, kinds)
        mode = ws.WS_APPEND_NORM_ROPE if mode is None else mode
        fn = self.cache.unit_attention if path == "video" else self.cache.audio_attention
        fn(q, out, mask, mode, pos, self.gq, self.wl.eps)
        torch.cuda.synchronize()
        return bf16_f64(from_dev(out))

    def oracle(self, q_bits, q_pos, q_unit, kinds, heads=None, min_unit=-(2 ** 31), mode=None):
        kind_mask = sum(1 << k for k in kinds)
        mode = oracle.MODE_NORM_ROPE if mode is None else mode
        out, _ = oracle.unit_attention(self.ocache, q_bits, q_unit, mode=mode, positions=q_pos,
                                       gamma=self.wl.gamma_q.astype(np.float64), eps=self.wl.eps,
                                       min_visible_unit=min_unit, kind_mask=kind_mask,
                                       heads=heads)
        return out

    def bound(self, q_bits, q_pos, q_unit, kinds, heads=None, min_unit=-(2 ** 31), mode=None):
        """rounding_bound for the same call as oracle()."""
        mode = oracle.MODE_NORM_ROPE if mode is None else mode
        return rounding_bound(self.ocache, q_bits, q_unit, mode=mode, positions=q_pos,
                              gamma=self.wl.gamma_q.astype(np.float64), eps=self.wl.eps,
                              min_visible_unit=min_unit, kind_mask=sum(1 << k for k in kinds), heads=heads)

    def close(self):
        self.cache.close()


def rounding_bound(ocache, q_bits, q_unit, *, mode=oracle.MODE_NORM_ROPE, positions=None, gamma=None,
                   eps=1e-6, scale=None, min_visible_unit=-(2 ** 31), kind_mask=0b011, heads=None):
    """The elementwise bound above for oracle.unit_attention's output with the
    same arguments: [n_q, len(heads), D] float64."""
    q_bits = np.asarray(q_bits, dtype=np.uint16)
    n_q, H, D = q_bits.shape
    heads = list(range(H)) if heads is None else list(heads)
    scale = 1.0 / np.sqrt(D) if scale is None else scale
    gamma = np.ones(D) if gamma is None else gamma
    u = ROUND_U
    out = np.zeros((n_q, len(heads), D))
    for hi, h in enumerate(heads):
        q = oracle.query_prologue(q_bits[:, h, :], mode, positions, gamma, eps, ocache.band_pairs, ocache.theta)
        k, v = ocache.keys_values(h, q_unit, min_visible_unit, kind_mask)
        n_k = k.shape[0]
        if n_k == 0:
            continue
        # float32 is ample for a bound (its own error is ~1e-7 relative)
        q32, k32, v32 = (x.astype(np.float32) for x in (q, k, v))
        logit = np.float32(scale) * (q32 @ k32.T)
        logit -= logit.max(axis=1, keepdims=True)
        p = np.exp(logit, out=logit)
        p /= p.sum(axis=1, keepdims=True)
        av = np.abs(v32)
        o = np.abs(p @ v32)
        a = p @ av
        w = np.abs(q32) @ np.abs(k32).T
        w *= np.float32(2 * u * scale)
        w += np.float32(u)
        w *= p
        b = w @ av + o * w.sum(axis=1, keepdims=True)
        out[:, hi, :] = 1.05 * ((2 * u + 2 * n_k * 2.0 ** -24) * a + b) + 1e-7
    return out


def errors(got, ref):
    d = np.abs(got - ref)
    return dict(max=float(d.max()), mean=float(d.mean()),
                frob=float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)))


def assert_gates(got, ref, strict=True, label="", scale=1.0, bound=None):
    """The contract gates; with strict, the Frobenius gate and the fitted
    elementwise one; with a bound (rounding_bound), |got - ref| <= bound
    everywhere as well."""
    assert np.isfinite(got).all(), f"{label}: non-finite output"
    e = errors(got, ref)
    if bound is not None:
        r = np.abs(got - ref) / bound
        e["bound_ratio"] = float(r.max())
        assert e["bound_ratio"] <= 1.0, f"{label}: rounding bound exceeded: {e}"
    rms = float(np.sqrt(np.mean(ref * ref)))
    bound = STRICT_REL * np.abs(ref) + STRICT_RMS * rms
    ratio = np.abs(got - ref) / np.maximum(bound, 1e-30)
    i = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
    e["worst_ratio"] = float(ratio[i])
    e["worst_ref"] = float(ref[i])
    msg = f"{label}: {e}"
    assert e["max"] <= scale * CONTRACT_MAX and e["mean"] <= scale * CONTRACT_MEAN, msg
    if strict:
        assert e["frob"] <= STRICT_FROB and e["worst_ratio"] <= 1.0, msg
    return e
