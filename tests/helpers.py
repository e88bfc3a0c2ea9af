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

    def close(self):
        self.cache.close()


def errors(got, ref):
    d = np.abs(got - ref)
    return dict(max=float(d.max()), mean=float(d.mean()),
                frob=float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)))


def assert_gates(got, ref, strict=True, label="", scale=1.0):
    assert np.isfinite(got).all(), f"{label}: non-finite output"
    e = errors(got, ref)
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
