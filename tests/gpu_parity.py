"""Helpers of the GPU parity tests: run the HIP path through the C ABI and
compare with the oracle on the same seeded inputs.

Comparison rules (tolerances derived in the design doc):
  records   oracle.pack(GPU codes, GPU metadata) reproduces the GPU words exactly
            (padding included); oracle-packed records unpack on the GPU exactly;
  metadata  fp16 zero-point/scale bit-equal, except adjacent fp16 values whose
            oracle pre-rounding value lies within META_TOL (relative) of the
            midpoint, at a rate of at most META_FRAC of (token, group) pairs
            (binomial bound on the sample, rate_allowance);
  codes     under the GPU's metadata, >= 99.99% equal; every mismatch is one level
            with the oracle's u within TIE_TOL of a half-integer;
  decode    relative L2 per stream <= 1e-3 vs the oracle's own encode/decode, and
            <= 1e-6 vs the oracle decode of the GPU's bytes;
  attention relative L2 per (sequence, query head) <= 2e-3 vs the oracle's own
            cache, <= ATTN_SAME_TOL vs the oracle over the GPU's bytes.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

import oracle as O
import paper_2608_07915_amd as S
import synth

TIE_TOL = 1e-3
META_TOL = 1e-5
META_FRAC = 1e-3
ATTN_SAME_TOL = 1e-5


def sparams(p: O.Params) -> S.Params:
    return S.Params(p.head_dim, p.group_size, p.b_max, p.meta_bits, p.centered, p.ratio, p.budget_bits)


def to_device(x: np.ndarray, dtype: str):
    """numpy stored values (float32 array or uint16 bf16 bits) -> torch device tensor."""
    import torch
    if dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).cuda().view(torch.bfloat16)


def values_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    return (x if dtype == "f32" else synth.bf16_bits_to_f32(x)).astype(np.float64)


def host_values(t) -> np.ndarray:
    """Device tensor (fp32 or bf16) -> numpy float64 values."""
    import torch
    return t.float().cpu().numpy().astype(np.float64) if t.dtype == torch.bfloat16 else t.cpu().numpy().astype(np.float64)


def records_of(packed, s: int, t0: int, n: int, t_cap: int, W: int) -> np.ndarray:
    """Logical records [n, W] of stream s, slots [t0, t0+n), from the tiled device words."""
    words = packed.cpu().numpy().view(np.uint32)
    t = np.arange(t0, t0 + n)
    out = np.zeros((n, W), dtype=np.uint32)
    for w in range(W):
        out[:, w] = words[O.physical_index(s, t, w, t_cap, W)]
    return out


def codec_state(codec: S.Codec, s: int):
    return (codec.basis[s].cpu().numpy(), codec.mean[s].cpu().numpy(),
            [int(b) for b in codec.bits[s].cpu().numpy()])


@dataclass
class EncodeReport:
    meta_mismatch: float
    code_mismatch: float
    n_codes: int
    meta_dist: float = 0.0   # largest relative distance of a differing fp16 value's pre-rounding value to the midpoint


def rate_allowance(n: int, rate: float, p_false: float = 1e-6) -> int:
    """Largest count of events that a rate of at most `rate` over n trials exceeds
    with probability below p_false (one-sided binomial bound): the bar for a mismatch
    rate measured on a finite sample."""
    from scipy.stats import binom
    return int(binom.isf(p_false, n, rate)) if n > 0 else 0


def _fp16_boundary_dist(pre: np.ndarray, got_bits: np.ndarray, want_bits: np.ndarray) -> np.ndarray:
    """Relative distance of `pre` to the rounding midpoint of two fp16 values; inf
    unless the two are adjacent."""
    a = O.f16_bits_to_f64(got_bits)
    b = O.f16_bits_to_f64(want_bits)
    adjacent = np.abs(got_bits.astype(np.int64) - want_bits.astype(np.int64)) == 1
    mid = 0.5 * (a + b)
    dist = np.abs(pre - mid) / np.maximum(np.abs(mid), 2.0 ** -24)
    return np.where(adjacent, dist, np.inf)


def check_encoded_stream(x64: np.ndarray, basis, mean, bits, p: O.Params, rec_gpu: np.ndarray,
                         dot_bound: bool = False, scale=None) -> EncodeReport:
    """P3-P5 for one stream: x64 [n, d] input values, rec_gpu [n, W] GPU records.

    dot_bound (long projections, d > 128): a code may differ only where the oracle's
    u = (c - z)/s lies within the forward error bound of the GPU's fp32 projection of
    a half-integer: |dc| <= n_r 2^-24 sum_k |x_k V_kj| + 2^-22 |c| (n_r = d/16 + 16
    sequential roundings: 16-term MFMA steps chained over d, then the chunk adds).
    scale: the square-root split factors f_j (the cached coordinate is (x V - m)_j f_j)."""
    W = O.record_words(p)
    coef = x64 @ basis.astype(np.float64) - mean.astype(np.float64)[None, :]
    fs = np.ones(coef.shape[1]) if scale is None else np.asarray(scale, np.float64)
    coef = coef * fs[None, :]
    codes_o, meta_o = O.quantize(coef, bits, p)
    codes_g, meta_g = O.unpack(rec_gpu, bits, p)
    # P5: re-packing the GPU's codes and metadata reproduces its words exactly
    assert np.array_equal(O.pack(codes_g, meta_g, bits, p), rec_gpu), "GPU record words are not the packed codes"
    n_pairs = 0
    bad_meta = 0
    meta_dist = 0.0
    g = p.group_size
    for G, b in enumerate(bits):
        if b == 0:
            continue
        c = coef[:, G * g:(G + 1) * g]
        lo, hi = c.min(axis=1), c.max(axis=1)
        zg, zo = meta_g[:, G] >> 16, meta_o[:, G] >> 16
        sg, so = meta_g[:, G] & 0xFFFF, meta_o[:, G] & 0xFFFF
        dz = zg != zo
        dist_z = _fp16_boundary_dist(lo[dz], zg[dz], zo[dz])
        ds = (sg != so) & ~dz
        pre_s = np.maximum(hi - O.f16_bits_to_f64(zo), 0.0) / float((1 << b) - 1)
        dist_s = _fp16_boundary_dist(pre_s[ds], sg[ds], so[ds])
        for dist in (dist_z, dist_s):
            if dist.size:
                meta_dist = max(meta_dist, float(dist.max()))
        bad_meta += int(np.count_nonzero(dz | (sg != so)))
        n_pairs += c.shape[0]
    meta_frac = bad_meta / max(n_pairs, 1)
    assert meta_dist <= META_TOL, f"fp16 metadata differs {meta_dist:.3g} (relative) away from a rounding midpoint"
    assert bad_meta <= rate_allowance(n_pairs, META_FRAC), f"metadata mismatch fraction {meta_frac} of {n_pairs}"
    # P4: codes under the GPU's metadata
    codes_r, u = O.quantize_given_meta(coef, meta_g, bits, p)
    kept = np.repeat(np.array(bits) > 0, g)
    diff = codes_r[:, kept].astype(np.int64) - codes_g[:, kept].astype(np.int64)
    mism = diff != 0
    n_codes = int(mism.size)
    frac = float(np.count_nonzero(mism)) / max(n_codes, 1)
    if np.any(mism):
        uu = u[:, kept][mism]
        assert np.all(np.abs(diff[mism]) == 1), "code off by more than one level"
        if dot_bound:
            d = x64.shape[1]
            A = np.abs(x64) @ np.abs(basis.astype(np.float64))
            s_tok = np.zeros_like(coef)
            for G, b in enumerate(bits):
                if b:
                    s_tok[:, G * g:(G + 1) * g] = O.f16_bits_to_f64(meta_g[:, G] & 0xFFFF)[:, None]
            dc = (d / 16 + 16) * 2.0 ** -24 * A * fs[None, :] + 2.0 ** -22 * np.abs(coef)
            bound = (dc[:, kept] / np.where(s_tok[:, kept] > 0, s_tok[:, kept], np.inf))[mism] + 1e-6
            assert np.all(np.abs(uu - np.floor(uu) - 0.5) <= bound), "code mismatch outside the fp32 projection bound"
        else:
            assert np.all(np.abs(uu - np.floor(uu) - 0.5) <= TIE_TOL), "code mismatch away from a rounding tie"
    assert frac <= 1e-4, f"code mismatch fraction {frac}"
    assert np.all(codes_g[:, ~kept] == 0)
    return EncodeReport(meta_frac, frac, n_codes, meta_dist)


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def oracle_attention(q64: np.ndarray, kh: np.ndarray, vh: np.ndarray) -> np.ndarray:
    """q [Hq, d]; kh, vh [Hkv, T, d] reconstructed caches -> [Hq, d] (Mode A)."""
    return O.attention_mode_a(q64, kh, vh)


def fit_and_encode(x_dev, p: O.Params, t_cap: int, fit: bool = True, codec=None):
    """Fit (unless a codec is given) and encode x_dev [S, T, d] into a new packed cache."""
    import torch
    if codec is None:
        codec = S.Codec(sparams(p), x_dev.shape[0])
    if fit:
        S.spectra_fit_basis(codec, x_dev)
    packed = codec.empty_packed(t_cap)
    S.spectra_encode(codec, x_dev, 0, packed, t_cap)
    torch.cuda.synchronize()
    return codec, packed
