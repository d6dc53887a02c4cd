"""Oracle of the SPECTRA codec: fit, allocation, quantize, pack, decode, attention.

Test infrastructure (see the package docstring). float64 throughout unless a
step is defined by a narrower format (fp32 basis storage, fp16 metadata).

Paper references are to arXiv 2608.07915:
  Sec. 3.1  caching a latent from a second-moment eigenbasis (Eqs. gsvd,
            second-moment-latent) and centering by measured means;
  Sec. 3.2  rate-distortion quantization: Eq. (waterfill), groups of g
            coordinates sharing one width, per-token min/max with an fp16 scale
            and zero-point per group, zero-bit groups stored as nothing;
  Sec. 3.3  Mode A (reconstruct then attend) and Mode B (latent attention);
  App. D    reverse water-filling derivation;
  App. E    latent-space attention identity q k^T = (q W_up^T) c^T;
  App. F    effective compression ratio 16 / b_eff counting payload and metadata.

Readings where the paper is silent are fixed in ``Params`` and in each
function's docstring (basis from the cache's own second moment per KV head,
orthonormal coefficients, exact integer allocation, record format).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from itertools import product
from typing import Optional, List, Sequence, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# Parameters and record geometry
# ----------------------------------------------------------------------------
@dataclass(frozen=True)
class Params:
    head_dim: int = 128
    group_size: int = 32
    b_max: int = 8
    meta_bits: int = 32        # fp16 scale + fp16 zero-point per kept group per token
    centered: bool = False     # False: eigenbasis of the uncentered second moment (Sec. 3.1)
    ratio: float = 8.0         # effective compression vs fp16 (App. F)
    budget_bits: int = 0       # >0 overrides ratio: bits per token per stream incl. metadata

    @property
    def n_groups(self) -> int:
        return self.head_dim // self.group_size


def record_budget_bits(p: Params) -> int:
    """Bits per token per stream, metadata included (App. F: ratio = 16 / b_eff).

    R = budget_bits if given, else floor(16 d / ratio + 1e-6); the 1e-6 guard
    keeps a ratio like 16/9 from flooring 1152 to 1151.
    """
    if p.budget_bits > 0:
        return int(p.budget_bits)
    return int(math.floor(16.0 * p.head_dim / p.ratio + 1e-6))


def record_words(p: Params) -> int:
    """Record width W in 32-bit words: floor(R / 32)."""
    return record_budget_bits(p) // 32


def split_budget(p: Params, kappa: float) -> Tuple[Params, Params]:
    """Asymmetric key/value split of the per-token budget (Sec. 3.1: r_k = kappa B,
    r_v = (1 - kappa) B; App. F: rates count payload and metadata).

    Reading: the allocation turns a bit budget into a kept rank (zero-bit groups
    are dropped, Sec. 3.2), so the paper's split of the rank budget between the
    key and value paths is realised as a split of the two records' combined
    per-token budget 2R. Keys get R_k = 32 * floor(kappa * 2R / 32 + 1/2) bits
    (whole words, nearest, halves up) and values R_v = 2R - R_k; each tensor is
    then allocated on its own budget. kappa = 1/2 gives the symmetric setting
    (App. F: 1/2 for the water-filling variant, 1/4 for the low-rank one). Both
    budgets must pay for at least one group (g + meta_bits bits).
    Returns (params_k, params_v) with budget_bits set.
    """
    if not (0.0 < kappa < 1.0):
        raise ValueError("kappa must lie in (0, 1)")
    total = 2 * record_budget_bits(p)
    rk = 32 * int(math.floor(kappa * total / 32 + 0.5))
    rv = total - rk
    one = p.group_size + p.meta_bits
    if rk < one or rv < one:
        raise ValueError("split leaves a tensor without a whole group")
    return replace(p, budget_bits=rk), replace(p, budget_bits=rv)


# ----------------------------------------------------------------------------
# fp16 helpers (IEEE binary16, round to nearest even, saturating at +-65504)
# ----------------------------------------------------------------------------
def fp16_rne_sat(x) -> np.ndarray:
    """Round float64 values once to binary16 (RNE), saturating at the largest finite."""
    x = np.clip(np.asarray(x, dtype=np.float64), -65504.0, 65504.0)
    return x.astype(np.float16)


def fp16_bits(h: np.ndarray) -> np.ndarray:
    return np.asarray(h, dtype=np.float16).view(np.uint16).astype(np.uint32)


def f16_bits_to_f64(b) -> np.ndarray:
    return np.asarray(b, dtype=np.uint32).astype(np.uint16).view(np.float16).astype(np.float64)


# ----------------------------------------------------------------------------
# O-1: fit (Sec. 3.1, Eqs. gsvd and second-moment-latent)
# ----------------------------------------------------------------------------
@dataclass
class FitResult:
    basis: np.ndarray     # [d, d] float32, column j = direction j (descending energy)
    mean: np.ndarray      # [d] float32, coefficient-space mean m = mu_hat . V32
    var: np.ndarray       # [d] float64, centered marginal variance of coefficient j
    eigvals: np.ndarray   # [d] float64, descending
    second_moment: np.ndarray  # [d, d] float64, the matrix that was diagonalised
    mu: np.ndarray        # [d] float64 token mean
    cov: np.ndarray       # [d, d] float64 centered covariance
    scale: Optional[np.ndarray] = None  # [d] float32 square-root split factors f_j (None: orthonormal latent)


def fit(x: np.ndarray, p: Params, latent_scale: bool = False) -> FitResult:
    """Per-stream spectral basis.

    Sec. 3.1 builds the latent from the G-weighted SVD M = G^{1/2} W = U S V^T.
    Because a key is k = h W, E[k^T k] = W^T G W = M^T M = V S^2 V^T: the right
    singular vectors are the eigenvectors of the keys' own uncentered second
    moment, and the rank-r reconstruction h W_down W_up equals k V_r V_r^T.
    This oracle therefore fits the eigenbasis of each stream's second moment
    directly (``centered=True`` uses the covariance instead). The latent is
    orthonormal (c = x V) rather than scaled by S^{-1/2}; Sec. 3.1 notes any
    split of S gives the same reconstruction.

    Steps: mu = mean_t x_t and S = (1/T) sum_t x_t^T x_t in fp64 (population
    normalisation; the paper is silent); eigendecompose; sort eigenvalues
    descending (stable by index); flip each eigenvector so its largest-|.|
    entry (lowest index on ties) is positive; store V32 = fp32(V). The
    coefficient mean m = fp32(mu . V32) and the centered marginal variances
    v_j = V32_j^T C V32_j (C the centered covariance) follow Sec. 3.1's
    instruction to subtract measured means and use centered variances.
    """
    x = np.asarray(x, dtype=np.float64)
    T, d = x.shape
    assert d == p.head_dim and T > 0
    mu = x.sum(axis=0) / T
    S = (x.T @ x) / T
    return _fit_from_moments(S, mu, p, latent_scale)


def fit_from_weights(W: np.ndarray, G: np.ndarray, hbar, p: Params, latent_scale: bool = False) -> FitResult:
    """Calibrate-once basis from a head's projection and its layer's input statistics
    (Sec. 3.1, Eqs. gweighted and gsvd; App. B).

    The paper whitens the weight, M = G^{1/2} W = U S V^T with G = E[h^T h], and keeps
    the top right singular directions. The keys the head produces, k = h W, have
    E[k^T k] = W^T G W = M^T M = V S^2 V^T and E[k] = hbar W (hbar = E[h]; None for
    zero), so the basis, coefficient mean, centered variances and widths are those
    of ``fit`` for a stream with exactly these moments: no pass over cached data.
    W [d_model, d], G [d_model, d_model], hbar [d_model]; all read as fp64.
    """
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    assert W.shape[1] == p.head_dim and G.shape == (W.shape[0], W.shape[0])
    S = W.T @ G @ W
    mu = np.zeros(p.head_dim) if hbar is None else np.asarray(hbar, dtype=np.float64) @ W
    return _fit_from_moments(S, mu, p, latent_scale)


def _fit_from_moments(S: np.ndarray, mu: np.ndarray, p: Params, latent_scale: bool = False) -> FitResult:
    """Steps of ``fit`` after the moments: second moment S and mean mu, fp64.

    latent_scale: the square-root split of Eq. gsvd. With M = G^{1/2} W = U Sig V^T the
    cached latent is h G^{-1/2} U Sig^{1/2} = (k V) Sig^{-1/2}, and Sig = diag(sqrt(lambda))
    for the eigenvalues lambda of E[k^T k]; so coordinate j of the orthonormal latent is
    multiplied by f_j = lambda_j^{-1/4}, which makes E[c^T c] = diag(sqrt(lambda)) (Eq.
    second-moment-latent). Reading: lambda_j is floored at lambda_0 2^-40 (a rank-deficient
    fit would otherwise scale noise without bound); the allocation receives the centered
    variances of the scaled coordinates, the quantities that are cached.
    """
    d = p.head_dim
    C = S - np.outer(mu, mu)
    M = C if p.centered else S
    M = 0.5 * (M + M.T)
    lam, vec = np.linalg.eigh(M)
    order = np.argsort(-lam, kind="stable")
    lam = lam[order]
    vec = vec[:, order]
    for j in range(d):
        i = int(np.argmax(np.abs(vec[:, j])))
        if vec[i, j] < 0:
            vec[:, j] = -vec[:, j]
    V32 = vec.astype(np.float32)
    V64 = V32.astype(np.float64)
    m = (mu @ V64).astype(np.float32)
    var = np.einsum("ij,ik,kj->j", V64, C, V64)
    if not latent_scale:
        return FitResult(V32, m, var, lam, M, mu, C)
    f = latent_scale_factors(lam)
    f64 = f.astype(np.float64)
    return FitResult(V32, m, var * f64 * f64, lam, M, mu, C, f)


def latent_scale_factors(lam: np.ndarray) -> np.ndarray:
    """f_j = max(lambda_j, lambda_0 2^-40)^(-1/4) as fp32 (1 where lambda_0 <= 0)."""
    lam = np.asarray(lam, dtype=np.float64)
    if lam[0] <= 0:
        return np.ones(lam.shape, np.float32)
    return (np.maximum(lam, lam[0] * 2.0 ** -40) ** -0.25).astype(np.float32)


# ----------------------------------------------------------------------------
# O-2: allocation (Sec. 3.2 Eq. waterfill, App. D; metadata counted per App. F)
# ----------------------------------------------------------------------------
_WSCALE = float(2 ** 39)


def _group_weights(var: Sequence[float], p: Params) -> List[int]:
    """Integer group energies w_G = floor(2^39 * D_G / max D), D_G = sum of the group's v_j.

    D_G (summed in ascending j, fp64) is g times the group's mean variance,
    the quantity Sec. 3.2 feeds to the allocation. Negative rounding residue
    is clamped to 0. The integer form makes the objective exact.
    """
    g, nG = p.group_size, p.n_groups
    D = []
    for G in range(nG):
        acc = 0.0
        for j in range(G * g, (G + 1) * g):
            acc += float(var[j])
        D.append(max(acc, 0.0))
    dmax = max(D)
    if not (dmax > 0.0):
        return [0] * nG
    return [int(math.floor((Dg / dmax) * _WSCALE)) for Dg in D]


def _cost(b: int, p: Params) -> int:
    return 0 if b == 0 else p.group_size * b + p.meta_bits


def _distortion(w: int, b: int) -> int:
    """w * 4^(8-b): proportional to v 2^{-2b} (App. D); b = 0 leaves the full energy."""
    return w << (2 * (8 - b))


def allocate_bits(var: Sequence[float], p: Params) -> List[int]:
    """Group bit widths minimising sum_G D_G 2^{-2 b_G} under the effective budget.

    App. D minimises sum_j v_j 2^{-2 b_j} at a fixed rate; Sec. 3.2 groups g
    coordinates under one width (from the group mean variance), drops zero-bit
    groups, and charges one fp16 scale + zero-point per kept group per token.
    The paper does not specify how the continuous water-filling widths are
    rounded to integers and corrected to the rate; this oracle takes the exact
    integer optimum of the same objective instead:

      minimise J(b) = sum_G w_G 4^(8-b_G), then cost C(b), then prefer the
      lexicographically largest b, subject to
      C(b) = sum_{b_G>0} (g b_G + meta_bits) <= R,  b_G in {0..b_max}.

    Solved by dynamic programming over groups (backwards) and remaining
    budget; for each group widths are tried from b_max down to 0 and replaced
    only on strict improvement of (J, C), which yields the lexicographically
    largest optimum. ``allocate_bits_bruteforce`` is the definition by search.
    """
    R = record_budget_bits(p)
    nG = p.n_groups
    w = _group_weights(var, p)
    # best[G][r] = (J, C, widths tuple) for groups G.. with budget r remaining
    budgets = range(R + 1)
    best_next = {r: (0, 0, ()) for r in budgets}
    for G in range(nG - 1, -1, -1):
        cur = {}
        for r in budgets:
            choice = None
            for b in range(p.b_max, -1, -1):
                c = _cost(b, p)
                if c > r:
                    continue
                J2, C2, tail = best_next[r - c]
                cand = (_distortion(w[G], b) + J2, c + C2, (b,) + tail)
                if choice is None or (cand[0], cand[1]) < (choice[0], choice[1]):
                    choice = cand
            cur[r] = choice
        best_next = cur
    return list(best_next[R][2])


def allocate_bits_bruteforce(var: Sequence[float], p: Params) -> List[int]:
    """Exhaustive search over all width vectors; same objective and tie rules."""
    R = record_budget_bits(p)
    w = _group_weights(var, p)
    best = None
    for b in product(range(p.b_max + 1), repeat=p.n_groups):
        C = sum(_cost(x, p) for x in b)
        if C > R:
            continue
        J = sum(_distortion(wg, x) for wg, x in zip(w, b))
        key = (J, C, tuple(-x for x in b))
        if best is None or key < best[0]:
            best = (key, b)
    return list(best[1])


# ----------------------------------------------------------------------------
# O-3: quantize (Sec. 3.2: per-token min/max per group, fp16 scale and zero-point)
# ----------------------------------------------------------------------------
def quantize(coef: np.ndarray, bits: Sequence[int], p: Params):
    """Quantize centered coefficients [T, d] group by group.

    For each token and kept group G at b bits: lo/hi = min/max of its g
    coefficients; z16 = fp16(lo) and s16 = fp16(max(hi - z, 0) / (2^b - 1)),
    each rounded once (RNE, saturating); with z = float(z16), s = float(s16):
    q = clamp(round_half_even((c - z) / s), 0, 2^b - 1), and q = 0 when s = 0.

    Returns codes [T, d] (uint8; 0 in dropped groups) and meta [T, nG] uint32
    (low 16 bits = s16 bits, high 16 bits = z16 bits; 0 for dropped groups).
    """
    coef = np.asarray(coef, dtype=np.float64)
    T, d = coef.shape
    g = p.group_size
    codes = np.zeros((T, d), dtype=np.uint8)
    meta = np.zeros((T, p.n_groups), dtype=np.uint32)
    for G, b in enumerate(bits):
        if b == 0:
            continue
        c = coef[:, G * g:(G + 1) * g]
        lo = c.min(axis=1)
        hi = c.max(axis=1)
        z16 = fp16_rne_sat(lo)
        z = z16.astype(np.float64)
        levels = float((1 << b) - 1)
        s16 = fp16_rne_sat(np.maximum(hi - z, 0.0) / levels)
        s = s16.astype(np.float64)
        safe = np.where(s > 0, s, 1.0)
        u = (c - z[:, None]) / safe[:, None]
        q = np.clip(np.rint(u), 0.0, levels)
        q[s == 0] = 0.0
        codes[:, G * g:(G + 1) * g] = q.astype(np.uint8)
        meta[:, G] = fp16_bits(s16) | (fp16_bits(z16) << np.uint32(16))
    return codes, meta


def quantize_given_meta(coef: np.ndarray, meta: np.ndarray, bits: Sequence[int], p: Params):
    """The quantization rule of ``quantize`` with the zero-point and scale taken
    from given metadata words (low 16 bits s16, high 16 bits z16).

    Returns codes [T, d] (0 in dropped groups) and the unrounded u = (c - z)/s
    [T, d] (NaN where s = 0 or the group is dropped), so a caller can tell
    rounding ties from other differences.
    """
    coef = np.asarray(coef, dtype=np.float64)
    T, d = coef.shape
    g = p.group_size
    codes = np.zeros((T, d), dtype=np.uint8)
    u_all = np.full((T, d), np.nan)
    for G, b in enumerate(bits):
        if b == 0:
            continue
        s = f16_bits_to_f64(meta[:, G] & 0xFFFF)
        z = f16_bits_to_f64(meta[:, G] >> 16)
        levels = float((1 << b) - 1)
        safe = np.where(s > 0, s, 1.0)
        u = (coef[:, G * g:(G + 1) * g] - z[:, None]) / safe[:, None]
        q = np.clip(np.rint(u), 0.0, levels)
        q[s == 0] = 0.0
        u[s == 0] = np.nan
        codes[:, G * g:(G + 1) * g] = q.astype(np.uint8)
        u_all[:, G * g:(G + 1) * g] = u
    return codes, u_all


def dequantize(codes: np.ndarray, meta: np.ndarray, bits: Sequence[int], p: Params) -> np.ndarray:
    """c_hat = z + s q on kept groups, 0 on dropped groups (Sec. 3.2)."""
    T = codes.shape[0]
    g = p.group_size
    out = np.zeros((T, p.head_dim), dtype=np.float64)
    for G, b in enumerate(bits):
        if b == 0:
            continue
        s = f16_bits_to_f64(meta[:, G] & 0xFFFF)
        z = f16_bits_to_f64(meta[:, G] >> 16)
        out[:, G * g:(G + 1) * g] = z[:, None] + s[:, None] * codes[:, G * g:(G + 1) * g].astype(np.float64)
    return out


# ----------------------------------------------------------------------------
# O-4: record format (Sec. 3.2 counts a payload plus an fp16 scale and
# zero-point per kept group and token; the bit layout is ours)
# ----------------------------------------------------------------------------
def pack(codes: np.ndarray, meta: np.ndarray, bits: Sequence[int], p: Params) -> np.ndarray:
    """Logical records [T, W] uint32.

    Words [0, |K|) hold the metadata of the kept groups K (ascending), then the
    payload of each kept group in order, g*b/32 words each; in-group code j
    occupies payload bits [j*b, (j+1)*b), least significant bit first, where
    payload bit p is bit p % 32 of payload word p // 32. Unused words are 0.
    """
    T = codes.shape[0]
    g = p.group_size
    W = record_words(p)
    kept = [G for G, b in enumerate(bits) if b > 0]
    used = len(kept) + sum(g * bits[G] // 32 for G in kept)
    assert used <= W, "allocation does not fit the record"
    rec = np.zeros((T, W), dtype=np.uint64)
    for k, G in enumerate(kept):
        rec[:, k] = meta[:, G]
    off = len(kept)
    for G in kept:
        b = bits[G]
        nbits = g * b
        stream = np.zeros((T, nbits), dtype=np.uint64)
        for j in range(g):
            cj = codes[:, G * g + j].astype(np.uint64)
            for i in range(b):
                stream[:, j * b + i] = (cj >> np.uint64(i)) & np.uint64(1)
        for wi in range(nbits // 32):
            word = np.zeros(T, dtype=np.uint64)
            for i in range(32):
                word |= stream[:, wi * 32 + i] << np.uint64(i)
            rec[:, off + wi] = word
        off += nbits // 32
    return rec.astype(np.uint32)


def unpack(rec: np.ndarray, bits: Sequence[int], p: Params):
    """Inverse of ``pack``: records [T, W] -> (codes [T, d] uint8, meta [T, nG] uint32)."""
    rec = np.asarray(rec, dtype=np.uint32)
    T = rec.shape[0]
    g = p.group_size
    kept = [G for G, b in enumerate(bits) if b > 0]
    codes = np.zeros((T, p.head_dim), dtype=np.uint8)
    meta = np.zeros((T, p.n_groups), dtype=np.uint32)
    for k, G in enumerate(kept):
        meta[:, G] = rec[:, k]
    off = len(kept)
    for G in kept:
        b = bits[G]
        nbits = g * b
        stream = np.zeros((T, nbits), dtype=np.uint64)
        for wi in range(nbits // 32):
            word = rec[:, off + wi].astype(np.uint64)
            for i in range(32):
                stream[:, wi * 32 + i] = (word >> np.uint64(i)) & np.uint64(1)
        for j in range(g):
            v = np.zeros(T, dtype=np.uint64)
            for i in range(b):
                v |= stream[:, j * b + i] << np.uint64(i)
            codes[:, G * g + j] = v.astype(np.uint8)
        off += nbits // 32
    return codes, meta


def physical_index(stream: int, t: np.ndarray, w: int, t_capacity: int, W: int) -> np.ndarray:
    """Word address of (stream, token t, word w) in the tiled device layout.

    Records are grouped in tiles of 64 tokens; inside a tile, word w of the 64
    tokens is contiguous: s*T_cap*W + (t // 64)*64*W + w*64 + (t % 64).
    """
    t = np.asarray(t, dtype=np.int64)
    return stream * t_capacity * W + (t // 64) * 64 * W + w * 64 + (t % 64)


# ----------------------------------------------------------------------------
# Encode / decode (Sec. 3.1-3.3, Mode A)
# ----------------------------------------------------------------------------
def encode(x: np.ndarray, basis32: np.ndarray, mean32: np.ndarray, bits: Sequence[int], p: Params, scale32=None):
    """Project (c = x V32 - m, fp64; times f_j under the square-root split), quantize and
    pack: returns (records, codes, meta, coef)."""
    x = np.asarray(x, dtype=np.float64)
    coef = x @ np.asarray(basis32, dtype=np.float64) - np.asarray(mean32, dtype=np.float64)[None, :]
    if scale32 is not None:
        coef = coef * np.asarray(scale32, dtype=np.float64)[None, :]
    codes, meta = quantize(coef, bits, p)
    return pack(codes, meta, bits, p), codes, meta, coef


def decode(rec: np.ndarray, basis32: np.ndarray, mean32: np.ndarray, bits: Sequence[int], p: Params,
           scale32=None) -> np.ndarray:
    """Mode A reconstruction x_hat = (c_hat + m) V32^T in fp64 (Sec. 3.3); under the
    square-root split c_hat / f_j takes the place of c_hat."""
    codes, meta = unpack(rec, bits, p)
    c_hat = dequantize(codes, meta, bits, p)
    if scale32 is not None:
        c_hat = c_hat / np.asarray(scale32, dtype=np.float64)[None, :]
    return (c_hat + np.asarray(mean32, np.float64)[None, :]) @ np.asarray(basis32, np.float64).T


# ----------------------------------------------------------------------------
# O-6: decode-step attention
# ----------------------------------------------------------------------------
def softmax_f64(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention_mode_a(q: np.ndarray, k_hat: np.ndarray, v_hat: np.ndarray, scale: float = 0.0) -> np.ndarray:
    """Standard single-step attention over a reconstructed cache (Mode A, Sec. 3.3).

    q [H_q, d]; k_hat, v_hat [H_kv, T, d]. Query head h reads KV head
    h // (H_q / H_kv) (grouped-query attention, Sec. 4.1). scale defaults to
    1/sqrt(d); no mask (a decode step sees every cached token).
    """
    q = np.asarray(q, np.float64)
    Hq, d = q.shape
    Hkv = k_hat.shape[0]
    nqh = Hq // Hkv
    sc = scale if scale > 0 else 1.0 / math.sqrt(d)
    out = np.zeros((Hq, d), dtype=np.float64)
    for h in range(Hq):
        kv = h // nqh
        s = sc * (np.asarray(k_hat[kv], np.float64) @ q[h])
        pr = softmax_f64(s)
        out[h] = pr @ np.asarray(v_hat[kv], np.float64)
    return out


def rope(x: np.ndarray, pos, inv_freq) -> np.ndarray:
    """Rotary position embedding of vectors x [..., d] at positions pos [...] (broadcast).

    Dimension i < d/2 is paired with i + d/2 (the pairing of Llama and Qwen) and the
    pair is rotated by the angle pos * inv_freq[i], computed exactly in fp64 from the
    given frequencies: x'_i = x_i cos - x_{i+d/2} sin, x'_{i+d/2} = x_{i+d/2} cos + x_i sin.
    """
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    w = np.asarray(inv_freq, np.float64)
    ang = np.asarray(pos, np.float64)[..., None] * w
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def attention_mode_a_rope(q: np.ndarray, k_hat: np.ndarray, v_hat: np.ndarray, inv_freq, q_pos: int,
                          scale: float = 0.0) -> np.ndarray:
    """Mode A with RoPE (Sec. 3.3): the cache holds latents of pre-RoPE keys, so each key
    is reconstructed and then rotated at its own position, which is what makes Mode A
    exact for rotary models. Key t sits at position t; the query at q_pos. Values are
    not rotated. Otherwise as ``attention_mode_a``.
    """
    q = np.asarray(q, np.float64)
    T = np.asarray(k_hat).shape[1]
    k_rot = rope(k_hat, np.arange(T)[None, :], inv_freq)
    q_rot = rope(q, q_pos, inv_freq)
    return attention_mode_a(q_rot, k_rot, v_hat, scale)


def attention_mode_b(q, ck_hat, cv_hat, basis_k, mean_k, basis_v, mean_v, scale: float = 0.0):
    """Latent-space attention (App. E): q' = q V_K once, scores q' (c_K + m_K), values in
    coefficient space, one inverse rotation per output. Equal to Mode A by linearity.

    ck_hat, cv_hat [H_kv, T, d] dequantized coefficients; basis_* [H_kv, d, d]; mean_* [H_kv, d].
    """
    q = np.asarray(q, np.float64)
    Hq, d = q.shape
    Hkv = ck_hat.shape[0]
    nqh = Hq // Hkv
    sc = scale if scale > 0 else 1.0 / math.sqrt(d)
    out = np.zeros((Hq, d), dtype=np.float64)
    for h in range(Hq):
        kv = h // nqh
        Vk = np.asarray(basis_k[kv], np.float64)
        Vv = np.asarray(basis_v[kv], np.float64)
        qp = sc * (q[h] @ Vk)
        s = (np.asarray(ck_hat[kv], np.float64) + np.asarray(mean_k[kv], np.float64)[None, :]) @ qp
        pr = softmax_f64(s)
        a = pr @ np.asarray(cv_hat[kv], np.float64)
        out[h] = (a + np.asarray(mean_v[kv], np.float64)) @ Vv.T
    return out
