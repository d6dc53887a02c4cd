"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test reaches the expected value by a route other than the oracle's own
code: closed forms, an SVD instead of an eigensolver, brute force with a real
valued objective, bit strings instead of integer packing, scipy's softmax, or
values printed in the paper (``tests/golden``).
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _tiny_stream(tensor, T=4096):
    return synth.numpy_stream(synth.WORKLOADS["tiny"], 0, 0, 0, tensor, n_tokens=T)


# ---------------------------------------------------------------------------
# O-1 fit: orthonormal basis that diagonalises the fitted second moment
# (Sec. 3.1, Eq. second-moment-latent)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("centered", [False, True])
@pytest.mark.parametrize("tensor", [0, 1])
def test_fit_basis_orthonormal_and_diagonalising(tensor, centered):
    p = O.Params(centered=centered)
    x = _tiny_stream(tensor)
    f = O.fit(x, p)
    V = f.basis.astype(np.float64)
    assert np.abs(V.T @ V - np.eye(128)).max() <= 1e-6
    # the matrix that was fitted, recomputed independently from the data
    xd = x.astype(np.float64)
    T = xd.shape[0]
    mu = xd.mean(axis=0)
    S = sum(np.outer(r, r) for r in xd[::1]) / T if T <= 512 else (xd.T @ xd) / T
    M = S - np.outer(mu, mu) if centered else S
    D = V.T @ M @ V
    lam_max = np.abs(np.diag(D)).max()
    off = D - np.diag(np.diag(D))
    assert np.abs(off).max() / lam_max <= 1e-6
    # eigenvalues descending, and they are the Rayleigh quotients of the basis
    assert np.all(np.diff(f.eigvals) <= 0)
    assert np.allclose(np.diag(D), f.eigvals, rtol=0, atol=1e-6 * lam_max)
    # residual ||M v - lambda v|| small for every direction
    res = np.linalg.norm(M @ V - V * f.eigvals[None, :], axis=0).max()
    assert res <= 1e-5 * lam_max


def test_fit_sign_and_order_convention_on_diagonal_data():
    # Data whose second moment is diagonal with known, distinct values: the
    # basis must be a permutation matrix with +1 entries, sorted by energy.
    rng = np.random.default_rng(7)
    d, T = 128, 256
    scales = rng.permutation(np.linspace(1.0, 3.0, d))
    # +-1 Rademacher columns with exactly zero cross products via Hadamard rows
    H = np.array([[1.0]])
    while H.shape[0] < T:
        H = np.block([[H, H], [H, -H]])
    x = H[:, 1:d + 1] * scales[None, :]          # columns orthogonal, mean zero
    f = O.fit(x, O.Params())
    expect_order = np.argsort(-scales, kind="stable")
    V = f.basis.astype(np.float64)
    P = np.zeros((d, d))
    P[expect_order, np.arange(d)] = 1.0
    assert np.abs(V - P).max() <= 1e-12
    assert np.allclose(f.eigvals, scales[expect_order] ** 2, rtol=1e-12)


def test_fit_matches_g_weighted_svd_of_the_weights():
    """Sec. 3.1 Eq. (gsvd): with k = h W and G = E[h^T h], the right singular
    vectors of M = G^{1/2} W are the eigenbasis of the keys' second moment and
    the rank-r reconstruction h W_down W_up equals k V_r V_r^T; the square-root
    split gives E[c^T c] = Sigma_r (Eq. second-moment-latent)."""
    rng = np.random.default_rng(11)
    T, dh = 4096, 256
    H = rng.standard_normal((T, dh)) @ np.diag(np.linspace(2.0, 0.2, dh)) + 0.3
    W = rng.standard_normal((dh, 128)) / math.sqrt(dh)
    K = H @ W
    G = H.T @ H / T
    evals, evecs = np.linalg.eigh(G)
    G_half = evecs @ np.diag(np.sqrt(evals)) @ evecs.T
    G_mhalf = evecs @ np.diag(1.0 / np.sqrt(evals)) @ evecs.T
    U, sig, Vt = np.linalg.svd(G_half @ W, full_matrices=False)
    f = O.fit(K, O.Params())
    Vo = f.basis.astype(np.float64)
    # same directions up to sign, same energies (eigenvalue = sigma^2)
    assert np.allclose(f.eigvals, sig ** 2, rtol=1e-9)
    cos = np.abs(np.sum(Vo * Vt.T, axis=0))
    assert np.all(cos >= 1 - 1e-6)
    for r in (8, 32, 64, 100):
        W_down = G_mhalf @ U[:, :r] @ np.diag(np.sqrt(sig[:r]))
        W_up = np.diag(np.sqrt(sig[:r])) @ Vt[:r]
        k_hat_paper = H @ W_down @ W_up
        k_hat_basis = K @ Vo[:, :r] @ Vo[:, :r].T
        rel = np.linalg.norm(k_hat_paper - k_hat_basis) / np.linalg.norm(K)
        assert rel <= 2e-6, (r, rel)
        c = H @ W_down
        Ec = c.T @ c / T
        assert np.allclose(Ec, np.diag(sig[:r]), atol=1e-9 * sig[0])


def test_fit_variance_and_mean_are_the_coefficient_statistics():
    x = _tiny_stream(0).astype(np.float64)
    f = O.fit(x, O.Params())
    c = x @ f.basis.astype(np.float64)
    # measured coordinate means (Sec. 3.1) and centered marginal variances
    assert np.allclose(f.mean, c.mean(axis=0), rtol=0, atol=1e-5 * np.abs(c).max())
    assert np.allclose(f.var, c.var(axis=0), rtol=1e-9, atol=1e-12)


# ---------------------------------------------------------------------------
# O-2 allocation: exact integer optimum of App. D's objective under App. F's
# effective rate
# ---------------------------------------------------------------------------
def _real_valued_best(var, p):
    """Independent brute force with the real-valued objective sum_G D_G 4^-b_G."""
    from itertools import product
    R = O.record_budget_bits(p)
    g = p.group_size
    Dg = [sum(var[G * g:(G + 1) * g]) for G in range(p.n_groups)]
    scored = []
    for b in product(range(p.b_max + 1), repeat=p.n_groups):
        cost = sum(0 if x == 0 else g * x + p.meta_bits for x in b)
        if cost > R:
            continue
        J = sum(d * 4.0 ** (-x) for d, x in zip(Dg, b))
        scored.append((J, cost, b))
    scored.sort(key=lambda s: (s[0], s[1]))
    return scored


def _random_var(rng, d):
    return np.exp(rng.uniform(-8, 3, size=d))


@pytest.mark.parametrize("g", [2, 4, 8])
@pytest.mark.parametrize("meta", [0, 32])
@pytest.mark.parametrize("b_max", [4, 8])
def test_allocation_dp_equals_bruteforce_d8(g, meta, b_max):
    rng = np.random.default_rng(100 + g * 7 + meta + b_max)
    cases = [_random_var(rng, 8) for _ in range(25)]
    cases += [np.zeros(8), np.ones(8), np.array([1e6, 1, 1, 1, 1, 1, 1, 1.0]),
              np.array([0, 0, 0, 0, 0, 0, 0, 5.0]), np.full(8, 3.25)]
    max_cost = (8 // g) * (g * b_max + meta)
    Rs = sorted(set([0, 1, g + meta - 1, g + meta, max_cost, max_cost + 5] +
                    list(rng.integers(0, max_cost + 1, size=12))))
    for v in cases:
        for R in Rs:
            p = O.Params(head_dim=8, group_size=g, b_max=b_max, meta_bits=meta, budget_bits=int(R))
            assert O.allocate_bits(v, p) == O.allocate_bits_bruteforce(v, p), (v, R)


def test_allocation_dp_equals_bruteforce_g1_small():
    rng = np.random.default_rng(5)
    for _ in range(6):
        v = _random_var(rng, 8)
        for R in (0, 3, 8, 13, 20, 32):
            p = O.Params(head_dim=8, group_size=1, b_max=4, meta_bits=0, budget_bits=R)
            assert O.allocate_bits(v, p) == O.allocate_bits_bruteforce(v, p)


def test_allocation_matches_real_valued_search_when_unique():
    rng = np.random.default_rng(9)
    checked = 0
    for _ in range(60):
        v = _random_var(rng, 128)
        for ratio in (4.0, 8.0, 12.0):
            p = O.Params(ratio=ratio)
            scored = _real_valued_best(v, p)
            best, second = scored[0], scored[1]
            if second[0] - best[0] <= 1e-6 * best[0]:
                continue  # near-tie: integer weights may order them either way
            assert tuple(O.allocate_bits(v, p)) == best[2]
            checked += 1
    assert checked > 100


def test_allocation_waterfill_closed_form():
    """Eq. (waterfill): with g = 1, no metadata and no active clamp the exact
    integer optimum spends d*b_bar bits and each b_j is within 1 of
    b_bar + 0.5 log2(v_j / GM(v))."""
    rng = np.random.default_rng(3)
    d = 8
    for _ in range(20):
        v = np.exp(rng.uniform(-1.0, 1.0, size=d))
        for b_bar in (3, 4, 5):
            p = O.Params(head_dim=d, group_size=1, b_max=8, meta_bits=0, budget_bits=d * b_bar)
            cont = b_bar + 0.5 * np.log2(v / np.exp(np.mean(np.log(v))))
            if cont.min() < 1 or cont.max() > 7:
                continue
            b = np.array(O.allocate_bits(v, p))
            assert b.sum() == d * b_bar
            assert np.all(np.abs(b - cont) <= 1.0)


def test_allocation_monotone_and_degenerate():
    rng = np.random.default_rng(4)
    v = _random_var(rng, 128)
    prev = None
    g, meta = 32, 32
    for R in range(0, 1200, 32):
        p = O.Params(budget_bits=R if R > 0 else 1)
        b = O.allocate_bits(v, p)
        J = sum(sum(v[G * g:(G + 1) * g]) * 4.0 ** (-x) for G, x in enumerate(b))
        if prev is not None:
            assert J <= prev + 1e-12 * prev
        prev = J
        if R < g + meta:
            assert b == [0, 0, 0, 0]
    # all groups at the cap when the budget allows it
    assert O.allocate_bits(v, O.Params(budget_bits=1152)) == [8, 8, 8, 8]
    # record widths at the three tiers (App. F accounting, 32-bit words)
    assert [O.record_words(O.Params(ratio=r)) for r in (4.0, 8.0, 12.0)] == [16, 8, 5]
    assert O.record_budget_bits(O.Params(ratio=16.0 / 9.0)) == 1152


def test_allocation_drops_low_energy_tail():
    # Sec. 3.2: zero-bit groups are dropped; low energy goes first
    v = np.concatenate([np.full(32, 10.0), np.full(32, 1.0), np.full(32, 1e-3), np.full(32, 1e-6)])
    b = O.allocate_bits(v, O.Params(ratio=8.0))
    assert b[2] == 0 and b[3] == 0 and b[0] >= b[1] >= 1


# ---------------------------------------------------------------------------
# Capacity table (App. E) pins the effective-rate accounting of App. F
# ---------------------------------------------------------------------------
def _fmt(n):
    if n >= 1e6:
        return f"{n / 1e6:.2f}M"
    return f"{round(n / 1e3):d}k"


def test_capacity_table_from_record_accounting():
    """The printed capacities follow App. F's effective ratio exactly:
    bytes/token = dense fp16 bytes / ratio with payload and metadata counted.
    The oracle's per-token record budget is that rate floored to whole bits."""
    g = json.load(open(os.path.join(GOLDEN, "capacity_table.json")))
    geo = g["geometry"]
    d = geo["head_dim"]
    dense = geo["n_layers"] * geo["n_kv_heads"] * d * 2 * 2
    assert dense == geo["dense_bytes_per_token"]
    for budget, cells in g["rows"].items():
        free = (float(budget) - geo["weights_gb"]) * geo["gb_unit_bytes"]
        for ratio, cell in zip(g["ratios"], cells):
            if ratio == "dense":
                per_tok = dense
            else:
                exact_bits = 16.0 * d / float(ratio)      # per token per stream
                R = O.record_budget_bits(O.Params(ratio=float(ratio)))
                assert exact_bits - 1 < R <= exact_bits
                per_tok = geo["n_layers"] * geo["n_kv_heads"] * 2 * exact_bits / 8.0
            assert _fmt(free / per_tok) == cell, (budget, ratio)
    # integral rates are kept exactly: 4x, 8x and 16/9 x
    for ratio, bits in ((4.0, 512), (8.0, 256), (16.0 / 9.0, 1152), (16.0, 128)):
        assert O.record_budget_bits(O.Params(ratio=ratio)) == bits


# ---------------------------------------------------------------------------
# fp16 metadata rounding (Sec. 3.2: one fp16 scale and zero-point per kept group
# and token; reading: each rounded once from the exact value, to nearest with
# ties to even, saturating at +-65504)
# ---------------------------------------------------------------------------
def _fp16_exact_bits(x: float) -> int:
    """Binary16 bits of x by exact rational arithmetic (no floating-point format
    conversion involved): sign, then the nearest multiple of the quantum of x's
    binade (2^-24 below 2^-14), ties to the even multiple; magnitudes >= 65504
    saturate to the largest finite value."""
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    a = Fraction(abs(x))
    if a >= 65504:
        return sign | 0x7BFF
    if a < Fraction(1, 2 ** 14):
        quantum = Fraction(1, 2 ** 24)
    else:
        e = a.numerator.bit_length() - a.denominator.bit_length()
        if Fraction(2) ** e > a:
            e -= 1
        quantum = Fraction(2) ** (e - 10)
    q = a / quantum
    n = q.numerator // q.denominator
    rem = q - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    v = n * quantum                      # exact value of the rounded magnitude
    if v == 0:
        return sign
    if v < Fraction(1, 2 ** 14):         # subnormal: the multiple of 2^-24 is the field
        return sign | int(v * 2 ** 24)
    e = v.numerator.bit_length() - v.denominator.bit_length()
    if Fraction(2) ** e > v:
        e -= 1
    mant = int(v / Fraction(2) ** (e - 10)) - 1024
    return sign | ((e + 15) << 10) | mant


# (value, expected bits, why)
_FP16_HAND = [
    (1.0 + 2.0 ** -11, 0x3C00, "midpoint of 1 and 1+2^-10: even mantissa 0"),
    (1.0 + 3 * 2.0 ** -11, 0x3C02, "midpoint of mantissas 1 and 2: even 2"),
    (1.0 + 2.0 ** -11 + 2.0 ** -40, 0x3C01, "just above a midpoint (through fp32 it would become the midpoint)"),
    (1.0 + 2.0 ** -11 - 2.0 ** -40, 0x3C00, "just below a midpoint"),
    (-(1.0 + 3 * 2.0 ** -11), 0xBC02, "negative midpoint, even mantissa 2"),
    (0.1, 0x2E66, "0.1 = 1638.4 quanta of 2^-14 -> 1638 = 0x400 + 0x266, exponent -4"),
    (2.0 ** -24, 0x0001, "smallest subnormal"),
    (2.0 ** -25, 0x0000, "half the smallest subnormal: tie to even zero"),
    (3 * 2.0 ** -25, 0x0002, "midpoint of subnormals 1 and 2: even 2"),
    (2.0 ** -25 + 2.0 ** -60, 0x0001, "just above the half-quantum"),
    (1023 * 2.0 ** -24, 0x03FF, "largest subnormal"),
    (2.0 ** -14 - 2.0 ** -25, 0x0400, "midpoint of the largest subnormal and 2^-14: even 0x400"),
    (-(2.0 ** -25), 0x8000, "negative tie to zero keeps the sign"),
    (65504.0, 0x7BFF, "largest finite"),
    (65519.99, 0x7BFF, "below the overflow midpoint"),
    (65520.0, 0x7BFF, "overflow midpoint: saturates (IEEE would give infinity)"),
    (1.0e6, 0x7BFF, "saturates"),
    (-1.0e6, 0xFBFF, "saturates negative"),
    (-65520.0, 0xFBFF, "negative overflow midpoint saturates"),
]


@pytest.mark.parametrize("x,bits,why", _FP16_HAND)
def test_fp16_rounding_hand_values(x, bits, why):
    assert _fp16_exact_bits(x) == bits, why
    assert int(O.fp16_bits(O.fp16_rne_sat(x))) == bits, why


def test_fp16_rounding_is_single_not_through_fp32():
    # rounding through fp32 first would collapse these onto fp16 midpoints
    differs = 0
    for k in range(0, 200):
        base = 1.0 + (2 * k + 1) * 2.0 ** -11          # midpoint of mantissas k and k + 1
        for off in (2.0 ** -40, -(2.0 ** -40)):
            x = base + off
            assert float(np.float32(x)) == base        # fp32 cannot hold the offset
            want = 0x3C00 + k + (1 if off > 0 else 0)  # the nearer neighbour
            assert _fp16_exact_bits(x) == want
            assert int(O.fp16_bits(O.fp16_rne_sat(x))) == want
            differs += _fp16_exact_bits(base) != want  # the tie through fp32 goes to the even one
    assert differs == 200


def test_fp16_rounding_matches_exact_reference():
    rng = np.random.default_rng(31)
    xs = list(rng.standard_normal(3000) * np.exp(rng.uniform(-25, 12, 3000)))
    # exact midpoints and their fp64 neighbours in normal and subnormal binades
    for e in range(-24, 16):
        quantum = 2.0 ** (max(e, -14) - 10) if e >= -14 else 2.0 ** -24
        for n in rng.integers(0, 1024, 8):
            lo = (1024 + int(n)) * quantum if e >= -14 else int(n) * quantum
            mid = lo + quantum / 2
            if abs(mid) > 65504:
                continue
            xs += [mid, np.nextafter(mid, np.inf), np.nextafter(mid, -np.inf), -mid]
    xs += [0.0, -0.0, 65504.0, 65520.0, 7e4, -7e4, np.nextafter(65520.0, 0.0)]
    got = O.fp16_bits(O.fp16_rne_sat(np.array(xs, dtype=np.float64)))
    want = np.array([_fp16_exact_bits(float(x)) for x in xs], dtype=np.uint32)
    assert np.array_equal(got, want)


# ---------------------------------------------------------------------------
# O-3 quantize (Sec. 3.2)
# ---------------------------------------------------------------------------
def test_quantize_hand_case_zero_point_not_representable():
    """Worked by hand: the zero-point is the fp16 rounding of the group minimum, so
    z != lo, and s is rounded from (hi - z)/(2^b - 1) with that z.

    [0.1, 0.3, 0.5, 0.7] at b = 2: z = fp16(0.1) = 1638 * 2^-14 = 0.0999755859375
    (0x2E66); (0.7 - z)/3 = 0.200008138... = 1638.47 quanta of 2^-13 -> s =
    1638 * 2^-13 = 0.199951171875 (0x3266); u = (c - z)/s = 1.2e-4, 1.00037,
    2.00061, 3.00085 -> q = [0, 1, 2, 3]; decoded z + s q = 0.0999755859375,
    0.2999267578125, 0.4998779296875, 0.6998291015625.

    [0.10003, 0.25, 0.6, 0.9] at b = 3: z = fp16(0.10003) = 1639 * 2^-14 =
    0.10003662109375 (0x2E67) lies above the minimum, so u_0 = -5.8e-5 clamps to 0;
    (0.9 - z)/7 = 0.1142805 = 1872.40 quanta of 2^-14 -> s = 1872 * 2^-14 =
    0.1142578125 (0x2F50); u = -5.8e-5, 1.3125, 4.37575, 7.00139 -> q = [0, 1, 4, 7].
    """
    p = O.Params(head_dim=4, group_size=4)
    codes, meta = O.quantize(np.array([[0.1, 0.3, 0.5, 0.7]]), [2], p)
    assert codes.tolist() == [[0, 1, 2, 3]]
    assert int(meta[0, 0]) == 0x2E663266
    rec = O.dequantize(codes, meta, [2], p)
    assert rec[0].tolist() == [0.0999755859375, 0.2999267578125, 0.4998779296875, 0.6998291015625]
    codes, meta = O.quantize(np.array([[0.10003, 0.25, 0.6, 0.9]]), [3], p)
    assert codes.tolist() == [[0, 1, 4, 7]]
    assert int(meta[0, 0]) == (0x2E67 << 16) | 0x2F50
    rec = O.dequantize(codes, meta, [3], p)
    assert rec[0].tolist() == [0.10003662109375, 0.10003662109375 + 0.1142578125,
                               0.10003662109375 + 4 * 0.1142578125, 0.10003662109375 + 7 * 0.1142578125]


def test_quantize_hand_vectors():
    p = O.Params(head_dim=4, group_size=4)
    codes, meta = O.quantize(np.array([[0.0, 1.0, 2.0, 3.0]]), [2], p)
    assert codes.tolist() == [[0, 1, 2, 3]]
    s = O.f16_bits_to_f64(meta[0, 0] & 0xFFFF)
    z = O.f16_bits_to_f64(meta[0, 0] >> 16)
    assert (s, z) == (1.0, 0.0)
    # ties round to even: u = 0.5 -> 0, 1.5 -> 2, 2.5 -> 2
    c2, m2 = O.quantize(np.array([[0.0, 0.5, 2.5, 3.0]]), [2], p)
    assert c2.tolist() == [[0, 0, 2, 3]]
    # constant group: s = 0, codes 0, reconstruction = z
    c3, m3 = O.quantize(np.array([[1.25, 1.25, 1.25, 1.25]]), [3], p)
    assert c3.tolist() == [[0, 0, 0, 0]]
    assert np.all(O.dequantize(c3, m3, [3], p) == 1.25)
    # dropped group stores nothing and dequantizes to 0
    c4, m4 = O.quantize(np.array([[5.0, 6, 7, 8]]), [0], p)
    assert c4.tolist() == [[0, 0, 0, 0]] and m4.tolist() == [[0]]
    assert np.all(O.dequantize(c4, m4, [0], p) == 0)


def test_quantize_range_and_error_bound():
    rng = np.random.default_rng(1)
    p = O.Params()
    coef = rng.standard_normal((512, 128)) * np.exp(rng.uniform(-3, 3, 128))[None, :]
    for b in range(1, 9):
        bits = [b, b, b, b]
        codes, meta = O.quantize(coef, bits, p)
        assert codes.max() <= (1 << b) - 1
        rec = O.dequantize(codes, meta, bits, p)
        for G in range(4):
            sl = slice(32 * G, 32 * G + 32)
            s = O.f16_bits_to_f64(meta[:, G] & 0xFFFF)[:, None]
            z = O.f16_bits_to_f64(meta[:, G] >> 16)[:, None]
            lo = coef[:, sl].min(axis=1, keepdims=True)
            top = z + s * ((1 << b) - 1)
            inside = (coef[:, sl] >= z) & (coef[:, sl] <= top)
            err = np.abs(rec[:, sl] - coef[:, sl])
            bound = s / 2 * (1 + 1e-12) + 1e-300
            assert np.all(err[inside] <= np.broadcast_to(bound, err.shape)[inside])
            # outside the representable range only by the fp16 rounding of z and s
            slack = np.abs(z - lo) + s * ((1 << b) - 1) * 2 ** -10 + s / 2
            assert np.all(err <= np.broadcast_to(slack, err.shape) + 1e-12)


# ---------------------------------------------------------------------------
# O-4 record format
# ---------------------------------------------------------------------------
def test_pack_hand_built_record():
    p = O.Params(budget_bits=256)           # W = 8
    codes = np.zeros((1, 128), np.uint8)
    codes[0, :32] = [j % 8 for j in range(32)]
    codes[0, 32:64] = [(3 * j + 1) % 4 for j in range(32)]
    meta = np.array([[0x3C00ABCD, 0x12345678, 0, 0]], dtype=np.uint32)
    rec = O.pack(codes, meta, [3, 2, 0, 0], p)
    expect = [0x3C00ABCD, 0x12345678,                 # metadata of kept groups 0, 1
              0x88FAC688, 0xC688FAC6, 0xFAC688FA,     # group 0 payload, 3-bit codes
              0xB1B1B1B1, 0xB1B1B1B1,                 # group 1 payload, 2-bit codes
              0x00000000]                             # padding
    assert rec[0].tolist() == expect
    c2, m2 = O.unpack(rec, [3, 2, 0, 0], p)
    assert np.array_equal(c2, codes) and m2[0, :2].tolist() == [0x3C00ABCD, 0x12345678]


@pytest.mark.parametrize("bits", [[1, 1, 1, 1], [2, 3, 0, 1], [8, 0, 0, 0], [5, 6, 7, 0], [4, 4, 4, 2],
                                  [0, 0, 0, 0], [0, 3, 0, 0]])
def test_pack_round_trip(bits):
    p = O.Params(budget_bits=1152)
    rng = np.random.default_rng(sum(bits) + 17)
    T = 70
    codes = np.zeros((T, 128), np.uint8)
    meta = np.zeros((T, 4), np.uint32)
    for G, b in enumerate(bits):
        if b:
            codes[:, 32 * G:32 * G + 32] = rng.integers(0, 1 << b, size=(T, 32))
            meta[:, G] = rng.integers(0, 2 ** 32, size=T, dtype=np.uint64).astype(np.uint32)
    rec = O.pack(codes, meta, bits, p)
    used = sum(1 for b in bits if b) + sum(b for b in bits)
    assert np.all(rec[:, used:] == 0)
    c2, m2 = O.unpack(rec, bits, p)
    assert np.array_equal(c2, codes) and np.array_equal(m2, meta)


def test_physical_index_tiles():
    W, Tcap = 5, 192
    idx = O.physical_index(2, np.array([0, 1, 63, 64, 130]), 3, Tcap, W)
    base = 2 * Tcap * W
    assert idx.tolist() == [base + 3 * 64 + 0, base + 3 * 64 + 1, base + 3 * 64 + 63,
                            base + 64 * W + 3 * 64, base + 2 * 64 * W + 3 * 64 + 2]
    # a tile of 64 tokens x W words is one contiguous block
    all_idx = np.array([O.physical_index(0, np.arange(64), w, Tcap, W) for w in range(W)]).ravel()
    assert sorted(all_idx.tolist()) == list(range(64 * W))


# ---------------------------------------------------------------------------
# O-3/O-5 reconstruction identities and limits
# ---------------------------------------------------------------------------
def _orthonormalised(f):
    q, r = np.linalg.qr(f.basis.astype(np.float64))
    return q * np.sign(np.diag(r))[None, :]


@pytest.mark.parametrize("tensor", [0, 1])
def test_parseval_mse_split(tensor):
    x = _tiny_stream(tensor).astype(np.float64)
    p = O.Params(ratio=8.0)
    f = O.fit(x, p)
    V = _orthonormalised(f)
    m = x.mean(axis=0) @ V
    bits = O.allocate_bits(f.var, p)
    rec, codes, meta, coef = O.encode(x, V, m, bits, p)
    xh = O.decode(rec, V, m, bits, p)
    c_hat = O.dequantize(codes, meta, bits, p)
    kept = np.repeat(np.array(bits) > 0, 32)
    lhs = np.sum((x - xh) ** 2)
    rhs = np.sum(coef[:, ~kept] ** 2) + np.sum((coef[:, kept] - c_hat[:, kept]) ** 2)
    assert abs(lhs - rhs) <= 1e-9 * lhs
    # on fit data the dropped energy per token is exactly the dropped variance
    dropped = np.sum(coef[:, ~kept] ** 2) / x.shape[0]
    var_exact = np.var(x @ V, axis=0)
    assert abs(dropped - var_exact[~kept].sum()) <= 1e-9 * max(dropped, 1e-30)
    # quantization noise ~ sum s^2 / 12 over kept entries (uniform-error model)
    s = np.stack([O.f16_bits_to_f64(meta[:, G] & 0xFFFF) for G in range(4)], axis=1)
    noise = np.sum((coef[:, kept] - c_hat[:, kept]) ** 2)
    model = sum(np.sum(s[:, G] ** 2) * 32 / 12.0 for G in range(4) if bits[G] >= 2)
    q_kept = [G for G in range(4) if bits[G] >= 2]
    if q_kept and all(bits[G] >= 2 for G in range(4) if bits[G]):
        assert 0.75 * model <= noise <= 1.25 * model


def test_near_lossless_and_bit_slope():
    x = _tiny_stream(0).astype(np.float64)
    f = O.fit(x, O.Params())
    V = _orthonormalised(f)
    m = x.mean(axis=0) @ V
    p8 = O.Params(budget_bits=1152)
    bits = O.allocate_bits(f.var, p8)
    assert bits == [8, 8, 8, 8]
    rec, *_ = O.encode(x, V, m, bits, p8)
    xh = O.decode(rec, V, m, bits, p8)
    assert np.linalg.norm(xh - x) / np.linalg.norm(x) <= 1e-2
    # MSE falls about 4x per extra bit at high rate (Sec. 3.2, App. D)
    mse = {}
    for b in (3, 4, 5, 6):
        r, *_ = O.encode(x, V, m, [b] * 4, p8)
        mse[b] = np.mean((O.decode(r, V, m, [b] * 4, p8) - x) ** 2)
    for b in (3, 4, 5):
        assert 3.0 <= mse[b] / mse[b + 1] <= 5.0


def test_zero_bits_reconstructs_the_mean():
    x = _tiny_stream(1).astype(np.float64)
    f = O.fit(x, O.Params())
    p = O.Params(budget_bits=16)
    bits = O.allocate_bits(f.var, p)
    assert bits == [0, 0, 0, 0]
    rec, *_ = O.encode(x[:10], f.basis, f.mean, bits, p)
    assert rec.shape == (10, 0)
    xh = O.decode(rec, f.basis, f.mean, bits, p)
    assert np.allclose(xh, x.mean(axis=0)[None, :], atol=1e-6 * np.abs(x).max())


# ---------------------------------------------------------------------------
# O-6 attention (Sec. 3.3 Mode A; App. E Mode B)
# ---------------------------------------------------------------------------
def _decoded_cache(rng, Hkv, T):
    out = []
    for _ in range(2):
        bases, means, chat = [], [], []
        for _ in range(Hkv):
            q, _r = np.linalg.qr(rng.standard_normal((128, 128)))
            bases.append(q.astype(np.float32))
            means.append(rng.standard_normal(128).astype(np.float32))
            chat.append(rng.standard_normal((T, 128)) * np.exp(-np.arange(128) / 40.0)[None, :])
        out.append((np.array(bases), np.array(means), np.array(chat)))
    return out


def test_mode_a_equals_mode_b_and_textbook_softmax():
    rng = np.random.default_rng(21)
    Hq, Hkv, T = 8, 2, 300
    (bk, mk, ck), (bv, mv, cv) = _decoded_cache(rng, Hkv, T)
    k_hat = np.einsum("htj,hij->hti", ck + mk[:, None, :], bk.astype(np.float64))
    v_hat = np.einsum("htj,hij->hti", cv + mv[:, None, :], bv.astype(np.float64))
    q = rng.standard_normal((Hq, 128))
    a = O.attention_mode_a(q, k_hat, v_hat)
    b = O.attention_mode_b(q, ck, cv, bk, mk, bv, mv)
    assert np.abs(a - b).max() <= 1e-12 * np.abs(a).max()
    for h in range(Hq):
        kv = h // (Hq // Hkv)
        pr = scipy.special.softmax(k_hat[kv] @ q[h] / math.sqrt(128))
        assert np.allclose(a[h], pr @ v_hat[kv], rtol=1e-12, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(22)
    k = rng.standard_normal((2, 1, 128))
    v = rng.standard_normal((2, 1, 128))
    q = rng.standard_normal((4, 128))
    out = O.attention_mode_a(q, k, v)
    # one token: the output is that token's value, for its KV head
    assert np.allclose(out[:2], v[0, 0][None, :]) and np.allclose(out[2:], v[1, 0][None, :])
    k = rng.standard_normal((1, 50, 128))
    v = rng.standard_normal((1, 50, 128))
    out = O.attention_mode_a(np.zeros((1, 128)), k, v)
    assert np.allclose(out[0], v[0].mean(axis=0), rtol=1e-12, atol=1e-12)


def test_end_to_end_oracle_attention_error_shrinks_with_rate():
    w = synth.WORKLOADS["tiny"]
    xk = synth.numpy_stream(w, 0, 0, 0, 0).astype(np.float64)
    xv = synth.numpy_stream(w, 0, 0, 0, 1).astype(np.float64)
    q = synth.numpy_query(w, 0, 0, 0).astype(np.float64)
    ref = O.attention_mode_a(q, xk[None], xv[None])
    errs = []
    for ratio in (12.0, 8.0, 4.0, 16.0 / 9.0):
        p = O.Params(ratio=ratio)
        fk, fv = O.fit(xk, p), O.fit(xv, p)
        bk, bv = O.allocate_bits(fk.var, p), O.allocate_bits(fv.var, p)
        rk, *_ = O.encode(xk, fk.basis, fk.mean, bk, p)
        rv, *_ = O.encode(xv, fv.basis, fv.mean, bv, p)
        kh = O.decode(rk, fk.basis, fk.mean, bk, p)
        vh = O.decode(rv, fv.basis, fv.mean, bv, p)
        out = O.attention_mode_a(q, kh[None], vh[None])
        errs.append(np.linalg.norm(out - ref) / np.linalg.norm(ref))
    assert errs == sorted(errs, reverse=True)
    assert errs[-1] < 1e-2


def test_quantize_given_meta_reproduces_quantize_and_hand_case():
    rng = np.random.default_rng(8)
    p = O.Params()
    coef = rng.standard_normal((300, 128)) * 3
    bits = [5, 0, 2, 8]
    codes, meta = O.quantize(coef, bits, p)
    codes2, u = O.quantize_given_meta(coef, meta, bits, p)
    assert np.array_equal(codes, codes2)
    assert np.all(np.isnan(u[:, 32:64]))
    # hand case: s = 0.5, z = -1 -> u = (c + 1) / 0.5; ties round to even
    p4 = O.Params(head_dim=4, group_size=4)
    meta = np.array([[int(O.fp16_bits(np.float16(0.5))) | (int(O.fp16_bits(np.float16(-1.0))) << 16)]], np.uint32)
    c, uu = O.quantize_given_meta(np.array([[-1.0, -0.75, 0.25, 9.0]]), meta, [3], p4)
    assert uu.tolist() == [[0.0, 0.5, 2.5, 20.0]]
    assert c.tolist() == [[0, 0, 2, 7]]
