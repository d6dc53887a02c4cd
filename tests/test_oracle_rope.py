"""Pins of the oracle's RoPE and Mode A with RoPE (Sec. 3.3: reconstruct, then rotate
each key at its own position) against closed forms and an independent complex-number
formulation. CPU only."""
import math

import numpy as np

import oracle as O


def _freqs(d=128, base=10000.0):
    return base ** (-np.arange(d // 2) / (d // 2))


def test_quarter_turn_by_hand():
    """d = 4: pair (0, 2) turned by a quarter turn maps e0 to e2 and e2 to -e0."""
    w = [math.pi / 2 / 3, 0.0]
    np.testing.assert_allclose(O.rope([1.0, 0, 0, 0], 3, w), [0, 0, 1, 0], atol=1e-15)
    np.testing.assert_allclose(O.rope([0, 0, 1.0, 0], 3, w), [-1, 0, 0, 0], atol=1e-15)
    np.testing.assert_allclose(O.rope([0, 5.0, 0, 7.0], 3, w), [0, 5, 0, 7], atol=1e-15)  # zero frequency


def test_rotation_group_and_norm():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 128))
    w = _freqs()
    np.testing.assert_allclose(O.rope(x, 0, w), x, atol=0)
    np.testing.assert_allclose(O.rope(O.rope(x, 17, w), 40, w), O.rope(x, 57, w), atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(O.rope(x, 123456, w), axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13)


def test_scores_depend_on_relative_position():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal(128), rng.standard_normal(128)
    w = _freqs()
    for P, t in ((100, 30), (131072, 5), (7, 7)):
        a = O.rope(q, P, w) @ O.rope(k, t, w)
        b = q @ O.rope(k, t - P, w)
        assert abs(a - b) <= 1e-10 * (abs(a) + 1)


def test_mode_a_rope_against_complex_formulation():
    """Pairs as complex numbers z = x_i + i x_{i+d/2}: the rotated score is
    Re(sum_i conj(z_q,i) z_k,i e^{i (t - P) w_i}); softmax and values as in Mode A."""
    rng = np.random.default_rng(3)
    Hq, Hkv, T, d = 4, 2, 50, 128
    q = rng.standard_normal((Hq, d))
    k = rng.standard_normal((Hkv, T, d))
    v = rng.standard_normal((Hkv, T, d))
    w = _freqs(base=500000.0)
    P = 1000
    got = O.attention_mode_a_rope(q, k, v, w, P)
    zq = q[:, :64] + 1j * q[:, 64:]
    zk = k[..., :64] + 1j * k[..., 64:]
    want = np.zeros((Hq, d))
    for h in range(Hq):
        kv = h // (Hq // Hkv)
        s = np.array([np.real(np.sum(np.conj(zq[h]) * zk[kv, t] * np.exp(1j * (t - P) * w))) for t in range(T)])
        s = s / math.sqrt(d)
        e = np.exp(s - s.max())
        want[h] = (e / e.sum()) @ v[kv]
    np.testing.assert_allclose(got, want, rtol=1e-11, atol=1e-12)


def test_zero_frequencies_reduce_to_mode_a():
    rng = np.random.default_rng(4)
    q, k, v = rng.standard_normal((2, 128)), rng.standard_normal((1, 20, 128)), rng.standard_normal((1, 20, 128))
    np.testing.assert_array_equal(O.attention_mode_a_rope(q, k, v, np.zeros(64), 19), O.attention_mode_a(q, k, v))
