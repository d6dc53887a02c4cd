"""Pins of the oracle's fit from weights (Sec. 3.1, Eqs. gweighted and gsvd; App. B)
against the whitened-weight SVD itself and against the fit of the keys the
weights produce. CPU only."""
import numpy as np
import pytest

import oracle as O
import synth


@pytest.fixture(scope="module")
def calib():
    return synth.calibration_layers(2, 2, 256, 4096, seed=3)


def _clear(eig):
    gap = np.minimum(np.abs(np.diff(eig, prepend=np.inf)), np.abs(np.diff(eig, append=-np.inf)))
    return gap > 1e-3 * eig[0]


def test_basis_is_right_singular_vectors_of_whitened_weight(calib):
    """M = G^{1/2} W = U S V^T (G^{1/2} from a symmetric eigendecomposition of G):
    eigenvalues S^2 and directions V up to sign."""
    H, G, hbar, W = calib
    p = O.Params(ratio=8.0)
    for s in (0, 3):
        Gl, Ws = G[s // 2], W[s].astype(np.float64)
        lam, Q = np.linalg.eigh(Gl)
        Ghalf = (Q * np.sqrt(np.clip(lam, 0, None))[None, :]) @ Q.T
        U, sv, Vt = np.linalg.svd(Ghalf @ Ws, full_matrices=False)
        f = O.fit_from_weights(Ws, Gl, hbar[s // 2], p)
        np.testing.assert_allclose(f.eigvals, sv ** 2, rtol=1e-10, atol=1e-12 * sv[0] ** 2)
        cos = np.abs(np.sum(f.basis.astype(np.float64) * Vt.T, axis=0))
        assert np.all(cos[_clear(f.eigvals)] >= 1 - 1e-6)


@pytest.mark.parametrize("centered", [False, True])
def test_equals_fit_of_the_produced_keys(calib, centered):
    """With G and hbar the sample moments of the inputs h, the fit from weights is the
    fit of the keys k = h W (the cache fit), to rounding."""
    H, G, hbar, W = calib
    p = O.Params(ratio=8.0, centered=centered)
    for s in range(4):
        l = s // 2
        f = O.fit_from_weights(W[s], G[l], hbar[l], p)
        g = O.fit(H[l] @ W[s].astype(np.float64), p)
        np.testing.assert_allclose(f.eigvals, g.eigvals, rtol=1e-9, atol=1e-12 * g.eigvals[0])
        assert np.abs(f.basis - g.basis).max() <= 1e-6
        np.testing.assert_allclose(f.var, g.var, rtol=1e-8, atol=1e-12 * g.var.max())
        assert np.abs(f.mean - g.mean).max() <= 1e-5 * np.abs(g.mean).max()
        assert O.allocate_bits(f.var, p) == O.allocate_bits(g.var, p)


def test_zero_mean_inputs(calib):
    """hbar = None is zero-mean input: coefficient means vanish and the centered and
    uncentered fits coincide."""
    H, G, hbar, W = calib
    f = O.fit_from_weights(W[1], G[0], None, O.Params(ratio=8.0))
    fc = O.fit_from_weights(W[1], G[0], None, O.Params(ratio=8.0, centered=True))
    assert np.all(f.mean == 0)
    np.testing.assert_allclose(f.var, fc.var, rtol=1e-12)
    np.testing.assert_allclose(f.var, f.eigvals, rtol=1e-6, atol=1e-9 * f.eigvals[0])
