"""Seeded synthetic layer inputs and key projections for the fit from weights.

Recipe per layer l (numpy ``default_rng([seed, 7, l])``): layer inputs
h = z diag(sqrt(lambda)) Q^T + mu with lambda_i = i^-alpha (i = 1..d_model,
normalised to mean 1), Q Haar-orthogonal, mu ~ N(0, 0.25)^d_model and z ~ N(0,1)
over n_tokens rows; then, per KV head, a projection W ~ N(0, 1/d_model)^{d_model x 128}
rounded to fp32. The calibration statistics are the sample second moment
G = h^T h / n_tokens and mean hbar = sum_t h_t / n_tokens (fp64), the quantities
a forward hook on the attention input accumulates (App. B). The inputs h are
returned too so that a consumer can form the keys k = h W itself.
"""
from __future__ import annotations

import numpy as np


def calibration_layers(n_layers: int, heads: int, d_model: int, n_tokens: int, alpha: float = 1.2,
                       seed: int = 0):
    """Returns (H [L][n_tokens][d_model] f64, G [L][d_model][d_model] f64, hbar [L][d_model] f64,
    W [L*heads][d_model][128] f32)."""
    Hs, Gs, hbars, Ws = [], [], [], []
    for layer in range(n_layers):
        rng = np.random.default_rng([seed, 7, layer])
        a = rng.standard_normal((d_model, d_model))
        q, r = np.linalg.qr(a)
        q = q * np.sign(np.diag(r))[None, :]
        lam = np.arange(1, d_model + 1, dtype=np.float64) ** (-alpha)
        lam *= d_model / lam.sum()
        mu = 0.5 * rng.standard_normal(d_model)
        z = rng.standard_normal((n_tokens, d_model))
        h = (z * np.sqrt(lam)[None, :]) @ q.T + mu
        Hs.append(h)
        Gs.append(h.T @ h / n_tokens)
        hbars.append(h.sum(axis=0) / n_tokens)
        for _ in range(heads):
            Ws.append((rng.standard_normal((d_model, 128)) / np.sqrt(d_model)).astype(np.float32))
    return np.stack(Hs), np.stack(Gs), np.stack(hbars), np.stack(Ws)
