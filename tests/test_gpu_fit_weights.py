"""GPU parity of the fit from weights (Sec. 3.1, Eqs. gweighted and gsvd; App. B):
spectra_fit_weights against the oracle's fit_from_weights, and against the GPU's
own data fit of the keys the weights produce (the equivalence the paper's
transform rests on, checked through the C ABI)."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import codec_state, sparams

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _clear(eig):
    gap = np.minimum(np.abs(np.diff(eig, prepend=np.inf)), np.abs(np.diff(eig, append=-np.inf)))
    return gap > 1e-3 * eig[0]


def _gpu_fit(W, G, hbar, p, spl):
    dev = torch.device("cuda:0")
    codec = S.Codec(sparams(p), W.shape[0])
    S.spectra_fit_weights(codec, torch.from_numpy(W).to(dev), torch.from_numpy(G).to(dev),
                          None if hbar is None else torch.from_numpy(hbar).to(dev), streams_per_layer=spl)
    return codec


@pytest.mark.parametrize("n_layers,heads,d_model,centered,with_mean",
                         [(2, 2, 256, False, True), (1, 4, 512, True, True), (3, 1, 192, False, False)])
def test_fit_weights_matches_oracle(n_layers, heads, d_model, centered, with_mean):
    H, G, hbar, W = synth.calibration_layers(n_layers, heads, d_model, 2048, seed=n_layers + d_model)
    p = O.Params(ratio=8.0, centered=centered)
    codec = _gpu_fit(W, G, hbar if with_mean else None, p, heads)
    for s in range(W.shape[0]):
        l = s // heads
        basis, mean, bits = codec_state(codec, s)
        f = O.fit_from_weights(W[s], G[l], hbar[l] if with_mean else None, p)
        V = basis.astype(np.float64)
        assert np.abs(V.T @ V - np.eye(128)).max() <= 1e-6
        D = V.T @ f.second_moment @ V
        assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-6 * f.eigvals[0]
        cos = np.sum(V * f.basis.astype(np.float64), axis=0)
        assert np.all(cos[_clear(f.eigvals)] >= 1 - 1e-6)        # same direction, same sign convention
        var = codec.var[s].cpu().numpy()
        assert np.allclose(var, f.var, rtol=1e-5, atol=1e-7 * f.var.max())
        assert np.abs(mean - f.mean).max() <= 1e-5 * np.abs(f.mean).max() + 1e-6
        assert bits == O.allocate_bits(f.var, p)


def test_fit_weights_equals_gpu_fit_of_produced_keys():
    """spectra_fit_weights(W, G = h^T h / N, hbar) against spectra_fit_basis over the
    keys k = h W (fp32): same widths, same directions where the spectrum is separated."""
    H, G, hbar, W = synth.calibration_layers(2, 2, 256, 4096, seed=11)
    p = O.Params(ratio=8.0)
    cw = _gpu_fit(W, G, hbar, p, 2)
    keys = np.stack([(H[s // 2] @ W[s].astype(np.float64)).astype(np.float32) for s in range(4)])
    cd = S.Codec(sparams(p), 4)
    S.spectra_fit_basis(cd, torch.from_numpy(keys).cuda())
    for s in range(4):
        bw, mw, bitw = codec_state(cw, s)
        bd, md, bitd = codec_state(cd, s)
        f = O.fit_from_weights(W[s], G[s // 2], hbar[s // 2], p)
        cos = np.sum(bw.astype(np.float64) * bd.astype(np.float64), axis=0)
        assert np.all(cos[_clear(f.eigvals)] >= 1 - 1e-5)
        assert bitw == bitd
        assert np.abs(mw - md).max() <= 1e-4 * np.abs(md).max()


def _layer_projection(W, heads, l):
    """The layer's whole projection: its KV heads' columns side by side, head-major."""
    return np.ascontiguousarray(np.concatenate([W[l * heads + h] for h in range(heads)], axis=1))


@pytest.mark.parametrize("latent_scale", [False, True])
def test_fit_weights_layer_geometry_matches_oracle(latent_scale):
    """The paper's own setting: one transform from a layer's whole key projection
    (d_kv = 4 x 128, groups of 64), with and without the square-root split."""
    heads, d_model, L = 4, 512, 2
    H, G, hbar, W = synth.calibration_layers(L, heads, d_model, 2048, seed=5)
    Wl = np.stack([_layer_projection(W, heads, l) for l in range(L)])
    d = heads * 128
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    dev = torch.device("cuda:0")
    codec = S.Codec(sparams(p), L, latent_scale=latent_scale)
    S.spectra_fit_weights(codec, torch.from_numpy(Wl).to(dev), torch.from_numpy(G).to(dev),
                          torch.from_numpy(hbar).to(dev), streams_per_layer=1)
    for l in range(L):
        basis, mean, bits = codec_state(codec, l)
        f = O.fit_from_weights(Wl[l], G[l], hbar[l], p, latent_scale=latent_scale)
        V = basis.astype(np.float64)
        assert np.abs(V.T @ V - np.eye(d)).max() <= 1e-6
        D = V.T @ f.second_moment @ V
        assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-6 * f.eigvals[0]
        cos = np.sum(V * f.basis.astype(np.float64), axis=0)
        assert np.all(cos[_clear(f.eigvals)] >= 1 - 1e-6)
        var = codec.var[l].cpu().numpy()
        assert np.allclose(var, f.var, rtol=1e-5, atol=1e-7 * f.var.max())
        assert np.abs(mean - f.mean).max() <= 1e-5 * np.abs(f.mean).max() + 1e-6
        assert bits == O.allocate_bits(f.var, p)
        if latent_scale:
            assert np.allclose(codec.lscale[l].cpu().numpy(), f.scale, rtol=1e-5)


def test_fit_weights_equals_gpu_fit_of_produced_keys_d1024():
    """Through the C ABI at the Llama-3.1-8B key width (8 KV heads side by side, d_kv =
    1024): the weight fit of a layer's projection W equals the GPU's data fit of the keys
    k = h W it produces (G = h^T h / N exactly), in widths and separated directions."""
    heads, d_model = 8, 1024
    H, G, hbar, W = synth.calibration_layers(1, heads, d_model, 4096, seed=23)
    Wl = _layer_projection(W, heads, 0)[None]
    d = heads * 128
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    dev = torch.device("cuda:0")
    cw = S.Codec(sparams(p), 1)
    S.spectra_fit_weights(cw, torch.from_numpy(Wl).to(dev), torch.from_numpy(G).to(dev),
                          torch.from_numpy(hbar).to(dev), streams_per_layer=1)
    keys = (H[0] @ Wl[0].astype(np.float64)).astype(np.float32)
    cd = S.Codec(sparams(p), 1)
    S.spectra_fit_basis(cd, torch.from_numpy(keys[None]).to(dev))
    bw, mw, bitw = codec_state(cw, 0)
    bd, md, bitd = codec_state(cd, 0)
    f = O.fit_from_weights(Wl[0], G[0], hbar[0], p)
    cos = np.sum(bw.astype(np.float64) * bd.astype(np.float64), axis=0)
    assert np.all(cos[_clear(f.eigvals)] >= 1 - 1e-5)
    assert np.abs(mw - md).max() <= 1e-4 * np.abs(md).max()
    assert bitw == bitd == O.allocate_bits(f.var, p)
