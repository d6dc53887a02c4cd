"""Pins of the oracle in the per-layer geometry of Sec. 4.1 and App. F: one
transform over a layer's whole KV vector (d_kv = 8 heads x 128 for Llama and
Mistral, 4 x 128 for Qwen) with latent groups of g = 64 coefficients.

The oracle's functions are written for any d and g; these tests pin them at
this geometry by routes other than the oracle's own code: per-block
eigenvalues from numpy, Ky Fan's maximum principle, brute force over widths,
and a record laid out bit by bit by hand.
"""
import numpy as np
import pytest

import oracle as O
import synth


def _spd(rng, n, scale):
    a = rng.standard_normal((n, n))
    q, _ = np.linalg.qr(a)
    lam = scale * np.sort(rng.uniform(0.05, 1.0, n))[::-1]
    return (q * lam) @ q.T


def test_block_diagonal_moment_splits_into_the_heads():
    # Heads that are exactly uncorrelated: the per-layer eigenbasis is the union of
    # the per-head eigenbases, each direction living inside one head's block.
    rng = np.random.default_rng(11)
    H, dh = 4, 128
    blocks = [_spd(rng, dh, 1.0 + h) for h in range(H)]
    S = np.zeros((H * dh, H * dh))
    for h, b in enumerate(blocks):
        S[h * dh:(h + 1) * dh, h * dh:(h + 1) * dh] = b
    p = O.Params(head_dim=H * dh, group_size=64)
    f = O.fit_from_weights(np.eye(H * dh), S, None, p)   # W = I: the moment is S itself
    want = np.sort(np.concatenate([np.linalg.eigvalsh(b) for b in blocks]))[::-1]
    assert np.allclose(f.eigvals, want, rtol=1e-12, atol=1e-12)
    V = f.basis.astype(np.float64)
    for j in range(H * dh):
        mass = [float(np.sum(V[h * dh:(h + 1) * dh, j] ** 2)) for h in range(H)]
        assert max(mass) >= 1 - 1e-6, f"direction {j} spans several heads"


def test_layer_transform_keeps_at_least_the_per_head_energy():
    # Ky Fan: the top-r eigen-directions of the layer's second moment capture at
    # least the energy of any r orthonormal directions, in particular of the best
    # r chosen among the per-head eigenbases. Cross-head correlation makes it strict.
    w = synth.WORKLOADS["qwen_layer_8x"]
    x = synth.bf16_bits_to_f32(synth.numpy_layer_stream(w, 0, 0, 0, 2048)).astype(np.float64)
    d = x.shape[1]
    p = O.Params(head_dim=d, group_size=64)
    f = O.fit(x, p)
    S = x.T @ x / x.shape[0]
    per_head = np.sort(np.concatenate([np.linalg.eigvalsh(S[h * 128:(h + 1) * 128, h * 128:(h + 1) * 128])
                                       for h in range(d // 128)]))[::-1]
    for r in (16, 32, 64, 128, 256, 384):
        layer_r = float(np.sum(f.eigvals[:r]))
        head_r = float(np.sum(per_head[:r]))
        assert layer_r >= head_r * (1 - 1e-12)
        if r <= 64:  # below the shared rank's reach the gain is clear (the steep tails make it tiny later)
            assert layer_r > head_r * 1.01, "the shared component should reward the per-layer transform"
    # energy check by a different route: trace of the projection onto the kept directions
    V = f.basis.astype(np.float64)[:, :128]
    assert abs(np.trace(V.T @ S @ V) - np.sum(f.eigvals[:128])) <= 1e-5 * np.sum(f.eigvals[:128])


@pytest.mark.parametrize("R", [256 + 64, 600, 1000, 1400])
def test_allocation_g64_equals_bruteforce(R):
    rng = np.random.default_rng(R)
    var = np.sort(rng.lognormal(0.0, 2.0, 256))[::-1]
    p = O.Params(head_dim=256, group_size=64, budget_bits=R)
    assert O.allocate_bits(var, p) == O.allocate_bits_bruteforce(var, p)


def test_pack_g64_hand_built_record():
    # d = 256, g = 64, widths (3, 0, 1, 0): metadata words of groups 0 and 2, then
    # 6 payload words of group 0 (64 x 3 bits) and 2 of group 2 (64 x 1 bit).
    p = O.Params(head_dim=256, group_size=64, budget_bits=32 * 12)
    bits = [3, 0, 1, 0]
    codes = np.zeros((1, 256), np.uint8)
    meta = np.zeros((1, 4), np.uint32)
    meta[0, 0], meta[0, 2] = 0x3C001234, 0xBC00ABCD
    codes[0, 42] = 5          # bits 126..128 of group 0's payload: straddles words 3 and 4
    codes[0, 63] = 7          # bits 189..191: top of word 5
    codes[0, 128 + 33] = 1    # group 2, code 33: bit 1 of its second payload word
    rec = O.pack(codes, meta, bits, p)[0]
    want = np.zeros(12, np.uint32)
    want[0], want[1] = 0x3C001234, 0xBC00ABCD
    want[2 + 3] = 1 << 30     # code 42 bit 0 -> payload bit 126; bit 1 (0) -> 127
    want[2 + 4] = 1           # code 42 bit 2 -> payload bit 128
    want[2 + 5] = 7 << 29     # code 63 -> payload bits 189, 190, 191
    want[8 + 1] = 1 << 1      # group 2 payload bit 33
    assert np.array_equal(rec, want)
    c2, m2 = O.unpack(rec[None, :], bits, p)
    assert np.array_equal(c2, codes) and np.array_equal(m2, meta)


def test_layer_capacity_at_8x():
    # App. F accounting at the Llama layer geometry: d_kv = 1024 at 8x is 2048 bits
    # (64 words) per token, and each kept 64-group costs one metadata word plus 2b words.
    p = O.Params(head_dim=1024, group_size=64, ratio=8.0)
    assert O.record_budget_bits(p) == 2048 and O.record_words(p) == 64
    rng = np.random.default_rng(3)
    var = np.sort(rng.lognormal(0.0, 2.0, 1024))[::-1]
    bits = O.allocate_bits(var, p)
    used = sum(1 + 2 * b for b in bits if b > 0)
    assert used <= 64
    assert bits == sorted(bits, reverse=True)


# ---------------------------------------------------------------------------
# Square-root latent scaling (Eqs. gsvd and second-moment-latent)
# ---------------------------------------------------------------------------
def test_square_root_split_matches_the_whitened_weight_svd():
    # The paper's latent c = h W_down with W_down = G^{-1/2} U_r S_r^{1/2} and
    # M = G^{1/2} W = U S V^T, formed here with numpy's SVD and eigh; the oracle's
    # scaled latent (h W V) * f must equal it up to the sign of each column.
    rng = np.random.default_rng(5)
    dm, d, T = 96, 64, 4000
    A = rng.standard_normal((dm, dm)) * (np.arange(1, dm + 1) ** -0.7)[None, :]
    G = A @ A.T / dm + 1e-3 * np.eye(dm)
    W = rng.standard_normal((dm, d)) / np.sqrt(dm)
    gw, gv = np.linalg.eigh(G)
    Gh = (gv * np.sqrt(gw)) @ gv.T
    Gmh = (gv / np.sqrt(gw)) @ gv.T
    U, Sg, Vt = np.linalg.svd(Gh @ W, full_matrices=False)
    W_down = Gmh @ U * np.sqrt(Sg)[None, :]
    h = rng.standard_normal((T, dm)) @ Gh            # E[h^T h] = G
    c_paper = h @ W_down
    p = O.Params(head_dim=d, group_size=16)
    f = O.fit_from_weights(W, G, None, p, latent_scale=True)
    c_or = (h @ W @ f.basis.astype(np.float64)) * f.scale.astype(np.float64)[None, :]
    sign = np.sign(np.sum(c_or * c_paper, axis=0))
    assert np.all(sign != 0)
    assert np.abs(c_or * sign[None, :] - c_paper).max() <= 1e-5 * np.abs(c_paper).max()
    # and the split's energies are the singular values of M
    assert np.allclose(f.scale.astype(np.float64) ** -2, Sg, rtol=1e-6)


def test_scaled_latent_second_moment_is_the_singular_values():
    # Eq. second-moment-latent: E[c^T c] = S (diagonal, descending) for the scaled latent,
    # S the singular values of the data matrix / sqrt(T) taken from numpy's SVD.
    w = synth.WORKLOADS["qwen_layer_8x"]
    x = synth.bf16_bits_to_f32(synth.numpy_layer_stream(w, 0, 0, 1, 3000)).astype(np.float64)
    d = x.shape[1]
    p = O.Params(head_dim=d, group_size=64)
    f = O.fit(x, p, latent_scale=True)
    sv = np.linalg.svd(x / np.sqrt(x.shape[0]), compute_uv=False)
    c = (x @ f.basis.astype(np.float64)) * f.scale.astype(np.float64)[None, :]
    Mc = c.T @ c / x.shape[0]
    keep = sv > sv[0] * 1e-3
    assert np.allclose(np.diag(Mc)[keep], sv[keep], rtol=1e-4)
    off = Mc - np.diag(np.diag(Mc))
    assert np.abs(off).max() <= 1e-5 * sv[0]


def test_scaled_fit_same_reconstruction_flatter_allocation():
    # Any split gives the same reconstruction (Sec. 3.1): at 8 bits per group the scaled
    # and orthonormal codecs both reconstruct to quantization accuracy; the scaled latent's
    # variances are sqrt(lambda)-like, so its allocation spreads bits over more groups.
    w = synth.WORKLOADS["qwen_layer_8x"]
    x = synth.bf16_bits_to_f32(synth.numpy_layer_stream(w, 0, 0, 0, 2048)).astype(np.float64)
    d = x.shape[1]
    p = O.Params(head_dim=d, group_size=64, ratio=8.0)
    fo, fs = O.fit(x, p), O.fit(x, p, latent_scale=True)
    assert np.array_equal(fo.basis, fs.basis) and np.array_equal(fo.mean, fs.mean)
    bo, bs = O.allocate_bits(fo.var, p), O.allocate_bits(fs.var, p)
    assert sum(b > 0 for b in bs) >= sum(b > 0 for b in bo)
    p8 = O.Params(head_dim=d, group_size=64, budget_bits=d * 8 + 32 * (d // 64))
    full = [8] * (d // 64)
    for f in (fo, fs):
        rec, *_ = O.encode(x[:256], f.basis, f.mean, full, p8, f.scale)
        xr = O.decode(rec, f.basis, f.mean, full, p8, f.scale)
        assert np.linalg.norm(xr - x[:256]) <= 2e-2 * np.linalg.norm(x[:256])
