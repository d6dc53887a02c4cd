"""GPU parity of fit, encode, decode and the record format against the oracle,
called through the C ABI. Sizes here let the oracle finish in seconds while
spanning several 64-token tiles and ragged tails."""
import numpy as np
import pytest

import oracle as O
import paper_2608_07915_amd as S
import synth
from gpu_parity import (check_encoded_stream, codec_state, fit_and_encode, records_of, rel_l2, sparams,
                        to_device, values_f64)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)


def _streams(w, tensor, T, n_streams=None, seed=0):
    """[S, T, d] stored values of the first n_streams (seq, layer, head) streams of a workload."""
    xs = []
    n = n_streams or w.n_kv_heads
    for i in range(n):
        seq, head = divmod(i, w.n_kv_heads)
        xs.append(synth.numpy_stream(w, seq % max(w.n_seq, 1), 0, head, tensor, n_tokens=T, seed=seed))
    return np.stack(xs)


# ---------------------------------------------------------------------------
# Fit (P2)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("tensor", [0, 1])
def test_fit_matches_oracle_tiny(tensor):
    w = synth.WORKLOADS["tiny"]
    x = _streams(w, tensor, 4096)
    p = O.Params(ratio=8.0)
    codec = S.Codec(sparams(p), 1)
    S.spectra_fit_basis(codec, to_device(x, w.dtype))
    basis, mean, bits = codec_state(codec, 0)
    f = O.fit(values_f64(x[0], w.dtype), p)
    V = basis.astype(np.float64)
    assert np.abs(V.T @ V - np.eye(128)).max() <= 1e-6
    D = V.T @ f.second_moment @ V
    assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-6 * f.eigvals[0]
    assert np.allclose(np.diag(D), f.eigvals, rtol=0, atol=1e-5 * f.eigvals[0])
    gap = np.minimum(np.abs(np.diff(f.eigvals, prepend=np.inf)), np.abs(np.diff(f.eigvals, append=-np.inf)))
    clear = gap > 1e-3 * f.eigvals[0]
    cos = np.sum(V * f.basis.astype(np.float64), axis=0)
    assert np.all(cos[clear] >= 1 - 1e-6)   # same direction and same sign convention
    var = codec.var[0].cpu().numpy()
    assert np.allclose(var, f.var, rtol=1e-5, atol=1e-7 * f.var.max())
    assert np.abs(mean - f.mean).max() <= 1e-5 * np.abs(f.mean).max() + 1e-6
    assert bits == O.allocate_bits(f.var, p)


def test_fit_bf16_several_streams_matches_oracle():
    w = synth.WORKLOADS["llama_layer_4x"]
    x = _streams(w, 0, 3000)  # 8 streams, ragged chunking
    p = O.Params(ratio=4.0)
    codec = S.Codec(sparams(p), 8)
    S.spectra_fit_basis(codec, to_device(x, w.dtype))
    for s in (0, 5, 7):
        basis, mean, bits = codec_state(codec, s)
        f = O.fit(values_f64(x[s], w.dtype), p)
        V = basis.astype(np.float64)
        D = V.T @ f.second_moment @ V
        assert np.abs(D - np.diag(np.diag(D))).max() <= 1e-6 * f.eigvals[0]
        assert bits == O.allocate_bits(f.var, p)


# ---------------------------------------------------------------------------
# Record format hooks (P5)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits", [[3, 2, 0, 0], [1, 1, 1, 1], [8, 0, 0, 0], [5, 7, 0, 2], [0, 6, 0, 4],
                                  [2, 3, 4, 5], [0, 0, 0, 0]])
def test_pack_unpack_hooks_bit_exact(bits):
    p = O.Params(budget_bits=1152)
    W = O.record_words(p)
    rng = np.random.default_rng(sum(bits) * 7 + 1)
    Sn, T, t_cap = 3, 150, 192
    codes = np.zeros((Sn, T, 128), np.uint8)
    meta = np.zeros((Sn, T, 4), np.uint32)
    for G, b in enumerate(bits):
        if b:
            codes[:, :, 32 * G:32 * G + 32] = rng.integers(0, 1 << b, size=(Sn, T, 32))
            meta[:, :, G] = rng.integers(0, 2 ** 32, size=(Sn, T), dtype=np.uint64).astype(np.uint32)
    codec = S.Codec(sparams(p), Sn)
    codec.bits.copy_(torch.tensor([bits] * Sn, dtype=torch.uint8))
    packed = codec.empty_packed(t_cap)
    packed.fill_(-1)
    S.spectra_pack_codes(codec, torch.from_numpy(codes).cuda(), torch.from_numpy(meta.view(np.int32)).cuda(),
                         packed, t_cap)
    torch.cuda.synchronize()
    for s in range(Sn):
        rec = records_of(packed, s, 0, T, t_cap, W)
        assert np.array_equal(rec, O.pack(codes[s], meta[s], bits, p))
    # slots beyond n_tokens untouched
    words = packed.cpu().numpy().view(np.uint32)
    tail = O.physical_index(0, np.arange(T, t_cap), 0, t_cap, W)
    assert np.all(words[tail] == 0xFFFFFFFF)
    # unpack of oracle-packed records
    host = np.full(codec.packed_words(t_cap), 0xFFFFFFFF, np.uint32)
    for s in range(Sn):
        rec = O.pack(codes[s], meta[s], bits, p)
        for w_ in range(W):
            host[O.physical_index(s, np.arange(T), w_, t_cap, W)] = rec[:, w_]
    c2, m2 = S.spectra_unpack_codes(codec, torch.from_numpy(host.view(np.int32)).cuda(), t_cap, T)
    assert np.array_equal(c2.cpu().numpy(), codes)
    kept = np.array(bits) > 0
    assert np.array_equal(m2.cpu().numpy().view(np.uint32)[:, :, kept], meta[:, :, kept])
    assert np.all(m2.cpu().numpy()[:, :, ~kept] == 0)


# ---------------------------------------------------------------------------
# Encode (P3, P4, P5) and decode (P6) at the three tiers and edge cases
# ---------------------------------------------------------------------------
CASES = [
    ("tiny", 0, 4096, 8.0),
    ("tiny", 1, 4096, 8.0),
    ("llama_layer_4x", 0, 2000, 4.0),
    ("llama_layer_4x", 1, 2000, 4.0),
    ("qwen_layer_8x", 0, 2500, 8.0),
    ("qwen_layer_8x", 1, 2500, 8.0),
    ("llama_batch16_12x", 0, 1500, 12.0),
    ("llama_batch16_12x", 1, 1500, 12.0),
    ("llama_model_131k_8x", 0, 1100, 8.0),
    ("llama_model_131k_8x", 1, 1100, 8.0),
    ("llama_layer_4x", 0, 700, 16.0 / 9.0),   # every group at 8 bits (near-lossless)
]


@pytest.mark.parametrize("name,tensor,T,ratio", CASES)
def test_encode_decode_parity(name, tensor, T, ratio):
    w = synth.WORKLOADS[name]
    x = _streams(w, tensor, T, n_streams=min(w.n_kv_heads, 4))
    p = O.Params(ratio=ratio)
    t_cap = (T + 63) // 64 * 64 + 64
    x_dev = to_device(x, w.dtype)
    codec, packed = fit_and_encode(x_dev, p, t_cap)
    W = O.record_words(p)
    dec_gpu = S.spectra_decode(codec, packed, t_cap, 0, T).cpu().numpy()
    for s in range(x.shape[0]):
        basis, mean, bits = codec_state(codec, s)
        if ratio < 2:
            assert bits == [8, 8, 8, 8]
        xs = values_f64(x[s], w.dtype)
        rec = records_of(packed, s, 0, T, t_cap, W)
        check_encoded_stream(xs, basis, mean, bits, p, rec)
        # P6 on identical bytes: arithmetic only
        dec_same = O.decode(rec, basis, mean, bits, p)
        assert rel_l2(dec_gpu[s], dec_same) <= 1e-6
        # P6 vs the oracle's own encode/decode
        rec_o, *_ = O.encode(xs, basis, mean, bits, p)
        dec_o = O.decode(rec_o, basis, mean, bits, p)
        assert rel_l2(dec_gpu[s], dec_o) <= 1e-3
        if ratio < 2:
            assert rel_l2(dec_gpu[s], xs) <= 1e-2


@pytest.mark.parametrize("ratio", [12.0, 8.0, 4.0, 3.0, 16.0 / 9.0])
def test_decode_many_super_tiles_per_workgroup(ratio):
    """Mode A decode of 32 streams over a window whose first and last 128-token
    super-tiles are partial: the decode grid gives each stream 16 workgroups, so some
    walk two super-tiles (records of up to 32 words double-buffered in LDS, wider ones
    through one buffer). P6 on identical bytes against the oracle for every stream."""
    w = synth.WORKLOADS["llama_batch16_12x"]
    T, t0, n = 2500, 37, 2400
    x = _streams(w, 0, T, n_streams=32)
    p = O.Params(ratio=ratio)
    t_cap = (T + 63) // 64 * 64
    codec, packed = fit_and_encode(to_device(x, w.dtype), p, t_cap)
    W = O.record_words(p)
    dec = S.spectra_decode(codec, packed, t_cap, t0, n).cpu().numpy()
    assert dec.shape == (32, n, 128)
    for s in range(32):
        basis, mean, bits = codec_state(codec, s)
        ref = O.decode(records_of(packed, s, t0, n, t_cap, W), basis, mean, bits, p)
        assert rel_l2(dec[s], ref) <= 1e-6, (ratio, s)


def test_encode_in_pieces_and_appends_equal_one_shot():
    """Slots outside [t0, t0+n) are untouched: pieces, ragged offsets and single-token
    appends give the same bytes as one call; encoding twice is bit-identical."""
    w = synth.WORKLOADS["llama_layer_4x"]
    T = 777
    x = _streams(w, 0, T, n_streams=3)
    p = O.Params(ratio=8.0)
    t_cap = 832
    x_dev = to_device(x, w.dtype)
    codec, packed1 = fit_and_encode(x_dev, p, t_cap)
    packed2 = codec.empty_packed(t_cap)
    packed2.fill_(0x5A5A5A5A)
    pieces = [(0, 100), (100, 1), (101, 63), (164, 500), (664, 50)] + [(t, 1) for t in range(714, 777)]
    for t0, n in pieces:
        S.spectra_encode(codec, x_dev[:, t0:t0 + n], t0, packed2, t_cap)
    torch.cuda.synchronize()
    W = O.record_words(p)
    for s in range(3):
        assert np.array_equal(records_of(packed1, s, 0, T, t_cap, W), records_of(packed2, s, 0, T, t_cap, W))
    packed3 = codec.empty_packed(t_cap)
    S.spectra_encode(codec, x_dev, 0, packed3, t_cap)
    torch.cuda.synchronize()
    assert torch.equal(packed1, packed3)
    # partial decode of a ragged window matches the full decode
    full = S.spectra_decode(codec, packed1, t_cap, 0, T)
    part = S.spectra_decode(codec, packed1, t_cap, 130, 77)
    assert torch.equal(full[:, 130:207], part)


def test_non_prefix_kept_groups_and_dropped_everything():
    """Width tables that keep non-adjacent groups, and a budget that drops all groups."""
    w = synth.WORKLOADS["tiny"]
    x = _streams(w, 1, 500)
    x_dev = to_device(x, w.dtype)
    p = O.Params(budget_bits=32 * 9)  # W = 9
    codec = S.Codec(sparams(p), 1)
    S.spectra_fit_basis(codec, x_dev)
    for bits in ([0, 3, 0, 4], [2, 0, 5, 0], [0, 0, 0, 7], [1, 1, 1, 0]):
        codec.bits.copy_(torch.tensor([bits], dtype=torch.uint8))
        t_cap = 512
        packed = codec.empty_packed(t_cap)
        S.spectra_encode(codec, x_dev, 0, packed, t_cap)
        torch.cuda.synchronize()
        basis, mean, _ = codec_state(codec, 0)
        rec = records_of(packed, 0, 0, 500, t_cap, 9)
        check_encoded_stream(values_f64(x[0], w.dtype), basis, mean, bits, p, rec)
        dec = S.spectra_decode(codec, packed, t_cap, 0, 500).cpu().numpy()[0]
        assert rel_l2(dec, O.decode(rec, basis, mean, bits, p)) <= 1e-6
    # budget below one group: nothing stored, decode returns the mean
    p0 = O.Params(budget_bits=40)
    c0 = S.Codec(sparams(p0), 1)
    S.spectra_fit_basis(c0, x_dev)
    assert c0.bits.cpu().numpy().tolist() == [[0, 0, 0, 0]]
    packed = c0.empty_packed(512)
    S.spectra_encode(c0, x_dev, 0, packed, 512)
    dec = S.spectra_decode(c0, packed, 512, 0, 10).cpu().numpy()[0]
    mu = values_f64(x[0], w.dtype).mean(axis=0)
    assert np.abs(dec - mu[None, :]).max() <= 1e-5 * np.abs(mu).max() + 1e-6


def test_fp32_and_bf16_inputs_agree_on_bf16_values():
    w = synth.WORKLOADS["llama_layer_4x"]
    x = _streams(w, 0, 300, n_streams=2)
    p = O.Params(ratio=8.0)
    xb = to_device(x, "bf16")
    xf = xb.float().contiguous()
    codec, pb = fit_and_encode(xb, p, 320)
    _, pf = fit_and_encode(xf, p, 320, fit=False, codec=codec)
    assert torch.equal(pb, pf)


def test_degenerate_groups_identity_basis():
    """Metadata and codes at the format's edges (Sec. 3.2 per-token min/max with fp16
    scale and zero-point): constant groups (s = 0, all codes 0), values beyond the
    fp16 range (z and s saturate at 65504), values in the fp16 subnormal range, and
    all-zero groups. The identity basis makes the coefficients the input itself."""
    T, t_cap = 300, 320
    bits = [4, 3, 8, 2]
    p = O.Params(budget_bits=32 * (4 + 4 + 3 + 8 + 2))   # metadata + payload words: W = 21
    rng = np.random.default_rng(5)
    x = np.zeros((T, 128), dtype=np.float32)
    x[:, 0:32] = rng.standard_normal((T, 32))
    const = np.arange(T) % 3 == 0
    # one fp16-representable value per token: z = min exactly, so s = 0 and all codes 0
    x[const, 0:32] = rng.standard_normal((int(const.sum()), 1)).astype(np.float16).astype(np.float32)
    x[:, 32:64] = rng.uniform(-2e5, 2e5, (T, 32))                      # beyond fp16: saturating z and s
    x[:, 64:96] = 1e-6 * rng.standard_normal((T, 32))                  # fp16 subnormal metadata
    # x[:, 96:128] stays zero
    codec = S.Codec(sparams(p), 1)
    codec.basis.copy_(torch.eye(128, dtype=torch.float32)[None])
    codec.mean.zero_()
    codec.var.fill_(1.0)
    codec.bits.copy_(torch.tensor([bits], dtype=torch.uint8))
    packed = codec.empty_packed(t_cap)
    xd = torch.from_numpy(x[None]).cuda()
    S.spectra_encode(codec, xd, 0, packed, t_cap)
    torch.cuda.synchronize()
    basis, mean, _ = codec_state(codec, 0)
    rec = records_of(packed, 0, 0, T, t_cap, O.record_words(p))
    check_encoded_stream(x.astype(np.float64), basis, mean, bits, p, rec)
    codes, meta = O.unpack(rec, bits, p)
    assert np.all(codes[const, 0:32] == 0) and np.all(meta[const, 0] & 0xFFFF == 0)    # s = 0 on constant groups
    assert np.all(codes[:, 96:128] == 0) and np.all(meta[:, 3] == 0)                    # zero groups
    assert np.any((meta[:, 1] >> 16) == 0xFBFF)                                          # z saturated at -65504
    dec = S.spectra_decode(codec, packed, t_cap, 0, T).cpu().numpy()[0]
    ref = O.decode(rec, basis, mean, bits, p)
    assert np.all(np.isfinite(dec))
    for g in range(4):
        sl = slice(32 * g, 32 * g + 32)
        scale = np.abs(ref[:, sl]).max()
        assert np.abs(dec[:, sl] - ref[:, sl]).max() <= 1e-6 * scale + 1e-30, g
