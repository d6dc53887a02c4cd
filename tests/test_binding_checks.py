"""The binding's shape and size checks: a tensor that does not match the codec
raises ValueError before anything reaches the C ABI (which sees pointers only)."""
import pytest

import paper_2608_07915_amd as S

torch = pytest.importorskip("torch")


def test_host_tensors_are_rejected_before_any_call():
    c = S.Codec(S.Params(ratio=8.0), 2, device="cpu")
    x = torch.zeros(2, 64, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        S.spectra_fit_basis(c, x)
    with pytest.raises(ValueError, match="device tensor"):
        S.spectra_encode(c, x, 0, torch.zeros(2 * 64 * 8, dtype=torch.int32), 64)


@pytest.mark.gpu
@pytest.mark.skipif(not torch.cuda.is_available(), reason="no GPU")
def test_mismatched_device_tensors_raise():
    dev = "cuda"
    p = S.Params(ratio=8.0)
    ck, cv = S.Codec(p, 4), S.Codec(p, 4)
    x = torch.zeros(4, 100, 128, dtype=torch.bfloat16, device=dev)
    pk, pv = ck.empty_packed(128), cv.empty_packed(128)
    with pytest.raises(ValueError, match="n_streams"):
        S.spectra_encode(ck, x[:3], 0, pk, 128)                       # fewer streams than the codec
    with pytest.raises(ValueError, match="n_tokens"):
        S.spectra_encode(ck, x, 0, pk, 128, n_tokens=101)             # more tokens than x holds
    with pytest.raises(ValueError, match="words"):
        S.spectra_encode(ck, x, 0, pk[:100], 128)                     # packed cache too small
    with pytest.raises(ValueError, match="words"):
        S.spectra_decode(ck, pk, 256, 0, 10)                          # capacity beyond the packed words
    q = torch.zeros(1, 16, 128, dtype=torch.bfloat16, device=dev)
    with pytest.raises(ValueError, match="streams"):
        S.spectra_decode_attention(ck, cv, pk, pv, 128, 100, q, 2)    # 1 x 2 KV heads != 4 streams
    with pytest.raises(ValueError, match="multiple"):
        S.spectra_decode_attention(ck, cv, pk, pv, 128, 100, q[:, :15].contiguous(), 4)
    kn = torch.zeros(1, 4, 128, dtype=torch.bfloat16, device=dev)
    with pytest.raises(ValueError, match="k_new"):
        S.spectra_decode_step(ck, cv, pk, pv, 128, 100, kn[:, :3].contiguous(), kn, q, 4)
    W = torch.zeros(4, 128, 128, device=dev)
    G = torch.zeros(2, 128, 128, dtype=torch.float64, device=dev)
    with pytest.raises(ValueError, match="G must be"):
        S.spectra_fit_weights(ck, W, G, streams_per_layer=1)          # 4 layers expected
