"""The oracle's rotary position encoding, pinned to sources outside the
oracle: the inverse-frequency schedule theta^(-2j/D) for every pair j
(not only j = 0), the rotate-half pairing (j, j + D/2) and the rotation's
sign.

* A hand-computed closed form at D = 4, theta = 500000: pair 0 turns by p
  radians and pair 1 by p * theta^(-1/2).
* The Llama rotary embedding of the transformers library (its inverse
  frequencies, rotate_half and apply_rotary_pos_emb) in float64 at
  head_dim 128, theta = 500000, for the query and key heads of the
  test-only layer and for the K state of an input row at its compressed
  position ("Positional Encoding under Token-Span Merging": the surrogate
  takes the compressed position, and RoPE acts on that position only).
A wrong exponent (say theta^(-j/D)) or a swapped pairing fails both."""
import numpy as np
import pytest


def _cache(orc, H, D, lengths, bs=16):
    mb = max(-(-L // bs) for L in lengths) + 1
    oc = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs,
                         num_blocks=len(lengths) * mb + 4, max_seqs=len(lengths), max_blocks_per_seq=mb)
    offs = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    z = np.zeros((int(offs[-1]), H, D), np.uint16)
    assert oc.append(np.arange(len(lengths)), offs, z, z) == orc.OK
    return oc


def test_second_pair_turns_by_theta_power(orc):
    # D = 4: pairs (0, 2) and (1, 3) with inverse frequencies 1 and
    # theta^(-2/4); an identity projection exposes the rotated RMS-normed x
    theta, p = 500000.0, 3
    x = np.array([[1.0, 2.0, -0.5, 0.25]])
    W = np.eye(4)
    q, k, v = orc.layer_qkv(x, [p], W, W, W, 1, 1, 4, rope_theta=theta, rms_eps=0.0)
    xn = x[0] / np.sqrt(np.mean(x[0] ** 2))
    a0, a1 = p * 1.0, p * theta ** -0.5          # 3 rad and 3 / sqrt(500000) rad
    want = np.array([xn[0] * np.cos(a0) - xn[2] * np.sin(a0),
                     xn[1] * np.cos(a1) - xn[3] * np.sin(a1),
                     xn[2] * np.cos(a0) + xn[0] * np.sin(a0),
                     xn[3] * np.cos(a1) + xn[1] * np.sin(a1)])
    np.testing.assert_allclose(q[0, 0], want, rtol=0, atol=1e-14)
    np.testing.assert_allclose(k[0, 0], want, rtol=0, atol=1e-14)
    np.testing.assert_allclose(v[0, 0], xn, rtol=0, atol=1e-14)    # V carries no position
    # the same through the K/V state at the cached length p
    oc = _cache(orc, 1, 4, [p])
    st, K, V = oc.kv_project([0], x, W, W, rope_theta=theta, rms_eps=0.0)
    assert st == orc.OK
    np.testing.assert_allclose(K[0, 0], want, rtol=0, atol=1e-14)
    # a wrong exponent would turn pair 1 by p * theta^(-1/4) instead
    wrong = xn[1] * np.cos(p * theta ** -0.25) - xn[3] * np.sin(p * theta ** -0.25)
    assert abs(K[0, 0, 1] - wrong) > 1e-3


def _transformers_rope():
    pytest.importorskip("transformers")
    import torch
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding, apply_rotary_pos_emb
    return torch, LlamaConfig, LlamaRotaryEmbedding, apply_rotary_pos_emb


def _reference_qk(xn, pos, Wq, Wk, Hq, Hk, D, theta):
    """Rotated q and k of RMS-normed rows by the transformers Llama rotary
    embedding: its inverse frequencies (widened to float64) and its
    apply_rotary_pos_emb, with cos / sin of float64 angles."""
    torch, LlamaConfig, LlamaRotaryEmbedding, apply_rotary_pos_emb = _transformers_rope()
    cfg = LlamaConfig(hidden_size=xn.shape[1], num_attention_heads=Hq, num_key_value_heads=Hk, head_dim=D,
                      rope_theta=theta, max_position_embeddings=1 << 20)
    inv = LlamaRotaryEmbedding(cfg).inv_freq.to(torch.float64)           # [D / 2]
    ang = torch.as_tensor(np.asarray(pos, np.float64))[:, None] * inv[None, :]
    emb = torch.cat((ang, ang), dim=-1)                                   # [T, D]
    cos, sin = emb.cos()[None], emb.sin()[None]                          # [1, T, D]
    x = torch.as_tensor(xn)
    qh = (x @ torch.as_tensor(Wq).T).view(len(pos), Hq, D).transpose(0, 1)[None]   # [1, Hq, T, D]
    kh = (x @ torch.as_tensor(Wk).T).view(len(pos), Hk, D).transpose(0, 1)[None]
    qr, kr = apply_rotary_pos_emb(qh, kh, cos, sin)
    return qr[0].transpose(0, 1).numpy(), kr[0].transpose(0, 1).numpy()


def test_layer_qkv_matches_transformers_llama_rope(orc):
    rng = np.random.RandomState(11)
    d, Hq, Hk, D, theta = 64, 4, 2, 128, 500000.0
    pos = [0, 1, 2, 7, 33, 64]
    x = rng.randn(len(pos), d)
    Wq, Wk, Wv = (rng.randn(H * D, d) / np.sqrt(d) for H in (Hq, Hk, Hk))
    q, k, v = orc.layer_qkv(x, pos, Wq, Wk, Wv, Hq, Hk, D, rope_theta=theta, rms_eps=1e-5)
    xn = x / np.sqrt(np.mean(x ** 2, axis=1, keepdims=True) + 1e-5)
    qr, kr = _reference_qk(xn, pos, Wq, Wk, Hq, Hk, D, theta)
    # the library's inverse frequencies are float32: angles agree to about
    # 64 * 2^-24 rad, far inside this bound and far below a schedule error
    np.testing.assert_allclose(q, qr, rtol=0, atol=2e-5)
    np.testing.assert_allclose(k, kr, rtol=0, atol=2e-5)
    np.testing.assert_allclose(v, (xn @ Wv.T).reshape(len(pos), Hk, D), rtol=0, atol=1e-12)


def test_kv_project_matches_transformers_llama_rope(orc):
    rng = np.random.RandomState(12)
    d, H, D, theta = 96, 2, 128, 500000.0
    lengths = [5, 0, 61]                        # the rows land at these compressed positions
    x = rng.randn(3, d)
    Wk, Wv = rng.randn(H * D, d) / np.sqrt(d), rng.randn(H * D, d) / np.sqrt(d)
    oc = _cache(orc, H, D, lengths)
    st, K, V = oc.kv_project([0, 1, 2], x, Wk, Wv, rope_theta=theta, rms_eps=1e-5)
    assert st == orc.OK
    xn = x / np.sqrt(np.mean(x ** 2, axis=1, keepdims=True) + 1e-5)
    _, kr = _reference_qk(xn, lengths, Wk, Wk, H, H, D, theta)
    np.testing.assert_allclose(K, kr, rtol=0, atol=2e-5)
    np.testing.assert_allclose(V, (xn @ Wv.T).reshape(3, H, D), rtol=0, atol=1e-12)
