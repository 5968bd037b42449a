"""The oracle's K/V state of an input row at its compressed position, pinned
by closed forms of its parts: a single rotary pair rotates by exactly p
radians, rotation keeps every pair's norm, scores depend only on the
relative position, V carries no position, RMSNorm is scale invariant, and
the position is the sequence's cached length."""
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


def test_single_pair_rotates_by_position(orc):
    # D = 2: one rotary pair with inverse frequency theta^0 = 1, so the key
    # at position p is the position-0 key turned by p radians
    d, p = 4, 7
    oc = _cache(orc, 1, 2, [p])
    Wk = np.array([[1.0, 0, 0, 0], [0, 1.0, 0, 0]])
    x = np.array([[3.0, 4.0, 0.0, 0.0]])
    st, K, V = oc.kv_project([0], x, Wk, Wk, rms_eps=0.0)
    assert st == orc.OK
    r = np.sqrt((9 + 16) / 4)                     # RMSNorm of x
    k1, k2 = 3 / r, 4 / r
    np.testing.assert_allclose(K[0, 0], [k1 * np.cos(p) - k2 * np.sin(p), k2 * np.cos(p) + k1 * np.sin(p)],
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(V[0, 0], [k1, k2], rtol=1e-12)   # V is not rotated


def test_norms_relative_position_and_scale(orc):
    rng = np.random.RandomState(0)
    H, D, d = 2, 16, 24
    Wk, Wv = rng.randn(H * D, d), rng.randn(H * D, d)
    x = rng.randn(2, d)
    oc0 = _cache(orc, H, D, [0, 0])
    _, K0, V0 = oc0.kv_project([0, 1], x, Wk, Wv, rope_theta=10000.0)
    oc = _cache(orc, H, D, [5, 2])
    _, Ka, Va = oc.kv_project([0, 1], x, Wk, Wv, rope_theta=10000.0)
    # rotation keeps the norm of every (i, i + D/2) pair
    half = D // 2
    for t in range(2):
        for h in range(H):
            n0 = K0[t, h, :half] ** 2 + K0[t, h, half:] ** 2
            na = Ka[t, h, :half] ** 2 + Ka[t, h, half:] ** 2
            np.testing.assert_allclose(na, n0, rtol=1e-12)
    np.testing.assert_allclose(Va, V0, rtol=1e-12)
    # q.k depends only on the position difference: (5, 2) and (13, 10)
    oc2 = _cache(orc, H, D, [13, 10])
    _, Kb, _ = oc2.kv_project([0, 1], x, Wk, Wv, rope_theta=10000.0)
    for h in range(H):
        assert np.isclose(Ka[0, h] @ Ka[1, h], Kb[0, h] @ Kb[1, h], rtol=1e-10)
    assert not np.isclose(Ka[0, h] @ Ka[1, h], K0[0, h] @ K0[1, h], rtol=1e-6)
    # RMSNorm: a positive rescale of the input changes nothing (eps = 0)
    _, Ks, Vs = oc.kv_project([0, 1], 3.7 * x, Wk, Wv, rope_theta=10000.0, rms_eps=0.0)
    _, Ku, Vu = oc.kv_project([0, 1], x, Wk, Wv, rope_theta=10000.0, rms_eps=0.0)
    np.testing.assert_allclose(Ks, Ku, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Vs, Vu, rtol=1e-12, atol=1e-12)


def test_position_is_the_cached_length(orc):
    rng = np.random.RandomState(1)
    H, D, d = 2, 8, 16
    Wk, Wv, Wq = rng.randn(H * D, d), rng.randn(H * D, d), rng.randn(H * D, d)
    x = rng.randn(3, d)
    oc = _cache(orc, H, D, [4, 0, 37])
    st, K, V = oc.kv_project([2, 0, 1], x, Wk, Wv)
    assert st == orc.OK
    _, k_ref, v_ref = orc.layer_qkv(x, [37, 4, 0], Wq, Wk, Wv, H, H, D)
    np.testing.assert_allclose(K, k_ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(V, v_ref, rtol=1e-12, atol=1e-12)
    st, *_ = oc.kv_project([3], x[:1], Wk, Wv)
    assert st == orc.EINVAL
