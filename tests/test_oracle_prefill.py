"""Pins of the oracle's prefill attention (CPU only).

Library routine: torch fp64 scaled_dot_product_attention with an explicit
boolean mask (query at cache position p sees keys 0..p) and the KV heads
repeated per group.  Closed forms: a full prefill's first row is V[0]; with
every key equal the scores tie and row p is the mean of V[0..p].
Consistency: each request's last row equals the decode attention of the
same sequence.  Bad requests are rejected.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F


def _filled(orc, rng, lens, H=2, D=64, bs=16, NB=256, bf16=False, K=None, V=None):
    order = rng.permutation(NB).astype(np.int32)
    c = orc.OracleCache(bf16=bf16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                        max_seqs=len(lens) + 1, max_blocks_per_seq=NB, free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    if K is None:
        K = rng.normal(size=(offs[-1], H, D)).astype(np.float32)
    if V is None:
        V = rng.normal(size=(offs[-1], H, D)).astype(np.float32)
    assert c.append(np.arange(len(lens)), offs, K, V) == orc.OK
    return c, K, V, offs


@pytest.mark.parametrize("Hq,H,ms", [(4, 4, "full"), (8, 2, "full"), (6, 3, "chunk"), (4, 1, "chunk")])
def test_matches_torch_sdpa_with_causal_mask(orc, Hq, H, ms):
    rng = np.random.RandomState(Hq * 7 + H)
    lens = [1, 17, 45, 100]
    c, K, V, offs = _filled(orc, rng, lens, H=H)
    m = list(lens) if ms == "full" else [1, 5, 45, 33]
    qo = np.concatenate([[0], np.cumsum(m)]).astype(np.int32)
    q = rng.normal(size=(qo[-1], Hq, 64))
    st, out = c.prefill_attention(np.arange(len(lens)), qo, q, Hq, 64 ** -0.5)
    assert st == orc.OK
    for i, L in enumerate(lens):
        k = torch.from_numpy(K[offs[i]:offs[i + 1]].astype(np.float64)).transpose(0, 1)
        v = torch.from_numpy(V[offs[i]:offs[i + 1]].astype(np.float64)).transpose(0, 1)
        k = k.repeat_interleave(Hq // H, dim=0).contiguous()
        v = v.repeat_interleave(Hq // H, dim=0).contiguous()
        qi = torch.from_numpy(q[qo[i]:qo[i + 1]]).transpose(0, 1).contiguous()  # [Hq, m, D]
        pos = L - m[i] + np.arange(m[i])
        mask = torch.from_numpy(np.arange(L)[None, :] <= pos[:, None])          # [m, L]
        ref = F.scaled_dot_product_attention(qi, k, v, attn_mask=mask)          # [Hq, m, D]
        np.testing.assert_allclose(out[qo[i]:qo[i + 1]], ref.transpose(0, 1).numpy(), rtol=1e-11, atol=1e-12)


def test_first_row_is_the_first_value(orc):
    rng = np.random.RandomState(3)
    c, K, V, offs = _filled(orc, rng, [30], H=1)
    q = rng.normal(size=(30, 2, 64)) * 10.0
    st, out = c.prefill_attention([0], [0, 30], q, 2, 0.125)
    assert st == orc.OK
    np.testing.assert_array_equal(out[0, 0], V[0, 0].astype(np.float64))
    np.testing.assert_array_equal(out[0, 1], V[0, 0].astype(np.float64))


def test_equal_keys_give_the_running_mean(orc):
    rng = np.random.RandomState(4)
    T = 50
    K = np.repeat(rng.normal(size=(1, 1, 64)).astype(np.float32), T, axis=0)
    c, K, V, offs = _filled(orc, rng, [T], H=1, K=K)
    q = rng.normal(size=(T, 1, 64))
    st, out = c.prefill_attention([0], [0, T], q, 1, 64 ** -0.5)
    assert st == orc.OK
    running = np.cumsum(V[:, 0].astype(np.float64), axis=0) / np.arange(1, T + 1)[:, None]
    np.testing.assert_allclose(out[:, 0], running, rtol=1e-12, atol=1e-13)


def test_last_row_is_the_decode_attention(orc):
    rng = np.random.RandomState(5)
    lens = [9, 64, 130]
    c, K, V, offs = _filled(orc, rng, lens, H=2)
    m = [9, 20, 7]
    qo = np.concatenate([[0], np.cumsum(m)]).astype(np.int32)
    q = rng.normal(size=(qo[-1], 8, 64))
    st, out = c.prefill_attention([0, 1, 2], qo, q, 8, 64 ** -0.5)
    assert st == orc.OK
    st2, dec = c.decode_attention([0, 1, 2], q[qo[1:] - 1], 8, 64 ** -0.5)
    assert st2 == orc.OK
    np.testing.assert_allclose(out[qo[1:] - 1], dec, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("bad", ["too_many_rows", "bad_id", "offsets"])
def test_bad_requests_are_rejected(orc, bad):
    rng = np.random.RandomState(6)
    c, K, V, offs = _filled(orc, rng, [10, 20], H=1)
    ids, qo = [0, 1], [0, 10, 30]
    if bad == "too_many_rows":
        qo = [0, 11, 31]
    elif bad == "bad_id":
        ids = [0, 5]
    else:
        qo = [1, 10, 30]
    q = np.zeros((qo[-1], 1, 64))
    st, _ = c.prefill_attention(ids, qo, q, 1, 0.125)
    assert st == orc.EINVAL
