"""Pins of the oracle's decode attention (CPU only).

Brute force: the full causal attention matrix of a tiny sequence, whose last
row is the decode step.  Library routine: torch fp64
scaled_dot_product_attention with the KV heads repeated per group
(repeat_interleave, i.e. query head h reads KV head h // G).  Invariant:
softmax rows sum to one.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F


def _filled(orc, rng, lens, H=2, D=64, bs=16, NB=128, bf16=False, shuffled=True):
    order = rng.permutation(NB).astype(np.int32) if shuffled else None
    c = orc.OracleCache(bf16=bf16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                        max_seqs=len(lens) + 1, max_blocks_per_seq=NB, free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K = rng.normal(size=(offs[-1], H, D)).astype(np.float32)
    V = rng.normal(size=(offs[-1], H, D)).astype(np.float32)
    assert c.append(np.arange(len(lens)), offs, K, V) == orc.OK
    return c, K, V, offs


def test_last_row_of_full_causal_attention(orc):
    rng = np.random.RandomState(0)
    T, H, D = 37, 1, 64
    c, K, V, _ = _filled(orc, rng, [T], H=H, D=D)
    Q = rng.normal(size=(T, 1, D))
    scale = D ** -0.5
    S = (Q[:, 0] @ K[:, 0].astype(np.float64).T) * scale
    S[np.triu_indices(T, 1)] = -np.inf          # causal mask
    P = np.exp(S - S.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    full = P @ V[:, 0].astype(np.float64)
    st, out = c.decode_attention([0], Q[-1:], 1, scale)
    assert st == orc.OK
    np.testing.assert_allclose(out[0, 0], full[-1], rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("Hq,H", [(4, 4), (8, 2), (7, 1), (6, 3)])
def test_grouped_query_matches_torch_sdpa(orc, Hq, H):
    rng = np.random.RandomState(Hq * 10 + H)
    lens = [1, 16, 45, 100]
    c, K, V, offs = _filled(orc, rng, lens, H=H, D=64)
    q = rng.normal(size=(len(lens), Hq, 64))
    st, out = c.decode_attention(np.arange(len(lens)), q, Hq, 64 ** -0.5)
    assert st == orc.OK
    for i, L in enumerate(lens):
        k = torch.from_numpy(K[offs[i]:offs[i + 1]].astype(np.float64)).transpose(0, 1)  # [H, L, D]
        v = torch.from_numpy(V[offs[i]:offs[i + 1]].astype(np.float64)).transpose(0, 1)
        k = k.repeat_interleave(Hq // H, dim=0).contiguous()
        v = v.repeat_interleave(Hq // H, dim=0).contiguous()
        ref = F.scaled_dot_product_attention(torch.from_numpy(q[i])[:, None, :], k, v)[:, 0]
        np.testing.assert_allclose(out[i], ref.numpy(), rtol=1e-11, atol=1e-12)


def test_softmax_rows_sum_to_one(orc):
    rng = np.random.RandomState(2)
    lens = [3, 64, 129]
    c, *_ = _filled(orc, rng, lens, H=2, D=64)
    q = rng.normal(0, 3.0, size=(3, 4, 64))
    st, out, probs = c.decode_attention([0, 1, 2], q, 4, 0.125, return_probs=True)
    assert st == orc.OK
    for i, L in enumerate(lens):
        np.testing.assert_allclose(probs[i, :, :L].sum(axis=1), 1.0, atol=1e-12)


def test_empty_sequence_and_bad_id(orc):
    rng = np.random.RandomState(3)
    c, *_ = _filled(orc, rng, [5, 0], H=1, D=64)
    st, out = c.decode_attention([1], rng.normal(size=(1, 1, 64)), 1, 0.125)
    assert st == orc.OK and np.all(out == 0)
    st, out = c.decode_attention([7], rng.normal(size=(1, 1, 64)), 1, 0.125)
    assert st == orc.EINVAL and np.all(out == 0)


def test_bf16_pool_reads_exact_values(orc):
    # bf16 storage widens exactly: a pool holding the bits of 1.5 and 2.0
    c = orc.OracleCache(bf16=True, num_kv_heads=1, head_dim=64, block_size=16, num_blocks=2,
                        max_seqs=1, max_blocks_per_seq=2)
    K = np.full((1, 1, 64), 0x3fc0, np.uint16)   # 1.5
    V = np.full((1, 1, 64), 0x4000, np.uint16)   # 2.0
    assert c.append([0], [0, 1], K, V) == orc.OK
    st, out = c.decode_attention([0], np.ones((1, 1, 64)), 1, 1.0)
    assert st == orc.OK and np.all(out == 2.0)
