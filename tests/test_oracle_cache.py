"""Pins of the oracle's paged KV cache (rollback / append), CPU only.

Closed form L_C' = L_C - (n-1) + 1 from the paper's decoding-time merge,
the invariant "roll back k entries and re-append them restores the cache
bit for bit", the invariant "rolling back a span and appending its surrogate
equals prefilling with the span replaced", and a brute-force comparison
against a plain list-of-rows model over random operation sequences.
"""
import numpy as np
import pytest

from conftest import load_golden


def _cache(orc, bf16=True, H=2, D=64, bs=16, NB=64, S=8, MB=16, order=None):
    return orc.OracleCache(bf16=bf16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                           max_seqs=S, max_blocks_per_seq=MB, free_order=order)


def _rows(rng, m, H, D, bf16=True):
    if bf16:
        return rng.randint(0, 0x7f80, size=(m, H, D)).astype(np.uint16)
    return rng.normal(size=(m, H, D)).astype(np.float32)


def _snapshot(c):
    top = int(c.free_top[0])
    return (c.k_pool.copy(), c.v_pool.copy(), c.block_table.copy(), c.lengths.copy(),
            c.free_stack[:top].copy(), top)


def _same(a, b):
    return all(np.array_equal(x, y) for x, y in zip(a, b))


def test_decode_merge_length_closed_form(orc):
    g = load_golden("decode_merge_lengths.json")
    rng = np.random.RandomState(0)
    for LC, n, expect in g["decode_cases"]:
        c = _cache(orc)
        assert c.append([3], [0, LC], _rows(rng, LC, 2, 64), _rows(rng, LC, 2, 64)) == orc.OK
        assert c.rollback([3], [n - 1]) == orc.OK          # crop the n-1 cached span tokens
        assert c.append([3], [0, 1], _rows(rng, 1, 2, 64), _rows(rng, 1, 2, 64)) == orc.OK  # surrogate
        assert c.lengths[3] == expect == LC - (n - 1) + 1


@pytest.mark.parametrize("bs", [16, 32])
@pytest.mark.parametrize("shuffled", [False, True])
def test_rollback_then_reappend_restores_cache(orc, bs, shuffled):
    rng = np.random.RandomState(bs + shuffled)
    order = rng.permutation(64).astype(np.int32) if shuffled else None
    c = _cache(orc, bs=bs, MB=1024 // bs, order=order)
    ids = [5, 1, 2]
    lens = [70, 33, 16]
    rows = {s: (_rows(rng, L, 2, 64), _rows(rng, L, 2, 64)) for s, L in zip(ids, lens)}
    offs = np.concatenate([[0], np.cumsum(lens)])
    K = np.concatenate([rows[s][0] for s in ids])
    V = np.concatenate([rows[s][1] for s in ids])
    assert c.append(ids, offs, K, V) == orc.OK
    before = _snapshot(c)
    ks = [17, 1, 16]
    assert c.rollback(ids, ks) == orc.OK
    # re-append the same rows, in the same request order
    K2 = np.concatenate([rows[s][0][L - k:] for s, L, k in zip(ids, lens, ks)])
    V2 = np.concatenate([rows[s][1][L - k:] for s, L, k in zip(ids, lens, ks)])
    assert c.append(ids, np.concatenate([[0], np.cumsum(ks)]), K2, V2) == orc.OK
    assert _same(before, _snapshot(c))


def test_random_ops_against_list_model(orc):
    rng = np.random.RandomState(42)
    H, D, bs, NB, S = 2, 64, 16, 80, 6
    c = _cache(orc, H=H, D=D, bs=bs, NB=NB, S=S, MB=40, order=rng.permutation(NB).astype(np.int32))
    model = {s: [] for s in range(S)}
    for step in range(120):
        ids = rng.choice(S, size=rng.randint(1, S + 1), replace=False).astype(np.int32)
        if rng.rand() < 0.55:
            m = rng.randint(0, 30, size=len(ids))
            offs = np.concatenate([[0], np.cumsum(m)]).astype(np.int32)
            K, V = _rows(rng, offs[-1], H, D), _rows(rng, offs[-1], H, D)
            need = sum(-(-(len(model[s]) + mm) // bs) - (-(-len(model[s]) // bs)) for s, mm in zip(ids, m))
            free = NB - sum(-(-len(model[s]) // bs) for s in range(S))
            st = c.append(ids, offs, K, V)
            if any(len(model[s]) + mm > 40 * bs for s, mm in zip(ids, m)):
                assert st == orc.ERANGE
            elif need > free:
                assert st == orc.ENOMEM
            else:
                assert st == orc.OK
                for i, s in enumerate(ids):
                    model[s] += [(K[r], V[r]) for r in range(offs[i], offs[i + 1])]
        else:
            k = np.array([rng.randint(0, len(model[s]) + 2) for s in ids], np.int32)
            st = c.rollback(ids, k)
            if any(kk > len(model[s]) for s, kk in zip(ids, k)):
                assert st == orc.ERANGE
            else:
                assert st == orc.OK
                for s, kk in zip(ids, k):
                    model[s] = model[s][:len(model[s]) - kk]
        # state equals the model; blocks are conserved and never shared
        mapped = []
        for s in range(S):
            L = len(model[s])
            assert c.lengths[s] == L
            nb = -(-L // bs)
            assert np.all(c.block_table[s, :nb] >= 0) and np.all(c.block_table[s, nb:] == -1)
            mapped += c.block_table[s, :nb].tolist()
            if L:
                Kl, Vl = c.logical_kv(s)
                np.testing.assert_array_equal(Kl, np.stack([r[0] for r in model[s]]))
                np.testing.assert_array_equal(Vl, np.stack([r[1] for r in model[s]]))
        top = int(c.free_top[0])
        assert sorted(mapped + c.free_stack[:top].tolist()) == list(range(NB))


def test_failed_calls_change_nothing(orc):
    rng = np.random.RandomState(3)
    c = _cache(orc, NB=8, MB=4)
    assert c.append([0, 1], [0, 20, 40], _rows(rng, 40, 2, 64), _rows(rng, 40, 2, 64)) == orc.OK
    snap = _snapshot(c)
    assert c.rollback([0], [21]) == orc.ERANGE               # k > length
    assert c.rollback([0, 0], [1, 1]) == orc.EINVAL          # duplicate id
    assert c.rollback([9], [1]) == orc.EINVAL                # id out of range
    assert c.rollback([1], [-1]) == orc.EINVAL               # negative k
    assert c.append([2], [0, 80], _rows(rng, 80, 2, 64), _rows(rng, 80, 2, 64)) == orc.ERANGE  # > 4 blocks
    assert c.append([2, 3], [0, 64, 128], _rows(rng, 128, 2, 64), _rows(rng, 128, 2, 64)) == orc.ENOMEM
    assert c.append([2, 2], [0, 1, 2], _rows(rng, 2, 2, 64), _rows(rng, 2, 2, 64)) == orc.EINVAL
    assert _same(snap, _snapshot(c))
    # k = 0 is a no-op, k = length empties the sequence
    assert c.rollback([0], [0]) == orc.OK
    assert _same(snap, _snapshot(c))
    assert c.rollback([0], [20]) == orc.OK and c.lengths[0] == 0


def test_rollback_and_surrogate_equals_prefill_with_surrogate(orc):
    """Merging equals prefilling the surrogate, on the test-only layer: a decode-time merge of the
    last n tokens (crop n-1 cached entries, append the surrogate's K/V at the
    compressed position) gives the cache of a prefill in which the span was
    replaced by the surrogate from the start; the surrogate's query then
    attends exactly like the last row of causal attention over that prefill."""
    rng = np.random.RandomState(7)
    d, Hq, H, D = 32, 4, 2, 16
    Wq, Wk, Wv = (rng.normal(0, 0.3, size=(o, d)) for o in (Hq * D, H * D, H * D))
    L, n = 23, 3
    x = rng.normal(size=(L, d))        # raw token embeddings; the last n form the span
    z = rng.normal(size=(1, d))        # its surrogate embedding
    f32 = lambda a: a.astype(np.float32)
    # A: raw prefill of the first L-1 tokens (the newest is not cached yet)
    qa, ka, va = orc.layer_qkv(x[:L - 1], np.arange(L - 1), Wq, Wk, Wv, Hq, H, D)
    A = _cache(orc, bf16=False, H=H, D=D, bs=16, NB=8, S=2, MB=4)
    assert A.append([0], [0, L - 1], f32(ka), f32(va)) == orc.OK
    assert A.rollback([0], [n - 1]) == orc.OK
    pos = int(A.lengths[0])            # compressed position of the surrogate
    qz, kz, vz = orc.layer_qkv(z, [pos], Wq, Wk, Wv, Hq, H, D)
    assert A.append([0], [0, 1], f32(kz), f32(vz)) == orc.OK
    # B: prefill of [x_0 .. x_{L-n-1}, z] at contiguous positions
    xb = np.concatenate([x[:L - n], z])
    qb, kb, vb = orc.layer_qkv(xb, np.arange(L - n + 1), Wq, Wk, Wv, Hq, H, D)
    B = _cache(orc, bf16=False, H=H, D=D, bs=16, NB=8, S=2, MB=4, order=np.arange(8)[::-1].copy())
    assert B.append([1], [0, L - n + 1], f32(kb), f32(vb)) == orc.OK
    assert A.lengths[0] == B.lengths[1] == L - (n - 1)
    KA, VA = A.logical_kv(0)
    KB, VB = B.logical_kv(1)
    np.testing.assert_array_equal(KA, KB)
    np.testing.assert_array_equal(VA, VB)
    # attention of the surrogate's query: oracle decode == causal last row
    st, oa = A.decode_attention([0], qz, Hq, D ** -0.5)
    assert st == orc.OK
    Kf, Vf = KB.astype(np.float64), VB.astype(np.float64)
    G = Hq // H
    for h in range(Hq):
        s = Kf[:, h // G] @ qb[-1, h] * D ** -0.5
        p = np.exp(s - s.max())
        p /= p.sum()
        np.testing.assert_allclose(oa[0, h], p @ Vf[:, h // G], rtol=1e-12, atol=1e-13)


def test_rope_offsets_unchanged_before_the_span(orc):
    # "Structural effect under RoPE": for two entries before the merged span,
    # q.k is the same whether or not the span was merged
    rng = np.random.RandomState(1)
    d, D = 16, 8
    Wq, Wk, Wv = (rng.normal(size=(D, d)) for _ in range(3))
    x = rng.normal(size=(6, d))
    q1, k1, _ = orc.layer_qkv(x, [0, 1, 2, 3, 4, 5], Wq, Wk, Wv, 1, 1, D)
    q2, k2, _ = orc.layer_qkv(x, [0, 1, 2, 2, 3, 4], Wq, Wk, Wv, 1, 1, D)  # tokens 2,3 merged
    assert np.isclose(q1[1, 0] @ k1[0, 0], q2[1, 0] @ k2[0, 0], rtol=1e-12)
    # pairs after the span share the same shift: their offsets are unchanged
    assert np.isclose(q1[5, 0] @ k1[4, 0], q2[5, 0] @ k2[4, 0], rtol=1e-12)
    # a pair across the span is shortened by one position
    assert not np.isclose(q1[5, 0] @ k1[0, 0], q2[5, 0] @ k2[0, 0], rtol=1e-9)


def test_crop_append_against_list_model(orc):
    """crop_append (the decode-time merge update as one step): every request
    goes from L to L - k + 1 entries, its logical K/V is its first L - k rows
    plus the new one, and blocks are conserved; when any check fails the
    whole cache is as before, even where the crop alone would have
    succeeded."""
    rng = np.random.RandomState(77)
    H, D, bs, NB, S = 2, 64, 16, 24, 6
    c = _cache(orc, H=H, D=D, bs=bs, NB=NB, S=S, MB=12, order=rng.permutation(NB).astype(np.int32))
    model = {s: [] for s in range(S)}
    n_ok = n_fail = 0
    for step in range(200):
        ids = rng.choice(S, size=rng.randint(1, S + 1), replace=False).astype(np.int32)
        if rng.rand() < 0.3:  # grow
            m = rng.randint(0, 40, size=len(ids))
            offs = np.concatenate([[0], np.cumsum(m)]).astype(np.int32)
            K, V = _rows(rng, offs[-1], H, D), _rows(rng, offs[-1], H, D)
            if c.append(ids, offs, K, V) == orc.OK:
                for i, s in enumerate(ids):
                    model[s] += [(K[r], V[r]) for r in range(offs[i], offs[i + 1])]
            continue
        k = np.array([rng.randint(0, min(len(model[s]), 9) + 1) if rng.rand() < 0.9 else len(model[s])
                      for s in ids], np.int32)
        if rng.rand() < 0.05:
            k[0] = len(model[ids[0]]) + 1          # crop longer than the cache
        K, V = _rows(rng, len(ids), H, D), _rows(rng, len(ids), H, D)
        snap = _snapshot(c)
        st = c.crop_append(ids, k, K, V)
        if any(kk > len(model[s]) for s, kk in zip(ids, k)):
            assert st == orc.ERANGE
        elif any(len(model[s]) - kk + 1 > 12 * bs for s, kk in zip(ids, k)):
            assert st == orc.ERANGE
        else:
            used = sum(-(-(len(model[s]) - kk + (s in ids and 1)) // bs) if s in ids else -(-len(model[s]) // bs)
                       for s, kk in zip(list(range(S)), [dict(zip(ids, k)).get(s, 0) for s in range(S)]))
            assert st == (orc.OK if used <= NB else orc.ENOMEM)
        if st == orc.OK:
            n_ok += 1
            for i, s in enumerate(ids):
                model[s] = model[s][:len(model[s]) - k[i]] + [(K[i], V[i])]
        else:
            n_fail += 1
            assert _same(snap, _snapshot(c))
        mapped = []
        for s in range(S):
            L = len(model[s])
            assert c.lengths[s] == L
            nb = -(-L // bs)
            mapped += c.block_table[s, :nb].tolist()
            assert np.all(c.block_table[s, nb:] == -1)
            if L:
                Kl, Vl = c.logical_kv(s)
                np.testing.assert_array_equal(Kl, np.stack([r[0] for r in model[s]]))
                np.testing.assert_array_equal(Vl, np.stack([r[1] for r in model[s]]))
        top = int(c.free_top[0])
        assert sorted(mapped + c.free_stack[:top].tolist()) == list(range(NB))
    assert n_ok > 50 and n_fail > 5


def test_crop_append_failure_after_a_good_crop_restores(orc):
    """The append fails for want of a block after the crop succeeded: the
    two separate calls would leave the crop applied; the one update leaves
    nothing."""
    rng = np.random.RandomState(5)
    c = _cache(orc, NB=6, MB=4, S=4)   # filled: no free block
    assert c.append([0, 1], [0, 32, 64], _rows(rng, 64, 2, 64), _rows(rng, 64, 2, 64)) == orc.OK
    assert c.append([2], [0, 32], _rows(rng, 32, 2, 64), _rows(rng, 32, 2, 64)) == orc.OK
    snap = _snapshot(c)
    # request 0 crops 1 (no block freed); requests 1 and 2 end pages and need 2 blocks, none free
    st = c.crop_append([0, 1, 2], [1, 0, 0], _rows(rng, 3, 2, 64), _rows(rng, 3, 2, 64))
    assert st == orc.ENOMEM
    assert _same(snap, _snapshot(c))
    # a crop that frees a page makes room: request 0 frees its second page, request 1 pops it
    st = c.crop_append([0, 1], [17, 0], _rows(rng, 2, 2, 64), _rows(rng, 2, 2, 64))
    assert st == orc.OK
    assert c.lengths[0] == 16 and c.lengths[1] == 33
    assert c.block_table[1, 2] == snap[2][0, 1]   # the block request 0 gave up
