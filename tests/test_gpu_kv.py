"""GPU kv_rollback / kv_append vs the oracle: block tables, lengths, free
stack and every pool byte must match bit for bit; error words must match the
oracle's status."""
import numpy as np
import pytest
import torch

from gpu_util import ERR_OF_STATUS, assert_same_state, dev, gpu_cache_like, i32, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _raw_rows(rng, m, H, D, dtype):
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((m, H, D), dtype, g)
    V = wl.randn((m, H, D), dtype, g)
    return K, V


def _append_both(orc, oc, c, ids, m, rng, dtype):
    offs = np.concatenate([[0], np.cumsum(m)]).astype(np.int32)
    K, V = _raw_rows(rng, int(offs[-1]), oc.H, oc.D, dtype)
    st = oc.append(ids, offs, wl.to_raw(K), wl.to_raw(V))
    sm.kv_append(c, i32(ids), i32(offs), K.to(dev()), V.to(dev()))
    return st


@pytest.mark.parametrize("dtype,H,D,bs", [(torch.bfloat16, 8, 128, 16), (torch.bfloat16, 4, 64, 32),
                                         (torch.float32, 4, 64, 512), (torch.float32, 2, 128, 16)])
def test_random_ops_bit_exact(orc, dtype, H, D, bs):
    rng = np.random.RandomState(H * 1000 + bs)
    NB, S, MB = 96, 8, 48
    oc = orc.OracleCache(bf16=dtype == torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=bs,
                         num_blocks=NB, max_seqs=S, max_blocks_per_seq=MB,
                         free_order=rng.permutation(NB).astype(np.int32))
    c = gpu_cache_like(oc, dtype)
    for step in range(60):
        ids = rng.choice(S, size=rng.randint(1, S + 1), replace=False).astype(np.int32)
        if rng.rand() < 0.6:
            m = rng.randint(0, 3 * bs // 2 + 2, size=len(ids))
            say("append", step, ids.tolist(), m.tolist())
            st = _append_both(orc, oc, c, ids, m, rng, dtype)
        else:
            k = np.array([rng.randint(0, int(oc.lengths[s]) + 3) for s in ids], np.int32)
            say("rollback", step, ids.tolist(), k.tolist())
            st = oc.rollback(ids, k)
            sm.kv_rollback(c, i32(ids), i32(k))
        torch.cuda.synchronize()
        assert c.error_bits() == ERR_OF_STATUS[st], (st, c.error_bits())
        c.clear_error()
        assert_same_state(c, oc)


def test_errors_leave_state_and_err_is_sticky(orc):
    rng = np.random.RandomState(5)
    dtype = torch.bfloat16
    oc = orc.OracleCache(bf16=True, num_kv_heads=2, head_dim=64, block_size=16, num_blocks=8,
                         max_seqs=4, max_blocks_per_seq=4)
    c = gpu_cache_like(oc, dtype)
    assert _append_both(orc, oc, c, [0, 1], [20, 20], rng, dtype) == orc.OK
    torch.cuda.synchronize()
    assert_same_state(c, oc)
    cases = [
        ("rollback", [0], [21]), ("rollback", [0, 0], [1, 1]), ("rollback", [3], [-1]),
        ("append", [2], [80]), ("append", [2, 3], [64, 64]), ("append", [2, 2], [1, 1]),
    ]
    for kind, ids, arg in cases:
        say("error case", kind, ids, arg)
        if kind == "rollback":
            st = oc.rollback(ids, arg)
            sm.kv_rollback(c, i32(ids), i32(arg))
        else:
            st = _append_both(orc, oc, c, np.array(ids, np.int32), np.array(arg), rng, dtype)
        torch.cuda.synchronize()
        assert st != orc.OK
        assert c.error_bits() == ERR_OF_STATUS[st]
        assert_same_state(c, oc)
        # sticky: a valid call does nothing while the word is set
        sm.kv_rollback(c, i32([0]), i32([1]))
        torch.cuda.synchronize()
        assert_same_state(c, oc)
        c.clear_error()
    # out-of-range sequence id
    say("error case bad id")
    sm.kv_rollback(c, i32([17]), i32([1]))
    torch.cuda.synchronize()
    assert c.error_bits() == sm.ERR_EINVAL
    c.clear_error()
    assert_same_state(c, oc)


def test_rollback_reappend_restores_gpu_cache(orc):
    rng = np.random.RandomState(11)
    dtype = torch.bfloat16
    oc = orc.OracleCache(bf16=True, num_kv_heads=8, head_dim=128, block_size=16, num_blocks=200,
                         max_seqs=16, max_blocks_per_seq=64,
                         free_order=rng.permutation(200).astype(np.int32))
    c = gpu_cache_like(oc, dtype)
    ids = np.array([3, 9, 0, 12], np.int32)
    lens = np.array([300, 17, 160, 33])
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    K, V = _raw_rows(rng, int(offs[-1]), 8, 128, dtype)
    sm.kv_append(c, i32(ids), i32(offs), K.to(dev()), V.to(dev()))
    torch.cuda.synchronize()
    snap = [t.clone() for t in (c.k_pool, c.v_pool, c.block_table, c.lengths)]
    top = int(c.free_top.item())
    stack = c.free_stack[:top].clone()
    k = np.array([45, 1, 16, 33], np.int32)
    sm.kv_rollback(c, i32(ids), i32(k))
    sel = np.concatenate([np.arange(offs[i + 1] - k[i], offs[i + 1]) for i in range(4)])
    K2, V2 = K[torch.as_tensor(sel)].contiguous(), V[torch.as_tensor(sel)].contiguous()
    sm.kv_append(c, i32(ids), i32(np.concatenate([[0], np.cumsum(k)])), K2.to(dev()), V2.to(dev()))
    torch.cuda.synchronize()
    assert c.error_bits() == 0
    for a, b in zip(snap, (c.k_pool, c.v_pool, c.block_table, c.lengths)):
        assert torch.equal(a, b)
    assert int(c.free_top.item()) == top and torch.equal(stack, c.free_stack[:top])


def test_bulk_prompt_append_llama3_8b_shape(orc):
    """Appending the compacted prompts of the 16 x 4096 workload (about 39k
    rows, 161 MB of K/V) in one call."""
    w = wl.WORKLOADS[2]
    P = wl.make_prompts(w)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    offs = res["packed_offsets"]
    rows = int(offs[-1])
    say("bulk append rows", rows)
    NB = rows // 16 + 16 * 17 + 64
    rng = np.random.RandomState(1)
    oc = orc.OracleCache(bf16=True, num_kv_heads=8, head_dim=128, block_size=16, num_blocks=NB,
                         max_seqs=16, max_blocks_per_seq=4096 // 16 + 32,
                         free_order=rng.permutation(NB).astype(np.int32))
    c = gpu_cache_like(oc, torch.bfloat16)
    K, V = _raw_rows(rng, rows, 8, 128, torch.bfloat16)
    assert oc.append(np.arange(16), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    sm.kv_append(c, i32(np.arange(16)), i32(offs), K.to(dev()), V.to(dev()))
    torch.cuda.synchronize()
    assert c.error_bits() == 0
    assert_same_state(c, oc)
