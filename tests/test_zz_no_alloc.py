"""sm_decode_step_noalloc (the fused decode step whose workspace is the
library's per-device scratch array) against sm_decode_step with a caller
workspace: identical outputs and cache state, bit for bit, on two calls in
a row (the second smaller), checked against the oracle as well; calls too
large for the array are refused before any launch."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_same_state, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _twin_caches(orc, rng, dtype, H, D, bs, lens, MB=None):
    need = sum(-(-L // bs) for L in lens)
    NB = need + 2 * len(lens) + 8
    MB = MB or max(-(-L // bs) for L in lens) + 4
    order = rng.permutation(NB).astype(np.int32)
    oc = orc.OracleCache(bf16=dtype == torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=bs,
                         num_blocks=NB, max_seqs=len(lens), max_blocks_per_seq=MB, free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((int(offs[-1]), H, D), dtype, g)
    V = wl.randn((int(offs[-1]), H, D), dtype, g)
    assert oc.append(np.arange(len(lens)), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    return oc, gpu_cache_like(oc, dtype), gpu_cache_like(oc, dtype)


def _inputs(rng, dtype, n, H, Hq, D):
    g = wl.generator(int(rng.randint(1 << 30)))
    return tuple(wl.randn(s, dtype, g).to(dev()) for s in ((n, H, D), (n, H, D), (n, Hq, D)))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_noalloc_step_equals_workspace_step(orc, dtype):
    Hq, H, D, bs = (32, 8, 128, 16) if dtype == torch.bfloat16 else (8, 4, 64, 16)
    rng = np.random.RandomState(707)
    lens = [2458] * 12 + [0, 1, 15, 16, 17, 1000] if dtype == torch.bfloat16 else [300, 0, 16, 255, 5]
    oc, ca, cb = _twin_caches(orc, rng, dtype, H, D, bs, lens)
    # call 1: every sequence; call 2: a smaller batch, shorter max_len
    calls = [(np.arange(len(lens)), max(lens) + 16), (np.array([4, 0, 2]), max(lens[i] for i in (4, 0, 2)) + 8)]
    for k, (ids, max_len) in enumerate(calls):
        n = len(ids)
        say("no-alloc step", dtype, "call", k, "n", n, "max_len", max_len)
        K, V, q = _inputs(rng, dtype, n, H, Hq, D)
        ws = torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
        out_a = torch.full((n, Hq, D), float("nan"), dtype=dtype, device=dev())
        out_b = torch.full((n, Hq, D), float("nan"), dtype=dtype, device=dev())
        sm.decode_step(ca, i32(ids), K, V, q, out_a, ws, max_len)
        sm.decode_step_noalloc(cb, i32(ids), K, V, q, out_b, max_len)
        torch.cuda.synchronize()
        assert ca.error_bits() == 0 and cb.error_bits() == 0
        assert torch.equal(out_a.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                           out_b.view(torch.int16 if dtype == torch.bfloat16 else torch.int32))
        st_a = oc.append(ids.astype(np.int32), np.arange(n + 1, dtype=np.int32), wl.to_raw(K.cpu()),
                         wl.to_raw(V.cpu()))
        st_d, ref = oc.decode_attention(ids.astype(np.int32), wl.to_f64(q.cpu()), Hq, D ** -0.5)
        assert st_a == orc.OK and st_d == orc.OK
        assert_same_state(ca, oc)
        assert_same_state(cb, oc)
        e = rel_l2_max(out_b.float().cpu().numpy(), ref)
        say("rel_l2_max vs oracle", e)
        assert e <= TOL[dtype]


def test_noalloc_refuses_calls_beyond_the_array(orc):
    # 256 sequences x 64 heads x 2 chunks (of 2048 entries at max_len 4096)
    # x 130 x 4 bytes = 17 MB > 8 MiB: refused on the host, nothing launched,
    # the cache untouched
    rng = np.random.RandomState(9)
    oc, ca, _ = _twin_caches(orc, rng, torch.bfloat16, 8, 128, 16, [16] * 256, MB=4096 // 16 + 1)
    n, Hq = 256, 64
    K, V, q = _inputs(rng, torch.bfloat16, n, 8, Hq, 128)
    out = torch.empty((n, Hq, 128), dtype=torch.bfloat16, device=dev())
    limit = sm.load().sm_decode_step_noalloc_max_bytes()
    assert limit == 8 << 20
    with pytest.raises(sm.SpanMergeError, match="status 1"):
        sm.decode_step_noalloc(ca, i32(np.arange(n)), K, V, q, out, 4096)
    torch.cuda.synchronize()
    assert ca.error_bits() == 0
    assert_same_state(ca, oc)
