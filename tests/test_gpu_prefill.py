"""GPU prefill attention (causal, grouped query, over the paged cache) vs the
oracle's prefill attention on the same cache and queries."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _cache(orc, rng, H, D, bs, lens, extra_seqs=1):
    need = sum(-(-L // bs) for L in lens)
    NB = need + len(lens) + 8
    MB = max([-(-L // bs) for L in lens] + [1]) + 2
    order = rng.permutation(NB).astype(np.int32)
    oc = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                         max_seqs=len(lens) + extra_seqs, max_blocks_per_seq=MB, free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    V = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    assert oc.append(np.arange(len(lens)), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    return oc, gpu_cache_like(oc, torch.bfloat16)


def _gpu_prefill(c, ids, qo, q, max_rows):
    out = torch.full(q.shape, float("nan"), dtype=torch.bfloat16, device=dev())
    sm.prefill_attention(c, i32(ids), i32(qo), q.to(dev()), out, max_rows)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


CASES = [
    # Hq, H, D, bs, lens, rows per request (None = the whole sequence)
    (8, 2, 128, 16, [1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 100, 255], None),
    (32, 8, 128, 16, [300, 77], None),
    (32, 8, 128, 16, [300, 77, 129], [1, 77, 40]),            # chunked: rows after earlier context
    (8, 8, 128, 16, [200, 33], None),                           # group of 1: 256 positions per workgroup
    (28, 4, 128, 16, [190, 64], None),                          # group of 7: 36 positions, 4 vectors idle
    (16, 1, 64, 16, [150, 20, 0], [150, 3, 0]),                 # group of 16, head_dim 64, an empty request
    (8, 4, 64, 128, [400, 129], [400, 100]),
    (4, 2, 128, 512, [700], [513]),
    (8, 2, 128, 32, [130, 64, 1], None),                        # two pages per 64-key tile
    (8, 2, 128, 64, [200, 65], [200, 1]),                       # one page per tile
    (12, 3, 64, 256, [300, 257], [300, 129]),                   # pages longer than a tile, D 64
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_prefill_matches_oracle(orc, case):
    Hq, H, D, bs, lens, ms = CASES[case]
    rng = np.random.RandomState(100 + case)
    ms = list(lens) if ms is None else ms
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.arange(len(lens), dtype=np.int32)
    qo = np.concatenate([[0], np.cumsum(ms)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    q = wl.randn((int(qo[-1]), Hq, D), torch.bfloat16, g)
    st, ref = oc.prefill_attention(ids, qo, wl.to_f64(q), Hq, D ** -0.5)
    assert st == orc.OK
    say("prefill", Hq, H, D, bs, lens, ms)
    out = _gpu_prefill(c, ids, qo, q, max(ms))
    assert c.error_bits() == 0
    e = rel_l2_max(out, ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


@pytest.mark.parametrize("scale", [-0.09, 0.0, 0.4])
def test_prefill_scale_values(orc, scale):
    """Negative, zero (the plain mean of the visible V rows) and large scales."""
    Hq, H, D, bs = 8, 2, 128, 16
    rng = np.random.RandomState(31)
    lens = [150, 70]
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.arange(len(lens), dtype=np.int32)
    qo = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(32)
    q = wl.randn((int(qo[-1]), Hq, D), torch.bfloat16, g)
    st, ref = oc.prefill_attention(ids, qo, wl.to_f64(q), Hq, scale)
    assert st == orc.OK
    say("prefill scale", scale)
    out = torch.full(q.shape, float("nan"), dtype=torch.bfloat16, device=dev())
    sm.prefill_attention(c, i32(ids), i32(qo), q.to(dev()), out, max(lens), scale=scale)
    torch.cuda.synchronize()
    assert c.error_bits() == 0
    e = rel_l2_max(out.float().cpu().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


def test_bad_requests_zero_their_rows_only(orc):
    """m > length and an out-of-range id give EINVAL and zero rows; the
    good request next to them is unaffected."""
    Hq, H, D, bs = 8, 2, 128, 16
    rng = np.random.RandomState(7)
    lens = [50, 90, 70]
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.array([0, 1, 99], dtype=np.int32)
    ms = [51, 90, 10]                      # request 0 asks for more rows than cached
    qo = np.concatenate([[0], np.cumsum(ms)]).astype(np.int32)
    g = wl.generator(8)
    q = wl.randn((int(qo[-1]), Hq, D), torch.bfloat16, g)
    say("prefill with bad requests")
    out = _gpu_prefill(c, ids, qo, q, 90)
    assert c.error_bits() == sm.ERR_EINVAL
    assert np.all(out[qo[0]:qo[1]] == 0) and np.all(out[qo[2]:qo[3]] == 0)
    st, ref = oc.prefill_attention([1], [0, 90], wl.to_f64(q[qo[1]:qo[2]]), Hq, D ** -0.5)
    assert st == orc.OK
    assert rel_l2_max(out[qo[1]:qo[2]], ref) <= TOL[torch.bfloat16]


def test_llama3_8b_prompt_batch_sampled(orc):
    """The compressed Llama-3-8B-shaped prompt batch (16 x 2458 positions, 32/8 heads,
    head_dim 128) at full size, launched as the bench launches it.  Checked
    on the last 12 rows of every request and on the first 40 rows of two
    requests (the oracle runs those as requests of their own over the same
    pages)."""
    w = wl.WORKLOADS[2]
    Hq, H, D, bs = w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size
    L0 = w.prompt_len - int(round(w.target * w.prompt_len))
    rng = np.random.RandomState(9)
    lens = [L0] * w.batch
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.arange(w.batch, dtype=np.int32)
    qo = np.arange(w.batch + 1, dtype=np.int32) * L0
    g = wl.generator(10)
    q = wl.randn((int(qo[-1]), Hq, D), torch.bfloat16, g)
    say("prefill 8B-shaped batch", w.batch, "x", L0)
    out = _gpu_prefill(c, ids, qo, q, L0)
    assert c.error_bits() == 0
    k = 12
    rows = np.concatenate([np.arange(qo[i + 1] - k, qo[i + 1]) for i in range(w.batch)])
    st, ref = oc.prefill_attention(ids, np.arange(w.batch + 1, dtype=np.int32) * k, wl.to_f64(q[rows]), Hq,
                                   D ** -0.5)
    assert st == orc.OK
    e_tail = rel_l2_max(out[rows], ref)
    # first 40 positions of requests 0 and 5: a shorter copy of their sequences
    head = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=oc.num_blocks,
                           max_seqs=oc.max_seqs, max_blocks_per_seq=oc.max_blocks)
    head.k_pool[:], head.v_pool[:], head.block_table[:] = oc.k_pool, oc.v_pool, oc.block_table
    head.lengths[:] = 0
    head.lengths[[0, 5]] = 40
    first = np.concatenate([np.arange(qo[0], qo[0] + 40), np.arange(qo[5], qo[5] + 40)])
    st, ref2 = head.prefill_attention([0, 5], [0, 40, 80], wl.to_f64(q[first]), Hq, D ** -0.5)
    assert st == orc.OK
    e_head = rel_l2_max(out[first], ref2)
    say("rel_l2_max last rows", e_tail, "first rows", e_head)
    assert e_tail <= TOL[torch.bfloat16] and e_head <= TOL[torch.bfloat16]


@pytest.mark.parametrize("wid", [3, 5])
def test_prompt_batch_full_size_sampled(orc, wid):
    """The compressed prompt batches of the long-context batch (4 x 19661
    positions over shuffled pages) and of the 70B-shaped batch (32 x 4915
    positions, 64 query heads, group 8) at full size; checked on the last 4
    rows of every request and the first 24 rows of one."""
    w = wl.WORKLOADS[wid]
    Hq, H, D, bs = w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size
    L0 = w.prompt_len - int(round(w.target * w.prompt_len))
    rng = np.random.RandomState(40 + wid)
    lens = [L0] * w.batch
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.arange(w.batch, dtype=np.int32)
    qo = np.arange(w.batch + 1, dtype=np.int32) * L0
    gq = wl.generator(50 + wid, "cuda")
    q = wl.randn((int(qo[-1]), Hq, D), torch.bfloat16, gq, device="cuda")
    out = torch.full(q.shape, float("nan"), dtype=torch.bfloat16, device=dev())
    say("prefill", w.name, w.batch, "x", L0)
    sm.prefill_attention(c, i32(ids), i32(qo), q, out, L0)
    torch.cuda.synchronize()
    assert c.error_bits() == 0
    k = 4
    rows = np.concatenate([np.arange(qo[i + 1] - k, qo[i + 1]) for i in range(w.batch)])
    rows_t = torch.as_tensor(rows, device=dev())
    st, ref = oc.prefill_attention(ids, np.arange(w.batch + 1, dtype=np.int32) * k,
                                   wl.to_f64(q[rows_t].cpu()), Hq, D ** -0.5)
    assert st == orc.OK
    e_tail = rel_l2_max(out[rows_t].float().cpu().numpy(), ref)
    head = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=oc.num_blocks,
                           max_seqs=oc.max_seqs, max_blocks_per_seq=oc.max_blocks)
    head.k_pool[:], head.v_pool[:], head.block_table[:] = oc.k_pool, oc.v_pool, oc.block_table
    head.lengths[:] = 0
    head.lengths[1] = 24
    first = torch.arange(int(qo[1]), int(qo[1]) + 24, device=dev())
    st, ref2 = head.prefill_attention([1], [0, 24], wl.to_f64(q[first].cpu()), Hq, D ** -0.5)
    assert st == orc.OK
    e_head = rel_l2_max(out[first].float().cpu().numpy(), ref2)
    say("rel_l2_max last rows", e_tail, "first rows", e_head)
    assert e_tail <= TOL[torch.bfloat16] and e_head <= TOL[torch.bfloat16]
