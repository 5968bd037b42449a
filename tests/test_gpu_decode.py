"""GPU decode attention vs the oracle (split + combine kernels)."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _setup(orc, rng, dtype, Hq, H, D, bs, lens, NB=None, shuffled=True, extra_seqs=1):
    bf16 = dtype == torch.bfloat16
    need = sum(-(-L // bs) for L in lens)
    NB = NB or need + 8
    MB = max(-(-L // bs) for L in lens) + 4
    order = rng.permutation(NB).astype(np.int32) if shuffled else None
    oc = orc.OracleCache(bf16=bf16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                         max_seqs=len(lens) + extra_seqs, max_blocks_per_seq=MB, free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((int(offs[-1]), H, D), dtype, g)
    V = wl.randn((int(offs[-1]), H, D), dtype, g)
    assert oc.append(np.arange(len(lens)), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    return oc, gpu_cache_like(oc, dtype)


def _run(orc, oc, c, dtype, Hq, seq_ids, max_len, rng, scale=None):
    D = oc.D
    n = len(seq_ids)
    q = wl.randn((n, Hq, D), dtype, wl.generator(int(rng.randint(1 << 30))))
    sc = D ** -0.5 if scale is None else scale
    st, ref = oc.decode_attention(seq_ids, wl.to_f64(q), Hq, sc)
    out = torch.full((n, Hq, D), float("nan"), dtype=dtype, device=dev())
    ws = torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
    sm.decode_attention(c, i32(seq_ids), q.to(dev()), out, ws, max_len, scale=sc)
    torch.cuda.synchronize()
    return st, ref, out.cpu()


CASES = [
    # dtype, Hq, H, D, bs, lens
    (torch.float32, 4, 4, 64, 512, [410]),
    (torch.float32, 4, 4, 64, 512, [0, 1, 33, 409, 1000, 256, 257]),
    (torch.float32, 8, 2, 128, 16, [5, 17, 300]),
    (torch.bfloat16, 32, 8, 128, 16, [1, 15, 16, 17, 31, 32, 33, 127, 128, 129, 1000, 2458]),
    (torch.bfloat16, 28, 4, 128, 16, [512, 700, 4096, 1]),
    (torch.bfloat16, 64, 8, 128, 16, [4915, 40]),
    (torch.bfloat16, 8, 8, 128, 16, [100, 3]),
    (torch.bfloat16, 16, 4, 64, 16, [77, 1024, 0]),
    (torch.bfloat16, 32, 8, 128, 32, [65, 500]),
    (torch.bfloat16, 32, 8, 128, 128, [1000, 129]),
    (torch.bfloat16, 4, 4, 64, 512, [410, 1030]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_decode_matches_oracle(orc, case):
    dtype, Hq, H, D, bs, lens = CASES[case]
    say("decode", case, dtype, Hq, H, D, bs, lens)
    rng = np.random.RandomState(100 + case)
    oc, c = _setup(orc, rng, dtype, Hq, H, D, bs, lens)
    ids = np.arange(len(lens))
    rng.shuffle(ids)
    max_len = max(lens) + int(rng.randint(0, 40))
    st, ref, out = _run(orc, oc, c, dtype, Hq, ids, max_len, rng)
    assert st == orc.OK
    assert c.error_bits() == 0
    err = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", err)
    assert err <= TOL[dtype]


def test_decode_repeated_ids_and_large_scores(orc):
    rng = np.random.RandomState(7)
    dtype = torch.bfloat16
    oc, c = _setup(orc, rng, dtype, 32, 8, 128, 16, [300, 2000])
    say("decode repeated ids, scale 0.5")
    st, ref, out = _run(orc, oc, c, dtype, 32, [1, 0, 1, 1], 2000, rng, scale=0.5)
    assert st == orc.OK and c.error_bits() == 0
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[dtype]


def test_decode_llama3_8b_shape(orc):
    """The benchmark's launch: 16 sequences of ~2458 compacted entries,
    32 query / 8 KV heads, 16-token pages, every row checked."""
    w = wl.WORKLOADS[2]
    rng = np.random.RandomState(2)
    lens = [2458] * 12 + [2714, 2600, 2459, 2457]
    say("decode llama3-8b shape", lens)
    oc, c = _setup(orc, rng, torch.bfloat16, w.num_q_heads, w.num_kv_heads, w.head_dim, 16, lens)
    st, ref, out = _run(orc, oc, c, torch.bfloat16, w.num_q_heads, np.arange(16), 2714, rng)
    assert st == orc.OK and c.error_bits() == 0
    err = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", err)
    assert err <= 1e-2


def test_decode_error_rows_are_zero(orc):
    rng = np.random.RandomState(9)
    dtype = torch.bfloat16
    oc, c = _setup(orc, rng, dtype, 8, 2, 128, 16, [50, 90])
    say("decode length above max_len -> ERANGE")
    st, ref, out = _run(orc, oc, c, dtype, 8, [0, 1], 60, rng)
    assert c.error_bits() == sm.ERR_ERANGE
    assert torch.all(out[1] == 0)
    assert rel_l2_max(out[0].float().numpy(), ref[0]) <= 1e-2
    c.clear_error()
    say("decode bad sequence id -> EINVAL")
    bad = oc.max_seqs + 3
    st, ref, out = _run(orc, oc, c, dtype, 8, [0, bad], 90, rng)
    assert st == orc.EINVAL
    assert c.error_bits() == sm.ERR_EINVAL
    assert torch.all(out[1] == 0)


def _ragged(rng, n, hi):
    """n cached lengths: the page edges 0, 1, 15, 16, 17, 31, 32, 33 and
    hi, the rest uniform in [0, hi]."""
    edges = [0, 1, 15, 16, 17, 31, 32, 33, hi]
    lens = list(rng.randint(0, hi + 1, size=n))
    lens[:len(edges)] = edges[:n]
    rng.shuffle(lens)
    return [int(x) for x in lens]


# More single-chunk (sequence, kv head) pairs than compute units: each
# workgroup takes its pair from the requests sorted by cached length
# (longest first), the first resident rounds dealt in alternating order.
# Cases: a partial second round (280 and 400 pairs), exactly two rounds
# (512), and more pairs than resident workgroups (2048: the rest are
# dispatched as compute units free up).
ORDERED = [
    # Hq, H, D, n, longest length
    (28, 4, 128, 70, 1500),
    (28, 4, 128, 100, 4096),
    (32, 8, 64, 64, 700),
    (32, 8, 64, 256, 400),
]


@pytest.mark.parametrize("case", range(len(ORDERED)))
def test_decode_pairs_dealt_by_length(orc, case):
    Hq, H, D, n, hi = ORDERED[case]
    rng = np.random.RandomState(300 + case)
    lens = _ragged(rng, n, hi)
    say("decode dealt by length: Hq", Hq, "H", H, "D", D, "n", n, "pairs", n * H, "longest", hi)
    oc, c = _setup(orc, rng, torch.bfloat16, Hq, H, D, 16, lens)
    ids = rng.permutation(n)
    st, ref, out = _run(orc, oc, c, torch.bfloat16, Hq, ids, hi + 5, rng)
    assert st == orc.OK and c.error_bits() == 0
    err = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", err)
    assert err <= TOL[torch.bfloat16]
    # requests that attend over nothing get zero rows
    for j, s in enumerate(ids):
        if lens[s] == 0:
            assert torch.all(out[j] == 0)


def test_decode_pairs_dealt_by_length_with_bad_ids(orc):
    """Ids out of range sort last (key -1) and get zero rows and EINVAL; a
    repeated id takes two ranks."""
    rng = np.random.RandomState(41)
    n, H, Hq, D = 90, 4, 28, 128
    lens = _ragged(rng, n, 900)
    oc, c = _setup(orc, rng, torch.bfloat16, Hq, H, D, 16, lens)
    ids = rng.permutation(n).astype(np.int64)
    ids[3] = oc.max_seqs + 7
    ids[50] = -1
    ids[60] = ids[61]
    say("decode dealt by length, bad ids at 3 and 50, repeated id at 60/61")
    st, ref, out = _run(orc, oc, c, torch.bfloat16, Hq, ids, 905, rng)
    assert st == orc.EINVAL
    assert c.error_bits() == sm.ERR_EINVAL
    assert torch.all(out[3] == 0) and torch.all(out[50] == 0)
    good = [j for j in range(n) if j not in (3, 50)]
    assert rel_l2_max(out[good].float().numpy(), ref[good]) <= TOL[torch.bfloat16]
