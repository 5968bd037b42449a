"""GPU decode-time merge step (crop k entries per request, append its row,
attend; one launch, one all-or-nothing update) vs the oracle's crop_append
(rollback then append, restored if either fails) followed by its attention.
Cache state is compared bit for bit, attention within the bf16 bar."""
import numpy as np
import pytest
import torch

from gpu_util import ERR_OF_STATUS, TOL, assert_same_state, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _cache(orc, rng, H, D, bs, lens, NB=None, MB=None, extra_seqs=1):
    need = sum(-(-L // bs) for L in lens)
    NB = NB or need + len(lens) + 8
    MB = MB or max([-(-L // bs) for L in lens] + [1]) + 4
    oc = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                         max_seqs=len(lens) + extra_seqs, max_blocks_per_seq=MB,
                         free_order=rng.permutation(NB).astype(np.int32))
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    V = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    assert oc.append(np.arange(len(lens)), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    return oc, gpu_cache_like(oc, torch.bfloat16)


def _inputs(rng, n, H, Hq, D):
    g = wl.generator(int(rng.randint(1 << 30)))
    return tuple(wl.randn(shape, torch.bfloat16, g) for shape in ((n, H, D), (n, H, D), (n, Hq, D)))


def _oracle(oc, ids, k, K, V, q, Hq):
    st_a = oc.crop_append(np.asarray(ids, np.int32), np.asarray(k, np.int32), wl.to_raw(K), wl.to_raw(V))
    st_d, ref = oc.decode_attention(np.asarray(ids, np.int32), wl.to_f64(q), Hq, oc.D ** -0.5)
    return st_a, ref


def _gpu(c, ids, k, K, V, q, max_len, ws=None):
    n, Hq, D = q.shape
    out = torch.full((n, Hq, D), float("nan"), dtype=q.dtype, device=dev())
    if ws is None:
        ws = torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
    sm.decode_merge_step(c, i32(ids), i32(k), K.to(dev()), V.to(dev()), q.to(dev()), out, ws, max_len)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(ws[:256 * 1024]).item()) == 0, "workspace counters not re-armed"
    return out.cpu(), ws


def _crops(rng, lens, hi=7):
    """Span crops n - 1 (1..7), some 0, some the whole cache."""
    k = [int(rng.randint(0, min(L, hi) + 1)) for L in lens]
    for j in rng.choice(len(lens), size=max(1, len(lens) // 8), replace=False):
        k[j] = int(lens[j])
    return k


CASES = [
    # Hq, H, D, bs, lens
    (32, 8, 128, 16, [0, 1, 15, 16, 17, 31, 32, 33, 127, 128, 1000, 2458]),
    (32, 8, 128, 16, [2458] * 16),
    (28, 4, 128, 16, [512, 700, 4096, 1, 4095, 18, 20]),
    (16, 4, 64, 16, [77, 1024, 0, 16, 48, 49]),
    (32, 8, 128, 32, [1000, 128, 255, 33, 64]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_merge_step_matches_oracle(orc, case):
    Hq, H, D, bs, lens = CASES[case]
    rng = np.random.RandomState(500 + case)
    oc, c = _cache(orc, rng, H, D, bs, lens)
    n = len(lens)
    ids = rng.permutation(n)
    ws = None
    for step in range(3):   # three merge steps in a row on one workspace
        cur = [int(oc.lengths[s]) for s in ids]
        k = _crops(rng, cur)
        K, V, q = _inputs(rng, n, H, Hq, D)
        st_a, ref = _oracle(oc, ids, k, K, V, q, Hq)
        assert st_a == orc.OK
        say("merge step case", case, "step", step, "crops", k[:12])
        out, ws = _gpu(c, ids, k, K, V, q, max(cur) + 1, ws)
        assert c.error_bits() == 0
        assert_same_state(c, oc)
        err = rel_l2_max(out.float().numpy(), ref)
        say("rel_l2_max", err)
        assert err <= TOL[torch.bfloat16]


def test_merge_step_freed_pages_are_popped_by_other_requests(orc):
    """Crops that free pages while other requests end pages: the append's
    pops take the freed pages (request 0's first, ascending), then the old
    stack; the stack has nothing else free."""
    Hq, H, D, bs = 8, 2, 64, 16
    rng = np.random.RandomState(9)
    lens = [40, 33, 64, 32, 48, 17, 80]
    NB = sum(-(-L // bs) for L in lens) + 1      # one block free beforehand
    oc, c = _cache(orc, rng, H, D, bs, lens, NB=NB)
    ids = np.arange(len(lens))
    k = [9, 1, 0, 0, 16, 1, 17]                  # frees pages of 0, 1, 4, 5, 6; 2, 3, 4, 5 end a page
    K, V, q = _inputs(rng, len(ids), H, Hq, D)
    st_a, ref = _oracle(oc, ids, k, K, V, q, Hq)
    assert st_a == orc.OK
    out, _ = _gpu(c, ids, k, K, V, q, max(lens))
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[torch.bfloat16]


def test_merge_step_all_zero_crops_equals_decode_step(orc):
    Hq, H, D, bs = 32, 8, 128, 16
    rng = np.random.RandomState(10)
    lens = [100, 2458, 15, 16, 0]
    oc, c = _cache(orc, rng, H, D, bs, lens)
    oc2, c2 = _cache(orc, np.random.RandomState(10), H, D, bs, lens)
    ids = np.arange(len(lens))
    K, V, q = _inputs(rng, len(ids), H, Hq, D)
    out, _ = _gpu(c, ids, [0] * len(ids), K, V, q, 2459)
    out2 = torch.empty_like(out, device=dev())
    ws2 = torch.zeros(sm.decode_workspace_bytes(len(ids), Hq, D, 2459), dtype=torch.uint8, device=dev())
    sm.decode_step(c2, i32(ids), K.to(dev()), V.to(dev()), q.to(dev()), out2, ws2, 2459)
    torch.cuda.synchronize()
    assert c.error_bits() == 0 and c2.error_bits() == 0
    for name in ("lengths", "block_table", "free_top", "k_pool", "v_pool"):
        assert torch.equal(getattr(c, name), getattr(c2, name)), name
    assert torch.equal(out, out2.cpu())


@pytest.mark.parametrize("n,H,Hq,D,hi", [(100, 4, 28, 128, 1500), (256, 2, 8, 64, 70), (200, 8, 32, 64, 90)])
def test_merge_step_many_requests(orc, n, H, Hq, D, hi):
    """Request counts past one 64-request slot per lane, and past the
    compute unit count in (sequence, head) pairs (dealt by length)."""
    bs = 16
    rng = np.random.RandomState(3000 + n)
    lens = list(rng.randint(0, hi + 1, size=n))
    lens[:6] = [0, 1, 16, 17, 32, hi]
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = rng.permutation(n)
    cur = [int(oc.lengths[s]) for s in ids]
    k = _crops(rng, cur)
    K, V, q = _inputs(rng, n, H, Hq, D)
    st_a, ref = _oracle(oc, ids, k, K, V, q, Hq)
    assert st_a == orc.OK
    say("merge step n", n, "pairs", n * H)
    out, _ = _gpu(c, ids, k, K, V, q, hi + 1)
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[torch.bfloat16]


def _snapshot(c):
    torch.cuda.synchronize()
    return {k: getattr(c, k).clone() for k in ("lengths", "block_table", "free_top", "free_stack", "k_pool", "v_pool")}


@pytest.mark.parametrize("kind", ["crop_too_long", "negative", "duplicate", "nomem_after_crop", "frozen",
                                  "range_no_crop"])
def test_failed_merge_step_changes_nothing(orc, kind):
    Hq, H, D, bs = 8, 2, 64, 16
    rng = np.random.RandomState(40 + len(kind))
    lens = [32, 48, 90, 96]                  # blocks 2 + 3 + 6 + 6 = 17
    NB = 17 if kind == "nomem_after_crop" else 17 + 8
    oc, c = _cache(orc, rng, H, D, bs, lens, NB=NB, MB=6 if kind == "range_no_crop" else 12)
    ids, k = {"crop_too_long": ([0, 1], [1, 49]),
              "negative": ([0, 1], [-1, 0]),
              "duplicate": ([0, 2, 0], [1, 1, 1]),
              "nomem_after_crop": ([0, 1, 2], [1, 0, 0]),   # 0 and 1 end pages after their crops, none free
              "frozen": ([0, 1], [2, 2]),
              "range_no_crop": ([2, 3], [0, 0])}[kind]       # sequence 3 is at capacity
    if kind == "frozen":
        c.err.fill_(sm.ERR_EINVAL)
    expect = {"crop_too_long": sm.ERR_ERANGE, "negative": sm.ERR_EINVAL, "duplicate": sm.ERR_EINVAL,
              "nomem_after_crop": sm.ERR_ENOMEM, "frozen": sm.ERR_EINVAL, "range_no_crop": sm.ERR_ERANGE}[kind]
    snap = _snapshot(c)
    K, V, q = _inputs(rng, len(ids), H, Hq, D)
    st_d, ref = oc.decode_attention(np.asarray(ids, np.int32), wl.to_f64(q), Hq, D ** -0.5)
    if kind != "frozen":
        st_a = oc.crop_append(np.asarray(ids, np.int32), np.asarray(k, np.int32), wl.to_raw(K), wl.to_raw(V))
        assert ERR_OF_STATUS[st_a] == expect
    say("merge step failing", kind, ids, k)
    out, _ = _gpu(c, ids, k, K, V, q, 96)
    for name, v in snap.items():
        assert torch.equal(getattr(c, name), v), name
    assert c.error_bits() == expect
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[torch.bfloat16]


def test_match_decode_crops_feed_the_merge_step(orc):
    """A rule match decides the crops: sm_match_decode without a cache
    writes k = n - 1 for every request whose new token completes a rule
    span, and the merge step applies them."""
    Hq, H, D, bs = 8, 2, 64, 16
    rng = np.random.RandomState(11)
    rules = np.array([[5, 6, 7, -1], [8, 9, -1, -1]], np.int32)
    table = sm.RuleTable(sm.RuleTable.capacity_for(len(rules)), device=dev())
    sm.rules_build(table, i32(rules))
    R = orc.OracleRules(rules)
    lens = [40, 33, 17]
    oc, c = _cache(orc, rng, H, D, bs, lens)
    ids = np.arange(3)
    state = torch.zeros((4, 4), dtype=torch.int32, device=dev())
    k_out = torch.empty(3, dtype=torch.int32, device=dev())
    r_out = torch.empty(3, dtype=torch.int32, device=dev())
    stream_tokens = [[5, 8, 1], [6, 9, 2], [7, 3, 3]]   # request 0 completes (5, 6, 7), request 1 (8, 9)
    for toks in stream_tokens:
        sm.match_decode(table, state, i32(ids), i32(toks), k_out, r_out, cache=None)
        want = [R.decode_step(int(s), int(y))[0] for s, y in zip(ids, toks)]
    torch.cuda.synchronize()
    k = k_out.cpu().numpy()
    assert k.tolist() == want == [2, 0, 0]
    K, V, q = _inputs(rng, 3, H, Hq, D)
    st_a, ref = _oracle(oc, ids, k, K, V, q, Hq)
    assert st_a == orc.OK
    out, _ = _gpu(c, ids, k, K, V, q, max(lens))
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[torch.bfloat16]
