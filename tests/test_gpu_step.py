"""GPU fused decode step (one appended K/V row per sequence, then attention,
in one launch) vs the oracle's append followed by its attention, and vs the
two separate GPU calls."""
import numpy as np
import pytest
import torch

from gpu_util import ERR_OF_STATUS, TOL, assert_same_state, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _cache(orc, rng, dtype, H, D, bs, lens, NB=None, MB=None, extra_seqs=1, shuffled=True):
    need = sum(-(-L // bs) for L in lens)
    NB = NB or need + len(lens) + 8
    MB = MB or max([-(-L // bs) for L in lens] + [1]) + 4
    order = rng.permutation(NB).astype(np.int32) if shuffled else None
    oc = orc.OracleCache(bf16=dtype == torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=bs,
                         num_blocks=NB, max_seqs=len(lens) + extra_seqs, max_blocks_per_seq=MB,
                         free_order=order)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(int(rng.randint(1 << 30)))
    K = wl.randn((int(offs[-1]), H, D), dtype, g)
    V = wl.randn((int(offs[-1]), H, D), dtype, g)
    assert oc.append(np.arange(len(lens)), offs, wl.to_raw(K), wl.to_raw(V)) == orc.OK
    return oc, gpu_cache_like(oc, dtype)


def _inputs(rng, dtype, n, H, Hq, D):
    g = wl.generator(int(rng.randint(1 << 30)))
    return (wl.randn((n, H, D), dtype, g), wl.randn((n, H, D), dtype, g), wl.randn((n, Hq, D), dtype, g))


def _oracle_step(orc, oc, ids, K, V, q, Hq):
    n = len(ids)
    st_a = oc.append(np.asarray(ids, np.int32), np.arange(n + 1, dtype=np.int32), wl.to_raw(K), wl.to_raw(V))
    st_d, ref = oc.decode_attention(np.asarray(ids, np.int32), wl.to_f64(q), Hq, oc.D ** -0.5)
    return st_a, st_d, ref


def _gpu_step(c, ids, K, V, q, max_len, ws=None):
    n, Hq, D = q.shape
    out = torch.full((n, Hq, D), float("nan"), dtype=q.dtype, device=dev())
    if ws is None:
        ws = torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
    sm.decode_step(c, i32(ids), K.to(dev()), V.to(dev()), q.to(dev()), out, ws, max_len)
    torch.cuda.synchronize()
    return out.cpu(), ws


def _counters_clear(ws):
    assert int(torch.count_nonzero(ws[:256 * 1024]).item()) == 0, "workspace counters not re-armed"


CASES = [
    # dtype, Hq, H, D, bs, lens
    (torch.bfloat16, 32, 8, 128, 16, [0, 1, 15, 16, 17, 31, 32, 33, 127, 128, 1000, 2458]),
    (torch.bfloat16, 32, 8, 128, 16, [2458] * 16),
    (torch.bfloat16, 28, 4, 128, 16, [512, 700, 4096, 1, 4095]),
    (torch.bfloat16, 64, 8, 128, 16, [4915, 40, 4096]),
    (torch.bfloat16, 16, 4, 64, 16, [77, 1024, 0, 16]),
    (torch.bfloat16, 32, 8, 128, 128, [1000, 128, 255]),
    (torch.bfloat16, 4, 4, 64, 512, [410, 1030, 512, 0]),
    (torch.float32, 4, 4, 64, 512, [410, 0, 511, 512]),
    (torch.float32, 8, 2, 128, 16, [5, 16, 300, 0, 255]),
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_step_matches_oracle_append_then_attention(orc, case):
    dtype, Hq, H, D, bs, lens = CASES[case]
    say("decode step", case, dtype, Hq, H, D, bs, lens)
    rng = np.random.RandomState(300 + case)
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = np.arange(len(lens))
    rng.shuffle(ids)
    K, V, q = _inputs(rng, dtype, len(ids), H, Hq, D)
    max_len = max(lens) + 1 + int(rng.randint(0, 40))
    st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
    assert st_a == orc.OK and st_d == orc.OK
    out, ws = _gpu_step(c, ids, K, V, q, max_len)
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    _counters_clear(ws)
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[dtype]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_many_steps_share_one_workspace(orc, dtype):
    """40 steps over short sequences (pages fill and new blocks are popped
    every few steps), one workspace for all of them and for a plain
    attention call in between."""
    Hq, H, D, bs = (32, 8, 128, 16) if dtype == torch.bfloat16 else (8, 4, 64, 16)
    rng = np.random.RandomState(41)
    lens = [14, 15, 16, 31, 0, 2]
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens, NB=64, MB=8)
    ids = np.array([3, 0, 5, 1, 4, 2])
    max_len = 128
    ws = torch.zeros(sm.decode_workspace_bytes(len(ids), Hq, D, max_len), dtype=torch.uint8, device=dev())
    say("decode step x40", dtype)
    for step in range(40):
        K, V, q = _inputs(rng, dtype, len(ids), H, Hq, D)
        st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
        assert st_a == orc.OK and st_d == orc.OK
        out, _ = _gpu_step(c, ids, K, V, q, max_len, ws)
        e = rel_l2_max(out.float().numpy(), ref)
        assert e <= TOL[dtype], (step, e)
        if step % 10 == 9:
            q2 = _inputs(rng, dtype, len(ids), H, Hq, D)[2]
            out2 = torch.empty((len(ids), Hq, D), dtype=dtype, device=dev())
            sm.decode_attention(c, i32(ids), q2.to(dev()), out2, ws, max_len)
            st2, ref2 = oc.decode_attention(ids.astype(np.int32), wl.to_f64(q2), Hq, D ** -0.5)
            torch.cuda.synchronize()
            assert rel_l2_max(out2.float().cpu().numpy(), ref2) <= TOL[dtype]
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    _counters_clear(ws)


def test_step_equals_the_two_calls():
    """Same initial cache: the fused call and kv_append + decode_attention
    leave bit-identical caches and outputs equal up to rounding order."""
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    rng = np.random.RandomState(5)
    lens = [2458, 2459, 2463, 2464, 16, 1, 0, 4000]
    n = len(lens)
    caches = []
    for _ in range(2):
        c = sm.PagedCache(dtype=dtype, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=1200,
                          max_seqs=n, max_blocks_per_seq=300, device=dev(),
                          free_order=torch.as_tensor(np.random.RandomState(9).permutation(1200).astype(np.int32)))
        caches.append(c)
    g = wl.generator(3, "cuda")
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    Kp = wl.randn((int(offs[-1]), H, D), dtype, g, device="cuda")
    Vp = wl.randn((int(offs[-1]), H, D), dtype, g, device="cuda")
    for c in caches:
        sm.kv_append(c, i32(np.arange(n)), i32(offs), Kp, Vp)
    ids = np.array([7, 2, 0, 5, 1, 3, 6, 4])
    K, V, q = _inputs(rng, dtype, n, H, Hq, D)
    max_len = 4001
    say("decode step vs two calls")
    out_f, _ = _gpu_step(caches[0], ids, K, V, q, max_len)
    sm.kv_append(caches[1], i32(ids), i32(np.arange(n + 1)), K.to(dev()), V.to(dev()))
    out_s = torch.empty_like(q, device=dev())
    ws = torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
    sm.decode_attention(caches[1], i32(ids), q.to(dev()), out_s, ws, max_len)
    torch.cuda.synchronize()
    a, b = caches
    for name in ("lengths", "block_table", "free_top", "k_pool", "v_pool"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    top = int(a.free_top.item())
    assert torch.equal(a.free_stack[:top], b.free_stack[:top])
    assert a.error_bits() == 0 and b.error_bits() == 0
    e = rel_l2_max(out_f.float().numpy(), out_s.float().cpu().numpy())
    say("fused vs two calls rel_l2_max", e)
    assert e <= 5e-3


def _snapshot(c):
    torch.cuda.synchronize()
    return {k: getattr(c, k).clone() for k in ("lengths", "block_table", "free_top", "free_stack", "k_pool", "v_pool")}


def _assert_unchanged(c, snap):
    torch.cuda.synchronize()
    for k, v in snap.items():
        assert torch.equal(getattr(c, k), v), k


@pytest.mark.parametrize("kind", ["duplicate", "nomem", "range", "frozen", "bad_id"])
def test_failed_append_leaves_cache_and_attends_over_it(orc, kind):
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    rng = np.random.RandomState(["duplicate", "nomem", "range", "frozen", "bad_id"].index(kind))
    lens = [32, 48, 90, 96]                 # blocks 2 + 3 + 6 + 6
    NB = 17 + 1 if kind == "nomem" else 17 + 8
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens, NB=NB, MB=6 if kind == "range" else 12)
    ids = {"duplicate": [0, 2, 0],
           "nomem": [0, 1, 2],              # two requests need a new block, one is free
           "range": [2, 3],                 # sequence 3 is at its capacity (6 pages)
           "frozen": [0, 1],
           "bad_id": [1, 99, 2]}[kind]
    if kind == "frozen":
        c.err.fill_(sm.ERR_EINVAL)
    expect = {"duplicate": sm.ERR_EINVAL, "nomem": sm.ERR_ENOMEM, "range": sm.ERR_ERANGE,
              "frozen": sm.ERR_EINVAL, "bad_id": sm.ERR_EINVAL}[kind]
    snap = _snapshot(c)
    K, V, q = _inputs(rng, dtype, len(ids), H, Hq, D)
    # the attention the step must give: over the cache as it was
    st_d, ref = oc.decode_attention(np.asarray(ids, np.int32), wl.to_f64(q), Hq, D ** -0.5)
    if kind != "frozen":  # the oracle agrees that the append fails
        st_a = oc.append(np.asarray(ids, np.int32), np.arange(len(ids) + 1, dtype=np.int32),
                         wl.to_raw(K), wl.to_raw(V))
        assert ERR_OF_STATUS[st_a] == expect
    say("decode step failing append", kind, ids)
    out, ws = _gpu_step(c, ids, K, V, q, 96)  # every length stays <= 96 (the append fails)
    _assert_unchanged(c, snap)
    assert c.error_bits() == expect
    _counters_clear(ws)
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e, "attention status", st_d)
    assert e <= TOL[dtype]


def test_length_beyond_max_len_after_append(orc):
    """The append succeeds; the sequence whose new length exceeds max_len
    gets zero rows and ERANGE, the others their attention."""
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    rng = np.random.RandomState(11)
    lens = [100, 64, 30]
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = [0, 1, 2]
    K, V, q = _inputs(rng, dtype, 3, H, Hq, D)
    st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
    assert st_a == orc.OK
    say("decode step with max_len = 100")
    out, ws = _gpu_step(c, ids, K, V, q, 100)
    assert_same_state(c, oc)
    assert c.error_bits() == sm.ERR_ERANGE
    _counters_clear(ws)
    assert float(out[0].float().abs().max()) == 0.0
    assert rel_l2_max(out[1:].float().numpy(), ref[1:]) <= TOL[dtype]


def test_length_at_max_len_and_failed_append(orc):
    """A sequence exactly at max_len: the append fails (a repeated id), so
    its attention over the unchanged cache is still within max_len."""
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    rng = np.random.RandomState(13)
    lens = [100, 64, 30]
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = [0, 1, 1]
    snap = _snapshot(c)
    K, V, q = _inputs(rng, dtype, 3, H, Hq, D)
    st_d, ref = oc.decode_attention(np.asarray(ids, np.int32), wl.to_f64(q), Hq, D ** -0.5)
    say("decode step at max_len with a failing append")
    out, ws = _gpu_step(c, ids, K, V, q, 100)
    _assert_unchanged(c, snap)
    assert c.error_bits() == sm.ERR_EINVAL
    _counters_clear(ws)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[dtype]


def test_full_request_count(orc):
    """256 requests (the most one call takes), lengths around page edges."""
    dtype, Hq, H, D, bs = torch.bfloat16, 8, 2, 64, 16
    rng = np.random.RandomState(12)
    lens = list(rng.randint(0, 70, size=256))
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = rng.permutation(256)
    K, V, q = _inputs(rng, dtype, 256, H, Hq, D)
    st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
    assert st_a == orc.OK
    say("decode step n=256")
    out, ws = _gpu_step(c, ids, K, V, q, 80)
    assert c.error_bits() == 0
    assert_same_state(c, oc)
    _counters_clear(ws)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[dtype]


@pytest.mark.parametrize("n,dup", [(64, None), (65, None), (130, None), (64, (5, 63)), (65, (0, 64)),
                                   (130, (3, 100)), (130, (70, 129))])
def test_request_slots_and_duplicates(orc, n, dup):
    """Request counts at the edges of one 64-request slot per lane (the plan
    takes a single-slot form up to 64 requests), with and without a repeated
    id in the same slot or across slots; lengths straddle page edges so that
    some requests pop a block."""
    dtype, Hq, H, D, bs = torch.bfloat16, 8, 2, 64, 16
    rng = np.random.RandomState(1000 + n + (dup[1] if dup else 0))
    lens = list(rng.randint(0, 70, size=n))
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = rng.permutation(n).astype(np.int32)
    if dup:
        ids[dup[1]] = ids[dup[0]]
    K, V, q = _inputs(rng, dtype, n, H, Hq, D)
    say("decode step n", n, "repeated id at", dup)
    if dup:
        snap = _snapshot(c)
        st_d, ref = oc.decode_attention(ids, wl.to_f64(q), Hq, D ** -0.5)
        st_a = oc.append(ids, np.arange(n + 1, dtype=np.int32), wl.to_raw(K), wl.to_raw(V))
        assert ERR_OF_STATUS[st_a] == sm.ERR_EINVAL
        out, ws = _gpu_step(c, ids, K, V, q, 80)
        _assert_unchanged(c, snap)
        assert c.error_bits() == sm.ERR_EINVAL
    else:
        st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
        assert st_a == orc.OK
        out, ws = _gpu_step(c, ids, K, V, q, 80)
        assert c.error_bits() == 0
        assert_same_state(c, oc)
    _counters_clear(ws)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[dtype]


def test_steps_on_four_streams_match_the_oracle(orc):
    """The benchmark's schedule: the resident batches' fused steps spread
    over four streams (batch r on stream r % 4, one workspace per stream),
    issued without host synchronisation so that launches of different
    streams overlap.  Every step's output and the final cache states match
    the oracle run step by step."""
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    R, NS, n, rounds = 8, 4, 16, 2
    rng = np.random.RandomState(77)
    caches = [_cache(orc, rng, dtype, H, D, bs, list(rng.randint(200, 900, size=n)), MB=64) for _ in range(R)]
    ids = [rng.permutation(n) for _ in range(R)]
    inputs = [[_inputs(rng, dtype, n, H, Hq, D) for _ in range(R)] for _ in range(rounds)]
    max_len = 1000
    streams = [torch.cuda.Stream() for _ in range(NS)]
    wss = [torch.zeros(sm.decode_workspace_bytes(n, Hq, D, max_len), dtype=torch.uint8, device=dev())
           for _ in range(NS)]
    dev_in = [[tuple(x.to(dev()) for x in inputs[s][r]) for r in range(R)] for s in range(rounds)]
    dev_ids = [i32(x) for x in ids]
    outs = [[torch.full((n, Hq, D), float("nan"), dtype=dtype, device=dev()) for _ in range(R)]
            for _ in range(rounds)]
    torch.cuda.synchronize()
    for st in streams:
        st.wait_stream(torch.cuda.current_stream())
    say("decode steps on", NS, "streams", R, "batches", rounds, "rounds")
    for s in range(rounds):
        for r in range(R):
            K, V, q = dev_in[s][r]
            sm.decode_step(caches[r][1], dev_ids[r], K, V, q, outs[s][r], wss[r % NS], max_len,
                           stream=streams[r % NS])
    torch.cuda.synchronize()
    for s in range(rounds):
        for r in range(R):
            K, V, q = inputs[s][r]
            st_a, st_d, ref = _oracle_step(orc, caches[r][0], ids[r], K, V, q, Hq)
            assert st_a == orc.OK and st_d == orc.OK
            e = rel_l2_max(outs[s][r].float().cpu().numpy(), ref)
            assert e <= TOL[dtype], (s, r, e)
    for oc, c in caches:
        assert c.error_bits() == 0
        assert_same_state(c, oc)
    for ws in wss:
        _counters_clear(ws)


def test_commit_wait_give_up_commits_nothing_and_reports_einval(orc):
    """The commit workgroup's bounded wait, forced from the host to give up
    after one poll (every kernel still exits normally: nothing waits on the
    commit workgroup): EINVAL, no metadata change, the logical cache intact.
    After the workspace counters are zeroed again and the error word
    cleared, the next step matches the oracle, which never saw the failed
    call."""
    dtype, Hq, H, D, bs = torch.bfloat16, 32, 8, 128, 16
    rng = np.random.RandomState(77)
    lens = [4000] * 16
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens)
    ids = np.arange(len(lens))
    max_len = max(lens) + 8
    snap = _snapshot(c)
    K, V, q = _inputs(rng, dtype, len(ids), H, Hq, D)
    L = sm.load()
    say("commit wait forced to give up")
    L.sm_set_commit_wait_limit(1)
    try:
        _, ws = _gpu_step(c, ids, K, V, q, max_len)
    finally:
        L.sm_set_commit_wait_limit(0)
    assert c.error_bits() == sm.ERR_EINVAL
    for k in ("lengths", "block_table", "free_top"):
        assert torch.equal(getattr(c, k), snap[k]), k
    top = int(c.free_top.item())
    assert torch.equal(c.free_stack[:top], snap["free_stack"][:top])
    ws.zero_()
    c.clear_error()
    K, V, q = _inputs(rng, dtype, len(ids), H, Hq, D)
    st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
    assert st_a == orc.OK and st_d == orc.OK
    out, _ = _gpu_step(c, ids, K, V, q, max_len, ws)
    assert c.error_bits() == 0
    assert_same_state(c, oc, pools=False)
    e = rel_l2_max(out.float().numpy(), ref)
    say("step after the give-up: rel_l2_max", e)
    assert e <= TOL[dtype]


@pytest.mark.parametrize("n,H,Hq,D,hi", [(100, 4, 28, 128, 3000), (128, 4, 28, 128, 300), (200, 8, 32, 64, 90)])
def test_step_pairs_dealt_by_length(orc, n, H, Hq, D, hi):
    """More single-chunk (sequence, kv head) pairs than compute units: the
    workgroups take the pairs longest first.  Lengths include 0, 1 and the
    page edges, so some requests pop a block; two steps in a row."""
    dtype, bs = torch.bfloat16, 16
    rng = np.random.RandomState(2000 + n)
    edges = [0, 1, 15, 16, 17, 31, 32, 33, hi]
    lens = list(rng.randint(0, hi + 1, size=n))
    lens[:len(edges)] = edges
    rng.shuffle(lens)
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens, MB=-(-(hi + 2) // bs) + 2)
    ids = rng.permutation(n)
    ws = None
    for step in range(2):
        K, V, q = _inputs(rng, dtype, n, H, Hq, D)
        st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
        assert st_a == orc.OK
        say("decode step dealt by length: n", n, "H", H, "pairs", n * H, "step", step)
        out, ws = _gpu_step(c, ids, K, V, q, hi + 2, ws)
        assert c.error_bits() == 0
        assert_same_state(c, oc)
        _counters_clear(ws)
        err = rel_l2_max(out.float().numpy(), ref)
        say("rel_l2_max", err)
        assert err <= TOL[dtype]


@pytest.mark.parametrize("dup", [None, (3, 69)])
def test_many_sequence_slots_duplicate_check(orc, dup):
    """More sequence slots (40,000) than the plan's LDS bitmap covers: the
    duplicate-id check compares ids instead; 70 requests, with and without
    a repeated id."""
    dtype, Hq, H, D, bs = torch.bfloat16, 8, 2, 64, 16
    rng = np.random.RandomState(4000 + (dup[1] if dup else 0))
    n = 70
    lens = list(rng.randint(0, 70, size=n))
    oc, c = _cache(orc, rng, dtype, H, D, bs, lens, extra_seqs=40000 - n)
    ids = rng.permutation(n).astype(np.int32)
    ids[5] = 39999 - 7   # a high slot (empty sequence)
    if dup:
        ids[dup[1]] = ids[dup[0]]
    K, V, q = _inputs(rng, dtype, n, H, Hq, D)
    say("decode step, 40000 slots, repeated id", dup)
    if dup:
        snap = _snapshot(c)
        st_d, ref = oc.decode_attention(ids, wl.to_f64(q), Hq, D ** -0.5)
        out, ws = _gpu_step(c, ids, K, V, q, 80)
        _assert_unchanged(c, snap)
        assert c.error_bits() == sm.ERR_EINVAL
    else:
        st_a, st_d, ref = _oracle_step(orc, oc, ids, K, V, q, Hq)
        assert st_a == orc.OK
        out, ws = _gpu_step(c, ids, K, V, q, 80)
        assert c.error_bits() == 0
        assert_same_state(c, oc)
    _counters_clear(ws)
    assert rel_l2_max(out.float().numpy(), ref) <= TOL[dtype]
