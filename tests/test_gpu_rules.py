"""GPU rule table and matching vs the oracle's rule set and matching, bit
for bit (integer outputs)."""
import numpy as np
import pytest
import torch

from gpu_util import dev, i32, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _small_rules(rng, count, V):
    out = np.full((count, 4), -1, np.int32)
    for i in range(count):
        n = rng.randint(2, 5)
        out[i, :n] = rng.randint(0, V, n)
    return out


def _table(rules):
    t = sm.RuleTable(sm.RuleTable.capacity_for(len(rules)), device=dev())
    sm.rules_build(t, i32(rules))
    return t


def _gpu_match(t, toks, offs):
    T, B = len(toks), len(offs) - 1
    cap = max(T // 2, 1)
    outs = [torch.full((cap,), -7, dtype=torch.int32, device=dev()) for _ in range(3)]
    sso = torch.full((B + 1,), -7, dtype=torch.int32, device=dev())
    ws = torch.empty(sm.match_prompt_workspace_bytes(B, T), dtype=torch.uint8, device=dev())
    sm.match_prompt(t, i32(toks), i32(offs), *outs, sso, ws)
    torch.cuda.synchronize()
    sso = sso.cpu().numpy()
    S = int(sso[-1])
    return [o[:S].cpu().numpy() for o in outs] + [sso]


@pytest.mark.parametrize("seed", range(3))
def test_lookup_matches_oracle(orc, seed):
    rng = np.random.RandomState(seed)
    rules = _small_rules(rng, 3000 + 1000 * seed, 40)       # many duplicates at this vocabulary
    R = orc.OracleRules(rules)
    t = _table(rules)
    grams = _small_rules(rng, 20000, 40)
    ids = torch.empty(len(grams), dtype=torch.int32, device=dev())
    sm.rules_lookup(t, i32(grams), ids)
    torch.cuda.synchronize()
    say("rules", len(rules), "distinct", R.count)
    assert t.error_bits() == 0
    want = np.array([R.find(g[g >= 0]) for g in grams], np.int32)
    assert np.array_equal(ids.cpu().numpy(), want)
    # every rule finds itself, with the first index among duplicates
    ids2 = torch.empty(len(rules), dtype=torch.int32, device=dev())
    sm.rules_lookup(t, i32(rules), ids2)
    want2 = np.array([R.find(g[g >= 0]) for g in rules], np.int32)
    assert np.array_equal(ids2.cpu().numpy(), want2)
    # the table holds exactly the distinct rules
    assert int((t.keys[:, 0] >= 0).sum().item()) == R.count


def test_malformed_rule_sets_einval():
    rules = np.array([[1, 2, -1, -1], [3, -1, 4, -1], [5, 6, 7, 8]], np.int32)
    t = _table(rules)
    assert t.error_bits() == sm.ERR_EINVAL
    ids = torch.empty(2, dtype=torch.int32, device=dev())
    sm.rules_lookup(t, i32(np.array([[1, 2, -1, -1], [5, 6, 7, 8]], np.int32)), ids)
    assert ids.cpu().tolist() == [0, 2]                     # the well-formed rules are in


CASES = [
    # vocabulary, rules, sequence lengths
    (8, 60, [0, 1, 2, 5, 33, 100]),
    (6, 40, [4095, 4096, 4097]),                           # one segment of 4096, ragged tails
    (10, 200, [9000, 1, 12289]),                           # several segments
    (4, 12, [3000]),                                       # dense: matches almost everywhere
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_match_prompt_matches_oracle(orc, case):
    V, nr, lens = CASES[case]
    rng = np.random.RandomState(20 + case)
    rules = _small_rules(rng, nr, V)
    R = orc.OracleRules(rules)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    toks = rng.randint(0, V, int(offs[-1])).astype(np.int32)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK
    t = _table(rules)
    say("match_prompt", V, nr, lens, "spans", len(s0))
    g0, gl, gr, gs = _gpu_match(t, toks, offs)
    assert t.error_bits() == 0
    assert np.array_equal(gs, sso)
    assert np.array_equal(g0, s0) and np.array_equal(gl, ln) and np.array_equal(gr, ru)


def test_match_prompt_negative_ids_and_bad_offsets(orc):
    rules = np.array([[1, 2, -1, -1], [3, 4, -1, -1]], np.int32)
    t = _table(rules)
    toks = np.array([5, 1, 2, 3, -1, 4, 3, 4], np.int32)
    g0, gl, gr, gs = _gpu_match(t, toks, np.array([0, 2, 5, 8], np.int32))
    assert g0.tolist() == [6] and gl.tolist() == [2] and gs.tolist() == [0, 0, 0, 1]
    assert t.error_bits() == 0
    g0, gl, gr, gs = _gpu_match(t, toks, np.array([0, 5, 3, 8], np.int32))   # out of order
    assert t.error_bits() == sm.ERR_EINVAL
    assert gs.tolist()[1] == gs.tolist()[2]                  # sequence 1 (5 > 3) got no spans


def test_match_prompt_llama3_8b_batch(orc):
    """The Llama-3-8B-shaped prompt batch (16 x 4096) with 2.17M synthetic rules of the
    Llama-3 rule counts, rules planted for a 40% reduction."""
    rules = wl.make_rules()
    toks, offs = wl.make_rule_prompts(rules, 16, 4096, 0.4, 128256, seed=3)
    R = orc.OracleRules(rules)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK
    t = _table(rules)
    say("8B-shaped batch: spans", len(s0), "reduction", float((ln - 1).sum()) / len(toks))
    g0, gl, gr, gs = _gpu_match(t, toks, offs)
    assert t.error_bits() == 0
    assert np.array_equal(gs, sso)
    assert np.array_equal(g0, s0) and np.array_equal(gl, ln) and np.array_equal(gr, ru)
    assert abs(float((ln - 1).sum()) / len(toks) - 0.4) < 0.01


@pytest.mark.parametrize("seed", range(3))
def test_match_decode_matches_oracle(orc, seed):
    rng = np.random.RandomState(70 + seed)
    V, B, steps, max_seqs = 5, 24, 60, 40
    rules = _small_rules(rng, 30, V)
    R = orc.OracleRules(rules)
    t = _table(rules)
    state = torch.zeros((max_seqs, 4), dtype=torch.int32, device=dev())
    seqs = rng.permutation(max_seqs)[:B].astype(np.int32)
    k_out = torch.empty(B, dtype=torch.int32, device=dev())
    r_out = torch.empty(B, dtype=torch.int32, device=dev())
    say("match_decode", B, steps)
    for step in range(steps):
        order = rng.permutation(B)                           # request order changes per step
        ids = seqs[order]
        toks = rng.randint(0, V, B).astype(np.int32)
        sm.match_decode(t, state, i32(ids), i32(toks), k_out, r_out)
        got_k, got_r = k_out.cpu().numpy(), r_out.cpu().numpy()
        want = [R.decode_step(int(s), int(y)) for s, y in zip(ids, toks)]
        assert got_k.tolist() == [w[0] for w in want], step
        assert got_r.tolist() == [w[1] for w in want], step
    assert t.error_bits() == 0


def test_match_decode_fused_rollback(orc):
    """The crop the merges imply, run by the same call: lengths, block tables
    and free stack equal the oracle's rollback with the oracle's k."""
    rng = np.random.RandomState(5)
    V, B, H, D, bs = 4, 8, 2, 64, 16
    rules = _small_rules(rng, 10, V)
    R = orc.OracleRules(rules)
    t = _table(rules)
    lens = rng.randint(20, 60, B)
    NB = int(sum(-(-L // bs) for L in lens)) + 8
    oc = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB, max_seqs=B,
                         max_blocks_per_seq=8)
    c = sm.PagedCache(dtype=torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB,
                      max_seqs=B, max_blocks_per_seq=8, device=dev())
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    g = wl.generator(6)
    K = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    Vv = wl.randn((int(offs[-1]), H, D), torch.bfloat16, g)
    ids = np.arange(B, dtype=np.int32)
    assert oc.append(ids, offs, wl.to_raw(K), wl.to_raw(Vv)) == orc.OK
    sm.kv_append(c, i32(ids), i32(offs), K.to(dev()), Vv.to(dev()))
    state = torch.zeros((B, 4), dtype=torch.int32, device=dev())
    k_out = torch.empty(B, dtype=torch.int32, device=dev())
    r_out = torch.empty(B, dtype=torch.int32, device=dev())
    merged = 0
    for step in range(12):
        toks = rng.randint(0, V, B).astype(np.int32)
        sm.match_decode(t, state, i32(ids), i32(toks), k_out, r_out, cache=c)
        want_k = np.array([R.decode_step(int(s), int(y))[0] for s, y in zip(ids, toks)], np.int32)
        assert k_out.cpu().numpy().tolist() == want_k.tolist()
        assert oc.rollback(ids, want_k) == orc.OK
        merged += int(want_k.sum())
    torch.cuda.synchronize()
    say("fused rollback: entries cropped", merged)
    assert merged > 0 and c.error_bits() == 0
    assert np.array_equal(c.lengths.cpu().numpy(), oc.lengths)
    assert np.array_equal(c.block_table.cpu().numpy(), oc.block_table)
    top = int(c.free_top.item())
    assert top == int(oc.free_top[0])
    assert np.array_equal(c.free_stack.cpu().numpy()[:top], oc.free_stack[:top])


def test_match_decode_repeated_id_changes_nothing(orc):
    rules = np.array([[1, 2, -1, -1]], np.int32)
    t = _table(rules)
    state = torch.zeros((4, 4), dtype=torch.int32, device=dev())
    k_out = torch.full((2,), 9, dtype=torch.int32, device=dev())
    r_out = torch.full((2,), 9, dtype=torch.int32, device=dev())
    sm.match_decode(t, state, i32([1, 2]), i32([1, 1]), k_out, r_out)
    before = state.clone()
    sm.match_decode(t, state, i32([1, 1]), i32([2, 2]), k_out, r_out)
    torch.cuda.synchronize()
    assert t.error_bits() == sm.ERR_EINVAL
    assert torch.equal(state, before) and k_out.cpu().tolist() == [0, 0] and r_out.cpu().tolist() == [-1, -1]


@pytest.mark.parametrize("B,T", [(4, 32768), (32, 8192)])
def test_match_prompt_long_and_wide_batches(orc, B, T):
    """The prompt shapes of the long-context (4 x 32768: eight scan passes
    per sequence) and 70B-shaped (32 x 8192) batches, 2.17M rules."""
    rules = wl.make_rules()
    toks, offs = wl.make_rule_prompts(rules, B, T, 0.4, 128256, seed=B)
    R = orc.OracleRules(rules)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK
    t = _table(rules)
    say("match_prompt", B, "x", T, "spans", len(s0))
    g0, gl, gr, gs = _gpu_match(t, toks, offs)
    assert t.error_bits() == 0
    assert np.array_equal(gs, sso)
    assert np.array_equal(g0, s0) and np.array_equal(gl, ln) and np.array_equal(gr, ru)
