"""GPU surrogate lookup and span dedupe vs the oracle: the gather and the
dedupe bit for bit, and the two prompt paths they enable (surrogates from a
per-rule table, merge of distinct spans only) against the oracle's merge of
every span in context."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, dev, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,d", [(torch.bfloat16, 4096), (torch.float32, 256), (torch.bfloat16, 72)])
def test_gather_matches_oracle(orc, dtype, d):
    rng = np.random.RandomState(d)
    g = wl.generator(d)
    emb = wl.randn((300, d), dtype, g)
    lut = wl.randn((50, d), dtype, g)
    n = 777
    rule = np.where(rng.rand(n) < 0.5, rng.randint(0, 50, n), -1).astype(np.int32)
    tok = rng.randint(0, 300, n).astype(np.int32)
    out = torch.full((n, d), float("nan"), dtype=dtype, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    say("gather", dtype, d, n)
    sm.gather_surrogates(lut.to(dev()), i32(rule), out, err, emb=emb.to(dev()), token_ids=i32(tok))
    st, ref = orc.gather_surrogates(wl.to_raw(emb), wl.to_raw(lut), tok, rule)
    assert st == orc.OK and int(err.item()) == 0
    assert np.array_equal(wl.to_raw(out.cpu()), ref)


def test_gather_out_of_range_rows_are_zero():
    d = 64
    lut = torch.ones((4, d), dtype=torch.bfloat16, device=dev())
    emb = torch.ones((8, d), dtype=torch.bfloat16, device=dev())
    out = torch.full((3, d), 7.0, dtype=torch.bfloat16, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.gather_surrogates(lut, i32([4, -1, 1]), out, err, emb=emb, token_ids=i32([0, 8, 0]))
    torch.cuda.synchronize()
    assert int(err.item()) == sm.ERR_EINVAL
    o = out.float().cpu()
    assert not o[0].any() and not o[1].any() and bool((o[2] == 1).all())


def _matched_spans(orc, rules, B, T, V, seed):
    toks, offs = wl.make_rule_prompts(rules, B, T, 0.4, V, seed)
    R = orc.OracleRules(rules)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK
    return toks, s0, ln, ru


def _gpu_dedupe(toks, s0, ln, ru, num_rules):
    S = len(s0)
    uniq = torch.full((S,), -7, dtype=torch.int32, device=dev())
    slot = torch.full((S,), -7, dtype=torch.int32, device=dev())
    rows = torch.full((int(ln.sum()),), -7, dtype=torch.int32, device=dev())
    offs = torch.full((S + 1,), -7, dtype=torch.int32, device=dev())
    nu = torch.zeros(1, dtype=torch.int32, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.span_dedupe(i32(ru), i32(s0), i32(ln), num_rules, i32(toks), uniq, slot, rows, offs, nu, err)
    torch.cuda.synchronize()
    U = int(nu.item())
    return U, uniq[:U].cpu().numpy(), slot.cpu().numpy(), offs[:U + 1].cpu().numpy(), rows, int(err.item())


@pytest.mark.parametrize("counts,B,T", [((4, 3, 2), 3, 200), ((300, 300, 300), 8, 1000), ((6, 0, 0), 1, 5000)])
def test_dedupe_matches_oracle(orc, counts, B, T):
    V = 64
    rules = wl.make_rules(counts=counts, vocab=V, seed=sum(counts))
    toks, s0, ln, ru = _matched_spans(orc, rules, B, T, V, seed=B)
    U, us, slot, uo, rows, err = _gpu_dedupe(toks, s0, ln, ru, len(rules))
    U0, us0, slot0, rows0, uo0 = orc.span_dedupe(ru, s0, ln, len(rules), toks)
    say("dedupe spans", len(s0), "unique", U0)
    assert err == 0 and U == U0
    assert np.array_equal(us, us0) and np.array_equal(slot, slot0) and np.array_equal(uo, uo0)
    assert np.array_equal(rows[:int(uo0[-1])].cpu().numpy(), rows0)


def test_dedupe_bad_rule_or_range():
    toks = np.arange(10, dtype=np.int32)
    for ru, s0, ln in (([0, 5], [0, 3], [2, 2]), ([0, 1], [0, 9], [2, 2])):   # rule 5 of 3; span past the end
        U, *_, err = _gpu_dedupe(toks, np.array(s0), np.array(ln), np.array(ru), 3)
        assert U == 0 and err == sm.ERR_EINVAL


def _setup_merge(d, h, V, seed):
    g = wl.generator(seed)
    emb = wl.randn((V, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, h, torch.bfloat16, g, spread=True)
    return emb, params


def _merge_gpu(emb, row_idx_dev, offs_np, params, h):
    S, d = len(offs_np) - 1, emb.shape[1]
    out = torch.full((S, d), float("nan"), dtype=torch.bfloat16, device=dev())
    ws = torch.empty(sm.merge_workspace_bytes(int(offs_np[-1]), S, d, torch.bfloat16), dtype=torch.uint8,
                     device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.merge_spans(emb, row_idx_dev, i32(offs_np), {k: v.to(dev()) for k, v in params.items()}, h, out, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return out


def _oracle_in_context(orc, emb, params, h, toks, s0, ln):
    rows = np.concatenate([toks[a:a + n] for a, n in zip(s0, ln)])
    st, ref = orc.merge_spans(wl.to_f64(emb), rows, np.concatenate([[0], np.cumsum(ln)]),
                              {k: wl.to_f64(v) for k, v in params.items()}, h)
    assert st == orc.OK
    return ref


def test_prompt_surrogates_from_rule_table(orc):
    """Table = M_phi over every rule (GPU); the prompt's span surrogates are
    looked up by the matched rule ids and compared with the oracle's merge
    of the spans in their prompts."""
    d, h, V = 1024, 4, 2000
    rules = wl.make_rules(counts=(150, 150, 150), vocab=V, seed=11)
    emb, params = _setup_merge(d, h, V, 12)
    toks, s0, ln, ru = _matched_spans(orc, rules, 4, 1500, V, seed=13)
    n_of = (rules >= 0).sum(1)
    lut = _merge_gpu(emb.to(dev()), i32(rules[rules >= 0]), np.concatenate([[0], np.cumsum(n_of)]).astype(np.int32),
                     params, h)
    z = torch.empty((len(s0), d), dtype=torch.bfloat16, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.gather_surrogates(lut, i32(ru), z, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = _oracle_in_context(orc, emb, params, h, toks, s0, ln)
    e = rel_l2_max(z.float().cpu().numpy(), ref)
    say("table surrogates: spans", len(s0), "rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


def test_prompt_surrogates_from_distinct_spans(orc):
    """Dedupe, merge only the distinct spans (GPU), spread back by slot."""
    d, h, V = 1024, 4, 500
    rules = wl.make_rules(counts=(20, 20, 20), vocab=V, seed=21)       # repeats in every prompt
    emb, params = _setup_merge(d, h, V, 22)
    toks, s0, ln, ru = _matched_spans(orc, rules, 4, 1500, V, seed=23)
    U, us, slot, uo, rows, err = _gpu_dedupe(toks, s0, ln, ru, len(rules))
    assert err == 0 and U < len(s0)
    zu = _merge_gpu(emb.to(dev()), rows[:int(uo[-1])].contiguous(), uo.astype(np.int32), params, h)
    z = torch.empty((len(s0), d), dtype=torch.bfloat16, device=dev())
    e_ = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.gather_surrogates(zu, i32(slot), z, e_)
    torch.cuda.synchronize()
    assert int(e_.item()) == 0
    ref = _oracle_in_context(orc, emb, params, h, toks, s0, ln)
    e = rel_l2_max(z.float().cpu().numpy(), ref)
    say("distinct spans", U, "of", len(s0), "rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]
