"""The oracle's surrogate lookup and span dedupe, pinned by the property the
paper gives for them (a span's surrogate depends on its tokens only, so a
table of per-rule surrogates and a merge of only the distinct spans both
reproduce the merge of every span), by first-occurrence brute force, and by
the fallback and range rules."""
import numpy as np
import pytest

from paper_2609_27233_amd import workload as wl


def _params(orc, d, h, seed):
    rng = np.random.RandomState(seed)
    p = {"Q": rng.randn(h, d // h), "W_kv": rng.randn(d, d) * 0.1, "b_kv": rng.randn(d) * 0.1,
         "g_kv": 1 + 0.1 * rng.randn(d), "beta_kv": 0.1 * rng.randn(d), "W_o": rng.randn(d, d) * 0.1,
         "b_o": rng.randn(d) * 0.1, "g_o": 1 + 0.1 * rng.randn(d), "beta_o": 0.1 * rng.randn(d)}
    return p


def _spans_from_rules(orc, rules, V, seed):
    toks, offs = wl.make_rule_prompts(rules, 3, 60, 0.4, V, seed)
    R = orc.OracleRules(rules)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK and len(s0) > 5
    return toks, s0, ln, ru


def test_lookup_table_reproduces_in_context_merge(orc):
    """Surrogates of every rule, computed once from the rule's own tokens,
    equal the merge of the same spans inside prompts (exactly, in fp64)."""
    d, h, V = 32, 4, 50
    rules = wl.make_rules(counts=(12, 10, 8), vocab=V, seed=1)
    emb = np.random.RandomState(2).randn(V, d)
    p = _params(orc, d, h, 3)
    n_of = (rules >= 0).sum(1)
    st, lut = orc.merge_spans(emb, rules[rules >= 0], np.concatenate([[0], np.cumsum(n_of)]), p, h)
    assert st == orc.OK
    toks, s0, ln, ru = _spans_from_rules(orc, rules, V, seed=4)
    rows = np.concatenate([toks[a:a + n] for a, n in zip(s0, ln)])
    st, z = orc.merge_spans(emb, rows, np.concatenate([[0], np.cumsum(ln)]), p, h)
    assert st == orc.OK
    st, got = orc.gather_surrogates(np.zeros((1, d)), lut, None, ru)
    assert st == orc.OK
    assert np.array_equal(got, z)


def test_dedupe_first_occurrence_and_merge_equivalence(orc):
    d, h, V = 32, 4, 40
    rules = wl.make_rules(counts=(4, 3, 2), vocab=V, seed=5)       # few rules: many repeats
    toks, s0, ln, ru = _spans_from_rules(orc, rules, V, seed=6)
    U, us, slot, urows, uoffs = orc.span_dedupe(ru, s0, ln, len(rules), toks)
    first = {}
    for s, r in enumerate(ru):
        first.setdefault(int(r), s)
    want_us = sorted(first.values())
    assert us.tolist() == want_us and U == len(want_us) < len(ru)
    assert [want_us[slot[s]] for s in range(len(ru))] == [first[int(r)] for r in ru]
    emb = np.random.RandomState(7).randn(V, d)
    p = _params(orc, d, h, 8)
    st, z_u = orc.merge_spans(emb, urows, uoffs, p, h)
    assert st == orc.OK
    rows = np.concatenate([toks[a:a + n] for a, n in zip(s0, ln)])
    st, z_all = orc.merge_spans(emb, rows, np.concatenate([[0], np.cumsum(ln)]), p, h)
    assert st == orc.OK
    assert np.array_equal(z_u[slot], z_all)


def test_gather_fallback_and_range(orc):
    rng = np.random.RandomState(9)
    emb = rng.randint(0, 65535, (20, 8)).astype(np.uint16)
    lut = rng.randint(0, 65535, (5, 8)).astype(np.uint16)
    st, out = orc.gather_surrogates(emb, lut, [3, 7, 19, 2], [-1, 4, -1, 0])
    assert st == orc.OK
    assert np.array_equal(out, np.stack([emb[3], lut[4], emb[19], lut[0]]))
    st, out = orc.gather_surrogates(emb, lut, [20, 1], [-1, 5])          # token and rule out of range
    assert st == orc.EINVAL and not out.any()


def test_dedupe_rejects_bad_rule_ids(orc):
    U, *_ = orc.span_dedupe([0, 3], [0, 2], [2, 2], 3, np.arange(4))
    assert U == -1
