"""The oracle's rule set and its two matching procedures, pinned by the
appendix's worked example and hand-worked cases (tests/golden), by the
paper's second statement of the prompt-time assignment (all matches sorted
by start, longer first, kept when they do not overlap a kept one), by
Python-set membership, and by a run-length form of the decode-time rule."""
import numpy as np
import pytest

from conftest import load_golden

pytestmark = pytest.mark.filterwarnings("ignore")


def _rules(orc, grams):
    R = orc.OracleRules(orc.rule_keys(grams))
    assert R.status == orc.OK
    return R


def test_worked_and_hand_examples(orc):
    g = load_golden("rule_matching_examples.json")
    for case in g["prompt_cases"]:
        R = _rules(orc, case["rules"])
        toks = case["tokens"]
        st, s0, ln, ru, sso = R.match_prompt(toks, [0, len(toks)])
        assert st == orc.OK
        assert [[int(a), int(b)] for a, b in zip(s0, ln)] == case["spans"], case["note"]
        # the paper's length formula: L~ = L - sum over spans (n - 1)
        assert len(toks) - int(np.sum(ln - 1)) == case["compressed_len"]
        for a, b, r in zip(s0, ln, ru):
            assert tuple(toks[a:a + b]) == tuple(case["rules"][r])
    for case in g["decode_cases"]:
        R = _rules(orc, case["rules"])
        ks = [R.decode_step(0, t)[0] for t in case["stream"]]
        assert ks == case["k"], case["note"]


def _all_matches_then_filter(toks, offs, ruleset):
    """The assignment as the 'Non-overlapping Assignment in a Sequence'
    paragraph states it: every occurrence of every rule, sorted by start and
    then by decreasing length, kept when it overlaps no kept one."""
    out = []
    for b in range(len(offs) - 1):
        x = toks[offs[b]:offs[b + 1]]
        cand = [(i, n) for i in range(len(x)) for n in (2, 3, 4)
                if i + n <= len(x) and tuple(x[i:i + n]) in ruleset]
        cand.sort(key=lambda c: (c[0], -c[1]))
        end = 0
        for i, n in cand:
            if i >= end:
                out.append((offs[b] + i, n))
                end = i + n
    return out


@pytest.mark.parametrize("seed", range(6))
def test_scan_equals_sorted_filter_statement(orc, seed):
    rng = np.random.RandomState(seed)
    V = 6 + seed                     # small vocabulary: dense matches and overlaps
    grams = set()
    for _ in range(40 + 10 * seed):
        n = rng.randint(2, 5)
        grams.add(tuple(int(t) for t in rng.randint(0, V, n)))
    grams = sorted(grams)
    R = _rules(orc, grams)
    lens = rng.randint(0, 60, size=5)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    toks = rng.randint(0, V, int(offs[-1])).astype(np.int32)
    st, s0, ln, ru, sso = R.match_prompt(toks, offs)
    assert st == orc.OK
    want = _all_matches_then_filter(list(toks), list(offs), set(grams))
    assert list(zip(s0.tolist(), ln.tolist())) == want
    # spans stay inside their sequence, in order, and the CSR ranges agree
    for b in range(len(lens)):
        for j in range(sso[b], sso[b + 1]):
            assert offs[b] <= s0[j] and s0[j] + ln[j] <= offs[b + 1]
    assert np.all(np.diff(s0) > 0) if len(s0) > 1 else True
    for a, n, r in zip(s0, ln, ru):
        assert tuple(toks[a:a + n].tolist()) == grams[r]


def test_find_matches_python_set(orc):
    rng = np.random.RandomState(3)
    grams = sorted({tuple(int(t) for t in rng.randint(0, 50, rng.randint(2, 5))) for _ in range(500)})
    R = _rules(orc, grams)
    assert R.count == len(grams)
    index = {g: i for i, g in enumerate(grams)}
    for _ in range(3000):
        q = tuple(int(t) for t in rng.randint(0, 50, rng.randint(2, 5)))
        assert R.find(list(q)) == index.get(q, -1)
    assert R.find([-1, 3]) == -1 and R.find([3]) == -1


def test_duplicates_keep_first_index(orc):
    R = _rules(orc, [(5, 6), (7, 8, 9), (5, 6), (7, 8, 9), (1, 2)])
    assert R.count == 3
    assert R.find([5, 6]) == 0 and R.find([7, 8, 9]) == 1 and R.find([1, 2]) == 4


@pytest.mark.parametrize("bad", [[[5, -1, -1, -1]], [[5, -1, 6, -1]], [[5, 6, -3, -1]], [[-1, 5, 6, -1]]])
def test_malformed_rules_rejected(orc, bad):
    R = orc.OracleRules(np.array(bad, np.int32))
    assert R.status == orc.EINVAL and R.count == 0


def test_no_match_across_sequences_or_through_negative_ids(orc):
    R = _rules(orc, [(1, 2), (3, 4)])
    st, s0, ln, ru, sso = R.match_prompt([5, 1, 2, 3, -1, 4, 3, 4], [0, 2, 5, 8])
    # (1, 2) straddles sequences 0/1; (3, -1) holds a negative id; (3, 4) in sequence 2 merges
    assert s0.tolist() == [6] and ln.tolist() == [2] and sso.tolist() == [0, 0, 0, 1]


def _decode_run_length(grams, stream):
    """Decode-time rule written with a run length: r = raw tokens since the
    last merge; the candidate suffixes are the last n <= min(r, 4) tokens."""
    ruleset = set(map(tuple, grams))
    hist, r, ks = [], 0, []
    for t in stream:
        hist.append(t)
        r += 1
        k = 0
        for n in (4, 3, 2):
            if n <= r and tuple(hist[-n:]) in ruleset:
                k, r = n - 1, 0
                break
        ks.append(k)
    return ks


@pytest.mark.parametrize("seed", range(5))
def test_decode_equals_run_length_form(orc, seed):
    rng = np.random.RandomState(50 + seed)
    V = 5
    grams = sorted({tuple(int(t) for t in rng.randint(0, V, rng.randint(2, 5))) for _ in range(25)})
    R = _rules(orc, grams)
    for seq in range(4):
        stream = rng.randint(0, V, 80).tolist()
        ks = [R.decode_step(seq, t)[0] for t in stream]
        assert ks == _decode_run_length(grams, stream)
        # the list keeps one entry per cached unit: raw tokens + merged markers
        assert len(R.state(seq)) == len(stream) - sum(ks)
