"""Pins of the oracle's prompt packing (CPU only).

Worked examples printed in the paper (golden fixtures), the closed forms
L~_p = L_p - sum(j - i - 1) and pi(t) = t - r(t), the RoPE relative-offset
property of compressed positions, and a brute-force left-to-right rebuild of
the compressed sequence.
"""
import numpy as np
import pytest

from conftest import load_golden
from paper_2609_27233_amd import workload as wl


def _pack_one(orc, T, spans):
    starts = np.array([s for s, _ in spans], np.int32)
    lens = np.array([n for _, n in spans], np.int32)
    return orc.pack_spans(np.array([0, T], np.int32), starts, lens,
                          np.array([0, len(spans)], np.int32))


def _units(res, names):
    return [names[s] if s >= 0 else "z%d" % (-1 - s) for s in res["packed_src"]]


def test_prompt_time_worked_example(orc):
    g = load_golden("prompt_merge_example.json")
    st, res = _pack_one(orc, len(g["tokens"]), g["spans"])
    assert st == orc.OK
    assert _units(res, g["tokens"]) == g["packed_units"]
    # the position of each packed unit is its index: contiguous positions
    assert list(range(res["packed_offsets"][1])) == g["packed_positions"]
    # a kept token sits at position pi; the surrogate at pi of its last token
    for t, name in enumerate(g["tokens"]):
        unit = _units(res, g["tokens"])[res["pi"][t]]
        assert unit == name or unit.startswith("z")


def test_mask_alignment_worked_example(orc):
    g = load_golden("mask_alignment_example.json")
    toks = g["tokens"]
    st, res = _pack_one(orc, len(toks), g["spans"])
    assert st == orc.OK
    units = _units(res, toks)
    assert units == g["packed_units"]
    # keep mask: the position a packed unit is anchored to (the token itself,
    # or the last token of a span)
    keep = np.zeros(len(toks), int)
    for r, src in enumerate(res["packed_src"]):
        if src >= 0:
            keep[src] = 1
        else:
            s0, n = g["spans"][-1 - src]
            keep[s0 + n - 1] = 1
    first = min(s for s, _ in g["spans"])
    teacher = keep * (np.arange(len(toks)) >= first)
    assert teacher.tolist() == g["teacher_mask"]
    L = int(res["packed_offsets"][1])
    assert [1] * L == g["attn_mask"]
    N = int(teacher.sum())
    student = [0] * (L - N) + [1] * N
    assert student == g["student_mask"]
    pairs = [[toks[t], units[res["pi"][t]]] for t in range(len(toks)) if teacher[t]]
    assert pairs == g["aligned_pairs"]


def test_packed_length_closed_form(orc):
    g = load_golden("decode_merge_lengths.json")
    for T, spans, expect in g["prompt_cases"]:
        st, res = _pack_one(orc, T, [(i, j - i) for i, j in spans])
        assert st == orc.OK
        assert res["packed_offsets"][1] == expect == T - sum(j - i - 1 for i, j in spans)


def _random_prompts(seed, B=3, T=300):
    w = wl.WORKLOADS[2]
    return wl.make_prompts(w, seed=seed, batch=B, prompt_len=T)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_pi_is_t_minus_removed_before(orc, seed):
    P = _random_prompts(seed)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    removed = np.zeros(P.seq_offsets[-1], bool)
    for s, n in zip(P.span_start, P.span_len):
        removed[s:s + n - 1] = True
    for b in range(len(P.seq_offsets) - 1):
        a, e = P.seq_offsets[b], P.seq_offsets[b + 1]
        for t in range(a, e):
            r_t = int(removed[a:t].sum())  # positions removed before t
            assert res["pi"][t] == (t - a) - r_t
        # packed length of each sequence
        nb = int(np.sum((P.span_start >= a) & (P.span_start < e)))
        spans_b = P.span_len[P.seq_span_offsets[b]:P.seq_span_offsets[b + 1]]
        assert nb == len(spans_b)
        assert res["packed_offsets"][b + 1] - res["packed_offsets"][b] == (e - a) - int(np.sum(spans_b - 1))


def test_relative_offsets_kept_inside_unmerged_regions(orc):
    # "Structural effect under RoPE": if r(i) = r(j) then pi(j) - pi(i) = j - i;
    # across merged spans the distance shrinks by exactly r(j) - r(i)
    P = _random_prompts(5, B=1, T=200)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    keep_t = [t for t in range(200) if not any(s <= t < s + n - 1 for s, n in zip(P.span_start, P.span_len))]
    removed = np.zeros(200, int)
    for s, n in zip(P.span_start, P.span_len):
        removed[s:s + n - 1] = 1
    r = np.concatenate([[0], np.cumsum(removed)])[:-1]
    for i in keep_t[::7]:
        for j in keep_t[::11]:
            if j <= i:
                continue
            d = res["pi"][j] - res["pi"][i]
            assert d == (j - i) - (r[j] - r[i])
            if r[i] == r[j]:
                assert d == j - i


def test_bruteforce_left_to_right_rebuild(orc):
    # walk the prompt left to right; at a span start emit the surrogate and
    # jump past the span, else emit the token (prompt-merging procedure)
    P = _random_prompts(9, B=4, T=257)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    start_of = {int(s): k for k, s in enumerate(P.span_start)}
    expect = []
    for b in range(4):
        t, e = int(P.seq_offsets[b]), int(P.seq_offsets[b + 1])
        while t < e:
            if t in start_of:
                k = start_of[t]
                expect.append(-1 - k)
                t += int(P.span_len[k])
            else:
                expect.append(t)
                t += 1
    assert res["packed_src"].tolist() == expect


def test_packed_rows_are_copies(orc):
    P = _random_prompts(11, B=2, T=64)
    rng = np.random.RandomState(0)
    d = 16
    emb = rng.randint(0, 65535, size=(wl.WORKLOADS[2].vocab, d)).astype(np.uint16)
    sur = rng.randint(0, 65535, size=(len(P.span_len), d)).astype(np.uint16)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets,
                             token_ids=P.token_ids, emb_raw=emb, surrogates_raw=sur)
    assert st == orc.OK
    for r, src in enumerate(res["packed_src"]):
        row = emb[P.token_ids[src]] if src >= 0 else sur[-1 - src]
        np.testing.assert_array_equal(res["packed"][r], row)


@pytest.mark.parametrize("spans", [
    [(1, 3), (2, 2)],   # overlapping
    [(3, 2), (0, 2)],   # unsorted
    [(7, 3)],           # runs past the sequence end
    [(2, 0)],           # empty span
])
def test_rejects_invalid_spans(orc, spans):
    st, _ = _pack_one(orc, 8, spans)
    assert st == orc.EINVAL


def test_generator_hits_targets():
    for wid in (1, 2):
        w = wl.WORKLOADS[wid]
        P = wl.make_prompts(w, batch=2)
        for b in range(2):
            lens = P.span_len[P.seq_span_offsets[b]:P.seq_span_offsets[b + 1]]
            if w.target_kind == "reduction":
                assert int(np.sum(lens - 1)) == round(w.target * w.prompt_len)
            else:
                assert int(np.sum(lens)) == round(w.target * w.prompt_len)
            assert set(lens.tolist()) <= set(w.span_n)
