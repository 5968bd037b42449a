"""GPU merge_spans (M_phi) vs the oracle."""
import math

import numpy as np
import pytest
import torch

from gpu_util import TOL, dev, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _gpu_merge(emb, row_idx, offs, params, h, dtype):
    S = len(offs) - 1
    d = emb.shape[1]
    out = torch.full((S, d), float("nan"), dtype=dtype, device=dev())
    ws = torch.empty(sm.merge_workspace_bytes(len(row_idx), S, d, dtype), dtype=torch.uint8, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    pd = {k: v.to(dev()) for k, v in params.items()}
    sm.merge_spans(emb, i32(row_idx), i32(offs), pd, h, out, ws, err)
    torch.cuda.synchronize()
    return out.cpu(), int(err.item())


def _oracle(orc, emb_rows_f64, row_idx, offs, params, h, sample=None):
    if sample is None:
        st, ref = orc.merge_spans(emb_rows_f64, row_idx, offs, {k: wl.to_f64(v) for k, v in params.items()}, h)
        assert st == orc.OK
        return ref
    # re-pack the sampled spans as their own CSR list
    rows = np.concatenate([row_idx[offs[s]:offs[s + 1]] for s in sample])
    so = np.concatenate([[0], np.cumsum([offs[s + 1] - offs[s] for s in sample])]).astype(np.int32)
    st, ref = orc.merge_spans(emb_rows_f64, rows, so, {k: wl.to_f64(v) for k, v in params.items()}, h)
    assert st == orc.OK
    return ref


@pytest.mark.parametrize("spread", [False, True])
def test_merge_tiny_f32(orc, spread):
    w = wl.WORKLOADS[1]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed)
    emb = wl.randn((w.vocab, w.d), torch.float32, g, std=0.02)
    params = wl.make_merge_params(w.d, w.h, torch.float32, g, spread=spread)
    say("merge f32 tiny spread", spread, "spans", len(P.span_len))
    out, err = _gpu_merge(emb.to(dev()), P.row_idx, P.span_offsets, params, w.h, torch.float32)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), P.row_idx, P.span_offsets, params, w.h)
    e = rel_l2_max(out.numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.float32]


@pytest.mark.parametrize("d,S,nmax,h", [(512, 50, 9, 8), (1024, 20, 5, 16), (768, 17, 3, 4)])
def test_merge_f32_heads(orc, d, S, nmax, h):
    """fp32 storage at several widths and head counts (768 takes the
    register form at 3 groups per lane)."""
    rng = np.random.RandomState(7 * d + S)
    lens = rng.randint(1, nmax + 1, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 500
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d + h)
    emb = wl.randn((vocab, d), torch.float32, g, std=0.02)
    params = wl.make_merge_params(d, h, torch.float32, g, spread=True)
    say("merge f32", d, S, nmax, h)
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, h, torch.float32)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, h)
    e = rel_l2_max(out.numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.float32]


@pytest.mark.parametrize("d,S,nmax,spread,h", [(512, 300, 8, True, 4), (1024, 129, 5, False, 4),
                                               (768, 37, 12, True, 4), (256, 1, 1, True, 4),
                                               (1024, 60, 6, True, 16), (2048, 40, 8, True, 8),
                                               (3584, 33, 5, True, 4), (1536, 20, 40, True, 2),
                                               (8192, 9, 4, True, 1)])
def test_merge_bf16_small(orc, d, S, nmax, spread, h):
    """Sizes cover the register-form pooling at 1..8 and 16 groups per lane,
    one to sixteen heads, spans longer than the four pooling waves, and the
    general form (d = 256 and 768 are not multiples of 512)."""
    rng = np.random.RandomState(d + S)
    lens = rng.randint(1, nmax + 1, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 2000
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d)
    emb = wl.randn((vocab, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, h, torch.bfloat16, g, spread=spread)
    say("merge bf16", d, S, nmax, spread, h)
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, h, torch.bfloat16)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, h)
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


def test_merge_bf16_large_tiles(orc):
    """Enough rows and spans that both projections take the 256 x 256-tile
    GEMM (at least 256 output tiles), with ragged last row tiles; the oracle
    checks a sample of spans from every part of the batch, the last ones
    included."""
    d, S = 512, 33000
    rng = np.random.RandomState(77)
    lens = rng.randint(1, 4, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 5000
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    assert (int(offs[-1]) + 255) // 256 * (d // 256) >= 256 and (S + 255) // 256 * (d // 256) >= 256
    assert int(offs[-1]) % 256 and S % 256
    g = wl.generator(d + 1)
    emb = wl.randn((vocab, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g, spread=True)
    say("merge bf16 large tiles", d, S, "rows", int(offs[-1]))
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, 4, torch.bfloat16)
    assert err == 0
    sample = np.unique(np.concatenate([rng.choice(S, 400, replace=False), np.arange(S - 300, S)]))
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, 4, sample=sample)
    e = rel_l2_max(out.float().numpy()[sample], ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


def test_merge_llama3_8b_prompt_batch(orc):
    """All ~9.7k spans of the 16 x 4096 workload in one call on the GPU; a
    seeded sample of spans checked against the oracle."""
    w = wl.WORKLOADS[2]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed, "cuda")
    emb = wl.randn((w.vocab, w.d), torch.bfloat16, g, device="cuda", std=0.02)
    params = wl.make_merge_params(w.d, w.h, torch.bfloat16, g, device="cuda")
    S = len(P.span_len)
    say("merge llama3-8b prompts, spans", S, "rows", len(P.row_idx))
    out, err = _gpu_merge(emb, P.row_idx, P.span_offsets, params, w.h, torch.bfloat16)
    assert err == 0
    rng = np.random.RandomState(0)
    sample = np.sort(rng.choice(S, size=24, replace=False))
    sample = np.unique(np.concatenate([sample, [0, S - 1]]))
    used = np.unique(np.concatenate([P.row_idx[P.span_offsets[s]:P.span_offsets[s + 1]] for s in sample]))
    # the oracle gets the used rows only (remapped), exact float64 copies
    remap = {int(r): i for i, r in enumerate(used)}
    emb_used = wl.to_f64(emb[torch.as_tensor(used, device="cuda")])
    sub_rows = np.concatenate([[remap[int(r)] for r in P.row_idx[P.span_offsets[s]:P.span_offsets[s + 1]]]
                               for s in sample]).astype(np.int32)
    so = np.concatenate([[0], np.cumsum([P.span_offsets[s + 1] - P.span_offsets[s] for s in sample])]).astype(np.int32)
    st, ref = orc.merge_spans(emb_used, sub_rows, so, {k: wl.to_f64(v) for k, v in params.items()}, w.h)
    assert st == orc.OK
    e = rel_l2_max(out[torch.as_tensor(sample)].float().numpy(), ref)
    say("rel_l2_max over", len(sample), "spans:", e)
    assert e <= TOL[torch.bfloat16]
    assert torch.isfinite(out.float()).all()


def test_merge_bad_row_index_sets_einval(orc):
    d = 256
    g = wl.generator(3)
    emb = wl.randn((10, d), torch.bfloat16, g)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g)
    say("merge bad row index")
    out, err = _gpu_merge(emb.to(dev()), np.array([1, 2, 99], np.int32), np.array([0, 2, 3], np.int32),
                          params, 4, torch.bfloat16)
    assert err == sm.ERR_EINVAL


def test_merge_sorted_rows_bad_ids_and_repeat(orc):
    """A bf16 batch large enough for the 256-tile first stage, which runs in
    token-id order (rows sorted by a counting sort, G1 read back through the
    inverse permutation): ids outside the table set EINVAL and are read as
    row 0, every other span is pooled as usual, and a second call gives the
    same bits (the permutation does not depend on timing)."""
    d, S, vocab = 512, 17000, 3000
    rng = np.random.RandomState(91)
    lens = rng.randint(1, 4, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    R = int(offs[-1])
    assert (R + 255) // 256 * (d // 256) >= 256 and R % 4096
    # a skewed id law: a tenth of the rows share 5 ids, so some buckets are large
    row_idx = rng.randint(0, vocab, size=R).astype(np.int32)
    hot = rng.rand(R) < 0.1
    row_idx[hot] = rng.randint(0, 5, size=int(hot.sum()))
    bad_spans = [5, S // 2, S - 1]
    bad_ids = [-7, vocab, vocab + 123]
    for s, b in zip(bad_spans, bad_ids):
        row_idx[offs[s]] = b
    g = wl.generator(d + 7)
    emb = wl.randn((vocab, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g, spread=True)
    say("merge sorted rows, bad ids and repeat", d, S, "rows", R)
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, 4, torch.bfloat16)
    assert err == sm.ERR_EINVAL
    out2, err2 = _gpu_merge(emb.to(dev()), row_idx, offs, params, 4, torch.bfloat16)
    assert err2 == sm.ERR_EINVAL and torch.equal(out.view(torch.int16), out2.view(torch.int16))
    fixed = row_idx.copy()
    fixed[(fixed < 0) | (fixed >= vocab)] = 0
    sample = np.unique(np.concatenate([rng.choice(S, 300, replace=False), bad_spans, [0, 1]]))
    ref = _oracle(orc, wl.to_f64(emb), fixed, offs, params, 4, sample=sample)
    e = rel_l2_max(out.float().numpy()[sample], ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


@pytest.mark.parametrize("d,S", [(4096, 16), (3584, 128), (8192, 4)])
def test_merge_decode_time_batches(orc, d, S):
    """Decode-time merges: one freshly completed span of n = 2..4 tokens per
    sequence (a few rows: the skinny GEMM path) at the model widths of the
    benchmark layers."""
    rng = np.random.RandomState(d + S)
    lens = rng.randint(2, 5, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 1500
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d + 1, "cuda")
    emb = wl.randn((vocab, d), torch.bfloat16, g, device="cuda", std=0.02)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g, device="cuda", spread=True)
    say("merge decode-time", d, S, "rows", int(offs[-1]))
    out, err = _gpu_merge(emb, row_idx, offs, params, 4, torch.bfloat16)
    assert err == 0
    sample = np.arange(S) if S <= 16 else np.sort(rng.choice(S, size=12, replace=False))
    used = np.unique(np.concatenate([row_idx[offs[s]:offs[s + 1]] for s in sample]))
    remap = {int(r): i for i, r in enumerate(used)}
    sub_rows = np.array([remap[int(r)] for s in sample for r in row_idx[offs[s]:offs[s + 1]]], np.int32)
    so = np.concatenate([[0], np.cumsum([offs[s + 1] - offs[s] for s in sample])]).astype(np.int32)
    st, ref = orc.merge_spans(wl.to_f64(emb[torch.as_tensor(used, device="cuda")]), sub_rows, so,
                              {k: wl.to_f64(v) for k, v in params.items()}, 4)
    assert st == orc.OK
    e = rel_l2_max(out[torch.as_tensor(sample)].float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


@pytest.mark.parametrize("d,h,lens", [
    (2048, 8, [1, 4, 5, 9, 64, 255, 256, 2, 3, 8, 1, 17]),  # one to 64 groups of four rows
    (6144, 6, [1, 2, 3, 4, 5, 6, 7, 13, 2, 4]),             # three groups per lane; heads straddle the quarters
    (8192, 16, [4, 8, 1, 3, 12]),                             # four groups per lane, four heads per quarter
])
def test_merge_slice_pooling_spans_and_heads(orc, d, h, lens):
    """The column-slice pooling kernel (d a multiple of 2048): spans from one
    row to the 256-row limit, so the online softmax folds from one to 64
    groups of rows, and head counts whose heads straddle the workgroup's
    column quarters (d = 6144, h = 6: 1024-column heads over 1536-column
    quarters)."""
    rng = np.random.RandomState(d + h)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 600
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d + 3 * h)
    emb = wl.randn((vocab, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, h, torch.bfloat16, g, spread=True)
    say("merge slice pooling", d, h, "spans", len(lens), "rows", int(offs[-1]))
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, h, torch.bfloat16)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, h)
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]


@pytest.mark.parametrize("d,h", [(1024, 4), (4096, 16)])
def test_merge_slice_pooling_rows_far_from_zero_f32(orc, d, h):
    """fp32 rows whose values sit far from zero (first-stage bias + 16, row
    spread about 0.6): LN_kv statistics formed as E[x^2] - E[x]^2 would lose
    about 2e-5 of relative precision here; the shifted sums of the slice
    pooling keep the result within the fp32 bar (d = 1024 and 4096: one and
    four 16-byte groups per lane)."""
    rng = np.random.RandomState(d)
    lens = rng.randint(1, 9, size=24)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    vocab = 300
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d + 11)
    emb = wl.randn((vocab, d), torch.float32, g, std=1.0)
    params = wl.make_merge_params(d, h, torch.float32, g, spread=True)
    params["b_kv"] = params["b_kv"] + 16.0
    say("merge f32 offset rows", d, h, "rows", int(offs[-1]))
    out, err = _gpu_merge(emb.to(dev()), row_idx, offs, params, h, torch.float32)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, h)
    e = rel_l2_max(out.numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.float32]


@pytest.mark.parametrize("d", [256, 2048])
def test_merge_empty_span_sets_einval(orc, d):
    """A span with no rows (CSR offsets 0, 3, 3, 5): EINVAL, a zero pooled
    vector for it (so its surrogate is LN_o(GELU(b_o))), and the other spans
    still pooled as the oracle does (d = 256: the one-workgroup-per-span
    kernel; d = 2048: the column-slice kernel)."""
    g = wl.generator(d + 21)
    emb = wl.randn((40, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g, spread=True)
    row_idx = np.array([3, 7, 11, 19, 23], np.int32)
    say("merge empty span", d)
    out, err = _gpu_merge(emb.to(dev()), row_idx, np.array([0, 3, 3, 5], np.int32), params, 4, torch.bfloat16)
    assert err == sm.ERR_EINVAL
    p64 = {k: wl.to_f64(v) for k, v in params.items()}
    y = p64["b_o"] * 0.5 * (1.0 + np.vectorize(math.erf)(p64["b_o"] / math.sqrt(2.0)))
    z_empty = (y - y.mean()) / np.sqrt(y.var() + 1e-5) * p64["g_o"] + p64["beta_o"]
    ref = _oracle(orc, wl.to_f64(emb), row_idx, np.array([0, 3, 5], np.int32), params, 4)
    ref = np.stack([ref[0], z_empty, ref[1]])
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]
