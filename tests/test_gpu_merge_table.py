"""GPU token table of M_phi's first stage and the tabled merge vs the
oracle (the table is exact: GELU(Linear_kv(e)) depends on the token alone)."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, dev, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _table(emb, params, h):
    table = torch.full_like(emb, float("nan"))
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.merge_token_table(emb, {k: v.to(dev()) for k, v in params.items()}, h, table, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return table


def _tabled(table, row_idx, offs, params, h):
    S = len(offs) - 1
    d = table.shape[1]
    out = torch.full((S, d), float("nan"), dtype=table.dtype, device=dev())
    ws = torch.empty(sm.merge_workspace_bytes(0, S, d, table.dtype), dtype=torch.uint8, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.merge_spans_tabled(table, i32(row_idx), i32(offs), {k: v.to(dev()) for k, v in params.items()}, h,
                          out, ws, err)
    torch.cuda.synchronize()
    return out.cpu(), int(err.item())


def _oracle(orc, emb_f64, row_idx, offs, params, h, sample):
    used = np.unique(np.concatenate([row_idx[offs[s]:offs[s + 1]] for s in sample]))
    remap = {int(r): k for k, r in enumerate(used)}
    rows = np.array([remap[int(r)] for s in sample for r in row_idx[offs[s]:offs[s + 1]]], np.int32)
    so = np.concatenate([[0], np.cumsum([offs[s + 1] - offs[s] for s in sample])]).astype(np.int32)
    st, ref = orc.merge_spans(emb_f64[used], rows, so, {k: wl.to_f64(v) for k, v in params.items()}, h)
    assert st == orc.OK
    return ref


@pytest.mark.parametrize("dtype,d,vocab", [(torch.float32, 256, 1000), (torch.bfloat16, 512, 40),
                                           (torch.bfloat16, 1024, 3000)])
def test_token_table_rows(dtype, d, vocab):
    """Table rows against GELU(emb W_kv^T + b_kv) computed in float64 on the
    CPU from the same stored inputs (the skinny, 128- and 256-tile GEMMs)."""
    g = wl.generator(d + vocab)
    emb = wl.randn((vocab, d), dtype, g, std=0.02)
    params = wl.make_merge_params(d, 4, dtype, g, spread=True)
    say("token table", dtype, d, vocab)
    table = _table(emb.to(dev()), params, 4).cpu()
    x = wl.to_f64(emb) @ wl.to_f64(params["W_kv"]).T + wl.to_f64(params["b_kv"])
    from scipy.special import erf
    ref = 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))
    e = rel_l2_max(table.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[dtype]


def test_tabled_merge_tiny_f32(orc):
    w = wl.WORKLOADS[1]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed)
    emb = wl.randn((w.vocab, w.d), torch.float32, g, std=0.02)
    params = wl.make_merge_params(w.d, w.h, torch.float32, g, spread=True)
    S = len(P.span_len)
    say("tabled merge f32 tiny, spans", S)
    table = _table(emb.to(dev()), params, w.h)
    out, err = _tabled(table, P.row_idx, P.span_offsets, params, w.h)
    assert err == 0
    ref = _oracle(orc, wl.to_f64(emb), P.row_idx, P.span_offsets, params, w.h, np.arange(S))
    e = rel_l2_max(out.numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.float32]


@pytest.mark.parametrize("S,nmin,nmax", [(16, 2, 4), (700, 2, 8)])
def test_tabled_merge_llama3_8b_width(orc, S, nmin, nmax):
    """A decode-time batch (16 spans of 2-4 tokens) and a prompt-time batch
    at d = 4096, vocab 3000; every span (or a sample with both ends) against
    the oracle, and against sm_merge_spans on the same inputs."""
    d, h, vocab = 4096, 4, 3000
    rng = np.random.RandomState(S)
    lens = rng.randint(nmin, nmax + 1, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    row_idx = rng.randint(0, vocab, size=int(offs[-1])).astype(np.int32)
    g = wl.generator(d + S, "cuda")
    emb = wl.randn((vocab, d), torch.bfloat16, g, device="cuda", std=0.02)
    params = wl.make_merge_params(d, h, torch.bfloat16, g, device="cuda", spread=True)
    say("tabled merge bf16 d 4096 spans", S, "rows", int(offs[-1]))
    table = _table(emb, params, h)
    out, err = _tabled(table, row_idx, offs, params, h)
    assert err == 0
    sample = np.arange(S) if S <= 16 else np.unique(np.concatenate([rng.choice(S, 20, replace=False), [0, S - 1]]))
    ref = _oracle(orc, wl.to_f64(emb), row_idx, offs, params, h, sample)
    e = rel_l2_max(out[torch.as_tensor(sample)].float().numpy(), ref)
    say("rel_l2_max vs oracle", e)
    assert e <= TOL[torch.bfloat16]
    # the untabled call on the same inputs
    ws = torch.empty(sm.merge_workspace_bytes(len(row_idx), S, d, torch.bfloat16), dtype=torch.uint8, device=dev())
    out2 = torch.empty((S, d), dtype=torch.bfloat16, device=dev())
    err2 = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.merge_spans(emb, i32(row_idx), i32(offs), {k: v.to(dev()) for k, v in params.items()}, h, out2, ws, err2)
    torch.cuda.synchronize()
    assert int(err2.item()) == 0
    e2 = rel_l2_max(out.float().numpy(), out2.float().cpu().numpy())
    say("rel_l2_max vs sm_merge_spans", e2)
    assert e2 <= TOL[torch.bfloat16]


@pytest.mark.parametrize("d", [256, 2048])
def test_tabled_merge_bad_token_sets_einval(orc, d):
    """A token id past the table: EINVAL, that row read as row 0, the other
    spans exact (d = 256: the one-workgroup-per-span pooling; d = 2048: the
    column-slice pooling)."""
    g = wl.generator(5 + d)
    emb = wl.randn((10, d), torch.bfloat16, g, std=0.02)
    params = wl.make_merge_params(d, 4, torch.bfloat16, g, spread=True)
    say("tabled merge bad token", d)
    table = _table(emb.to(dev()), params, 4)
    out, err = _tabled(table, np.array([1, 2, 10, 4, 5], np.int32), np.array([0, 2, 3, 5], np.int32), params, 4)
    assert err == sm.ERR_EINVAL
    assert torch.isfinite(out.float()).all()
    # the bad id is read as row 0, so span 1 pools row 0
    ref = _oracle(orc, wl.to_f64(emb), np.array([1, 2, 0, 4, 5], np.int32), np.array([0, 2, 3, 5], np.int32),
                  params, 4, np.arange(3))
    e = rel_l2_max(out.float().numpy(), ref)
    say("rel_l2_max", e)
    assert e <= TOL[torch.bfloat16]
