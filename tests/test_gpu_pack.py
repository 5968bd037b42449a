"""GPU pack_spans vs the oracle: compressed positions, packed offsets and
sources bit-exact; packed rows are byte copies."""
import numpy as np
import pytest
import torch

from gpu_util import dev, i32, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _gpu_pack(P, emb=None, surrogates=None):
    total = int(P.seq_offsets[-1])
    B = len(P.seq_offsets) - 1
    pi = torch.full((max(total, 1),), -7, dtype=torch.int32, device=dev())
    po = torch.full((B + 1,), -7, dtype=torch.int32, device=dev())
    ps = torch.full((max(total, 1),), -7, dtype=torch.int32, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    packed = None
    if emb is not None:
        packed = torch.zeros((max(total, 1), emb.shape[1]), dtype=emb.dtype, device=dev())
    sm.pack_spans(i32(P.seq_offsets), i32(P.span_start), i32(P.span_len), i32(P.seq_span_offsets),
                  pi, po, ps, err, total,
                  token_ids=i32(P.token_ids) if emb is not None else None,
                  emb=emb, surrogates=surrogates, packed=packed)
    torch.cuda.synchronize()
    return int(err.item()), pi.cpu().numpy()[:total], po.cpu().numpy(), ps.cpu().numpy(), packed


@pytest.mark.parametrize("wid,B", [(1, 1), (2, 16), (3, 4), (5, 3)])
def test_pack_indices_bit_exact(orc, wid, B):
    w = wl.WORKLOADS[wid]
    P = wl.make_prompts(w, batch=B)
    say("pack", w.name, "B", B, "spans", len(P.span_len))
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    err, pi, po, ps, _ = _gpu_pack(P)
    assert err == 0
    np.testing.assert_array_equal(pi, res["pi"])
    np.testing.assert_array_equal(po, res["packed_offsets"])
    np.testing.assert_array_equal(ps[:po[-1]], res["packed_src"])


@pytest.mark.parametrize("dtype,d", [(torch.bfloat16, 4096), (torch.float32, 256), (torch.bfloat16, 8192)])
def test_pack_rows_are_copies(orc, dtype, d):
    w = wl.WORKLOADS[2]
    P = wl.make_prompts(w, seed=77, batch=3, prompt_len=700)
    vocab = 3000
    P.token_ids[:] = P.token_ids % vocab
    g = wl.generator(5)
    emb = wl.randn((vocab, d), dtype, g, std=0.02)
    sur = wl.randn((len(P.span_len), d), dtype, g)
    say("pack rows", dtype, d, "spans", len(P.span_len))
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets,
                             token_ids=P.token_ids, emb_raw=wl.to_raw(emb), surrogates_raw=wl.to_raw(sur))
    assert st == orc.OK
    err, pi, po, ps, packed = _gpu_pack(P, emb.to(dev()), sur.to(dev()))
    assert err == 0
    n = int(po[-1])
    assert np.array_equal(wl.to_raw(packed[:n]), res["packed"])


def test_pack_edge_cases(orc):
    # a sequence with no spans, an empty sequence, a span covering a whole
    # sequence, single-token spans and back-to-back spans
    seq_offsets = np.array([0, 5, 5, 9, 17], np.int32)
    spans = [(5, 4), (9, 1), (10, 2), (12, 3), (16, 1)]
    P = wl.Prompts(token_ids=np.arange(17, dtype=np.int32), seq_offsets=seq_offsets,
                   span_start=np.array([s for s, _ in spans], np.int32),
                   span_len=np.array([n for _, n in spans], np.int32),
                   seq_span_offsets=np.array([0, 0, 0, 1, 5], np.int32))
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    err, pi, po, ps, _ = _gpu_pack(P)
    assert err == 0
    np.testing.assert_array_equal(pi, res["pi"])
    np.testing.assert_array_equal(po, res["packed_offsets"])
    np.testing.assert_array_equal(ps[:po[-1]], res["packed_src"])


def test_pack_invalid_spans_set_einval(orc):
    P = wl.Prompts(token_ids=np.arange(10, dtype=np.int32), seq_offsets=np.array([0, 10], np.int32),
                   span_start=np.array([2, 3], np.int32), span_len=np.array([3, 2], np.int32),
                   seq_span_offsets=np.array([0, 2], np.int32))
    st, _ = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.EINVAL
    err, *_ = _gpu_pack(P)
    assert err == sm.ERR_EINVAL
