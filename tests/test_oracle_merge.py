"""Pins of the oracle's merge module M_phi (CPU only).

The oracle follows the appendix form (Linear -> GELU -> LayerNorm, per-head
learned-query pooling with P as key and value, Linear -> GELU -> LayerNorm).
It is pinned here by
  * a composition of independent library routines (torch fp64 F.linear,
    F.gelu, F.layer_norm and scaled_dot_product_attention, which with one
    query and key = value = P_i is exactly the pooling of one head),
  * closed-form special cases (zero projection, a single-row span),
  * invariants (permutation invariance, duplicated rows, weights sum to 1),
  * the paper's parameter count |phi| = 2d^2 + 7d.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import erf

from conftest import load_golden
from paper_2609_27233_amd import workload as wl


def _params(d, h, seed, spread=True):
    g = wl.generator(seed)
    p = wl.make_merge_params(d, h, torch.float32, g, spread=spread)
    return {k: wl.to_f64(v) for k, v in p.items()}


def _torch_merge(E, p, h, eps=1e-5):
    """M_phi of one span [n, d] built from torch library routines (fp64)."""
    t = {k: torch.from_numpy(v) for k, v in p.items()}
    E = torch.from_numpy(E)
    n, d = E.shape
    dh = d // h
    P = F.layer_norm(F.gelu(F.linear(E, t["W_kv"], t["b_kv"])), (d,), t["g_kv"], t["beta_kv"], eps)
    Ph = P.view(n, h, dh).transpose(0, 1).contiguous()          # [h, n, dh]
    o = F.scaled_dot_product_attention(t["Q"].view(h, 1, dh), Ph, Ph)  # [h, 1, dh]
    c = o.reshape(d)
    z = F.layer_norm(F.gelu(F.linear(c, t["W_o"], t["b_o"])), (d,), t["g_o"], t["beta_o"], eps)
    return z.numpy()


def _spans(rng, S, nmax, rows):
    lens = rng.randint(1, nmax + 1, size=S)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    row_idx = rng.randint(0, rows, size=offs[-1]).astype(np.int32)
    return row_idx, offs


@pytest.mark.parametrize("d,h", [(64, 4), (256, 4), (96, 3)])
def test_matches_torch_library_composition(orc, d, h):
    rng = np.random.RandomState(d + h)
    emb = rng.normal(0, 0.5, size=(50, d))
    p = _params(d, h, seed=d)
    row_idx, offs = _spans(rng, 12, 6, 50)
    st, out = orc.merge_spans(emb, row_idx, offs, p, h)
    assert st == orc.OK
    for s in range(len(offs) - 1):
        ref = _torch_merge(emb[row_idx[offs[s]:offs[s + 1]]], p, h)
        np.testing.assert_allclose(out[s], ref, rtol=1e-11, atol=1e-11)


def test_pooling_weights_are_softmax_over_span(orc):
    d, h = 64, 4
    rng = np.random.RandomState(3)
    emb = rng.normal(0, 1.0, size=(20, d))
    p = _params(d, h, seed=9)
    row_idx, offs = _spans(rng, 10, 5, 20)
    st, _, w = orc.merge_spans(emb, row_idx, offs, p, h, return_weights=True)
    assert st == orc.OK
    for s in range(10):
        n = offs[s + 1] - offs[s]
        np.testing.assert_allclose(w[s, :, :n].sum(axis=1), 1.0, atol=1e-13)
        assert np.all(w[s, :, :n] > 0)


def test_zero_projection_closed_form(orc):
    # W_kv = 0, b_kv = 0: GELU(0) = 0 and LayerNorm of a constant row is beta,
    # so P_j = beta_kv for every j, the pooled row is beta_kv (weights sum to
    # 1) and z = LN_o(GELU(W_o beta_kv + b_o)).  With W_o = 0 as well,
    # z = gamma_o (u - mean u) / sqrt(var u + eps) + beta_o, u = GELU(b_o).
    d, h, eps = 128, 4, 1e-5
    p = _params(d, h, seed=4)
    p["W_kv"][:] = 0
    p["b_kv"][:] = 0
    p["W_o"][:] = 0
    rng = np.random.RandomState(5)
    emb = rng.normal(size=(7, d))
    st, out = orc.merge_spans(emb, np.arange(7, dtype=np.int32), np.array([0, 3, 7], np.int32), p, h)
    assert st == orc.OK
    u = 0.5 * p["b_o"] * (1 + erf(p["b_o"] / np.sqrt(2)))
    ref = p["g_o"] * (u - u.mean()) / np.sqrt(u.var() + eps) + p["beta_o"]
    np.testing.assert_allclose(out[0], ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(out[1], ref, rtol=1e-12, atol=1e-12)


def test_single_row_span_weight_is_one(orc):
    d, h = 64, 4
    rng = np.random.RandomState(6)
    emb = rng.normal(size=(4, d))
    p = _params(d, h, seed=6)
    st, out, w = orc.merge_spans(emb, np.array([2], np.int32), np.array([0, 1], np.int32), p, h,
                                 return_weights=True)
    assert st == orc.OK
    np.testing.assert_array_equal(w[0, :, 0], 1.0)


def test_permutation_invariant(orc):
    # pooling has no positional term: shuffling a span's tokens keeps z
    d, h = 128, 4
    rng = np.random.RandomState(7)
    emb = rng.normal(0, 0.3, size=(30, d))
    p = _params(d, h, seed=7)
    rows = rng.randint(0, 30, size=6).astype(np.int32)
    perm = rng.permutation(6)
    st, out = orc.merge_spans(emb, np.concatenate([rows, rows[perm]]), np.array([0, 6, 12], np.int32), p, h)
    assert st == orc.OK
    np.testing.assert_allclose(out[0], out[1], rtol=1e-12, atol=1e-13)


def test_duplicated_rows_independent_of_n(orc):
    # n copies of one embedding pool to that embedding's P for every n
    d, h = 64, 4
    rng = np.random.RandomState(8)
    emb = rng.normal(size=(5, d))
    p = _params(d, h, seed=8)
    rows = np.array([3] * 1 + [3] * 2 + [3] * 5, np.int32)
    st, out = orc.merge_spans(emb, rows, np.array([0, 1, 3, 8], np.int32), p, h)
    assert st == orc.OK
    np.testing.assert_allclose(out[1], out[0], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out[2], out[0], rtol=1e-12, atol=1e-13)


def test_bare_form_is_eq1(orc):
    # flag 1 drops GELU, LayerNorm and biases: the main text's Eq. 1,
    # M(E) = W^o [o_1; ...; o_h], o_i = softmax(q_i^T (W^kv E)_i / sqrt(d_h)) (W^kv E)_i^T
    d, h = 64, 2
    rng = np.random.RandomState(10)
    emb = rng.normal(size=(6, d))
    p = _params(d, h, seed=10)
    st, out = orc.merge_spans(emb, np.arange(6, dtype=np.int32), np.array([0, 6], np.int32), p, h, flags=1)
    assert st == orc.OK
    K = emb @ p["W_kv"].T  # [n, d]: row j is W^kv e_j
    dh = d // h
    cols = []
    for i in range(h):
        Ki = K[:, i * dh:(i + 1) * dh]
        a = Ki @ p["Q"][i] / np.sqrt(dh)
        a = np.exp(a - a.max())
        a /= a.sum()
        cols.append(a @ Ki)
    ref = p["W_o"] @ np.concatenate(cols)
    np.testing.assert_allclose(out[0], ref, rtol=1e-12, atol=1e-13)


def test_parameter_count_matches_paper():
    gold = load_golden("param_count.json")
    # the generated parameter set has exactly the paper's shapes ...
    for d in (64, 256):
        p = wl.make_merge_params(d, 4, torch.float32, wl.generator(0))
        assert sum(v.numel() for v in p.values()) == 2 * d * d + 7 * d
    # ... and the closed form gives the paper's count at d = 4096
    d = gold["d"]
    assert 2 * d * d + 7 * d == gold["exact"]
    assert round((2 * d * d + 7 * d) / 1e6, 1) == gold["approx_millions"]


def test_rejects_bad_spans(orc):
    d, h = 64, 4
    p = _params(d, h, seed=1)
    emb = np.zeros((4, d))
    assert orc.merge_spans(emb, np.array([0, 9], np.int32), np.array([0, 2], np.int32), p, h)[0] == orc.EINVAL
    assert orc.merge_spans(emb, np.array([0, 1], np.int32), np.array([0, 0, 2], np.int32), p, h)[0] == orc.EINVAL


@pytest.mark.parametrize("d,h,spread", [(64, 4, True), (256, 4, False), (96, 3, True)])
def test_rows_form_matches_the_c_oracle_and_torch(orc, d, h, spread):
    """The batched-rows form used for full-size samples equals the C oracle
    span by span, and the torch library composition."""
    rng = np.random.RandomState(3 * d + h)
    emb = rng.normal(0, 0.5, size=(40, d))
    p = _params(d, h, seed=d + 1, spread=spread)
    row_idx, offs = _spans(rng, 20, 8, 40)
    offs = np.asarray(offs, np.int32)
    st, out = orc.merge_spans(emb, row_idx, offs, p, h)
    assert st == orc.OK
    rows = orc.merge_spans_rows(emb, row_idx, offs, p, h)
    np.testing.assert_allclose(rows, out, rtol=1e-11, atol=1e-11)
    for s in (0, 7, len(offs) - 2):
        np.testing.assert_allclose(rows[s], _torch_merge(emb[row_idx[offs[s]:offs[s + 1]]], p, h),
                                   rtol=1e-11, atol=1e-11)
    # a single-row span takes the whole weight; permuting a span's rows changes nothing
    one = orc.merge_spans_rows(emb, row_idx[:1], np.array([0, 1], np.int32), p, h)
    np.testing.assert_allclose(one[0], _torch_merge(emb[row_idx[:1]], p, h), rtol=1e-11, atol=1e-11)
    a, b = offs[3], offs[4]
    perm = row_idx.copy()
    perm[a:b] = perm[a:b][::-1]
    np.testing.assert_allclose(orc.merge_spans_rows(emb, perm, offs, p, h)[3], rows[3], rtol=1e-11, atol=1e-12)
