"""Parity at the five workloads, at their full sizes.

Each test runs the workload's job on the GPU and on the oracle in lock
step: prompt compression (merge, pack, bulk append of the compressed
prompt's K/V), then decode steps with decode-time merges (merge module,
rollback of n-1 entries, append of the surrogate's K/V) or plain token
appends, and decode attention after every step.  Integer state (block
tables, lengths, free stack, pools) is compared bit for bit after every
cache update; floating outputs are compared on every sequence for the small
workloads and on a seeded sample of sequences / spans for the large
ones.
"""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_same_state, dev, gpu_cache_like, i32, rel_l2_max, say
from paper_2609_27233_amd import lib as sm
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def _merge_check(orc, emb, params, h, row_idx, offs, out, sample, tol):
    """Oracle M_phi on the sampled spans (with only the embedding rows they
    use) against the GPU surrogates of those spans.  Large samples take the
    oracle's batched-rows form (the same definition, weights streamed once
    per call)."""
    used = np.unique(np.concatenate([row_idx[offs[s]:offs[s + 1]] for s in sample]))
    remap = {int(r): k for k, r in enumerate(used)}
    rows = np.array([remap[int(r)] for s in sample for r in row_idx[offs[s]:offs[s + 1]]], np.int32)
    so = np.concatenate([[0], np.cumsum([offs[s + 1] - offs[s] for s in sample])]).astype(np.int32)
    emb_used = wl.to_f64(emb[torch.as_tensor(used, device=emb.device)])
    p64 = {k: wl.to_f64(v) for k, v in params.items()}
    if len(sample) > 64:
        ref = orc.merge_spans_rows(emb_used, rows, so, p64, h)
    else:
        st, ref = orc.merge_spans(emb_used, rows, so, p64, h)
        assert st == orc.OK
    e = rel_l2_max(out[torch.as_tensor(sample, device=out.device)].float().cpu().numpy(), ref)
    say("merge rel_l2_max over", len(sample), "spans:", e)
    assert e <= tol


def _gpu_merge(emb, row_idx, offs, params, h, dtype):
    S = len(offs) - 1
    d = emb.shape[1]
    out = torch.empty((S, d), dtype=dtype, device=dev())
    ws = torch.empty(sm.merge_workspace_bytes(len(row_idx), S, d, dtype), dtype=torch.uint8, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.merge_spans(emb, i32(row_idx), i32(offs), params, h, out, ws, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    return out


class Lockstep:
    """A GPU paged cache and its oracle twin driven by the same calls."""

    def __init__(self, orc, w, num_blocks, max_blocks, free_order=None):
        self.orc, self.w = orc, w
        self.oc = orc.OracleCache(bf16=w.dtype == "bf16", num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
                                  block_size=w.block_size, num_blocks=num_blocks, max_seqs=w.batch,
                                  max_blocks_per_seq=max_blocks, free_order=free_order)
        self.c = gpu_cache_like(self.oc, w.torch_dtype)
        self.ws = None

    def append(self, ids, offs, K, V):
        st = self.oc.append(ids, offs, wl.to_raw(K), wl.to_raw(V))
        assert st == self.orc.OK
        sm.kv_append(self.c, i32(ids), i32(offs), K.to(dev()), V.to(dev()))

    def rollback(self, ids, k):
        assert self.oc.rollback(ids, k) == self.orc.OK
        sm.kv_rollback(self.c, i32(ids), i32(k))

    def check_state(self, pools=True):
        torch.cuda.synchronize()
        assert self.c.error_bits() == 0
        assert_same_state(self.c, self.oc, pools=pools)

    def step(self, K, V, q, max_len, sample, crop=None):
        """One fused decode step on the GPU (sm_decode_step: append a row per
        sequence, attend; with `crop`, sm_decode_merge_step: first drop
        crop[i] entries); the oracle appends (crop_append), and attends for
        the sampled sequences (every query head of each)."""
        w = self.w
        n = w.batch
        if self.ws is None:
            self.ws = torch.zeros(sm.decode_workspace_bytes(n, w.num_q_heads, w.head_dim, max_len),
                                  dtype=torch.uint8, device=dev())
        out = torch.empty((n, w.num_q_heads, w.head_dim), dtype=w.torch_dtype, device=dev())
        if crop is None:
            sm.decode_step(self.c, i32(np.arange(n)), K.to(dev()), V.to(dev()), q.to(dev()), out, self.ws, max_len)
            assert self.oc.append(np.arange(n), np.arange(n + 1), wl.to_raw(K), wl.to_raw(V)) == self.orc.OK
        else:
            sm.decode_merge_step(self.c, i32(np.arange(n)), i32(crop), K.to(dev()), V.to(dev()), q.to(dev()), out,
                                 self.ws, max_len)
            assert self.oc.crop_append(np.arange(n), np.asarray(crop, np.int32), wl.to_raw(K),
                                       wl.to_raw(V)) == self.orc.OK
        torch.cuda.synchronize()
        assert self.c.error_bits() == 0
        if len(sample):
            st, ref = self.oc.decode_attention(sample, wl.to_f64(q[torch.as_tensor(sample)]), w.num_q_heads,
                                               w.head_dim ** -0.5)
            assert st == self.orc.OK
            e = rel_l2_max(out[torch.as_tensor(sample, device=dev())].float().cpu().numpy(), ref)
            assert e <= TOL[w.torch_dtype], e
            return e
        return 0.0

    def attention(self, q, max_len, sample):
        w = self.w
        n = w.batch
        if self.ws is None:
            self.ws = torch.zeros(sm.decode_workspace_bytes(n, w.num_q_heads, w.head_dim, max_len),
                                  dtype=torch.uint8, device=dev())
        out = torch.empty((n, w.num_q_heads, w.head_dim), dtype=w.torch_dtype, device=dev())
        sm.decode_attention(self.c, i32(np.arange(n)), q.to(dev()), out, self.ws, max_len)
        torch.cuda.synchronize()
        assert self.c.error_bits() == 0
        st, ref = self.oc.decode_attention(sample, wl.to_f64(q[torch.as_tensor(sample)]), w.num_q_heads,
                                           w.head_dim ** -0.5)
        assert st == self.orc.OK
        e = rel_l2_max(out[torch.as_tensor(sample, device=dev())].float().cpu().numpy(), ref)
        say("attention rel_l2_max over", len(sample), "sequences:", e)
        assert e <= TOL[w.torch_dtype]


def _prompt_phase(orc, w, ls, P, emb, params, g, merge_sample):
    """Merge every prompt span (GPU; oracle on a sample), pack (indices
    bit-exact), append the compressed prompts' K/V on both sides."""
    out = _gpu_merge(emb, P.row_idx, P.span_offsets, params, w.h, w.torch_dtype)
    _merge_check(orc, emb, params, w.h, P.row_idx, P.span_offsets, out, merge_sample, TOL[w.torch_dtype])
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    assert st == orc.OK
    total = int(P.seq_offsets[-1])
    pi = torch.empty(total, dtype=torch.int32, device=dev())
    po = torch.empty(w.batch + 1, dtype=torch.int32, device=dev())
    ps = torch.empty(total, dtype=torch.int32, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.pack_spans(i32(P.seq_offsets), i32(P.span_start), i32(P.span_len), i32(P.seq_span_offsets),
                  pi, po, ps, err, total)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    np.testing.assert_array_equal(pi.cpu().numpy(), res["pi"])
    np.testing.assert_array_equal(po.cpu().numpy(), res["packed_offsets"])
    rows = int(res["packed_offsets"][-1])
    np.testing.assert_array_equal(ps.cpu().numpy()[:rows], res["packed_src"])
    say("prompt rows after compression", rows, "of", total)
    K = wl.randn((rows, w.num_kv_heads, w.head_dim), w.torch_dtype, g)
    V = wl.randn((rows, w.num_kv_heads, w.head_dim), w.torch_dtype, g)
    ls.append(np.arange(w.batch), res["packed_offsets"], K, V)
    ls.check_state()
    return res


def _decode_phase(orc, w, ls, emb, params, g, steps, max_len, attn_sample, check_every, merge_sample_size):
    rng = np.random.RandomState(w.seed + 21)
    B, H, D = w.batch, w.num_kv_heads, w.head_dim
    for s in range(steps):
        merging = w.merge_every and s % w.merge_every == w.merge_every - 1
        if merging:
            n = wl.decode_merge_lengths(w, s)
            offs = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
            row_idx = rng.randint(0, w.vocab, size=int(offs[-1])).astype(np.int32)
            z = _gpu_merge(emb, row_idx, offs, params, w.h, w.torch_dtype)
            sample = np.arange(B) if B <= merge_sample_size else np.sort(rng.choice(B, merge_sample_size, replace=False))
            _merge_check(orc, emb, params, w.h, row_idx, offs, z, sample, TOL[w.torch_dtype])
            say("step", s, "decode-time merge, rollback", (n - 1).tolist()[:8], "...")
            ls.rollback(np.arange(B), n - 1)
        K = wl.randn((B, H, D), w.torch_dtype, g)
        V = wl.randn((B, H, D), w.torch_dtype, g)
        ls.append(np.arange(B), np.arange(B + 1), K, V)
        ls.check_state(pools=(s % check_every == check_every - 1) or s == steps - 1)
        q = wl.randn((B, w.num_q_heads, D), w.torch_dtype, g)
        if merging or s == 0 or s == steps - 1:
            ls.attention(q, max_len, attn_sample)


def test_tiny_f32_workload_full_chain(orc):
    """The tiny fp32 workload (1 x 512 tokens, d = 256): every output compared.  Prompt compression, the prompt K/V
    from the test-only layer at compressed positions, then one decode-time
    merge (crop n-1, append the surrogate's K/V at its compressed position,
    attend with the surrogate's query) and one ordinary decode step."""
    w = wl.WORKLOADS[1]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed)
    emb = wl.randn((w.vocab, w.d), torch.float32, g, std=0.02).to(dev())
    params = {k: v.to(dev()) for k, v in wl.make_merge_params(w.d, w.h, torch.float32, g).items()}
    say("tiny fp32 workload: spans", len(P.span_len))
    z = _gpu_merge(emb, P.row_idx, P.span_offsets, params, w.h, torch.float32)
    _merge_check(orc, emb, params, w.h, P.row_idx, P.span_offsets, z, np.arange(len(P.span_len)), 1e-5)
    # oracle surrogates feed the test-only layer on both sides
    st, zref = orc.merge_spans(wl.to_f64(emb), P.row_idx, P.span_offsets,
                               {k: wl.to_f64(v) for k, v in params.items()}, w.h)
    z32 = zref.astype(np.float32)
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets,
                             token_ids=P.token_ids, emb_raw=wl.to_raw(emb), surrogates_raw=z32)
    assert st == orc.OK
    total = int(P.seq_offsets[-1])
    pi = torch.empty(total, dtype=torch.int32, device=dev())
    po = torch.empty(2, dtype=torch.int32, device=dev())
    ps = torch.empty(total, dtype=torch.int32, device=dev())
    packed = torch.empty((total, w.d), dtype=torch.float32, device=dev())
    err = torch.zeros(1, dtype=torch.int32, device=dev())
    sm.pack_spans(i32(P.seq_offsets), i32(P.span_start), i32(P.span_len), i32(P.seq_span_offsets), pi, po, ps,
                  err, total, token_ids=i32(P.token_ids), emb=emb, surrogates=torch.from_numpy(z32).to(dev()),
                  packed=packed)
    torch.cuda.synchronize()
    rows = int(res["packed_offsets"][-1])
    assert int(err.item()) == 0 and int(po[-1].item()) == rows
    assert np.array_equal(packed[:rows].cpu().numpy(), res["packed"])
    # prompt K/V from the test-only layer at compressed positions 0..rows-1
    rng = np.random.RandomState(3)
    Wq, Wk, Wv = (rng.normal(0, 0.5 / np.sqrt(w.d), size=(o, w.d))
                  for o in (w.num_q_heads * w.head_dim, w.num_kv_heads * w.head_dim, w.num_kv_heads * w.head_dim))
    q, k, v = orc.layer_qkv(res["packed"].astype(np.float64), np.arange(rows), Wq, Wk, Wv,
                            w.num_q_heads, w.num_kv_heads, w.head_dim)
    ls = Lockstep(orc, w, num_blocks=4, max_blocks=2)
    ls.append([0], [0, rows], torch.from_numpy(k.astype(np.float32)), torch.from_numpy(v.astype(np.float32)))
    ls.check_state()
    # generated tokens: n-1 ordinary steps, then the n-th completes a span
    n = int(np.random.RandomState(w.seed).choice([2, 3, 4]))
    toks = np.random.RandomState(w.seed + 1).randint(0, w.vocab, size=n + 1).astype(np.int32)
    pos = rows
    gen_x = wl.to_f64(emb[torch.as_tensor(toks, device=dev())])
    for j in range(n - 1):
        qj, kj, vj = orc.layer_qkv(gen_x[j:j + 1], [pos], Wq, Wk, Wv, w.num_q_heads, w.num_kv_heads, w.head_dim)
        ls.append([0], [0, 1], torch.from_numpy(kj.astype(np.float32)), torch.from_numpy(vj.astype(np.float32)))
        pos += 1
        ls.attention(torch.from_numpy(qj.astype(np.float32)), 1024, [0])
    # the span: merge its n tokens, roll back the n-1 cached ones, append the surrogate
    zs = _gpu_merge(emb, toks[:n], np.array([0, n], np.int32), params, w.h, torch.float32)
    st, zr = orc.merge_spans(wl.to_f64(emb), toks[:n], np.array([0, n], np.int32),
                             {kk: wl.to_f64(vv) for kk, vv in params.items()}, w.h)
    assert rel_l2_max(zs.cpu().numpy(), zr) <= 1e-5
    ls.rollback([0], [n - 1])
    pos = int(ls.oc.lengths[0])
    assert pos == rows  # L_C' = L_C - (n - 1) + 1 once the surrogate is appended
    qz, kz, vz = orc.layer_qkv(zr, [pos], Wq, Wk, Wv, w.num_q_heads, w.num_kv_heads, w.head_dim)
    ls.append([0], [0, 1], torch.from_numpy(kz.astype(np.float32)), torch.from_numpy(vz.astype(np.float32)))
    ls.check_state()
    ls.attention(torch.from_numpy(qz.astype(np.float32)), 1024, [0])
    # one ordinary decode step after the merge
    qn, kn, vn = orc.layer_qkv(gen_x[n:n + 1], [pos + 1], Wq, Wk, Wv, w.num_q_heads, w.num_kv_heads, w.head_dim)
    ls.append([0], [0, 1], torch.from_numpy(kn.astype(np.float32)), torch.from_numpy(vn.astype(np.float32)))
    ls.check_state()
    ls.attention(torch.from_numpy(qn.astype(np.float32)), 1024, [0])


def _full_decode(orc, w, ls, emb, params, g, steps, max_len, pool_every, seqs_per_step):
    """The workload's whole decode run with the fused steps (the merge
    steps crop, append and attend in one sm_decode_merge_step): every
    decode-time merge's spans all checked, integer state after every step,
    pools every `pool_every` steps, attention of every sequence at the first
    step, every merge step and the last step, and of `seqs_per_step`
    sampled sequences (every query head) at the others."""
    rng = np.random.RandomState(w.seed + 31)
    B, H, D = w.batch, w.num_kv_heads, w.head_dim
    everyone = np.arange(B)
    worst = 0.0
    for s in range(steps):
        merging = bool(w.merge_every) and s % w.merge_every == w.merge_every - 1
        if merging:
            n = wl.decode_merge_lengths(w, s)
            offs = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
            row_idx = rng.randint(0, w.vocab, size=int(offs[-1])).astype(np.int32)
            z = _gpu_merge(emb, row_idx, offs, params, w.h, w.torch_dtype)
            _merge_check(orc, emb, params, w.h, row_idx, offs, z, everyone, TOL[w.torch_dtype])
        K = wl.randn((B, H, D), w.torch_dtype, g)
        V = wl.randn((B, H, D), w.torch_dtype, g)
        q = wl.randn((B, w.num_q_heads, D), w.torch_dtype, g)
        full = merging or s == 0 or s == steps - 1
        sample = everyone if full else np.sort(rng.choice(B, seqs_per_step, replace=False))
        # a merge step crops the span's n - 1 entries in the step's own launch
        worst = max(worst, ls.step(K, V, q, max_len, sample, crop=(n - 1) if merging else None))
        ls.check_state(pools=(s % pool_every == pool_every - 1) or s == steps - 1)
        if s % 32 == 31 or s == steps - 1:
            say("step", s, "lengths", ls.oc.lengths[:4].tolist(), "worst attention rel_l2 so far", worst)


def test_llama3_8b_batch_prompt_compression_and_separate_decode_calls(orc):
    """The Llama-3-8B-shaped batch (16 x 4096-token prompts) at full size: all spans merged in one call (oracle on a
    sample), pack and bulk append bit-exact, then 9 decode steps through the
    separate append and attention calls, a decode-time merge at step 7.
    (The benchmark's own job, with the fused step for all 256 steps, is
    tests/test_gpu_job.py.)"""
    w = wl.WORKLOADS[2]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed, "cuda")
    emb = wl.randn((w.vocab, w.d), w.torch_dtype, g, device="cuda", std=0.02)
    params = wl.make_merge_params(w.d, w.h, w.torch_dtype, g, device="cuda")
    S = len(P.span_len)
    say(w.name, "spans", S, "rows", len(P.row_idx))
    rng = np.random.RandomState(2)
    merge_sample = np.unique(np.concatenate([[0, S - 1], rng.choice(S, 254, replace=False)]))
    L0 = w.prompt_len - int(round(w.target * w.prompt_len))
    steps = 9
    max_len = L0 + steps
    nb_seq = -(-max_len // w.block_size) + 2
    NB = w.batch * nb_seq
    ls = Lockstep(orc, w, NB, nb_seq, free_order=wl.free_order(NB, w.shuffled_pages, w.seed))
    gk = wl.generator(w.seed + 3)
    _prompt_phase(orc, w, ls, P, emb, params, gk, merge_sample)
    attn_sample = np.sort(rng.choice(w.batch, 4, replace=False))
    _decode_phase(orc, w, ls, emb, params, gk, steps, max_len, attn_sample, check_every=4, merge_sample_size=4)


@pytest.mark.parametrize("wid", [3, 5])
def test_prompt_compression_and_full_decode(orc, wid):
    """The long-context batch (4 x 32,768-token prompts, shuffled pages) and
    the Llama-3-70B-shaped batch (32 x 8192) at full size for their whole runs: every prompt span
    merged in one call (1024 sampled spans plus the first and last checked),
    pack and bulk append bit-exact, then all decode steps (128 with a
    decode-time merge every 8 steps for the long-context batch, 64 for the
    70B-shaped one) with the
    fused step; at least 64 (sequence, head) rows checked per step."""
    w = wl.WORKLOADS[wid]
    P = wl.make_prompts(w)
    g = wl.generator(w.seed, "cuda")
    emb = wl.randn((w.vocab, w.d), w.torch_dtype, g, device="cuda", std=0.02)
    params = wl.make_merge_params(w.d, w.h, w.torch_dtype, g, device="cuda")
    S = len(P.span_len)
    say(w.name, "spans", S, "rows", len(P.row_idx))
    rng = np.random.RandomState(wid)
    merge_sample = np.unique(np.concatenate([[0, S - 1], rng.choice(S, 1024, replace=False)]))
    L0 = w.prompt_len - int(round(w.target * w.prompt_len))
    steps = w.decode_steps
    max_len = L0 + steps
    nb_seq = -(-max_len // w.block_size) + 2
    NB = w.batch * nb_seq
    ls = Lockstep(orc, w, NB, nb_seq, free_order=wl.free_order(NB, w.shuffled_pages, w.seed))
    gk = wl.generator(w.seed + 3)
    _prompt_phase(orc, w, ls, P, emb, params, gk, merge_sample)
    _full_decode(orc, w, ls, emb, params, gk, steps, max_len, pool_every=32 if wid == 3 else 16,
                 seqs_per_step=-(-64 // w.num_q_heads))


def test_qwen2_ragged_contexts_with_frequent_rollback(orc):
    """The Qwen2-7B-shaped ragged batch: 128 sequences with contexts uniform in [512, 4096], all 256
    decode steps with the fused step, a decode-time merge (k ~ U{2,3,4},
    n = k + 1 tokens at d = 3584, all 128 spans checked) and crop every
    4 steps, attention over the ragged cache (3 sequences x 28 heads per
    step, every sequence at merge steps and the first and last)."""
    w = wl.WORKLOADS[4]
    lens = wl.context_lengths(w)
    g = wl.generator(w.seed, "cuda")
    emb = wl.randn((w.vocab, w.d), w.torch_dtype, g, device="cuda", std=0.02)
    params = wl.make_merge_params(w.d, w.h, w.torch_dtype, g, device="cuda")
    steps = w.decode_steps
    max_len = int(lens.max()) + steps
    nb_seq = -(-max_len // w.block_size) + 2
    NB = int(np.sum(-(-(lens + steps) // w.block_size))) + w.batch + 8
    ls = Lockstep(orc, w, NB, nb_seq)
    gk = wl.generator(w.seed + 3)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    say("ragged batch prefill rows", int(offs[-1]))
    K = wl.randn((int(offs[-1]), w.num_kv_heads, w.head_dim), w.torch_dtype, gk)
    V = wl.randn((int(offs[-1]), w.num_kv_heads, w.head_dim), w.torch_dtype, gk)
    ls.append(np.arange(w.batch), offs, K, V)
    ls.check_state()
    del K, V
    _full_decode(orc, w, ls, emb, params, gk, steps, max_len, pool_every=32, seqs_per_step=3)
