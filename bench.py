#!/usr/bin/env python
"""Benchmark of the span-merging inference hot path on one MI355X.

Workload: one Llama-3-8B-shaped attention layer (d = 4096, 32 query / 8 KV
heads, head_dim 128, bf16), batch 16, 4096-token prompts compressed by span
merging (spans of 2-8 tokens, 40% effective-length reduction -> 2458 cached
entries per sequence), then 256 decode steps.  Every 8th decode step each
sequence merges a freshly completed span of n = 2..4 tokens (merge module ->
roll back n-1 entries -> append the surrogate's K/V); the other steps append
the new token's K/V.  The append and the step's decode attention over the
compacted paged cache (16-token pages) are one fused launch
(sm_decode_step).

One benchmark step runs that whole job for R resident batches ("replicas")
of 16 sequences, served round-robin the way a server alternates between
batches; R * (bytes per attention launch) is several times the 256 MB
Infinity Cache, so no attention launch finds its KV in the MALL.  The
batches' decode steps are spread over four streams ("lanes": batch r on
stream r % 4, each with its own workspaces), so that one launch's drain and
combine overlap other launches' streaming.  The merge module's first
stage comes from the token table (built once, at set up); a stream's
batches reach their merge steps together, so their fresh spans go to the
merge module together, 64 spans per call.

Printed: one JSON line with the whole-job decode throughput, the fused
append + decode attention kernel's achieved HBM bandwidth against the 8 TB/s
roofline (its launch duration measured live with HIP events around each
decode step's back-to-back launches in a one-stream pass of the same job;
`roofline.overlapped` gives the rate of the lanes' overlapped launches), and the CPU oracle timed on a bounded sample of the same job.
"""
from __future__ import annotations

import argparse
import ctypes as C
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
METRIC = "decode-attention tokens/s + achieved HBM GB/s over span-compacted KV cache"

# HBM traffic of the fused step kernel from rocprofv3 --pmc FETCH_SIZE and
# WRITE_SIZE runs (see profiles/decode_step_llama3-8b-layer.md): scaled
# measured bytes per launch divided by the algorithmic bytes of the same
# launches.  Valid only for the kernel source it was measured on.
TRAFFIC_RATIO = 1.0156
TRAFFIC_SOURCE_SHA256 = {"decode_attn.hip": "7ebac19459e1d185ca656f1d77649011df215d63ea84b769a15ccf7f6932dd37", "common.hpp": "3a781c03722dbc429c51a46492495ab49231891a56fcc322a70bd2033200c04d"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def decode_bytes(w, lens, fused=True):
    """Algorithmic HBM bytes of one fused step launch ending at lengths
    `lens`: K and V of every entry attended to (the cached ones from the
    pool, the appended one from its input row), the appended rows' stores,
    the queries, the outputs and the block table entries read (fused=False:
    a plain attention launch, no stores)."""
    es = 2 if w.dtype == "bf16" else 4
    lens = np.asarray(lens, np.int64)
    row = w.num_kv_heads * w.head_dim * es
    kv = 2 * int(np.sum(lens)) * row
    new_rows = 2 * len(lens) * row if fused else 0
    qo = 2 * len(lens) * w.num_q_heads * w.head_dim * es
    bt = 4 * int(np.sum(-(-lens // w.block_size)))
    return kv + new_rows + qo + bt


class Job:
    """Device state of R resident batches of one workload."""

    def __init__(self, w, R, dev, seed_base=0, token_table=True, lanes=1):
        import torch
        from paper_2609_27233_amd import lib as sm
        from paper_2609_27233_amd import workload as wl

        self.w, self.R, self.dev = w, R, dev
        self.sm, self.L = sm, sm.load()
        bf = w.torch_dtype
        B, H, D, Hq, bs = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads, w.block_size
        T = w.prompt_len
        g = wl.generator(w.seed + seed_base, dev)
        t0 = time.time()
        self.emb = wl.randn((w.vocab, w.d), bf, g, device=dev, std=0.02)
        self.params = wl.make_merge_params(w.d, w.h, bf, g, device=dev)
        i32 = lambda a: torch.as_tensor(np.asarray(a, np.int32)).to(dev)

        self.prompts = [wl.make_prompts(w, seed=w.seed + 97 * r + seed_base) for r in range(R)]
        self.dev_prompts = []
        for P in self.prompts:
            self.dev_prompts.append(dict(
                row_idx=i32(P.row_idx), span_offsets=i32(P.span_offsets), seq_offsets=i32(P.seq_offsets),
                span_start=i32(P.span_start), span_len=i32(P.span_len),
                seq_span_offsets=i32(P.seq_span_offsets), token_ids=i32(P.token_ids),
                S=len(P.span_len), rows=len(P.row_idx)))
        removed = [int(np.sum(P.span_len - 1)) for P in self.prompts]
        self.packed_rows = [B * T - r for r in removed]
        self.L0 = T - int(round(w.target * T))          # cached entries per sequence after compression
        assert all(pr == B * self.L0 for pr in self.packed_rows)

        steps = w.decode_steps
        self.max_len = self.L0 + steps
        nb_seq = -(-self.max_len // bs) + 2
        self.caches = [sm.PagedCache(dtype=bf, num_kv_heads=H, head_dim=D, block_size=bs,
                                     num_blocks=B * nb_seq, max_seqs=B, max_blocks_per_seq=nb_seq,
                                     device=dev) for _ in range(R)]
        Smax = max(p["S"] for p in self.dev_prompts)
        rows_max = max(p["rows"] for p in self.dev_prompts)
        self.z = torch.empty((Smax, w.d), dtype=bf, device=dev)
        self.merge_ws = torch.empty(sm.merge_workspace_bytes(rows_max, Smax, w.d, bf), dtype=torch.uint8, device=dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.pi = torch.empty(B * T, dtype=torch.int32, device=dev)
        self.po = torch.empty(B + 1, dtype=torch.int32, device=dev)
        self.ps = torch.empty(B * T, dtype=torch.int32, device=dev)
        self.packed = torch.empty((B * T, w.d), dtype=bf, device=dev)
        # prompt K/V (what the frozen backbone would produce for the packed rows)
        self.Kp = wl.randn((self.packed_rows[0], H, D), bf, g, device=dev)
        self.Vp = wl.randn((self.packed_rows[0], H, D), bf, g, device=dev)
        # per-step inputs, cycled
        self.nin = 16
        self.Kt = [wl.randn((B, H, D), bf, g, device=dev) for _ in range(self.nin)]
        self.Vt = [wl.randn((B, H, D), bf, g, device=dev) for _ in range(self.nin)]
        self.q = [wl.randn((B, Hq, D), bf, g, device=dev) for _ in range(self.nin)]
        # batch r's decode steps run on lane (stream) r % lanes; each lane has
        # its own output, decode workspace and decode-time merge buffers, so
        # that the lanes' launches can overlap
        self.lanes = NL = max(1, min(lanes, R))
        self.out = [torch.empty((B, Hq, D), dtype=bf, device=dev) for _ in range(NL)]
        self.dec_ws = [torch.zeros(sm.decode_workspace_bytes(B, Hq, D, self.max_len), dtype=torch.uint8, device=dev)
                       for _ in range(NL)]
        self.ids = i32(np.arange(B))
        self.one_row = i32(np.arange(B + 1))
        self.kreset = torch.empty(B, dtype=torch.int32, device=dev)
        # prompt compression buffers per lane (lane 0's are the ones above),
        # so that every lane compresses its own batches' prompts
        self.cbuf = [dict(z=self.z, merge_ws=self.merge_ws, pi=self.pi, po=self.po, ps=self.ps,
                          packed=self.packed, kreset=self.kreset)]
        for _ in range(1, NL):
            self.cbuf.append(dict(z=torch.empty_like(self.z), merge_ws=torch.empty_like(self.merge_ws),
                                  pi=torch.empty_like(self.pi), po=torch.empty_like(self.po),
                                  ps=torch.empty_like(self.ps), packed=torch.empty_like(self.packed),
                                  kreset=torch.empty_like(self.kreset)))
        # decode-time merges: n per sequence per merge step, spans drawn from
        # a synthetic generated-token stream
        self.merge_steps = [s for s in range(steps) if w.merge_every and s % w.merge_every == w.merge_every - 1]
        rng = np.random.RandomState(w.seed + 5)
        # the resident batches reach a merge step together: the fresh spans
        # of a lane's batches go to the merge module together, 64 spans (4
        # batches of 16) per call (the skinny GEMM's row limit), each batch
        # then rolls back its own cache
        self.merge_group = max(1, 64 // B)
        G = self.merge_group
        self.merge_groups = []
        for lane in range(NL):
            rs = list(range(lane, R, NL))
            self.merge_groups.append([rs[i:i + G] for i in range(0, len(rs), G)])
        self.dmerge = {}
        for s in self.merge_steps:
            n = wl.decode_merge_lengths(w, s)
            offs = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
            rows = int(offs[-1])
            row_idx = rng.randint(0, w.vocab, size=rows)
            goffs = np.concatenate([offs[:-1] + j * rows for j in range(G)] + [[G * rows]]).astype(np.int32)
            self.dmerge[s] = dict(n=n, k=i32(n - 1), rows=rows, g_offs=i32(goffs), g_row_idx=i32(np.tile(row_idx, G)))
        self.zdec = [torch.empty((G * B, w.d), dtype=bf, device=dev) for _ in range(NL)]
        self.dmerge_ws = [torch.empty(sm.merge_workspace_bytes(G * B * max(w.merge_n), G * B, w.d, bf),
                                      dtype=torch.uint8, device=dev) for _ in range(NL)]
        # host-side copy of the length schedule (for the algorithmic bytes)
        self.len_sched = []
        lens = np.full(B, self.L0, np.int64)
        for s in range(steps):
            if s in self.dmerge:
                lens = lens - (self.dmerge[s]["n"] - 1) + 1
            else:
                lens = lens + 1
            self.len_sched.append(lens.copy())
        torch.cuda.synchronize()
        self._prep_ctypes()
        # the merge module's first stage for every vocabulary row, built once
        # (as at model load) when the job uses the token table
        self.table, self.table_ms = None, None
        if token_table:
            self.table = torch.empty_like(self.emb)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            rc = self.L.sm_merge_token_table(self.emb.data_ptr(), self.emb.shape[0], C.byref(self.mp), sm.SM_BF16,
                                             self.table.data_ptr(), self.err.data_ptr(),
                                             torch.cuda.current_stream().cuda_stream)
            e1.record()
            torch.cuda.synchronize()
            if rc or int(self.err.item()):
                raise RuntimeError(f"sm_merge_token_table failed: {rc}")
            self.table_ms = e0.elapsed_time(e1)
        log(f"setup {time.time() - t0:.1f}s: R={R}, spans/batch={Smax}, packed rows/batch={self.packed_rows[0]}, "
            f"L0={self.L0}, max_len={self.max_len}")

    def _prep_ctypes(self):
        sm = self.sm
        w = self.w
        p = self.params
        self.mp = sm.MergeParams(w.d, w.h, 1e-5, *(p[k].data_ptr() for k in
                                 ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")))
        self.descs = [C.byref(c.desc) for c in self.caches]

    def decode_bytes(self, lens, fused=True):
        return decode_bytes(self.w, lens, fused)

    def _merge_call(self, row_idx, rows, offs, S, z, ws, st):
        """M_phi over one CSR batch of spans: from the token table when the
        job has one, else from the embeddings."""
        L, bf = self.L, self.sm.SM_BF16
        if self.table is not None:
            return L.sm_merge_spans_tabled(self.table.data_ptr(), self.table.shape[0], row_idx, rows, offs, S,
                                           C.byref(self.mp), bf, z, ws.data_ptr(), ws.numel(),
                                           self.err.data_ptr(), st)
        return L.sm_merge_spans(self.emb.data_ptr(), self.emb.shape[0], row_idx, rows, offs, S,
                                C.byref(self.mp), bf, z, ws.data_ptr(), ws.numel(), self.err.data_ptr(), st)

    def _merge(self, rs, s, lane, st):
        """Decode-time merge of batches rs (at most merge_group of them, all
        on `lane`) before decode step s: the merge module on every
        sequence's freshly completed span, in one call.  The crop of the
        span's n-1 cached entries happens in the step's own launch."""
        w = self.w
        B = w.batch
        m = self.dmerge[s]
        S = len(rs) * B
        rc = self._merge_call(m["g_row_idx"].data_ptr(), len(rs) * m["rows"], m["g_offs"].data_ptr(), S,
                              self.zdec[lane].data_ptr(), self.dmerge_ws[lane], st)
        if rc:
            raise RuntimeError(f"decode-time merge launch failed at step {s}: {rc}")

    def _step(self, r, s, st):
        """Decode step s of batch r in one launch: append the step's K/V row
        (new token, or at a merge step the surrogate's after cropping the
        span's n-1 entries) and attend."""
        L, w = self.L, self.w
        j = s % self.nin
        lane = r % self.lanes
        ws = self.dec_ws[lane]
        if s in self.dmerge:
            rc = L.sm_decode_merge_step(self.descs[r], self.ids.data_ptr(), self.dmerge[s]["k"].data_ptr(), w.batch,
                                        self.Kt[j].data_ptr(), self.Vt[j].data_ptr(), self.q[j].data_ptr(),
                                        w.num_q_heads, w.head_dim ** -0.5, self.max_len,
                                        self.out[lane].data_ptr(), ws.data_ptr(), ws.numel(), st)
        else:
            rc = L.sm_decode_step(self.descs[r], self.ids.data_ptr(), w.batch, self.Kt[j].data_ptr(),
                                  self.Vt[j].data_ptr(), self.q[j].data_ptr(), w.num_q_heads, w.head_dim ** -0.5,
                                  self.max_len, self.out[lane].data_ptr(), ws.data_ptr(), ws.numel(), st)
        if rc:
            raise RuntimeError(f"decode step launch failed at step {s}: {rc}")

    def run(self, streams, events=None, hook=None):
        """One benchmark step: the whole job for every resident batch.

        Lane l's batches (r % lanes == l) run their prompt compression,
        decode steps and decode-time merges, in order, on
        streams[l % len(streams)]; the lanes share nothing, so their
        launches overlap: one lane's workgroups stream their KV while
        another's launch drains its last tiles and combines, or compresses
        its prompts.  With `events` (one stream only) each step's launches
        are bracketed by events[0][s] and events[1][s].  `hook` (tests
        only) is called after the prompt compression ("prompt", None),
        after each merge step's merges ("merge", s) and after each decode
        step's launches ("step", s); it may synchronize and read state, and
        changes none of the launches."""
        import torch
        L, w = self.L, self.w
        B = w.batch
        R = self.R
        if events is not None and len(streams) != 1:
            raise ValueError("per-step events need a single stream")
        s0 = streams[0]
        lane_st = [streams[l % len(streams)] for l in range(self.lanes)]
        # prompt compression of every batch, on its lane (after its previous
        # job's last decode step)
        for r in range(R):
            dp = self.dev_prompts[r]
            c = self.caches[r]
            lane = r % self.lanes
            cb, st = self.cbuf[lane], lane_st[lane]
            sb = st.cuda_stream
            with torch.cuda.stream(st):
                cb["kreset"].copy_(c.lengths[:B])   # evict the previous job's sequences
            rc = L.sm_kv_rollback(self.descs[r], self.ids.data_ptr(), cb["kreset"].data_ptr(), B, sb)
            rc |= self._merge_call(dp["row_idx"].data_ptr(), dp["rows"], dp["span_offsets"].data_ptr(), dp["S"],
                                   cb["z"].data_ptr(), cb["merge_ws"], sb)
            rc |= L.sm_pack_spans(B, dp["seq_offsets"].data_ptr(), B * w.prompt_len, dp["S"],
                                  dp["span_start"].data_ptr(), dp["span_len"].data_ptr(),
                                  dp["seq_span_offsets"].data_ptr(), cb["pi"].data_ptr(), cb["po"].data_ptr(),
                                  cb["ps"].data_ptr(), dp["token_ids"].data_ptr(), self.emb.data_ptr(),
                                  self.emb.shape[0], cb["z"].data_ptr(), w.d, self.sm.SM_BF16,
                                  cb["packed"].data_ptr(), self.err.data_ptr(), sb)
            rc |= L.sm_kv_append(self.descs[r], self.ids.data_ptr(), cb["po"].data_ptr(), B, self.packed_rows[r],
                                 self.Kp.data_ptr(), self.Vp.data_ptr(), sb)
            if rc:
                raise RuntimeError(f"prompt compression launch failed: {rc}")
        if hook is not None:
            hook("prompt", None)
        for s in range(w.decode_steps):
            if s in self.dmerge:
                for lane, groups in enumerate(self.merge_groups):
                    for rs in groups:
                        self._merge(rs, s, lane, lane_st[lane].cuda_stream)
                if hook is not None:
                    hook("merge", s)
            if events is not None:
                events[0][s].record(s0)
            for r in range(R):
                self._step(r, s, lane_st[r % self.lanes].cuda_stream)
            if events is not None:
                events[1][s].record(s0)
            if hook is not None:
                hook("step", s)

    def check_errors(self):
        bits = [c.error_bits() for c in self.caches] + [int(self.err.item())]
        if any(bits):
            raise RuntimeError(f"device error bits set: {bits}")


def lanes_report(job, streams, rounds):
    """Fused decode steps of every resident batch back to back over the
    job's caches as the job left them, on one stream and then on the job's
    lanes: the rate at which the overlapped launches move the kernel's
    algorithmic bytes.  Each round appends one row per sequence; every pass
    rolls its rows back, so the caches end as the job left them.  Rounds
    are limited by the caches' spare capacity (None if there is none)."""
    import torch
    w, B = job.w, job.w.batch
    spare = job.max_len - max(int(c.lengths[:B].max()) for c in job.caches)
    rounds = min(rounds, spare)
    if rounds < 1:
        return None
    res = {}
    for name, sts in (("one_stream", streams[:1]), ("lanes", streams)):
        lane_st = [sts[l % len(sts)] for l in range(job.lanes)]
        for timed in (False, True):
            lens0 = np.stack([c.lengths[:B].cpu().numpy().astype(np.int64) for c in job.caches])
            n = rounds if timed else 1
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(sts[0])
            for st in sts[1:]:
                st.wait_event(e0)
            for it in range(n):
                for r in range(job.R):
                    job._step(r, it, lane_st[r % job.lanes].cuda_stream)
            for st in sts[1:]:
                sts[0].wait_stream(st)
            e1.record(sts[0])
            torch.cuda.synchronize()
            k = torch.full((B,), n, dtype=torch.int32, device=job.dev)
            for r in range(job.R):
                if job.L.sm_kv_rollback(job.descs[r], job.ids.data_ptr(), k.data_ptr(), B,
                                        sts[0].cuda_stream):
                    raise RuntimeError("roll back after the lanes measurement failed")
            torch.cuda.synchronize()
        nbytes = sum(job.decode_bytes(lens0[r] + it + 1) for it in range(n) for r in range(job.R))
        us = e0.elapsed_time(e1) * 1e3 / (n * job.R)
        res[name] = {"us_per_launch": round(us, 3), "achieved": round(nbytes / (us * 1e-6 * n * job.R) / 1e9, 1)}
        mean_len = float(lens0.mean()) + (n + 1) / 2
    job.check_errors()
    ach = res["lanes"]["achieved"]
    return {"lanes": job.lanes, "us_per_launch": res["lanes"]["us_per_launch"], "achieved": ach,
            "frac": round(ach / PEAK_HBM_GBS, 4), "one_stream_us_per_launch": res["one_stream"]["us_per_launch"],
            "mean_cache_len": round(mean_len, 1),
            "note": "the fused step of every resident batch, %d rounds back to back over the job's caches, batch r "
                    "on stream r %% %d: bytes of all launches over the time from the first start to the last end; "
                    "overlapping launches have no duration of their own" % (rounds, job.lanes)}


def graph_report(job, rounds):
    """The fused step of every resident batch, R launches back to back on one
    stream, captured once as a HIP graph and replayed `rounds` times (each
    replay appends one row per sequence; the rows are rolled back
    afterwards), against the same launches issued eagerly: the time per
    launch including the gaps between launches.  None if the caches have no
    spare capacity."""
    import torch
    w, B = job.w, job.w.batch
    spare = job.max_len - max(int(c.lengths[:B].max()) for c in job.caches)
    rounds = min(rounds, spare // 2)
    if rounds < 1:
        return None
    stream = torch.cuda.Stream()
    res = {}
    with torch.cuda.stream(stream):
        torch.cuda.synchronize()
        lens0 = [c.lengths[:B].clone() for c in job.caches]
        # eager, one stream
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(rounds):
            for r in range(job.R):
                job._step(r, 0, stream.cuda_stream)
        e1.record(stream)
        torch.cuda.synchronize()
        res["eager_us_per_launch"] = round(e0.elapsed_time(e1) * 1e3 / (rounds * job.R), 3)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for r in range(job.R):
                job._step(r, 0, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(rounds - 1):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        res["graph_us_per_launch"] = round(e0.elapsed_time(e1) * 1e3 / ((rounds - 1) * job.R), 3) if rounds > 1 \
            else None
        for r, c in enumerate(job.caches):
            grown = (c.lengths[:B] - lens0[r]).to(torch.int32).contiguous()
            if int(grown.min()) != 2 * rounds - 1 or int(grown.max()) != 2 * rounds - 1:
                raise RuntimeError("graph replays did not append one row per sequence each")
            if job.L.sm_kv_rollback(job.descs[r], job.ids.data_ptr(), grown.data_ptr(), B, stream.cuda_stream):
                raise RuntimeError("roll back after the graph measurement failed")
        torch.cuda.synchronize()
    job.check_errors()
    res["rounds"] = rounds
    res["note"] = ("one decode step of all %d resident batches (R fused launches) on one stream: eager issue "
                   "against one captured HIP graph replayed; HIP events around all rounds" % job.R)
    return res


def _time(fn, stream, reps):
    """Average ms of fn() over reps calls, HIP events on `stream`."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def extras_report(job, stream, attn_us):
    """Side measurements named in the workload description: the same
    attention over the uncompressed cache (control), the merge module at the
    70B-shaped prompt batch (MFMA utilisation), and the cache operations."""
    import torch
    from paper_2609_27233_amd import workload as wl
    sm, L, w, dev = job.sm, job.L, job.w, job.dev
    B, H, D, Hq, bs = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads, w.block_size
    st = stream.cuda_stream
    out = {}
    g = wl.generator(77, dev)
    ids = job.ids

    # --- the attention kernel alone (no append) over the job's caches as the
    # job left them: the plain decode_attention entry point
    descs0 = [C.byref(c.desc) for c in job.caches]
    ws0 = torch.zeros(sm.decode_workspace_bytes(B, Hq, D, job.max_len), dtype=torch.uint8, device=dev)

    def attn_job():
        for d0 in descs0:
            L.sm_decode_attention(d0, ids.data_ptr(), B, job.q[0].data_ptr(), Hq, D ** -0.5, job.max_len,
                                  job.out[0].data_ptr(), ws0.data_ptr(), ws0.numel(), st)
    ms0 = _time(attn_job, stream, 16) / job.R
    lens_end = job.caches[0].lengths[:B].cpu().numpy().astype(np.int64)
    b0 = job.decode_bytes(lens_end, fused=False)
    out["attention_only"] = {
        "kernel": "decode_split_bf16<128> (decode_attention, no append)",
        "mean_cache_len": round(float(lens_end.mean()), 1), "avg_launch_us": round(ms0 * 1e3, 3),
        "achieved_GBps": round(b0 / (ms0 * 1e-3) / 1e9, 1), "frac": round(b0 / (ms0 * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "note": "the plain attention kernel over the same caches at the end of the job; HIP events around "
                "back-to-back launches"}
    del ws0
    log("extras: attention-only done")

    # --- uncompressed control: same launch shape, cache length = prompt + 128
    Lu = w.prompt_len + 128
    nb = -(-Lu // bs) + 1
    caches = []
    Ku = wl.randn((B * Lu, H, D), w.torch_dtype, g, device=dev)
    Vu = wl.randn((B * Lu, H, D), w.torch_dtype, g, device=dev)
    offs = torch.as_tensor(np.arange(B + 1, dtype=np.int32) * Lu).to(dev)
    for r in range(job.R):
        c = sm.PagedCache(dtype=w.torch_dtype, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=B * nb,
                          max_seqs=B, max_blocks_per_seq=nb, device=dev)
        sm.kv_append(c, ids, offs, Ku, Vu, stream=stream)
        caches.append(c)
    del Ku, Vu
    ws = torch.zeros(sm.decode_workspace_bytes(B, Hq, D, Lu), dtype=torch.uint8, device=dev)
    descs = [C.byref(c.desc) for c in caches]

    def attn_all():
        for d in descs:
            L.sm_decode_attention(d, ids.data_ptr(), B, job.q[0].data_ptr(), Hq, D ** -0.5, Lu,
                                  job.out[0].data_ptr(), ws.data_ptr(), ws.numel(), st)
    ms = _time(attn_all, stream, 16) / job.R
    ubytes = job.decode_bytes(np.full(B, Lu), fused=False)
    out["uncompressed_control"] = {
        "cache_len": Lu, "avg_launch_us": round(ms * 1e3, 3),
        "achieved_GBps": round(ubytes / (ms * 1e-3) / 1e9, 1),
        "compacted_avg_launch_us": round(attn_us, 3),
        "speedup_per_step": round(ms * 1e3 / attn_us, 3),
        "note": "per decode step of the same batch: uncompressed cache (prompt 4096 + 128) vs span-compacted "
                "cache (mean over the job's 256 steps)"}
    assert all(c.error_bits() == 0 for c in caches)
    log("extras: uncompressed control done")
    del caches, descs, ws
    torch.cuda.empty_cache()

    out["cache_ops"] = cache_ops_report(job, stream)
    out["configs"] = configs_report(dev, stream, (2, 3, 4, 5))

    out["merge_spans_70b_prompt_batch"] = merge_70b_report(job.sm, job.L, dev, stream)
    out["prefill_attention"] = prefill_report(job.sm, job.L, dev, stream)
    out["rule_matching"] = rules_report(job.sm, job.L, dev, stream)
    out["surrogate_lookup"] = lut_report(job.sm, job.L, dev, stream)
    out["kv_projection"] = kvproj_report(job.sm, job.L, dev, stream)
    return out


def _time_each(fn, undo, stream, reps):
    """Average ms of fn() alone over reps calls, each bracketed by its own
    HIP events on `stream`; undo() (untimed) runs after each call."""
    import torch
    fn()
    undo()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for e0, e1 in evs:
        e0.record(stream)
        fn()
        e1.record(stream)
        undo()
    torch.cuda.synchronize()
    return sum(e0.elapsed_time(e1) for e0, e1 in evs) / reps


def cache_ops_report(job, stream):
    """The cache operations of one batch, as separate calls on a fresh cache
    of the job's shape: the bulk append of a compressed prompt batch, pack,
    the per-step append, rollback and a decode-time merge update."""
    import torch
    sm, L, w, dev = job.sm, job.L, job.w, job.dev
    B, H, D, bs = w.batch, w.num_kv_heads, w.head_dim, w.block_size
    st = stream.cuda_stream
    ids = job.ids
    c = sm.PagedCache(dtype=w.torch_dtype, num_kv_heads=H, head_dim=D, block_size=bs,
                      num_blocks=job.caches[0].num_blocks, max_seqs=B,
                      max_blocks_per_seq=job.caches[0].max_blocks, device=dev)
    d = C.byref(c.desc)
    rows = job.packed_rows[0]
    kfull = torch.full((B,), job.L0, dtype=torch.int32, device=dev)
    # packed offsets of batch 0 for the bulk append
    po = np.concatenate([[0], np.cumsum(np.full(B, job.L0))]).astype(np.int32)
    job.po.copy_(torch.as_tensor(po))

    def bulk():
        L.sm_kv_append(d, ids.data_ptr(), job.po.data_ptr(), B, rows, job.Kp.data_ptr(), job.Vp.data_ptr(), st)

    def roll_all():
        L.sm_kv_rollback(d, ids.data_ptr(), kfull.data_ptr(), B, st)
    t_bulk = _time_each(bulk, roll_all, stream, 10)
    t_bulk_roll = _time(lambda: (bulk(), roll_all()), stream, 5)
    bulk()

    def step_append():
        L.sm_kv_append(d, ids.data_ptr(), job.one_row.data_ptr(), B, B, job.Kt[0].data_ptr(),
                       job.Vt[0].data_ptr(), st)
    t_app = _time(step_append, stream, 100)          # 101 appends: L0 + 101 entries per sequence
    k1 = torch.ones(B, dtype=torch.int32, device=dev)
    k3 = torch.full((B,), 3, dtype=torch.int32, device=dev)
    t_roll = _time(lambda: L.sm_kv_rollback(d, ids.data_ptr(), k1.data_ptr(), B, st), stream, 40)

    def merge_update():                              # one decode-time merge of n = 4: crop 3, append 1
        L.sm_kv_rollback(d, ids.data_ptr(), k3.data_ptr(), B, st)
        L.sm_kv_append(d, ids.data_ptr(), job.one_row.data_ptr(), B, B, job.Kt[1].data_ptr(),
                       job.Vt[1].data_ptr(), st)
    t_mu = _time(merge_update, stream, 20)
    dp = job.dev_prompts[0]

    def pack():
        L.sm_pack_spans(B, dp["seq_offsets"].data_ptr(), B * w.prompt_len, dp["S"], dp["span_start"].data_ptr(),
                        dp["span_len"].data_ptr(), dp["seq_span_offsets"].data_ptr(), job.pi.data_ptr(),
                        job.po.data_ptr(), job.ps.data_ptr(), dp["token_ids"].data_ptr(), job.emb.data_ptr(),
                        job.emb.shape[0], job.z.data_ptr(), w.d, sm.SM_BF16, job.packed.data_ptr(),
                        job.err.data_ptr(), st)
    t_pack = _time(pack, stream, 10)
    assert c.error_bits() == 0 and int(job.err.item()) == 0
    row_bytes = H * D * 2
    append_bytes = 4 * rows * row_bytes                 # read and write of K and V
    pack_bytes = 2 * rows * w.d * 2 + 8 * B * w.prompt_len
    del c
    torch.cuda.empty_cache()
    log("cache operations done")
    return {
        "bulk_append_rows": rows,
        "bulk_append_us": round(t_bulk * 1e3, 2),
        "bulk_append_GBps": round(append_bytes / (t_bulk * 1e-3) / 1e9, 1),
        "bulk_append_frac": round(append_bytes / (t_bulk * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "bulk_append_plus_full_rollback_ms": round(t_bulk_roll, 4),
        "decode_append_16_rows_us": round(t_app * 1e3, 2),
        "rollback_16_seqs_k1_us": round(t_roll * 1e3, 2),
        "merge_update_16_seqs_us": round(t_mu * 1e3, 2),
        "pack_prompt_batch_us": round(t_pack * 1e3, 1),
        "pack_GBps": round(pack_bytes / (t_pack * 1e-3) / 1e9, 1),
        "pack_frac": round(pack_bytes / (t_pack * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "note": "bulk append: HIP events around each call (metadata + copy launches), a full rollback between "
                "calls; the rest: events around back-to-back calls on one stream; merge update = roll back 3 "
                "entries and append the surrogate's K/V for each of 16 sequences; bytes: append reads and "
                "writes K and V, pack reads and writes the packed rows plus 8 B of indices per token"}


# resident replicas per configuration: R x (bytes per attention launch) is
# at least 1 GiB, so no launch finds its cache in the 256 MB MALL
CONFIG_REPLICAS = {2: 8, 3: 4, 4: 2, 5: 2}


def config_start_lengths(w):
    """Cached entries per sequence when decoding starts: the compressed
    prompt length, or the seeded ragged contexts."""
    if w.ctx_range is not None:
        return wl_mod().context_lengths(w).astype(np.int64)
    return np.full(w.batch, w.prompt_len - int(round(w.target * w.prompt_len)), np.int64)


def wl_mod():
    from paper_2609_27233_amd import workload as wl
    return wl


def config_decode_report(cid, dev, stream, reps=3, merge_every=None):
    """Decode attention of one configuration at its full size: R resident
    replicas of the batch's paged cache at the configuration's starting
    lengths (random K/V; values do not change the traffic), then the
    configuration's decode steps, each one fused append + attention launch
    per replica (sm_decode_step), with the configuration's decode-time
    rollback of k entries before every merge step (the appended row is
    then the surrogate's).  Timed on one stream: tokens/s of the loop, and
    the step kernel's launch duration from HIP events around each step's R
    back-to-back launches."""
    import dataclasses
    import torch
    from paper_2609_27233_amd import lib as sm
    wl = wl_mod()
    L = sm.load()
    w = wl.WORKLOADS[cid]
    if merge_every is not None:
        w = dataclasses.replace(w, merge_every=merge_every)
    B, H, D, Hq, bs = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads, w.block_size
    dt = w.torch_dtype
    R = CONFIG_REPLICAS[cid]
    S = w.decode_steps
    st = stream.cuda_stream
    lens0 = config_start_lengths(w)
    # host copy of the length schedule: k per merge step, lengths after each step
    ks, sched = {}, []
    lens = lens0.copy()
    for s_ in range(S):
        if w.merge_every and s_ % w.merge_every == w.merge_every - 1:
            k = (wl.decode_merge_lengths(w, s_) - 1).astype(np.int64)
            ks[s_] = k
            lens = lens - k
        lens = lens + 1
        sched.append(lens.copy())
    max_len = int(max(x.max() for x in sched))
    peak = np.max(np.stack([lens0] + sched), axis=0)
    nb_seq = -(-max_len // bs) + 1
    NB = int(np.sum(-(-peak // bs))) + B
    g = wl.generator(w.seed + 500, dev)
    offs = torch.as_tensor(np.concatenate([[0], np.cumsum(lens0)]).astype(np.int32)).to(dev)
    rows = int(lens0.sum())
    K0 = wl.randn((rows, H, D), dt, g, device=dev)
    V0 = wl.randn((rows, H, D), dt, g, device=dev)
    ids = torch.arange(B, dtype=torch.int32, device=dev)
    caches = []
    for r in range(R):
        c = sm.PagedCache(dtype=dt, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=NB, max_seqs=B,
                          max_blocks_per_seq=nb_seq, device=dev,
                          free_order=wl.free_order(NB, w.shuffled_pages, w.seed + r))
        sm.kv_append(c, ids, offs, K0, V0, stream=stream)
        caches.append(c)
    del K0, V0
    nin = 8
    Kt = [wl.randn((B, H, D), dt, g, device=dev) for _ in range(nin)]
    Vt = [wl.randn((B, H, D), dt, g, device=dev) for _ in range(nin)]
    q = [wl.randn((B, Hq, D), dt, g, device=dev) for _ in range(nin)]
    out = torch.empty((B, Hq, D), dtype=dt, device=dev)
    ws = torch.zeros(sm.decode_workspace_bytes(B, Hq, D, max_len), dtype=torch.uint8, device=dev)
    kdev = {s_: torch.as_tensor(k.astype(np.int32)).to(dev) for s_, k in ks.items()}
    restore = torch.as_tensor((sched[-1] - lens0).astype(np.int32)).to(dev)
    descs = [C.byref(c.desc) for c in caches]
    scale = D ** -0.5
    torch.cuda.synchronize()

    def loop(ev=None):
        for s_ in range(S):
            j = s_ % nin
            if ev is not None:
                ev[0][s_].record(stream)
            for d in descs:
                if s_ in kdev:  # crop the span's n - 1 entries, append the surrogate's row, attend
                    rc = L.sm_decode_merge_step(d, ids.data_ptr(), kdev[s_].data_ptr(), B, Kt[j].data_ptr(),
                                                Vt[j].data_ptr(), q[j].data_ptr(), Hq, scale, max_len,
                                                out.data_ptr(), ws.data_ptr(), ws.numel(), st)
                else:
                    rc = L.sm_decode_step(d, ids.data_ptr(), B, Kt[j].data_ptr(), Vt[j].data_ptr(), q[j].data_ptr(),
                                          Hq, scale, max_len, out.data_ptr(), ws.data_ptr(), ws.numel(), st)
                if rc:
                    raise RuntimeError(f"decode step failed at config {cid} step {s_}: {rc}")
            if ev is not None:
                ev[1][s_].record(stream)

    def undo():
        for d in descs:
            L.sm_kv_rollback(d, ids.data_ptr(), restore.data_ptr(), B, st)

    loop()
    undo()
    torch.cuda.synchronize()
    elapsed, kern, per_merge, per_plain = [], [], [], []
    for _ in range(reps):
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(S)] for _ in range(2)]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        loop(ev)
        e1.record(stream)
        undo()
        torch.cuda.synchronize()
        elapsed.append(e0.elapsed_time(e1))
        per = [a.elapsed_time(b) for a, b in zip(ev[0], ev[1])]
        kern.append(sum(per))
        per_merge.append(sum(per[x] for x in kdev) / max(1, len(kdev)))
        per_plain.append(sum(per[x] for x in range(S) if x not in kdev) / max(1, S - len(kdev)))
    bad = [c.error_bits() for c in caches]
    if any(bad):
        raise RuntimeError(f"config {cid}: device error bits {bad}")
    step_bytes = [decode_bytes(w, x) for x in sched]
    t_loop = min(elapsed) * 1e-3
    t_kern = min(kern) * 1e-3
    launch_us = t_kern / (S * R) * 1e6
    gbps = sum(step_bytes) * R / t_kern / 1e9
    res = {
        "workload": w.name, "batch": B, "q_heads": Hq, "kv_heads": H, "head_dim": D,
        "start_len_mean": round(float(lens0.mean()), 1), "start_len_min": int(lens0.min()),
        "start_len_max": int(lens0.max()), "end_len_mean": round(float(sched[-1].mean()), 1),
        "decode_steps": S, "merge_every": w.merge_every, "replicas": R, "shuffled_pages": w.shuffled_pages,
        "tokens_per_s": round(B * S * R / t_loop, 1),
        "avg_launch_us": round(launch_us, 3),
        "algorithmic_MB_per_launch": round(sum(step_bytes) / S / 1e6, 2),
        "achieved_GBps": round(gbps, 1), "frac": round(gbps / PEAK_HBM_GBS, 4),
        "merge_step_launch_us": round(min(per_merge) * 1e3 / R, 3) if kdev else None,
        "plain_step_launch_us": round(min(per_plain) * 1e3 / R, 3),
        "note": "one stream; tokens/s = B x steps x replicas over the loop's time (best of %d); a merge step is "
                "one sm_decode_merge_step launch per replica (crop n-1, append, attend), the others "
                "sm_decode_step; launch time from HIP events around each step's back-to-back launches" % reps}
    del caches, ws
    torch.cuda.empty_cache()
    log(f"config {cid}: {res['avg_launch_us']} us per launch, {res['achieved_GBps']} GB/s")
    return res


def configs_report(dev, stream, cids=(3, 4, 5)):
    out = {}
    for cid in cids:
        if cid == 2:
            out["2_without_decode_merges"] = config_decode_report(2, dev, stream, merge_every=0)
        else:
            out[str(cid)] = config_decode_report(cid, dev, stream)
    return out


def merge_70b_report(sm, L, dev, stream, reps=3):
    """The merge module over every span of the 32 x 8192 Llama-3-70B-shaped
    prompt batch in one call: time and MFMA utilisation."""
    import torch
    from paper_2609_27233_amd import workload as wl
    st = stream.cuda_stream
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    w5 = wl.WORKLOADS[5]
    P5 = wl.make_prompts(w5)
    g5 = wl.generator(w5.seed, dev)
    emb5 = wl.randn((w5.vocab, w5.d), torch.bfloat16, g5, device=dev, std=0.02)
    par5 = wl.make_merge_params(w5.d, w5.h, torch.bfloat16, g5, device=dev)
    S5, R5 = len(P5.span_len), len(P5.row_idx)
    i32 = lambda a: torch.as_tensor(np.asarray(a, np.int32)).to(dev)
    ri, so = i32(P5.row_idx), i32(P5.span_offsets)
    z5 = torch.empty((S5, w5.d), dtype=torch.bfloat16, device=dev)
    ws5 = torch.empty(sm.merge_workspace_bytes(R5, S5, w5.d, torch.bfloat16), dtype=torch.uint8, device=dev)
    mp5 = sm.MergeParams(w5.d, w5.h, 1e-5, *(par5[k].data_ptr() for k in
                         ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")))

    def merge5():
        rc = L.sm_merge_spans(emb5.data_ptr(), emb5.shape[0], ri.data_ptr(), R5, so.data_ptr(), S5, C.byref(mp5),
                              sm.SM_BF16, z5.data_ptr(), ws5.data_ptr(), ws5.numel(), err.data_ptr(), st)
        if rc:
            raise RuntimeError(f"sm_merge_spans failed: {rc}")
    torch.cuda.synchronize()
    log(f"extras: merge module inputs ready ({S5} spans, {R5} rows)")
    t5 = _time(merge5, stream, reps)
    flop5 = 2.0 * w5.d * w5.d * (R5 + S5)
    assert int(err.item()) == 0
    # the same surrogates from the token table: the table (vocab x d) is one
    # GEMM, built once; each call then runs the span-level stages only
    z5t = torch.empty_like(z5)
    table5 = torch.empty_like(emb5)

    def table_build():
        rc = L.sm_merge_token_table(emb5.data_ptr(), emb5.shape[0], C.byref(mp5), sm.SM_BF16, table5.data_ptr(),
                                    err.data_ptr(), st)
        if rc:
            raise RuntimeError(f"sm_merge_token_table failed: {rc}")

    def merge5t():
        rc = L.sm_merge_spans_tabled(table5.data_ptr(), table5.shape[0], ri.data_ptr(), R5, so.data_ptr(), S5,
                                     C.byref(mp5), sm.SM_BF16, z5t.data_ptr(), ws5.data_ptr(), ws5.numel(),
                                     err.data_ptr(), st)
        if rc:
            raise RuntimeError(f"sm_merge_spans_tabled failed: {rc}")
    tb = _time(table_build, stream, 2)
    tt = _time(merge5t, stream, reps)
    assert int(err.item()) == 0
    flop_tb = 2.0 * w5.d * w5.d * emb5.shape[0]
    flop_t = 2.0 * w5.d * w5.d * S5
    agree = float((z5t.float() - z5.float()).norm(dim=1).div(z5.float().norm(dim=1)).max())
    del table5
    # context, not part of the path: the library GEMM (torch.nn.functional.linear,
    # hipBLASLt on ROCm) on the first projection's plain product over the
    # same rows, gathered beforehand (no gather, bias or GELU in the timed call)
    with torch.cuda.stream(stream):
        ag = emb5.index_select(0, ri.long())
        w_kv = par5["W_kv"]
        t_lib = _time(lambda: torch.nn.functional.linear(ag, w_kv), stream, reps)
    del ag
    flop_lib = 2.0 * w5.d * w5.d * R5
    return {
        "spans": S5, "rows": R5, "d": w5.d, "ms": round(t5, 3),
        "TFLOPs": round(flop5 / (t5 * 1e-3) / 1e12, 1),
        "frac_of_bf16_peak": round(flop5 / (t5 * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "token_table": {
            "build_ms": round(tb, 3), "build_TFLOPs": round(flop_tb / (tb * 1e-3) / 1e12, 1),
            "table_GB": round(emb5.numel() * 2 / 1e9, 2),
            "tabled_merge_ms": round(tt, 3), "tabled_speedup": round(t5 / tt, 2),
            "tabled_TFLOPs_second_projection": round(flop_t / (tt * 1e-3) / 1e12, 1),
            "max_rel_l2_vs_direct": round(agree, 5),
            "note": "sm_merge_token_table over the 128256-row vocabulary, once; sm_merge_spans_tabled over the "
                    "same spans reads the first stage by token id"},
        "library_gemm_reference": {
            "ms": round(t_lib, 3), "TFLOPs": round(flop_lib / (t_lib * 1e-3) / 1e12, 1),
            "note": "context only: torch.nn.functional.linear (hipBLASLt) on the first projection's plain product, rows gathered "
                    "beforehand, no bias or GELU"},
        "note": "one sm_merge_spans call over every span of the 32 x 8192 prompts; FLOP = 2 d^2 (rows + spans) "
                "for the two projections (pooling and LayerNorm are O(d) per row)"}


def prefill_report(sm, L, dev, stream, reps=10):
    """Prefill attention (one layer, all 32 query heads) over the 16-prompt
    batch: the span-compacted prompts (2458 positions) against the same
    batch uncompressed (4096).  FLOP = 4 Hq D sum over rows of (position + 1)
    for the two causal products."""
    import torch
    from paper_2609_27233_amd import workload as wl
    w = wl.WORKLOADS[2]
    B, H, D, Hq, bs = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads, w.block_size
    st = stream.cuda_stream
    g = wl.generator(91, dev)
    res = {}
    for name, Lp in (("compacted", w.prompt_len - int(round(w.target * w.prompt_len))), ("uncompressed", w.prompt_len)):
        nb = -(-Lp // bs)
        c = sm.PagedCache(dtype=torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=bs, num_blocks=B * nb,
                          max_seqs=B, max_blocks_per_seq=nb, device=dev)
        offs = torch.arange(B + 1, dtype=torch.int32, device=dev) * Lp
        ids = torch.arange(B, dtype=torch.int32, device=dev)
        K = wl.randn((B * Lp, H, D), torch.bfloat16, g, device=dev)
        V = wl.randn((B * Lp, H, D), torch.bfloat16, g, device=dev)
        sm.kv_append(c, ids, offs, K, V, stream=stream)
        del K, V
        q = wl.randn((B * Lp, Hq, D), torch.bfloat16, g, device=dev)
        out = torch.empty_like(q)
        d = C.byref(c.desc)

        def call():
            rc = L.sm_prefill_attention(d, ids.data_ptr(), B, offs.data_ptr(), B * Lp, q.data_ptr(), Hq,
                                        D ** -0.5, Lp, out.data_ptr(), st)
            if rc:
                raise RuntimeError(f"sm_prefill_attention failed: {rc}")
        t = _time(call, stream, reps)
        assert c.error_bits() == 0
        flop = 4.0 * Hq * D * B * Lp * (Lp + 1) / 2
        res[name] = {"positions": Lp, "ms": round(t, 4), "TFLOPs": round(flop / (t * 1e-3) / 1e12, 1),
                     "frac_of_bf16_peak": round(flop / (t * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}
        del c, q, out
        torch.cuda.empty_cache()
        log(f"extras: prefill attention over {Lp} positions done")
    res["speedup"] = round(res["uncompressed"]["ms"] / res["compacted"]["ms"], 3)
    res["kernel"] = "prefill_bf16<128>: causal grouped-query attention of 16 prompts x 32 heads over the paged cache"
    res["note"] = "HIP events around back-to-back calls; one layer's attention, K/V already appended"
    return res


def rules_report(sm, L, dev, stream, reps=20):
    """Rule matching over the 16 x 4096 prompt batch with 2.17M synthetic
    rules (the Llama-3 rule counts), rules planted for a 40% reduction: table
    build, the prompt scan, and one decode-time check of 16 sequences."""
    import torch
    from paper_2609_27233_amd import workload as wl
    st = stream.cuda_stream
    rules_np = wl.make_rules()
    toks_np, offs_np = wl.make_rule_prompts(rules_np, 16, 4096, 0.4, 128256, seed=3)
    i32 = lambda a: torch.as_tensor(np.asarray(a, np.int32)).to(dev)
    rules, toks, offs = i32(rules_np), i32(toks_np), i32(offs_np)
    t = sm.RuleTable(sm.RuleTable.capacity_for(len(rules_np)), device=dev)
    ws_b = torch.empty(L.sm_rules_build_workspace_bytes(t.capacity), dtype=torch.uint8, device=dev)
    d = C.byref(t.desc)

    def build():
        if L.sm_rules_build(rules.data_ptr(), len(rules_np), d, ws_b.data_ptr(), ws_b.numel(), st):
            raise RuntimeError("sm_rules_build failed")
    t_build = _time(build, stream, 3)
    T, B = len(toks_np), len(offs_np) - 1
    outs = [torch.empty(T // 2, dtype=torch.int32, device=dev) for _ in range(3)]
    sso = torch.empty(B + 1, dtype=torch.int32, device=dev)
    ws_m = torch.empty(L.sm_match_prompt_workspace_bytes(B, T), dtype=torch.uint8, device=dev)

    def match():
        if L.sm_match_prompt(d, toks.data_ptr(), offs.data_ptr(), B, T, outs[0].data_ptr(), outs[1].data_ptr(),
                             outs[2].data_ptr(), sso.data_ptr(), ws_m.data_ptr(), ws_m.numel(), st):
            raise RuntimeError("sm_match_prompt failed")
    t_match = _time(match, stream, reps)
    S = int(sso[-1].item())
    removed = int((outs[1][:S] - 1).sum().item())
    state = torch.zeros((B, 4), dtype=torch.int32, device=dev)
    ids = torch.arange(B, dtype=torch.int32, device=dev)
    gen = torch.as_tensor(np.random.RandomState(4).randint(0, 128256, (64, B)).astype(np.int32)).to(dev)
    k_out = torch.empty(B, dtype=torch.int32, device=dev)
    r_out = torch.empty(B, dtype=torch.int32, device=dev)
    step = [0]

    def dec():
        y = gen[step[0] % 64]
        step[0] += 1
        if L.sm_match_decode(d, state.data_ptr(), B, ids.data_ptr(), y.data_ptr(), B, k_out.data_ptr(),
                             r_out.data_ptr(), None, st):
            raise RuntimeError("sm_match_decode failed")
    t_dec = _time(dec, stream, 100)
    assert t.error_bits() == 0
    return {
        "rules": len(rules_np), "table_slots": t.capacity, "build_ms": round(t_build, 3),
        "prompt_tokens": T, "spans": S, "reduction": round(removed / T, 4),
        "match_prompt_us": round(t_match * 1e3, 1), "match_prompt_Mtokens_per_s": round(T / (t_match * 1e-3) / 1e6, 1),
        "decode_match_16_seqs_us": round(t_dec * 1e3, 2),
        "note": "HIP events around back-to-back calls; the prompt scan is 4 launches (longest rule per position, "
                "per-sequence chain scan, CSR offsets, compaction); latency-bound hash probes into a "
                f"{t.capacity * 20 / 2**20:.0f} MiB table"}


def lut_report(sm, L, dev, stream, reps=20):
    """Surrogates of the 16 x 4096 prompt batch's matched spans (d = 4096,
    bf16): looked up by rule id in a table of all 2.17M rules (17.8 GB),
    against the merge module over the same spans; the decode-step input of
    16 sequences; and the dedupe of a batch whose rules follow a Zipf law."""
    import torch
    from paper_2609_27233_amd import workload as wl
    st = stream.cuda_stream
    w = wl.WORKLOADS[2]
    d, h = w.d, w.h
    rules_np = wl.make_rules()
    R = len(rules_np)
    i32 = lambda a: torch.as_tensor(np.asarray(a, np.int32)).to(dev)
    toks_np, offs_np = wl.make_rule_prompts(rules_np, 16, 4096, 0.4, w.vocab, seed=3)
    t = sm.RuleTable(sm.RuleTable.capacity_for(R), device=dev)
    sm.rules_build(t, i32(rules_np))
    T, B = len(toks_np), 16
    toks, offs = i32(toks_np), i32(offs_np)
    s0, ln, ru = (torch.empty(T // 2, dtype=torch.int32, device=dev) for _ in range(3))
    sso = torch.empty(B + 1, dtype=torch.int32, device=dev)
    sm.match_prompt(t, toks, offs, s0, ln, ru, sso,
                    torch.empty(sm.match_prompt_workspace_bytes(B, T), dtype=torch.uint8, device=dev))
    S = int(sso[-1].item())
    g = wl.generator(5, dev)
    emb = wl.randn((w.vocab, d), torch.bfloat16, g, device=dev, std=0.02)
    lut = torch.empty((R, d), dtype=torch.bfloat16, device=dev)      # values do not change a copy's cost
    z = torch.empty((S, d), dtype=torch.bfloat16, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def gather():
        if L.sm_gather_surrogates(None, 0, lut.data_ptr(), R, None, ru.data_ptr(), S, d, sm.SM_BF16, z.data_ptr(),
                                  err.data_ptr(), st):
            raise RuntimeError("sm_gather_surrogates failed")
    t_g = _time(gather, stream, reps)
    # the merge module over the same spans
    ln_h, s0_h = ln[:S].cpu().numpy(), s0[:S].cpu().numpy()
    rows = i32(np.concatenate([toks_np[a:a + n] for a, n in zip(s0_h, ln_h)]))
    so = i32(np.concatenate([[0], np.cumsum(ln_h)]))
    par = wl.make_merge_params(d, h, torch.bfloat16, g, device=dev)
    ws = torch.empty(sm.merge_workspace_bytes(rows.numel(), S, d, torch.bfloat16), dtype=torch.uint8, device=dev)
    mp = sm.MergeParams(d, h, 1e-5, *(par[k].data_ptr() for k in
                        ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")))

    def merge():
        if L.sm_merge_spans(emb.data_ptr(), emb.shape[0], rows.data_ptr(), rows.numel(), so.data_ptr(), S,
                            C.byref(mp), sm.SM_BF16, z.data_ptr(), ws.data_ptr(), ws.numel(), err.data_ptr(), st):
            raise RuntimeError("sm_merge_spans failed")
    t_m = _time(merge, stream, 3)
    del ws
    # decode step inputs: 16 sequences, half of them just merged
    rid16 = i32(np.where(np.arange(16) % 2 == 0, np.arange(16) * 1000, -1))
    tok16 = i32(np.arange(16) * 7)
    x16 = torch.empty((16, d), dtype=torch.bfloat16, device=dev)

    def step_in():
        if L.sm_gather_surrogates(emb.data_ptr(), emb.shape[0], lut.data_ptr(), R, tok16.data_ptr(),
                                  rid16.data_ptr(), 16, d, sm.SM_BF16, x16.data_ptr(), err.data_ptr(), st):
            raise RuntimeError("sm_gather_surrogates failed")
    t_s = _time(step_in, stream, 100)
    del lut
    torch.cuda.empty_cache()
    # dedupe of a batch with Zipf-distributed rules
    tz_np, oz_np = wl.make_rule_prompts(rules_np, 16, 4096, 0.4, w.vocab, seed=9, zipf_a=1.2)
    tz = i32(tz_np)
    sm.match_prompt(t, tz, i32(oz_np), s0, ln, ru, sso,
                    torch.empty(sm.match_prompt_workspace_bytes(B, T), dtype=torch.uint8, device=dev))
    Sz = int(sso[-1].item())
    nsum = int(ln[:Sz].sum().item())
    uq, slot = (torch.empty(Sz, dtype=torch.int32, device=dev) for _ in range(2))
    urows, uoffs = torch.empty(nsum, dtype=torch.int32, device=dev), torch.empty(Sz + 1, dtype=torch.int32, device=dev)
    nu = torch.zeros(1, dtype=torch.int32, device=dev)
    wsd = torch.empty(L.sm_span_dedupe_workspace_bytes(Sz, R), dtype=torch.uint8, device=dev)

    def dedupe():
        if L.sm_span_dedupe(ru.data_ptr(), s0.data_ptr(), ln.data_ptr(), Sz, R, tz.data_ptr(), T, uq.data_ptr(),
                            slot.data_ptr(), urows.data_ptr(), uoffs.data_ptr(), nu.data_ptr(), wsd.data_ptr(),
                            wsd.numel(), err.data_ptr(), st):
            raise RuntimeError("sm_span_dedupe failed")
    t_d = _time(dedupe, stream, reps)
    U = int(nu.item())
    assert int(err.item()) == 0 and t.error_bits() == 0
    gbytes = 2.0 * S * d * 2
    return {
        "spans": S, "table_rows": R, "table_GB": round(R * d * 2 / 1e9, 1),
        "gather_us": round(t_g * 1e3, 1), "gather_GBps": round(gbytes / (t_g * 1e-3) / 1e9, 1),
        "gather_frac_of_hbm_peak": round(gbytes / (t_g * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "merge_module_same_spans_ms": round(t_m, 3), "lookup_speedup": round(t_m / t_g, 1),
        "decode_step_inputs_16_us": round(t_s * 1e3, 2),
        "zipf_batch_spans": Sz, "zipf_batch_distinct": U, "dedupe_us": round(t_d * 1e3, 1),
        "note": "HIP events around back-to-back calls; gather bytes = read + write of the span rows; the table "
                "is allocated at full size (values do not change a copy); dedupe on a batch whose planted rules "
                "follow Zipf(1.2) over the rule list"}


def kvproj_report(sm, L, dev, stream, reps=50):
    """The step inputs' K/V states (RMSNorm, W_k / W_v of the Llama-3-8B
    layer: 1024 x 4096 each, bf16, RoPE at the compressed position) for the
    16 decode sequences and for the 128 of the Qwen-shaped config, with and
    without the append."""
    import torch
    from paper_2609_27233_amd import workload as wl
    st = stream.cuda_stream
    res = {}
    for wid, name in ((2, "llama3_8b_16_seqs"), (4, "qwen2_7b_128_seqs")):
        w = wl.WORKLOADS[wid]
        n, d, H, D = w.batch, w.d, w.num_kv_heads, w.head_dim
        HD = H * D
        g = wl.generator(31, dev)
        x = wl.randn((n, d), torch.bfloat16, g, device=dev)
        Wk = wl.randn((HD, d), torch.bfloat16, g, device=dev, std=d ** -0.5)
        Wv = wl.randn((HD, d), torch.bfloat16, g, device=dev, std=d ** -0.5)
        c = sm.PagedCache(dtype=torch.bfloat16, num_kv_heads=H, head_dim=D, block_size=w.block_size,
                          num_blocks=n * (reps + 8), max_seqs=n, max_blocks_per_seq=reps + 8, device=dev)
        ids = torch.arange(n, dtype=torch.int32, device=dev)
        K = torch.empty((n, H, D), dtype=torch.bfloat16, device=dev)
        V = torch.empty_like(K)
        ws = torch.empty(sm.kv_project_workspace_bytes(n, d, H, D), dtype=torch.uint8, device=dev)
        p = sm.KVProjParams(d, Wk.data_ptr(), Wv.data_ptr(), 500000.0, 1e-5)
        dsc = C.byref(c.desc)

        def proj():
            if L.sm_kv_project(dsc, ids.data_ptr(), n, x.data_ptr(), C.byref(p), K.data_ptr(), V.data_ptr(),
                               ws.data_ptr(), ws.numel(), st):
                raise RuntimeError("sm_kv_project failed")

        def proj_append():
            if L.sm_kv_append_projected(dsc, ids.data_ptr(), n, x.data_ptr(), C.byref(p), ws.data_ptr(), ws.numel(),
                                        st):
                raise RuntimeError("sm_kv_append_projected failed")
        t_p = _time(proj, stream, reps)
        t_a = _time(proj_append, stream, reps)      # appends reps + 1 rows per sequence
        assert c.error_bits() == 0
        wbytes = 2 * HD * d * 2
        byts = wbytes + n * d * 2 + 2 * n * HD * 2
        res[name] = {"rows": n, "d": d, "kv_features": 2 * HD, "weights_MB": round(wbytes / 1e6, 1),
                     "project_us": round(t_p * 1e3, 2), "project_GBps": round(byts / (t_p * 1e-3) / 1e9, 1),
                     "project_frac_of_hbm_peak": round(byts / (t_p * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                     "project_and_append_us": round(t_a * 1e3, 2)}
        del c, ws
        torch.cuda.empty_cache()
    res["note"] = ("HIP events around back-to-back calls; bytes = W_k + W_v + the input rows + the K/V rows; "
                   "the weights stream from HBM once per call (they do not stay in the 4 MB L2 of an XCD)")
    return res


def traffic_bytes(alg_bytes):
    """Measured HBM bytes per attention launch, or None when the kernel
    sources differ from the ones the counters were taken on."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2609_27233_amd", "csrc")
    for name, digest in TRAFFIC_SOURCE_SHA256.items():
        with open(os.path.join(csrc, name), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return int(alg_bytes * TRAFFIC_RATIO)


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(job):
    """The oracle (plain fp64 C, OpenMP) timed on this host's cores on a
    bounded sample of one batch's job, scaled to the whole job.

    Threads: len(os.sched_getaffinity(0)) (the cores this process may run
    on).  Timed parts, on the job's own inputs:
      (i)   decode attention (append one row per sequence, then attention)
            of the full 16-sequence batch at the first decode step and at the
            last step's lengths; the job's 256 steps are estimated from the
            two by the step lengths (attention cost is linear in length);
      (ii)  the merge module on a seeded sample of min(S, 2048) prompt spans,
            extrapolated linearly to all S spans;
      (iii) pack and bulk append of the batch's prompt (full size).
    The decode-time merges (16 spans of 2-4 tokens every 8 steps) are
    extrapolated from (ii) per span.  A one-thread figure repeats (i) at the
    first step and (ii) on 64 spans."""
    import torch
    import oracle as orc
    from paper_2609_27233_amd import workload as wl

    w = job.w
    B, H, D, Hq = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads
    threads = len(os.sched_getaffinity(0))
    orc.set_num_threads(threads)
    P = job.prompts[0]
    S = len(P.span_len)
    params = {k: wl.to_f64(v) for k, v in job.params.items()}
    t_all = time.time()

    def merge_time(ns, seed):
        rng = np.random.RandomState(seed)
        sample = np.sort(rng.choice(S, ns, replace=False))
        offs = P.span_offsets
        rows = np.concatenate([P.row_idx[offs[s_]:offs[s_ + 1]] for s_ in sample])
        uniq, inv = np.unique(rows, return_inverse=True)
        emb_s = wl.to_f64(job.emb[torch.as_tensor(uniq, device=job.dev)])
        so = np.concatenate([[0], np.cumsum([offs[s_ + 1] - offs[s_] for s_ in sample])]).astype(np.int32)
        t = time.time()
        st, _ = orc.merge_spans(emb_s, inv.astype(np.int32), so, params, w.h)
        assert st == 0
        return (time.time() - t) / ns, float(np.mean(np.diff(so)))

    ns = min(S, 2048)
    t_span, mean_n = merge_time(ns, 11)
    t_merge = t_span * S
    # pack of the whole batch (indices) and bulk append of its K/V
    t = time.time()
    st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets)
    t_pack = time.time() - t
    assert st == 0
    nb_seq = -(-job.max_len // w.block_size) + 2
    oc = orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=w.block_size,
                         num_blocks=B * nb_seq, max_seqs=B, max_blocks_per_seq=nb_seq)
    t = time.time()
    st = oc.append(np.arange(B), res["packed_offsets"], wl.to_raw(job.Kp), wl.to_raw(job.Vp))
    t_append = time.time() - t
    assert st == 0
    Kt, Vt = wl.to_raw(job.Kt[0]), wl.to_raw(job.Vt[0])
    q = wl.to_f64(job.q[0])
    ids = np.arange(B)

    def step_time():
        t = time.time()
        assert oc.append(ids, np.arange(B + 1), Kt, Vt) == 0
        assert oc.decode_attention(ids, q, Hq, D ** -0.5)[0] == 0
        return time.time() - t

    t_first = step_time()
    # grow the cache to the last step's lengths (the job's schedule), then time that step
    last = job.len_sched[-1]
    grow = int(last.max()) - int(oc.lengths[:B].max()) - 1
    for _ in range(max(grow, 0)):
        oc.append(ids, np.arange(B + 1), Kt, Vt)
    t_last = step_time()
    first_len = float(job.L0 + 1)
    last_len = float(np.mean(oc.lengths[:B]))
    mean_len = float(np.mean([np.mean(x) for x in job.len_sched]))
    slope = (t_last - t_first) / max(last_len - first_len, 1.0)
    t_dec_job = w.decode_steps * (t_first + slope * (mean_len - first_len))
    n_dec_spans = B * len(job.dmerge)
    t_dec_merge = t_span * n_dec_spans * (3.0 / mean_n)   # decode-time spans hold 2-4 tokens (+ 1 output row)
    t_job = t_merge + t_pack + t_append + t_dec_job + t_dec_merge
    tokens = B * w.decode_steps
    measured = time.time() - t_all
    # one thread: the first decode step and 64 spans
    orc.set_num_threads(1)
    t_span1, _ = merge_time(min(S, 64), 12)
    oc.rollback(ids, np.full(B, int(oc.lengths[0]) - job.L0, np.int32))
    t_first1 = step_time()
    orc.set_num_threads(threads)
    t_job1 = (t_span1 * S + t_pack + t_append * 1.0 + t_dec_job * t_first1 / t_first
              + t_span1 * n_dec_spans * (3.0 / mean_n))
    return {
        "value": round(tokens / t_job, 2),
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": _cpu_model(),
        "value_1_thread": round(tokens / t_job1, 3),
        "sample": (f"fp64 oracle, {threads} threads (sched_getaffinity), on one 16-sequence batch of the job: "
                   f"(i) append + attention of all 16 sequences at the first decode step ({t_first:.3f} s, "
                   f"length {first_len:.0f}) and at the last step's lengths ({t_last:.3f} s, {last_len:.0f}), "
                   f"256 steps estimated linearly in length; (ii) M_phi on {ns} of {S} prompt spans, "
                   f"extrapolated to all spans and to the {n_dec_spans} decode-time spans; (iii) pack and "
                   f"bulk append of the batch ({job.packed_rows[0]} rows, full size); job estimate "
                   f"{t_job:.1f} s from {measured:.1f} s measured.  One thread: M_phi on 64 spans and the "
                   f"first decode step ({t_first1:.3f} s), same scaling (pack/append as measured)"),
        "parts_s": {"merge_prompt_extrapolated": round(t_merge, 2), "pack": round(t_pack, 3),
                    "bulk_append": round(t_append, 3), "decode_steps": round(t_dec_job, 2),
                    "decode_merges_extrapolated": round(t_dec_merge, 2)},
        "seconds_measured": round(measured, 2),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--replicas", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="skip the side measurements")
    ap.add_argument("--decode-steps", type=int, default=None,
                    help="decode steps per job (default: the workload's 256; shorter only for counter runs)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES three times (scales HBM counters) and exit")
    ap.add_argument("--merge-only", action="store_true",
                    help="only time the merge module over the 70B-shaped prompt batch and print that")
    ap.add_argument("--kvproj-only", action="store_true",
                    help="only time the K/V projection of the step inputs (with and without the append)")
    ap.add_argument("--lut-only", action="store_true",
                    help="only time the surrogate lookup, the merge module on the same spans, and the dedupe")
    ap.add_argument("--rules-only", action="store_true",
                    help="only time the rule table build and the prompt / decode matching")
    ap.add_argument("--configs-only", type=str, default=None, metavar="IDS",
                    help="only time the decode steps of these configurations (comma list of 2-5; 2 = without "
                         "decode-time merges)")
    ap.add_argument("--cache-ops-only", action="store_true",
                    help="only time the cache operations (bulk append, pack, step append, rollback) of one batch")
    ap.add_argument("--prefill-only", action="store_true",
                    help="only time the prefill attention over the compacted and uncompressed prompt batch")
    ap.add_argument("--no-token-table", action="store_true",
                    help="run the job's merges from the embeddings (sm_merge_spans) instead of the token table")
    ap.add_argument("--lanes", type=int, default=4,
                    help="streams the resident batches' decode steps are spread over (batch r on stream r %% lanes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: it measures the hot path on a single GPU "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    import dataclasses
    import torch
    from paper_2609_27233_amd import workload as wl

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration // 4
        a = torch.ones(n, dtype=torch.int32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"copied {n * 4} bytes three times")
        return
    if args.merge_only:
        from paper_2609_27233_amd import lib as sm
        print(json.dumps(merge_70b_report(sm, sm.load(), dev, torch.cuda.current_stream(), reps=5)), flush=True)
        return
    if args.kvproj_only:
        from paper_2609_27233_amd import lib as sm
        print(json.dumps(kvproj_report(sm, sm.load(), dev, torch.cuda.current_stream())), flush=True)
        return
    if args.lut_only:
        from paper_2609_27233_amd import lib as sm
        print(json.dumps(lut_report(sm, sm.load(), dev, torch.cuda.current_stream())), flush=True)
        return
    if args.rules_only:
        from paper_2609_27233_amd import lib as sm
        print(json.dumps(rules_report(sm, sm.load(), dev, torch.cuda.current_stream())), flush=True)
        return
    if args.prefill_only:
        from paper_2609_27233_amd import lib as sm
        print(json.dumps(prefill_report(sm, sm.load(), dev, torch.cuda.current_stream())), flush=True)
        return
    if args.configs_only:
        cids = tuple(int(x) for x in args.configs_only.split(","))
        print(json.dumps(configs_report(dev, torch.cuda.current_stream(), cids)), flush=True)
        return
    w = wl.WORKLOADS[2]
    if args.cache_ops_only:
        job = Job(dataclasses.replace(w, decode_steps=128), 1, dev, token_table=False, lanes=1)
        print(json.dumps(cache_ops_report(job, torch.cuda.current_stream())), flush=True)
        return
    if args.decode_steps is not None:
        w = dataclasses.replace(w, decode_steps=args.decode_steps)
    job = Job(w, args.replicas, dev, token_table=not args.no_token_table, lanes=args.lanes)
    stream = torch.cuda.current_stream()
    # one stream per lane, default priority
    streams = [stream] + [torch.cuda.Stream() for _ in range(job.lanes - 1)]
    nlaunch = w.decode_steps * job.R

    for i in range(args.warmup):
        job.run(streams)
        torch.cuda.synchronize()
        log(f"warmup {i} done")
    job.check_errors()

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        t_issue = time.perf_counter()
        job.run(streams)
        log(f"step {i} issued in {(time.perf_counter() - t_issue) * 1e3:.1f} ms of host time")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log("timed steps done")
    job.check_errors()

    # the kernel's own launch duration: the same job once more on one
    # stream, HIP events around each decode step's back-to-back launches
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(w.decode_steps)] for _ in range(2)]
    job.run([stream], events=ev)
    torch.cuda.synchronize()
    attn_ms = sum(a.elapsed_time(b) for a, b in zip(ev[0], ev[1]))
    job.check_errors()
    log("single-stream pass done")

    ms_per_step = elapsed * 1e3 / args.steps
    tokens = job.R * w.batch * w.decode_steps
    value = tokens * args.steps / elapsed
    bytes_per_step = sum(job.decode_bytes(l) for l in job.len_sched) * job.R
    avg_launch_us = attn_ms * 1e3 / nlaunch
    achieved = bytes_per_step / (attn_ms * 1e-3) / 1e9
    mean_bytes = bytes_per_step / nlaunch
    overlapped = lanes_report(job, streams, rounds=8) if job.lanes > 1 else None
    graph = graph_report(job, rounds=16)

    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: 40% span-merged prompts (L0={job.L0}), {w.decode_steps} decode steps, "
                        f"decode-time merge every {w.merge_every} steps, {job.R} resident batches",
            "batch": w.batch, "prompt_len": w.prompt_len, "compacted_len": job.L0,
            "decode_steps": w.decode_steps, "resident_batches": job.R,
            "decode_lanes": job.lanes,
            "merge_first_stage": ("token table (sm_merge_token_table once, %.2f ms; sm_merge_spans_tabled per call)"
                                  % job.table_ms) if job.table is not None else "per call (sm_merge_spans)",
            "layer": {"d": w.d, "q_heads": w.num_q_heads, "kv_heads": w.num_kv_heads, "head_dim": w.head_dim},
            "block_size": w.block_size,
        },
        "roofline": {
            "kernel": "decode_split_bf16<128, step>: one fused append + attention launch per decode step and "
                      "batch; HIP events around each step's back-to-back launches on one stream (a pass of the "
                      "same job after the timed steps), divided by the launch count",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic_bytes(mean_bytes),
            "avg_launch_us": round(avg_launch_us, 3),
            "algorithmic_bytes_per_launch": int(mean_bytes),
        },
    }
    if overlapped is not None:
        result["roofline"]["overlapped"] = overlapped
    if graph is not None:
        result["roofline"]["graph"] = graph
    if not args.no_extras and args.decode_steps is None:
        try:
            result["extras"] = extras_report(job, stream, avg_launch_us)
        except Exception as e:          # side measurements never hide the main line
            log(f"extras failed: {e!r}")
            result["extras"] = {"error": repr(e)}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(job)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
