"""The benchmark's own job end to end against the oracle: bench.Job for the
Llama-3-8B-shaped configuration (16 x 4096-token prompts, 40% merged, 256
decode steps with a decode-time merge every 8 steps), four resident
batches on four streams, exactly as bench.py schedules them:

* the merge module's first stage from the token table over the whole
  128,256-row vocabulary, sm_merge_spans_tabled for the prompt spans and
  for every decode-time merge;
* sm_pack_spans and the bulk sm_kv_append of the compressed prompts;
* every decode step one fused launch per batch: sm_decode_step, or at a
  merge step sm_decode_merge_step (crop n - 1 entries per sequence, append
  the surrogate's row, attend).

The job's test hook synchronizes after each phase and the oracle replays it:
pack indices and packed rows bit for bit; 256 sampled prompt surrogates per
batch and all 16 surrogates of every decode-time merge within the bf16 bar;
lengths, block tables and free stacks bit for bit after every step; the
pools bit for bit after the prompt and every 32 steps; attention outputs of
all 16 sequences at step 0, every merge step and step 255."""
import numpy as np
import pytest
import torch

from gpu_util import TOL, assert_same_state, dev, rel_l2_max, say
from paper_2609_27233_amd import workload as wl

pytestmark = pytest.mark.gpu


def test_bench_job_all_256_steps_on_four_streams(orc):
    import bench
    w = wl.WORKLOADS[2]
    R, lanes = 4, 4
    say("bench job: 16 x 4096-token batches", R, "lanes", lanes)
    job = bench.Job(w, R, dev(), token_table=True, lanes=lanes)
    B, H, D, Hq = w.batch, w.num_kv_heads, w.head_dim, w.num_q_heads
    tol = TOL[torch.bfloat16]
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(lanes - 1)]
    params64 = {k: wl.to_f64(v) for k, v in job.params.items()}
    ocs = [orc.OracleCache(bf16=True, num_kv_heads=H, head_dim=D, block_size=w.block_size,
                           num_blocks=c.num_blocks, max_seqs=B, max_blocks_per_seq=c.max_blocks)
           for c in job.caches]
    ids = np.arange(B)
    rng = np.random.RandomState(2024)
    Kt = [wl.to_raw(x) for x in job.Kt]
    Vt = [wl.to_raw(x) for x in job.Vt]
    q64 = [wl.to_f64(x) for x in job.q]
    emb_raw = wl.to_raw(job.emb)
    counts = dict(attention=0, prompt_spans=0, decode_spans=0, pools=0, meta=0)

    def merge_ref(row_idx, offs):
        used, inv = np.unique(row_idx, return_inverse=True)
        rows = wl.to_f64(job.emb[torch.as_tensor(used, device=dev())])
        return orc.merge_spans_rows(rows, inv.astype(np.int32), offs, params64, w.h)

    def meta(r):
        assert job.caches[r].error_bits() == 0
        assert_same_state(job.caches[r], ocs[r], pools=False)
        counts["meta"] += 1

    def pools(r):
        assert_same_state(job.caches[r], ocs[r], pools=True)
        counts["pools"] += 1

    def hook(kind, s):
        torch.cuda.synchronize()
        if kind == "prompt":
            for r in range(R):
                P, cb = job.prompts[r], job.cbuf[r % lanes]
                z = cb["z"][:len(P.span_len)]
                st, res = orc.pack_spans(P.seq_offsets, P.span_start, P.span_len, P.seq_span_offsets,
                                         token_ids=P.token_ids, emb_raw=emb_raw, surrogates_raw=wl.to_raw(z))
                assert st == orc.OK
                rows = int(res["packed_offsets"][-1])
                np.testing.assert_array_equal(cb["pi"].cpu().numpy(), res["pi"])
                np.testing.assert_array_equal(cb["po"].cpu().numpy(), res["packed_offsets"])
                np.testing.assert_array_equal(cb["ps"][:rows].cpu().numpy(), res["packed_src"])
                assert np.array_equal(wl.to_raw(cb["packed"][:rows]), res["packed"]), "packed rows differ"
                S = len(P.span_len)
                samp = np.sort(rng.choice(S, 256, replace=False))
                offs = P.span_offsets
                row_idx = np.concatenate([P.row_idx[offs[k]:offs[k + 1]] for k in samp])
                so = np.concatenate([[0], np.cumsum([offs[k + 1] - offs[k] for k in samp])]).astype(np.int32)
                e = rel_l2_max(z[torch.as_tensor(samp, device=dev())].float().cpu().numpy(), merge_ref(row_idx, so))
                say("batch", r, "prompt surrogates rel_l2_max over", len(samp), "spans:", e)
                assert e <= tol
                counts["prompt_spans"] += len(samp)
                assert ocs[r].append(ids, res["packed_offsets"], wl.to_raw(job.Kp), wl.to_raw(job.Vp)) == orc.OK
                meta(r)
                pools(r)
        elif kind == "merge":
            m = job.dmerge[s]
            rows = m["rows"]
            row_idx = m["g_row_idx"][:rows].cpu().numpy()
            offs = m["g_offs"][:B + 1].cpu().numpy().astype(np.int32)
            ref = merge_ref(row_idx, offs)
            for lane in range(lanes):
                e = rel_l2_max(job.zdec[lane][:B].float().cpu().numpy(), ref)
                assert e <= tol, (s, lane, e)
            counts["decode_spans"] += lanes * B
            for r in range(R):
                meta(r)   # the crop comes with the step's launch
        else:
            j = s % job.nin
            check_attn = s == 0 or s in job.dmerge or s == w.decode_steps - 1
            for r in range(R):
                if s in job.dmerge:
                    st = ocs[r].crop_append(ids, job.dmerge[s]["n"] - 1, Kt[j], Vt[j])
                else:
                    st = ocs[r].append(ids, np.arange(B + 1), Kt[j], Vt[j])
                assert st == orc.OK
                meta(r)
                if check_attn:
                    st, ref = ocs[r].decode_attention(ids, q64[j], Hq, D ** -0.5)
                    assert st == orc.OK
                    e = rel_l2_max(job.out[r % lanes].float().cpu().numpy(), ref)
                    assert e <= tol, (s, r, e)
                    counts["attention"] += 1
                if s % 32 == 31:
                    pools(r)
            if s % 32 == 31:
                say("step", s, "lengths", job.caches[0].lengths[:4].tolist(), counts)

    job.run(streams, hook=hook)
    torch.cuda.synchronize()
    job.check_errors()
    say("bench job checks", counts)
    assert counts["attention"] == R * len({0, w.decode_steps - 1} | set(job.dmerge))
    assert counts["decode_spans"] == lanes * B * len(job.dmerge)
