"""The C ABI library loads and exports every declared symbol; host-side
argument checks return their status without touching a GPU."""
import ctypes as C
import os
import re

import pytest

from conftest import ROOT
from paper_2609_27233_amd import lib as sm


def _declared():
    src = open(os.path.join(ROOT, "include", "spanmerge.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sm_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    return sm.load()


def test_every_declared_symbol_is_exported(L):
    names = _declared()
    assert set(names) == set(sm.EXPORTED)
    for n in names:
        assert hasattr(L, n), n


def test_no_other_exports():
    # symbols are hidden by default; only the sm_ entry points are visible
    out = os.popen("nm -D --defined-only %s" % sm.LIB_PATH).read()
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    assert {n for n in exported if n.startswith("sm_")} == set(sm.EXPORTED)


def test_status_strings(L):
    assert L.sm_status_string(0) == b"ok"
    assert b"argument" in L.sm_status_string(1)


def test_missing_library_fails_loudly(tmp_path):
    saved = sm._lib
    sm._lib = None
    try:
        with pytest.raises(sm.SpanMergeError):
            sm.load(str(tmp_path / "nope.so"))
    finally:
        sm._lib = saved


def _desc(**kw):
    base = dict(dtype=sm.SM_BF16, num_kv_heads=8, head_dim=128, block_size=16, num_blocks=64,
                max_seqs=4, max_blocks_per_seq=16, k_pool=1, v_pool=1, block_table=1,
                lengths=1, free_stack=1, free_top=1, err=1)
    base.update(kw)
    return sm.PagedCacheDesc(*base.values())


@pytest.mark.parametrize("kw", [dict(head_dim=96), dict(block_size=24), dict(block_size=8),
                                dict(dtype=7), dict(k_pool=None), dict(num_blocks=0)])
def test_cache_descriptor_checks(L, kw):
    d = _desc(**kw)
    assert L.sm_kv_rollback(C.byref(d), 1, 1, 1, None) == sm.SM_EINVAL
    assert L.sm_kv_append(C.byref(d), 1, 1, 1, 1, 1, 1, None) == sm.SM_EINVAL
    assert L.sm_decode_attention(C.byref(d), 1, 1, 1, 8, 1.0, 16, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_step(C.byref(d), 1, 1, 1, 1, 1, 8, 1.0, 16, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_merge_step(C.byref(d), 1, 1, 1, 1, 1, 1, 8, 1.0, 16, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_prefill_attention(C.byref(d), 1, 1, 1, 16, 1, 8, 1.0, 16, 1, None) == sm.SM_EINVAL


def test_prefill_argument_checks(L):
    d = _desc()
    pf = lambda d, n=1, rows=16, hq=32, max_rows=16: L.sm_prefill_attention(C.byref(d), 1, n, 1, rows, 1, hq, 1.0,
                                                                           max_rows, 1, None)
    assert pf(d, n=0) == sm.SM_OK                         # nothing to do
    assert pf(d, n=-1) == sm.SM_EINVAL
    assert pf(d, rows=-1) == sm.SM_EINVAL
    assert pf(d, max_rows=-1) == sm.SM_EINVAL
    assert pf(d, hq=12) == sm.SM_EINVAL                   # Hq % Hkv
    assert pf(d, hq=8 * 17) == sm.SM_EINVAL               # group > 16
    assert pf(_desc(dtype=sm.SM_F32)) == sm.SM_EINVAL     # bf16 only
    assert pf(_desc(head_dim=32)) == sm.SM_EINVAL
    assert pf(_desc(max_blocks_per_seq=4097)) == sm.SM_EINVAL
    assert L.sm_prefill_attention(C.byref(d), None, 1, 1, 16, 1, 32, 1.0, 16, 1, None) == sm.SM_EINVAL
    assert L.sm_prefill_attention(C.byref(d), 1, 1, None, 16, 1, 32, 1.0, 16, 1, None) == sm.SM_EINVAL
    assert L.sm_prefill_attention(C.byref(d), 1, 1, 1, 16, 1, 32, 1.0, 16, None, None) == sm.SM_EINVAL
    for bad in (float("nan"), float("inf"), -float("inf")):                   # the scale must be finite
        assert L.sm_prefill_attention(C.byref(d), 1, 1, 1, 16, 1, 32, bad, 16, 1, None) == sm.SM_EINVAL
    # one page over all kv heads must stay below 4 GiB: 8 heads x 2^22 tokens x 128 dims x 2 bytes = 8 GiB
    assert pf(_desc(block_size=1 << 22)) == sm.SM_EINVAL


def test_request_count_and_workspace_checks(L):
    d = _desc()
    assert L.sm_kv_rollback(C.byref(d), 1, 1, 5, None) == sm.SM_EINVAL       # n > max_seqs
    assert L.sm_kv_rollback(C.byref(d), 1, 1, 0, None) == sm.SM_OK           # nothing to do
    assert L.sm_decode_attention(C.byref(d), 1, 1, 1, 12, 1.0, 16, 1, 1, 1 << 30, None) == sm.SM_EINVAL  # Hq % Hkv
    assert L.sm_decode_attention(C.byref(d), 1, 1, 1, 8 * 17, 1.0, 16, 1, 1, 1 << 30, None) == sm.SM_EINVAL  # G > 16
    need = L.sm_decode_workspace_bytes(1, 32, 128, 256)
    assert need > 0
    assert L.sm_decode_attention(C.byref(d), 1, 1, 1, 32, 1.0, 256, 1, 1, need - 1, None) == sm.SM_EINVAL
    assert L.sm_decode_attention(C.byref(d), 1, 1, 1, 32, 1.0, 257, 1, 1, 1 << 30, None) == sm.SM_EINVAL  # > capacity
    # the fused step: at most 256 requests, new rows required, same workspace rule
    assert L.sm_decode_step(C.byref(d), 1, 0, None, None, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_OK
    assert L.sm_decode_step(C.byref(d), 1, 257, 1, 1, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_step(C.byref(d), 1, 1, None, 1, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_step(C.byref(d), 1, 1, 1, None, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_step(C.byref(d), 1, 1, 1, 1, 1, 32, 1.0, 256, 1, 1, need - 1, None) == sm.SM_EINVAL
    assert L.sm_decode_step(C.byref(d), 1, 1, 1, 1, 1, 32, 1.0, 257, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    # the merge step: the same rules, a crop array required, bf16 caches only
    assert L.sm_decode_merge_step(C.byref(d), 1, 1, 0, None, None, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_OK
    assert L.sm_decode_merge_step(C.byref(d), 1, None, 1, 1, 1, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_merge_step(C.byref(d), 1, 1, 257, 1, 1, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL
    assert L.sm_decode_merge_step(C.byref(d), 1, 1, 1, 1, 1, 1, 32, 1.0, 256, 1, 1, need - 1, None) == sm.SM_EINVAL
    f = _desc(dtype=sm.SM_F32)
    assert L.sm_decode_merge_step(C.byref(f), 1, 1, 1, 1, 1, 1, 32, 1.0, 256, 1, 1, 1 << 30, None) == sm.SM_EINVAL


def test_merge_argument_checks(L):
    p = sm.MergeParams(4096, 4, 1e-5, *([1] * 9))
    ws = L.sm_merge_workspace_bytes(100, 30, 4096, sm.SM_BF16)
    assert ws >= 100 * 4096 * 2 + 30 * 4096 * 6
    assert L.sm_merge_spans(1, 10, 1, 100, 1, 30, C.byref(p), sm.SM_BF16, 1, 1, ws - 1, 1, None) == sm.SM_EINVAL
    bad = sm.MergeParams(4000, 4, 1e-5, *([1] * 9))   # d % 256 != 0
    assert L.sm_merge_spans(1, 10, 1, 100, 1, 30, C.byref(bad), sm.SM_BF16, 1, 1, 1 << 40, 1, None) == sm.SM_EINVAL
    assert L.sm_merge_spans(1, 10, 1, 10, 1, 30, C.byref(p), sm.SM_BF16, 1, 1, 1 << 40, 1, None) == sm.SM_EINVAL  # rows < spans
    assert L.sm_merge_spans(1, 10, 1, 0, 1, 0, C.byref(p), sm.SM_BF16, 1, 1, 0, 1, None) == sm.SM_OK


def test_pack_argument_checks(L):
    assert L.sm_pack_spans(-1, 1, 0, 0, 1, 1, 1, 1, 1, 1, None, None, 0, None, 0, 1, None, 1, None) == sm.SM_EINVAL
    assert L.sm_pack_spans(0, 1, 0, 0, 1, 1, 1, 1, 1, 1, None, None, 0, None, 0, 1, None, 1, None) == sm.SM_OK
    # rows requested without an embedding table
    assert L.sm_pack_spans(2, 1, 8, 1, 1, 1, 1, 1, 1, 1, None, None, 0, None, 64, 1, 1, 1, None) == sm.SM_EINVAL


def test_rule_call_argument_checks(L):
    good = sm.RuleTableDesc(1024, 1, 1, 1)
    bad_cap = sm.RuleTableDesc(1000, 1, 1, 1)               # not a power of two
    assert L.sm_rules_build_workspace_bytes(1024) == 8192
    assert L.sm_rules_build(1, 10, C.byref(bad_cap), 1, 1 << 20, None) == sm.SM_EINVAL
    assert L.sm_rules_build(1, 769, C.byref(good), 1, 1 << 20, None) == sm.SM_EINVAL   # load above 3/4
    assert L.sm_rules_build(1, 10, C.byref(good), 1, 8191, None) == sm.SM_EINVAL       # workspace
    assert L.sm_rules_build(1, 10, C.byref(good), None, 1 << 20, None) == sm.SM_EINVAL
    assert L.sm_rules_build(None, 10, C.byref(good), 1, 1 << 20, None) == sm.SM_EINVAL
    assert L.sm_rules_lookup(C.byref(good), 1, 0, 1, None) == sm.SM_OK                 # nothing to do
    assert L.sm_rules_lookup(C.byref(bad_cap), 1, 4, 1, None) == sm.SM_EINVAL
    assert L.sm_rules_lookup(C.byref(good), None, 4, 1, None) == sm.SM_EINVAL
    need = L.sm_match_prompt_workspace_bytes(16, 65536)
    assert need >= 17 * 65536
    mp = lambda ws_bytes, B=16, T=65536, tbl=good, sso=1: L.sm_match_prompt(
        C.byref(tbl), 1, 1, B, T, 1, 1, 1, sso, 1, ws_bytes, None)
    assert mp(need - 1) == sm.SM_EINVAL
    assert mp(need, B=70000) == sm.SM_EINVAL
    assert mp(need, tbl=bad_cap) == sm.SM_EINVAL
    assert mp(need, sso=None) == sm.SM_EINVAL
    md = lambda n, ids=1, cache=None: L.sm_match_decode(C.byref(good), 1, 64, ids, 1, n, 1, 1, cache, None)
    assert md(0) == sm.SM_OK
    assert md(1025) == sm.SM_EINVAL
    assert md(4, ids=None) == sm.SM_EINVAL
    assert md(4, cache=C.byref(_desc(head_dim=96))) == sm.SM_EINVAL                      # the rollback's checks
    assert md(5, cache=C.byref(_desc())) == sm.SM_EINVAL                                 # n > max_seqs (4)


def test_lut_call_argument_checks(L):
    g = lambda n=4, d=64, dt=sm.SM_BF16, rule=1, out=1, err=1: L.sm_gather_surrogates(
        1, 10, 1, 10, 1, rule, n, d, dt, out, err, None)
    assert g(n=0) == sm.SM_OK
    assert g(n=-1) == sm.SM_EINVAL
    assert g(d=4) == sm.SM_EINVAL                       # 8 bytes: not a multiple of 16
    assert g(dt=7) == sm.SM_EINVAL
    assert g(rule=None) == sm.SM_EINVAL and g(out=None) == sm.SM_EINVAL and g(err=None) == sm.SM_EINVAL
    need = L.sm_span_dedupe_workspace_bytes(100, 1000)
    assert need >= 4 * 1100
    dd = lambda ws_bytes=need, S=100, rule=1: L.sm_span_dedupe(rule, 1, 1, S, 1000, 1, 500, 1, 1, 1, 1, 1, 1,
                                                               ws_bytes, 1, None)
    assert dd(ws_bytes=need - 1) == sm.SM_EINVAL
    assert dd(S=-1) == sm.SM_EINVAL
    assert dd(rule=None) == sm.SM_EINVAL


def test_kv_project_argument_checks(L):
    d = _desc()
    p = sm.KVProjParams(4096, 1, 1, 500000.0, 1e-5)
    need = L.sm_kv_project_workspace_bytes(4, 4096, 8, 128)
    assert need >= 16 * 4 * 2048 * 4
    assert L.sm_kv_project_workspace_bytes(4, 4000, 8, 128) == 0               # d not a multiple of 256
    kp = lambda desc=d, n=4, prm=p, ws_bytes=need, K=1: L.sm_kv_project(C.byref(desc), 1, n, 1, C.byref(prm), K, 1,
                                                                       1, ws_bytes, None)
    assert kp(n=0) == sm.SM_OK
    assert kp(ws_bytes=need - 1) == sm.SM_EINVAL
    assert kp(n=5) == sm.SM_EINVAL                                             # n > max_seqs (4)
    assert kp(desc=_desc(dtype=sm.SM_F32)) == sm.SM_EINVAL                     # bf16 caches only
    assert kp(prm=sm.KVProjParams(4000, 1, 1, 500000.0, 1e-5)) == sm.SM_EINVAL
    assert kp(prm=sm.KVProjParams(4096, 1, 1, 0.0, 1e-5)) == sm.SM_EINVAL      # theta must be > 0
    assert kp(prm=sm.KVProjParams(4096, None, 1, 500000.0, 1e-5)) == sm.SM_EINVAL
    assert kp(K=None) == sm.SM_EINVAL
    ap = lambda desc=d, n=4, ws_bytes=need: L.sm_kv_append_projected(C.byref(desc), 1, n, 1, C.byref(p), 1,
                                                                      ws_bytes, None)
    assert ap(n=0) == sm.SM_OK
    assert ap(ws_bytes=need - 1) == sm.SM_EINVAL
    assert ap(desc=_desc(head_dim=96)) == sm.SM_EINVAL
