"""Thin ctypes binding of ``libspanmerge.so`` (argument marshalling only).

Every function mirrors one C entry point of ``include/spanmerge.h`` and takes
torch tensors that already live on the GPU; the work itself runs in the HIP
kernels.  There is no CPU fallback: loading fails loudly when the library
has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspanmerge.so")

SM_F32, SM_BF16 = 0, 1
SM_OK, SM_EINVAL, SM_ERANGE, SM_ENOMEM, SM_EHIP = 0, 1, 2, 3, 4
ERR_EINVAL, ERR_ERANGE, ERR_ENOMEM = 1, 2, 4
MAX_REQUESTS = 1024

_P, _I, _L, _F, _Z = C.c_void_p, C.c_int, C.c_int64, C.c_float, C.c_size_t

EXPORTED = ("sm_status_string", "sm_merge_workspace_bytes", "sm_merge_spans",
            "sm_merge_token_table", "sm_merge_spans_tabled",
            "sm_pack_spans", "sm_kv_rollback", "sm_kv_append",
            "sm_decode_workspace_bytes", "sm_decode_attention", "sm_decode_step", "sm_decode_merge_step",
            "sm_decode_step_noalloc_max_bytes", "sm_decode_step_noalloc", "sm_set_commit_wait_limit",
            "sm_prefill_attention", "sm_rules_build_workspace_bytes", "sm_rules_build",
            "sm_rules_lookup", "sm_match_prompt_workspace_bytes", "sm_match_prompt",
            "sm_match_decode", "sm_gather_surrogates", "sm_span_dedupe_workspace_bytes", "sm_span_dedupe",
            "sm_kv_project_workspace_bytes", "sm_kv_project", "sm_kv_append_projected")


class MergeParams(C.Structure):
    _fields_ = [("d", _I), ("h", _I), ("ln_eps", _F), ("Q", _P), ("W_kv", _P),
                ("b_kv", _P), ("g_kv", _P), ("beta_kv", _P), ("W_o", _P),
                ("b_o", _P), ("g_o", _P), ("beta_o", _P)]


class PagedCacheDesc(C.Structure):
    _fields_ = [("dtype", _I), ("num_kv_heads", _I), ("head_dim", _I),
                ("block_size", _I), ("num_blocks", _I), ("max_seqs", _I),
                ("max_blocks_per_seq", _I), ("k_pool", _P), ("v_pool", _P),
                ("block_table", _P), ("lengths", _P), ("free_stack", _P),
                ("free_top", _P), ("err", _P)]


class RuleTableDesc(C.Structure):
    _fields_ = [("capacity", _I), ("keys", _P), ("ids", _P), ("err", _P)]


class KVProjParams(C.Structure):
    _fields_ = [("d", _I), ("W_k", _P), ("W_v", _P), ("rope_theta", _F), ("rms_eps", _F)]


class SpanMergeError(RuntimeError):
    pass


_lib = None


def load(path: str = LIB_PATH):
    """Load the HIP library (raises if it is missing: no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise SpanMergeError(
            f"{path} is missing; build it with `python -m paper_2609_27233_amd.build`")
    L = C.CDLL(path)
    L.sm_status_string.argtypes = [_I]
    L.sm_status_string.restype = C.c_char_p
    L.sm_merge_workspace_bytes.argtypes = [_I, _I, _I, _I]
    L.sm_merge_workspace_bytes.restype = _Z
    L.sm_merge_spans.argtypes = [_P, _L, _P, _I, _P, _I, C.POINTER(MergeParams), _I,
                                 _P, _P, _Z, _P, _P]
    L.sm_merge_spans.restype = _I
    L.sm_merge_token_table.argtypes = [_P, _L, C.POINTER(MergeParams), _I, _P, _P, _P]
    L.sm_merge_token_table.restype = _I
    L.sm_merge_spans_tabled.argtypes = [_P, _L, _P, _I, _P, _I, C.POINTER(MergeParams), _I,
                                        _P, _P, _Z, _P, _P]
    L.sm_merge_spans_tabled.restype = _I
    L.sm_pack_spans.argtypes = [_I, _P, _I, _I, _P, _P, _P, _P, _P, _P, _P, _P, _L,
                                _P, _I, _I, _P, _P, _P]
    L.sm_pack_spans.restype = _I
    L.sm_kv_rollback.argtypes = [C.POINTER(PagedCacheDesc), _P, _P, _I, _P]
    L.sm_kv_rollback.restype = _I
    L.sm_kv_append.argtypes = [C.POINTER(PagedCacheDesc), _P, _P, _I, _I, _P, _P, _P]
    L.sm_kv_append.restype = _I
    L.sm_decode_workspace_bytes.argtypes = [_I, _I, _I, _I]
    L.sm_decode_workspace_bytes.restype = _Z
    L.sm_decode_attention.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, _I, _F,
                                      _I, _P, _P, _Z, _P]
    L.sm_decode_attention.restype = _I
    L.sm_decode_step.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, _P, _P, _I, _F,
                                 _I, _P, _P, _Z, _P]
    L.sm_decode_step.restype = _I
    L.sm_decode_merge_step.argtypes = [C.POINTER(PagedCacheDesc), _P, _P, _I, _P, _P, _P, _I, _F,
                                       _I, _P, _P, _Z, _P]
    L.sm_decode_merge_step.restype = _I
    L.sm_decode_step_noalloc_max_bytes.argtypes = []
    L.sm_decode_step_noalloc_max_bytes.restype = _Z
    L.sm_decode_step_noalloc.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, _P, _P, _I, _F, _I, _P, _P]
    L.sm_decode_step_noalloc.restype = _I
    L.sm_set_commit_wait_limit.argtypes = [_I]
    L.sm_set_commit_wait_limit.restype = None
    L.sm_prefill_attention.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, _I, _P, _I, _F, _I, _P, _P]
    L.sm_prefill_attention.restype = _I
    L.sm_rules_build_workspace_bytes.argtypes = [_I]
    L.sm_rules_build_workspace_bytes.restype = _Z
    L.sm_rules_build.argtypes = [_P, _I, C.POINTER(RuleTableDesc), _P, _Z, _P]
    L.sm_rules_build.restype = _I
    L.sm_rules_lookup.argtypes = [C.POINTER(RuleTableDesc), _P, _I, _P, _P]
    L.sm_rules_lookup.restype = _I
    L.sm_match_prompt_workspace_bytes.argtypes = [_I, _I]
    L.sm_match_prompt_workspace_bytes.restype = _Z
    L.sm_match_prompt.argtypes = [C.POINTER(RuleTableDesc), _P, _P, _I, _I, _P, _P, _P, _P, _P, _Z, _P]
    L.sm_match_prompt.restype = _I
    L.sm_match_decode.argtypes = [C.POINTER(RuleTableDesc), _P, _I, _P, _P, _I, _P, _P,
                                  C.POINTER(PagedCacheDesc), _P]
    L.sm_match_decode.restype = _I
    L.sm_gather_surrogates.argtypes = [_P, _L, _P, _L, _P, _P, _I, _I, _I, _P, _P, _P]
    L.sm_gather_surrogates.restype = _I
    L.sm_span_dedupe_workspace_bytes.argtypes = [_I, _I]
    L.sm_span_dedupe_workspace_bytes.restype = _Z
    L.sm_span_dedupe.argtypes = [_P, _P, _P, _I, _I, _P, _I, _P, _P, _P, _P, _P, _P, _Z, _P, _P]
    L.sm_span_dedupe.restype = _I
    L.sm_kv_project_workspace_bytes.argtypes = [_I, _I, _I, _I]
    L.sm_kv_project_workspace_bytes.restype = _Z
    L.sm_kv_project.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, C.POINTER(KVProjParams), _P, _P, _P, _Z, _P]
    L.sm_kv_project.restype = _I
    L.sm_kv_append_projected.argtypes = [C.POINTER(PagedCacheDesc), _P, _I, _P, C.POINTER(KVProjParams), _P, _Z, _P]
    L.sm_kv_append_projected.restype = _I
    _lib = L
    return L


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise SpanMergeError("expected a GPU tensor")
    if not t.is_contiguous():
        raise SpanMergeError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _check(st: int, what: str):
    if st != SM_OK:
        msg = load().sm_status_string(st).decode()
        raise SpanMergeError(f"{what}: {msg} (status {st})")


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return SM_BF16
    if dt == torch.float32:
        return SM_F32
    raise SpanMergeError(f"unsupported dtype {dt}")


# --------------------------------------------------------------------------
# merge_spans

def merge_workspace_bytes(total_rows: int, num_spans: int, d: int, dtype: torch.dtype) -> int:
    return load().sm_merge_workspace_bytes(total_rows, num_spans, d, dtype_code(dtype))


def merge_spans(emb, row_idx, span_offsets, params: dict, h: int, out, ws, err,
                ln_eps: float = 1e-5, total_rows: Optional[int] = None, stream=None):
    """z_s = M_phi(emb[row_idx[span s]]) for every span; writes ``out``."""
    S = span_offsets.numel() - 1
    R = row_idx.numel() if total_rows is None else total_rows
    p = MergeParams(emb.shape[1], h, ln_eps, *(_ptr(params[k]) for k in
                    ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")))
    st = load().sm_merge_spans(_ptr(emb), emb.shape[0], _ptr(row_idx), R,
                               _ptr(span_offsets), S, C.byref(p), dtype_code(emb.dtype),
                               _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                               _ptr(err), _stream(stream))
    _check(st, "sm_merge_spans")


def _merge_params(d: int, h: int, params: dict, ln_eps: float):
    return MergeParams(d, h, ln_eps, *(_ptr(params[k]) for k in
                       ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")))


def merge_token_table(emb, params: dict, h: int, table, err, ln_eps: float = 1e-5, stream=None):
    """table[v] = GELU(Linear_kv(emb[v])) for every row of ``emb``."""
    p = _merge_params(emb.shape[1], h, params, ln_eps)
    st = load().sm_merge_token_table(_ptr(emb), emb.shape[0], C.byref(p), dtype_code(emb.dtype),
                                     _ptr(table), _ptr(err), _stream(stream))
    _check(st, "sm_merge_token_table")


def merge_spans_tabled(table, row_idx, span_offsets, params: dict, h: int, out, ws, err,
                       ln_eps: float = 1e-5, total_rows: Optional[int] = None, stream=None):
    """The surrogates of merge_spans, the first stage read from ``table``
    (rows = token ids)."""
    S = span_offsets.numel() - 1
    R = row_idx.numel() if total_rows is None else total_rows
    p = _merge_params(table.shape[1], h, params, ln_eps)
    st = load().sm_merge_spans_tabled(_ptr(table), table.shape[0], _ptr(row_idx), R,
                                      _ptr(span_offsets), S, C.byref(p), dtype_code(table.dtype),
                                      _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                      _ptr(err), _stream(stream))
    _check(st, "sm_merge_spans_tabled")


# --------------------------------------------------------------------------
# pack_spans

def pack_spans(seq_offsets, span_start, span_len, seq_span_offsets, pi,
               packed_offsets, packed_src, err, total_tokens: int,
               token_ids=None, emb=None, surrogates=None, packed=None, stream=None):
    B = seq_offsets.numel() - 1
    S = span_start.numel()
    d = emb.shape[1] if emb is not None else 0
    dt = dtype_code(emb.dtype) if emb is not None else SM_BF16
    st = load().sm_pack_spans(B, _ptr(seq_offsets), total_tokens, S, _ptr(span_start),
                              _ptr(span_len), _ptr(seq_span_offsets), _ptr(pi),
                              _ptr(packed_offsets), _ptr(packed_src), _ptr(token_ids),
                              _ptr(emb), emb.shape[0] if emb is not None else 0,
                              _ptr(surrogates), d, dt, _ptr(packed), _ptr(err),
                              _stream(stream))
    _check(st, "sm_pack_spans")


# --------------------------------------------------------------------------
# paged cache

class PagedCache:
    """Device buffers of one paged KV cache (allocated with torch) and the
    descriptor the C calls take.  Pools: K [NB, Hkv, bs, D], V [NB, Hkv, D, bs]."""

    def __init__(self, *, dtype: torch.dtype, num_kv_heads: int, head_dim: int,
                 block_size: int, num_blocks: int, max_seqs: int,
                 max_blocks_per_seq: int, device="cuda", free_order=None):
        self.dtype = dtype
        self.H, self.D, self.bs = num_kv_heads, head_dim, block_size
        self.num_blocks, self.max_seqs, self.max_blocks = num_blocks, max_seqs, max_blocks_per_seq
        self.k_pool = torch.zeros((num_blocks, num_kv_heads, block_size, head_dim), dtype=dtype, device=device)
        self.v_pool = torch.zeros((num_blocks, num_kv_heads, head_dim, block_size), dtype=dtype, device=device)
        self.block_table = torch.full((max_seqs, max_blocks_per_seq), -1, dtype=torch.int32, device=device)
        self.lengths = torch.zeros(max_seqs, dtype=torch.int32, device=device)
        order = (torch.arange(num_blocks, dtype=torch.int32) if free_order is None
                 else torch.as_tensor(free_order, dtype=torch.int32))
        # the top of the stack (last element) is handed out first
        self.free_stack = order.flip(0).contiguous().to(device)
        self.free_top = torch.tensor([num_blocks], dtype=torch.int32, device=device)
        self.err = torch.zeros(1, dtype=torch.int32, device=device)
        self.desc = PagedCacheDesc(dtype_code(dtype), num_kv_heads, head_dim, block_size,
                                   num_blocks, max_seqs, max_blocks_per_seq,
                                   _ptr(self.k_pool), _ptr(self.v_pool), _ptr(self.block_table),
                                   _ptr(self.lengths), _ptr(self.free_stack), _ptr(self.free_top),
                                   _ptr(self.err))

    def error_bits(self) -> int:
        return int(self.err.item())

    def clear_error(self):
        self.err.zero_()


def kv_rollback(cache: PagedCache, seq_ids, k, stream=None):
    st = load().sm_kv_rollback(C.byref(cache.desc), _ptr(seq_ids), _ptr(k), seq_ids.numel(),
                               _stream(stream))
    _check(st, "sm_kv_rollback")


def kv_append(cache: PagedCache, seq_ids, row_offsets, K, V, total_rows: Optional[int] = None,
              stream=None):
    R = K.shape[0] if total_rows is None else total_rows
    st = load().sm_kv_append(C.byref(cache.desc), _ptr(seq_ids), _ptr(row_offsets),
                             seq_ids.numel(), R, _ptr(K), _ptr(V), _stream(stream))
    _check(st, "sm_kv_append")


def decode_workspace_bytes(n: int, num_q_heads: int, head_dim: int, max_len: int) -> int:
    return load().sm_decode_workspace_bytes(n, num_q_heads, head_dim, max_len)


def decode_attention(cache: PagedCache, seq_ids, q, out, ws, max_len: int,
                     scale: Optional[float] = None, stream=None):
    n, Hq, D = q.shape
    sc = D ** -0.5 if scale is None else scale
    st = load().sm_decode_attention(C.byref(cache.desc), _ptr(seq_ids), n, _ptr(q), Hq, sc,
                                    max_len, _ptr(out), _ptr(ws),
                                    ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "sm_decode_attention")


def decode_step(cache: PagedCache, seq_ids, K, V, q, out, ws, max_len: int,
                scale: Optional[float] = None, stream=None):
    """Append one K/V row per sequence and attend, in one launch: the same
    as kv_append(cache, seq_ids, arange(n + 1), K, V) then decode_attention."""
    n, Hq, D = q.shape
    sc = D ** -0.5 if scale is None else scale
    st = load().sm_decode_step(C.byref(cache.desc), _ptr(seq_ids), n, _ptr(K), _ptr(V), _ptr(q), Hq, sc,
                               max_len, _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                               _stream(stream))
    _check(st, "sm_decode_step")


def decode_merge_step(cache: PagedCache, seq_ids, crop, K, V, q, out, ws, max_len: int,
                      scale: Optional[float] = None, stream=None):
    """The decode step at which spans complete: drop crop[i] cached entries
    of each request, append its row and attend, in one launch (the same as
    kv_rollback(cache, seq_ids, crop) then decode_step, made whole or not at
    all)."""
    n, Hq, D = q.shape
    sc = D ** -0.5 if scale is None else scale
    st = load().sm_decode_merge_step(C.byref(cache.desc), _ptr(seq_ids), _ptr(crop), n, _ptr(K), _ptr(V), _ptr(q),
                                     Hq, sc, max_len, _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                     _stream(stream))
    _check(st, "sm_decode_merge_step")


def decode_step_noalloc(cache: PagedCache, seq_ids, K, V, q, out, max_len: int,
                        scale: Optional[float] = None, stream=None):
    """decode_step with the library's own per-device scratch array as its
    workspace (no allocation in the call; calls on one device must not
    overlap)."""
    n, Hq, D = q.shape
    sc = D ** -0.5 if scale is None else scale
    st = load().sm_decode_step_noalloc(C.byref(cache.desc), _ptr(seq_ids), n, _ptr(K), _ptr(V), _ptr(q), Hq, sc,
                                       max_len, _ptr(out), _stream(stream))
    _check(st, "sm_decode_step_noalloc")


def prefill_attention(cache: PagedCache, seq_ids, q_offsets, q, out, max_rows: int,
                      scale: Optional[float] = None, stream=None):
    """Causal attention of each request's last m_i cached positions:
    q, out [rows, Hq, D] bf16; q_offsets [n + 1] int32 row ranges."""
    rows, Hq, D = q.shape
    sc = D ** -0.5 if scale is None else scale
    st = load().sm_prefill_attention(C.byref(cache.desc), _ptr(seq_ids), seq_ids.numel(), _ptr(q_offsets), rows,
                                     _ptr(q), Hq, sc, max_rows, _ptr(out), _stream(stream))
    _check(st, "sm_prefill_attention")


# --------------------------------------------------------------------------
# merge rules

class RuleTable:
    """Device buffers of the rule hash table (allocated with torch) and its
    descriptor.  capacity: a power of two >= 4/3 x the number of rules."""

    def __init__(self, capacity: int, device="cuda"):
        self.capacity = capacity
        self.keys = torch.full((capacity, 4), -1, dtype=torch.int32, device=device)
        self.ids = torch.full((capacity,), -1, dtype=torch.int32, device=device)
        self.err = torch.zeros(1, dtype=torch.int32, device=device)
        self.desc = RuleTableDesc(capacity, _ptr(self.keys), _ptr(self.ids), _ptr(self.err))

    @staticmethod
    def capacity_for(count: int) -> int:
        c = 16
        while 3 * c < 4 * count:
            c *= 2
        return c

    def error_bits(self) -> int:
        return int(self.err.item())

    def clear_error(self):
        self.err.zero_()


def rules_build(table: RuleTable, rules, ws=None, stream=None):
    """rules: [count, 4] int32 on the GPU (n >= 2 ids, then -1)."""
    need = load().sm_rules_build_workspace_bytes(table.capacity)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=rules.device)
    st = load().sm_rules_build(_ptr(rules), rules.shape[0], C.byref(table.desc), _ptr(ws),
                               ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "sm_rules_build")


def rules_lookup(table: RuleTable, grams, ids, stream=None):
    st = load().sm_rules_lookup(C.byref(table.desc), _ptr(grams), grams.shape[0], _ptr(ids), _stream(stream))
    _check(st, "sm_rules_lookup")


def match_prompt_workspace_bytes(B: int, total_tokens: int) -> int:
    return load().sm_match_prompt_workspace_bytes(B, total_tokens)


def match_prompt(table: RuleTable, token_ids, seq_offsets, span_start, span_len, span_rule,
                 seq_span_offsets, ws, stream=None):
    B = seq_offsets.numel() - 1
    st = load().sm_match_prompt(C.byref(table.desc), _ptr(token_ids), _ptr(seq_offsets), B, token_ids.numel(),
                                _ptr(span_start), _ptr(span_len), _ptr(span_rule), _ptr(seq_span_offsets),
                                _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "sm_match_prompt")


def match_decode(table: RuleTable, state, seq_ids, new_tokens, k_out, rule_out,
                 cache: Optional[PagedCache] = None, stream=None):
    """state [max_seqs, 4] int32 (zeroed when a sequence starts generating)."""
    st = load().sm_match_decode(C.byref(table.desc), _ptr(state), state.shape[0], _ptr(seq_ids),
                                _ptr(new_tokens), seq_ids.numel(), _ptr(k_out), _ptr(rule_out),
                                None if cache is None else C.byref(cache.desc), _stream(stream))
    _check(st, "sm_match_decode")


# --------------------------------------------------------------------------
# surrogate lookup and span dedupe

def gather_surrogates(lut, rule_ids, out, err, emb=None, token_ids=None, stream=None):
    """out[i] = lut[rule_ids[i]] if rule_ids[i] >= 0 else emb[token_ids[i]]."""
    n, d = out.shape
    st = load().sm_gather_surrogates(_ptr(emb), 0 if emb is None else emb.shape[0], _ptr(lut), lut.shape[0],
                                     _ptr(token_ids), _ptr(rule_ids), n, d, dtype_code(out.dtype), _ptr(out),
                                     _ptr(err), _stream(stream))
    _check(st, "sm_gather_surrogates")


def span_dedupe(span_rule, span_start, span_len, num_rules, token_ids, uniq_span, span_slot, uniq_row_idx,
                uniq_span_offsets, num_uniq, err, ws=None, stream=None):
    S = span_rule.numel()
    need = load().sm_span_dedupe_workspace_bytes(S, num_rules)
    if ws is None:
        ws = torch.empty(need, dtype=torch.uint8, device=span_rule.device)
    st = load().sm_span_dedupe(_ptr(span_rule), _ptr(span_start), _ptr(span_len), S, num_rules, _ptr(token_ids),
                               token_ids.numel(), _ptr(uniq_span), _ptr(span_slot), _ptr(uniq_row_idx),
                               _ptr(uniq_span_offsets), _ptr(num_uniq), _ptr(ws), ws.numel() * ws.element_size(),
                               _ptr(err), _stream(stream))
    _check(st, "sm_span_dedupe")


# --------------------------------------------------------------------------
# K/V state of an input row at its compressed position

def _proj_params(W_k, W_v, rope_theta, rms_eps):
    return KVProjParams(W_k.shape[1], _ptr(W_k), _ptr(W_v), rope_theta, rms_eps)


def kv_project_workspace_bytes(n: int, d: int, num_kv_heads: int, head_dim: int) -> int:
    return load().sm_kv_project_workspace_bytes(n, d, num_kv_heads, head_dim)


def kv_project(cache: PagedCache, seq_ids, x, W_k, W_v, K, V, ws=None, rope_theta=500000.0, rms_eps=1e-5,
               stream=None):
    """K, V [n, Hkv, D] bf16 of the rows x [n, d] at positions lengths[seq_ids]."""
    n = seq_ids.numel()
    if ws is None:
        ws = torch.empty(kv_project_workspace_bytes(n, x.shape[1], cache.H, cache.D), dtype=torch.uint8,
                         device=x.device)
    p = _proj_params(W_k, W_v, rope_theta, rms_eps)
    st = load().sm_kv_project(C.byref(cache.desc), _ptr(seq_ids), n, _ptr(x), C.byref(p), _ptr(K), _ptr(V),
                              _ptr(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "sm_kv_project")


def kv_append_projected(cache: PagedCache, seq_ids, x, W_k, W_v, ws=None, rope_theta=500000.0, rms_eps=1e-5,
                        stream=None):
    n = seq_ids.numel()
    if ws is None:
        ws = torch.empty(kv_project_workspace_bytes(n, x.shape[1], cache.H, cache.D), dtype=torch.uint8,
                         device=x.device)
    p = _proj_params(W_k, W_v, rope_theta, rms_eps)
    st = load().sm_kv_append_projected(C.byref(cache.desc), _ptr(seq_ids), n, _ptr(x), C.byref(p), _ptr(ws),
                                       ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "sm_kv_append_projected")
