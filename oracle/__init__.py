"""CPU oracle of the span-merging inference hot path (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  It wraps ``liboracle.so`` (plain C, double
precision, OpenMP) with ctypes and numpy; it never imports the GPU package
and the GPU package never imports it.  Inputs reach both sides only through
the seeded generators.

Floating inputs are passed as float64 (bf16 and fp32 values widen exactly);
cache pools hold raw storage elements (uint16 bf16 bit patterns or float32)
so that copies compare bit for bit.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
# a test may point the wrapper at another build of the same source (the
# sanitized one); nothing else sets this
_LIB_OVERRIDE = os.environ.get("ORACLE_LIB")

OK, EINVAL, ERANGE, ENOMEM = 0, 1, 2, 3


_CFLAGS = ["-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(force: bool = True) -> str:
    """Compile liboracle.so next to its source (gcc, -O2, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", *_CFLAGS, _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def build_sanitized(path: str) -> str:
    """Compile the same source with AddressSanitizer and UndefinedBehavior-
    Sanitizer (host code, gcc; any finding aborts) into ``path``.  A process
    loads it through ORACLE_LIB with libasan preloaded."""
    cmd = ["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", *_CFLAGS, _SRC, "-o", path, "-lm"]
    subprocess.run(cmd, check=True)
    return path


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            _lib = C.CDLL(_LIB_OVERRIDE)
            _declare(_lib)
            return _lib
        if not os.path.exists(_LIB_PATH):
            build()
        _lib = C.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


_P = C.c_void_p
_I = C.c_int
_L = C.c_int64
_D = C.c_double


class _Cache(C.Structure):
    _fields_ = [("is_bf16", _I), ("num_kv_heads", _I), ("head_dim", _I),
                ("block_size", _I), ("num_blocks", _I), ("max_seqs", _I),
                ("max_blocks_per_seq", _I), ("k_pool", _P), ("v_pool", _P),
                ("block_table", _P), ("lengths", _P), ("free_stack", _P),
                ("free_top", _P)]


class _Rules(C.Structure):
    _fields_ = [("count", _I), ("keys", _P), ("ids", _P)]


def _declare(L):
    L.orc_merge_spans.argtypes = [_I, _I, _D, _P, _L, _P, _P, _I, _P, _P, _P,
                                  _P, _P, _P, _P, _P, _P, _I, _P, _P, _I]
    L.orc_merge_spans.restype = _I
    L.orc_pack_spans.argtypes = [_I, _P, _I, _P, _P, _P, _P, _P, _P, _P, _P,
                                 _L, _P, _I, _I, _P]
    L.orc_pack_spans.restype = _I
    L.orc_kv_rollback.argtypes = [C.POINTER(_Cache), _P, _P, _I]
    L.orc_kv_rollback.restype = _I
    L.orc_kv_append.argtypes = [C.POINTER(_Cache), _P, _P, _I, _P, _P]
    L.orc_kv_append.restype = _I
    L.orc_decode_attention.argtypes = [C.POINTER(_Cache), _P, _I, _P, _I, _D,
                                       _P, _P, _I]
    L.orc_decode_attention.restype = _I
    L.orc_prefill_attention.argtypes = [C.POINTER(_Cache), _P, _I, _P, _P, _I, _D, _P]
    L.orc_prefill_attention.restype = _I
    L.orc_layer_qkv.argtypes = [_I, _I, _P, _P, _I, _I, _I, _D, _D, _P, _P,
                                _P, _P, _P, _P]
    L.orc_layer_qkv.restype = None
    L.orc_rules_init.argtypes = [C.POINTER(_Rules), _P, _I]
    L.orc_rules_init.restype = _I
    L.orc_rules_free.argtypes = [C.POINTER(_Rules)]
    L.orc_rules_free.restype = None
    L.orc_rules_find.argtypes = [C.POINTER(_Rules), _P, _I]
    L.orc_rules_find.restype = _I
    L.orc_match_prompt.argtypes = [C.POINTER(_Rules), _I, _P, _P, _P, _P, _P, _P]
    L.orc_match_prompt.restype = _I
    L.orc_match_decode_step.argtypes = [C.POINTER(_Rules), _P, C.POINTER(_I), C.c_int32, C.POINTER(C.c_int32),
                                        C.POINTER(C.c_int32)]
    L.orc_match_decode_step.restype = None
    L.orc_gather_surrogates.argtypes = [_P, _L, _P, _L, _P, _P, _I, _I, _I, _P]
    L.orc_gather_surrogates.restype = _I
    L.orc_span_dedupe.argtypes = [_P, _P, _P, _I, _I, _P, _P, _P, _P, _P]
    L.orc_span_dedupe.restype = _I
    L.orc_kv_project.argtypes = [C.POINTER(_Cache), _P, _I, _P, _I, _P, _P, _D, _D, _P, _P]
    L.orc_kv_project.restype = _I
    L.orc_num_threads.argtypes = []
    L.orc_num_threads.restype = _I
    L.orc_set_num_threads.argtypes = [_I]
    L.orc_set_num_threads.restype = None


def _ptr(a):
    return None if a is None else a.ctypes.data


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def num_threads() -> int:
    return lib().orc_num_threads()


def set_num_threads(n: int) -> None:
    lib().orc_set_num_threads(int(n))


# --------------------------------------------------------------------------
# merge module

PARAM_NAMES = ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o",
               "beta_o")


def merge_spans(emb, row_idx, span_offsets, params, h, ln_eps=1e-5, flags=0,
                return_weights=False):
    """M_phi for every span; returns float64 [S, d] (and pooling weights
    [S, h, max_n] when asked).  ``params`` maps PARAM_NAMES to arrays."""
    emb = _f64(emb)
    d = emb.shape[1]
    row_idx = _i32(row_idx)
    span_offsets = _i32(span_offsets)
    S = span_offsets.shape[0] - 1
    p = {k: _f64(params[k]) for k in PARAM_NAMES}
    out = np.zeros((max(S, 0), d), dtype=np.float64)
    n_max = int(np.max(np.diff(span_offsets))) if S > 0 else 1
    w = np.zeros((max(S, 0), h, n_max)) if return_weights else None
    st = lib().orc_merge_spans(
        d, h, ln_eps, _ptr(emb), emb.shape[0], _ptr(row_idx),
        _ptr(span_offsets), S, *(_ptr(p[k]) for k in PARAM_NAMES), flags,
        _ptr(out), _ptr(w), n_max)
    if return_weights:
        return st, out, w
    return st, out


def _gelu_erf(x):
    from scipy.special import erf
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def _layer_norm_rows(x, g, b, eps):
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)          # biased variance
    return g * (x - mean) / np.sqrt(var + eps) + b


def merge_spans_rows(emb, row_idx, span_offsets, params, h, ln_eps=1e-5):
    """The same M_phi as merge_spans (appendix "Attention-based Pooling
    Architecture"), for large calls: each of the two Linear layers is applied
    to every row of the call as one float64 matrix product (each row's
    Linear_kv, and each span's Linear_o, is independent of the others), so
    the d x d weights stream once per call instead of once per row.  GELU,
    LayerNorm over all d features and the per-head learned-query pooling
    (P as key and value, scale 1/sqrt(d_h), head-major concatenation) follow
    the definition element by element.  Returns float64 [S, d]."""
    emb = np.asarray(emb, np.float64)
    row_idx = _i32(row_idx)
    offs = _i32(span_offsets)
    p = {k: np.asarray(params[k], np.float64) for k in PARAM_NAMES}
    d = emb.shape[1]
    dh = d // h
    S = len(offs) - 1
    if S <= 0:
        return np.zeros((0, d))
    E = emb[row_idx]                                                # [R, d]
    P = _layer_norm_rows(_gelu_erf(E @ p["W_kv"].T + p["b_kv"]), p["g_kv"], p["beta_kv"], ln_eps)
    lens = np.diff(offs)
    nmax = int(lens.max())
    # spans padded to nmax rows; padded rows take no weight
    idx = offs[:-1, None] + np.arange(nmax)[None, :]                 # [S, nmax]
    valid = np.arange(nmax)[None, :] < lens[:, None]
    Pp = P[np.where(valid, idx, 0)].reshape(S, nmax, h, dh)         # [S, nmax, h, dh]
    sc = np.einsum("snhk,hk->snh", Pp, p["Q"]) / np.sqrt(dh)
    sc = np.where(valid[:, :, None], sc, -np.inf)
    sc = sc - sc.max(axis=1, keepdims=True)
    a = np.exp(sc)
    a = a / a.sum(axis=1, keepdims=True)                            # softmax over the span's rows
    c = np.einsum("snh,snhk->shk", a, Pp).reshape(S, d)             # concat in head order
    Y = _gelu_erf(c @ p["W_o"].T + p["b_o"])
    return _layer_norm_rows(Y, p["g_o"], p["beta_o"], ln_eps)


# --------------------------------------------------------------------------
# prompt packing

def pack_spans(seq_offsets, span_start, span_len, seq_span_offsets,
               token_ids=None, emb_raw=None, surrogates_raw=None):
    """Returns (status, dict(pi, packed_offsets, packed_src, packed)).
    ``emb_raw`` / ``surrogates_raw`` are raw-storage arrays (uint16 for bf16,
    float32 for fp32) of shape [rows, d]; packed rows are byte copies."""
    seq_offsets = _i32(seq_offsets)
    B = seq_offsets.shape[0] - 1
    total = int(seq_offsets[-1])
    span_start, span_len = _i32(span_start), _i32(span_len)
    seq_span_offsets = _i32(seq_span_offsets)
    S = span_start.shape[0]
    pi = np.full(total, -7, dtype=np.int32)
    packed_offsets = np.full(B + 1, -7, dtype=np.int32)
    packed_src = np.full(total, -7, dtype=np.int32)
    packed = None
    d, eb, emb_rows = 0, 0, 0
    if emb_raw is not None:
        emb_raw = np.ascontiguousarray(emb_raw)
        surrogates_raw = np.ascontiguousarray(surrogates_raw)
        token_ids = _i32(token_ids)
        d = emb_raw.shape[1]
        eb = emb_raw.dtype.itemsize
        emb_rows = emb_raw.shape[0]
        packed = np.zeros((total, d), dtype=emb_raw.dtype)
    st = lib().orc_pack_spans(
        B, _ptr(seq_offsets), S, _ptr(span_start), _ptr(span_len),
        _ptr(seq_span_offsets), _ptr(pi), _ptr(packed_offsets),
        _ptr(packed_src), _ptr(token_ids), _ptr(emb_raw), emb_rows,
        _ptr(surrogates_raw), d, eb, _ptr(packed))
    res = dict(pi=pi, packed_offsets=packed_offsets, packed_src=packed_src)
    if st == OK:
        n = int(packed_offsets[-1])
        res["packed_src"] = packed_src[:n].copy()
        if packed is not None:
            res["packed"] = packed[:n].copy()
    return st, res


# --------------------------------------------------------------------------
# paged KV cache

class OracleCache:
    """Paged cache held in numpy arrays, driven by the C oracle."""

    def __init__(self, *, bf16, num_kv_heads, head_dim, block_size,
                 num_blocks, max_seqs, max_blocks_per_seq, free_order=None):
        self.is_bf16 = bool(bf16)
        self.H, self.D, self.bs = num_kv_heads, head_dim, block_size
        self.num_blocks, self.max_seqs = num_blocks, max_seqs
        self.max_blocks = max_blocks_per_seq
        dt = np.uint16 if bf16 else np.float32
        self.k_pool = np.zeros((num_blocks, num_kv_heads, block_size, head_dim), dtype=dt)
        self.v_pool = np.zeros((num_blocks, num_kv_heads, head_dim, block_size), dtype=dt)
        self.block_table = np.full((max_seqs, max_blocks_per_seq), -1, dtype=np.int32)
        self.lengths = np.zeros(max_seqs, dtype=np.int32)
        # the stack pops from the top: free_stack[top-1] is handed out first
        order = np.arange(num_blocks, dtype=np.int32) if free_order is None else _i32(free_order)
        self.free_stack = order[::-1].copy()
        self.free_top = np.array([num_blocks], dtype=np.int32)

    def _struct(self):
        return _Cache(int(self.is_bf16), self.H, self.D, self.bs,
                      self.num_blocks, self.max_seqs, self.max_blocks,
                      _ptr(self.k_pool), _ptr(self.v_pool),
                      _ptr(self.block_table), _ptr(self.lengths),
                      _ptr(self.free_stack), _ptr(self.free_top))

    def rollback(self, seq_ids, k):
        seq_ids, k = _i32(seq_ids), _i32(k)
        s = self._struct()
        return lib().orc_kv_rollback(C.byref(s), _ptr(seq_ids), _ptr(k), seq_ids.shape[0])

    def append(self, seq_ids, row_offsets, K, V):
        """K, V: raw-storage arrays [rows, H, D] (uint16 bf16 bits or float32)."""
        seq_ids, row_offsets = _i32(seq_ids), _i32(row_offsets)
        dt = np.uint16 if self.is_bf16 else np.float32
        K = np.ascontiguousarray(K, dtype=dt)
        V = np.ascontiguousarray(V, dtype=dt)
        s = self._struct()
        return lib().orc_kv_append(C.byref(s), _ptr(seq_ids), _ptr(row_offsets),
                                   seq_ids.shape[0], _ptr(K), _ptr(V))

    def crop_append(self, seq_ids, k, K, V):
        """The decode-time merge update of the cache ("Decoding-Time Merging
        and KV-Cache Update"): request i drops its last k[i] entries, then
        its one row K[i], V[i] is appended (L -> L - k + 1).  The two steps
        are rollback() and append() as they stand, taken as one update: if
        either fails, every array is put back as it was and that step's
        status is returned."""
        saved = [a.copy() for a in (self.lengths, self.block_table, self.free_stack, self.free_top,
                                    self.k_pool, self.v_pool)]
        n = len(seq_ids)
        st = self.rollback(seq_ids, k)
        if st == OK:
            st = self.append(seq_ids, np.arange(n + 1, dtype=np.int32), K, V)
        if st != OK:
            for a, b in zip((self.lengths, self.block_table, self.free_stack, self.free_top,
                             self.k_pool, self.v_pool), saved):
                a[...] = b
        return st

    def decode_attention(self, seq_ids, q, num_q_heads, scale, return_probs=False):
        seq_ids = _i32(seq_ids)
        q = _f64(q)
        n = seq_ids.shape[0]
        out = np.zeros((n, num_q_heads, self.D))
        probs = None
        stride = 1
        if return_probs:
            stride = max(1, int(self.lengths[seq_ids].max()) if n else 1)
            probs = np.zeros((n, num_q_heads, stride))
        s = self._struct()
        st = lib().orc_decode_attention(C.byref(s), _ptr(seq_ids), n, _ptr(q),
                                        num_q_heads, scale, _ptr(out), _ptr(probs), stride)
        if return_probs:
            return st, out, probs
        return st, out

    def prefill_attention(self, seq_ids, q_offsets, q, num_q_heads, scale):
        """Causal attention of each request's last m_i cached positions;
        q [rows, Hq, D] (any float), returns (status, out [rows, Hq, D])."""
        seq_ids, q_offsets = _i32(seq_ids), _i32(q_offsets)
        q = _f64(q)
        out = np.zeros(q.shape)
        s = self._struct()
        st = lib().orc_prefill_attention(C.byref(s), _ptr(seq_ids), seq_ids.shape[0],
                                         _ptr(q_offsets), _ptr(q), num_q_heads, scale, _ptr(out))
        return st, out

    def kv_project(self, seq_ids, x, W_k, W_v, rope_theta=500000.0, rms_eps=1e-5):
        """(status, K, V) [n, H, D]: the rows' K/V at position lengths[s]."""
        seq_ids, x = _i32(seq_ids), _f64(x)
        n, d = x.shape
        K = np.zeros((n, self.H, self.D))
        V = np.zeros((n, self.H, self.D))
        s = self._struct()
        st = lib().orc_kv_project(C.byref(s), _ptr(seq_ids), n, _ptr(x), d, _ptr(_f64(W_k)), _ptr(_f64(W_v)),
                                  rope_theta, rms_eps, _ptr(K), _ptr(V))
        return st, K, V

    # logical view helpers (pure indexing, used by tests)
    def logical_kv(self, s):
        """Raw K [L, H, D] and V [L, H, D] of sequence s in cache order."""
        L = int(self.lengths[s])
        j = np.arange(L)
        blk = self.block_table[s, j // self.bs]
        slot = j % self.bs
        K = self.k_pool[blk, :, slot, :]
        V = self.v_pool[blk, :, :, slot]
        return K, V


# --------------------------------------------------------------------------
# test-only layer input side

def layer_qkv(x, pos, W_q, W_k, W_v, num_q_heads, num_kv_heads, head_dim,
              rope_theta=500000.0, rms_eps=1e-5):
    x = _f64(x)
    T, d = x.shape
    pos = _i32(pos)
    q = np.zeros((T, num_q_heads, head_dim))
    k = np.zeros((T, num_kv_heads, head_dim))
    v = np.zeros((T, num_kv_heads, head_dim))
    lib().orc_layer_qkv(T, d, _ptr(x), _ptr(pos), num_q_heads, num_kv_heads,
                        head_dim, rope_theta, rms_eps, _ptr(_f64(W_q)),
                        _ptr(_f64(W_k)), _ptr(_f64(W_v)), _ptr(q), _ptr(k), _ptr(v))
    return q, k, v


# --------------------------------------------------------------------------
# merge rules and matching

MERGED = -2  # a surrogate in the decode-time generated-state list


def rule_keys(grams):
    """[m, 4] int32 keys of n-grams given as sequences (unused tail -1)."""
    out = np.full((len(grams), 4), -1, dtype=np.int32)
    for i, g in enumerate(grams):
        out[i, :len(g)] = g
    return out


class OracleRules:
    """The rule set R (sorted, searched by bisection) and the two matching
    procedures of the appendix."""

    def __init__(self, keys):
        self.keys_in = _i32(np.asarray(keys).reshape(-1, 4))
        self._r = _Rules()
        self.status = lib().orc_rules_init(C.byref(self._r), _ptr(self.keys_in), self.keys_in.shape[0])
        self._states = {}

    def __del__(self):
        try:
            lib().orc_rules_free(C.byref(self._r))
        except Exception:
            pass

    @property
    def count(self):
        return self._r.count

    def find(self, gram):
        g = _i32(gram)
        return lib().orc_rules_find(C.byref(self._r), _ptr(g), g.shape[0])

    def match_prompt(self, token_ids, seq_offsets):
        """(status, span_start, span_len, span_rule, seq_span_offsets)."""
        tok, so = _i32(token_ids), _i32(seq_offsets)
        B = so.shape[0] - 1
        cap = max(int(so[-1]) // 2, 1)
        st_, ln, ru = (np.zeros(cap, np.int32) for _ in range(3))
        sso = np.zeros(B + 1, np.int32)
        st = lib().orc_match_prompt(C.byref(self._r), B, _ptr(so), _ptr(tok), _ptr(st_), _ptr(ln), _ptr(ru),
                                    _ptr(sso))
        S = int(sso[-1])
        return st, st_[:S].copy(), ln[:S].copy(), ru[:S].copy(), sso

    def decode_step(self, seq, token):
        """Feed one generated token of sequence `seq`; returns (k, rule id)."""
        buf, n = self._states.get(seq, (np.zeros(16, np.int32), 0))
        if n + 1 > buf.shape[0]:
            nb = np.zeros(2 * buf.shape[0], np.int32)
            nb[:n] = buf[:n]
            buf = nb
        ln = C.c_int(n)
        k, rule = C.c_int32(0), C.c_int32(-1)
        lib().orc_match_decode_step(C.byref(self._r), _ptr(buf), C.byref(ln), int(token), C.byref(k),
                                    C.byref(rule))
        self._states[seq] = (buf, ln.value)
        return k.value, rule.value

    def state(self, seq):
        buf, n = self._states.get(seq, (np.zeros(0, np.int32), 0))
        return buf[:n].copy()


# --------------------------------------------------------------------------
# surrogate lookup and span dedupe

def gather_surrogates(emb, lut, token_ids, rule_ids):
    """out[i] = lut[rule_ids[i]] if rule_ids[i] >= 0 else emb[token_ids[i]];
    emb, lut: raw element arrays [rows, d] of one dtype.  (status, out)."""
    emb, lut = np.ascontiguousarray(emb), np.ascontiguousarray(lut)
    rule_ids = _i32(rule_ids)
    tok = None if token_ids is None else _i32(token_ids)
    n, d = rule_ids.shape[0], lut.shape[1]
    out = np.zeros((n, d), dtype=lut.dtype)
    st = lib().orc_gather_surrogates(_ptr(emb), emb.shape[0], _ptr(lut), lut.shape[0], _ptr(tok),
                                     _ptr(rule_ids), n, d, lut.dtype.itemsize, _ptr(out))
    return st, out


def span_dedupe(span_rule, span_start, span_len, num_rules, token_ids):
    """(U, uniq_span [U], span_slot [S], uniq_row_idx, uniq_span_offsets [U+1])."""
    r, st_, ln, tok = _i32(span_rule), _i32(span_start), _i32(span_len), _i32(token_ids)
    S = r.shape[0]
    us, slot = np.zeros(max(S, 1), np.int32), np.zeros(max(S, 1), np.int32)
    rows = np.zeros(max(int(ln.sum()), 1), np.int32)
    offs = np.zeros(S + 1, np.int32)
    U = lib().orc_span_dedupe(_ptr(r), _ptr(st_), _ptr(ln), S, num_rules, _ptr(tok), _ptr(us), _ptr(slot),
                              _ptr(rows), _ptr(offs))
    if U < 0:
        return U, None, None, None, None
    return U, us[:U].copy(), slot[:S].copy(), rows[:offs[U]].copy(), offs[:U + 1].copy()
