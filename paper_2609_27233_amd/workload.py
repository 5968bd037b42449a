"""Seeded synthetic workloads for the span-merging hot path.

This module only draws inputs: token ids, span layouts, merge-module
parameters, K/V rows and queries.  It holds none of the method's arithmetic,
and both the GPU path and the CPU oracle receive exactly the arrays it
returns.  Integer structure is drawn with numpy on the host; floating tensors
are drawn with torch generators on the requested device (the oracle then gets
an exact float64 copy).

The five workloads stand in for the paper's data (WikiText-103 segments,
long documents, a controlled merge ratio for throughput): spans are laid out
like the left-to-right non-overlapping assignment of the prompt-merging
procedure, with lengths and reduction ratios matching the paper's operating
points ("up to 40%" effective-length reduction, 2-8 token spans).
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    dtype: str                    # "f32" or "bf16"
    d: int                        # model width (also the merge module's)
    h: int                        # merge-module pooling heads
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    batch: int
    prompt_len: Optional[int]     # fixed prompt length, or None
    ctx_range: Optional[tuple]    # (lo, hi) uniform context lengths, or None
    vocab: int
    span_n: tuple                 # allowed span lengths
    span_law: str                 # "uniform" or "inv" (P(n) ~ 1/(n-1))
    target_kind: Optional[str]    # "coverage" | "reduction" | None
    target: float
    block_size: int
    shuffled_pages: bool
    decode_steps: int
    merge_every: int              # decode-time merge cadence (0 = never)
    merge_n: tuple                # decode-time span lengths n (k = n - 1)
    seed: int

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def group(self):
        return self.num_q_heads // self.num_kv_heads


WORKLOADS = {
    1: Workload(1, "tiny-f32-d256-B1-T512", "f32", 256, 4, 4, 4, 64, 1, 512,
                None, 1000, (2, 3, 4), "uniform", "coverage", 0.30, 512,
                False, 1, 0, (2, 3, 4), 1001),
    2: Workload(2, "llama3-8b-layer-B16-T4096", "bf16", 4096, 4, 32, 8, 128,
                16, 4096, None, 128256, tuple(range(2, 9)), "inv",
                "reduction", 0.40, 16, False, 256, 8, (2, 3, 4), 1002),
    3: Workload(3, "llama3-8b-layer-B4-T32768-shuffled", "bf16", 4096, 4, 32,
                8, 128, 4, 32768, None, 128256, tuple(range(2, 9)), "inv",
                "reduction", 0.40, 16, True, 128, 8, (2, 3, 4), 1003),
    4: Workload(4, "qwen2-7b-layer-B128-ctx512-4096", "bf16", 3584, 4, 28, 4,
                128, 128, None, (512, 4096), 152064, (), "uniform", None, 0.0,
                16, False, 256, 4, (3, 4, 5), 1004),
    5: Workload(5, "llama3-70b-layer-B32-T8192", "bf16", 8192, 4, 64, 8, 128,
                32, 8192, None, 128256, tuple(range(2, 9)), "inv",
                "reduction", 0.40, 16, False, 64, 0, (2, 3, 4), 1005),
}


# --------------------------------------------------------------------------
# span layouts

def _span_probs(ns: Sequence[int], law: str) -> np.ndarray:
    ns = np.asarray(ns, dtype=np.float64)
    w = np.ones_like(ns) if law == "uniform" else 1.0 / (ns - 1.0)
    return w / w.sum()


def draw_span_lengths(rng: np.random.RandomState, ns, law, kind, amount):
    """Span lengths whose removed positions sum(n - 1) (kind="reduction") or
    covered tokens sum(n) (kind="coverage") equal ``amount`` exactly."""
    ns = list(ns)
    p = _span_probs(ns, law)
    lens = []
    cum = 0
    cost = (lambda n: n - 1) if kind == "reduction" else (lambda n: n)
    while cum < amount:
        n = int(rng.choice(ns, p=p))
        if cum + cost(n) > amount:
            rem = amount - cum
            n = rem + 1 if kind == "reduction" else rem
            if n < min(ns):
                # coverage left a single token: lengthen an earlier span
                for i in range(len(lens) - 1, -1, -1):
                    if lens[i] < max(ns):
                        lens[i] += rem
                        break
                else:
                    raise ValueError("cannot place spans exactly")
                cum += rem
                continue
        lens.append(n)
        cum += cost(n)
    return lens


def layout_spans(rng: np.random.RandomState, T: int, lens: Sequence[int]):
    """Place spans of the given lengths (in order) at random non-overlapping
    positions of a T-token sequence; returns sorted (starts, lens)."""
    lens = np.asarray(lens, dtype=np.int64)
    S = len(lens)
    free = T - int(lens.sum())
    if free < 0:
        raise ValueError("spans do not fit")
    # uniform random composition of `free` gap tokens into S + 1 gaps
    cuts = np.sort(rng.choice(free + S, size=S, replace=False)) if S else np.zeros(0, np.int64)
    gaps = np.diff(np.concatenate([[-1], cuts, [free + S]])) - 1
    starts = np.zeros(S, dtype=np.int64)
    pos = 0
    for i in range(S):
        pos += int(gaps[i])
        starts[i] = pos
        pos += int(lens[i])
    return starts.astype(np.int32), lens.astype(np.int32)


@dataclasses.dataclass
class Prompts:
    """Batch of prompts with their merge spans (global token indices)."""
    token_ids: np.ndarray         # [sum T] int32
    seq_offsets: np.ndarray       # [B + 1]
    span_start: np.ndarray        # [S] global token index
    span_len: np.ndarray          # [S]
    seq_span_offsets: np.ndarray  # [B + 1]

    @property
    def row_idx(self):
        """Embedding rows of every span token, spans back to back (CSR)."""
        idx = np.concatenate([np.arange(s, s + n) for s, n in
                              zip(self.span_start, self.span_len)]) if len(self.span_len) else np.zeros(0, np.int64)
        return self.token_ids[idx].astype(np.int32)

    @property
    def span_offsets(self):
        return np.concatenate([[0], np.cumsum(self.span_len)]).astype(np.int32)


def make_prompts(w: Workload, seed: Optional[int] = None, batch: Optional[int] = None,
                 prompt_len: Optional[int] = None) -> Prompts:
    rng = np.random.RandomState(w.seed if seed is None else seed)
    B = w.batch if batch is None else batch
    T = w.prompt_len if prompt_len is None else prompt_len
    toks, starts, lens, sso = [], [], [], [0]
    base = 0
    for _ in range(B):
        toks.append(rng.randint(0, w.vocab, size=T).astype(np.int32))
        if w.target_kind is None:
            st, ln = np.zeros(0, np.int32), np.zeros(0, np.int32)
        else:
            amount = int(round(w.target * T))
            ls = draw_span_lengths(rng, w.span_n, w.span_law, w.target_kind, amount)
            rng.shuffle(ls)
            st, ln = layout_spans(rng, T, ls)
        starts.append(st + base)
        lens.append(ln)
        sso.append(sso[-1] + len(ln))
        base += T
    return Prompts(
        token_ids=np.concatenate(toks).astype(np.int32),
        seq_offsets=(np.arange(B + 1) * T).astype(np.int32),
        span_start=np.concatenate(starts).astype(np.int32),
        span_len=np.concatenate(lens).astype(np.int32),
        seq_span_offsets=np.asarray(sso, dtype=np.int32))


# --------------------------------------------------------------------------
# merge rules: a synthetic stand-in for the rule set mined from WikiText-103

# 2-, 3- and 4-gram rules kept for the Llama-3 tokenizer (the paper's
# rule-count table, threshold tau = 5)
RULE_COUNTS_LLAMA3 = (216_700, 684_793, 1_266_080)


def make_rules(counts=RULE_COUNTS_LLAMA3, vocab: int = 128256, seed: int = 7) -> np.ndarray:
    """Distinct uniform random n-grams, counts[n - 2] of each n in 2..4, as
    [sum(counts), 4] int32 (unused tail -1), in shuffled order."""
    rng = np.random.RandomState(seed)
    out = []
    for n, c in zip((2, 3, 4), counts):
        got = np.zeros((0, n), np.int64)
        while len(got) < c:
            draw = np.concatenate([got, rng.randint(0, vocab, size=(int((c - len(got)) * 1.05) + 16, n))])
            rows = np.ascontiguousarray(draw).view(np.dtype((np.void, 8 * n))).ravel()
            _, first = np.unique(rows, return_index=True)          # distinct rows
            got = draw[np.sort(first)]
        got = got[rng.permutation(len(got))[:c]]
        pad = np.full((c, 4), -1, np.int64)
        pad[:, :n] = got
        out.append(pad)
    rules = np.concatenate(out) if out else np.zeros((0, 4), np.int64)
    return rules[rng.permutation(len(rules))].astype(np.int32)


def make_rule_prompts(rules: np.ndarray, B: int, T: int, removal: float, vocab: int, seed: int,
                      zipf_a: Optional[float] = None):
    """B prompts of T tokens: uniform random ids with randomly chosen rules
    planted at random non-overlapping places until sum(n - 1) reaches
    removal x T (the last rule may overshoot by up to 2).  Rules are drawn
    uniformly, or with zipf_a by a Zipf law over the rule list's order (a
    stand-in for n-gram frequencies of real text).  Returns
    (token_ids [B T] int32, seq_offsets [B + 1] int32)."""
    rng = np.random.RandomState(seed)
    n_of = (rules >= 0).sum(1)
    toks = rng.randint(0, vocab, size=B * T).astype(np.int32)
    target = int(round(removal * T))
    for b in range(B):
        picked, cost = [], 0
        while cost < target and len(rules):
            r = int(rng.randint(len(rules))) if zipf_a is None else int(rng.zipf(zipf_a) - 1) % len(rules)
            picked.append(r)
            cost += int(n_of[r]) - 1
        starts, _ = layout_spans(rng, T, n_of[picked])
        for st, r in zip(starts, picked):
            toks[b * T + st:b * T + st + n_of[r]] = rules[r, :n_of[r]]
    return toks, (np.arange(B + 1) * T).astype(np.int32)


# --------------------------------------------------------------------------
# floating tensors

def generator(seed: int, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def randn(shape, dtype, gen, device="cpu", std=1.0, mean=0.0):
    """Normal draws in fp32, then rounded once to the storage dtype."""
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mean != 0.0:
        x.add_(mean)
    return x.to(dtype)


PARAM_NAMES = ("Q", "W_kv", "b_kv", "g_kv", "beta_kv", "W_o", "b_o", "g_o", "beta_o")


def make_merge_params(d: int, h: int, dtype, gen, device="cpu", std=0.02,
                      spread: bool = False):
    """Random-init merge-module parameters.  Default: Q, W, b ~ N(0, std^2)
    with LayerNorm gain 1 and bias 0.  ``spread=True`` draws the LayerNorm
    affine terms too and a unit-variance Q, so pooling weights are far from
    uniform (used by the parity tests)."""
    dh = d // h
    p = {
        "Q": randn((h, dh), dtype, gen, device, std=1.0 if spread else std),
        "W_kv": randn((d, d), dtype, gen, device, std=std),
        "b_kv": randn((d,), dtype, gen, device, std=std),
        "W_o": randn((d, d), dtype, gen, device, std=std),
        "b_o": randn((d,), dtype, gen, device, std=std),
    }
    if spread:
        p["g_kv"] = randn((d,), dtype, gen, device, std=0.1, mean=1.0)
        p["beta_kv"] = randn((d,), dtype, gen, device, std=0.1)
        p["g_o"] = randn((d,), dtype, gen, device, std=0.1, mean=1.0)
        p["beta_o"] = randn((d,), dtype, gen, device, std=0.1)
    else:
        p["g_kv"] = torch.ones(d, dtype=dtype, device=device)
        p["beta_kv"] = torch.zeros(d, dtype=dtype, device=device)
        p["g_o"] = torch.ones(d, dtype=dtype, device=device)
        p["beta_o"] = torch.zeros(d, dtype=dtype, device=device)
    return p


def context_lengths(w: Workload, seed: Optional[int] = None) -> np.ndarray:
    """Per-sequence cached lengths for workloads without prompt spans."""
    rng = np.random.RandomState((w.seed if seed is None else seed) + 7)
    lo, hi = w.ctx_range
    return rng.randint(lo, hi + 1, size=w.batch).astype(np.int32)


def free_order(num_blocks: int, shuffled: bool, seed: int) -> np.ndarray:
    """Order in which physical blocks are handed out by the free stack."""
    if not shuffled:
        return np.arange(num_blocks, dtype=np.int32)
    return np.random.RandomState(seed + 11).permutation(num_blocks).astype(np.int32)


def decode_merge_lengths(w: Workload, step: int, seed: Optional[int] = None) -> np.ndarray:
    """Span length n per sequence for a decode-time merge at ``step``."""
    rng = np.random.RandomState(((w.seed if seed is None else seed) * 1009 + step) % (2 ** 31))
    return rng.choice(np.asarray(w.merge_n), size=w.batch).astype(np.int32)


# --------------------------------------------------------------------------
# raw-storage views for the oracle

def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact float64 copy of a fp32 / bf16 tensor."""
    return t.detach().to("cpu", torch.float64).numpy()


def to_raw(t: torch.Tensor) -> np.ndarray:
    """Storage bit pattern: uint16 for bf16, float32 for fp32."""
    t = t.detach().to("cpu").contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy().astype(np.float32, copy=False)


def from_raw(a: np.ndarray, device="cpu") -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)
