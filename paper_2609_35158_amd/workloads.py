"""Seeded synthetic inputs for paged-KV attention workloads.

This module only builds inputs: sequence lengths, a randomly permuted page
pool, block tables, and bf16 Q/K/V drawn from N(0, 1).  It performs none of
the attention arithmetic, and both the HIP path and the CPU oracle consume the
same bytes produced here.

The workload shapes follow the paper's setting: multi-turn agentic rollout in
which each turn appends new tokens to a growing context (Background, the
p_{t+1} = p_t + r_t + o_t recurrence), served with prefix caching and chunked
prefill batched with decode (Motivation, PD colocation), on Qwen3-8B and
Qwen3-30B-A3B attention shapes (Evaluation setup: group 16, batch 64, 32K
maximum trajectory).  All sizes below are synthetic stand-ins; no benchmark
content is used.

Conventions shared with the library (the boundary, not the method):
  * page size 16 tokens; token position p lives in logical page p // 16,
    slot p % 16 (standard paged semantics);
  * K and V pools are bf16 [num_pages][H_kv][16][d];
  * q / k_new / v_new are bf16 [total_q][H][d]; lengths are int32.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np
import torch

PAGE = 16


@dataclasses.dataclass
class Case:
    """One synthetic batch.  Tensors live on ``device``; lengths also on host."""

    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    ctx_lens: np.ndarray          # int32 [B] tokens already cached
    q_lens: np.ndarray            # int32 [B] new tokens this call
    block_table: torch.Tensor     # int32 [B][bt_stride]
    k_pool: torch.Tensor          # bf16 [num_pages][H_kv][16][d] (context filled)
    v_pool: torch.Tensor
    k_new: torch.Tensor           # bf16 [total_q][H_kv][d]
    v_new: torch.Tensor
    q: torch.Tensor               # bf16 [total_q][H_q][d]
    scale: float                  # fp32 softmax scale 1/sqrt(d)
    extra: Dict[str, object] = dataclasses.field(default_factory=dict)

    @property
    def batch(self) -> int:
        return int(self.ctx_lens.shape[0])

    @property
    def cu_q_lens(self) -> np.ndarray:
        cu = np.zeros(self.batch + 1, dtype=np.int32)
        cu[1:] = np.cumsum(self.q_lens)
        return cu

    @property
    def total_q(self) -> int:
        return int(self.q_lens.sum())

    @property
    def kv_lens(self) -> np.ndarray:
        return (self.ctx_lens + self.q_lens).astype(np.int32)

    @property
    def num_pages(self) -> int:
        return int(self.k_pool.shape[0])


def _fill_normal_bf16(shape, gen: torch.Generator, device, chunk_elems: int = 1 << 27) -> torch.Tensor:
    """N(0,1) float32 draws rounded to bf16 (torch's conversion is round-to-nearest-even).

    Drawn in chunks so host memory stays bounded for multi-GB pools."""
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        flat[s:e] = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
    return out


def _sentinel_fill(t: torch.Tensor, value_bits: int = 0x7FC1) -> None:
    """Fill with a NaN bit pattern so stray reads/writes are visible."""
    t.view(torch.int16).fill_(np.int16(np.uint16(value_bits).view(np.int16)))


def build_case(name: str, seed: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
               ctx_lens, q_lens, device="cpu", pool_pages: Optional[int] = None,
               sentinel_unused: bool = True, extra_pages: int = 0,
               shared_prefix_groups: int = 0) -> Case:
    """Generic builder.

    Order of draws (fixed): page permutation (numpy PCG64 on ``seed``), then on a
    torch generator seeded with ``seed``: K pool, V pool, k_new, v_new, q.

    Pages: every sequence b owns ceil((ctx+q)/16) logical pages; physical ids are
    a random permutation of the pool assigned in (sequence, logical page) order.
    Pages not owned by any sequence are sentinel-filled (NaN pattern).
    Context slots (positions < ctx) hold N(0,1) bf16; slots at positions >= ctx
    (where this call's tokens will be appended, and unused tails) are sentinel.
    """
    ctx = np.asarray(ctx_lens, dtype=np.int64)
    ql = np.asarray(q_lens, dtype=np.int64)
    B = ctx.shape[0]
    assert ql.shape[0] == B
    kv = ctx + ql
    pages_per_seq = (kv + PAGE - 1) // PAGE
    need = int(pages_per_seq.sum())
    num_pages = need + extra_pages if pool_pages is None else int(pool_pages)
    assert num_pages >= need
    rng = np.random.default_rng(seed)
    perm = rng.permutation(num_pages).astype(np.int32)
    bt_stride = max(1, int(pages_per_seq.max()) if B else 1)
    bt = np.zeros((B, bt_stride), dtype=np.int32)
    owned = np.zeros(num_pages, dtype=bool)
    pos = 0
    for b in range(B):
        n = int(pages_per_seq[b])
        bt[b, :n] = perm[pos:pos + n]
        owned[perm[pos:pos + n]] = True
        pos += n
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    H_kv, d = num_kv_heads, head_dim
    k_pool = _fill_normal_bf16((num_pages, H_kv, PAGE, d), gen, device)
    v_pool = _fill_normal_bf16((num_pages, H_kv, PAGE, d), gen, device)
    # Positions >= ctx are not yet written: mark them (and unowned pages) with sentinels.
    bt_t = torch.from_numpy(bt).to(device)
    if sentinel_unused:
        if (~owned).any():
            idx = torch.from_numpy(np.nonzero(~owned)[0]).to(device)
            _sentinel_fill_rows(k_pool, idx)
            _sentinel_fill_rows(v_pool, idx)
        for b in range(B):
            c, n = int(ctx[b]), int(pages_per_seq[b])
            first = c // PAGE
            if first >= n:
                continue
            # partial page: slots c%16.. of logical page `first`; then whole pages after it
            pg = int(bt[b, first])
            s0 = c % PAGE
            _sentinel_fill(k_pool[pg, :, s0:, :])
            _sentinel_fill(v_pool[pg, :, s0:, :])
            if first + 1 < n:
                idx = bt_t[b, first + 1:n].long()
                _sentinel_fill_rows(k_pool, idx)
                _sentinel_fill_rows(v_pool, idx)
    total_q = int(ql.sum())
    k_new = _fill_normal_bf16((total_q, H_kv, d), gen, device)
    v_new = _fill_normal_bf16((total_q, H_kv, d), gen, device)
    q = _fill_normal_bf16((total_q, num_q_heads, d), gen, device)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    return Case(name=name, seed=seed, num_q_heads=num_q_heads, num_kv_heads=H_kv, head_dim=d,
                ctx_lens=ctx.astype(np.int32), q_lens=ql.astype(np.int32), block_table=bt_t,
                k_pool=k_pool, v_pool=v_pool, k_new=k_new, v_new=v_new, q=q, scale=scale)


def _sentinel_fill_rows(pool: torch.Tensor, idx: torch.Tensor) -> None:
    sub = torch.empty((idx.numel(),) + tuple(pool.shape[1:]), dtype=pool.dtype, device=pool.device)
    _sentinel_fill(sub)
    pool.index_copy_(0, idx.to(pool.device), sub)


# ----------------------------------------------------------------------------------------------
# Named workloads.  Integer draws are uniform on inclusive ranges; lognormal lengths are rounded
# to the nearest integer and then clipped.
# ----------------------------------------------------------------------------------------------

def tiny_prefill(device="cpu") -> Case:
    """2 sequences with cached contexts of 100 and 37 tokens; 4 q-heads, 2 kv-heads (GQA 2), d=64;
    a 32-page pool, randomly permuted.  The turn appends 20 tokens per sequence (causal
    prefill-append); ``extra`` holds 8 further single-token decode steps (q, k, v per step, shape
    [2][H][d]).  Pages are owned for the final lengths 128 and 65 (8 + 5 = 13 of 32 pages); the
    other 19 pages stay sentinel-filled."""
    ctx = np.array([100, 37])
    n_turn, n_dec = 20, 8
    full = build_case("tiny", 0, 4, 2, 64, ctx, np.full(2, n_turn + n_dec), device=device, pool_pages=32)
    per = n_turn + n_dec
    turn_rows = np.concatenate([np.arange(b * per, b * per + n_turn) for b in range(2)])
    sel = torch.from_numpy(turn_rows).to(device)
    dec_q, dec_k, dec_v = [], [], []
    for t in range(n_dec):
        rows = torch.from_numpy(np.array([b * per + n_turn + t for b in range(2)])).to(device)
        dec_q.append(full.q[rows].contiguous())
        dec_k.append(full.k_new[rows].contiguous())
        dec_v.append(full.v_new[rows].contiguous())
    full.q = full.q[sel].contiguous()
    full.k_new = full.k_new[sel].contiguous()
    full.v_new = full.v_new[sel].contiguous()
    full.q_lens = np.full(2, n_turn, dtype=np.int32)
    full.extra.update(decode_q=dec_q, decode_k=dec_k, decode_v=dec_v)
    return full


def qwen3_8b_decode(device="cpu", batch=64, seed=1, lo=2048, hi=16384, num_q_heads=32,
                    num_kv_heads=8) -> Case:
    """Qwen3-8B attention shape (32 q-heads, 8 kv-heads, d=128); `batch` sequences with cached
    contexts uniform in [lo, hi]; one new token each; pool sized to the total context.  With
    16 q-heads and 4 kv-heads it is one GPU's share under tensor parallelism 2 (same lengths and
    page placement)."""
    rng = np.random.default_rng(seed + 1_000_003)
    ctx = rng.integers(lo, hi, size=batch, endpoint=True)
    name = "qwen3-8b-decode" if (num_q_heads, num_kv_heads) == (32, 8) else \
        "qwen3-8b-decode-h%d-%d" % (num_q_heads, num_kv_heads)
    return build_case(name, seed, num_q_heads, num_kv_heads, 128, ctx, np.ones(batch, np.int64), device=device)


def qwen3_8b_prefill_append(device="cpu", batch=16, seed=2, ctx_lo=4096, ctx_hi=24576,
                            n_lo=256, n_hi=2048) -> Case:
    """Qwen3-8B shape; `batch` sequences with cached context uniform in [ctx_lo, ctx_hi] and a new
    turn chunk uniform in [n_lo, n_hi] tokens (causal within the chunk, full attention to the
    context).  The chunk goes into randomly placed pages after the context."""
    rng = np.random.default_rng(seed + 1_000_003)
    ctx = rng.integers(ctx_lo, ctx_hi, size=batch, endpoint=True)
    ql = rng.integers(n_lo, n_hi, size=batch, endpoint=True)
    return build_case("qwen3-8b-prefill-append", seed, 32, 8, 128, ctx, ql, device=device)


def lognormal_lengths(rng: np.random.Generator, n: int, median: float, sigma: float,
                      lo: int, hi: int) -> np.ndarray:
    x = rng.lognormal(mean=math.log(median), sigma=sigma, size=n)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


def qwen3_30b_decode(device="cpu", batch=256, seed=None, median=6144, sigma=0.75,
                     lo=1024, hi=32768) -> Case:
    """Qwen3-30B-A3B attention shape (32 q-heads, 4 kv-heads, GQA 8, d=128); lognormal cached
    context (median 6144, sigma 0.75, clipped to [1024, 32768]); one new token per sequence."""
    if seed is None:
        seed = {256: 40, 128: 41, 32: 42}.get(batch, 43)
    rng = np.random.default_rng(seed + 1_000_003)
    ctx = lognormal_lengths(rng, batch, median, sigma, lo, hi)
    case = build_case("qwen3-30b-a3b-decode-b%d" % batch, seed, 32, 4, 128, ctx,
                      np.ones(batch, np.int64), device=device)
    case.extra["sigma"] = sigma
    return case


def mixed_colocated(device="cpu", seed=5, n_prefill=8, chunk=512, prefill_ctx=8192,
                    n_decode=192, dec_lo=2048, dec_hi=32768) -> Case:
    """Colocated batch on the Qwen3-30B-A3B shape: `n_prefill` chunks of `chunk` new tokens on
    `prefill_ctx`-token contexts, then `n_decode` single-token decodes with contexts uniform in
    [dec_lo, dec_hi]; one shared randomly permuted pool."""
    rng = np.random.default_rng(seed + 1_000_003)
    dctx = rng.integers(dec_lo, dec_hi, size=n_decode, endpoint=True)
    ctx = np.concatenate([np.full(n_prefill, prefill_ctx), dctx])
    ql = np.concatenate([np.full(n_prefill, chunk), np.ones(n_decode, np.int64)])
    case = build_case("mixed-colocated", seed, 32, 4, 128, ctx, ql, device=device)
    case.extra["n_prefill"] = n_prefill
    return case


def sub_batch(case: Case, seqs, q_lens=None, name: Optional[str] = None) -> Case:
    """A batch made of some sequences of ``case``, sharing its pools: sequence ``seqs[i]`` keeps its
    cached context and block-table row and takes the first ``q_lens[i]`` of its new tokens (all of
    them when ``q_lens`` is None).  Used to sweep batch composition over one generated pool."""
    dev = case.q.device
    seqs = np.asarray(seqs, dtype=np.int64)
    full = case.q_lens[seqs].astype(np.int64)
    ql = full if q_lens is None else np.asarray(q_lens, dtype=np.int64)
    assert ql.shape == full.shape and np.all(ql >= 0) and np.all(ql <= full)
    cu = case.cu_q_lens
    parts = [np.arange(cu[b], cu[b] + n) for b, n in zip(seqs, ql)]
    rows = torch.from_numpy(np.concatenate(parts) if parts else np.zeros(0, np.int64)).to(dev)
    return Case(name=name or case.name + "-sub", seed=case.seed, num_q_heads=case.num_q_heads,
                num_kv_heads=case.num_kv_heads, head_dim=case.head_dim,
                ctx_lens=case.ctx_lens[seqs].astype(np.int32), q_lens=ql.astype(np.int32),
                block_table=case.block_table.index_select(0, torch.from_numpy(seqs).to(dev)).contiguous(),
                k_pool=case.k_pool, v_pool=case.v_pool,
                k_new=case.k_new.index_select(0, rows).contiguous(),
                v_new=case.v_new.index_select(0, rows).contiguous(),
                q=case.q.index_select(0, rows).contiguous(), scale=case.scale)


def random_small(seed: int, device="cpu", batch=None, H_kv=None, G=None, d=None,
                 max_ctx=300, max_q=40, decode_only=False, allow_zero_q=False) -> Case:
    """Small random shapes for fuzzing: ragged contexts (including 0) and chunk lengths."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 5)) if batch is None else batch
    H_kv = int(rng.choice([1, 2, 4])) if H_kv is None else H_kv
    G = int(rng.choice([1, 2, 4, 8])) if G is None else G
    d = int(rng.choice([64, 128])) if d is None else d
    ctx = rng.integers(0, max_ctx, size=B, endpoint=True)
    if decode_only:
        ql = np.ones(B, np.int64)
    else:
        ql = rng.integers(0 if allow_zero_q else 1, max_q, size=B, endpoint=True)
    # keep at least one key visible per sequence with new tokens
    return build_case("random-small", seed, H_kv * G, H_kv, d, ctx, ql, device=device,
                      extra_pages=int(rng.integers(0, 4)))
