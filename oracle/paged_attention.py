"""CPU oracle for paged-KV GQA attention (append, prefill-append, decode, mixed).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that the HIP
library is checked against.  Only tests, the smoke check and the benchmark's CPU
baseline may import it; the library never calls it and it shares no code with
the library (it imports numpy and nothing else).

What is computed, and where the paper fixes it
----------------------------------------------
* Multi-turn rollout grows each trajectory's context by appending the previous
  response and the new environment observation to the prompt (Background,
  section "Agentic RL and Asynchronous Training": p_{t+1} = p_t + r_t + o_t).
  Serving engines keep the K/V of the already-processed prefix (prefix caching,
  Motivation section "Efficiency Degradation under PD Colocation") and only the
  new tokens are prefilled (Evaluation, "Scale-in recovery"; Related work,
  "append-prefill").  The new tokens' K/V are appended to the cache
  (`kv_append`), then the new tokens attend causally within the chunk and fully
  to the cached prefix (`attention`).
* Decode is the same function with one new token per sequence; its per-sequence
  marginal cost is the KV-cache read (section 4.3, Eq. 1, the term b).
* Chunked prefill is batched with decode on one GPU under PD colocation
  (Motivation, same section; section 4.3, Eq. 1): a mixed batch is a batch in
  which each sequence has its own number of new tokens.

The paper prints no attention formula; the function below is standard scaled
dot-product attention with grouped-query heads.  The readings taken where the
paper is silent (inclusive causal mask, contiguous GQA grouping q-head h ->
kv-head h // G, softmax scale passed in as fp32, natural-log LSE, page p // 16 and
slot p % 16 for token position p) are listed with the design notes.

Precision: inputs are bf16 bit patterns (uint16); they are widened exactly to
float64 and every product, sum, exp and division is float64.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

PAGE = 16


# ------------------------------------------------------------------------------------------
# bf16 <-> float64
# ------------------------------------------------------------------------------------------

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening: a bf16 value is the upper 16 bits of the float32 with the same value."""
    b = np.ascontiguousarray(bits).view(np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 to the nearest bf16, ties to even, in one step from the float64 bits (no
    intermediate float32 rounding).  Values outside bf16's normal range go through float32.
    Used only to report results in bf16 units."""
    x = np.asarray(x, dtype=np.float64)
    u = x.view(np.uint64)
    sign = (u >> np.uint64(63)).astype(np.uint64)
    e64 = ((u >> np.uint64(52)) & np.uint64(0x7FF)).astype(np.int64)
    # keep 7 of the 52 mantissa bits: round-half-even on the dropped 45 bits
    mag = u & np.uint64(0x7FFFFFFFFFFFFFFF)
    keep_lsb = (mag >> np.uint64(45)) & np.uint64(1)
    r = (mag + np.uint64((1 << 44) - 1) + keep_lsb) >> np.uint64(45)   # 11-bit exp + 7-bit mant
    e_r = (r >> np.uint64(7)).astype(np.int64)
    mant = (r & np.uint64(0x7F)).astype(np.uint64)
    e_bf = e_r - 1023 + 127
    out = ((sign << np.uint64(15)) | (np.clip(e_bf, 0, 255).astype(np.uint64) << np.uint64(7)) | mant)
    out = out.astype(np.uint16)
    normal = (e64 > 0) & (e_bf >= 1) & (e_bf <= 254)
    zero = (mag == 0)
    out[zero] = (sign[zero] << np.uint64(15)).astype(np.uint16)
    other = ~(normal | zero)
    if other.any():
        f32 = x[other].astype(np.float32).view(np.uint32)
        out[other] = ((f32 + np.uint32(0x7FFF) + ((f32 >> 16) & 1)) >> 16).astype(np.uint16)
    return out


# ------------------------------------------------------------------------------------------
# Paged addressing (standard paged semantics: position p -> logical page p // 16, slot p % 16)
# ------------------------------------------------------------------------------------------

def _page_slot(block_table_row: np.ndarray, positions: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    return block_table_row[positions // PAGE], positions % PAGE


def _kv_head_of(h: int, group: int) -> int:
    """Contiguous grouped-query mapping: q-heads [g*G, (g+1)*G) share kv-head g."""
    return h // group


def _visible(ctx_len: int, i: int) -> int:
    """Number of keys visible to new token i of a sequence whose cache held ctx_len tokens:
    its absolute position is ctx_len + i and the causal mask is inclusive (keys 0..pos)."""
    return ctx_len + i + 1


def _q_lens(cu_q_lens: Optional[np.ndarray], batch: int) -> np.ndarray:
    if cu_q_lens is None:
        return np.ones(batch, dtype=np.int64)
    cu = np.asarray(cu_q_lens, dtype=np.int64)
    return cu[1:] - cu[:-1]


def _q_starts(cu_q_lens: Optional[np.ndarray], batch: int) -> np.ndarray:
    if cu_q_lens is None:
        return np.arange(batch, dtype=np.int64)
    return np.asarray(cu_q_lens, dtype=np.int64)[:-1]


# ------------------------------------------------------------------------------------------
# kv_append: a bit copy of each new token's K and V rows into (page, slot)
# ------------------------------------------------------------------------------------------

def kv_append(k_pool: np.ndarray, v_pool: np.ndarray, k_new: np.ndarray, v_new: np.ndarray,
              block_table: np.ndarray, ctx_lens: np.ndarray,
              cu_q_lens: Optional[np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """Return copies of the pools after appending the new tokens.

    For sequence b and new token t (absolute position ctx_lens[b] + t), the K row of
    kv-head h is written to k_pool[page, h, slot, :] with (page, slot) from the block
    table; V likewise.  Pools are uint16 [num_pages][H_kv][16][d]; k_new / v_new are
    uint16 [total_q][H_kv][d].  Nothing else changes."""
    kp = np.array(k_pool, dtype=np.uint16, copy=True)
    vp = np.array(v_pool, dtype=np.uint16, copy=True)
    B = len(ctx_lens)
    ql = _q_lens(cu_q_lens, B)
    qs = _q_starts(cu_q_lens, B)
    for b in range(B):
        for t in range(int(ql[b])):
            pos = int(ctx_lens[b]) + t
            page = int(block_table[b][pos // PAGE])
            slot = pos % PAGE
            kp[page, :, slot, :] = k_new[qs[b] + t]
            vp[page, :, slot, :] = v_new[qs[b] + t]
    return kp, vp


# ------------------------------------------------------------------------------------------
# KV transfer between pools (PD disaggregation: the prefill pool hands each turn's new-token
# K/V to the decode pool; section 4.3, Eq. 3, the B * dL * K / BW transfer term)
# ------------------------------------------------------------------------------------------

def kv_pack(k_pool: np.ndarray, v_pool: np.ndarray, block_table: np.ndarray, ctx_lens: np.ndarray,
            cu_q_lens: Optional[np.ndarray]) -> np.ndarray:
    """Gather token rows out of the pools into a contiguous transfer buffer.

    For sequence b the rows of positions ctx_lens[b] .. ctx_lens[b] + n_b - 1 (n_b from
    cu_q_lens; one row each when it is None) go to buffer rows cu_q_lens[b] + t, for every
    kv-head.  Returns uint16 [2][total][H_kv][d]: K rows, then V rows."""
    B = len(ctx_lens)
    ql = _q_lens(cu_q_lens, B)
    qs = _q_starts(cu_q_lens, B)
    total = int(ql.sum())
    H_kv, d = k_pool.shape[1], k_pool.shape[3]
    buf = np.zeros((2, total, H_kv, d), dtype=np.uint16)
    for b in range(B):
        row = np.asarray(block_table[b])
        for t in range(int(ql[b])):
            page, slot = _page_slot(row, np.int64(int(ctx_lens[b]) + t))
            buf[0, qs[b] + t] = k_pool[int(page), :, int(slot), :]
            buf[1, qs[b] + t] = v_pool[int(page), :, int(slot), :]
    return buf


def kv_unpack(k_pool: np.ndarray, v_pool: np.ndarray, buf: np.ndarray, block_table: np.ndarray,
              ctx_lens: np.ndarray, cu_q_lens: Optional[np.ndarray]) -> Tuple[np.ndarray, np.ndarray]:
    """Scatter a transfer buffer (as made by kv_pack) into pools with their own block table:
    the append of its K half and V half at positions ctx_lens[b] + t."""
    return kv_append(k_pool, v_pool, buf[0], buf[1], block_table, ctx_lens, cu_q_lens)


# ------------------------------------------------------------------------------------------
# attention over the paged cache
# ------------------------------------------------------------------------------------------

def gather_kv(k_pool: np.ndarray, v_pool: np.ndarray, block_table_row: np.ndarray,
              kv_len: int, kv_head: int) -> Tuple[np.ndarray, np.ndarray]:
    """Explicit per-key gather of keys 0..kv_len-1 of one sequence and kv-head, float64 [kv_len][d]."""
    pos = np.arange(kv_len, dtype=np.int64)
    pages, slots = _page_slot(np.asarray(block_table_row, dtype=np.int64), pos)
    K = bf16_bits_to_f64(k_pool[pages, kv_head, slots, :])
    V = bf16_bits_to_f64(v_pool[pages, kv_head, slots, :])
    return K, V


def attention_unit(q_rows: np.ndarray, K: np.ndarray, V: np.ndarray, ctx_len: int,
                   scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Attention of the new tokens of one sequence for one q-head.

    q_rows: float64 [n][d] (new token i sits at position ctx_len + i); K, V: float64 [kv][d].
    For token i the visible keys are 0..ctx_len+i.  Returns (o [n][d], lse [n]):
      s_j = scale * q.k_j;  m = max_j s_j;  w_j = exp(s_j - m);  l = sum_j w_j;
      o = (sum_j w_j v_j) / l;  lse = m + ln l."""
    n = q_rows.shape[0]
    d = K.shape[1]
    o = np.empty((n, d), dtype=np.float64)
    lse = np.empty(n, dtype=np.float64)
    # rows are processed in blocks to keep the score matrix small; each row uses only its
    # own visible prefix (explicit slicing, no mask arithmetic)
    for i in range(n):
        vis = _visible(ctx_len, i)
        s = scale * (K[:vis] @ q_rows[i])
        m = s.max()
        w = np.exp(s - m)
        l = w.sum()
        o[i] = (w @ V[:vis]) / l
        lse[i] = m + math.log(l)
    return o, lse


def attention(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray, block_table: np.ndarray,
              ctx_lens: np.ndarray, cu_q_lens: Optional[np.ndarray], scale: float,
              seqs: Optional[Sequence[int]] = None, heads: Optional[Sequence[int]] = None,
              tokens: Optional[dict] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Paged GQA attention of every new token (prefill-append, decode and mixed batches alike).

    q: uint16 [total_q][H_q][d]; pools uint16 [num_pages][H_kv][16][d] AFTER the append (the
    new tokens' own K/V are in the cache); block_table int32 [B][*]; ctx_lens [B] = tokens
    cached before this call's tokens; cu_q_lens [B+1] prefix sums of new tokens, or None for
    one token per sequence.  `scale` is the float32 value the library receives.

    Returns float64 (o [total_q][H_q][d], lse [total_q][H_q]); entries of sequences/heads not
    selected by `seqs` / `heads` (or, per sequence b, new-token indices not in `tokens[b]`)
    are NaN."""
    q = np.asarray(q)
    total_q, H_q, d = q.shape
    H_kv = k_pool.shape[1]
    assert H_q % H_kv == 0
    G = H_q // H_kv
    B = len(ctx_lens)
    ql = _q_lens(cu_q_lens, B)
    qs = _q_starts(cu_q_lens, B)
    scale = float(np.float32(scale))
    o = np.full((total_q, H_q, d), np.nan)
    lse = np.full((total_q, H_q), np.nan)
    seqs = range(B) if seqs is None else seqs
    heads = range(H_q) if heads is None else heads
    for b in seqs:
        n = int(ql[b])
        if n == 0:
            continue
        L = int(ctx_lens[b])
        by_kv = {}
        for h in heads:
            by_kv.setdefault(_kv_head_of(h, G), []).append(h)
        for g, hs in by_kv.items():
            K, V = gather_kv(k_pool, v_pool, block_table[b], L + n, g)
            sel = list(range(n)) if tokens is None or b not in tokens else list(tokens[b])
            for h in hs:
                for i in sel:
                    row = bf16_bits_to_f64(q[qs[b] + i, h, :])[None, :]
                    vis = _visible(L, i)
                    ob, lb = attention_unit(row, K[:vis], V[:vis], vis - 1, scale)
                    o[qs[b] + i, h, :] = ob[0]
                    lse[qs[b] + i, h] = lb[0]
    return o, lse


# ------------------------------------------------------------------------------------------
# split-context form: partial softmax states over key ranges, merged by log-sum-exp
# ------------------------------------------------------------------------------------------

def partial_state(q_row: np.ndarray, K: np.ndarray, V: np.ndarray, lo: int, hi: int,
                  scale: float) -> Tuple[np.ndarray, float, float]:
    """Softmax state of one query over keys [lo, hi): (unnormalised o~ = sum w_j v_j, m, l)
    with w_j = exp(s_j - m), m the range maximum.  An empty range is (0, -inf, 0)."""
    if hi <= lo:
        return np.zeros(K.shape[1]), -math.inf, 0.0
    s = scale * (K[lo:hi] @ q_row)
    m = float(s.max())
    w = np.exp(s - m)
    return w @ V[lo:hi], m, float(w.sum())


def merge_states(states: List[Tuple[np.ndarray, float, float]]) -> Tuple[np.ndarray, float]:
    """m* = max m_s;  l* = sum l_s e^{m_s - m*};  o = sum e^{m_s - m*} o~_s / l*;  lse = m* + ln l*."""
    m_star = max(m for _, m, _ in states)
    l_star = sum(l * math.exp(m - m_star) for _, m, l in states if l > 0)
    acc = sum(o * math.exp(m - m_star) for o, m, l in states if l > 0)
    return acc / l_star, m_star + math.log(l_star)


def attention_split(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray, block_table: np.ndarray,
                    ctx_lens: np.ndarray, cu_q_lens: Optional[np.ndarray], scale: float,
                    bounds_for: "callable") -> Tuple[np.ndarray, np.ndarray]:
    """Same result as `attention`, computed by splitting each query's visible keys into the ranges
    given by ``bounds_for(b, i, visible)`` (a sorted list of cut points inside (0, visible)) and
    merging the partial states."""
    total_q, H_q, d = q.shape
    H_kv = k_pool.shape[1]
    G = H_q // H_kv
    B = len(ctx_lens)
    ql = _q_lens(cu_q_lens, B)
    qs = _q_starts(cu_q_lens, B)
    scale = float(np.float32(scale))
    o = np.full((total_q, H_q, d), np.nan)
    lse = np.full((total_q, H_q), np.nan)
    for b in range(B):
        n = int(ql[b])
        L = int(ctx_lens[b])
        for g in range(H_kv):
            if n == 0:
                continue
            K, V = gather_kv(k_pool, v_pool, block_table[b], L + n, g)
            for h in range(g * G, (g + 1) * G):
                for i in range(n):
                    vis = _visible(L, i)
                    cuts = [0] + list(bounds_for(b, i, vis)) + [vis]
                    qr = bf16_bits_to_f64(q[qs[b] + i, h, :])
                    st = [partial_state(qr, K, V, cuts[k], cuts[k + 1], scale) for k in range(len(cuts) - 1)]
                    o[qs[b] + i, h], lse[qs[b] + i, h] = merge_states(st)
    return o, lse


# ------------------------------------------------------------------------------------------
# a second, independent formulation for brute-force cross-checks on tiny inputs
# ------------------------------------------------------------------------------------------

def attention_scalar_loops(q, k_pool, v_pool, block_table, ctx_lens, cu_q_lens, scale):
    """Pure-Python scalar loops (math.exp, no numpy reductions).  Only for tiny inputs."""
    total_q, H_q, d = q.shape
    H_kv = k_pool.shape[1]
    G = H_q // H_kv
    B = len(ctx_lens)
    ql = _q_lens(cu_q_lens, B)
    qs = _q_starts(cu_q_lens, B)
    scale = float(np.float32(scale))
    qf = bf16_bits_to_f64(q)
    kf = bf16_bits_to_f64(k_pool)
    vf = bf16_bits_to_f64(v_pool)
    o = np.full((total_q, H_q, d), np.nan)
    lse = np.full((total_q, H_q), np.nan)
    for b in range(B):
        for i in range(int(ql[b])):
            row = int(qs[b]) + i
            last = int(ctx_lens[b]) + i
            for h in range(H_q):
                g = h // G
                scores = []
                for j in range(last + 1):
                    page = int(block_table[b][j // PAGE])
                    kk = kf[page, g, j % PAGE]
                    s = 0.0
                    for c in range(d):
                        s += float(qf[row, h, c]) * float(kk[c])
                    scores.append(scale * s)
                m = max(scores)
                ws = [math.exp(s - m) for s in scores]
                l = sum(ws)
                acc = [0.0] * d
                for j, w in enumerate(ws):
                    page = int(block_table[b][j // PAGE])
                    vv = vf[page, g, j % PAGE]
                    for c in range(d):
                        acc[c] += w * float(vv[c])
                o[row, h] = np.array(acc) / l
                lse[row, h] = m + math.log(l)
    return o, lse


# ------------------------------------------------------------------------------------------
# comparison helpers (reporting only)
# ------------------------------------------------------------------------------------------

def compare(gpu_bf16_bits: np.ndarray, ref_f64: np.ndarray) -> dict:
    """Max / mean absolute error of bf16 results against float64 reference values (finite
    reference entries only), plus the max error in bf16 ulps of the reference value."""
    g = bf16_bits_to_f64(gpu_bf16_bits)
    mask = np.isfinite(ref_f64)
    diff = np.abs(g[mask] - ref_f64[mask])
    ref = ref_f64[mask]
    if diff.size == 0:
        return {"max_abs": 0.0, "mean_abs": 0.0, "max_ulp": 0.0, "n": 0, "nonfinite_gpu": 0}
    exp = np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126)))
    ulp = 2.0 ** (exp - 7)
    return {"max_abs": float(diff.max()), "mean_abs": float(diff.mean()),
            "max_ulp": float((diff / ulp).max()), "n": int(diff.size),
            "nonfinite_gpu": int((~np.isfinite(g[mask])).sum())}
