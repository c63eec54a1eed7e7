"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI on a synthetic
case, and run the CPU oracle on the same bytes (whole case or sampled sequences)."""
from __future__ import annotations

import sys
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads

# Tolerance for bf16 outputs against the float64 oracle (bf16 inputs/outputs, fp32 accumulation).
MAX_ABS = 1e-2
MEAN_ABS = 1e-3
LSE_ABS = 1e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def dev_lengths(case: workloads.Case):
    dev = case.q.device
    ctx = torch.from_numpy(case.ctx_lens.astype(np.int32)).to(dev)
    cu = torch.from_numpy(case.cu_q_lens.astype(np.int32)).to(dev)
    return ctx, cu


def bounds(case: workloads.Case) -> Tuple[int, int]:
    max_q = int(case.q_lens.max()) if case.batch else 0
    max_kv = int(case.kv_lens.max()) if case.batch else 0
    return max_q, max_kv


def gpu_append(case: workloads.Case, decode_layout: bool = False) -> None:
    ctx, cu = dev_lengths(case)
    max_q, max_kv = bounds(case)
    pa.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, ctx,
                 None if decode_layout else cu, max_q, max_kv)


def gpu_attend(case: workloads.Case, mode: str, return_lse: bool = True, max_kv_len: Optional[int] = None):
    ctx, cu = dev_lengths(case)
    max_q, max_kv = bounds(case)
    if max_kv_len is not None:
        max_kv = max_kv_len
    if mode == "decode":
        return pa.decode(case.q, case.k_pool, case.v_pool, case.block_table, ctx, max_kv,
                         scale=case.scale, return_lse=return_lse)
    if mode == "prefill":
        return pa.prefill_append(case.q, case.k_pool, case.v_pool, case.block_table, ctx, cu, max_q,
                                 max_kv, scale=case.scale, return_lse=return_lse)
    if mode == "mixed":
        return pa.mixed(case.q, case.k_pool, case.v_pool, case.block_table, ctx, cu, max_q, max_kv,
                        scale=case.scale, return_lse=return_lse)
    raise ValueError(mode)


def oracle_full(case: workloads.Case, k_pool_bits=None, v_pool_bits=None):
    kp = bits(case.k_pool) if k_pool_bits is None else k_pool_bits
    vp = bits(case.v_pool) if v_pool_bits is None else v_pool_bits
    return oracle.attention(bits(case.q), kp, vp, case.block_table.cpu().numpy(), case.ctx_lens,
                            case.cu_q_lens, case.scale)


def oracle_sampled(case: workloads.Case, seqs: Sequence[int], tokens: Optional[Dict[int, List[int]]] = None,
                   heads: Optional[Sequence[int]] = None):
    """Oracle on a subset of sequences: gather only their pages (compact pool, remapped block
    table) so multi-GB pools need not be copied to the host."""
    bt = case.block_table.cpu().numpy()
    npages = (case.kv_lens + 15) // 16
    rows, cols = [], []
    for b in seqs:
        rows.append(bt[b, :npages[b]])
    uniq = np.unique(np.concatenate(rows)) if rows else np.zeros(0, np.int64)
    remap = {int(p): i for i, p in enumerate(uniq)}
    idx = torch.from_numpy(uniq.astype(np.int64)).to(case.k_pool.device)
    kp = bits(case.k_pool.index_select(0, idx))
    vp = bits(case.v_pool.index_select(0, idx))
    sub_bt = np.zeros((len(seqs), max(1, int(npages[list(seqs)].max()))), np.int32)
    for i, b in enumerate(seqs):
        sub_bt[i, :npages[b]] = [remap[int(p)] for p in bt[b, :npages[b]]]
    cu = case.cu_q_lens
    q_all = bits(case.q)
    # per selected sequence, build its own rows
    out_o, out_l = {}, {}
    for i, b in enumerate(seqs):
        n = int(case.q_lens[b])
        qb = q_all[cu[b]:cu[b] + n]
        sel = None if tokens is None else {0: tokens[b]}
        o, l = oracle.attention(qb, kp, vp, sub_bt[i:i + 1], case.ctx_lens[b:b + 1],
                                np.array([0, n], np.int32), case.scale, heads=heads, tokens=sel)
        out_o[b], out_l[b] = o, l
    return out_o, out_l


def oracle_workers() -> int:
    """Threads for whole-batch oracle runs: the host's CPU share, at most 16."""
    import os
    return max(1, min(16, len(os.sched_getaffinity(0))))


def oracle_every_sequence(case: workloads.Case, tokens: Optional[Dict[int, List[int]]] = None,
                          seqs: Optional[Sequence[int]] = None):
    """The oracle on every sequence of a full-size batch (or on `seqs`), each sequence evaluated
    on its own (its rows of q, its block-table row; `tokens[b]` selects new-token indices) in a
    pool of threads over one host copy of the pools.  numpy releases the interpreter lock inside
    its array kernels, and BLAS runs one thread per worker, so the sequences run in parallel.
    Returns {b: (o [n_b][H_q][d], lse [n_b][H_q])}; unselected tokens are NaN."""
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits
    kp, vp = bits(case.k_pool), bits(case.v_pool)
    bt = case.block_table.cpu().numpy()
    q_all = bits(case.q)
    cu = case.cu_q_lens
    seqs = list(range(case.batch)) if seqs is None else list(seqs)

    def one(b):
        n = int(case.q_lens[b])
        sel = None if tokens is None else {0: tokens[b]}
        return b, oracle.attention(q_all[cu[b]:cu[b] + n], kp, vp, bt[b:b + 1], case.ctx_lens[b:b + 1],
                                   np.array([0, n], np.int32), case.scale, tokens=sel)

    with threadpool_limits(limits=1):
        with ThreadPoolExecutor(max_workers=oracle_workers()) as ex:
            res = dict(ex.map(one, seqs))
    return res


def tile_edge_tokens(n: int, tokens_per_tile: int, extra: int, rng) -> List[int]:
    """New-token indices of a prefill chunk of n tokens: the first and last token of every q-tile
    plus `extra` random ones."""
    picks = set()
    for t0 in range(0, n, tokens_per_tile):
        picks.add(t0)
        picks.add(min(n, t0 + tokens_per_tile) - 1)
    picks.update(int(x) for x in rng.integers(0, n, size=extra))
    return sorted(picks)


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |x| (8 significant bits)."""
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -126)))
    return 2.0 ** (e - 7)


def peaked_bound(ref_o: np.ndarray, vmax: float) -> np.ndarray:
    """Per-element error bound of the bf16 path when a few keys dominate each softmax row (stress
    inputs with a large score range), derived from its rounding steps:
      * the fp32 result is rounded to bf16: at most half an ulp of o;
      * the weights enter P.V rounded to bf16 (8 significant bits, round to nearest even:
        relative error <= 2^-8 each) while l sums the fp32 weights, so o moves by at most
        2^-8 sum_j w_j |v_j| / l <= 2^-8 max_j |v_j|; with many comparable weights these
        errors average out, with one or two dominant keys they do not;
      * fp32 rounding of the scores, the sums and the normalisation: below 1e-4 at these sizes.
    The bar is the larger of the plain 1e-2 and this bound."""
    return np.maximum(MAX_ABS, 0.5 * bf16_ulp(ref_o) + vmax * 2.0 ** -8 + 1e-4)


def assert_close(gpu_o_bits: np.ndarray, ref_o: np.ndarray, gpu_lse: Optional[np.ndarray] = None,
                 ref_lse: Optional[np.ndarray] = None, what: str = "", peaked_vmax: Optional[float] = None) -> dict:
    """Outputs within max-abs 1e-2 and mean-abs 1e-3 of the float64 oracle.  peaked_vmax (stress
    inputs whose softmax rows are dominated by one or two keys; the largest |v| of the case)
    replaces the max-abs bar by the derived per-element bound of peaked_bound()."""
    st = oracle.compare(gpu_o_bits, ref_o)
    say("   parity %s: n=%d max_abs=%.3e mean_abs=%.3e max_ulp=%.1f" % (what, st["n"], st["max_abs"],
                                                                          st["mean_abs"], st["max_ulp"]))
    assert st["n"] > 0, "nothing compared"
    assert st["nonfinite_gpu"] == 0, "non-finite GPU outputs (%s)" % what
    if peaked_vmax is not None:
        g = oracle.bf16_bits_to_f64(gpu_o_bits)
        m = np.isfinite(ref_o)
        r = ref_o[m]
        excess = np.abs(g[m] - r) - peaked_bound(r, peaked_vmax)
        k = int(np.argmax(excess))
        say("   peaked bound %s: vmax=%.3f worst margin %.3e at |o|=%.4f" % (what, peaked_vmax, -excess[k], abs(r[k])))
        assert excess.max() <= 0, "max excess over the derived bound: %.3e at |o|=%.4f (%s)" % (
            excess.max(), abs(r[k]), what)
    else:
        assert st["max_abs"] <= MAX_ABS, "max_abs %.3e > %.1e (%s)" % (st["max_abs"], MAX_ABS, what)
    assert st["mean_abs"] <= MEAN_ABS, "mean_abs %.3e > %.1e (%s)" % (st["mean_abs"], MEAN_ABS, what)
    if gpu_lse is not None and ref_lse is not None:
        m = np.isfinite(ref_lse)
        d = np.abs(gpu_lse[m].astype(np.float64) - ref_lse[m])
        say("   lse %s: max_abs=%.3e" % (what, d.max() if d.size else 0.0))
        assert np.all(np.isfinite(gpu_lse[m]))
        assert d.size == 0 or d.max() <= LSE_ABS, "lse max_abs %.3e (%s)" % (d.max(), what)
    return st
