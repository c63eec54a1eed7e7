"""Parity at the benchmark's full sizes and launch configuration (Qwen3-8B / Qwen3-30B-A3B shapes):
the whole batch runs on the GPU and the oracle recomputes every decode sequence, and, for every
prefill chunk, the first and last token of every q-tile plus 32 random tokens (a pool of host
threads; see oracle_every_sequence).  Also checks every output is finite and that kv_append wrote
exactly the sampled rows.  Per-workload max/mean errors are printed."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_35158_amd import workloads
from gpu_helpers import (assert_close, bits, gpu_append, gpu_attend, oracle_every_sequence, oracle_sampled, say,
                         tile_edge_tokens)

pytestmark = pytest.mark.gpu


def _pick(lengths, k, rng):
    order = np.argsort(lengths)
    picks = {int(order[0]), int(order[-1])}
    while len(picks) < min(k, len(lengths)):
        picks.add(int(rng.integers(0, len(lengths))))
    return sorted(picks)


def _appended_rows_match(case, seqs):
    """The appended K/V rows of sampled sequences read back exactly through the block table."""
    bt = case.block_table.cpu().numpy()
    kp = case.k_pool
    cu = case.cu_q_lens
    for b in seqs:
        for t in (0, int(case.q_lens[b]) - 1):
            p = int(case.ctx_lens[b]) + t
            got = bits(kp[int(bt[b][p // 16]), :, p % 16, :])
            assert np.array_equal(got, bits(case.k_new[cu[b] + t])), (b, t)


def _check_every(case, out, lse, tokens=None, what=""):
    """Every sequence of the batch (tokens[b] of each prefill chunk) against the oracle; each
    sequence must pass the bar, and the aggregate statistics are printed."""
    res = oracle_every_sequence(case, tokens)
    cu = case.cu_q_lens
    ob, lb = bits(out), lse.cpu().numpy()
    worst, total, n_all = 0.0, 0.0, 0
    for b in range(case.batch):
        o_ref, l_ref = res[b]
        n = int(case.q_lens[b])
        sel = list(range(n)) if tokens is None else tokens[b]
        rows = [cu[b] + t for t in sel]
        st = assert_close(ob[rows], o_ref[sel], lb[rows], l_ref[sel], what="%s seq %d" % (what, b))
        worst = max(worst, st["max_abs"])
        total += st["mean_abs"] * st["n"]
        n_all += st["n"]
    say("   %s: every sequence compared: %d outputs, max_abs=%.3e mean_abs=%.3e" % (what, n_all, worst, total / n_all))


@pytest.mark.parametrize("heads", [(32, 8), (16, 4)])
def test_qwen3_8b_decode_fullsize(heads):
    """The headline batch, and one GPU's share of it under tensor parallelism 2 (half the heads)."""
    batch = 64
    say("case: qwen3-8b decode B=%d heads %s full size" % (batch, heads))
    case = workloads.qwen3_8b_decode("cuda", batch=batch, num_q_heads=heads[0], num_kv_heads=heads[1])
    gpu_append(case)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    seqs = _pick(case.ctx_lens, 6, np.random.default_rng(1))
    _appended_rows_match(case, seqs)
    _check_every(case, out, lse, what="8b decode heads %d/%d" % heads)


def test_qwen3_8b_prefill_append_fullsize():
    say("case: qwen3-8b prefill-append B=16 full size")
    case = workloads.qwen3_8b_prefill_append("cuda")
    gpu_append(case)
    out, lse = gpu_attend(case, "prefill")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    rng = np.random.default_rng(2)
    _appended_rows_match(case, range(case.batch))
    T = 256 // (case.num_q_heads // case.num_kv_heads)          # tokens per q-tile
    tokens = {b: tile_edge_tokens(int(case.q_lens[b]), T, 32, rng) for b in range(case.batch)}
    _check_every(case, out, lse, tokens, what="8b prefill")


@pytest.mark.parametrize("batch", [256, 128, 32])
def test_qwen3_30b_decode_fullsize(batch):
    say("case: qwen3-30b-a3b decode B=%d full size" % batch)
    case = workloads.qwen3_30b_decode("cuda", batch=batch)
    gpu_append(case)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    _check_every(case, out, lse, what="30b decode B=%d" % batch)


def test_mixed_colocated_fullsize():
    say("case: mixed colocated full size (8 x 512 prefill + 192 decode)")
    case = workloads.mixed_colocated("cuda")
    gpu_append(case)
    out, lse = gpu_attend(case, "mixed")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    rng = np.random.default_rng(5)
    _appended_rows_match(case, range(case.batch))
    T = 256 // (case.num_q_heads // case.num_kv_heads)
    tokens = {b: (tile_edge_tokens(int(case.q_lens[b]), T, 32, rng) if case.q_lens[b] > 1 else [0])
              for b in range(case.batch)}
    _check_every(case, out, lse, tokens, what="mixed")


def test_pd_interference_sweep_points():
    """The interference sweep's extreme points: 16 chunks of 2048 tokens and 1 chunk of 256 tokens
    on 8192-token contexts, batched with 192 decodes in one mixed launch, on sub-batches of one
    shared pool (as the benchmark builds them)."""
    say("case: pd-interference sweep points (16 x 2048 and 1 x 256 prefill + 192 decode)")
    base = workloads.mixed_colocated("cuda", n_prefill=16, chunk=2048)
    gpu_append(base)
    dec = list(range(16, base.batch))
    rng = np.random.default_rng(7)
    for k, s in ((16, 2048), (1, 256)):
        case = workloads.sub_batch(base, list(range(k)) + dec, [s] * k + [1] * len(dec))
        out, lse = gpu_attend(case, "mixed")
        torch.cuda.synchronize()
        assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
        pre = sorted({0, k - 1})
        dsel = k + np.array(_pick(case.ctx_lens[k:], 3, rng))
        tokens = {b: sorted({0, s - 1, s // 2, 255, 256 % s}) for b in pre}
        for b in dsel:
            tokens[int(b)] = [0]
        seqs = pre + [int(b) for b in dsel]
        o_ref, l_ref = oracle_sampled(case, seqs, tokens)
        cu = case.cu_q_lens
        ob, lb = bits(out), lse.cpu().numpy()
        for b in seqs:
            rows = [cu[b] + t for t in tokens[b]]
            assert_close(ob[rows], o_ref[b][tokens[b]], lb[rows], l_ref[b][tokens[b]],
                         what="pd k=%d s=%d seq %d" % (k, s, b))
        del case, out, lse
