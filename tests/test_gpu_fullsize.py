"""Parity at the benchmark's full sizes and launch configuration (Qwen3-8B / Qwen3-30B-A3B shapes):
the whole batch runs on the GPU; sampled sequences / tokens are recomputed by the oracle.
Also checks every output is finite and that kv_append wrote exactly the sampled rows."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_35158_amd import workloads
from gpu_helpers import assert_close, bits, gpu_append, gpu_attend, oracle_sampled, say

pytestmark = pytest.mark.gpu


def _check_sampled(case, out, lse, seqs, tokens=None, what=""):
    o_ref, l_ref = oracle_sampled(case, seqs, tokens)
    cu = case.cu_q_lens
    ob = bits(out)
    lb = lse.cpu().numpy()
    for b in seqs:
        n = int(case.q_lens[b])
        assert_close(ob[cu[b]:cu[b] + n], o_ref[b], lb[cu[b]:cu[b] + n], l_ref[b], what="%s seq %d" % (what, b))


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
    _check_sampled(case, out, lse, seqs, what="8b decode")


def test_qwen3_8b_prefill_append_fullsize():
    say("case: qwen3-8b prefill-append B=16 full size")
    case = workloads.qwen3_8b_prefill_append("cuda")
    gpu_append(case)
    out, lse = gpu_attend(case, "prefill")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    rng = np.random.default_rng(2)
    seqs = _pick(case.ctx_lens + case.q_lens, 3, rng)
    _appended_rows_match(case, seqs)
    tokens = {}
    for b in seqs:
        n = int(case.q_lens[b])
        tokens[b] = sorted({0, n - 1, n // 2, 255 % n, 256 % n} | set(int(x) for x in rng.integers(0, n, 3)))
    o_ref, l_ref = oracle_sampled(case, seqs, tokens)
    cu = case.cu_q_lens
    ob, lb = bits(out), lse.cpu().numpy()
    for b in seqs:
        rows = [cu[b] + t for t in tokens[b]]
        assert_close(ob[rows], o_ref[b][tokens[b]], lb[rows], l_ref[b][tokens[b]], what="8b prefill seq %d" % b)


@pytest.mark.parametrize("batch", [256, 128, 32])
def test_qwen3_30b_decode_fullsize(batch):
    say("case: qwen3-30b-a3b decode B=%d full size" % batch)
    case = workloads.qwen3_30b_decode("cuda", batch=batch)
    gpu_append(case)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    seqs = _pick(case.ctx_lens, 5, np.random.default_rng(batch))
    _check_sampled(case, out, lse, seqs, what="30b decode")


def test_mixed_colocated_fullsize():
    say("case: mixed colocated full size (8 x 512 prefill + 192 decode)")
    case = workloads.mixed_colocated("cuda")
    gpu_append(case)
    out, lse = gpu_attend(case, "mixed")
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(lse).all()
    rng = np.random.default_rng(5)
    pre = [0, 7]
    dec = 8 + np.array(_pick(case.ctx_lens[8:], 4, rng))
    tokens = {b: [0, 255, 256, 511] for b in pre}
    for b in dec:
        tokens[int(b)] = [0]
    seqs = pre + [int(b) for b in dec]
    _appended_rows_match(case, seqs)
    o_ref, l_ref = oracle_sampled(case, seqs, tokens)
    cu = case.cu_q_lens
    ob, lb = bits(out), lse.cpu().numpy()
    for b in seqs:
        rows = [cu[b] + t for t in tokens[b]]
        assert_close(ob[rows], o_ref[b][tokens[b]], lb[rows], l_ref[b][tokens[b]], what="mixed seq %d" % b)


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
