"""One decode step with its append (pearl_attn_decode_append: the attention kernel takes the new
token's K/V from k_new / v_new and writes them into the pools) against pearl_kv_append followed
by pearl_attn_decode: outputs, LSE and both pools bit for bit, and the oracle within tolerance.
Contexts cover a new token at the first and last slot of a page, an empty context, sequences of
several splits, and a batch above the in-kernel planning limit (which appends by a separate
launch)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads
from gpu_helpers import assert_close, bits, say

pytestmark = pytest.mark.gpu


def _run_both(case):
    ctx_d = torch.from_numpy(case.ctx_lens.astype(np.int32)).cuda()
    max_kv = int(case.kv_lens.max())
    k0, v0 = bits(case.k_pool), bits(case.v_pool)
    kp2, vp2 = case.k_pool.clone(), case.v_pool.clone()
    pa.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, ctx_d, None, 1, max_kv)
    ref, ref_lse = pa.decode(case.q, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv,
                             scale=case.scale, return_lse=True)
    out = torch.full_like(case.q, 7.0)
    got, got_lse = pa.decode_append(case.q, case.k_new, case.v_new, kp2, vp2, case.block_table, ctx_d, max_kv,
                                    scale=case.scale, return_lse=True, out=out)
    torch.cuda.synchronize()
    kr, vr = oracle.kv_append(k0, v0, bits(case.k_new), bits(case.v_new), case.block_table.cpu().numpy(),
                              case.ctx_lens, None)
    assert np.array_equal(bits(kp2), kr) and np.array_equal(bits(vp2), vr), "fused append differs from the oracle"
    assert np.array_equal(bits(case.k_pool), kr) and np.array_equal(bits(case.v_pool), vr)
    assert np.array_equal(bits(got), bits(ref)), "outputs differ from append + decode"
    assert torch.equal(got_lse, ref_lse), "LSE differs from append + decode"
    return got, got_lse, kr, vr


@pytest.mark.parametrize("seed", range(6))
def test_decode_append_matches_append_then_decode(seed):
    rng = np.random.default_rng(5100 + seed)
    G = [1, 2, 4, 8][seed % 4]
    d = [128, 64][(seed // 2) % 2]
    H_kv = [2, 4, 1, 8][seed % 4]
    B = int(rng.integers(8, 40))
    ctx = rng.integers(0, 700, size=B, endpoint=True)
    ctx[:6] = (0, 15, 16, 31, 4096, int(rng.integers(9000, 14000)))   # first/last slot, empty, multi-split
    say("case: decode_append seed=%d G=%d d=%d H_kv=%d B=%d" % (seed, G, d, H_kv, B))
    case = workloads.build_case("dec-append", 5200 + seed, H_kv * G, H_kv, d, ctx, np.ones(B, np.int64),
                                device="cuda", extra_pages=3)
    got, got_lse, kr, vr = _run_both(case)
    o_ref, l_ref = oracle.attention(bits(case.q), kr, vr, case.block_table.cpu().numpy(), case.ctx_lens, None,
                                    case.scale)
    assert_close(bits(got), o_ref, got_lse.cpu().numpy(), l_ref, what="decode_append seed %d" % seed)


def test_decode_append_full_size_and_above_the_planning_limit():
    say("case: decode_append on the 8B headline batch")
    case = workloads.qwen3_8b_decode("cuda")
    _run_both(case)
    say("case: decode_append on 1100 sequences (appended by a separate launch)")
    rng = np.random.default_rng(5300)
    ctx = rng.integers(0, 200, size=1100, endpoint=True)
    case = workloads.build_case("dec-append-big", 5301, 8, 2, 64, ctx, np.ones(1100, np.int64), device="cuda")
    got, got_lse, kr, vr = _run_both(case)
    o_ref, l_ref = oracle.attention(bits(case.q), kr, vr, case.block_table.cpu().numpy(), case.ctx_lens, None,
                                    case.scale, seqs=range(0, 1100, 37))
    rows = list(range(0, 1100, 37))
    assert_close(bits(got)[rows], o_ref[rows], got_lse.cpu().numpy()[rows], l_ref[rows], what="1100-sequence")
