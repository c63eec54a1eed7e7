"""The allocation-free decode (pearl_attn_decode_static, the library's static per-GPU workspace)
against pearl_attn_decode with a caller workspace: two calls in a row on one GPU, the second on
a smaller batch, each bit-identical to the allocating call and within the oracle's tolerance.
Both calls go through the C ABI."""
import numpy as np
import pytest
import torch

from gpu_helpers import assert_close, bits, dev_lengths, oracle_sampled, say
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import binding as bd
from paper_2609_35158_amd import workloads


def _decode_case(name, seed, batch, lo, hi):
    rng = np.random.default_rng(seed)
    ctx = rng.integers(lo, hi, size=batch, endpoint=True)
    case = workloads.build_case(name, seed, 32, 8, 128, ctx, np.ones(batch, np.int64), device="cuda")
    ctx_d, _ = dev_lengths(case)
    pa.kv_append(case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, ctx_d, None, 1,
                 int(case.kv_lens.max()))
    return case, ctx_d


@pytest.mark.gpu
def test_decode_static_matches_decode_on_two_calls():
    assert bd.decode_static_max_bytes() == 32 << 20
    for name, seed, batch, lo, hi in (("static-a", 911, 48, 900, 9000), ("static-b", 912, 11, 0, 700)):
        say("case: %s batch=%d ctx U[%d,%d]" % (name, batch, lo, hi))
        case, ctx_d = _decode_case(name, seed, batch, lo, hi)
        max_kv = int(case.kv_lens.max())
        desc = bd.make_desc(case.block_table, ctx_d, None, batch, 1, max_kv)
        assert bd.workspace_bytes(32, case.k_pool, desc) <= bd.decode_static_max_bytes()
        ref, ref_lse = pa.decode(case.q, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv,
                                 scale=case.scale, return_lse=True)
        out = torch.full_like(case.q, 3.0)
        lse = torch.full((batch, 32), 5.0, dtype=torch.float32, device="cuda")
        got, got_lse = bd.decode_static(case.q, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv,
                                        scale=case.scale, out=out, lse=lse)
        torch.cuda.synchronize()
        assert got.data_ptr() == out.data_ptr() and got_lse.data_ptr() == lse.data_ptr()
        assert np.array_equal(bits(got), bits(ref)), name
        assert torch.equal(got_lse, ref_lse), name
        seqs = sorted({0, batch - 1, int(np.argmax(case.ctx_lens)), int(np.argmin(case.ctx_lens))})
        o_ref, l_ref = oracle_sampled(case, seqs)
        for b in seqs:
            assert_close(bits(got[b:b + 1]), o_ref[b], got_lse[b:b + 1].cpu().numpy(), l_ref[b],
                         what="%s seq %d" % (name, b))
