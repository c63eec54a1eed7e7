"""Head layouts that the seeded random cases do not pair (there the kv-head count moves with G):
every G in {1, 2, 4, 8} with one and with eight kv-heads, at d = 64 and 128, through the fused
decode step (pearl_attn_decode_append), prefill-append and the mixed launch, against the oracle on
the same inputs.  Pools after the appends are compared bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads
from gpu_helpers import assert_close, bits, gpu_append, gpu_attend, oracle_full, say

pytestmark = pytest.mark.gpu

LAYOUTS = [(G, H_kv, d) for G in (1, 2, 4, 8) for H_kv in (1, 8) for d in (64, 128)]


@pytest.mark.parametrize("G,H_kv,d", LAYOUTS)
def test_head_layout(G, H_kv, d):
    seed = 7000 + 100 * G + 10 * H_kv + d // 64
    rng = np.random.default_rng(seed)
    tag = "G=%d H_kv=%d d=%d" % (G, H_kv, d)

    # one decode step with its append fused; the first sequence long enough for several splits
    ctx = rng.integers(0, 300, size=4, endpoint=True)
    ctx[0] = int(rng.integers(2000, 4000))
    say("case: head layout %s, decode_append ctx=%s" % (tag, ctx))
    case = workloads.build_case("grid-dec", seed, H_kv * G, H_kv, d, ctx, np.ones(4, np.int64), device="cuda",
                                extra_pages=2)
    k0, v0 = bits(case.k_pool), bits(case.v_pool)
    ctx_d = torch.from_numpy(case.ctx_lens.astype(np.int32)).cuda()
    out, lse = pa.decode_append(case.q, case.k_new, case.v_new, case.k_pool, case.v_pool, case.block_table, ctx_d,
                                int(case.kv_lens.max()), scale=case.scale, return_lse=True)
    torch.cuda.synchronize()
    bt = case.block_table.cpu().numpy()
    kr, vr = oracle.kv_append(k0, v0, bits(case.k_new), bits(case.v_new), bt, case.ctx_lens, None)
    assert np.array_equal(bits(case.k_pool), kr) and np.array_equal(bits(case.v_pool), vr), \
        "pools after the fused append differ from the oracle (%s)" % tag
    o_ref, l_ref = oracle.attention(bits(case.q), kr, vr, bt, case.ctx_lens, None, case.scale)
    assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="decode_append " + tag)

    # prefill-append and the mixed launch: ragged chunks, the first longer than one 256-row tile
    ctx = rng.integers(0, 200, size=3, endpoint=True)
    ql = rng.integers(1, 30, size=3, endpoint=True)
    ql[0] = 256 // G + int(rng.integers(1, 40))
    say("case: head layout %s, prefill ctx=%s q=%s" % (tag, ctx, ql))
    case = workloads.build_case("grid-pre", seed + 1, H_kv * G, H_kv, d, ctx, ql, device="cuda", extra_pages=2)
    k0, v0 = bits(case.k_pool), bits(case.v_pool)
    gpu_append(case)
    torch.cuda.synchronize()
    kr, vr = oracle.kv_append(k0, v0, bits(case.k_new), bits(case.v_new), case.block_table.cpu().numpy(),
                              case.ctx_lens, case.cu_q_lens)
    assert np.array_equal(bits(case.k_pool), kr) and np.array_equal(bits(case.v_pool), vr), \
        "pools after kv_append differ from the oracle (%s)" % tag
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="%s %s" % (mode, tag))
