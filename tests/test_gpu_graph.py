"""The decode step (kv_append + decode attention, or the two fused in pearl_attn_decode_append)
needs no host synchronisation or allocation, so it can be captured once in a HIP graph and
replayed (the paper notes graph recapture as part of a reconfiguration's cost; section 4.3.2).  Each replay, with eager work and synchronisations in
between, must equal the eager call bit for bit and the oracle within tolerance."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads
from gpu_helpers import assert_close, bits, say

pytestmark = pytest.mark.gpu


def _bf16(shape, gen):
    return torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)


@pytest.mark.parametrize("fused", [False, True], ids=["append+decode", "decode_append"])
def test_decode_step_graph_replays_match_eager(fused):
    say("case: decode step (%s) captured in a graph, 3 replays" % ("decode_append" if fused else "append + decode"))
    rng = np.random.default_rng(61)
    ctx = rng.integers(500, 4000, size=6, endpoint=True)
    case = workloads.build_case("graph", 6100, 8, 2, 128, ctx, np.ones(6, np.int64), device="cuda")
    ctx_d = torch.from_numpy(case.ctx_lens.astype(np.int32)).cuda()
    max_kv = int(case.kv_lens.max())
    from paper_2609_35158_amd import binding as bd
    desc = bd.make_desc(case.block_table, ctx_d, None, case.batch, 1, max_kv)
    nbytes = bd.workspace_bytes(case.num_q_heads, case.k_pool, desc)
    q_s, k_s, v_s = case.q.clone(), case.k_new.clone(), case.v_new.clone()
    out_g = torch.empty_like(q_s)
    lse_g = torch.empty((case.batch, case.num_q_heads), dtype=torch.float32, device="cuda")
    ws_g = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    out_e, lse_e = torch.empty_like(out_g), torch.empty_like(lse_g)
    ws_e = torch.empty_like(ws_g)

    def step(q, k, v, out, lse, ws):
        if fused:
            pa.decode_append(q, k, v, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv, scale=case.scale,
                             out=out, lse=lse, workspace=ws)
            return
        pa.kv_append(k, v, case.k_pool, case.v_pool, case.block_table, ctx_d, None, 1, max_kv)
        pa.decode(q, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv, scale=case.scale,
                  out=out, lse=lse, workspace=ws)

    # eager warm-up (first calls query the device), then capture
    step(q_s, k_s, v_s, out_e, lse_e, ws_e)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(q_s, k_s, v_s, out_g, lse_g, ws_g)
    torch.cuda.synchronize()
    gen = torch.Generator(device="cuda")
    gen.manual_seed(62)
    bt = case.block_table.cpu().numpy()
    for r in range(3):
        q_s.copy_(_bf16(q_s.shape, gen))
        k_s.copy_(_bf16(k_s.shape, gen))
        v_s.copy_(_bf16(v_s.shape, gen))
        graph.replay()
        torch.cuda.synchronize()
        got, got_lse = bits(out_g), lse_g.cpu().numpy()
        # eager work between replays: the same step on other output buffers
        step(q_s, k_s, v_s, out_e, lse_e, ws_e)
        torch.cuda.synchronize()
        assert np.array_equal(got, bits(out_e)), "replay %d differs from the eager call" % r
        assert np.array_equal(got_lse, lse_e.cpu().numpy())
        o_ref, l_ref = oracle.attention(bits(q_s), bits(case.k_pool), bits(case.v_pool), bt, case.ctx_lens,
                                        None, case.scale)
        assert_close(got, o_ref, got_lse, l_ref, what="graph replay %d" % r)
