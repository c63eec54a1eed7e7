"""HIP path vs the CPU oracle on the same seeded inputs, through the C ABI (needs an MI355X).

Bars: kv_append and block-table indexing bit-exact; attention outputs within max-abs 1e-2 and
mean-abs 1e-3 of the float64 oracle (bf16 in/out, fp32 accumulation); LSE within 1e-3."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads
from gpu_helpers import (assert_close, bits, bounds, dev_lengths, gpu_append, gpu_attend, oracle_full,
                         say)

pytestmark = pytest.mark.gpu


def _append_and_check(case):
    k0, v0 = bits(case.k_pool), bits(case.v_pool)
    gpu_append(case)
    torch.cuda.synchronize()
    kr, vr = oracle.kv_append(k0, v0, bits(case.k_new), bits(case.v_new), case.block_table.cpu().numpy(),
                              case.ctx_lens, case.cu_q_lens)
    assert np.array_equal(bits(case.k_pool), kr), "k_pool differs from the oracle append"
    assert np.array_equal(bits(case.v_pool), vr), "v_pool differs from the oracle append"
    return kr, vr


def test_tiny_turn_then_decode_steps():
    """2 sequences (contexts 100 and 37), GQA 2, d 64, 32-page permuted pool: a 20-token
    prefill-append turn, then 8 single-token decode steps."""
    say("case: tiny turn (seed 0)")
    case = workloads.tiny_prefill("cuda")
    kr, vr = _append_and_check(case)
    bt = case.block_table.cpu().numpy()
    o_ref, l_ref = oracle.attention(bits(case.q), kr, vr, bt, case.ctx_lens, case.cu_q_lens, case.scale)
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="tiny " + mode)
    ctx_now = case.ctx_lens + case.q_lens
    for t in range(8):
        q_t = case.extra["decode_q"][t]
        k_t, v_t = case.extra["decode_k"][t], case.extra["decode_v"][t]
        ctx_d = torch.from_numpy(ctx_now.astype(np.int32)).cuda()
        max_kv = int(ctx_now.max()) + 1
        k0, v0 = bits(case.k_pool), bits(case.v_pool)
        pa.kv_append(k_t, v_t, case.k_pool, case.v_pool, case.block_table, ctx_d, None, 1, max_kv)
        out, lse = pa.decode(q_t, case.k_pool, case.v_pool, case.block_table, ctx_d, max_kv,
                             scale=case.scale, return_lse=True)
        torch.cuda.synchronize()
        kr, vr = oracle.kv_append(k0, v0, bits(k_t), bits(v_t), bt, ctx_now, None)
        assert np.array_equal(bits(case.k_pool), kr) and np.array_equal(bits(case.v_pool), vr)
        o_ref, l_ref = oracle.attention(bits(q_t), kr, vr, bt, ctx_now, None, case.scale)
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="tiny decode step %d" % t)
        ctx_now = ctx_now + 1
    assert list(ctx_now) == [128, 65]


@pytest.mark.parametrize("seed", range(12))
def test_random_small_prefill_and_mixed(seed):
    """Random ragged shapes: G in {1,2,4,8}, d in {64,128}, contexts 0..300, chunks 1..40 plus a
    long chunk to span several 256-row tiles."""
    rng = np.random.default_rng(1000 + seed)
    G = [1, 2, 4, 8][seed % 4]
    d = [64, 128][(seed // 4) % 2]
    H_kv = [1, 2, 4][seed % 3]
    B = int(rng.integers(1, 5))
    ctx = rng.integers(0, 300, size=B, endpoint=True)
    ql = rng.integers(1, 40, size=B, endpoint=True)
    ql[0] = int(rng.integers(200, 700))          # several tiles and a ragged tail
    say("case: random prefill seed=%d G=%d d=%d H_kv=%d B=%d ctx=%s q=%s" % (seed, G, d, H_kv, B, ctx, ql))
    case = workloads.build_case("rand", 2000 + seed, H_kv * G, H_kv, d, ctx, ql, device="cuda", extra_pages=3)
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="%s seed %d" % (mode, seed))


@pytest.mark.parametrize("seed", range(8))
def test_random_small_decode(seed):
    """Decode on random shapes, including contexts long enough for many splits."""
    rng = np.random.default_rng(3000 + seed)
    G = [1, 2, 4, 8][seed % 4]
    d = [128, 64][(seed // 4) % 2]
    H_kv = [2, 1, 4, 8][seed % 4]
    B = int(rng.integers(1, 6))
    ctx = rng.integers(0, 300, size=B, endpoint=True)
    ctx[0] = int(rng.integers(3000, 9000))
    say("case: random decode seed=%d G=%d d=%d H_kv=%d ctx=%s" % (seed, G, d, H_kv, ctx))
    case = workloads.build_case("rand-dec", 4000 + seed, H_kv * G, H_kv, d, ctx, np.ones(B, np.int64),
                                device="cuda", extra_pages=2)
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in ("decode", "mixed", "prefill"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="%s seed %d" % (mode, seed))


@pytest.mark.parametrize("batch", [1, 63, 64, 65])
def test_decode_planner_boundary(batch):
    """Decode batches of at most 64 sequences are planned by one wave, larger ones by all 8 waves;
    both lists must cover every split exactly once.  Contexts give several full splits per
    sequence and short last splits of many sizes (and one sequence of a single key)."""
    rng = np.random.default_rng(9100 + batch)
    ctx = rng.integers(0, 2600, size=batch, endpoint=True)
    ctx[0] = 0
    if batch > 1:
        ctx[1] = 16 * 64 - 1
    say("case: decode planner boundary B=%d" % batch)
    case = workloads.build_case("plan-bound", 9200 + batch, 8, 2, 128, ctx, np.ones(batch, np.int64), device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="decode B=%d" % batch)


def test_split_plans_agree():
    """The same decode with different split plans (a larger max_kv_len bound gives larger splits)
    agrees within tolerance; the same plan twice is bit-identical."""
    say("case: split plans")
    ctx = np.array([20000, 7000, 15, 1, 33000])
    case = workloads.build_case("splits", 77, 32, 4, 128, ctx, np.ones(5, np.int64), device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    # widen the block table so the larger host bounds stay legal (extra columns are never read)
    bt = case.block_table
    case.block_table = torch.cat([bt, torch.zeros(bt.shape[0], 2000000 // 16 - bt.shape[1],
                                                  dtype=bt.dtype, device=bt.device)], 1).contiguous()
    outs = []
    for bound in (33001, 33001, 200000, 2000000):
        out, lse = gpu_attend(case, "decode", max_kv_len=bound)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="bound %d" % bound)
        outs.append(bits(out))
    assert np.array_equal(outs[0], outs[1])


def test_page_permutation_bit_identical():
    """Permuting the physical pages and rewriting the block table gives bit-identical outputs."""
    say("case: page permutation")
    ctx = np.array([500, 31, 1200]); ql = np.array([70, 1, 300])
    case = workloads.build_case("perm", 5, 16, 4, 128, ctx, ql, device="cuda", extra_pages=7)
    gpu_append(case)
    out1 = {m: bits(gpu_attend(case, m, return_lse=False)) for m in ("prefill", "mixed")}
    n = case.num_pages
    sigma = torch.randperm(n, generator=torch.Generator().manual_seed(9)).cuda()
    kp2 = torch.empty_like(case.k_pool); vp2 = torch.empty_like(case.v_pool)
    kp2[sigma] = case.k_pool; vp2[sigma] = case.v_pool
    case.k_pool, case.v_pool = kp2, vp2
    case.block_table = sigma[case.block_table.long()].to(torch.int32).contiguous()
    for m in ("prefill", "mixed"):
        out2 = bits(gpu_attend(case, m, return_lse=False))
        assert np.array_equal(out1[m], out2), m


def test_single_key_returns_v_exactly():
    """Empty context, one new token: the output equals v bit for bit."""
    say("case: single key")
    case = workloads.build_case("one", 6, 32, 8, 128, np.zeros(3, np.int64), np.ones(3, np.int64), device="cuda")
    gpu_append(case)
    for mode in ("decode", "prefill", "mixed"):
        out = gpu_attend(case, mode, return_lse=False)
        torch.cuda.synchronize()
        v = case.v_new.repeat_interleave(4, dim=1)
        assert torch.equal(out.view(torch.int16), v.view(torch.int16)), mode


def test_position_encoded_v_exact():
    """q = 0 gives uniform weights; V[j,:] = j makes each output exactly (position)/2, pinning the
    causal boundary and the page gather on the GPU."""
    say("case: position-encoded V")
    ctx = np.array([0, 13, 100, 200]); ql = np.array([57, 1, 30, 56])
    case = workloads.build_case("posv", 8, 8, 2, 64, ctx, ql, device="cuda")
    bt = case.block_table.cpu().numpy()
    vp = case.v_pool.float()
    for b in range(4):
        for j in range(int(ctx[b])):
            vp[bt[b][j // 16], :, j % 16, :] = j
    case.v_pool = vp.to(torch.bfloat16)
    tot = case.total_q
    case.v_new = (torch.cat([torch.arange(int(c), int(c + n)) for c, n in zip(ctx, ql)])
                  .float()[:, None, None].expand(tot, 2, 64).to(torch.bfloat16).cuda().contiguous())
    case.q = torch.zeros_like(case.q)
    gpu_append(case)
    exp = torch.cat([torch.arange(int(c), int(c + n)) for c, n in zip(ctx, ql)]).double() / 2
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        got = out.double().cpu()
        assert torch.equal(got, exp[:, None, None].expand_as(got)), mode
        want_lse = torch.log(exp * 2 + 1)
        assert torch.allclose(lse.double().cpu(), want_lse[:, None].expand_as(lse.cpu()), atol=1e-5)


def test_gqa_mapping_exact():
    """V of kv-head g is the constant g+1, so q-head h must output exactly h//G + 1."""
    say("case: GQA mapping")
    for G, H_kv in ((8, 4), (4, 8), (2, 2), (1, 4)):
        ctx = np.array([40, 300]); ql = np.array([30, 1])
        case = workloads.build_case("gqa", 10 + G, G * H_kv, H_kv, 128, ctx, ql, device="cuda")
        consts = torch.arange(1, H_kv + 1, dtype=torch.float32)[None, :, None, None]
        case.v_pool = consts.expand_as(case.v_pool.float()).to(torch.bfloat16).cuda().contiguous()
        case.v_new = consts[:, :, 0].expand(case.total_q, H_kv, 128).to(torch.bfloat16).cuda().contiguous()
        gpu_append(case)
        for mode in ("prefill", "mixed"):
            out = gpu_attend(case, mode, return_lse=False).float().cpu()
            want = (torch.arange(G * H_kv) // G + 1).float()[None, :, None].expand_as(out)
            # weights enter P.V in bf16 while the normaliser is fp32: equal up to ~2^-9 relative
            assert torch.allclose(out, want, atol=0, rtol=2 ** -8), (G, H_kv, mode, (out - want).abs().max())


def test_empty_and_zero_length_sequences():
    """Sequences with no new tokens are skipped (their output rows do not exist); an empty
    context is a plain causal prefill."""
    say("case: empty chunks")
    ctx = np.array([0, 50, 0, 17]); ql = np.array([0, 5, 33, 0])
    case = workloads.build_case("empty", 12, 16, 2, 128, ctx, ql, device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="empty " + mode)


def test_mixed_matches_standalone():
    """In one mixed launch each sequence matches its standalone decode or prefill result."""
    say("case: mixed vs standalone")
    ctx = np.array([3000, 10, 900, 5000, 64]); ql = np.array([300, 1, 1, 77, 1])
    case = workloads.build_case("mix", 13, 32, 4, 128, ctx, ql, device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    out_m, lse_m = gpu_attend(case, "mixed")
    out_p, lse_p = gpu_attend(case, "prefill")
    torch.cuda.synchronize()
    assert_close(bits(out_m), o_ref, lse_m.cpu().numpy(), l_ref, what="mixed")
    assert_close(bits(out_p), o_ref, lse_p.cpu().numpy(), l_ref, what="prefill")
    # decode-only sub-batch standalone
    dec = [1, 2, 4]
    sub = workloads.Case(name="sub", seed=0, num_q_heads=32, num_kv_heads=4, head_dim=128,
                         ctx_lens=case.ctx_lens[dec], q_lens=case.q_lens[dec],
                         block_table=case.block_table[dec].contiguous(), k_pool=case.k_pool,
                         v_pool=case.v_pool, k_new=None, v_new=None,
                         q=case.q[torch.tensor([int(case.cu_q_lens[b]) for b in dec]).cuda()].contiguous(),
                         scale=case.scale)
    out_d, lse_d = gpu_attend(sub, "decode")
    torch.cuda.synchronize()
    rows = [int(case.cu_q_lens[b]) for b in dec]
    diff = (out_d.float() - out_m[torch.tensor(rows).cuda()].float()).abs().max().item()
    say("   mixed vs standalone decode max diff %.3e" % diff)
    assert diff <= 1e-2


def test_device_length_violation_reports_and_writes_nothing():
    """A device length that breaks the host bounds makes the call write nothing; with
    PEARL_DEBUG=1 the call reports it."""
    import os
    say("case: bound violation")
    ctx = np.array([100, 40]); ql = np.array([1, 1])
    case = workloads.build_case("viol", 14, 8, 2, 64, ctx, ql, device="cuda")
    gpu_append(case)
    ctx_d = torch.from_numpy(np.array([100, 40], np.int32)).cuda()
    out = torch.full_like(case.q, 7.0)
    # max_kv_len bound of 64 is violated by the 101-key sequence
    pa.decode(case.q, case.k_pool, case.v_pool, case.block_table, ctx_d, 101, scale=case.scale, out=out)
    out2 = torch.full_like(case.q, 7.0)
    os.environ["PEARL_DEBUG"] = "1"
    try:
        with pytest.raises(pa.PearlError):
            pa.decode(case.q, case.k_pool, case.v_pool, case.block_table, ctx_d, 64, scale=case.scale, out=out2)
    finally:
        del os.environ["PEARL_DEBUG"]
    torch.cuda.synchronize()
    assert torch.all(out2 == 7.0)
    assert not torch.all(out == 7.0)


@pytest.mark.parametrize("pattern", ["ramp", "ramp_down", "large"])
def test_score_range_and_running_max(pattern):
    """Scores that grow (or shrink) steadily along the context make the running maximum move on
    every tile; large-magnitude q/k give scores far outside exp's fp32 range without the max
    subtraction.  All modes must still match the oracle."""
    say("case: score pattern %s" % pattern)
    ctx = np.array([1500, 700, 3000]); ql = np.array([90, 1, 1])
    case = workloads.build_case("range", 21, 32, 4, 128, ctx, ql, device="cuda")
    gen = torch.Generator(device="cuda").manual_seed(5)
    if pattern in ("ramp", "ramp_down"):
        sign = 1.0 if pattern == "ramp" else -1.0
        # q . k_j grows linearly with the key position j through the first coordinate
        bt = case.block_table.cpu().numpy()
        kp = case.k_pool.float()
        for b in range(3):
            n = int(ctx[b])
            pos = torch.arange(n, dtype=torch.float32, device="cuda")
            pages = torch.from_numpy(bt[b][np.arange(n) // 16].astype(np.int64)).cuda()
            slots = torch.from_numpy((np.arange(n) % 16).astype(np.int64)).cuda()
            kp[pages, :, slots, 0] = (sign * pos * 0.03)[:, None]
        case.k_pool = kp.to(torch.bfloat16)
        qf = case.q.float()
        qf[..., 0] = 8.0
        case.q = qf.to(torch.bfloat16).contiguous()
        kn = case.k_new.float()
        kn[..., 0] = sign * (torch.from_numpy(np.concatenate([np.arange(c, c + n) for c, n in zip(ctx, ql)]))
                             .float().cuda()[:, None] * 0.03)
        case.k_new = kn.to(torch.bfloat16).contiguous()
    else:
        case.q = (case.q.float() * 6.0).to(torch.bfloat16).contiguous()
        case.k_pool = (case.k_pool.float() * 4.0).to(torch.bfloat16)
        case.k_new = (case.k_new.float() * 4.0).to(torch.bfloat16).contiguous()
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    # the largest |v| the case holds (unwritten pool slots hold NaN sentinels)
    vv = oracle.bf16_bits_to_f64(vr)
    vmax = float(np.abs(vv[np.isfinite(vv)]).max()) if pattern == "large" else None
    for mode in ("prefill", "mixed"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="%s %s" % (pattern, mode),
                     peaked_vmax=vmax)
    dec = [1, 2]
    sub = workloads.Case(name="sub", seed=0, num_q_heads=32, num_kv_heads=4, head_dim=128,
                         ctx_lens=case.ctx_lens[dec], q_lens=case.q_lens[dec],
                         block_table=case.block_table[dec].contiguous(), k_pool=case.k_pool,
                         v_pool=case.v_pool, k_new=None, v_new=None,
                         q=case.q[torch.tensor([int(case.cu_q_lens[b]) for b in dec]).cuda()].contiguous(),
                         scale=case.scale)
    out_d, lse_d = gpu_attend(sub, "decode")
    torch.cuda.synchronize()
    rows = [int(case.cu_q_lens[b]) for b in dec]
    assert_close(bits(out_d), o_ref[rows], lse_d.cpu().numpy(), l_ref[rows], what="%s decode" % pattern,
                 peaked_vmax=vmax)


def _attend_with_workspace(case, mode):
    """Attention through the C ABI with a caller-owned workspace, returned for inspection."""
    from paper_2609_35158_amd import binding as bd
    ctx, cu = dev_lengths(case)
    max_q, max_kv = bounds(case)
    desc = bd.make_desc(case.block_table, ctx, cu, case.total_q, max_q, max_kv)
    ws = torch.empty(bd.workspace_bytes(case.num_q_heads, case.k_pool, desc), dtype=torch.uint8, device="cuda")
    fn = {"prefill": pa.prefill_append, "mixed": pa.mixed}[mode]
    out, lse = fn(case.q, case.k_pool, case.v_pool, case.block_table, ctx, cu, max_q, max_kv,
                  scale=case.scale, return_lse=True, workspace=ws)
    return out, lse, ws


PREFILL_SPLIT_CASES = [
    # (G, H_kv, d, contexts, chunk lengths, modes)
    (8, 4, 128, [8000], [100], ("prefill", "mixed")),
    (4, 2, 64, [3000, 1500], [60, 5], ("prefill", "mixed")),
    (1, 1, 128, [2500], [300], ("prefill", "mixed")),
    (2, 8, 128, [5000, 0, 2000], [33, 17, 1], ("prefill", "mixed")),
    (8, 1, 64, [1030, 4097], [1, 250], ("prefill",)),
]


@pytest.mark.parametrize("idx", range(len(PREFILL_SPLIT_CASES)))
def test_prefill_key_splits(idx):
    """Few prefill tiles on long contexts: the planner splits each tile's keys (checked in the
    workspace header) and the prefill merge combines the partial states; outputs and LSE against
    the oracle.  Contexts end mid-page and chunks span ragged tiles."""
    G, H_kv, d, ctx, ql, modes = PREFILL_SPLIT_CASES[idx]
    say("case: prefill key splits G=%d H_kv=%d d=%d ctx=%s q=%s" % (G, H_kv, d, ctx, ql))
    case = workloads.build_case("pre-split", 9100 + idx, H_kv * G, H_kv, d, np.array(ctx), np.array(ql),
                                device="cuda", extra_pages=2)
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in modes:
        out, lse, ws = _attend_with_workspace(case, mode)
        torch.cuda.synchronize()
        hdr = ws[:64 * 4].view(torch.int32).cpu().numpy()
        say("   %s: keys per split %d, split tiles %d" % (mode, hdr[5], hdr[6]))
        if mode == "prefill":
            assert hdr[5] > 0 and hdr[6] > 0, "expected the planner to split prefill tiles"
        assert hdr[3] == 0
        assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="%s split case %d" % (mode, idx))


def test_prefill_key_splits_long_context_sampled():
    """One 256-token chunk on a 30000-token context (Qwen3-30B-A3B shape): splits larger than the
    minimum; sampled tokens against the oracle."""
    from gpu_helpers import oracle_sampled
    say("case: prefill key splits, 256 tokens on 30000")
    case = workloads.build_case("pre-split-long", 9200, 32, 4, 128, np.array([30000]), np.array([256]),
                                device="cuda")
    gpu_append(case)
    out, lse, ws = _attend_with_workspace(case, "prefill")
    torch.cuda.synchronize()
    hdr = ws[:64 * 4].view(torch.int32).cpu().numpy()
    say("   keys per split %d, split tiles %d" % (hdr[5], hdr[6]))
    assert hdr[5] > 1024 and hdr[6] == 8
    toks = [0, 1, 31, 32, 100, 200, 254, 255]
    o_ref, l_ref = oracle_sampled(case, [0], {0: toks})
    assert_close(bits(out)[toks], o_ref[0][toks], lse.cpu().numpy()[toks], l_ref[0][toks], what="long split")


def test_batches_larger_than_one_planner_chunk():
    """More sequences than one pass of the planners' threads: the block scans carry offsets from
    one chunk of sequences to the next.  Decode of 800 sequences long enough for several full
    splits each is planned inside the attention kernel (512 sequences per chunk), so its full
    splits, short last splits and their size classes span chunks; decode of 1500 sequences (above
    the in-kernel limit) and a mixed batch of 1100 sequences with ragged chunks go through the
    planner kernel (256 sequences per chunk)."""
    say("case: 800-sequence decode with multi-split sequences")
    rng = np.random.default_rng(78)
    ctx = rng.integers(0, 3000, size=800, endpoint=True)
    ctx[:5] = (16 * 64, 16 * 64 - 1, 16 * 128, 0, 1)      # split-size multiples and edges
    ctx[600:605] = (16 * 160 - 1, 16 * 160, 0, 2999, 1)  # and in the second chunk
    case = workloads.build_case("big-batch-splits", 7703, 8, 2, 64, ctx, np.ones(800, np.int64), device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="800-sequence multi-split decode")
    say("case: 1500-sequence decode and 1100-sequence mixed batch")
    rng = np.random.default_rng(77)
    ctx = rng.integers(0, 90, size=1500, endpoint=True)
    case = workloads.build_case("big-batch-dec", 7701, 8, 2, 64, ctx, np.ones(1500, np.int64), device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    out, lse = gpu_attend(case, "decode")
    torch.cuda.synchronize()
    assert_close(bits(out), o_ref, lse.cpu().numpy(), l_ref, what="1500-sequence decode")
    ctx = rng.integers(0, 60, size=1100, endpoint=True)
    ql = np.where(rng.random(1100) < 0.5, 1, rng.integers(0, 9, size=1100, endpoint=True))
    case = workloads.build_case("big-batch-mixed", 7702, 8, 2, 64, ctx, ql, device="cuda")
    kr, vr = _append_and_check(case)
    o_ref, l_ref = oracle_full(case, kr, vr)
    for mode in ("mixed", "prefill"):
        out, lse = gpu_attend(case, mode)
        torch.cuda.synchronize()
        m = np.isfinite(o_ref).all(axis=(1, 2))
        assert_close(bits(out)[m], o_ref[m], lse.cpu().numpy()[m], l_ref[m], what="1100-sequence " + mode)


def test_prefill_tile_order_spans_chunks():
    """Prefill of 300 sequences with up to 4 tiles each and no key splits: tiles are written by
    size class across the whole launch, a sequence's run of tiles in one class claimed together,
    and the classes and runs span the planner's 256-sequence chunks.  Every row's LSE (preset to
    NaN) must be written, and sampled sequences match the oracle."""
    from gpu_helpers import oracle_sampled
    from paper_2609_35158_amd import binding as bd
    say("case: 300-sequence prefill, tiles ordered by size class")
    rng = np.random.default_rng(79)
    ctx = rng.integers(0, 2000, size=300, endpoint=True)
    ql = rng.integers(1, 256, size=300, endpoint=True)
    ctx[:4] = (0, 2000, 0, 1999)
    ql[:4] = (256, 256, 1, 65)
    case = workloads.build_case("prefill-order", 7704, 8, 2, 64, ctx, ql, device="cuda")
    gpu_append(case)
    dctx, cu = dev_lengths(case)
    max_q, max_kv = bounds(case)
    desc = bd.make_desc(case.block_table, dctx, cu, case.total_q, max_q, max_kv)
    ws = torch.empty(bd.workspace_bytes(case.num_q_heads, case.k_pool, desc), dtype=torch.uint8, device="cuda")
    lse = torch.full((case.total_q, case.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
    out, lse = pa.prefill_append(case.q, case.k_pool, case.v_pool, case.block_table, dctx, cu, max_q, max_kv,
                                 scale=case.scale, return_lse=True, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    hdr = ws[:64 * 4].view(torch.int32).cpu().numpy()
    assert hdr[5] == 0, "expected no key splits"
    lse_np = lse.cpu().numpy()
    assert np.isfinite(lse_np).all(), "rows left unwritten: %d" % int((~np.isfinite(lse_np)).sum())
    seqs = [0, 1, 2, 3] + sorted(int(x) for x in rng.choice(np.arange(4, 300), 20, replace=False))
    o_ref, l_ref = oracle_sampled(case, seqs)
    o = bits(out)
    for b in seqs:
        r = slice(int(case.cu_q_lens[b]), int(case.cu_q_lens[b] + case.q_lens[b]))
        assert_close(o[r], o_ref[b], lse_np[r], l_ref[b], what="prefill-order sequence %d" % b)
