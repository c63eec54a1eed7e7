"""KV transfer pack/unpack between two pools (PD disaggregation, Eq. 3 transfer term) through
the C ABI (needs an MI355X).  Bar: bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_35158_amd as pa
from paper_2609_35158_amd import workloads
from gpu_helpers import assert_close, bits, gpu_append, gpu_attend, oracle_full, say

pytestmark = pytest.mark.gpu

PAGE = 16


def _permuted_table(rng, lens, extra):
    pages = (np.asarray(lens) + PAGE - 1) // PAGE
    num_pages = int(pages.sum()) + extra
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.zeros((len(lens), max(1, int(pages.max()))), np.int32)
    pos = 0
    for b, n in enumerate(pages):
        bt[b, :n] = perm[pos:pos + n]
        pos += n
    return bt, num_pages


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).astype(np.int32)).cuda()


@pytest.mark.parametrize("seed", range(6))
def test_pack_and_unpack_match_oracle(seed):
    """Ragged token ranges (starting mid-page, empty ranges, whole contexts) packed out of pool A
    and unpacked into pool B with a different page placement; both results bit-exact."""
    rng = np.random.default_rng(500 + seed)
    H_kv = [1, 2, 4, 8, 3, 8][seed]
    d = [64, 128][seed % 2]
    B = int(rng.integers(1, 6))
    lens = rng.integers(1, 400, size=B, endpoint=True)
    start = np.array([int(rng.integers(0, n)) for n in lens])
    if seed % 3 == 0:
        start[0] = 0                       # a whole context
    n = lens - start
    if B > 1 and seed % 2:
        n[1] = 0                           # an empty range
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    total = int(cu[-1])
    say("case: kv transfer seed=%d H_kv=%d d=%d lens=%s start=%s n=%s" % (seed, H_kv, d, lens, start, n))
    case = workloads.build_case("xfer", 600 + seed, H_kv, H_kv, d, lens, np.zeros(B, np.int64),
                                device="cuda", extra_pages=3)
    kp_a, vp_a = bits(case.k_pool), bits(case.v_pool)
    bt_a = case.block_table.cpu().numpy()
    max_q, max_kv = int(max(n.max(), 1)), int(lens.max())
    buf = pa.kv_pack(case.k_pool, case.v_pool, case.block_table, _dev(start), _dev(cu), total, max_q, max_kv)
    torch.cuda.synchronize()
    ref = oracle.kv_pack(kp_a, vp_a, bt_a, start, cu)
    assert np.array_equal(bits(buf), ref), "pack differs from the oracle"
    # receiving pool: its own placement, pre-filled with random bits
    bt_b, np_b = _permuted_table(rng, lens, extra=5)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(700 + seed)
    shape = (np_b, H_kv, PAGE, d)
    kp_b = torch.randint(-32768, 32767, shape, generator=gen, device="cuda", dtype=torch.int16).view(torch.bfloat16)
    vp_b = torch.randint(-32768, 32767, shape, generator=gen, device="cuda", dtype=torch.int16).view(torch.bfloat16)
    kb0, vb0 = bits(kp_b), bits(vp_b)
    pa.kv_unpack(buf, kp_b, vp_b, _dev(bt_b), _dev(start), _dev(cu), max_q, max_kv)
    torch.cuda.synchronize()
    kr, vr = oracle.kv_unpack(kb0, vb0, ref, bt_b, start, cu)
    assert np.array_equal(bits(kp_b), kr) and np.array_equal(bits(vp_b), vr), "unpack differs from the oracle"


def test_one_row_per_sequence_without_cu():
    """cu_q_lens NULL: one row per sequence, position ctx_lens[b] (a decode step's new token)."""
    say("case: kv transfer, one row per sequence")
    lens = np.array([17, 1, 64, 300])
    case = workloads.build_case("xfer1", 31, 8, 8, 128, lens, np.zeros(4, np.int64), device="cuda")
    pos = lens - 1
    buf = pa.kv_pack(case.k_pool, case.v_pool, case.block_table, _dev(pos), None, 4, 1, int(lens.max()))
    torch.cuda.synchronize()
    ref = oracle.kv_pack(bits(case.k_pool), bits(case.v_pool), case.block_table.cpu().numpy(), pos, None)
    assert np.array_equal(bits(buf), ref)


def test_transfer_then_attention_is_bit_identical():
    """Move whole contexts from a prefill pool to a decode pool with another page placement: the
    decode output on the receiving pool is bit-identical to the one on the sending pool (same
    lengths, so the same split plan) and matches the oracle."""
    say("case: transfer then decode")
    ctx = np.array([3000, 77, 1500, 16])
    case = workloads.build_case("xfer-dec", 41, 32, 8, 128, ctx, np.ones(4, np.int64), device="cuda")
    gpu_append(case)
    lens = case.kv_lens
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    zeros = np.zeros(4, np.int64)
    buf = pa.kv_pack(case.k_pool, case.v_pool, case.block_table, _dev(zeros), _dev(cu), int(cu[-1]),
                     int(lens.max()), int(lens.max()))
    rng = np.random.default_rng(42)
    bt_b, np_b = _permuted_table(rng, lens, extra=9)
    kp_b = torch.zeros((np_b,) + tuple(case.k_pool.shape[1:]), dtype=torch.bfloat16, device="cuda")
    vp_b = torch.zeros_like(kp_b)
    pa.kv_unpack(buf, kp_b, vp_b, _dev(bt_b), _dev(zeros), _dev(cu), int(lens.max()), int(lens.max()))
    out_a, lse_a = gpu_attend(case, "decode")
    moved = workloads.Case(name="moved", seed=case.seed, num_q_heads=32, num_kv_heads=8, head_dim=128,
                           ctx_lens=case.ctx_lens, q_lens=case.q_lens, block_table=_dev(bt_b),
                           k_pool=kp_b, v_pool=vp_b, k_new=case.k_new, v_new=case.v_new, q=case.q,
                           scale=case.scale)
    out_b, lse_b = gpu_attend(moved, "decode")
    torch.cuda.synchronize()
    assert np.array_equal(bits(out_a), bits(out_b))
    assert torch.equal(lse_a, lse_b)
    o_ref, l_ref = oracle_full(moved)
    assert_close(bits(out_b), o_ref, lse_b.cpu().numpy(), l_ref, what="decode on the receiving pool")


def test_full_context_transfer_fullsize():
    """The Qwen3-8B decode batch (64 contexts, 2.4 GB of K/V) packed and unpacked into a second
    pool: sampled sequences' buffer rows bit-exact against the oracle; every moved row of the
    receiving pool equals its source row; packing the receiving pool returns the same buffer."""
    say("case: full-context transfer, qwen3-8b decode batch")
    case = workloads.qwen3_8b_decode("cuda")
    B = case.batch
    lens = case.ctx_lens.astype(np.int64)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    total, max_kv = int(cu[-1]), int(lens.max())
    zeros = _dev(np.zeros(B, np.int64))
    buf = pa.kv_pack(case.k_pool, case.v_pool, case.block_table, zeros, _dev(cu), total, max_kv, max_kv)
    rng = np.random.default_rng(8)
    bt_b, np_b = _permuted_table(rng, lens, extra=0)
    kp_b = torch.empty((np_b,) + tuple(case.k_pool.shape[1:]), dtype=torch.bfloat16, device="cuda")
    vp_b = torch.empty_like(kp_b)
    bt_b_dev = _dev(bt_b)
    pa.kv_unpack(buf, kp_b, vp_b, bt_b_dev, zeros, _dev(cu), max_kv, max_kv)
    buf2 = pa.kv_pack(kp_b, vp_b, bt_b_dev, zeros, _dev(cu), total, max_kv, max_kv)
    torch.cuda.synchronize()
    assert torch.equal(buf.view(torch.int16), buf2.view(torch.int16))
    bt_a = case.block_table.cpu().numpy()
    order = np.argsort(lens)
    for b in sorted({int(order[0]), int(order[-1]), 5, 33}):
        npg = (int(lens[b]) + PAGE - 1) // PAGE
        ia = torch.from_numpy(bt_a[b, :npg].astype(np.int64)).cuda()
        ib = torch.from_numpy(bt_b[b, :npg].astype(np.int64)).cuda()
        ka, va = bits(case.k_pool.index_select(0, ia)), bits(case.v_pool.index_select(0, ia))
        ref = oracle.kv_pack(ka, va, np.arange(npg, dtype=np.int32)[None, :], np.zeros(1, np.int64),
                             np.array([0, lens[b]], np.int32))
        rows = bits(buf[:, cu[b]:cu[b + 1]])
        assert np.array_equal(rows, ref), "sequence %d" % b
        kb, vb = bits(kp_b.index_select(0, ib)), bits(vp_b.index_select(0, ib))
        L = int(lens[b])
        flat = lambda x: x.transpose(0, 2, 1, 3).reshape(npg * PAGE, x.shape[1], x.shape[3])[:L]
        assert np.array_equal(flat(kb), flat(ka)) and np.array_equal(flat(vb), flat(va)), "sequence %d" % b


def test_out_of_range_pages_pack_zeros_and_unpack_skips():
    """Documented behaviour for block-table entries outside [0, num_pages): a pack writes zero rows
    for them and an unpack leaves the pools untouched for them (no access happens: the kernel
    checks the id before addressing the pool)."""
    say("case: kv transfer with out-of-range page ids")
    lens = np.array([40, 20])
    case = workloads.build_case("xfer-oob", 51, 4, 4, 64, lens, np.zeros(2, np.int64), device="cuda")
    bt = case.block_table.cpu().numpy().copy()
    bt[0, 1] = -1                       # positions 16..31 of sequence 0
    bt[1, 0] = case.num_pages           # positions 0..15 of sequence 1
    bt_d = _dev(bt)
    cu = np.array([0, 40, 60], np.int32)
    zeros = _dev(np.zeros(2, np.int64))
    buf = pa.kv_pack(case.k_pool, case.v_pool, bt_d, zeros, _dev(cu), 60, 40, 40)
    torch.cuda.synchronize()
    got = bits(buf)
    ref_bt = case.block_table.cpu().numpy()
    ref = oracle.kv_pack(bits(case.k_pool), bits(case.v_pool), ref_bt, np.zeros(2, np.int64), cu)
    bad_rows = list(range(16, 32)) + list(range(40, 56))
    good_rows = [r for r in range(60) if r not in bad_rows]
    assert np.all(got[:, bad_rows] == 0)
    assert np.array_equal(got[:, good_rows], ref[:, good_rows])
    k0, v0 = bits(case.k_pool), bits(case.v_pool)
    pa.kv_unpack(buf.flip(-1).contiguous(), case.k_pool, case.v_pool, bt_d, zeros, _dev(cu), 40, 40)
    torch.cuda.synchronize()
    # the oracle takes the valid table; only rows whose id is valid in `bt` are compared, and the
    # pages behind the two invalid ids must be unchanged
    kr, vr = oracle.kv_unpack(k0, v0, bits(buf.flip(-1).contiguous()), ref_bt, np.zeros(2, np.int64), cu)
    kg, vg = bits(case.k_pool), bits(case.v_pool)
    for pg in (int(ref_bt[0, 1]), int(ref_bt[1, 0])):
        assert np.array_equal(kg[pg], k0[pg]) and np.array_equal(vg[pg], v0[pg])
    for b, L in ((0, 40), (1, 20)):
        for p in range(L):
            if bt[b, p // 16] < 0 or bt[b, p // 16] >= case.num_pages:
                continue
            pg, sl = bt[b, p // 16], p % 16
            assert np.array_equal(kg[pg, :, sl], kr[pg, :, sl]) and np.array_equal(vg[pg, :, sl], vr[pg, :, sl])
