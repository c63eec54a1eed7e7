"""Pins that tie the CPU oracle to facts fixed independently of it.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with a closed form, an
invariant, a hand-worked example or an independent library routine.  They are run as ordinary
tests (``test_oracle_pins.py``) and again under planted mistakes (``test_oracle_mutations.py``)
to show that each plausible slip in the oracle is caught by at least one of them.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

import oracle
from oracle import paged_attention as pa

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
PAGE = 16


def bits(x) -> np.ndarray:
    """float -> bf16 bit patterns via torch (round to nearest even); exact for the small
    integers and dyadic values used by the closed-form pins."""
    t = torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=np.float32)))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def place(per_seq, block_table, num_pages, H_kv, d, fill=np.nan) -> np.ndarray:
    """Lay out per-sequence rows [len][H_kv][d] into a bf16 pool through the block table
    (position p -> physical page block_table[b][p // 16], slot p % 16)."""
    pool = np.full((num_pages, H_kv, PAGE, d), fill, dtype=np.float32)
    for b, arr in enumerate(per_seq):
        arr = np.asarray(arr, dtype=np.float32)
        for j in range(arr.shape[0]):
            pool[block_table[b][j // PAGE], :, j % PAGE, :] = arr[j]
    return bits(pool)


def rand_layout(rng, lens, extra=3):
    pages = [(n + PAGE - 1) // PAGE for n in lens]
    num_pages = sum(pages) + extra
    perm = rng.permutation(num_pages)
    bt = np.zeros((len(lens), max(1, max(pages))), dtype=np.int32)
    pos = 0
    for b, n in enumerate(pages):
        bt[b, :n] = perm[pos:pos + n]
        pos += n
    return bt, num_pages


def _eval(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {"e": math.e, "exp": math.exp, "ln": math.log}))


# --------------------------------------------------------------------------------------------
# pins
# --------------------------------------------------------------------------------------------

def pin_golden_worked_example():
    """Hand-derived closed forms (tests/golden/two_keys_worked_example.json)."""
    spec = json.load(open(os.path.join(GOLDEN, "two_keys_worked_example.json")))
    sh = spec["shape"]
    bt = np.array(spec["block_table"], dtype=np.int32)
    for case in spec["cases"]:
        L = case["ctx_len"]
        n = len(case["new_k"])
        d = sh["head_dim"]
        cached_k = np.array(case["cached_k"], dtype=np.float32).reshape(L, 1, d)
        cached_v = np.array(case["cached_v"], dtype=np.float32).reshape(L, 1, d)
        kp = place([cached_k], bt, sh["num_pages"], 1, d, fill=0.0)
        vp = place([cached_v], bt, sh["num_pages"], 1, d, fill=0.0)
        cu = np.array([0, n], dtype=np.int32)
        k_new = bits(np.array(case["new_k"], dtype=np.float32).reshape(n, 1, d))
        v_new = bits(np.array(case["new_v"], dtype=np.float32).reshape(n, 1, d))
        kp, vp = oracle.kv_append(kp, vp, k_new, v_new, bt, np.array([L]), cu)
        q = bits(np.array(case["q"], dtype=np.float32).reshape(n, 1, d))
        o, lse = oracle.attention(q, kp, vp, bt, np.array([L]), cu, spec["scale"])
        exp_o = np.array([[_eval(x) for x in row] for row in case["expected_o"]])
        exp_lse = np.array([_eval(x) for x in case["expected_lse"]])
        assert np.allclose(o[:, 0, :], exp_o, rtol=0, atol=1e-14), (case["name"], o[:, 0, :], exp_o)
        assert np.allclose(lse[:, 0], exp_lse, rtol=0, atol=1e-14), (case["name"], lse, exp_lse)


def pin_kv_append_roundtrip_and_sentinel():
    """Appended rows read back exactly through the block table; every other byte is unchanged."""
    rng = np.random.default_rng(11)
    H_kv, d = 2, 64
    ctx = np.array([5, 16, 31, 0])
    ql = np.array([20, 1, 3, 17])
    bt, num_pages = rand_layout(rng, ctx + ql, extra=4)
    kp = rng.integers(0, 65536, size=(num_pages, H_kv, PAGE, d)).astype(np.uint16)
    vp = rng.integers(0, 65536, size=(num_pages, H_kv, PAGE, d)).astype(np.uint16)
    total = int(ql.sum())
    k_new = rng.integers(0, 65536, size=(total, H_kv, d)).astype(np.uint16)
    v_new = rng.integers(0, 65536, size=(total, H_kv, d)).astype(np.uint16)
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    kp2, vp2 = oracle.kv_append(kp, vp, k_new, v_new, bt, ctx, cu)
    touched = np.zeros((num_pages, PAGE), dtype=bool)
    for b in range(len(ctx)):
        for t in range(ql[b]):
            p = ctx[b] + t
            pg, sl = bt[b][p // PAGE], p % PAGE
            assert np.array_equal(kp2[pg, :, sl, :], k_new[cu[b] + t])
            assert np.array_equal(vp2[pg, :, sl, :], v_new[cu[b] + t])
            touched[pg, sl] = True
    assert touched.sum() == total
    untouched = ~touched
    assert np.array_equal(kp2.transpose(0, 2, 1, 3)[untouched], kp.transpose(0, 2, 1, 3)[untouched])
    assert np.array_equal(vp2.transpose(0, 2, 1, 3)[untouched], vp.transpose(0, 2, 1, 3)[untouched])


def pin_single_key_returns_v():
    """Empty context, one new token: softmax over one key is 1, so o = v exactly."""
    rng = np.random.default_rng(3)
    H_kv, G, d = 2, 4, 64
    bt = np.array([[5]], dtype=np.int32)
    kp = bits(np.zeros((8, H_kv, PAGE, d)))
    vp = bits(np.zeros((8, H_kv, PAGE, d)))
    k_new = bits(rng.standard_normal((1, H_kv, d)))
    v_new = bits(rng.standard_normal((1, H_kv, d)))
    kp, vp = oracle.kv_append(kp, vp, k_new, v_new, bt, np.array([0]), None)
    q = bits(rng.standard_normal((1, H_kv * G, d)))
    o, lse = oracle.attention(q, kp, vp, bt, np.array([0]), None, 0.125)
    vf = oracle.bf16_bits_to_f64(v_new)
    for h in range(H_kv * G):
        assert np.array_equal(o[0, h], vf[0, h // G])
        s = 0.125 * float(oracle.bf16_bits_to_f64(q[0, h]) @ oracle.bf16_bits_to_f64(k_new[0, h // G]))
        assert abs(lse[0, h] - s) < 1e-12


def pin_identical_keys_mean_of_v():
    """All keys equal: uniform weights; o = mean of v_0..v_p, lse = scale q.k + ln(p+1)."""
    rng = np.random.default_rng(4)
    H_kv, G, d = 1, 2, 64
    L, n = 37, 9
    bt, num_pages = rand_layout(rng, [L + n])
    kvec = rng.standard_normal(d)
    K = np.tile(kvec, (L + n, H_kv, 1))
    V = rng.standard_normal((L + n, H_kv, d))
    kp = place([K], bt, num_pages, H_kv, d)
    vp = place([V], bt, num_pages, H_kv, d)
    q = bits(rng.standard_normal((n, H_kv * G, d)))
    cu = np.array([0, n], dtype=np.int32)
    o, lse = oracle.attention(q, kp, vp, bt, np.array([L]), cu, 0.125)
    Vb = oracle.bf16_bits_to_f64(bits(V))
    kb = oracle.bf16_bits_to_f64(bits(kvec))
    for i in range(n):
        p = L + i
        for h in range(H_kv * G):
            assert np.allclose(o[i, h], Vb[:p + 1, 0].mean(axis=0), atol=1e-13, rtol=0)
            s = 0.125 * float(oracle.bf16_bits_to_f64(q[i, h]) @ kb)
            assert abs(lse[i, h] - (s + math.log(p + 1))) < 1e-12


def pin_gqa_mapping():
    """V of kv-head g is the constant g+1: q-head h must return floor(h/G)+1 exactly."""
    rng = np.random.default_rng(5)
    H_kv, G, d = 4, 4, 64
    L, n = 20, 3
    bt, num_pages = rand_layout(rng, [L + n])
    K = rng.standard_normal((L + n, H_kv, d))
    V = np.zeros((L + n, H_kv, d))
    for g in range(H_kv):
        V[:, g, :] = g + 1
    kp = place([K], bt, num_pages, H_kv, d)
    vp = place([V], bt, num_pages, H_kv, d)
    q = bits(rng.standard_normal((n, H_kv * G, d)))
    o, _ = oracle.attention(q, kp, vp, bt, np.array([L]), np.array([0, n]), 0.125)
    for h in range(H_kv * G):
        assert np.allclose(o[:, h, :], h // G + 1, atol=1e-13, rtol=0), h


def pin_position_encoded_v():
    """q = 0 gives uniform weights; with V[j,:] = j (exact in bf16 for j <= 256) the output of
    the token at position p is the prefix mean p/2 exactly.  Pins the mask boundary, the page
    gather and the q-row offsets of a ragged batch."""
    rng = np.random.default_rng(6)
    H_kv, G, d = 2, 2, 64
    ctx = np.array([0, 13, 40, 100])
    ql = np.array([17, 1, 30, 5])
    bt, num_pages = rand_layout(rng, ctx + ql, extra=5)
    per_k, per_v = [], []
    for b in range(4):
        n = ctx[b] + ql[b]
        per_k.append(rng.standard_normal((n, H_kv, d)))
        per_v.append(np.broadcast_to(np.arange(n, dtype=np.float64)[:, None, None], (n, H_kv, d)))
    kp = place(per_k, bt, num_pages, H_kv, d)
    vp = place(per_v, bt, num_pages, H_kv, d)
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    q = bits(np.zeros((int(ql.sum()), H_kv * G, d)))
    o, lse = oracle.attention(q, kp, vp, bt, ctx, cu, 0.125)
    for b in range(4):
        for i in range(ql[b]):
            p = ctx[b] + i
            assert np.allclose(o[cu[b] + i], p / 2.0, atol=1e-12, rtol=0), (b, i)
            assert np.allclose(lse[cu[b] + i], math.log(p + 1), atol=1e-12, rtol=0)


def pin_page_permutation_invariance():
    """Permuting physical pages and rewriting the block table leaves every output identical."""
    rng = np.random.default_rng(7)
    H_kv, G, d = 2, 4, 64
    ctx = np.array([50, 3, 77])
    ql = np.array([6, 1, 12])
    bt, num_pages = rand_layout(rng, ctx + ql, extra=2)
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    vp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    q = bits(rng.standard_normal((int(ql.sum()), H_kv * G, d)))
    o1, l1 = oracle.attention(q, kp, vp, bt, ctx, cu, 0.125)
    sigma = rng.permutation(num_pages)          # new physical id of old page i is sigma[i]
    kp2 = np.empty_like(kp); vp2 = np.empty_like(vp)
    kp2[sigma] = kp; vp2[sigma] = vp
    bt2 = sigma[bt].astype(np.int32)
    o2, l2 = oracle.attention(q, kp2, vp2, bt2, ctx, cu, 0.125)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    # and a different layout is actually different (the gather matters)
    o3, _ = oracle.attention(q, kp2, vp2, bt, ctx, cu, 0.125)
    assert not np.allclose(o1, o3)


def pin_prefill_equals_sequential_decode():
    """A causal prefill-append of n tokens equals n single-token decode steps on the same cache."""
    rng = np.random.default_rng(8)
    H_kv, G, d = 2, 2, 64
    L, n = 29, 7
    bt, num_pages = rand_layout(rng, [L + n])
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    vp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    k_new = bits(rng.standard_normal((n, H_kv, d)))
    v_new = bits(rng.standard_normal((n, H_kv, d)))
    q = bits(rng.standard_normal((n, H_kv * G, d)))
    cu = np.array([0, n], dtype=np.int32)
    kpa, vpa = oracle.kv_append(kp, vp, k_new, v_new, bt, np.array([L]), cu)
    o_pre, l_pre = oracle.attention(q, kpa, vpa, bt, np.array([L]), cu, 0.088388347648)
    kps, vps = kp, vp
    for t in range(n):
        kps, vps = oracle.kv_append(kps, vps, k_new[t:t + 1], v_new[t:t + 1], bt, np.array([L + t]), None)
        o_t, l_t = oracle.attention(q[t:t + 1], kps, vps, bt, np.array([L + t]), None, 0.088388347648)
        assert np.allclose(o_t[0], o_pre[t], atol=1e-12, rtol=0)
        assert np.allclose(l_t[0], l_pre[t], atol=1e-12, rtol=0)
    assert np.array_equal(kps, kpa) and np.array_equal(vps, vpa)


def pin_split_merge_equals_unsplit():
    """Splitting the visible keys into random ranges and merging by log-sum-exp is exact."""
    rng = np.random.default_rng(9)
    H_kv, G, d = 1, 4, 64
    ctx = np.array([90, 33])
    ql = np.array([4, 1])
    bt, num_pages = rand_layout(rng, ctx + ql)
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)) * 3)
    vp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    q = bits(rng.standard_normal((int(ql.sum()), H_kv * G, d)))
    o1, l1 = oracle.attention(q, kp, vp, bt, ctx, cu, 0.125)

    def cuts(b, i, vis):
        k = int(rng.integers(1, 6))
        return sorted(set(int(c) for c in rng.integers(1, vis, size=k)))
    o2, l2 = oracle.attention_split(q, kp, vp, bt, ctx, cu, 0.125, cuts)
    assert np.allclose(o1, o2, atol=1e-12, rtol=0) and np.allclose(l1, l2, atol=1e-12, rtol=0)


def pin_sdpa_reduction():
    """Contiguous pages: equals torch's scaled_dot_product_attention in float64 with K/V repeated
    over the group and an explicit boolean mask j <= L + i (bottom-right aligned causal)."""
    rng = np.random.default_rng(10)
    H_kv, G, d = 2, 4, 128
    for L, n in [(0, 24), (45, 10)]:
        kv = L + n
        npg = (kv + PAGE - 1) // PAGE
        bt = np.arange(npg, dtype=np.int32)[None, :]
        kp = bits(rng.standard_normal((npg, H_kv, PAGE, d)))
        vp = bits(rng.standard_normal((npg, H_kv, PAGE, d)))
        q = bits(rng.standard_normal((n, H_kv * G, d)))
        scale = float(np.float32(1 / math.sqrt(d)))
        o, lse = oracle.attention(q, kp, vp, bt, np.array([L]), np.array([0, n]), scale)
        Kc = oracle.bf16_bits_to_f64(kp).transpose(1, 0, 2, 3).reshape(H_kv, -1, d)[:, :kv]
        Vc = oracle.bf16_bits_to_f64(vp).transpose(1, 0, 2, 3).reshape(H_kv, -1, d)[:, :kv]
        Qt = torch.from_numpy(oracle.bf16_bits_to_f64(q).transpose(1, 0, 2).copy())[None]
        Kt = torch.from_numpy(Kc.copy()).repeat_interleave(G, dim=0)[None]
        Vt = torch.from_numpy(Vc.copy()).repeat_interleave(G, dim=0)[None]
        mask = torch.from_numpy(np.arange(kv)[None, :] <= (L + np.arange(n))[:, None])
        ref = torch.nn.functional.scaled_dot_product_attention(Qt, Kt, Vt, attn_mask=mask, scale=scale)
        ref = ref[0].numpy().transpose(1, 0, 2)
        assert np.allclose(o, ref, atol=1e-12, rtol=0), np.abs(o - ref).max()
        # lse against a direct logsumexp
        s = torch.einsum("hnd,hkd->hnk", Qt[0], Kt[0]) * scale
        s = s.masked_fill(~mask, -math.inf)
        ref_lse = torch.logsumexp(s, dim=-1).numpy().T
        assert np.allclose(lse, ref_lse, atol=1e-12, rtol=0)


def pin_linearity_in_v():
    """o(V1 + V2) = o(V1) + o(V2) for fixed Q, K."""
    rng = np.random.default_rng(12)
    H_kv, G, d = 2, 2, 64
    ctx = np.array([21]); ql = np.array([5])
    bt, num_pages = rand_layout(rng, ctx + ql)
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    v1 = rng.integers(-8, 8, size=(num_pages, H_kv, PAGE, d)).astype(np.float64)
    v2 = rng.integers(-8, 8, size=(num_pages, H_kv, PAGE, d)).astype(np.float64)
    q = bits(rng.standard_normal((5, H_kv * G, d)))
    cu = np.array([0, 5])
    oa, _ = oracle.attention(q, kp, bits(v1), bt, ctx, cu, 0.125)
    ob, _ = oracle.attention(q, kp, bits(v2), bt, ctx, cu, 0.125)
    oc, _ = oracle.attention(q, kp, bits(v1 + v2), bt, ctx, cu, 0.125)
    assert np.allclose(oa + ob, oc, atol=1e-12, rtol=0)


def pin_brute_force_scalar_loops():
    """On a tiny ragged batch, the numpy oracle equals pure-Python scalar loops."""
    rng = np.random.default_rng(13)
    H_kv, G, d = 2, 2, 64
    ctx = np.array([19, 0, 33]); ql = np.array([3, 2, 1])
    bt, num_pages = rand_layout(rng, ctx + ql, extra=1)
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    vp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    q = bits(rng.standard_normal((int(ql.sum()), H_kv * G, d)))
    o1, l1 = oracle.attention(q, kp, vp, bt, ctx, cu, 0.125)
    o2, l2 = oracle.attention_scalar_loops(q, kp, vp, bt, ctx, cu, 0.125)
    assert np.allclose(o1, o2, atol=1e-12, rtol=0) and np.allclose(l1, l2, atol=1e-12, rtol=0)


def pin_mixed_batch_independence():
    """Each sequence of a mixed batch (prefill chunks, decodes, empty) equals its own
    single-sequence call."""
    rng = np.random.default_rng(14)
    H_kv, G, d = 2, 4, 64
    ctx = np.array([40, 7, 0, 64]); ql = np.array([9, 1, 0, 1])
    bt, num_pages = rand_layout(rng, ctx + ql)
    kp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    vp = bits(rng.standard_normal((num_pages, H_kv, PAGE, d)))
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    q = bits(rng.standard_normal((int(ql.sum()), H_kv * G, d)))
    o, l = oracle.attention(q, kp, vp, bt, ctx, cu, 0.125)
    for b in range(4):
        if ql[b] == 0:
            continue
        ob, lb = oracle.attention(q[cu[b]:cu[b + 1]], kp, vp, bt[b:b + 1], ctx[b:b + 1],
                                  np.array([0, ql[b]]), 0.125)
        assert np.array_equal(ob, o[cu[b]:cu[b + 1]]) and np.array_equal(lb, l[cu[b]:cu[b + 1]])


def pin_bf16_rounding():
    """The reporting helper rounds to nearest, ties to even (checked on exact ties and on values
    next to ties), and widening is exact."""
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -30, -(1.0 + 3 * 2 ** -8), 0.1])
    b = oracle.f64_to_bf16_bits(x)
    assert [int(v) for v in b[:4]] == [0x3F80, 0x3F82, 0x3F81, 0xBF82]
    assert abs(oracle.bf16_bits_to_f64(b[4:5])[0] - 0.1) <= 2 ** -4 * 2 ** -8


def pin_kv_pack_closed_form():
    """Pools whose every row encodes its own address (K: page, head, slot, 0; V: the negatives
    minus one): packed row cu[b] + t of kv-head h must read (bt[b][p // 16], h, p % 16) with
    p = ctx[b] + t.  All codes are small integers, exact in bf16."""
    rng = np.random.default_rng(23)
    H_kv, d = 3, 4
    ctx = np.array([0, 15, 16, 40, 7])
    ql = np.array([17, 2, 16, 0, 1])
    bt, num_pages = rand_layout(rng, ctx + ql, extra=2)
    code = np.zeros((num_pages, H_kv, PAGE, d), dtype=np.float32)
    code[..., 0] = np.arange(num_pages)[:, None, None]
    code[..., 1] = np.arange(H_kv)[None, :, None]
    code[..., 2] = np.arange(PAGE)[None, None, :]
    kp, vp = bits(code), bits(-code - 1)
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    buf = pa.kv_pack(kp, vp, bt, ctx, cu)
    assert buf.shape == (2, int(ql.sum()), H_kv, d)
    got_k = oracle.bf16_bits_to_f64(buf[0])
    got_v = oracle.bf16_bits_to_f64(buf[1])
    for b in range(len(ctx)):
        for t in range(ql[b]):
            p = ctx[b] + t
            for h in range(H_kv):
                want = np.array([bt[b][p // PAGE], h, p % PAGE, 0.0])
                assert np.array_equal(got_k[cu[b] + t, h], want), (b, t, h)
                assert np.array_equal(got_v[cu[b] + t, h], -want - 1), (b, t, h)
    # one row per sequence when cu_q_lens is None: row b holds position ctx[b]
    one = pa.kv_pack(kp, vp, bt, ctx, None)
    for b in range(len(ctx)):
        p = ctx[b]
        assert np.array_equal(oracle.bf16_bits_to_f64(one[0, b, 2]), [bt[b][p // PAGE], 2, p % PAGE, 0.0])


def pin_kv_pack_unpack_transfer():
    """A transfer between two pools with different page placements: packing token ranges out of
    pool A and unpacking them into pool B makes B's gathered rows equal A's, leaves every other
    byte of B unchanged, and packing B again returns the same buffer."""
    rng = np.random.default_rng(29)
    H_kv, d = 2, 8
    ctx = np.array([3, 33, 0])
    ql = np.array([30, 1, 16])
    lens = ctx + ql
    bt_a, np_a = rand_layout(rng, lens, extra=1)
    bt_b, np_b = rand_layout(rng, lens, extra=5)
    kp_a = rng.integers(0, 65536, size=(np_a, H_kv, PAGE, d)).astype(np.uint16)
    vp_a = rng.integers(0, 65536, size=(np_a, H_kv, PAGE, d)).astype(np.uint16)
    kp_b = rng.integers(0, 65536, size=(np_b, H_kv, PAGE, d)).astype(np.uint16)
    vp_b = rng.integers(0, 65536, size=(np_b, H_kv, PAGE, d)).astype(np.uint16)
    cu = np.concatenate([[0], np.cumsum(ql)]).astype(np.int32)
    buf = pa.kv_pack(kp_a, vp_a, bt_a, ctx, cu)
    kb2, vb2 = pa.kv_unpack(kp_b, vp_b, buf, bt_b, ctx, cu)
    touched = np.zeros((np_b, PAGE), dtype=bool)
    for b in range(len(ctx)):
        for p in range(ctx[b], lens[b]):
            pa_, pb_, sl = bt_a[b][p // PAGE], bt_b[b][p // PAGE], p % PAGE
            assert np.array_equal(kb2[pb_, :, sl, :], kp_a[pa_, :, sl, :])
            assert np.array_equal(vb2[pb_, :, sl, :], vp_a[pa_, :, sl, :])
            touched[pb_, sl] = True
    keep = ~touched
    assert np.array_equal(kb2.transpose(0, 2, 1, 3)[keep], kp_b.transpose(0, 2, 1, 3)[keep])
    assert np.array_equal(vb2.transpose(0, 2, 1, 3)[keep], vp_b.transpose(0, 2, 1, 3)[keep])
    assert np.array_equal(pa.kv_pack(kb2, vb2, bt_b, ctx, cu), buf)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
