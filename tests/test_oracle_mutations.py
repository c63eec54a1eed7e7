"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins catch each one."""
import numpy as np
import pytest

from oracle import paged_attention as pa
from oracle_pins import ALL_PINS


def _fails_some_pin():
    failed = []
    for pin in ALL_PINS:
        try:
            pin()
        except Exception:  # AssertionError or an indexing error caused by the mutation
            failed.append(pin.__name__)
    return failed


_orig_unit = pa.attention_unit
_orig_gather = pa.gather_kv
_orig_merge = pa.merge_states


def _unit_no_scale(q_rows, K, V, ctx_len, scale):
    return _orig_unit(q_rows, K, V, ctx_len, 1.0)


def _gather_v_is_k(k_pool, v_pool, row, kv_len, kv_head):
    K, V = _orig_gather(k_pool, v_pool, row, kv_len, kv_head)
    return K, K


def _unit_lse_without_max(q_rows, K, V, ctx_len, scale):
    o, lse = _orig_unit(q_rows, K, V, ctx_len, scale)
    n = q_rows.shape[0]
    for i in range(n):
        vis = ctx_len + i + 1
        lse[i] -= (scale * (K[:vis] @ q_rows[i])).max()
    return o, lse


def _merge_drops_rescale(states):
    l_star = sum(l for _, m, l in states if l > 0)
    acc = sum(o for o, m, l in states if l > 0)
    m_star = max(m for _, m, _ in states)
    return acc / l_star, m_star + np.log(l_star)


_orig_pack = pa.kv_pack


def _pack_k_v_swapped(k_pool, v_pool, block_table, ctx_lens, cu_q_lens):
    return _orig_pack(k_pool, v_pool, block_table, ctx_lens, cu_q_lens)[::-1]


def _pack_rows_shifted(k_pool, v_pool, block_table, ctx_lens, cu_q_lens):
    return _orig_pack(k_pool, v_pool, block_table, np.asarray(ctx_lens) + 1, cu_q_lens)


MUTATIONS = {
    "gqa_mod_instead_of_div": ("_kv_head_of", lambda h, group: h % group),
    "exclusive_causal_mask": ("_visible", lambda ctx_len, i: ctx_len + i),
    "mask_one_too_many": ("_visible", lambda ctx_len, i: ctx_len + i + 2),
    "page_slot_swapped": ("_page_slot", lambda row, pos: (row[pos % 16], pos // 16)),
    "slot_from_wrong_page_size": ("_page_slot", lambda row, pos: (row[pos // 16], pos % 8)),
    "q_rows_offset_by_one_seq": ("_q_starts", lambda cu, batch: (np.arange(batch) if cu is None
                                                                 else np.asarray(cu)[1:])),
    "scale_dropped": ("attention_unit", _unit_no_scale),
    "v_operand_is_k": ("gather_kv", _gather_v_is_k),
    "lse_missing_max": ("attention_unit", _unit_lse_without_max),
    "merge_without_rescale": ("merge_states", _merge_drops_rescale),
    "pack_k_v_swapped": ("kv_pack", _pack_k_v_swapped),
    "pack_rows_shifted": ("kv_pack", _pack_rows_shifted),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(pa, attr, fn)
    failed = _fails_some_pin()
    assert failed, "mutation %s passed every pin" % name
