"""Plant plausible mistakes in the PD decision-engine oracle (on the CPU) and check that the pins
catch each one."""
import pytest

from oracle import pd_model as pm
from pd_pins import ALL_PINS

_decode_path = pm.decode_path
_prefill_path = pm.prefill_path
_coloc = pm.makespan_coloc
_plan = pm.plan_min_change
_feasible = pm.feasible_dis
_decide = pm.decide


def _decode_without_bubble_factor(p, N_D):
    return _decode_path(p, N_D) / (1.0 + p["theta"])


def _decode_bubbles_on_b(p, N_D):
    th = p["theta"]
    return p["S"] * p["r"] * (p["A"] + p["b"] * p["B"] / N_D) * (1.0 + th)


def _transfer_split_over_prefill_workers(p, N_P):
    return p["S"] * (p["B"] * p["dL"] / N_P * p["t_prefill"] + p["B"] * p["dL"] * p["K"] / p["BW"] / N_P)


def _coloc_without_overhead(p, N):
    return _coloc(dict(p, T_over=0.0), N)


def _plan_ignores_current_roles(cur_role, target_active, n_dst):
    blank = [pm.ROLE_NONE if a else r for r, a in zip(cur_role, target_active)]
    new, _, _ = _plan(blank, target_active, n_dst)
    dw, dr = pm.change_count(cur_role, new)
    return new, dw, dr


def _feasible_ignores_kv(p, N_P, N_D):
    return _feasible(dict(p, K_seq=0.0), N_P, N_D)


def _decide_absolute_threshold(p, N, current, delta_mode, delta_ratio):
    # thresholds taken as seconds instead of fractions
    if current is None:
        return _decide(p, N, current, delta_mode, delta_ratio)
    T = pm.makespan_coloc(p, N) if current[0] == pm.COLOC else pm.makespan_dis(p, current[1], current[2])
    return _decide(p, N, current, delta_mode / T, delta_ratio / T)


MUTATIONS = {
    "decode_path_without_bubble_factor": ("decode_path", _decode_without_bubble_factor),
    "bubbles_scale_b_not_A": ("decode_path", _decode_bubbles_on_b),
    "transfer_term_divided_by_N_P": ("prefill_path", _transfer_split_over_prefill_workers),
    "coloc_without_T_over": ("makespan_coloc", _coloc_without_overhead),
    "plan_ignores_current_roles": ("plan_min_change", _plan_ignores_current_roles),
    "capacity_ignores_kv": ("feasible_dis", _feasible_ignores_kv),
    "hysteresis_absolute": ("decide", _decide_absolute_threshold),
}


def _fails_some_pin():
    failed = []
    for pin in ALL_PINS:
        try:
            pin()
        except Exception:
            failed.append(pin.__name__)
    return failed


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pd_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(pm, attr, fn)
    assert _fails_some_pin(), "mutation %s passed every pin" % name
