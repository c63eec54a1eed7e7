"""Pins that tie the PD decision-engine oracle (oracle/pd_model.py) to facts fixed independently of
it: a hand-worked example, algebraic identities of Eqs. 1-3, the capacity boundaries, the
hysteresis rules, exhaustive search for the minimal-change plan (the optimality argument of
section 4.4.2), the gate of Eq. 7 at its boundary, and exact recovery of noiseless refits.

Each ``pin_*`` raises AssertionError on a disagreement; ``test_pd_pins.py`` runs them and
``test_pd_mutations.py`` plants plausible mistakes in the oracle and checks that one fails."""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np

from oracle import pd_model as pm

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _ev(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {}))


def _params(**over):
    p = {"B": 64.0, "S": 4.0, "dL": 1000.0, "r": 500.0, "theta": 0.5, "A": 0.01, "b": 0.0005,
         "t_prefill": 1e-4, "T_over": 1.0, "T_env": 50.0, "K": 65536.0, "BW": 1.6384e10,
         "K_seq": 2e9, "H_max": 4e10, "u_max": 1.0}
    p.update(over)
    return p


def pin_golden_makespans():
    """Hand-worked makespans, feasibility and decisions (tests/golden/pd_makespan_worked_example.json)."""
    spec = json.load(open(os.path.join(GOLDEN, "pd_makespan_worked_example.json")))
    for case in spec["cases"]:
        p = {k: float(v) for k, v in case["params"].items()}
        N = case["N"]
        assert math.isclose(pm.makespan_coloc(p, N), _ev(case["coloc"]), rel_tol=1e-13), case["name"]
        for d in case["dis"]:
            pre, dec = _ev(d["prefill_path"]), _ev(d["decode_path"])
            assert math.isclose(pm.prefill_path(p, d["N_P"]), pre, rel_tol=1e-13), (case["name"], d)
            assert math.isclose(pm.decode_path(p, d["N_D"]), dec, rel_tol=1e-13), (case["name"], d)
            assert math.isclose(pm.makespan_dis(p, d["N_P"], d["N_D"]), max(pre, dec) + p["T_env"], rel_tol=1e-13)
            assert pm.feasible_dis(p, d["N_P"], d["N_D"]) == d["feasible"], (case["name"], d)
        best, _, _ = pm.best_config(p, N)
        want = case["decision"]
        assert best[0] == (pm.DIS if want["mode"] == "dis" else pm.COLOC), case["name"]
        if want["mode"] == "dis":
            assert (best[1], best[2]) == (want["N_P"], want["N_D"]), (case["name"], best)
        else:
            assert best[3] == N


def pin_no_bubbles_decode_path_is_colocated_decode_term():
    """theta = 0: Eq. 2 reduces to S r (A + b B / N_D), the decode term of Eq. 1 at N = N_D
    (Eq. 1 with dL = 0, T_over = 0, T_env = 0)."""
    for N_D in (1, 3, 8):
        p = _params(theta=0.0)
        q = _params(theta=0.0, dL=0.0, T_over=0.0, T_env=0.0)
        assert math.isclose(pm.decode_path(p, N_D), pm.makespan_coloc(q, N_D), rel_tol=1e-14)


def pin_bubbles_cost_fixed_iteration_time():
    """Eq. 2 is linear in theta with slope S r A: bubbles cost the fixed per-iteration time of the
    extra iterations, while the per-sequence term b B / N_D is unchanged."""
    p0, p1 = _params(theta=0.0), _params(theta=1.5)
    for N_D in (2, 5):
        slope = (pm.decode_path(p1, N_D) - pm.decode_path(p0, N_D)) / 1.5
        assert math.isclose(slope, p0["S"] * p0["r"] * p0["A"], rel_tol=1e-12)


def pin_transfer_term_is_volume_over_bandwidth():
    """Eq. 3's second term: doubling BW halves it, and it does not depend on N_P."""
    p, q = _params(), _params(BW=2 * 1.6384e10)
    t = p["S"] * p["B"] * p["dL"] * p["K"] / p["BW"]
    for N_P in (1, 4):
        assert math.isclose(pm.prefill_path(p, N_P) - pm.prefill_path(q, N_P), t / 2, rel_tol=1e-12)
    assert math.isclose(pm.prefill_path(_params(t_prefill=0.0), 1), t, rel_tol=1e-14)
    assert math.isclose(pm.prefill_path(_params(t_prefill=0.0), 7), t, rel_tol=1e-14)


def pin_capacity_boundaries():
    """B K_seq <= N_D H_max holds with equality; the prefill keep-pace test flips where
    lambda_P t_prefill / N_P crosses u_max * T_decode."""
    p = _params(K_seq=2e9, H_max=3.2e10, B=64.0)        # needs exactly N_D >= 4
    assert pm.feasible_dis(p, 1, 4) and not pm.feasible_dis(p, 1, 3)
    assert not pm.feasible_dis(p, 0, 8) and not pm.feasible_dis(p, 8, 0)
    q = _params(theta=0.0, r=50.0, A=0.01, b=0.0005, K_seq=1.0)
    dec = q["S"] * q["r"] * (q["A"] + q["b"] * q["B"] / 3)
    load = q["B"] * q["S"] * q["dL"] * q["t_prefill"]
    q_at = dict(q, u_max=load / 2 / dec)                # N_P = 2: busy time equals the cap
    assert pm.feasible_dis(q_at, 2, 3)
    assert not pm.feasible_dis(dict(q_at, u_max=q_at["u_max"] * (1 - 1e-9)), 2, 3)


def pin_enumeration_is_exhaustive_argmin():
    """The decision equals an exhaustive search over every split of N workers (colocation
    preferred on ties, then the smallest N_P), for random parameters."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        p = _params(theta=float(rng.uniform(0, 3)), T_over=float(rng.uniform(0, 10)),
                    r=float(rng.uniform(10, 2000)), dL=float(rng.uniform(100, 4000)),
                    BW=float(rng.uniform(1e9, 1e11)), K_seq=float(rng.uniform(1e8, 8e9)),
                    u_max=float(rng.uniform(0.5, 2.0)))
        N = int(rng.integers(2, 17))
        cands = [(pm.makespan_coloc(p, N), 0, pm.COLOC)]
        for N_P in range(1, N):
            if pm.feasible_dis(p, N_P, N - N_P):
                cands.append((pm.makespan_dis(p, N_P, N - N_P), 1 + N_P, pm.DIS))
        T, key, mode = min(cands)
        best, _, _ = pm.best_config(p, N)
        assert best[0] == mode and math.isclose(best[4], T, rel_tol=0, abs_tol=0)
        if mode == pm.DIS:
            assert best[1] == key - 1


def pin_hysteresis_rules():
    """A ratio change within disaggregation needs more than delta_ratio of gain, a mode switch
    more than delta_mode; an infeasible current topology forces the optimum."""
    p = _params(theta=0.1, T_over=20.0, K_seq=1e8)
    N = 8
    best, t_coloc, best_dis = pm.best_config(p, N)
    assert best[0] == pm.DIS
    cur = None
    for N_P in range(1, N):                              # a feasible non-optimal split
        if (N_P, N - N_P) != best[1:3] and pm.feasible_dis(p, N_P, N - N_P):
            cur = (pm.DIS, N_P, N - N_P)
            break
    gain = 1 - best[4] / pm.makespan_dis(p, cur[1], cur[2])
    assert gain > 0
    cfg, why = pm.decide(p, N, cur, delta_mode=1.0, delta_ratio=gain * 1.01)
    assert why == "keep" and cfg[1:3] == cur[1:3]
    cfg, why = pm.decide(p, N, cur, delta_mode=1.0, delta_ratio=gain * 0.99)
    assert why == "switch" and cfg[1:3] == best[1:3]
    # colocated now: disaggregation must beat it by delta_mode
    mode_gain = 1 - best[4] / t_coloc
    cfg, why = pm.decide(p, N, (pm.COLOC, 0, 0), delta_mode=mode_gain * 1.01, delta_ratio=0.0)
    assert why == "keep" and cfg[0] == pm.COLOC
    cfg, why = pm.decide(p, N, (pm.COLOC, 0, 0), delta_mode=mode_gain * 0.99, delta_ratio=0.0)
    assert why == "switch" and cfg[0] == pm.DIS
    # the current split no longer adds up to the budget, or breaks a capacity constraint
    cfg, why = pm.decide(p, N - 2, cur, delta_mode=1.0, delta_ratio=1.0)
    assert why == "forced" and cfg == pm.best_config(p, N - 2)[0]
    tight = dict(p, K_seq=p["H_max"] * 1.5 / p["B"])    # needs N_D >= 2
    cfg, why = pm.decide(tight, N, (pm.DIS, N - 1, 1), delta_mode=1.0, delta_ratio=1.0)
    assert why == "forced"
    assert pm.decide(p, N, None, 0.1, 0.05)[1] == "initial"


def _tables(rng, n_slots):
    cur = [int(x) for x in rng.integers(0, 4, size=n_slots)]
    target = [bool(x) for x in rng.integers(0, 2, size=n_slots)]
    m = sum(target)
    cuts = sorted(int(x) for x in rng.integers(0, m + 1, size=2))
    n_dst = {pm.ROLE_PREFILL: cuts[0], pm.ROLE_DECODE: cuts[1] - cuts[0], pm.ROLE_COLOC: m - cuts[1]}
    return cur, target, n_dst


def pin_plan_attains_the_minimum():
    """On enumerated small worker tables the plan meets the target counts, adds exactly W' \\ W,
    removes exactly W \\ W', and its change count equals both the exhaustive minimum and
    D_worker + D_role from Eqs. 5 and 6."""
    rng = np.random.default_rng(9)
    for trial in range(300):
        cur, target, n_dst = _tables(rng, int(rng.integers(1, 8)))
        new, dw, dr = pm.plan_min_change(cur, target, n_dst)
        for r in pm.ROLES:
            assert sum(1 for x in new if x == r) == n_dst[r]
        for w in range(len(cur)):
            assert (new[w] != pm.ROLE_NONE) == target[w]
        assert pm.change_count(cur, new) == (dw, dr)
        assert (dw, dr) == pm.eq5_eq6(cur, target, n_dst)
        assert dw + dr == pm.min_change_brute_force(cur, target, n_dst), (cur, target, n_dst)


def pin_plan_keeps_unaffected_workers():
    """A role-count change touching one worker changes one role; a departure with unchanged
    counts elsewhere changes membership only."""
    P, D, C = pm.ROLE_PREFILL, pm.ROLE_DECODE, pm.ROLE_COLOC
    cur = [P, P, D, D, D, D]
    new, dw, dr = pm.plan_min_change(cur, [True] * 6, {P: 1, D: 5, C: 0})
    assert (dw, dr) == (0, 1) and new == [P, D, D, D, D, D]
    new, dw, dr = pm.plan_min_change(cur, [True, True, True, True, True, False], {P: 2, D: 3, C: 0})
    assert (dw, dr) == (1, 0) and new[:5] == cur[:5] and new[5] == pm.ROLE_NONE
    new, dw, dr = pm.plan_min_change([0, 0, P, D], [True, True, True, True], {P: 1, D: 1, C: 2})
    assert (dw, dr) == (2, 0) and new == [C, C, P, D]


def pin_toggle_gate_boundary():
    """Eq. 7 is strict: equality does not borrow."""
    assert not pm.toggle_gate(32, 64, 110.0, 100.0, 5.0)         # (1/2) * 10 = 5
    assert pm.toggle_gate(33, 64, 110.0, 100.0, 5.0)
    assert not pm.toggle_gate(64, 64, 100.0, 110.0, 0.0)          # no gain
    p = _params()
    enable, T_ded, T_full = pm.toggle_decide(p, 4, 8, 64.0, 0.0)
    assert T_full <= T_ded and enable == (T_full < T_ded)


def pin_refits_recover_noiseless_parameters():
    """Least-squares refits return the generating A, b and t_prefill exactly (to rounding) on
    noiseless telemetry; theta(f = 1/2) = 1 and theta(f = 1) = 0."""
    c = np.array([8, 16, 32, 64, 128], dtype=np.float64)
    A, b = pm.fit_decode_cost(c, 0.012 + 3.5e-5 * c)
    assert math.isclose(A, 0.012, rel_tol=1e-10) and math.isclose(b, 3.5e-5, rel_tol=1e-10)
    tok = np.array([100.0, 1000.0, 5000.0])
    assert math.isclose(pm.fit_prefill_cost(tok, 2.5e-5 * tok), 2.5e-5, rel_tol=1e-12)
    assert pm.bubble_ratio(0.5) == 1.0 and pm.bubble_ratio(1.0) == 0.0
    assert pm.ema(10.0, 20.0, 0.25) == 12.5


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
