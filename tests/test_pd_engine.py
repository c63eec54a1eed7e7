"""The native PD decision engine, plan generator and toggle gate (include/pearl_pd.h, through
the C ABI) against the oracle (oracle/pd_model.py).  Host code only: runs without a GPU.

Both sides evaluate the equations in double precision in the written order, so makespans and
feasibility must agree exactly and decisions must be identical; the least-squares refits use
different (equivalent) formulas and agree to 1e-9 relative."""
import json
import math
import os

import numpy as np
import pytest

from oracle import pd_model as pm
from paper_2609_35158_amd import pd
from paper_2609_35158_amd.binding import PearlError

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rand_params(rng):
    return {"B": float(rng.choice([16, 32, 64, 96, 128])), "S": float(rng.integers(1, 60)),
            "dL": float(rng.uniform(50, 8000)), "r": float(rng.uniform(20, 4000)),
            "theta": float(rng.uniform(0, 4)), "A": float(rng.uniform(0.002, 0.05)),
            "b": float(rng.uniform(1e-6, 1e-3)), "t_prefill": float(rng.uniform(1e-6, 5e-4)),
            "T_over": float(rng.uniform(0, 30)), "T_env": float(rng.uniform(0, 600)),
            "K": float(rng.choice([65536, 98304, 147456])), "BW": float(rng.uniform(5e9, 1e11)),
            "K_seq": float(rng.uniform(1e8, 1e10)), "H_max": float(rng.uniform(1e10, 8e10)),
            "u_max": float(rng.uniform(0.3, 2.0))}


def test_golden_example_through_the_native_engine():
    spec = json.load(open(os.path.join(GOLDEN, "pd_makespan_worked_example.json")))
    for case in spec["cases"]:
        p = {k: float(v) for k, v in case["params"].items()}
        N = case["N"]
        assert pd.makespan_coloc(p, N) == pm.makespan_coloc(p, N)
        for d in case["dis"]:
            assert pd.prefill_path(p, d["N_P"]) == pm.prefill_path(p, d["N_P"])
            assert pd.decode_path(p, d["N_D"]) == pm.decode_path(p, d["N_D"])
            assert pd.feasible_dis(p, d["N_P"], d["N_D"]) == d["feasible"]
        assert pd.best_config(p, N) == pm.best_config(p, N)


@pytest.mark.parametrize("seed", range(4))
def test_models_and_enumeration_match_exactly(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(400):
        p = _rand_params(rng)
        N = int(rng.integers(1, 33))
        assert pd.makespan_coloc(p, N) == pm.makespan_coloc(p, N)
        for n_p in range(1, N):
            n_d = N - n_p
            assert pd.prefill_path(p, n_p) == pm.prefill_path(p, n_p)
            assert pd.decode_path(p, n_d) == pm.decode_path(p, n_d)
            assert pd.makespan_dis(p, n_p, n_d) == pm.makespan_dis(p, n_p, n_d)
            assert pd.feasible_dis(p, n_p, n_d) == pm.feasible_dis(p, n_p, n_d)
        assert pd.best_config(p, N) == pm.best_config(p, N)


@pytest.mark.parametrize("seed", range(4))
def test_decisions_match(seed):
    rng = np.random.default_rng(200 + seed)
    reasons = set()
    for _ in range(500):
        p = _rand_params(rng)
        N = int(rng.integers(2, 25))
        dm, dr = float(rng.uniform(0, 0.3)), float(rng.uniform(0, 0.1))
        kind = int(rng.integers(0, 4))
        if kind == 0:
            cur = None
        elif kind == 1:
            cur = (pm.COLOC, 0, 0)
        else:
            Nc = N if kind == 2 else int(rng.integers(2, 25))
            n_p = int(rng.integers(1, Nc))
            cur = (pm.DIS, n_p, Nc - n_p)
        want = pm.decide(p, N, cur, dm, dr)
        got = pd.decide(p, N, cur, dm, dr)
        assert got == want, (p, N, cur, dm, dr)
        reasons.add(want[1])
    assert reasons == {"initial", "keep", "switch", "forced"}


def test_plans_match_and_are_minimal():
    rng = np.random.default_rng(7)
    for _ in range(500):
        n = int(rng.integers(0, 40))
        cur = [int(x) for x in rng.integers(0, 4, size=n)]
        target = [bool(x) for x in rng.integers(0, 2, size=n)]
        m = sum(target)
        cuts = sorted(int(x) for x in rng.integers(0, m + 1, size=2))
        counts = (cuts[0], cuts[1] - cuts[0], m - cuts[1])
        n_dst = dict(zip(pm.ROLES, counts))
        want = pm.plan_min_change(cur, target, n_dst)
        got = pd.plan_min_change(cur, target, *counts)
        assert got == tuple(want) or list(got) == list(want), (cur, target, counts)
        assert (got[1], got[2]) == pm.eq5_eq6(cur, target, n_dst)
    # exhaustive minimum on small tables
    for _ in range(100):
        n = int(rng.integers(1, 7))
        cur = [int(x) for x in rng.integers(0, 4, size=n)]
        target = [bool(x) for x in rng.integers(0, 2, size=n)]
        m = sum(target)
        cuts = sorted(int(x) for x in rng.integers(0, m + 1, size=2))
        counts = (cuts[0], cuts[1] - cuts[0], m - cuts[1])
        new, dw, dr = pd.plan_min_change(cur, target, *counts)
        assert dw + dr == pm.min_change_brute_force(cur, target, dict(zip(pm.ROLES, counts)))


def test_toggle_gate_and_decision_match():
    rng = np.random.default_rng(11)
    for _ in range(300):
        R, B = float(rng.integers(0, 129)), float(rng.choice([32, 64, 128]))
        a, c, t = (float(x) for x in rng.uniform(0, 500, size=3))
        assert pd.toggle_gate(R, B, a, c, t) == pm.toggle_gate(R, B, a, c, t)
    for _ in range(200):
        p = _rand_params(rng)
        n_ded, n_ov = int(rng.integers(1, 9)), int(rng.integers(0, 9))
        R, Tt = float(rng.uniform(0, p["B"])), float(rng.uniform(0, 200))
        got = pd.toggle_decide(p, n_ded, n_ov, R, Tt)
        assert got == pm.toggle_decide(p, n_ded, n_ov, R, Tt)


def test_refits_match():
    rng = np.random.default_rng(13)
    for _ in range(100):
        x = rng.uniform(1, 256, size=int(rng.integers(2, 20)))
        y = 0.01 + 4e-5 * x + rng.normal(0, 1e-4, size=x.size)
        A0, b0 = pm.fit_decode_cost(x, y)
        A1, b1 = pd.fit_decode_cost(x, y)
        assert math.isclose(A0, A1, rel_tol=1e-9, abs_tol=1e-15) and math.isclose(b0, b1, rel_tol=1e-9)
        tok = rng.uniform(1, 1e4, size=x.size)
        tim = 3e-5 * tok * rng.uniform(0.9, 1.1, size=x.size)
        assert math.isclose(pm.fit_prefill_cost(tok, tim), pd.fit_prefill_cost(tok, tim), rel_tol=1e-12)
    for f in (0.1, 0.5, 0.75, 1.0):
        assert pd.bubble_ratio(f) == pm.bubble_ratio(f)
    assert math.isnan(pd.bubble_ratio(0.0))
    assert pd.ema(3.0, 7.0, 0.125) == pm.ema(3.0, 7.0, 0.125)


def test_invalid_arguments_are_rejected():
    p = _rand_params(np.random.default_rng(1))
    with pytest.raises(PearlError):
        pd.best_config(dict(p, BW=0.0), 4)
    with pytest.raises(PearlError):
        pd.best_config(dict(p, theta=float("nan")), 4)
    with pytest.raises(PearlError):
        pd.best_config(p, 0)
    with pytest.raises(PearlError):
        pd.decide(p, 4, None, 1.5, 0.0)
    with pytest.raises(PearlError):
        pd.plan_min_change([1, 2], [True, True], 1, 0, 0)          # counts do not add up to |W'|
    with pytest.raises(PearlError):
        pd.plan_min_change([7], [True], 1, 0, 0)                    # not a role
    with pytest.raises(PearlError):
        pd.fit_decode_cost([4, 4, 4], [1.0, 2.0, 3.0])              # one distinct concurrency
    assert math.isnan(pd.makespan_coloc(dict(p, B=-1.0), 4))
    with pytest.raises(PearlError):
        pd.feasible_dis(dict(p, u_max=0.0), 1, 1)
