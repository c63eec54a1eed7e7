"""CPU oracle for the PD decision engine, the minimal-change orchestration plan and the
intra-scale toggle gate.

TEST INFRASTRUCTURE ONLY.  This is the plain reference that the library's native decision
engine is checked against.  Only tests, the smoke check and the benchmark may import it; it
imports numpy and nothing else, and shares no code with the library.

Everything here is double precision, evaluated in the order the equations are written.

What is computed (paper, section 4: Design)
-------------------------------------------
* Colocated batch makespan, Eq. 1:
      T_coloc = S [ (B dL / N) t_prefill + r (A + b B / N) + T_over ] + T_env
* Disaggregated decode path, Eq. 2 (bubble ratio theta = (1 - f) / f):
      T_decode = S r (A + b B / (N_D (1 + theta))) (1 + theta)
* Disaggregated prefill path, Eq. 3:
      T_prefill = S ( (B dL / N_P) t_prefill + B dL K / BW )
  and T_dis = max(T_prefill, T_decode) + T_env.
* Capacity constraints (section 4.2): the decode pool holds the batch's KV cache,
  B K_seq <= N_D H_max; the prefill pool keeps up with the prefill token load
  lambda_P = B S dL.
* Decision (section 4.3.2): enumerate N_P in [1, N - 1] with N_D = N - N_P, drop infeasible
  ones, compare the best against colocation, with mode-dependent hysteresis.
* Minimal-change plan (section 4.4.2, Eqs. 5 and 6): D_worker = |W' \\ W| + |W \\ W'|,
  D_role = sum_r [n_src(r) - min(n_src(r), n_dst(r))]; keeping each survivor's role up to the
  target count and filling deficits with added and reassigned workers attains the minimum.
* Toggle gate (section 4.6, Eq. 7): borrow when (R / B)(T_ded - T_full) > T_toggle.
* Runtime refits (section 4.3.2 and Implementation, runtime statistics): A and b from
  (concurrency, iteration time) telemetry, t_prefill from (tokens, time) telemetry, theta from
  the active-decode fraction f, and an exponential moving average for the toggle cost.

Readings where the paper is silent
----------------------------------
* Prefill capacity: lambda_P t_prefill / N_P <= u_max * T_decode(N_D), i.e. the prefill pool's
  busy time per step must not exceed the decode path it feeds (u_max, a utilisation cap, is an
  input; 1 means "keeps pace").
* Colocation is always feasible (the paper's fallback).
* Ties: colocation unless a disaggregated configuration is strictly faster; among
  disaggregated configurations the smallest N_P wins.
* Hysteresis thresholds are relative: a candidate c different from the current configuration
  is admitted when T(c) < T(cur) (1 - delta), delta = delta_mode for a colocation <->
  disaggregation switch and delta_ratio for a ratio change; the admitted candidate with the
  smallest makespan wins, else the current configuration is kept.  A disaggregated current
  configuration whose counts do not add up to N, or that violates a capacity constraint, forces
  a switch to the unconstrained optimum.  A colocated current configuration is valid at any N.
* Plan determinism: survivors keep their role in ascending slot order; deficits are filled role
  by role (prefill, decode, colocated), first with reassigned survivors, then with added
  workers, each in ascending slot order.
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

COLOC, DIS = 0, 1
ROLE_NONE, ROLE_PREFILL, ROLE_DECODE, ROLE_COLOC = 0, 1, 2, 3
ROLES = (ROLE_PREFILL, ROLE_DECODE, ROLE_COLOC)

PARAM_KEYS = ("B", "S", "dL", "r", "theta", "A", "b", "t_prefill", "T_over", "T_env", "K", "BW",
              "K_seq", "H_max", "u_max")


# ------------------------------------------------------------------------------------------
# makespan models
# ------------------------------------------------------------------------------------------

def makespan_coloc(p: Dict[str, float], N: int) -> float:
    """Eq. 1."""
    t_pre_turn = p["B"] * p["dL"] / N * p["t_prefill"]
    t_dec_turn = p["r"] * (p["A"] + p["b"] * p["B"] / N)
    return p["S"] * (t_pre_turn + t_dec_turn + p["T_over"]) + p["T_env"]


def decode_path(p: Dict[str, float], N_D: int) -> float:
    """Eq. 2."""
    th = p["theta"]
    return p["S"] * p["r"] * (p["A"] + p["b"] * p["B"] / (N_D * (1.0 + th))) * (1.0 + th)


def prefill_path(p: Dict[str, float], N_P: int) -> float:
    """Eq. 3."""
    return p["S"] * (p["B"] * p["dL"] / N_P * p["t_prefill"] + p["B"] * p["dL"] * p["K"] / p["BW"])


def makespan_dis(p: Dict[str, float], N_P: int, N_D: int) -> float:
    return max(prefill_path(p, N_P), decode_path(p, N_D)) + p["T_env"]


def feasible_dis(p: Dict[str, float], N_P: int, N_D: int) -> bool:
    """Capacity constraints of a disaggregated configuration (section 4.2)."""
    if N_P < 1 or N_D < 1:
        return False
    holds_kv = p["B"] * p["K_seq"] <= N_D * p["H_max"]
    lam = p["B"] * p["S"] * p["dL"]
    keeps_pace = lam * p["t_prefill"] / N_P <= p["u_max"] * decode_path(p, N_D)
    return bool(holds_kv and keeps_pace)


# ------------------------------------------------------------------------------------------
# decision engine
# ------------------------------------------------------------------------------------------

def best_config(p: Dict[str, float], N: int):
    """Enumeration over N_P in [1, N-1]; returns (best, T_coloc, best_dis) where configurations
    are tuples (mode, N_P, N_D, N_C, T) and best_dis is None when none is feasible."""
    t_coloc = makespan_coloc(p, N)
    best_dis = None
    for N_P in range(1, N):
        N_D = N - N_P
        if not feasible_dis(p, N_P, N_D):
            continue
        T = makespan_dis(p, N_P, N_D)
        if best_dis is None or T < best_dis[4]:
            best_dis = (DIS, N_P, N_D, 0, T)
    best = (COLOC, 0, 0, N, t_coloc)
    if best_dis is not None and best_dis[4] < t_coloc:
        best = best_dis
    return best, t_coloc, best_dis


def decide(p: Dict[str, float], N: int, current: Optional[Tuple[int, int, int]], delta_mode: float,
           delta_ratio: float):
    """Target configuration for budget N given the current one ((mode, N_P, N_D) or None).
    Returns (config, reason) with reason 'initial', 'forced', 'switch' or 'keep'."""
    best, t_coloc, best_dis = best_config(p, N)
    if current is None:
        return best, "initial"
    mode, cp, cd = current
    if mode == DIS and (cp + cd != N or not feasible_dis(p, cp, cd)):
        return best, "forced"
    if mode == COLOC:
        cur = (COLOC, 0, 0, N, t_coloc)
    else:
        cur = (DIS, cp, cd, 0, makespan_dis(p, cp, cd))
    admitted = None
    for cand in ((COLOC, 0, 0, N, t_coloc), best_dis):
        if cand is None or cand[:4] == cur[:4]:
            continue
        delta = delta_mode if cand[0] != cur[0] else delta_ratio
        if cand[4] < cur[4] * (1.0 - delta):
            if admitted is None or cand[4] < admitted[4]:
                admitted = cand
    if admitted is None:
        return cur, "keep"
    return admitted, "switch"


# ------------------------------------------------------------------------------------------
# minimal-change plan
# ------------------------------------------------------------------------------------------

def plan_min_change(cur_role: Sequence[int], target_active: Sequence[bool], n_dst: Dict[int, int]):
    """Role table after the transition: cur_role[w] in {0 (not active), 1, 2, 3}; target_active[w]
    says whether slot w is in W'.  n_dst maps each role to its target count, and the counts must
    add up to |W'|.  Returns (new_role, D_worker, D_role)."""
    n = len(cur_role)
    assert len(target_active) == n
    active_now = [cur_role[w] != ROLE_NONE for w in range(n)]
    assert sum(n_dst.get(r, 0) for r in ROLES) == sum(bool(a) for a in target_active)
    survivors = [w for w in range(n) if active_now[w] and target_active[w]]
    added = [w for w in range(n) if not active_now[w] and target_active[w]]
    removed = [w for w in range(n) if active_now[w] and not target_active[w]]
    new_role = [ROLE_NONE] * n
    kept = {r: 0 for r in ROLES}
    excess = []
    for w in survivors:
        r = cur_role[w]
        if kept[r] < n_dst.get(r, 0):
            new_role[w] = r
            kept[r] += 1
        else:
            excess.append(w)
    pool = excess + added
    i = 0
    for r in ROLES:
        for _ in range(n_dst.get(r, 0) - kept[r]):
            new_role[pool[i]] = r
            i += 1
    assert i == len(pool)
    d_worker = len(added) + len(removed)
    d_role = len(excess)
    return new_role, d_worker, d_role


def change_count(cur_role: Sequence[int], new_role: Sequence[int]) -> Tuple[int, int]:
    """(membership changes, role changes among survivors) of a transition, counted directly."""
    d_worker = sum(1 for a, b in zip(cur_role, new_role) if (a == ROLE_NONE) != (b == ROLE_NONE))
    d_role = sum(1 for a, b in zip(cur_role, new_role) if a != ROLE_NONE and b != ROLE_NONE and a != b)
    return d_worker, d_role


def min_change_brute_force(cur_role: Sequence[int], target_active: Sequence[bool], n_dst: Dict[int, int]) -> int:
    """Smallest D_worker + D_role over every assignment of roles to W' with the target counts."""
    targets = [w for w in range(len(cur_role)) if target_active[w]]
    multiset = []
    for r in ROLES:
        multiset += [r] * n_dst.get(r, 0)
    best = None
    for perm in set(itertools.permutations(multiset)):
        new_role = [ROLE_NONE] * len(cur_role)
        for w, r in zip(targets, perm):
            new_role[w] = r
        dw, dr = change_count(cur_role, new_role)
        if best is None or dw + dr < best:
            best = dw + dr
    return 0 if best is None else best


def eq5_eq6(cur_role: Sequence[int], target_active: Sequence[bool], n_dst: Dict[int, int]) -> Tuple[int, int]:
    """D_worker and D_role evaluated straight from Eqs. 5 and 6."""
    W = {w for w, r in enumerate(cur_role) if r != ROLE_NONE}
    W2 = {w for w, a in enumerate(target_active) if a}
    S = W & W2
    d_worker = len(W2 - W) + len(W - W2)
    d_role = 0
    for r in ROLES:
        n_src = sum(1 for w in S if cur_role[w] == r)
        d_role += n_src - min(n_src, n_dst.get(r, 0))
    return d_worker, d_role


# ------------------------------------------------------------------------------------------
# toggle gate and runtime refits
# ------------------------------------------------------------------------------------------

def toggle_gate(R: float, B: float, T_ded: float, T_full: float, T_toggle: float) -> bool:
    """Eq. 7."""
    return (R / B) * (T_ded - T_full) > T_toggle


def toggle_decide(p: Dict[str, float], n_ded: int, n_overlap: int, R: float, T_toggle: float):
    """Eq. 7 with T_ded and T_full the best predicted makespans on the dedicated workers alone and
    on dedicated plus overlap workers."""
    T_ded = best_config(p, n_ded)[0][4]
    T_full = best_config(p, n_ded + n_overlap)[0][4]
    return toggle_gate(R, p["B"], T_ded, T_full, T_toggle), T_ded, T_full


def fit_decode_cost(concurrency: Sequence[float], iter_time: Sequence[float]) -> Tuple[float, float]:
    """Least-squares line iter_time = A + b * concurrency (the decode term of Eq. 1)."""
    x = np.asarray(concurrency, dtype=np.float64)
    y = np.asarray(iter_time, dtype=np.float64)
    M = np.stack([np.ones_like(x), x], axis=1)
    (A, b), *_ = np.linalg.lstsq(M, y, rcond=None)
    return float(A), float(b)


def fit_prefill_cost(tokens: Sequence[float], time: Sequence[float]) -> float:
    """Least-squares t_prefill with time = tokens * t_prefill (per-token prefill time)."""
    x = np.asarray(tokens, dtype=np.float64)
    y = np.asarray(time, dtype=np.float64)
    return float((x * y).sum() / (x * x).sum())


def bubble_ratio(f: float) -> float:
    """theta = (1 - f) / f for an active-decode fraction f (section 4.3.1)."""
    return (1.0 - f) / f


def ema(prev: float, obs: float, alpha: float) -> float:
    """Exponential moving average step."""
    return alpha * obs + (1.0 - alpha) * prev
