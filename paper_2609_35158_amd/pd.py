"""ctypes binding of the PD decision engine, minimal-change plan and toggle gate
(include/pearl_pd.h).  Argument marshalling only: every decision is computed by the native
library; there is no Python fallback.

Parameters are dicts with the keys of ``PARAM_KEYS``; configurations are tuples
(mode, N_P, N_D, N_C, makespan) with mode COLOC = 0 or DIS = 1."""
from __future__ import annotations

import ctypes
from typing import Dict, Optional, Sequence, Tuple

from .binding import PearlError, last_error, load as _load_lib

COLOC, DIS, NONE = 0, 1, -1
ROLE_NONE, ROLE_PREFILL, ROLE_DECODE, ROLE_COLOC = 0, 1, 2, 3
REASONS = {0: "initial", 1: "keep", 2: "switch", 3: "forced"}
PARAM_KEYS = ("B", "S", "dL", "r", "theta", "A", "b", "t_prefill", "T_over", "T_env", "K", "BW",
              "K_seq", "H_max", "u_max")

EXPORTED = ("pearl_pd_makespan_coloc", "pearl_pd_decode_path", "pearl_pd_prefill_path",
            "pearl_pd_makespan_dis", "pearl_pd_feasible_dis", "pearl_pd_best", "pearl_pd_decide",
            "pearl_plan_min_change", "pearl_toggle_gate", "pearl_toggle_decide",
            "pearl_pd_fit_decode_cost", "pearl_pd_fit_prefill_cost", "pearl_pd_bubble_ratio",
            "pearl_pd_ema")


class PdParams(ctypes.Structure):
    _fields_ = [(k, ctypes.c_double) for k in PARAM_KEYS]


class PdConfig(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("n_p", ctypes.c_int32), ("n_d", ctypes.c_int32),
                ("n_c", ctypes.c_int32), ("makespan", ctypes.c_double)]


_typed = False


def load():
    global _typed
    lib = _load_lib()
    if _typed:
        return lib
    P, D, I = ctypes.POINTER, ctypes.c_double, ctypes.c_int32
    for name, args in (("pearl_pd_makespan_coloc", [P(PdParams), I]), ("pearl_pd_decode_path", [P(PdParams), I]),
                       ("pearl_pd_prefill_path", [P(PdParams), I]),
                       ("pearl_pd_makespan_dis", [P(PdParams), I, I])):
        f = getattr(lib, name)
        f.restype, f.argtypes = D, args
    lib.pearl_pd_feasible_dis.restype = I
    lib.pearl_pd_feasible_dis.argtypes = [P(PdParams), I, I]
    lib.pearl_pd_best.restype = ctypes.c_int
    lib.pearl_pd_best.argtypes = [P(PdParams), I, P(PdConfig), P(PdConfig), P(D)]
    lib.pearl_pd_decide.restype = ctypes.c_int
    lib.pearl_pd_decide.argtypes = [P(PdParams), I, P(PdConfig), D, D, P(PdConfig), P(I)]
    lib.pearl_plan_min_change.restype = ctypes.c_int
    lib.pearl_plan_min_change.argtypes = [I, P(I), P(ctypes.c_uint8), I, I, I, P(I), P(I), P(I)]
    lib.pearl_toggle_gate.restype = I
    lib.pearl_toggle_gate.argtypes = [D, D, D, D, D]
    lib.pearl_toggle_decide.restype = ctypes.c_int
    lib.pearl_toggle_decide.argtypes = [P(PdParams), I, I, D, D, P(I), P(D), P(D)]
    lib.pearl_pd_fit_decode_cost.restype = ctypes.c_int
    lib.pearl_pd_fit_decode_cost.argtypes = [P(D), P(D), I, P(D), P(D)]
    lib.pearl_pd_fit_prefill_cost.restype = ctypes.c_int
    lib.pearl_pd_fit_prefill_cost.argtypes = [P(D), P(D), I, P(D)]
    lib.pearl_pd_bubble_ratio.restype = D
    lib.pearl_pd_bubble_ratio.argtypes = [D]
    lib.pearl_pd_ema.restype = D
    lib.pearl_pd_ema.argtypes = [D, D, D]
    _typed = True
    return lib


def _params(p: Dict[str, float]) -> PdParams:
    missing = [k for k in PARAM_KEYS if k not in p]
    if missing:
        raise KeyError("missing parameters: %s" % ", ".join(missing))
    return PdParams(*[float(p[k]) for k in PARAM_KEYS])


def _check(st: int, func: str) -> None:
    if st != 0:
        raise PearlError(st, func, last_error())


def _tuple(c: PdConfig):
    if c.mode == NONE:
        return None
    return (int(c.mode), int(c.n_p), int(c.n_d), int(c.n_c), float(c.makespan))


def makespan_coloc(p, n: int) -> float:
    return load().pearl_pd_makespan_coloc(ctypes.byref(_params(p)), n)


def decode_path(p, n_d: int) -> float:
    return load().pearl_pd_decode_path(ctypes.byref(_params(p)), n_d)


def prefill_path(p, n_p: int) -> float:
    return load().pearl_pd_prefill_path(ctypes.byref(_params(p)), n_p)


def makespan_dis(p, n_p: int, n_d: int) -> float:
    return load().pearl_pd_makespan_dis(ctypes.byref(_params(p)), n_p, n_d)


def feasible_dis(p, n_p: int, n_d: int) -> bool:
    r = load().pearl_pd_feasible_dis(ctypes.byref(_params(p)), n_p, n_d)
    if r < 0:
        raise PearlError(1, "pearl_pd_feasible_dis", "invalid parameters")
    return bool(r)


def best_config(p, n: int):
    """(best, T_coloc, best_dis or None)."""
    best, bd, tc = PdConfig(), PdConfig(), ctypes.c_double()
    _check(load().pearl_pd_best(ctypes.byref(_params(p)), n, ctypes.byref(best), ctypes.byref(bd),
                                ctypes.byref(tc)), "pearl_pd_best")
    return _tuple(best), float(tc.value), _tuple(bd)


def decide(p, n: int, current: Optional[Tuple[int, int, int]], delta_mode: float, delta_ratio: float):
    """(target config, reason) for budget n given the current (mode, N_P, N_D) or None."""
    cur = None
    if current is not None:
        mode, n_p, n_d = current
        cur = PdConfig(mode, n_p, n_d, n if mode == COLOC else 0, 0.0)
    tgt, why = PdConfig(), ctypes.c_int32()
    _check(load().pearl_pd_decide(ctypes.byref(_params(p)), n, None if cur is None else ctypes.byref(cur),
                                  delta_mode, delta_ratio, ctypes.byref(tgt), ctypes.byref(why)), "pearl_pd_decide")
    return _tuple(tgt), REASONS[why.value]


def plan_min_change(cur_role: Sequence[int], target_active: Sequence[bool], n_prefill: int, n_decode: int,
                    n_coloc: int):
    """(new_role list, D_worker, D_role)."""
    n = len(cur_role)
    cr = (ctypes.c_int32 * max(n, 1))(*cur_role)
    ta = (ctypes.c_uint8 * max(n, 1))(*[1 if a else 0 for a in target_active])
    out = (ctypes.c_int32 * max(n, 1))()
    dw, dr = ctypes.c_int32(), ctypes.c_int32()
    _check(load().pearl_plan_min_change(n, cr, ta, n_prefill, n_decode, n_coloc, out, ctypes.byref(dw),
                                        ctypes.byref(dr)), "pearl_plan_min_change")
    return [int(out[i]) for i in range(n)], int(dw.value), int(dr.value)


def toggle_gate(R: float, B: float, T_ded: float, T_full: float, T_toggle: float) -> bool:
    r = load().pearl_toggle_gate(R, B, T_ded, T_full, T_toggle)
    if r < 0:
        raise PearlError(1, "pearl_toggle_gate", "invalid arguments")
    return bool(r)


def toggle_decide(p, n_ded: int, n_overlap: int, R: float, T_toggle: float):
    """(enable, T_ded, T_full)."""
    en, td, tf = ctypes.c_int32(), ctypes.c_double(), ctypes.c_double()
    _check(load().pearl_toggle_decide(ctypes.byref(_params(p)), n_ded, n_overlap, R, T_toggle, ctypes.byref(en),
                                      ctypes.byref(td), ctypes.byref(tf)), "pearl_toggle_decide")
    return bool(en.value), float(td.value), float(tf.value)


def _darr(xs):
    xs = [float(x) for x in xs]
    return (ctypes.c_double * max(len(xs), 1))(*xs), len(xs)


def fit_decode_cost(concurrency, iter_time) -> Tuple[float, float]:
    x, n = _darr(concurrency)
    y, m = _darr(iter_time)
    if n != m:
        raise ValueError("concurrency and iter_time differ in length")
    A, b = ctypes.c_double(), ctypes.c_double()
    _check(load().pearl_pd_fit_decode_cost(x, y, n, ctypes.byref(A), ctypes.byref(b)), "pearl_pd_fit_decode_cost")
    return float(A.value), float(b.value)


def fit_prefill_cost(tokens, time) -> float:
    x, n = _darr(tokens)
    y, m = _darr(time)
    if n != m:
        raise ValueError("tokens and time differ in length")
    t = ctypes.c_double()
    _check(load().pearl_pd_fit_prefill_cost(x, y, n, ctypes.byref(t)), "pearl_pd_fit_prefill_cost")
    return float(t.value)


def bubble_ratio(f: float) -> float:
    return load().pearl_pd_bubble_ratio(f)


def ema(prev: float, obs: float, alpha: float) -> float:
    return load().pearl_pd_ema(prev, obs, alpha)
