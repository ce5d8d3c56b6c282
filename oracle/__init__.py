"""fp64 CPU oracle for the R-iKFAD optimiser step (ctypes binding).

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this module.  It wraps the
plain C implementation in ``rikfad_oracle.c`` (built by ``oracle.build``),
which follows the paper's App. A Table of sub-step updates literally in
fp64, and ``adafm_oracle.c``, the paper's Adafactor-m baseline step.  It shares no code with the GPU package and never imports it.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("RIKFAD_ORACLE_LIB") or os.path.join(_HERE, "liboracle_rikfad.so")

_lib = None


class _HP(ctypes.Structure):
    _fields_ = [("h", ctypes.c_double), ("gamma", ctypes.c_double),
                ("alpha", ctypes.c_double), ("mu", ctypes.c_double),
                ("eps_stab", ctypes.c_double)]


class _AdaHP(ctypes.Structure):
    _fields_ = [("h", ctypes.c_double), ("beta1", ctypes.c_double),
                ("decay_rate", ctypes.c_double), ("eps1", ctypes.c_double),
                ("eps2", ctypes.c_double), ("clip_threshold", ctypes.c_double),
                ("scale_parameter", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class _Tensor(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("x_unrounded", ctypes.c_void_p),
                ("g", ctypes.c_void_p), ("p", ctypes.c_void_p),
                ("r", ctypes.c_void_p), ("c", ctypes.c_void_p),
                ("m", ctypes.c_int64), ("n", ctypes.c_int64),
                ("x_bf16", ctypes.c_int32), ("reserved", ctypes.c_int32)]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"oracle library {LIB_PATH} is not built; run oracle.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        hp = ctypes.POINTER(_HP)
        L.orc_coefficients.argtypes = [hp, vp]
        L.orc_rank1_friction.argtypes = [i64, i64, vp, vp, ctypes.c_double, vp]
        L.orc_rikfad_matrix_step.argtypes = [i64, i64, i32, vp, vp, vp, vp, vp, vp, hp]
        L.orc_ikfad_step.argtypes = [i64, i32, vp, vp, vp, vp, vp, hp]
        L.orc_rikfad_step_list.argtypes = [i64, vp, hp, ctypes.c_int]
        L.orc_round_bf16.argtypes = [ctypes.c_double]
        L.orc_round_bf16.restype = ctypes.c_double
        L.orc_round_bf16_array.argtypes = [vp, vp, i64]
        L.orc_round_bf16_array.restype = None
        L.orc_quadratic_run.argtypes = [i64, i64, vp, vp, vp, vp, vp, hp, i64, i64,
                                        vp, vp]
        ahp = ctypes.POINTER(_AdaHP)
        L.orc_adafm_beta2.argtypes = [i64, ctypes.c_double]
        L.orc_adafm_beta2.restype = ctypes.c_double
        L.orc_adafm_matrix_step.argtypes = [i64, i64, i64, i32, vp, vp, vp, vp, vp, vp, ahp]
        L.orc_adafm_vector_step.argtypes = [i64, i64, i32, vp, vp, vp, vp, vp, ahp]
        L.orc_adafm_step_list.argtypes = [i64, vp, i64, ahp, ctypes.c_int]
        for fn in (L.orc_coefficients, L.orc_rank1_friction, L.orc_rikfad_matrix_step,
                   L.orc_ikfad_step, L.orc_rikfad_step_list, L.orc_quadratic_run,
                   L.orc_adafm_matrix_step, L.orc_adafm_vector_step, L.orc_adafm_step_list):
            fn.restype = ctypes.c_int
        _lib = L
    return _lib


@dataclass
class HParams:
    h: float
    gamma: float = 0.0
    alpha: float = 0.1
    mu: float = 1.0
    eps_stab: float = 1e-8

    def _c(self):
        return _HP(self.h, self.gamma, self.alpha, self.mu, self.eps_stab)


def _f64(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    return a


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def coefficients(hp: HParams):
    """(exp(-alpha h), (1 - exp(-alpha h))/(mu alpha), exp(-gamma h))."""
    out = np.zeros(3)
    _check(lib().orc_coefficients(ctypes.byref(hp._c()), out.ctypes.data), "coefficients")
    return tuple(out)


def rank1_friction(r, c, eps_stab):
    r, c = _f64(r), _f64(c)
    xi = np.empty((r.size, c.size))
    _check(lib().orc_rank1_friction(r.size, c.size, r.ctypes.data, c.ctypes.data,
                                    float(eps_stab), xi.ctypes.data), "rank1_friction")
    return xi


def round_bf16(v):
    v = _f64(v)
    out = np.empty_like(v)
    lib().orc_round_bf16_array(v.ctypes.data, out.ctypes.data, v.size)
    return out


def _need_f64(name, a):
    if a.dtype != np.float64 or not a.flags.c_contiguous:
        raise TypeError(f"{name} must be a C-contiguous float64 array")


def rikfad_matrix_step(x, g, p, r, c, hp: HParams, x_bf16=False, x_unrounded=None):
    """One BACD step on an m x n matrix; x, p, r, c (float64) updated in place."""
    m, n = x.shape
    for nm, a in (("x", x), ("p", p), ("r", r), ("c", c)):
        _need_f64(nm, a)
    g = _f64(g)
    if x_unrounded is not None:
        _need_f64("x_unrounded", x_unrounded)
    _check(lib().orc_rikfad_matrix_step(m, n, int(bool(x_bf16)), x.ctypes.data,
                                        _ptr(x_unrounded), g.ctypes.data, p.ctypes.data,
                                        r.ctypes.data, c.ctypes.data,
                                        ctypes.byref(hp._c())), "matrix step")


def ikfad_step(x, g, p, xi, hp: HParams, x_bf16=False, x_unrounded=None):
    """One element-wise iKFAD step; x, p, xi (float64) updated in place."""
    for nm, a in (("x", x), ("p", p), ("xi", xi)):
        _need_f64(nm, a)
    g = _f64(g)
    if x_unrounded is not None:
        _need_f64("x_unrounded", x_unrounded)
    _check(lib().orc_ikfad_step(x.size, int(bool(x_bf16)), x.ctypes.data,
                                _ptr(x_unrounded), g.ctypes.data, p.ctypes.data,
                                xi.ctypes.data, ctypes.byref(hp._c())), "ikfad step")


@dataclass
class OracleTensor:
    """State of one parameter tensor in fp64.  For a vector (m == 1 or n == 1)
    the element-wise friction lives in ``c`` when m == 1, else in ``r``."""
    m: int
    n: int
    bf16: bool
    x: np.ndarray
    p: np.ndarray
    r: np.ndarray
    c: np.ndarray
    x_unrounded: np.ndarray = field(default=None)

    @property
    def is_vector(self):
        return self.m == 1 or self.n == 1

    @property
    def xi(self):
        return self.c if self.m == 1 else self.r


def make_tensor(x0, bf16=False, p0=None, r0=None, c0=None, track_unrounded=False):
    """Oracle state from a 2-D initial parameter array (values are taken exactly)."""
    x0 = np.asarray(x0)
    m, n = x0.shape
    x = np.array(x0, dtype=np.float64, order="C")
    p = np.zeros((m, n)) if p0 is None else np.array(p0, dtype=np.float64, order="C")
    r = np.zeros(m) if r0 is None else np.array(r0, dtype=np.float64)
    c = np.zeros(n) if c0 is None else np.array(c0, dtype=np.float64)
    xu = np.zeros((m, n)) if track_unrounded else None
    return OracleTensor(m, n, bool(bf16), x, p, r, c, xu)


def step_list(tensors, grads, hp: HParams, threads=1):
    """One R-iKFAD step over a list of OracleTensor with matching gradients."""
    arr = (_Tensor * max(1, len(tensors)))()
    keep = []
    for i, (t, g) in enumerate(zip(tensors, grads)):
        g = _f64(g)
        if g.size != t.m * t.n:
            raise ValueError("gradient size mismatch")
        keep.append(g)
        arr[i] = _Tensor(t.x.ctypes.data, _ptr(t.x_unrounded), g.ctypes.data,
                         t.p.ctypes.data, t.r.ctypes.data, t.c.ctypes.data,
                         t.m, t.n, int(t.bf16), 0)
    _check(lib().orc_rikfad_step_list(len(tensors), ctypes.addressof(arr),
                                      ctypes.byref(hp._c()), int(threads)), "step_list")


def quadratic_run(A, x, p, r, c, hp: HParams, nsteps, every):
    """Integrate the quadratic test problem; returns (energies, max relative
    increase of the modified energy).  x, p are m x n float64 (updated)."""
    m, n = x.shape
    A = _f64(A)
    for nm, a in (("x", x), ("p", p), ("r", r), ("c", c)):
        _need_f64(nm, a)
    energy = np.empty(nsteps // every + 1)
    worst = ctypes.c_double(0.0)
    _check(lib().orc_quadratic_run(m, n, A.ctypes.data, x.ctypes.data, p.ctypes.data,
                                   r.ctypes.data, c.ctypes.data, ctypes.byref(hp._c()),
                                   int(nsteps), int(every), energy.ctypes.data,
                                   ctypes.byref(worst)), "quadratic_run")
    return energy, worst.value


def friction_report(xi, eps_stab):
    """Rank-1 friction statistics of a full iKFAD friction tensor (Section 4,
    "How Close is xi~ to the Best Rank-1 Friction?"), from their definitions:
    shadow factors R = xi 1 and C = xi^T 1 (the R-iKFAD filter fed by the
    same P^(1), started at zero, is linear and equals these sums), rank-1
    friction xi~ = R C^T / (1^T R + eps_stab) (0 if the denominator is 0),
    relative error |xi - xi~|_F / |xi|_F, leading singular value sigma_1
    from numpy's SVD, Eckart-Young floor sqrt(1 - sigma_1^2 / |xi|_F^2) and
    stable rank |xi|_F^2 / sigma_1^2.  fp64."""
    xi = np.asarray(xi, dtype=np.float64)
    r = xi.sum(axis=1)
    c = xi.sum(axis=0)
    s = r.sum()
    denom = s + eps_stab
    xit = np.outer(r, c) / denom if denom != 0.0 else np.zeros_like(xi)
    fro2 = float(np.sum(xi * xi))
    err2 = float(np.sum((xi - xit) ** 2))
    sigma1 = float(np.linalg.svd(xi, compute_uv=False)[0])
    ratio = sigma1 ** 2 / fro2 if fro2 > 0 else 1.0
    return {"xi_fro2": fro2, "err_fro2": err2, "sum_r": float(s), "sigma1": sigma1,
            "rel_err": float(np.sqrt(err2 / fro2)) if fro2 > 0 else 0.0,
            "eckart_young_floor": float(np.sqrt(max(0.0, 1.0 - ratio))),
            "stable_rank": fro2 / sigma1 ** 2 if sigma1 > 0 else 0.0}


# ------------------------------------------------------------- Adafactor-m

@dataclass
class AdafmHParams:
    """Adafactor-m hyperparameters: step size h, first-moment decay beta1,
    second-moment schedule beta2_t = 1 - t^decay_rate, eps1 added to G^2,
    eps2 floor of RMS(X) for the optional parameter scale, update clipping
    threshold (<= 0: off)."""
    h: float
    beta1: float = 0.9
    decay_rate: float = -0.8
    eps1: float = 1e-30
    eps2: float = 1e-3
    clip_threshold: float = 1.0
    scale_parameter: bool = False

    def _c(self):
        return _AdaHP(self.h, self.beta1, self.decay_rate, self.eps1, self.eps2,
                      self.clip_threshold, int(bool(self.scale_parameter)), 0)


def adafm_beta2(t, decay_rate=-0.8):
    """Second-moment decay of step t: 1 - t^decay_rate."""
    return lib().orc_adafm_beta2(int(t), float(decay_rate))


def adafm_matrix_step(x, g, mom, r, c, t, hp: AdafmHParams, x_bf16=False, x_unrounded=None):
    """Adafactor-m step t on an m x n matrix; x, mom, r, c updated in place."""
    m, n = x.shape
    for nm, a in (("x", x), ("mom", mom), ("r", r), ("c", c)):
        _need_f64(nm, a)
    g = _f64(g)
    if x_unrounded is not None:
        _need_f64("x_unrounded", x_unrounded)
    _check(lib().orc_adafm_matrix_step(m, n, int(t), int(bool(x_bf16)), x.ctypes.data,
                                       _ptr(x_unrounded), g.ctypes.data, mom.ctypes.data,
                                       r.ctypes.data, c.ctypes.data, ctypes.byref(hp._c())),
           "adafm matrix step")


def adafm_vector_step(x, g, mom, v, t, hp: AdafmHParams, x_bf16=False, x_unrounded=None):
    """Adafactor-m step t on a non-2D parameter (unfactored second moment v)."""
    for nm, a in (("x", x), ("mom", mom), ("v", v)):
        _need_f64(nm, a)
    g = _f64(g)
    if x_unrounded is not None:
        _need_f64("x_unrounded", x_unrounded)
    _check(lib().orc_adafm_vector_step(x.size, int(t), int(bool(x_bf16)), x.ctypes.data,
                                       _ptr(x_unrounded), g.ctypes.data, mom.ctypes.data,
                                       v.ctypes.data, ctypes.byref(hp._c())),
           "adafm vector step")


def adafm_step_list(tensors, grads, t, hp: AdafmHParams, threads=1):
    """Adafactor-m step t over a list of OracleTensor (p = first moment; a
    vector keeps its second moment in ``xi``)."""
    arr = (_Tensor * max(1, len(tensors)))()
    keep = []
    for i, (T, g) in enumerate(zip(tensors, grads)):
        g = _f64(g)
        if g.size != T.m * T.n:
            raise ValueError("gradient size mismatch")
        keep.append(g)
        arr[i] = _Tensor(T.x.ctypes.data, _ptr(T.x_unrounded), g.ctypes.data,
                         T.p.ctypes.data, T.r.ctypes.data, T.c.ctypes.data,
                         T.m, T.n, int(T.bf16), 0)
    _check(lib().orc_adafm_step_list(len(tensors), ctypes.addressof(arr), int(t),
                                     ctypes.byref(hp._c()), int(threads)), "adafm step_list")
