"""CPU oracle for YOSO attention (fp64, plain loops in C).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of
the bench are the only users.  The product path (the HIP library and its Python
binding) never imports this package, and this package imports nothing from it.

Each wrapper converts its inputs to contiguous fp64 / uint16 arrays and calls the
matching routine in ``yoso_oracle.c``; see that file for the paper passages the
routines follow.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "yoso_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math: fp64 operations stay as written)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-D_DEFAULT_SOURCE", "-fPIC", "-shared",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I64, I32 = ctypes.c_int64, ctypes.c_int
        lib.oracle_hash.argtypes = [P, I64, I64, I32, P, I32, I32, P, P]
        lib.oracle_forward.argtypes = [P, P, P, I64, I64, I64, I32, I32, I32, P]
        lib.oracle_backward.argtypes = [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, P, P, P]
        lib.oracle_backward_d2.argtypes = [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, P, P]
        lib.oracle_expectation.argtypes = [P, P, P, P, I64, I64, I64, I32, I32, ctypes.c_double, P, P, P, P, P, P]
        lib.oracle_backward_star.argtypes = [P, P, P, P, P, P, I64, I64, I64, I32, I32, I32, ctypes.c_double,
                                             P, P, P]
        lib.oracle_l2_normalize.argtypes = [P, I64, I32, P]
        lib.oracle_l2_normalize_backward.argtypes = [P, P, I64, I32, P]
        lib.oracle_hadamard.argtypes = [I32, P]
        lib.oracle_fast_hyperplanes.argtypes = [P, I32, I32, I32, P]
        lib.oracle_collision_prob.argtypes = [ctypes.c_double, I32]
        lib.oracle_collision_prob.restype = ctypes.c_double
        for fn in ("oracle_hash", "oracle_forward", "oracle_backward", "oracle_backward_d2", "oracle_backward_star",
                   "oracle_expectation", "oracle_l2_normalize", "oracle_l2_normalize_backward",
                   "oracle_hadamard", "oracle_fast_hyperplanes"):
            getattr(lib, fn).restype = None
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _u16(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint16)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def hash_codes(x, R, m: int, tau: int, with_margin: bool = False):
    """codes[bh, m, n] (uint16) of rows x[bh, n, d] under hyperplanes R[d, m*tau].

    With ``with_margin`` also returns min_b |projection| per (bh, h, i)."""
    x = _f64(x)
    R = _f64(R)
    bh, n, d = x.shape
    assert R.shape == (d, m * tau)
    codes = np.zeros((bh, m, n), np.uint16)
    margin = np.zeros((bh, m, n), np.float64) if with_margin else None
    _load().oracle_hash(_ptr(x), bh, n, d, _ptr(R), m, tau, _ptr(codes),
                        _ptr(margin) if with_margin else None)
    return (codes, margin) if with_margin else codes


def forward(qc, kc, v, m: int, tau: int) -> np.ndarray:
    qc, kc, v = _u16(qc), _u16(kc), _f64(v)
    bh, nk, d = v.shape
    nq = qc.shape[2]
    assert qc.shape == (bh, m, nq) and kc.shape == (bh, m, nk)
    y = np.zeros((bh, nq, d), np.float64)
    _load().oracle_forward(_ptr(qc), _ptr(kc), _ptr(v), bh, nq, nk, d, m, tau, _ptr(y))
    return y


def backward(qc, kc, q, k, v, dy, m: int, tau: int):
    """(dq, dk, dv) of the sampled surrogate backward, pairwise bucket form."""
    qc, kc = _u16(qc), _u16(kc)
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    bh, nq, d = q.shape
    nk = k.shape[1]
    dq = np.zeros((bh, nq, d))
    dk = np.zeros((bh, nk, d))
    dv = np.zeros((bh, nk, d))
    _load().oracle_backward(_ptr(qc), _ptr(kc), _ptr(q), _ptr(k), _ptr(v), _ptr(dy),
                            bh, nq, nk, d, m, tau, _ptr(dq), _ptr(dk), _ptr(dv))
    return dq, dk, dv


def backward_d2(qc, kc, q, k, v, dy, m: int, tau: int):
    """(dq, dk) of the same surrogate via d runs of the bucket-table subroutine."""
    qc, kc = _u16(qc), _u16(kc)
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    bh, nq, d = q.shape
    nk = k.shape[1]
    dq = np.zeros((bh, nq, d))
    dk = np.zeros((bh, nk, d))
    _load().oracle_backward_d2(_ptr(qc), _ptr(kc), _ptr(q), _ptr(k), _ptr(v), _ptr(dy),
                               bh, nq, nk, d, m, tau, _ptr(dq), _ptr(dk))
    return dq, dk


# Bound of 1 - x^2 in *YOSO's weight 1/(pi sqrt(1 - x^2)) (|x| <= 0.99216, at most
# 8/pi): the reading taken here of the divergence that Sec. 3.3 points out.
STAR_FLOOR = 1.0 / 64.0


def backward_star(qc, kc, q, k, v, dy, m: int, tau: int, floor: float = STAR_FLOOR):
    """(dq, dk, dv) of *YOSO: the sampled estimate of the true gradient of
    eq. (gradient-q) (pairs whose codes agree on all bits but at most one), and
    dv of eq. (gradient-v)."""
    qc, kc = _u16(qc), _u16(kc)
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    bh, nq, d = q.shape
    nk = k.shape[1]
    assert qc.shape == (bh, m, nq) and kc.shape == (bh, m, nk)
    dq = np.zeros((bh, nq, d))
    dk = np.zeros((bh, nk, d))
    dv = np.zeros((bh, nk, d))
    _load().oracle_backward_star(_ptr(qc), _ptr(kc), _ptr(q), _ptr(k), _ptr(v), _ptr(dy),
                                 bh, nq, nk, d, m, tau, float(floor), _ptr(dq), _ptr(dk), _ptr(dv))
    return dq, dk, dv


def expectation(q, k, v, dy, tau: int, true_grad: bool = False, floor: float = 0.0):
    """E[Y], E[dV], E[dQ], E[dK] over hash functions; with ``true_grad`` also the
    true gradients of eq. (gradient-q) for Q and K, their 1 - cos^2 raised to at
    least ``floor``."""
    q, k, v, dy = _f64(q), _f64(k), _f64(v), _f64(dy)
    bh, nq, d = q.shape
    nk = k.shape[1]
    ey = np.zeros((bh, nq, d))
    edv = np.zeros((bh, nk, d))
    edq = np.zeros((bh, nq, d))
    edk = np.zeros((bh, nk, d))
    tdq = np.zeros((bh, nq, d)) if true_grad else None
    tdk = np.zeros((bh, nk, d)) if true_grad else None
    _load().oracle_expectation(_ptr(q), _ptr(k), _ptr(v), _ptr(dy), bh, nq, nk, d, tau, float(floor),
                               _ptr(ey), _ptr(edv), _ptr(edq), _ptr(edk),
                               _ptr(tdq) if true_grad else None, _ptr(tdk) if true_grad else None)
    out = (ey, edv, edq, edk)
    return out + (tdq, tdk) if true_grad else out


def l2_normalize(x) -> np.ndarray:
    """Rows of x[..., d] divided by their Euclidean norms (zero rows stay zero)."""
    x = _f64(x)
    d = x.shape[-1]
    y = np.zeros_like(x)
    _load().oracle_l2_normalize(_ptr(x), x.size // d if d else 0, d, _ptr(y))
    return y


def l2_normalize_backward(x, dy) -> np.ndarray:
    """Gradient w.r.t. x of <dy, l2_normalize(x)>, row by row, from the explicit Jacobian."""
    x, dy = _f64(x), _f64(dy)
    assert x.shape == dy.shape
    d = x.shape[-1]
    dx = np.zeros_like(x)
    _load().oracle_l2_normalize_backward(_ptr(x), _ptr(dy), x.size // d if d else 0, d, _ptr(dx))
    return dx


def hadamard(d: int) -> np.ndarray:
    """Sylvester's Walsh-Hadamard matrix of order d (a power of two)."""
    assert d >= 1 and d & (d - 1) == 0
    H = np.zeros((d, d), np.float64)
    _load().oracle_hadamard(d, _ptr(H))
    return H


def fast_hyperplanes(signs, d: int, m: int, tau: int) -> np.ndarray:
    """R[d, m*tau] of the fast hash: the rows of the pseudo-random rotations
    (1/d) H D3 H D2 H D1, rotation r giving columns r*d .. r*d+d-1.
    ``signs``: uint64[ceil(m*tau/d), 3]; bit l of signs[r, i] negates coordinate l in D_{i+1}."""
    assert d >= 1 and d & (d - 1) == 0 and d <= 64
    nrot = (m * tau + d - 1) // d
    signs = np.ascontiguousarray(signs, dtype=np.uint64).reshape(-1)
    assert signs.size == 3 * nrot
    R = np.zeros((d, m * tau), np.float64)
    _load().oracle_fast_hyperplanes(_ptr(signs), d, m, tau, _ptr(R))
    return R


def fast_hash_codes(x, signs, m: int, tau: int, with_margin: bool = False):
    """The fast hash: the sign hash of x under the hyperplanes of fast_hyperplanes."""
    d = np.shape(x)[-1]
    return hash_codes(x, fast_hyperplanes(signs, d, m, tau), m, tau, with_margin=with_margin)


def collision_prob(x: float, tau: int) -> float:
    return _load().oracle_collision_prob(float(x), int(tau))


def run_all(inp: dict, m: int, tau: int, heads: Optional[slice] = None):
    """Hash + forward + backward for a batch of heads; returns a dict of fp64 arrays."""
    sl = heads if heads is not None else slice(None)
    q, k, v, dy = inp["q"][sl], inp["k"][sl], inp["v"][sl], inp["dy"][sl]
    qc = hash_codes(q, inp["R"], m, tau)
    kc = hash_codes(k, inp["R"], m, tau)
    y = forward(qc, kc, v, m, tau)
    dq, dk, dv = backward(qc, kc, q, k, v, dy, m, tau)
    return dict(qc=qc, kc=kc, y=y, dq=dq, dk=dk, dv=dv)
