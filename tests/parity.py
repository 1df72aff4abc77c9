"""Error measures shared by the GPU parity tests.

Two figures per output tensor, both required to stay within the tolerance
(1e-4 for fp32 storage, 2e-2 for bf16):

  frob  per head, ||gpu - ref||_F / ||ref||_F, the largest over the heads;
  elem  over every element, |gpu - ref| / (|ref| + rms(ref row)), where rms is
        the root mean square of the element's reference row (the 64 features of
        one token).  Small entries of a row are judged against the row's scale,
        large ones against themselves.  A reference row that is exactly zero must
        come back exactly zero.
"""
from __future__ import annotations

import sys

import numpy as np

TOL = {"f32": 1e-4, "bf16": 2e-2}

# (tag, tensor, frob, elem, tol) of every check in this session; the terminal
# summary of tests/conftest.py prints them, so a passing run still shows them.
RECORD = []


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def frob_error(gpu, ref) -> float:
    out = []
    for g, r in zip(gpu, ref):
        nr = np.linalg.norm(r)
        ng = np.linalg.norm(g - r)
        out.append(ng / nr if nr > 0 else (0.0 if ng == 0 else np.inf))
    return max(out) if out else 0.0


def elem_error(gpu, ref) -> float:
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    if r.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(r * r, axis=-1, keepdims=True))
    den = np.abs(r) + rms
    diff = np.abs(g - r)
    zero_rows = np.broadcast_to(rms == 0, diff.shape)
    if np.any(diff[zero_rows] != 0):
        return float("inf")
    safe = np.where(den > 0, den, 1.0)
    return float(np.max(np.where(zero_rows, 0.0, diff / safe)))


def errors(gpu, ref):
    return frob_error(gpu, ref), elem_error(gpu, ref)


def check_all(tag: str, pairs, tol: float) -> dict:
    """pairs: iterable of (name, gpu, ref).  Logs both figures of every tensor,
    then asserts them."""
    errs = {name: errors(g, r) for name, g, r in pairs}
    log(f"[{tag}] " + " ".join(f"{k}: frob {f:.2e} elem {e:.2e}" for k, (f, e) in errs.items()))
    RECORD.extend((tag, k, f, e, tol) for k, (f, e) in errs.items())
    for name, (f, e) in errs.items():
        assert f <= tol and e <= tol, (tag, name, f, e, tol)
    return errs
