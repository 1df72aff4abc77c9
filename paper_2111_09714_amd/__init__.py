"""MI355X (gfx950) YOSO attention: Python binding of libyoso.so.

The binding only marshals arguments: every step of the computation runs in the
HIP kernels behind the C ABI declared in include/yoso.h.  There is no fallback:
if the library is missing or a call fails, an exception is raised.

Function names follow the C ABI:
    yoso_hash(x, R, m, tau, codes)                     codes[bh, n, m] (int16/uint16 storage)
    yoso_fast_hyperplanes(signs, m, tau, R)            R of the fast hash's pseudo-random rotations
    yoso_fast_hash(x, signs, m, tau, codes)            the fast hash (Walsh-Hadamard rotations per row)
    yoso_forward(qcodes, kcodes, v, m, tau, y, ws)     y = (1/m) sum_h B_h v
    yoso_backward(qcodes, kcodes, q, k, v, dy, m, tau, dq, dk, dv, ws)
    yoso_workspace_bytes(op, bh, n_q, n_k, d, m, tau, dtype) -> bytes
Tensors are torch tensors on one GPU, contiguous, [bh, n, 64], all float32 or all
bfloat16 (R is float32, codes 16-bit).  Work is enqueued on the current torch
stream unless `stream` is given.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = [
    "YosoError", "F32", "BF16", "OP_HASH", "OP_FORWARD", "OP_BACKWARD", "OP_BACKWARD_STAR",
    "lib", "lib_path", "yoso_workspace_bytes", "yoso_status_str", "yoso_hash", "yoso_fast_hyperplanes", "yoso_fast_hash", "yoso_forward",
    "yoso_backward", "yoso_backward_star", "backward_star", "yoso_backward_noalloc", "yoso_backward_noalloc_limit", "yoso_backward_table_threshold", "yoso_l2_normalize", "yoso_l2_normalize_backward", "yoso_expectation_forward",
    "yoso_expectation_backward",
    "yoso_timing_enable", "yoso_timing_reset", "yoso_timing_query",
    "workspace", "hash_qk", "fast_hash_qk", "forward", "backward",
]

F32, BF16 = 0, 1
OP_HASH, OP_FORWARD, OP_BACKWARD, OP_BACKWARD_STAR = 0, 1, 2, 3
STATUS = {0: "YOSO_OK", 1: "YOSO_ERR_NULL", 2: "YOSO_ERR_SHAPE", 3: "YOSO_ERR_TAU", 4: "YOSO_ERR_DTYPE",
          5: "YOSO_ERR_ALIGN", 6: "YOSO_ERR_WORKSPACE", 7: "YOSO_ERR_DEVICE", 8: "YOSO_ERR_OP"}

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_PKG, "libyoso.so")
_lib = None


class YosoError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{STATUS.get(status, status)}: {detail}")


def lib_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """The loaded libyoso.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2111_09714_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
        L.yoso_hash.argtypes = [P, I32, I64, I64, I32, P, I32, I32, P, P]
        L.yoso_fast_hyperplanes.argtypes = [P, I32, I32, I32, P, P]
        L.yoso_fast_hash.argtypes = [P, I32, I64, I64, I32, P, I32, I32, P, P]
        L.yoso_forward.argtypes = [P, P, P, I32, I64, I64, I64, I32, I32, I32, P, P, SZ, P]
        L.yoso_backward.argtypes = [P, P, P, P, P, P, I32, I64, I64, I64, I32, I32, I32, P, P, P, P, SZ, P]
        L.yoso_backward_star.argtypes = [P, P, P, P, P, P, I32, I64, I64, I64, I32, I32, I32, P, P, P, P, SZ, P]
        L.yoso_backward_star.restype = ctypes.c_int
        L.yoso_backward_noalloc.argtypes = [P, P, P, P, P, P, I32, I64, I64, I64, I32, I32, I32, P, P, P, P]
        L.yoso_backward_noalloc.restype = ctypes.c_int
        L.yoso_backward_noalloc_limit.argtypes = []
        L.yoso_backward_noalloc_limit.restype = SZ
        L.yoso_backward_table_threshold.argtypes = []
        L.yoso_backward_table_threshold.restype = ctypes.c_int32
        L.yoso_workspace_bytes.argtypes = [I32, I64, I64, I64, I32, I32, I32, I32]
        L.yoso_workspace_bytes.restype = SZ
        L.yoso_l2_normalize.argtypes = [P, I32, I64, I32, P, P]
        L.yoso_expectation_forward.argtypes = [P, P, P, I32, I64, I64, I64, I32, I32, P, P]
        L.yoso_expectation_backward.argtypes = [P, P, P, P, I32, I64, I64, I64, I32, I32, P, P, P, P]
        L.yoso_l2_normalize_backward.argtypes = [P, P, I32, I64, I32, P, P]
        for fn in ("yoso_hash", "yoso_forward", "yoso_backward"):
            getattr(L, fn).restype = ctypes.c_int
        L.yoso_status_str.argtypes = [ctypes.c_int]
        L.yoso_status_str.restype = ctypes.c_char_p
        L.yoso_last_error.argtypes = []
        L.yoso_last_error.restype = ctypes.c_char_p
        L.yoso_timing_enable.argtypes = [I32]
        L.yoso_timing_reset.argtypes = []
        L.yoso_timing_query.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64)]
        for fn in ("yoso_timing_enable", "yoso_timing_reset", "yoso_timing_query"):
            getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise YosoError(status, lib().yoso_last_error().decode())


# ------------------------------------------------------------------ tensor marshalling

def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr() if t.numel() > 0 else None


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _codes_ok(c) -> None:
    import torch
    if c.dtype not in (torch.int16, torch.uint16):
        raise TypeError("codes must be int16 or uint16 tensors (16-bit storage)")


def _same(ref, named) -> None:
    """Every tensor in `named` ((tensor, name) pairs) must have the storage type of
    `ref` and live on its device: the kernels read and write every buffer with the
    element size of the one dtype code passed to the C ABI."""
    for t, name in named:
        if t is None:
            continue
        if t.dtype != ref.dtype:
            raise TypeError(f"{name} is {t.dtype}, expected {ref.dtype} like the other data tensors")
        if t.device != ref.device:
            raise ValueError(f"{name} is on {t.device}, expected {ref.device}")


def _on(ref, named) -> None:
    """Tensors of other types (codes, R, signs, workspace) must share ref's device."""
    for t, name in named:
        if t is not None and t.device != ref.device:
            raise ValueError(f"{name} is on {t.device}, expected {ref.device}")


def _f32(t, name: str) -> None:
    import torch
    if t.dtype != torch.float32:
        raise TypeError(f"{name} must be float32")


def _expect(t, shape, name: str) -> None:
    """The C ABI cannot see buffer sizes, so shapes are checked here before any launch."""
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def yoso_workspace_bytes(op: int, bh: int, n_q: int, n_k: int, d: int, m: int, tau: int, dtype: int) -> int:
    out = lib().yoso_workspace_bytes(op, bh, n_q, n_k, d, m, tau, dtype)
    if out == ctypes.c_size_t(-1).value:
        raise YosoError(-1, lib().yoso_last_error().decode())
    return out


def yoso_status_str(status: int) -> str:
    return lib().yoso_status_str(status).decode()


def yoso_hash(x, R, m: int, tau: int, codes, stream=None) -> None:
    """codes[b, i, h] = sum_t [x[b, i] . R[:, h*tau + t] > 0] << t."""
    _codes_ok(codes)
    _f32(R, "R")
    _on(x, ((R, "R"), (codes, "codes")))
    bh, n, d = x.shape
    _expect(R, (d, m * tau), "R")
    _expect(codes, (bh, n, m), "codes")
    _check(lib().yoso_hash(_ptr(x), _dtype_code(x), bh, n, d, _ptr(R), m, tau, _ptr(codes), _stream(stream)))


def yoso_fast_hyperplanes(signs, m: int, tau: int, R, stream=None) -> None:
    """R[:, 64 r + l] = row l of (1/64) H D3 H D2 H D1 of rotation r (the fast hash's
    hyperplanes); signs[r, i] (64-bit, int64 or uint64 storage) holds D_{i+1}'s negations."""
    import torch
    if signs.dtype not in (torch.int64, torch.uint64):
        raise TypeError("signs must be an int64 or uint64 tensor (64-bit masks)")
    _f32(R, "R")
    _on(R, ((signs, "signs"),))
    _expect(signs, ((m * tau + 63) // 64, 3), "signs")
    _expect(R, (64, m * tau), "R")
    _check(lib().yoso_fast_hyperplanes(_ptr(signs), 64, m, tau, _ptr(R), _stream(stream)))


def yoso_fast_hash(x, signs, m: int, tau: int, codes, stream=None) -> None:
    """codes[b, i, h]: the signs of the rows of x under the rotations H D3 H D2 H D1 of ``signs``."""
    import torch
    _codes_ok(codes)
    if signs.dtype not in (torch.int64, torch.uint64):
        raise TypeError("signs must be an int64 or uint64 tensor (64-bit masks)")
    _on(x, ((signs, "signs"), (codes, "codes")))
    bh, n, d = x.shape
    _expect(signs, ((m * tau + 63) // 64, 3), "signs")
    _expect(codes, (bh, n, m), "codes")
    _check(lib().yoso_fast_hash(_ptr(x), _dtype_code(x), bh, n, d, _ptr(signs), m, tau, _ptr(codes),
                                _stream(stream)))


def yoso_forward(qcodes, kcodes, v, m: int, tau: int, y, ws=None, stream=None) -> None:
    """y = (1/m) sum_h B_h v with B_h(i, j) = [qcodes[:, i, h] == kcodes[:, j, h]]."""
    _codes_ok(qcodes)
    _codes_ok(kcodes)
    _same(v, ((y, "y"),))
    _on(v, ((qcodes, "qcodes"), (kcodes, "kcodes"), (ws, "ws")))
    bh, n_k, d = v.shape
    n_q = y.shape[1]
    _expect(y, (bh, n_q, d), "y")
    _expect(qcodes, (bh, n_q, m), "qcodes")
    _expect(kcodes, (bh, n_k, m), "kcodes")
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().yoso_forward(_ptr(qcodes), _ptr(kcodes), _ptr(v), _dtype_code(v), bh, n_q, n_k, d, m, tau,
                              _ptr(y), _ptr(ws), nbytes, _stream(stream)))


def yoso_backward(qcodes, kcodes, q, k, v, dy, m: int, tau: int, dq, dk, dv, ws, stream=None) -> None:
    """dv = (1/m) sum_h B_h^T dy;  dq, dk = tau/(2m) sum_h [(dy v^T) .* B_h] k, ...^T q."""
    _codes_ok(qcodes)
    _codes_ok(kcodes)
    _same(q, ((k, "k"), (v, "v"), (dy, "dy"), (dq, "dq"), (dk, "dk"), (dv, "dv")))
    _on(q, ((qcodes, "qcodes"), (kcodes, "kcodes"), (ws, "ws")))
    bh, n_q, d = q.shape
    n_k = k.shape[1]
    for t, shape, name in ((k, (bh, n_k, d), "k"), (v, (bh, n_k, d), "v"), (dy, (bh, n_q, d), "dy"),
                           (dq, (bh, n_q, d), "dq"), (dk, (bh, n_k, d), "dk"), (dv, (bh, n_k, d), "dv"),
                           (qcodes, (bh, n_q, m), "qcodes"), (kcodes, (bh, n_k, m), "kcodes")):
        _expect(t, shape, name)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().yoso_backward(_ptr(qcodes), _ptr(kcodes), _ptr(q), _ptr(k), _ptr(v), _ptr(dy), _dtype_code(q),
                               bh, n_q, n_k, d, m, tau, _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws), nbytes,
                               _stream(stream)))


def yoso_backward_star(qcodes, kcodes, q, k, v, dy, m: int, tau: int, dq, dk, dv, ws, stream=None) -> None:
    """*YOSO: dq, dk estimate the true gradient of eq. (gradient-q) (pairs whose codes
    agree on all bits but at most one, weighted 1/(pi sqrt(max(1 - (q.k)^2, 1/64))));
    dv as yoso_backward."""
    _codes_ok(qcodes)
    _codes_ok(kcodes)
    _same(q, ((k, "k"), (v, "v"), (dy, "dy"), (dq, "dq"), (dk, "dk"), (dv, "dv")))
    _on(q, ((qcodes, "qcodes"), (kcodes, "kcodes"), (ws, "ws")))
    bh, n_q, d = q.shape
    n_k = k.shape[1]
    for t, shape, name in ((k, (bh, n_k, d), "k"), (v, (bh, n_k, d), "v"), (dy, (bh, n_q, d), "dy"),
                           (dq, (bh, n_q, d), "dq"), (dk, (bh, n_k, d), "dk"), (dv, (bh, n_k, d), "dv"),
                           (qcodes, (bh, n_q, m), "qcodes"), (kcodes, (bh, n_k, m), "kcodes")):
        _expect(t, shape, name)
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().yoso_backward_star(_ptr(qcodes), _ptr(kcodes), _ptr(q), _ptr(k), _ptr(v), _ptr(dy),
                                    _dtype_code(q), bh, n_q, n_k, d, m, tau, _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws),
                                    nbytes, _stream(stream)))


def yoso_backward_noalloc(qcodes, kcodes, q, k, v, dy, m: int, tau: int, dq, dk, dv, stream=None) -> None:
    """yoso_backward on the library's fixed per-GPU scratch (no workspace, no
    allocation); shapes needing more than yoso_backward_noalloc_limit() bytes are
    refused.  Calls that overlap on one GPU race."""
    _codes_ok(qcodes)
    _codes_ok(kcodes)
    _same(q, ((k, "k"), (v, "v"), (dy, "dy"), (dq, "dq"), (dk, "dk"), (dv, "dv")))
    _on(q, ((qcodes, "qcodes"), (kcodes, "kcodes")))
    bh, n_q, d = q.shape
    n_k = k.shape[1]
    for t, shape, name in ((k, (bh, n_k, d), "k"), (v, (bh, n_k, d), "v"), (dy, (bh, n_q, d), "dy"),
                           (dq, (bh, n_q, d), "dq"), (dk, (bh, n_k, d), "dk"), (dv, (bh, n_k, d), "dv"),
                           (qcodes, (bh, n_q, m), "qcodes"), (kcodes, (bh, n_k, m), "kcodes")):
        _expect(t, shape, name)
    _check(lib().yoso_backward_noalloc(_ptr(qcodes), _ptr(kcodes), _ptr(q), _ptr(k), _ptr(v), _ptr(dy),
                                       _dtype_code(q), bh, n_q, n_k, d, m, tau, _ptr(dq), _ptr(dk), _ptr(dv),
                                       _stream(stream)))


def yoso_backward_noalloc_limit() -> int:
    return lib().yoso_backward_noalloc_limit()


def yoso_backward_table_threshold() -> int:
    """T of the backward's rule: a bucket takes the table form when b_q b_k > T (b_q + b_k)."""
    return lib().yoso_backward_table_threshold()


def yoso_l2_normalize(x, y, stream=None) -> None:
    """y = x / ||x|| row by row over the last dimension (zero rows stay zero)."""
    d = x.shape[-1]
    _expect(y, x.shape, "y")
    _same(x, ((y, "y"),))
    rows = x.numel() // d if d else 0
    _check(lib().yoso_l2_normalize(_ptr(x), _dtype_code(x), rows, d, _ptr(y), _stream(stream)))


def yoso_l2_normalize_backward(x, dy, dx, stream=None) -> None:
    """dx = (dy - y (y . dy)) / ||x||, y = x / ||x||, row by row (x is the forward's input)."""
    d = x.shape[-1]
    _expect(dy, x.shape, "dy")
    _expect(dx, x.shape, "dx")
    _same(x, ((dy, "dy"), (dx, "dx")))
    rows = x.numel() // d if d else 0
    _check(lib().yoso_l2_normalize_backward(_ptr(x), _ptr(dy), _dtype_code(x), rows, d, _ptr(dx), _stream(stream)))


def yoso_expectation_forward(q, k, v, tau: int, y, stream=None) -> None:
    """YOSO-E: y = P v with P_ij = (1 - arccos(cos(q_i, k_j))/pi)^tau."""
    bh, n_q, d = q.shape
    n_k = k.shape[1]
    _same(q, ((k, "k"), (v, "v"), (y, "y")))
    for t, shape, name in ((k, (bh, n_k, d), "k"), (v, (bh, n_k, d), "v"), (y, (bh, n_q, d), "y")):
        _expect(t, shape, name)
    _check(lib().yoso_expectation_forward(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), bh, n_q, n_k, d, tau, _ptr(y),
                                          _stream(stream)))


def yoso_expectation_backward(q, k, v, dy, tau: int, dq, dk, dv, stream=None) -> None:
    """YOSO-E backward: dv = P^T dy, dq = (tau/2)[(dy v^T) .* P] k, dk = (tau/2)[(dy v^T) .* P]^T q."""
    bh, n_q, d = q.shape
    n_k = k.shape[1]
    _same(q, ((k, "k"), (v, "v"), (dy, "dy"), (dq, "dq"), (dk, "dk"), (dv, "dv")))
    for t, shape, name in ((k, (bh, n_k, d), "k"), (v, (bh, n_k, d), "v"), (dy, (bh, n_q, d), "dy"),
                           (dq, (bh, n_q, d), "dq"), (dk, (bh, n_k, d), "dk"), (dv, (bh, n_k, d), "dv")):
        _expect(t, shape, name)
    _check(lib().yoso_expectation_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(dy), _dtype_code(q), bh, n_q, n_k, d, tau,
                                           _ptr(dq), _ptr(dk), _ptr(dv), _stream(stream)))


def yoso_timing_enable(capacity: int) -> None:
    _check(lib().yoso_timing_enable(capacity))


def yoso_timing_reset() -> None:
    _check(lib().yoso_timing_reset())


def yoso_timing_query(kernel: str):
    """(total_ms, launches) recorded for `kernel` since the last reset (synchronises)."""
    ms, n = ctypes.c_double(0.0), ctypes.c_int64(0)
    _check(lib().yoso_timing_query(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ------------------------------------------------------------------ allocating conveniences

def workspace(op: int, x, m: int, tau: int, n_k: Optional[int] = None):
    """A uint8 device tensor large enough for `op` on tensors shaped like x ([bh, n_q, 64])."""
    import torch
    bh, n_q, d = x.shape
    n_k = n_q if n_k is None else n_k
    nbytes = yoso_workspace_bytes(op, bh, n_q, n_k, d, m, tau, _dtype_code(x))
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=x.device)


def hash_qk(q, k, R, m: int, tau: int):
    """Codes of Q and K under the same hyperplanes (fresh int16 tensors)."""
    import torch
    qc = torch.empty((q.shape[0], q.shape[1], m), dtype=torch.int16, device=q.device)
    kc = torch.empty((k.shape[0], k.shape[1], m), dtype=torch.int16, device=k.device)
    yoso_hash(q, R, m, tau, qc)
    yoso_hash(k, R, m, tau, kc)
    return qc, kc


def fast_hash_qk(q, k, signs, m: int, tau: int):
    """Codes of Q and K under the fast hash of the rotations in ``signs`` (fresh int16 tensors)."""
    import torch
    qc = torch.empty((q.shape[0], q.shape[1], m), dtype=torch.int16, device=q.device)
    kc = torch.empty((k.shape[0], k.shape[1], m), dtype=torch.int16, device=k.device)
    yoso_fast_hash(q, signs, m, tau, qc)
    yoso_fast_hash(k, signs, m, tau, kc)
    return qc, kc


def forward(qcodes, kcodes, v, m: int, tau: int, n_q: Optional[int] = None):
    import torch
    n_q = qcodes.shape[1] if n_q is None else n_q
    y = torch.empty((v.shape[0], n_q, v.shape[2]), dtype=v.dtype, device=v.device)
    ws = workspace(OP_FORWARD, y, m, tau, n_k=v.shape[1])
    yoso_forward(qcodes, kcodes, v, m, tau, y, ws)
    return y


def backward(qcodes, kcodes, q, k, v, dy, m: int, tau: int):
    import torch
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = workspace(OP_BACKWARD, q, m, tau, n_k=k.shape[1])
    yoso_backward(qcodes, kcodes, q, k, v, dy, m, tau, dq, dk, dv, ws)
    return dq, dk, dv


def backward_star(qcodes, kcodes, q, k, v, dy, m: int, tau: int):
    import torch
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = workspace(OP_BACKWARD_STAR, q, m, tau, n_k=k.shape[1])
    yoso_backward_star(qcodes, kcodes, q, k, v, dy, m, tau, dq, dk, dv, ws)
    return dq, dk, dv
