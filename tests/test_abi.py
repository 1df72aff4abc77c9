"""Host-side checks of the C ABI: the library loads, exports what include/yoso.h
declares, and rejects every bad argument before touching the device.

No call here reaches a kernel: each one carries at least one invalid argument, and
the library validates everything on the host before its first HIP call.  The
device pointers are fake (never dereferenced)."""
import ctypes
import os
import re

import pytest

import paper_2111_09714_amd as Y
from paper_2111_09714_amd import build as ybuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # 16-byte aligned, never dereferenced


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(Y.lib_path()):
        ybuild.build()
    return Y.lib()


def _declared_symbols():
    text = open(os.path.join(ROOT, "include", "yoso.h")).read()
    return sorted(set(re.findall(r"\b(yoso_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = _declared_symbols()
    assert {"yoso_hash", "yoso_forward", "yoso_backward", "yoso_workspace_bytes",
            "yoso_status_str", "yoso_last_error"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    for s in range(9):
        assert L.yoso_status_str(s)
    assert L.yoso_status_str(0) == b"ok"
    assert Y.yoso_status_str(3) == "tau or m out of range"


def _hash(L, x=FAKE, dtype=0, bh=2, n=128, d=64, R=FAKE, m=32, tau=8, codes=FAKE):
    return L.yoso_hash(x, dtype, bh, n, d, R, m, tau, codes, None)


def _fwd(L, qc=FAKE, kc=FAKE, v=FAKE, dtype=0, bh=2, nq=128, nk=128, d=64, m=32, tau=8, y=FAKE,
         ws=FAKE, wsb=1 << 30):
    return L.yoso_forward(qc, kc, v, dtype, bh, nq, nk, d, m, tau, y, ws, wsb, None)


def _bwd(L, dtype=0, bh=2, nq=128, nk=128, d=64, m=32, tau=8, ws=FAKE, wsb=1 << 30, **ptrs):
    p = dict(qc=FAKE, kc=FAKE, q=FAKE, k=FAKE, v=FAKE, dy=FAKE, dq=FAKE, dk=FAKE, dv=FAKE)
    p.update(ptrs)
    return L.yoso_backward(p["qc"], p["kc"], p["q"], p["k"], p["v"], p["dy"], dtype, bh, nq, nk, d, m, tau,
                           p["dq"], p["dk"], p["dv"], ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 4),
    (dict(d=32), 2),
    (dict(bh=-1), 2),
    (dict(n=65537), 2),
    (dict(n=-3), 2),
    (dict(tau=0), 3),
    (dict(tau=13), 3),
    (dict(m=0), 3),
    (dict(m=65), 3),
    (dict(m=64, tau=9), 3),   # m*tau = 576 > 512
    (dict(x=None), 1),
    (dict(R=None), 1),
    (dict(codes=None), 1),
    (dict(x=FAKE + 4), 5),
    (dict(codes=FAKE + 2), 5),
])
def test_hash_rejects(L, kw, status):
    assert _hash(L, **kw) == status
    assert L.yoso_last_error()


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=2), 4),
    (dict(d=128), 2),
    (dict(nq=70000), 2),
    (dict(nk=-1), 2),
    (dict(tau=20), 3),
    (dict(qc=None), 1),
    (dict(kc=None), 1),
    (dict(v=None), 1),
    (dict(y=None), 1),
    (dict(v=FAKE + 8), 5),
])
def test_forward_rejects(L, kw, status):
    assert _fwd(L, **kw) == status


def test_forward_workspace_checks(L):
    # past the dense form's 1024 rows, tau = 12 needs several hash groups of tables,
    # and bf16 output needs an fp32 accumulator
    need = Y.yoso_workspace_bytes(Y.OP_FORWARD, 2, 2048, 2048, 64, 32, 12, Y.BF16)
    assert need > 0
    big = dict(dtype=1, tau=12, nq=2048, nk=2048)
    assert _fwd(L, ws=None, wsb=0, **big) == 6
    assert _fwd(L, ws=FAKE, wsb=need - 1, **big) == 6
    assert _fwd(L, ws=FAKE + 4, wsb=need, **big) == 5


def test_dense_forward_needs_no_workspace(L):
    # many heads of short sequences: the forward counts collisions pair by pair and
    # needs no workspace; over few heads it takes the tables, and bf16 output with
    # several groups of tau = 12 tables needs an fp32 accumulator
    for n_q, n_k in ((1, 1), (100, 1024), (512, 512), (1024, 1)):
        for tau, m, dt in ((12, 32, Y.BF16), (8, 64, Y.F32), (1, 1, Y.F32)):
            assert Y.yoso_workspace_bytes(Y.OP_FORWARD, 1024, n_q, n_k, 64, m, tau, dt) == 0
    assert Y.yoso_workspace_bytes(Y.OP_FORWARD, 4, 512, 512, 64, 32, 12, Y.BF16) > 0
    assert Y.yoso_workspace_bytes(Y.OP_FORWARD, 1024, 1025, 1024, 64, 32, 12, Y.BF16) > 0


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=-1), 4),
    (dict(d=0), 2),
    (dict(m=100), 3),
    (dict(q=None), 1),
    (dict(dy=None), 1),
    (dict(dk=None), 1),
    (dict(dv=FAKE + 1), 5),
    (dict(ws=None), 6),
    (dict(wsb=16), 6),
])
def test_backward_rejects(L, kw, status):
    assert _bwd(L, **kw) == status


def test_noalloc_refuses_shapes_beyond_its_scratch(L):
    """yoso_backward_noalloc checks the workspace its shapes need against its fixed
    64 MiB scratch before any HIP call."""
    assert L.yoso_backward_noalloc_limit() == 64 << 20
    assert L.yoso_backward_table_threshold() >= 16  # table buckets span more than one 16-row tile
    p = [FAKE] * 6
    # 32 heads of 4096 rows at m = 32 need about 0.9 GB
    st = L.yoso_backward_noalloc(*p, 0, 32, 4096, 4096, 64, 32, 8, FAKE, FAKE, FAKE, None)
    assert st == 6 and b"scratch" in L.yoso_last_error()
    assert L.yoso_backward_noalloc(*p, 0, 1, 128, 128, 32, 32, 8, FAKE, FAKE, FAKE, None) == 2  # d
    assert L.yoso_backward_noalloc(*p, 0, 1, 128, 128, 64, 32, 13, FAKE, FAKE, FAKE, None) == 3  # tau
    assert L.yoso_backward_noalloc(FAKE, None, *p[2:], 0, 1, 128, 128, 64, 32, 8, FAKE, FAKE, FAKE, None) == 1


def _star(L, dtype=0, bh=2, nq=128, nk=128, d=64, m=32, tau=8, ws=FAKE, wsb=1 << 40, **ptrs):
    p = dict(qc=FAKE, kc=FAKE, q=FAKE, k=FAKE, v=FAKE, dy=FAKE, dq=FAKE, dk=FAKE, dv=FAKE)
    p.update(ptrs)
    return L.yoso_backward_star(p["qc"], p["kc"], p["q"], p["k"], p["v"], p["dy"], dtype, bh, nq, nk, d, m, tau,
                                p["dq"], p["dk"], p["dv"], ws, wsb, None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=3), 4),
    (dict(d=16), 2),
    (dict(tau=13), 3),
    (dict(m=64, tau=9), 3),
    (dict(dk=None), 1),
    (dict(q=FAKE + 2), 5),
    (dict(ws=None), 6),
    (dict(wsb=1024), 6),
])
def test_backward_star_rejects(L, kw, status):
    assert _star(L, **kw) == status


def test_backward_star_workspace():
    """*YOSO runs the pair passes over m*tau derived hashes of tau-1 bits: its
    workspace is the backward layout of those, plus the derived codes."""
    bh, nq, nk, m, tau = 2, 512, 300, 32, 8
    star = Y.yoso_workspace_bytes(Y.OP_BACKWARD_STAR, bh, nq, nk, 64, m, tau, Y.F32)
    mh = m * tau                                           # derived hashes
    partials = bh * (nq + nk) * mh * (64 * 3 + 1)          # 24-bit rows + exponents
    index = bh * mh * (2 * (2 ** (tau - 1) + 1) * 4 + (nq + 16 + nk + 16) * 4)
    split = 4 * bh * (nq + nk) // 2 * 64 * 4
    codes = 2 * bh * (nq + nk) * mh * 2                    # the derived codes, then transposed
    need = partials + index + split + codes
    assert need <= star < 1.02 * need + (1 << 16)


def test_empty_tensors_need_no_pointers(L):
    # zero-sized tensors are valid and their pointers may be NULL; with every size 0
    # nothing is launched, so these calls return OK even without a GPU.
    assert _hash(L, bh=0, x=None, codes=None) == 0
    assert _hash(L, n=0, x=None, codes=None) == 0
    assert _fwd(L, bh=0, qc=None, kc=None, v=None, y=None, ws=None, wsb=0) == 0


def test_workspace_sizes():
    # backward workspace: bucket offsets + sorted entries, the codes transposed for the
    # sort, the fp16 (hi, lo) copies of Q, K, V, dY (4 bytes per element) and one
    # partial row per (row, hash) for dq and dk in 24-bit fixed point (64 int16 high
    # parts, 64 low bytes and one exponent byte); bf16 outputs take 16-bit rows
    # (no low bytes)
    f32 = Y.yoso_workspace_bytes(Y.OP_BACKWARD, 32, 4096, 4096, 64, 32, 8, Y.F32)
    bf = Y.yoso_workspace_bytes(Y.OP_BACKWARD, 32, 4096, 4096, 64, 32, 8, Y.BF16)
    units = 32 * 32
    index = units * (2 * 257 * 4 + 2 * 4096 * 4 + 2 * 4096 * 2)
    split = 4 * 32 * 4096 * 64 * 4
    partials = 2 * 32 * 4096 * 32 * (64 * 3 + 1)
    assert f32 >= index + split + partials
    assert f32 < 1.05 * (index + split + partials) + (1 << 20)
    # bf16: no low parts and no exponent arrays (16-bit rows carry their exponents)
    low = 2 * 32 * 4096 * 32 * 64
    exps = 2 * 32 * 4096 * 32
    assert f32 - low - exps - (1 << 12) <= bf <= f32 - low - exps
    assert Y.yoso_workspace_bytes(Y.OP_HASH, 32, 4096, 4096, 64, 32, 8, Y.F32) == 0
    assert Y.yoso_workspace_bytes(Y.OP_FORWARD, 32, 4096, 4096, 64, 32, 8, Y.F32) == 0
    with pytest.raises(Y.YosoError):
        Y.yoso_workspace_bytes(9, 1, 1, 1, 64, 1, 1, Y.F32)


def test_workspace_bytes_rejects_bad_arguments(L):
    bad = ctypes.c_size_t(-1).value
    # op, bh, n_q, n_k, d, m, tau, dtype
    for args in ((9, 1, 1, 1, 64, 1, 1, 0), (2, 1, 1, 1, 32, 1, 1, 0), (2, 1, 1, 1, 64, 1, 13, 0),
                 (2, 1, 1, 1, 64, 65, 1, 0), (2, -1, 1, 1, 64, 1, 1, 0), (2, 1, 70000, 1, 64, 1, 1, 0),
                 (2, 1, 1, 1, 64, 1, 1, 5)):
        assert L.yoso_workspace_bytes(*args) == bad, args
        assert L.yoso_last_error()


def test_binding_refuses_mixed_dtypes_and_devices():
    """The C ABI takes one dtype code for all data tensors: a tensor of another type
    (or R that is not fp32) would be read or written with the wrong element size, so
    the binding refuses it before any call."""
    torch = pytest.importorskip("torch")
    f, b = torch.float32, torch.bfloat16
    x = torch.zeros(1, 16, 64)
    codes = torch.zeros(1, 16, 2, dtype=torch.int16)
    with pytest.raises(TypeError):
        Y.yoso_hash(x, torch.zeros(64, 16, dtype=b), 2, 8, codes)
    with pytest.raises(TypeError):
        Y.yoso_forward(codes, codes, torch.zeros(1, 16, 64, dtype=f), 2, 8, torch.zeros(1, 16, 64, dtype=b))
    q = torch.zeros(1, 16, 64, dtype=f)
    for bad in range(6):
        ts = [torch.zeros(1, 16, 64, dtype=f) for _ in range(6)]
        ts[bad] = ts[bad].to(b)
        k, v, dy, dq, dk, dv = ts
        with pytest.raises(TypeError):
            Y.yoso_backward(codes, codes, q, k, v, dy, 2, 8, dq, dk, dv, None)
    with pytest.raises(TypeError):
        Y.yoso_l2_normalize(q, torch.zeros(1, 16, 64, dtype=b))
    with pytest.raises(TypeError):
        Y.yoso_l2_normalize_backward(q, q, torch.zeros(1, 16, 64, dtype=b))
    with pytest.raises(TypeError):
        Y.yoso_expectation_forward(q, q, q, 8, torch.zeros(1, 16, 64, dtype=b))
    with pytest.raises(TypeError):
        Y.yoso_expectation_backward(q, q.to(b), q, q, 8, q, q, q)
    with pytest.raises(TypeError):
        Y.yoso_fast_hyperplanes(torch.zeros(1, 3, dtype=torch.int64), 8, 8, torch.zeros(64, 64, dtype=b))


def test_binding_refuses_host_tensors():
    torch = pytest.importorskip("torch")
    x = torch.zeros(1, 16, 64)
    with pytest.raises(ValueError):
        Y.yoso_hash(x, torch.zeros(64, 16), 2, 8, torch.zeros(1, 16, 2, dtype=torch.int16))


def _l2(L, x=FAKE, dtype=0, rows=100, d=64, y=FAKE):
    return L.yoso_l2_normalize(x, dtype, rows, d, y, None)


def _l2b(L, x=FAKE, dy=FAKE, dtype=0, rows=100, d=64, dx=FAKE):
    return L.yoso_l2_normalize_backward(x, dy, dtype, rows, d, dx, None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=2), 4),
    (dict(d=63), 2),
    (dict(rows=-1), 2),
    (dict(x=None), 1),
    (dict(y=None), 1),
    (dict(x=FAKE + 8), 5),
    (dict(y=FAKE + 4), 5),
])
def test_l2_normalize_rejects(L, kw, status):
    assert _l2(L, **kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=-1), 4),
    (dict(d=128), 2),
    (dict(rows=-5), 2),
    (dict(dy=None), 1),
    (dict(dx=None), 1),
    (dict(dy=FAKE + 2), 5),
])
def test_l2_normalize_backward_rejects(L, kw, status):
    assert _l2b(L, **kw) == status


def test_l2_empty_is_a_no_op(L):
    # zero rows: valid with NULL pointers, nothing launched
    assert L.yoso_l2_normalize(None, 0, 0, 64, None, None) == 0
    assert L.yoso_l2_normalize_backward(None, None, 1, 0, 64, None, None) == 0


def _efwd(L, q=FAKE, k=FAKE, v=FAKE, dtype=0, bh=2, nq=64, nk=64, d=64, tau=8, y=FAKE):
    return L.yoso_expectation_forward(q, k, v, dtype, bh, nq, nk, d, tau, y, None)


def _ebwd(L, dtype=0, bh=2, nq=64, nk=64, d=64, tau=8, **ptrs):
    p = dict(q=FAKE, k=FAKE, v=FAKE, dy=FAKE, dq=FAKE, dk=FAKE, dv=FAKE)
    p.update(ptrs)
    return L.yoso_expectation_backward(p["q"], p["k"], p["v"], p["dy"], dtype, bh, nq, nk, d, tau,
                                       p["dq"], p["dk"], p["dv"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=3), 4),
    (dict(d=16), 2),
    (dict(bh=-2), 2),
    (dict(nq=70000), 2),
    (dict(tau=0), 3),
    (dict(tau=13), 3),
    (dict(q=None), 1),
    (dict(y=None), 1),
    (dict(v=FAKE + 4), 5),
])
def test_expectation_forward_rejects(L, kw, status):
    assert _efwd(L, **kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=9), 4),
    (dict(nk=-1), 2),
    (dict(tau=20), 3),
    (dict(dy=None), 1),
    (dict(dk=None), 1),
    (dict(dq=FAKE + 12), 5),
])
def test_expectation_backward_rejects(L, kw, status):
    assert _ebwd(L, **kw) == status


def _fhp(L, signs=FAKE, d=64, m=32, tau=8, R=FAKE):
    return L.yoso_fast_hyperplanes(signs, d, m, tau, R, None)


@pytest.mark.parametrize("kw,status", [
    (dict(d=32), 2),
    (dict(tau=0), 3),
    (dict(tau=13), 3),
    (dict(m=0), 3),
    (dict(m=65), 3),
    (dict(m=64, tau=9), 3),      # m*tau = 576 > 512
    (dict(signs=None), 1),
    (dict(R=None), 1),
    (dict(signs=FAKE + 8), 5),
    (dict(R=FAKE + 4), 5),
])
def test_fast_hyperplanes_rejects(L, kw, status):
    assert _fhp(L, **kw) == status


def _fh(L, x=FAKE, dtype=0, bh=2, n=128, d=64, signs=FAKE, m=32, tau=8, codes=FAKE):
    return L.yoso_fast_hash(x, dtype, bh, n, d, signs, m, tau, codes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=2), 4),
    (dict(d=32), 2),
    (dict(bh=-1), 2),
    (dict(n=70000), 2),
    (dict(tau=13), 3),
    (dict(m=65), 3),
    (dict(x=None), 1),
    (dict(signs=None), 1),
    (dict(codes=None), 1),
    (dict(signs=FAKE + 8), 5),
    (dict(codes=FAKE + 2), 5),
])
def test_fast_hash_rejects(L, kw, status):
    assert _fh(L, **kw) == status


def test_fast_hash_empty_is_a_no_op(L):
    # zero rows: x and codes may be NULL (signs, like R for yoso_hash, is still required)
    assert L.yoso_fast_hash(None, 0, 0, 128, 64, FAKE, 32, 8, None, None) == 0
