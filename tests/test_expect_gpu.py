"""Parity of YOSO-E (the exact expectation over hash functions, forward and the
surrogate backward) with the fp64 oracle, plus closed-form special cases.

Bar: per head ||gpu - ref||_F / ||ref||_F and, element by element,
|gpu - ref| / (|ref| + rms(ref row)), both <= 1e-4 for fp32 storage, 2e-2 for bf16
(tests/parity.py).
"""

import numpy as np
import pytest

import oracle
from parity import TOL, check_all, log
from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2111_09714_amd as Y  # noqa: E402

@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    Y.lib()


def to_dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    return t.to(device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def run_gpu(q, k, v, dy, tau):
    y = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    Y.yoso_expectation_forward(q, k, v, tau, y)
    Y.yoso_expectation_backward(q, k, v, dy, tau, dq, dk, dv)
    torch.cuda.synchronize()
    return host(y), host(dq), host(dk), host(dv)


def unit(a):
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


@pytest.mark.parametrize("bh,nq,nk,tau,dtype", [(2, 100, 77, 8, "f32"), (1, 64, 64, 1, "f32"),
                                                (1, 130, 200, 12, "f32"), (2, 65, 129, 4, "bf16"),
                                                (1, 1, 1, 3, "f32"), (3, 257, 63, 9, "f32")])
def test_expectation_small(bh, nq, nk, tau, dtype):
    g = np.random.default_rng(1000 + nq + nk + tau)
    q = unit(g.standard_normal((bh, nq, 64)))
    k = unit(g.standard_normal((bh, nk, 64)))
    v = g.standard_normal((bh, nk, 64))
    dy = g.standard_normal((bh, nq, 64))
    qd, kd, vd, dyd = (to_dev(a, dtype) for a in (q, k, v, dy))
    y, dq, dk, dv = run_gpu(qd, kd, vd, dyd, tau)
    # the oracle sees the values the GPU read (bf16-rounded for bf16 storage)
    ey, edv, edq, edk = oracle.expectation(host(qd), host(kd), host(vd), host(dyd), tau)
    check_all(f"yoso-e bh{bh} nq{nq} nk{nk} tau{tau} {dtype}",
              [("y", y, ey), ("dq", dq, edq), ("dk", dk, edk), ("dv", dv, edv)], TOL[dtype])


@pytest.mark.parametrize("what,scale", [("dy", 1e-6), ("dy", 1e3), ("v", 1e-5), ("rows", None)])
def test_expectation_far_from_unit_scale(what, scale):
    """Gradients and values far from unit size (training gradients are small): the
    per-row and per-tile power-of-two scalings before the fp16 (hi, lo) split keep
    every output at the fp32 bar; "rows" gives every row of dY and V its own scale
    (10^-4 .. 1 and 10^-3 .. 10)."""
    g = np.random.default_rng(4000 + len(what))
    bh, nq, nk, tau = 2, 200, 150, 8
    q = unit(g.standard_normal((bh, nq, 64)))
    k = unit(g.standard_normal((bh, nk, 64)))
    v = g.standard_normal((bh, nk, 64))
    dy = g.standard_normal((bh, nq, 64))
    if what == "rows":
        dy = dy * 10.0 ** g.uniform(-4, 0, size=(bh, nq, 1))
        v = v * 10.0 ** g.uniform(-3, 1, size=(bh, nk, 1))
    elif what == "dy":
        dy = dy * scale
    else:
        v = v * scale
    qd, kd, vd, dyd = (to_dev(a, "f32") for a in (q, k, v, dy))
    y, dq, dk, dv = run_gpu(qd, kd, vd, dyd, tau)
    ey, edv, edq, edk = oracle.expectation(host(qd), host(kd), host(vd), host(dyd), tau)
    check_all(f"yoso-e scaled {what} {scale}", [("y", y, ey), ("dq", dq, edq), ("dk", dk, edk), ("dv", dv, edv)],
              TOL["f32"])


def test_expectation_closed_forms():
    """P = 1 for identical directions, 2^-tau for orthogonal ones, 0 for opposite ones."""
    tau = 5
    e = np.eye(64)
    q = np.stack([e[0], e[1], -e[2] * 3.0])[None]            # the scale of a row does not matter
    k = np.stack([2.0 * e[0], e[2]])[None]
    v = np.random.default_rng(3).standard_normal((1, 2, 64))
    dy = np.random.default_rng(4).standard_normal((1, 3, 64))
    y, dq, dk, dv = run_gpu(to_dev(q, "f32"), to_dev(k, "f32"), to_dev(v, "f32"), to_dev(dy, "f32"), tau)
    P = np.array([[1.0, 2.0 ** -tau], [2.0 ** -tau, 2.0 ** -tau], [2.0 ** -tau, 0.0]])
    np.testing.assert_allclose(y[0], P @ v[0], rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(dv[0], P.T @ dy[0], rtol=1e-5, atol=1e-6)
    G = dy[0] @ v[0].T
    np.testing.assert_allclose(dq[0], (tau / 2) * (G * P) @ k[0], rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(dk[0], (tau / 2) * (G * P).T @ q[0], rtol=1e-5, atol=1e-5)


def test_expectation_empty():
    for bh, nq, nk in [(0, 4, 4), (1, 0, 5), (1, 5, 0)]:
        q = torch.randn(bh, nq, 64, device="cuda")
        k = torch.randn(bh, nk, 64, device="cuda")
        v = torch.randn(bh, nk, 64, device="cuda")
        dy = torch.randn(bh, nq, 64, device="cuda")
        y, dq, dk, dv = run_gpu(q, k, v, dy, 4)
        for t in (y, dq, dk, dv):
            assert t.size == 0 or not t.any()


def test_expectation_full_size_head():
    """The long-sequence workload (32 heads of n = 4096) on the GPU; the oracle
    recomputes one head (heads are independent)."""
    w = WORKLOADS["lra_n4096"]
    inp = make_inputs(w)
    q, k, v, dy = (to_dev(inp[s], "f32") for s in ("q", "k", "v", "dy"))
    y, dq, dk, dv = run_gpu(q, k, v, dy, w.tau)
    h = w.bh - 1
    sl = slice(h, h + 1)
    ey, edv, edq, edk = oracle.expectation(inp["q"][sl], inp["k"][sl], inp["v"][sl], inp["dy"][sl], w.tau)
    check_all("yoso-e lra head", [("y", y[sl], ey), ("dq", dq[sl], edq), ("dk", dk[sl], edk), ("dv", dv[sl], edv)],
              TOL["f32"])
