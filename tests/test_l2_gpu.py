"""Parity of the l2 normalisation calls (N-YOSO's output normalisation and the Q/K
normalisation before hashing) with the fp64 oracle, alone and composed with the
hash / forward / backward calls into the normalised attention and its gradients.

Bars: per tensor (or per head) ||gpu - ref||_F / ||ref||_F and, element by element,
|gpu - ref| / (|ref| + rms(ref row)) (tests/parity.py), both <= 1e-5 for the fp32
row operations alone, 1e-4 for the fp32 composition, 2e-2 with bf16 storage; zero
rows must come out exactly zero.
"""

import numpy as np
import pytest

import oracle
import workloads
from parity import check_all, log
from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2111_09714_amd as Y  # noqa: E402

TOL_ROW = {"f32": 1e-5, "bf16": 2e-2}
TOL = {"f32": 1e-4, "bf16": 2e-2}
MARGIN = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    Y.lib()


def to_dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    return t.to(device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def row_inputs(rows, seed):
    g = np.random.default_rng(seed)
    x = g.standard_normal((rows, 64)) * np.exp(g.uniform(-4, 4, size=(rows, 1)))
    x[:: max(1, rows // 5)] = 0.0  # some zero rows
    dy = g.standard_normal((rows, 64))
    return x, dy


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rows", [1, 3, 1000, 4097])
def test_l2_rows(rows, dtype):
    x, dy = row_inputs(rows, 100 + rows)
    xd, dyd = to_dev(x, dtype), to_dev(dy, dtype)
    y = torch.empty_like(xd)
    dx = torch.empty_like(xd)
    Y.yoso_l2_normalize(xd, y)
    Y.yoso_l2_normalize_backward(xd, dyd, dx)
    torch.cuda.synchronize()
    # the oracle sees exactly the values the GPU read (bf16-rounded for bf16 storage)
    xs, dys = host(xd), host(dyd)
    y_ref = oracle.l2_normalize(xs)
    dx_ref = oracle.l2_normalize_backward(xs, dys)
    check_all(f"l2 rows={rows} {dtype}", [("y", host(y)[None], y_ref[None]), ("dx", host(dx)[None], dx_ref[None])],
              TOL_ROW[dtype])
    zero = np.all(xs == 0, axis=1)
    assert not host(y)[zero].any() and not host(dx)[zero].any()
    # in place: y may be x
    xi = xd.clone()
    Y.yoso_l2_normalize(xi, xi)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(xi), host(y))


def test_l2_empty_and_shape_checks():
    x = torch.empty((0, 64), device="cuda")
    Y.yoso_l2_normalize(x, torch.empty_like(x))
    Y.yoso_l2_normalize_backward(x, torch.empty_like(x), torch.empty_like(x))
    bad = torch.randn(4, 32, device="cuda")
    with pytest.raises(Y.YosoError):
        Y.yoso_l2_normalize(bad, torch.empty_like(bad))


def test_l2_full_size_rows():
    """The Q rows of the long-sequence workload (32 x 4096 rows), all compared."""
    w = WORKLOADS["lra_n4096"]
    inp = make_inputs(w)
    x = inp["q"] * np.random.default_rng(5).uniform(0.5, 2.0, size=(w.bh, w.n, 1))
    xd = to_dev(x, "f32")
    dyd = to_dev(inp["dy"], "f32")
    y, dx = torch.empty_like(xd), torch.empty_like(xd)
    Y.yoso_l2_normalize(xd, y)
    Y.yoso_l2_normalize_backward(xd, dyd, dx)
    torch.cuda.synchronize()
    xs = host(xd)
    check_all("l2 lra rows", [("y", host(y), oracle.l2_normalize(xs)),
                              ("dx", host(dx), oracle.l2_normalize_backward(xs, host(dyd)))], TOL_ROW["f32"])


def codes_np(t):
    return np.ascontiguousarray(t.cpu().numpy().view(np.uint16).transpose(0, 2, 1))


@pytest.mark.parametrize("bh,n,m,tau,dtype", [(2, 300, 16, 6, "f32"), (1, 1000, 32, 8, "f32"),
                                              (2, 257, 8, 5, "bf16")])
def test_normalised_attention_composite(bh, n, m, tau, dtype):
    """N-YOSO with l2-normalised queries and keys, forward and backward:
         qh = l2(q), kh = l2(k); z = YOSO(qh, kh, v); y = l2(z)
         dz = l2'(z) dy; (dqh, dkh, dv) = YOSO backward(qh, kh, v, dz)
         dq = l2'(q) dqh, dk = l2'(k) dkh
    The oracle evaluates the same chain on the GPU's codes after checking them
    bit for bit wherever the oracle's projection margin exceeds 1e-4."""
    g = np.random.default_rng(7 + n + m)
    q = g.standard_normal((bh, n, 64)) * g.uniform(0.2, 5.0, size=(bh, n, 1))
    k = g.standard_normal((bh, n, 64)) * g.uniform(0.2, 5.0, size=(bh, n, 1))
    v = g.standard_normal((bh, n, 64))
    dy = g.standard_normal((bh, n, 64))
    R = g.standard_normal((64, m * tau)).astype(np.float32)
    qd, kd, vd, dyd = (to_dev(a, dtype) for a in (q, k, v, dy))
    Rd = torch.from_numpy(R).cuda()
    qh, kh = torch.empty_like(qd), torch.empty_like(kd)
    Y.yoso_l2_normalize(qd, qh)
    Y.yoso_l2_normalize(kd, kh)
    qc, kc = Y.hash_qk(qh, kh, Rd, m, tau)
    z = Y.forward(qc, kc, vd, m, tau, n_q=n)
    y = torch.empty_like(z)
    Y.yoso_l2_normalize(z, y)
    dz = torch.empty_like(z)
    Y.yoso_l2_normalize_backward(z, dyd, dz)
    dqh, dkh, dv = Y.backward(qc, kc, qh, kh, vd, dz, m, tau)
    dq, dk = torch.empty_like(qd), torch.empty_like(kd)
    Y.yoso_l2_normalize_backward(qd, dqh, dq)
    Y.yoso_l2_normalize_backward(kd, dkh, dk)
    torch.cuda.synchronize()

    qs, ks, vs, dys = host(qd), host(kd), host(vd), host(dyd)
    qho, kho = oracle.l2_normalize(qs), oracle.l2_normalize(ks)
    if dtype == "bf16":
        # the normalised rows are stored (and then hashed) as bf16: round the oracle's
        # the same way (round to nearest even) before it hashes and differentiates
        rnd = lambda a: torch.from_numpy(a).to(torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
        qho, kho = rnd(qho), rnd(kho)
    gq, gk = codes_np(qc), codes_np(kc)
    for x, gc in ((qho, gq), (kho, gk)):
        ref, margin = oracle.hash_codes(x, R.astype(np.float64), m, tau, with_margin=True)
        sure = margin > MARGIN
        assert not ((ref != gc) & sure).any()
    zo = oracle.forward(gq, gk, vs, m, tau)
    yo = oracle.l2_normalize(zo)
    dzo = oracle.l2_normalize_backward(zo, dys)
    dqho, dkho, dvo = oracle.backward(gq, gk, qho, kho, vs, dzo, m, tau)
    dqo = oracle.l2_normalize_backward(qs, dqho)
    dko = oracle.l2_normalize_backward(ks, dkho)
    check_all(f"nyoso bh{bh} n{n} m{m} tau{tau} {dtype}",
              [(key, host(gt), ref) for key, gt, ref in (("y", y, yo), ("dq", dq, dqo), ("dk", dk, dko), ("dv", dv, dvo))],
              TOL[dtype])
