"""Parity of the fast hash (Sec. 3.2 "Speed-up": pseudo-random rotations
H D3 H D2 H D1 in place of a Gaussian R) with the fp64 oracle.

Bars: the expanded hyperplanes are exact (every entry is a multiple of 1/64), so R
must match bit for bit; codes must match bit for bit wherever the oracle's
smallest |projection| of the hash exceeds 1e-4; the attention computed on the
fast codes meets the usual 1e-4 relative bar (fp32).
"""
import sys

import numpy as np
import pytest

import oracle
import workloads
from parity import check_all
from workloads import WORKLOADS, make_inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
import paper_2111_09714_amd as Y  # noqa: E402

MARGIN = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    Y.lib()


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def signs_dev(s):
    return torch.from_numpy(np.ascontiguousarray(s, np.uint64).view(np.int64)).cuda()


def to_dev(a, dtype):
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32))
    return t.to(device="cuda", dtype=torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()


def host(t):
    return t.float().cpu().numpy().astype(np.float64)


def codes_np(t):
    return np.ascontiguousarray(t.cpu().numpy().view(np.uint16).transpose(0, 2, 1))


def rand_signs(seed, m, tau):
    nrot = (m * tau + 63) // 64
    return np.random.default_rng(seed).integers(0, 2**64, size=(nrot, 3), dtype=np.uint64)


@pytest.mark.parametrize("m,tau", [(32, 8), (30, 9), (1, 1), (64, 8), (7, 5), (16, 12)])
def test_fast_hyperplanes_exact(m, tau):
    s = rand_signs(m * 100 + tau, m, tau)
    R = torch.full((64, m * tau), float("nan"), device="cuda")
    Y.yoso_fast_hyperplanes(signs_dev(s), m, tau, R)
    torch.cuda.synchronize()
    ref = oracle.fast_hyperplanes(s, 64, m, tau)
    log(f"[fast R m{m} tau{tau}] max |diff| {np.abs(host(R) - ref).max():.1e}")
    np.testing.assert_array_equal(host(R), ref)


def test_fast_hyperplanes_without_signs_are_hadamard():
    """No negations: M = H, so R's first 64 columns are the Hadamard matrix."""
    R = torch.empty((64, 64), device="cuda")
    Y.yoso_fast_hyperplanes(torch.zeros((1, 3), dtype=torch.int64, device="cuda"), 8, 8, R)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(R), oracle.hadamard(64))


def check_codes(x, signs, m, tau, got):
    ref, margin = oracle.fast_hash_codes(x, signs, m, tau, with_margin=True)
    sure = margin > MARGIN
    bad = int(((ref != got) & sure).sum())
    unsure = float((~sure).mean())
    return bad, unsure


@pytest.mark.parametrize("bh,n,m,tau,dtype", [(2, 300, 32, 8, "f32"), (1, 1000, 30, 9, "f32"),
                                              (3, 129, 16, 6, "bf16"), (1, 1, 1, 1, "f32"),
                                              (2, 65, 64, 8, "f32"), (1, 77, 7, 5, "f32"),
                                              (2, 300, 32, 9, "bf16"), (1, 200, 20, 2, "f32"),
                                              (1, 257, 33, 4, "bf16"), (1, 130, 64, 1, "f32")])
def test_fast_hash_codes(bh, n, m, tau, dtype):
    g = np.random.default_rng(7 * n + m + tau)
    q = g.standard_normal((bh, n, 64))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k = g.standard_normal((bh, n + 3, 64))            # a different length for K
    s = rand_signs(n + tau, m, tau)
    qd, kd = to_dev(q, dtype), to_dev(k, dtype)
    qc, kc = Y.fast_hash_qk(qd, kd, signs_dev(s), m, tau)
    torch.cuda.synchronize()
    for name, xd, c in (("q", qd, qc), ("k", kd, kc)):
        bad, unsure = check_codes(host(xd), s, m, tau, codes_np(c))
        log(f"[fast hash {name} bh{bh} n{n} m{m} tau{tau} {dtype}] mismatches {bad}, unchecked {unsure:.2e}")
        assert bad == 0


def test_fast_hash_full_size():
    """All 32 heads of the 4096-token workload hashed on the GPU; the oracle checks
    the first and last head of Q and K (heads are independent)."""
    w = WORKLOADS["lra_n4096"]
    inp = make_inputs(w)
    qd, kd = to_dev(inp["q"], "f32"), to_dev(inp["k"], "f32")
    qc, kc = Y.fast_hash_qk(qd, kd, signs_dev(inp["signs"]), w.m, w.tau)
    torch.cuda.synchronize()
    for name, x, c in (("q", inp["q"], qc), ("k", inp["k"], kc)):
        for h in (0, w.bh - 1):
            bad, unsure = check_codes(x[h:h + 1], inp["signs"], w.m, w.tau, codes_np(c[h:h + 1]))
            log(f"[fast hash lra {name} head {h}] mismatches {bad}, unchecked {unsure:.2e}")
            assert bad == 0


def test_fast_hash_full_size_bf16():
    """The 32768-token bf16 workload (tau = 9: the general, straddling extraction),
    two of its 24 heads, Q and K, all rows checked."""
    w = WORKLOADS["bf16_n32768"]
    inp = make_inputs(w, heads=[0, w.bh - 1])
    sd = signs_dev(inp["signs"])
    for name in ("q", "k"):
        xd = torch.from_numpy(inp[name + "_bits"].view(np.int16)).cuda().view(torch.bfloat16).contiguous()
        c = torch.empty((2, w.n, w.m), dtype=torch.int16, device="cuda")
        Y.yoso_fast_hash(xd, sd, w.m, w.tau, c)
        torch.cuda.synchronize()
        bad, unsure = check_codes(inp[name], inp["signs"], w.m, w.tau, codes_np(c))
        log(f"[fast hash bf16_n32768 {name}] mismatches {bad}, unchecked {unsure:.2e}")
        assert bad == 0


def test_attention_on_fast_codes():
    """Hash with the fast hash, then forward and backward; the oracle recomputes the
    attention and its gradients from the same codes (after checking them)."""
    w = WORKLOADS["single_head_n512"]
    inp = make_inputs(w, n=700)
    q, k, v, dy = (to_dev(inp[s], "f32") for s in ("q", "k", "v", "dy"))
    qc, kc = Y.fast_hash_qk(q, k, signs_dev(inp["signs"]), w.m, w.tau)
    y = Y.forward(qc, kc, v, w.m, w.tau)
    dq, dk, dv = Y.backward(qc, kc, q, k, v, dy, w.m, w.tau)
    torch.cuda.synchronize()
    gq, gk = codes_np(qc), codes_np(kc)
    for x, c in ((inp["q"], gq), (inp["k"], gk)):
        assert check_codes(x, inp["signs"], w.m, w.tau, c)[0] == 0
    yo = oracle.forward(gq, gk, inp["v"], w.m, w.tau)
    dqo, dko, dvo = oracle.backward(gq, gk, inp["q"], inp["k"], inp["v"], inp["dy"], w.m, w.tau)
    check_all("attention on fast codes",
              [(name, host(a), b) for name, a, b in (("y", y, yo), ("dq", dq, dqo), ("dk", dk, dko), ("dv", dv, dvo))],
              1e-4)


def test_fast_hash_matches_dense_hash_of_expanded_rotations():
    """Both GPU routes to the fast hash agree: the per-row Walsh-Hadamard kernel and
    the dense hash kernel on the expanded rotations (except near-zero projections)."""
    w = WORKLOADS["lra_n4096"]
    inp = make_inputs(w, heads=[3, 17])
    q = to_dev(inp["q"], "f32")
    sd = signs_dev(inp["signs"])
    R = torch.empty((64, w.m * w.tau), device="cuda")
    Y.yoso_fast_hyperplanes(sd, w.m, w.tau, R)
    dense = torch.empty((2, w.n, w.m), dtype=torch.int16, device="cuda")
    fast = torch.empty_like(dense)
    Y.yoso_hash(q, R, w.m, w.tau, dense)
    Y.yoso_fast_hash(q, sd, w.m, w.tau, fast)
    torch.cuda.synchronize()
    _, margin = oracle.fast_hash_codes(inp["q"], inp["signs"], w.m, w.tau, with_margin=True)
    differ = codes_np(dense) != codes_np(fast)
    log(f"[fast vs dense route] differing codes {int(differ.sum())}, all near zero: {bool((margin[differ] <= MARGIN).all())}")
    assert (margin[differ] <= MARGIN).all()


def test_fast_hash_empty():
    s = torch.zeros((4, 3), dtype=torch.int64, device="cuda")
    for bh, n in ((0, 5), (2, 0)):
        x = torch.randn(bh, n, 64, device="cuda")
        c = torch.empty((bh, n, 32), dtype=torch.int16, device="cuda")
        Y.yoso_fast_hash(x, s, 32, 8, c)
    torch.cuda.synchronize()
