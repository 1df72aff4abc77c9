"""Pins of the CPU oracle against facts the paper and the mathematics fix.

None of these re-types the oracle's own formula: each check is a hand-worked
example, a closed form, a special case, an invariant, a brute-force count on tiny
inputs, or a Monte-Carlo law of the hash family.  Together they are chosen so
that a dropped term, a wrong sign, a swapped index or a transposed operand in
any oracle routine fails at least one of them.
"""
import math

import numpy as np
import pytest

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


def _unit(a):
    return a / np.linalg.norm(a, axis=-1, keepdims=True)


def _rand_problem(seed, bh=2, nq=23, nk=19, d=5, m=3, tau=3):
    g = _rng(seed)
    q = _unit(g.standard_normal((bh, nq, d)))
    k = _unit(g.standard_normal((bh, nk, d)))
    v = g.standard_normal((bh, nk, d))
    dy = g.standard_normal((bh, nq, d))
    R = g.standard_normal((d, m * tau))
    return q, k, v, dy, R


def _brute_collisions(qc, kc):
    """B[bh, h, i, j] = [qc_h(i) == kc_h(j)] by direct comparison of every pair."""
    return (qc[:, :, :, None] == kc[:, :, None, :]).astype(np.float64)


# ---------------------------------------------------------------- worked examples

def test_hash_worked_example(golden):
    g = golden["hash"]
    x = np.array(g["x"])[None]
    codes = oracle.hash_codes(x, np.array(g["R"]), g["m"], g["tau"])
    np.testing.assert_array_equal(codes[0], np.array(g["codes"]))


def test_forward_backward_worked_example(golden):
    g = golden["forward_backward"]
    m, tau = g["m"], g["tau"]
    qc = np.array(g["qc"], np.uint16)[None]
    kc = np.array(g["kc"], np.uint16)[None]
    q, k, v, dy = (np.array(g[s])[None] for s in ("q", "k", "v", "dy"))
    np.testing.assert_allclose(oracle.forward(qc, kc, v, m, tau)[0], g["y"], rtol=0, atol=1e-12)
    dq, dk, dv = oracle.backward(qc, kc, q, k, v, dy, m, tau)
    np.testing.assert_allclose(dv[0], g["dv"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dq[0], g["dq"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk[0], g["dk"], rtol=0, atol=1e-12)
    dq2, dk2 = oracle.backward_d2(qc, kc, q, k, v, dy, m, tau)
    np.testing.assert_allclose(dq2[0], g["dq"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk2[0], g["dk"], rtol=0, atol=1e-12)


# ---------------------------------------------------------------- hash special cases

def test_hash_basis_vectors_read_signs_of_R():
    """For x = e_l the projection on column c is R[l, c] itself, so bit b of hash h
    must be [R[l, h*tau+b] > 0] and -e_l must give the complement."""
    d, m, tau = 8, 4, 5
    R = _rng(1).standard_normal((d, m * tau))
    x = np.eye(d)[None]
    codes = oracle.hash_codes(x, R, m, tau)
    neg = oracle.hash_codes(-x, R, m, tau)
    for l in range(d):
        for h in range(m):
            want = sum(1 << b for b in range(tau) if R[l, h * tau + b] > 0)
            assert codes[0, h, l] == want
            assert neg[0, h, l] == (~want) & ((1 << tau) - 1)


def test_hash_scale_invariance_and_margin():
    q, _, _, _, R = _rand_problem(2, bh=1, nq=50, d=16, m=6, tau=7)
    c1, margin = oracle.hash_codes(q, R, 6, 7, with_margin=True)
    c2 = oracle.hash_codes(q * 3.75, R, 6, 7)
    np.testing.assert_array_equal(c1, c2)
    # the margin is the smallest |projection| over the tau hyperplanes of a hash
    proj = q[0] @ R
    want = np.abs(proj).reshape(50, 6, 7).min(axis=2).T
    np.testing.assert_allclose(margin[0], want, rtol=1e-12)


# ---------------------------------------------------------------- hash law

def _angle_pair(theta, d, seed):
    g = _rng(seed)
    a = _unit(g.standard_normal(d))
    b = g.standard_normal(d)
    b = _unit(b - (b @ a) * a)
    return np.stack([a, math.cos(theta) * a + math.sin(theta) * b])


@pytest.mark.parametrize("d", [3, 64])
@pytest.mark.parametrize("tau", [1, 8, 9])
@pytest.mark.parametrize("theta", [0.05, math.pi / 4, math.pi / 2, 2 * math.pi / 3, math.pi - 0.05])
def test_collision_frequency_matches_closed_form(d, tau, theta):
    """Per-code collision probability of tau concatenated hyperplane hashes is
    (1 - theta/pi)^tau (eq. yoso-expectation; tau = 1 is Charikar's 1 - theta/pi)."""
    S = 100_000 if tau > 1 else 20_000
    x = _angle_pair(theta, d, seed=int(theta * 1000) + d + tau)
    R = _rng(10 + d + tau).standard_normal((d, S * tau))
    codes = oracle.hash_codes(x[None], R, S, tau)[0]
    hits = codes[:, 0] == codes[:, 1]
    p = (1 - theta / math.pi) ** tau
    assert abs(hits.mean() - p) <= 5 * math.sqrt(p * (1 - p) / S) + 1e-12
    # hashes use disjoint columns, so collisions of consecutive hashes are independent
    joint = (hits[0::2] & hits[1::2]).mean()
    half = S // 2
    assert abs(joint - p * p) <= 5 * math.sqrt(p * p * (1 - p * p) / half) + 1e-12


def test_collision_prob_closed_form_points():
    """Fig. 2: p(1) = 1, p(0) = 2^-tau, p(-1) = 0, and p is increasing."""
    for tau in (1, 2, 8, 9):
        assert oracle.collision_prob(1.0, tau) == 1.0
        assert abs(oracle.collision_prob(0.0, tau) - 2.0 ** -tau) < 1e-15
        assert oracle.collision_prob(-1.0, tau) == 0.0
        xs = np.linspace(-1, 1, 101)
        ps = [oracle.collision_prob(x, tau) for x in xs]
        assert all(b >= a for a, b in zip(ps, ps[1:]))


def test_surrogate_is_lower_bound_of_true_derivative():
    """Sec. 3.3 / Fig. 2: (tau/2) p(x) <= p'(x) on (-1, 1), p'(x) = tau (1-acos(x)/pi)^(tau-1) / (pi sqrt(1-x^2))."""
    for tau in (1, 2, 4, 8, 9, 16):
        xs = np.linspace(-0.999999, 0.999999, 20001)
        p1 = 1 - np.arccos(xs) / math.pi
        dp = tau * p1 ** (tau - 1) / (math.pi * np.sqrt(1 - xs ** 2))
        assert np.all(tau / 2 * p1 ** tau <= dp * (1 + 1e-12))


# ---------------------------------------------------------------- forward

def test_forward_matches_brute_force_pairs():
    q, k, v, dy, R = _rand_problem(3)
    m, tau = 3, 3
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    B = _brute_collisions(qc, kc)
    want = np.einsum("bhij,bjd->bid", B, v) / m
    np.testing.assert_allclose(oracle.forward(qc, kc, v, m, tau), want, rtol=0, atol=1e-12)


def test_forward_ones_counts_collisions():
    """Plugging V = 1 gives B 1 (Sec. 3.1, normalising attention): integer counts / m."""
    q, k, _, _, R = _rand_problem(4, nq=40, nk=31, d=6, m=5, tau=2)
    m, tau = 5, 2
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    y = oracle.forward(qc, kc, np.ones(k.shape), m, tau) * m
    np.testing.assert_allclose(y, np.round(y), rtol=0, atol=1e-12)
    y = np.round(y)
    counts = sum((qc[:, h, :, None] == kc[:, h, None, :]).sum(-1) for h in range(m))
    np.testing.assert_array_equal(y[..., 0], counts)


def test_forward_keys_equal_queries_collide_with_themselves():
    q, _, _, _, R = _rand_problem(5, nq=17, d=4, m=7, tau=4)
    m, tau = 7, 4
    c = oracle.hash_codes(q, R, m, tau)
    e = np.zeros((q.shape[0], 17, 17))
    e[:, np.arange(17), np.arange(17)] = 1.0   # v_j = e_j reads column j of C
    y = oracle.forward(c, c, e, m, tau) * m
    np.testing.assert_allclose(np.diagonal(y, axis1=1, axis2=2), m, rtol=0, atol=1e-12)


def test_antipodal_keys_never_collide():
    """K = -Q negates every projection, so (all margins being nonzero) every code of
    a key is the complement of its query's code: a row never collides with its own
    antipode, and a query whose only key is its antipode gathers exactly zero."""
    q, _, v, _, R = _rand_problem(30, bh=1, nq=40, nk=40, d=8, m=6, tau=5)
    qc, margin = oracle.hash_codes(q, R, 6, 5, with_margin=True)
    assert margin.min() > 0
    kc = oracle.hash_codes(-q, R, 6, 5)
    np.testing.assert_array_equal(kc, (~qc) & 31)
    # (other pairs may still collide; a row and its antipode never do)
    np.testing.assert_array_equal(np.diagonal(_brute_collisions(qc, kc)[0], axis1=1, axis2=2), 0.0)
    # with a single query and its antipode as the only key, nothing is ever gathered
    y = oracle.forward(qc[:, :, :1], kc[:, :, :1], v[:, :1], 6, 5)
    assert np.all(y == 0.0)


def test_forward_table_sums_are_the_value_sums():
    """One query per bucket (codes 0 .. 2^tau - 1) with m = 1: each query reads one
    bucket's table row, so the queries' outputs add up to the sum of all values
    (every key lands in exactly one bucket: sum_c H[c] = sum_j V_j)."""
    g = _rng(31)
    tau, nk, d = 4, 57, 5
    v = g.standard_normal((2, nk, d))
    kc = g.integers(0, 2 ** tau, size=(2, 1, nk)).astype(np.uint16)
    qc = np.tile(np.arange(2 ** tau, dtype=np.uint16), (2, 1, 1))
    y = oracle.forward(qc, kc, v, 1, tau)
    np.testing.assert_allclose(y.sum(axis=1), v.sum(axis=1), rtol=1e-12, atol=1e-12)
    # and each bucket's row is the sum of exactly its keys
    for b in range(2):
        for c in range(2 ** tau):
            np.testing.assert_allclose(y[b, c], v[b][kc[b, 0] == c].sum(axis=0), rtol=1e-12, atol=1e-12)


def test_forward_empty_keys_give_zero():
    qc = np.zeros((1, 2, 5), np.uint16)
    kc = np.zeros((1, 2, 0), np.uint16)
    y = oracle.forward(qc, kc, np.zeros((1, 0, 3)), 2, 4)
    assert y.shape == (1, 5, 3) and not y.any()


# ---------------------------------------------------------------- backward

def test_dv_is_adjoint_of_forward():
    """Y is linear in V, so <dY, Y> = <dV, V> exactly (eq. gradient-v, sampled)."""
    q, k, v, dy, R = _rand_problem(6)
    m, tau = 3, 3
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    y = oracle.forward(qc, kc, v, m, tau)
    _, _, dv = oracle.backward(qc, kc, q, k, v, dy, m, tau)
    assert abs(np.sum(dy * y) - np.sum(dv * v)) < 1e-10
    # finite difference of the sampled forward in V along a random direction
    e = _rng(7).standard_normal(v.shape)
    fd = np.sum(dy * (oracle.forward(qc, kc, v + 0.5 * e, m, tau) - y)) / 0.5
    assert abs(fd - np.sum(dv * e)) < 1e-9


def test_dqdk_pairwise_equals_backward_d2():
    """eq. (pseudo-gradient-q) evaluated pair by pair equals eq. (backward-d2)."""
    q, k, v, dy, R = _rand_problem(8, nq=29, nk=33, d=6, m=4, tau=2)
    m, tau = 4, 2
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    dq, dk, _ = oracle.backward(qc, kc, q, k, v, dy, m, tau)
    dq2, dk2 = oracle.backward_d2(qc, kc, q, k, v, dy, m, tau)
    np.testing.assert_allclose(dq, dq2, rtol=0, atol=1e-11)
    np.testing.assert_allclose(dk, dk2, rtol=0, atol=1e-11)


def test_backward_matches_dense_masked_brute_force():
    q, k, v, dy, R = _rand_problem(9)
    m, tau = 3, 3
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    C = _brute_collisions(qc, kc).sum(axis=1)            # [bh, nq, nk]
    S = np.einsum("bid,bjd->bij", dy, v)                  # dY V^T
    W = tau / (2 * m) * S * C
    dq, dk, dv = oracle.backward(qc, kc, q, k, v, dy, m, tau)
    np.testing.assert_allclose(dq, np.einsum("bij,bjd->bid", W, k), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dk, np.einsum("bij,bid->bjd", W, q), rtol=0, atol=1e-11)
    np.testing.assert_allclose(dv, np.einsum("bij,bid->bjd", C / m, dy), rtol=0, atol=1e-11)


def test_dq_dk_inner_products_agree():
    """<dQ, Q> = <dK, K> = tau/(2m) sum_ij C_ij (dY_i.V_j)(Q_i.K_j) for the surrogate."""
    q, k, v, dy, R = _rand_problem(10, nq=31, nk=27, d=7, m=5, tau=2)
    m, tau = 5, 2
    qc, kc = oracle.hash_codes(q, R, m, tau), oracle.hash_codes(k, R, m, tau)
    dq, dk, _ = oracle.backward(qc, kc, q, k, v, dy, m, tau)
    a, b = np.sum(dq * q), np.sum(dk * k)
    assert abs(a - b) < 1e-10 * max(1.0, abs(a))


# ---------------------------------------------------------------- Monte-Carlo laws

def _mc_batches(q, k, v, dy, tau, hashes, batches, seed):
    """Average of the sampled forward/backward over `hashes` fresh hash functions,
    repeated for `batches` independent batches."""
    d = q.shape[-1]
    outs = []
    g = _rng(seed)
    for _ in range(batches):
        R = g.standard_normal((d, hashes * tau))
        qc, kc = oracle.hash_codes(q, R, hashes, tau), oracle.hash_codes(k, R, hashes, tau)
        y = oracle.forward(qc, kc, v, hashes, tau)
        dq, dk, dv = oracle.backward(qc, kc, q, k, v, dy, hashes, tau)
        outs.append(np.stack([y, dq, dk, dv]))
    return np.stack(outs)  # [batches, 4, bh, n, d]


def test_monte_carlo_mean_converges_to_expectation():
    """YOSO-m -> YOSO-E (Sec. 3.1): the average over many hashes tends to P V, and the
    backward average to P^T dY and (tau/2)[(dY V^T) .* P] K (eqs. gradient-v,
    pseudo-gradient-q).  Fig. 1 setting: n = 32 keys in 3 dimensions."""
    g = _rng(11)
    tau = 4
    q = _unit(g.standard_normal((1, 32, 3)))
    k = _unit(g.standard_normal((1, 32, 3)))
    v = g.standard_normal((1, 32, 3))
    dy = g.standard_normal((1, 32, 3))
    ey, edv, edq, edk = oracle.expectation(q, k, v, dy, tau)
    want = np.stack([ey, edq, edk, edv])
    samples = _mc_batches(q, k, v, dy, tau, hashes=256, batches=40, seed=12)
    mean = samples.mean(0)
    se = samples.std(0, ddof=1) / math.sqrt(samples.shape[0])
    z = np.abs(mean - want) / np.maximum(se, 1e-12)
    assert np.all(z < 6.0), z.max()
    # error falls roughly like 1/sqrt(number of hashes)
    small = _mc_batches(q, k, v, dy, tau, hashes=64, batches=1, seed=13)[0]
    large = _mc_batches(q, k, v, dy, tau, hashes=4096, batches=1, seed=14)[0]
    e_small = np.linalg.norm(small - want)
    e_large = np.linalg.norm(large - want)
    assert e_large < e_small / 3.0  # sqrt(64) = 8 in expectation


def test_true_gradient_matches_finite_difference_of_expectation():
    """eq. (gradient-q): the derivative of <dY, P V> in q_i along a tangent direction."""
    g = _rng(15)
    tau, d = 3, 5
    q = _unit(g.standard_normal((1, 4, d)))
    k = _unit(g.standard_normal((1, 6, d)))
    v = g.standard_normal((1, 6, d))
    dy = g.standard_normal((1, 4, d))
    _, _, _, _, tdq, _ = oracle.expectation(q, k, v, dy, tau, true_grad=True)
    i = 2
    t = g.standard_normal(d)
    t -= (t @ q[0, i]) * q[0, i]
    t /= np.linalg.norm(t)
    def loss(eps):
        qq = q.copy()
        qq[0, i] = _unit(q[0, i] + eps * t)
        return np.sum(dy * oracle.expectation(qq, k, v, dy, tau)[0])
    h = 1e-5
    fd = (loss(h) - loss(-h)) / (2 * h)
    assert abs(fd - tdq[0, i] @ t) < 1e-6 * max(1.0, abs(fd))


def test_true_gradient_of_keys_matches_finite_difference_of_expectation():
    """The K counterpart of eq. (gradient-q): the derivative of <dY, P V> in k_j."""
    g = _rng(16)
    tau, d = 4, 6
    q = _unit(g.standard_normal((1, 5, d)))
    k = _unit(g.standard_normal((1, 3, d)))
    v = g.standard_normal((1, 3, d))
    dy = g.standard_normal((1, 5, d))
    _, _, _, _, _, tdk = oracle.expectation(q, k, v, dy, tau, true_grad=True)
    j = 1
    t = g.standard_normal(d)
    t -= (t @ k[0, j]) * k[0, j]
    t /= np.linalg.norm(t)
    def loss(eps):
        kk = k.copy()
        kk[0, j] = _unit(k[0, j] + eps * t)
        return np.sum(dy * oracle.expectation(q, kk, v, dy, tau)[0])
    h = 1e-5
    fd = (loss(h) - loss(-h)) / (2 * h)
    assert abs(fd - tdk[0, j] @ t) < 1e-6 * max(1.0, abs(fd))


# ---------------------------------------------------------------- *YOSO (true-gradient estimator)

def test_star_worked_example(golden):
    g = golden["star_backward"]
    m, tau = g["m"], g["tau"]
    qc = np.array(g["qc"], np.uint16)[None]
    kc = np.array(g["kc"], np.uint16)[None]
    q, k, v, dy = (np.array(g[s])[None] for s in ("q", "k", "v", "dy"))
    dq, dk, dv = oracle.backward_star(qc, kc, q, k, v, dy, m, tau)
    np.testing.assert_allclose(dq[0] * math.pi, g["dq_times_pi"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk[0] * math.pi, g["dk_times_pi"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dv[0], g["dv"], rtol=0, atol=1e-12)
    f = g["floored"]
    qc = np.array(f["qc"], np.uint16)[None]
    kc = np.array(f["kc"], np.uint16)[None]
    q, k, v, dy = (np.array(f[s])[None] for s in ("q", "k", "v", "dy"))
    dq, dk, _ = oracle.backward_star(qc, kc, q, k, v, dy, 1, f["tau"])
    np.testing.assert_allclose(dq[0] * math.pi, f["dq_times_pi"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(dk[0] * math.pi, f["dk_times_pi"], rtol=0, atol=1e-12)


def test_star_is_exact_at_tau_one():
    """With one bit per hash every pair collides after dropping that bit, so the
    estimator is the true gradient of eq. (gradient-q) at tau = 1 for any draw."""
    q, k, v, dy, R = _rand_problem(20, nq=13, nk=11, d=6, m=3, tau=1)
    qc, kc = oracle.hash_codes(q, R, 3, 1), oracle.hash_codes(k, R, 3, 1)
    dq, dk, _ = oracle.backward_star(qc, kc, q, k, v, dy, 3, 1)
    _, _, _, _, tdq, tdk = oracle.expectation(q, k, v, dy, 1, true_grad=True, floor=oracle.STAR_FLOOR)
    np.testing.assert_allclose(dq, tdq, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dk, tdk, rtol=1e-12, atol=1e-12)


def test_star_pairs_two_bits_apart_contribute_nothing():
    """Codes that differ in two or more bits are never counted; dV stays the
    sampled eq. (gradient-v), which is zero without equal codes."""
    q, k, v, dy, _ = _rand_problem(21, bh=1, nq=5, nk=4, d=4)
    qc = np.zeros((1, 2, 5), np.uint16)
    kc = np.full((1, 2, 4), 0b0110, np.uint16)
    dq, dk, dv = oracle.backward_star(qc, kc, q, k, v, dy, 2, 4)
    assert not dq.any() and not dk.any() and not dv.any()
    kc[0, 1, 2] = 0b0100  # one bit away from 0 in hash 1 only: key 2 meets every query once
    dq, dk, _ = oracle.backward_star(qc, kc, q, k, v, dy, 2, 4)
    assert np.abs(dk[0, [0, 1, 3]]).max() == 0 and np.abs(dk[0, 2]).max() > 0
    assert np.all(np.abs(dq[0]).max(axis=1) > 0)


def test_star_inner_products_agree():
    """<dQ*, Q> = <dK*, K>: both are (1/m) sum C_h(i,j) w_ij (dY_i.V_j)(Q_i.K_j)."""
    q, k, v, dy, R = _rand_problem(22, nq=29, nk=31, d=7, m=4, tau=3)
    qc, kc = oracle.hash_codes(q, R, 4, 3), oracle.hash_codes(k, R, 4, 3)
    dq, dk, _ = oracle.backward_star(qc, kc, q, k, v, dy, 4, 3)
    a, b = np.sum(dq * q), np.sum(dk * k)
    assert abs(a) > 1e-3 and abs(a - b) < 1e-10 * abs(a)


def test_star_monte_carlo_mean_converges_to_true_gradient():
    """*YOSO is unbiased for eq. (gradient-q): over many hash draws its mean tends
    to tau (1 - theta/pi)^(tau-1) / (pi sqrt(max(1 - x^2, 1/64))) weighting, for Q and
    K.  One query-key pair is nearly parallel (x = 0.998) so that the bound is active."""
    g = _rng(23)
    tau, d = 4, 3
    q = _unit(g.standard_normal((1, 12, d)))
    k = _unit(g.standard_normal((1, 10, d)))
    k[0, 0] = _unit(q[0, 0] + 0.063 * _unit(g.standard_normal(d)))
    assert 1 - (q[0, 0] @ k[0, 0]) ** 2 < oracle.STAR_FLOOR
    v = g.standard_normal((1, 10, d))
    dy = g.standard_normal((1, 12, d))
    _, _, _, _, tdq, tdk = oracle.expectation(q, k, v, dy, tau, true_grad=True, floor=oracle.STAR_FLOOR)
    want = np.concatenate([tdq.ravel(), tdk.ravel()])
    outs = []
    for _ in range(40):
        R = g.standard_normal((d, 256 * tau))
        qc, kc = oracle.hash_codes(q, R, 256, tau), oracle.hash_codes(k, R, 256, tau)
        dq, dk, _ = oracle.backward_star(qc, kc, q, k, v, dy, 256, tau)
        outs.append(np.concatenate([dq.ravel(), dk.ravel()]))
    samples = np.stack(outs)
    mean = samples.mean(0)
    se = samples.std(0, ddof=1) / math.sqrt(samples.shape[0])
    z = np.abs(mean - want) / np.maximum(se, 1e-12)
    assert np.all(z < 6.0), z.max()
    # and the surrogate of eq. (pseudo-gradient-q) is a different quantity
    _, _, edq, _ = oracle.expectation(q, k, v, dy, tau)
    assert np.linalg.norm(edq - tdq) > 10 * np.linalg.norm(se[:tdq.size])


# ---------------------------------------------------------------- l2 normalisation (N-YOSO, Q/K prologue)
def _l2_inputs(seed, rows=7, d=64):
    g = _rng(seed)
    x = g.standard_normal((rows, d)) * g.uniform(1e-3, 1e3, size=(rows, 1))
    x[2] = 0.0  # the zero row
    return x


def test_l2_normalize_unit_rows_and_zero_row():
    x = _l2_inputs(11)
    y = oracle.l2_normalize(x)
    n = np.linalg.norm(y, axis=-1)
    assert np.allclose(np.delete(n, 2), 1.0, atol=1e-14)
    assert np.all(y[2] == 0.0)
    # direction kept: y is a positive multiple of x
    for r in (0, 1, 3):
        assert np.allclose(y[r] * np.linalg.norm(x[r]), x[r], rtol=1e-12, atol=0)


def test_l2_normalize_scale_and_sign_invariance():
    x = _l2_inputs(12)
    y = oracle.l2_normalize(x)
    assert np.allclose(oracle.l2_normalize(3.7 * x), y, atol=1e-15)
    assert np.allclose(oracle.l2_normalize(-x), -y, atol=1e-15)
    # a basis vector and a two-hot vector have known normalisations
    e = np.zeros((2, 64))
    e[0, 5] = 4.0
    e[1, [1, 2]] = 3.0, 4.0
    ye = oracle.l2_normalize(e)
    assert ye[0, 5] == 1.0 and np.count_nonzero(ye[0]) == 1
    assert np.allclose(ye[1, [1, 2]], [0.6, 0.8], atol=1e-15)


def test_l2_backward_matches_central_differences():
    g = _rng(13)
    x = g.standard_normal((3, 64))
    dy = g.standard_normal((3, 64))
    dx = oracle.l2_normalize_backward(x, dy)
    h = 1e-6
    fd = np.zeros_like(x)
    for r in range(x.shape[0]):
        for j in range(x.shape[1]):
            xp, xm = x.copy(), x.copy()
            xp[r, j] += h
            xm[r, j] -= h
            fd[r, j] = (np.sum(dy * oracle.l2_normalize(xp)) - np.sum(dy * oracle.l2_normalize(xm))) / (2 * h)
    assert np.allclose(dx, fd, rtol=1e-6, atol=1e-8)


def test_l2_backward_matches_autograd():
    torch = pytest.importorskip("torch")
    x = _l2_inputs(14)
    g = _rng(15).standard_normal(x.shape)
    xt = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    nz = xt.norm(dim=-1, keepdim=True)
    yt = torch.where(nz > 0, xt / nz.clamp_min(1e-300), torch.zeros_like(xt))
    (yt * torch.tensor(g)).sum().backward()
    dx = oracle.l2_normalize_backward(x, g)
    ref = xt.grad.numpy()
    ref[2] = 0.0
    assert np.allclose(dx, ref, rtol=1e-10, atol=1e-300)


def test_l2_backward_invariants():
    x = _l2_inputs(16)
    g = _rng(17).standard_normal(x.shape)
    dx = oracle.l2_normalize_backward(x, g)
    # the gradient is orthogonal to x (moving along x does not change x/||x||) ...
    dots = np.sum(dx * x, axis=-1) / (np.linalg.norm(x, axis=-1) * np.linalg.norm(dx, axis=-1) + 1e-300)
    assert np.all(np.abs(np.delete(dots, 2)) < 1e-12)
    # ... scales as 1/||x|| ...
    assert np.allclose(oracle.l2_normalize_backward(2.0 * x, g), 0.5 * dx, rtol=1e-12, atol=0)
    # ... passes a gradient orthogonal to x through scaled by 1/||x||, and kills one along x
    r = 0
    u = x[r] / np.linalg.norm(x[r])
    gp = g[r] - u * np.dot(u, g[r])
    assert np.allclose(oracle.l2_normalize_backward(x[r:r + 1], gp[None])[0], gp / np.linalg.norm(x[r]), rtol=1e-11)
    assert np.allclose(oracle.l2_normalize_backward(x[r:r + 1], u[None])[0], 0.0, atol=1e-15)
    assert np.all(dx[2] == 0.0)


# ---------------------------------------------------------------- fast hash (Sec. 3.2 "Speed-up")

def _signs(seed, nrot):
    return _rng(seed).integers(0, 2**64, size=(nrot, 3), dtype=np.uint64)


def test_hadamard_is_sylvester():
    """The oracle's Walsh-Hadamard matrix equals scipy's Sylvester construction, and
    H H^T = d I."""
    sl = pytest.importorskip("scipy.linalg")
    for d in (1, 2, 4, 8, 16, 32, 64):
        H = oracle.hadamard(d)
        np.testing.assert_array_equal(H, sl.hadamard(d))
        np.testing.assert_array_equal(H @ H.T, d * np.eye(d))


def test_fast_hyperplanes_hand_worked_d2():
    """d = 2, D1 = diag(1, -1), D2 = D3 = I, worked by hand:
         H D1 = [[1, -1], [1, 1]],  H H D1 = [[2, 0], [0, -2]],  H H H D1 = [[2, -2], [2, 2]],
       so M = [[1, -1], [1, 1]] and R (column l = row l of M) = [[1, 1], [-1, 1]].
       Hashing e_0 gives projections (1, 1) -> code 3; e_1 gives (-1, 1) -> code 2."""
    signs = np.array([[0b10, 0, 0]], np.uint64)
    R = oracle.fast_hyperplanes(signs, 2, 1, 2)
    np.testing.assert_array_equal(R, [[1.0, 1.0], [-1.0, 1.0]])
    codes = oracle.fast_hash_codes(np.eye(2)[None], signs, 1, 2)
    np.testing.assert_array_equal(codes[0, 0], [3, 2])


def test_fast_hyperplanes_without_signs_are_hadamard_rows():
    """With no negations M = H^3 / d = H (H^2 = d I), so hashing the basis vector e_j
    reads row l = c mod d of H at column j: bit = [(-1)^popcount(l & j) > 0]."""
    d, m, tau = 64, 20, 7                       # 140 columns: three rotations, the last partial
    nrot = (m * tau + d - 1) // d
    codes = oracle.fast_hash_codes(np.eye(d)[None], np.zeros((nrot, 3), np.uint64), m, tau)
    for j in range(d):
        for h in range(m):
            want = sum(1 << b for b in range(tau) if bin(((h * tau + b) % d) & j).count("1") % 2 == 0)
            assert codes[0, h, j] == want


def test_fast_hyperplanes_rotations_are_orthogonal():
    """Each rotation (1/d) H D3 H D2 H D1 has orthogonal rows of length sqrt(d); the
    columns of R it supplies are those rows, the last rotation only its first ones."""
    d, m, tau = 64, 30, 9                       # 270 columns: 4 full rotations + 14 rows
    R = oracle.fast_hyperplanes(_signs(21, 5), d, m, tau)
    for r in range(5):
        blk = R[:, r * d:(r + 1) * d]
        np.testing.assert_allclose(blk.T @ blk, d * np.eye(blk.shape[1]), atol=1e-12)
    # distinct rotations are not aligned with each other
    assert np.abs(R[:, :d].T @ R[:, d:2 * d]).max() > 1.0


def test_fast_hash_sign_flip_invariances():
    """D1 acts on the input: negating coordinate j in D1 is the same as negating x_j.
    Negating every coordinate of any one D_i negates every projection, so every code
    is complemented (all margins here are nonzero)."""
    d, m, tau = 64, 16, 8
    x = _unit(_rng(22).standard_normal((1, 40, d)))
    s = _signs(23, 2)
    base, margin = oracle.fast_hash_codes(x, s, m, tau, with_margin=True)
    assert margin.min() > 0
    for j in (0, 5, 63):
        s1 = s.copy()
        s1[0, 0] ^= np.uint64(1) << np.uint64(j)
        s1[1, 0] ^= np.uint64(1) << np.uint64(j)
        xj = x.copy()
        xj[..., j] = -xj[..., j]
        np.testing.assert_array_equal(oracle.fast_hash_codes(x, s1, m, tau), oracle.fast_hash_codes(xj, s, m, tau))
        assert (oracle.fast_hash_codes(x, s1, m, tau) != base).any()
    for i in range(3):
        sf = s.copy()
        sf[:, i] = ~sf[:, i]
        np.testing.assert_array_equal(oracle.fast_hash_codes(x, sf, m, tau), (~base) & ((1 << tau) - 1))


@pytest.mark.parametrize("theta", [math.pi / 6, math.pi / 3, math.pi / 2, 2 * math.pi / 3])
def test_fast_hash_collision_law(theta):
    """The pseudo-random rotation stands in for a random rotation (Sec. 3.2 "Speed-up",
    after Andoni et al. 2015), so its bits follow the hyperplane law 1 - theta/pi and a
    4-bit code (1 - theta/pi)^4.  The pair is sparse (x = e_0, y in span(e_0, e_1)),
    where fewer than three D/H rounds visibly fail (one round gives collision 1 or 1/2
    per bit; two give a 4-bit code rate of ~0.26 at theta = pi/2 instead of 0.0625)."""
    d, tau, nrot = 64, 4, 1500
    x = np.zeros((1, 2, d))
    x[0, 0, 0] = 1.0
    x[0, 1, 0], x[0, 1, 1] = math.cos(theta), math.sin(theta)
    R = oracle.fast_hyperplanes(_signs(24, nrot), d, nrot * d // tau, tau)
    z = x[0] @ R                                  # projections of both rows on every column
    bit_hits = (z[0] > 0) == (z[1] > 0)
    codes = oracle.hash_codes(x, R, nrot * d // tau, tau)[0]
    code_hits = codes[:, 0] == codes[:, 1]
    p = 1 - theta / math.pi
    assert abs(bit_hits.mean() - p) <= 0.03
    assert abs(code_hits.mean() - p ** tau) <= 0.015
