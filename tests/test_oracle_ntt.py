"""Pins for oracle/ntt.py and oracle/poly.py.

The NTT definition (evaluation at psi^(2*brv(i)+1), bit-reversed order) is
checked by Horner evaluation of the polynomial at those roots, by the
convolution theorem against the schoolbook negacyclic product, and by round
trips; the fast oracle route is checked against the definition.
"""
import numpy as np
import pytest

from oracle import ntt as O
from oracle import params, poly


def _setup(log_n, L=2):
    # primes = 1 mod 2^11 are also = 1 mod 2N for every smaller N
    qs = params.moduli(max(log_n, 10), L)
    return qs, [params.psi(q, log_n) for q in qs]


def _rand(rng, q, shape):
    return rng.integers(0, q, size=shape, dtype=np.uint64)


@pytest.mark.parametrize("log_n", [3, 4, 5, 6])
def test_direct_ntt_is_evaluation_at_the_odd_roots(log_n):
    n = 1 << log_n
    qs, psis = _setup(log_n)
    rng = np.random.default_rng(log_n)
    for q, psi in zip(qs, psis):
        a = _rand(rng, q, n)
        got = O.ntt_direct(a, q, psi, log_n)
        pts = [pow(psi, 2 * params.brv(i, log_n) + 1, q) for i in range(n)]
        assert len(set(pts)) == n and all(pow(x, n, q) == q - 1 for x in pts)
        for i, x in enumerate(pts):
            acc = 0
            for coef in reversed(a.tolist()):        # Horner
                acc = (acc * x + int(coef)) % q
            assert int(got[i]) == acc


@pytest.mark.parametrize("log_n", [3, 4, 5, 6])
def test_convolution_theorem_against_schoolbook(log_n):
    n = 1 << log_n
    qs, psis = _setup(log_n)
    rng = np.random.default_rng(100 + log_n)
    for q, psi in zip(qs, psis):
        a, b = _rand(rng, q, n), _rand(rng, q, n)
        prod = poly.negacyclic_mul(a, b, q)
        lhs = (O.ntt_direct(a, q, psi, log_n) * O.ntt_direct(b, q, psi, log_n)) % np.uint64(q)
        assert np.array_equal(lhs, O.ntt_direct(prod, q, psi, log_n))


def test_convolution_theorem_n1024_fast_route():
    log_n = 10
    qs, psis = _setup(log_n)
    rng = np.random.default_rng(7)
    q, psi = qs[0], psis[0]
    a, b = _rand(rng, q, 1024), _rand(rng, q, 1024)
    prod = poly.negacyclic_mul(a, b, q)
    lhs = (O.ntt(a, q, psi, log_n) * O.ntt(b, q, psi, log_n)) % np.uint64(q)
    assert np.array_equal(lhs, O.ntt(prod, q, psi, log_n))
    assert np.array_equal(O.intt(lhs, q, psi, log_n), prod)


@pytest.mark.parametrize("log_n", [3, 6, 10])
def test_round_trips_and_fast_equals_direct(log_n):
    n = 1 << log_n
    qs, psis = _setup(log_n)
    rng = np.random.default_rng(200 + log_n)
    for q, psi in zip(qs, psis):
        a = _rand(rng, q, (3, n))
        d = O.ntt_direct(a, q, psi, log_n)
        assert np.array_equal(O.intt_direct(d, q, psi, log_n), a)
        assert np.array_equal(O.ntt(a, q, psi, log_n), d)
        assert np.array_equal(O.intt(d, q, psi, log_n), a)


@pytest.mark.parametrize("log_n,L", [(14, 4), (15, 6), (16, 8)])
def test_fast_equals_direct_at_sampled_points_full_size(log_n, L):
    n = 1 << log_n
    qs = params.moduli(log_n, L)
    rng = np.random.default_rng(300 + log_n)
    for l in (0, L - 1):
        q, psi = qs[l], params.psi(qs[l], log_n)
        a = _rand(rng, q, n)
        fast = O.ntt(a, q, psi, log_n)
        pts = np.concatenate([[0, 1, n - 1], rng.choice(n, size=61, replace=False)])
        assert np.array_equal(fast[pts], O.ntt_direct(a, q, psi, log_n, points=pts))
        back = O.intt(fast, q, psi, log_n)
        assert np.array_equal(back, a)
        assert np.array_equal(back[pts], O.intt_direct(fast, q, psi, log_n, points=pts))


def test_ntt_special_values():
    log_n = 10
    n = 1 << log_n
    qs, psis = _setup(log_n)
    q, psi = qs[0], psis[0]
    one = np.zeros(n, dtype=np.uint64)
    one[0] = 1
    assert np.all(O.ntt(one, q, psi, log_n) == 1)
    x = np.zeros(n, dtype=np.uint64)
    x[1] = 1                                   # NTT(X)[i] is the i-th evaluation point
    got = O.ntt(x, q, psi, log_n)
    assert [int(v) for v in got[:8]] == [pow(psi, 2 * params.brv(i, log_n) + 1, q) for i in range(8)]


def test_schoolbook_hand_cases():
    q = 97
    n = 8
    xn1 = [0] * n
    xn1[n - 1] = 1
    x1 = [0] * n
    x1[1] = 1
    assert poly.negacyclic_mul(xn1, x1, q).tolist() == [q - 1] + [0] * (n - 1)   # X^(N-1) X = -1
    assert poly.negacyclic_mul_z(xn1, x1) == [-1] + [0] * (n - 1)
    # (1 + X)(1 - X) = 1 - X^2
    assert poly.negacyclic_mul_z([1, 1] + [0] * 6, [1, -1] + [0] * 6) == [1, 0, -1] + [0] * 5


def test_schoolbook_ring_laws():
    rng = np.random.default_rng(11)
    q, n = params.moduli(10, 1)[0], 32
    a, b, c = (_rand(rng, q, n) for _ in range(3))
    ab = poly.negacyclic_mul(a, b, q)
    assert np.array_equal(ab, poly.negacyclic_mul(b, a, q))
    assert np.array_equal(poly.negacyclic_mul(ab, c, q), poly.negacyclic_mul(a, poly.negacyclic_mul(b, c, q), q))
    z = poly.negacyclic_mul_z(a.tolist(), b.tolist())
    assert [v % q for v in z] == ab.tolist()
