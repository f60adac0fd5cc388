"""Pins for oracle/params.py: the modulus chain and the roots of unity.

The paper is silent on prime and root choice for these workloads; the reading
(L largest NTT-friendly 30-bit primes, minimal primitive 2N-th root) is checked
here against sympy's primality test, exhaustive scans and brute-force search.
"""
import numpy as np
import pytest
import sympy

from oracle import params

CASES = [(10, 2), (11, 3), (12, 3), (14, 4), (15, 6), (16, 8)]


@pytest.mark.parametrize("log_n,L", CASES)
def test_moduli_are_the_largest_ntt_primes(log_n, L):
    qs = params.moduli(log_n, L)
    two_n = 2 << log_n
    assert len(qs) == L
    assert list(qs) == sorted(qs, reverse=True)
    for q in qs:
        assert (1 << 29) < q < (1 << 30)
        assert q % two_n == 1
        assert sympy.isprime(q)
    # every skipped candidate k*2N+1 between q_{L-1} and 2^30 is composite
    cand = ((1 << 30) - 2) // two_n * two_n + 1
    while cand > qs[-1]:
        assert (cand in qs) == sympy.isprime(cand)
        cand -= two_n


def test_miller_rabin_agrees_with_sympy_on_a_range():
    lo = (1 << 30) - 20000
    for n in range(lo, lo + 20000, 3):
        assert params.is_prime(n) == sympy.isprime(n)


def _pow_vec(x: np.ndarray, e: int, q: int) -> np.ndarray:
    r = np.ones_like(x)
    b = x.copy()
    while e:
        if e & 1:
            r = (r * b) % np.uint64(q)
        b = (b * b) % np.uint64(q)
        e >>= 1
    return r


@pytest.mark.parametrize("log_n,L", CASES)
def test_psi_is_the_minimal_primitive_2n_th_root(log_n, L):
    n = 1 << log_n
    for q in params.moduli(log_n, L):
        psi = params.psi(q, log_n)
        assert pow(psi, n, q) == q - 1          # order exactly 2N (2N a power of two)
        smaller = np.arange(2, psi, dtype=np.uint64)
        if len(smaller):
            assert not np.any(_pow_vec(smaller, n, q) == q - 1)


def test_generator_has_full_order():
    for q in params.moduli(12, 3):
        g = params.smallest_generator(q)
        assert sympy.n_order(g, q) == q - 1
        assert all(sympy.n_order(h, q) != q - 1 for h in range(2, g))


def test_brv_and_crt():
    assert [params.brv(i, 3) for i in range(8)] == [0, 4, 2, 6, 1, 5, 3, 7]
    qs = params.moduli(10, 3)
    Q = qs[0] * qs[1] * qs[2]
    rng = np.random.default_rng(5)
    vals = [int(x) for x in rng.integers(0, 2**62, size=20)] + [0, Q - 1, 12345]
    res = [[v % q for v in vals] for q in qs]
    assert params.crt_lift(res, qs) == [v % Q for v in vals]
    assert params.centre(Q - 1, Q) == -1 and params.centre(5, Q) == 5
