"""Modulus chain, roots of unity and index helpers (CPU oracle; test infrastructure only).

The paper fixes the ring R_Q = Z_Q[X]/(X^N+1) with Q a product of RNS primes,
N a power of two, and rescaling that drops one prime per level (section 2.1).
Its own parameter set (N = 8192, primes of [60,30,30,30] bits, scale 2^30,
section 4.2) needs 64-bit residues; the workloads here use all-30-bit primes,
and the paper is silent on how they are chosen.  Readings taken:

* primes: q_0 > q_1 > ... > q_{L-1} are the L largest primes in (2^29, 2^30)
  with q = 1 (mod 2N); rescaling drops q_{L-1}, the smallest;
* psi_l: the smallest primitive 2N-th root of unity mod q_l (found as
  g^((q-1)/2N) for the smallest generator g of Z_q^*, then the minimum over all
  odd powers of that root).

Parity: pinned (tests/test_oracle_params.py) by sympy primality, exhaustive
scans of the skipped candidates, and a brute-force search for smaller roots.
"""
from __future__ import annotations

from functools import lru_cache

# Deterministic Miller-Rabin for n < 3,215,031,751 (Jaeschke 1993: bases 2, 3, 5, 7).
_MR_BASES = (2, 3, 5, 7)


def is_prime(n: int) -> bool:
    """Miller-Rabin, deterministic for n < 3.2e9 with bases 2, 3, 5, 7."""
    if n < 2:
        return False
    for p in (2, 3, 5, 7, 11, 13):
        if n % p == 0:
            return n == p
    d, s = n - 1, 0
    while d % 2 == 0:
        d //= 2
        s += 1
    for a in _MR_BASES:
        x = pow(a, d, n)
        if x in (1, n - 1):
            continue
        for _ in range(s - 1):
            x = x * x % n
            if x == n - 1:
                break
        else:
            return False
    return True


@lru_cache(maxsize=None)
def moduli(log_n: int, num_limbs: int) -> tuple[int, ...]:
    """The num_limbs largest primes q in (2^29, 2^30) with q = 1 mod 2N, descending."""
    two_n = 2 << log_n
    out = []
    # largest candidate of the form k*2N + 1 below 2^30
    q = ((1 << 30) - 2) // two_n * two_n + 1
    while len(out) < num_limbs:
        if q <= (1 << 29):
            raise ValueError("not enough primes in (2^29, 2^30) for this N")
        if is_prime(q):
            out.append(q)
        q -= two_n
    return tuple(out)


def _prime_factors(n: int) -> list[int]:
    fs, p = [], 2
    while p * p <= n:
        if n % p == 0:
            fs.append(p)
            while n % p == 0:
                n //= p
        p += 1
    if n > 1:
        fs.append(n)
    return fs


@lru_cache(maxsize=None)
def smallest_generator(q: int) -> int:
    """Smallest g whose multiplicative order mod prime q is q-1."""
    fs = _prime_factors(q - 1)
    g = 2
    while any(pow(g, (q - 1) // f, q) == 1 for f in fs):
        g += 1
    return g


@lru_cache(maxsize=None)
def psi(q: int, log_n: int) -> int:
    """Minimal primitive 2N-th root of unity mod q."""
    two_n = 2 << log_n
    if (q - 1) % two_n:
        raise ValueError("q is not 1 mod 2N")
    root = pow(smallest_generator(q), (q - 1) // two_n, q)
    best = min(pow(root, k, q) for k in range(1, two_n, 2))
    assert pow(best, two_n // 2, q) == q - 1
    return best


def brv(i: int, bits: int) -> int:
    """Reverse the low `bits` bits of i."""
    r = 0
    for _ in range(bits):
        r = (r << 1) | (i & 1)
        i >>= 1
    return r


def modinv(a: int, q: int) -> int:
    return pow(a % q, -1, q)


def crt_lift(residues, qs) -> list[int]:
    """CRT: the unique C in [0, Q) with C = r_l mod q_l (residues given per limb, same length)."""
    Q = 1
    for q in qs:
        Q *= q
    coeffs = []
    for q in qs:
        Qi = Q // q
        coeffs.append(Qi * modinv(Qi, q))
    n = len(residues[0])
    out = []
    for k in range(n):
        c = 0
        for l, q in enumerate(qs):
            c += int(residues[l][k]) * coeffs[l]
        out.append(c % Q)
    return out


def centre(c: int, Q: int) -> int:
    """Representative of c mod Q in (-Q/2, Q/2]."""
    c %= Q
    return c - Q if c > Q // 2 else c
