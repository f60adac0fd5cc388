"""Schoolbook negacyclic products in Z_q[X]/(X^N+1) and Z[X]/(X^N+1) (CPU oracle; test infrastructure only).

The ring is the one of section 2.1.  Products are computed by the schoolbook
rule X^a * X^b = X^(a+b), with X^N = -1; no transform is involved, so these
functions are what the NTT's convolution theorem is checked against.

Parity: pinned (tests/test_oracle_ntt.py) by hand-checkable monomial cases
(X^(N-1) * X = -1) and by commutativity/associativity on random inputs.
"""
from __future__ import annotations

import numpy as np


def negacyclic_mul(a, b, q: int) -> np.ndarray:
    """c = a * b mod (X^N + 1, q); a, b are residue vectors of length N."""
    qq = np.uint64(q)
    a = np.asarray(a, dtype=np.uint64) % qq
    b = np.asarray(b, dtype=np.uint64) % qq
    n = a.shape[-1]
    c = np.zeros(n, dtype=np.uint64)
    for k in range(n):
        ak = a[k]
        if ak == 0:
            continue
        t = (b * ak) % qq                      # a_k * X^k * b(X): coefficient m lands on m + k
        c[k:] = (c[k:] + t[:n - k]) % qq       # no wrap
        if k:
            c[:k] = (c[:k] + (qq - t[n - k:]) % qq) % qq   # wrapped past X^N: sign flips
    return c


def negacyclic_mul_z(a, b) -> list[int]:
    """Exact product over Z[X]/(X^N+1) with Python integers (small N only)."""
    n = len(a)
    c = [0] * n
    for k in range(n):
        ak = int(a[k])
        if ak == 0:
            continue
        for m in range(n):
            v = ak * int(b[m])
            p = k + m
            if p < n:
                c[p] += v
            else:
                c[p - n] -= v
    return c
