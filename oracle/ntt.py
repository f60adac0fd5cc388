"""Negacyclic NTT / INTT per RNS limb (CPU oracle; test infrastructure only).

The paper's ring is R_Q = Z_Q[X]/(X^N+1) (section 2.1) and its accelerator
kernels work on ciphertexts in NTT form (section 4.2 names the NTT kernels).
The paper is silent on ordering and scaling; the reading taken is

    NTT(a)[i]  = sum_k a_k * psi^((2*brv(i)+1)*k)          mod q   (unscaled)
    INTT(b)[k] = N^-1 * sum_i b_i * psi^(-(2*brv(i)+1)*k)  mod q

i.e. evaluation of a(X) at the 2N-th primitive roots psi^(2j+1), listed in
bit-reversed order of j.

``ntt_direct`` / ``intt_direct`` are that definition written out (O(N^2)).
``ntt`` / ``intt`` are a textbook route for large N: twist by psi^k, a cyclic
radix-2 decimation-in-time DFT with omega = psi^2 (Cormen et al., iterative
FFT), then the bit-reversal read-out.  The tests pin ``ntt`` to
``ntt_direct`` at every point for N <= 2^10 and at sampled points up to 2^16,
and pin ``ntt_direct`` itself by Horner evaluation and by the convolution
theorem against the schoolbook negacyclic product.

All arrays are numpy uint64 with residues in [0, q); products stay < 2^60.
"""
from __future__ import annotations

from functools import lru_cache

import numpy as np

from .params import brv


@lru_cache(maxsize=256)
def _pow_table(base: int, count: int, q: int) -> np.ndarray:
    """base^e mod q for e < count (cached, read-only)."""
    out = np.empty(count, dtype=np.uint64)
    x = 1
    for e in range(count):
        out[e] = x
        x = x * base % q
    out.flags.writeable = False
    return out


@lru_cache(maxsize=32)
def brv_perm(log_n: int) -> np.ndarray:
    out = np.array([brv(i, log_n) for i in range(1 << log_n)], dtype=np.int64)
    out.flags.writeable = False
    return out


def ntt_direct(a, q: int, psi: int, log_n: int, points=None) -> np.ndarray:
    """NTT(a)[i] for i in `points` (default: all i < N), straight from the definition.

    `a` has shape (..., N).  Returns shape (..., len(points)).
    """
    n = 1 << log_n
    a = np.asarray(a, dtype=np.uint64) % np.uint64(q)
    pw = _pow_table(psi, 2 * n, q)
    pts = np.arange(n) if points is None else np.asarray(points, dtype=np.int64)
    k = np.arange(n, dtype=np.int64)
    out = np.empty(a.shape[:-1] + (len(pts),), dtype=np.uint64)
    chunk = max(1, (1 << 20) // n)
    for c0 in range(0, len(pts), chunk):
        sel = pts[c0:c0 + chunk]
        ex = np.array([2 * brv(int(i), log_n) + 1 for i in sel], dtype=np.int64)
        e = np.outer(ex, k) % (2 * n)                      # (chunk, N)
        terms = (a[..., None, :] * pw[e]) % np.uint64(q)   # (..., chunk, N), each < q
        out[..., c0:c0 + len(sel)] = terms.sum(axis=-1) % np.uint64(q)
    return out


def intt_direct(b, q: int, psi: int, log_n: int, points=None) -> np.ndarray:
    """INTT(b)[k] for k in `points` (default all), straight from the definition."""
    n = 1 << log_n
    b = np.asarray(b, dtype=np.uint64) % np.uint64(q)
    psi_inv = pow(psi, -1, q)
    n_inv = pow(n, -1, q)
    pw = _pow_table(psi_inv, 2 * n, q)
    pts = np.arange(n) if points is None else np.asarray(points, dtype=np.int64)
    ex = np.array([2 * brv(i, log_n) + 1 for i in range(n)], dtype=np.int64)
    out = np.empty(b.shape[:-1] + (len(pts),), dtype=np.uint64)
    chunk = max(1, (1 << 20) // n)
    for c0 in range(0, len(pts), chunk):
        sel = pts[c0:c0 + chunk]
        e = np.outer(sel, ex) % (2 * n)                    # (chunk, N): exponent for (k, i)
        terms = (b[..., None, :] * pw[e]) % np.uint64(q)
        s = terms.sum(axis=-1) % np.uint64(q)
        out[..., c0:c0 + len(sel)] = (s * np.uint64(n_inv)) % np.uint64(q)
    return out


def _cyclic_dft(x, omega: int, q: int) -> np.ndarray:
    """A_m = sum_k x_k omega^(m k) mod q over the last axis (length N, omega of order N).

    Iterative radix-2 decimation in time: bit-reverse the input, then merge
    pairs of half-length transforms with the twiddles omega_{2m}^j.
    """
    n = x.shape[-1]
    log_n = n.bit_length() - 1
    qq = np.uint64(q)
    y = np.ascontiguousarray(x[..., brv_perm(log_n)])
    lead = y.shape[:-1]
    m = 1
    while m < n:
        w_2m = pow(omega, n // (2 * m), q)                 # primitive 2m-th root
        tw = _pow_table(w_2m, m, q)
        y = y.reshape(lead + (n // (2 * m), 2, m))
        even = y[..., 0, :]
        t = (y[..., 1, :] * tw) % qq
        y = np.stack([(even + t) % qq, (even + qq - t) % qq], axis=-2)
        m *= 2
    return y.reshape(lead + (n,))


def ntt(a, q: int, psi: int, log_n: int) -> np.ndarray:
    """Fast oracle NTT over the last axis (same result as ntt_direct)."""
    n = 1 << log_n
    qq = np.uint64(q)
    a = np.asarray(a, dtype=np.uint64) % qq
    twist = _pow_table(psi, n, q)
    cyc = _cyclic_dft((a * twist) % qq, psi * psi % q, q)
    return np.ascontiguousarray(cyc[..., brv_perm(log_n)])


def intt(b, q: int, psi: int, log_n: int) -> np.ndarray:
    """Fast oracle INTT over the last axis (same result as intt_direct)."""
    n = 1 << log_n
    qq = np.uint64(q)
    b = np.asarray(b, dtype=np.uint64) % qq
    psi_inv = pow(psi, -1, q)
    cyc = b[..., brv_perm(log_n)]                            # A_m = b_brv(m)
    x = _cyclic_dft(cyc, psi_inv * psi_inv % q, q)
    untwist = (_pow_table(psi_inv, n, q) * np.uint64(pow(n, -1, q))) % qq
    return (x * untwist) % qq
