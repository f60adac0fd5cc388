"""CKKS encoding and decoding by direct canonical-embedding sums (CPU oracle; test infrastructure only).

The paper's plaintexts pack N/2 complex slots into one element of
R = Z[X]/(X^N+1) (section 2.1, CKKS as cited there); its weights are encoded
once and kept resident, or re-encoded per call when they do not fit (section
4.2; fallback encoding is 34.4% of Qwen3 decode in the cost-breakdown table of
section 6.1).  The paper is silent on the slot order and rounding; readings:

* slot j is the value at zeta_j = exp(i*pi*e_j/N), e_j = 5^j mod 2N, j < N/2
  (the standard CKKS ordering; the conjugate slots are implied);
* the inverse embedding is m_k = (2/N) * Re sum_j z_j * zeta_j^(-k), k < N;
* rounding is IEEE round-half-to-even (numpy.rint), p_k = rint(Delta * m_k);
* scalar weights are the constant polynomial rint(w * Delta), so their RNS
  residues are rint(w * Delta) mod q_l.

Exponents are reduced mod 2N (as integers) before the cos/sin lookup.  Sums
are plain fp64 sums (a matmul against the gathered cos/sin table).

Parity: pinned (tests/test_oracle_encode.py) by the constant-slot closed form,
Parseval's identity, evaluation of the encoded polynomial at the roots via
numpy's FFT, and the decode(encode(z)) rounding bound.
"""
from __future__ import annotations

import numpy as np

from .ntt import ntt


def slot_exponents(log_n: int) -> np.ndarray:
    """e_j = 5^j mod 2N for j < N/2."""
    n = 1 << log_n
    out = np.empty(n // 2, dtype=np.int64)
    x = 1
    for j in range(n // 2):
        out[j] = x
        x = x * 5 % (2 * n)
    return out


def _trig_tables(log_n: int):
    n = 1 << log_n
    t = np.arange(2 * n, dtype=np.float64)
    return np.cos(np.pi * t / n), np.sin(np.pi * t / n)


def encode_coeffs(z, log_n: int, ks=None) -> np.ndarray:
    """Real coefficients m_k (fp64) of the inverse canonical embedding of slots z (..., N/2),
    for every k < N, or only for the indices ks (..., len(ks))."""
    n = 1 << log_n
    z = np.asarray(z)
    zr = np.real(z).astype(np.float64).reshape(-1, n // 2)
    zi = np.imag(z).astype(np.float64).reshape(-1, n // 2) if np.iscomplexobj(z) else None
    cos_t, sin_t = _trig_tables(log_n)
    e = slot_exponents(log_n)
    kall = np.arange(n, dtype=np.int64) if ks is None else np.asarray(ks, dtype=np.int64)
    out = np.empty((zr.shape[0], len(kall)), dtype=np.float64)
    chunk = max(1, (1 << 22) // (n // 2))
    for c0 in range(0, len(kall), chunk):
        k = kall[c0:c0 + chunk]
        t = np.outer(e, k) % (2 * n)                      # (N/2, chunk): exponent of zeta_j^k
        # Re(z * zeta^-k) = Re(z) cos(theta) + Im(z) sin(theta), theta = pi t / N
        acc = zr @ cos_t[t]
        if zi is not None:
            acc += zi @ sin_t[t]
        out[:, c0:c0 + len(k)] = acc * (2.0 / n)
    return out.reshape(z.shape[:-1] + (len(kall),))


def round_coeffs(m, delta: float) -> np.ndarray:
    """p_k = rint(Delta * m_k) (ties to even), as int64."""
    v = np.rint(np.asarray(m, dtype=np.float64) * delta)
    if np.any(np.abs(v) >= 2.0 ** 62):
        raise OverflowError("encoded coefficient beyond 2^62")
    return v.astype(np.int64)


def to_residues(p, qs) -> np.ndarray:
    """Signed integers (...,) -> residues (..., L) in [0, q_l)."""
    p = np.asarray(p, dtype=np.int64)
    return np.stack([np.mod(p, q).astype(np.uint64) for q in qs], axis=-1)


def encode_scalar(w, delta: float, qs) -> np.ndarray:
    """Scalar weights w (...) -> residues (..., L) of the constant polynomial rint(w*Delta)."""
    return to_residues(round_coeffs(w, delta), qs)


def encode_poly(z, delta: float, qs, psis, log_n: int) -> np.ndarray:
    """Slot vectors z (..., N/2) -> NTT-form plaintext residues (..., L, N)."""
    p = round_coeffs(encode_coeffs(z, log_n), delta)          # (..., N)
    res = to_residues(p, qs)                                   # (..., N, L)
    res = np.moveaxis(res, -1, -2)                             # (..., L, N)
    out = np.empty_like(res)
    for l, (q, ps) in enumerate(zip(qs, psis)):
        out[..., l, :] = ntt(res[..., l, :], q, ps, log_n)
    return out


def decode(m, delta: float, log_n: int) -> np.ndarray:
    """Slots z_j = (1/Delta) sum_k m_k zeta_j^k for integer (or real) coefficients m.

    m is one coefficient vector (N,) or a batch (B, N); returns (N/2,) or (B, N/2).
    """
    n = 1 << log_n
    single = np.ndim(m) == 1 if not isinstance(m, list) else not isinstance(m[0], (list, np.ndarray))
    rows = [m] if single else list(m)
    mf = np.array([[float(x) for x in row] for row in rows], dtype=np.float64).T      # (N, B)
    cos_t, sin_t = _trig_tables(log_n)
    e = slot_exponents(log_n)
    k = np.arange(n, dtype=np.int64)
    out = np.empty((n // 2, mf.shape[1]), dtype=np.complex128)
    chunk = max(1, (1 << 22) // n)
    for j0 in range(0, n // 2, chunk):
        ej = e[j0:j0 + chunk]
        t = np.outer(ej, k) % (2 * n)
        out[j0:j0 + len(ej)] = (cos_t[t] @ mf + 1j * (sin_t[t] @ mf)) / delta
    out = out.T
    return out[0] if single else out
