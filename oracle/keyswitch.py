"""Galois automorphisms, key switching and slot rotations (CPU oracle; test infrastructure only).

The paper's FHE linear path is HEonGPU's baby-step / giant-step (BSGS) matrix-vector
product over pre-encoded weight diagonals (sections 4.1 and 4.2), and rotations of a
ciphertext are automorphisms followed by key switching under a special prime (section
4.2's parameter set has one special prime for key switching; section 2.1 notes that
rotations and key switching are explicit costs in CKKS).  The paper gives no formulas
for them; the readings taken are the standard ones:

* Automorphism sigma_g (g odd, taken mod 2N) maps a(X) to a(X^g) in Z[X]/(X^N + 1):
  coefficient k moves to position k*g mod 2N, negated when that position is N or more
  (X^N = -1).  With slot j at the root zeta^(5^j) (the slot order of the encoder),
  sigma_(5^r) puts old slot j + r at slot j: a left rotation of the slots by r.
* Key switching is the hybrid form with one special prime P and one digit per
  ciphertext limb.  Digit i of an NTT-form polynomial c over q_0 .. q_{L-1} is the
  centred coefficient vector of limb i (|d_i| < q_i / 2); the switching key from
  s_from to s_to has, per digit, the pair

      ksk_i = (-a_i * s_to + e_i + P * g_i * s_from,  a_i)    over q_0 .. q_{L-1}, P,

  with g_i the CRT idempotent of limb i (1 mod q_i, 0 mod the other q_j; P * g_i is 0
  mod P).  Then sum_i d_i * ksk_i decrypts under s_to to P * c * s_from + sum_i d_i e_i
  (mod Q P), and dividing by P, which is the rescale that drops the last prime (by its
  CRT definition, ``linear.rescale``), leaves c * s_from plus a small error.
* The special prime is a 30-bit prime (the next prime of the same chain, placed last)
  instead of the paper's 60-bit one, so that every residue stays below 2^30.  The error
  that key switching adds is then at most sum_i N (q_i / 2) |e|_max / P + N / 2 + 1 / 2
  per coefficient (about L * N * 10 for the error bound 19 used by the generators).
* Rotation by r: g = 5^r mod 2N; out = (sigma_g(c0) + u0, u1) where (u0, u1) switches
  sigma_g(c1) from the key sigma_g(s) back to s.

The random draws of key generation (a_i uniform in NTT form, e_i small integers) are
inputs, as for encryption.

Parity: pinned (tests/test_oracle_keyswitch.py) by the evaluation homomorphism
sigma_g(a)(w) = a(w^g) at roots mod q, group laws of the automorphisms, slot rotation
and conjugation through the decoder, the index form of the automorphism on NTT values,
and decryption of switched and rotated ciphertexts within the error bound above.
"""
from __future__ import annotations

import numpy as np

from .linear import rescale
from .ntt import intt, ntt


def galois_element(r: int, log_n: int) -> int:
    """g = 5^r mod 2N for a slot rotation by r (left; negative r rotates right)."""
    n = 1 << log_n
    return pow(5, r % (n // 2), 2 * n)


def automorphism_int(a, g: int, log_n: int) -> np.ndarray:
    """sigma_g on signed integer coefficient vectors (..., N) (int64 or object)."""
    n = 1 << log_n
    a = np.asarray(a)
    if g % 2 == 0:
        raise ValueError("g must be odd")
    k = np.arange(n, dtype=np.int64)
    t = (k * (g % (2 * n))) % (2 * n)
    out = np.zeros_like(a)
    pos = t < n
    out[..., t[pos]] = a[..., k[pos]]
    out[..., t[~pos] - n] = -a[..., k[~pos]]
    return out


def automorphism_mod(a, g: int, q: int, log_n: int) -> np.ndarray:
    """sigma_g on coefficient residues (..., N) mod q."""
    a = np.asarray(a, dtype=np.uint64) % np.uint64(q)
    signed = automorphism_int(a.astype(np.int64), g, log_n)
    return np.mod(signed, q).astype(np.uint64)


def automorphism_ntt(b, g: int, q: int, psi: int, log_n: int) -> np.ndarray:
    """sigma_g on NTT-form residues (..., N): back to coefficients, permute, forward."""
    return ntt(automorphism_mod(intt(b, q, psi, log_n), g, q, log_n), q, psi, log_n)


def _res(v, q: int) -> np.ndarray:
    v = np.asarray(v)
    if v.dtype == object:
        return np.vectorize(lambda x: int(x) % q, otypes=[np.uint64])(v)
    return np.mod(v.astype(np.int64), q).astype(np.uint64)


def keygen_switch(s_from, s_to, a_ntt, e, qs_p, psis_p, log_n: int) -> np.ndarray:
    """Switching key from s_from to s_to (integer coefficient vectors (N,)).

    qs_p / psis_p: the ciphertext primes q_0 .. q_{L-1} followed by the special prime P.
    a_ntt: uniform residues (L, L+1, N) in NTT form; e: integers (L, N).
    Returns ksk (L, 2, L+1, N): ksk[i, 0] = -a_i s_to + e_i + P g_i s_from, ksk[i, 1] = a_i.
    """
    L = len(qs_p) - 1
    P = qs_p[-1]
    n = 1 << log_n
    ksk = np.empty((L, 2, L + 1, n), dtype=np.uint64)
    for j, (p, ps) in enumerate(zip(qs_p, psis_p)):
        pp = np.uint64(p)
        st_hat = ntt(_res(s_to, p), p, ps, log_n)
        sf_hat = ntt(_res(s_from, p), p, ps, log_n)
        for i in range(L):
            a = np.asarray(a_ntt[i, j], dtype=np.uint64) % pp
            b = (ntt(_res(e[i], p), p, ps, log_n) + pp - (a * st_hat) % pp) % pp
            if j == i:                                     # P * g_i is P mod q_i, 0 mod the rest
                b = (b + (np.uint64(P % p) * sf_hat) % pp) % pp
            ksk[i, 0, j] = b
            ksk[i, 1, j] = a
    return ksk


def rotation_key(s, r: int, a_ntt, e, qs_p, psis_p, log_n: int) -> np.ndarray:
    """Key switching sigma_g(s) -> s for g = 5^r (rotation by r slots)."""
    g = galois_element(r, log_n)
    return keygen_switch(automorphism_int(np.asarray(s, dtype=np.int64), g, log_n), s, a_ntt, e,
                         qs_p, psis_p, log_n)


def decompose(c, qs, psis, log_n: int):
    """Digits of an NTT-form polynomial c (L, N): the centred coefficients of each limb."""
    out = []
    for i in range(c.shape[0]):
        q = qs[i]
        v = intt(np.asarray(c[i], dtype=np.uint64), q, psis[i], log_n).astype(np.int64)
        out.append(np.where(v > q // 2, v - q, v))
    return out


def keyswitch_ext(c, ksk, qs_p, psis_p, log_n: int) -> np.ndarray:
    """The key-switching inner product of the NTT-form polynomial c (L, N) over
    q_0 .. q_{L-1} with ksk (L, 2, L+1, N), before the division by P: returns
    (a0, a1) (2, L+1, N) over q_0 .. q_{L-1}, P with a0 + a1 s_to = P c s_from +
    sum_i d_i e_i (mod Q P).
    """
    L = c.shape[0]
    if L != len(qs_p) - 1:
        raise ValueError("key switching runs with every ciphertext limb and the special prime last")
    n = 1 << log_n
    digits = decompose(c, qs_p, psis_p, log_n)
    acc = np.zeros((1, 2, L + 1, n), dtype=np.uint64)
    for j, (p, ps) in enumerate(zip(qs_p, psis_p)):
        pp = np.uint64(p)
        for i in range(L):
            d_hat = ntt(_res(digits[i], p), p, ps, log_n)
            for k in range(2):
                acc[0, k, j] = (acc[0, k, j] + (d_hat * (np.asarray(ksk[i, k, j], dtype=np.uint64) % pp)) % pp) % pp
    return acc[0]


def keyswitch(c, ksk, qs_p, psis_p, log_n: int) -> np.ndarray:
    """Switch the NTT-form polynomial c (L, N) over q_0 .. q_{L-1} with ksk (L, 2, L+1, N).

    Returns (u0, u1) (2, L, N) with u0 + u1 s_to = c s_from + small error.
    """
    ext = keyswitch_ext(c, ksk, qs_p, psis_p, log_n)
    return rescale(ext[None], qs_p, psis_p, log_n)[0]     # division by P: drop the last prime


def automorphism_ct(ct, g: int, qs, psis, log_n: int) -> np.ndarray:
    """sigma_g on both components of an NTT-form ciphertext (2, L, N)."""
    L = ct.shape[1]
    sig = np.empty((2, L, 1 << log_n), dtype=np.uint64)
    for c in range(2):
        for l in range(L):
            sig[c, l] = automorphism_ntt(ct[c, l], g, qs[l], psis[l], log_n)
    return sig


def rotate(ct, r: int, ksk, qs_p, psis_p, log_n: int) -> np.ndarray:
    """Rotate the slots of an NTT-form ciphertext (2, L, N) left by r, with ksk = rotation_key(s, r)."""
    L = ct.shape[1]
    sig = automorphism_ct(ct, galois_element(r, log_n), qs_p, psis_p, log_n)
    u = keyswitch(sig[1], ksk, qs_p, psis_p, log_n)
    q = np.array(qs_p[:L], dtype=np.uint64)[:, None]
    return np.stack([(sig[0] + u[0]) % q, u[1]])
