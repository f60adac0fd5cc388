"""Symmetric-key RLWE encryption / decryption over the RNS chain (CPU oracle; test infrastructure only).

The paper's accelerator only ever sees ciphertexts; encryption and decryption
run in the trusted CPU domain on either side of each accelerator linear call
(sections 3.2 and 4.2; the decrypt-then-encrypt refresh ct' = Enc(Dec(ct)) of
section 3.2).  Those steps are not on the accelerator path; they exist here to
make valid encrypted inputs and to check outputs by decryption.  The paper
writes public-key encryption; the ct x pt path is indifferent to how the RLWE
ciphertext was made, so the symmetric form is used (reading):

    ct = (c0, c1) = (-a*s + m + e, a)            per limb, in NTT form,

with s ternary, e a rounded Gaussian (sigma = 3.2, |e| <= 19) and a uniform.
Because the NTT is a bijection of Z_q^N, drawing a uniformly in NTT form is
the same distribution as drawing it in coefficient form; the random draws are
inputs (they come from the seeded generators, never from here).

Decryption is m + e' = INTT(c0 + c1 (.) NTT(s)), lifted by CRT to centred
integers.

Decrypt-then-encrypt refresh (the DtE equation of section 3.2, ct' =
Enc(Dec(ct))): the plaintext polynomial m + e' of a ciphertext at any level is
recovered exactly from its first two limbs by CRT to centred integers (valid
while |m + e'| < q_0 q_1 / 2), then encrypted afresh, with new randomness,
under a chosen number of limbs (reading: the refresh acts on the integer
plaintext polynomial; decoding to slots and re-encoding would round it again).

Parity: pinned (tests/test_oracle_rlwe.py) against the coefficient-domain
definition -a*s + m + e with the schoolbook product at small N, by round
trips, and (refresh) against a direct fresh encryption of the known m + e.
"""
from __future__ import annotations

import numpy as np

from .ntt import intt, ntt
from .params import centre, crt_lift


def _residues(v, q: int) -> np.ndarray:
    """Integer vector(s) (any shape, Python ints or int64) -> residues mod q (uint64)."""
    v = np.asarray(v)
    if v.dtype == object:
        return np.vectorize(lambda x: int(x) % q, otypes=[np.uint64])(v)
    return np.mod(v.astype(np.int64), q).astype(np.uint64)


def encrypt(m, s, a_ntt, e, qs, psis, log_n: int) -> np.ndarray:
    """m, e: integer coefficient vectors (N,) or batches (B, N); s: secret (N,);
    a_ntt: uniform residues (L, N) or (B, L, N).

    Returns the ciphertext(s) (2, L, N) or (B, 2, L, N) in NTT form.
    """
    m = np.asarray(m, dtype=object if isinstance(m, list) else None)
    single = m.ndim == 1
    m2 = m[None] if single else m
    e2 = np.asarray(e)[None] if single else np.asarray(e)
    a2 = np.asarray(a_ntt)[None] if single else np.asarray(a_ntt)
    B, L, n = m2.shape[0], len(qs), 1 << log_n
    ct = np.empty((B, 2, L, n), dtype=np.uint64)
    for l, (q, ps) in enumerate(zip(qs, psis)):
        qq = np.uint64(q)
        s_hat = ntt(_residues(s, q), q, ps, log_n)
        me_hat = ntt((_residues(m2, q) + _residues(e2, q)) % qq, q, ps, log_n)     # (B, N)
        a = a2[:, l].astype(np.uint64) % qq
        ct[:, 1, l] = a
        ct[:, 0, l] = (me_hat + qq - (a * s_hat) % qq) % qq
    return ct[0] if single else ct


def decrypt_residues(ct, s, qs, psis, log_n: int) -> np.ndarray:
    """Coefficient residues (L', N) of c0 + c1*s for a ciphertext (2, L', N) in NTT form."""
    L = ct.shape[1]
    out = np.empty((L, 1 << log_n), dtype=np.uint64)
    for l in range(L):
        q, ps = qs[l], psis[l]
        qq = np.uint64(q)
        s_hat = ntt(_residues(s, q), q, ps, log_n)
        v = (np.asarray(ct[0, l], dtype=np.uint64) + (np.asarray(ct[1, l], dtype=np.uint64) * s_hat) % qq) % qq
        out[l] = intt(v, q, ps, log_n)
    return out


def decrypt(ct, s, qs, psis, log_n: int) -> list[int]:
    """Centred integer coefficients of the decrypted plaintext (CRT over all limbs of ct)."""
    L = ct.shape[1]
    res = decrypt_residues(ct, s, qs, psis, log_n)
    Q = 1
    for q in qs[:L]:
        Q *= q
    return [centre(c, Q) for c in crt_lift(res, qs[:L])]


def refresh(ct, s, a_ntt, e, qs, psis, log_n: int, limbs_out: int) -> np.ndarray:
    """Decrypt-then-encrypt (section 3.2): ct (B, 2, L_in, N) in NTT form, L_in >= 2.

    Decrypts with limbs 0 and 1 (CRT over q_0 q_1, centred), then returns
    encrypt(m + e', s, a_ntt, e) under q_0 .. q_{limbs_out-1}: shape
    (B, 2, limbs_out, N).  a_ntt (B, limbs_out, N) and e (B, N) are the fresh
    randomness (inputs).
    """
    ct = np.asarray(ct)
    B = ct.shape[0]
    Q2 = qs[0] * qs[1]
    out = np.empty((B, 2, limbs_out, 1 << log_n), dtype=np.uint64)
    for b in range(B):
        res = decrypt_residues(ct[b, :, :2], s, qs[:2], psis[:2], log_n)
        m = [centre(c, Q2) for c in crt_lift(res, qs[:2])]
        out[b] = encrypt(m, s, np.asarray(a_ntt)[b], np.asarray(e)[b], qs[:limbs_out], psis[:limbs_out], log_n)
    return out
