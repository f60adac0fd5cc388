"""The ct x pt linear layer and rescaling (CPU oracle; test infrastructure only).

The paper evaluates regular projection and FFN layers homomorphically on the
accelerator, with public plaintext weights and encrypted activations (sections
3.2 and 3.5; FHE_Linear in the PD-split serving algorithm, Algorithm 3).  The
packing used here is one ciphertext per input feature, with scalar weights
(one constant per (output, input) pair) or full-polynomial weights (one slot
vector per pair); the paper's own rotation-based packing is not this one.  In
both cases output ciphertext j is

    out_j = sum_i pt_ji * ct_i          in R_Q,

which in NTT form and per RNS limb l is the slot-wise modular sum

    out[j, c, l, k] = sum_i w[j, i, l] * ct[i, c, l, k]          mod q_l   (scalar)
    out[j, c, l, k] = sum_i pt[j, i, l, k] * ct[i, c, l, k]      mod q_l   (full poly)

computed here by direct modular sums (each product reduced before adding).

Rescaling (section 2.1: divide by the last prime, drop one level) is given by
its plain definition: lift the coefficients by CRT to C in [0, Q), take
round(C / q_{L-1}) (q_{L-1} is odd, so there are no ties) and reduce it mod the
remaining primes.  ``rescale_ntt_formula`` is the per-limb NTT-domain route
the accelerator takes; the tests pin it to the definition.

Parity: pinned (tests/test_oracle_linear.py) by identity and one-hot weights,
linearity, CRT consistency with signed integer weights over Z_Q, brute force
on tiny shapes, and the rescale special cases C = q_{L-1} * D.
"""
from __future__ import annotations

import numpy as np

from .ntt import intt, ntt


def _q_col(qs, ndim_tail: int) -> np.ndarray:
    """Moduli as a uint64 array broadcastable over (..., L) + (1,)*ndim_tail."""
    return np.array(qs, dtype=np.uint64).reshape((len(qs),) + (1,) * ndim_tail)


def mac_scalar(w_enc, ct, qs, rows=None) -> np.ndarray:
    """w_enc (d_out, d_in, L) residues; ct (d_in, 2, L, N) residues -> (len(rows), 2, L, N)."""
    w_enc = np.asarray(w_enc, dtype=np.uint64)
    ct = np.asarray(ct)
    d_out, d_in, L = w_enc.shape
    rows = range(d_out) if rows is None else rows
    q = _q_col(qs[:L], 1)                                     # (L, 1)
    out = np.empty((len(rows), 2, L, ct.shape[-1]), dtype=np.uint64)
    for r, j in enumerate(rows):
        acc = np.zeros((2, L, ct.shape[-1]), dtype=np.uint64)
        for i in range(d_in):
            prod = (w_enc[j, i][:, None] * ct[i].astype(np.uint64)) % q
            acc = (acc + prod) % q
        out[r] = acc
    return out


def mac_poly(pt, ct, qs, rows=None) -> np.ndarray:
    """pt (d_out, d_in, L, N) NTT-form residues; ct (d_in, 2, L, N) -> (len(rows), 2, L, N)."""
    pt = np.asarray(pt)
    ct = np.asarray(ct)
    d_out, d_in, L, n = pt.shape
    rows = range(d_out) if rows is None else rows
    q = _q_col(qs[:L], 1)
    out = np.empty((len(rows), 2, L, n), dtype=np.uint64)
    for r, j in enumerate(rows):
        acc = np.zeros((2, L, n), dtype=np.uint64)
        for i in range(d_in):
            prod = (pt[j, i].astype(np.uint64)[None] * ct[i].astype(np.uint64)) % q
            acc = (acc + prod) % q
        out[r] = acc
    return out


def _crt_constants(qs):
    Q = 1
    for q in qs:
        Q *= q
    return Q, [(Q // q) * pow(Q // q, -1, q) for q in qs]


def rescale(ct, qs, psis, log_n: int) -> np.ndarray:
    """Rescale NTT-form ciphertexts (count, 2, L, N) -> (count, 2, L-1, N) by the CRT definition."""
    ct = np.asarray(ct, dtype=np.uint64)
    count, _, L, n = ct.shape
    Q, coef = _crt_constants(qs[:L])
    ql = qs[L - 1]
    out = np.empty((count, 2, L - 1, n), dtype=np.uint64)
    for b in range(count):
        for c in range(2):
            C = np.zeros(n, dtype=object)
            for l in range(L):
                res = intt(ct[b, c, l], qs[l], psis[l], log_n)
                C = C + res.astype(object) * coef[l]
            C = C % Q                                          # C in [0, Q)
            D = (2 * C + ql) // (2 * ql)                       # round(C / q_{L-1}), no ties (q odd)
            for l in range(L - 1):
                d_l = np.array([int(x) % qs[l] for x in D], dtype=np.uint64)
                out[b, c, l] = ntt(d_l, qs[l], psis[l], log_n)
    return out


def rescale_ntt_formula(ct, qs, psis, log_n: int) -> np.ndarray:
    """Per-limb NTT-domain route to the same result:

    r = centred INTT_{L-1}(c_{L-1});  out_l = (c_l - NTT_l(r mod q_l)) * q_{L-1}^-1  mod q_l.
    """
    ct = np.asarray(ct, dtype=np.uint64)
    count, _, L, n = ct.shape
    ql = qs[L - 1]
    out = np.empty((count, 2, L - 1, n), dtype=np.uint64)
    for b in range(count):
        for c in range(2):
            r = intt(ct[b, c, L - 1], ql, psis[L - 1], log_n).astype(np.int64)
            r = np.where(r > ql // 2, r - ql, r)              # centred in (-q/2, q/2)
            for l in range(L - 1):
                q = qs[l]
                qq = np.uint64(q)
                r_hat = ntt(np.mod(r, q).astype(np.uint64), q, psis[l], log_n)
                inv = np.uint64(pow(ql, -1, q))
                out[b, c, l] = ((ct[b, c, l] + qq - r_hat) % qq * inv) % qq
    return out
