"""Pins for oracle/rlwe.py: the NTT-form encryption equals the coefficient-domain
definition c0 = -a*s + m + e (schoolbook product), and decryption inverts it."""
import numpy as np
import pytest

from oracle import params, poly, rlwe
from oracle.ntt import intt
from workloads import gen


@pytest.mark.parametrize("log_n,L", [(4, 2), (6, 3)])
def test_encrypt_matches_coefficient_definition(log_n, L):
    n = 1 << log_n
    qs = params.moduli(10, L)
    psis = [params.psi(q, log_n) for q in qs]
    st = gen.streams(99, log_n)
    s = gen.ternary_secret(st["secret"], n)
    e = gen.gaussian_error(st["error"], n)
    m = st["activations"].integers(-2**40, 2**40, n)
    a_ntt = np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs])
    ct = rlwe.encrypt(m, s, a_ntt, e, qs, psis, log_n)
    for l, (q, ps) in enumerate(zip(qs, psis)):
        a = intt(ct[1, l], q, ps, log_n)
        c0 = intt(ct[0, l], q, ps, log_n)
        s_res = np.mod(s, q).astype(np.uint64)
        as_ = poly.negacyclic_mul(a, s_res, q)
        want = (np.mod(m + e, q).astype(np.uint64) + np.uint64(q) - as_) % np.uint64(q)
        assert np.array_equal(c0, want)


def test_decrypt_round_trip():
    log_n, L, n = 10, 3, 1024
    qs = params.moduli(10, L)
    psis = [params.psi(q, log_n) for q in qs]
    st = gen.streams(98)
    s = gen.ternary_secret(st["secret"], n)
    e = gen.gaussian_error(st["error"], n)
    assert np.abs(e).max() <= 19
    m = st["activations"].integers(-2**50, 2**50, n)
    a_ntt = np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs])
    ct = rlwe.encrypt(m, s, a_ntt, e, qs, psis, log_n)
    assert rlwe.decrypt(ct, s, qs, psis, log_n) == [int(x) + int(y) for x, y in zip(m, e)]
    # two limbs are enough while |m + e| < q0 q1 / 2
    assert rlwe.decrypt(ct[:, :2], s, qs, psis, log_n) == [int(x) + int(y) for x, y in zip(m, e)]


def _keys(log_n, L, seed):
    n = 1 << log_n
    qs = params.moduli(log_n if log_n >= 10 else 10, L)
    psis = [params.psi(q, log_n) for q in qs]
    st = gen.streams(seed, log_n)
    s = gen.ternary_secret(st["secret"], n)
    return n, qs, psis, s, st


@pytest.mark.parametrize("log_n,L_in,L_out", [(6, 2, 4), (6, 3, 3), (10, 3, 4)])
def test_refresh_equals_fresh_encryption_of_the_decrypted_polynomial(log_n, L_in, L_out):
    """A ciphertext of m with error e, refreshed with fresh (a', e''), is bit for
    bit the fresh encryption of the integer polynomial m + e under (a', e'')."""
    n, qs, psis, s, st = _keys(log_n, 4, 91)
    B = 2
    m = st["activations"].integers(-2**45, 2**45, (B, n))
    e = gen.gaussian_error(st["error"], (B, n))
    a = np.stack([np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs[:L_in]]) for _ in range(B)])
    ct = rlwe.encrypt(m, s, a, e, qs[:L_in], psis[:L_in], log_n)
    a2 = np.stack([np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs[:L_out]]) for _ in range(B)])
    e2 = gen.gaussian_error(st["error"], (B, n))
    got = rlwe.refresh(ct, s, a2, e2, qs, psis, log_n, L_out)
    want = rlwe.encrypt(m + e, s, a2, e2, qs[:L_out], psis[:L_out], log_n)
    assert got.shape == (B, 2, L_out, n)
    assert np.array_equal(got, want)
    # and it decrypts (over all L_out limbs) to m + e + e''
    for b in range(B):
        assert rlwe.decrypt(got[b], s, qs[:L_out], psis[:L_out], log_n) == [int(x) for x in m[b] + e[b] + e2[b]]


def test_refresh_of_a_rescaled_ciphertext_restores_the_level():
    """After a rescale (2 limbs left) the refresh brings the ciphertext back to 4
    limbs and the rounded plaintext survives: decrypt(refresh(rescale(ct))) =
    round(decrypt(ct) / q_last) + e''."""
    from oracle import linear
    log_n, L = 6, 3
    n, qs, psis, s, st = _keys(log_n, 4, 92)
    m = st["activations"].integers(-2**50, 2**50, (1, n))
    e = gen.gaussian_error(st["error"], (1, n))
    a = np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs[:L]])[None]
    ct = rlwe.encrypt(m, s, a, e, qs[:L], psis[:L], log_n)
    r = linear.rescale(ct, qs[:L], psis[:L], log_n)            # 2 limbs
    dec_r = rlwe.decrypt(r[0], s, qs[:L - 1], psis[:L - 1], log_n)
    a2 = np.stack([st["residues"].integers(0, q, n, dtype=np.uint64) for q in qs])[None]
    e2 = gen.gaussian_error(st["error"], (1, n))
    f = rlwe.refresh(r, s, a2, e2, qs, psis, log_n, 4)
    assert rlwe.decrypt(f[0], s, qs, psis, log_n) == [x + int(y) for x, y in zip(dec_r, e2[0])]
    # the rescaled plaintext is m + e divided by q_last, up to the rescale's rounding error
    want = (m[0] + e[0]) / qs[L - 1]
    assert np.max(np.abs(np.array(dec_r, dtype=np.float64) - want)) < n
