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
