"""Pins for oracle/encode.py.

The direct O(N^2) canonical-embedding sums are checked against numpy's FFT
evaluation of the polynomial at the 2N-th roots, against the constant-slot
closed form and Parseval's identity, and by the decode(encode(z)) rounding bound.
"""
import numpy as np
import pytest

from oracle import encode as E
from oracle import params
from oracle.ntt import ntt


def _eval_at_roots_fft(m, log_n):
    """m(omega^(2u+1)) for u < N, omega = exp(i pi / N), via numpy's inverse FFT."""
    n = 1 << log_n
    k = np.arange(n)
    twisted = np.asarray(m, dtype=np.complex128) * np.exp(1j * np.pi * k / n)
    return np.fft.ifft(twisted) * n          # sum_k (m_k w^k) e^{2 pi i u k / N}


@pytest.mark.parametrize("log_n", [4, 6, 10])
def test_slot_exponents_cover_half_the_odd_residues(log_n):
    n = 1 << log_n
    e = E.slot_exponents(log_n)
    s = set(int(x) for x in e) | set(int((2 * n - x) % (2 * n)) for x in e)
    assert s == set(range(1, 2 * n, 2))


@pytest.mark.parametrize("log_n", [4, 6, 10])
def test_encoded_polynomial_takes_the_slot_values_at_the_roots(log_n):
    n = 1 << log_n
    rng = np.random.default_rng(log_n)
    z = rng.uniform(-1, 1, n // 2) + 1j * rng.uniform(-1, 1, n // 2)
    m = E.encode_coeffs(z, log_n)
    vals = _eval_at_roots_fft(m, log_n)
    e = E.slot_exponents(log_n)
    assert np.allclose(vals[(e - 1) // 2], z, atol=1e-11)
    assert np.allclose(vals[(2 * n - e - 1) // 2], np.conj(z), atol=1e-11)


@pytest.mark.parametrize("log_n", [4, 10])
def test_decode_matches_fft_evaluation(log_n):
    n = 1 << log_n
    rng = np.random.default_rng(40 + log_n)
    m = rng.integers(-2**40, 2**40, n)
    delta = 2.0 ** 30
    got = E.decode(m.tolist(), delta, log_n)
    e = E.slot_exponents(log_n)
    ref = _eval_at_roots_fft(m.astype(np.float64), log_n)[(e - 1) // 2] / delta
    assert np.allclose(got, ref, rtol=0, atol=1e-9 * np.abs(ref).max())


def test_constant_slots_encode_to_the_constant_polynomial():
    log_n, delta = 10, 2.0 ** 25
    for c in (0.75, -0.3125, 0.01):
        m = E.encode_coeffs(np.full(512, c), log_n)
        assert abs(m[0] - c) < 1e-13 and np.max(np.abs(m[1:])) < 1e-13
        p = E.round_coeffs(m, delta)
        assert p[0] == int(np.rint(c * delta)) and not np.any(p[1:])
    qs = params.moduli(10, 2)
    psis = [params.psi(q, 10) for q in qs]
    pt = E.encode_poly(np.full(512, -0.3125), delta, qs, psis, 10)
    sc = E.encode_scalar(np.array(-0.3125), delta, qs)
    for l in range(2):
        assert np.all(pt[l] == sc[l])            # NTT of a constant is constant


@pytest.mark.parametrize("log_n", [6, 10])
def test_parseval(log_n):
    n = 1 << log_n
    rng = np.random.default_rng(9)
    z = rng.normal(size=n // 2) + 1j * rng.normal(size=n // 2)
    m = E.encode_coeffs(z, log_n)
    assert np.isclose(np.sum(np.abs(z) ** 2), (n / 2) * np.sum(m ** 2), rtol=1e-12)


def test_decode_encode_within_rounding_bound():
    log_n, n, delta = 10, 1024, 2.0 ** 25
    rng = np.random.default_rng(3)
    z = rng.uniform(-1, 1, n // 2)
    p = E.round_coeffs(E.encode_coeffs(z, log_n), delta)
    err = E.decode(p.tolist(), delta, log_n) - z
    sd = np.sqrt(n / 12) / delta                 # per-slot std of the rounding error (complex)
    assert np.max(np.abs(err)) < 6 * sd
    assert np.sqrt(np.mean(np.abs(err) ** 2)) < 1.5 * sd


def test_scalar_encode_rounds_half_to_even_and_wraps_negatives():
    qs = params.moduli(10, 2)
    delta = 2.0 ** 4
    w = np.array([1.5, 2.5, -1.5, -2.5, 0.0, 3.0]) / delta   # w*Delta exact
    r = E.encode_scalar(w, delta, qs)
    for l, q in enumerate(qs):
        assert r[:, l].tolist() == [2, 2, q - 2, q - 2, 0, 3]


def test_encode_poly_is_ntt_of_rounded_coefficients():
    log_n, delta = 10, 2.0 ** 30
    qs = params.moduli(10, 3)
    psis = [params.psi(q, 10) for q in qs]
    rng = np.random.default_rng(21)
    z = rng.normal(0, 0.02, 512)
    pt = E.encode_poly(z, delta, qs, psis, log_n)
    p = E.round_coeffs(E.encode_coeffs(z, log_n), delta)
    for l, q in enumerate(qs):
        assert np.array_equal(pt[l], ntt(np.mod(p, q).astype(np.uint64), q, psis[l], log_n))


def test_slot_order_is_powers_of_five():
    """Slot j sits at exp(i pi 5^j / N): evaluate the encoded polynomial there directly."""
    log_n = 6
    n = 1 << log_n
    rng = np.random.default_rng(12)
    z = rng.uniform(-1, 1, n // 2) + 1j * rng.uniform(-1, 1, n // 2)
    m = E.encode_coeffs(z, log_n)
    for j in (0, 1, 2, 3, 7, n // 2 - 1):
        point = np.exp(1j * np.pi * pow(5, j, 2 * n) / n)
        assert abs(np.polyval(m[::-1], point) - z[j]) < 1e-11


def test_selected_coefficients_match_the_full_sum():
    """encode_coeffs(z, log_n, ks) gives column ks of the full inverse embedding
    (the full form is pinned above), including k = 0, N/2 and N - 1."""
    log_n = 8
    n = 1 << log_n
    z = np.random.default_rng(5).normal(0, 0.02, (2, n // 2))
    ks = np.array([0, 1, 7, n // 4, n // 2, n // 2 + 3, n - 1])
    assert np.array_equal(E.encode_coeffs(z, log_n, ks), E.encode_coeffs(z, log_n)[:, ks])
