"""Pins for oracle/linear.py: the modular MAC and rescaling."""
import numpy as np
import pytest

from oracle import encode, linear, params, poly
from oracle.ntt import intt, ntt
from workloads import gen


def _ctx(log_n, L):
    qs = params.moduli(max(log_n, 10), L)
    return qs, [params.psi(q, log_n) for q in qs]


def _rand_ct(rng, count, qs, n):
    return np.stack([np.stack([np.stack([rng.integers(0, q, n, dtype=np.uint64) for q in qs])
                               for _ in range(2)]) for _ in range(count)])


def test_mac_identity_and_one_hot():
    qs, _ = _ctx(10, 3)
    rng = np.random.default_rng(1)
    ct = _rand_ct(rng, 5, qs, 64)
    eye = np.zeros((5, 5, 3), dtype=np.uint64)
    for i in range(5):
        eye[i, i, :] = 1
    assert np.array_equal(linear.mac_scalar(eye, ct, qs), ct)
    hot = np.zeros((2, 5, 3), dtype=np.uint64)
    hot[0, 3, :] = 1
    hot[1, 1, :] = [q - 1 for q in qs]            # weight -1
    out = linear.mac_scalar(hot, ct, qs)
    assert np.array_equal(out[0], ct[3])
    for l, q in enumerate(qs):
        assert np.array_equal(out[1, :, l], (np.uint64(q) - ct[1, :, l]) % np.uint64(q))


def test_mac_brute_force_and_crt_consistency():
    qs, _ = _ctx(10, 3)
    Q = qs[0] * qs[1] * qs[2]
    rng = np.random.default_rng(2)
    d_out, d_in, n = 3, 4, 8
    w = rng.normal(0, 0.02, (d_out, d_in))
    delta = 2.0 ** 26
    w_signed = [[int(np.rint(x * delta)) for x in row] for row in w]
    w_enc = encode.encode_scalar(w, delta, qs)
    ct = _rand_ct(rng, d_in, qs, n)
    out = linear.mac_scalar(w_enc, ct, qs)
    for j in range(d_out):
        for c in range(2):
            for k in range(n):
                for l, q in enumerate(qs):       # brute force with Python ints
                    assert int(out[j, c, l, k]) == sum(int(w_enc[j, i, l]) * int(ct[i, c, l, k]) for i in range(d_in)) % q
                # CRT consistency: the limbs together are the product over Z_Q with signed weights
                lifted_out = params.crt_lift([[int(out[j, c, l, k])] for l in range(3)], qs)[0]
                lifted_in = [params.crt_lift([[int(ct[i, c, l, k])] for l in range(3)], qs)[0] for i in range(d_in)]
                assert lifted_out == sum(w_signed[j][i] * lifted_in[i] for i in range(d_in)) % Q


def test_mac_linearity():
    qs, _ = _ctx(10, 2)
    rng = np.random.default_rng(3)
    w = np.stack([np.stack([rng.integers(0, q, 6, dtype=np.uint64) for q in qs], -1) for _ in range(4)])
    a, b = _rand_ct(rng, 6, qs, 32), _rand_ct(rng, 6, qs, 32)
    q = np.array(qs, dtype=np.uint64)[:, None]
    s = (a + b) % q
    lhs = linear.mac_scalar(w, s, qs)
    rhs = (linear.mac_scalar(w, a, qs) + linear.mac_scalar(w, b, qs)) % q
    assert np.array_equal(lhs, rhs)


def test_mac_poly_constant_weights_equal_scalar_path():
    qs, psis = _ctx(10, 3)
    rng = np.random.default_rng(4)
    d_out, d_in, delta = 3, 5, 2.0 ** 30
    w = rng.normal(0, 0.02, (d_out, d_in))
    w_enc = encode.encode_scalar(w, delta, qs)
    pt = encode.encode_poly(np.repeat(w[..., None], 512, axis=-1), delta, qs, psis, 10)
    ct = _rand_ct(rng, d_in, qs, 1024)
    assert np.array_equal(linear.mac_poly(pt, ct, qs), linear.mac_scalar(w_enc, ct, qs))


def test_mac_poly_is_negacyclic_product_in_coefficients():
    log_n, n = 4, 16
    qs, psis = _ctx(log_n, 2)
    rng = np.random.default_rng(5)
    pt = np.stack([np.stack([np.stack([rng.integers(0, q, n, dtype=np.uint64) for q in qs]) for _ in range(3)])
                   for _ in range(2)])                                    # (2, 3, L, n)
    ct = _rand_ct(rng, 3, qs, n)
    out = linear.mac_poly(pt, ct, qs)
    for j in range(2):
        for c in range(2):
            for l, (q, ps) in enumerate(zip(qs, psis)):
                acc = np.zeros(n, dtype=np.uint64)
                for i in range(3):
                    prod = poly.negacyclic_mul(intt(pt[j, i, l], q, ps, log_n), intt(ct[i, c, l], q, ps, log_n), q)
                    acc = (acc + prod) % np.uint64(q)
                assert np.array_equal(intt(out[j, c, l], q, ps, log_n), acc)


@pytest.mark.parametrize("log_n,L", [(4, 2), (4, 4), (10, 3)])
def test_rescale_special_case_exact_multiple(log_n, L):
    n = 1 << log_n
    qs, psis = _ctx(log_n, L)
    rng = np.random.default_rng(6 + L)
    Q = 1
    for q in qs:
        Q *= q
    ql = qs[-1]
    # C = q_{L-1} * D + r with |r| < q_{L-1}/2 (r = 0 for the first component): rescale gives D
    D = [int(x) for x in rng.integers(-2**40, 2**40, (2, n)).ravel()]
    R = [0] * n + [int(x) for x in rng.integers(-(ql // 2), ql // 2, n)]
    ct = np.empty((1, 2, L, n), dtype=np.uint64)
    for c in range(2):
        for l, (q, ps) in enumerate(zip(qs, psis)):
            coef = np.array([(ql * D[c * n + k] + R[c * n + k]) % q for k in range(n)], dtype=np.uint64)
            ct[0, c, l] = ntt(coef, q, ps, log_n)
    out = linear.rescale(ct, qs, psis, log_n)
    for c in range(2):
        for l, (q, ps) in enumerate(zip(qs[:-1], psis[:-1])):
            got = intt(out[0, c, l], q, ps, log_n)
            assert got.tolist() == [D[c * n + k] % q for k in range(n)]


@pytest.mark.parametrize("log_n,L", [(4, 2), (5, 3), (10, 4)])
def test_rescale_ntt_formula_equals_definition(log_n, L):
    n = 1 << log_n
    qs, psis = _ctx(log_n, L)
    rng = np.random.default_rng(7 + log_n)
    ct = _rand_ct(rng, 2, qs, n)
    assert np.array_equal(linear.rescale_ntt_formula(ct, qs, psis, log_n), linear.rescale(ct, qs, psis, log_n))


def test_rescale_constant_polynomial():
    log_n, n, L = 10, 1024, 3
    qs, psis = _ctx(log_n, L)
    val = 123456789 * qs[-1] + 17                       # rounds to 123456789
    ct = np.empty((1, 2, L, n), dtype=np.uint64)
    for l, q in enumerate(qs):
        ct[0, :, l, :] = val % q                        # NTT of a constant is that constant
    out = linear.rescale(ct, qs, psis, log_n)
    for l, q in enumerate(qs[:-1]):
        assert np.all(out[0, :, l] == 123456789 % q)


def test_sample_rows_generator():
    rows = gen.sample_rows(gen.streams(2)["sample"], 768)
    assert rows[0] == 0 and rows[-1] == 767 and len(set(rows)) == 16
    assert gen.sample_rows(gen.streams(1)["sample"], 16) == list(range(16))
