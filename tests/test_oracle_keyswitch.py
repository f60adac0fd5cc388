"""Pins for oracle/keyswitch.py and oracle/bsgs.py: automorphisms against the
evaluation homomorphism and the slot decoder, key switching and rotation by
decryption within the stated error bound, and the BSGS product against numpy's
W @ x."""
import numpy as np
import pytest

from oracle import bsgs, params, rlwe
from oracle import encode as OE
from oracle import keyswitch as KS
from oracle.ntt import intt, ntt
from workloads import gen


def _chain(log_n, L, seed):
    """L ciphertext primes and the special prime last (the next prime of the chain)."""
    n = 1 << log_n
    qs_p = list(params.moduli(max(log_n, 10), L + 1))
    psis_p = [params.psi(q, log_n) for q in qs_p]
    st = gen.streams(seed, log_n)
    s = gen.ternary_secret(st["secret"], n)
    return n, qs_p, psis_p, s, st


def _key(st, s_from, s_to, qs_p, psis_p, log_n):
    L, n = len(qs_p) - 1, 1 << log_n
    a = gen.uniform_residues(st["residues"], (L,), qs_p, n)            # (L, L+1, N)
    e = gen.gaussian_error(st["error"], (L, n))
    return KS.keygen_switch(s_from, s_to, a, e, qs_p, psis_p, log_n)


def _switch_bound(qs, n):
    P = qs[-1]
    return sum(n * (q // 2) * 19 for q in qs[:-1]) / P + n / 2 + 1


def _centred_lift(res, qs):
    Q = 1
    for q in qs:
        Q *= q
    return np.array([params.centre(c, Q) for c in params.crt_lift(res, qs)], dtype=object)


@pytest.mark.parametrize("g", [3, 5, 25, 127, 2 * 64 - 1])
def test_automorphism_is_the_evaluation_homomorphism(g):
    """sigma_g(a)(w) = a(w^g) at the roots w = psi^(2j+1), by Horner in Python integers."""
    log_n, n = 6, 64
    q = params.moduli(10, 1)[0]
    psi = params.psi(q, log_n)
    a = np.random.default_rng(g).integers(0, q, n).astype(np.uint64)
    b = KS.automorphism_mod(a, g, q, log_n)

    def ev(c, w):
        acc = 0
        for x in reversed([int(v) for v in c]):
            acc = (acc * w + x) % q
        return acc

    for j in (0, 1, 7, 31, 63):
        w = pow(psi, 2 * j + 1, q)
        assert ev(b, w) == ev(a, pow(w, g, q))


def test_automorphism_group_laws():
    log_n, n = 7, 128
    a = np.random.default_rng(1).integers(-1000, 1000, n)
    for g, h in ((5, 3), (25, 129), (255, 5)):
        gh = g * h % (2 * n)
        assert np.array_equal(KS.automorphism_int(KS.automorphism_int(a, h, log_n), g, log_n),
                              KS.automorphism_int(a, gh, log_n))
        g_inv = pow(g, -1, 2 * n)
        assert np.array_equal(KS.automorphism_int(KS.automorphism_int(a, g, log_n), g_inv, log_n), a)
    assert np.array_equal(KS.automorphism_int(a, 1, log_n), a)
    assert KS.galois_element(n // 2, log_n) == 1                   # 5 has order N/2 mod 2N
    assert KS.galois_element(-1, log_n) * 5 % (2 * n) == 1


def test_automorphism_on_ntt_values_is_an_index_permutation():
    """NTT(sigma_g a)[i] = NTT(a)[i'] with 2 brv(i') + 1 = (2 brv(i) + 1) g mod 2N."""
    log_n, n = 8, 256
    q = params.moduli(10, 1)[0]
    psi = params.psi(q, log_n)
    b = np.random.default_rng(2).integers(0, q, n).astype(np.uint64)
    for g in (5, 5 ** 7 % (2 * n), 2 * n - 1):
        got = KS.automorphism_ntt(b, g, q, psi, log_n)
        src = [params.brv((((2 * params.brv(i, log_n) + 1) * g) % (2 * n) - 1) // 2, log_n) for i in range(n)]
        assert np.array_equal(got, b[src])


@pytest.mark.parametrize("r", [1, 3, 17, -2])
def test_rotation_element_rotates_the_slots(r):
    log_n, n = 7, 128
    z = np.random.default_rng(r + 10).normal(0, 1, n // 2)
    m = OE.round_coeffs(OE.encode_coeffs(z, log_n), 2.0 ** 30)
    got = OE.decode(KS.automorphism_int(m, KS.galois_element(r, log_n), log_n), 2.0 ** 30, log_n)
    want = np.roll(OE.decode(m, 2.0 ** 30, log_n), -r)
    assert np.max(np.abs(got - want)) < 1e-9
    assert np.max(np.abs(got.real - np.roll(z, -r))) < 1e-6
    conj = OE.decode(KS.automorphism_int(m, 2 * n - 1, log_n), 2.0 ** 30, log_n)
    assert np.max(np.abs(conj - np.conj(OE.decode(m, 2.0 ** 30, log_n)))) < 1e-9


@pytest.mark.parametrize("log_n,L", [(6, 2), (8, 3), (10, 4)])
def test_keyswitch_decrypts_to_c_times_s_from(log_n, L):
    n, qs_p, psis_p, s, st = _chain(log_n, L, 40 + log_n)
    s2 = gen.ternary_secret(st["secret"], n)
    ksk = _key(st, s2, s, qs_p, psis_p, log_n)
    assert ksk.shape == (L, 2, L + 1, n)
    c = gen.uniform_residues(st["residues"], (), qs_p[:L], n)          # (L, N)
    u = KS.keyswitch(c, ksk, qs_p, psis_p, log_n)
    assert u.shape == (2, L, n)
    got, want = [], []
    for l in range(L):
        q, ps = qs_p[l], psis_p[l]
        qq = np.uint64(q)
        s_hat = ntt(np.mod(s, q).astype(np.uint64), q, ps, log_n)
        s2_hat = ntt(np.mod(s2, q).astype(np.uint64), q, ps, log_n)
        got.append(intt((u[0, l] + (u[1, l] * s_hat) % qq) % qq, q, ps, log_n))
        want.append(intt((c[l].astype(np.uint64) * s2_hat) % qq, q, ps, log_n))
    diff = _centred_lift(np.stack(got), qs_p[:L]) - _centred_lift(np.stack(want), qs_p[:L])
    err = max(abs(int(x)) for x in diff)
    assert err <= _switch_bound(qs_p, n)
    assert err > 0                                           # the key's error is really there


@pytest.mark.parametrize("log_n,L", [(6, 2), (8, 3)])
def test_keyswitch_ext_decrypts_to_p_times_c_times_s_from(log_n, L):
    """Before the division by P: a0 + a1 s_to = P c s_from + sum_i d_i e_i over all L + 1
    primes, |d_i| <= q_i / 2 and |e_i| <= 19 per coefficient, so the CRT-lifted difference
    stays within sum_i N (q_i/2) 19 (the same bound as after the division, times P)."""
    n, qs_p, psis_p, s, st = _chain(log_n, L, 50 + log_n)
    s2 = gen.ternary_secret(st["secret"], n)
    ksk = _key(st, s2, s, qs_p, psis_p, log_n)
    c = gen.uniform_residues(st["residues"], (), qs_p[:L], n)
    ext = KS.keyswitch_ext(c, ksk, qs_p, psis_p, log_n)
    assert ext.shape == (2, L + 1, n)
    P = qs_p[-1]
    got, want = [], []
    c_int = _centred_lift(np.stack([intt(c[l].astype(np.uint64), qs_p[l], psis_p[l], log_n) for l in range(L)]),
                          qs_p[:L])                                 # c as centred integers
    for l in range(L + 1):
        q, ps = qs_p[l], psis_p[l]
        qq = np.uint64(q)
        s_hat = ntt(np.mod(s, q).astype(np.uint64), q, ps, log_n)
        s2_hat = ntt(np.mod(s2, q).astype(np.uint64), q, ps, log_n)
        c_hat = ntt(np.array([int(x) % q for x in c_int], dtype=np.uint64), q, ps, log_n)
        got.append(intt((ext[0, l] + (ext[1, l] * s_hat) % qq) % qq, q, ps, log_n))
        want.append(intt((((c_hat * s2_hat) % qq) * np.uint64(P % q)) % qq, q, ps, log_n))
    diff = _centred_lift(np.stack(got), qs_p) - _centred_lift(np.stack(want), qs_p)
    err = max(abs(int(x)) for x in diff)
    assert err <= sum(n * (q // 2) * 19 for q in qs_p[:-1])
    assert err > n * 19                                       # the digits' error terms are really there


def test_keyswitch_with_a_wrong_key_fails_the_bound():
    """A key for a different s_from gives an error of the order of Q, far past the bound."""
    log_n, L = 6, 2
    n, qs_p, psis_p, s, st = _chain(log_n, L, 47)
    s2 = gen.ternary_secret(st["secret"], n)
    s3 = gen.ternary_secret(st["secret"], n)
    ksk = _key(st, s3, s, qs_p, psis_p, log_n)
    c = gen.uniform_residues(st["residues"], (), qs_p[:L], n)
    u = KS.keyswitch(c, ksk, qs_p, psis_p, log_n)
    got, want = [], []
    for l in range(L):
        q, ps = qs_p[l], psis_p[l]
        qq = np.uint64(q)
        s_hat = ntt(np.mod(s, q).astype(np.uint64), q, ps, log_n)
        s2_hat = ntt(np.mod(s2, q).astype(np.uint64), q, ps, log_n)
        got.append(intt((u[0, l] + (u[1, l] * s_hat) % qq) % qq, q, ps, log_n))
        want.append(intt((c[l].astype(np.uint64) * s2_hat) % qq, q, ps, log_n))
    diff = _centred_lift(np.stack(got), qs_p[:L]) - _centred_lift(np.stack(want), qs_p[:L])
    assert max(abs(int(x)) for x in diff) > 1000 * _switch_bound(qs_p, n)


@pytest.mark.parametrize("log_n,L,r", [(6, 2, 1), (8, 3, 5), (8, 3, -1), (10, 4, 33)])
def test_rotation_decrypts_to_the_rotated_plaintext(log_n, L, r):
    n, qs_p, psis_p, s, st = _chain(log_n, L, 60 + log_n + r)
    qs, psis = qs_p[:L], psis_p[:L]
    z = st["activations"].normal(0, 1, n // 2)
    delta = 2.0 ** 26
    m = OE.round_coeffs(OE.encode_coeffs(z, log_n), delta)
    e = gen.gaussian_error(st["error"], n)
    a = gen.uniform_residues(st["residues"], (), qs, n)
    ct = rlwe.encrypt(m, s, a, e, qs, psis, log_n)
    g = KS.galois_element(r, log_n)
    ka = gen.uniform_residues(st["residues"], (L,), qs_p, n)
    ke = gen.gaussian_error(st["error"], (L, n))
    ksk = KS.rotation_key(s, r, ka, ke, qs_p, psis_p, log_n)
    rot = KS.rotate(ct, r, ksk, qs_p, psis_p, log_n)
    dec = np.array(rlwe.decrypt(rot, s, qs, psis, log_n), dtype=object)
    want = KS.automorphism_int((m + e).astype(object), g, log_n)
    assert max(abs(int(x)) for x in dec - want) <= _switch_bound(qs_p, n)
    slots = OE.decode(np.array(dec, dtype=np.float64), delta, log_n).real
    assert np.max(np.abs(slots - np.roll(z, -r))) < 1e-3


def test_diagonal_split_identity_in_plaintext():
    """sum_j rot(sum_i pt[j, i] (.) rot(z, i), j n1) = W x, replicated, for the slot vectors of diagonal_slots."""
    rng = np.random.default_rng(5)
    for d, n1, slots in ((8, 2, 32), (16, 4, 64), (12, 3, 48), (16, 16, 16)):
        W = rng.normal(size=(d, d))
        x = rng.normal(size=d)
        pt = bsgs.diagonal_slots(W, n1, slots)
        z = bsgs.replicate(x, slots)
        acc = np.zeros(slots)
        for j in range(d // n1):
            inner = sum(pt[j, i] * np.roll(z, -i) for i in range(n1))
            acc += np.roll(inner, -j * n1)
        assert np.allclose(acc, bsgs.replicate(W @ x, slots), atol=1e-12)


@pytest.mark.parametrize("log_n,L,d,n1", [(6, 3, 8, 4), (7, 3, 16, 4), (7, 3, 16, 8)])
def test_bsgs_matvec_decrypts_to_w_times_x(log_n, L, d, n1):
    n, qs_p, psis_p, s, st = _chain(log_n, L, 80 + d + n1)
    qs, psis = qs_p[:L], psis_p[:L]
    slots = n // 2
    n2 = d // n1
    W = st["weights"].normal(0, 0.5, (d, d))
    x = st["activations"].normal(0, 1, d)
    delta = 2.0 ** 25
    pt = OE.encode_poly(bsgs.diagonal_slots(W, n1, slots), delta, qs, psis, log_n)     # (n2, n1, L, N)
    m = OE.round_coeffs(OE.encode_coeffs(bsgs.replicate(x, slots), log_n), delta)
    ct = rlwe.encrypt(m, s, gen.uniform_residues(st["residues"], (), qs, n), gen.gaussian_error(st["error"], n),
                      qs, psis, log_n)
    keys = {}
    for r in list(range(1, n1)) + [j * n1 for j in range(1, n2)]:
        keys[r] = KS.rotation_key(s, r, gen.uniform_residues(st["residues"], (L,), qs_p, n),
                                  gen.gaussian_error(st["error"], (L, n)), qs_p, psis_p, log_n)
    out = bsgs.matvec(pt, ct, n1, keys, qs_p, psis_p, log_n)
    assert out.shape == (2, L - 1, n)
    dec = np.array(rlwe.decrypt(out, s, qs[:L - 1], psis[:L - 1], log_n), dtype=np.float64)
    y = OE.decode(dec, delta * delta / qs[L - 1], log_n).real
    assert np.max(np.abs(y - bsgs.replicate(W @ x, slots))) < 1e-3


def test_tiled_product_decodes_to_w_times_x():
    """A 2 x 2 grid of 8 x 8 tiles: block i of the output decodes to (W x)[block i]."""
    log_n, L, n1, t = 6, 3, 4, 2
    n, qs_p, psis_p, s, st = _chain(log_n, L, 91)
    qs, psis = qs_p[:L], psis_p[:L]
    slots, d = n // 2, 8
    W = st["weights"].normal(0, 0.5, (t * d, t * d))
    x = st["activations"].normal(0, 1, t * d)
    delta = 2.0 ** 25
    tiles = bsgs.tile_slots(W, t, t, n1, slots)                     # (t, t, n2, n1, slots)
    pt = OE.encode_poly(tiles, delta, qs, psis, log_n)
    cts = []
    for j in range(t):
        m = OE.round_coeffs(OE.encode_coeffs(bsgs.replicate(x[j * d:(j + 1) * d], slots), log_n), delta)
        cts.append(rlwe.encrypt(m, s, gen.uniform_residues(st["residues"], (), qs, n),
                                gen.gaussian_error(st["error"], n), qs, psis, log_n))
    keys = {r: KS.rotation_key(s, r, gen.uniform_residues(st["residues"], (L,), qs_p, n),
                               gen.gaussian_error(st["error"], (L, n)), qs_p, psis_p, log_n) for r in (1, 2, 3, 4)}
    out = bsgs.tiled_matvec(pt, np.stack(cts), n1, keys, qs_p, psis_p, log_n)
    assert out.shape == (t, 2, L - 1, n)
    y = W @ x
    for i in range(t):
        dec = np.array(rlwe.decrypt(out[i], s, qs[:L - 1], psis[:L - 1], log_n), dtype=np.float64)
        got = OE.decode(dec, delta * delta / qs[L - 1], log_n).real
        assert np.max(np.abs(got - bsgs.replicate(y[i * d:(i + 1) * d], slots))) < 1e-3


def _dec_diff(a, b, s, qs, psis, log_n):
    """Centred coefficients of dec(a) - dec(b) mod Q (both (2, L, N) NTT form)."""
    Q = 1
    for q in qs:
        Q *= q
    da = rlwe.decrypt(a, s, qs, psis, log_n)
    db = rlwe.decrypt(b, s, qs, psis, log_n)
    out = []
    for x, y in zip(da, db):
        v = (int(x) - int(y)) % Q
        out.append(v - Q if v > Q // 2 else v)
    return out


@pytest.mark.parametrize("log_n,L,d,n1,seed", [(6, 3, 16, 4, 95), (7, 3, 32, 4, 96), (6, 4, 16, 2, 97)])
def test_lazy_schedule_within_the_bound_of_the_eager_product(log_n, L, d, n1, seed):
    """matvec (every giant-step rotation divided by P on its own, the plain formula)
    and matvec_lazy (giant steps summed before one division by P) on uniform residues.
    Before the closing rescale the sums differ (the roundings are not the same) and
    their decryptions by at most (n2 / 2)(N + 1) per coefficient; after it, by at most
    eager_lazy_bound (N + 1).  A misplaced giant-step term leaves a difference spread
    over all of Z_Q."""
    n2 = d // n1
    n, qs_p, psis_p, s, st = _chain(log_n, L, seed)
    qs, psis = qs_p[:L], psis_p[:L]
    pt = gen.uniform_residues(st["residues"], (n2, n1), qs, n)
    ct = gen.uniform_residues(st["residues"], (2,), qs, n)
    keys = {r: KS.rotation_key(s, r, gen.uniform_residues(st["residues"], (L,), qs_p, n),
                               gen.gaussian_error(st["error"], (L, n)), qs_p, psis_p, log_n)
            for r in list(range(1, n1)) + [j * n1 for j in range(1, n2)]}
    z_e = bsgs.matvec(pt, ct, n1, keys, qs_p, psis_p, log_n, rescaled=False)
    z_l = bsgs.matvec_lazy(pt, ct, n1, keys, qs_p, psis_p, log_n, rescaled=False)
    assert not np.array_equal(z_l, z_e)
    pre = _dec_diff(z_l, z_e, s, qs, psis, log_n)
    assert 0 < max(abs(v) for v in pre) <= (n2 * (n + 1)) // 2
    eager = bsgs.matvec(pt, ct, n1, keys, qs_p, psis_p, log_n)
    lazy = bsgs.matvec_lazy(pt, ct, n1, keys, qs_p, psis_p, log_n)
    bound = bsgs.eager_lazy_bound(n2, log_n, qs[L - 1])
    assert bound == n + 1
    diff = _dec_diff(lazy, eager, s, qs[:L - 1], psis[:L - 1], log_n)
    assert max(abs(v) for v in diff) <= bound
    # one giant-step term left out of the lazy sum is far outside the bound
    keys_wrong = dict(keys)
    keys_wrong[n1] = keys[1] if n1 > 1 else keys[n1]
    wrong = bsgs.matvec_lazy(pt, ct, n1, keys_wrong, qs_p, psis_p, log_n)
    diff_w = _dec_diff(wrong, eager, s, qs[:L - 1], psis[:L - 1], log_n)
    assert max(abs(v) for v in diff_w) > 1000 * bound


def test_eager_product_is_the_composition_of_single_rotations():
    """matvec equals rotations of the inner sums added one by one, each through
    keyswitch.rotate (the pinned single rotation), then the pinned rescale."""
    from oracle import linear as OL
    log_n, L, d, n1 = 6, 3, 12, 3
    n2 = d // n1
    n, qs_p, psis_p, s, st = _chain(log_n, L, 98)
    qs, psis = qs_p[:L], psis_p[:L]
    pt = gen.uniform_residues(st["residues"], (n2, n1), qs, n)
    ct = gen.uniform_residues(st["residues"], (2,), qs, n)
    keys = {r: KS.rotation_key(s, r, gen.uniform_residues(st["residues"], (L,), qs_p, n),
                               gen.gaussian_error(st["error"], (L, n)), qs_p, psis_p, log_n)
            for r in list(range(1, n1)) + [j * n1 for j in range(1, n2)]}
    got = bsgs.matvec(pt, ct, n1, keys, qs_p, psis_p, log_n)
    q = np.array(qs, dtype=np.uint64)[:, None]
    acc = np.zeros((2, L, n), dtype=np.uint64)
    for j in range(n2):
        y = np.zeros((2, L, n), dtype=np.uint64)
        for i in range(n1):
            xi = ct.astype(np.uint64) if i == 0 else KS.rotate(ct, i, keys[i], qs_p, psis_p, log_n)
            y = (y + (pt[j, i].astype(np.uint64)[None] * xi) % q) % q
        acc = (acc + (y if j == 0 else KS.rotate(y, j * n1, keys[j * n1], qs_p, psis_p, log_n))) % q
    want = OL.rescale(acc[None], qs, psis[:L], log_n)[0]
    assert np.array_equal(got, want)
