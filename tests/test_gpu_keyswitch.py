"""GPU parity of the automorphism, rotation-key generation, rotation (hoisted
and per-input) and BSGS entry points against the oracle, and the BSGS product
end to end against numpy's W @ x.

The automorphism, the keys and single rotations are unique results and are
compared bit for bit.  The BSGS product is judged against the oracle's plain
formula (oracle.bsgs.matvec: every giant-step rotation a complete key switch
with its own division by P): the two decrypt, under the test's secret, to
values within oracle.bsgs.eager_lazy_bound (N + 1) of each other in every
coefficient, and the number of residues that differ is reported.  The kernel
sums its giant steps before one division by P, which the oracle also states
as oracle.bsgs.matvec_lazy; against that schedule the product is compared bit
for bit as well.

The context holds the ciphertext primes and the special prime last; every
expected value is computed by the oracle from host-side integers."""
import numpy as np
import pytest

from oracle import bsgs as OB
from oracle import encode as OE
from oracle import keyswitch as KS
from oracle import rlwe as OR
from workloads import gen

pytestmark = pytest.mark.gpu

_CTX = {}


def ctx_for(ck, log_n, L):
    """Context with L ciphertext primes and the special prime (L + 1 primes)."""
    key = (log_n, L)
    if key not in _CTX:
        _CTX[key] = ck.Context(log_n, L + 1)
    return _CTX[key]


def setup(ck, log_n, L, seed):
    ctx = ctx_for(ck, log_n, L)
    qs_p, psis_p, n = list(ctx.moduli), list(ctx.roots), ctx.n
    st = gen.streams(seed, log_n)
    s = gen.ternary_secret(st["secret"], n)
    s_ntt = ck.to_device(np.stack([np.mod(s, q) for q in qs_p]).astype(np.uint32))
    ck.ckks_ntt(ctx, s_ntt, 1, L + 1)
    return ctx, qs_p, psis_p, n, st, s, s_ntt


def dec_diff(a, b, s, qs, psis, log_n):
    """Centred coefficients of dec(a) - dec(b) mod Q (ciphertexts (2, L, N), NTT form)."""
    Q = 1
    for q in qs:
        Q *= q
    out = []
    for x, y in zip(OR.decrypt(a, s, qs, psis, log_n), OR.decrypt(b, s, qs, psis, log_n)):
        v = (int(x) - int(y)) % Q
        out.append(v - Q if v > Q // 2 else v)
    return out


def check_product(got, want_eager, want_lazy, s, qs_p, psis_p, log_n, n2, terms=1, where=""):
    """got against the plain formula (decryption within the bound, summed over `terms`
    products) and against the kernel's schedule (bit for bit).  Returns the number of
    residues that differ from the plain formula."""
    Lo = got.shape[-2]
    qs, psis = qs_p[:Lo], psis_p[:Lo]
    bound = terms * OB.eager_lazy_bound(n2, log_n, qs_p[Lo])
    worst = max(abs(v) for v in dec_diff(got.astype(np.uint64), want_eager, s, qs, psis, log_n))
    assert worst <= bound, f"{where}: decryption differs from the plain BSGS formula by {worst} > {bound}"
    assert np.array_equal(got, want_lazy.astype(np.uint32)), f"{where}: differs from the lazy schedule"
    mism = int(np.count_nonzero(got != want_eager.astype(np.uint32)))
    print(f"{where}: residues differing from the plain formula: {mism} of {got.size}; "
          f"max decryption difference {worst} (bound {bound})", flush=True)
    return mism


def oracle_keys(st, s, steps, qs_p, psis_p, log_n):
    L, n = len(qs_p) - 1, 1 << log_n
    out = []
    for r in steps:
        a = gen.uniform_residues(st["residues"], (L,), qs_p, n)
        e = gen.gaussian_error(st["error"], (L, n))
        out.append(KS.rotation_key(s, r, a, e, qs_p, psis_p, log_n))
    return np.stack(out).astype(np.uint32)                        # (keys, L, 2, L+1, N)


@pytest.mark.parametrize("log_n", [10, 13, 16])
def test_automorphism_bit_exact(gpu_lib, log_n):
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, 2, 700 + log_n)
    rows = gen.uniform_residues(st["residues"], (2,), qs_p, n)           # (2, 3, N): row r uses prime r % 3
    d_in = ck.to_device(rows)
    d_out = ck.empty_u32(rows.shape)
    for g in (KS.galois_element(1, log_n), KS.galois_element(77, log_n), 2 * n - 1):
        ck.ckks_automorphism(ctx, d_in, 6, g, d_out)
        got = ck.to_host_u32(d_out)
        for c in range(2):
            for l in range(3):
                want = KS.automorphism_ntt(rows[c, l], g, qs_p[l], psis_p[l], log_n)
                assert np.array_equal(got[c, l], want.astype(np.uint32)), (g, c, l)


@pytest.mark.parametrize("log_n,L,r0,r_step,count", [(10, 2, 1, 1, 3), (13, 4, 8, 8, 2)])
def test_keygen_rotation_bit_exact(gpu_lib, log_n, L, r0, r_step, count):
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 720 + log_n)
    a = gen.uniform_residues(st["residues"], (count, L), qs_p, n)         # (count, L, L+1, N)
    e = gen.gaussian_error(st["error"], (count, L, n)).astype(np.int32)
    ksk = ck.empty_u32((count, L, 2, L + 1, n))
    ck.ckks_keygen_rotation(ctx, s_ntt, r0, r_step, count, ck.to_device(a), ck.to_device(e), ksk)
    got = ck.to_host_u32(ksk)
    for k in range(count):
        want = KS.rotation_key(s, r0 + k * r_step, a[k], e[k], qs_p, psis_p, log_n)
        assert np.array_equal(got[k], want.astype(np.uint32)), k


@pytest.mark.parametrize("log_n,L,hoisted,steps", [(10, 2, True, (1, 2, 3)), (10, 3, False, (5, 9)),
                                                   (12, 3, True, (4, 8)), (13, 2, True, (1, 2, 3)),
                                                   (14, 3, False, (2, 6)), (16, 2, False, (1,)),
                                                   (10, 2, True, (511,)),                  # a left rotation by N/2 - 1 = right by 1
                                                   (14, 3, False, tuple(range(1, 23))),    # 264 ModUp groups: two-launch form
                                                   (10, 5, True, (1, 2))])                 # 5 digits: keys re-read per use
def test_rotate_bit_exact(gpu_lib, log_n, L, hoisted, steps):
    """Bit-exact against the oracle.  The ModUp runs fused while its (input, digit, prime)
    workgroups number at most one per CU (256), else in two launches (22 inputs x 3 digits
    x 4 primes at 2^14), and at 2^16 as the four-launch pass route.  The key-switching
    inner product holds the keys in registers for 2 to 4 digits, and re-reads them for
    more (5 here)."""
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 740 + log_n + L)
    count = len(steps)
    r0, r_step = steps[0], (steps[1] - steps[0]) if count > 1 else 1
    assert list(steps) == [r0 + k * r_step for k in range(count)]
    cts = gen.uniform_residues(st["residues"], (1 if hoisted else count, 2), qs_p[:L], n)
    keys = oracle_keys(st, s, steps, qs_p, psis_p, log_n)
    ws = ck.empty_workspace(ck.rotate_workspace_bytes(ctx, count, hoisted))
    out = ck.empty_u32((count, 2, L, n))
    ck.ckks_rotate(ctx, ck.to_device(cts), count, r0, r_step, hoisted, ck.to_device(keys), ws, out)
    got = ck.to_host_u32(out)
    for k, r in enumerate(steps):
        src = cts[0] if hoisted else cts[k]
        want = KS.rotate(src.astype(np.uint64), r, keys[k], qs_p, psis_p, log_n)
        assert np.array_equal(got[k], want.astype(np.uint32)), (k, r)


@pytest.mark.parametrize("log_n,L,n1,n2,count", [(10, 2, 4, 4, 2), (11, 3, 3, 5, 1), (10, 3, 1, 4, 1),
                                                 (10, 2, 4, 1, 1), (10, 2, 2, 3, 6), (10, 2, 2, 2, 65),
                                                 (15, 2, 2, 2, 1), (16, 2, 2, 2, 1), (11, 3, 2, 10, 3),
                                                 (12, 3, 8, 17, 5), (10, 4, 16, 2, 20)])
def test_bsgs_matches_the_oracle(gpu_lib, log_n, L, n1, n2, count):
    """Any residues: uniform plaintexts and ciphertexts, the product checked against the
    plain formula (decryption within N + 1) and against the lazy schedule bit for bit.
    The closing pair of rescales (division by P, then by q_(L-1)) runs as one launch
    for few inputs up to 2^15 and as
    two rescales for 65 inputs (more than a quarter of 256 CUs) and at 2^16.  Several
    inputs take the register-tiled MAC (8 rows by 2 inputs per thread): n2 = 10 and 17
    and 3 or 5 inputs leave partial tiles in both directions.  With 20 inputs, n1 = 16 and
    4 digits at 2^10 the key-switching loop over each baby key's 20 uses is cut into
    chunks that do not divide it evenly (14 on 256 CUs)."""
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 760 + n1 * 7 + n2)
    pt = gen.uniform_residues(st["residues"], (n2, n1), qs_p[:L], n)
    cts = gen.uniform_residues(st["residues"], (count, 2), qs_p[:L], n)
    steps = list(range(1, n1)) + [j * n1 for j in range(1, n2)]
    keys = oracle_keys(st, s, steps, qs_p, psis_p, log_n) if steps else None
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, count, n1, n2))
    out = ck.empty_u32((count, 2, L - 1, n))
    ck.ckks_linear_bsgs(ctx, ck.to_device(pt), ck.to_device(cts), count, n1, n2,
                        ck.to_device(keys) if keys is not None else None, ws, out)
    got = ck.to_host_u32(out)
    kd = {r: keys[i] for i, r in enumerate(steps)}
    for b in range(count):
        x = cts[b].astype(np.uint64)
        check_product(got[b], OB.matvec(pt, x, n1, kd, qs_p, psis_p, log_n),
                      OB.matvec_lazy(pt, x, n1, kd, qs_p, psis_p, log_n), s, qs_p, psis_p, log_n, n2,
                      where=f"input {b}")


def test_bsgs_end_to_end_matches_w_times_x(gpu_lib):
    """Diagonals encoded and keys generated on the GPU; the decrypted, decoded
    product equals numpy's W @ x for every slot (d = 64, N = 2^12)."""
    ck = gpu_lib
    log_n, L, d, n1 = 12, 3, 64, 8
    n2 = d // n1
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 781)
    qs, psis, slots = qs_p[:L], psis_p[:L], n // 2
    delta = float(2 ** 26)
    W = st["weights"].normal(0, 0.1, (d, d))
    x = st["activations"].normal(0, 1, d)
    diag = OB.diagonal_slots(W, n1, slots).reshape(n2 * n1, slots)
    pt = ck.empty_u32((n2, n1, L, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(diag), n2 * n1, L, delta, pt)
    m = OE.round_coeffs(OE.encode_coeffs(OB.replicate(x, slots), log_n), delta)
    ct = OR.encrypt(m, s, gen.uniform_residues(st["residues"], (), qs, n), gen.gaussian_error(st["error"], n),
                    qs, psis, log_n).astype(np.uint32)
    steps_b, steps_g = n1 - 1, n2 - 1
    a = gen.uniform_residues(st["residues"], (steps_b + steps_g, L), qs_p, n)
    e = gen.gaussian_error(st["error"], (steps_b + steps_g, L, n)).astype(np.int32)
    ksk = ck.empty_u32((steps_b + steps_g, L, 2, L + 1, n))
    key_words = L * 2 * (L + 1) * n
    flat = ksk.view(-1)
    ck.ckks_keygen_rotation(ctx, s_ntt, 1, 1, steps_b, ck.to_device(a[:steps_b]), ck.to_device(e[:steps_b]),
                            flat[: steps_b * key_words])
    ck.ckks_keygen_rotation(ctx, s_ntt, n1, n1, steps_g, ck.to_device(a[steps_b:]), ck.to_device(e[steps_b:]),
                            flat[steps_b * key_words:])
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, 1, n1, n2))
    out = ck.empty_u32((1, 2, L - 1, n))
    ck.ckks_linear_bsgs(ctx, pt, ck.to_device(ct[None]), 1, n1, n2, ksk, ws, out)
    res = ck.to_host_u32(out)[0].astype(np.uint64)
    dec = np.array(OR.decrypt(res, s, qs[:L - 1], psis[:L - 1], log_n), dtype=np.float64)
    y = OE.decode(dec, delta * delta / qs[L - 1], log_n).real
    assert np.max(np.abs(y - OB.replicate(W @ x, slots))) < 1e-3


def test_rotation_argument_errors(gpu_lib):
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, 10, 2, 790)
    ct = ck.empty_u32((1, 2, 2, n))
    out = ck.empty_u32((2, 2, 2, n))
    ksk = ck.empty_u32((2, 2, 2, 3, n))
    small = ck.empty_workspace(64)
    with pytest.raises(ck.CkksError) as ex:
        ck.ckks_rotate(ctx, ct, 2, 1, 1, True, ksk, small, out)
    assert ex.value.code == ck.CKKS_E_WORKSPACE
    with pytest.raises(ck.CkksError) as ex:
        ck.ckks_automorphism(ctx, ct, 4, 6, out)                       # even element
    assert ex.value.code == ck.CKKS_E_INVALID_ARG
    import ctypes
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    ws = ck.empty_workspace(1 << 20)
    rc = ck._lib.ckks_linear_bsgs(ctx.handle, P(ksk), P(ct), 1, 32, 32, P(ksk), P(ws), 1 << 20, P(out), None)
    assert rc == ck.CKKS_E_INVALID_ARG and "n1 n2 <= N/2" in ck.ckks_last_error()   # d = 1024 > N/2
    two = ck.Context(10, 2)
    with pytest.raises(ck.CkksError) as ex:                              # no room for the special prime
        ck.ckks_rotate(two, ck.empty_u32((1, 2, 1, n)), 1, 1, 1, True, ck.empty_u32((1, 1, 2, 2, n)), small,
                       ck.empty_u32((1, 2, 1, n)))
    assert ex.value.code == ck.CKKS_E_INVALID_ARG


def test_add_bit_exact(gpu_lib):
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, 11, 3, 795)
    a = gen.uniform_residues(st["residues"], (5, 2), qs_p[:3], n)
    b = gen.uniform_residues(st["residues"], (5, 2), qs_p[:3], n)
    q = np.array(qs_p[:3], dtype=np.uint64)[:, None]
    want = ((a.astype(np.uint64) + b) % q).astype(np.uint32)
    da, db = ck.to_device(a), ck.to_device(b)
    out = ck.empty_u32(a.shape)
    ck.ckks_add(ctx, da, db, 5, 3, out)
    assert np.array_equal(ck.to_host_u32(out), want)
    ck.ckks_add(ctx, da, db, 5, 3, da)                                   # in place
    assert np.array_equal(ck.to_host_u32(da), want)


def test_tiled_product_matches_the_oracle(gpu_lib):
    """A 2 x 3 grid of tiles: per-tile BSGS calls and ciphertext additions on the GPU
    against the oracle's tiled product (uniform residues): decryptions within 3 (N + 1)
    of the plain formula's (three tile products per block), bit for bit against the
    lazy schedule."""
    ck = gpu_lib
    log_n, L, n1, n2, t_o, t_i, count = 10, 2, 2, 2, 2, 3, 1
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 797)
    pt = gen.uniform_residues(st["residues"], (t_o, t_i, n2, n1), qs_p[:L], n)
    cts = gen.uniform_residues(st["residues"], (t_i, 2), qs_p[:L], n)
    steps = [1, 2]
    keys = oracle_keys(st, s, steps, qs_p, psis_p, log_n)
    d_keys, d_pt, d_ct = ck.to_device(keys), ck.to_device(pt), ck.to_device(cts)
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, count, n1, n2))
    out = ck.empty_u32((t_o, 2, L - 1, n))
    part = ck.empty_u32((2, L - 1, n))
    for i in range(t_o):
        ck.ckks_linear_bsgs(ctx, d_pt[i, 0], d_ct[0:1], 1, n1, n2, d_keys, ws, out[i])
        for j in range(1, t_i):
            ck.ckks_linear_bsgs(ctx, d_pt[i, j], d_ct[j:j + 1], 1, n1, n2, d_keys, ws, part)
            ck.ckks_add(ctx, out[i], part, 1, L - 1, out[i])
    kd = {1: keys[0], 2: keys[1]}
    x = cts.astype(np.uint64)
    eager = OB.tiled_matvec(pt, x, n1, kd, qs_p, psis_p, log_n)
    lazy = OB.tiled_matvec(pt, x, n1, kd, qs_p, psis_p, log_n, product=OB.matvec_lazy)
    got = ck.to_host_u32(out)
    for i in range(got.shape[0]):
        check_product(got[i], eager[i], lazy[i], s, qs_p, psis_p, log_n, pt.shape[2], terms=pt.shape[1],
                      where=f"output block {i}")


def test_bsgs_full_size(gpu_lib):
    """The benchmarked call's shape: d = 1024 (n1 = n2 = 32) at N = 2^13 with 4 ciphertext
    primes and the special prime, one input; uniform residues, oracle keys, checked against
    the plain formula (decryption within N + 1) and the lazy schedule (bit for bit)."""
    ck = gpu_lib
    log_n, L, n1, n2 = 13, 4, 32, 32
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 799)
    pt = gen.uniform_residues(st["residues"], (n2, n1), qs_p[:L], n)
    ct = gen.uniform_residues(st["residues"], (1, 2), qs_p[:L], n)
    steps = list(range(1, n1)) + [j * n1 for j in range(1, n2)]
    keys = oracle_keys(st, s, steps, qs_p, psis_p, log_n)
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, 1, n1, n2))
    out = ck.empty_u32((1, 2, L - 1, n))
    ck.ckks_linear_bsgs(ctx, ck.to_device(pt), ck.to_device(ct), 1, n1, n2, ck.to_device(keys), ws, out)
    kd = {r: keys[i] for i, r in enumerate(steps)}
    x = ct[0].astype(np.uint64)
    check_product(ck.to_host_u32(out)[0], OB.matvec(pt, x, n1, kd, qs_p, psis_p, log_n),
                  OB.matvec_lazy(pt, x, n1, kd, qs_p, psis_p, log_n), s, qs_p, psis_p, log_n, n2,
                  where="d = 1024, N = 2^13")


def test_add_rejects_partial_overlap(gpu_lib):
    ck = gpu_lib
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, 10, 2, 801)
    buf = ck.empty_u32((3, 2, 2, n))
    with pytest.raises(ck.CkksError) as ex:
        ck.ckks_add(ctx, buf[0:2], buf[1:3], 2, 2, buf[1:3])   # out aliases b exactly, overlaps a partly
    assert ex.value.code == ck.CKKS_E_INVALID_ARG


def test_bsgs_one_by_one(gpu_lib):
    """d = 1 (n1 = n2 = 1): no rotations, no keys; the product is pt (.) x, rescaled."""
    ck = gpu_lib
    log_n, L = 10, 3
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 803)
    pt = gen.uniform_residues(st["residues"], (1, 1), qs_p[:L], n)
    ct = gen.uniform_residues(st["residues"], (2, 2), qs_p[:L], n)
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, 2, 1, 1))
    out = ck.empty_u32((2, 2, L - 1, n))
    ck.ckks_linear_bsgs(ctx, ck.to_device(pt), ck.to_device(ct), 2, 1, 1, None, ws, out)
    for b in range(2):
        want = OB.matvec(pt, ct[b].astype(np.uint64), 1, {}, qs_p, psis_p, log_n)
        assert np.array_equal(ck.to_host_u32(out)[b], want.astype(np.uint32))   # no rotation: unique


def test_tiled_product_at_the_benchmarked_shape(gpu_lib):
    """The sweep's 2x2 configuration for one row: 512 x 512 tiles (n1 = 32, n2 = 16) at
    N = 2^12, four limbs and the special prime; per-tile BSGS calls and ciphertext
    additions against the oracle's tiled product (uniform residues): decryptions within
    2 (N + 1) of the plain formula's, bit for bit against the lazy schedule."""
    ck = gpu_lib
    log_n, L, n1, n2, t = 12, 4, 32, 16, 2
    ctx, qs_p, psis_p, n, st, s, s_ntt = setup(ck, log_n, L, 807)
    pt = gen.uniform_residues(st["residues"], (t, t, n2, n1), qs_p[:L], n)
    cts = gen.uniform_residues(st["residues"], (t, 2), qs_p[:L], n)
    steps = list(range(1, n1)) + [j * n1 for j in range(1, n2)]
    keys = oracle_keys(st, s, steps, qs_p, psis_p, log_n)
    d_keys, d_pt, d_ct = ck.to_device(keys), ck.to_device(pt), ck.to_device(cts)
    ws = ck.empty_workspace(ck.bsgs_workspace_bytes(ctx, 1, n1, n2))
    out = ck.empty_u32((t, 2, L - 1, n))
    part = ck.empty_u32((2, L - 1, n))
    for i in range(t):
        ck.ckks_linear_bsgs(ctx, d_pt[i, 0], d_ct[0:1], 1, n1, n2, d_keys, ws, out[i])
        for j in range(1, t):
            ck.ckks_linear_bsgs(ctx, d_pt[i, j], d_ct[j:j + 1], 1, n1, n2, d_keys, ws, part)
            ck.ckks_add(ctx, out[i], part, 1, L - 1, out[i])
    kd = {r: keys[k] for k, r in enumerate(steps)}
    x = cts.astype(np.uint64)
    eager = OB.tiled_matvec(pt, x, n1, kd, qs_p, psis_p, log_n)
    lazy = OB.tiled_matvec(pt, x, n1, kd, qs_p, psis_p, log_n, product=OB.matvec_lazy)
    got = ck.to_host_u32(out)
    for i in range(t):
        check_product(got[i], eager[i], lazy[i], s, qs_p, psis_p, log_n, n2, terms=t, where=f"output block {i}")
