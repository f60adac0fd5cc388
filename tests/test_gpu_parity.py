"""GPU parity on small shapes: every C-ABI entry point against the CPU oracle.

Integer work (NTT, scalar encode, both MACs, rescale) must be bit-exact.  The
full-polynomial encode runs its spectral transform in fp64, so residues may
differ by one near rounding ties; it is held to a decoded-slot error of at
most 2^-20 relative to the oracle's decoded values, and its mismatch count is
reported.  Inputs come from the seeded generators (and, for the encrypted
cases, from the oracle's encoder and encryptor).
"""
import numpy as np
import pytest

from oracle import encode as OE
from oracle import linear as OL
from oracle import ntt as ON
from oracle import params as OP
from tests.cases import build_layer, check_decrypted
from workloads import gen, get

pytestmark = pytest.mark.gpu

_CTX = {}


def ctx_for(ck, log_n, limbs):
    key = (log_n, limbs)
    if key not in _CTX:
        _CTX[key] = ck.Context(log_n, limbs)
    return _CTX[key]


def rand_residues(seed, prefix, qs, n):
    return gen.uniform_residues(np.random.default_rng(seed), prefix, qs, n)


@pytest.mark.parametrize("log_n,limbs", [(10, 2), (14, 4), (15, 6), (16, 8)])
def test_context_chain_matches_oracle(gpu_lib, log_n, limbs):
    ctx = ctx_for(gpu_lib, log_n, limbs)
    assert ctx.moduli == OP.moduli(log_n, limbs)
    assert ctx.roots == tuple(OP.psi(q, log_n) for q in ctx.moduli)


@pytest.mark.parametrize("log_n", [10, 11, 12, 13, 14, 15, 16])
def test_ntt_and_intt_bit_exact(gpu_lib, log_n):
    ck = gpu_lib
    limbs = 3
    ctx = ctx_for(ck, log_n, limbs)
    qs, n, count = ctx.moduli, 1 << log_n, 2
    a = rand_residues(log_n, (count,), qs, n)                    # (count, limbs, n)
    d = ck.to_device(a)
    ck.ckks_ntt(ctx, d, count, limbs)
    got = ck.to_host_u32(d).reshape(count, limbs, n)
    for l in range(limbs):
        want = ON.ntt(a[:, l].astype(np.uint64), qs[l], ctx.roots[l], log_n)
        assert np.array_equal(got[:, l], want), f"ntt limb {l}"
    ck.ckks_intt(ctx, d, count, limbs)
    assert np.array_equal(ck.to_host_u32(d).reshape(a.shape), a)
    # inverse alone against the oracle
    d2 = ck.to_device(a)
    ck.ckks_intt(ctx, d2, count, limbs)
    got = ck.to_host_u32(d2).reshape(count, limbs, n)
    for l in range(limbs):
        assert np.array_equal(got[:, l], ON.intt(a[:, l].astype(np.uint64), qs[l], ctx.roots[l], log_n))


def test_longest_chain_16_limbs(gpu_lib):
    """The longest modulus chain the context accepts (16 limbs), at N = 2^10:
    the chain and roots, the transforms, scalar encode, both scalar MAC kernels
    and the poly MAC, each against the oracle."""
    ck = gpu_lib
    log_n, limbs = 10, 16
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, 1 << log_n
    assert qs == OP.moduli(log_n, limbs)
    assert ctx.roots == tuple(OP.psi(q, log_n) for q in qs)
    a = rand_residues(161, (2,), qs, n)
    d = ck.to_device(a)
    ck.ckks_ntt(ctx, d, 2, limbs)
    got = ck.to_host_u32(d).reshape(a.shape)
    for l in range(limbs):
        assert np.array_equal(got[:, l], ON.ntt(a[:, l].astype(np.uint64), qs[l], ctx.roots[l], log_n)), l
    ck.ckks_intt(ctx, d, 2, limbs)
    assert np.array_equal(ck.to_host_u32(d).reshape(a.shape), a)
    rng = np.random.default_rng(162)
    w = rng.normal(0, 0.02, (40, 37))
    w_enc = ck.empty_u32((40, 37, limbs))
    ck.ckks_linear_encode_scalar(ctx, ck.to_device(w), 40, 37, limbs, 2.0**28, w_enc)
    want_w = OE.encode_scalar(w, 2.0**28, qs).astype(np.uint32)
    assert np.array_equal(ck.to_host_u32(w_enc), want_w)
    ct = rand_residues(163, (37, 2), qs, n)
    want = OL.mac_scalar(want_w, ct, qs).astype(np.uint32)
    for algo in (ck.CKKS_MAC_VALU, ck.CKKS_MAC_MFMA):
        ck.ckks_ctx_set_mac_algo(ctx, algo)
        try:
            ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, 40, 37, limbs)
            ws = ck.empty_u32((max(ws_bytes, 16) // 4 + 4,))
            out = ck.empty_u32((40, 2, limbs, n))
            ck.ckks_linear_mac_scalar(ctx, w_enc, ck.to_device(ct), out, 40, 37, limbs, ws)
            assert np.array_equal(ck.to_host_u32(out), want), algo
        finally:
            ck.ckks_ctx_set_mac_algo(ctx, ck.CKKS_MAC_AUTO)
    pt = rand_residues(164, (5, 4), qs, n)
    ct2 = rand_residues(165, (4, 2), qs, n)
    out = ck.empty_u32((5, 2, limbs, n))
    ck.ckks_linear_mac_poly(ctx, ck.to_device(pt), ck.to_device(ct2), out, 5, 4, limbs)
    assert np.array_equal(ck.to_host_u32(out), OL.mac_poly(pt, ct2, qs).astype(np.uint32))


def test_ntt_limb_subset_and_empty(gpu_lib):
    ck = gpu_lib
    ctx = ctx_for(ck, 12, 4)
    a = rand_residues(5, (3,), ctx.moduli[:2], 4096)
    d = ck.to_device(a)
    ck.ckks_ntt(ctx, d, 3, 2)
    got = ck.to_host_u32(d).reshape(a.shape)
    for l in range(2):
        assert np.array_equal(got[:, l], ON.ntt(a[:, l].astype(np.uint64), ctx.moduli[l], ctx.roots[l], 12))
    ck.ckks_ntt(ctx, d, 0, 2)                                   # empty batch: no-op
    assert np.array_equal(ck.to_host_u32(d).reshape(a.shape), got)


def test_encode_scalar_bit_exact(gpu_lib):
    ck = gpu_lib
    ctx = ctx_for(ck, 14, 4)
    rng = np.random.default_rng(3)
    w = rng.normal(0, 0.02, (37, 53))
    w[0, :6] = np.array([1.5, 2.5, -1.5, -2.5, 0.0, -0.0]) / 2**26      # exact ties and zeros
    w[1, 0] = 3.0e7 / 2**26 * 2**20                                     # large magnitude
    for scale in (2.0**26, 2.0**30):
        dw = ck.to_device(w)
        out = ck.empty_u32((37, 53, 4))
        ck.ckks_linear_encode_scalar(ctx, dw, 37, 53, 4, scale, out)
        assert np.array_equal(ck.to_host_u32(out), OE.encode_scalar(w, scale, ctx.moduli).astype(np.uint32))


@pytest.mark.parametrize("log_n,limbs,d_in,d_out", [(10, 1, 5, 3), (10, 2, 16, 16), (11, 3, 33, 17),
                                                  (12, 2, 70, 9), (10, 3, 1, 1)])
@pytest.mark.parametrize("algo", ["valu", "mfma"])
def test_mac_scalar_bit_exact(gpu_lib, log_n, limbs, d_in, d_out, algo):
    ck = gpu_lib
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, 1 << log_n
    rng = np.random.default_rng(log_n * 100 + d_in)
    # general residues (not only small signed weights), plus extremes
    w = np.stack([rng.integers(0, q, (d_out, d_in), dtype=np.uint64) for q in qs], -1).astype(np.uint32)
    w[0, 0, :] = [q - 1 for q in qs]
    ct = rand_residues(d_in, (d_in, 2), qs, n)
    ct[0, 0, :, :7] = np.array(qs, dtype=np.uint32)[:, None] - 1
    want = OL.mac_scalar(w, ct, qs).astype(np.uint32)
    ck.ckks_ctx_set_mac_algo(ctx, ck.CKKS_MAC_VALU if algo == "valu" else ck.CKKS_MAC_MFMA)
    try:
        ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d_out, d_in, limbs)
        ws = ck.empty_u32((max(ws_bytes, 16) // 4 + 4,))
        out = ck.empty_u32((d_out, 2, limbs, n))
        ck.ckks_linear_mac_scalar(ctx, ck.to_device(w), ck.to_device(ct), out, d_out, d_in, limbs, ws)
        assert np.array_equal(ck.to_host_u32(out), want)
    finally:
        ck.ckks_ctx_set_mac_algo(ctx, ck.CKKS_MAC_AUTO)


def test_mac_scalar_zero_inputs_and_empty_outputs(gpu_lib):
    ck = gpu_lib
    ctx = ctx_for(ck, 10, 2)
    out = ck.to_device(np.full((3, 2, 2, 1024), 7, dtype=np.uint32))
    ck.ckks_linear_mac_scalar(ctx, None, None, out, 3, 0, 2)             # d_in = 0 writes zeros
    assert not ck.to_host_u32(out).any()
    ck.ckks_linear_mac_scalar(ctx, None, None, None, 0, 5, 2)            # d_out = 0: no-op


@pytest.mark.parametrize("log_n,limbs,d_in,d_out", [(10, 3, 8, 8), (11, 2, 5, 3), (10, 1, 1, 2)])
def test_mac_poly_bit_exact(gpu_lib, log_n, limbs, d_in, d_out):
    ck = gpu_lib
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, 1 << log_n
    pt = rand_residues(7 + d_in, (d_out, d_in), qs, n)
    ct = rand_residues(8 + d_in, (d_in, 2), qs, n)
    out = ck.empty_u32((d_out, 2, limbs, n))
    ck.ckks_linear_mac_poly(ctx, ck.to_device(pt), ck.to_device(ct), out, d_out, d_in, limbs)
    assert np.array_equal(ck.to_host_u32(out), OL.mac_poly(pt, ct, qs).astype(np.uint32))


@pytest.mark.parametrize("log_n,limbs,count", [(10, 2, 3), (11, 3, 2), (12, 4, 1), (13, 2, 1), (14, 3, 1),
                                               (15, 2, 1), (16, 3, 1), (10, 4, 70), (12, 3, 65)])
def test_rescale_bit_exact(gpu_lib, log_n, limbs, count):
    ck = gpu_lib
    ctx = ctx_for(ck, log_n, max(limbs, 3))
    qs, psis, n = ctx.moduli[:limbs], ctx.roots[:limbs], 1 << log_n
    ct = rand_residues(log_n + count, (count, 2), qs, n)
    ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_RESCALE, count, 0, limbs)
    ws = ck.empty_u32((max(ws_bytes, 16) // 4,))
    out = ck.empty_u32((count, 2, limbs - 1, n))
    ck.ckks_rescale(ctx, ck.to_device(ct), out, count, limbs, ws)
    assert np.array_equal(ck.to_host_u32(out), OL.rescale(ct, qs, psis, log_n).astype(np.uint32))


def test_rescale_rejects_one_limb_and_small_workspace(gpu_lib):
    ck = gpu_lib
    ctx = ctx_for(ck, 16, 8)
    x = ck.empty_u32((2, 2, 65536))
    with pytest.raises(ck.CkksError) as e:
        ck.ckks_rescale(ctx, x, ck.empty_u32((1,)), 1, 1)
    assert e.value.code == ck.CKKS_E_INVALID_ARG
    x = ck.empty_u32((1, 2, 2, 65536))
    with pytest.raises(ck.CkksError) as e:
        ck.ckks_rescale(ctx, x, ck.empty_u32((2, 65536)), 1, 2, ck.empty_u32((16,)))
    assert e.value.code == ck.CKKS_E_WORKSPACE


def test_misaligned_and_out_of_range_arguments(gpu_lib):
    ck = gpu_lib
    ctx = ctx_for(ck, 10, 2)
    buf = ck.empty_u32((2 * 2 * 1024 + 1,))
    with pytest.raises(ck.CkksError) as e:
        ck.ckks_ntt(ctx, buf[1:], 1, 2)                                  # 4-byte offset
    assert e.value.code == ck.CKKS_E_INVALID_ARG
    with pytest.raises(ck.CkksError) as e:
        ck.ckks_ntt(ctx, buf, 1, 3)                                      # limbs > L
    assert e.value.code == ck.CKKS_E_INVALID_ARG
    with pytest.raises(ValueError):
        ck.ckks_ntt(ctx, ck.empty_u32((100,)), 1, 2)                     # buffer too small
    with pytest.raises(ck.CkksError) as e:
        ck.Context(12, 2, moduli=[1073707009, 1073707009])               # not = 1 mod 2^13 / repeated
    assert e.value.code == ck.CKKS_E_INVALID_ARG


def _decode_rows(pt_ntt, qs, psis, log_n, delta):
    """Oracle decode of NTT-form single-limb-lifted plaintexts (rows, L, N) -> slots."""
    out = []
    Q = 1
    for q in qs:
        Q *= q
    for row in pt_ntt:
        coef = [ON.intt(row[l].astype(np.uint64), qs[l], psis[l], log_n) for l in range(len(qs))]
        lifted = [OP.centre(c, Q) for c in OP.crt_lift(coef, qs)]
        out.append(OE.decode(lifted, delta, log_n))
    return np.array(out)


@pytest.mark.parametrize("log_n,limbs,count", [(10, 3, 6), (12, 2, 2), (13, 4, 2), (14, 4, 1), (15, 2, 1)])
def test_encode_poly_within_tolerance(gpu_lib, log_n, limbs, count):
    ck = gpu_lib
    ctx = ctx_for(ck, log_n, max(limbs, 3))
    qs, psis, n = ctx.moduli[:limbs], ctx.roots[:limbs], 1 << log_n
    delta = 2.0 ** 30
    z = gen.poly_weights(np.random.default_rng(log_n), 1, count, n // 2)[0]
    z[0, :] = 0.25                                                       # constant slots: exact closed form
    pt = ck.empty_u32((count, limbs, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(z), count, limbs, delta, pt)
    got = ck.to_host_u32(pt)
    want = OE.encode_poly(z, delta, qs, psis, log_n).astype(np.uint32)
    assert np.all(got[0] == np.uint32(round(0.25 * delta) % np.array(qs, dtype=np.int64)[:, None]))
    # compare coefficients (a one-off rounding difference would touch every NTT slot)
    coef_got = np.stack([[ON.intt(got[b, l].astype(np.uint64), qs[l], psis[l], log_n) for l in range(limbs)]
                         for b in range(count)])
    coef_want = np.stack([[ON.intt(want[b, l].astype(np.uint64), qs[l], psis[l], log_n) for l in range(limbs)]
                          for b in range(count)])
    mismatches = int(np.sum(np.any(coef_got != coef_want, axis=1)))
    print(f"encode_poly N=2^{log_n} L={limbs} count={count}: {mismatches} coefficient mismatches")
    sl_got = _decode_rows(got, qs, psis, log_n, delta)
    sl_want = _decode_rows(want, qs, psis, log_n, delta)
    err = np.max(np.abs(sl_got - sl_want))
    assert err <= 2.0 ** -20 * max(1.0, np.max(np.abs(sl_want))), err
    assert mismatches <= max(2, count * n // 100000)


@pytest.mark.parametrize("log_scale", [30, 40])
def test_encode_poly_n16_sampled_coefficients(gpu_lib, log_scale):
    """N = 2^16 (split spectral transform, then the batched 2^16 NTT): constant
    slots give the constant polynomial exactly in every NTT slot; for random
    slots every limb's plaintext, taken back to coefficients by the oracle's
    inverse transform, equals the oracle's rounded coefficients at 1024 sampled
    indices (k = 0, 1, N/2 - 1, N/2, N/2 + 1, N - 1 and random ones, both
    parities and all four quarters), except at fp64 rounding ties."""
    ck = gpu_lib
    log_n, limbs, count = 16, 3, 2
    ctx = ctx_for(ck, log_n, limbs)
    qs, psis, n = ctx.moduli, ctx.roots, 1 << log_n
    delta = 2.0 ** log_scale
    z = gen.poly_weights(np.random.default_rng(160 + log_scale), 1, count, n // 2)[0]
    if log_scale == 40:
        z = z + 4.0                                           # coefficients near 2^42
    z[0, :] = 0.25
    pt = ck.empty_u32((count, limbs, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(z), count, limbs, delta, pt)
    got = ck.to_host_u32(pt)
    c0 = round(0.25 * delta)
    for l in range(limbs):
        assert np.all(got[0, l] == np.uint32(c0 % qs[l])), l
    rng = np.random.default_rng(7)
    ks = np.unique(np.concatenate([[0, 1, n // 2 - 1, n // 2, n // 2 + 1, n - 1],
                                   rng.choice(n, 1018, replace=False)]))
    want = OE.round_coeffs(OE.encode_coeffs(z[1], log_n, ks), delta)
    bad = 0
    for l in range(limbs):
        coef = ON.intt(got[1, l].astype(np.uint64), qs[l], psis[l], log_n).astype(np.int64)
        w = np.mod(want, qs[l])
        diff = np.mod(coef[ks] - w, qs[l])
        off = diff != 0
        assert np.all((diff[off] == 1) | (diff[off] == qs[l] - 1)), (l, diff[off][:8])
        bad += int(np.sum(off))
    print(f"encode_poly N=2^16 scale 2^{log_scale}: {bad} of {limbs * len(ks)} sampled residues off by one")
    assert bad <= 2


@pytest.mark.parametrize("log_n,limbs", [(10, 3), (14, 3), (15, 2)])
def test_encode_poly_large_coefficients(gpu_lib, log_n, limbs):
    """Slots offset by 4.0 at scale 2^30: coefficients beyond 2^31 take the
    encoder's wide path (every limb's coefficient residues written first, then
    transformed in place); bit-exact against the oracle's NTT-form residues
    except at fp64 rounding ties, held to the same decoded-slot bound."""
    ck = gpu_lib
    ctx = ctx_for(ck, log_n, max(limbs, 3))
    qs, psis, n = ctx.moduli[:limbs], ctx.roots[:limbs], 1 << log_n
    delta = 2.0 ** 30
    z = 4.0 + gen.poly_weights(np.random.default_rng(log_n + 5), 1, 2, n // 2)[0]
    pt = ck.empty_u32((2, limbs, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(z), 2, limbs, delta, pt)
    got = ck.to_host_u32(pt)
    want = OE.encode_poly(z, delta, qs, psis, log_n).astype(np.uint32)
    assert np.max(np.abs(OE.round_coeffs(OE.encode_coeffs(z, log_n), delta))) >= 2 ** 31
    sl_got = _decode_rows(got, qs, psis, log_n, delta)
    sl_want = _decode_rows(want, qs, psis, log_n, delta)
    err = np.max(np.abs(sl_got - sl_want))
    assert err <= 2.0 ** -20 * max(1.0, np.max(np.abs(sl_want))), err
    rows_equal = int(sum(np.array_equal(got[b, l], want[b, l]) for b in range(2) for l in range(limbs)))
    print(f"encode_poly large N=2^{log_n}: {rows_equal} of {2 * limbs} limb rows identical")


def test_encode_poly_mixed_batch_wide_vectors(gpu_lib):
    """A batch with a few slot vectors whose coefficients pass 2^31 (offset by 4.0
    at scale 2^30) among CKKS-scaled ones: each workgroup takes its own vector's
    path.  The wide vectors match the oracle within the decoded-slot bound and
    their own encoding alone; every other vector is bit-identical to a batch
    without wide neighbours; no output word lies outside [0, q)."""
    ck = gpu_lib
    log_n, limbs, count = 10, 2, 600
    ctx = ctx_for(ck, log_n, 3)
    qs, psis, n = ctx.moduli[:limbs], ctx.roots[:limbs], 1 << log_n
    delta = 2.0 ** 30
    z = gen.poly_weights(np.random.default_rng(1010), 1, count, n // 2)[0]
    wide = [0, 1, 255, 256, 511, count - 1]
    z_mixed = z.copy()
    z_mixed[wide] += 4.0
    pt = ck.empty_u32((count, limbs, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(z_mixed), count, limbs, delta, pt)
    got = ck.to_host_u32(pt)
    pt_plain = ck.empty_u32((count, limbs, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(z), count, limbs, delta, pt_plain)
    plain = ck.to_host_u32(pt_plain)
    assert np.all(got.astype(np.uint64) < np.array(qs, dtype=np.uint64)[None, :, None]), "a word outside [0, q)"
    others = np.setdiff1d(np.arange(count), wide)
    assert np.array_equal(got[others], plain[others]), "a fitting vector changed beside wide ones"
    one = ck.empty_u32((1, limbs, n))
    for v in wide:
        ck.ckks_linear_encode_poly(ctx, ck.to_device(z_mixed[v:v + 1]), 1, limbs, delta, one)
        assert np.array_equal(got[v], ck.to_host_u32(one)[0]), f"wide vector {v} differs from its own encoding"
    for v in (wide[0], wide[3], wide[-1]):
        want = OE.encode_poly(z_mixed[v:v + 1], delta, qs, psis, log_n).astype(np.uint32)
        assert np.max(np.abs(OE.round_coeffs(OE.encode_coeffs(z_mixed[v:v + 1], log_n), delta))) >= 2 ** 31
        sl_got = _decode_rows(got[v:v + 1], qs, psis, log_n, delta)
        sl_want = _decode_rows(want, qs, psis, log_n, delta)
        err = np.max(np.abs(sl_got - sl_want))
        assert err <= 2.0 ** -20 * max(1.0, np.max(np.abs(sl_want))), (v, err)


def test_tiny_layer_end_to_end(gpu_lib):
    """Tiny encrypted layer: GPU encode + MAC + rescale bit-exact, then decrypts to W.x."""
    ck = gpu_lib
    cfg = get("c1")
    layer = build_layer(cfg)
    ctx = ctx_for(ck, cfg.log_n, cfg.limbs)
    L, n = cfg.limbs, cfg.n
    w_enc = ck.empty_u32((cfg.d_out, cfg.d_in, L))
    ck.ckks_linear_encode_scalar(ctx, ck.to_device(layer.W), cfg.d_out, cfg.d_in, L, cfg.scale, w_enc)
    want_w = OE.encode_scalar(layer.W, cfg.scale, layer.qs)
    assert np.array_equal(ck.to_host_u32(w_enc), want_w.astype(np.uint32))
    for algo in (ck.CKKS_MAC_VALU, ck.CKKS_MAC_AUTO):
        ck.ckks_ctx_set_mac_algo(ctx, algo)
        ws = ck.empty_u32((max(16, ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, 16, 16, L)) // 4,))
        mac = ck.empty_u32((cfg.d_out, 2, L, n))
        ck.ckks_linear_mac_scalar(ctx, w_enc, ck.to_device(layer.ct), mac, cfg.d_out, cfg.d_in, L, ws)
        want_mac = OL.mac_scalar(want_w, layer.ct, layer.qs)
        assert np.array_equal(ck.to_host_u32(mac), want_mac.astype(np.uint32))
    ck.ckks_ctx_set_mac_algo(ctx, ck.CKKS_MAC_AUTO)
    res = ck.empty_u32((cfg.d_out, 2, L - 1, n))
    ck.ckks_rescale(ctx, mac, res, cfg.d_out, L)
    got = ck.to_host_u32(res)
    assert np.array_equal(got, OL.rescale(want_mac, layer.qs, layer.psis, cfg.log_n).astype(np.uint32))
    scale_out = ck.ckks_rescaled_scale(ctx, cfg.scale * cfg.scale, L)
    assert scale_out == cfg.scale * cfg.scale / layer.qs[-1]
    chk = check_decrypted(layer, got, range(cfg.d_out), layer.W @ layer.X, scale_out)
    assert chk["ok"], chk


def test_full_polynomial_twin_end_to_end(gpu_lib):
    """N=2^10, L=3, 8 -> 8 full-polynomial weights encoded on the GPU, MAC, rescale, decrypt."""
    ck = gpu_lib
    cfg = get("c5")
    log_n, L, d = 10, 3, 8
    layer = build_layer(cfg, log_n=log_n, limbs=L, d_in=d, d_out=d)
    ctx = ctx_for(ck, log_n, L)
    n = 1 << log_n
    pt = ck.empty_u32((d, d, L, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(np.ascontiguousarray(layer.W)), d * d, L, cfg.scale, pt)
    pt_h = ck.to_host_u32(pt)
    mac = ck.empty_u32((d, 2, L, n))
    ck.ckks_linear_mac_poly(ctx, pt, ck.to_device(layer.ct), mac, d, d, L)
    want_mac = OL.mac_poly(pt_h, layer.ct, layer.qs)                      # oracle MAC on the GPU's plaintext
    assert np.array_equal(ck.to_host_u32(mac), want_mac.astype(np.uint32))
    res = ck.empty_u32((d, 2, L - 1, n))
    ck.ckks_rescale(ctx, mac, res, d, L)
    got = ck.to_host_u32(res)
    assert np.array_equal(got, OL.rescale(want_mac, layer.qs, layer.psis, log_n).astype(np.uint32))
    scale_out = cfg.scale * cfg.scale / layer.qs[-1]
    ref = np.einsum("jis,is->js", layer.W, layer.X)
    chk = check_decrypted(layer, got, range(d), ref, scale_out)
    assert chk["ok"], chk
