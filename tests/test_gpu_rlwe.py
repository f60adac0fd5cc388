"""GPU parity of the batched RLWE entry points (encrypt, decrypt and the
decrypt-then-encrypt refresh of section 3.2) against the oracle, bit for bit.

Inputs come from the seeded generators.  The secret and the plaintext are
taken to NTT form on the GPU with ckks_ntt (the library's own API); every
expected value is computed by the oracle from the host-side integers alone.
"""
import numpy as np
import pytest

from oracle import linear as OL
from oracle import rlwe as OR
from workloads import gen

pytestmark = pytest.mark.gpu

_CTX = {}


def ctx_for(ck, log_n, limbs):
    key = (log_n, limbs)
    if key not in _CTX:
        _CTX[key] = ck.Context(log_n, limbs)
    return _CTX[key]


def residues_of(v, qs):
    """Integer array (..., N) -> residues (..., L, N) uint32."""
    v = np.asarray(v, dtype=np.int64)
    return np.stack([np.mod(v, q) for q in qs], axis=-2).astype(np.uint32)


def setup(ck, log_n, limbs, count, seed):
    ctx = ctx_for(ck, log_n, limbs)
    qs, psis, n = ctx.moduli, ctx.roots, ctx.n
    st = gen.streams(seed, log_n)
    s = gen.ternary_secret(st["secret"], n)
    s_ntt = ck.to_device(residues_of(s, qs))
    ck.ckks_ntt(ctx, s_ntt, 1, limbs)
    m = st["activations"].integers(-2**40, 2**40, (count, n))
    e = gen.gaussian_error(st["error"], (count, n)).astype(np.int32)
    a = gen.uniform_residues(st["residues"], (count,), qs, n)
    return ctx, qs, psis, n, st, s, s_ntt, m, e, a


@pytest.mark.parametrize("log_n,limbs,count", [(10, 3, 5), (14, 4, 3), (16, 3, 2)])
def test_encrypt_bit_exact(gpu_lib, log_n, limbs, count):
    ck = gpu_lib
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, limbs, count, 300 + log_n)
    pt = ck.to_device(residues_of(m, qs))
    ck.ckks_ntt(ctx, pt, count, limbs)
    ct = ck.empty_u32((count, 2, limbs, n))
    ck.ckks_encrypt(ctx, pt, s_ntt, ck.to_device(a), ck.to_device(e), count, limbs, ct)
    want = OR.encrypt(m, s, a, e, qs, psis, log_n).astype(np.uint32)
    assert np.array_equal(ck.to_host_u32(ct), want)


def test_encrypt_zero_plaintext(gpu_lib):
    ck = gpu_lib
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, 11, 2, 3, 311)
    ct = ck.empty_u32((3, 2, 2, n))
    ck.ckks_encrypt(ctx, None, s_ntt, ck.to_device(a), ck.to_device(e), 3, 2, ct)
    want = OR.encrypt(np.zeros((3, n), dtype=np.int64), s, a, e, qs, psis, 11).astype(np.uint32)
    assert np.array_equal(ck.to_host_u32(ct), want)


@pytest.mark.parametrize("log_n,limbs,count", [(10, 2, 4), (14, 4, 3), (16, 2, 2)])
def test_decrypt_bit_exact(gpu_lib, log_n, limbs, count):
    ck = gpu_lib
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, limbs, count, 320 + log_n)
    ct = OR.encrypt(m, s, a, e, qs, psis, log_n).astype(np.uint32)
    out = ck.empty_u32((count, limbs, n))
    ck.ckks_decrypt(ctx, ck.to_device(ct), s_ntt, count, limbs, out)
    got = ck.to_host_u32(out)
    for b in range(count):
        assert np.array_equal(got[b], OR.decrypt_residues(ct[b], s, qs, psis, log_n).astype(np.uint32)), b
    # and the residues are those of the integer polynomial m + e
    assert np.array_equal(got, residues_of(m + e, qs))


# Routes on 256 CUs: fused for N <= 2^13 with at most 256 (ciphertext, output limb) pairs
# (64 x 4 at 2^13 is the largest), the two-kernel route otherwise (every 2^14 and
# 2^15 case), pointwise passes at 2^16.
@pytest.mark.parametrize("log_n,L,limbs_in,limbs_out,count", [(10, 4, 2, 4, 4), (14, 4, 3, 4, 3), (12, 5, 4, 2, 2),
                                                              (16, 3, 2, 3, 2), (10, 3, 2, 3, 160), (13, 4, 3, 4, 200),
                                                              (13, 4, 3, 4, 64), (15, 5, 3, 5, 3)])
def test_refresh_bit_exact(gpu_lib, log_n, L, limbs_in, limbs_out, count):
    ck = gpu_lib
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, L, count, 340 + log_n)
    ct = OR.encrypt(m, s, a[:, :limbs_in], e, qs[:limbs_in], psis[:limbs_in], log_n).astype(np.uint32)
    a2 = gen.uniform_residues(st["residues"], (count,), qs[:limbs_out], n)
    e2 = gen.gaussian_error(st["error"], (count, n)).astype(np.int32)
    out = ck.empty_u32((count, 2, limbs_out, n))
    ck.ckks_refresh(ctx, ck.to_device(ct), limbs_in, s_ntt, ck.to_device(a2), ck.to_device(e2), count, limbs_out, out)
    want = OR.refresh(ct, s, a2, e2, qs, psis, log_n, limbs_out).astype(np.uint32)
    assert np.array_equal(ck.to_host_u32(out), want)


def test_refresh_after_rescale_restores_the_level(gpu_lib):
    """The pipeline's use: a ciphertext rescaled to 2 limbs is refreshed back to
    4 limbs on the GPU; it equals the oracle's refresh of the oracle's rescale."""
    ck = gpu_lib
    log_n, L, count = 12, 4, 3
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, L, count, 361)
    ct = OR.encrypt(m * 2**20, s, a[:, :3], e, qs[:3], psis[:3], log_n).astype(np.uint32)
    r_dev = ck.empty_u32((count, 2, 2, n))
    ck.ckks_rescale(ctx, ck.to_device(ct), r_dev, count, 3)
    a2 = gen.uniform_residues(st["residues"], (count,), qs, n)
    e2 = gen.gaussian_error(st["error"], (count, n)).astype(np.int32)
    out = ck.empty_u32((count, 2, L, n))
    ck.ckks_refresh(ctx, r_dev, 2, s_ntt, ck.to_device(a2), ck.to_device(e2), count, L, out)
    r_host = OL.rescale(ct, qs[:3], psis[:3], log_n)
    want = OR.refresh(r_host, s, a2, e2, qs, psis, log_n, L).astype(np.uint32)
    assert np.array_equal(ck.to_host_u32(out), want)


def test_round_trip_on_gpu(gpu_lib):
    """decrypt(encrypt(pt)) = NTT^-1(pt) + e, all on the GPU, at a ragged count."""
    ck = gpu_lib
    log_n, limbs, count = 13, 3, 7
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, limbs, count, 371)
    pt = ck.to_device(residues_of(m, qs))
    ck.ckks_ntt(ctx, pt, count, limbs)
    ct = ck.empty_u32((count, 2, limbs, n))
    ck.ckks_encrypt(ctx, pt, s_ntt, ck.to_device(a), ck.to_device(e), count, limbs, ct)
    out = ck.empty_u32((count, limbs, n))
    ck.ckks_decrypt(ctx, ct, s_ntt, count, limbs, out)
    assert np.array_equal(ck.to_host_u32(out), residues_of(m + e, qs))


def test_rlwe_argument_errors(gpu_lib):
    ck = gpu_lib
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, 10, 3, 2, 381)
    ct = ck.empty_u32((2, 2, 3, n))
    d_a, d_e = ck.to_device(a), ck.to_device(e)
    ck.ckks_encrypt(ctx, None, s_ntt, d_a, d_e, 0, 3, ct)                  # count 0: no-op
    with pytest.raises(ck.CkksError) as ex:
        ck.ckks_refresh(ctx, ct, 1, s_ntt, d_a, d_e, 2, 3, ck.empty_u32((2, 2, 3, n)))
    assert ex.value.code == ck.CKKS_E_INVALID_ARG                          # limbs_in < 2
    with pytest.raises(ck.CkksError) as ex:
        ck.ckks_refresh(ctx, ct, 3, s_ntt, d_a, d_e, 2, 3, ct)              # ct_out aliases ct_in
    assert ex.value.code == ck.CKKS_E_INVALID_ARG
    # limbs > L: rejected by the library itself (the binding's size checks would stop it first)
    import ctypes
    big = ck.empty_u32((2, 2, 4, n))
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    assert ck._lib.ckks_encrypt(ctx.handle, None, P(s_ntt), P(d_a), P(d_e), 2, 4, P(big), None) == ck.CKKS_E_INVALID_ARG
    assert "limbs=4" in ck.ckks_last_error()


def test_refresh_at_the_benchmarked_size(gpu_lib):
    """The refresh workload's shape: 768 ciphertexts at N = 2^14 refreshed from 3 to 4
    limbs (the two-kernel route); 16 sampled ciphertexts compared with the oracle bit
    for bit."""
    ck = gpu_lib
    log_n, L, count = 14, 4, 768
    ctx, qs, psis, n, st, s, s_ntt, m, e, a = setup(ck, log_n, L, count, 391)
    ct = gen.uniform_residues(st["residues"], (count, 2), qs[:3], n)       # any residues: exact arithmetic
    a2 = gen.uniform_residues(st["residues"], (count,), qs, n)
    e2 = gen.gaussian_error(st["error"], (count, n)).astype(np.int32)
    out = ck.empty_u32((count, 2, L, n))
    ck.ckks_refresh(ctx, ck.to_device(ct), 3, s_ntt, ck.to_device(a2), ck.to_device(e2), count, L, out)
    got = ck.to_host_u32(out)
    rows = gen.sample_rows(st["sample"], count, count=16)
    want = OR.refresh(ct[rows].astype(np.uint64), s, a2[rows], e2[rows], qs, psis, log_n, L).astype(np.uint32)
    assert np.array_equal(got[rows], want)
