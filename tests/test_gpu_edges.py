"""GPU parity at the edges of the kernels' tilings and arithmetic bounds.

* The matrix-core MAC over several row, column and k tiles with ragged tails
  in every dimension, on both sides of the d_in at which its contraction
  changes form, with three- and four-digit weight tiles mixed, and at the
  largest d_in its exact epilogue allows
  (4096), with operands that make the shift-class sums as large as valid
  residues can; one past that limit the library refuses the matrix-core path
  and its automatic choice takes the VALU kernel.
* Rescale at the largest chain (16 limbs) and, at N = 2^16, over more
  polynomials than one staging chunk holds (a ragged second chunk).
* The poly MAC with an output count that is not a multiple of its row group.

Everything is compared with the CPU oracle, bit for bit.
"""
import numpy as np
import pytest

from oracle import linear as OL
from workloads import gen

pytestmark = pytest.mark.gpu

_CTX = {}


def ctx_for(ck, log_n, limbs):
    key = (log_n, limbs)
    if key not in _CTX:
        _CTX[key] = ck.Context(log_n, limbs)
    return _CTX[key]


def residues(seed, prefix, qs, n):
    return gen.uniform_residues(np.random.default_rng(seed), prefix, qs, n)


def run_mac(ck, ctx, w, ct, d_out, d_in, limbs, algo):
    ck.ckks_ctx_set_mac_algo(ctx, algo)
    try:
        ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d_out, d_in, limbs)
        ws = ck.empty_u32((max(ws_bytes, 16) // 4 + 4,))
        out = ck.empty_u32((d_out, 2, limbs, ctx.n))
        ck.ckks_linear_mac_scalar(ctx, ck.to_device(w), ck.to_device(ct), out, d_out, d_in, limbs, ws)
        return ck.to_host_u32(out)
    finally:
        ck.ckks_ctx_set_mac_algo(ctx, ck.CKKS_MAC_AUTO)


@pytest.mark.parametrize("algo", ["valu", "mfma"])
def test_mac_scalar_multitile_ragged(gpu_lib, algo):
    """300 outputs (3 row tiles, the last 44 rows), 200 inputs (4 k-steps, the
    last 8 deep), 64 column tiles, 3 limbs; general residues as weights."""
    ck = gpu_lib
    log_n, limbs, d_in, d_out = 10, 3, 200, 300
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    rng = np.random.default_rng(4242)
    w = np.stack([rng.integers(0, q, (d_out, d_in), dtype=np.uint64) for q in qs], -1).astype(np.uint32)
    ct = residues(4243, (d_in, 2), qs, n)
    got = run_mac(ck, ctx, w, ct, d_out, d_in, limbs, ck.CKKS_MAC_VALU if algo == "valu" else ck.CKKS_MAC_MFMA)
    assert np.array_equal(got, OL.mac_scalar(w, ct, qs).astype(np.uint32))


@pytest.mark.parametrize("d_in,d_out", [(1024, 300), (1025, 150)])
def test_mac_mfma_both_contraction_forms(gpu_lib, d_in, d_out):
    """d_in = 1024 is the largest the column-stationary contraction takes (16
    k-steps held in LDS; 10 wave tiles of 32 rows, so two of the 8 waves take a
    second one, the last 12 rows deep); d_in = 1025 the smallest the streamed
    contraction takes (17 k-steps, the last one row deep).  The 32-row wave
    tiles alternate between small centred weights (three digits) and general
    residues (four digits)."""
    ck = gpu_lib
    log_n, limbs = 10, 2
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    rng = np.random.default_rng(d_in * 7 + d_out)
    small = rng.integers(-0x7F7F7F, 0x7F7F7F + 1, (d_out, d_in), dtype=np.int64)
    w = np.stack([np.mod(small, q) for q in qs], -1).astype(np.uint32)
    general = np.stack([rng.integers(0, q, (d_out, d_in), dtype=np.uint64) for q in qs], -1).astype(np.uint32)
    odd_tile = (np.arange(d_out) // 32) % 2 == 1
    w[odd_tile] = general[odd_tile]
    ct = residues(d_in + 1, (d_in, 2), qs, n)
    got = run_mac(ck, ctx, w, ct, d_out, d_in, limbs, ck.CKKS_MAC_MFMA)
    assert np.array_equal(got, OL.mac_scalar(w, ct, qs).astype(np.uint32))


@pytest.mark.parametrize("case", ["most_negative", "most_positive", "random"])
def test_mac_mfma_at_the_exactness_bound(gpu_lib, case):
    """d_in = 4096, the largest the exact digit-split epilogue allows.  Weights
    whose centred values are -(q-1)/2 or (q-1)/2 (four large digits) against
    residues q - 1 drive every shift-class sum to its largest magnitude for
    valid inputs; random residues cover general digit patterns."""
    ck = gpu_lib
    log_n, limbs, d_in, d_out = 10, 2, 4096, 16
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    if case == "random":
        rng = np.random.default_rng(77)
        w = np.stack([rng.integers(0, q, (d_out, d_in), dtype=np.uint64) for q in qs], -1).astype(np.uint32)
        ct = residues(78, (d_in, 2), qs, n)
    else:
        wv = [(q + 1) // 2 if case == "most_negative" else (q - 1) // 2 for q in qs]
        w = np.empty((d_out, d_in, limbs), dtype=np.uint32)
        w[:] = np.array(wv, dtype=np.uint32)
        ct = np.empty((d_in, 2, limbs, n), dtype=np.uint32)
        ct[:] = (np.array(qs, dtype=np.uint32) - 1)[:, None]
    got = run_mac(ck, ctx, w, ct, d_out, d_in, limbs, ck.CKKS_MAC_MFMA)
    assert np.array_equal(got, OL.mac_scalar(w, ct, qs).astype(np.uint32))


def test_mac_above_the_matrix_core_limit(gpu_lib):
    """d_in = 4097: the matrix-core path is refused; the automatic choice runs
    the VALU kernel and is exact."""
    ck = gpu_lib
    log_n, limbs, d_in, d_out = 10, 1, 4097, 2
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    rng = np.random.default_rng(99)
    w = rng.integers(0, qs[0], (d_out, d_in, 1), dtype=np.uint64).astype(np.uint32)
    ct = residues(100, (d_in, 2), qs[:1], n)
    with pytest.raises(ck.CkksError) as e:
        run_mac(ck, ctx, w, ct, d_out, d_in, limbs, ck.CKKS_MAC_MFMA)
    assert e.value.code == ck.CKKS_E_UNSUPPORTED
    assert ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d_out, d_in, limbs) == 0
    got = run_mac(ck, ctx, w, ct, d_out, d_in, limbs, ck.CKKS_MAC_AUTO)
    assert np.array_equal(got, OL.mac_scalar(w, ct, qs[:1]).astype(np.uint32))


def test_rescale_longest_chain(gpu_lib):
    ck = gpu_lib
    log_n, limbs, count = 10, 16, 2
    ctx = ctx_for(ck, log_n, limbs)
    qs, psis, n = ctx.moduli, ctx.roots, ctx.n
    ct = residues(1616, (count, 2), qs, n)
    out = ck.empty_u32((count, 2, limbs - 1, n))
    ck.ckks_rescale(ctx, ck.to_device(ct), out, count, limbs)
    assert np.array_equal(ck.to_host_u32(out), OL.rescale(ct, qs, psis, log_n).astype(np.uint32))


def test_rescale_n16_across_staging_chunks(gpu_lib):
    """130 ciphertexts = 260 polynomials at N = 2^16: one full staging chunk of
    256 and a ragged one of 4; sampled ciphertexts from both are checked."""
    ck = gpu_lib
    log_n, limbs, count = 16, 3, 130
    ctx = ctx_for(ck, log_n, limbs)
    qs, psis, n = ctx.moduli, ctx.roots, ctx.n
    ct = residues(6516, (count, 2), qs, n)
    ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_RESCALE, count, 0, limbs)
    ws = ck.empty_u32((ws_bytes // 4,))
    out = ck.empty_u32((count, 2, limbs - 1, n))
    ck.ckks_rescale(ctx, ck.to_device(ct), out, count, limbs, ws)
    got = ck.to_host_u32(out)
    for b in (0, 127, 128, 129):
        want = OL.rescale(ct[b:b + 1], qs, psis, log_n)[0].astype(np.uint32)
        assert np.array_equal(got[b], want), f"ciphertext {b}"


def test_mac_poly_ragged_row_group(gpu_lib):
    """7 outputs of a narrow launch (the two-row kernel): three full groups of
    two rows and a ragged group of one."""
    ck = gpu_lib
    log_n, limbs, d_in, d_out = 11, 2, 6, 7
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    pt = residues(71, (d_out, d_in), qs, n)
    ct = residues(72, (d_in, 2), qs, n)
    out = ck.empty_u32((d_out, 2, limbs, n))
    ck.ckks_linear_mac_poly(ctx, ck.to_device(pt), ck.to_device(ct), out, d_out, d_in, limbs)
    assert np.array_equal(ck.to_host_u32(out), OL.mac_poly(pt, ct, qs).astype(np.uint32))


def test_mac_poly_wide_launch_ragged_row_group(gpu_lib):
    """87 outputs at N = 2^14, 6 limbs: 22 row groups x 96 (limb, slot block)
    workgroups fill 8 per CU on 256 CUs, so the four-row kernel runs (its
    non-temporal plaintext loads); the last group has three rows, and its
    missing row's loads re-read row 0, whose sums must not be stored."""
    ck = gpu_lib
    log_n, limbs, d_in, d_out = 14, 6, 2, 87
    ctx = ctx_for(ck, log_n, limbs)
    qs, n = ctx.moduli, ctx.n
    pt = residues(73, (d_out, d_in), qs, n)
    ct = residues(74, (d_in, 2), qs, n)
    out = ck.empty_u32((d_out + 1, 2, limbs, n))
    out.fill_(-1)  # a guard ciphertext past the last output stays untouched
    ck.ckks_linear_mac_poly(ctx, ck.to_device(pt), ck.to_device(ct), out, d_out, d_in, limbs)
    got = ck.to_host_u32(out)
    assert np.array_equal(got[:d_out], OL.mac_poly(pt, ct, qs).astype(np.uint32))
    assert np.all(got[d_out] == 0xFFFFFFFF)


def _expect_invalid(ck, fn, *args, **kw):
    with pytest.raises(ck.CkksError) as e:
        fn(*args, **kw)
    assert e.value.code == ck.CKKS_E_INVALID_ARG, e.value


def test_overlapping_outputs_are_rejected(gpu_lib):
    """Outputs that share bytes with an input (in place, or offset by one
    ciphertext) and workspaces that share bytes with a data buffer are refused on
    the host with CKKS_E_INVALID_ARG, before any launch."""
    import torch
    ck = gpu_lib
    log_n, L, d = 10, 3, 4
    ctx = ctx_for(ck, log_n, L)
    n = ctx.n
    ct_words = 2 * L * n
    big = ck.empty_u32((4 * d * ct_words,))
    w = ck.empty_u32((d, d, L))
    ws_bytes = ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d, d, L)
    ws = ck.empty_u32((ws_bytes // 4 + 4,))
    ct_in = big[: d * ct_words]
    mac = ck.ckks_linear_mac_scalar
    _expect_invalid(ck, mac, ctx, w, ct_in, ct_in, d, d, L, ws)                                  # in place
    _expect_invalid(ck, mac, ctx, w, ct_in, big[ct_words: (d + 1) * ct_words], d, d, L, ws)      # partial
    w_words = ck.empty_u32((d * ct_words,))
    _expect_invalid(ck, mac, ctx, w_words[: d * d * L], ck.empty_u32((d * ct_words,)), w_words, d, d, L, ws)
    out = big[d * ct_words: 2 * d * ct_words]
    _expect_invalid(ck, mac, ctx, w, ct_in, out, d, d, L, big[2 * d * ct_words - 8:])           # ws over ct_out
    _expect_invalid(ck, mac, ctx, w, ct_in, out, d, d, L, big[: ws_bytes // 4 + 4])            # ws over ct_in
    pt = ck.empty_u32((d, d, L, n))
    _expect_invalid(ck, ck.ckks_linear_mac_poly, ctx, pt, ct_in, ct_in, d, d, L)
    _expect_invalid(ck, ck.ckks_linear_mac_poly, ctx, pt, ct_in, big[ct_words: (d + 1) * ct_words], d, d, L)
    _expect_invalid(ck, ck.ckks_linear_mac_poly, ctx, pt, ct_in, pt.view(-1)[: d * ct_words], d, d, L)
    _expect_invalid(ck, ck.ckks_rescale, ctx, ct_in, ct_in, d, L)
    _expect_invalid(ck, ck.ckks_rescale, ctx, ct_in, big[ct_words // 2: ct_words // 2 + d * 2 * (L - 1) * n], d, L)
    wf = ck.empty_u32((2 * d * d * L,))
    _expect_invalid(ck, ck.ckks_linear_encode_scalar, ctx, wf.view(torch.float64), d, d, L, 2.0 ** 20, wf[: d * d * L])
    slots = torch.empty((2, n // 2), dtype=torch.float64, device="cuda")
    _expect_invalid(ck, ck.ckks_linear_encode_poly, ctx, slots, 2, 1, 2.0 ** 20, slots.view(torch.int32))
    # disjoint buffers still work
    mac(ctx, w, ct_in, out, d, d, L, ws)


def test_mac_rejects_oversized_d_in(gpu_lib):
    """d_in above 2^24 is refused on the host (CKKS_E_INVALID_ARG); the shape check
    runs before any buffer is looked at, so tiny buffers suffice."""
    import ctypes
    ck = gpu_lib
    ctx = ctx_for(ck, 10, 2)
    buf = ck.empty_u32((64,))
    rc = ck._lib.ckks_linear_mac_scalar(ctx.handle, ctypes.c_void_p(buf.data_ptr()), ctypes.c_void_p(buf.data_ptr()),
                                        ctypes.c_void_p(buf.data_ptr() + 128), 1, (1 << 24) + 1, 2, None, 0,
                                        ctypes.c_void_p(0))
    assert rc == ck.CKKS_E_INVALID_ARG
    assert "d_in" in ck.ckks_last_error()
