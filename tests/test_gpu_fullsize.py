"""GPU parity at the full workload sizes, in the launch configuration bench.py
times (default MAC kernel, i.e. the int8 matrix-core path).

The oracle cannot evaluate whole layers of this size, so outputs are checked
on seeded samples (first row, last row and random rows, each on all
components, limbs and NTT slots), computed one by one by the oracle, plus
properties over every output (all residues reduced, NTT round trips).
Inputs are the same seeded draws bench.py uses.
"""
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

from oracle import encode as OE
from oracle import linear as OL
from oracle import ntt as ON
from oracle import params as OP
from tests.cases import build_layer, check_decrypted
from workloads import gen, get

pytestmark = pytest.mark.gpu
POOL = 16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _rows_host(ck, t, rows):
    import torch
    idx = torch.tensor(rows, device=t.device)
    return ck.to_host_u32(t.index_select(0, idx).contiguous())


def _all_reduced(t, qs, limb_axis=2):
    """Every residue of a [count][2][limbs][N] device tensor is below its modulus."""
    import torch
    for l, q in enumerate(qs):
        v = t.select(limb_axis, l).view(torch.int32)
        if int(v.min()) < 0 or int(v.max()) >= q:
            return False
    return True


@pytest.mark.parametrize("key", ["c2", "c3", "c4"])
def test_scalar_layer_full_size(gpu_lib, key):
    import torch
    ck = gpu_lib
    cfg = get(key)
    t0 = time.time()
    ctx = ck.Context(cfg.log_n, cfg.limbs)
    qs = ctx.moduli
    assert qs == OP.moduli(cfg.log_n, cfg.limbs)
    psis = list(ctx.roots)
    st = gen.streams(cfg.index)
    W = gen.scalar_weights(st["weights"], cfg.d_out, cfg.d_in)
    ct = gen.uniform_residues(st["residues"], (cfg.d_in, 2), qs, cfg.n)
    rows = gen.sample_rows(st["sample"], cfg.d_out)
    say(f"[{key}] inputs ready {time.time() - t0:.1f}s rows={rows}")
    L, n = cfg.limbs, cfg.n
    w_enc = ck.empty_u32((cfg.d_out, cfg.d_in, L))
    ck.ckks_linear_encode_scalar(ctx, ck.to_device(W), cfg.d_out, cfg.d_in, L, cfg.scale, w_enc)
    d_ct = ck.to_device(ct)
    mac = ck.empty_u32((cfg.d_out, 2, L, n))
    ws = ck.empty_u32((ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, cfg.d_out, cfg.d_in, L) // 4 + 4,))
    ck.ckks_linear_mac_scalar(ctx, w_enc, d_ct, mac, cfg.d_out, cfg.d_in, L, ws)
    res = ck.empty_u32((cfg.d_out, 2, L - 1, n))
    wr = ck.empty_u32((max(16, ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_RESCALE, cfg.d_out, 0, L)) // 4,))
    ck.ckks_rescale(ctx, mac, res, cfg.d_out, L, wr)
    torch.cuda.synchronize()
    say(f"[{key}] gpu done {time.time() - t0:.1f}s")
    w_ref = OE.encode_scalar(W, cfg.scale, qs)
    assert np.array_equal(ck.to_host_u32(w_enc), w_ref.astype(np.uint32))
    mac_rows = _rows_host(ck, mac, rows)
    res_rows = _rows_host(ck, res, rows)
    assert _all_reduced(mac, qs) and _all_reduced(res, qs[:-1])
    with ThreadPoolExecutor(POOL) as ex:
        refs = list(ex.map(lambda j: OL.mac_scalar(w_ref, ct, qs, rows=[j])[0], rows))
    say(f"[{key}] oracle MAC done {time.time() - t0:.1f}s")
    for r, j in enumerate(rows):
        assert np.array_equal(mac_rows[r], refs[r].astype(np.uint32)), f"MAC row {j}"
    with ThreadPoolExecutor(POOL) as ex:
        rres = list(ex.map(lambda r: OL.rescale(refs[r][None], qs, psis, cfg.log_n)[0], range(len(rows))))
    say(f"[{key}] oracle rescale of all {len(rows)} sampled rows done {time.time() - t0:.1f}s")
    for r, j in enumerate(rows):
        assert np.array_equal(res_rows[r], rres[r].astype(np.uint32)), f"rescale row {j}"

    if key == "c3":
        # standalone batched transforms over all 3072*2*6 output polynomials
        polys = mac.clone()
        count = cfg.d_out * 2
        ck.ckks_intt(ctx, polys, count, L)
        back = polys.clone()
        ck.ckks_ntt(ctx, back, count, L)
        torch.cuda.synchronize()
        assert torch.equal(back, mac), "NTT(INTT(x)) != x"
        inv_rows = _rows_host(ck, polys, rows)
        rng = np.random.default_rng(33)
        picks = [(r, c, l) for r in range(len(rows)) for c in range(2) for l in range(L)]
        picks = [picks[i] for i in rng.choice(len(picks), size=64, replace=False)]
        with ThreadPoolExecutor(POOL) as ex:
            outs = list(ex.map(lambda p: ON.intt(mac_rows[p[0], p[1], p[2]].astype(np.uint64), qs[p[2]],
                                                 psis[p[2]], cfg.log_n), picks))
        for p, want in zip(picks, outs):
            assert np.array_equal(inv_rows[p[0], p[1], p[2]], want), f"intt {p}"
        say(f"[{key}] standalone NTT/INTT checked {time.time() - t0:.1f}s")
    ctx.close()


def test_fallback_layer_full_size(gpu_lib):
    """The full-polynomial layer (64 x 64 slot-vector weights, N = 2^15, 6 limbs, scale
    2^30) encoded on the GPU per call, MAC, rescale."""
    import torch
    ck = gpu_lib
    cfg = get("c5")
    t0 = time.time()
    layer = build_layer(cfg)                                    # encrypted inputs (oracle encoder/encryptor)
    say(f"[c5] inputs ready {time.time() - t0:.1f}s")
    ctx = ck.Context(cfg.log_n, cfg.limbs)
    assert ctx.moduli == layer.qs
    L, n, d = cfg.limbs, cfg.n, cfg.d_in
    pt = ck.empty_u32((d, d, L, n))
    ck.ckks_linear_encode_poly(ctx, ck.to_device(np.ascontiguousarray(layer.W)), d * d, L, cfg.scale, pt)
    mac = ck.empty_u32((d, 2, L, n))
    ck.ckks_linear_mac_poly(ctx, pt, ck.to_device(layer.ct), mac, d, d, L)
    res = ck.empty_u32((d, 2, L - 1, n))
    ck.ckks_rescale(ctx, mac, res, d, L)
    torch.cuda.synchronize()
    say(f"[c5] gpu done {time.time() - t0:.1f}s")
    pt_h = ck.to_host_u32(pt)
    mac_h = ck.to_host_u32(mac)
    res_h = ck.to_host_u32(res)
    # encode: 16 sampled weights against the O(N^2) oracle, compared on coefficients
    rng = gen.streams(cfg.index)["sample"]
    picks = sorted(set([0, d * d - 1] + [int(x) for x in rng.choice(d * d, size=14, replace=False)]))
    zs = layer.W.reshape(d * d, n // 2)[picks]
    p_ref = OE.round_coeffs(OE.encode_coeffs(zs, cfg.log_n), cfg.scale)            # (16, N) signed
    diff_l1 = 0
    for r, w in enumerate(picks):
        coef0 = ON.intt(pt_h.reshape(d * d, L, n)[w, 0].astype(np.uint64), layer.qs[0], layer.psis[0], cfg.log_n)
        got = np.where(coef0 > layer.qs[0] // 2, coef0.astype(np.int64) - layer.qs[0], coef0.astype(np.int64))
        diff_l1 = max(diff_l1, int(np.abs(got - p_ref[r]).sum()))
        for l in range(1, L):      # every limb holds the same integer polynomial
            cl = ON.intt(pt_h.reshape(d * d, L, n)[w, l].astype(np.uint64), layer.qs[l], layer.psis[l], cfg.log_n)
            assert np.array_equal(cl, np.mod(got, layer.qs[l]).astype(np.uint64))
    # |slot error| <= sum_k |coefficient difference| / Delta (|zeta^k| = 1)
    bound = diff_l1 / cfg.scale
    say(f"[c5] encode: max L1 coefficient difference {diff_l1}, slot error bound {bound:.3g}")
    assert bound <= 2.0 ** -20 * max(1.0, float(np.abs(zs).max()))
    # MAC: every output against the oracle on the GPU's plaintexts
    with ThreadPoolExecutor(POOL) as ex:
        refs = list(ex.map(lambda j: OL.mac_poly(pt_h, layer.ct, layer.qs, rows=[j])[0], range(d)))
    for j in range(d):
        assert np.array_equal(mac_h[j], refs[j].astype(np.uint32)), f"MAC row {j}"
    say(f"[c5] oracle MAC done {time.time() - t0:.1f}s")
    with ThreadPoolExecutor(POOL) as ex:
        rres = list(ex.map(lambda j: OL.rescale(refs[j][None], layer.qs, layer.psis, cfg.log_n)[0], range(d)))
    for j in range(d):
        assert np.array_equal(res_h[j], rres[j].astype(np.uint32)), f"rescale row {j}"
    say(f"[c5] oracle rescale of all {d} outputs done {time.time() - t0:.1f}s")
    sub = [0, 17, 40, d - 1]
    # decrypt sampled outputs: slot-wise sum_i W[j,i] * x_i within the rescale noise
    scale_out = cfg.scale * cfg.scale / layer.qs[-1]
    ref = np.stack([np.einsum("is,is->s", layer.W[j], layer.X) for j in sub])
    chk = check_decrypted(layer, res_h[sub], sub, ref, scale_out)
    say(f"[c5] decrypt check {chk} {time.time() - t0:.1f}s")
    assert chk["ok"], chk
    ctx.close()


def test_fallback_encode_every_weight_constant_slots(gpu_lib):
    """The full-polynomial layer's shape, every one of its 64 x 64 weights through the full-polynomial
    encode on a call of its own: with constant slot vectors (slot value W[j, i]) the
    encoding is the constant polynomial rint(W[j, i] scale), whose NTT is that constant
    in every slot, i.e. exactly the scalar encoding.  So all 4096 plaintexts must equal
    the oracle's scalar encodings broadcast over the N slots, and the poly MAC over them
    must equal the scalar MAC bit for bit on all 64 outputs (and the oracle's scalar MAC
    on sampled outputs)."""
    import torch
    ck = gpu_lib
    cfg = get("c5")
    t0 = time.time()
    ctx = ck.Context(cfg.log_n, cfg.limbs)
    qs = ctx.moduli
    L, n, d = cfg.limbs, cfg.n, cfg.d_in
    st = gen.streams(cfg.index, 77)
    Wc = gen.scalar_weights(st["weights"], d, d)                        # (64, 64) N(0, 0.02^2)
    ct = gen.uniform_residues(st["residues"], (d, 2), qs, n)
    w_ref = OE.encode_scalar(Wc, cfg.scale, qs)                          # (64, 64, L) oracle
    slots = ck.to_device(Wc.reshape(d * d, 1)).expand(d * d, n // 2).contiguous()
    pt = ck.empty_u32((d, d, L, n))
    ck.ckks_linear_encode_poly(ctx, slots, d * d, L, cfg.scale, pt)
    del slots
    want = ck.to_device(w_ref.astype(np.uint32)).view(d, d, L, 1)
    bad = int((pt != want).sum())
    say(f"[c5 constant slots] {d * d} weights x {L} limbs x {n} slots encoded; mismatches {bad} "
        f"{time.time() - t0:.1f}s")
    assert bad == 0
    d_ct = ck.to_device(ct)
    out_poly = ck.empty_u32((d, 2, L, n))
    ck.ckks_linear_mac_poly(ctx, pt, d_ct, out_poly, d, d, L)
    w_enc = ck.empty_u32((d, d, L))
    ck.ckks_linear_encode_scalar(ctx, ck.to_device(Wc), d, d, L, cfg.scale, w_enc)
    ws = ck.empty_u32((ck.ckks_workspace_bytes(ctx, ck.CKKS_OP_MAC_SCALAR, d, d, L) // 4 + 4,))
    out_scalar = ck.empty_u32((d, 2, L, n))
    ck.ckks_linear_mac_scalar(ctx, w_enc, d_ct, out_scalar, d, d, L, ws)
    torch.cuda.synchronize()
    assert np.array_equal(ck.to_host_u32(w_enc), w_ref.astype(np.uint32))
    assert torch.equal(out_poly, out_scalar), "poly MAC over constant-slot plaintexts != scalar MAC"
    rows = gen.sample_rows(st["sample"], d, count=4)
    got = _rows_host(ck, out_poly, rows)
    with ThreadPoolExecutor(POOL) as ex:
        refs = list(ex.map(lambda j: OL.mac_scalar(w_ref, ct, qs, rows=[j])[0], rows))
    for r, j in enumerate(rows):
        assert np.array_equal(got[r], refs[r].astype(np.uint32)), f"MAC row {j}"
    say(f"[c5 constant slots] poly MAC = scalar MAC on all {d} outputs, oracle rows {rows} "
        f"{time.time() - t0:.1f}s")
    ctx.close()
