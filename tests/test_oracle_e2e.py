"""The tiny 16 -> 16 layer (N = 2^10, 2 limbs) end to end on the oracle alone: encode + encrypt activations, scalar
weights, MAC, rescale, decrypt, decode, and compare with fp64 W.x within the
analytic noise bound (rescale rounding dominates: sd ~ 1.6e-4 per slot)."""
import numpy as np

from oracle import encode, linear
from tests.cases import build_layer, check_decrypted
from workloads import get


def test_tiny_layer_decrypts_to_w_times_x():
    cfg = get("c1")
    layer = build_layer(cfg)
    w_enc = encode.encode_scalar(layer.W, cfg.scale, layer.qs)
    out = linear.mac_scalar(w_enc, layer.ct, layer.qs)
    res = linear.rescale(out, layer.qs, layer.psis, cfg.log_n)
    scale_out = cfg.scale * cfg.scale / layer.qs[-1]
    ref = layer.W @ layer.X                                   # (d_out, N/2)
    chk = check_decrypted(layer, res, range(cfg.d_out), ref, scale_out)
    assert chk["ok"], chk
    assert 0.5 * chk["sd"] < chk["rms_re"]                    # the noise is really there


def test_full_polynomial_twin_decrypts_to_slotwise_products():
    """Full-polynomial weights: out_j = sum_i W[j,i] (.) x_i slot-wise."""
    cfg = get("c5")
    layer = build_layer(cfg, log_n=10, limbs=3, d_in=4, d_out=3)
    pt = encode.encode_poly(layer.W, cfg.scale, layer.qs, layer.psis, 10)
    out = linear.mac_poly(pt, layer.ct, layer.qs)
    res = linear.rescale(out, layer.qs, layer.psis, 10)
    scale_out = cfg.scale * cfg.scale / layer.qs[-1]
    ref = np.einsum("jis,is->js", layer.W, layer.X)
    chk = check_decrypted(layer, res, range(3), ref, scale_out)
    assert chk["ok"], chk
