"""Input builders shared by the oracle tests, the GPU parity tests and smoke().

Inputs come from the seeded generators in ``workloads.gen``; where a workload
needs real encryptions (configs 1 and 5 and their small twins) the CPU oracle
encodes and encrypts them.  Nothing here reads anything the GPU produced.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from oracle import encode, params, rlwe
from workloads import gen
from workloads.configs import Config


@dataclass
class Layer:
    log_n: int
    qs: tuple
    psis: list
    delta: float
    W: np.ndarray          # fp64 weights: (d_out, d_in) scalar or (d_out, d_in, N/2) slots
    X: np.ndarray | None   # fp64 activation slots (d_in, N/2) when encrypted
    s: np.ndarray | None   # secret (N,)
    ct: np.ndarray         # uint32 (d_in, 2, L, N) NTT form


def moduli_and_roots(log_n: int, limbs: int):
    qs = params.moduli(log_n, limbs)
    return qs, [params.psi(q, log_n) for q in qs]


def build_layer(cfg: Config, *, log_n=None, limbs=None, d_in=None, d_out=None,
                encrypted=None, seed_extra=()) -> Layer:
    """Inputs for `cfg`, optionally shrunk (a 'twin' with the same recipe)."""
    log_n = cfg.log_n if log_n is None else log_n
    limbs = cfg.limbs if limbs is None else limbs
    d_in = cfg.d_in if d_in is None else d_in
    d_out = cfg.d_out if d_out is None else d_out
    encrypted = cfg.encrypted if encrypted is None else encrypted
    n = 1 << log_n
    qs, psis = moduli_and_roots(log_n, limbs)
    st = gen.streams(cfg.index, *seed_extra)
    if cfg.weights == "scalar":
        W = gen.scalar_weights(st["weights"], d_out, d_in)
    else:
        W = gen.poly_weights(st["weights"], d_out, d_in, n // 2)
    if not encrypted:
        ct = gen.uniform_residues(st["residues"], (d_in, 2), qs, n)
        return Layer(log_n, qs, psis, cfg.scale, W, None, None, ct)
    X = gen.activations(st["activations"], d_in, n // 2)
    s = gen.ternary_secret(st["secret"], n)
    a = gen.uniform_residues(st["residues"], (d_in,), qs, n)
    e = gen.gaussian_error(st["error"], (d_in, n))
    m_all = encode.round_coeffs(encode.encode_coeffs(X, log_n), cfg.scale)     # (d_in, N), one pass
    ct = rlwe.encrypt(m_all, s, a, e, qs, psis, log_n).astype(np.uint32)       # (d_in, 2, L, N)
    return Layer(log_n, qs, psis, cfg.scale, W, X, s, ct)


def rescale_noise_sd(log_n: int, scale_out: float) -> float:
    """Per-slot std (real part) of the rescale rounding noise tau0 + tau1*s, ternary s,
    averaged over the secret: sqrt(N/2 * (N/18 + 1/12)) / scale."""
    n = 1 << log_n
    return float(np.sqrt(n / 2 * (n / 18 + 1 / 12)) / scale_out)


def slot_noise_sd(layer: Layer, scale_out: float) -> np.ndarray:
    """Per-slot std (real or imaginary part) of tau0(zeta_j) + tau1(zeta_j) s(zeta_j) given the secret.

    The rounding polynomials tau0, tau1 have independent U(-1/2, 1/2) coefficients, so
    tau(zeta) is close to a circular Gaussian with E|tau(zeta)|^2 = N/12; the product with
    the fixed value s(zeta_j) scales it by |s(zeta_j)|.  Unconditionally the error is a
    product of two near-Gaussians and has heavy tails, so the bound is taken per slot.
    """
    n = 1 << layer.log_n
    s_at = encode.decode([int(x) for x in layer.s], 1.0, layer.log_n)     # s(zeta_j)
    return np.sqrt(n / 24 * (1 + np.abs(s_at) ** 2)) / scale_out


def check_decrypted(layer: Layer, out_ct, rows, ref_slots, scale_out: float) -> dict:
    """Decrypt + decode rescaled outputs and compare with fp64 reference slots.

    Accepts when every slot error (real part and imaginary part) is within 6 of its
    per-slot std given the secret, and the RMS over all slots is within 1.5x the
    secret-averaged std.
    """
    sd = rescale_noise_sd(layer.log_n, scale_out)
    sd_j = slot_noise_sd(layer, scale_out)
    worst, rms_re, rms_im = 0.0, [], []
    ms = [rlwe.decrypt(np.asarray(out_ct[r], dtype=np.uint64), layer.s, layer.qs, layer.psis, layer.log_n)
          for r in range(len(rows))]
    zs = encode.decode(ms, scale_out, layer.log_n)                       # (rows, N/2), one pass
    for r, j in enumerate(rows):
        z = zs[r]
        err_re = z.real - ref_slots[r]
        worst = max(worst, np.max(np.abs(err_re) / sd_j), np.max(np.abs(z.imag) / sd_j))
        rms_re.append(np.mean(err_re ** 2))
        rms_im.append(np.mean(z.imag ** 2))
    res = {"sd": sd, "max_over_slot_sd": float(worst), "rms_re": float(np.sqrt(np.mean(rms_re))),
           "rms_im": float(np.sqrt(np.mean(rms_im)))}
    res["ok"] = bool(res["max_over_slot_sd"] <= 6 and res["rms_re"] <= 1.5 * sd and res["rms_im"] <= 1.5 * sd)
    return res
