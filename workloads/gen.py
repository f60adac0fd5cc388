"""Seeded synthetic inputs (shared by the GPU path and the CPU oracle).

Every draw comes from numpy's PCG64 seeded with
``SeedSequence([2606, 17421, cfg_index, *extra])``, spawned into independent
child streams in a fixed order: weights, activations, residues (ciphertext
residues or the RLWE ``a`` polynomial), secret, error.  Nothing here encodes,
transforms or reduces: moduli are passed in by the caller and residues are
drawn uniformly below them.
"""
from __future__ import annotations

import numpy as np

STREAMS = ("weights", "activations", "residues", "secret", "error", "sample")

WEIGHT_STD = 0.02      # N(0, 0.02^2) stand-in for trained weights
ERROR_SIGMA = 3.2      # RLWE error standard deviation
ERROR_BOUND = 19       # floor(6 sigma)


def streams(cfg_index: int, *extra: int) -> dict[str, np.random.Generator]:
    ss = np.random.SeedSequence([2606, 17421, cfg_index, *extra])
    return {name: np.random.default_rng(child) for name, child in zip(STREAMS, ss.spawn(len(STREAMS)))}


def scalar_weights(rng: np.random.Generator, d_out: int, d_in: int, std: float = WEIGHT_STD) -> np.ndarray:
    return rng.normal(0.0, std, size=(d_out, d_in))


def poly_weights(rng: np.random.Generator, d_out: int, d_in: int, slots: int,
                 std: float = WEIGHT_STD) -> np.ndarray:
    return rng.normal(0.0, std, size=(d_out, d_in, slots))


def activations(rng: np.random.Generator, count: int, slots: int) -> np.ndarray:
    """Real activation slot vectors, uniform in [-1, 1]."""
    return rng.uniform(-1.0, 1.0, size=(count, slots))


def uniform_residues(rng: np.random.Generator, prefix: tuple, moduli, n: int) -> np.ndarray:
    """uint32 array prefix + (L, n); limb l uniform in [0, moduli[l])."""
    out = np.empty(tuple(prefix) + (len(moduli), n), dtype=np.uint32)
    for l, q in enumerate(moduli):
        out[..., l, :] = rng.integers(0, int(q), size=tuple(prefix) + (n,), dtype=np.uint32)
    return out


def ternary_secret(rng: np.random.Generator, n: int) -> np.ndarray:
    return rng.integers(-1, 2, size=n).astype(np.int64)


def gaussian_error(rng: np.random.Generator, shape) -> np.ndarray:
    e = np.rint(rng.normal(0.0, ERROR_SIGMA, size=shape))
    return np.clip(e, -ERROR_BOUND, ERROR_BOUND).astype(np.int64)


def sample_rows(rng: np.random.Generator, d_out: int, count: int = 16) -> list[int]:
    """Rows checked at full size: first, last, and (count - 2) distinct random others."""
    if d_out <= count:
        return list(range(d_out))
    middle = rng.choice(np.arange(1, d_out - 1), size=count - 2, replace=False)
    return [0] + sorted(int(x) for x in middle) + [d_out - 1]
