"""Baby-step / giant-step diagonal matrix-vector product (CPU oracle; test infrastructure only).

The paper's accelerator linear call is a BSGS matrix-vector product over weight
diagonals that are encoded once and kept on the device (sections 4.1 and 4.2: the
BSGS-GEMM objects, 500 to 800 ms per call on its GPU).  The paper does not spell the
method out; the reading is the Halevi-Shoup diagonal method with the baby-step /
giant-step split:

* A d x d weight matrix W (d divides the slot count n = N/2) acts on a vector x that
  is packed d-periodically into the slots: z[t] = x[t mod d].
* Diagonal k of W, extended d-periodically: diag_k[t] = W[t mod d, (t + k) mod d].
  Then (W x)[t mod d] = sum_{k < d} diag_k[t] * z[t + k], i.e.
  W x = sum_k diag_k (.) rot(z, k), where rot(v, r)[t] = v[t + r] (left rotation).
* With d = n1 * n2 and k = j n1 + i, rot(z, j n1 + i) = rot(rot(z, i), j n1), so

      W x = sum_{j < n2} rot( sum_{i < n1} rot(diag_{j n1 + i}, -j n1) (.) rot(z, i),  j n1 ).

  The plaintexts pt[j, i] = Encode(rot(diag_{j n1 + i}, -j n1)) are the pre-encoded
  objects; one call takes n1 - 1 baby-step rotations of the input, n2 ct x pt inner
  sums (the full-polynomial MAC), n2 - 1 giant-step rotations, a sum, and one rescale.
* The giant-step rotations are summed before their division by P (a lazy ModDown, as
  BSGS implementations commonly do): with y_j the inner sums and (a0_j, a1_j) the
  key-switching inner product of sigma_j(c1 of y_j) over q_0 .. q_{L-1}, P,

      z = ModDown( P y_0 + sum_{j >= 1} ( (P sigma_j(c0 of y_j), 0) + (a0_j, a1_j) ) ),

  which equals the sum of the n2 rotated inner sums up to the rounding of one
  division by P instead of n2 - 1 of them (P y is exact in the extended basis:
  ModDown(P y + a) = y + ModDown(a)).  Then z is rescaled once.

Tiling (section 3.3's small-ring tiles, section 6's GEMM tiling experiment): a
D x K weight matrix cut into a t_o x t_i grid of d x d tiles (d = D / t_o = K / t_i)
acts on the input cut into t_i sub-vectors, each encrypted on its own; output block i
is the homomorphic sum over j of the tile products W_ij x_j (ciphertext additions, mod
q_l per limb), each tile product a BSGS product as above.

Parity: pinned (tests/test_oracle_keyswitch.py) by decrypting and decoding the result
against numpy's W @ x, by the plaintext identity of the diagonal split on random
matrices, and (tiles) by decoding the aggregated blocks against W @ x.
"""
from __future__ import annotations

import numpy as np

from .keyswitch import automorphism_ct, galois_element, keyswitch_ext, rotate
from .linear import mac_poly, rescale


def diagonal_slots(W, n1: int, slots: int) -> np.ndarray:
    """Slot vectors (n2, n1, slots) of rot(diag_{j n1 + i}, -j n1) for a d x d matrix W."""
    W = np.asarray(W, dtype=np.float64)
    d = W.shape[0]
    if W.shape != (d, d) or slots % d or d % n1:
        raise ValueError("need a square d x d matrix with d | slots and n1 | d")
    n2 = d // n1
    t = np.arange(slots)
    out = np.empty((n2, n1, slots), dtype=np.float64)
    for j in range(n2):
        for i in range(n1):
            k = j * n1 + i
            diag = W[t % d, (t + k) % d]
            out[j, i] = np.roll(diag, j * n1)          # rot(v, -r) = v shifted right by r
    return out


def replicate(x, slots: int) -> np.ndarray:
    """z[t] = x[t mod d]."""
    x = np.asarray(x)
    return x[np.arange(slots) % len(x)]


def matvec(pt, ct, n1: int, keys, qs_p, psis_p, log_n: int) -> np.ndarray:
    """BSGS product of the encoded diagonals pt (n2, n1, L, N) with ct (2, L, N).

    keys: rotation keys by step r (rotation_key(s, r)) for r = 1 .. n1-1 and
    r = j n1, j = 1 .. n2-1; qs_p / psis_p: the L ciphertext primes and the special
    prime last.  Returns the rescaled result (2, L-1, N).
    """
    pt = np.asarray(pt)
    n2 = pt.shape[0]
    L = ct.shape[1]
    qs = qs_p[:L]
    baby = [np.asarray(ct, dtype=np.uint64)]
    for i in range(1, n1):
        baby.append(rotate(baby[0], i, keys[i], qs_p, psis_p, log_n))
    inner = mac_poly(pt, np.stack(baby), qs)              # (n2, 2, L, N)
    P = qs_p[-1]
    qp = np.array(qs_p, dtype=np.uint64)[:, None]
    ext = np.zeros((2, L + 1, 1 << log_n), dtype=np.uint64)    # over q_0 .. q_{L-1}, P

    def add_times_p(comp, x):                                  # ext[comp] += P x (x over the q_l)
        for l in range(L):
            ql = np.uint64(qs[l])
            ext[comp, l] = (ext[comp, l] + (np.uint64(P % qs[l]) * (np.asarray(x[l], dtype=np.uint64) % ql)) % ql) % ql

    add_times_p(0, inner[0][0])
    add_times_p(1, inner[0][1])
    for j in range(1, n2):
        sig = automorphism_ct(inner[j], galois_element(j * n1, log_n), qs_p, psis_p, log_n)
        add_times_p(0, sig[0])
        ext = (ext + keyswitch_ext(sig[1], keys[j * n1], qs_p, psis_p, log_n)) % qp
    z = rescale(ext[None], qs_p, psis_p, log_n)[0]              # one division by P
    return rescale(z[None], qs, psis_p[:L], log_n)[0]


def tile_slots(W, t_o: int, t_i: int, n1: int, slots: int) -> np.ndarray:
    """Diagonal slot vectors (t_o, t_i, n2, n1, slots) of the d x d tiles of W (D x K)."""
    W = np.asarray(W, dtype=np.float64)
    d = W.shape[0] // t_o
    if W.shape != (t_o * d, t_i * d):
        raise ValueError("W must be a t_o x t_i grid of square tiles")
    return np.stack([np.stack([diagonal_slots(W[i * d:(i + 1) * d, j * d:(j + 1) * d], n1, slots)
                               for j in range(t_i)]) for i in range(t_o)])


def tiled_matvec(pt, cts, n1: int, keys, qs_p, psis_p, log_n: int) -> np.ndarray:
    """Tile products summed per output block: pt (t_o, t_i, n2, n1, L, N), cts (t_i, 2, L, N)
    (the encrypted input blocks).  Returns (t_o, 2, L-1, N)."""
    pt = np.asarray(pt)
    t_o, t_i = pt.shape[:2]
    L = cts.shape[2]
    q = np.array(qs_p[:L - 1], dtype=np.uint64)[:, None]
    out = []
    for i in range(t_o):
        acc = None
        for j in range(t_i):
            y = matvec(pt[i, j], cts[j], n1, keys, qs_p, psis_p, log_n)
            acc = y if acc is None else (acc + y) % q
        out.append(acc)
    return np.stack(out)
