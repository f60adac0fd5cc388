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
* ``matvec`` is that formula as written: every rotation, baby or giant, is a complete
  rotation (automorphism, then key switching with its own division by P, exactly
  ``keyswitch.rotate``), the rotated inner sums are added mod Q, and the sum is
  rescaled once.  It is the reference.
* ``matvec_lazy`` is a schedule of the same product that an accelerator may prefer:
  the giant-step rotations are summed before their division by P.  With y_j the inner
  sums and (a0_j, a1_j) the key-switching inner product of sigma_j(c1 of y_j) over
  q_0 .. q_{L-1}, P,

      z = ModDown( P y_0 + sum_{j >= 1} ( (P sigma_j(c0 of y_j), 0) + (a0_j, a1_j) ) ).

  P y is exact in the extended basis (ModDown(P y + a) = y + ModDown(a)), so z differs
  from the eager sum only in rounding: one division by P of the summed inner products
  instead of one per giant step, at most n2 / 2 per coefficient of each component.
  After the closing rescale the two results decrypt to values at most N + 1 apart per
  coefficient (both rescale roundings included); ``eager_lazy_bound`` states it and the
  tests pin it.  The lazy form is an implementation choice, not a reading of the paper.

Tiling (section 3.3's small-ring tiles, section 6's GEMM tiling experiment): a
D x K weight matrix cut into a t_o x t_i grid of d x d tiles (d = D / t_o = K / t_i)
acts on the input cut into t_i sub-vectors, each encrypted on its own; output block i
is the homomorphic sum over j of the tile products W_ij x_j (ciphertext additions, mod
q_l per limb), each tile product a BSGS product as above.

Parity: pinned (tests/test_oracle_keyswitch.py) by decrypting and decoding the result
against numpy's W @ x, by the plaintext identity of the diagonal split on random
matrices, by the eager product's agreement with an independent composition of single
rotations (``keyswitch.rotate``) and plaintext products, and (tiles) by decoding the
aggregated blocks against W @ x.
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


def _baby_and_inner(pt, ct, n1: int, keys, qs_p, psis_p, log_n: int):
    """The baby-step rotations rot(x, i), i < n1, and the n2 inner sums
    y_j = sum_i pt[j, i] (.) rot(x, i) (2, L, N) each."""
    L = ct.shape[1]
    baby = [np.asarray(ct, dtype=np.uint64)]
    for i in range(1, n1):
        baby.append(rotate(baby[0], i, keys[i], qs_p, psis_p, log_n))
    return mac_poly(pt, np.stack(baby), qs_p[:L])          # (n2, 2, L, N)


def matvec(pt, ct, n1: int, keys, qs_p, psis_p, log_n: int, rescaled: bool = True) -> np.ndarray:
    """BSGS product of the encoded diagonals pt (n2, n1, L, N) with ct (2, L, N), every
    rotation complete (its own key switch and division by P), then one rescale.

    keys: rotation keys by step r (rotation_key(s, r)) for r = 1 .. n1-1 and
    r = j n1, j = 1 .. n2-1; qs_p / psis_p: the L ciphertext primes and the special
    prime last.  Returns the rescaled result (2, L-1, N), or with rescaled=False the
    sum before the closing rescale (2, L, N).
    """
    pt = np.asarray(pt)
    n2 = pt.shape[0]
    L = ct.shape[1]
    qs = qs_p[:L]
    inner = _baby_and_inner(pt, ct, n1, keys, qs_p, psis_p, log_n)
    q = np.array(qs, dtype=np.uint64)[:, None]
    z = inner[0] % q
    for j in range(1, n2):
        z = (z + rotate(inner[j], j * n1, keys[j * n1], qs_p, psis_p, log_n)) % q
    return rescale(z[None], qs, psis_p[:L], log_n)[0] if rescaled else z


def eager_lazy_bound(n2: int, log_n: int, q_last: int) -> int:
    """Largest difference, per coefficient, between the decryptions (under the ternary
    key s) of ``matvec`` and ``matvec_lazy`` on the same inputs.

    Before the closing rescale the two sums differ by delta with |delta_c| <= n2 / 2 per
    coefficient of each component c (n2 - 1 roundings of a division by P against one),
    so their decryptions differ by at most (n2 / 2)(1 + N).  Rescaling z to (z - r) / q
    with centred remainders |r_c| <= (q - 1) / 2 gives decryptions
    (dec(z) - r_0 - r_1 s) / q, so the results differ by at most
    ((n2 / 2) (1 + N) + (q - 1)(1 + N)) / q < (N + 1)(1 + n2 / (2 q)), i.e. N + 1 when
    n2 < q / (N + 1).  (The rescaled results are in fact bit-identical unless a
    coefficient of the sum lies within n2 / 2 of a rounding boundary of the closing
    rescale, which happens with probability about 2 N n2 / q per product.)"""
    n = 1 << log_n
    num = (n2 * (1 + n) + 1) // 2 + (q_last - 1) * (1 + n)
    return num // q_last                                    # the difference is an integer


def matvec_lazy(pt, ct, n1: int, keys, qs_p, psis_p, log_n: int, rescaled: bool = True) -> np.ndarray:
    """The same product with the giant-step rotations summed before one division by P
    (see the module text); equal to ``matvec`` within ``eager_lazy_bound`` after
    decryption.  rescaled=False: the sum before the closing rescale."""
    pt = np.asarray(pt)
    n2 = pt.shape[0]
    L = ct.shape[1]
    qs = qs_p[:L]
    inner = _baby_and_inner(pt, ct, n1, keys, qs_p, psis_p, log_n)
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
    return rescale(z[None], qs, psis_p[:L], log_n)[0] if rescaled else z


def tile_slots(W, t_o: int, t_i: int, n1: int, slots: int) -> np.ndarray:
    """Diagonal slot vectors (t_o, t_i, n2, n1, slots) of the d x d tiles of W (D x K)."""
    W = np.asarray(W, dtype=np.float64)
    d = W.shape[0] // t_o
    if W.shape != (t_o * d, t_i * d):
        raise ValueError("W must be a t_o x t_i grid of square tiles")
    return np.stack([np.stack([diagonal_slots(W[i * d:(i + 1) * d, j * d:(j + 1) * d], n1, slots)
                               for j in range(t_i)]) for i in range(t_o)])


def tiled_matvec(pt, cts, n1: int, keys, qs_p, psis_p, log_n: int, product=None) -> np.ndarray:
    """Tile products summed per output block: pt (t_o, t_i, n2, n1, L, N), cts (t_i, 2, L, N)
    (the encrypted input blocks).  product: the per-tile BSGS product (``matvec`` by
    default).  Returns (t_o, 2, L-1, N)."""
    product = matvec if product is None else product
    pt = np.asarray(pt)
    t_o, t_i = pt.shape[:2]
    L = cts.shape[2]
    q = np.array(qs_p[:L - 1], dtype=np.uint64)[:, None]
    out = []
    for i in range(t_o):
        acc = None
        for j in range(t_i):
            y = product(pt[i, j], cts[j], n1, keys, qs_p, psis_p, log_n)
            acc = y if acc is None else (acc + y) % q
        out.append(acc)
    return np.stack(out)
