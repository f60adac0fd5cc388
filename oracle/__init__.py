"""CPU oracle for the CKKS ciphertext x plaintext linear layer.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
reference that the GPU library is checked against.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import or call it; the product path (``paper_2606_17421_amd``) never does, and
the two share no code.

Contents, each following the paper's statement of the problem (CKKS over
R_Q = Z_Q[X]/(X^N+1) with RNS limbs, levels and rescaling, paper section 2.1;
ciphertext x public-plaintext linear layers on the accelerator with encoded
weights that are either resident or re-encoded per call, sections 3.2, 4.2 and
the FHE decode cost-breakdown table of section 6.1):

* ``params``  -- modulus chain and roots of unity (readings where the paper is
  silent: the L largest primes in (2^29, 2^30) with q = 1 mod 2N, the minimal
  primitive 2N-th root).
* ``ntt``     -- the negacyclic number-theoretic transform by its definition
  (evaluation at the odd powers of psi, bit-reversed order), plus a textbook
  twisted radix-2 version for large N that the tests pin to the definition.
* ``poly``    -- schoolbook negacyclic products.
* ``encode``  -- CKKS canonical-embedding encode/decode by direct O(N^2) sums.
* ``rlwe``    -- symmetric RLWE encryption / decryption used to make and check
  the encrypted inputs of the end-to-end checks.
* ``linear``  -- the modular MAC (scalar and full-polynomial weights) by direct
  modular sums, and rescaling by its CRT closed form.

Parity status per function is recorded in each module header.  Every function
here is pinned by a test under ``tests/test_oracle_*.py`` against something
other than itself (brute force, closed forms, library routines, invariants).
"""
