/*
 * ckks_linear.h -- C ABI of the MI355X (gfx950) CKKS ciphertext x plaintext
 * linear-layer library.
 *
 * The operation is the accelerator side of a hybrid TEE/FHE serving design:
 * projection and FFN layers evaluated on encrypted activations with public
 * plaintext weights (paper section 3.2 and the threat model of section 3.5),
 * with weights either encoded once and kept resident or re-encoded per call
 * (section 4.2; fallback encoding is 34.4% of Qwen3-0.6B decode in the cost
 * breakdown table of section 6.1), over CKKS in R_Q = Z_Q[X]/(X^N+1) with RNS
 * limbs, levels and rescaling (section 2.1).
 *
 * Data model (all device buffers are caller-owned; the library keeps no
 * pointer to them after a call returns):
 *   - residues are uint32 in [0, q_l); every output is fully reduced;
 *   - a ciphertext is two polynomials (c0, c1), each stored as `limbs`
 *     contiguous rows of N residues:  ct[count][2][limbs][N];
 *   - polynomials handed to the transforms are poly[count][limbs][N];
 *     row r of a batch uses modulus q_(r mod limbs);
 *   - "NTT form" is the negacyclic NTT of section 2.1's ring, unscaled, in
 *     bit-reversed order:  A[i] = sum_k a_k psi^((2 brv(i) + 1) k) mod q,
 *     psi the smallest primitive 2N-th root of unity mod q;
 *   - `limbs` (1..L of the context) selects q_0 .. q_(limbs-1); rescaling
 *     drops q_(limbs-1).
 *
 * Moduli: unless given, q_0 > q_1 > ... are the L largest primes in
 * (2^29, 2^30) with q = 1 mod 2N.
 *
 * Errors: every entry point returns CKKS_OK (0) or a negative status and
 * never throws.  Argument errors are detected on the host before any launch.
 * Kernels run asynchronously on `stream` (a hipStream_t; NULL = the default
 * stream), so device-side faults surface at the caller's next synchronisation.
 * ckks_last_error() returns a thread-local description of the last failure.
 * Device pointers must be 16-byte aligned.  Entry points taking a context are
 * safe to call concurrently on different streams; outputs must not alias
 * inputs unless stated.
 */
#ifndef CKKS_LINEAR_H
#define CKKS_LINEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ckks_ctx ckks_ctx;

enum ckks_status {
  CKKS_OK = 0,
  CKKS_E_INVALID_ARG = -1, /* bad shape, pointer, alignment or modulus          */
  CKKS_E_UNSUPPORTED = -2, /* valid request the library does not implement    */
  CKKS_E_HIP = -3,         /* a HIP runtime call or launch failed              */
  CKKS_E_WORKSPACE = -4    /* workspace missing or smaller than required       */
};

/* Operations that take a workspace (see ckks_workspace_bytes). */
enum ckks_op {
  CKKS_OP_MAC_SCALAR = 1, /* a = d_out, b = d_in  */
  CKKS_OP_RESCALE = 2,    /* a = count, b unused  */
  CKKS_OP_ENCODE_POLY = 3, /* a = count, b unused  */
  CKKS_OP_ROTATE = 4       /* a = count, b = hoisted (0 or 1); limbs = L - 1 */
};

/* MAC kernel selection for ckks_linear_mac_scalar (ckks_ctx_set_mac_algo). */
enum ckks_mac_algo {
  CKKS_MAC_AUTO = 0, /* library choice (int8 MFMA digit split)               */
  CKKS_MAC_VALU = 1, /* u32 x u32 -> u64 vector multiply-add                 */
  CKKS_MAC_MFMA = 2  /* exact int8 digit-split contractions on matrix cores  */
};

/* Context: the RNS modulus chain of one ring degree and its device tables
 * (twiddles with Shoup companions, rescale inverses, encode FFT tables).
 * The paper keeps one CKKS context per projection shape (section 4.2); here
 * one context serves every shape that shares (N, chain).
 *   out        receives the new context (host pointer); unchanged on error.
 *   log_n      log2 N, 10..16.
 *   num_limbs  L, 1..16.
 *   moduli     host array of L distinct primes in (2^29, 2^30), each = 1 mod
 *              2N, or NULL for the default chain.  Checked: CKKS_E_INVALID_ARG.
 *   device     HIP device ordinal the tables live on; all later calls with
 *              this context must run on that device.
 * Allocates device memory (the only entry point that does, with destroy
 * freeing it). */
int ckks_ctx_create(ckks_ctx** out, uint32_t log_n, uint32_t num_limbs,
                    const uint32_t* moduli, int device);
int ckks_ctx_destroy(ckks_ctx* ctx);
/* Host copies of the chain: moduli q_l and roots psi_l (length L each). */
int ckks_ctx_moduli(const ckks_ctx* ctx, uint32_t* out);
int ckks_ctx_roots(const ckks_ctx* ctx, uint32_t* out);
int ckks_ctx_info(const ckks_ctx* ctx, uint32_t* log_n, uint32_t* num_limbs);
/* Select the scalar-weight MAC kernel (ckks_mac_algo); applies to later calls. */
int ckks_ctx_set_mac_algo(ckks_ctx* ctx, int algo);

/* Forward / inverse negacyclic NTT (section 2.1 ring; definition above),
 * in place on polys[count][limbs][N] (device).  The inverse includes N^-1.
 * count == 0 is a no-op. */
int ckks_ntt(const ckks_ctx* ctx, uint32_t* polys, uint32_t count, uint32_t limbs,
             void* stream);
int ckks_intt(const ckks_ctx* ctx, uint32_t* polys, uint32_t count, uint32_t limbs,
              void* stream);

/* Scalar weight encoding (weights as constant plaintexts, section 4.2's
 * pre-encoded GPU-resident weights in the one-ciphertext-per-feature
 * packing):  w_enc[j][i][l] = rint(w[j][i] * scale) mod q_l, rint rounding
 * half to even.
 *   w      device fp64 [d_out][d_in]; |w * scale| < 2^63 and finite.
 *   w_enc  device uint32 [d_out][d_in][limbs]; must not overlap w
 *          (CKKS_E_INVALID_ARG). */
int ckks_linear_encode_scalar(const ckks_ctx* ctx, const double* w, uint32_t d_out,
                              uint32_t d_in, uint32_t limbs, double scale,
                              uint32_t* w_enc, void* stream);

/* Full-polynomial encoding of real slot vectors (the per-call fallback
 * encode of section 4.2): the inverse canonical embedding with slot j at
 * exp(i pi 5^j / N), m_k = (2/N) Re sum_j z_j exp(-i pi 5^j k / N), then
 * p_k = rint(scale * m_k), reduced mod each q_l and taken to NTT form.
 *   slots  device fp64 [count][N/2] (real slot values).
 *   pt     device uint32 [count][limbs][N], NTT form; must not overlap slots.
 * Every supported N (at N = 2^16 count x limbs <= 2^31 / 64, else
 * CKKS_E_INVALID_ARG).  The spectral transform runs in fp64, so a coefficient
 * whose scaled value lies within about 1e-9 of a rounding tie may differ by
 * one from an exact evaluation. */
int ckks_linear_encode_poly(const ckks_ctx* ctx, const double* slots, uint32_t count,
                            uint32_t limbs, double scale, uint32_t* pt, void* stream);

/* ct x pt MAC with scalar weights (FHE_Linear of Algorithm 3 in the
 * one-ciphertext-per-feature packing): for every output j, component c,
 * limb l and NTT slot k
 *     ct_out[j][c][l][k] = sum_i w_enc[j][i][l] * ct_in[i][c][l][k]  mod q_l.
 *   w_enc    device uint32 [d_out][d_in][limbs], residues < q_l.
 *   ct_in    device uint32 [d_in][2][limbs][N].
 *   ct_out   device uint32 [d_out][2][limbs][N]; must not overlap ct_in or
 *            w_enc (checked: CKKS_E_INVALID_ARG).
 *   workspace / workspace_bytes: device scratch of at least
 *            ckks_workspace_bytes(ctx, CKKS_OP_MAC_SCALAR, d_out, d_in, limbs)
 *            bytes (may be 0 for the VALU kernel); else CKKS_E_WORKSPACE.  It
 *            must not overlap ct_in, ct_out or w_enc (CKKS_E_INVALID_ARG).
 * d_out <= 524280 and d_in <= 2^24 (else CKKS_E_INVALID_ARG); the matrix-core
 * kernel takes d_in <= 4096 (above it CKKS_MAC_AUTO runs the VALU kernel and
 * CKKS_MAC_MFMA returns CKKS_E_UNSUPPORTED).
 * d_out == 0 is a no-op; d_in == 0 writes zeros. */
int ckks_linear_mac_scalar(const ckks_ctx* ctx, const uint32_t* w_enc,
                           const uint32_t* ct_in, uint32_t* ct_out, uint32_t d_out,
                           uint32_t d_in, uint32_t limbs, void* workspace,
                           size_t workspace_bytes, void* stream);

/* ckks_linear_mac_scalar without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, result and errors as
 * ckks_linear_mac_scalar; the matrix-core kernel's workspace (the weight digit
 * fragments and per-tile flags, ckks_workspace_bytes(ctx, CKKS_OP_MAC_SCALAR,
 * d_out, d_in, limbs) bytes) is instead a library-owned device array of
 * CKKS_NOALLOC_SCRATCH_BYTES (64 MiB) on each GPU the library runs on, held
 * until the process ends.  The call allocates nothing.  Requests needing more
 * scratch than that return CKKS_E_WORKSPACE (the fragments take 4 bytes per
 * weight and limb, rows rounded up to 128 and d_in to 64: at 4 limbs up to
 * 3968 x 1024 weights, for any N).  Every call on one GPU shares that GPU's array,
 * which keeps the last call's contents: calls that overlap in time on one GPU
 * (different streams, or different host threads) race and must be serialised
 * by the caller.  The kernels overwrite every scratch byte they read, so
 * nothing needs clearing between calls. */
#define CKKS_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int ckks_linear_mac_scalar_noalloc(const ckks_ctx* ctx, const uint32_t* w_enc,
                                   const uint32_t* ct_in, uint32_t* ct_out,
                                   uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                   void* stream);

/* ct x pt MAC with full-polynomial NTT-form weights (the fallback-encode
 * path of section 4.2): slot-wise
 *     ct_out[j][c][l][k] = sum_i pt[j][i][l][k] * ct_in[i][c][l][k]  mod q_l,
 * i.e. a negacyclic product per pair in the coefficient domain.
 *   pt      device uint32 [d_out][d_in][limbs][N] (NTT form).
 *   ct_in   device uint32 [d_in][2][limbs][N];  ct_out [d_out][2][limbs][N],
 *           which must not overlap pt or ct_in (CKKS_E_INVALID_ARG). */
int ckks_linear_mac_poly(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* ct_in,
                         uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                         void* stream);

/* Rescale (section 2.1: divide by the last prime, drop one level), NTT form
 * in and out.  Per polynomial, with C the CRT lift of the coefficients over
 * q_0..q_(limbs-1):  out = NTT_l( round(C / q_(limbs-1)) mod q_l ), l < limbs-1,
 * computed as (c_l - NTT_l([INTT(c_(limbs-1))]_centred mod q_l)) * q_(limbs-1)^-1.
 *   ct_in   device uint32 [count][2][limbs][N], limbs >= 2.
 *   ct_out  device uint32 [count][2][limbs-1][N]; must not overlap ct_in
 *           (checked: CKKS_E_INVALID_ARG).
 *   workspace: ckks_workspace_bytes(ctx, CKKS_OP_RESCALE, count, 0, limbs)
 *           bytes (0 for log_n <= 15), not overlapping ct_in or ct_out. */
int ckks_rescale(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t* ct_out,
                 uint32_t count, uint32_t limbs, void* workspace, size_t workspace_bytes,
                 void* stream);

/* Symmetric RLWE encryption, decryption and decrypt-then-encrypt refresh,
 * batched.  In the paper these are the steps on the trusted side of each
 * accelerator call (section 3.2: decrypt-compute-encrypt windows and the DtE
 * refresh ct' = Enc(Dec(ct)); section 4.2 quotes about 30 ms each for the
 * CPU-side encrypt and decrypt of one call).  They take the secret key as an
 * input buffer, so calling them on a device puts that device inside the
 * trust boundary: they serve deployments where it is (a trusted
 * accelerator) and the generation and checking of encrypted workloads.
 *   s_ntt  device uint32 [limbs][N]: the secret (ternary, or any integer
 *          polynomial) reduced mod q_l and taken to NTT form (ckks_ntt).
 *   a      device uint32 [count][limbs][N]: fresh uniform residues, NTT form.
 *   e      device int32 [count][N]: fresh error coefficients, |e| < q_l.
 * Encryption, per limb:  c0 = pt + NTT(e) - a (.) s,  c1 = a.
 *   pt     device uint32 [count][limbs][N] (NTT form, e.g. ckks_linear_encode_poly
 *          output), or NULL for a zero plaintext.
 *   ct     device uint32 [count][2][limbs][N]; must not overlap the inputs. */
int ckks_encrypt(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* s_ntt,
                 const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs,
                 uint32_t* ct, void* stream);

/* Decryption to coefficient residues:  m[c][l] = INTT(c0 + c1 (.) s) mod q_l.
 *   ct  device uint32 [count][2][limbs][N];  m  device uint32 [count][limbs][N]
 *   (must not overlap ct).  Lifting to integers (CRT) and decoding are the
 *   caller's. */
int ckks_decrypt(const ckks_ctx* ctx, const uint32_t* ct, const uint32_t* s_ntt,
                 uint32_t count, uint32_t limbs, uint32_t* m, void* stream);

/* Decrypt-then-encrypt refresh (the DtE equation of section 3.2): the integer
 * plaintext polynomial of ct_in is recovered from limbs 0 and 1 (CRT over
 * q_0 q_1, centred; exact while every coefficient of the decrypted polynomial
 * is below q_0 q_1 / 2 in magnitude, about 2^59) and encrypted afresh with
 * (a, e) under limbs_out limbs.  The scale is unchanged (the caller carries it).
 *   ct_in   device uint32 [count][2][limbs_in][N], 2 <= limbs_in <= L.
 *   s_ntt   [limbs_out][N] (limbs_out >= 2);  a [count][limbs_out][N];  e [count][N].
 *   ct_out  device uint32 [count][2][limbs_out][N], 2 <= limbs_out <= L; must
 *           not overlap ct_in (its c1 rows serve as scratch during the call). */
int ckks_refresh(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t limbs_in,
                 const uint32_t* s_ntt, const uint32_t* a, const int32_t* e, uint32_t count,
                 uint32_t limbs_out, uint32_t* ct_out, void* stream);

/* ---- Rotations and the BSGS diagonal matrix-vector product -----------------
 *
 * The paper's accelerator linear call is a baby-step / giant-step product of
 * pre-encoded weight diagonals with rotated copies of the input ciphertext
 * (sections 4.1 and 4.2), rotations being Galois automorphisms followed by key
 * switching under one special prime (section 4.2's parameter set).
 *
 * Key-switching context: the LAST prime of the context is the special prime P.
 * Ciphertexts that are rotated, and the BSGS input, carry the other
 * Lk = L - 1 limbs (L = the context's limb count, at least 3).  Switching keys
 * are [Lk][2][L][N] words per key (digit i, then the pair (b, a), then every
 * prime including P), NTT form: ksk_i = (-a_i s + e_i + P g_i s_from, a_i)
 * with g_i the CRT idempotent of limb i.  Key switching uses one digit per limb
 * (the centred coefficients of limb i), the digits lifted to every prime,
 * an inner product with the key and the division by P (the rescale that drops
 * P).  Rotation by r slots: g = 5^r mod 2N; slot j + r moves to slot j.
 */

/* sigma_g on NTT-form polynomials: out = the polynomial a(X^g) for each of
 * `rows` rows of N words (any limb; the permutation does not depend on the
 * prime).  galois odd, below 2N (5^r mod 2N rotates by r; 2N - 1 conjugates).
 * in and out must not overlap. */
int ckks_automorphism(const ckks_ctx* ctx, const uint32_t* in, uint32_t rows, uint32_t galois, uint32_t* out,
                      void* stream);

/* Rotation keys for steps r0, r0 + r_step, ..., (count keys), under the
 * secret s_ntt [L][N] (NTT form over every prime of the context, P included).
 * a: uniform residues [count][Lk][L][N] (NTT form); e: small error
 * coefficients [count][Lk][N].  ksk: [count][Lk][2][L][N].  Runs on the trusted
 * side (the secret is an input).  Steps are taken mod N/2. */
int ckks_keygen_rotation(const ckks_ctx* ctx, const uint32_t* s_ntt, uint32_t r0, uint32_t r_step, uint32_t count,
                         const uint32_t* a, const int32_t* e, uint32_t* ksk, void* stream);

/* `count` rotations of ciphertexts [..][2][Lk][N]: rotation k is by step
 * r0 + k r_step with key ksk[k] ([count][Lk][2][L][N]).  hoisted = 1: all count
 * rotations act on the one ciphertext ct_in (its digits are lifted once);
 * hoisted = 0: rotation k acts on ct_in[k].  ct_out [count][2][Lk][N] must not
 * overlap the inputs.  workspace: ckks_workspace_bytes(ctx, CKKS_OP_ROTATE,
 * count, hoisted, Lk) bytes of device memory, 256-byte aligned. */
int ckks_rotate(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t count, uint32_t r0, uint32_t r_step,
                int hoisted, const uint32_t* ksk, void* workspace, size_t workspace_bytes, uint32_t* ct_out,
                void* stream);

/* BSGS product y = W x of a d x d weight matrix, d = n1 n2, with x packed
 * d-periodically in the slots of each of `count` input ciphertexts ct_in
 * [count][2][Lk][N] (Halevi-Shoup diagonals with the baby-step / giant-step
 * split):  y = sum_j rot( sum_i pt[j][i] (.) rot(x, i), j n1 ), then one rescale.
 * Schedule: the giant-step rotations are summed before their division by P
 * (the sum is formed over the L primes: P times the unrotated term and the
 * rotated c0 parts, plus the key-switching inner products, then divided by P
 * once).  Against the formula with every rotation complete (its own division
 * by P) this changes only roundings: the two results decrypt to values at
 * most N + 1 apart per coefficient, and they are bit-identical unless a
 * coefficient of the sum lies within n2/2 of a rounding boundary of the
 * closing rescale.
 * pt [n2][n1][Lk][N]: NTT-form encodings of rot(diag_(j n1 + i), -j n1) (the
 * slot vectors diag_k[t] = W[t mod d][(t + k) mod d]; ckks_linear_encode_poly
 * makes them).  ksk: n1 - 1 rotation keys for steps 1 .. n1-1 followed by
 * n2 - 1 keys for steps n1, 2 n1, .., (n2-1) n1 ([n1 + n2 - 2][Lk][2][L][N]).
 * ct_out [count][2][Lk - 1][N] (scale: scale_pt scale_ct / q_(Lk-1)).
 * workspace: ckks_bsgs_workspace_bytes(ctx, count, n1, n2), 256-byte aligned.
 * d must divide N/2 (not checked by the library: the caller's packing). */
int ckks_linear_bsgs(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* ct_in, uint32_t count, uint32_t n1,
                     uint32_t n2, const uint32_t* ksk, void* workspace, size_t workspace_bytes, uint32_t* ct_out,
                     void* stream);

/* Workspace of ckks_linear_bsgs in bytes ((size_t)-1 for an invalid request). */
size_t ckks_bsgs_workspace_bytes(const ckks_ctx* ctx, uint32_t count, uint32_t n1, uint32_t n2);

/* Homomorphic addition ct_out = ct_a + ct_b of `count` ciphertexts
 * [count][2][limbs][N] (NTT form, same scale): the aggregation of tile outputs
 * when a large product is cut into tiles (section 3.3, tiling of large
 * homomorphic GEMMs).  ct_out may alias ct_a or ct_b exactly (in place), but
 * must not partially overlap either. */
int ckks_add(const ckks_ctx* ctx, const uint32_t* ct_a, const uint32_t* ct_b, uint32_t count, uint32_t limbs,
             uint32_t* ct_out, void* stream);

/* Workspace size in bytes for `op` (ckks_op) with the given sizes; 0 when
 * none is needed; (size_t)-1 for an invalid request. */
size_t ckks_workspace_bytes(const ckks_ctx* ctx, int op, uint32_t a, uint32_t b,
                            uint32_t limbs);

/* Scale after rescaling a ciphertext of scale `scale_in` at `limbs` limbs:
 * scale_in / q_(limbs-1) (the caller carries the scale). */
double ckks_rescaled_scale(const ckks_ctx* ctx, double scale_in, uint32_t limbs);

/* Thread-local text of the last error ("" if none). */
const char* ckks_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CKKS_LINEAR_H */
