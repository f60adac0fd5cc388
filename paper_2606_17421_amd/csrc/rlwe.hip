// Symmetric RLWE encryption, decryption and the decrypt-then-encrypt refresh
// (gfx950), batched over ciphertexts [count][2][limbs][N] in NTT form.
//
// Encryption (the ciphertext form of section 2.1, made by the trusted side in
// section 3.2): c0 = pt + NTT(e) - a (.) s, c1 = a, per limb, with the
// secret s and the fresh randomness a (uniform, NTT form) and e (small
// integer coefficients) supplied by the caller.  Decryption: the coefficient
// residues INTT(c0 + c1 (.) s) per limb.  Refresh (the DtE equation of
// section 3.2, ct' = Enc(Dec(ct))): the integer plaintext polynomial is
// recovered from limbs 0 and 1 by CRT to centred integers (exact while its
// coefficients lie within q0 q1 / 2 in magnitude) and encrypted afresh under
// limbs_out limbs.
//
// Encryption and decryption run the batched NTT kernels over the c0 rows (or
// the output rows) through their row-group stride, with pointwise passes
// around them, 16 bytes per thread and limb.  The refresh, up to N = 2^15, is
// two transform kernels (decrypt + inverse, lift + forward + combine), or up to
// 2^13 for decode-size counts one fused kernel split by output limb; at 2^16
// (a row exceeds the LDS) it is the pass structure of encryption and decryption.
#include "ntt_core.hpp"

namespace ckks {
namespace {

constexpr int kThreads = 256;

// 16-byte accesses use native vector types: written with the HIP uint4
// struct, the read-modify-write loop of the encrypt combine compiled to an
// empty kernel.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int32_t v4s __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4u ld4(const uint32_t* p) { return *reinterpret_cast<const v4u*>(p); }
__device__ __forceinline__ v4s ld4(const int32_t* p) { return *reinterpret_cast<const v4s*>(p); }
__device__ __forceinline__ void st4(uint32_t* p, v4u v) { *reinterpret_cast<v4u*>(p) = v; }

// Signed 64-bit x mod q, in [0, q).
__device__ __forceinline__ uint32_t reduce_i64(int64_t x, uint32_t q, double qr) {
  const uint64_t ax = static_cast<uint64_t>(x < 0 ? -x : x);
  const uint32_t r = reduce_u64(ax, q, qr);
  return (x < 0 && r != 0) ? q - r : r;
}

// floor(w 2^32 / q) for w < q (the Shoup companion of w): the fp64 estimate is
// within one of it, and one remainder check fixes it.
__device__ __forceinline__ uint32_t shoup_const(uint32_t w, uint32_t q, double qr) {
  uint32_t ws = static_cast<uint32_t>(static_cast<double>(w) * 4294967296.0 * qr);
  const int64_t r = static_cast<int64_t>((static_cast<uint64_t>(w) << 32) - static_cast<uint64_t>(ws) * q);
  if (r < 0) --ws;
  else if (r >= static_cast<int64_t>(q)) ++ws;
  return ws;
}

// (x0 + q0 k - [neg] q0 q1 + e) mod q_l, the refreshed residue of one
// coefficient: x0 < q0 and k < q1 are the CRT digits, neg the centring flag,
// e in [-19, 19] the fresh error.  With ka = k + [neg](2 q - q1) (< 2^32; 2 q >
// q1) the centring folds into the product q0 ka = q0 k - [neg] q0 q1 (mod q);
// the lazy Shoup product lies in [0, 2q), so x0 mod q + product + e + q lies
// in [q - 19, 4q + 19) < 2^32 and three conditional subtractions finish.
struct LiftConst {
  uint32_t q, q0l, q0ls, d2;
};
__device__ __forceinline__ LiftConst lift_const(uint32_t q0, uint32_t q1, uint32_t q, double qr) {
  LiftConst c;
  c.q = q;
  c.q0l = q0 >= q ? q0 - q : q0;  // q0 < 2q
  c.q0ls = shoup_const(c.q0l, q, qr);
  c.d2 = 2 * q - q1;
  return c;
}
__device__ __forceinline__ uint32_t lift_residue(const LiftConst& c, uint32_t x0, uint32_t k, bool neg, int32_t e) {
  const uint32_t ka = neg ? k + c.d2 : k;
  const uint32_t p = mul_shoup_lazy(ka, c.q0l, c.q0ls, c.q);
  const uint32_t x0l = min(x0, x0 - c.q);
  uint32_t t = x0l + p + static_cast<uint32_t>(e + static_cast<int32_t>(c.q));
  t = min(t, t - 2 * c.q);
  t = min(t, t - c.q);
  return min(t, t - c.q);
}

// Buffer resource over one row of N words (row bases live in scalar
// registers; per-lane offsets and per-element constants index into it).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void* base, uint32_t n) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n * 4, 0x00020000);
}

// Thread -> (ciphertext c, coefficient quad k4) over count * N/4 quads.
struct Quad {
  size_t c;
  uint32_t k;
  bool ok;
};
__device__ __forceinline__ Quad quad_of(uint32_t n, uint32_t count) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x;
  const uint32_t per = n >> 2;
  Quad r;
  r.c = i / per;
  r.k = static_cast<uint32_t>(i % per) * 4;
  r.ok = r.c < count;
  return r;
}

// ct[c][0][l][k] = e[c][k] mod q_l for every limb (coefficient form).
__global__ __launch_bounds__(kThreads) void err_rows_kernel(Tables tb, const int32_t* __restrict__ e,
                                                            uint32_t count, uint32_t limbs,
                                                            uint32_t* __restrict__ ct) {
  const uint32_t n = tb.n;
  const Quad p = quad_of(n, count);
  if (!p.ok) return;
  const v4s ev = ld4(e + p.c * n + p.k);
  for (uint32_t l = 0; l < limbs; ++l) {
    const uint32_t q = tb.q[l];
    v4u r;
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = ev[j] < 0 ? q - static_cast<uint32_t>(-ev[j]) : static_cast<uint32_t>(ev[j]);
    st4(ct + ((p.c * 2) * limbs + l) * n + p.k, r);
  }
}

// c0 <- c0 + pt - a (.) s, c1 <- a  (pt == nullptr: no plaintext term).
__global__ __launch_bounds__(kThreads) void enc_combine_kernel(Tables tb, const uint32_t* __restrict__ pt,
                                                               const uint32_t* __restrict__ s_ntt,
                                                               const uint32_t* __restrict__ a, uint32_t count,
                                                               uint32_t limbs, uint32_t* __restrict__ ct) {
  const uint32_t n = tb.n;
  const Quad p = quad_of(n, count);
  if (!p.ok) return;
  for (uint32_t l = 0; l < limbs; ++l) {
    const uint32_t q = tb.q[l], mu = tb.barrett[l];
    const size_t row = (p.c * limbs + l) * n + p.k;
    uint32_t* c0p = ct + ((p.c * 2) * limbs + l) * n + p.k;
    uint32_t* c1p = c0p + static_cast<size_t>(limbs) * n;
    const v4u c0 = ld4(c0p);
    const v4u av = ld4(a + row);
    const v4u sv = ld4(s_ntt + static_cast<size_t>(l) * n + p.k);
    const v4u pv = pt ? ld4(pt + row) : v4u{0, 0, 0, 0};
    v4u o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = sub_mod(add_mod(c0[j], pv[j], q), mul_mod_barrett(av[j], sv[j], q, mu), q);
    st4(c0p, o);
    st4(c1p, av);
  }
}

// out row (c * out_gstride + out_off + l) <- c0 + c1 (.) s of ciphertext c,
// limb l < limbs_used, read from ct[count][2][ct_limbs][N] (NTT form).
__global__ __launch_bounds__(kThreads) void dec_pointwise_kernel(Tables tb, const uint32_t* __restrict__ ct,
                                                                 uint32_t ct_limbs, const uint32_t* __restrict__ s_ntt,
                                                                 uint32_t count, uint32_t limbs_used,
                                                                 uint32_t* __restrict__ out, uint32_t out_gstride,
                                                                 uint32_t out_off) {
  const uint32_t n = tb.n;
  const Quad p = quad_of(n, count);
  if (!p.ok) return;
  for (uint32_t l = 0; l < limbs_used; ++l) {
    const uint32_t q = tb.q[l], mu = tb.barrett[l];
    const uint32_t* c0p = ct + ((p.c * 2) * ct_limbs + l) * n + p.k;
    const v4u c0 = ld4(c0p);
    const v4u c1 = ld4(c0p + static_cast<size_t>(ct_limbs) * n);
    const v4u sv = ld4(s_ntt + static_cast<size_t>(l) * n + p.k);
    v4u o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = add_mod(c0[j], mul_mod_barrett(c1[j], sv[j], q, mu), q);
    st4(out + (p.c * out_gstride + out_off + l) * n + p.k, o);
  }
}

// Refresh lift.  dec rows (c * 2 limbs_out + limbs_out + {0, 1}) hold the
// decrypted coefficient residues mod q0, q1.  x = r0 + q0 ((r1 - r0) q0^-1
// mod q1) is the CRT value in [0, q0 q1); centred, plus the fresh error, it
// is written mod q_l into the c0 rows of ct_out for l < limbs_out.
__global__ __launch_bounds__(kThreads) void dte_lift_kernel(Tables tb, const int32_t* __restrict__ e,
                                                            uint32_t count, uint32_t limbs_out,
                                                            uint32_t* __restrict__ ct_out) {
  const uint32_t n = tb.n;
  const Quad p = quad_of(n, count);
  if (!p.ok) return;
  const uint32_t q0 = tb.q[0], q1 = tb.q[1];
  const uint32_t w = tb.qinv[0 * tb.L + 1], ws = tb.qinv_shoup[0 * tb.L + 1];  // q0^-1 mod q1
  const uint64_t Q2 = static_cast<uint64_t>(q0) * q1;
  const uint32_t* d0 = ct_out + ((p.c * 2) * limbs_out + limbs_out) * n + p.k;
  const v4u r0v = ld4(d0);
  const v4u r1v = ld4(d0 + n);
  const v4s ev = ld4(e + p.c * n + p.k);
  int64_t m[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t r0 = r0v[j];
    const uint32_t r0m = r0 >= q1 ? r0 - q1 : r0;  // r0 < q0 < 2 q1
    const uint32_t t = mul_shoup(sub_mod(r1v[j], r0m, q1), w, ws, q1);
    const uint64_t x = static_cast<uint64_t>(r0) + static_cast<uint64_t>(q0) * t;  // [0, q0 q1)
    const int64_t xc = x > Q2 / 2 ? static_cast<int64_t>(x) - static_cast<int64_t>(Q2) : static_cast<int64_t>(x);
    m[j] = xc + ev[j];
  }
  for (uint32_t l = 0; l < limbs_out; ++l) {
    const uint32_t q = tb.q[l];
    const double qr = tb.q_recip[l];
    v4u o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = reduce_i64(m[j], q, qr);
    st4(ct_out + ((p.c * 2) * limbs_out + l) * n + p.k, o);
  }
}

// Fused refresh for N <= 2^13 and at most one workgroup per CU (a decode-size
// group): one workgroup per ciphertext and output limb.  Limbs 0
// and 1 of c0 + c1 (.) s are read coalesced and inverse-transformed in LDS;
// the CRT value over q0 q1 is kept as its two digits x = x0 + q0 k (k with the
// centring flag in bit 31) in the group-0 layout that the forward transform
// starts from, rebuilt mod q_l with 32-bit Barrett products, the fresh error
// added, transformed, combined with a and s and written coalesced.  The two
// inverse transforms are repeated per output limb, so the chain per workgroup
// is three transforms on limbs_out times the workgroups.  16 residues per
// thread (1024 threads at 2^14) keeps the live state in registers.
template <int LOGN>
struct RefreshPlan {
  static_assert(LOGN <= 13, "the fused refresh serves N <= 2^13");
  static constexpr int LOGE = 4;
  using P = Plan<LOGN, LOGE>;
  static constexpr int kWavesPerSimd = 4;
};

template <int LOGN>
__global__ __launch_bounds__(RefreshPlan<LOGN>::P::T, RefreshPlan<LOGN>::kWavesPerSimd) void refresh_kernel(
    Tables tb, const uint32_t* __restrict__ ct_in, uint32_t limbs_in, const uint32_t* __restrict__ s_ntt,
    const uint32_t* __restrict__ a, const int32_t* __restrict__ e, uint32_t limbs_out,
    uint32_t* __restrict__ ct_out) {
  using P = typename RefreshPlan<LOGN>::P;
  constexpr int LOGE = RefreshPlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const size_t c = blockIdx.x;
  const uint32_t t = threadIdx.x;
  const uint32_t vofs = pos_coalesced<LOGE>(t, 0) * 4;  // byte offset of element 0 in the coalesced layout

  uint32_t x0[P::E], v[P::E];
#pragma unroll
  for (int l = 0; l < 2; ++l) {
    const uint32_t q = tb.q[l], mu = tb.barrett[l];
    const auto r_c0 = row_rsrc(ct_in + ((c * 2) * limbs_in + l) * N, N);
    const auto r_c1 = row_rsrc(ct_in + ((c * 2 + 1) * limbs_in + l) * N, N);
    const auto r_s = row_rsrc(s_ntt + static_cast<size_t>(l) * N, N);
    if (l == 1) __syncthreads();  // the last (workgroup-wide) exchange of limb 0 is read out
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      const uint32_t c0 = __builtin_amdgcn_raw_buffer_load_b32(r_c0, vofs, j << 8, 0);
      const uint32_t c1 = __builtin_amdgcn_raw_buffer_load_b32(r_c1, vofs, j << 8, 0);
      const uint32_t sv = __builtin_amdgcn_raw_buffer_load_b32(r_s, vofs, j << 8, 0);
      v[j] = add_mod(c0, mul_mod_barrett(c1, sv, q, mu), q);
    }
    wave_relayout<LOGN, LOGE, true>(v, t, lds);
    const size_t tl = static_cast<size_t>(l) << LOGN;
    inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + tl, tb.inv_shoup + tl, q, lds);
    const uint32_t ni = tb.ninv[l], nis = tb.ninv_shoup[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      v[j] = mul_shoup(v[j], ni, nis, q);
      if (l == 0) x0[j] = v[j];
    }
  }
  // CRT digits: x = x0 + q0 k in [0, q0 q1), k = (r1 - r0) q0^-1 mod q1;
  // bit 31 of kf marks x > q0 q1 / 2 (centred value x - q0 q1).
  const uint32_t q0 = tb.q[0], q1 = tb.q[1];
  const uint32_t w = tb.qinv[0 * tb.L + 1], ws = tb.qinv_shoup[0 * tb.L + 1];  // q0^-1 mod q1
  const uint64_t half = static_cast<uint64_t>(q0) * q1 / 2;
  uint32_t kf[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t r0m = x0[j] >= q1 ? x0[j] - q1 : x0[j];  // x0 < q0 < 2 q1
    const uint32_t k = mul_shoup(sub_mod(v[j], r0m, q1), w, ws, q1);
    const uint64_t x = static_cast<uint64_t>(x0[j]) + static_cast<uint64_t>(q0) * k;
    kf[j] = k | (x > half ? 0x80000000u : 0u);
  }
  // the error row through a buffer resource: the per-j offsets j T are scalar constants
  const auto er = row_rsrc(e + c * N, N);
  {
    const uint32_t l = blockIdx.y;
    const uint32_t q = tb.q[l], mu = tb.barrett[l];
    const LiftConst lc = lift_const(q0, q1, q, tb.q_recip[l]);
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      const int32_t ev = static_cast<int32_t>(
          __builtin_amdgcn_raw_buffer_load_b32(er, t * 4, P::template pos<0>(0, j) * 4, 0));
      v[j] = lift_residue(lc, x0[j], kf[j] & 0x7fffffffu, (kf[j] >> 31) != 0, ev);
    }
    const size_t tl = static_cast<size_t>(l) << LOGN;
    fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);
    wave_relayout<LOGN, LOGE, false>(v, t, lds);
    const auto r_o0 = row_rsrc(ct_out + ((c * 2) * limbs_out + l) * N, N);
    const auto r_o1 = row_rsrc(ct_out + ((c * 2 + 1) * limbs_out + l) * N, N);
    const auto r_a = row_rsrc(a + (c * limbs_out + l) * N, N);
    const auto r_s = row_rsrc(s_ntt + static_cast<size_t>(l) * N, N);
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      const uint32_t av = __builtin_amdgcn_raw_buffer_load_b32(r_a, vofs, j << 8, 0);
      const uint32_t sv = __builtin_amdgcn_raw_buffer_load_b32(r_s, vofs, j << 8, 0);
      __builtin_amdgcn_raw_buffer_store_b32(sub_mod(v[j], mul_mod_barrett(av, sv, q, mu), q), r_o0, vofs, j << 8, 0);
      __builtin_amdgcn_raw_buffer_store_b32(av, r_o1, vofs, j << 8, 0);
    }
  }
}

// Two-kernel refresh for N <= 2^15: the same arithmetic as the fused kernel,
// with each transform in a workgroup of its own and the whole-row plan's
// occupancy (two workgroups per CU up to 2^14, one at 2^15).
// (1) per (ciphertext, limb 0 or 1): c0 + c1 (.) s read coalesced, inverse
//     transform, the coefficient residues written to c1 row 0 / 1 of ct_out
//     (scratch);
// (2) per (ciphertext, output limb): the CRT digits of the two scratch rows,
//     the value mod q_l plus the fresh error, the forward transform, and
//     c0 = . - a (.) s written coalesced;
// c1 = a: rows from 2 on by (2), rows 0 and 1 (the scratch) copied afterwards.
template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN>::P::T), (WholePlan<LOGN>::kWavesPerSimd)) void dte_dec_intt_kernel(
    Tables tb, const uint32_t* __restrict__ ct_in, uint32_t limbs_in, const uint32_t* __restrict__ s_ntt,
    uint32_t limbs_out, uint32_t* __restrict__ ct_out) {
  using P = typename WholePlan<LOGN>::P;
  constexpr int LOGE = WholePlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const size_t c = blockIdx.x >> 1;
  const uint32_t l = blockIdx.x & 1, t = threadIdx.x;
  const uint32_t q = tb.q[l], mu = tb.barrett[l];
  const uint32_t vofs = pos_coalesced<LOGE>(t, 0) * 4;
  const auto r_c0 = row_rsrc(ct_in + ((c * 2) * limbs_in + l) * N, N);
  const auto r_c1 = row_rsrc(ct_in + ((c * 2 + 1) * limbs_in + l) * N, N);
  const auto r_s = row_rsrc(s_ntt + static_cast<size_t>(l) * N, N);
  uint32_t v[P::E], xb[P::E], xs[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    v[j] = __builtin_amdgcn_raw_buffer_load_b32(r_c0, vofs, j << 8, 0);
    xb[j] = __builtin_amdgcn_raw_buffer_load_b32(r_c1, vofs, j << 8, 0);
    xs[j] = __builtin_amdgcn_raw_buffer_load_b32(r_s, vofs, j << 8, 0);
  }
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = add_mod(v[j], mul_mod_barrett(xb[j], xs[j], q, mu), q);
  wave_relayout<LOGN, LOGE, true>(v, t, lds);
  const size_t tl = static_cast<size_t>(l) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + tl, tb.inv_shoup + tl, q, lds);
  const uint32_t ni = tb.ninv[l], nis = tb.ninv_shoup[l];
  uint32_t* r = ct_out + ((c * 2 + 1) * limbs_out + l) * N;
#pragma unroll
  for (int j = 0; j < P::E; ++j) r[P::template pos<0>(t, j)] = mul_shoup(v[j], ni, nis, q);
}

template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN>::P::T), (WholePlan<LOGN>::kWavesPerSimd)) void dte_lift_ntt_kernel(
    Tables tb, const int32_t* __restrict__ e, const uint32_t* __restrict__ s_ntt, const uint32_t* __restrict__ a,
    uint32_t limbs_out, uint32_t* __restrict__ ct_out) {
  using P = typename WholePlan<LOGN>::P;
  constexpr int LOGE = WholePlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  // logical id = c * limbs_out + l.  Consecutive workgroup ids alternate XCDs, so
  // each XCD is given a contiguous range of logical ids: the limbs of one
  // ciphertext then run together on one XCD and read its two scratch rows and
  // its error row from HBM once, the other limbs from that XCD's L2.
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const size_t c = lid / limbs_out;
  const uint32_t l = lid % limbs_out, t = threadIdx.x;
  // scratch rows: coefficient residues mod q0, q1; element j of thread t of the
  // group-0 layout sits at t + T j (buffer loads: the offset j T is a constant)
  const auto rr0 = row_rsrc(ct_out + ((c * 2 + 1) * limbs_out) * N, N);
  const auto rr1 = row_rsrc(ct_out + ((c * 2 + 1) * limbs_out + 1) * N, N);
  const auto rer = row_rsrc(e + c * N, N);
  const uint32_t q0 = tb.q[0], q1 = tb.q[1];
  const uint32_t w = tb.qinv[0 * tb.L + 1], ws = tb.qinv_shoup[0 * tb.L + 1];  // q0^-1 mod q1
  const uint64_t half = static_cast<uint64_t>(q0) * q1 / 2;
  const uint32_t q = tb.q[l], mu = tb.barrett[l];
  const LiftConst lc = lift_const(q0, q1, q, tb.q_recip[l]);
  uint32_t v[P::E];
  // keeps the element loads below the per-limb constants: scheduled above them,
  // the loads' live ranges spill registers
  __builtin_amdgcn_sched_barrier(0);
  // loads in batches of 8 elements, each batch issued before the previous one is
  // used (group 0: element j of thread t at t + T j)
  constexpr int kB = 8;
  uint32_t xa[2][kB], xb[2][kB];
  int32_t ea[2][kB];
  auto load = [&](int set, int j0) {
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      const uint32_t jo = P::template pos<0>(0, j0 + i) * 4;
      xa[set][i] = __builtin_amdgcn_raw_buffer_load_b32(rr0, t * 4, jo, 0);
      xb[set][i] = __builtin_amdgcn_raw_buffer_load_b32(rr1, t * 4, jo, 0);
      ea[set][i] = static_cast<int32_t>(__builtin_amdgcn_raw_buffer_load_b32(rer, t * 4, jo, 0));
    }
  };
  load(0, 0);
#pragma unroll
  for (int j0 = 0; j0 < P::E; j0 += kB) {
    const int cur = (j0 / kB) & 1;
    if (j0 + kB < P::E) load(cur ^ 1, j0 + kB);
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      const uint32_t x0 = xa[cur][i];
      const uint32_t r0m = x0 >= q1 ? x0 - q1 : x0;                          // x0 < q0 < 2 q1
      const uint32_t k = mul_shoup(sub_mod(xb[cur][i], r0m, q1), w, ws, q1);
      const bool neg = static_cast<uint64_t>(x0) + static_cast<uint64_t>(q0) * k > half;
      v[j0 + i] = lift_residue(lc, x0, k, neg, ea[cur][i]);
    }
  }
  const size_t tl = static_cast<size_t>(l) << LOGN;
  fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);
  wave_relayout<LOGN, LOGE, false>(v, t, lds);
  __builtin_amdgcn_sched_barrier(0);  // the combine's loads stay after the transform
  const uint32_t vofs = pos_coalesced<LOGE>(t, 0) * 4;
  const auto ra = row_rsrc(a + (c * limbs_out + l) * N, N);
  const auto rs = row_rsrc(s_ntt + static_cast<size_t>(l) * N, N);
  const auto ro = row_rsrc(ct_out + ((c * 2) * limbs_out + l) * N, N);
  const auto ro1 = row_rsrc(ct_out + ((c * 2 + 1) * limbs_out + l) * N, N);  // c1 row l (rows 0, 1 are the scratch)
  uint32_t ya[2][kB], ys[2][kB];
  auto load_as = [&](int set, int j0) {
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      ya[set][i] = __builtin_amdgcn_raw_buffer_load_b32(ra, vofs, (j0 + i) << 8, 0);
      ys[set][i] = __builtin_amdgcn_raw_buffer_load_b32(rs, vofs, (j0 + i) << 8, 0);
    }
  };
  load_as(0, 0);
#pragma unroll
  for (int j0 = 0; j0 < P::E; j0 += kB) {
    const int cur = (j0 / kB) & 1;
    if (j0 + kB < P::E) load_as(cur ^ 1, j0 + kB);
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      const uint32_t ax = ya[cur][i];
      __builtin_amdgcn_raw_buffer_store_b32(sub_mod(v[j0 + i], mul_mod_barrett(ax, ys[cur][i], q, mu), q), ro, vofs,
                                            (j0 + i) << 8, 0);
      if (l >= 2) __builtin_amdgcn_raw_buffer_store_b32(ax, ro1, vofs, (j0 + i) << 8, 0);
    }
  }
}

template <int LOGN>
hipError_t launch_refresh_two(const Tables& t, const uint32_t* ct_in, uint32_t limbs_in, const uint32_t* s_ntt,
                              const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs_out,
                              uint32_t* ct_out, hipStream_t s) {
  constexpr uint32_t T = WholePlan<LOGN>::P::T;
  dte_dec_intt_kernel<LOGN><<<dim3(2 * count), T, 0, s>>>(t, ct_in, limbs_in, s_ntt, limbs_out, ct_out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  dte_lift_ntt_kernel<LOGN><<<dim3(count * limbs_out), T, 0, s>>>(t, e, s_ntt, a, limbs_out, ct_out);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  // c1 rows 0 and 1 (the scratch) = a rows 0 and 1; the kernel wrote the others
  const size_t ct_bytes = static_cast<size_t>(2) * limbs_out * t.n * 4, a_bytes = ct_bytes / 2;
  return hipMemcpy2DAsync(ct_out + static_cast<size_t>(limbs_out) * t.n, ct_bytes, a, a_bytes, 2 * t.n * 4, count,
                          hipMemcpyDeviceToDevice, s);
}

template <int LOGN>
hipError_t launch_refresh_fused(const Tables& t, const uint32_t* ct_in, uint32_t limbs_in, const uint32_t* s_ntt,
                                const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs_out,
                                uint32_t* ct_out, hipStream_t s) {
  refresh_kernel<LOGN><<<dim3(count, limbs_out), RefreshPlan<LOGN>::P::T, 0, s>>>(t, ct_in, limbs_in, s_ntt, a, e,
                                                                                 limbs_out, ct_out);
  return hipGetLastError();
}

uint32_t quad_grid(uint32_t n, uint32_t count) {
  const size_t quads = static_cast<size_t>(count) * (n / 4);
  return static_cast<uint32_t>((quads + kThreads - 1) / kThreads);
}

}  // namespace

hipError_t launch_encrypt(const Tables& t, const uint32_t* pt, const uint32_t* s_ntt, const uint32_t* a,
                          const int32_t* e, uint32_t count, uint32_t limbs, uint32_t* ct, hipStream_t s) {
  const uint32_t grid = quad_grid(t.n, count);
  err_rows_kernel<<<grid, kThreads, 0, s>>>(t, e, count, limbs, ct);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  err = launch_ntt(t, ct, static_cast<size_t>(count) * limbs, limbs, false, s, 2 * limbs);  // c0 rows
  if (err != hipSuccess) return err;
  enc_combine_kernel<<<grid, kThreads, 0, s>>>(t, pt, s_ntt, a, count, limbs, ct);
  return hipGetLastError();
}

hipError_t launch_decrypt(const Tables& t, const uint32_t* ct, const uint32_t* s_ntt, uint32_t count,
                          uint32_t limbs, uint32_t* m, hipStream_t s) {
  dec_pointwise_kernel<<<quad_grid(t.n, count), kThreads, 0, s>>>(t, ct, limbs, s_ntt, count, limbs, m, limbs, 0);
  const hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_ntt(t, m, static_cast<size_t>(count) * limbs, limbs, true, s);
}

hipError_t launch_refresh(const Tables& t, const uint32_t* ct_in, uint32_t limbs_in, const uint32_t* s_ntt,
                          const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs_out,
                          uint32_t* ct_out, hipStream_t s) {
  // Up to 2^13, launches of at most one fused workgroup (ciphertext x output
  // limb) per CU take the fused kernel split by output limb, whose chain is
  // three transforms (64 ciphertexts x 4 limbs at 2^13: 26.7 against 30.7 us);
  // larger ones, and every count at 2^14 (its fused workgroup is 1024
  // threads), the two-kernel route (32 ciphertexts at 2^14: 40.9 against
  // 41.8 us; 128: 62.5 against 89.5 us; 768: 0.36 against 0.52 ms).  At 2^15
  // it replaces the pointwise passes (768 ciphertexts x 4 limbs: 0.79 against
  // 1.01 ms; 32: 66 against 72 us).
  if (t.log_n >= 14 || static_cast<size_t>(count) * limbs_out > t.num_cus) {
    switch (t.log_n) {
      case 10: return launch_refresh_two<10>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      case 11: return launch_refresh_two<11>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      case 12: return launch_refresh_two<12>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      case 13: return launch_refresh_two<13>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      case 14: return launch_refresh_two<14>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      case 15: return launch_refresh_two<15>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
      default: break;
    }
  }
  switch (t.log_n) {
    case 10: return launch_refresh_fused<10>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
    case 11: return launch_refresh_fused<11>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
    case 12: return launch_refresh_fused<12>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
    case 13: return launch_refresh_fused<13>(t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out, s);
    default: break;
  }
  // N = 2^16 (a row exceeds the LDS): pointwise passes around the batched
  // transforms
  const uint32_t grid = quad_grid(t.n, count);
  const uint32_t gs = 2 * limbs_out;
  // 1. limbs 0 and 1 of c0 + c1 (.) s into the c1 rows 0, 1 of ct_out (scratch), then INTT them
  dec_pointwise_kernel<<<grid, kThreads, 0, s>>>(t, ct_in, limbs_in, s_ntt, count, 2, ct_out, gs, limbs_out);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  err = launch_ntt(t, ct_out + static_cast<size_t>(limbs_out) * t.n, static_cast<size_t>(count) * 2, 2, true, s, gs);
  if (err != hipSuccess) return err;
  // 2. CRT lift + fresh error, reduced under limbs_out limbs, into the c0 rows; NTT them
  dte_lift_kernel<<<grid, kThreads, 0, s>>>(t, e, count, limbs_out, ct_out);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  err = launch_ntt(t, ct_out, static_cast<size_t>(count) * limbs_out, limbs_out, false, s, gs);
  if (err != hipSuccess) return err;
  // 3. c0 -= a (.) s, c1 = a (overwrites the scratch rows)
  enc_combine_kernel<<<grid, kThreads, 0, s>>>(t, nullptr, s_ntt, a, count, limbs_out, ct_out);
  return hipGetLastError();
}

}  // namespace ckks
