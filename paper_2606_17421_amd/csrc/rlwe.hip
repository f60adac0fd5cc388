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
// The transforms are the batched NTT kernels, run over the c0 rows (or a
// pair of scratch rows) of the ciphertext buffer through their row-group
// stride; the kernels here are the pointwise passes around them, 16 bytes
// per thread and limb.
#include "ckks_internal.hpp"

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

// a * b mod q for residues a, b < q.
__device__ __forceinline__ uint32_t mul_mod(uint32_t a, uint32_t b, uint32_t q, double qr) {
  return reduce_u64(static_cast<uint64_t>(a) * b, q, qr);
}

// Signed 64-bit x mod q, in [0, q).
__device__ __forceinline__ uint32_t reduce_i64(int64_t x, uint32_t q, double qr) {
  const uint64_t ax = static_cast<uint64_t>(x < 0 ? -x : x);
  const uint32_t r = reduce_u64(ax, q, qr);
  return (x < 0 && r != 0) ? q - r : r;
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
    const uint32_t q = tb.q[l];
    const double qr = tb.q_recip[l];
    const size_t row = (p.c * limbs + l) * n + p.k;
    uint32_t* c0p = ct + ((p.c * 2) * limbs + l) * n + p.k;
    uint32_t* c1p = c0p + static_cast<size_t>(limbs) * n;
    const v4u c0 = ld4(c0p);
    const v4u av = ld4(a + row);
    const v4u sv = ld4(s_ntt + static_cast<size_t>(l) * n + p.k);
    const v4u pv = pt ? ld4(pt + row) : v4u{0, 0, 0, 0};
    v4u o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = sub_mod(add_mod(c0[j], pv[j], q), mul_mod(av[j], sv[j], q, qr), q);
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
    const uint32_t q = tb.q[l];
    const double qr = tb.q_recip[l];
    const uint32_t* c0p = ct + ((p.c * 2) * ct_limbs + l) * n + p.k;
    const v4u c0 = ld4(c0p);
    const v4u c1 = ld4(c0p + static_cast<size_t>(ct_limbs) * n);
    const v4u sv = ld4(s_ntt + static_cast<size_t>(l) * n + p.k);
    v4u o;
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = add_mod(c0[j], mul_mod(c1[j], sv[j], q, qr), q);
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
