// Weight encoding kernels (gfx950): scalar constants and full-polynomial
// slot vectors (the per-call fallback encode).
//
// Full-polynomial route for real slots.  With e_j = 5^j mod 2N, each slot
// exponent e_j or 2N - e_j is an odd t = 2u + 1 < N, and the coefficients of
// the inverse canonical embedding reduce to a DCT-II of length M = N/2:
//     m_k = (2/N) X_k,  X_k = sum_{u<M} y_u cos(pi (2u+1) k / N),  y_u = z_{j(u)},
// with m_{N/2} = 0 and m_{N-k} = -m_k.  X is computed with Makhoul's
// reordering (v_n = y_2n, v_{M-1-n} = y_{2n+1}; X_k = Re(exp(-i pi k/2M) V_k),
// V = DFT_M(v)), and the real DFT of length M is folded into one complex DFT
// of length P = M/2, run in LDS in fp64 (radix-2 decimation in frequency).
#include "ckks_internal.hpp"

namespace ckks {
namespace {

constexpr int kEncScalarThreads = 256;

__global__ __launch_bounds__(kEncScalarThreads) void encode_scalar_kernel(
    const uint32_t* __restrict__ q, const double* __restrict__ q_recip,
    const double* __restrict__ w, size_t count, uint32_t limbs, double scale,
    uint32_t* __restrict__ w_enc) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kEncScalarThreads + threadIdx.x;
  if (i >= count) return;
  const double v = rint(w[i] * scale);
  for (uint32_t l = 0; l < limbs; ++l) w_enc[i * limbs + l] = reduce_f64_int(v, q[l], q_recip[l]);
}

__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
  return make_double2(fma(a.x, b.x, -a.y * b.y), fma(a.x, b.y, a.y * b.x));
}
__device__ __forceinline__ double2 cadd(double2 a, double2 b) { return make_double2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ double2 csub(double2 a, double2 b) { return make_double2(a.x - b.x, a.y - b.y); }

template <int LOGN>
struct EncPlan {
  static constexpr int N = 1 << LOGN;
  static constexpr int M = N / 2;
  static constexpr int LOGP = LOGN - 2;
  static constexpr int P = N / 4;
  static constexpr int T = P / 2 < 1024 ? P / 2 : 1024;
};

// One workgroup per slot vector: writes coefficient-form residues pt[b][l][0..N).
template <int LOGN>
__global__ __launch_bounds__(EncPlan<LOGN>::T) void encode_poly_coeffs_kernel(
    Tables tb, const double* __restrict__ slots, uint32_t limbs, double scale,
    uint32_t* __restrict__ pt) {
  using EP = EncPlan<LOGN>;
  constexpr int N = EP::N, M = EP::M, P = EP::P, T = EP::T;
  __shared__ double2 a[P];
  const size_t b = blockIdx.x;
  const double* z = slots + b * M;
  uint32_t* out = pt + b * static_cast<size_t>(limbs) * N;

  // c_n = v_2n + i v_2n+1, v_m = y_{u(m)}, u(m) = 2m (m < M/2) or 2(M-1-m)+1.
  for (int n = threadIdx.x; n < P; n += T) {
    const int m0 = 2 * n, m1 = 2 * n + 1;
    const int u0 = m0 < M / 2 ? 2 * m0 : 2 * (M - 1 - m0) + 1;
    const int u1 = m1 < M / 2 ? 2 * m1 : 2 * (M - 1 - m1) + 1;
    a[n] = make_double2(z[tb.slot_perm[u0]], z[tb.slot_perm[u1]]);
  }
  __syncthreads();

  // Radix-2 DIF DFT of length P (forward sign); output in bit-reversed order.
  for (int s = 0; s < EP::LOGP; ++s) {
    const int d = P >> (s + 1);
    for (int idx = threadIdx.x; idx < P / 2; idx += T) {
      const int i = idx & (d - 1);
      const int x = ((idx >> (EP::LOGP - 1 - s)) << (EP::LOGP - s)) | i;  // (idx / d) * 2d + i
      const double2 U = a[x], V = a[x + d];
      a[x] = cadd(U, V);
      a[x + d] = cmul(csub(U, V), tb.fft_tw[i << s]);
    }
    __syncthreads();
  }

  const double two_over_n = 2.0 / N;
  for (int k = threadIdx.x; k < P; k += T) {
    const int kr = static_cast<int>(__brev(static_cast<uint32_t>(k)) >> (32 - EP::LOGP));
    const int km = (P - k) & (P - 1);
    const int kmr = static_cast<int>(__brev(static_cast<uint32_t>(km)) >> (32 - EP::LOGP));
    const double2 ck = a[kr];
    const double2 cm = a[kmr];
    const double2 cmc = make_double2(cm.x, -cm.y);
    const double2 e = make_double2(0.5 * (ck.x + cmc.x), 0.5 * (ck.y + cmc.y));
    const double2 dd = csub(ck, cmc);                      // O = dd / (2i) = (dd.y, -dd.x) / 2
    const double2 o = make_double2(0.5 * dd.y, -0.5 * dd.x);
    const double2 wo = cmul(tb.rfft_tw[k], o);
    const double2 v_lo = cadd(e, wo);                      // V_k
    const double2 v_hi = csub(e, wo);                      // V_{k+P}
    const double2 t_lo = tb.dct_tw[k], t_hi = tb.dct_tw[k + P];
    const double x_lo = t_lo.x * v_lo.x - t_lo.y * v_lo.y;  // Re(exp(-i pi k/2M) V_k)
    const double x_hi = t_hi.x * v_hi.x - t_hi.y * v_hi.y;
    const double p_lo = rint(scale * (two_over_n * x_lo));
    const double p_hi = rint(scale * (two_over_n * x_hi));
    const int k_hi = k + P;
    for (uint32_t l = 0; l < limbs; ++l) {
      const uint32_t q = tb.q[l];
      const double qr = tb.q_recip[l];
      uint32_t* row = out + static_cast<size_t>(l) * N;
      const uint32_t r_lo = reduce_f64_int(p_lo, q, qr);
      const uint32_t r_hi = reduce_f64_int(p_hi, q, qr);
      row[k] = r_lo;
      row[k_hi] = r_hi;
      // m_{N-k} = -m_k for 0 < k < M; m_{N/2} = 0.
      if (k == 0) row[M] = 0;
      else row[N - k] = r_lo ? q - r_lo : 0;
      row[N - k_hi] = r_hi ? q - r_hi : 0;
    }
  }
}

template <int LOGN>
hipError_t launch_poly(const Tables& t, const double* slots, uint32_t count, uint32_t limbs,
                       double scale, uint32_t* pt, hipStream_t s) {
  encode_poly_coeffs_kernel<LOGN><<<count, EncPlan<LOGN>::T, 0, s>>>(t, slots, limbs, scale, pt);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_encode_scalar(const Tables& t, const double* w, size_t count, uint32_t limbs,
                                double scale, uint32_t* w_enc, hipStream_t s) {
  if (count == 0) return hipSuccess;
  const size_t grid = (count + kEncScalarThreads - 1) / kEncScalarThreads;
  encode_scalar_kernel<<<static_cast<uint32_t>(grid), kEncScalarThreads, 0, s>>>(
      t.q, t.q_recip, w, count, limbs, scale, w_enc);
  return hipGetLastError();
}

hipError_t launch_encode_poly_coeffs(const Tables& t, const double* slots, uint32_t count,
                                     uint32_t limbs, double scale, uint32_t* pt, hipStream_t s) {
  if (count == 0) return hipSuccess;
  switch (t.log_n) {
    case 10: return launch_poly<10>(t, slots, count, limbs, scale, pt, s);
    case 11: return launch_poly<11>(t, slots, count, limbs, scale, pt, s);
    case 12: return launch_poly<12>(t, slots, count, limbs, scale, pt, s);
    case 13: return launch_poly<13>(t, slots, count, limbs, scale, pt, s);
    case 14: return launch_poly<14>(t, slots, count, limbs, scale, pt, s);
    case 15: return launch_poly<15>(t, slots, count, limbs, scale, pt, s);
    default: return hipErrorNotSupported;
  }
}

}  // namespace ckks
