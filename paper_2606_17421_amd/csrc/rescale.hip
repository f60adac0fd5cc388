// Rescale kernels (gfx950): divide by the last prime q_t (t = limbs - 1) and
// drop it (section 2.1), in NTT form:
//     r     = centred INTT_t(c_t)              (|r| < q_t / 2)
//     out_l = (c_l - NTT_l(r mod q_l)) * q_t^-1   mod q_l,   l < t.
//
// N <= 2^15: one workgroup per polynomial (ciphertext component).  The last
// limb is inverse-transformed through the register-group NTT, and the centred
// residues stay in registers (group-0 layout, which is also the forward
// transform's starting layout) while each remaining limb is forward-
// transformed and combined with c_l on the way out.  HBM traffic is the
// minimum: read limbs rows, write limbs - 1 rows.
// N = 2^16: staged through a workspace with the two-pass NTT.
#include "ntt_core.hpp"

namespace ckks {
namespace {

template <int LOGN>
__global__ __launch_bounds__(WholePlan<LOGN>::P::T, WholePlan<LOGN>::kWavesPerSimd) void rescale_kernel(
    Tables tb, const uint32_t* __restrict__ in, uint32_t* __restrict__ out, uint32_t limbs) {
  using P = typename WholePlan<LOGN>::P;
  constexpr int LOGE = WholePlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const size_t poly = blockIdx.x;  // ciphertext * 2 + component
  const uint32_t t = threadIdx.x;
  const uint32_t* src = in + poly * limbs * N;
  uint32_t* dst = out + poly * (limbs - 1) * N;
  const uint32_t top = limbs - 1;
  const uint32_t qt = tb.q[top];

  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = src[static_cast<size_t>(top) * N + P::template pos<P::NG - 1>(t, j)];
  const size_t ttop = static_cast<size_t>(top) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + ttop, tb.inv_shoup + ttop, qt, lds);
  const uint32_t ni = tb.ninv[top], nis = tb.ninv_shoup[top];
  int32_t r[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t x = mul_shoup(v[j], ni, nis, qt);
    r[j] = x > (qt >> 1) ? static_cast<int32_t>(x) - static_cast<int32_t>(qt) : static_cast<int32_t>(x);
  }

  for (uint32_t l = 0; l < top; ++l) {
    const uint32_t q = tb.q[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = static_cast<uint32_t>(r[j] < 0 ? r[j] + static_cast<int32_t>(q) : r[j]);
    const size_t tl = static_cast<size_t>(l) << LOGN;
    fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);
    const uint32_t qi = tb.qinv[top * tb.L + l], qis = tb.qinv_shoup[top * tb.L + l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      const size_t x = static_cast<size_t>(l) * N + P::template pos<P::NG - 1>(t, j);
      dst[x] = mul_shoup(sub_mod(src[x], v[j], q), qi, qis, q);
    }
  }
}

// ---- N = 2^16 staging kernels (rows of 2^16 residues) ----------------------
constexpr int kT = 256;

// A[p] = in[p][top]  for p < polys
__global__ __launch_bounds__(kT) void gather_top_kernel(const uint32_t* __restrict__ in,
                                                        uint32_t* __restrict__ A, uint32_t limbs,
                                                        size_t polys) {
  const size_t words = polys << 16;
  const size_t stride = static_cast<size_t>(gridDim.x) * kT;
  for (size_t i = static_cast<size_t>(blockIdx.x) * kT + threadIdx.x; i < words; i += stride) {
    const size_t p = i >> 16, k = i & 0xFFFF;
    A[i] = in[((p * limbs) + limbs - 1) * 65536 + k];
  }
}

// B = centred(A) mod q_l, A holding residues mod q_top
__global__ __launch_bounds__(kT) void centre_reduce_kernel(Tables tb, const uint32_t* __restrict__ A,
                                                           uint32_t* __restrict__ B, uint32_t top,
                                                           uint32_t l, size_t words) {
  const uint32_t qt = tb.q[top], q = tb.q[l];
  const size_t stride = static_cast<size_t>(gridDim.x) * kT;
  for (size_t i = static_cast<size_t>(blockIdx.x) * kT + threadIdx.x; i < words; i += stride) {
    const uint32_t x = A[i];
    const int32_t r = x > (qt >> 1) ? static_cast<int32_t>(x) - static_cast<int32_t>(qt) : static_cast<int32_t>(x);
    B[i] = static_cast<uint32_t>(r < 0 ? r + static_cast<int32_t>(q) : r);
  }
}

// out[p][l] = (in[p][l] - B[p]) * q_top^-1 mod q_l
__global__ __launch_bounds__(kT) void combine_kernel(Tables tb, const uint32_t* __restrict__ in,
                                                     const uint32_t* __restrict__ B,
                                                     uint32_t* __restrict__ out, uint32_t limbs,
                                                     uint32_t l, size_t polys) {
  const uint32_t top = limbs - 1;
  const uint32_t q = tb.q[l], qi = tb.qinv[top * tb.L + l], qis = tb.qinv_shoup[top * tb.L + l];
  const size_t words = polys << 16;
  const size_t stride = static_cast<size_t>(gridDim.x) * kT;
  for (size_t i = static_cast<size_t>(blockIdx.x) * kT + threadIdx.x; i < words; i += stride) {
    const size_t p = i >> 16, k = i & 0xFFFF;
    const uint32_t c = in[(p * limbs + l) * 65536 + k];
    out[(p * (limbs - 1) + l) * 65536 + k] = mul_shoup(sub_mod(c, B[i], q), qi, qis, q);
  }
}

constexpr size_t kChunkPolys16 = 1024;  // polynomials staged per pass for N = 2^16

uint32_t grid_for(size_t words) {
  size_t g = (words + kT - 1) / kT;
  return static_cast<uint32_t>(g > 16384 ? 16384 : g);
}

// Tables restricted to limb l (so a one-limb batch transforms with q_l).
Tables limb_view(const Tables& t, uint32_t l) {
  Tables v = t;
  const size_t off = static_cast<size_t>(l) << t.log_n;
  v.q += l;
  v.fwd += off;
  v.fwd_shoup += off;
  v.inv += off;
  v.inv_shoup += off;
  v.ninv += l;
  v.ninv_shoup += l;
  return v;
}

hipError_t rescale16(const Tables& t, const uint32_t* in, uint32_t* out, uint32_t count,
                     uint32_t limbs, void* workspace, hipStream_t s) {
  const size_t polys_total = static_cast<size_t>(count) * 2;
  const size_t chunk = polys_total < kChunkPolys16 ? polys_total : kChunkPolys16;
  uint32_t* A = static_cast<uint32_t*>(workspace);  // [chunk][2^16]
  uint32_t* B = A + (chunk << 16);                  // [chunk][2^16]
  const uint32_t top = limbs - 1;
  for (size_t p0 = 0; p0 < polys_total; p0 += chunk) {
    const size_t np = polys_total - p0 < chunk ? polys_total - p0 : chunk;
    const uint32_t* src = in + p0 * limbs * 65536;
    uint32_t* dst = out + p0 * (limbs - 1) * 65536;
    gather_top_kernel<<<grid_for(np << 16), kT, 0, s>>>(src, A, limbs, np);
    hipError_t e = launch_ntt(limb_view(t, top), A, np, 1, true, s);
    if (e != hipSuccess) return e;
    for (uint32_t l = 0; l < top; ++l) {
      centre_reduce_kernel<<<grid_for(np << 16), kT, 0, s>>>(t, A, B, top, l, np << 16);
      e = launch_ntt(limb_view(t, l), B, np, 1, false, s);
      if (e != hipSuccess) return e;
      combine_kernel<<<grid_for(np << 16), kT, 0, s>>>(t, src, B, dst, limbs, l, np);
    }
  }
  return hipGetLastError();
}

template <int LOGN>
hipError_t launch_rescale_whole(const Tables& t, const uint32_t* in, uint32_t* out, uint32_t count,
                                uint32_t limbs, hipStream_t s) {
  rescale_kernel<LOGN><<<dim3(2 * count), WholePlan<LOGN>::P::T, 0, s>>>(t, in, out, limbs);
  return hipGetLastError();
}

}  // namespace

size_t rescale_workspace_bytes(const Tables& t, uint32_t count) {
  if (t.log_n < 16) return 0;
  const size_t polys = static_cast<size_t>(count) * 2;
  const size_t chunk = polys < kChunkPolys16 ? polys : kChunkPolys16;
  return 2 * (chunk << 16) * sizeof(uint32_t);
}

hipError_t launch_rescale(const Tables& t, const uint32_t* ct_in, uint32_t* ct_out, uint32_t count,
                          uint32_t limbs, void* workspace, hipStream_t s) {
  if (count == 0) return hipSuccess;
  switch (t.log_n) {
    case 10: return launch_rescale_whole<10>(t, ct_in, ct_out, count, limbs, s);
    case 11: return launch_rescale_whole<11>(t, ct_in, ct_out, count, limbs, s);
    case 12: return launch_rescale_whole<12>(t, ct_in, ct_out, count, limbs, s);
    case 13: return launch_rescale_whole<13>(t, ct_in, ct_out, count, limbs, s);
    case 14: return launch_rescale_whole<14>(t, ct_in, ct_out, count, limbs, s);
    case 15: return launch_rescale_whole<15>(t, ct_in, ct_out, count, limbs, s);
    case 16: return rescale16(t, ct_in, ct_out, count, limbs, workspace, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ckks
