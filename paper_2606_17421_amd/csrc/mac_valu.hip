// Vector-ALU modular MAC kernels (gfx950).
//
// Scalar weights: per limb a modular GEMM (d_out x d_in) . (d_in x 2N); each
// thread owns one (component, NTT slot) column and kRows output rows, keeps
// u64 accumulators fed by v_mad_u64_u32, and reduces every 15 products
// (15 * 2^60 + 2^30 < 2^64).  Weights are wave-uniform (scalar loads).
// Full-polynomial weights: slot-wise products, the plaintexts streamed once
// from HBM; each thread owns one (limb, slot), both ciphertext components and
// a group of output rows.
#include "ckks_internal.hpp"

namespace ckks {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = 8;
constexpr int kLazy = 15;

__global__ __launch_bounds__(kThreads) void mac_scalar_valu_kernel(
    Tables tb, const uint32_t* __restrict__ w_enc, const uint32_t* __restrict__ ct_in,
    uint32_t* __restrict__ ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  const uint32_t n = tb.n;
  const uint32_t col = blockIdx.x * kThreads + threadIdx.x;  // < 2N
  const uint32_t c = col >> tb.log_n;
  const uint32_t k = col & (n - 1);
  const uint32_t l = blockIdx.z;
  const uint32_t j0 = blockIdx.y * kRows;
  const uint32_t q = tb.q[l];
  const double qr = tb.q_recip[l];
  const size_t in_stride = 2ull * limbs * n;
  const uint32_t* x_ptr = ct_in + (static_cast<size_t>(c) * limbs + l) * n + k;
  size_t w_row[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const uint32_t j = min(j0 + r, d_out - 1);  // clamp: rows past d_out are computed, not stored
    w_row[r] = static_cast<size_t>(j) * d_in * limbs + l;
  }
  uint64_t acc[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) acc[r] = 0;
  uint32_t i = 0;
  while (i < d_in) {
    const uint32_t stop = min(d_in, i + kLazy);
    for (; i < stop; ++i) {
      const uint64_t x = x_ptr[i * in_stride];
#pragma unroll
      for (int r = 0; r < kRows; ++r) acc[r] += x * w_enc[w_row[r] + static_cast<size_t>(i) * limbs];
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) acc[r] = reduce_u64(acc[r], q, qr);
  }
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const uint32_t j = j0 + r;
    if (j < d_out)
      ct_out[((static_cast<size_t>(j) * 2 + c) * limbs + l) * n + k] = static_cast<uint32_t>(acc[r]);
  }
}

// Full-polynomial weights: thread = (limb l, slots k .. k+3) for kPolyRows
// outputs j0 .. j0 + kPolyRows - 1, with 16-byte loads.  Each ciphertext
// residue quad is loaded once per kPolyRows outputs; every plaintext residue
// is read exactly once.  Workgroups with the same (l, slot block) and
// consecutive row groups are adjacent in logical order, and each XCD runs a
// contiguous range of logical ids, so the shared ciphertext columns are
// fetched once into that XCD's L2.  Four rows per thread when the grid
// still holds at least 8 workgroups per CU; narrower layers (the 32-output
// groups of a decode stack or a BSGS giant-step set) take two rows per thread
// for twice the workgroups: 47.7 -> 32.2 us at 32 x 32, 4 limbs, N = 2^13
// (2.8 -> 4.2 TB/s of plaintext stream).  Per input the row loads are all
// issued before the first product (a ragged last group re-reads row 0 for its
// missing rows and discards those sums), so a wave waits on memory once per
// input instead of once per row: 31.1 -> 24.9 us at 32 x 32, 2^13, 4 limbs.
// The 4-row kernel (wide layers) loads the plaintexts, which are read once,
// non-temporally, so that they do not displace the ciphertext columns every
// row group re-reads from L2: 669 -> 623 us at 64 x 64, 2^15, 6 limbs.  At
// 32 x 32 the non-temporal loads were slower, so the 2-row kernel keeps plain
// loads.  Both kernels store their outputs non-temporally (written once): 621
// -> 600 us at 64 x 64, 2^15, 6 limbs; 53 -> 49.5 us at 32 x 32, 2^14, 4 limbs.
constexpr int kPolySlots = 4;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <bool kNonTemporal>
__device__ __forceinline__ uint4 load_pt(const uint4* p) {
  if constexpr (kNonTemporal) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    return *p;
  }
}

template <int kPolyRows>
__global__ __launch_bounds__(kThreads) void mac_poly_kernel(
    Tables tb, const uint32_t* __restrict__ pt, const uint32_t* __restrict__ ct_in,
    uint32_t* __restrict__ ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  const uint32_t n = tb.n;
  const uint32_t groups = (d_out + kPolyRows - 1) / kPolyRows;
  const uint32_t blocks_per_row = n / (kThreads * kPolySlots);
  // blockIdx.x = (l * blocks_per_row + kb) * groups + g
  // Consecutive workgroup ids alternate XCDs: each XCD takes a contiguous
  // range of logical ids, so the row groups sharing a column block meet in one L2.
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const uint32_t g = lid % groups;
  const uint32_t lk = lid / groups;
  const uint32_t l = lk / blocks_per_row;
  const uint32_t k = ((lk % blocks_per_row) * kThreads + threadIdx.x) * kPolySlots;
  const uint32_t j0 = g * kPolyRows;
  const uint32_t rows = d_out - j0 < kPolyRows ? d_out - j0 : kPolyRows;  // workgroup-uniform
  const uint32_t q = tb.q[l];
  const double qr = tb.q_recip[l];
  const size_t ln = static_cast<size_t>(limbs) * n;
  const uint4* p_ptr = reinterpret_cast<const uint4*>(pt + (static_cast<size_t>(j0) * d_in * limbs + l) * n + k);
  const size_t p_row = static_cast<size_t>(d_in) * ln / 4;  // one output's plaintexts, in uint4
  const size_t ln4 = ln / 4;
  const uint4* x_ptr = reinterpret_cast<const uint4*>(ct_in + static_cast<size_t>(l) * n + k);
  uint64_t a0[kPolyRows][kPolySlots], a1[kPolyRows][kPolySlots];
#pragma unroll
  for (int r = 0; r < kPolyRows; ++r)
#pragma unroll
    for (int e = 0; e < kPolySlots; ++e) a0[r][e] = a1[r][e] = 0;
  uint32_t i = 0;
  while (i < d_in) {
    const uint32_t stop = min(d_in, i + kLazy);
    for (; i < stop; ++i) {
      const uint4 x0 = x_ptr[(2ull * i) * ln4], x1 = x_ptr[(2ull * i + 1) * ln4];
      uint4 pv[kPolyRows];
#pragma unroll
      for (int r = 0; r < kPolyRows; ++r) {
        const uint32_t rr = r < rows ? r : 0;  // rows >= 1; sums of rows past d_out are not stored
        pv[r] = load_pt<kPolyRows == 4>(&p_ptr[rr * p_row + static_cast<size_t>(i) * ln4]);
      }
      const uint32_t xs0[4] = {x0.x, x0.y, x0.z, x0.w}, xs1[4] = {x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int r = 0; r < kPolyRows; ++r) {
        const uint32_t ps[4] = {pv[r].x, pv[r].y, pv[r].z, pv[r].w};
#pragma unroll
        for (int e = 0; e < kPolySlots; ++e) {
          a0[r][e] += static_cast<uint64_t>(ps[e]) * xs0[e];
          a1[r][e] += static_cast<uint64_t>(ps[e]) * xs1[e];
        }
      }
    }
#pragma unroll
    for (int r = 0; r < kPolyRows; ++r)
#pragma unroll
      for (int e = 0; e < kPolySlots; ++e) {
        a0[r][e] = reduce_u64(a0[r][e], q, qr);
        a1[r][e] = reduce_u64(a1[r][e], q, qr);
      }
  }
#pragma unroll
  for (int r = 0; r < kPolyRows; ++r) {
    if (r < rows) {
      u32x4* o = reinterpret_cast<u32x4*>(ct_out + ((static_cast<size_t>(j0 + r) * 2) * limbs + l) * n + k);
      __builtin_nontemporal_store(u32x4{static_cast<uint32_t>(a0[r][0]), static_cast<uint32_t>(a0[r][1]),
                                        static_cast<uint32_t>(a0[r][2]), static_cast<uint32_t>(a0[r][3])}, &o[0]);
      __builtin_nontemporal_store(u32x4{static_cast<uint32_t>(a1[r][0]), static_cast<uint32_t>(a1[r][1]),
                                        static_cast<uint32_t>(a1[r][2]), static_cast<uint32_t>(a1[r][3])}, &o[ln4]);
    }
  }
}

__global__ __launch_bounds__(kThreads) void zero_kernel(uint32_t* p, size_t words) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x;
  const size_t stride = static_cast<size_t>(gridDim.x) * kThreads;
  for (size_t k = i; k < words; k += stride) p[k] = 0;
}

}  // namespace

hipError_t launch_mac_scalar_valu(const Tables& t, const uint32_t* w_enc, const uint32_t* ct_in,
                                  uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                  hipStream_t s) {
  dim3 grid(2 * t.n / kThreads, (d_out + kRows - 1) / kRows, limbs);
  mac_scalar_valu_kernel<<<grid, kThreads, 0, s>>>(t, w_enc, ct_in, ct_out, d_out, d_in, limbs);
  return hipGetLastError();
}

hipError_t launch_mac_poly(const Tables& t, const uint32_t* pt, const uint32_t* ct_in,
                           uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                           hipStream_t s) {
  const size_t blocks = static_cast<size_t>(limbs) * (t.n / (kThreads * kPolySlots));
  const size_t grid4 = static_cast<size_t>((d_out + 3) / 4) * blocks;
  if (grid4 >= 8 * static_cast<size_t>(t.num_cus)) {
    mac_poly_kernel<4><<<static_cast<uint32_t>(grid4), kThreads, 0, s>>>(t, pt, ct_in, ct_out, d_out, d_in, limbs);
  } else {
    const size_t grid2 = static_cast<size_t>((d_out + 1) / 2) * blocks;
    mac_poly_kernel<2><<<static_cast<uint32_t>(grid2), kThreads, 0, s>>>(t, pt, ct_in, ct_out, d_out, d_in, limbs);
  }
  return hipGetLastError();
}

hipError_t launch_zero(uint32_t* p, size_t words, hipStream_t s) {
  if (words == 0) return hipSuccess;
  size_t grid = (words + kThreads - 1) / kThreads;
  if (grid > 65536) grid = 65536;
  zero_kernel<<<static_cast<uint32_t>(grid), kThreads, 0, s>>>(p, words);
  return hipGetLastError();
}

}  // namespace ckks
