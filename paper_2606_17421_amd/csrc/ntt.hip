// Batched negacyclic NTT / INTT kernels (gfx950).
//
// N <= 2^15: one workgroup per polynomial row; the row is read from HBM once
// in group-0 layout (coalesced), transformed through register groups and
// padded-LDS exchanges (at most 132 KiB of LDS), and written once.  Both
// accesses cover whole cache lines per wave and are non-temporal (36,864 rows
// of 2^15: forward 2.97-3.02 -> 2.88 ms, inverse 3.57 -> 3.43 ms).
// N = 2^16 (256 KiB per row, above the 160 KiB LDS): two passes over HBM,
// a column pass over the top 6 index bits (64 residues per thread, twiddles
// uniform across the workgroup) and a block pass over 1024-point blocks, also
// with non-temporal whole-line accesses (16,384 rows: forward 3.39-3.50 ->
// 3.34 ms, inverse 3.60 -> 3.26 ms).
//
// Logical row r uses limb r % limbs and lives at physical row
// (r / limbs) * gstride + r % limbs: gstride = limbs for packed
// [count][limbs][N] rows, 2 * limbs for one component of [count][2][limbs][N]
// ciphertexts.
#include "ntt_core.hpp"

namespace ckks {
namespace {

__device__ __forceinline__ size_t phys_row(size_t r, uint32_t limbs, uint32_t gstride) {
  return (r / limbs) * gstride + r % limbs;
}

template <int LOGN, bool INV, bool LAT>
__global__ __launch_bounds__((WholePlan<LOGN, LAT>::P::T), (WholePlan<LOGN, LAT>::kWavesPerSimd)) void ntt_whole_kernel(
    Tables tb, uint32_t* rows, uint32_t limbs, uint32_t gstride) {
  using P = typename WholePlan<LOGN, LAT>::P;
  constexpr int LOGE = WholePlan<LOGN, LAT>::LOGE;
  __shared__ uint32_t lds[P::lds_words];
  const size_t r = blockIdx.x;
  const uint32_t l = static_cast<uint32_t>(r % limbs);
  const uint32_t t = threadIdx.x;
  uint32_t* a = rows + phys_row(r, limbs, gstride) * P::B;
  const uint32_t q = tb.q[l];
  const size_t toff = static_cast<size_t>(l) << LOGN;
  uint32_t v[P::E];
  if constexpr (!INV) {
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&a[P::template pos<0>(t, j)]);
    fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + toff, tb.fwd_shoup + toff, q, lds);
    wave_relayout<LOGN, LOGE, false>(v, t, lds);
    uint32_t* ac = a + pos_coalesced<LOGE>(t, 0);
#pragma unroll
    for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(v[j], &ac[j << 6]);
  } else {
    const uint32_t* ac = a + pos_coalesced<LOGE>(t, 0);
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&ac[j << 6]);
    wave_relayout<LOGN, LOGE, true>(v, t, lds);
    inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + toff, tb.inv_shoup + toff, q, lds);
    const uint32_t ni = tb.ninv[l], nis = tb.ninv_shoup[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(mul_shoup(v[j], ni, nis, q), &a[P::template pos<0>(t, j)]);
  }
}

// N = 2^16, top 6 bits: thread owns column c (low 10 bits) of one row.
constexpr int kColLogE = 6;
constexpr int kColThreads = 256;

template <bool INV>
// Two workgroups per CU (two waves per SIMD, at most 256 registers each).
__global__ __launch_bounds__(kColThreads, 2) void ntt16_cols_kernel(Tables tb, uint32_t* rows,
                                                                 uint32_t limbs, uint32_t gstride) {
  using P = Plan<16, kColLogE>;
  constexpr int kColsPerRow = 1 << (16 - kColLogE);
  const size_t r = blockIdx.x / (kColsPerRow / kColThreads);
  const uint32_t c = (blockIdx.x % (kColsPerRow / kColThreads)) * kColThreads + threadIdx.x;
  const uint32_t l = static_cast<uint32_t>(r % limbs);
  uint32_t* a = rows + (phys_row(r, limbs, gstride) << 16);
  const uint32_t q = tb.q[l];
  const size_t toff = static_cast<size_t>(l) << 16;
  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&a[P::template pos<0>(c, j)]);
  if constexpr (!INV) {
    fwd_group<16, 16, kColLogE, 0>(v, c, 0, tb.fwd + toff, tb.fwd_shoup + toff, q);
  } else {
    inv_group<16, 16, kColLogE, 0>(v, c, 0, tb.inv + toff, tb.inv_shoup + toff, q);
    const uint32_t ni = tb.ninv[l], nis = tb.ninv_shoup[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = mul_shoup(v[j], ni, nis, q);
  }
#pragma unroll
  for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(v[j], &a[P::template pos<0>(c, j)]);
}

// N = 2^16, low 10 bits: one 64-thread workgroup per 1024-point block.
constexpr int kBlkLogB = 10;
constexpr int kBlkLogE = 4;

template <bool INV>
__global__ __launch_bounds__(1 << (kBlkLogB - kBlkLogE)) void ntt16_blocks_kernel(Tables tb,
                                                                                 uint32_t* rows,
                                                                                 uint32_t limbs,
                                                                                 uint32_t gstride) {
  using P = Plan<kBlkLogB, kBlkLogE>;
  __shared__ uint32_t lds[P::lds_words];
  constexpr int kBlocksPerRow = 1 << (16 - kBlkLogB);
  const size_t r = blockIdx.x / kBlocksPerRow;
  const uint32_t blk = blockIdx.x % kBlocksPerRow;
  const uint32_t l = static_cast<uint32_t>(r % limbs);
  const uint32_t t = threadIdx.x;
  uint32_t* a = rows + (phys_row(r, limbs, gstride) << 16) + (static_cast<size_t>(blk) << kBlkLogB);
  const uint32_t q = tb.q[l];
  const size_t toff = static_cast<size_t>(l) << 16;
  uint32_t v[P::E];
  if constexpr (!INV) {
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&a[P::template pos<0>(t, j)]);
    fwd_block<16, kBlkLogB, kBlkLogE>(v, t, blk, tb.fwd + toff, tb.fwd_shoup + toff, q, lds);
    wave_relayout<kBlkLogB, kBlkLogE, false>(v, t, lds);
#pragma unroll
    for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(v[j], &a[t + 64 * j]);  // coalesced (one wave per block)
  } else {
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&a[t + 64 * j]);
    wave_relayout<kBlkLogB, kBlkLogE, true>(v, t, lds);
    inv_block<16, kBlkLogB, kBlkLogE>(v, t, blk, tb.inv + toff, tb.inv_shoup + toff, q, lds);
#pragma unroll
    for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(v[j], &a[P::template pos<0>(t, j)]);
  }
}

template <int LOGN, bool LAT>
hipError_t launch_whole_plan(const Tables& t, uint32_t* rows, size_t count, uint32_t limbs, bool inv,
                             hipStream_t s, uint32_t gs) {
  using P = typename WholePlan<LOGN, LAT>::P;
  if (inv)
    ntt_whole_kernel<LOGN, true, LAT><<<dim3(static_cast<uint32_t>(count)), P::T, 0, s>>>(t, rows, limbs, gs);
  else
    ntt_whole_kernel<LOGN, false, LAT><<<dim3(static_cast<uint32_t>(count)), P::T, 0, s>>>(t, rows, limbs, gs);
  return hipGetLastError();
}

// Fewer rows than CUs: the latency form (each row has a CU to itself).
template <int LOGN>
hipError_t launch_whole(const Tables& t, uint32_t* rows, size_t count, uint32_t limbs, bool inv,
                        hipStream_t s, uint32_t gs) {
  if ((LOGN == 13 || LOGN == 14) && count < t.num_cus) return launch_whole_plan<LOGN, true>(t, rows, count, limbs, inv, s, gs);
  return launch_whole_plan<LOGN, false>(t, rows, count, limbs, inv, s, gs);
}

hipError_t launch_ntt16(const Tables& t, uint32_t* rows, size_t count, uint32_t limbs, bool inv,
                        hipStream_t s, uint32_t gs) {
  const uint32_t col_grid = static_cast<uint32_t>(count * ((1 << (16 - kColLogE)) / kColThreads));
  const uint32_t blk_grid = static_cast<uint32_t>(count * (1 << (16 - kBlkLogB)));
  constexpr int blk_threads = 1 << (kBlkLogB - kBlkLogE);
  if (!inv) {
    ntt16_cols_kernel<false><<<col_grid, kColThreads, 0, s>>>(t, rows, limbs, gs);
    ntt16_blocks_kernel<false><<<blk_grid, blk_threads, 0, s>>>(t, rows, limbs, gs);
  } else {
    ntt16_blocks_kernel<true><<<blk_grid, blk_threads, 0, s>>>(t, rows, limbs, gs);
    ntt16_cols_kernel<true><<<col_grid, kColThreads, 0, s>>>(t, rows, limbs, gs);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_ntt(const Tables& t, uint32_t* rows, size_t count_rows, uint32_t limbs,
                      bool inverse, hipStream_t s, uint32_t gstride) {
  if (count_rows == 0) return hipSuccess;
  const uint32_t gs = gstride ? gstride : limbs;
  switch (t.log_n) {
    case 10: return launch_whole<10>(t, rows, count_rows, limbs, inverse, s, gs);
    case 11: return launch_whole<11>(t, rows, count_rows, limbs, inverse, s, gs);
    case 12: return launch_whole<12>(t, rows, count_rows, limbs, inverse, s, gs);
    case 13: return launch_whole<13>(t, rows, count_rows, limbs, inverse, s, gs);
    case 14: return launch_whole<14>(t, rows, count_rows, limbs, inverse, s, gs);
    case 15: return launch_whole<15>(t, rows, count_rows, limbs, inverse, s, gs);
    case 16: return launch_ntt16(t, rows, count_rows, limbs, inverse, s, gs);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ckks
