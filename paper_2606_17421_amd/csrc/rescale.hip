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
// minimum: read limbs rows, write limbs - 1 rows.  When the polynomials are
// fewer than half the CUs (the key-switch ModDown of a few rotations, a
// decode-size layer), each workgroup instead takes one output limb of one
// polynomial (kSplit): the inverse transform is repeated per limb, but the
// chain per workgroup is two transforms instead of limbs, on limbs - 1 times
// the workgroups, and with the latency plan (more lanes per transform).  Rows
// are read and written in the wave-coalesced layout.
// N = 2^16: three passes through a workspace (see below).
#include "ntt_core.hpp"

namespace ckks {
namespace {

template <int LOGN, bool kSplit>
__global__ __launch_bounds__((WholePlan<LOGN, kSplit>::P::T), (WholePlan<LOGN, kSplit>::kWavesPerSimd)) void rescale_kernel(
    Tables tb, const uint32_t* __restrict__ in, uint32_t* __restrict__ out, uint32_t limbs) {
  using P = typename WholePlan<LOGN, kSplit>::P;
  constexpr int LOGE = WholePlan<LOGN, kSplit>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const size_t poly = blockIdx.x;  // ciphertext * 2 + component
  const uint32_t t = threadIdx.x;
  const uint32_t* src = in + poly * limbs * N;
  uint32_t* dst = out + poly * (limbs - 1) * N;
  const uint32_t top = limbs - 1;
  const uint32_t qt = tb.q[top];

  // The rows are read and written in the wave-coalesced layout (re-laid out
  // through each wave's LDS region), non-temporally when one workgroup takes a
  // whole polynomial (each row is touched once).  The split route re-reads the
  // top row in every limb's workgroup and keeps all its accesses cached
  // (non-temporal there: 12.3 -> 13.3-13.8 us for 32 ciphertexts at 2^13, 4
  // limbs).  At 2^15 the coalesced path spills a few registers and still wins:
  // 3.66-3.70 -> 3.33 ms for 3072 ciphertexts of 6 limbs, 147.5 -> 129.4 us
  // for 64 (split), against loads and stores in the last group's layout, where
  // a wave's access to one element index spans 64 cache lines.
  uint32_t v[P::E];
  const uint32_t* stop = src + static_cast<size_t>(top) * N + pos_coalesced<LOGE>(t, 0);
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = kSplit ? stop[j << 6] : __builtin_nontemporal_load(&stop[j << 6]);
  wave_relayout<LOGN, LOGE, true>(v, t, lds);
  const size_t ttop = static_cast<size_t>(top) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + ttop, tb.inv_shoup + ttop, qt, lds);
  const uint32_t ni = tb.ninv[top], nis = tb.ninv_shoup[top];
  int32_t r[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t x = mul_shoup(v[j], ni, nis, qt);
    r[j] = x > (qt >> 1) ? static_cast<int32_t>(x) - static_cast<int32_t>(qt) : static_cast<int32_t>(x);
  }

  const uint32_t l_begin = kSplit ? blockIdx.y : 0, l_end = kSplit ? blockIdx.y + 1 : top;
  for (uint32_t l = l_begin; l < l_end; ++l) {
    const uint32_t q = tb.q[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = static_cast<uint32_t>(r[j] < 0 ? r[j] + static_cast<int32_t>(q) : r[j]);
    const size_t tl = static_cast<size_t>(l) << LOGN;
    fwd_block<LOGN, LOGN, LOGE, 0, false>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);  // [0, 4q)
    const uint32_t qi = tb.qinv[top * tb.L + l], qis = tb.qinv_shoup[top * tb.L + l];
    wave_relayout<LOGN, LOGE, false>(v, t, lds);
    const uint32_t* sl = src + static_cast<size_t>(l) * N + pos_coalesced<LOGE>(t, 0);
    uint32_t* dl = dst + static_cast<size_t>(l) * N + pos_coalesced<LOGE>(t, 0);
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      if constexpr (kSplit) dl[j << 6] = sub_lazy_mul_shoup(sl[j << 6], v[j], qi, qis, q);
      else __builtin_nontemporal_store(sub_lazy_mul_shoup(__builtin_nontemporal_load(&sl[j << 6]), v[j], qi, qis, q),
                                       &dl[j << 6]);
    }
  }
}

// Two rescales in one launch: divide by the last prime q_t (t = limbs - 1) and
// then by q_u (u = t - 1), dropping both.  With
//     r1 = centred INTT_t(c_t),
//     r2 = centred ((INTT_u(c_u) - r1) q_t^-1 mod q_u)   (the coefficients of
//          the first rescale's limb u),
// the second rescale's output limb l < u is
//     ((c_l - NTT_l(r1)) q_t^-1 - NTT_l(r2)) q_u^-1
//   = (c_l q_t^-1 - NTT_l(r1 q_t^-1 + r2)) q_u^-1     mod q_l,
// the same residues as the two rescales in turn.  For launches of few
// polynomials (the key-switched sum of the BSGS giant steps: its division by
// the special prime, then the product's own rescale), in two launches whose
// chains are one transform each:
//   rescale2_inv_kernel, one workgroup per polynomial and row (t or u): the
//     inverse transform of that row, r1 (centred) or INTT_u(c_u) stored to the
//     workspace in the plan's register order (element e of thread t at
//     e * T + t, coalesced both ways, read back by the same plan's threads);
//   rescale2_fwd_kernel, one workgroup per polynomial and output limb l: r2
//     from the two stored rows, then NTT_l(r1 q_t^-1 + r2) and the combine.
// (One launch doing all three transforms per workgroup took 20.5 us for one
// ciphertext at 2^13; a loop over the limbs would also hold r1, r2 and the row
// in registers at once and spill.)
template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN, true>::P::T), (WholePlan<LOGN, true>::kWavesPerSimd)) void
rescale2_inv_kernel(Tables tb, const uint32_t* __restrict__ in, uint32_t limbs, uint32_t* __restrict__ ws) {
  using P = typename WholePlan<LOGN, true>::P;
  constexpr int LOGE = WholePlan<LOGN, true>::LOGE;
  constexpr int N = P::B;
  constexpr bool kCoalesce = LOGN <= 14;
  __shared__ uint32_t lds[P::lds_words];
  const size_t poly = blockIdx.x;                     // ciphertext * 2 + component
  const uint32_t which = blockIdx.y;                  // 0: row t (r1), 1: row u
  const uint32_t m = limbs - 1 - which;
  const uint32_t t = threadIdx.x;
  const uint32_t* src = in + (poly * limbs + m) * N;
  uint32_t v[P::E];
  if constexpr (kCoalesce) {
    const uint32_t* sm = src + pos_coalesced<LOGE>(t, 0);
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = sm[j << 6];
    wave_relayout<LOGN, LOGE, true>(v, t, lds);
  } else {
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = src[P::template pos<P::NG - 1>(t, j)];
  }
  const size_t tm = static_cast<size_t>(m) << LOGN;
  const uint32_t qm = tb.q[m];
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + tm, tb.inv_shoup + tm, qm, lds);
  const uint32_t ni = tb.ninv[m], nis = tb.ninv_shoup[m];
  uint32_t* dst = ws + (poly * 2 + which) * N + t;
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t x = mul_shoup(v[j], ni, nis, qm);
    // row t: the centred value as a two's-complement word; row u: the residue
    dst[j * P::T] = which == 0 && x > (qm >> 1) ? x - qm : x;
  }
}

template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN, true>::P::T), (WholePlan<LOGN, true>::kWavesPerSimd)) void
rescale2_fwd_kernel(Tables tb, const uint32_t* __restrict__ in, const uint32_t* __restrict__ ws, uint32_t limbs,
                    uint32_t* __restrict__ out) {
  using P = typename WholePlan<LOGN, true>::P;
  constexpr int LOGE = WholePlan<LOGN, true>::LOGE;
  constexpr int N = P::B;
  constexpr bool kCoalesce = LOGN <= 14;
  __shared__ uint32_t lds[P::lds_words];
  const size_t poly = blockIdx.x;
  const uint32_t t = threadIdx.x;
  const uint32_t* src = in + poly * limbs * N;
  uint32_t* dst = out + poly * (limbs - 2) * N;
  const uint32_t top = limbs - 1, mid = limbs - 2;
  auto lift = [](int32_t r, uint32_t q) {   // |r| < 2^29 < q
    return static_cast<uint32_t>(r < 0 ? r + static_cast<int32_t>(q) : r);
  };
  const uint32_t* w1 = ws + (poly * 2) * N + t;
  const uint32_t* w2 = w1 + N;
  int32_t r1[P::E], r2[P::E];
  {
    const uint32_t qu = tb.q[mid];
    const uint32_t ti = tb.qinv[top * tb.L + mid], tis = tb.qinv_shoup[top * tb.L + mid];
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      r1[j] = static_cast<int32_t>(w1[j * P::T]);
      const uint32_t x = mul_shoup(sub_mod(w2[j * P::T], lift(r1[j], qu), qu), ti, tis, qu);
      r2[j] = x > (qu >> 1) ? static_cast<int32_t>(x) - static_cast<int32_t>(qu) : static_cast<int32_t>(x);
    }
  }
  const uint32_t l = blockIdx.y, q = tb.q[l];
  const uint32_t ti = tb.qinv[top * tb.L + l], tis = tb.qinv_shoup[top * tb.L + l];
  const uint32_t ui = tb.qinv[mid * tb.L + l], uis = tb.qinv_shoup[mid * tb.L + l];
  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = add_mod(mul_shoup(lift(r1[j], q), ti, tis, q), lift(r2[j], q), q);
  const size_t tl = static_cast<size_t>(l) << LOGN;
  fwd_block<LOGN, LOGN, LOGE, 0, false>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);  // [0, 4q)
  if constexpr (kCoalesce) {
    wave_relayout<LOGN, LOGE, false>(v, t, lds);
    const uint32_t* sl = src + static_cast<size_t>(l) * N + pos_coalesced<LOGE>(t, 0);
    uint32_t* dl = dst + static_cast<size_t>(l) * N + pos_coalesced<LOGE>(t, 0);
#pragma unroll
    for (int j = 0; j < P::E; ++j) dl[j << 6] = sub_lazy_mul_shoup(mul_shoup(sl[j << 6], ti, tis, q), v[j], ui, uis, q);
  } else {
#pragma unroll
    for (int j = 0; j < P::E; ++j) {
      const size_t x = static_cast<size_t>(l) * N + P::template pos<P::NG - 1>(t, j);
      dst[x] = sub_lazy_mul_shoup(mul_shoup(src[x], ti, tis, q), v[j], ui, uis, q);
    }
  }
}

// ---- N = 2^16: three passes over a chunk of polynomials --------------------
// A row of 2^16 residues (256 KiB) exceeds the LDS, so each transform splits
// into a column pass over the top 6 index bits (64 residues per thread,
// column c = low 10 bits) and a block pass over 1024-point blocks, as in the
// standalone NTT.  Per chunk of polynomials:
//   1. top_blocks: inverse block stages of limb top, ct_in -> A;
//   2. cols: inverse column stages of A, N^-1, centring, then for every
//      lower limb l the forward column stages of r mod q_l -> B[l]
//      (the centred coefficients stay in registers across the limbs);
//   3. blocks_combine: forward block stages of B[l], then
//      (c_l - .) q_top^-1 mod q_l -> ct_out.
// HBM traffic per polynomial: 2 + 2 (top) + 4 (per lower limb) row transfers
// instead of the minimum 1 + 2 per lower limb.  The streams touched once per
// chunk (the top row of ct_in, B written and read back, c_l, ct_out) are
// loaded and stored non-temporally, the intermediate top row A normally:
// 21.6-21.7 -> 20.6 ms for 6144 ciphertexts of 8 limbs (non-temporal loads
// alone, or stores alone, gained nothing).
constexpr int kColLogE = 6;
constexpr int kColThreads = 256;
constexpr int kBlkLogB = 10;
constexpr int kBlkLogE = 4;
constexpr int kBlkThreads = 1 << (kBlkLogB - kBlkLogE);
constexpr int kBlocksPerRow = 1 << (16 - kBlkLogB);
constexpr uint32_t kChunkPolys16 = 1024;  // polynomials per pass: workspace (1 + top) x 256 MiB; 2048
                                          // ciphertexts x 8 limbs: 7.77 ms at 256, 7.13 ms at 1024


__global__ __launch_bounds__(kBlkThreads) void rescale16_top_blocks_kernel(Tables tb, const uint32_t* __restrict__ in,
                                                                          uint32_t* __restrict__ A, uint32_t limbs,
                                                                          size_t p0) {
  using P = Plan<kBlkLogB, kBlkLogE>;
  __shared__ uint32_t lds[P::lds_words];
  const size_t r = blockIdx.x / kBlocksPerRow;
  const uint32_t blk = blockIdx.x % kBlocksPerRow;
  const uint32_t t = threadIdx.x;
  const uint32_t top = limbs - 1;
  const uint32_t* a = in + ((p0 + r) * limbs + top) * 65536 + (static_cast<size_t>(blk) << kBlkLogB);
  uint32_t* o = A + (r << 16) + (static_cast<size_t>(blk) << kBlkLogB);
  const size_t toff = static_cast<size_t>(top) << 16;
  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&a[t + 64 * j]);  // coalesced
  wave_relayout<kBlkLogB, kBlkLogE, true>(v, t, lds);
  inv_block<16, kBlkLogB, kBlkLogE>(v, t, blk, tb.inv + toff, tb.inv_shoup + toff, tb.q[top], lds);
#pragma unroll
  for (int j = 0; j < P::E; ++j) o[P::template pos<0>(t, j)] = v[j];
}

// Two workgroups per CU (two waves per SIMD, at most 256 registers each).
__global__ __launch_bounds__(kColThreads, 2) void rescale16_cols_kernel(Tables tb, const uint32_t* __restrict__ A,
                                                                    uint32_t* __restrict__ B, uint32_t limbs,
                                                                    size_t chunk_words) {
  using P = Plan<16, kColLogE>;
  constexpr int kColsPerRow = 1 << (16 - kColLogE);
  const size_t r = blockIdx.x / (kColsPerRow / kColThreads);
  const uint32_t c = (blockIdx.x % (kColsPerRow / kColThreads)) * kColThreads + threadIdx.x;
  const uint32_t top = limbs - 1;
  const uint32_t qt = tb.q[top];
  const uint32_t* a = A + (r << 16) + c;
  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = a[P::template pos<0>(0, j)];
  const size_t ttop = static_cast<size_t>(top) << 16;
  inv_group<16, 16, kColLogE, 0>(v, c, 0, tb.inv + ttop, tb.inv_shoup + ttop, qt);  // [0, 2q)
  const uint32_t ni = tb.ninv[top], nis = tb.ninv_shoup[top];
  int32_t rc[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t x = mul_shoup(v[j], ni, nis, qt);
    rc[j] = x > (qt >> 1) ? static_cast<int32_t>(x) - static_cast<int32_t>(qt) : static_cast<int32_t>(x);
  }
  for (uint32_t l = 0; l < top; ++l) {
    const uint32_t q = tb.q[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = static_cast<uint32_t>(rc[j] < 0 ? rc[j] + static_cast<int32_t>(q) : rc[j]);
    const size_t tl = static_cast<size_t>(l) << 16;
    fwd_group<16, 16, kColLogE, 0>(v, c, 0, tb.fwd + tl, tb.fwd_shoup + tl, q);  // [0, 4q)
    uint32_t* o = B + l * chunk_words + (r << 16) + c;
#pragma unroll
    for (int j = 0; j < P::E; ++j) __builtin_nontemporal_store(v[j], &o[P::template pos<0>(0, j)]);
  }
}

__global__ __launch_bounds__(kBlkThreads) void rescale16_blocks_combine_kernel(
    Tables tb, const uint32_t* __restrict__ in, const uint32_t* __restrict__ B, uint32_t* __restrict__ out,
    uint32_t limbs, size_t p0, size_t np, size_t chunk_words) {
  using P = Plan<kBlkLogB, kBlkLogE>;
  __shared__ uint32_t lds[P::lds_words];
  const size_t per_limb = np * kBlocksPerRow;
  const uint32_t l = static_cast<uint32_t>(blockIdx.x / per_limb);
  const size_t rem = blockIdx.x % per_limb;
  const size_t r = rem / kBlocksPerRow;
  const uint32_t blk = static_cast<uint32_t>(rem % kBlocksPerRow);
  const uint32_t t = threadIdx.x;
  const uint32_t top = limbs - 1;
  const uint32_t q = tb.q[l];
  const size_t boff = static_cast<size_t>(blk) << kBlkLogB;
  const uint32_t* b = B + l * chunk_words + (r << 16) + boff;
  uint32_t v[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = __builtin_nontemporal_load(&b[P::template pos<0>(t, j)]);
  const size_t tl = static_cast<size_t>(l) << 16;
  fwd_block<16, kBlkLogB, kBlkLogE, 0, false>(v, t, blk, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);  // [0, 4q)
  const uint32_t qi = tb.qinv[top * tb.L + l], qis = tb.qinv_shoup[top * tb.L + l];
  const uint32_t* c = in + ((p0 + r) * limbs + l) * 65536 + boff;
  uint32_t* o = out + ((p0 + r) * (limbs - 1) + l) * 65536 + boff;
  wave_relayout<kBlkLogB, kBlkLogE, false>(v, t, lds);
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t x = t + 64 * j;  // coalesced
    __builtin_nontemporal_store(sub_lazy_mul_shoup(__builtin_nontemporal_load(&c[x]), v[j], qi, qis, q), &o[x]);
  }
}

size_t chunk16(size_t polys) { return polys < kChunkPolys16 ? polys : kChunkPolys16; }

hipError_t rescale16(const Tables& t, const uint32_t* in, uint32_t* out, uint32_t count,
                     uint32_t limbs, void* workspace, hipStream_t s) {
  const size_t polys_total = static_cast<size_t>(count) * 2;
  const size_t chunk = chunk16(polys_total);
  const size_t chunk_words = chunk << 16;
  uint32_t* A = static_cast<uint32_t*>(workspace);  // [chunk][2^16]
  uint32_t* B = A + chunk_words;                    // [limbs - 1][chunk][2^16]
  const uint32_t top = limbs - 1;
  for (size_t p0 = 0; p0 < polys_total; p0 += chunk) {
    const size_t np = polys_total - p0 < chunk ? polys_total - p0 : chunk;
    rescale16_top_blocks_kernel<<<static_cast<uint32_t>(np * kBlocksPerRow), kBlkThreads, 0, s>>>(t, in, A, limbs, p0);
    rescale16_cols_kernel<<<static_cast<uint32_t>(np * ((1 << (16 - kColLogE)) / kColThreads)), kColThreads, 0, s>>>(
        t, A, B, limbs, chunk_words);
    rescale16_blocks_combine_kernel<<<static_cast<uint32_t>(top * np * kBlocksPerRow), kBlkThreads, 0, s>>>(
        t, in, B, out, limbs, p0, np, chunk_words);
  }
  return hipGetLastError();
}

template <int LOGN>
hipError_t launch_rescale_whole(const Tables& t, const uint32_t* in, uint32_t* out, uint32_t count,
                                uint32_t limbs, hipStream_t s) {
  if (4 * static_cast<size_t>(count) <= t.num_cus && limbs > 2)
    rescale_kernel<LOGN, true><<<dim3(2 * count, limbs - 1), WholePlan<LOGN, true>::P::T, 0, s>>>(t, in, out, limbs);
  else
    rescale_kernel<LOGN, false><<<dim3(2 * count), WholePlan<LOGN>::P::T, 0, s>>>(t, in, out, limbs);
  return hipGetLastError();
}

}  // namespace

size_t rescale_workspace_bytes(const Tables& t, uint32_t count, uint32_t limbs) {
  if (t.log_n < 16) return 0;
  return static_cast<size_t>(limbs) * (chunk16(static_cast<size_t>(count) * 2) << 16) * sizeof(uint32_t);
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

// Two rescales in turn (limbs -> limbs - 2): rescale2_inv_kernel then
// rescale2_fwd_kernel for fewer than num_cus / 4 ciphertexts up to 2^15 (their
// 4 count N words of rows in `mid`), else the two rescales with the
// intermediate [count][2][limbs-1][N] in `mid`.  `mid` is caller-provided.
hipError_t launch_rescale2(const Tables& t, const uint32_t* ct_in, uint32_t* mid, uint32_t* ct_out, uint32_t count,
                           uint32_t limbs, void* workspace, hipStream_t s) {
  if (count == 0) return hipSuccess;
  if (limbs < 3) return hipErrorInvalidValue;
  if (t.log_n <= 15 && 4 * static_cast<size_t>(count) <= t.num_cus) {
    const dim3 gi(2 * count, 2), gf(2 * count, limbs - 2);
    switch (t.log_n) {
#define CKKS_R2(LN)                                                                                     \
  case LN:                                                                                              \
    rescale2_inv_kernel<LN><<<gi, WholePlan<LN, true>::P::T, 0, s>>>(t, ct_in, limbs, mid);             \
    rescale2_fwd_kernel<LN><<<gf, WholePlan<LN, true>::P::T, 0, s>>>(t, ct_in, mid, limbs, ct_out);     \
    break;
      CKKS_R2(10)
      CKKS_R2(11)
      CKKS_R2(12)
      CKKS_R2(13)
      CKKS_R2(14)
      default: CKKS_R2(15)
#undef CKKS_R2
    }
    return hipGetLastError();
  }
  const hipError_t err = launch_rescale(t, ct_in, mid, count, limbs, workspace, s);
  return err != hipSuccess ? err : launch_rescale(t, mid, ct_out, count, limbs - 1, workspace, s);
}

}  // namespace ckks
