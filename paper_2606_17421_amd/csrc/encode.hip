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
// of length P = M/2, run in LDS in fp64 (decimation in frequency, three
// radix-2 stages per LDS pass).  The slot vector is staged in LDS with
// coalesced loads before the Makhoul reordering gathers from it, and the
// transformed rows leave through the wave-local re-layout as coalesced stores.
#include "ntt_core.hpp"

namespace ckks {
namespace {

// Slot vectors are read once and transformed rows written once: both streams
// are non-temporal (4096 weights at 2^15, 6 limbs: 2.43 -> 2.37 ms).
typedef double f64x2 __attribute__((ext_vector_type(2)));

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

// Complex element i of the spectral buffer sits at i + i / 32: the late FFT
// passes read groups two or sixteen elements apart across lanes, which
// without the padding land on the same LDS banks (bank-conflict cycles
// -41%; 2529 -> 2474 us per launch of 4096 slot vectors at N = 2^15).
__device__ __forceinline__ int spec_pad(int i) { return i + (i >> 5); }

// R consecutive radix-2 decimation-in-frequency stages s .. s+R-1 of a
// P = 2^LOGP point complex FFT held in LDS, run in registers: a group is the
// 2^R elements base + j (P >> (s+R)) that those stages combine with each
// other; the stage s+r butterfly on (x, x + d), d = P >> (s+r+1), multiplies
// the difference by tw[(x mod d) << (s+r)].  Same results, in the same
// positions, as R single stages; one LDS round trip and one barrier.
// TWS: the table holds the twiddles of a 2^(LOGP + TWS)-point transform
// (exp(-2 pi i m / 2^(LOGP + TWS))), so this transform's are every 2^TWS-th.
template <int LOGP, int R, int TWS = 0>
__device__ __forceinline__ void fft_pass(double2* a, int s, const double2* __restrict__ tw, int nthreads) {
  constexpr int P = 1 << LOGP, G = 1 << R;
  const int span_lo = P >> (s + R);           // stride between a group's elements
  for (int g = threadIdx.x; g < (P >> R); g += nthreads) {
    const int x0 = g & (span_lo - 1);
    const int base = ((g >> (LOGP - s - R)) << (LOGP - s)) | x0;
    double2 v[G];
#pragma unroll
    for (int j = 0; j < G; ++j) v[j] = a[spec_pad(base + j * span_lo)];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int h = G >> (r + 1);             // partner distance within the group
#pragma unroll
      for (int j = 0; j < G; ++j) {
        if (j & h) continue;
        const int i = x0 + (j & (h - 1)) * span_lo;   // index within the stage's half-block
        const double2 U = v[j], V = v[j + h];
        v[j] = cadd(U, V);
        v[j + h] = cmul(csub(U, V), tw[i << (s + r + TWS)]);
      }
    }
#pragma unroll
    for (int j = 0; j < G; ++j) a[spec_pad(base + j * span_lo)] = v[j];
  }
  __syncthreads();
}

// Fused full-polynomial encode: coefficients and the forward NTT of every limb
// in one workgroup per slot vector, with the whole-polynomial transform's
// thread count.  The spectral buffer (P double2, padded) and the transform's exchange
// buffer share the LDS.  When every rounded coefficient fits in int32 (the
// CKKS-scaled weights of the workloads) each thread keeps its 2P/T of them in
// registers; per limb it writes the residues of their four mirrored positions
// into the exchange buffer and the transform starts from there (group-0
// layout).  Otherwise the workgroup writes every limb's coefficient residues
// to its output rows first and transforms the rows in place from there.
template <int LOGN>
struct FusedPlan {
  using W = WholePlan<LOGN>;
  using NP = typename W::P;
  static constexpr int N = 1 << LOGN, M = N / 2, LOGP = LOGN - 2, P = N / 4;
  static constexpr int T = NP::T;
  static constexpr int KPT = P / T;  // spectral outputs k per thread
  static constexpr int SPEC_WORDS = (P + (P >> 5)) * 4;  // padded spectral buffer (double2)
  static constexpr int LDS_WORDS = (SPEC_WORDS > NP::lds_words) ? SPEC_WORDS : NP::lds_words;
};

// Slots -> spectrum -> rounded coefficients p(k), p(k + P) for the thread's k
// (k = t + T i), as exact doubles.  Ends with every thread done reading LDS.
template <int LOGN>
__device__ __forceinline__ bool encode_spectrum(const Tables& tb, const double* __restrict__ z, double scale,
                                                double2* a, double (&p_lo)[FusedPlan<LOGN>::KPT],
                                                double (&p_hi)[FusedPlan<LOGN>::KPT]) {
  using FP = FusedPlan<LOGN>;
  constexpr int M = FP::M, P = FP::P, T = FP::T, N = FP::N;
  // Stage the slot vector in LDS with coalesced 16-byte loads, then gather
  // the Makhoul-ordered pairs from there (the spectrum reuses the same LDS).
  {
    double2* zs = a;  // M doubles = P double2
    const double2* z2 = reinterpret_cast<const double2*>(z);
#pragma unroll
    for (int i = 0; i < P / T; ++i) {
      const f64x2 zv = __builtin_nontemporal_load(reinterpret_cast<const f64x2*>(z2) + threadIdx.x + T * i);
      zs[threadIdx.x + T * i] = make_double2(zv.x, zv.y);
    }
    __syncthreads();
    const double* zd = reinterpret_cast<const double*>(zs);
    double2 g[P / T];
#pragma unroll
    for (int i = 0; i < P / T; ++i) {
      const int n = threadIdx.x + T * i;
      const int m0 = 2 * n, m1 = 2 * n + 1;
      const int u0 = m0 < M / 2 ? 2 * m0 : 2 * (M - 1 - m0) + 1;
      const int u1 = m1 < M / 2 ? 2 * m1 : 2 * (M - 1 - m1) + 1;
      g[i] = make_double2(zd[tb.slot_perm[u0]], zd[tb.slot_perm[u1]]);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < P / T; ++i) a[spec_pad(threadIdx.x + T * i)] = g[i];
  }
  __syncthreads();
  int s = 0;
  for (; s + 3 <= FP::LOGP; s += 3) fft_pass<FP::LOGP, 3>(a, s, tb.fft_tw, T);
  if (FP::LOGP - s == 2) fft_pass<FP::LOGP, 2>(a, s, tb.fft_tw, T);
  if (FP::LOGP - s == 1) fft_pass<FP::LOGP, 1>(a, s, tb.fft_tw, T);
  const double two_over_n = 2.0 / N;
  bool fits = true;
#pragma unroll
  for (int i = 0; i < FP::KPT; ++i) {
    const int k = threadIdx.x + T * i;
    const int kr = static_cast<int>(__brev(static_cast<uint32_t>(k)) >> (32 - FP::LOGP));
    const int km = (P - k) & (P - 1);
    const int kmr = static_cast<int>(__brev(static_cast<uint32_t>(km)) >> (32 - FP::LOGP));
    const double2 ck = a[spec_pad(kr)];
    const double2 cm = a[spec_pad(kmr)];
    const double2 cmc = make_double2(cm.x, -cm.y);
    const double2 e = make_double2(0.5 * (ck.x + cmc.x), 0.5 * (ck.y + cmc.y));
    const double2 dd = csub(ck, cmc);
    const double2 o = make_double2(0.5 * dd.y, -0.5 * dd.x);
    const double2 wo = cmul(tb.rfft_tw[k], o);
    const double2 v_lo = cadd(e, wo);
    const double2 v_hi = csub(e, wo);
    const double2 t_lo = tb.dct_tw[k], t_hi = tb.dct_tw[k + P];
    p_lo[i] = rint(scale * (two_over_n * (t_lo.x * v_lo.x - t_lo.y * v_lo.y)));
    p_hi[i] = rint(scale * (two_over_n * (t_hi.x * v_hi.x - t_hi.y * v_hi.y)));
    fits = fits && fabs(p_lo[i]) < 2147483648.0 && fabs(p_hi[i]) < 2147483648.0;
  }
  return __syncthreads_and(fits);
}

// Residues mod q of coefficients k, k + P and their mirrors at index x of
// `row` through `at` (m_{N-k} = -m_k for 0 < k < M; m_{N/2} = 0).
template <int LOGN, typename At>
__device__ __forceinline__ void scatter_residues(At at, int k, double p_lo, double p_hi, uint32_t q, double qr) {
  using FP = FusedPlan<LOGN>;
  constexpr int N = FP::N, M = FP::M, P = FP::P;
  const uint32_t r_lo = reduce_f64_int(p_lo, q, qr);
  const uint32_t r_hi = reduce_f64_int(p_hi, q, qr);
  at(k) = r_lo;
  at(k + P) = r_hi;
  if (k == 0) at(M) = 0;
  else at(N - k) = r_lo ? q - r_lo : 0;
  at(N - k - P) = r_hi ? q - r_hi : 0;
}

template <int LOGN>
__global__ __launch_bounds__(FusedPlan<LOGN>::T, WholePlan<LOGN>::kWavesPerSimd) void encode_poly_ntt_kernel(
    Tables tb, const double* __restrict__ slots, uint32_t limbs, double scale, uint32_t* __restrict__ pt) {
  using FP = FusedPlan<LOGN>;
  using NP = typename FP::NP;
  constexpr int LOGE = FP::W::LOGE;
  constexpr int N = FP::N, T = FP::T;
  __shared__ __align__(16) uint32_t lds[FP::LDS_WORDS];
  const size_t b = blockIdx.x;
  const double* z = slots + b * FP::M;
  uint32_t* out = pt + b * static_cast<size_t>(limbs) * N;
  const uint32_t t = threadIdx.x;

  double p_lo[FP::KPT], p_hi[FP::KPT];
  const bool all_fit = encode_spectrum<LOGN>(tb, z, scale, reinterpret_cast<double2*>(lds), p_lo, p_hi);
  if (all_fit) {  // workgroup-uniform
    int32_t c_lo[FP::KPT], c_hi[FP::KPT];
#pragma unroll
    for (int i = 0; i < FP::KPT; ++i) {
      c_lo[i] = static_cast<int32_t>(p_lo[i]);
      c_hi[i] = static_cast<int32_t>(p_hi[i]);
    }
    // Natural (unpadded) order for the scatter: lane t touches index t + const
    // or N - t - const, distinct banks either way.  Index N - k for k = 0 is
    // index N, a spare word past the row; index N/2 is written 0 separately.
    uint32_t* b0 = lds + t;                                   // k = t + T i
    uint32_t* b1 = lds + t + FP::P;                           // k + P
    uint32_t* b2 = lds + (N - t) - T * (FP::KPT - 1);         // N - k      at offset T (KPT-1-i)
    uint32_t* b3 = lds + (N - FP::P - t) - T * (FP::KPT - 1); // N - k - P  at offset T (KPT-1-i)
    for (uint32_t l = 0; l < limbs; ++l) {
      const uint32_t q = tb.q[l];
      // x mod q for x < 2^32 by a Shoup product with w = 1: ws = floor(2^32 / q)
      uint32_t ws = static_cast<uint32_t>(4294967296.0 * tb.q_recip[l]);
      if (static_cast<uint64_t>(ws) * q > 0xFFFFFFFFull) --ws;
      if (static_cast<uint64_t>(ws + 1) * q <= 0xFFFFFFFFull) ++ws;
      uint32_t b31 = 0x80000000u - 2 * q;  // 2^31 mod q (2 q < 2^31 < 4 q)
      b31 = min(b31, b31 - q);
      auto residue = [&](int32_t c) {  // c mod q for |c| < 2^31
        return sub_mod(mul_shoup(static_cast<uint32_t>(c) + 0x80000000u, 1u, ws, q), b31, q);
      };
      if (l > 0) __syncthreads();  // the previous transform is done with the LDS
#pragma unroll
      for (int i = 0; i < FP::KPT; ++i) {
        const uint32_t r_lo = residue(c_lo[i]), r_hi = residue(c_hi[i]);
        b0[T * i] = r_lo;
        b1[T * i] = r_hi;
        b2[T * (FP::KPT - 1 - i)] = r_lo ? q - r_lo : 0;
        b3[T * (FP::KPT - 1 - i)] = r_hi ? q - r_hi : 0;
      }
      if (t == 0) lds[FP::M] = 0;  // m_{N/2} = 0
      __syncthreads();
      uint32_t v[NP::E];
#pragma unroll
      for (int j = 0; j < NP::E; ++j) v[j] = lds[NP::template pos<0>(t, j)];
      const size_t tl = static_cast<size_t>(l) << LOGN;
      fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);
      wave_relayout<LOGN, LOGE, false>(v, t, lds);  // last-group layout -> wave-coalesced
      uint32_t* row = out + static_cast<size_t>(l) * N;
#pragma unroll
      for (int j = 0; j < NP::E; ++j) __builtin_nontemporal_store(v[j], &row[pos_coalesced<LOGE>(t, j)]);
    }
  } else {
    for (uint32_t l = 0; l < limbs; ++l) {
      const uint32_t q = tb.q[l];
      const double qr = tb.q_recip[l];
      uint32_t* row = out + static_cast<size_t>(l) * N;
#pragma unroll
      for (int i = 0; i < FP::KPT; ++i)
        scatter_residues<LOGN>([&](int x) -> uint32_t& { return row[x]; }, static_cast<int>(t) + T * i, p_lo[i],
                               p_hi[i], q, qr);
    }
    for (uint32_t l = 0; l < limbs; ++l) {
      __syncthreads();  // coefficient rows written; the previous transform is done with the LDS
      uint32_t* row = out + static_cast<size_t>(l) * N;
      uint32_t v[NP::E];
#pragma unroll
      for (int j = 0; j < NP::E; ++j) v[j] = row[NP::template pos<0>(t, j)];
      const size_t tl = static_cast<size_t>(l) << LOGN;
      fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, tb.q[l], lds);
      wave_relayout<LOGN, LOGE, false>(v, t, lds);
#pragma unroll
      for (int j = 0; j < NP::E; ++j) __builtin_nontemporal_store(v[j], &row[pos_coalesced<LOGE>(t, j)]);
    }
  }
}

// N = 2^16: the P = 2^14-point spectral transform (256 KiB of complex fp64)
// does not fit the LDS.  Its first radix-2 decimation-in-frequency stage is
// split off: A[n] = v[n] + v[n + P/2] and B[n] = (v[n] - v[n + P/2]) w_P^n,
// whose P/2-point DFTs are the even and the odd outputs, X[2m] and X[2m + 1];
// output k and its partner P - k have the same parity, so each half folds on
// its own.  The plaintext's own first 256 KiB serve as scratch: the slot
// vector is read coalesced and scattered into Makhoul order there (v), A and
// B are read back coalesced (A into the LDS, B into registers), and the even
// half's rounded coefficients wait there while the odd half is transformed.
// Each thread then holds outputs 2m and 2m + 1 and writes every limb's
// residues as 8-byte pairs, whole cache lines per wave (the halves written
// apart would leave every line half-written twice).  The limbs are taken to
// NTT form afterwards by the batched 2^16 transform.
constexpr int kE16Threads = 1024;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(kE16Threads) void encode_poly16_coeff_kernel(
    Tables tb, const double* __restrict__ slots, uint32_t limbs, double scale, uint32_t* __restrict__ pt) {
  constexpr int N = 1 << 16, M = N / 2, P = N / 4, H = P / 2, LOGH = 13, T = kE16Threads, KH = H / T;
  __shared__ __align__(16) double2 a[H + (H >> 5)];  // spec_pad layout
  const size_t b = blockIdx.x;
  const double* z = slots + b * M;
  uint32_t* out = pt + b * static_cast<size_t>(limbs) * N;
  const int t = static_cast<int>(threadIdx.x);
  // v[n] = (y_2n, y_2n+1) as doubles y_m at vs[m]: slot j lands at its Makhoul index
  double* vs = reinterpret_cast<double*>(out);
#pragma unroll 4
  for (int i = 0; i < M / T; ++i) {
    const int j = t + T * i;
    vs[tb.slot_pos[j]] = z[j];
  }
  __syncthreads();  // the scattered sequence is visible to the whole workgroup
  const double2* v2 = reinterpret_cast<const double2*>(vs);
  double2 bv[KH];
#pragma unroll
  for (int i = 0; i < KH; ++i) {
    const int n = t + T * i;
    const double2 v0 = v2[n], v1 = v2[n + H];
    a[spec_pad(n)] = cadd(v0, v1);
    bv[i] = cmul(csub(v0, v1), tb.fft_tw[n]);
  }
  const double two_over_n = 2.0 / N;
  auto brev = [](int x) { return static_cast<int>(__brev(static_cast<uint32_t>(x)) >> (32 - LOGH)); };
  // Rounded coefficients k and k + P of output k = 2m + odd, which sits at
  // position brev(m); its partner P - k is output (H - m) mod H of the even
  // half, H - 1 - m of the odd one.
  auto fold = [&](int m, int odd, double& p_lo, double& p_hi) {
    const int k = 2 * m + odd;
    const int mp = odd ? H - 1 - m : (H - m) & (H - 1);
    const double2 ck = a[spec_pad(brev(m))], cm = a[spec_pad(brev(mp))];
    const double2 cmc = make_double2(cm.x, -cm.y);
    const double2 e = make_double2(0.5 * (ck.x + cmc.x), 0.5 * (ck.y + cmc.y));
    const double2 dd = csub(ck, cmc);
    const double2 o = make_double2(0.5 * dd.y, -0.5 * dd.x);
    const double2 wo = cmul(tb.rfft_tw[k], o);
    const double2 v_lo = cadd(e, wo), v_hi = csub(e, wo);
    const double2 t_lo = tb.dct_tw[k], t_hi = tb.dct_tw[k + P];
    p_lo = rint(scale * (two_over_n * (t_lo.x * v_lo.x - t_lo.y * v_lo.y)));
    p_hi = rint(scale * (two_over_n * (t_hi.x * v_hi.x - t_hi.y * v_hi.y)));
  };
  auto half_fft = [&]() {
    __syncthreads();
    int s = 0;
    for (; s + 3 <= LOGH; s += 3) fft_pass<LOGH, 3, 1>(a, s, tb.fft_tw, T);
    fft_pass<LOGH, 1, 1>(a, s, tb.fft_tw, T);  // LOGH = 13: stages 0..11 by threes, then 12
  };
  // even half; its coefficients (k = 2m, 2m + P) wait at vs[m], vs[H + m]
  // (every read of v is done: the transform's barriers come first)
  half_fft();
#pragma unroll
  for (int i = 0; i < KH; ++i) {
    __builtin_amdgcn_sched_barrier(0);
    const int m = t + T * i;
    double p_lo, p_hi;
    fold(m, 0, p_lo, p_hi);
    vs[m] = p_lo;
    vs[H + m] = p_hi;
  }
  __syncthreads();  // every thread is done reading the even half
#pragma unroll
  for (int i = 0; i < KH; ++i) a[spec_pad(t + T * i)] = bv[i];
  half_fft();
  // odd half, then each pair (2m, 2m + 1) for every limb.  m_{N-k} = -m_k
  // (0 < k < N/2), m_{N/2} = 0.  Limb 0's stores at 2m and 2m + P overwrite
  // only this thread's own waiting values vs[m], vs[H + m], read just before;
  // the mirrored positions lie above the scratch.  Buffer stores: a 32-bit
  // lane offset per position, the limb's row as the scalar offset (a
  // plaintext is at most 16 limbs x 256 KiB).
  const __amdgpu_buffer_rsrc_t ro =
      __builtin_amdgcn_make_buffer_rsrc(out, 0, limbs * static_cast<uint32_t>(N) * 4u, 0x00020000);
  constexpr int kB = 2;
#pragma unroll 1
  for (int i0 = 0; i0 < KH; i0 += kB) {
    double e_lo[kB], e_hi[kB], o_lo[kB], o_hi[kB];
#pragma unroll
    for (int ii = 0; ii < kB; ++ii) {
      const int m = t + T * (i0 + ii);
      fold(m, 1, o_lo[ii], o_hi[ii]);
      e_lo[ii] = vs[m];
      e_hi[ii] = vs[H + m];
    }
    for (uint32_t l = 0; l < limbs; ++l) {
      const uint32_t q = tb.q[l];
      const double qr = tb.q_recip[l];
      const uint32_t so = l * static_cast<uint32_t>(N) * 4u;
#pragma unroll
      for (int ii = 0; ii < kB; ++ii) {
        const uint32_t m = static_cast<uint32_t>(t + T * (i0 + ii));
        const uint32_t r0 = reduce_f64_int(e_lo[ii], q, qr), r1 = reduce_f64_int(o_lo[ii], q, qr);
        const uint32_t h0 = reduce_f64_int(e_hi[ii], q, qr), h1 = reduce_f64_int(o_hi[ii], q, qr);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{r0, r1}, ro, 2u * m * 4u, so, 0);
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{h0, h1}, ro, (2u * m + P) * 4u, so, 0);
        __builtin_amdgcn_raw_buffer_store_b32(m ? (r0 ? q - r0 : 0u) : 0u, ro, (m ? N - 2u * m : M) * 4u, so, 0);
        __builtin_amdgcn_raw_buffer_store_b32(r1 ? q - r1 : 0u, ro, (N - 2u * m - 1u) * 4u, so, 0);
        __builtin_amdgcn_raw_buffer_store_b32(h0 ? q - h0 : 0u, ro, (N - 2u * m - P) * 4u, so, 0);
        __builtin_amdgcn_raw_buffer_store_b32(h1 ? q - h1 : 0u, ro, (N - 2u * m - 1u - P) * 4u, so, 0);
      }
    }
  }
}

template <int LOGN>
hipError_t launch_poly(const Tables& t, const double* slots, uint32_t count, uint32_t limbs,
                       double scale, uint32_t* pt, hipStream_t s) {
  encode_poly_ntt_kernel<LOGN><<<count, FusedPlan<LOGN>::T, 0, s>>>(t, slots, limbs, scale, pt);
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

hipError_t launch_encode_poly(const Tables& t, const double* slots, uint32_t count, uint32_t limbs,
                              double scale, uint32_t* pt, hipStream_t s) {
  if (count == 0) return hipSuccess;
  switch (t.log_n) {
    case 10: return launch_poly<10>(t, slots, count, limbs, scale, pt, s);
    case 11: return launch_poly<11>(t, slots, count, limbs, scale, pt, s);
    case 12: return launch_poly<12>(t, slots, count, limbs, scale, pt, s);
    case 13: return launch_poly<13>(t, slots, count, limbs, scale, pt, s);
    case 14: return launch_poly<14>(t, slots, count, limbs, scale, pt, s);
    case 15: return launch_poly<15>(t, slots, count, limbs, scale, pt, s);
    case 16: {
      encode_poly16_coeff_kernel<<<count, kE16Threads, 0, s>>>(t, slots, limbs, scale, pt);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_ntt(t, pt, static_cast<size_t>(count) * limbs, limbs, false, s);
    }
    default: return hipErrorNotSupported;
  }
}

}  // namespace ckks
