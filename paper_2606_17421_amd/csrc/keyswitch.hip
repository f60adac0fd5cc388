// Galois automorphisms, hybrid key switching and slot rotations, and the
// baby-step / giant-step (BSGS) diagonal matrix-vector product on top of them
// (gfx950).  The paper's accelerator linear call is a BSGS product over
// pre-encoded weight diagonals (sections 4.1 and 4.2), with rotations done by
// automorphisms and key switching under one special prime (section 4.2).
//
// Conventions.  The context's last prime P is the special prime; ciphertexts
// that are rotated carry the other t.L - 1 limbs (L below).  NTT value i is
// the evaluation at psi^(2 brv(i) + 1), so sigma_g (a(X) -> a(X^g)) permutes
// NTT values: out[i] = in[brv(u g + (g - 1) / 2 mod N)] with u = brv(i).
// Rotation by r slots uses g = 5^r mod 2N.
//
// Key switching (hybrid, one digit per limb): the digits of c1 are the centred
// coefficient vectors of its limbs, lifted to every prime of q_0..q_{L-1}, P
// (ModUp: an INTT per digit, then a lifted NTT per digit and prime, in one,
// two or four launches by size).  A rotation then needs only its key and an
// index permutation: sigma_g commutes with the digit decomposition exactly
// (the centred lift is odd-symmetric for odd q), so the inner product reads
// the unrotated digits through the permutation.  All rotations of one
// ciphertext share one ModUp (hoisting).  The division by P (ModDown) is the
// rescale that drops the last prime, fused with the rotation's combine up to
// 2^14; the BSGS giant steps sum their inner products first and divide once.
#include "ntt_core.hpp"

namespace ckks {
namespace {

constexpr int kThreads = 256;

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int32_t v4s __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4u ld4(const uint32_t* p) { return *reinterpret_cast<const v4u*>(p); }
__device__ __forceinline__ v4s ld4(const int32_t* p) { return *reinterpret_cast<const v4s*>(p); }
__device__ __forceinline__ void st4(uint32_t* p, v4u v) { *reinterpret_cast<v4u*>(p) = v; }

uint32_t grid_for(size_t threads) { return static_cast<uint32_t>((threads + kThreads - 1) / kThreads); }

// g = 5^r mod 2N (r reduced mod N/2, the order of 5).
__host__ __device__ __forceinline__ uint32_t galois_of(uint32_t r, uint32_t log_n) {
  const uint32_t two_n_mask = (2u << log_n) - 1;
  uint32_t e = r & ((1u << (log_n - 1)) - 1), b = 5, g = 1;
  while (e) {
    if (e & 1) g = (g * b) & two_n_mask;
    b = (b * b) & two_n_mask;
    e >>= 1;
  }
  return g;
}

// Source index of NTT value i under sigma_g.
__device__ __forceinline__ uint32_t perm_src(uint32_t i, uint32_t g, uint32_t log_n) {
  const uint32_t shift = 32 - log_n;
  const uint32_t u = __builtin_bitreverse32(i) >> shift;
  const uint32_t v = (u * g + (g >> 1)) & ((1u << log_n) - 1);
  return __builtin_bitreverse32(v) >> shift;
}

// Four consecutive outputs c .. c+3 (c a multiple of 4) read from one aligned
// quad of the source row: their indices' low two bits are the top two of
// u = brv(c + e), and u g + (g-1)/2 mod N keeps the low log N - 2 bits of u
// fixed, so the sources share all bits above the low two.  A thread loads the
// quad once (16 bytes) and selects within it, instead of four scattered words.
struct QuadSrc {
  uint32_t base;   // the quad's first index
  uint32_t sel[4];
};
__device__ __forceinline__ QuadSrc quad_src(uint32_t c, uint32_t g, uint32_t log_n) {
  QuadSrc x;
  uint32_t s[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) s[e] = perm_src(c + e, g, log_n);
  x.base = s[0] & ~3u;
#pragma unroll
  for (int e = 0; e < 4; ++e) x.sel[e] = s[e] & 3u;
  return x;
}
__device__ __forceinline__ uint32_t pick(const v4u& v, uint32_t k) {
  return k == 0 ? v[0] : k == 1 ? v[1] : k == 2 ? v[2] : v[3];
}

// A sequence of ciphertexts [2][L][N] in memory: element m sits at ciphertext
// position (m / grp) * grp_stride + off + m % grp from the base.
struct Seq {
  uint32_t grp, grp_stride, off;
};
__host__ __device__ __forceinline__ size_t seq_pos(size_t m, Seq q) {
  return (m / q.grp) * q.grp_stride + q.off + m % q.grp;
}
inline Seq contiguous() { return Seq{1, 1, 0}; }

// Rotation k: input m = k / per_input, key slot k % key_period, step
// r0 + slot * r_step (or the fixed element galois_fixed when nonzero).
struct RotPlan {
  uint32_t per_input, key_period, r0, r_step, galois_fixed;
};
struct RotIndex {
  uint32_t m, slot, g;
};
__device__ __forceinline__ RotIndex rot_index(uint32_t k, RotPlan p, uint32_t log_n) {
  RotIndex x;
  x.m = k / p.per_input;
  x.slot = k % p.key_period;
  x.g = p.galois_fixed ? p.galois_fixed : galois_of(p.r0 + x.slot * p.r_step, log_n);
  return x;
}

// out[c][p][l][i] = in[c][p][l][perm_g(i)] for rows of N words, one g.
__global__ __launch_bounds__(kThreads) void automorphism_kernel(Tables tb, const uint32_t* __restrict__ in,
                                                                size_t rows, uint32_t g,
                                                                uint32_t* __restrict__ out) {
  const size_t i = static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x;
  const size_t row = i >> tb.log_n;
  if (row >= rows) return;
  const uint32_t k = static_cast<uint32_t>(i & (tb.n - 1));
  out[i] = in[(row << tb.log_n) + perm_src(k, g, tb.log_n)];
}

// ModUp, step 1: T[m][i] = limb i of c1 of input m (to be inverse-transformed).
__global__ __launch_bounds__(kThreads) void c1_copy_kernel(Tables tb, const uint32_t* __restrict__ ct, Seq in_seq,
                                                           uint32_t inputs, uint32_t L, uint32_t* __restrict__ T) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const size_t per = static_cast<size_t>(L) << tb.log_n;
  const size_t m = i / per;
  if (m >= inputs) return;
  const size_t off = i % per;
  st4(T + i, ld4(ct + seq_pos(m, in_seq) * 2 * per + per + off));
}

// ModUp, step 2: D[b][i][j] = centred(T[b][i] mod q_i) mod p_j for every prime
// j <= L (coefficient form).  Every prime exceeds 2^29 > q_i / 2, so the
// centred value needs no reduction: v or p_j - (q_i - v).
__global__ __launch_bounds__(kThreads) void modup_lift_kernel(Tables tb, const uint32_t* __restrict__ T, uint32_t count,
                                                              uint32_t L, uint32_t* __restrict__ D) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const size_t rowsz = tb.n;
  const size_t row = i >> tb.log_n;                        // b * L + digit
  if (row >= static_cast<size_t>(count) * L) return;
  const uint32_t digit = static_cast<uint32_t>(row % L);
  const uint32_t k = static_cast<uint32_t>(i & (tb.n - 1));
  const uint32_t qi = tb.q[digit], half = qi >> 1;
  const v4u v = ld4(T + i);
  uint32_t* dst = D + (row * (L + 1)) * rowsz + k;
  for (uint32_t j = 0; j <= L; ++j) {
    const uint32_t pj = tb.q[j];
    v4u o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = v[e] > half ? pj - (qi - v[e]) : v[e];
    st4(dst + j * rowsz, o);
  }
}

// ModUp in one kernel for small launches (N <= 2^14): a workgroup takes
// digit i of input m and one target prime p_j.  It reads limb i of c1
// coalesced, inverse-transforms it, centres it (|d| < q_i / 2) and writes
// NTT_j(d mod p_j) to D[m][i][j]; for j == i that is limb i itself, copied.
// The same values as the copy / batched INTT / lift / batched NTT route, with
// a chain of two transforms per workgroup instead of four launches.
template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN, true>::P::T), (WholePlan<LOGN, true>::kWavesPerSimd)) void
modup_fused_kernel(Tables tb, const uint32_t* __restrict__ ct, Seq in_seq, uint32_t L, uint32_t* __restrict__ D) {
  using P = typename WholePlan<LOGN, true>::P;
  constexpr int LOGE = WholePlan<LOGN, true>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const uint32_t m = blockIdx.x / L, i = blockIdx.x % L, j = blockIdx.y;
  const uint32_t t = threadIdx.x;
  const uint32_t Lp = L + 1;
  const uint32_t c_base = pos_coalesced<LOGE>(t, 0);
  const uint32_t* src = ct + (seq_pos(m, in_seq) * 2 + 1) * L * N + static_cast<size_t>(i) * N + c_base;
  uint32_t* dst = D + ((static_cast<size_t>(m) * L + i) * Lp + j) * N + c_base;
  uint32_t v[P::E];
#pragma unroll
  for (int e = 0; e < P::E; ++e) v[e] = src[e << 6];
  if (j == i) {                                             // workgroup-uniform
#pragma unroll
    for (int e = 0; e < P::E; ++e) dst[e << 6] = v[e];
    return;
  }
  wave_relayout<LOGN, LOGE, true>(v, t, lds);
  const uint32_t qi = tb.q[i];
  const size_t ti = static_cast<size_t>(i) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + ti, tb.inv_shoup + ti, qi, lds);
  const uint32_t ni = tb.ninv[i], nis = tb.ninv_shoup[i];
  const uint32_t pj = tb.q[j];
#pragma unroll
  for (int e = 0; e < P::E; ++e) {
    const uint32_t y = mul_shoup(v[e], ni, nis, qi);
    v[e] = y > (qi >> 1) ? pj - (qi - y) : y;               // centred digit mod p_j
  }
  const size_t tj = static_cast<size_t>(j) << LOGN;
  fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tj, tb.fwd_shoup + tj, pj, lds);
  wave_relayout<LOGN, LOGE, false>(v, t, lds);
#pragma unroll
  for (int e = 0; e < P::E; ++e) dst[e << 6] = v[e];
}

// ModUp in two launches for larger batches (N <= 2^14), without the
// round trips of the copy / batched INTT / lift / batched NTT route:
//   modup_intt_kernel, one workgroup per digit (input m, limb i of c1): read
//     the limb coalesced, inverse-transform it, scale by N^-1 and write the
//     coefficients to T[m][i] in the plan's group-0 register order (element e
//     of thread t at e * T + t: coalesced both ways, read back by the same
//     plan's threads);
//   modup_ntt_kernel, one workgroup per (digit, prime p_j): centre the digit,
//     lift it to p_j and forward-transform it into D[m][i][j] (for j == i the
//     limb itself, copied).
// One inverse transform per digit instead of one per (digit, prime) as in
// modup_fused_kernel, whose workgroups then outnumber the CUs.
template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN>::P::T), (WholePlan<LOGN>::kWavesPerSimd)) void modup_intt_kernel(
    Tables tb, const uint32_t* __restrict__ ct, Seq in_seq, uint32_t L, uint32_t* __restrict__ T) {
  using P = typename WholePlan<LOGN>::P;
  constexpr int LOGE = WholePlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const uint32_t m = blockIdx.x / L, i = blockIdx.x % L;
  const uint32_t t = threadIdx.x;
  const uint32_t* src = ct + (seq_pos(m, in_seq) * 2 + 1) * L * N + static_cast<size_t>(i) * N + pos_coalesced<LOGE>(t, 0);
  uint32_t v[P::E];
#pragma unroll
  for (int e = 0; e < P::E; ++e) v[e] = src[e << 6];
  wave_relayout<LOGN, LOGE, true>(v, t, lds);
  const uint32_t qi = tb.q[i];
  const size_t ti = static_cast<size_t>(i) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + ti, tb.inv_shoup + ti, qi, lds);
  const uint32_t ni = tb.ninv[i], nis = tb.ninv_shoup[i];
  uint32_t* dst = T + static_cast<size_t>(blockIdx.x) * N + t;
#pragma unroll
  for (int e = 0; e < P::E; ++e) dst[e * P::T] = mul_shoup(v[e], ni, nis, qi);
}

template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN>::P::T), (WholePlan<LOGN>::kWavesPerSimd)) void modup_ntt_kernel(
    Tables tb, const uint32_t* __restrict__ ct, Seq in_seq, const uint32_t* __restrict__ T, uint32_t L,
    uint32_t* __restrict__ D) {
  using P = typename WholePlan<LOGN>::P;
  constexpr int LOGE = WholePlan<LOGN>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const uint32_t m = blockIdx.x / L, i = blockIdx.x % L, j = blockIdx.y;
  const uint32_t t = threadIdx.x;
  const uint32_t c_base = pos_coalesced<LOGE>(t, 0);
  uint32_t* dst = D + ((static_cast<size_t>(m) * L + i) * (L + 1) + j) * N + c_base;
  uint32_t v[P::E];
  if (j == i) {                                             // workgroup-uniform
    const uint32_t* src = ct + (seq_pos(m, in_seq) * 2 + 1) * L * N + static_cast<size_t>(i) * N + c_base;
#pragma unroll
    for (int e = 0; e < P::E; ++e) dst[e << 6] = src[e << 6];
    return;
  }
  const uint32_t* src = T + static_cast<size_t>(blockIdx.x) * N + t;
  const uint32_t qi = tb.q[i], pj = tb.q[j];
#pragma unroll
  for (int e = 0; e < P::E; ++e) {
    const uint32_t y = src[e * P::T];
    v[e] = y > (qi >> 1) ? pj - (qi - y) : y;               // centred digit mod p_j
  }
  const size_t tj = static_cast<size_t>(j) << LOGN;
  fwd_block<LOGN, LOGN, LOGE>(v, t, 0, tb.fwd + tj, tb.fwd_shoup + tj, pj, lds);
  wave_relayout<LOGN, LOGE, false>(v, t, lds);
#pragma unroll
  for (int e = 0; e < P::E; ++e) dst[e << 6] = v[e];
}

// Key-switch inner product for rotation k (input m, Galois element g):
//   acc[k][p][j][n] = sum_i D[m][i][j][perm_g(n)] * K[slot][i][p][j][n]   mod p_j,  p in {0, 1}.
// Products are below 2^60 and at most 15 are summed, so one reduction of the
// 64-bit sums finishes.  A thread serves one key slot and loops over the
// rotations that use that key (k = u * key_period + slot, one per input of a
// batch), so each key is streamed from HBM once per call and re-read from
// cache by the same thread.  When keys x primes x N/4 threads are too few to
// fill the chip (small rings, large batches), the loop over u is cut into
// `chunks` ranges on as many workgroups (blockIdx.x / blocks_per_chunk).
// With KL = L > 0 (L <= 4) the thread's 8 L key words stay in registers for
// the whole loop instead of being re-read per use (past L2 once the keys of
// a rotation set outgrow it); KL = 0 takes any L.
template <int KL>
__global__ __launch_bounds__(kThreads) void ks_inner_kernel(Tables tb, const uint32_t* __restrict__ D,
                                                            const uint32_t* __restrict__ ksk, uint32_t L,
                                                            uint32_t rotations, RotPlan plan,
                                                            uint32_t blocks_per_chunk, uint32_t chunks,
                                                            uint32_t* __restrict__ acc) {
  const uint32_t chunk = blockIdx.x / blocks_per_chunk;
  const size_t i = (static_cast<size_t>(blockIdx.x % blocks_per_chunk) * kThreads + threadIdx.x) * 4;
  const uint32_t log_n = tb.log_n, n = tb.n;
  const size_t row = i >> log_n;                           // slot * (L + 1) + j
  const uint32_t Lp = L + 1;
  if (row >= static_cast<size_t>(plan.key_period) * Lp) return;
  const uint32_t slot = static_cast<uint32_t>(row / Lp), j = static_cast<uint32_t>(row % Lp);
  const uint32_t c = static_cast<uint32_t>(i & (n - 1));
  const RotIndex x0 = rot_index(slot, plan, log_n);        // the element depends on the slot only
  const QuadSrc qs = quad_src(c, x0.g, log_n);
  const size_t key_stride = static_cast<size_t>(2) * Lp * n;        // one digit of one key
  const uint32_t* key = ksk + static_cast<size_t>(slot) * L * key_stride + static_cast<size_t>(j) * n + c;
  const uint32_t pj = tb.q[j];
  const double pr = tb.q_recip[j];
  const uint32_t uses = rotations / plan.key_period;        // rotations per key
  const uint32_t u_begin = static_cast<uint32_t>(static_cast<uint64_t>(uses) * chunk / chunks);
  const uint32_t u_end = static_cast<uint32_t>(static_cast<uint64_t>(uses) * (chunk + 1) / chunks);
  constexpr int KR = KL > 0 ? KL : 1;
  v4u kr0[KR], kr1[KR];
  if constexpr (KL > 0) {
#pragma unroll
    for (int d = 0; d < KL; ++d) {
      kr0[d] = ld4(key + d * key_stride);
      kr1[d] = ld4(key + d * key_stride + static_cast<size_t>(Lp) * n);
    }
  }
  for (uint32_t k = slot + u_begin * plan.key_period; k < u_end * plan.key_period; k += plan.key_period) {
    const uint32_t m = k / plan.per_input;
    const uint32_t* dig = D + (static_cast<size_t>(m) * L * Lp + j) * n;
    uint64_t a0[4] = {0, 0, 0, 0}, a1[4] = {0, 0, 0, 0};
    auto digit = [&](uint32_t d, const v4u& k0, const v4u& k1) {
      const v4u dq = ld4(dig + static_cast<size_t>(d) * Lp * n + qs.base);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint64_t dv = pick(dq, qs.sel[e]);
        a0[e] += dv * k0[e];
        a1[e] += dv * k1[e];
      }
    };
    if constexpr (KL > 0) {
#pragma unroll
      for (int d = 0; d < KL; ++d) digit(d, kr0[d], kr1[d]);
    } else {
      for (uint32_t d = 0; d < L; ++d)
        digit(d, ld4(key + d * key_stride), ld4(key + d * key_stride + static_cast<size_t>(Lp) * n));
    }
    v4u o0, o1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o0[e] = reduce_u64(a0[e], pj, pr);
      o1[e] = reduce_u64(a1[e], pj, pr);
    }
    uint32_t* out = acc + ((static_cast<size_t>(k) * 2) * Lp + j) * n + c;
    st4(out, o0);
    st4(out + static_cast<size_t>(Lp) * n, o1);
  }
}

// Rotation k's result: out[k] = (sigma_g(c0_m) + u0, u1), u = ModDown(acc[k]) (tmp[k][2][L][N]);
// at 2^15 and 2^16, after the separate ModDown.
__global__ __launch_bounds__(kThreads) void rot_combine_kernel(Tables tb, const uint32_t* __restrict__ ct, Seq in_seq,
                                                               const uint32_t* __restrict__ tmp, uint32_t L,
                                                               uint32_t rotations, RotPlan plan,
                                                               uint32_t* __restrict__ out, Seq out_seq) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const uint32_t log_n = tb.log_n, n = tb.n;
  const size_t row = i >> log_n;                           // k * L + l
  if (row >= static_cast<size_t>(rotations) * L) return;
  const uint32_t k = static_cast<uint32_t>(row / L), l = static_cast<uint32_t>(row % L);
  const uint32_t c = static_cast<uint32_t>(i & (n - 1));
  const RotIndex x = rot_index(k, plan, log_n);
  const size_t ctw = static_cast<size_t>(2) * L * n;
  const uint32_t* c0 = ct + seq_pos(x.m, in_seq) * ctw + static_cast<size_t>(l) * n;
  const size_t base = (static_cast<size_t>(k) * 2 * L + l) * n + c;
  const v4u u0 = ld4(tmp + base);
  const v4u u1 = ld4(tmp + base + static_cast<size_t>(L) * n);
  const uint32_t q = tb.q[l];
  const QuadSrc qs = quad_src(c, x.g, log_n);
  const v4u cq = ld4(c0 + qs.base);
  v4u o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = add_mod(pick(cq, qs.sel[e]), u0[e], q);
  uint32_t* dst = out + seq_pos(k, out_seq) * ctw + static_cast<size_t>(l) * n + c;
  st4(dst, o);
  st4(dst + static_cast<size_t>(L) * n, u1);
}

// ModDown of the key-switching inner products fused with the rotations' final
// step (N <= 2^14): for rotation k (input m, Galois element g) and component p,
//     r   = centred INTT_P(acc[k][p][P row]),
//     u_l = (acc[k][p][l] - NTT_l(r mod q_l)) P^-1   mod q_l,
//     out[k] = (sigma_g(c0_m) + u0, u1),
// the rescale's arithmetic (the P row is the last of the L + 1) with the
// combine as its store, so u never goes through memory.  One workgroup per
// polynomial acc[k][p] and output limb l (blockIdx.y), latency plan, as the
// split rescale, at every batch size: two transforms per workgroup where a
// loop over the limbs would take 1 + L per polynomial, but no intermediate
// rows and no second launch (measured: 4% faster for 1920 rotations at 2^10,
// 2% slower for 3968 at 2^13).  (A loop over the limbs would also spill with
// the permuted c0 loads in its store.)
template <int LOGN>
__global__ __launch_bounds__((WholePlan<LOGN, true>::P::T), (WholePlan<LOGN, true>::kWavesPerSimd)) void
moddown_combine_kernel(Tables tb, const uint32_t* __restrict__ acc, const uint32_t* __restrict__ ct, Seq in_seq,
                       uint32_t L, uint32_t rotations, RotPlan plan, uint32_t* __restrict__ out, Seq out_seq,
                       Seq copy_seq) {
  using P = typename WholePlan<LOGN, true>::P;
  constexpr int LOGE = WholePlan<LOGN, true>::LOGE;
  constexpr int N = P::B;
  __shared__ uint32_t lds[P::lds_words];
  const uint32_t t = threadIdx.x;
  const uint32_t c_base = pos_coalesced<LOGE>(t, 0);
  if (blockIdx.x >= 2 * rotations) {
    // workgroups past the rotations copy limb blockIdx.y of component p of
    // input m unchanged to element m of copy_seq (the BSGS baby slot 0), so
    // that copy needs no launch of its own; the whole workgroup returns here
    const uint32_t idx = blockIdx.x - 2 * rotations, m = idx >> 1, pc = idx & 1;
    const size_t row = static_cast<size_t>(pc) * L * N + static_cast<size_t>(blockIdx.y) * N + c_base;
    const uint32_t* cs = ct + seq_pos(m, in_seq) * 2 * L * N + row;
    uint32_t* cd = out + seq_pos(m, copy_seq) * 2 * L * N + row;
#pragma unroll
    for (int j = 0; j < P::E; ++j) cd[j << 6] = cs[j << 6];
    return;
  }
  const uint32_t poly = blockIdx.x;                         // k * 2 + p
  const uint32_t k = poly >> 1, p = poly & 1;
  const uint32_t top = L;                                   // the special prime's row
  const uint32_t* src = acc + static_cast<size_t>(poly) * (L + 1) * N + c_base;
  const RotIndex x = rot_index(k, plan, LOGN);
  const size_t ctw = static_cast<size_t>(2) * L * N;
  const uint32_t* c0 = ct + seq_pos(x.m, in_seq) * ctw;
  uint32_t* dst = out + seq_pos(k, out_seq) * ctw + static_cast<size_t>(p) * L * N + c_base;

  uint32_t v[P::E];
  const uint32_t* stop = src + static_cast<size_t>(top) * N;
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = stop[j << 6];
  wave_relayout<LOGN, LOGE, true>(v, t, lds);
  const uint32_t qt = tb.q[top];
  const size_t ttop = static_cast<size_t>(top) << LOGN;
  inv_block<LOGN, LOGN, LOGE>(v, t, 0, tb.inv + ttop, tb.inv_shoup + ttop, qt, lds);
  const uint32_t ni = tb.ninv[top], nis = tb.ninv_shoup[top];
  int32_t r[P::E];
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    const uint32_t y = mul_shoup(v[j], ni, nis, qt);
    r[j] = y > (qt >> 1) ? static_cast<int32_t>(y) - static_cast<int32_t>(qt) : static_cast<int32_t>(y);
  }

  {
    const uint32_t l = blockIdx.y, q = tb.q[l];
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = static_cast<uint32_t>(r[j] < 0 ? r[j] + static_cast<int32_t>(q) : r[j]);
    const size_t tl = static_cast<size_t>(l) << LOGN;
    fwd_block<LOGN, LOGN, LOGE, 0, false>(v, t, 0, tb.fwd + tl, tb.fwd_shoup + tl, q, lds);  // [0, 4q)
    wave_relayout<LOGN, LOGE, false>(v, t, lds);
    const uint32_t pi = tb.qinv[top * tb.L + l], pis = tb.qinv_shoup[top * tb.L + l];
    const uint32_t* sl = src + static_cast<size_t>(l) * N;
    uint32_t* dl = dst + static_cast<size_t>(l) * N;
    if (p == 0) {                                           // workgroup-uniform
      const uint32_t* c0l = c0 + static_cast<size_t>(l) * N;
#pragma unroll
      for (int j = 0; j < P::E; ++j) {
        const uint32_t u = sub_lazy_mul_shoup(sl[j << 6], v[j], pi, pis, q);
        dl[j << 6] = add_mod(u, c0l[perm_src(c_base + (j << 6), x.g, LOGN)], q);
      }
    } else {
#pragma unroll
      for (int j = 0; j < P::E; ++j) dl[j << 6] = sub_lazy_mul_shoup(sl[j << 6], v[j], pi, pis, q);
    }
  }
}

// Rotation keys, after the error rows have been forward-transformed in the
// b rows: b_i[j] += -a_i[j] s[j] (+ P s_g[j] when j == i), with s_g = sigma_g(s)
// read through the permutation of the NTT-form secret.
__global__ __launch_bounds__(kThreads) void keygen_combine_kernel(Tables tb, const uint32_t* __restrict__ s_ntt,
                                                                  const uint32_t* __restrict__ a, uint32_t L,
                                                                  uint32_t keys, uint32_t r0, uint32_t r_step,
                                                                  uint32_t* __restrict__ ksk) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const uint32_t log_n = tb.log_n, n = tb.n, Lp = L + 1;
  const size_t row = i >> log_n;                           // (key * L + digit) * Lp + j
  if (row >= static_cast<size_t>(keys) * L * Lp) return;
  const uint32_t j = static_cast<uint32_t>(row % Lp);
  const size_t kd = row / Lp;                              // key * L + digit
  const uint32_t digit = static_cast<uint32_t>(kd % L), key = static_cast<uint32_t>(kd / L);
  const uint32_t c = static_cast<uint32_t>(i & (n - 1));
  const uint32_t q = tb.q[j], mu = tb.barrett[j];
  const v4u av = ld4(a + row * n + c);
  const v4u sv = ld4(s_ntt + static_cast<size_t>(j) * n + c);
  uint32_t* b = ksk + ((kd * 2) * Lp + j) * n + c;
  const v4u bv = ld4(b);
  v4u o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = sub_mod(bv[e], mul_mod_barrett(av[e], sv[e], q, mu), q);
  if (j == digit) {
    const uint32_t g = galois_of(r0 + key * r_step, log_n);
    const uint32_t pm = tb.q[L] % q;                        // P mod q_i
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t sg = s_ntt[static_cast<size_t>(j) * n + perm_src(c + e, g, log_n)];
      o[e] = add_mod(o[e], mul_mod_barrett(pm, sg, q, mu), q);
    }
  }
  st4(b, o);
  st4(b + static_cast<size_t>(Lp) * n, av);
}

// ksk[key][i][0][j] = e[key][i] mod p_j (coefficient form; transformed next).
__global__ __launch_bounds__(kThreads) void keygen_err_kernel(Tables tb, const int32_t* __restrict__ e, uint32_t L,
                                                              uint32_t keys, uint32_t* __restrict__ ksk) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const uint32_t n = tb.n, Lp = L + 1;
  const size_t row = i >> tb.log_n;                        // key * L + digit
  if (row >= static_cast<size_t>(keys) * L) return;
  const uint32_t c = static_cast<uint32_t>(i & (n - 1));
  const v4s ev = ld4(e + row * n + c);
  for (uint32_t j = 0; j < Lp; ++j) {
    const uint32_t q = tb.q[j];
    v4u r;
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = ev[k] < 0 ? q - static_cast<uint32_t>(-ev[k]) : static_cast<uint32_t>(ev[k]);
    st4(ksk + ((row * 2) * Lp + j) * n + c, r);
  }
}

// Giant-step sum in the extended basis q_0 .. q_{L-1}, P, ahead of its one
// ModDown: for input b,
//   ext[b] = P ( inner[b][0] + sum_{j>=1} (sigma_gj(c0 of inner[b][j]), 0) ) + sum_{j>=1} acc[b (n2-1) + j - 1],
// acc[k] [2][L+1][N] the giant rotations' key-switching inner products (P last),
// g_j = g1^j with g1 = 5^n1.  P y is exact in the extended basis, so one
// division by P after the sum stands for the n2 - 1 divisions of the rotations.
// A workgroup takes 64 consecutive coefficients of one row; its 4 waves sum the
// terms j = 1 + w, 5 + w, .. (independent loads in flight) and combine through LDS.
__global__ __launch_bounds__(kThreads) void giant_ext_kernel(Tables tb, const uint32_t* __restrict__ inner,
                                                             const uint32_t* __restrict__ acc, uint32_t L,
                                                             uint32_t count, uint32_t n2, uint32_t g1,
                                                             uint32_t* __restrict__ ext) {
  __shared__ uint32_t part[2][3][64];
  const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const size_t i = static_cast<size_t>(blockIdx.x) * 64 + lane;
  const uint32_t log_n = tb.log_n, n = tb.n, Lp = L + 1;
  const size_t ctw = static_cast<size_t>(2) * L * n, extw = static_cast<size_t>(2) * Lp * n;
  const size_t b = i / extw;                                // workgroup-uniform (64 | N)
  if (b >= count) return;
  const size_t off = i % extw;                              // (p * (L + 1) + l) * N + c
  const uint32_t pl = static_cast<uint32_t>(off >> log_n);
  const uint32_t p = pl / Lp, l = pl % Lp, c = static_cast<uint32_t>(off & (n - 1));
  const uint32_t q = tb.q[l];
  const bool carries_sigma = p == 0 && l < L;               // rows with the rotated c0 terms
  const uint32_t* in_b = inner + b * n2 * ctw;
  const uint32_t* acc_b = acc + b * (n2 - 1) * extw + off;
  const uint32_t mask = (2u << log_n) - 1;
  uint32_t g = 1, g4 = 1;
  for (uint32_t e = 0; e <= w; ++e) g = (g * g1) & mask;   // g1^(1 + w)
  for (int e = 0; e < 4; ++e) g4 = (g4 * g1) & mask;       // g1^4
  uint32_t sy = (w == 0 && l < L) ? in_b[(static_cast<size_t>(p) * L + l) * n + c] : 0;
  uint32_t sa = 0;
  // the row kind is workgroup-uniform: one loop per kind, no branch inside
  if (carries_sigma) {
#pragma unroll 4
    for (uint32_t j = 1 + w; j < n2; j += 4) {
      sa = add_mod(sa, acc_b[(j - 1) * extw], q);
      sy = add_mod(sy, in_b[j * ctw + static_cast<size_t>(l) * n + perm_src(c, g, log_n)], q);
      g = (g * g4) & mask;
    }
  } else {
#pragma unroll 4
    for (uint32_t j = 1 + w; j < n2; j += 4) sa = add_mod(sa, acc_b[(j - 1) * extw], q);
  }
  if (w > 0) {
    part[0][w - 1][lane] = sy;
    part[1][w - 1][lane] = sa;
  }
  __syncthreads();
  if (w == 0) {
    sy = add_mod(add_mod(sy, part[0][0][lane], q), add_mod(part[0][1][lane], part[0][2][lane], q), q);
    sa = add_mod(add_mod(sa, part[1][0][lane], q), add_mod(part[1][1][lane], part[1][2][lane], q), q);
    const uint32_t p_mod = tb.q[L] % q;                     // 0 on the P row, where sy is 0 too
    ext[i] = add_mod(sa, reduce_u64(static_cast<uint64_t>(sy) * p_mod, q, tb.q_recip[l]), q);
  }
}

// Batched full-polynomial MAC of the BSGS inner sums, for several inputs that
// share the plaintexts: inner[b][j] = sum_i pt[j][i] (.) baby[b][i], per
// coefficient a (n2 x n1) by (n1 x 2 count) product.  A thread takes one
// coefficient of one limb and a register tile of kTileJ rows j by kTileB
// inputs b (both components): per i it loads kTileJ plaintext residues and
// 2 kTileB input residues for 2 kTileJ kTileB products, so the plaintexts are
// read count / kTileB times and the inputs n2 / kTileJ times (the previous
// form, one row by four inputs, re-read every input n2 times and was bound by
// that L2 traffic).  64-bit sums, folded every 11 products.  Workgroups that
// share a plaintext tile (consecutive b tiles) or an input tile are numbered
// together and placed on one XCD.
constexpr int kTileJ = 8, kTileB = 2;
__global__ __launch_bounds__(kThreads) void bsgs_mac_tile_kernel(Tables tb, const uint32_t* __restrict__ pt,
                                                                 const uint32_t* __restrict__ baby, uint32_t count,
                                                                 uint32_t n1, uint32_t n2, uint32_t L,
                                                                 uint32_t* __restrict__ inner) {
  const uint32_t n = tb.n;
  const uint32_t G = gridDim.x, bid = blockIdx.x;
  const uint32_t lid = (G & 7) ? bid : (bid & 7) * (G >> 3) + (bid >> 3);   // XCD-contiguous numbering
  const uint32_t btiles = (count + kTileB - 1) / kTileB, jtiles = (n2 + kTileJ - 1) / kTileJ;
  const uint32_t cblocks = n / kThreads;
  // lid = ((l * cblocks + cb) * jtiles + jt) * btiles + bt
  const uint32_t bt = lid % btiles;
  uint32_t rest = lid / btiles;
  const uint32_t jt = rest % jtiles;
  rest /= jtiles;
  const uint32_t cb = rest % cblocks, l = rest / cblocks;
  const uint32_t c = cb * kThreads + threadIdx.x;
  const uint32_t j0 = jt * kTileJ, b0 = bt * kTileB;
  const uint32_t jn = n2 - j0 < static_cast<uint32_t>(kTileJ) ? n2 - j0 : kTileJ;   // workgroup-uniform
  const uint32_t bn = count - b0 < static_cast<uint32_t>(kTileB) ? count - b0 : kTileB;
  const uint32_t q = tb.q[l];
  const double qr = tb.q_recip[l];
  const size_t ln = static_cast<size_t>(L) * n, ctw = 2 * ln;
  // row pointers are workgroup-uniform (scalar); the lane adds its coefficient c
  const uint32_t* prow = pt + (static_cast<size_t>(j0) * n1 * L + l) * n;         // + (jj n1 + i) L N
  const uint32_t* xrow = baby + static_cast<size_t>(b0) * n1 * ctw + static_cast<size_t>(l) * n;   // + (bb n1 + i) ctw
  const size_t pj_stride = static_cast<size_t>(n1) * ln, xb_stride = static_cast<size_t>(n1) * ctw;
  // Sums are folded every kFold products: a = hi 2^32 + lo -> hi (2^32 mod q) + lo
  // (exact mod q) is below 2^62 + 2^32, and kFold = 11 further products below
  // 2^60 keep it below 2^64; one full reduction at the end.
  constexpr uint32_t kFold = 11;
  const uint32_t c32 = reduce_u64(uint64_t{1} << 32, q, qr);
  uint64_t a[kTileJ][2 * kTileB];
#pragma unroll
  for (int jj = 0; jj < kTileJ; ++jj)
#pragma unroll
    for (int x = 0; x < 2 * kTileB; ++x) a[jj][x] = 0;
  uint32_t since = 0;
  for (uint32_t i = 0; i < n1; ++i) {
    // every load is issued (rows past a partial tile read the tile's first
    // row, in bounds) and its value zeroed by a select, so the 12 loads go
    // out back to back instead of one branch each
    uint32_t xv[2 * kTileB], pv[kTileJ];
#pragma unroll
    for (int bb = 0; bb < kTileB; ++bb) {
      const bool in = static_cast<uint32_t>(bb) < bn;
      const uint32_t* xp = xrow + (in ? bb : 0) * xb_stride + static_cast<size_t>(i) * ctw;
      const uint32_t x0 = xp[c], x1 = (xp + ln)[c];
      xv[2 * bb] = in ? x0 : 0;
      xv[2 * bb + 1] = in ? x1 : 0;
    }
#pragma unroll
    for (int jj = 0; jj < kTileJ; ++jj) {
      const bool in = static_cast<uint32_t>(jj) < jn;
      const uint32_t p = (prow + (in ? jj : 0) * pj_stride + static_cast<size_t>(i) * ln)[c];
      pv[jj] = in ? p : 0;
    }
#pragma unroll
    for (int jj = 0; jj < kTileJ; ++jj)
#pragma unroll
      for (int x = 0; x < 2 * kTileB; ++x) a[jj][x] += static_cast<uint64_t>(pv[jj]) * xv[x];
    if (++since == kFold) {
      since = 0;
#pragma unroll
      for (int jj = 0; jj < kTileJ; ++jj)
#pragma unroll
        for (int x = 0; x < 2 * kTileB; ++x)
          a[jj][x] = static_cast<uint64_t>(static_cast<uint32_t>(a[jj][x] >> 32)) * c32 +
                     static_cast<uint32_t>(a[jj][x]);
    }
  }
#pragma unroll
  for (int jj = 0; jj < kTileJ; ++jj)
#pragma unroll
    for (int x = 0; x < 2 * kTileB; ++x) a[jj][x] = reduce_u64(a[jj][x], q, qr);
#pragma unroll
  for (int bb = 0; bb < kTileB; ++bb) {
    if (static_cast<uint32_t>(bb) >= bn) continue;
    uint32_t* o = inner + (static_cast<size_t>(b0 + bb) * n2 + j0) * ctw + static_cast<size_t>(l) * n + c;
#pragma unroll
    for (int jj = 0; jj < kTileJ; ++jj) {
      if (static_cast<uint32_t>(jj) >= jn) continue;
      o[jj * ctw] = static_cast<uint32_t>(a[jj][2 * bb]);
      o[jj * ctw + ln] = static_cast<uint32_t>(a[jj][2 * bb + 1]);
    }
  }
}

// Workspace of rotate(): T [inputs][L][N], D [inputs][L][L+1][N],
// acc [rotations][2][L+1][N], tmp [rotations][2][L][N] (the separate ModDown's
// output, 2^15 and 2^16), rescale scratch.
struct RotWs {
  uint32_t *T, *D, *acc, *tmp;
  void* rs;
  size_t bytes;
};

RotWs rot_layout(const Tables& t, uint32_t inputs, uint32_t rotations, void* base) {
  const size_t n = t.n, L = t.L - 1;
  RotWs w;
  uint8_t* p = static_cast<uint8_t*>(base);
  size_t off = 0;
  auto take = [&](size_t words) {
    uint8_t* q = p ? p + off : nullptr;
    off += ((words * 4 + 255) / 256) * 256;
    return reinterpret_cast<uint32_t*>(q);
  };
  w.T = take(inputs * L * n);
  w.D = take(inputs * L * (L + 1) * n);
  w.acc = take(rotations * 2 * (L + 1) * n);
  w.tmp = take(rotations * 2 * L * n);
  const size_t rs = rescale_workspace_bytes(t, rotations, static_cast<uint32_t>(L + 1));
  w.rs = p ? p + off : nullptr;
  off += ((rs + 255) / 256) * 256;
  w.bytes = off;
  return w;
}

// out = a + b, elementwise mod q_l over ciphertexts [count][2][limbs][N].
__global__ __launch_bounds__(kThreads) void ct_add_kernel(Tables tb, const uint32_t* __restrict__ a,
                                                          const uint32_t* __restrict__ b, uint32_t count,
                                                          uint32_t limbs, uint32_t* __restrict__ out) {
  const size_t i = (static_cast<size_t>(blockIdx.x) * kThreads + threadIdx.x) * 4;
  const size_t total = static_cast<size_t>(count) * 2 * limbs << tb.log_n;
  if (i >= total) return;
  const uint32_t l = static_cast<uint32_t>((i >> tb.log_n) % limbs);
  const uint32_t q = tb.q[l];
  const v4u x = ld4(a + i), y = ld4(b + i);
  v4u o;
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = add_mod(x[e], y[e], q);
  st4(out + i, o);
}

}  // namespace

hipError_t launch_ct_add(const Tables& t, const uint32_t* a, const uint32_t* b, uint32_t count, uint32_t limbs,
                         uint32_t* out, hipStream_t s) {
  if (count == 0) return hipSuccess;
  ct_add_kernel<<<grid_for((static_cast<size_t>(count) * 2 * limbs << t.log_n) / 4), kThreads, 0, s>>>(t, a, b, count,
                                                                                                     limbs, out);
  return hipGetLastError();
}

size_t rotate_workspace_bytes(const Tables& t, uint32_t inputs, uint32_t rotations) {
  return rot_layout(t, inputs, rotations, nullptr).bytes;
}

hipError_t launch_automorphism(const Tables& t, const uint32_t* in, size_t rows, uint32_t galois, uint32_t* out,
                               hipStream_t s) {
  if (rows == 0) return hipSuccess;
  automorphism_kernel<<<grid_for(rows << t.log_n), kThreads, 0, s>>>(t, in, rows, galois, out);
  return hipGetLastError();
}

// `rotations` rotations of `inputs` ciphertexts (element m of in_seq from ct):
// rotation k acts on input k / plan.per_input with key ksk[k % key_period]
// ([key_period][L][2][L+1][N]) and is written as element k of out_seq.  Each
// input is decomposed once (ModUp), however many rotations read it.
// With out == nullptr the rotations stop before ModDown: the key-switching
// inner product acc[k] ([2][L+1][N], P last) is left in the workspace's acc
// region (rot_layout(..).acc) for a consumer that sums before dividing by P.
hipError_t launch_rotate_seq(const Tables& t, const uint32_t* ct, Seq in_seq, uint32_t inputs, uint32_t rotations,
                             RotPlan plan, const uint32_t* ksk, void* workspace, uint32_t* out, Seq out_seq,
                             hipStream_t s, const Seq* copy_inputs) {
  if (rotations == 0) return hipSuccess;
  if (rotations % plan.key_period != 0) return hipErrorInvalidValue;   // every key serves whole batches
  const uint32_t L = t.L - 1, Lp = L + 1;
  const size_t n = t.n;
  RotWs w = rot_layout(t, inputs, rotations, workspace);
  hipError_t err;
  // ModUp: one fused launch while its workgroups (one per input, digit and prime)
  // number at most one per CU (the baby steps of one vector at d = 1024: 20),
  // else up to 2^14 the two-launch form (the giant steps: 124 inverse and 620
  // forward workgroups), else copy / batched INTT / lift / batched NTT
  const size_t fused_groups = static_cast<size_t>(inputs) * L * Lp;
  const dim3 grid(inputs * L, Lp);
  if (t.log_n <= 14 && fused_groups <= static_cast<size_t>(t.num_cus)) {
    switch (t.log_n) {
      case 10: modup_fused_kernel<10><<<grid, WholePlan<10, true>::P::T, 0, s>>>(t, ct, in_seq, L, w.D); break;
      case 11: modup_fused_kernel<11><<<grid, WholePlan<11, true>::P::T, 0, s>>>(t, ct, in_seq, L, w.D); break;
      case 12: modup_fused_kernel<12><<<grid, WholePlan<12, true>::P::T, 0, s>>>(t, ct, in_seq, L, w.D); break;
      case 13: modup_fused_kernel<13><<<grid, WholePlan<13, true>::P::T, 0, s>>>(t, ct, in_seq, L, w.D); break;
      default: modup_fused_kernel<14><<<grid, WholePlan<14, true>::P::T, 0, s>>>(t, ct, in_seq, L, w.D); break;
    }
    if ((err = hipGetLastError()) != hipSuccess) return err;
  } else if (t.log_n <= 14) {
    switch (t.log_n) {
#define CKKS_MODUP2(LN)                                                                           \
  case LN:                                                                                        \
    modup_intt_kernel<LN><<<inputs * L, WholePlan<LN>::P::T, 0, s>>>(t, ct, in_seq, L, w.T);      \
    if ((err = hipGetLastError()) != hipSuccess) return err;                                      \
    modup_ntt_kernel<LN><<<grid, WholePlan<LN>::P::T, 0, s>>>(t, ct, in_seq, w.T, L, w.D);        \
    break;
      CKKS_MODUP2(10)
      CKKS_MODUP2(11)
      CKKS_MODUP2(12)
      CKKS_MODUP2(13)
      default: CKKS_MODUP2(14)
#undef CKKS_MODUP2
    }
    if ((err = hipGetLastError()) != hipSuccess) return err;
  } else {
    c1_copy_kernel<<<grid_for(inputs * L * n / 4), kThreads, 0, s>>>(t, ct, in_seq, inputs, L, w.T);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    err = launch_ntt(t, w.T, static_cast<size_t>(inputs) * L, L, true, s);
    if (err != hipSuccess) return err;
    modup_lift_kernel<<<grid_for(inputs * L * n / 4), kThreads, 0, s>>>(t, w.T, inputs, L, w.D);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    err = launch_ntt(t, w.D, static_cast<size_t>(inputs) * L * Lp, Lp, false, s);
    if (err != hipSuccess) return err;
  }
  {
    // every key's uses split over enough workgroups for about 4 per CU
    const uint32_t blocks = grid_for(static_cast<size_t>(plan.key_period) * Lp * n / 4);
    const uint32_t uses = rotations / plan.key_period;
    const uint32_t want = (4 * t.num_cus + blocks - 1) / blocks;
    const uint32_t chunks = want < 1 ? 1 : (want > uses ? uses : want);
    const dim3 g(blocks * chunks);
    switch (L) {
      case 2: ks_inner_kernel<2><<<g, kThreads, 0, s>>>(t, w.D, ksk, L, rotations, plan, blocks, chunks, w.acc); break;
      case 3: ks_inner_kernel<3><<<g, kThreads, 0, s>>>(t, w.D, ksk, L, rotations, plan, blocks, chunks, w.acc); break;
      case 4: ks_inner_kernel<4><<<g, kThreads, 0, s>>>(t, w.D, ksk, L, rotations, plan, blocks, chunks, w.acc); break;
      default: ks_inner_kernel<0><<<g, kThreads, 0, s>>>(t, w.D, ksk, L, rotations, plan, blocks, chunks, w.acc); break;
    }
  }
  if ((err = hipGetLastError()) != hipSuccess || out == nullptr) return err;
  if (t.log_n <= 14) {
    const uint32_t copies = copy_inputs ? inputs : 0;
    const Seq cseq = copy_inputs ? *copy_inputs : contiguous();
    const dim3 grid(2 * (rotations + copies), L);
    switch (t.log_n) {
#define CKKS_MDC(LN)                                                                                       \
  case LN:                                                                                                 \
    moddown_combine_kernel<LN><<<grid, WholePlan<LN, true>::P::T, 0, s>>>(t, w.acc, ct, in_seq, L, rotations, \
                                                                          plan, out, out_seq, cseq);       \
    break;
      CKKS_MDC(10)
      CKKS_MDC(11)
      CKKS_MDC(12)
      CKKS_MDC(13)
      default: CKKS_MDC(14)
#undef CKKS_MDC
    }
    return hipGetLastError();
  }
  if (copy_inputs != nullptr) return hipErrorInvalidValue;   // the input copy rides on the fused form only
  err = launch_rescale(t, w.acc, w.tmp, rotations, Lp, w.rs, s);
  if (err != hipSuccess) return err;
  rot_combine_kernel<<<grid_for(static_cast<size_t>(rotations) * L * n / 4), kThreads, 0, s>>>(
      t, ct, in_seq, w.tmp, L, rotations, plan, out, out_seq);
  return hipGetLastError();
}

hipError_t launch_keygen_rotation(const Tables& t, const uint32_t* s_ntt, uint32_t r0, uint32_t r_step,
                                  uint32_t keys, const uint32_t* a, const int32_t* e, uint32_t* ksk,
                                  hipStream_t s) {
  if (keys == 0) return hipSuccess;
  const uint32_t L = t.L - 1, Lp = L + 1;
  const size_t n = t.n;
  keygen_err_kernel<<<grid_for(static_cast<size_t>(keys) * L * n / 4), kThreads, 0, s>>>(t, e, L, keys, ksk);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  // the b rows: logical row (key * L + digit) * Lp + j is physical row (.. / Lp) * 2 Lp + j
  err = launch_ntt(t, ksk, static_cast<size_t>(keys) * L * Lp, Lp, false, s, 2 * Lp);
  if (err != hipSuccess) return err;
  keygen_combine_kernel<<<grid_for(static_cast<size_t>(keys) * L * Lp * n / 4), kThreads, 0, s>>>(
      t, s_ntt, a, L, keys, r0, r_step, ksk);
  return hipGetLastError();
}

// Workspace of the BSGS product for `count` input ciphertexts: baby rotations
// [count][n1][2][L][N], inner sums [count][n2][2][L][N], the giant-step sum in
// the extended basis [count][2][L+1][N], and the largest of the two rotation
// workspaces and the two closing rescales'.
size_t bsgs_workspace_bytes(const Tables& t, uint32_t count, uint32_t n1, uint32_t n2) {
  const size_t ct = static_cast<size_t>(2) * (t.L - 1) * t.n * 4;
  const size_t fixed = ct * count * (static_cast<size_t>(n1) + n2) + static_cast<size_t>(2) * t.L * t.n * 4 * count;
  size_t scratch = rotate_workspace_bytes(t, count, count * (n1 - 1));
  const size_t rot2 = rotate_workspace_bytes(t, count * (n2 - 1), count * (n2 - 1));
  size_t rs = rescale_workspace_bytes(t, count, t.L);             // the ModDown of the sum
  const size_t rs2 = rescale_workspace_bytes(t, count, t.L - 1);  // the closing rescale
  rs = rs > rs2 ? rs : rs2;
  scratch = scratch > rot2 ? scratch : rot2;
  return fixed + (scratch > rs ? scratch : rs);
}

hipError_t launch_rotate(const Tables& t, const uint32_t* ct, uint32_t count, uint32_t r0, uint32_t r_step,
                         uint32_t galois, bool hoisted, const uint32_t* ksk, void* workspace, uint32_t* out,
                         hipStream_t s) {
  // hoisted: count rotations of one input; else rotation k of input k
  RotPlan plan{hoisted ? count : 1u, count, r0, r_step, galois};
  return launch_rotate_seq(t, ct, contiguous(), hoisted ? 1 : count, count, plan, ksk, workspace, out, contiguous(),
                           s, nullptr);
}

// y = sum_j rot( sum_i pt[j][i] (.) rot(x, i), j n1 ), rescaled, for each of
// `count` inputs.  pt [n2][n1][L][N]; ksk: n1 - 1 baby keys (steps 1 .. n1-1)
// then n2 - 1 giant keys (steps n1, 2 n1, ..); out [count][2][L-1][N].
hipError_t launch_bsgs(const Tables& t, const uint32_t* pt, const uint32_t* ct, uint32_t count, uint32_t n1,
                       uint32_t n2, const uint32_t* ksk, void* workspace, uint32_t* out, hipStream_t s) {
  if (count == 0) return hipSuccess;
  const uint32_t L = t.L - 1;
  const size_t n = t.n, ctw = 2 * L * n;
  const size_t key_words = static_cast<size_t>(L) * 2 * (L + 1) * n;
  uint32_t* baby = static_cast<uint32_t*>(workspace);
  uint32_t* inner = baby + static_cast<size_t>(count) * n1 * ctw;
  uint32_t* ext = inner + static_cast<size_t>(count) * n2 * ctw;
  void* rws = ext + static_cast<size_t>(count) * 2 * (L + 1) * n;
  // baby steps: element 0 of each input's group is the input itself, then its
  // rotations by 1 .. n1-1 (one ModUp per input).  Up to 2^14 the input's copy
  // into slot 0 rides on the rotations' ModDown launch; else it is a copy of its own.
  hipError_t err = hipSuccess;
  const bool copy_in_rotation = n1 > 1 && t.log_n <= 14;
  if (!copy_in_rotation) {
    err = hipMemcpy2DAsync(baby, n1 * ctw * 4, ct, ctw * 4, ctw * 4, count, hipMemcpyDeviceToDevice, s);
    if (err != hipSuccess) return err;
  }
  if (n1 > 1) {
    RotPlan plan{n1 - 1, n1 - 1, 1, 1, 0};
    const Seq slot0{1, n1, 0};
    err = launch_rotate_seq(t, ct, contiguous(), count, count * (n1 - 1), plan, ksk, rws, baby,
                            Seq{n1 - 1, n1, 1}, s, copy_in_rotation ? &slot0 : nullptr);
    if (err != hipSuccess) return err;
  }
  // inner sums: the full-polynomial MAC (one input), or the register-tiled
  // batched form
  if (count == 1) {
    err = launch_mac_poly(t, pt, baby, inner, n2, n1, L, s);
  } else {
    const size_t grid = static_cast<size_t>(L) * (n / kThreads) * ((n2 + kTileJ - 1) / kTileJ) *
                        ((count + kTileB - 1) / kTileB);
    bsgs_mac_tile_kernel<<<static_cast<uint32_t>(grid), kThreads, 0, s>>>(t, pt, baby, count, n1, n2, L, inner);
    err = hipGetLastError();
  }
  if (err != hipSuccess) return err;
  if (n2 == 1) return launch_rescale(t, inner, out, count, L, rws, s);
  // giant steps: inner sum j >= 1 of every input rotated by j n1, up to the
  // key-switching inner product; the terms summed in the extended basis; its
  // ModDown and the product's rescale in one launch (at 2^16 two, through the
  // baby region, free after the MAC)
  RotPlan plan{1, n2 - 1, n1, n1, 0};
  err = launch_rotate_seq(t, inner, Seq{n2 - 1, n2, 1}, count * (n2 - 1), count * (n2 - 1), plan,
                          ksk + static_cast<size_t>(n1 - 1) * key_words, rws, nullptr, contiguous(), s, nullptr);
  if (err != hipSuccess) return err;
  const uint32_t* acc = rot_layout(t, count * (n2 - 1), count * (n2 - 1), rws).acc;
  giant_ext_kernel<<<static_cast<uint32_t>(count * 2 * (L + 1) * n / 64), kThreads, 0, s>>>(
      t, inner, acc, L, count, n2, galois_of(n1, t.log_n), ext);
  if ((err = hipGetLastError()) != hipSuccess) return err;
  return launch_rescale2(t, ext, baby, out, count, L + 1, rws, s);
}

}  // namespace ckks
