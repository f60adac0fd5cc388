// Register-group negacyclic NTT building blocks for gfx950.
//
// Transform (ring of section 2.1, NTT form as declared in ckks_linear.h):
// merged-twiddle Cooley-Tukey (forward) and Gentleman-Sande (inverse), stage
// s = 0..log N - 1 pairing index bits b = log N - 1 - s, twiddle index
// 2^s + (x >> (b + 1)) into the bit-reversed power tables.
//
// A transform (or a 2^LOGB-point block of one) is split into groups of LOGE
// consecutive index bits.  For one group a thread owns E = 2^LOGE residues
// whose indices differ only in the group's window of bits, and runs all the
// group's stages in registers (a radix-E butterfly network).  Butterflies are
// lazy (Harvey): forward values stay in [0, 4q) and inverse values in [0, 2q)
// (4q < 2^32 for q < 2^30), and a block normalises to [0, q) when it ends; a
// forward group run on its own (the N = 2^16 column pass) leaves [0, 4q),
// which the next forward stage accepts.  Between groups
// the residues are exchanged through LDS, padded by one word per 32 so that
// power-of-two strides spread across banks.  Group 0 covers the top bits, so
// its window is a stride-T pattern (coalesced HBM access) and the last group's
// window is contiguous per thread.
#pragma once

#include "ckks_internal.hpp"

namespace ckks {

__device__ __forceinline__ uint32_t lds_pad(uint32_t x) { return x + (x >> 5); }

template <int LOGB, int LOGE>
struct Plan {
  static constexpr int B = 1 << LOGB;
  static constexpr int LOGT = LOGB - LOGE;
  static constexpr int T = 1 << LOGT;
  static constexpr int E = 1 << LOGE;
  static constexpr int NG = (LOGB + LOGE - 1) / LOGE;
  static constexpr int lds_words = B + (B >> 5);
  static constexpr int hi(int g) { return LOGB - 1 - g * LOGE; }
  static constexpr int lo(int g) { return LOGB - (g + 1) * LOGE > 0 ? LOGB - (g + 1) * LOGE : 0; }
  // Index (within the block) of element j of thread t in group g's layout.
  template <int G>
  static __device__ __forceinline__ uint32_t pos(uint32_t t, uint32_t j) {
    constexpr int w = lo(G);
    return (t & ((1u << w) - 1u)) | (j << w) | ((t >> w) << (w + LOGE));
  }
};

// Forward stages of group G (bits hi..lo, descending).  LOGN is the full
// transform size (for the stage number); blk is the block index above the
// block's LOGB bits (0 for a whole-polynomial block).
template <int LOGN, int LOGB, int LOGE, int G>
__device__ __forceinline__ void fwd_group(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t blk,
                                          const uint32_t* __restrict__ tw,
                                          const uint32_t* __restrict__ tws, uint32_t q) {
  using P = Plan<LOGB, LOGE>;
  constexpr int w = P::lo(G);
  const uint32_t q2 = 2 * q;
#pragma unroll
  for (int b = P::hi(G); b >= P::lo(G); --b) {
    const int s = LOGN - 1 - b;
    const int lb = b - w;
    // In group 0 a thread id below 2^w has t >> w = 0: the twiddles are then
    // workgroup-uniform (scalar loads).
    const uint32_t base = (1u << s) + (blk << (LOGB - 1 - b)) +
                          (w >= P::LOGT ? 0u : ((t >> w) << (w + LOGE - b - 1)));
#pragma unroll
    for (int u = 0; u < (P::E >> (lb + 1)); ++u) {
      const uint32_t idx = base + u;
      const uint32_t wv = tw[idx], wsv = tws[idx];
#pragma unroll
      for (int low = 0; low < (1 << lb); ++low) {
        const int j0 = (u << (lb + 1)) | low;
        const int j1 = j0 | (1 << lb);
        uint32_t U = v[j0];
        U = min(U, U - q2);                               // [0, 2q)
        // The lazy Shoup product V = a w - floor(a ws / 2^32) q lies in [0, 2q);
        // formed negated (Vn = 2^32 - V), the two outputs take one subtraction
        // and one three-input addition.
        const uint32_t a = v[j1];
        const uint32_t Vn = __umulhi(a, wsv) * q - a * wv;
        v[j0] = U - Vn;                                   // U + V in [0, 4q)
        v[j1] = U + Vn + q2;                              // U - V + 2q in (0, 4q)
      }
    }
  }
}

// Inverse stages of group G (bits lo..hi, ascending).
template <int LOGN, int LOGB, int LOGE, int G>
__device__ __forceinline__ void inv_group(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t blk,
                                          const uint32_t* __restrict__ tw,
                                          const uint32_t* __restrict__ tws, uint32_t q) {
  using P = Plan<LOGB, LOGE>;
  constexpr int w = P::lo(G);
  const uint32_t q2 = 2 * q;
#pragma unroll
  for (int b = P::lo(G); b <= P::hi(G); ++b) {
    const int s = LOGN - 1 - b;
    const int lb = b - w;
    // In group 0 a thread id below 2^w has t >> w = 0: the twiddles are then
    // workgroup-uniform (scalar loads).
    const uint32_t base = (1u << s) + (blk << (LOGB - 1 - b)) +
                          (w >= P::LOGT ? 0u : ((t >> w) << (w + LOGE - b - 1)));
#pragma unroll
    for (int u = 0; u < (P::E >> (lb + 1)); ++u) {
      const uint32_t idx = base + u;
      const uint32_t wv = tw[idx], wsv = tws[idx];
#pragma unroll
      for (int low = 0; low < (1 << lb); ++low) {
        const int j0 = (u << (lb + 1)) | low;
        const int j1 = j0 | (1 << lb);
        const uint32_t U = v[j0], V = v[j1];
        const uint32_t S = U + V;                         // [0, 4q)
        v[j0] = min(S, S - q2);                           // [0, 2q)
        v[j1] = mul_shoup_lazy(U - V + q2, wv, wsv, q);   // [0, 2q)
      }
    }
  }
}

// Move the thread's residues from group GF's layout to group GT's through LDS.
// When both groups keep at most 6 low index bits in the thread id (lo(g) <= 6),
// the 64 threads of a wave hold the same index set in both layouts (all
// indices whose bits from LOGE + 6 up equal the wave number), so the exchange
// stays inside the wave's own LDS region: no workgroup barrier, only the
// wave's in-order LDS accesses (wave_barrier keeps the compiler from moving
// them).  Any other exchange is workgroup-wide and synchronises; it also
// orders every earlier wave-local access before its writes.
template <int LOGB, int LOGE, int GF, int GT>
__device__ __forceinline__ void exchange(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t* lds) {
  using P = Plan<LOGB, LOGE>;
  constexpr bool wave_local = P::lo(GF) <= 6 && P::lo(GT) <= 6;
  if constexpr (wave_local) {
    __builtin_amdgcn_wave_barrier();
  } else {
    __syncthreads();  // earlier readers of lds are done
  }
  // t's bits and j's bits of a position are disjoint, so the padded position
  // splits into a per-thread base and a compile-time offset per j.
  uint32_t* wb = lds + lds_pad(P::template pos<GF>(t, 0));
#pragma unroll
  for (int j = 0; j < P::E; ++j) wb[lds_pad(P::template pos<GF>(0, j))] = v[j];
  if constexpr (wave_local) {
    __builtin_amdgcn_wave_barrier();
  } else {
    __syncthreads();
  }
  const uint32_t* rb = lds + lds_pad(P::template pos<GT>(t, 0));
#pragma unroll
  for (int j = 0; j < P::E; ++j) v[j] = rb[lds_pad(P::template pos<GT>(0, j))];
}

// Wave-coalesced layout: element j of lane i of wave a is index
// a 2^(LOGE+6) + 64 j + i, so a load or store of element j by a wave touches
// 64 consecutive words.  Each wave holds the same index set in it as in the
// last group's layout (index t 2^LOGE + j; all indices whose bits from
// LOGE + 6 up equal a), so the two convert through the wave's own LDS region
// without a workgroup barrier.  Needs T >= 64 (every plan here).
template <int LOGE>
__device__ __forceinline__ uint32_t pos_coalesced(uint32_t t, uint32_t j) {
  return ((t >> 6) << (LOGE + 6)) + (j << 6) + (t & 63);
}

template <int LOGB, int LOGE, bool TO_LAST>
__device__ __forceinline__ void wave_relayout(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t* lds) {
  using P = Plan<LOGB, LOGE>;
  static_assert(P::T >= 64 && P::lo(P::NG - 1) == 0, "whole waves; last group keeps no thread bits low");
  // t's bits and j's bits of either position are disjoint: base + constant.
  uint32_t* cb = lds + lds_pad(pos_coalesced<LOGE>(t, 0));
  uint32_t* lb = lds + lds_pad(P::template pos<P::NG - 1>(t, 0));
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    if constexpr (TO_LAST) cb[lds_pad(j << 6)] = v[j];
    else lb[lds_pad(P::template pos<P::NG - 1>(0, j))] = v[j];
  }
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int j = 0; j < P::E; ++j) {
    if constexpr (TO_LAST) v[j] = lb[lds_pad(P::template pos<P::NG - 1>(0, j))];
    else v[j] = cb[lds_pad(j << 6)];
  }
  __builtin_amdgcn_wave_barrier();
}

// Forward transform of one block held in registers in group-0 layout; on
// return the registers hold group NG-1 layout, in [0, q) (kNorm) or left in
// the lazy range [0, 4q) for a consumer that reduces anyway.
template <int LOGN, int LOGB, int LOGE, int G = 0, bool kNorm = true>
__device__ __forceinline__ void fwd_block(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t blk,
                                          const uint32_t* __restrict__ tw,
                                          const uint32_t* __restrict__ tws, uint32_t q,
                                          uint32_t* lds) {
  using P = Plan<LOGB, LOGE>;
  if constexpr (G > 0) exchange<LOGB, LOGE, G - 1, G>(v, t, lds);
  fwd_group<LOGN, LOGB, LOGE, G>(v, t, blk, tw, tws, q);
  if constexpr (G + 1 < P::NG) {
    fwd_block<LOGN, LOGB, LOGE, G + 1, kNorm>(v, t, blk, tw, tws, q, lds);
  } else if constexpr (kNorm) {
#pragma unroll
    for (int j = 0; j < P::E; ++j) {  // [0, 4q) -> [0, q)
      uint32_t x = min(v[j], v[j] - 2 * q);
      v[j] = min(x, x - q);
    }
  }
}

// (c - v) w mod q in [0, q) for c in [0, q) and a lazy forward output v in
// [0, 4q), w < q with its Shoup companion ws: v mod 2q, then c + 2q - v in
// (0, 3q) < 2^32 through the lazy Shoup product and one conditional
// subtraction (10 operations against 14 with v normalised first).
__device__ __forceinline__ uint32_t sub_lazy_mul_shoup(uint32_t c, uint32_t v, uint32_t w, uint32_t ws,
                                                       uint32_t q) {
  const uint32_t r = min(v, v - 2 * q);
  const uint32_t y = mul_shoup_lazy(c + 2 * q - r, w, ws, q);
  return min(y, y - q);
}

// Inverse transform (without the N^-1 factor) of one block held in group
// NG-1 layout; on return the registers hold group-0 layout.
template <int LOGN, int LOGB, int LOGE, int G = Plan<LOGB, LOGE>::NG - 1>
__device__ __forceinline__ void inv_block(uint32_t (&v)[1 << LOGE], uint32_t t, uint32_t blk,
                                          const uint32_t* __restrict__ tw,
                                          const uint32_t* __restrict__ tws, uint32_t q,
                                          uint32_t* lds) {
  using P = Plan<LOGB, LOGE>;
  if constexpr (G < P::NG - 1) exchange<LOGB, LOGE, G + 1, G>(v, t, lds);
  inv_group<LOGN, LOGB, LOGE, G>(v, t, blk, tw, tws, q);
  if constexpr (G > 0) {
    inv_block<LOGN, LOGB, LOGE, G - 1>(v, t, blk, tw, tws, q, lds);
  } else {
#pragma unroll
    for (int j = 0; j < P::E; ++j) v[j] = min(v[j], v[j] - q);  // [0, 2q) -> [0, q)
  }
}

// Per-N choice of residues per thread for whole-polynomial blocks.  Kernels
// over whole polynomials ask for 4 waves per SIMD (a 128-register budget):
// two 2^14 workgroups, or one 2^15 workgroup, fill a CU's LDS.  The latency
// form (LAT) is for launches with fewer workgroups than CUs, where each
// transform has a CU to itself: 16 residues per thread at 2^13 and 2^14, so
// twice the lanes share each transform's chain.
template <int LOGN, bool LAT = false>
struct WholePlan {
  static constexpr int LOGE = (LOGN <= 12 || (LAT && LOGN <= 14)) ? 4 : 5;
  using P = Plan<LOGN, LOGE>;
  static constexpr int kWavesPerSimd = 4;
};

}  // namespace ckks
