// Scalar-weight ct x pt MAC on the gfx950 matrix cores, exact, via int8 digit
// splitting.
//
// Per limb l the MAC is the modular GEMM  C = A . B mod q  with A the weights
// (d_out x d_in) and B the ciphertext residues (d_in x 2N).  Both operands are
// written in balanced base-256 digits that fit int8:
//   B: x in [0, 2^30)          x = sum_b d_b 256^b,  b < 4  (d_3 in [0, 64])
//   A: v = centred w in (-q/2, q/2]   v = sum_a e_a 256^a,  a < 4 (e_3 = 0 when
//      -0x808080 <= v <= 0x7f7f7f, which holds for CKKS-scaled weights)
// using (u + 0x80808080) ^ 0x80808080, whose bytes read as int8 are the digits.
// Then  sum_i v_i x_i = sum_s 256^s S_s,  S_s = sum_{a+b=s} sum_i e_a(i) d_b(i),
// where each S_s is an exact i32 contraction on v_mfma_i32_16x16x64_i8
// (|S_s| <= 4 * d_in * 2^14 <= 2^28 for d_in <= 4096).  The epilogue folds the
// classes exactly in signed 64-bit integers, with 256^s mod q for s >= 4, and
// reduces the sum mod q through one fp64 quotient estimate.
// Digit products: 12 per modular MAC with 3 weight digits, 16 with 4.
//
// A prep kernel lays the weights out as MFMA fragments (16 bytes per lane, the
// lane order of v_mfma_i32_16x16x64_i8) per 16-row tile and 64-deep k-step,
// with a flag for tiles that need a fourth digit.
//
// Every wave owns 32 rows x 32 columns of one limb (2 x 2 MFMA tiles x 6 or
// 7 shift-class accumulators) and reads its weight fragments from global
// memory (L2 resident, one k-step ahead).  Two contraction forms:
//  * column-stationary (d_in <= 1024): a 512-thread workgroup owns 32 columns
//    and converts all of their residues once into digit fragments for every
//    k-step, held in LDS (<= 128 KiB, one workgroup per CU); its 8 waves then
//    walk the row tiles with no further synchronisation.  Each residue is
//    loaded and converted once per call.
//  * streamed (1024 < d_in <= 4096): a 256-thread workgroup computes a 128 x
//    32 tile; per k-step it converts the residues of its 32 columns (loads
//    issued two steps ahead) into an LDS double buffer and synchronises, two
//    workgroups per CU; XCD-aware grouped order keeps a row group's weights
//    and the columns its row tiles share in one XCD's L2.
// In both, rows past d_in read as zero through the buffer range check, and a
// wave-uniform branch per tile selects three or four weight digits.
#include <mutex>

#include "ckks_internal.hpp"

// Workspace of the no-allocation MAC entry point: one array per GPU, owned by
// the library for the life of the process.  Its name is a host-side stand-in;
// kernels receive the device address that hipGetSymbolAddress returns for the
// current device (see noalloc_scratch below).
static __device__ __align__(256) unsigned char scratch[ckks::kNoAllocScratchBytes];

namespace ckks {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBM = 128;       // rows per workgroup tile
constexpr int kBN = 32;        // columns per workgroup tile
constexpr int kBK = 64;        // K per MFMA step
constexpr int kMT = 2;         // 16-row MFMA tiles per wave
constexpr int kNT = kBN / 16;  // 16-column MFMA tiles per wave
constexpr int kFragsPerStep = kNT * 4 * 64;  // 16-byte ciphertext fragments per k-step
constexpr int kGroupM = 8;                   // row tiles per L2-resident weight group
constexpr uint32_t kBias = 0x80808080u;
constexpr uint32_t kMaxDin = 4096;
constexpr int kRsrcWord3 = 0x00020000;  // buffer resource word 3: 32-bit raw data, range-checked
typedef __amdgpu_buffer_rsrc_t rsrc_t;


// o[b] byte e = p[e] byte b (4x4 byte transpose, eight v_perm_b32).
// __builtin_amdgcn_perm(hi, lo, sel): selector byte values 0-3 pick bytes of
// lo, 4-7 bytes of hi.
__device__ __forceinline__ void transpose4(uint32_t p0, uint32_t p1, uint32_t p2, uint32_t p3,
                                           uint32_t (&o)[4]) {
  const uint32_t x01l = __builtin_amdgcn_perm(p1, p0, 0x05010400u);  // p0.0 p1.0 p0.1 p1.1
  const uint32_t x01h = __builtin_amdgcn_perm(p1, p0, 0x07030602u);  // p0.2 p1.2 p0.3 p1.3
  const uint32_t x23l = __builtin_amdgcn_perm(p3, p2, 0x05010400u);
  const uint32_t x23h = __builtin_amdgcn_perm(p3, p2, 0x07030602u);
  o[0] = __builtin_amdgcn_perm(x23l, x01l, 0x05040100u);            // p0.0 p1.0 p2.0 p3.0
  o[1] = __builtin_amdgcn_perm(x23l, x01l, 0x07060302u);            // p0.1 p1.1 p2.1 p3.1
  o[2] = __builtin_amdgcn_perm(x23h, x01h, 0x05040100u);
  o[3] = __builtin_amdgcn_perm(x23h, x01h, 0x07060302u);
}

// 16 residues (consecutive k) -> one 16-byte digit fragment per digit b:
// byte i of fragment b is digit b of residue i.  The bias is added before
// the byte transpose and removed after it (both are bytewise).
__device__ __forceinline__ void to_fragments(const uint32_t (&x)[16], v4i (&f)[4]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    uint32_t o[4];
    transpose4(x[4 * g] + kBias, x[4 * g + 1] + kBias, x[4 * g + 2] + kBias, x[4 * g + 3] + kBias, o);
#pragma unroll
    for (int b = 0; b < 4; ++b) f[b][g] = static_cast<int>(o[b] ^ kBias);
  }
}

// Weight digits: adig[((l * mt_total + mt) * ks_total + ks) * 4 + a][lane] holds
// e_a(w[mt*16 + lane%16][ks*64 + (lane/16)*16 + i]) in byte i (zero-padded);
// flags[l * mt_total + mt] != 0 when any e_3 of that 16-row tile is non-zero.
// One workgroup per (tile, limb).  The limbs of a weight are adjacent in w_enc,
// so the workgroups of one tile read the same cache lines: their logical ids
// are consecutive and each XCD runs a contiguous range of them, so a tile's
// rows come from HBM once into that XCD's L2 (with the limb as the slow grid
// dimension every line was fetched about once per limb).
__global__ __launch_bounds__(kThreads) void mfma_prep_kernel(
    const uint32_t* __restrict__ qtab, const uint32_t* __restrict__ w_enc, uint32_t d_out,
    uint32_t d_in, uint32_t limbs, uint32_t mt_total, uint32_t ks_total, v4i* __restrict__ adig,
    uint32_t* __restrict__ flags) {
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const uint32_t mt = lid / limbs, l = lid - mt * limbs;
  const uint32_t q = qtab[l];
  uint32_t top = 0;
  for (uint32_t idx = threadIdx.x; idx < ks_total * 64; idx += kThreads) {
    const uint32_t ks = idx >> 6, lane = idx & 63;
    const uint32_t row = mt * 16 + (lane & 15);
    const uint32_t k0 = ks * kBK + (lane >> 4) * 16;
    uint32_t p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t k = k0 + i;
      uint32_t w = 0;
      if (row < d_out && k < d_in) w = w_enc[(static_cast<size_t>(row) * d_in + k) * limbs + l];
      p[i] = w > (q >> 1) ? w - q : w;  // centred, two's complement
    }
    v4i f[4];
    to_fragments(p, f);
    const size_t base = ((static_cast<size_t>(l) * mt_total + mt) * ks_total + ks) * 4;
#pragma unroll
    for (int a = 0; a < 4; ++a) adig[(base + a) * 64 + lane] = f[a];
    top |= static_cast<uint32_t>(f[3][0] | f[3][1] | f[3][2] | f[3][3]);
  }
  const int any = __syncthreads_or(top != 0);
  if (threadIdx.x == 0) flags[l * mt_total + mt] = any ? 1u : 0u;
}

// K loop.  The workgroup converts each 64-deep k-step of its 32 ciphertext
// columns into digit fragments in LDS (thread: one column, 8 consecutive k);
// the other workgroup resident on the CU runs its contractions meanwhile.
// Step ks: issue the residue loads of step ks+2 (register set ks%2) and the
// weight fragments of step ks+1; contract step ks out of LDS buffer ks%2;
// convert the residues of step ks+1 (issued two steps earlier) into LDS
// buffer (ks+1)%2; synchronise once.
template <int NDA>
__device__ __forceinline__ void mac_loop(const v4i* __restrict__ adig_wave, uint32_t ks_total,
                                         const uint32_t* __restrict__ bsrc, uint32_t row_bytes,
                                         uint32_t d_in, v4i (*bs)[kFragsPerStep],
                                         v4i (&acc)[kMT][kNT][NDA + 3]) {
  const uint32_t tid = threadIdx.x;
  const uint32_t lane = tid & 63;
  const uint32_t col = tid % kBN;       // staging: column of the tile
  const uint32_t kg = tid / kBN;        // staging: 8-k group within the step (0..7)
  uint32_t raw[2][8];
  v4i af[2][kMT][NDA];
  // LDS byte offset of this thread's 8 bytes of digit-b fragment: fragment
  // (nt, b), MFMA lane col%16 + 16*(kg/2), bytes 8*(kg%2)..+8.
  const uint32_t frag_lane = (col & 15) + 16 * (kg >> 1);
  const uint32_t nt_s = col >> 4;
  const uint32_t half = kg & 1;
  uint32_t voff[8];  // byte offset of (row kg*8+i, this column) from the step's first row
#pragma unroll
  for (int i = 0; i < 8; ++i) voff[i] = (kg * 8 + i) * row_bytes + col * 4;
  const uint32_t row_words = row_bytes >> 2;

  // Rows at or past d_in fall outside the step's buffer range and read as 0.
  auto load_b = [&](uint32_t (&r)[8], uint32_t ks) {
    const uint32_t rows = d_in - ks * kBK < kBK ? d_in - ks * kBK : kBK;
    const rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint32_t*>(bsrc) + static_cast<size_t>(ks) * kBK * row_words, 0, rows * row_bytes, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, voff[i], 0, 0);
  };
  auto store_b = [&](const uint32_t (&r)[8], int buf) {
    uint32_t lo[4], hi[4];
    transpose4(r[0] + kBias, r[1] + kBias, r[2] + kBias, r[3] + kBias, lo);
    transpose4(r[4] + kBias, r[5] + kBias, r[6] + kBias, r[7] + kBias, hi);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      uint2* dst = reinterpret_cast<uint2*>(&bs[buf][(nt_s * 4 + b) * 64 + frag_lane]) + half;
      *dst = make_uint2(lo[b] ^ kBias, hi[b] ^ kBias);
    }
  };
  const rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<v4i*>(adig_wave), 0,
                                                      kMT * ks_total * 4 * 64 * 16, kRsrcWord3);
  auto load_a = [&](v4i (&a)[kMT][NDA], uint32_t ks) {
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
      for (int d = 0; d < NDA; ++d)
        a[mt][d] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(ra, lane * 16, ((mt * ks_total + ks) * 4 + d) * 1024, 0);
  };
  auto step = [&](uint32_t ks, uint32_t (&r_issue)[8], const uint32_t (&r_store)[8], v4i (&a_cur)[kMT][NDA],
                  v4i (&a_nxt)[kMT][NDA]) {
    const int buf = ks & 1;
    load_b(r_issue, ks + 2 < ks_total ? ks + 2 : ks_total - 1);
    load_a(a_nxt, ks + 1 < ks_total ? ks + 1 : ks_total - 1);
    __builtin_amdgcn_sched_barrier(0);  // keep the prefetches ahead of the contractions
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      v4i bf[kNT];
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) bf[nt] = bs[buf][(nt * 4 + b) * 64 + lane];
      // within one digit b the NDA * kMT * kNT contractions hit distinct accumulators
#pragma unroll
      for (int d = 0; d < NDA; ++d)
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
          for (int nt = 0; nt < kNT; ++nt)
            acc[mt][nt][d + b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a_cur[mt][d], bf[nt], acc[mt][nt][d + b], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    store_b(r_store, buf ^ 1);
    __syncthreads();
  };

  load_b(raw[0], 0);
  load_b(raw[1], ks_total > 1 ? 1 : 0);
  load_a(af[0], 0);
  store_b(raw[0], 0);
  __syncthreads();
  uint32_t ks = 0;
  for (; ks + 1 < ks_total; ks += 2) {
    step(ks, raw[0], raw[1], af[0], af[1]);      // issues ks+2 into set 0, converts ks+1 from set 1
    step(ks + 1, raw[1], raw[0], af[1], af[0]);  // issues ks+3 into set 1, converts ks+2 from set 0
  }
  if (ks < ks_total) step(ks, raw[0], raw[1], af[0], af[1]);
}

// out = sum_s S_s 256^s mod q, exactly.  T = sum_{s<4} S_s 2^(8s) +
// sum_{s>=4} S_s (256^s mod q) is an exact signed 64-bit sum (|T| < 2^59.7 for
// |S_s| <= 2^28 and q < 2^30).  The quotient estimate floor(T / q) from fp64
// (T rounded once, then times 1/q) is within one of the true quotient and below
// 2^31 in magnitude (q > 2^29), so r = T - qt q lies in [-q, 2q) and its low 32
// bits are exact; r + q in [0, 3q) then takes two conditional subtractions.
template <int NDA>
__device__ __forceinline__ void epilogue(const v4i (&acc)[kMT][kNT][NDA + 3], const Tables& tb, uint32_t l,
                                         uint32_t lane, const rsrc_t& out, uint32_t row_bytes) {
  const uint32_t q = tb.q[l];
  const double qr = tb.q_recip[l];
  const uint32_t* pw = tb.pow256 + l * 8;
  // 256^s mod q as signed multipliers (2^(8s) itself for s < 4, since 2^24 < q)
  int32_t cs[NDA + 3];
#pragma unroll
  for (int s = 1; s < NDA + 3; ++s) cs[s] = static_cast<int32_t>(pw[s]);
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      // output row mt*16 + 4*(lane/16) + r of the wave; rows past d_out are out of range
      const uint32_t voff = (mt * 16 + 4 * (lane >> 4) + r) * row_bytes + (lane & 15) * 4;
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) {
        const v4i* a = acc[mt][nt];
        int64_t t = a[0][r];
#pragma unroll
        for (int s = 1; s < NDA + 3; ++s) t += static_cast<int64_t>(a[s][r]) * static_cast<int64_t>(cs[s]);
        const double tf = static_cast<double>(t);
        const int32_t qt = static_cast<int32_t>(floor(tf * qr));
        uint32_t u = static_cast<uint32_t>(t) - static_cast<uint32_t>(qt) * q + q;  // r + q, in [0, 3q)
        u = min(u, u - q);
        u = min(u, u - q);
        __builtin_amdgcn_raw_buffer_store_b32(u, out, voff, nt * 64, 0);
      }
    }
  }
}

// One workgroup-uniform branch per row tile: tiles whose weights need a fourth
// digit (flag set) take the NDA = 4 contraction, the others NDA = 3.
template <int NDA>
__device__ __forceinline__ void mac_tile(const Tables& tb, const v4i* __restrict__ adig_wave, uint32_t ks_total,
                                         const uint32_t* __restrict__ bsrc, uint32_t row_bytes, uint32_t d_in,
                                         v4i (*bs)[kFragsPerStep], const rsrc_t& out, uint32_t l, uint32_t lane) {
  v4i acc[kMT][kNT][NDA + 3];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
      for (int s = 0; s < NDA + 3; ++s) acc[mt][nt][s] = v4i{0, 0, 0, 0};
  mac_loop<NDA>(adig_wave, ks_total, bsrc, row_bytes, d_in, bs, acc);
  epilogue<NDA>(acc, tb, l, lane, out, row_bytes);
}

__global__ __launch_bounds__(kThreads, 2) void mac_mfma_kernel(
    Tables tb, const v4i* __restrict__ adig, const uint32_t* __restrict__ flags,
    const uint32_t* __restrict__ ct_in, uint32_t* __restrict__ ct_out, uint32_t d_out, uint32_t d_in,
    uint32_t limbs, uint32_t mt_total, uint32_t ks_total, uint32_t tiles_m, uint32_t tiles_n) {
  __shared__ v4i bs[2][kFragsPerStep];  // ciphertext digit fragments of one k-step, double buffered

  // Tile order: consecutive workgroup ids alternate XCDs, so each XCD is given a
  // contiguous range of logical tiles.  Logical order: limb, then groups of up
  // to kGroupM row tiles (their weight digits, <= 1024 x d_in x 4 bytes, stay in
  // the XCD's L2), then column tile, then row tile within the group.
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const uint32_t per_limb = tiles_m * tiles_n;
  const uint32_t l = lid / per_limb;
  uint32_t rem = lid - l * per_limb;
  const uint32_t grp = rem / (kGroupM * tiles_n);           // full groups first
  const uint32_t g0 = grp * kGroupM;
  const uint32_t gsize = tiles_m - g0 < kGroupM ? tiles_m - g0 : kGroupM;
  rem -= g0 * tiles_n;
  const uint32_t ntile = rem / gsize;
  const uint32_t mtile = g0 + rem % gsize;

  uint32_t top = 0;
#pragma unroll
  for (int i = 0; i < kBM / 16; ++i) top |= flags[l * mt_total + mtile * (kBM / 16) + i];

  const uint32_t n = tb.n;
  const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const uint32_t col0 = ntile * kBN;  // column in [0, 2N): component c = col0 / N
  const uint32_t c = col0 >> tb.log_n, k0 = col0 & (n - 1);
  const uint32_t row_bytes = 2u * limbs * n * 4u;  // one ciphertext, input and output alike
  const uint32_t* bsrc = ct_in + (static_cast<size_t>(c) * limbs + l) * n + k0;
  const uint32_t mt_wave = mtile * (kBM / 16) + wave * kMT;
  const v4i* adig_wave = adig + (static_cast<size_t>(l) * mt_total + mt_wave) * ks_total * 4 * 64;
  const uint32_t row0 = mt_wave * 16;
  const uint32_t rows = row0 < d_out ? (d_out - row0 < kMT * 16 ? d_out - row0 : kMT * 16) : 0;
  uint32_t* dst = ct_out + ((static_cast<size_t>(row0) * 2 + c) * limbs + l) * n + k0;
  const rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(dst, 0, rows * row_bytes, kRsrcWord3);
  if (top != 0)
    mac_tile<4>(tb, adig_wave, ks_total, bsrc, row_bytes, d_in, bs, out, l, lane);
  else
    mac_tile<3>(tb, adig_wave, ks_total, bsrc, row_bytes, d_in, bs, out, l, lane);
}

// Column-stationary contraction (d_in <= kCsMaxDin).  The workgroup converts
// the residues of its 32 columns for every k-step into LDS, synchronises once,
// and its 8 waves walk the 32-row wave tiles (wave w takes tiles w, w + 8,
// ...; at any time the workgroup covers 256 adjacent rows, so workgroups on one
// XCD moving through the rows together share their weight fragments in L2).
// Converting the whole column strip once replaces the streamed form's per-tile
// reload, conversion and per-k-step barrier (1024 -> 6144 at N = 2^16 with 8
// limbs: 65-68 ms per call against 82-85 ms, bit-identical).
constexpr uint32_t kCsMaxDin = 1024;
constexpr int kCsMaxKs = kCsMaxDin / kBK;
constexpr int kCsThreads = 512;
constexpr int kCsWaves = kCsThreads / 64;

template <int NDA>
__device__ __forceinline__ void cs_loop(const v4i* __restrict__ adig_wave, uint32_t ks_total,
                                        const v4i (*bs)[kFragsPerStep], v4i (&acc)[kMT][kNT][NDA + 3],
                                        uint32_t lane) {
  const rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(const_cast<v4i*>(adig_wave), 0,
                                                      kMT * ks_total * 4 * 64 * 16, kRsrcWord3);
  v4i af[2][kMT][NDA];
  auto load_a = [&](v4i (&a)[kMT][NDA], uint32_t ks) {
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
      for (int d = 0; d < NDA; ++d)
        a[mt][d] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(ra, lane * 16, ((mt * ks_total + ks) * 4 + d) * 1024, 0);
  };
  auto step = [&](uint32_t ks, v4i (&a_cur)[kMT][NDA], v4i (&a_nxt)[kMT][NDA]) {
    load_a(a_nxt, ks + 1 < ks_total ? ks + 1 : ks_total - 1);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      v4i bf[kNT];
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) bf[nt] = bs[ks][(nt * 4 + b) * 64 + lane];
#pragma unroll
      for (int d = 0; d < NDA; ++d)
#pragma unroll
        for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
          for (int nt = 0; nt < kNT; ++nt)
            acc[mt][nt][d + b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a_cur[mt][d], bf[nt], acc[mt][nt][d + b], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  load_a(af[0], 0);
  uint32_t ks = 0;
  for (; ks + 1 < ks_total; ks += 2) {
    step(ks, af[0], af[1]);
    step(ks + 1, af[1], af[0]);
  }
  if (ks < ks_total) step(ks, af[0], af[1]);
}

template <int NDA>
__device__ __forceinline__ void cs_tile(const Tables& tb, const v4i* __restrict__ adig_wave, uint32_t ks_total,
                                        const v4i (*bs)[kFragsPerStep], const rsrc_t& out, uint32_t l, uint32_t lane,
                                        uint32_t row_bytes) {
  v4i acc[kMT][kNT][NDA + 3];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
      for (int s = 0; s < NDA + 3; ++s) acc[mt][nt][s] = v4i{0, 0, 0, 0};
  cs_loop<NDA>(adig_wave, ks_total, bs, acc, lane);
  epilogue<NDA>(acc, tb, l, lane, out, row_bytes);
}

__global__ __launch_bounds__(kCsThreads, 1) void mac_cs_kernel(
    Tables tb, const v4i* __restrict__ adig, const uint32_t* __restrict__ flags,
    const uint32_t* __restrict__ ct_in, uint32_t* __restrict__ ct_out, uint32_t d_out, uint32_t d_in,
    uint32_t limbs, uint32_t mt_total, uint32_t ks_total, uint32_t tiles_n) {
  __shared__ v4i bs[kCsMaxKs][kFragsPerStep];  // residue digit fragments of every k-step (128 KiB)
  // Consecutive workgroup ids alternate XCDs: each XCD takes a contiguous range
  // of (limb, column tile), so the workgroups resident on one XCD share a limb's
  // weight fragments in its L2.
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const uint32_t l = lid / tiles_n, ntile = lid - l * tiles_n;
  const uint32_t n = tb.n;
  const uint32_t col0 = ntile * kBN;  // column in [0, 2N): component c = col0 / N
  const uint32_t c = col0 >> tb.log_n, k0 = col0 & (n - 1);
  const uint32_t row_bytes = 2u * limbs * n * 4u;
  const uint32_t* bsrc = ct_in + (static_cast<size_t>(c) * limbs + l) * n + k0;
  const uint32_t row_words = row_bytes >> 2;
  const uint32_t tid = threadIdx.x;

  // Fill: thread (half h, k group kg, column col) converts 8 consecutive k of
  // one column for every k-step ks = h, h + 2, ...; all loads are issued first.
  {
    const uint32_t col = tid % kBN, kg = (tid / kBN) & 7, h = tid / 256;  // h is wave-uniform
    const uint32_t frag_lane = (col & 15) + 16 * (kg >> 1), nt_s = col >> 4, half = kg & 1;
    uint32_t raw[kCsMaxKs / 2][8];
#pragma unroll
    for (int i = 0; i < kCsMaxKs / 2; ++i) {
      const uint32_t ks = 2 * i + h;
      if (ks < ks_total) {
        const uint32_t rows = d_in - ks * kBK < kBK ? d_in - ks * kBK : kBK;
        const rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<uint32_t*>(bsrc) + static_cast<size_t>(ks) * kBK * row_words, 0, rows * row_bytes, kRsrcWord3);
#pragma unroll
        for (int r = 0; r < 8; ++r)
          raw[i][r] = __builtin_amdgcn_raw_buffer_load_b32(rs, (kg * 8 + r) * row_bytes + col * 4, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < kCsMaxKs / 2; ++i) {
      const uint32_t ks = 2 * i + h;
      if (ks < ks_total) {
        uint32_t lo[4], hi[4];
        transpose4(raw[i][0] + kBias, raw[i][1] + kBias, raw[i][2] + kBias, raw[i][3] + kBias, lo);
        transpose4(raw[i][4] + kBias, raw[i][5] + kBias, raw[i][6] + kBias, raw[i][7] + kBias, hi);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          uint2* dst = reinterpret_cast<uint2*>(&bs[ks][(nt_s * 4 + b) * 64 + frag_lane]) + half;
          *dst = make_uint2(lo[b] ^ kBias, hi[b] ^ kBias);
        }
      }
    }
  }
  __syncthreads();

  const uint32_t wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const uint32_t wtiles = (d_out + kMT * 16 - 1) / (kMT * 16);
  for (uint32_t wt = wave; wt < wtiles; wt += kCsWaves) {
    const uint32_t mt_wave = wt * kMT;
    uint32_t top = 0;
#pragma unroll
    for (int i = 0; i < kMT; ++i) top |= flags[l * mt_total + mt_wave + i];
    top = __builtin_amdgcn_readfirstlane(top);
    const v4i* adig_wave = adig + (static_cast<size_t>(l) * mt_total + mt_wave) * ks_total * 4 * 64;
    const uint32_t row0 = mt_wave * 16;
    const uint32_t rows = d_out - row0 < kMT * 16 ? d_out - row0 : kMT * 16;
    uint32_t* dst = ct_out + ((static_cast<size_t>(row0) * 2 + c) * limbs + l) * n + k0;
    const rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(dst, 0, rows * row_bytes, kRsrcWord3);
    if (top != 0)
      cs_tile<4>(tb, adig_wave, ks_total, bs, out, l, lane, row_bytes);
    else
      cs_tile<3>(tb, adig_wave, ks_total, bs, out, l, lane, row_bytes);
  }
}

struct Shape {
  uint32_t tiles_m, tiles_n, mt_total, ks_total;
  size_t adig_bytes, flag_bytes;
};

Shape shape_of(uint32_t n, uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  Shape s;
  s.tiles_m = (d_out + kBM - 1) / kBM;
  s.tiles_n = 2 * n / kBN;
  s.mt_total = s.tiles_m * (kBM / 16);
  s.ks_total = (d_in + kBK - 1) / kBK;
  s.adig_bytes = static_cast<size_t>(limbs) * s.mt_total * s.ks_total * 4 * 64 * sizeof(v4i);
  s.flag_bytes = ((static_cast<size_t>(limbs) * s.mt_total * 4) + 255) & ~size_t(255);
  return s;
}

}  // namespace

hipError_t noalloc_scratch(int device, void** out) {
  // Resolved once per device, with that device current (the caller's guard).
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[device]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[device] = p;
  }
  *out = addr[device];
  return hipSuccess;
}

size_t mac_mfma_workspace_bytes(uint32_t n, uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  if (d_out == 0 || d_in == 0 || d_in > kMaxDin) return 0;
  const Shape s = shape_of(n, d_out, d_in, limbs);
  return s.adig_bytes + s.flag_bytes;
}

bool mac_mfma_supported(uint32_t d_in) { return d_in >= 1 && d_in <= kMaxDin; }

hipError_t launch_mac_scalar_mfma(const Tables& t, const uint32_t* w_enc, const uint32_t* ct_in,
                                  uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                  void* workspace, hipStream_t st) {
  const Shape s = shape_of(t.n, d_out, d_in, limbs);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  v4i* adig = reinterpret_cast<v4i*>(ws);
  uint32_t* flags = reinterpret_cast<uint32_t*>(ws + s.adig_bytes);
  mfma_prep_kernel<<<dim3(s.mt_total * limbs), kThreads, 0, st>>>(t.q, w_enc, d_out, d_in, limbs, s.mt_total,
                                                                  s.ks_total, adig, flags);
  const size_t grid = static_cast<size_t>(limbs) * s.tiles_n * s.tiles_m;
  if (grid >= (size_t(1) << 31)) return hipErrorInvalidValue;  // tile indices are 32-bit
  if (d_in <= kCsMaxDin) {
    const size_t cgrid = static_cast<size_t>(limbs) * s.tiles_n;
    if (cgrid >= (size_t(1) << 31)) return hipErrorInvalidValue;
    mac_cs_kernel<<<static_cast<uint32_t>(cgrid), kCsThreads, 0, st>>>(t, adig, flags, ct_in, ct_out, d_out, d_in,
                                                                      limbs, s.mt_total, s.ks_total, s.tiles_n);
    return hipGetLastError();
  }
  mac_mfma_kernel<<<static_cast<uint32_t>(grid), kThreads, 0, st>>>(t, adig, flags, ct_in, ct_out, d_out, d_in, limbs,
                                                                   s.mt_total, s.ks_total, s.tiles_m, s.tiles_n);
  return hipGetLastError();
}

}  // namespace ckks
