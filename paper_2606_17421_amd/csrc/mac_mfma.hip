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
// (|S_s| <= 4 * d_in * 2^14 <= 2^30 for d_in <= 16384).  The epilogue folds
// the classes in i64 (classes 0..3 with their exact weights 2^(8s), classes
// 4..6 with 256^s mod q; |sum| < 2^62) and reduces once mod q.
// Digit products: 12 per modular MAC with 3 weight digits, 16 with 4.
//
// Tiling: a 256-thread workgroup computes a 128 (rows) x 64 (columns) tile of
// one limb; each wave owns 32 rows x 64 columns (2 x 4 MFMA tiles x 6 or 7
// shift-class accumulators).  Weight digit fragments are pre-arranged in
// MFMA lane order by a prep kernel and read straight from global memory (L2
// resident); ciphertext residues are staged through LDS, converted to digit
// fragments once per workgroup.  Workgroups are ordered (limb, column tile,
// row tile) with row tiles fastest and remapped so that each XCD runs a
// contiguous range: tiles sharing a B tile, and a whole limb's A, stay in one
// XCD's L2.
#include "ckks_internal.hpp"

namespace ckks {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBM = 128;       // rows per workgroup tile
constexpr int kBN = 64;        // columns per workgroup tile
constexpr int kBK = 64;        // K per MFMA step
constexpr int kMT = 2;         // 16-row MFMA tiles per wave
constexpr int kNT = kBN / 16;  // 16-column MFMA tiles per wave
constexpr uint32_t kBias = 0x80808080u;
constexpr uint32_t kMaxDin = 16384;

__device__ __forceinline__ uint32_t digits4(uint32_t u) { return (u + kBias) ^ kBias; }

// o[b] byte e = p[e] byte b  (4x4 byte transpose)
__device__ __forceinline__ void transpose4(const uint32_t (&p)[4], uint32_t (&o)[4]) {
#pragma unroll
  for (int b = 0; b < 4; ++b)
    o[b] = ((p[0] >> (8 * b)) & 0xffu) | (((p[1] >> (8 * b)) & 0xffu) << 8) |
           (((p[2] >> (8 * b)) & 0xffu) << 16) | (((p[3] >> (8 * b)) & 0xffu) << 24);
}

// 16 packed digit words (consecutive k) -> one 16-byte fragment per digit.
__device__ __forceinline__ void to_fragments(const uint32_t (&p)[16], v4i (&f)[4]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const uint32_t in[4] = {p[4 * g], p[4 * g + 1], p[4 * g + 2], p[4 * g + 3]};
    uint32_t o[4];
    transpose4(in, o);
#pragma unroll
    for (int b = 0; b < 4; ++b) f[b][g] = static_cast<int>(o[b]);
  }
}

// Weight digits: adig[((l * mt_total + mt) * ks_total + ks) * 4 + a][lane] holds
// e_a(w[mt*16 + lane%16][ks*64 + (lane/16)*16 + i]) in byte i (zero-padded);
// flags[l * mt_total + mt] != 0 when any e_3 of that 16-row tile is non-zero.
__global__ __launch_bounds__(kThreads) void mfma_prep_kernel(
    const uint32_t* __restrict__ qtab, const uint32_t* __restrict__ w_enc, uint32_t d_out,
    uint32_t d_in, uint32_t limbs, uint32_t mt_total, uint32_t ks_total, v4i* __restrict__ adig,
    uint32_t* __restrict__ flags) {
  const uint32_t mt = blockIdx.x, l = blockIdx.y;
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
      const uint32_t v = w > (q >> 1) ? w - q : w;  // centred, two's complement
      p[i] = digits4(v);
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

// K loop, software pipelined: while the MFMAs of step ks run, the raw
// ciphertext residues and the weight fragments of step ks+1 are in flight;
// the residues are then converted to digit fragments into the other LDS
// buffer, so each step needs one barrier.
template <int NDA>
__device__ __forceinline__ void mac_loop(const v4i* __restrict__ adig_wave, uint32_t ks_total,
                                         const uint32_t* __restrict__ bsrc, size_t bstride,
                                         uint32_t d_in, v4i (*bs)[kNT][4][64],
                                         v4i (&acc)[kMT][kNT][7]) {
  const uint32_t tid = threadIdx.x;
  const uint32_t lane = tid & 63;
  const uint32_t col = tid & 63;  // staging: column within the tile
  const uint32_t g = tid >> 6;    // staging: 16-k group
  uint32_t raw[16];
  v4i a_cur[kMT][NDA], a_nxt[kMT][NDA];

  auto load_b = [&](uint32_t ks) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      uint32_t k = ks * kBK + g * 16 + i;
      k = k < d_in ? k : d_in - 1;  // padded k: any in-bounds value (its weight digits are 0)
      raw[i] = bsrc[static_cast<size_t>(k) * bstride + col];
    }
  };
  auto store_b = [&](int buf) {
    uint32_t p[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) p[i] = digits4(raw[i]);
    v4i f[4];
    to_fragments(p, f);
#pragma unroll
    for (int b = 0; b < 4; ++b) bs[buf][col >> 4][b][(col & 15) + 16 * g] = f[b];
  };
  auto load_a = [&](v4i (&a)[kMT][NDA], uint32_t ks) {
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
      for (int d = 0; d < NDA; ++d)
        a[mt][d] = adig_wave[((static_cast<size_t>(mt) * ks_total + ks) * 4 + d) * 64 + lane];
  };

  load_b(0);
  load_a(a_cur, 0);
  store_b(0);
  __syncthreads();
  for (uint32_t ks = 0; ks < ks_total; ++ks) {
    const int buf = ks & 1;
    const bool more = ks + 1 < ks_total;
    if (more) {
      load_b(ks + 1);
      load_a(a_nxt, ks + 1);
    }
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt) {
      v4i bf[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) bf[b] = bs[buf][nt][b][lane];
#pragma unroll
      for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
        for (int d = 0; d < NDA; ++d)
#pragma unroll
          for (int b = 0; b < 4; ++b)
            acc[mt][nt][d + b] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a_cur[mt][d], bf[b], acc[mt][nt][d + b], 0, 0, 0);
    }
    if (more) store_b(buf ^ 1);
    __syncthreads();
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
      for (int d = 0; d < NDA; ++d) a_cur[mt][d] = a_nxt[mt][d];
  }
}

__global__ __launch_bounds__(kThreads) void mac_mfma_kernel(
    Tables tb, const v4i* __restrict__ adig, const uint32_t* __restrict__ flags,
    const uint32_t* __restrict__ ct_in, uint32_t* __restrict__ ct_out, uint32_t d_out, uint32_t d_in,
    uint32_t limbs, uint32_t mt_total, uint32_t ks_total, uint32_t tiles_m, uint32_t tiles_n) {
  __shared__ v4i bs[2][kNT][4][64];  // B digit fragments, double buffered (32 KiB)

  // XCD-aware order: consecutive workgroup ids alternate XCDs; give each XCD a
  // contiguous range of logical tiles (row tile fastest, then column, then limb).
  const uint32_t G = gridDim.x;
  uint32_t lid = blockIdx.x;
  if ((G & 7u) == 0) lid = (lid & 7u) * (G >> 3) + (lid >> 3);
  const uint32_t mtile = lid % tiles_m;
  lid /= tiles_m;
  const uint32_t ntile = lid % tiles_n;
  const uint32_t l = lid / tiles_n;

  const uint32_t n = tb.n;
  const uint32_t wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint32_t col0 = ntile * kBN;  // column in [0, 2N): component c = col0 / N
  const uint32_t c = col0 >> tb.log_n, k0 = col0 & (n - 1);
  const size_t bstride = 2ull * limbs * n;  // one input ciphertext
  const uint32_t* bsrc = ct_in + (static_cast<size_t>(c) * limbs + l) * n + k0;
  const uint32_t mt_wave = mtile * (kBM / 16) + wave * kMT;
  const v4i* adig_wave = adig + (static_cast<size_t>(l) * mt_total + mt_wave) * ks_total * 4 * 64;

  uint32_t top = 0;
#pragma unroll
  for (int i = 0; i < kBM / 16; ++i) top |= flags[l * mt_total + mtile * (kBM / 16) + i];

  v4i acc[kMT][kNT][7];
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int nt = 0; nt < kNT; ++nt)
#pragma unroll
      for (int s = 0; s < 7; ++s) acc[mt][nt][s] = v4i{0, 0, 0, 0};

  if (top) mac_loop<4>(adig_wave, ks_total, bsrc, bstride, d_in, bs, acc);
  else mac_loop<3>(adig_wave, ks_total, bsrc, bstride, d_in, bs, acc);

  // ---- epilogue: out = sum_s S_s 256^s  mod q ----
  // Classes 0..3 enter with their exact weights 2^(8s); classes 4..6 with
  // 256^s mod q.  |v| < 2^62: the fp64 quotient estimate is within one of the
  // true quotient, so the remainder, formed in 32 bits, lies in [-q, 2q).
  const uint32_t q = tb.q[l];
  const double qr = tb.q_recip[l];
  const int64_t c4 = static_cast<int64_t>((1ull << 32) % q);
  const int64_t c5 = static_cast<int64_t>((static_cast<uint64_t>(c4) << 8) % q);
  const int64_t c6 = static_cast<int64_t>((static_cast<uint64_t>(c5) << 8) % q);
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t j = (mt_wave + mt) * 16 + 4 * (lane >> 4) + r;
      if (j >= d_out) continue;
      uint32_t* orow = ct_out + ((static_cast<size_t>(j) * 2 + c) * limbs + l) * n + k0 + (lane & 15);
#pragma unroll
      for (int nt = 0; nt < kNT; ++nt) {
        const v4i* a = acc[mt][nt];
        int64_t v = static_cast<int64_t>(a[0][r]) + (static_cast<int64_t>(a[1][r]) << 8) +
                    (static_cast<int64_t>(a[2][r]) << 16) + (static_cast<int64_t>(a[3][r]) << 24) +
                    static_cast<int64_t>(a[4][r]) * c4 + static_cast<int64_t>(a[5][r]) * c5 +
                    static_cast<int64_t>(a[6][r]) * c6;
        const int64_t qt = static_cast<int64_t>(floor(static_cast<double>(v) * qr));
        int32_t rem = static_cast<int32_t>(static_cast<uint32_t>(v) - static_cast<uint32_t>(qt) * q);
        rem += rem < 0 ? static_cast<int32_t>(q) : 0;
        rem -= rem >= static_cast<int32_t>(q) ? static_cast<int32_t>(q) : 0;
        orow[nt * 16] = static_cast<uint32_t>(rem);
      }
    }
  }
}

struct Shape {
  uint32_t tiles_m, mt_total, ks_total;
  size_t adig_bytes, flag_bytes;
};

Shape shape_of(uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  Shape s;
  s.tiles_m = (d_out + kBM - 1) / kBM;
  s.mt_total = s.tiles_m * (kBM / 16);
  s.ks_total = (d_in + kBK - 1) / kBK;
  s.adig_bytes = static_cast<size_t>(limbs) * s.mt_total * s.ks_total * 4 * 64 * sizeof(v4i);
  s.flag_bytes = ((static_cast<size_t>(limbs) * s.mt_total * 4) + 255) & ~size_t(255);
  return s;
}

}  // namespace

size_t mac_mfma_workspace_bytes(uint32_t d_out, uint32_t d_in, uint32_t limbs) {
  if (d_out == 0 || d_in == 0 || d_in > kMaxDin) return 0;
  const Shape s = shape_of(d_out, d_in, limbs);
  return s.adig_bytes + s.flag_bytes;
}

bool mac_mfma_supported(uint32_t d_in) { return d_in >= 1 && d_in <= kMaxDin; }

hipError_t launch_mac_scalar_mfma(const Tables& t, const uint32_t* w_enc, const uint32_t* ct_in,
                                  uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                  void* workspace, hipStream_t st) {
  const Shape s = shape_of(d_out, d_in, limbs);
  v4i* adig = static_cast<v4i*>(workspace);
  uint32_t* flags = reinterpret_cast<uint32_t*>(static_cast<unsigned char*>(workspace) + s.adig_bytes);
  mfma_prep_kernel<<<dim3(s.mt_total, limbs), kThreads, 0, st>>>(t.q, w_enc, d_out, d_in, limbs, s.mt_total,
                                                                 s.ks_total, adig, flags);
  const uint32_t tiles_n = 2 * t.n / kBN;
  const size_t grid = static_cast<size_t>(limbs) * tiles_n * s.tiles_m;
  mac_mfma_kernel<<<static_cast<uint32_t>(grid), kThreads, 0, st>>>(t, adig, flags, ct_in, ct_out, d_out, d_in,
                                                                   limbs, s.mt_total, s.ks_total, s.tiles_m,
                                                                   tiles_n);
  return hipGetLastError();
}

}  // namespace ckks
