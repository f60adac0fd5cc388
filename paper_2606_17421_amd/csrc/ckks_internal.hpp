// Internal declarations of the gfx950 CKKS linear-layer library: the device
// table bundle that every kernel receives by value, 30-bit modular arithmetic
// helpers, and the launchers each kernel file exports to the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ckks {

constexpr int kMaxLimbs = 16;
constexpr int kMinLogN = 10;
constexpr int kMaxLogN = 16;
constexpr uint32_t kMaxMacDin = 1u << 24;  // largest d_in of the scalar MAC entry point
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;  // per-GPU workspace of the no-allocation MAC
constexpr int kMaxDevices = 64;

// Per-context device tables.  All arrays live in one device allocation owned
// by the context; [L][N] arrays are limb-major.
struct Tables {
  uint32_t log_n;
  uint32_t n;
  uint32_t L;
  uint32_t num_cus;            // compute units of the context's device
  const uint32_t* q;           // [L]
  const uint32_t* fwd;         // [L][N]  psi_l^brv(k)         (forward twiddles)
  const uint32_t* fwd_shoup;   // [L][N]  floor(fwd * 2^32 / q)
  const uint32_t* inv;         // [L][N]  psi_l^-brv(k)        (inverse twiddles)
  const uint32_t* inv_shoup;   // [L][N]
  const uint32_t* ninv;        // [L]     N^-1 mod q_l
  const uint32_t* ninv_shoup;  // [L]
  const uint32_t* qinv;        // [L][L]  qinv[m*L + l] = q_m^-1 mod q_l (0 on the diagonal)
  const uint32_t* qinv_shoup;  // [L][L]
  const double* q_recip;       // [L]     1.0 / q_l rounded to nearest
  const uint32_t* barrett;     // [L]     floor(2^61 / q_l) (< 2^32 for q_l > 2^29)
  const uint32_t* pow256;      // [L][8]  256^s mod q_l, s < 8
  // Encode tables (M = N/2, P = N/4).
  const uint32_t* slot_perm;   // [M]  slot index j whose odd exponent is 2u+1 (up to sign)
  const uint32_t* slot_pos;    // [M]  index m of slot j in the Makhoul-ordered real sequence
  const double2* fft_tw;       // [P/2] exp(-2 pi i m / P)
  const double2* rfft_tw;      // [P]   exp(-2 pi i k / M)
  const double2* dct_tw;       // [M]   exp(-i pi k / (2M))
};

// ---------------------------------------------------------------------------
// 30-bit modular arithmetic (q < 2^30, all operands fully reduced unless noted)
// ---------------------------------------------------------------------------

// Shoup product: w < q, ws = floor(w 2^32 / q); any a < 2^32.  Result in [0, q).
__device__ __forceinline__ uint32_t mul_shoup(uint32_t a, uint32_t w, uint32_t ws, uint32_t q) {
  uint32_t hi = __umulhi(a, ws);
  uint32_t r = a * w - hi * q;  // in [0, 2q)
  return min(r, r - q);
}

// Lazy Shoup product: any a < 2^32, w < q, ws = floor(w 2^32 / q).  The
// quotient estimate floor(a ws / 2^32) is within one of floor(a w / q), so the
// result lies in [0, 2q).
__device__ __forceinline__ uint32_t mul_shoup_lazy(uint32_t a, uint32_t w, uint32_t ws, uint32_t q) {
  return a * w - __umulhi(a, ws) * q;
}

__device__ __forceinline__ uint32_t add_mod(uint32_t a, uint32_t b, uint32_t q) {
  uint32_t s = a + b;
  return min(s, s - q);
}

__device__ __forceinline__ uint32_t sub_mod(uint32_t a, uint32_t b, uint32_t q) {
  uint32_t d = a - b + q;
  return min(d, d - q);
}

// a * b mod q for a < 2^30, b < q, with mu = floor(2^61 / q) (Barrett, 32-bit
// operations only).  With x = a b < 2^60, t = floor(x / 2^29) and qt =
// floor(t mu / 2^32), x/q - 2 < qt <= x/q, so x - qt q lies in [0, 3q) and its
// low 32 bits are exact (3q < 2^32); two conditional subtractions finish.
__device__ __forceinline__ uint32_t mul_mod_barrett(uint32_t a, uint32_t b, uint32_t q, uint32_t mu) {
  const uint32_t lo = a * b, hi = __umulhi(a, b);
  const uint32_t t = __builtin_amdgcn_alignbit(hi, lo, 29);  // bits 29..60 of a b
  uint32_t r = lo - __umulhi(t, mu) * q;
  r = min(r, r - q);
  return min(r, r - q);
}

// x mod q for any x < 2^64, with qr = 1.0/q.  The fp64 quotient estimate is
// within one of floor(x/q) (relative error < 2^-51 on a quotient < 2^35), so
// the 64-bit remainder lies in [-q, 2q) before the two corrections.
__device__ __forceinline__ uint32_t reduce_u64(uint64_t x, uint32_t q, double qr) {
  double qt = floor(static_cast<double>(x) * qr);
  uint64_t qi = static_cast<uint64_t>(qt);
  int64_t r = static_cast<int64_t>(x - qi * static_cast<uint64_t>(q));
  r += (r < 0) ? static_cast<int64_t>(q) : 0;
  r -= (r >= static_cast<int64_t>(q)) ? static_cast<int64_t>(q) : 0;
  return static_cast<uint32_t>(r);
}

// v mod q for an integer-valued double v (|v| < 2^63), result in [0, q).
__device__ __forceinline__ uint32_t reduce_f64_int(double v, uint32_t q, double qr) {
  if (fabs(v) < 4503599627370496.0) {  // 2^52: v and the remainder are exact in fp64
    double qt = floor(v * qr);
    double r = fma(-qt, static_cast<double>(q), v);
    r += (r < 0.0) ? static_cast<double>(q) : 0.0;
    r -= (r >= static_cast<double>(q)) ? static_cast<double>(q) : 0.0;
    return static_cast<uint32_t>(r);
  }
  int64_t iv = static_cast<int64_t>(v);
  int64_t r = iv % static_cast<int64_t>(q);
  return static_cast<uint32_t>(r < 0 ? r + static_cast<int64_t>(q) : r);
}

// ---------------------------------------------------------------------------
// Launchers (each returns hipSuccess or the launch error)
// ---------------------------------------------------------------------------

// In-place forward / inverse NTT of count_rows rows; logical row r uses limb
// r % limbs and is physical row (r / limbs) * gstride + r % limbs of
// rows[][N] (gstride 0 means limbs: packed [count][limbs][N]).
hipError_t launch_ntt(const Tables& t, uint32_t* rows, size_t count_rows, uint32_t limbs,
                      bool inverse, hipStream_t s, uint32_t gstride = 0);

hipError_t launch_encode_scalar(const Tables& t, const double* w, size_t count, uint32_t limbs,
                                double scale, uint32_t* w_enc, hipStream_t s);

// NTT-form residues pt[count][limbs][N] of the encoded slot vectors.
hipError_t launch_encode_poly(const Tables& t, const double* slots, uint32_t count, uint32_t limbs,
                              double scale, uint32_t* pt, hipStream_t s);

hipError_t launch_mac_scalar_valu(const Tables& t, const uint32_t* w_enc, const uint32_t* ct_in,
                                  uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                  hipStream_t s);

size_t mac_mfma_workspace_bytes(uint32_t n, uint32_t d_out, uint32_t d_in, uint32_t limbs);
// Device address, on `device` (which must be current), of the library's
// kNoAllocScratchBytes array that the no-allocation MAC uses as its workspace.
hipError_t noalloc_scratch(int device, void** out);
bool mac_mfma_supported(uint32_t d_in);
hipError_t launch_mac_scalar_mfma(const Tables& t, const uint32_t* w_enc, const uint32_t* ct_in,
                                  uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                                  void* workspace, hipStream_t s);

hipError_t launch_mac_poly(const Tables& t, const uint32_t* pt, const uint32_t* ct_in,
                           uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                           hipStream_t s);

size_t rescale_workspace_bytes(const Tables& t, uint32_t count, uint32_t limbs);
hipError_t launch_rescale(const Tables& t, const uint32_t* ct_in, uint32_t* ct_out, uint32_t count,
                          uint32_t limbs, void* workspace, hipStream_t s);
hipError_t launch_rescale2(const Tables& t, const uint32_t* ct_in, uint32_t* mid, uint32_t* ct_out, uint32_t count,
                           uint32_t limbs, void* workspace, hipStream_t s);

hipError_t launch_zero(uint32_t* p, size_t words, hipStream_t s);

// Symmetric RLWE over ciphertexts [count][2][limbs][N], NTT form (rlwe.hip).
hipError_t launch_encrypt(const Tables& t, const uint32_t* pt, const uint32_t* s_ntt, const uint32_t* a,
                          const int32_t* e, uint32_t count, uint32_t limbs, uint32_t* ct, hipStream_t s);
hipError_t launch_decrypt(const Tables& t, const uint32_t* ct, const uint32_t* s_ntt, uint32_t count,
                          uint32_t limbs, uint32_t* m, hipStream_t s);
hipError_t launch_refresh(const Tables& t, const uint32_t* ct_in, uint32_t limbs_in, const uint32_t* s_ntt,
                          const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs_out,
                          uint32_t* ct_out, hipStream_t s);

// Rotations and the BSGS product (keyswitch.hip).  The context's last prime is
// the special prime; rotated ciphertexts carry t.L - 1 limbs.
hipError_t launch_automorphism(const Tables& t, const uint32_t* in, size_t rows, uint32_t galois, uint32_t* out,
                               hipStream_t s);
size_t rotate_workspace_bytes(const Tables& t, uint32_t inputs, uint32_t rotations);
hipError_t launch_rotate(const Tables& t, const uint32_t* ct, uint32_t count, uint32_t r0, uint32_t r_step,
                         uint32_t galois, bool hoisted, const uint32_t* ksk, void* workspace, uint32_t* out,
                         hipStream_t s);
hipError_t launch_keygen_rotation(const Tables& t, const uint32_t* s_ntt, uint32_t r0, uint32_t r_step,
                                  uint32_t keys, const uint32_t* a, const int32_t* e, uint32_t* ksk,
                                  hipStream_t s);
size_t bsgs_workspace_bytes(const Tables& t, uint32_t count, uint32_t n1, uint32_t n2);
hipError_t launch_ct_add(const Tables& t, const uint32_t* a, const uint32_t* b, uint32_t count, uint32_t limbs,
                         uint32_t* out, hipStream_t s);
hipError_t launch_bsgs(const Tables& t, const uint32_t* pt, const uint32_t* ct, uint32_t count, uint32_t n1,
                       uint32_t n2, const uint32_t* ksk, void* workspace, uint32_t* out, hipStream_t s);

}  // namespace ckks
