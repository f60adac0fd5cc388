// C ABI of the CKKS ct x pt linear-layer library: context creation (modulus
// chain, roots, device tables), argument validation and kernel dispatch.
// Declarations and contracts: include/ckks_linear.h.
#include "ckks_linear.h"

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "ckks_internal.hpp"

static_assert(CKKS_NOALLOC_SCRATCH_BYTES == ckks::kNoAllocScratchBytes, "scratch size in the header and the library");

struct ckks_ctx {
  int device = 0;
  uint32_t log_n = 0, n = 0, L = 0;
  std::vector<uint32_t> q, psi;
  int mac_algo = CKKS_MAC_AUTO;
  void* dev = nullptr;
  void* scratch = nullptr;            // the device's no-allocation MAC workspace (library-owned)
  hipError_t scratch_status = hipSuccess;
  ckks::Tables t{};
};

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return CKKS_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(CKKS_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

// ---- host number theory (q < 2^30, so products fit in 64 bits) ------------

uint64_t powmod(uint64_t b, uint64_t e, uint64_t m) {
  uint64_t r = 1 % m;
  b %= m;
  while (e) {
    if (e & 1) r = r * b % m;
    b = b * b % m;
    e >>= 1;
  }
  return r;
}

// Deterministic Miller-Rabin for n < 3,215,031,751 with bases 2, 3, 5, 7.
bool is_prime(uint64_t n) {
  if (n < 2) return false;
  for (uint64_t p : {2ull, 3ull, 5ull, 7ull, 11ull, 13ull})
    if (n % p == 0) return n == p;
  uint64_t d = n - 1;
  int s = 0;
  while ((d & 1) == 0) {
    d >>= 1;
    ++s;
  }
  for (uint64_t a : {2ull, 3ull, 5ull, 7ull}) {
    uint64_t x = powmod(a, d, n);
    if (x == 1 || x == n - 1) continue;
    bool comp = true;
    for (int r = 1; r < s; ++r) {
      x = x * x % n;
      if (x == n - 1) {
        comp = false;
        break;
      }
    }
    if (comp) return false;
  }
  return true;
}

bool default_moduli(uint32_t log_n, uint32_t L, std::vector<uint32_t>& out) {
  const uint64_t two_n = 2ull << log_n;
  uint64_t c = ((1ull << 30) - 2) / two_n * two_n + 1;
  out.clear();
  while (out.size() < L) {
    if (c <= (1ull << 29)) return false;
    if (is_prime(c)) out.push_back(static_cast<uint32_t>(c));
    c -= two_n;
  }
  return true;
}

// Smallest primitive 2N-th root of unity: g^((q-1)/2N) for the smallest
// generator g of Z_q^*, minimised over its odd powers.
uint32_t min_root(uint32_t q, uint32_t log_n) {
  std::vector<uint64_t> fs;
  uint64_t m = q - 1;
  for (uint64_t p = 2; p * p <= m; ++p) {
    if (m % p == 0) {
      fs.push_back(p);
      while (m % p == 0) m /= p;
    }
  }
  if (m > 1) fs.push_back(m);
  uint64_t g = 2;
  for (;; ++g) {
    bool gen = true;
    for (uint64_t f : fs)
      if (powmod(g, (q - 1) / f, q) == 1) {
        gen = false;
        break;
      }
    if (gen) break;
  }
  const uint64_t two_n = 2ull << log_n;
  const uint64_t root = powmod(g, (q - 1) / two_n, q);
  const uint64_t root2 = root * root % q;
  uint64_t x = root, best = root;
  for (uint64_t k = 3; k < two_n; k += 2) {
    x = x * root2 % q;
    if (x < best) best = x;
  }
  return static_cast<uint32_t>(best);
}

uint32_t brv(uint32_t x, uint32_t bits) {
  uint32_t r = 0;
  for (uint32_t i = 0; i < bits; ++i) {
    r = (r << 1) | (x & 1);
    x >>= 1;
  }
  return r;
}

uint32_t shoup(uint32_t w, uint32_t q) {
  return static_cast<uint32_t>((static_cast<uint64_t>(w) << 32) / q);
}

struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      ok = false;
      return;
    }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Layout builder for the single device allocation holding all tables.
struct Blob {
  std::vector<unsigned char> bytes;
  size_t add(const void* src, size_t n) {
    size_t off = (bytes.size() + 255) & ~size_t(255);
    bytes.resize(off + n);
    std::memcpy(bytes.data() + off, src, n);
    return off;
  }
};

// Byte ranges [x, x + xb) and [y, y + yb) share at least one byte.
bool overlaps(const void* x, size_t xb, const void* y, size_t yb) {
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(x), b0 = reinterpret_cast<uintptr_t>(y);
  return xb != 0 && yb != 0 && a0 < b0 + yb && b0 < a0 + xb;
}

int check_ctx(const ckks_ctx* ctx) {
  if (!ctx) return fail(CKKS_E_INVALID_ARG, "null context");
  return CKKS_OK;
}

int check_limbs(const ckks_ctx* ctx, uint32_t limbs, uint32_t min_limbs) {
  if (limbs < min_limbs || limbs > ctx->L)
    return fail(CKKS_E_INVALID_ARG, "limbs=%u outside [%u, %u]", limbs, min_limbs, ctx->L);
  return CKKS_OK;
}

int check_ptr(const void* p, const char* name) {
  if (!p) return fail(CKKS_E_INVALID_ARG, "%s is null", name);
  if (!aligned16(p)) return fail(CKKS_E_INVALID_ARG, "%s is not 16-byte aligned", name);
  return CKKS_OK;
}

}  // namespace

extern "C" {

int ckks_ctx_create(ckks_ctx** out, uint32_t log_n, uint32_t num_limbs, const uint32_t* moduli,
                    int device) {
  if (!out) return fail(CKKS_E_INVALID_ARG, "out is null");
  if (log_n < ckks::kMinLogN || log_n > ckks::kMaxLogN)
    return fail(CKKS_E_INVALID_ARG, "log_n=%u outside [10, 16]", log_n);
  if (num_limbs < 1 || num_limbs > static_cast<uint32_t>(ckks::kMaxLimbs))
    return fail(CKKS_E_INVALID_ARG, "num_limbs=%u outside [1, 16]", num_limbs);
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
    return fail(CKKS_E_INVALID_ARG, "device %d not available (%d devices)", device, ndev);

  ckks_ctx* c = new ckks_ctx();
  c->device = device;
  c->log_n = log_n;
  c->n = 1u << log_n;
  c->L = num_limbs;
  const uint64_t two_n = 2ull << log_n;
  if (moduli) {
    c->q.assign(moduli, moduli + num_limbs);
    for (uint32_t i = 0; i < num_limbs; ++i) {
      const uint32_t q = c->q[i];
      if (q <= (1u << 29) || q >= (1u << 30) || q % two_n != 1 || !is_prime(q)) {
        delete c;
        return fail(CKKS_E_INVALID_ARG, "modulus %u is not a prime in (2^29, 2^30) with q = 1 mod 2N", q);
      }
      for (uint32_t k = 0; k < i; ++k)
        if (c->q[k] == q) {
          delete c;
          return fail(CKKS_E_INVALID_ARG, "modulus %u repeated", q);
        }
    }
  } else if (!default_moduli(log_n, num_limbs, c->q)) {
    delete c;
    return fail(CKKS_E_UNSUPPORTED, "not enough 30-bit NTT primes for N=2^%u", log_n);
  }
  const uint32_t n = c->n, L = num_limbs;
  for (uint32_t q : c->q) c->psi.push_back(min_root(q, log_n));

  // ---- host tables ----
  std::vector<uint32_t> fwd(size_t(L) * n), fwds(size_t(L) * n), inv(size_t(L) * n), invs(size_t(L) * n);
  std::vector<uint32_t> ninv(L), ninvs(L), qinv(size_t(L) * L, 0), qinvs(size_t(L) * L, 0);
  std::vector<double> qrec(L);
  std::vector<uint32_t> bar(L);
  std::vector<uint32_t> p256(size_t(L) * 8);
  for (uint32_t l = 0; l < L; ++l) {
    const uint64_t q = c->q[l];
    const uint64_t ps = c->psi[l];
    const uint64_t psi_inv = powmod(ps, q - 2, q);
    // powers in natural order, then scatter to bit-reversed positions
    uint64_t x = 1, y = 1;
    for (uint32_t k = 0; k < n; ++k) {
      const uint32_t r = brv(k, log_n);
      fwd[size_t(l) * n + r] = static_cast<uint32_t>(x);
      inv[size_t(l) * n + r] = static_cast<uint32_t>(y);
      x = x * ps % q;
      y = y * psi_inv % q;
    }
    for (uint32_t k = 0; k < n; ++k) {
      fwds[size_t(l) * n + k] = shoup(fwd[size_t(l) * n + k], c->q[l]);
      invs[size_t(l) * n + k] = shoup(inv[size_t(l) * n + k], c->q[l]);
    }
    ninv[l] = static_cast<uint32_t>(powmod(n, q - 2, q));
    ninvs[l] = shoup(ninv[l], c->q[l]);
    qrec[l] = 1.0 / static_cast<double>(q);
    bar[l] = static_cast<uint32_t>((uint64_t(1) << 61) / q);
    uint64_t pw = 1;
    for (int e = 0; e < 8; ++e) {
      p256[size_t(l) * 8 + e] = static_cast<uint32_t>(pw);
      pw = (pw << 8) % q;
    }
    for (uint32_t m = 0; m < L; ++m) {
      if (m == l) continue;
      const uint32_t v = static_cast<uint32_t>(powmod(c->q[m] % q, q - 2, q));
      qinv[size_t(m) * L + l] = v;
      qinvs[size_t(m) * L + l] = shoup(v, c->q[l]);
    }
  }

  Blob blob;
  const size_t o_q = blob.add(c->q.data(), L * 4);
  const size_t o_fwd = blob.add(fwd.data(), fwd.size() * 4);
  const size_t o_fwds = blob.add(fwds.data(), fwds.size() * 4);
  const size_t o_inv = blob.add(inv.data(), inv.size() * 4);
  const size_t o_invs = blob.add(invs.data(), invs.size() * 4);
  const size_t o_ninv = blob.add(ninv.data(), L * 4);
  const size_t o_ninvs = blob.add(ninvs.data(), L * 4);
  const size_t o_qinv = blob.add(qinv.data(), qinv.size() * 4);
  const size_t o_qinvs = blob.add(qinvs.data(), qinvs.size() * 4);
  const size_t o_qrec = blob.add(qrec.data(), L * 8);
  const size_t o_bar = blob.add(bar.data(), L * 4);
  const size_t o_p256 = blob.add(p256.data(), p256.size() * 4);
  size_t o_perm = 0, o_pos = 0, o_fft = 0, o_rfft = 0, o_dct = 0;
  {  // encode tables (every supported N)
    const uint32_t M = n / 2, P = n / 4;
    std::vector<uint32_t> perm(M), pos(M);
    uint64_t e = 1;
    for (uint32_t j = 0; j < M; ++j) {
      const uint64_t t = e < n ? e : two_n - e;  // odd, < N
      perm[(t - 1) / 2] = j;
      e = e * 5 % two_n;
    }
    // Makhoul order: y_m = z at perm[u], u = 2m (m < M/2) or 2(M - 1 - m) + 1
    for (uint32_t u = 0; u < M; ++u) pos[perm[u]] = (u % 2 == 0) ? u / 2 : M - 1 - (u - 1) / 2;
    const long double pi = 3.141592653589793238462643383279502884L;
    std::vector<double2> fft(P / 2), rfft(P), dct(M);
    for (uint32_t m = 0; m < P / 2; ++m) {
      const long double a = -2.0L * pi * m / P;
      fft[m] = make_double2(static_cast<double>(cosl(a)), static_cast<double>(sinl(a)));
    }
    for (uint32_t k = 0; k < P; ++k) {
      const long double a = -2.0L * pi * k / M;
      rfft[k] = make_double2(static_cast<double>(cosl(a)), static_cast<double>(sinl(a)));
    }
    for (uint32_t k = 0; k < M; ++k) {
      const long double a = -pi * k / (2.0L * M);
      dct[k] = make_double2(static_cast<double>(cosl(a)), static_cast<double>(sinl(a)));
    }
    o_perm = blob.add(perm.data(), perm.size() * 4);
    o_pos = blob.add(pos.data(), pos.size() * 4);
    o_fft = blob.add(fft.data(), fft.size() * sizeof(double2));
    o_rfft = blob.add(rfft.data(), rfft.size() * sizeof(double2));
    o_dct = blob.add(dct.data(), dct.size() * sizeof(double2));
  }

  DeviceGuard guard(device);
  if (!guard.ok) {
    delete c;
    return fail(CKKS_E_HIP, "cannot select device %d", device);
  }
  hipError_t he = hipMalloc(&c->dev, blob.bytes.size());
  if (he != hipSuccess) {
    delete c;
    return hip_fail(he, "hipMalloc(context tables)");
  }
  he = hipMemcpy(c->dev, blob.bytes.data(), blob.bytes.size(), hipMemcpyHostToDevice);
  if (he != hipSuccess) {
    (void)hipFree(c->dev);
    delete c;
    return hip_fail(he, "hipMemcpy(context tables)");
  }
  int cus = 0;
  he = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (he != hipSuccess || cus <= 0) {
    (void)hipFree(c->dev);
    delete c;
    return hip_fail(he == hipSuccess ? hipErrorInvalidDevice : he, "hipDeviceGetAttribute(compute units)");
  }
  // The no-allocation MAC's workspace: this device's copy of the library's
  // scratch array, resolved here with the device current.
  c->scratch_status = ckks::noalloc_scratch(device, &c->scratch);
  if (c->scratch_status != hipSuccess) c->scratch = nullptr;
  auto* base = static_cast<unsigned char*>(c->dev);
  ckks::Tables& t = c->t;
  t.log_n = log_n;
  t.n = n;
  t.L = L;
  t.num_cus = static_cast<uint32_t>(cus);
  t.q = reinterpret_cast<const uint32_t*>(base + o_q);
  t.fwd = reinterpret_cast<const uint32_t*>(base + o_fwd);
  t.fwd_shoup = reinterpret_cast<const uint32_t*>(base + o_fwds);
  t.inv = reinterpret_cast<const uint32_t*>(base + o_inv);
  t.inv_shoup = reinterpret_cast<const uint32_t*>(base + o_invs);
  t.ninv = reinterpret_cast<const uint32_t*>(base + o_ninv);
  t.ninv_shoup = reinterpret_cast<const uint32_t*>(base + o_ninvs);
  t.qinv = reinterpret_cast<const uint32_t*>(base + o_qinv);
  t.qinv_shoup = reinterpret_cast<const uint32_t*>(base + o_qinvs);
  t.q_recip = reinterpret_cast<const double*>(base + o_qrec);
  t.barrett = reinterpret_cast<const uint32_t*>(base + o_bar);
  t.pow256 = reinterpret_cast<const uint32_t*>(base + o_p256);
  {
    t.slot_perm = reinterpret_cast<const uint32_t*>(base + o_perm);
    t.slot_pos = reinterpret_cast<const uint32_t*>(base + o_pos);
    t.fft_tw = reinterpret_cast<const double2*>(base + o_fft);
    t.rfft_tw = reinterpret_cast<const double2*>(base + o_rfft);
    t.dct_tw = reinterpret_cast<const double2*>(base + o_dct);
  }
  *out = c;
  return ok();
}

int ckks_ctx_destroy(ckks_ctx* ctx) {
  if (!ctx) return ok();
  int rc = CKKS_OK;
  {
    DeviceGuard guard(ctx->device);
    if (ctx->dev) {
      hipError_t e = hipFree(ctx->dev);
      if (e != hipSuccess) rc = hip_fail(e, "hipFree(context tables)");
    }
  }
  delete ctx;
  return rc == CKKS_OK ? ok() : rc;
}

int ckks_ctx_moduli(const ckks_ctx* ctx, uint32_t* out) {
  if (int rc = check_ctx(ctx)) return rc;
  if (!out) return fail(CKKS_E_INVALID_ARG, "out is null");
  std::memcpy(out, ctx->q.data(), ctx->L * 4);
  return ok();
}

int ckks_ctx_roots(const ckks_ctx* ctx, uint32_t* out) {
  if (int rc = check_ctx(ctx)) return rc;
  if (!out) return fail(CKKS_E_INVALID_ARG, "out is null");
  std::memcpy(out, ctx->psi.data(), ctx->L * 4);
  return ok();
}

int ckks_ctx_info(const ckks_ctx* ctx, uint32_t* log_n, uint32_t* num_limbs) {
  if (int rc = check_ctx(ctx)) return rc;
  if (log_n) *log_n = ctx->log_n;
  if (num_limbs) *num_limbs = ctx->L;
  return ok();
}

int ckks_ctx_set_mac_algo(ckks_ctx* ctx, int algo) {
  if (int rc = check_ctx(ctx)) return rc;
  if (algo != CKKS_MAC_AUTO && algo != CKKS_MAC_VALU && algo != CKKS_MAC_MFMA)
    return fail(CKKS_E_INVALID_ARG, "unknown MAC algorithm %d", algo);
  ctx->mac_algo = algo;
  return ok();
}

static int do_ntt(const ckks_ctx* ctx, uint32_t* polys, uint32_t count, uint32_t limbs, void* stream,
                  bool inverse) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (count == 0) return ok();
  if (int rc = check_ptr(polys, "polys")) return rc;
  const size_t rows = static_cast<size_t>(count) * limbs;
  if (rows > 0x7FFFFFFFull / (ctx->log_n == 16 ? 64 : 1))
    return fail(CKKS_E_INVALID_ARG, "too many polynomials (%zu rows)", rows);
  DeviceGuard guard(ctx->device);
  hipError_t e = ckks::launch_ntt(ctx->t, polys, rows, limbs, inverse, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ok() : hip_fail(e, inverse ? "intt launch" : "ntt launch");
}

int ckks_ntt(const ckks_ctx* ctx, uint32_t* polys, uint32_t count, uint32_t limbs, void* stream) {
  return do_ntt(ctx, polys, count, limbs, stream, false);
}

int ckks_intt(const ckks_ctx* ctx, uint32_t* polys, uint32_t count, uint32_t limbs, void* stream) {
  return do_ntt(ctx, polys, count, limbs, stream, true);
}

int ckks_linear_encode_scalar(const ckks_ctx* ctx, const double* w, uint32_t d_out, uint32_t d_in,
                              uint32_t limbs, double scale, uint32_t* w_enc, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (!(scale > 0.0) || !std::isfinite(scale)) return fail(CKKS_E_INVALID_ARG, "scale must be finite and > 0");
  const size_t count = static_cast<size_t>(d_out) * d_in;
  if (count == 0) return ok();
  if (int rc = check_ptr(w, "w")) return rc;
  if (int rc = check_ptr(w_enc, "w_enc")) return rc;
  if (overlaps(w_enc, count * limbs * 4, w, count * 8)) return fail(CKKS_E_INVALID_ARG, "w_enc overlaps w");
  DeviceGuard guard(ctx->device);
  hipError_t e = ckks::launch_encode_scalar(ctx->t, w, count, limbs, scale, w_enc,
                                            static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "encode_scalar launch");
}

int ckks_linear_encode_poly(const ckks_ctx* ctx, const double* slots, uint32_t count, uint32_t limbs,
                            double scale, uint32_t* pt, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (!(scale > 0.0) || !std::isfinite(scale)) return fail(CKKS_E_INVALID_ARG, "scale must be finite and > 0");
  if (count == 0) return ok();
  if (int rc = check_ptr(slots, "slots")) return rc;
  if (int rc = check_ptr(pt, "pt")) return rc;
  if (overlaps(pt, size_t(count) * limbs * ctx->n * 4, slots, size_t(count) * (ctx->n / 2) * 8))
    return fail(CKKS_E_INVALID_ARG, "pt overlaps slots");
  // at N = 2^16 the rows go through the batched transform (64 workgroups per row)
  if (ctx->log_n == 16 && size_t(count) * limbs > 0x7FFFFFFFull / 64)
    return fail(CKKS_E_INVALID_ARG, "count x limbs = %zu rows too many", size_t(count) * limbs);
  DeviceGuard guard(ctx->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = ckks::launch_encode_poly(ctx->t, slots, count, limbs, scale, pt, s);
  return e == hipSuccess ? ok() : hip_fail(e, "encode_poly launch");
}

// Shape limits of the scalar MAC: the VALU kernel's grid has ceil(d_out / 8)
// rows (at most 65535), and d_in is bounded so that every weight and fragment
// offset of both kernels stays far inside its index type.
static int check_mac_shapes(uint32_t d_out, uint32_t d_in) {
  if (d_out > (65535u * 8u)) return fail(CKKS_E_INVALID_ARG, "d_out=%u too large (max %u)", d_out, 65535u * 8u);
  if (d_in > ckks::kMaxMacDin) return fail(CKKS_E_INVALID_ARG, "d_in=%u too large (max %u)", d_in, ckks::kMaxMacDin);
  return CKKS_OK;
}

// The scalar MAC behind both entry points.  noalloc: the matrix-core workspace
// is the context device's library-owned scratch array instead of the caller's.
static int mac_scalar_impl(const ckks_ctx* ctx, const uint32_t* w_enc, const uint32_t* ct_in, uint32_t* ct_out,
                           uint32_t d_out, uint32_t d_in, uint32_t limbs, void* workspace, size_t workspace_bytes,
                           void* stream, bool noalloc) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (int rc = check_mac_shapes(d_out, d_in)) return rc;
  if (d_out == 0) return ok();
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t ct_row = size_t(2) * limbs * ctx->n * 4;  // bytes of one ciphertext
  const size_t out_b = size_t(d_out) * ct_row, in_b = size_t(d_in) * ct_row;
  const size_t w_b = size_t(d_out) * d_in * limbs * 4;
  if (d_in > 0) {
    if (int rc = check_ptr(w_enc, "w_enc")) return rc;
    if (int rc = check_ptr(ct_in, "ct_in")) return rc;
    if (overlaps(ct_out, out_b, ct_in, in_b) || overlaps(ct_out, out_b, w_enc, w_b))
      return fail(CKKS_E_INVALID_ARG, "ct_out overlaps ct_in or w_enc");
  }
  DeviceGuard guard(ctx->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (d_in == 0) {
    e = ckks::launch_zero(ct_out, static_cast<size_t>(d_out) * 2 * limbs * ctx->n, s);
    return e == hipSuccess ? ok() : hip_fail(e, "zero launch");
  }
  const bool mfma_ok = ckks::mac_mfma_supported(d_in);
  if (ctx->mac_algo == CKKS_MAC_MFMA && !mfma_ok)
    return fail(CKKS_E_UNSUPPORTED, "matrix-core MAC needs d_in <= 4096 (got %u)", d_in);
  const bool use_mfma = ctx->mac_algo == CKKS_MAC_MFMA || (ctx->mac_algo == CKKS_MAC_AUTO && mfma_ok);
  if (use_mfma) {
    const size_t need = ckks::mac_mfma_workspace_bytes(ctx->n, d_out, d_in, limbs);
    if (noalloc) {
      if (!ctx->scratch)
        return hip_fail(ctx->scratch_status, "no-allocation MAC scratch (hipGetSymbolAddress at context creation)");
      if (need > ckks::kNoAllocScratchBytes)
        return fail(CKKS_E_WORKSPACE,
                    "no-allocation MAC needs %zu bytes of scratch for d_out=%u, d_in=%u, limbs=%u; its array holds %zu",
                    need, d_out, d_in, limbs, ckks::kNoAllocScratchBytes);
      workspace = ctx->scratch;
      workspace_bytes = ckks::kNoAllocScratchBytes;
    }
    if (!workspace || workspace_bytes < need)
      return fail(CKKS_E_WORKSPACE, "MAC workspace %zu bytes < %zu required", workspace_bytes, need);
    if (!aligned16(workspace)) return fail(CKKS_E_INVALID_ARG, "workspace is not 16-byte aligned");
    if (overlaps(workspace, need, ct_out, out_b) || overlaps(workspace, need, ct_in, in_b) ||
        overlaps(workspace, need, w_enc, w_b))
      return fail(CKKS_E_INVALID_ARG, "workspace overlaps ct_in, ct_out or w_enc");
    e = ckks::launch_mac_scalar_mfma(ctx->t, w_enc, ct_in, ct_out, d_out, d_in, limbs, workspace, s);
  } else {
    e = ckks::launch_mac_scalar_valu(ctx->t, w_enc, ct_in, ct_out, d_out, d_in, limbs, s);
  }
  return e == hipSuccess ? ok() : hip_fail(e, "mac_scalar launch");
}

int ckks_linear_mac_scalar(const ckks_ctx* ctx, const uint32_t* w_enc, const uint32_t* ct_in,
                           uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                           void* workspace, size_t workspace_bytes, void* stream) {
  return mac_scalar_impl(ctx, w_enc, ct_in, ct_out, d_out, d_in, limbs, workspace, workspace_bytes, stream, false);
}

int ckks_linear_mac_scalar_noalloc(const ckks_ctx* ctx, const uint32_t* w_enc, const uint32_t* ct_in,
                                   uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs, void* stream) {
  return mac_scalar_impl(ctx, w_enc, ct_in, ct_out, d_out, d_in, limbs, nullptr, 0, stream, true);
}

int ckks_linear_mac_poly(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* ct_in,
                         uint32_t* ct_out, uint32_t d_out, uint32_t d_in, uint32_t limbs,
                         void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (d_out == 0) return ok();
  if (static_cast<uint64_t>(d_out) * limbs * (ctx->n / 256) > 0x7FFFFFFFull)
    return fail(CKKS_E_INVALID_ARG, "d_out=%u too large", d_out);
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  if (d_in > 0) {
    if (int rc = check_ptr(pt, "pt")) return rc;
    if (int rc = check_ptr(ct_in, "ct_in")) return rc;
    const size_t ct_row = size_t(2) * limbs * ctx->n * 4, out_b = size_t(d_out) * ct_row;
    if (overlaps(ct_out, out_b, ct_in, size_t(d_in) * ct_row) ||
        overlaps(ct_out, out_b, pt, size_t(d_out) * d_in * limbs * ctx->n * 4))
      return fail(CKKS_E_INVALID_ARG, "ct_out overlaps ct_in or pt");
  }
  DeviceGuard guard(ctx->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = d_in == 0 ? ckks::launch_zero(ct_out, static_cast<size_t>(d_out) * 2 * limbs * ctx->n, s)
                           : ckks::launch_mac_poly(ctx->t, pt, ct_in, ct_out, d_out, d_in, limbs, s);
  return e == hipSuccess ? ok() : hip_fail(e, "mac_poly launch");
}

int ckks_rescale(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t* ct_out, uint32_t count,
                 uint32_t limbs, void* workspace, size_t workspace_bytes, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 2)) return rc;
  if (count == 0) return ok();
  if (count > 0x3FFFFFFFu) return fail(CKKS_E_INVALID_ARG, "count=%u too large", count);
  if (int rc = check_ptr(ct_in, "ct_in")) return rc;
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t need = ckks::rescale_workspace_bytes(ctx->t, count, limbs);
  if (need && (!workspace || workspace_bytes < need))
    return fail(CKKS_E_WORKSPACE, "rescale workspace %zu bytes < %zu required", workspace_bytes, need);
  if (need && !aligned16(workspace)) return fail(CKKS_E_INVALID_ARG, "workspace is not 16-byte aligned");
  const size_t in_b = size_t(count) * 2 * limbs * ctx->n * 4, out_b = size_t(count) * 2 * (limbs - 1) * ctx->n * 4;
  if (overlaps(ct_out, out_b, ct_in, in_b)) return fail(CKKS_E_INVALID_ARG, "ct_out overlaps ct_in");
  if (need && (overlaps(workspace, need, ct_in, in_b) || overlaps(workspace, need, ct_out, out_b)))
    return fail(CKKS_E_INVALID_ARG, "workspace overlaps ct_in or ct_out");
  DeviceGuard guard(ctx->device);
  hipError_t e = ckks::launch_rescale(ctx->t, ct_in, ct_out, count, limbs, workspace,
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ok() : hip_fail(e, "rescale launch");
}

// Rows handed to the batched transforms must keep their grids below 2^31
// workgroups (64 per row in the N = 2^16 block pass).
static int check_rows(const ckks_ctx* ctx, uint32_t count, uint32_t limbs) {
  const size_t rows = static_cast<size_t>(count) * limbs;
  if (rows > 0x7FFFFFFFull / (ctx->log_n == 16 ? 64 : 1))
    return fail(CKKS_E_INVALID_ARG, "too many polynomials (%zu rows)", rows);
  return CKKS_OK;
}

int ckks_encrypt(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* s_ntt, const uint32_t* a,
                 const int32_t* e, uint32_t count, uint32_t limbs, uint32_t* ct, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (count == 0) return ok();
  if (int rc = check_rows(ctx, count, limbs)) return rc;
  if (int rc = check_ptr(s_ntt, "s_ntt")) return rc;
  if (int rc = check_ptr(a, "a")) return rc;
  if (int rc = check_ptr(e, "e")) return rc;
  if (int rc = check_ptr(ct, "ct")) return rc;
  if (pt && !aligned16(pt)) return fail(CKKS_E_INVALID_ARG, "pt is not 16-byte aligned");
  const size_t n = ctx->n, ct_bytes = size_t(count) * 2 * limbs * n * 4;
  if (overlaps(ct, ct_bytes, a, size_t(count) * limbs * n * 4) || overlaps(ct, ct_bytes, e, size_t(count) * n * 4) ||
      overlaps(ct, ct_bytes, s_ntt, size_t(limbs) * n * 4) || (pt && overlaps(ct, ct_bytes, pt, size_t(count) * limbs * n * 4)))
    return fail(CKKS_E_INVALID_ARG, "ct overlaps an input");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_encrypt(ctx->t, pt, s_ntt, a, e, count, limbs, ct, static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "encrypt launch");
}

int ckks_decrypt(const ckks_ctx* ctx, const uint32_t* ct, const uint32_t* s_ntt, uint32_t count, uint32_t limbs,
                 uint32_t* m, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (count == 0) return ok();
  if (int rc = check_rows(ctx, count, limbs)) return rc;
  if (int rc = check_ptr(ct, "ct")) return rc;
  if (int rc = check_ptr(s_ntt, "s_ntt")) return rc;
  if (int rc = check_ptr(m, "m")) return rc;
  const size_t n = ctx->n;
  if (overlaps(m, size_t(count) * limbs * n * 4, ct, size_t(count) * 2 * limbs * n * 4))
    return fail(CKKS_E_INVALID_ARG, "m overlaps ct");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_decrypt(ctx->t, ct, s_ntt, count, limbs, m, static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "decrypt launch");
}

int ckks_refresh(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t limbs_in, const uint32_t* s_ntt,
                 const uint32_t* a, const int32_t* e, uint32_t count, uint32_t limbs_out, uint32_t* ct_out,
                 void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs_in, 2)) return rc;
  if (int rc = check_limbs(ctx, limbs_out, 2)) return rc;
  if (count == 0) return ok();
  if (int rc = check_rows(ctx, count, limbs_in > limbs_out ? limbs_in : limbs_out)) return rc;
  if (int rc = check_ptr(ct_in, "ct_in")) return rc;
  if (int rc = check_ptr(s_ntt, "s_ntt")) return rc;
  if (int rc = check_ptr(a, "a")) return rc;
  if (int rc = check_ptr(e, "e")) return rc;
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t n = ctx->n, out_bytes = size_t(count) * 2 * limbs_out * n * 4;
  if (overlaps(ct_out, out_bytes, ct_in, size_t(count) * 2 * limbs_in * n * 4) ||
      overlaps(ct_out, out_bytes, a, size_t(count) * limbs_out * n * 4) ||
      overlaps(ct_out, out_bytes, e, size_t(count) * n * 4) || overlaps(ct_out, out_bytes, s_ntt, size_t(limbs_out) * n * 4))
    return fail(CKKS_E_INVALID_ARG, "ct_out overlaps an input");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_refresh(ctx->t, ct_in, limbs_in, s_ntt, a, e, count, limbs_out, ct_out,
                                       static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "refresh launch");
}

// ---- rotations and the BSGS product ----------------------------------------

static int check_ks_ctx(const ckks_ctx* ctx) {
  if (int rc = check_ctx(ctx)) return rc;
  if (ctx->L < 3) return fail(CKKS_E_INVALID_ARG, "key switching needs a context of at least 3 primes (got %u)", ctx->L);
  return CKKS_OK;
}

static bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255) == 0; }

int ckks_automorphism(const ckks_ctx* ctx, const uint32_t* in, uint32_t rows, uint32_t galois, uint32_t* out,
                      void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if ((galois & 1) == 0 || galois >= 2 * ctx->n) return fail(CKKS_E_INVALID_ARG, "galois=%u not odd below 2N", galois);
  if (rows == 0) return ok();
  if (int rc = check_ptr(in, "in")) return rc;
  if (int rc = check_ptr(out, "out")) return rc;
  const size_t bytes = size_t(rows) * ctx->n * 4;
  if (overlaps(in, bytes, out, bytes)) return fail(CKKS_E_INVALID_ARG, "out overlaps in");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_automorphism(ctx->t, in, rows, galois, out, static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "automorphism launch");
}

int ckks_keygen_rotation(const ckks_ctx* ctx, const uint32_t* s_ntt, uint32_t r0, uint32_t r_step, uint32_t count,
                         const uint32_t* a, const int32_t* e, uint32_t* ksk, void* stream) {
  if (int rc = check_ks_ctx(ctx)) return rc;
  if (count == 0) return ok();
  const size_t L = ctx->L, Lk = L - 1, n = ctx->n;
  if (int rc = check_rows(ctx, count, static_cast<uint32_t>(Lk * L))) return rc;
  if (int rc = check_ptr(s_ntt, "s_ntt")) return rc;
  if (int rc = check_ptr(a, "a")) return rc;
  if (int rc = check_ptr(e, "e")) return rc;
  if (int rc = check_ptr(ksk, "ksk")) return rc;
  const size_t kb = size_t(count) * Lk * 2 * L * n * 4;
  if (overlaps(ksk, kb, s_ntt, L * n * 4) || overlaps(ksk, kb, a, size_t(count) * Lk * L * n * 4) ||
      overlaps(ksk, kb, e, size_t(count) * Lk * n * 4))
    return fail(CKKS_E_INVALID_ARG, "ksk overlaps an input");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_keygen_rotation(ctx->t, s_ntt, r0, r_step, count, a, e, ksk,
                                               static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "keygen_rotation launch");
}

int ckks_rotate(const ckks_ctx* ctx, const uint32_t* ct_in, uint32_t count, uint32_t r0, uint32_t r_step,
                int hoisted, const uint32_t* ksk, void* workspace, size_t workspace_bytes, uint32_t* ct_out,
                void* stream) {
  if (int rc = check_ks_ctx(ctx)) return rc;
  if (hoisted != 0 && hoisted != 1) return fail(CKKS_E_INVALID_ARG, "hoisted=%d not 0 or 1", hoisted);
  if (count == 0) return ok();
  const size_t L = ctx->L, Lk = L - 1, n = ctx->n;
  if (int rc = check_rows(ctx, count, static_cast<uint32_t>(Lk * L))) return rc;
  if (int rc = check_ptr(ct_in, "ct_in")) return rc;
  if (int rc = check_ptr(ksk, "ksk")) return rc;
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t need = ckks::rotate_workspace_bytes(ctx->t, hoisted ? 1 : count, count);
  if (!workspace || workspace_bytes < need)
    return fail(CKKS_E_WORKSPACE, "rotate workspace %zu bytes < %zu required", workspace_bytes, need);
  if (!aligned256(workspace)) return fail(CKKS_E_INVALID_ARG, "workspace is not 256-byte aligned");
  const size_t ctb = 2 * Lk * n * 4, out_b = size_t(count) * ctb;
  const size_t in_b = (hoisted ? 1 : size_t(count)) * ctb;
  if (overlaps(ct_out, out_b, ct_in, in_b) || overlaps(ct_out, out_b, ksk, size_t(count) * Lk * 2 * L * n * 4) ||
      overlaps(workspace, need, ct_in, in_b) || overlaps(workspace, need, ct_out, out_b))
    return fail(CKKS_E_INVALID_ARG, "ct_out or workspace overlaps another buffer");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_rotate(ctx->t, ct_in, count, r0, r_step, 0, hoisted == 1, ksk, workspace, ct_out,
                                      static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "rotate launch");
}

size_t ckks_bsgs_workspace_bytes(const ckks_ctx* ctx, uint32_t count, uint32_t n1, uint32_t n2) {
  if (!ctx || ctx->L < 3 || n1 == 0 || n2 == 0 || n1 > 65536 || n2 > 65536) return static_cast<size_t>(-1);
  return ckks::bsgs_workspace_bytes(ctx->t, count, n1, n2);
}

int ckks_linear_bsgs(const ckks_ctx* ctx, const uint32_t* pt, const uint32_t* ct_in, uint32_t count, uint32_t n1,
                     uint32_t n2, const uint32_t* ksk, void* workspace, size_t workspace_bytes, uint32_t* ct_out,
                     void* stream) {
  if (int rc = check_ks_ctx(ctx)) return rc;
  const size_t L = ctx->L, Lk = L - 1, n = ctx->n;
  if (n1 == 0 || n2 == 0 || size_t(n1) * n2 > n / 2)
    return fail(CKKS_E_INVALID_ARG, "n1=%u, n2=%u: need n1, n2 >= 1 and n1 n2 <= N/2", n1, n2);
  if (count == 0) return ok();
  if (int rc = check_rows(ctx, count, static_cast<uint32_t>(Lk * L * (n1 > n2 ? n1 : n2)))) return rc;
  if (static_cast<uint64_t>(n2) * Lk * (n / 256) > 0x7FFFFFFFull) return fail(CKKS_E_INVALID_ARG, "n2=%u too large", n2);
  if (int rc = check_ptr(pt, "pt")) return rc;
  if (int rc = check_ptr(ct_in, "ct_in")) return rc;
  if (n1 + n2 > 2 && check_ptr(ksk, "ksk")) return CKKS_E_INVALID_ARG;
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t need = ckks::bsgs_workspace_bytes(ctx->t, count, n1, n2);
  if (!workspace || workspace_bytes < need)
    return fail(CKKS_E_WORKSPACE, "bsgs workspace %zu bytes < %zu required", workspace_bytes, need);
  if (!aligned256(workspace)) return fail(CKKS_E_INVALID_ARG, "workspace is not 256-byte aligned");
  const size_t in_b = size_t(count) * 2 * Lk * n * 4, out_b = size_t(count) * 2 * (Lk - 1) * n * 4;
  if (overlaps(ct_out, out_b, ct_in, in_b) || overlaps(ct_out, out_b, pt, size_t(n1) * n2 * Lk * n * 4) ||
      overlaps(workspace, need, ct_in, in_b) || overlaps(workspace, need, ct_out, out_b) ||
      overlaps(workspace, need, pt, size_t(n1) * n2 * Lk * n * 4))
    return fail(CKKS_E_INVALID_ARG, "ct_out or workspace overlaps another buffer");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_bsgs(ctx->t, pt, ct_in, count, n1, n2, ksk, workspace, ct_out,
                                    static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "bsgs launch");
}

int ckks_add(const ckks_ctx* ctx, const uint32_t* ct_a, const uint32_t* ct_b, uint32_t count, uint32_t limbs,
             uint32_t* ct_out, void* stream) {
  if (int rc = check_ctx(ctx)) return rc;
  if (int rc = check_limbs(ctx, limbs, 1)) return rc;
  if (count == 0) return ok();
  if (int rc = check_rows(ctx, count, 2 * limbs)) return rc;
  if (int rc = check_ptr(ct_a, "ct_a")) return rc;
  if (int rc = check_ptr(ct_b, "ct_b")) return rc;
  if (int rc = check_ptr(ct_out, "ct_out")) return rc;
  const size_t bytes = size_t(count) * 2 * limbs * ctx->n * 4;
  if ((ct_out != ct_a && overlaps(ct_out, bytes, ct_a, bytes)) || (ct_out != ct_b && overlaps(ct_out, bytes, ct_b, bytes)))
    return fail(CKKS_E_INVALID_ARG, "ct_out partially overlaps an input");
  DeviceGuard guard(ctx->device);
  hipError_t he = ckks::launch_ct_add(ctx->t, ct_a, ct_b, count, limbs, ct_out, static_cast<hipStream_t>(stream));
  return he == hipSuccess ? ok() : hip_fail(he, "add launch");
}

size_t ckks_workspace_bytes(const ckks_ctx* ctx, int op, uint32_t a, uint32_t b, uint32_t limbs) {
  if (!ctx || limbs < 1 || limbs > ctx->L) return static_cast<size_t>(-1);
  switch (op) {
    case CKKS_OP_MAC_SCALAR:
      return ctx->mac_algo == CKKS_MAC_VALU ? 0 : ckks::mac_mfma_workspace_bytes(ctx->n, a, b, limbs);
    case CKKS_OP_RESCALE:
      return limbs < 2 ? static_cast<size_t>(-1) : ckks::rescale_workspace_bytes(ctx->t, a, limbs);
    case CKKS_OP_ENCODE_POLY:
      return 0;
    case CKKS_OP_ROTATE:
      if (ctx->L < 3 || limbs != ctx->L - 1 || b > 1) return static_cast<size_t>(-1);
      return ckks::rotate_workspace_bytes(ctx->t, b ? 1 : a, a);
    default:
      return static_cast<size_t>(-1);
  }
}

double ckks_rescaled_scale(const ckks_ctx* ctx, double scale_in, uint32_t limbs) {
  if (!ctx || limbs < 2 || limbs > ctx->L) return NAN;
  return scale_in / static_cast<double>(ctx->q[limbs - 1]);
}

const char* ckks_last_error(void) { return g_err.c_str(); }

}  // extern "C"
