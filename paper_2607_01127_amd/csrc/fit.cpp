// Host side of liblogbq: the per-tensor fit (Sec. 3.1 Eq. 3-4, Sec. 3.2 Eq. 5), the exact
// encoding thresholds, status strings.
//
// Built with g++ -O2 -ffp-contract=off and without -ffast-math: every float64 operation
// below must round exactly as written (no fused multiply-add, no reassociation), because
// the fitted parameters are compared bit for bit with an independent implementation.

#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <new>
#include <system_error>
#include <thread>
#include <vector>

#include "fit_detail.h"
#include "logbq.h"

namespace {

inline uint32_t f2u(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }
inline float u2f(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }

// LSD radix sort of non-negative float32 bit patterns (their integer order is their value
// order). Three 11-bit passes; passes whose digit is constant over the input are skipped. Each
// pass splits the input into T contiguous ranges: per-range digit counts give every (range,
// digit) its own output offsets, and each range is scattered in order, so the sort is stable
// and its result is the same for any T.
// Ranges per pass: LOGBQ_HOST_THREADS (1..16) when set, else the hardware threads (at most
// 16); one range below 2^20 weights.
unsigned sort_ranges(size_t n) {
  unsigned nt = std::thread::hardware_concurrency();
  if (const char* env = std::getenv("LOGBQ_HOST_THREADS")) {
    const long v = std::strtol(env, nullptr, 10);
    if (v >= 1) nt = (unsigned)v;
  }
  nt = nt < 1 ? 1 : (nt > 16 ? 16 : nt);
  if (n < (size_t(1) << 20)) nt = 1;
  return nt;
}

void radix_sort_u32(std::vector<uint32_t>& a) {
  const size_t n = a.size();
  const unsigned nt = sort_ranges(n);
  std::vector<uint32_t> tmp(n);
  uint32_t* src = a.data();
  uint32_t* dst = tmp.data();
  std::vector<size_t> cnt((size_t)nt * 2048);
  // Range t runs on a thread of its own, or on the calling thread when no thread can be
  // started (the ranges are independent, so the result does not depend on where they run).
  auto run = [&](auto&& fn) {
    if (nt == 1) { fn(0u); return; }
    std::vector<std::thread> th;
    th.reserve(nt);
    unsigned started = 0;
    try {
      for (; started < nt; ++started) th.emplace_back(fn, started);
    } catch (const std::system_error&) {
    }
    for (unsigned t = started; t < nt; ++t) fn(t);
    for (auto& x : th) x.join();
  };
  auto lo = [&](unsigned t) { return n * t / nt; };
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass * 11;
    std::fill(cnt.begin(), cnt.end(), size_t(0));
    run([&](unsigned t) {
      size_t* c = cnt.data() + (size_t)t * 2048;
      for (size_t i = lo(t); i < lo(t + 1); ++i) c[(src[i] >> shift) & 2047u]++;
    });
    bool constant = false;
    size_t next = 0;
    for (int d = 0; d < 2048; ++d) {
      size_t tot = 0;
      for (unsigned t = 0; t < nt; ++t) {
        const size_t c = cnt[(size_t)t * 2048 + d];
        cnt[(size_t)t * 2048 + d] = next + tot;   // output offset of (range t, digit d)
        tot += c;
      }
      if (tot == n) constant = true;
      next += tot;
    }
    if (constant) continue;
    run([&](unsigned t) {
      size_t* o = cnt.data() + (size_t)t * 2048;
      for (size_t i = lo(t); i < lo(t + 1); ++i) dst[o[(src[i] >> shift) & 2047u]++] = src[i];
    });
    std::swap(src, dst);
  }
  if (src != a.data()) std::memcpy(a.data(), src, n * sizeof(uint32_t));
}

// ---- small unsigned big integer, enough for exact threshold tests -----------------------
struct Big {
  std::vector<uint32_t> d;  // little-endian 32-bit limbs
  explicit Big(uint64_t v = 0) { while (v) { d.push_back(uint32_t(v)); v >>= 32; } }
  void mul_small(uint64_t m) {  // m < 2^64
    const uint32_t mlo = uint32_t(m), mhi = uint32_t(m >> 32);
    std::vector<uint32_t> r(d.size() + 3, 0);
    for (size_t i = 0; i < d.size(); ++i) {
      unsigned __int128 carry = 0;
      unsigned __int128 t = (unsigned __int128)d[i] * mlo + r[i] + carry;
      r[i] = uint32_t(t);
      carry = t >> 32;
      t = (unsigned __int128)d[i] * mhi + r[i + 1] + carry;
      r[i + 1] = uint32_t(t);
      carry = t >> 32;
      size_t j = i + 2;
      while (carry) { t = (unsigned __int128)r[j] + carry; r[j] = uint32_t(t); carry = t >> 32; ++j; }
    }
    d.swap(r);
    trim();
  }
  void shl(int64_t bits) {
    if (d.empty() || bits <= 0) return;
    const size_t limbs = size_t(bits / 32);
    const int rem = int(bits % 32);
    std::vector<uint32_t> r(d.size() + limbs + 1, 0);
    for (size_t i = 0; i < d.size(); ++i) {
      uint64_t v = uint64_t(d[i]) << rem;
      r[i + limbs] |= uint32_t(v);
      r[i + limbs + 1] |= uint32_t(v >> 32);
    }
    d.swap(r);
    trim();
  }
  void add(const Big& o) {
    if (o.d.size() > d.size()) d.resize(o.d.size(), 0);
    uint64_t carry = 0;
    for (size_t i = 0; i < d.size(); ++i) {
      const uint64_t t = uint64_t(d[i]) + (i < o.d.size() ? o.d[i] : 0u) + carry;
      d[i] = uint32_t(t);
      carry = t >> 32;
    }
    if (carry) d.push_back(uint32_t(carry));
  }
  Big mul(const Big& o) const {
    Big r;
    if (d.empty() || o.d.empty()) return r;
    r.d.assign(d.size() + o.d.size(), 0);
    for (size_t i = 0; i < d.size(); ++i) {
      uint64_t carry = 0;
      for (size_t j = 0; j < o.d.size(); ++j) {
        const uint64_t t = uint64_t(d[i]) * o.d[j] + r.d[i + j] + carry;
        r.d[i + j] = uint32_t(t);
        carry = t >> 32;
      }
      size_t k = i + o.d.size();
      while (carry) {
        const uint64_t t = uint64_t(r.d[k]) + carry;
        r.d[k] = uint32_t(t);
        carry = t >> 32;
        ++k;
      }
    }
    r.trim();
    return r;
  }
  // floor(this / 2^bits), plus one if any discarded bit was set (the ceiling).
  void shr_ceil(int64_t bits) {
    if (d.empty() || bits <= 0) return;
    const size_t limbs = size_t(bits / 32);
    const int rem = int(bits % 32);
    bool lost = false;
    for (size_t i = 0; i < limbs && i < d.size(); ++i) lost |= d[i] != 0;
    if (limbs < d.size() && rem) lost |= (d[limbs] & ((1u << rem) - 1u)) != 0;
    std::vector<uint32_t> r(d.size() > limbs ? d.size() - limbs : 0, 0);
    for (size_t i = 0; i < r.size(); ++i) {
      uint64_t v = d[i + limbs] >> rem;
      if (rem && i + limbs + 1 < d.size()) v |= uint64_t(d[i + limbs + 1]) << (32 - rem);
      r[i] = uint32_t(v);
    }
    d.swap(r);
    trim();
    if (lost) add(Big(1));
  }
  void trim() { while (!d.empty() && d.back() == 0) d.pop_back(); }
  static int cmp(const Big& a, const Big& b) {
    if (a.d.size() != b.d.size()) return a.d.size() < b.d.size() ? -1 : 1;
    for (size_t i = a.d.size(); i-- > 0;)
      if (a.d[i] != b.d[i]) return a.d[i] < b.d[i] ? -1 : 1;
    return 0;
  }
};

// f = F * 2^ef for a finite non-negative float32.
void split_f32(float f, uint64_t& F, int64_t& ef) {
  const uint32_t u = f2u(f);
  const uint32_t e = (u >> 23) & 0xFFu, m = u & 0x7FFFFFu;
  if (e == 0) { F = m; ef = -149; }
  else { F = m | 0x800000u; ef = int64_t(e) - 150; }
}

// b = B * 2^eb for a finite positive double.
void split_f64(double b, uint64_t& B, int64_t& eb) {
  uint64_t u; std::memcpy(&u, &b, 8);
  const uint64_t e = (u >> 52) & 0x7FFu, m = u & ((uint64_t(1) << 52) - 1);
  if (e == 0) { B = m; eb = -1074; }
  else { B = m | (uint64_t(1) << 52); eb = int64_t(e) - 1075; }
}

// B^e (e >= 0) by repeated squaring.
Big pow_big(uint64_t B, int64_t e) {
  Big r(1), x(B);
  while (e > 0) {
    if (e & 1) r = r.mul(x);
    e >>= 1;
    if (e > 0) x = x.mul(x);
  }
  return r;
}

// Exact test f >= b^(n/2) for odd n, i.e. f^2 >= b^n (f >= 0 finite, b > 1 finite), given
// pw = B^|n| where b = B 2^eb.
bool ge_half_power(float f, double b, int64_t n, const Big& pw) {
  uint64_t F, B; int64_t ef, eb;
  split_f32(f, F, ef);
  if (F == 0) return false;
  split_f64(b, B, eb);
  if (n >= 0) {
    // F^2 2^(2ef) >= B^n 2^(n eb)
    Big lhs(F); lhs.mul_small(F);
    Big rhs = pw;
    const int64_t d = 2 * ef - n * eb;
    if (d >= 0) lhs.shl(d); else rhs.shl(-d);
    return Big::cmp(lhs, rhs) >= 0;
  }
  // F^2 2^(2ef) B^m 2^(m eb) >= 1  with m = -n
  const int64_t m = -n;
  Big lhs = pw;
  lhs.mul_small(F);
  lhs.mul_small(F);
  const int64_t e = -2 * ef - m * eb;   // need lhs >= 2^e
  if (e <= 0) return true;              // lhs >= 1
  Big rhs(1); rhs.shl(e);
  return Big::cmp(lhs, rhs) >= 0;
}

// Smallest float32 t with t >= b^(k + 1/2 - s); +inf beyond the float32 range. pw = B^|n| for
// n = 2k + 1 - 2s, b = B 2^eb.
float exact_threshold(double b, int32_t s, int k, const Big& pw) {
  const int64_t n = 2 * int64_t(k) + 1 - 2 * int64_t(s);
  const long double approx = powl((long double)b, (long double)k + 0.5L - (long double)s);
  if (!(approx <= (long double)FLT_MAX * 2)) return std::numeric_limits<float>::infinity();
  float f = approx > (long double)FLT_MAX ? FLT_MAX : (float)approx;
  const float inf = std::numeric_limits<float>::infinity();
  while (!ge_half_power(f, b, n, pw)) {
    f = std::nextafter(f, inf);
    if (std::isinf(f)) return f;
  }
  while (f > 0.0f) {
    const float g = std::nextafter(f, 0.0f);
    if (ge_half_power(g, b, n, pw)) f = g; else break;
  }
  return f;
}

// Code of x under the asymmetric linear quantizer: round(x / s) - z with ties up, clamped.
int uniform_code(float x, double s, int32_t z) {
  const double v = (double)x / s;
  if (std::isnan(v)) return 0;
  if (std::isinf(v)) return v > 0 ? 15 : 0;
  const double q = std::floor(v + 0.5) - (double)z;
  return q < 0.0 ? 0 : (q > 15.0 ? 15 : (int)q);
}

// Smallest float32 whose code is at least j: start at the real boundary s (j + z - 1/2) and
// walk neighbouring float32 values (the code is non-decreasing in x).
float uniform_threshold(double s, int32_t z, int j) {
  float t = (float)(s * ((double)j + (double)z - 0.5));
  if (!std::isfinite(t)) return t;
  while (uniform_code(t, s, z) >= j) t = std::nextafterf(t, -INFINITY);
  while (uniform_code(t, s, z) < j) {
    t = std::nextafterf(t, INFINITY);
    if (!std::isfinite(t)) break;
  }
  return t;
}

int32_t finish_params(int32_t bits, double eps, double wmin, double wmax, int64_t istar,
                      logbq_params* out);

}  // namespace

extern "C" {

int32_t logbq_fit_uniform(const float* w_host, int64_t numel, int32_t bits, logbq_uniform* out) {
  if (!w_host || !out || numel < 2) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4) return LOGBQ_ERR_UNSUPPORTED;
  float lo = INFINITY, hi = -INFINITY;
  for (int64_t i = 0; i < numel; ++i) {
    const float v = w_host[i];
    if (!std::isfinite(v)) return LOGBQ_ERR_NONFINITE;
    lo = v < lo ? v : lo;
    hi = v > hi ? v : hi;
  }
  if (!(hi > lo)) return LOGBQ_ERR_DEGENERATE;
  const double s = ((double)hi - (double)lo) / 15.0;
  const double zf = std::floor((double)lo / s + 0.5);
  if (!(zf > -1e9 && zf < 1e9)) return LOGBQ_ERR_DEGENERATE;
  logbq_uniform u;
  std::memset(&u, 0, sizeof(u));
  u.bits = bits;
  u.zero = (int32_t)zf;
  u.wmin = lo;
  u.wmax = hi;
  u.scale = s;
  for (int q = 0; q < 16; ++q) u.codebook[q] = (float)(s * (double)(q + u.zero));
  for (int j = 1; j < 16; ++j) u.thresholds[j - 1] = uniform_threshold(s, u.zero, j);
  *out = u;
  return LOGBQ_OK;
}


int32_t logbq_abi_version(void) { return LOGBQ_ABI_VERSION; }

const char* logbq_status_str(int32_t status) {
  switch (status) {
    case LOGBQ_OK: return "ok";
    case LOGBQ_ERR_INVALID_ARG: return "invalid argument";
    case LOGBQ_ERR_NONFINITE: return "non-finite weight";
    case LOGBQ_ERR_DEGENERATE: return "degenerate weight range";
    case LOGBQ_ERR_UNSUPPORTED: return "unsupported shape, alignment or bit width";
    case LOGBQ_ERR_HIP: return "HIP runtime error";
    case LOGBQ_ERR_HOST_RESOURCE: return "host memory could not be allocated";
    default: return "unknown status";
  }
}

}  // extern "C"

namespace {

int32_t fit_sequential(const float* w_host, int64_t numel, int32_t bits, double eps,
                       logbq_params* out) {

  // |w| as float32 bit patterns (sign cleared); reject NaN / Inf.
  std::vector<uint32_t> a((size_t)numel);
  for (int64_t i = 0; i < numel; ++i) {
    const uint32_t u = f2u(w_host[i]) & 0x7FFFFFFFu;
    if (u >= 0x7F800000u) return LOGBQ_ERR_NONFINITE;
    a[(size_t)i] = u;
  }
  radix_sort_u32(a);
  const double wmax = (double)u2f(a.back());
  if (wmax == 0.0) return LOGBQ_ERR_DEGENERATE;

  // Eq. 5 with sequential float64 prefix sums in ascending |w| order; squares of float32
  // values are exact in float64.
  double total = 0.0;
  for (size_t i = 0; i < a.size(); ++i) {
    const double v = (double)u2f(a[i]);
    total += v * v;
  }
  double prefix = 0.0;
  size_t istar = a.size() - 1;
  for (size_t i = 0; i < a.size(); ++i) {
    const double v = (double)u2f(a[i]);
    prefix += v * v;
    if (prefix / total >= eps) { istar = i; break; }
  }
  const double wmin = (double)u2f(a[istar]);
  return finish_params(bits, eps, wmin, wmax, (int64_t)istar, out);
}

}  // namespace

extern "C" int32_t logbq_fit(const float* w_host, int64_t numel, int32_t bits, double eps,
                             logbq_params* out) {
  if (!w_host || !out || numel < 2) return LOGBQ_ERR_INVALID_ARG;
  if (!(eps > 0.0 && eps < 1.0)) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  try {
    return fit_sequential(w_host, numel, bits, eps, out);
  } catch (...) {   // host scratch (4 numel bytes twice) could not be allocated
    return LOGBQ_ERR_HOST_RESOURCE;
  }
}

namespace {

// Eq. 3 and Eq. 4 from w_min and w_max, then the codebook (Eq. 2) and the exact thresholds.
int32_t finish_params(int32_t bits, double eps, double wmin, double wmax, int64_t istar,
                      logbq_params* out) {
  const int32_t qmax = (1 << (bits - 1)) - 1;
  if (!(wmin < wmax)) return LOGBQ_ERR_DEGENERATE;

  // Eq. 3 and Eq. 4 (floor taken exactly: largest J with b^J <= w_max).
  const double b = std::pow(wmax / wmin, 1.0 / (double)qmax);
  if (!(b > 1.0)) return LOGBQ_ERR_DEGENERATE;
  int64_t J = (int64_t)std::floor(std::log(wmax) / std::log(b));
  while (std::pow(b, (double)(J + 1)) <= wmax) ++J;
  while (std::pow(b, (double)J) > wmax) --J;
  const int64_t s = qmax - J;
  if (s > INT32_MAX / 4 || s < INT32_MIN / 4) return LOGBQ_ERR_DEGENERATE;

  logbq_params p;
  std::memset(&p, 0, sizeof(p));
  p.bits = bits;
  p.qmax = qmax;
  p.eps = eps;
  p.wmin = wmin;
  p.wmax = wmax;
  p.base = b;
  p.shift = (int32_t)s;
  p.wmin_index = istar;
  const int half = 1 << (bits - 1);
  for (int k = 1; k <= qmax; ++k) {
    const float v = (float)std::pow(b, (double)(k - p.shift));
    p.codebook[k] = v;
    p.codebook[half + k] = -v;
  }
  p.codebook[0] = 0.0f;
  p.codebook[half] = 0.0f;
  const int nthr = (int)(sizeof(p.thresholds) / sizeof(p.thresholds[0]));
  for (int k = qmax; k < nthr; ++k) p.thresholds[k] = std::numeric_limits<float>::infinity();
  // B^|n_k| for n_k = 2k + 1 - 2s (odd, never 0). The k with n_k > 0 are taken upward from the
  // smallest such k, those with n_k < 0 downward from the largest: |n_k| grows by 2 per step
  // in both sweeps, so each sweep squares once and then multiplies by B^2 per step.
  uint64_t B;
  int64_t eb;
  split_f64(b, B, eb);
  auto nk = [&](int k) { return 2 * int64_t(k) + 1 - 2 * int64_t(p.shift); };
  int kpos = 0;
  while (kpos < qmax && nk(kpos) < 0) ++kpos;
  if (kpos < qmax) {
    Big pw = pow_big(B, nk(kpos));
    for (int k = kpos; k < qmax; ++k) {
      if (k > kpos) {
        pw.mul_small(B);
        pw.mul_small(B);
      }
      p.thresholds[k] = exact_threshold(b, p.shift, k, pw);
    }
  }
  if (kpos > 0) {
    Big pw = pow_big(B, -nk(kpos - 1));
    for (int k = kpos - 1; k >= 0; --k) {
      if (k < kpos - 1) {
        pw.mul_small(B);
        pw.mul_small(B);
      }
      p.thresholds[k] = exact_threshold(b, p.shift, k, pw);
    }
  }
  *out = p;
  return LOGBQ_OK;
}

}  // namespace

// ---- exact selection of the device fit ---------------------------------------------------

namespace {

// Energy of a bin in units of 2^-298 (the square of the smallest float32 subnormal):
// (hi * 2^24 + lo) * 2^(2 ef + 298), where |w| = m * 2^ef for every weight of the bin.
Big bin_energy(uint64_t hi, uint64_t lo, uint32_t exp_field) {
  const int64_t ef = exp_field == 0 ? -149 : int64_t(exp_field) - 150;
  Big e(hi);
  e.shl(24);
  e.add(Big(lo));
  e.shl(2 * ef + 298);
  return e;
}

}  // namespace

namespace logbq_detail {

int32_t fit_from_passes(int32_t bits, double eps, FitPassFn run, void* ctx, logbq_params* out) {
  FitPassResult r{};
  int32_t st = run(ctx, 1, 0, &r);
  if (st != LOGBQ_OK) return st;
  if (r.nonfinite) return LOGBQ_ERR_NONFINITE;
  if (r.max_key == 0) return LOGBQ_ERR_DEGENERATE;
  const double wmax = (double)u2f(r.max_key);

  // eps = N 2^e exactly (e < 0): an integer energy P reaches eps T iff P 2^-e >= N T, i.e.
  // iff P >= ceil(N T 2^e).
  uint64_t N;
  int64_t e;
  split_f64(eps, N, e);
  Big total;
  for (int b = 0; b < kFitBins1; ++b)
    if (r.bins[3 * b]) total.add(bin_energy(r.bins[3 * b + 1], r.bins[3 * b + 2], uint32_t(b) >> 3));
  Big target = total;
  target.mul_small(N);
  target.shr_ceil(-e);
  auto reaches = [&](const Big& p) { return Big::cmp(p, target) >= 0; };

  // Energy and count of all weights below the current selection.
  Big below;
  uint64_t count_below = 0;
  // First bin at which the running energy reaches the target; below / count_below then cover
  // the bins before it.
  auto pick = [&](const FitPassResult& pr, int nbins, uint32_t exp_field, bool per_bin_exp) {
    for (int b = 0; b < nbins; ++b) {
      const uint64_t* w = pr.bins + 3 * b;
      if (w[0] == 0) continue;
      Big run_e = below;
      run_e.add(bin_energy(w[1], w[2], per_bin_exp ? uint32_t(b) >> 3 : exp_field));
      if (reaches(run_e)) return b;
      below.d.swap(run_e.d);
      count_below += w[0];
    }
    return -1;
  };

  const int b1 = pick(r, kFitBins1, 0, true);
  if (b1 < 0) return LOGBQ_ERR_HIP;
  const uint32_t exp_field = uint32_t(b1) >> 3;
  st = run(ctx, 2, uint32_t(b1), &r);
  if (st != LOGBQ_OK) return st;
  const int b2 = pick(r, kFitBins2, exp_field, false);
  if (b2 < 0) return LOGBQ_ERR_HIP;
  const uint32_t sel = (uint32_t(b1) << 9) | uint32_t(b2);
  st = run(ctx, 3, sel, &r);
  if (st != LOGBQ_OK) return st;
  const int b3 = pick(r, kFitBins3, exp_field, false);
  if (b3 < 0) return LOGBQ_ERR_HIP;

  // w_min is the value of the chosen single-value bin; its position is the first of its
  // copies at which the running energy reaches the target.
  const uint32_t key = (sel << 11) | uint32_t(b3);
  const uint64_t copies = r.bins[3 * b3];
  uint64_t F;
  int64_t ef;
  split_f32(u2f(key), F, ef);
  Big v2(F);
  v2.mul_small(F);
  v2.shl(2 * ef + 298);
  uint64_t lo = 1, hi = copies;   // reaches(below + copies v^2) holds
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo) / 2;
    Big p = v2;
    p.mul_small(mid);
    p.add(below);
    if (reaches(p)) hi = mid; else lo = mid + 1;
  }
  const int64_t istar = (int64_t)(count_below + lo - 1);
  return finish_params(bits, eps, (double)u2f(key), wmax, istar, out);
}

}  // namespace logbq_detail

// ---- the device fit's passes on the host -------------------------------------------------

namespace {

struct HostPassCtx {
  const float* w;
  int64_t n;
  std::vector<uint64_t> bins;
};

// The three radix-selection passes of fit_detail.h over host weights, one weight at a time.
int32_t host_pass(void* vctx, int pass, uint32_t sel, logbq_detail::FitPassResult* res) {
  HostPassCtx& c = *static_cast<HostPassCtx*>(vctx);
  const int nb = pass == 1 ? logbq_detail::kFitBins1
               : pass == 2 ? logbq_detail::kFitBins2 : logbq_detail::kFitBins3;
  c.bins.assign(3 * (size_t)nb, 0);
  uint32_t kmax = 0, bad = 0;
  for (int64_t i = 0; i < c.n; ++i) {
    const uint32_t key = f2u(c.w[i]) & 0x7FFFFFFFu;
    uint32_t bin;
    if (pass == 1) {
      kmax = key > kmax ? key : kmax;
      bad |= key >= 0x7F800000u ? 1u : 0u;
      bin = key >> 20;
    } else if (pass == 2) {
      if ((key >> 20) != sel) continue;
      bin = (key >> 11) & 0x1FFu;
    } else {
      if ((key >> 11) != sel) continue;
      bin = key & 0x7FFu;
    }
    const uint64_t m = (key & 0x7FFFFFu) | (key >= 0x800000u ? 0x800000u : 0u);
    const uint64_t q = m * m;
    c.bins[3 * bin] += 1;
    c.bins[3 * bin + 1] += q >> 24;
    c.bins[3 * bin + 2] += q & 0xFFFFFFu;
  }
  res->bins = c.bins.data();
  res->max_key = kmax;
  res->nonfinite = bad;
  return LOGBQ_OK;
}

}  // namespace

extern "C" int32_t logbq_fit_exact(const float* w_host, int64_t numel, int32_t bits, double eps,
                                   logbq_params* out) {
  if (!w_host || !out || numel < 2) return LOGBQ_ERR_INVALID_ARG;
  if (!(eps > 0.0 && eps < 1.0)) return LOGBQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return LOGBQ_ERR_UNSUPPORTED;
  if (numel >= (int64_t(1) << 40)) return LOGBQ_ERR_UNSUPPORTED;
  try {
    HostPassCtx c{w_host, numel, {}};
    return logbq_detail::fit_from_passes(bits, eps, host_pass, &c, out);
  } catch (...) {   // host scratch could not be allocated
    return LOGBQ_ERR_HOST_RESOURCE;
  }
}
