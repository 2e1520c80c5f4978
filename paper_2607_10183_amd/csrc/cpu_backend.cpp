// Host-CPU backend of the hybrid execution (Sec. 4.3-4.4: a tensor the
// placement keeps off the GPU runs on the host CPU unless the round promotes
// it).  The product is the block-int4 linear of Sec. 4.1: y[m][n] =
// sum_k (u[n][k] - 8) * s[n][k/32] * x[m][k] with fp32 sums; outputs are
// rounded to fp16 (round to nearest even) by the caller's epilogue.
//
// Layout of the hot loop (AVX2): one 16-byte load gives a group's 32 codes;
// the low nibbles are the 16 even inputs and the high nibbles the 16 odd
// ones, so the activations are re-ordered once per call to match (the 16
// even inputs of a group, then its 16 odd inputs) and each code byte is used
// where it lies.  Codes become exact signed integers (u - 8) before the
// conversion to fp32, so no offset correction is subtracted later.  Up to
// four tokens share each unpacked group.  CPUs without AVX2/FMA/F16C take a
// plain loop with the same sums per group.
#include "cpu_backend.h"

#include <immintrin.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>

#include "../../include/atsi.h"

namespace atsi {
namespace cpu {

// ---------------------------------------------------------------- pool

// Waiting for the next job: pause-spin briefly, then yield the core (so that
// under oversubscription a preempted thread of this pool gets it), then sleep.
constexpr auto kPauseSpin = std::chrono::microseconds(20);
constexpr auto kYieldSpin = std::chrono::microseconds(2000);

Pool::Pool(int threads) : n_(std::max(1, threads)) {
  for (int i = 1; i < n_; ++i) threads_.emplace_back(&Pool::worker, this, i);
}

Pool::~Pool() {
  {
    std::lock_guard<std::mutex> lk(mu_);
    stop_.store(true);
  }
  go_.notify_all();
  for (auto& t : threads_) t.join();
}

void Pool::worker(int id) {
  uint64_t seen = 0;
  for (;;) {
    const auto t0 = std::chrono::steady_clock::now();
    int spins = 0;
    while (gen_.load() == seen && !stop_.load()) {
      if (++spins < 64) {
        _mm_pause();
        continue;
      }
      spins = 0;
      const auto dt = std::chrono::steady_clock::now() - t0;
      if (dt < kPauseSpin) continue;
      if (dt < kYieldSpin) {
        std::this_thread::yield();
        continue;
      }
      std::unique_lock<std::mutex> lk(mu_);
      sleepers_.fetch_add(1);
      go_.wait(lk, [&] { return gen_.load() != seen || stop_.load(); });
      sleepers_.fetch_sub(1);
    }
    if (stop_.load()) return;
    seen = gen_.load();
    (*fn_)(id);
    pending_.fetch_sub(1);
  }
}

void Pool::run(const std::function<void(int)>& fn) {
  std::lock_guard<std::mutex> one(run_mu_);
  fn_ = &fn;
  pending_.store(n_ - 1);
  gen_.fetch_add(1);  // publishes fn_ (sequentially consistent)
  if (sleepers_.load() > 0) {
    std::lock_guard<std::mutex> lk(mu_);
    go_.notify_all();
  }
  fn(0);
  const auto t0 = std::chrono::steady_clock::now();
  int spins = 0;
  while (pending_.load() != 0) {
    if (++spins < 64) {
      _mm_pause();
      continue;
    }
    spins = 0;
    if (std::chrono::steady_clock::now() - t0 >= kPauseSpin) std::this_thread::yield();
  }
}

// ---------------------------------------------------------------- fp16

// IEEE binary16 -> binary32 (exact).
float half_to_float(uint16_t h) {
  const uint32_t sign = (uint32_t)(h >> 15) << 31;
  const uint32_t e = (h >> 10) & 0x1f, m = h & 0x3ff;
  uint32_t bits;
  if (e == 0) {
    const float v = std::ldexp((float)m, -24);  // zero or subnormal: m * 2^-24, exact
    std::memcpy(&bits, &v, 4);
    bits |= sign;
  } else if (e == 31) {
    bits = sign | 0x7f800000u | (m << 13);
  } else {
    bits = sign | ((e + 112u) << 23) | (m << 13);  // rebias 15 -> 127
  }
  float f;
  std::memcpy(&f, &bits, 4);
  return f;
}

// binary32 -> binary16, round to nearest, ties to even.
uint16_t float_to_half_rn(float f) {
  uint32_t a;
  std::memcpy(&a, &f, 4);
  const uint16_t sign = (uint16_t)((a >> 16) & 0x8000u);
  a &= 0x7fffffffu;
  if (a >= 0x7f800000u) return sign | 0x7c00u | (a > 0x7f800000u ? 0x200u : 0u);  // inf, NaN
  if (a >= 0x477ff000u) return sign | 0x7c00u;  // >= 65520 rounds past the largest finite half
  if (a < 0x38800000u) {                          // below 2^-14: a multiple of 2^-24
    float v;
    std::memcpy(&v, &a, 4);
    return sign | (uint16_t)std::nearbyint(v * 16777216.0f);  // exact scaling; current mode is nearest-even
  }
  uint32_t h = (((a >> 23) - 112u) << 10) | ((a >> 13) & 0x3ffu);
  const uint32_t rest = a & 0x1fffu;
  if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) ++h;  // a carry moves into the exponent correctly
  return sign | (uint16_t)h;
}

// ---------------------------------------------------------------- product

void prepare_x(const uint16_t* x, int64_t M, int64_t K, float* xf) {
  for (int64_t m = 0; m < M; ++m)
    for (int64_t g = 0; g < K / 32; ++g) {
      const uint16_t* src = x + m * K + 32 * g;
      float* dst = xf + m * K + 32 * g;
      for (int j = 0; j < 16; ++j) {
        dst[j] = half_to_float(src[2 * j]);
        dst[16 + j] = half_to_float(src[2 * j + 1]);
      }
    }
}

namespace {

void rows_plain(const uint8_t* codes, const uint16_t* scales, int64_t K, const float* xf, int64_t M, int64_t n0,
                int64_t n1, float* acc, int64_t ldacc) {
  const int64_t G = K / 32;
  for (int64_t n = n0; n < n1; ++n) {
    const uint8_t* cr = codes + n * (K / 2);
    for (int64_t m = 0; m < M; ++m) {
      const float* xr = xf + m * K;
      float sum = 0.f;
      for (int64_t g = 0; g < G; ++g) {
        float p = 0.f;
        for (int j = 0; j < 16; ++j) {
          const uint8_t b = cr[16 * g + j];
          p += (float)((int)(b & 15) - 8) * xr[32 * g + j];
          p += (float)((int)(b >> 4) - 8) * xr[32 * g + 16 + j];
        }
        sum += half_to_float(scales[n * G + g]) * p;
      }
      acc[m * ldacc + n] = sum;
    }
  }
}

__attribute__((target("avx2,fma,f16c"))) inline float hsum(__m256 v) {
  __m128 s = _mm_add_ps(_mm256_castps256_ps128(v), _mm256_extractf128_ps(v, 1));
  s = _mm_add_ps(s, _mm_movehl_ps(s, s));
  s = _mm_add_ss(s, _mm_movehdup_ps(s));
  return _mm_cvtss_f32(s);
}

template <int MB>
__attribute__((target("avx2,fma,f16c"))) void rows_avx2_block(const uint8_t* codes, const uint16_t* scales, int64_t K,
                                                               const float* xf, int64_t n0, int64_t n1, float* acc,
                                                               int64_t ldacc) {
  const int64_t G = K / 32;
  const __m128i low = _mm_set1_epi8(0x0f), eight = _mm_set1_epi8(8);
  for (int64_t n = n0; n < n1; ++n) {
    const uint8_t* cr = codes + n * (K / 2);
    const uint16_t* sr = scales + n * G;
    __m256 a[MB];
    for (int t = 0; t < MB; ++t) a[t] = _mm256_setzero_ps();
    for (int64_t g = 0; g < G; ++g) {
      const __m128i b = _mm_loadu_si128(reinterpret_cast<const __m128i*>(cr + 16 * g));
      const __m128i qe = _mm_sub_epi8(_mm_and_si128(b, low), eight);                      // even inputs
      const __m128i qo = _mm_sub_epi8(_mm_and_si128(_mm_srli_epi16(b, 4), low), eight);  // odd inputs
      const __m256 q0 = _mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(qe));
      const __m256 q1 = _mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(_mm_srli_si128(qe, 8)));
      const __m256 q2 = _mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(qo));
      const __m256 q3 = _mm256_cvtepi32_ps(_mm256_cvtepi8_epi32(_mm_srli_si128(qo, 8)));
      const __m256 s = _mm256_set1_ps(_cvtsh_ss(sr[g]));
      for (int t = 0; t < MB; ++t) {
        const float* xg = xf + (int64_t)t * K + 32 * g;
        __m256 p = _mm256_mul_ps(q0, _mm256_loadu_ps(xg));
        p = _mm256_fmadd_ps(q1, _mm256_loadu_ps(xg + 8), p);
        p = _mm256_fmadd_ps(q2, _mm256_loadu_ps(xg + 16), p);
        p = _mm256_fmadd_ps(q3, _mm256_loadu_ps(xg + 24), p);
        a[t] = _mm256_fmadd_ps(s, p, a[t]);
      }
    }
    for (int t = 0; t < MB; ++t) acc[(int64_t)t * ldacc + n] = hsum(a[t]);
  }
}

// ATSI_CPU_PLAIN=1 (read once) takes the plain loop on any CPU.
bool have_avx2() {
  static const bool ok = __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma") &&
                         __builtin_cpu_supports("f16c") && !(getenv("ATSI_CPU_PLAIN") && atoi(getenv("ATSI_CPU_PLAIN")) == 1);
  return ok;
}

}  // namespace

void rows(const uint8_t* codes, const uint16_t* scales, int64_t K, const float* xf, int64_t M, int64_t n0,
          int64_t n1, float* acc, int64_t ldacc) {
  if (!have_avx2()) {
    rows_plain(codes, scales, K, xf, M, n0, n1, acc, ldacc);
    return;
  }
  for (int64_t m0 = 0; m0 < M; m0 += 4) {
    const float* x = xf + m0 * K;
    float* out = acc + m0 * ldacc;
    switch (std::min<int64_t>(4, M - m0)) {
      case 1: rows_avx2_block<1>(codes, scales, K, x, n0, n1, out, ldacc); break;
      case 2: rows_avx2_block<2>(codes, scales, K, x, n0, n1, out, ldacc); break;
      case 3: rows_avx2_block<3>(codes, scales, K, x, n0, n1, out, ldacc); break;
      default: rows_avx2_block<4>(codes, scales, K, x, n0, n1, out, ldacc); break;
    }
  }
}

void linear(Pool& pool, const uint8_t* codes, const uint16_t* scales, int64_t N, int64_t K, const float* xf,
            int64_t M, float* acc) {
  const int T = pool.size();
  pool.run([&](int t) {
    const int64_t n0 = N * t / T, n1 = N * (t + 1) / T;
    if (n1 > n0) rows(codes, scales, K, xf, M, n0, n1, acc, N);
  });
}

}  // namespace cpu
void set_context_free_error(const char* msg);
}  // namespace atsi

namespace {
atsi_status refuse(atsi_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  atsi::set_context_free_error(buf);
  return st;
}
}  // namespace

extern "C" {

atsi_status atsi_cpu_pool_create(int32_t threads, atsi_cpu_pool** out) {
  if (!out) return refuse(ATSI_E_INVALID, "out is NULL");
  *out = nullptr;
  if (threads < 1 || threads > 1024) return refuse(ATSI_E_INVALID, "threads = %d outside 1..1024", threads);
  atsi_cpu_pool* p = new (std::nothrow) atsi_cpu_pool(threads);
  if (!p) return refuse(ATSI_E_INVALID, "out of host memory");
  *out = p;
  return ATSI_OK;
}

atsi_status atsi_cpu_pool_destroy(atsi_cpu_pool* p) {
  if (!p) return ATSI_E_INVALID;
  delete p;
  return ATSI_OK;
}

atsi_status atsi_cpu_linear(atsi_cpu_pool* p, const uint8_t* codes, const uint16_t* scales, int64_t N, int64_t K,
                            const uint16_t* x, int64_t M, uint16_t* y) {
  if (!p || !codes || !scales || !x || !y) return refuse(ATSI_E_INVALID, "pool, codes, scales, x and y must be non-null");
  if (K < 32 || K % 32 != 0 || K > (1 << 20)) return refuse(ATSI_E_SHAPE, "K=%lld must be a positive multiple of 32 up to 2^20", (long long)K);
  if (N < 1 || N > (1 << 24)) return refuse(ATSI_E_SHAPE, "N=%lld outside 1..2^24", (long long)N);
  if (M < 1 || M > 65536) return refuse(ATSI_E_SHAPE, "M=%lld outside 1..65536", (long long)M);
  std::vector<float> xf((size_t)(M * K)), acc((size_t)(M * N));
  atsi::cpu::prepare_x(x, M, K, xf.data());
  atsi::cpu::linear(p->pool, codes, scales, N, K, xf.data(), M, acc.data());
  for (size_t i = 0; i < acc.size(); ++i) y[i] = atsi::cpu::float_to_half_rn(acc[i]);
  return ATSI_OK;
}

atsi_status atsi_debug_cpu_f16(const float* in, int64_t n, uint16_t* out, float* back) {
  if (!in || n < 0) return refuse(ATSI_E_INVALID, "in is NULL or n < 0");
  for (int64_t i = 0; i < n; ++i) {
    const uint16_t h = atsi::cpu::float_to_half_rn(in[i]);
    if (out) out[i] = h;
    if (back) back[i] = atsi::cpu::half_to_float(h);
  }
  return ATSI_OK;
}

}  // extern "C"
