/*
 * Plain fp64 CPU oracle of the block-int4 quantised linear layer.
 *
 * TEST INFRASTRUCTURE ONLY: built and called by the test suite and by the
 * benchmark's CPU-baseline leg, never by the GPU library.  It shares no code
 * with the HIP path.
 *
 * y[m][n] = sum_k x[m][k] * s[n][k/32] * q[n][k], every product and sum in
 * double precision, with
 *   q[n][k] = ((codes[n][k/2] >> (4 * (k % 2))) & 15) - 8   (offset-binary
 *             nibbles, the even input in the low nibble), and
 *   s[n][g] = the IEEE binary16 value of scales[n][g], decoded below from its
 *             bits (sign, 5-bit exponent with bias 15, 10-bit fraction;
 *             subnormals when the exponent field is 0).
 * This is the paper's per-tensor quantised linear operator (Sec. 4.1-4.2;
 * INT4 weights, Sec. 5.1) under the block-int4 reading: one signed 4-bit
 * code per weight and one fp16 scale per 32 consecutive inputs.
 *
 * Plain loops, no blocking and no library calls; output rows are split over
 * `threads` POSIX threads (each thread owns a contiguous range of n, so the
 * result does not depend on the thread count).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>

static double half_bits_to_double(uint16_t h) {
  const int sign = (h >> 15) & 1, e = (h >> 10) & 31, f = h & 1023;
  double v;
  if (e == 0)
    v = ldexp((double)f, -24); /* subnormal: f * 2^-10 * 2^-14 */
  else if (e == 31)
    v = f ? NAN : INFINITY;
  else
    v = ldexp(1024.0 + f, e - 25); /* (1 + f/1024) * 2^(e-15) */
  return sign ? -v : v;
}

typedef struct {
  const uint8_t* codes;
  const uint16_t* scales;
  int64_t N, K, M, n0, n1;
  const double* x;
  double* y;
} job_t;

static void* run(void* arg) {
  const job_t* j = (const job_t*)arg;
  const int64_t G = j->K / 32;
  for (int64_t n = j->n0; n < j->n1; ++n) {
    const uint8_t* row = j->codes + n * (j->K / 2);
    const uint16_t* srow = j->scales + n * G;
    for (int64_t m = 0; m < j->M; ++m) {
      const double* xm = j->x + m * j->K;
      double acc = 0.0;
      for (int64_t k = 0; k < j->K; ++k) {
        const int q = ((row[k / 2] >> (4 * (k % 2))) & 15) - 8;
        acc += xm[k] * (half_bits_to_double(srow[k / 32]) * (double)q);
      }
      j->y[m * j->N + n] = acc;
    }
  }
  return NULL;
}

/* y[M][N] (row-major, fp64) from codes[N][K/2], scales[N][K/32] (fp16 bits)
 * and x[M][K] (fp64); K % 32 == 0.  Returns 0, or -1 for bad arguments. */
int q4_linear_f64(const uint8_t* codes, const uint16_t* scales, int64_t N, int64_t K, const double* x, int64_t M,
                  double* y, int threads) {
  if (!codes || !scales || !x || !y || N < 1 || K < 32 || K % 32 || M < 1) return -1;
  if (threads < 1) threads = 1;
  if (threads > N) threads = (int)N;
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * threads);
  job_t* jobs = (job_t*)malloc(sizeof(job_t) * threads);
  if (!th || !jobs) {
    free(th);
    free(jobs);
    return -1;
  }
  for (int t = 0; t < threads; ++t) {
    job_t j = {codes, scales, N, K, M, N * t / threads, N * (t + 1) / threads, x, y};
    jobs[t] = j;
  }
  char* live = (char*)calloc((size_t)threads, 1);
  if (!live) {
    free(th);
    free(jobs);
    return -1;
  }
  for (int t = 1; t < threads; ++t) {
    if (pthread_create(&th[t], NULL, run, &jobs[t]) == 0)
      live[t] = 1;
    else
      run(&jobs[t]); /* no thread: do that range here */
  }
  run(&jobs[0]);
  for (int t = 1; t < threads; ++t)
    if (live[t]) pthread_join(th[t], NULL);
  free(live);
  free(th);
  free(jobs);
  return 0;
}
