// Host-CPU backend: a thread pool and the block-int4 matrix-vector product
// the CPU-placed tensors run on (the paper's hybrid: tensors without a GPU
// copy execute on the host CPU, Sec. 4.3-4.4).  Host code only; no HIP here.
#pragma once

#include <stdint.h>

#include <atomic>
#include <condition_variable>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

namespace atsi {
namespace cpu {

// A fixed set of worker threads; run(fn) calls fn(0..n-1) once each, the
// calling thread taking part as worker 0, and returns when all are done.
// One run at a time per pool (run serialises its callers).  Workers spin on
// the job counter for a while after each job (decode rounds hand the pool a
// new product every few tens of microseconds) and then sleep on a condition
// variable.
class Pool {
 public:
  explicit Pool(int threads);
  ~Pool();
  int size() const { return n_; }
  void run(const std::function<void(int)>& fn);

 private:
  void worker(int id);
  int n_;
  std::vector<std::thread> threads_;
  std::mutex run_mu_;  // one run at a time
  std::mutex mu_;      // guards sleeping
  std::condition_variable go_;
  const std::function<void(int)>* fn_ = nullptr;
  std::atomic<uint64_t> gen_{0};
  std::atomic<int> pending_{0};
  std::atomic<int> sleepers_{0};
  std::atomic<bool> stop_{false};
};

// acc[m * ldacc + n] = sum_k q[n][k] * s[n][k / 32] * x[m][k] in fp32 for
// rows n in [n0, n1): codes [N][K/2] (even input in the low nibble, code
// u = q + 8), scales fp16 bits [N][K/32], xf the fp32 activations [M][K]
// re-ordered per 32-input group as the 16 even inputs then the 16 odd ones
// (prepare_x).  Each product q * x is exact in fp32 when x came from fp16;
// the sums and the scaling are fp32.
void prepare_x(const uint16_t* x, int64_t M, int64_t K, float* xf);
void rows(const uint8_t* codes, const uint16_t* scales, int64_t K, const float* xf, int64_t M, int64_t n0,
          int64_t n1, float* acc, int64_t ldacc);

// acc[M][N] for all rows of one tensor, split over the pool's threads.
void linear(Pool& pool, const uint8_t* codes, const uint16_t* scales, int64_t N, int64_t K, const float* xf,
            int64_t M, float* acc);

float half_to_float(uint16_t h);
uint16_t float_to_half_rn(float f);

}  // namespace cpu
}  // namespace atsi

// The C-ABI handle of a pool.
struct atsi_cpu_pool {
  atsi::cpu::Pool pool;
  explicit atsi_cpu_pool(int threads) : pool(threads) {}
};
