// Dynamic transfer scheduling (Sec. 4.4.1-4.4.2, Alg. 2) and load-aware
// re-scheduling (Sec. 4.4.3, Alg. 3).  Host code only.
//
// A round runs tensors 0..n-1 in execution order.  Tensors the static
// placement keeps on the GPU (b_i = GPU) run there; a CPU-placed tensor
// either runs on the CPU or is promoted: its weights are copied to the GPU,
// issued from a CPU-side endpoint j, and it runs on the GPU.  Only the part
// of the copy that the window seg(j, i) (the default path's time strictly
// between j and i) does not hide is exposed: delta_i = max(w_i - seg(j,i), 0).
// The program minimises the round latency
//   T(rb) = sum_i t_i^{rb_i} + sum_{i>=1} c_i [rb_{i-1} != rb_i] + sum_promoted delta_i.
//
// dp[i][k] is the least latency of tensors 0..i with tensor i on backend k.
// Extending a state by one tensor adds its time and, on a backend change,
// c_i.  A promotion of i starts from a CPU-side endpoint: the round start
// (a virtual point with latency 0) or a state dp[j][CPU], with tensors j+1..
// i-1 on their default backends; it then waits for max(w_i, seg(j, i)), pays
// the switch into i when tensor i-1 runs on the CPU, and adds t^g_i.  With
// prefix sums P of the default path (times plus switches), seg(j, i) =
// P[i] - P[j+1], so each promotion scans its candidate endpoints once:
// O(n^2) time, O(n) memory (one endpoint and one predecessor bit per tensor
// for the backtrack).
//
// Readings (the paper leaves them open): the round start is an endpoint, so
// the first CPU-placed tensor can be promoted with its copy hidden behind
// everything before it; the switch charged on promotion is the one T(rb)
// charges (tensor i-1 on the CPU), not the printed condition on b_{i-1} =
// GPU, which would make the program minimise something other than T(rb);
// two promoted tensors need a CPU-run tensor between them, as the program's
// transitions imply.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <new>
#include <vector>

#include "../../include/atsi.h"

namespace atsi {
void set_context_free_error(const char* msg);
}

namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();
constexpr int32_t kMaxTensors = 1 << 16;
constexpr int kCpu = 0, kGpu = 1;

atsi_status refuse(atsi_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  atsi::set_context_free_error(buf);
  return st;
}

atsi_status check_problem(const atsi_transfer_problem* p) {
  if (!p) return refuse(ATSI_E_INVALID, "transfer problem is NULL");
  if (p->n < 1 || p->n > kMaxTensors) return refuse(ATSI_E_SHAPE, "n = %d outside 1..%d", p->n, kMaxTensors);
  if (!p->on_gpu || !p->t_gpu || !p->t_cpu || !p->c || !p->w)
    return refuse(ATSI_E_INVALID, "on_gpu, t_gpu, t_cpu, c and w must be non-null");
  for (int32_t i = 0; i < p->n; ++i) {
    if (p->on_gpu[i] > 1) return refuse(ATSI_E_INVALID, "on_gpu[%d] = %d is not 0 or 1", i, p->on_gpu[i]);
    const double v[4] = {p->t_gpu[i], p->t_cpu[i], p->c[i], p->w[i]};
    for (double x : v)
      if (!(x >= 0.0) || !std::isfinite(x))
        return refuse(ATSI_E_INVALID, "times of tensor %d must be finite and >= 0", i);
  }
  return ATSI_OK;
}

// Alg. 2.  rb[i] = 1 where tensor i runs on the GPU.  Returns T*.
double solve(const atsi_transfer_problem* p, uint8_t* rb) {
  const int n = p->n;
  const uint8_t* b = p->on_gpu;
  auto t = [&](int i, int k) { return k == kGpu ? p->t_gpu[i] : p->t_cpu[i]; };
  auto sw = [&](int i) { return i >= 1 ? p->c[i] : 0.0; };
  // P[i]: default-path time of tensors 0..i-1 including the switches inside
  std::vector<double> P(n + 1, 0.0);
  for (int i = 0; i < n; ++i) P[i + 1] = P[i] + t(i, b[i]) + ((i >= 1 && b[i - 1] != b[i]) ? p->c[i] : 0.0);
  std::vector<double> dp(2 * (size_t)n, kInf);
  std::vector<uint8_t> pred(2 * (size_t)n, 0);  // backend of i-1 for an extended state
  std::vector<int32_t> from(n, -2);             // endpoint of a promotion (-1: round start), -2: none
  auto D = [&](int i, int k) -> double& { return dp[2 * (size_t)i + k]; };
  for (int i = 0; i < n; ++i) {
    if (b[i] == kGpu) {
      // a GPU-placed tensor extends either state
      double best = kInf;
      uint8_t pk = 0;
      if (i == 0) {
        best = 0.0;
      } else {
        const double fc = D(i - 1, kCpu) + sw(i), fg = D(i - 1, kGpu);
        best = fc <= fg ? fc : fg;  // ties: the CPU predecessor
        pk = fc <= fg ? kCpu : kGpu;
      }
      D(i, kGpu) = best + t(i, kGpu);
      pred[2 * (size_t)i + kGpu] = pk;
      continue;
    }
    // CPU-placed: stay on the CPU ...
    {
      double best = 0.0;
      uint8_t pk = 0;
      if (i > 0) {
        const double fc = D(i - 1, kCpu), fg = D(i - 1, kGpu) + sw(i);
        best = fc <= fg ? fc : fg;
        pk = fc <= fg ? kCpu : kGpu;
      }
      D(i, kCpu) = best + t(i, kCpu);
      pred[2 * (size_t)i + kCpu] = pk;
    }
    // ... or be promoted from the earliest-ending endpoint
    double best = std::max(p->w[i], P[i]);  // round start: seg = P[i] - P[0]
    int32_t arg = -1;
    for (int j = 0; j < i; ++j) {
      if (b[j] != kCpu) continue;
      const double v = D(j, kCpu) + std::max(p->w[i], P[i] - P[j + 1]);
      if (v < best) {
        best = v;
        arg = j;
      }
    }
    const bool switch_in = i >= 1 && b[i - 1] == kCpu;
    D(i, kGpu) = best + (switch_in ? p->c[i] : 0.0) + t(i, kGpu);
    from[i] = arg;
  }
  int k = D(n - 1, kCpu) <= D(n - 1, kGpu) ? kCpu : kGpu;
  const double total = D(n - 1, k);
  int i = n - 1;
  while (i >= 0) {
    if (k == kGpu && b[i] == kCpu) {  // a promotion: i on the GPU, back to its endpoint on the default path
      rb[i] = 1;
      const int j = from[i];
      for (int q = i - 1; q > j; --q) rb[q] = b[q];
      if (j < 0) break;
      i = j;
      k = kCpu;
      continue;
    }
    rb[i] = (uint8_t)k;
    k = pred[2 * (size_t)i + k];
    --i;
  }
  return total;
}

}  // namespace

struct atsi_rescheduler {
  int32_t n = 0;
  double eps = 0.0, tau_tpot = 0.0;
  bool have_prev = false;
  double t_last = 0.0;
  std::vector<uint8_t> b, rb;
  std::vector<double> tg, tc, c, w;  // the snapshot the last scheduling used
};

extern "C" {

atsi_status atsi_schedule_transfers(const atsi_transfer_problem* p, uint8_t* rb_out, double* latency_out) {
  atsi_status st = check_problem(p);
  if (st) return st;
  if (!rb_out) return refuse(ATSI_E_INVALID, "rb_out is NULL");
  const double T = solve(p, rb_out);
  if (latency_out) *latency_out = T;
  return ATSI_OK;
}

atsi_status atsi_transfer_latency(const atsi_transfer_problem* p, const uint8_t* rb, double* latency_out) {
  atsi_status st = check_problem(p);
  if (st) return st;
  if (!rb || !latency_out) return refuse(ATSI_E_INVALID, "rb and latency_out must be non-null");
  const int n = p->n;
  const uint8_t* b = p->on_gpu;
  for (int i = 0; i < n; ++i) {
    if (rb[i] > 1) return refuse(ATSI_E_INVALID, "rb[%d] = %d is not 0 or 1", i, rb[i]);
    if (b[i] == kGpu && rb[i] == kCpu) return refuse(ATSI_E_INVALID, "tensor %d is placed on the GPU", i);
  }
  // walk the round: the default-path prefix P gives seg(j, i) = P[i] - P[j+1]
  std::vector<double> P(n + 1, 0.0);
  for (int i = 0; i < n; ++i)
    P[i + 1] = P[i] + (b[i] == kGpu ? p->t_gpu[i] : p->t_cpu[i]) + ((i >= 1 && b[i - 1] != b[i]) ? p->c[i] : 0.0);
  double T = 0.0;
  int start = -1;        // endpoint of the next promotion: -1 round start, -2 none yet after a promotion
  for (int i = 0; i < n; ++i) {
    T += rb[i] == kGpu ? p->t_gpu[i] : p->t_cpu[i];
    if (i >= 1 && rb[i - 1] != rb[i]) T += p->c[i];
    if (b[i] == kCpu && rb[i] == kGpu) {
      if (start == -2) {
        *latency_out = kInf;  // two promotions with no CPU-run tensor between
        return ATSI_OK;
      }
      T += std::max(p->w[i] - (P[i] - P[start + 1]), 0.0);
      start = -2;
    } else if (rb[i] == kCpu && start == -2) {
      start = i;
    }
  }
  *latency_out = T;
  return ATSI_OK;
}

atsi_status atsi_rescheduler_create(int32_t n, double eps, double tau_tpot, atsi_rescheduler** out) {
  if (!out) return refuse(ATSI_E_INVALID, "out is NULL");
  *out = nullptr;
  if (n < 1 || n > kMaxTensors) return refuse(ATSI_E_SHAPE, "n = %d outside 1..%d", n, kMaxTensors);
  if (!(eps >= 0.0) || !std::isfinite(eps) || !(tau_tpot >= 0.0) || !std::isfinite(tau_tpot))
    return refuse(ATSI_E_INVALID, "eps and the interval multiple must be finite and >= 0");
  atsi_rescheduler* r = new (std::nothrow) atsi_rescheduler;
  if (!r) return refuse(ATSI_E_INVALID, "out of host memory");
  r->n = n;
  r->eps = eps;
  r->tau_tpot = tau_tpot;
  *out = r;
  return ATSI_OK;
}

atsi_status atsi_rescheduler_destroy(atsi_rescheduler* r) {
  if (!r) return ATSI_E_INVALID;
  delete r;
  return ATSI_OK;
}

atsi_status atsi_rescheduler_step(atsi_rescheduler* r, const atsi_transfer_problem* cur, double now_s,
                                  double tpot_s, uint8_t* rb_out, int32_t* rescheduled_out, double* deviation_out) {
  if (!r) return refuse(ATSI_E_INVALID, "rescheduler is NULL");
  atsi_status st = check_problem(cur);
  if (st) return st;
  if (cur->n != r->n) return refuse(ATSI_E_SHAPE, "snapshot of %d tensors, rescheduler made for %d", cur->n, r->n);
  if (!rb_out) return refuse(ATSI_E_INVALID, "rb_out is NULL");
  if (!std::isfinite(now_s) || !(tpot_s >= 0.0) || !std::isfinite(tpot_s))
    return refuse(ATSI_E_INVALID, "now and the recent TPOT must be finite (TPOT >= 0)");
  const int n = r->n;
  // ComputeDeviation: the largest relative change of a measured series' total
  double d = 0.0;
  bool same_b = r->have_prev;
  if (r->have_prev) {
    const double* prev[4] = {r->tg.data(), r->tc.data(), r->c.data(), r->w.data()};
    const double* now[4] = {cur->t_gpu, cur->t_cpu, cur->c, cur->w};
    for (int s = 0; s < 4; ++s) {
      double sp = 0.0, sq = 0.0;
      for (int i = 0; i < n; ++i) {
        sp += prev[s][i];
        sq += now[s][i];
      }
      if (sp > 0.0)
        d = std::max(d, std::fabs(sq - sp) / sp);
      else if (sq > 0.0)
        d = kInf;
    }
    same_b = std::equal(r->b.begin(), r->b.end(), cur->on_gpu);
  }
  // Alg. 3: keep the previous assignment below eps or within tau of the last
  // re-scheduling; the first round and a changed placement always schedule
  const bool keep = same_b && (d < r->eps || now_s - r->t_last < r->tau_tpot * tpot_s);
  if (deviation_out) *deviation_out = d;
  if (rescheduled_out) *rescheduled_out = keep ? 0 : 1;
  if (!keep) {
    r->rb.assign(n, 0);
    solve(cur, r->rb.data());
    r->b.assign(cur->on_gpu, cur->on_gpu + n);
    r->tg.assign(cur->t_gpu, cur->t_gpu + n);
    r->tc.assign(cur->t_cpu, cur->t_cpu + n);
    r->c.assign(cur->c, cur->c + n);
    r->w.assign(cur->w, cur->w + n);
    r->t_last = now_s;
    r->have_prev = true;
  }
  std::memcpy(rb_out, r->rb.data(), (size_t)n);
  return ATSI_OK;
}

}  // extern "C"
