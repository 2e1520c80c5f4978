// Static tensor placement (Sec. 4.3; Alg. 1): which tensors stay resident in
// GPU memory.  Host code only.
//
// Tensors come in execution order.  Keeping tensor i on the GPU saves r_i of
// latency; running neighbours i-1 and i on different backends costs c_i.  The
// placement maximises sum r_i [b_i = GPU] - sum_{i>=1} c_i [b_i != b_{i-1}]
// with the GPU-resident sizes inside the budget.  As in the paper, sizes and
// the budget are counted in units of a granularity (MB there): sizes rounded
// up, the budget rounded down.
//
// The solver is the knapsack dynamic program the paper names, with the
// backend of the previous tensor as a second state coordinate so the switch
// penalty is exact: best[m][k] is the best objective of the tensors so far
// with m budget units used and the last one on backend k.  One bit per state
// and tensor records the predecessor's backend for the backtrack.  O(n W)
// time for W budget units (W is capped at the total size of the tensors the
// program chooses among, so an ample budget costs nothing), O(n W / 4) bytes.
//
// MoE models (Alg. 1): when the budget covers every non-expert tensor, those
// are all GPU-resident and the program chooses experts in what remains;
// otherwise every expert stays on the CPU and the program chooses among the
// non-expert tensors.  The tensors it does not choose among keep their fixed
// backend while the program optimises the whole objective, switches at their
// boundaries included.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <limits>
#include <vector>

#include "atsi.h"

namespace atsi {
void set_context_free_error(const char* msg);

namespace {

constexpr double kNone = -std::numeric_limits<double>::infinity();
constexpr uint64_t kMaxCells = 1ull << 31;  // tensors x budget units the program may visit

atsi_status refuse(atsi_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  set_context_free_error(buf);
  return st;
}

// forced[i]: -1 chosen by the program, 0 fixed on the CPU, 1 fixed on the GPU.
// w[i]: budget units of a chosen tensor.  Writes the best placement to b.
void solve(int n, const std::vector<int8_t>& forced, const std::vector<int64_t>& w, int64_t W, const double* r,
           const double* c, uint8_t* b) {
  const size_t cols = (size_t)W + 1;
  std::vector<double> cur(2 * cols, kNone), nxt(2 * cols, kNone);
  std::vector<uint64_t> back(((size_t)n * cols * 2 + 63) / 64, 0);  // predecessor backend bits
  auto bit = [&](int i, size_t m, int k) { return ((size_t)i * cols + m) * 2 + (size_t)k; };
  auto units = [&](int i, int k) -> int64_t { return (k == 1 && forced[i] < 0) ? w[i] : 0; };
  auto allowed = [&](int i, int k) { return forced[i] < 0 || forced[i] == k; };

  int64_t reach = 0;  // most units any state can have used so far
  for (int k = 0; k < 2; ++k)
    if (allowed(0, k) && units(0, k) <= W) cur[(size_t)units(0, k) * 2 + k] = k ? r[0] : 0.0;
  reach = std::min<int64_t>(W, units(0, 1));
  for (int i = 1; i < n; ++i) {
    const int64_t next_reach = std::min<int64_t>(W, reach + units(i, 1));
    for (size_t m = 0; m <= (size_t)next_reach; ++m) nxt[2 * m] = nxt[2 * m + 1] = kNone;
    for (size_t m = 0; m <= (size_t)reach; ++m)
      for (int kp = 0; kp < 2; ++kp) {
        const double v = cur[2 * m + kp];
        if (v == kNone) continue;
        for (int k = 0; k < 2; ++k) {
          if (!allowed(i, k)) continue;
          const size_t m2 = m + (size_t)units(i, k);
          if (m2 > (size_t)W) continue;
          const double v2 = v + (k ? r[i] : 0.0) - (k != kp ? c[i] : 0.0);
          // strictly better only: on ties the CPU predecessor and the fewer units win
          if (v2 > nxt[2 * m2 + k]) {
            nxt[2 * m2 + k] = v2;
            const size_t x = bit(i, m2, k);
            if (kp) back[x / 64] |= 1ull << (x % 64); else back[x / 64] &= ~(1ull << (x % 64));
          }
        }
      }
    reach = next_reach;
    cur.swap(nxt);
  }
  size_t bm = 0;
  int bk = 0;
  double best = kNone;
  for (size_t m = 0; m <= (size_t)reach; ++m)
    for (int k = 0; k < 2; ++k)
      if (cur[2 * m + k] > best) {
        best = cur[2 * m + k];
        bm = m;
        bk = k;
      }
  for (int i = n - 1; i >= 0; --i) {
    b[i] = (uint8_t)bk;
    if (i == 0) break;
    const size_t x = bit(i, bm, bk);
    const int kp = (int)((back[x / 64] >> (x % 64)) & 1ull);
    bm -= (size_t)units(i, bk);
    bk = kp;
  }
}

}  // namespace
}  // namespace atsi

extern "C" atsi_status atsi_solve_placement(const atsi_placement_problem* p, uint8_t* on_gpu_out,
                                            double* objective_out) {
  using namespace atsi;
  if (!p || !on_gpu_out) return refuse(ATSI_E_INVALID, "placement problem and output must be non-null");
  const int n = p->n;
  if (n < 1) return refuse(ATSI_E_SHAPE, "placement of %d tensors", n);
  if (!p->size_bytes || !p->r || !p->c) return refuse(ATSI_E_INVALID, "size_bytes, r and c must be non-null");
  const double g = p->granularity_bytes, M = p->budget_bytes;
  if (!(g > 0.0) || !std::isfinite(g)) return refuse(ATSI_E_INVALID, "granularity %g must be positive", g);
  if (!(M >= 0.0) || !std::isfinite(M)) return refuse(ATSI_E_INVALID, "budget %g must be finite and >= 0", M);
  for (int i = 0; i < n; ++i) {
    const double s = p->size_bytes[i];
    if (!(s >= 0.0) || !std::isfinite(s)) return refuse(ATSI_E_INVALID, "size of tensor %d is %g", i, s);
    if (!std::isfinite(p->r[i]) || !std::isfinite(p->c[i]))
      return refuse(ATSI_E_INVALID, "r or c of tensor %d is not finite", i);
  }

  // Alg. 1's dense / MoE branch
  std::vector<int8_t> forced(n, -1);
  double budget = M;
  if (p->is_expert) {
    double s_nonexp = 0.0;
    for (int i = 0; i < n; ++i)
      if (!p->is_expert[i]) s_nonexp += p->size_bytes[i];
    if (M >= s_nonexp) {
      for (int i = 0; i < n; ++i)
        if (!p->is_expert[i]) forced[i] = 1;
      budget = M - s_nonexp;
    } else {
      for (int i = 0; i < n; ++i)
        if (p->is_expert[i]) forced[i] = 0;
    }
  }
  std::vector<int64_t> w(n, 0);
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    if (forced[i] >= 0) continue;
    const double u = std::ceil(p->size_bytes[i] / g);
    if (u > 4e18) return refuse(ATSI_E_SHAPE, "tensor %d is %g granules", i, u);
    w[i] = (int64_t)u;
    total += w[i];
    if (total < 0 || total > (int64_t)4e18) return refuse(ATSI_E_SHAPE, "sizes overflow the unit count");
  }
  const double wb = budget > 0.0 ? std::floor(budget / g) : 0.0;
  const int64_t W = wb >= (double)total ? total : (int64_t)wb;  // a budget beyond every size never binds
  if ((uint64_t)n * (uint64_t)(W + 1) > kMaxCells)
    return refuse(ATSI_E_SHAPE, "%d tensors x %lld budget units is too fine a granularity (at most %llu states)", n,
                  (long long)(W + 1), (unsigned long long)kMaxCells);
  solve(n, forced, w, W, p->r, p->c, on_gpu_out);
  if (objective_out) {
    double gain = 0.0, sw = 0.0;
    for (int i = 0; i < n; ++i)
      if (on_gpu_out[i]) gain += p->r[i];
    for (int i = 1; i < n; ++i)
      if (on_gpu_out[i] != on_gpu_out[i - 1]) sw += p->c[i];
    *objective_out = gain - sw;
  }
  return ATSI_OK;
}
