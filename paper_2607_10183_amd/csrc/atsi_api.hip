// C-ABI layer: context, tensor registry, placement, the host-streaming engine
// and dispatch to the kernels.
//
// Streaming engine (Sec. 4.2.1-4.2.2 of the paper): host-resident tensors are
// copied from pinned memory into GPU temporary buffers ("slots") on the
// transfer stream and consumed on the compute stream.  Per slot two events
// order the streams: `ready` (recorded on the transfer stream after the copy,
// waited on by the compute stream before the consumer) and `free` (recorded
// on the compute stream after the consumer, waited on by the transfer stream
// before the slot is overwritten), so a slot is never reused early.  Copies
// start as early as a free slot allows: an explicit prefetch, or the schedule
// (the execution order of tensors) lets the engine run the transfer stream
// ahead of compute by up to n_slots - 1 tensors.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/atsi.h"
#include "common.h"

using namespace atsi;

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }

struct Tensor {
  int64_t K = 0, N = 0;
  const uint8_t* dcodes = nullptr;
  const uint16_t* dscales = nullptr;
  const uint8_t* hcodes = nullptr;
  const uint16_t* hscales = nullptr;
  bool on_host = false;
  size_t codes_bytes() const { return (size_t)(K / 2) * (size_t)N; }
  size_t scales_bytes() const { return (size_t)(K / kGroup) * (size_t)N * 2; }
  size_t slot_need() const { return align_up(codes_bytes()) + align_up(scales_bytes()); }
};

struct Slot {
  char* base = nullptr;
  hipEvent_t ready = nullptr;
  hipEvent_t free = nullptr;
  bool free_recorded = false;
  int tid = -1;         // tensor whose copy the slot holds or receives
  bool armed = false;   // copy issued ahead of its consumer, not yet consumed
  uint64_t seq = 0;     // issue order of the armed copy
  uint64_t last = 0;    // last use (issue or consume), for round-robin reuse
};

thread_local std::string g_create_error;

}  // namespace

struct atsi_ctx {
  int device = 0;
  hipStream_t cs = nullptr;  // compute stream
  hipStream_t ts = nullptr;  // transfer stream
  char* ws = nullptr;
  size_t ws_bytes = 0;
  int n_slots = 0;
  std::vector<Tensor> tensors;
  std::vector<Slot> slots;
  size_t slot_bytes = 0;
  size_t scratch_off = 0;
  std::vector<atsi_tid> schedule;
  size_t sched_pos = 0;     // next schedule position whose host tensor is not yet prefetched
  uint64_t clock = 0;
  std::string err;
  atsi_status latched = ATSI_OK;
  std::string latched_msg;
};

namespace {

atsi_status fail(atsi_ctx* c, atsi_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c) c->err = buf; else g_create_error = buf;
  return st;
}

atsi_status hip_fail(atsi_ctx* c, hipError_t e, const char* what) {
  atsi_status st = fail(c, ATSI_E_HIP, "%s: %s", what, hipGetErrorString(e));
  if (c && c->latched == ATSI_OK) {
    c->latched = ATSI_E_HIP;
    c->latched_msg = c->err;
  }
  return st;
}

#define HIP_TRY(ctx, expr)                                   \
  do {                                                       \
    hipError_t e_ = (expr);                                  \
    if (e_ != hipSuccess) return hip_fail((ctx), e_, #expr); \
  } while (0)

atsi_status enter(atsi_ctx* c) {
  if (!c) return ATSI_E_INVALID;
  if (c->latched != ATSI_OK) {
    c->err = c->latched_msg;
    return c->latched;
  }
  hipError_t e = hipSetDevice(c->device);
  if (e != hipSuccess) return hip_fail(c, e, "hipSetDevice");
  return ATSI_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

atsi_status check_tid(atsi_ctx* c, atsi_tid t) {
  if (t < 0 || (size_t)t >= c->tensors.size())
    return fail(c, ATSI_E_UNKNOWN_TENSOR, "unknown tensor id %d (registered: %zu)", t, c->tensors.size());
  return ATSI_OK;
}

// Lay out n_slots slots sized for the largest host-resident tensor.
atsi_status layout_slots(atsi_ctx* c) {
  size_t need = 0;
  for (const Tensor& t : c->tensors)
    if (t.on_host) need = std::max(need, t.slot_need());
  if (need > 0 && (size_t)c->n_slots * need > c->ws_bytes)
    return fail(c, ATSI_E_WORKSPACE, "workspace %zu B < %d slots x %zu B", c->ws_bytes, c->n_slots, need);
  HIP_TRY(c, hipStreamSynchronize(c->cs));
  HIP_TRY(c, hipStreamSynchronize(c->ts));
  c->slot_bytes = need;
  for (int i = 0; i < c->n_slots; ++i) {
    Slot& s = c->slots[i];
    s.base = c->ws + (size_t)i * need;
    s.free_recorded = false;
    s.tid = -1;
    s.armed = false;
    s.last = 0;
  }
  c->scratch_off = align_up((size_t)c->n_slots * need);
  c->sched_pos = 0;
  return ATSI_OK;
}

// Issue the H2D copy of host tensor `tid` into a reusable slot; returns its index.
atsi_status issue_copy(atsi_ctx* c, atsi_tid tid, int* slot_out) {
  int best = -1;
  for (int i = 0; i < c->n_slots; ++i) {
    const Slot& s = c->slots[i];
    if (s.armed) continue;
    if (best < 0 || s.last < c->slots[best].last) best = i;
  }
  if (best < 0) return fail(c, ATSI_E_STATE, "all %d slots hold prefetched tensors not yet consumed", c->n_slots);
  Slot& s = c->slots[best];
  const Tensor& t = c->tensors[tid];
  if (s.free_recorded) HIP_TRY(c, hipStreamWaitEvent(c->ts, s.free, 0));
  HIP_TRY(c, hipMemcpyAsync(s.base, t.hcodes, t.codes_bytes(), hipMemcpyHostToDevice, c->ts));
  HIP_TRY(c, hipMemcpyAsync(s.base + align_up(t.codes_bytes()), t.hscales, t.scales_bytes(),
                            hipMemcpyHostToDevice, c->ts));
  HIP_TRY(c, hipEventRecord(s.ready, c->ts));
  s.tid = tid;
  s.armed = true;
  s.seq = ++c->clock;
  s.last = s.seq;
  *slot_out = best;
  return ATSI_OK;
}

// Keep the transfer stream ahead: prefetch the next host tensors of the schedule.
atsi_status topup(atsi_ctx* c) {
  if (c->schedule.empty()) return ATSI_OK;
  int armed = 0;
  for (const Slot& s : c->slots) armed += s.armed ? 1 : 0;
  size_t guard = 0;
  while (armed < c->n_slots - 1 && guard++ < c->schedule.size()) {
    atsi_tid t = c->schedule[c->sched_pos % c->schedule.size()];
    c->sched_pos++;
    if (!c->tensors[t].on_host) continue;
    int si;
    atsi_status st = issue_copy(c, t, &si);
    if (st) return st;
    ++armed;
    guard = 0;
  }
  return ATSI_OK;
}

// Resolve where tensor `tid` is read from for the next kernel; for a host
// tensor this makes the compute stream wait for its copy.  *slot = -1 for HBM.
atsi_status acquire(atsi_ctx* c, atsi_tid tid, QView* v, int* slot) {
  const Tensor& t = c->tensors[tid];
  v->K = (int)t.K;
  v->N = (int)t.N;
  *slot = -1;
  if (!t.on_host) {
    v->codes = t.dcodes;
    v->scales = t.dscales;
    return ATSI_OK;
  }
  int si = -1;
  for (int i = 0; i < c->n_slots; ++i) {
    const Slot& s = c->slots[i];
    if (s.armed && s.tid == tid && (si < 0 || s.seq < c->slots[si].seq)) si = i;
  }
  if (si < 0) {
    atsi_status st = issue_copy(c, tid, &si);
    if (st) return st;
  }
  Slot& s = c->slots[si];
  HIP_TRY(c, hipStreamWaitEvent(c->cs, s.ready, 0));
  v->codes = reinterpret_cast<const uint8_t*>(s.base);
  v->scales = reinterpret_cast<const uint16_t*>(s.base + align_up(t.codes_bytes()));
  *slot = si;
  return ATSI_OK;
}

// After the consumer kernel of a slot has been enqueued.
atsi_status release(atsi_ctx* c, int slot) {
  if (slot < 0) return ATSI_OK;
  Slot& s = c->slots[slot];
  HIP_TRY(c, hipEventRecord(s.free, c->cs));
  s.free_recorded = true;
  s.armed = false;
  s.last = ++c->clock;
  return topup(c);
}

atsi_status launched(atsi_ctx* c, hipError_t e, const char* what) {
  if (e != hipSuccess) return hip_fail(c, e, what);
  return ATSI_OK;
}

}  // namespace

extern "C" {

atsi_status atsi_create(int device, void* compute_stream, void* transfer_stream, void* workspace,
                        size_t workspace_bytes, int n_slots, atsi_ctx** out) {
  if (!out) return fail(nullptr, ATSI_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!compute_stream || !transfer_stream || compute_stream == transfer_stream)
    return fail(nullptr, ATSI_E_INVALID, "compute and transfer streams must be distinct and non-null");
  if (!workspace || ((uintptr_t)workspace % kAlign) != 0)
    return fail(nullptr, ATSI_E_INVALID, "workspace must be non-null and 256-byte aligned");
  if (n_slots < 2 || n_slots > 64) return fail(nullptr, ATSI_E_INVALID, "n_slots %d outside 2..64", n_slots);
  if (device < 0) return fail(nullptr, ATSI_E_INVALID, "device %d < 0", device);
  int ndev = 0;
  hipError_t e = hipGetDeviceCount(&ndev);
  if (e != hipSuccess || ndev <= device)
    return fail(nullptr, ATSI_E_HIP, "no usable GPU %d (hipGetDeviceCount: %s, count %d)", device,
                hipGetErrorString(e), ndev);
  e = hipSetDevice(device);
  if (e != hipSuccess) return fail(nullptr, ATSI_E_HIP, "hipSetDevice: %s", hipGetErrorString(e));
  atsi_ctx* c = new (std::nothrow) atsi_ctx;
  if (!c) return fail(nullptr, ATSI_E_INVALID, "out of host memory");
  c->device = device;
  c->cs = (hipStream_t)compute_stream;
  c->ts = (hipStream_t)transfer_stream;
  c->ws = (char*)workspace;
  c->ws_bytes = workspace_bytes;
  c->n_slots = n_slots;
  c->slots.resize(n_slots);
  for (Slot& s : c->slots) {
    if (hipEventCreateWithFlags(&s.ready, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&s.free, hipEventDisableTiming) != hipSuccess) {
      fail(nullptr, ATSI_E_HIP, "hipEventCreate failed");
      atsi_destroy(c);
      return ATSI_E_HIP;
    }
  }
  *out = c;
  return ATSI_OK;
}

atsi_status atsi_destroy(atsi_ctx* c) {
  if (!c) return ATSI_E_INVALID;
  hipSetDevice(c->device);
  if (c->cs) hipStreamSynchronize(c->cs);
  if (c->ts) hipStreamSynchronize(c->ts);
  for (Slot& s : c->slots) {
    if (s.ready) hipEventDestroy(s.ready);
    if (s.free) hipEventDestroy(s.free);
  }
  delete c;
  return ATSI_OK;
}

const char* atsi_last_error(const atsi_ctx* c) { return c ? c->err.c_str() : g_create_error.c_str(); }

atsi_status atsi_tensor_register(atsi_ctx* c, const atsi_qtensor* t, atsi_tid* out) {
  if (!c) return ATSI_E_INVALID;
  if (!t || !out) return fail(c, ATSI_E_INVALID, "tensor descriptor or out is NULL");
  if (t->group != kGroup) return fail(c, ATSI_E_SHAPE, "group %d unsupported (must be 32)", t->group);
  if (t->K < kGroup || t->K % kGroup != 0 || t->K > (1 << 20))
    return fail(c, ATSI_E_SHAPE, "K=%lld must be a positive multiple of 32 up to 2^20", (long long)t->K);
  if (t->N < 1 || t->N > (1 << 24)) return fail(c, ATSI_E_SHAPE, "N=%lld outside 1..2^24", (long long)t->N);
  const bool has_dev = t->dev_codes && t->dev_scales;
  const bool has_host = t->host_codes && t->host_scales;
  if ((t->dev_codes != nullptr) != (t->dev_scales != nullptr) ||
      (t->host_codes != nullptr) != (t->host_scales != nullptr))
    return fail(c, ATSI_E_INVALID, "codes and scales of a location must both be given or both be NULL");
  if (!has_dev && !has_host) return fail(c, ATSI_E_NO_COPY, "tensor has neither an HBM nor a host copy");
  if (has_dev && (!aligned16(t->dev_codes) || ((uintptr_t)t->dev_scales & 1u)))
    return fail(c, ATSI_E_INVALID, "device codes must be 16-byte aligned, scales 2-byte aligned");
  Tensor r;
  r.K = t->K;
  r.N = t->N;
  r.dcodes = t->dev_codes;
  r.dscales = t->dev_scales;
  r.hcodes = t->host_codes;
  r.hscales = t->host_scales;
  r.on_host = !has_dev;
  atsi_status st = enter(c);
  if (st) return st;
  c->tensors.push_back(r);
  *out = (atsi_tid)(c->tensors.size() - 1);
  if (r.on_host && r.slot_need() > c->slot_bytes) {
    st = layout_slots(c);
    if (st) {
      c->tensors.pop_back();
      *out = -1;
      return st;
    }
  }
  return ATSI_OK;
}

atsi_status atsi_set_placement(atsi_ctx* c, const uint8_t* host_mask, int32_t n) {
  if (!c) return ATSI_E_INVALID;
  if (!host_mask) return fail(c, ATSI_E_INVALID, "host_mask is NULL");
  if (n != (int32_t)c->tensors.size())
    return fail(c, ATSI_E_INVALID, "mask length %d != %zu registered tensors", n, c->tensors.size());
  for (int32_t i = 0; i < n; ++i) {
    const Tensor& t = c->tensors[i];
    if (host_mask[i] > 1) return fail(c, ATSI_E_INVALID, "mask[%d]=%d is not 0 or 1", i, host_mask[i]);
    if (host_mask[i] && !(t.hcodes && t.hscales))
      return fail(c, ATSI_E_NO_COPY, "tensor %d placed on host but has no host copy", i);
    if (!host_mask[i] && !(t.dcodes && t.dscales))
      return fail(c, ATSI_E_NO_COPY, "tensor %d placed in HBM but has no HBM copy", i);
  }
  atsi_status st = enter(c);
  if (st) return st;
  std::vector<bool> old(n);
  for (int32_t i = 0; i < n; ++i) {
    old[i] = c->tensors[i].on_host;
    c->tensors[i].on_host = host_mask[i] != 0;
  }
  st = layout_slots(c);
  if (st) {
    for (int32_t i = 0; i < n; ++i) c->tensors[i].on_host = old[i];
    return st;
  }
  return ATSI_OK;
}

atsi_status atsi_linear(atsi_ctx* c, atsi_tid w, const void* x, int64_t M, void* y) {
  if (!c) return ATSI_E_INVALID;
  if (!x || !y) return fail(c, ATSI_E_INVALID, "x or y is NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(c, ATSI_E_INVALID, "x and y must be 16-byte aligned");
  if (M < 1 || M > 65536) return fail(c, ATSI_E_SHAPE, "M=%lld outside 1..65536", (long long)M);
  atsi_status st = check_tid(c, w);
  if (st) return st;
  st = enter(c);
  if (st) return st;
  QView v;
  int slot;
  st = acquire(c, w, &v, &slot);
  if (st) return st;
  const __half* xh = (const __half*)x;
  __half* yh = (__half*)y;
  hipError_t e = (M <= 4) ? launch_gemv(v, xh, (int)M, yh, v.N, kStore, nullptr, c->cs)
                          : launch_gemm(v, xh, (int)M, yh, v.N, kStore, nullptr, c->cs);
  st = launched(c, e, M <= 4 ? "q4 gemv launch" : "q4 gemm launch");
  if (st) return st;
  return release(c, slot);
}

atsi_status atsi_sync(atsi_ctx* c) {
  if (!c) return ATSI_E_INVALID;
  hipError_t e = hipSetDevice(c->device);
  if (e == hipSuccess) e = hipStreamSynchronize(c->ts);
  if (e == hipSuccess) e = hipStreamSynchronize(c->cs);
  if (e != hipSuccess) hip_fail(c, e, "stream synchronize");
  if (c->latched != ATSI_OK) {
    c->err = c->latched_msg;
    return c->latched;
  }
  return ATSI_OK;
}

atsi_status atsi_debug_unpack(atsi_ctx* c, atsi_tid w, int8_t* q_out) {
  if (!c) return ATSI_E_INVALID;
  if (!q_out) return fail(c, ATSI_E_INVALID, "q_out is NULL");
  atsi_status st = check_tid(c, w);
  if (st) return st;
  st = enter(c);
  if (st) return st;
  QView v;
  int slot;
  st = acquire(c, w, &v, &slot);
  if (st) return st;
  st = launched(c, launch_unpack(v, q_out, c->cs), "unpack launch");
  if (st) return st;
  return release(c, slot);
}

}  // extern "C"
