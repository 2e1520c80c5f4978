// C-ABI layer: context, tensor registry, placement, the host-streaming engine
// and dispatch to the kernels.
//
// Streaming engine (Sec. 4.2.1-4.2.2 of the paper): host-resident tensors are
// copied from pinned memory into GPU temporary buffers ("slots") on the
// transfer stream and consumed on the compute stream.  Two kinds of events
// order the work: `ready` (recorded on the transfer stream after a copy,
// waited on by the compute stream before the consumer) and `free` (recorded
// on the compute stream after the consumer; the host checks it before the
// slot receives another copy), so a slot is never overwritten while read.
// Every slot records its own ready event after each copy into it, so a wait
// on a slot's event always names that slot's latest copy.
// Copies start as soon as a free slot allows: an explicit prefetch, or the
// schedule (the execution order of tensors) lets the transfer stream run
// ahead of compute by up to n_slots - 1 tensors.  A call that needs a copy
// while every slot is still being read waits on the host for the oldest
// reader to finish.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <deque>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/atsi.h"
#include "common.h"
#include "cpu_backend.h"
#include "layer.h"
#include "moe.h"

using namespace atsi;

namespace {

constexpr size_t kAlign = 256;
// Batch-1 decode of an all-resident 8B-shaped layer can run as one persistent
// launch (q4_layer.hip, the same bits as the four fused launches).  It is
// slower on MI355X than the four launches, so a context takes it only when
// ATSI_FUSED_DECODE_LAYER=1 is set at atsi_create.
inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }

struct Tensor {
  int64_t K = 0, N = 0;
  const uint8_t* dcodes = nullptr;
  const uint16_t* dscales = nullptr;
  const uint8_t* hcodes = nullptr;
  const uint16_t* hscales = nullptr;
  // device addresses of the host copy (mapped pinned memory), or null
  const uint8_t* zcodes = nullptr;
  const uint16_t* zscales = nullptr;
  bool on_host = false;
  bool on_cpu = false;  // runtime backend: runs on the CPU backend (a host tensor only)
  // a host tensor that runs on the GPU is copied into a slot for each use
  bool streamed() const { return on_host && !on_cpu; }
  size_t codes_bytes() const { return (size_t)(K / 2) * (size_t)N; }
  size_t scales_bytes() const { return (size_t)(K / kGroup) * (size_t)N * 2; }
  size_t bytes() const { return codes_bytes() + scales_bytes(); }
  // a slot holds the codes followed directly by the scales (16-byte aligned:
  // K/2 * N is a multiple of 16), the same layout as a contiguous host copy
  size_t slot_need() const { return align_up(bytes()); }
  bool host_contiguous() const { return hcodes && hcodes + codes_bytes() == reinterpret_cast<const uint8_t*>(hscales); }
};

// A slot is free (may receive a copy now), armed (a copy of `tid` has been
// issued into it and not consumed yet) or pending (its consumer is enqueued
// on the compute stream; it turns free once that launch's `free` event has
// completed).  Slots filled by one copy share its ready event and slots read
// by one launch share its free event.
struct Slot {
  char* base = nullptr;
  hipEvent_t ready = nullptr;     // owned; recorded after every copy into this slot
  hipEvent_t free = nullptr;      // owned
  hipEvent_t free_ev = nullptr;   // event of the launch that last read the slot
  uint64_t ready_rec = 0;         // number of the copy that fills the slot (slots of one run share it)
  bool armed = false;
  bool pending = false;
  int tid = -1;         // tensor whose copy the slot holds or receives
  uint64_t seq = 0;     // issue order of the armed copy
  uint64_t last = 0;    // last use (issue or consume), for round-robin reuse
  bool usable() const { return !armed && !pending; }
};

thread_local std::string g_create_error;

// Scratch of the allocation-free SwiGLU entry point (atsi_ffn_swiglu_noalloc):
// a file-scope device array, so each GPU the library runs on holds one copy
// until the process ends.  Host code never uses the array's name as an
// address: atsi_create looks up each device's copy once, with that device
// current, and calls pass that address to the kernels.  Calls on one GPU
// share the array (and see the last call's contents); overlapping calls on
// one GPU race.
constexpr size_t kStaticScratchBytes = 16u << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// The device address of this GPU's scratch array (device current), or null
// with *e set.
char* device_scratch(int device, hipError_t* e) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  *e = hipSuccess;
  if (device < 0 || device >= kMaxDevices) {
    *e = hipErrorInvalidDevice;
    return nullptr;
  }
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    *e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (*e != hipSuccess) return nullptr;
    g_scratch_ptr[device] = static_cast<char*>(p);
  }
  return g_scratch_ptr[device];
}

}  // namespace

namespace atsi {
// the message atsi_last_error(NULL) returns, for calls made without a context
void set_context_free_error(const char* msg) { g_create_error = msg; }
}  // namespace atsi

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
  size_t scratch_top = 0;  // end of the scratch the current call has taken
  std::vector<atsi_tid> schedule;  // execution order of tensors, repeated cyclically
  size_t sched_pos = 0;            // next schedule position not yet queued
  std::deque<atsi_tid> queue;      // host tensors to copy ahead, in consumption order
  std::deque<int> pending;         // pending slots in release order
  uint64_t clock = 0;
  // MoE expert tables, stacked down from the top of the workspace
  struct MoeTable {
    std::vector<atsi_tid> key;  // gate ids, up ids, down ids
    size_t off = 0;             // ExpertW[E] then uint8 resident[E]
    uint64_t version = ~0ull;   // placement version it was written for
    int n_streamed = 0;         // experts with a host-resident tensor
  };
  std::vector<MoeTable> tables;
  size_t table_floor = 0;       // lowest byte used by tables (ws_bytes if none)
  uint64_t placement_version = 0;
  unsigned* layer_bar = nullptr;  // barrier words of the fused decode layer (top of the workspace)
  unsigned* route_count = nullptr;  // the router's finished-workgroup count, after the barrier words
  float* row_inv = nullptr;       // per-row 1/rms for normalised prefill GEMMs (below the barrier words)
  bool layer_launched = false;    // a fused layer ran since the last atsi_sync
  bool fused_layer = false;       // batch-1 decode layers take the single persistent launch
  uint32_t debug = 0;             // ATSI_DEBUG_* flags (atsi_set_debug)
  bool zero_copy = false;         // decode experts on host are read in place (atsi_set_zero_copy)
  int moe_light_rows = -1;        // prefill experts routed at most this many pairs take the light kernels (-1: by call size)
  char* static_scratch = nullptr;  // this device's copy of the allocation-free entry point's scratch array
  hipStream_t ts2 = nullptr;      // the caller's second transfer stream, or null: copies alternate between ts and ts2
  unsigned copy_turn = 0;
  uint64_t copy_rec = 0;          // copies issued (numbers the ready records)
  int32_t* pinned = nullptr;    // caller's pinned host buffer for the per-expert counts, or null
  hipEvent_t counts_ev = nullptr;
  atsi_stats stats{};           // transfer counters (atsi_get_stats)
  // CPU backend (atsi_set_cpu_backend): the caller's pool and pinned staging
  atsi::cpu::Pool* pool = nullptr;
  char* staging = nullptr;
  char* staging_dev = nullptr;         // its device address (mapped pinned memory), or null
  size_t staging_bytes = 0;
  hipEvent_t cpu_ev = nullptr;         // a CPU launch's inputs have reached staging
  std::vector<float> cpu_x, cpu_acc;   // re-ordered fp32 inputs, fp32 products
  // timing (atsi_set_timing): event pairs resolved into per-tensor figures
  struct TimeRec {
    hipEvent_t a, b;
    int kind;  // offset of the field in atsi_tensor_timing, in doubles
    int n;
    atsi_tid tid[3];
    double share[3];
  };
  bool timing = false;
  std::vector<hipEvent_t> tev;          // timing events (created when timing is first enabled)
  size_t tev_used = 0;
  std::vector<TimeRec> trecs;
  std::vector<atsi_tensor_timing> timings;
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
  c->scratch_top = c->scratch_off;
  return ATSI_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

atsi_status check_tid(atsi_ctx* c, atsi_tid t) {
  if (t < 0 || (size_t)t >= c->tensors.size())
    return fail(c, ATSI_E_UNKNOWN_TENSOR, "unknown tensor id %d (registered: %zu)", t, c->tensors.size());
  return ATSI_OK;
}

// ---- timing (atsi_set_timing) ----
// Fields of atsi_tensor_timing, in doubles.
constexpr int kTimeGpu = 0, kTimeCpu = 1, kTimeD2H = 2, kTimeH2D = 3, kTimeW = 4;
constexpr size_t kTimingEvents = 2048;

double* timing_field(atsi_ctx* c, atsi_tid t, int kind) {
  if ((size_t)t >= c->timings.size()) {
    const double nan = std::numeric_limits<double>::quiet_NaN();
    c->timings.resize(c->tensors.size(), atsi_tensor_timing{nan, nan, nan, nan, nan});
  }
  return reinterpret_cast<double*>(&c->timings[t]) + kind;
}

// Shares of a multi-tensor operation, by byte size.
void byte_shares(atsi_ctx* c, const atsi_tid* tids, int n, double* share) {
  double tot = 0.0;
  for (int i = 0; i < n; ++i) tot += (double)c->tensors[tids[i]].bytes();
  for (int i = 0; i < n; ++i) share[i] = tot > 0.0 ? (double)c->tensors[tids[i]].bytes() / tot : 1.0 / n;
}

// Turn the recorded event pairs into per-tensor figures (drains the streams).
atsi_status resolve_timing(atsi_ctx* c) {
  if (c->trecs.empty()) return ATSI_OK;
  HIP_TRY(c, hipStreamSynchronize(c->cs));
  HIP_TRY(c, hipStreamSynchronize(c->ts));
  if (c->ts2) HIP_TRY(c, hipStreamSynchronize(c->ts2));
  for (const auto& r : c->trecs) {
    float ms = 0.f;
    HIP_TRY(c, hipEventElapsedTime(&ms, r.a, r.b));
    for (int i = 0; i < r.n; ++i) *timing_field(c, r.tid[i], r.kind) = (double)ms * 1e-3 * r.share[i];
  }
  c->trecs.clear();
  c->tev_used = 0;
  return ATSI_OK;
}

// Start timing an operation of `kind` on tensors tids (at most 3) on stream
// s; *rec = the record to close with time_end, or -1 with timing off.
atsi_status time_begin(atsi_ctx* c, int kind, const atsi_tid* tids, int n, hipStream_t s, int* rec) {
  *rec = -1;
  if (!c->timing || n < 1) return ATSI_OK;
  if (c->tev_used + 2 > c->tev.size()) {
    atsi_status st = resolve_timing(c);
    if (st) return st;
  }
  atsi_ctx::TimeRec r{};
  r.a = c->tev[c->tev_used++];
  r.b = c->tev[c->tev_used++];
  r.kind = kind;
  r.n = std::min(n, 3);
  for (int i = 0; i < r.n; ++i) r.tid[i] = tids[i];
  byte_shares(c, r.tid, r.n, r.share);
  HIP_TRY(c, hipEventRecord(r.a, s));
  c->trecs.push_back(r);
  *rec = (int)c->trecs.size() - 1;
  return ATSI_OK;
}

atsi_status time_end(atsi_ctx* c, int rec, hipStream_t s) {
  if (rec >= 0) HIP_TRY(c, hipEventRecord(c->trecs[rec].b, s));
  return ATSI_OK;
}

// Lay out n_slots slots sized for the largest host-resident tensor.
atsi_status layout_slots(atsi_ctx* c) {
  size_t need = 0;
  for (const Tensor& t : c->tensors)
    if (t.on_host) need = std::max(need, t.slot_need());
  if (need > 0 && (size_t)c->n_slots * need > c->table_floor)
    return fail(c, ATSI_E_WORKSPACE, "workspace %zu B (%zu B free of expert tables) < %d slots x %zu B",
                c->ws_bytes, c->table_floor, c->n_slots, need);
  HIP_TRY(c, hipStreamSynchronize(c->cs));
  HIP_TRY(c, hipStreamSynchronize(c->ts));
  if (c->ts2) HIP_TRY(c, hipStreamSynchronize(c->ts2));
  c->slot_bytes = need;
  for (int i = 0; i < c->n_slots; ++i) {
    Slot& s = c->slots[i];
    s.base = c->ws + (size_t)i * need;
    s.armed = false;
    s.pending = false;
    s.tid = -1;
    s.last = 0;
  }
  c->scratch_off = align_up((size_t)c->n_slots * need);
  c->sched_pos = 0;
  c->queue.clear();
  c->pending.clear();
  return ATSI_OK;
}

// Turn pending slots whose readers have finished back into free ones.  The
// compute stream completes launches in release order, so the scan stops at
// the first unfinished one.  With `block`, wait for the oldest pending launch
// first.  Reuse is decided here, on the host, rather than by making the
// transfer stream wait for compute-stream events: on ROCm such cross-stream
// waits in front of DMA copies have stalled the enqueueing thread for
// milliseconds.
atsi_status retire(atsi_ctx* c, bool block) {
  while (!c->pending.empty()) {
    const hipEvent_t ev = c->slots[c->pending.front()].free_ev;
    hipError_t e = hipEventQuery(ev);
    if (e == hipErrorNotReady) {
      if (!block) break;
      e = hipEventSynchronize(ev);
      block = false;
    }
    if (e != hipSuccess) return hip_fail(c, e, "free-event wait");
    while (!c->pending.empty() && c->slots[c->pending.front()].free_ev == ev) {
      c->slots[c->pending.front()].pending = false;
      c->pending.pop_front();
    }
  }
  return ATSI_OK;
}

// Poison mode: every byte of a slot about to receive a copy becomes 0xFF first
// (codes q = 7, scales fp16 NaN), on the transfer stream ahead of the copy, so
// a launch that read the slot before its copy landed would show NaN.  A fill
// kernel rather than a memset node, so that captured streams stay valid.
__global__ void poison_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
    p[i] = make_uint4(~0u, ~0u, ~0u, ~0u);
}

// The stream of the next copy: copies alternate between the two transfer
// streams, so two are in flight at once (a copy of a few MB spends a sizeable
// part of its time outside the transfer itself).  A copy's poison fill, copy
// and ready event all go on its stream.
hipStream_t copy_stream(atsi_ctx* c) { return (c->ts2 && (c->copy_turn++ & 1u)) ? c->ts2 : c->ts; }

// Before a copy into `bytes` at base (slot-aligned, whole slots) on stream xs:
// poison it, and in serialise mode let every launch already enqueued finish
// first.
atsi_status before_copy(atsi_ctx* c, char* base, size_t bytes, hipStream_t xs) {
  if (c->debug & ATSI_DEBUG_SERIALIZE) HIP_TRY(c, hipStreamSynchronize(c->cs));
  if (c->debug & ATSI_DEBUG_POISON) {
    const size_t n16 = bytes / 16;
    const unsigned blocks = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
    hipLaunchKernelGGL(poison_kernel, dim3(blocks), dim3(256), 0, xs, reinterpret_cast<uint4*>(base), n16);
    HIP_TRY(c, hipGetLastError());
  }
  return ATSI_OK;
}

// In serialise mode a copy completes before the host goes on.
atsi_status after_copy(atsi_ctx* c, hipStream_t xs) {
  if (c->debug & ATSI_DEBUG_SERIALIZE) HIP_TRY(c, hipStreamSynchronize(xs));
  return ATSI_OK;
}

// Copy host tensor t into slot s on the transfer stream: one copy when its
// host codes and scales are contiguous (small copies cost far more than their
// bytes), else two.  The slot must be free.
atsi_status copy_into(atsi_ctx* c, atsi_tid tid, Slot& s, hipStream_t xs) {
  const Tensor& t = c->tensors[tid];
  atsi_status st = before_copy(c, s.base, c->slot_bytes, xs);
  if (st) return st;
  int tr;
  if ((st = time_begin(c, kTimeW, &tid, 1, xs, &tr))) return st;
  if (t.host_contiguous()) {
    HIP_TRY(c, hipMemcpyAsync(s.base, t.hcodes, t.bytes(), hipMemcpyHostToDevice, xs));
    c->stats.h2d_copies += 1;
  } else {
    HIP_TRY(c, hipMemcpyAsync(s.base, t.hcodes, t.codes_bytes(), hipMemcpyHostToDevice, xs));
    HIP_TRY(c, hipMemcpyAsync(s.base + t.codes_bytes(), t.hscales, t.scales_bytes(), hipMemcpyHostToDevice, xs));
    c->stats.h2d_copies += 2;
  }
  if ((st = time_end(c, tr, xs))) return st;
  c->stats.h2d_bytes += t.bytes();
  c->stats.h2d_tensors += 1;
  return after_copy(c, xs);
}

void arm(atsi_ctx* c, Slot& s, atsi_tid tid, uint64_t rec) {
  s.tid = tid;
  s.armed = true;
  s.ready_rec = rec;
  s.seq = ++c->clock;
  s.last = s.seq;
}

bool held_by(const std::vector<int>& held, int i) { return std::find(held.begin(), held.end(), i) != held.end(); }

// Pick a slot for a new copy (never one in `held`).  Prefers the least
// recently used free slot.  Without `block`, returns -1 when none is free
// yet; with it, waits for pending slots and, when every other slot holds a
// prefetched copy, drops the copy furthest in the future and queues its
// tensor again.
atsi_status pick_slot(atsi_ctx* c, const std::vector<int>& held, bool block, int* out) {
  atsi_status st;
  for (;;) {
    int best = -1;
    for (int i = 0; i < c->n_slots; ++i) {
      const Slot& s = c->slots[i];
      if (s.usable() && !held_by(held, i) && (best < 0 || s.last < c->slots[best].last)) best = i;
    }
    if (best >= 0) {
      *out = best;
      return ATSI_OK;
    }
    const size_t before = c->pending.size();
    if (before > 0) {
      if ((st = retire(c, false))) return st;
      if (c->pending.size() < before) continue;
      if (!block) {
        *out = -1;
        return ATSI_OK;
      }
      if ((st = retire(c, true))) return st;
      continue;
    }
    if (!block) {
      *out = -1;
      return ATSI_OK;
    }
    for (int i = 0; i < c->n_slots; ++i) {
      const Slot& s = c->slots[i];
      if (s.armed && !held_by(held, i) && (best < 0 || s.seq > c->slots[best].seq)) best = i;
    }
    if (best < 0)
      return fail(c, ATSI_E_STATE, "one launch needs more streamed tensors than the %d slots", c->n_slots);
    // the dropped copy may still be in flight, possibly on the other transfer
    // stream than the copy that will replace it: let it land first, so it can
    // never overwrite the new contents
    HIP_TRY(c, hipEventSynchronize(c->slots[best].ready));
    c->queue.push_front(c->slots[best].tid);
    c->slots[best].armed = false;
    *out = best;
    return ATSI_OK;
  }
}

// Issue the H2D copy of host tensor `tid` into a slot; *slot_out is -1 when
// `block` is false and no slot is free.
atsi_status issue_copy(atsi_ctx* c, atsi_tid tid, bool block, const std::vector<int>& held, int* slot_out) {
  int si;
  atsi_status st = pick_slot(c, held, block, &si);
  if (st) return st;
  *slot_out = si;
  if (si < 0) return ATSI_OK;
  Slot& s = c->slots[si];
  hipStream_t xs = copy_stream(c);
  if ((st = copy_into(c, tid, s, xs))) return st;
  HIP_TRY(c, hipEventRecord(s.ready, xs));
  arm(c, s, tid, ++c->copy_rec);
  return ATSI_OK;
}

// Tensors registered back to back in one host buffer, each exactly one slot in
// size, can move with a single copy into adjacent free slots (an expert's
// gate, up and down, for instance).
bool run_candidate(atsi_ctx* c, const atsi_tid* tids, int n) {
  if (n < 2) return false;
  for (int i = 0; i < n; ++i) {
    const Tensor& t = c->tensors[tids[i]];
    if (!t.streamed() || !t.host_contiguous() || t.bytes() != c->slot_bytes) return false;
    if (i && c->tensors[tids[i - 1]].hcodes + c->slot_bytes != t.hcodes) return false;
  }
  return true;
}

// First slot of n adjacent free slots, in slot-aligned groups (first slot a
// multiple of n) so that runs never fragment each other; -1 if none.
int find_run(atsi_ctx* c, int n) {
  for (int j = 0; j + n <= c->n_slots; j += n) {
    bool ok = true;
    for (int i = 0; i < n && ok; ++i) ok = c->slots[j + i].usable();
    if (ok) return j;
  }
  return -1;
}

// Copy a run (see run_candidate) with one hipMemcpyAsync.  *issued is false
// when no aligned group of free slots exists (after retiring what finished).
atsi_status issue_run(atsi_ctx* c, const atsi_tid* tids, int n, bool* issued) {
  *issued = false;
  int first = find_run(c, n);
  if (first < 0) {
    atsi_status st = retire(c, false);
    if (st) return st;
    first = find_run(c, n);
  }
  if (first < 0) return ATSI_OK;
  Slot& s0 = c->slots[first];
  hipStream_t xs = copy_stream(c);
  atsi_status st = before_copy(c, s0.base, (size_t)n * c->slot_bytes, xs);
  if (st) return st;
  int tr;
  if ((st = time_begin(c, kTimeW, tids, n, xs, &tr))) return st;
  HIP_TRY(c, hipMemcpyAsync(s0.base, c->tensors[tids[0]].hcodes, (size_t)n * c->slot_bytes, hipMemcpyHostToDevice,
                            xs));
  if ((st = time_end(c, tr, xs))) return st;
  c->stats.h2d_copies += 1;
  c->stats.h2d_bytes += (uint64_t)n * c->slot_bytes;
  c->stats.h2d_tensors += (uint64_t)n;
  const uint64_t rec = ++c->copy_rec;
  for (int i = 0; i < n; ++i) {
    HIP_TRY(c, hipEventRecord(c->slots[first + i].ready, xs));
    arm(c, c->slots[first + i], tids[i], rec);
  }
  *issued = true;
  return after_copy(c, xs);
}

// Keep the transfer stream ahead of compute without waiting: copy queued (or
// scheduled) host tensors into free slots, leaving one slot for on-demand
// copies.
atsi_status topup(atsi_ctx* c) {
  int armed = 0;
  for (const Slot& s : c->slots) armed += s.armed ? 1 : 0;
  size_t guard = 0;
  atsi_status st;
  while (armed < c->n_slots - 1) {
    if (c->queue.empty()) {
      if (c->schedule.empty() || guard++ >= c->schedule.size()) break;
      atsi_tid t = c->schedule[c->sched_pos % c->schedule.size()];
      c->sched_pos++;
      if (c->tensors[t].streamed()) c->queue.push_back(t);
      continue;
    }
    if (c->queue.size() >= 3) {
      const atsi_tid run[3] = {c->queue[0], c->queue[1], c->queue[2]};
      if (run_candidate(c, run, 3)) {
        // an expert moves as one copy or waits for three aligned free slots
        bool issued = false;
        if (armed + 3 > c->n_slots - 1) break;
        if ((st = issue_run(c, run, 3, &issued))) return st;
        if (!issued) break;
        c->queue.erase(c->queue.begin(), c->queue.begin() + 3);
        armed += 3;
        guard = 0;
        continue;
      }
    }
    const atsi_tid t = c->queue.front();
    if (!c->tensors[t].streamed()) {
      c->queue.pop_front();
      continue;
    }
    int si;
    if ((st = issue_copy(c, t, false, {}, &si))) return st;
    if (si < 0) break;
    c->queue.pop_front();
    ++armed;
    guard = 0;
  }
  return ATSI_OK;
}

// Without a schedule, a multi-tensor call queues its own host tensors so their
// copies start before the first of them is needed.
atsi_status prefetch_call(atsi_ctx* c, const atsi_tid* tids, int n) {
  if (!c->schedule.empty()) return topup(c);
  for (int i = 0; i < n; ++i) {
    const atsi_tid t = tids[i];
    if (!c->tensors[t].streamed()) continue;
    bool have = std::find(c->queue.begin(), c->queue.end(), t) != c->queue.end();
    for (const Slot& s : c->slots) have = have || (s.armed && s.tid == t);
    if (!have) c->queue.push_back(t);
  }
  return topup(c);
}

int armed_slot(atsi_ctx* c, atsi_tid tid, const std::vector<int>& held) {
  int si = -1;
  for (int i = 0; i < c->n_slots; ++i) {
    const Slot& s = c->slots[i];
    if (s.armed && s.tid == tid && !held_by(held, i) && (si < 0 || s.seq < c->slots[si].seq)) si = i;
  }
  return si;
}

// Resolve where tensor `tid` is read from for the launch being assembled;
// for a host tensor the compute stream waits for its copy.  The slot index is
// appended to `held` (HBM tensors hold none).  A queued tensor is copied in
// queue order, waiting for slots to free up as needed.
atsi_status acquire(atsi_ctx* c, atsi_tid tid, QView* v, std::vector<int>& held) {
  const Tensor& t = c->tensors[tid];
  v->K = (int)t.K;
  v->N = (int)t.N;
  if (!t.on_host) {
    v->codes = t.dcodes;
    v->scales = t.dscales;
    return ATSI_OK;
  }
  atsi_status st;
  int si = armed_slot(c, tid, held);
  while (si < 0 && std::find(c->queue.begin(), c->queue.end(), tid) != c->queue.end()) {
    if ((st = topup(c))) return st;
    if ((si = armed_slot(c, tid, held)) >= 0 || c->pending.empty()) break;
    if ((st = retire(c, true))) return st;
  }
  if (si < 0) {
    auto q = std::find(c->queue.begin(), c->queue.end(), tid);
    if (q != c->queue.end()) c->queue.erase(q);
    if ((st = issue_copy(c, tid, true, held, &si))) return st;
  }
  Slot& s = c->slots[si];
  // one wait per copy: slots filled by one copy (a run) share its number
  bool waited = false;
  for (int h : held) waited = waited || c->slots[h].ready_rec == s.ready_rec;
  if (!waited) HIP_TRY(c, hipStreamWaitEvent(c->cs, s.ready, 0));
  v->codes = reinterpret_cast<const uint8_t*>(s.base);
  v->scales = reinterpret_cast<const uint16_t*>(s.base + t.codes_bytes());
  held.push_back(si);
  c->stats.host_reads += 1;
  c->stats.host_read_bytes += t.bytes();
  return ATSI_OK;
}

// After the consumer launch of the held slots has been enqueued.
atsi_status release(atsi_ctx* c, std::vector<int>& held) {
  if (!held.empty()) {
    const hipEvent_t ev = c->slots[held[0]].free;
    HIP_TRY(c, hipEventRecord(ev, c->cs));
    for (int si : held) {
      Slot& s = c->slots[si];
      s.free_ev = ev;
      s.armed = false;
      s.pending = true;
      s.last = ++c->clock;
      c->pending.push_back(si);
    }
  }
  held.clear();
  return topup(c);
}

// Bump allocator over the scratch region of the workspace (after the slots).
struct Scratch {
  atsi_ctx* c;
  size_t off;
  explicit Scratch(atsi_ctx* ctx) : c(ctx), off(ctx->scratch_off) {}
  __half* take(size_t elems, size_t elem_bytes = 2) {
    size_t need = align_up(elems * elem_bytes);
    if (off + need > c->table_floor) return nullptr;
    char* p = c->ws + off;
    off += need;
    c->scratch_top = std::max(c->scratch_top, off);
    return reinterpret_cast<__half*>(p);
  }
};

// Device table of expert weights for one MoE layer, cached at the top of the
// workspace and rewritten (by kernel, no host staging) when placement changes.
atsi_status get_table(atsi_ctx* c, const atsi_moe* m, atsi_ctx::MoeTable** out) {
  const int E = m->n_experts;
  std::vector<atsi_tid> key(3 * E);
  for (int e = 0; e < E; ++e) {
    key[e] = m->gate[e];
    key[E + e] = m->up[e];
    key[2 * E + e] = m->down[e];
  }
  atsi_ctx::MoeTable* tb = nullptr;
  for (auto& t : c->tables)
    if (t.key == key) tb = &t;
  if (!tb) {
    const size_t need = align_up((size_t)E * sizeof(ExpertW)) + align_up((size_t)E);
    if (c->table_floor < need || c->table_floor - need < c->scratch_off)
      return fail(c, ATSI_E_WORKSPACE, "no workspace left for a %d-expert table", E);
    c->table_floor -= need;
    c->tables.push_back(atsi_ctx::MoeTable{key, c->table_floor, ~0ull, 0});
    tb = &c->tables.back();
  }
  if (tb->version != c->placement_version) {
    ExpertW* dev = reinterpret_cast<ExpertW*>(c->ws + tb->off);
    uint8_t* res = reinterpret_cast<uint8_t*>(c->ws + tb->off + align_up((size_t)E * sizeof(ExpertW)));
    tb->n_streamed = 0;
    for (int e0 = 0; e0 < E; e0 += 16) {
      const int n = std::min(16, E - e0);
      ExpertW w[16];
      uint8_t r[16];
      for (int i = 0; i < n; ++i) {
        const Tensor* ts[3] = {&c->tensors[m->gate[e0 + i]], &c->tensors[m->up[e0 + i]], &c->tensors[m->down[e0 + i]]};
        QView* qv[3] = {&w[i].gate, &w[i].up, &w[i].down};
        bool resident = true;
        for (int j = 0; j < 3; ++j) {
          // a host tensor's entry is its mapped host copy in zero-copy mode
          // (read in place by the pair-indexed decode launches only)
          const bool z = ts[j]->on_host && c->zero_copy;
          *qv[j] = QView{z ? ts[j]->zcodes : ts[j]->dcodes, z ? ts[j]->zscales : ts[j]->dscales, (int)ts[j]->K,
                         (int)ts[j]->N};
          resident = resident && !ts[j]->on_host;
        }
        r[i] = resident ? 1 : 0;
        tb->n_streamed += resident ? 0 : 1;
      }
      hipError_t e = launch_table_patch(dev, res, e0, n, w, r, c->cs);
      if (e != hipSuccess) return hip_fail(c, e, "expert table patch");
    }
    tb->version = c->placement_version;
  }
  *out = tb;
  return ATSI_OK;
}

// Acquire the tensors of a fused launch (segment order; SwiGLU: gate, up),
// launch the GEMV (M <= 4) or the GEMM, release the slots.
atsi_status run_gpu_op(atsi_ctx* c, LinOp& op, const atsi_tid* tids, int ntids, bool workspace_scratch) {
  std::vector<int> held;
  atsi_status st;
  for (int i = 0; i < ntids; ++i) {
    QView v;
    st = acquire(c, tids[i], &v, held);
    if (st) return st;
    if (op.swiglu) {
      if (i == 0) op.seg[0].w = v; else op.seg[0].w2 = v;
    } else {
      op.seg[i].w = v;
    }
  }
  // Prefill on 512-row tiles (each weight dequantised once per 512 rows).  A
  // normalised input needs 1/rms per row from a small pass over x (the main
  // loop has no registers to spare for the sums); a launch with K ranges
  // needs their fp32 partial sums above the scratch this call has taken,
  // which nothing else uses until its reduction has run on the stream.
  int tr;  // timed from after the copy waits: the launch alone
  if ((st = time_begin(c, kTimeGpu, tids, ntids, c->cs, &tr))) return st;
  int wide = (op.norm && !c->row_inv) ? 0 : gemm_wide_splits(op);
  float* part = nullptr;
  if (wide > 1 && !workspace_scratch) wide = 0;  // no partial sums outside the workspace
  if (wide > 1) {
    const size_t at = align_up(c->scratch_top), need = gemm_wide_part_bytes(op, wide);
    if (at + need <= c->table_floor)
      part = reinterpret_cast<float*>(c->ws + at);
    else
      wide = 0;
  }
  if (wide) {
    if (op.norm) {
      hipError_t e = launch_rms_inv(op.x, op.M, op.K, op.eps, c->row_inv, c->cs);
      if (e != hipSuccess) return hip_fail(c, e, "row rms launch");
      op.rinv = c->row_inv;
    }
    hipError_t e = launch_gemm_wide(op, wide, part, c->cs);
    if (e != hipSuccess) return hip_fail(c, e, "q4 wide gemm launch");
    if ((st = time_end(c, tr, c->cs))) return st;
    return release(c, held);
  }
  // decode sizes: one token runs the GEMV, 2 to 16 the batched-decode kernel
  // on the matrix cores (both read the codes once); where that kernel does
  // not apply (K not a multiple of 128), up to 4 tokens run as GEMV launches
  // of at most gemv_tokens(K) tokens each; larger batches run the MFMA GEMM
  const int mt = gemv_tokens(op.K);
  const bool skinny = op.M >= kSkinnyMinTokens && op.M <= kSkinnyMaxTokens && skinny_supported(op);
  if (!skinny && op.M <= kGemvMaxTokens && mt > 0) {
    for (int m0 = 0; m0 < op.M; m0 += mt) {
      LinOp sub = op;
      sub.M = std::min(mt, op.M - m0);
      sub.x = op.x + (size_t)m0 * op.K;
      for (int s = 0; s < op.nseg; ++s) sub.seg[s].y = op.seg[s].y + (size_t)m0 * op.seg[s].ldy;
      if (op.res) sub.res = op.res + (size_t)m0 * op.seg[0].ldy;
      if (op.y32) sub.y32 = op.y32 + (size_t)m0 * op.seg[0].ldy;
      hipError_t e = launch_gemv(sub, c->cs);
      if (e != hipSuccess) return hip_fail(c, e, "q4 gemv launch");
    }
  } else if (skinny) {
    hipError_t e = launch_skinny(op, c->cs);
    if (e != hipSuccess) return hip_fail(c, e, "q4 batched-decode launch");
  } else {
    hipError_t e = launch_gemm(op, c->cs);
    if (e != hipSuccess) return hip_fail(c, e, "q4 gemm launch");
  }
  if ((st = time_end(c, tr, c->cs))) return st;
  return release(c, held);
}

// ---- CPU backend part of a launch ----
// Activation transfers of a CPU-run launch (the paper's copy kernel): GPU
// threads copy rows between device memory and mapped pinned staging, on the
// compute stream, so these small transfers never queue behind weight copies
// on the DMA engines.  rows x row_bytes, each side with its own pitch;
// 16-byte units where rows, pitches and both bases allow, else 2-byte units.
__global__ void stage_rows_kernel(const uint8_t* __restrict__ src, size_t spitch, uint8_t* __restrict__ dst,
                                  size_t dpitch, size_t row_bytes, int rows, int vec16) {
  const size_t per_row = vec16 ? row_bytes / 16 : row_bytes / 2;
  const size_t total = per_row * (size_t)rows;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const size_t r = i / per_row, col = i % per_row;
    if (vec16)
      *reinterpret_cast<uint4*>(dst + r * dpitch + col * 16) =
          *reinterpret_cast<const uint4*>(src + r * spitch + col * 16);
    else
      *reinterpret_cast<uint16_t*>(dst + r * dpitch + col * 2) =
          *reinterpret_cast<const uint16_t*>(src + r * spitch + col * 2);
  }
  __threadfence_system();  // host-side readers wait on an event recorded after the launch
}

// Copy rows on the compute stream: by the copy kernel when staging is mapped,
// else by the DMA engines.  host_side: the staging address (host pointer).
atsi_status stage_rows(atsi_ctx* c, const void* src, size_t spitch, void* dst, size_t dpitch, size_t row_bytes,
                       int rows, bool to_host) {
  if (rows <= 0 || row_bytes == 0) return ATSI_OK;
  if (!c->staging_dev) {
    HIP_TRY(c, hipMemcpy2DAsync(dst, dpitch, src, spitch, row_bytes, (size_t)rows,
                                to_host ? hipMemcpyDeviceToHost : hipMemcpyHostToDevice, c->cs));
    return ATSI_OK;
  }
  // the staging side is addressed through its device mapping
  auto dev = [&](const void* h) { return c->staging_dev + (static_cast<const char*>(h) - c->staging); };
  const uint8_t* s = static_cast<const uint8_t*>(to_host ? src : dev(src));
  uint8_t* d = reinterpret_cast<uint8_t*>(to_host ? dev(dst) : dst);
  const bool v16 = row_bytes % 16 == 0 && spitch % 16 == 0 && dpitch % 16 == 0 && ((uintptr_t)s % 16) == 0 &&
                   ((uintptr_t)d % 16) == 0;
  const size_t units = (v16 ? row_bytes / 16 : row_bytes / 2) * (size_t)rows;
  const unsigned blocks = (unsigned)std::min<size_t>((units + 255) / 256, 1024);
  hipLaunchKernelGGL(stage_rows_kernel, dim3(blocks), dim3(256), 0, c->cs, s, spitch, d, dpitch, row_bytes, rows,
                     v16 ? 1 : 0);
  HIP_TRY(c, hipGetLastError());
  return ATSI_OK;
}

// Staging regions of the CPU segments of one launch: the input rows, the
// residual (segment 0), and one packed output block per CPU segment.
struct CpuPlan {
  int seg[kMaxSeg];
  int n = 0;
  atsi_tid tids[kMaxSeg + 1];  // the CPU tensors (a SwiGLU pair counts two)
  int ntids = 0;
  char* x = nullptr;
  char* res = nullptr;
  char* out[kMaxSeg] = {};
  int N[kMaxSeg] = {};      // outputs of the segment's tensor
  int width[kMaxSeg] = {};  // output columns per row (N, or N * expand)
  int elem[kMaxSeg] = {};   // 2 (fp16) or 4 (fp32)
};

atsi_status cpu_plan(atsi_ctx* c, const LinOp& op, const bool* cpu, const atsi_tid* tids, CpuPlan* p) {
  if (!c->pool || !c->staging) return fail(c, ATSI_E_STATE, "a tensor runs on the CPU but no CPU backend is attached");
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* r = c->staging + off;
    off += align_up(bytes);
    return r;
  };
  const size_t M = (size_t)op.M;
  p->x = take(M * op.K * 2);
  for (int s = 0; s < op.nseg; ++s) {
    if (!cpu[s]) continue;
    const Seg& sg = op.seg[s];
    const int i = p->n++;
    p->seg[i] = s;
    if (op.swiglu) {
      p->tids[p->ntids++] = tids[0];
      p->tids[p->ntids++] = tids[1];
    } else {
      p->tids[p->ntids++] = tids[s];
    }
    // the launch's views are filled in only when a GPU part acquires them:
    // sizes come from the registered tensor
    p->N[i] = (int)c->tensors[op.swiglu ? tids[0] : tids[s]].N;
    p->width[i] = sg.expand > 1 ? p->N[i] * sg.expand : p->N[i];
    p->elem[i] = (s == 0 && op.y32) ? 4 : 2;
    p->out[i] = take(M * p->width[i] * p->elem[i]);
    if (s == 0 && op.res) p->res = take(M * p->N[i] * 2);
  }
  if (off > c->staging_bytes)
    return fail(c, ATSI_E_WORKSPACE, "CPU backend staging of %zu B < %zu B this %d-row launch needs",
                c->staging_bytes, off, op.M);
  return ATSI_OK;
}

// Inputs of the CPU part to staging, on the compute stream (after everything
// that produces them), then the event the host waits on.
atsi_status cpu_fetch(atsi_ctx* c, const LinOp& op, const CpuPlan& p) {
  atsi_status st;
  int tr;
  if ((st = time_begin(c, kTimeD2H, p.tids, p.ntids, c->cs, &tr))) return st;
  const size_t xrow = (size_t)op.K * 2;
  if ((st = stage_rows(c, op.x, xrow, p.x, xrow, xrow, op.M, true))) return st;
  if (p.res) {  // segment 0 is then the plan's first
    const size_t row = (size_t)p.N[0] * 2;
    if ((st = stage_rows(c, op.res, (size_t)op.seg[0].ldy * 2, p.res, row, row, op.M, true))) return st;
  }
  if ((st = time_end(c, tr, c->cs))) return st;
  HIP_TRY(c, hipEventRecord(c->cpu_ev, c->cs));
  return ATSI_OK;
}

// The CPU part proper: wait for the inputs, run the products on the pool,
// apply the launch's epilogue (the same semantics as the GPU's: RMS norm of
// the input, SwiGLU, grouped-query expansion, residual, fp32 or fp16 output)
// and copy the outputs back on the compute stream.
atsi_status cpu_finish(atsi_ctx* c, const LinOp& op, const CpuPlan& p) {
  // poll (a blocking wait wakes up tens of microseconds late), then block
  {
    hipError_t e = hipEventQuery(c->cpu_ev);
    const auto t0 = std::chrono::steady_clock::now();
    while (e == hipErrorNotReady && std::chrono::steady_clock::now() - t0 < std::chrono::milliseconds(20)) {
      std::this_thread::yield();
      e = hipEventQuery(c->cpu_ev);
    }
    if (e == hipErrorNotReady) e = hipEventSynchronize(c->cpu_ev);
    if (e != hipSuccess) return hip_fail(c, e, "waiting for a CPU launch's inputs");
  }
  const int M = op.M, K = op.K;
  c->cpu_x.resize((size_t)M * K);
  atsi::cpu::prepare_x(reinterpret_cast<const uint16_t*>(p.x), M, K, c->cpu_x.data());
  std::vector<float> inv((size_t)M, 1.f);
  if (op.norm)
    for (int m = 0; m < M; ++m) {
      double ss = 0.0;
      for (int k = 0; k < K; ++k) ss += (double)c->cpu_x[(size_t)m * K + k] * c->cpu_x[(size_t)m * K + k];
      inv[m] = (float)(1.0 / std::sqrt(ss / K + (double)op.eps));
    }
  const uint16_t* res = reinterpret_cast<const uint16_t*>(p.res);
  for (int i = 0; i < p.n; ++i) {
    const int s = p.seg[i];
    const Seg& sg = op.seg[s];
    const int N = p.N[i];
    const atsi_tid t0 = op.swiglu ? p.tids[0] : p.tids[i];
    const Tensor& w = c->tensors[t0];
    c->cpu_acc.resize((size_t)(op.swiglu ? 2 : 1) * M * N);
    float* acc = c->cpu_acc.data();
    const auto t_start = std::chrono::steady_clock::now();
    atsi::cpu::linear(*c->pool, w.hcodes, w.hscales, N, K, c->cpu_x.data(), M, acc);
    if (op.swiglu) {
      const Tensor& u = c->tensors[p.tids[1]];
      atsi::cpu::linear(*c->pool, u.hcodes, u.hscales, N, K, c->cpu_x.data(), M, acc + (size_t)M * N);
    }
    uint16_t* o16 = reinterpret_cast<uint16_t*>(p.out[i]);
    float* o32 = reinterpret_cast<float*>(p.out[i]);
    const int W = p.width[i];
    // the epilogue over rows [m0, m1); split over the pool when it is large
    auto epilogue = [&](int m0, int m1) {
    for (int m = m0; m < m1; ++m)
      for (int n = 0; n < N; ++n) {
        float v = acc[(size_t)m * N + n] * inv[m];
        if (op.swiglu) {
          const float u = acc[(size_t)(M + m) * N + n] * inv[m];
          v = v / (1.f + std::exp(-v)) * u;
        }
        if (sg.expand > 1) {
          const int hd = op.head_dim, jh = n / hd, d = n % hd;
          const uint16_t h = atsi::cpu::float_to_half_rn(v);
          for (int g = 0; g < sg.expand; ++g) o16[(size_t)m * W + (size_t)(jh * sg.expand + g) * hd + d] = h;
          continue;
        }
        if (s == 0 && res) v += atsi::cpu::half_to_float(res[(size_t)m * N + n]);
        if (p.elem[i] == 4)
          o32[(size_t)m * W + n] = v;
        else
          o16[(size_t)m * W + n] = atsi::cpu::float_to_half_rn(v);
      }
    };
    if ((size_t)M * N < (1u << 16) || M < 2) {
      epilogue(0, M);
    } else {
      const int T = c->pool->size();
      c->pool->run([&](int t) { epilogue((int)((int64_t)M * t / T), (int)((int64_t)M * (t + 1) / T)); });
    }
    const double secs = std::chrono::duration<double>(std::chrono::steady_clock::now() - t_start).count();
    if (c->timing) {
      double share[2] = {1.0, 0.0};
      const int nt = op.swiglu ? 2 : 1;
      const atsi_tid tt[2] = {t0, op.swiglu ? p.tids[1] : t0};
      if (nt == 2) byte_shares(c, tt, 2, share);
      for (int j = 0; j < nt; ++j) *timing_field(c, tt[j], kTimeCpu) = secs * share[j];
    }
  }
  atsi_status st;
  int tr;
  if ((st = time_begin(c, kTimeH2D, p.tids, p.ntids, c->cs, &tr))) return st;
  for (int i = 0; i < p.n; ++i) {
    const Seg& sg = op.seg[p.seg[i]];
    void* dst = (p.seg[i] == 0 && op.y32) ? (void*)op.y32 : (void*)sg.y;
    const size_t row = (size_t)p.width[i] * p.elem[i];
    if ((st = stage_rows(c, p.out[i], row, dst, (size_t)sg.ldy * p.elem[i], row, M, false))) return st;
  }
  return time_end(c, tr, c->cs);
}

// Run one fused launch: segments whose tensors are assigned to the CPU run
// on the CPU backend, the rest as one GPU launch that overlaps the CPU part.
atsi_status run_op(atsi_ctx* c, LinOp& op, const atsi_tid* tids, int ntids, bool workspace_scratch = true) {
  bool cpu[kMaxSeg] = {};
  int ncpu = 0;
  for (int s = 0; s < op.nseg; ++s) {
    const atsi_tid t = op.swiglu ? tids[0] : tids[s];
    cpu[s] = c->tensors[t].on_cpu;
    if (op.swiglu && c->tensors[tids[1]].on_cpu != cpu[s])
      return fail(c, ATSI_E_STATE, "gate %d and up %d of a SwiGLU pair must share a backend", tids[0], tids[1]);
    ncpu += cpu[s] ? 1 : 0;
  }
  if (ncpu == 0) return run_gpu_op(c, op, tids, ntids, workspace_scratch);
  if (!workspace_scratch) return fail(c, ATSI_E_STATE, "this entry point runs no tensor on the CPU backend");
  if (ncpu < op.nseg && (op.res || op.y32 || op.swiglu))
    return fail(c, ATSI_E_STATE, "a launch with a residual or fp32 output runs on one backend");
  CpuPlan p;
  atsi_status st = cpu_plan(c, op, cpu, tids, &p);
  if (st) return st;
  if ((st = cpu_fetch(c, op, p))) return st;
  if (ncpu < op.nseg) {
    LinOp g = op;
    g.nseg = 0;
    atsi_tid gt[kMaxSeg];
    for (int s = 0; s < op.nseg; ++s)
      if (!cpu[s]) {
        gt[g.nseg] = tids[s];
        g.seg[g.nseg++] = op.seg[s];
      }
    if ((st = run_gpu_op(c, g, gt, g.nseg, workspace_scratch))) return st;
  }
  return cpu_finish(c, op, p);
}

atsi_status check_act(atsi_ctx* c, const void* p, const char* what) {
  if (!p) return fail(c, ATSI_E_INVALID, "%s is NULL", what);
  if (!aligned16(p)) return fail(c, ATSI_E_INVALID, "%s must be 16-byte aligned", what);
  return ATSI_OK;
}

atsi_status check_m(atsi_ctx* c, int64_t M) {
  if (M < 1 || M > kMaxCallRows) return fail(c, ATSI_E_SHAPE, "M=%lld outside 1..%d", (long long)M, kMaxCallRows);
  return ATSI_OK;
}

// Attention half of a pre-norm decoder layer (tensors ids[0..3] = q, k, v, o):
//   1. q, k, v = rms(h) Wq, Wk, Wv in one launch; v goes straight to the
//      attention output of every query head of its group (context length 1);
//   2. h = h + attn Wo.
atsi_status run_attention(atsi_ctx* c, const atsi_tid* ids, int n_heads, int n_kv, int head_dim, float eps,
                          __half* hh, int Mi, __half* qb, __half* kb, __half* oin) {
  const Tensor &tq = c->tensors[ids[0]], &tk = c->tensors[ids[1]], &to = c->tensors[ids[3]];
  atsi_status st;
  LinOp a{};
  a.nseg = 3;
  a.x = hh; a.M = Mi; a.K = (int)tq.K; a.norm = 1; a.eps = eps; a.head_dim = head_dim;
  a.seg[0] = Seg{QView{}, QView{}, qb, (int)tq.N, 1};
  a.seg[1] = Seg{QView{}, QView{}, kb, (int)tk.N, 1};
  a.seg[2] = Seg{QView{}, QView{}, oin, (int)tq.N, n_heads / n_kv};
  if ((st = run_op(c, a, ids, 3))) return st;
  LinOp o = plain_op(QView{nullptr, nullptr, (int)to.K, (int)to.N}, oin, Mi, hh);
  o.res = hh;
  return run_op(c, o, &ids[3], 1);
}

// Shapes of the attention tensors of a layer with hidden H.
atsi_status check_attention(atsi_ctx* c, const atsi_tid* ids, int n_heads, int n_kv, int head_dim, float eps) {
  atsi_status st;
  for (int i = 0; i < 4; ++i)
    if ((st = check_tid(c, ids[i]))) return st;
  if (n_heads < 1 || n_kv < 1 || head_dim < 1 || n_heads % n_kv != 0 || !(eps >= 0.f))
    return fail(c, ATSI_E_SHAPE, "heads %d / kv heads %d / head_dim %d / eps invalid", n_heads, n_kv, head_dim);
  const Tensor &tq = c->tensors[ids[0]], &tk = c->tensors[ids[1]], &tv = c->tensors[ids[2]], &to = c->tensors[ids[3]];
  const int64_t H = tq.K, Hq = (int64_t)n_heads * head_dim, Hkv = (int64_t)n_kv * head_dim;
  if (tq.N != Hq || tk.K != H || tv.K != H || tk.N != Hkv || tv.N != Hkv || to.K != Hq || to.N != H)
    return fail(c, ATSI_E_SHAPE, "attention tensor shapes do not match hidden %lld, heads %d x %d", (long long)H,
                n_heads, head_dim);
  return ATSI_OK;
}

// Debug buffers must be 16-byte aligned device memory.
atsi_status check_layer_debug(atsi_ctx* c, const atsi_layer_debug* d) {
  if (d && ((d->attn && !aligned16(d->attn)) || (d->h_attn && !aligned16(d->h_attn)) ||
            (d->act && !aligned16(d->act)) || (d->sum32 && !aligned16(d->sum32))))
    return fail(c, ATSI_E_INVALID, "layer debug buffers must be 16-byte aligned");
  return ATSI_OK;
}

atsi_status check_moe_debug(atsi_ctx* c, const atsi_moe_debug* d) {
  if (d && ((d->expert_h && !aligned16(d->expert_h)) || (d->expert_out && !aligned16(d->expert_out))))
    return fail(c, ATSI_E_INVALID, "expert_h / expert_out must be 16-byte aligned");
  return ATSI_OK;
}

// The residual stream after the attention block, for a caller that asked.
atsi_status copy_h_attn(atsi_ctx* c, const atsi_layer_debug* d, const __half* hh, int M, int64_t H) {
  if (d && d->h_attn)
    HIP_TRY(c, hipMemcpyAsync(d->h_attn, hh, (size_t)M * H * 2, hipMemcpyDeviceToDevice, c->cs));
  return ATSI_OK;
}

// Validate an MoE descriptor and its experts' shapes.
atsi_status check_moe(atsi_ctx* c, const atsi_moe* m) {
  if (!m) return fail(c, ATSI_E_INVALID, "moe descriptor is NULL");
  const int E = m->n_experts, k = m->top_k;
  if (E < 16 || E > kMaxExperts || E % 16 != 0 || k < 1 || k > kMaxTopK || k > E)
    return fail(c, ATSI_E_SHAPE, "n_experts %d (multiple of 16, <= %d) / top_k %d (1..16) unsupported", E,
                kMaxExperts, k);
  if (m->hidden < 32 || m->hidden % 32 || m->inter < 32 || m->inter % 32)
    return fail(c, ATSI_E_SHAPE, "hidden %lld / inter %lld must be positive multiples of 32", (long long)m->hidden,
                (long long)m->inter);
  if (!m->router_w_f16 || !aligned16(m->router_w_f16) || !m->gate || !m->up || !m->down)
    return fail(c, ATSI_E_INVALID, "router weights (16-byte aligned) and expert id arrays are required");
  const int H = (int)m->hidden, I = (int)m->inter;
  atsi_status st;
  for (int e = 0; e < E; ++e) {
    if ((st = check_tid(c, m->gate[e])) || (st = check_tid(c, m->up[e])) || (st = check_tid(c, m->down[e]))) return st;
    const Tensor &g = c->tensors[m->gate[e]], &u = c->tensors[m->up[e]], &d = c->tensors[m->down[e]];
    if (g.K != H || g.N != I || u.K != H || u.N != I || d.K != I || d.N != H)
      return fail(c, ATSI_E_SHAPE, "expert %d: gate/up must be %d x %d and down %d x %d", e, H, I, I, H);
    if (g.on_cpu || u.on_cpu || d.on_cpu)
      return fail(c, ATSI_E_STATE, "expert %d is assigned to the CPU backend; experts run on the GPU only", e);
  }
  return ATSI_OK;
}

// The SwiGLU activations of the routed pairs in pair order, for a caller that
// asked: row i of h belongs to pair perm[i] (bucketed) or to pair i.
atsi_status gather_expert_h(atsi_ctx* c, const atsi_moe_debug* d, const __half* h, const int32_t* perm, int rows,
                            int I) {
  if (!d || !d->expert_h) return ATSI_OK;
  hipError_t e = launch_gather_rows(h, perm, rows, I, (__half*)d->expert_h, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "expert activation gather");
  return ATSI_OK;
}

// The routed MoE FFN (validated descriptor): y = sum_j p_j FFN_{e_j}(x) for
// each token, plus res when res is given (y may then alias res but not x);
// with inv_r the input is x * inv_r[t] per token (make_inv: the factors are
// computed here into inv_r, with eps), the factor applied to the
// router logits and the expert gate/up products.
atsi_status run_moe(atsi_ctx* c, const atsi_moe* m, const __half* x, int Mi, __half* y, const atsi_moe_debug* dbg,
                    float* inv_r, bool make_inv, float eps, const __half* res, Scratch& sc) {
  atsi_status st;
  if (!c->pinned && !(Mi <= 4 && c->zero_copy))
    for (int e = 0; e < m->n_experts; ++e)
      if (c->tensors[m->gate[e]].on_host || c->tensors[m->up[e]].on_host || c->tensors[m->down[e]].on_host)
        return fail(c, ATSI_E_STATE, "streamed experts need the pinned host_counts buffer given to atsi_create");
  atsi_ctx::MoeTable* tb;
  if ((st = get_table(c, m, &tb))) return st;
  const int E = m->n_experts, k = m->top_k;
  const int H = (int)m->hidden, I = (int)m->inter;
  const int Mk = Mi * k;
  const bool gemv = Mi <= 4;
  const int bm = expert_tile_rows(gemv);
  // experts routed at most `light` pairs run on the light-expert kernels (by
  // default all of them: faster than the grouped GEMM at 64, 512 and 2048
  // tokens of the 128-expert layer on MI355X)
  int light = c->moe_light_rows < 0 ? kMoeLightRowsMax : c->moe_light_rows;
  if (gemv || !light_supported(H, I) || (size_t)Mk * std::max(H, I) * 2 >= ((size_t)1 << 31)) light = 0;
  // taller tiles pay off once experts are routed many tokens; below that the
  // extra launches' latency costs more than they save (MI355X: 16-row tiles
  // only up to 16 pairs per expert on average).  Where the shape allows only
  // 16-row tiles, large calls keep the grouped GEMM by default: heavy experts
  // would be streamed once per 16 of their rows.
  const bool tall = Mk > kLightTallPairs * E;
  if (tall && c->moe_light_rows < 0 && light && light_mtmax(H, I) < 2) light = 0;
  const int lmt = !light ? 0 : (tall ? light_mtmax(H, I) : 1);
  float* part = (float*)sc.take(router_partial_floats(Mi, H, E), 4);
  int32_t* idx = dbg && dbg->idx ? dbg->idx : (int32_t*)sc.take(Mk, 4);
  float* p = dbg && dbg->p ? dbg->p : (float*)sc.take(Mk, 4);
  int32_t* counts = dbg && dbg->counts ? dbg->counts : (int32_t*)sc.take(E, 4);
  int32_t* offsets = dbg && dbg->offsets ? dbg->offsets : (int32_t*)sc.take(E + 1, 4);
  int32_t* perm = dbg && dbg->perm ? dbg->perm : (int32_t*)sc.take(Mk, 4);
  int32_t* inv = dbg && dbg->inv_perm ? dbg->inv_perm : (int32_t*)sc.take(Mk, 4);
  int32_t* order = (int32_t*)sc.take(E, 4);
  int32_t* tiles = (int32_t*)sc.take(2 * ((size_t)Mk / bm + E + 1), 4);
  int32_t* ntiles = (int32_t*)sc.take(1, 4);
  int32_t* ltiles = light ? (int32_t*)sc.take(2 * ((size_t)Mk / kLightTileRows + E + 1), 4) : nullptr;
  int32_t* nltiles = light ? (int32_t*)sc.take(kLightClasses, 4) : nullptr;
  __half* h = sc.take((size_t)Mk * I);
  __half* out = dbg && dbg->expert_out ? (__half*)dbg->expert_out : sc.take((size_t)Mk * H);
  if (!part || !idx || !p || !counts || !offsets || !perm || !inv || !order || !tiles || !ntiles || !h || !out ||
      (light && (!ltiles || !nltiles)))
    return fail(c, ATSI_E_WORKSPACE, "scratch too small for a %d-token MoE layer", Mi);
  const ExpertW* table = reinterpret_cast<const ExpertW*>(c->ws + tb->off);
  const uint8_t* resident = reinterpret_cast<const uint8_t*>(c->ws + tb->off + align_up((size_t)E * sizeof(ExpertW)));

  hipError_t e = launch_router(x, make_inv ? nullptr : inv_r, make_inv ? inv_r : nullptr, eps,
                               (const __half*)m->router_w_f16, m->router_bias, Mi, H, E, k, part, idx, p,
                               dbg ? dbg->logits : nullptr, c->route_count, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "router launch");
  // decode with every expert resident, or with host experts read in place
  // (zero-copy): the expert launches index routed pairs directly, and the
  // bucketing only runs when the caller asks for its output
  const bool by_pair = gemv && (tb->n_streamed == 0 || c->zero_copy);
  const bool want_buckets = dbg && (dbg->counts || dbg->offsets || dbg->perm || dbg->inv_perm);
  if (!by_pair || want_buckets) {
    e = launch_bucket(idx, Mi, k, E, resident, bm, light, lmt, counts, offsets, perm, inv, order, tiles, ntiles,
                      ltiles, nltiles, c->cs);
    if (e != hipSuccess) return hip_fail(c, e, "bucket launch");
  }
  if (tb->n_streamed > 0 && !by_pair) {
    HIP_TRY(c, hipMemcpyAsync(c->pinned, counts, E * sizeof(int32_t), hipMemcpyDeviceToHost, c->cs));
    HIP_TRY(c, hipEventRecord(c->counts_ev, c->cs));
  }
  MoeArgs a{};
  a.table = table;
  a.tiles = tiles;
  a.n_tiles = ntiles;
  a.counts = counts;
  a.offsets = offsets;
  a.perm = perm;
  a.x = x;
  a.h = h;
  a.out = out;
  a.inv_r = inv_r;
  a.k = k;
  a.M = Mi;
  a.H = H;
  a.I = I;
  if (by_pair) {
    a.pair_expert = idx;
    a.n_pairs = Mk;
    a.n_experts = E;
  }
  // HBM-resident experts first: they run while the host learns which
  // streamed experts are needed.  Grid bounds: tiles of bm rows over experts
  // routed more than `light` pairs, and light tiles over the others.
  const int heavy = std::min(E, Mk / (light + 1));  // experts that can be routed more than `light` pairs
  const int bound = bm == 1 ? Mk : (heavy > 0 ? Mk / bm + heavy : 0);
  const int lbound = light ? std::min(Mk / kLightTileRows + E, E * ((light + kLightTileRows - 1) / kLightTileRows)) : 0;
  MoeArgs al = a;
  al.tiles = ltiles;
  al.n_tiles = nltiles;
  if ((e = launch_expert_gateup(a, bound, gemv, c->cs)) != hipSuccess) return hip_fail(c, e, "expert gate/up launch");
  // one launch for every light tile height the shape allows
  if (lmt && (e = launch_light_all_gateup(al, lmt, lbound, c->cs)) != hipSuccess)
    return hip_fail(c, e, "light expert gate/up launch");
  if (by_pair) {  // every expert resident: the down launch also combines
    a.store_out = dbg && dbg->expert_out;
    if ((e = launch_expert_down_combine(a, Mi, p, res, y, c->cs)) != hipSuccess)
      return hip_fail(c, e, "expert down/combine launch");
    return gather_expert_h(c, dbg, h, nullptr, Mk, I);
  }
  if ((e = launch_expert_down(a, bound, gemv, c->cs)) != hipSuccess) return hip_fail(c, e, "expert down launch");
  if (lmt && (e = launch_light_all_down(al, lmt, lbound, c->cs)) != hipSuccess)
    return hip_fail(c, e, "light expert down launch");

  if (tb->n_streamed > 0) {
    HIP_TRY(c, hipEventSynchronize(c->counts_ev));
    std::vector<int> act;
    for (int ex = 0; ex < E; ++ex) {
      const Tensor &g = c->tensors[m->gate[ex]], &u = c->tensors[m->up[ex]], &d = c->tensors[m->down[ex]];
      if ((g.on_host || u.on_host || d.on_host) && c->pinned[ex] > 0) act.push_back(ex);
    }
    std::stable_sort(act.begin(), act.end(), [&](int l, int r) { return c->pinned[l] > c->pinned[r]; });
    for (int ex : act)
      for (const atsi_tid t : {m->gate[ex], m->up[ex], m->down[ex]})
        if (c->tensors[t].on_host) c->queue.push_back(t);
    if ((st = topup(c))) return st;
    const int B = std::max(1, std::min(kBatchExp, c->n_slots / 3));
    for (size_t b0 = 0; b0 < act.size(); b0 += B) {
      std::vector<int> held;
      MoeArgs ba = a;  // tiles of bm rows / light tiles of each class of the batch
      ba.nb = 0;
      MoeArgs bl[kLightClasses] = {a, a, a};
      for (MoeArgs& q : bl) q.nb = 0;
      const int nbx = (int)std::min<size_t>(B, act.size() - b0);
      for (int b = 0; b < nbx; ++b) {
        const int ex = act[b0 + b];
        ba.bexp[b] = ex;
        if ((st = acquire(c, m->gate[ex], &ba.bw[b].gate, held)) || (st = acquire(c, m->up[ex], &ba.bw[b].up, held)) ||
            (st = acquire(c, m->down[ex], &ba.bw[b].down, held)))
          return st;
        for (MoeArgs& q : bl) {
          q.bexp[b] = ex;
          q.bw[b] = ba.bw[b];
        }
      }
      auto flush = [&]() -> atsi_status {
        hipError_t fe = hipSuccess;
        if (ba.nb > 0) fe = launch_expert_gateup(ba, ba.nb, gemv, c->cs);
        for (int q = 0; q < kLightClasses; ++q)
          if (fe == hipSuccess && bl[q].nb > 0) fe = launch_light_gateup(bl[q], q, bl[q].nb, c->cs);
        if (fe == hipSuccess && ba.nb > 0) fe = launch_expert_down(ba, ba.nb, gemv, c->cs);
        for (int q = 0; q < kLightClasses; ++q)
          if (fe == hipSuccess && bl[q].nb > 0) fe = launch_light_down(bl[q], q, bl[q].nb, c->cs);
        if (fe != hipSuccess) return hip_fail(c, fe, "streamed expert launch");
        ba.nb = 0;
        for (MoeArgs& q : bl) q.nb = 0;
        return ATSI_OK;
      };
      for (int b = 0; b < nbx; ++b) {
        // the same tiles as a resident expert with this count gets
        const int cnt = c->pinned[act[b0 + b]];
        const bool lt = cnt <= light;
        const int lmtb = lt ? light_mt(cnt, lmt) : 0;
        MoeArgs& dst = lt ? bl[light_class(lmtb)] : ba;
        for (int r0 = 0; r0 < cnt; r0 += lt ? kLightTileRows * lmtb : bm) {
          if (dst.nb == kBatchTiles && (st = flush())) return st;
          dst.btiles[dst.nb++] = make_int2(b, r0);
        }
      }
      if ((st = flush())) return st;
      if ((st = release(c, held))) return st;
    }
  }
  e = launch_combine(out, p, Mi, k, H, res, y, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "combine launch");
  return gather_expert_h(c, dbg, h, perm, Mk, I);
}

}  // namespace

extern "C" {

atsi_status atsi_create(int device, void* compute_stream, void* transfer_stream, void* transfer_stream2,
                        void* workspace, size_t workspace_bytes, int32_t* host_counts, int n_slots, atsi_ctx** out) {
  if (!out) return fail(nullptr, ATSI_E_INVALID, "out is NULL");
  *out = nullptr;
  if (!compute_stream || !transfer_stream || compute_stream == transfer_stream)
    return fail(nullptr, ATSI_E_INVALID, "compute and transfer streams must be distinct and non-null");
  if (transfer_stream2 && (transfer_stream2 == compute_stream || transfer_stream2 == transfer_stream))
    return fail(nullptr, ATSI_E_INVALID, "the second transfer stream must differ from the other two");
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
  c->ts2 = (hipStream_t)transfer_stream2;
  c->pinned = host_counts;
  c->static_scratch = device_scratch(device, &e);
  if (!c->static_scratch) {
    delete c;
    return fail(nullptr, ATSI_E_HIP, "hipGetSymbolAddress of the static scratch: %s", hipGetErrorString(e));
  }
  if (const char* f = getenv("ATSI_FUSED_DECODE_LAYER")) c->fused_layer = atoi(f) == 1;
  c->table_floor = workspace_bytes / kAlign * kAlign;
  const size_t bar_bytes = align_up((kLayerBarrierWords + 1) * sizeof(unsigned));
  if (c->table_floor < bar_bytes) {
    delete c;
    return fail(nullptr, ATSI_E_WORKSPACE, "workspace of %zu B is too small", workspace_bytes);
  }
  c->table_floor -= bar_bytes;
  c->layer_bar = reinterpret_cast<unsigned*>(c->ws + c->table_floor);
  c->route_count = c->layer_bar + kLayerBarrierWords;
  // one float per activation row of the largest call (M <= 65536); left out of
  // small workspaces, where normalised prefill GEMMs keep the 128-row tiles
  const size_t rinv_bytes = align_up((size_t)kMaxCallRows * sizeof(float));
  if (c->table_floor >= 2 * rinv_bytes) {
    c->table_floor -= rinv_bytes;
    c->row_inv = reinterpret_cast<float*>(c->ws + c->table_floor);
  }
  c->slots.resize(n_slots);
  if (hipEventCreateWithFlags(&c->counts_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->cpu_ev, hipEventDisableTiming) != hipSuccess) {
    fail(nullptr, ATSI_E_HIP, "hipEventCreate failed");
    atsi_destroy(c);
    return ATSI_E_HIP;
  }
  for (Slot& s : c->slots) {
    if (hipEventCreateWithFlags(&s.ready, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&s.free, hipEventDisableTiming) != hipSuccess) {
      fail(nullptr, ATSI_E_HIP, "hipEventCreate failed");
      atsi_destroy(c);
      return ATSI_E_HIP;
    }
  }
  // the fused decode layer's barrier and the router's count start from zeroed
  // words and leave them so
  if (hipMemsetAsync(c->layer_bar, 0, bar_bytes, c->cs) != hipSuccess || hipStreamSynchronize(c->cs) != hipSuccess) {
    fail(nullptr, ATSI_E_HIP, "clearing the workspace barrier words failed");
    atsi_destroy(c);
    return ATSI_E_HIP;
  }
  *out = c;
  return ATSI_OK;
}

atsi_status atsi_destroy(atsi_ctx* c) {
  if (!c) return ATSI_E_INVALID;
  (void)hipSetDevice(c->device);
  if (c->cs) (void)hipStreamSynchronize(c->cs);
  if (c->ts) (void)hipStreamSynchronize(c->ts);
  if (c->ts2) (void)hipStreamSynchronize(c->ts2);
  for (Slot& s : c->slots) {
    if (s.ready) (void)hipEventDestroy(s.ready);
    if (s.free) (void)hipEventDestroy(s.free);
  }
  if (c->counts_ev) (void)hipEventDestroy(c->counts_ev);
  if (c->cpu_ev) (void)hipEventDestroy(c->cpu_ev);
  for (hipEvent_t e : c->tev) (void)hipEventDestroy(e);
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
  if (has_host) {
    void *zc = nullptr, *zs = nullptr;
    if (hipHostGetDevicePointer(&zc, const_cast<uint8_t*>(t->host_codes), 0) == hipSuccess &&
        hipHostGetDevicePointer(&zs, const_cast<uint16_t*>(t->host_scales), 0) == hipSuccess) {
      r.zcodes = static_cast<const uint8_t*>(zc);
      r.zscales = static_cast<const uint16_t*>(zs);
    } else {
      (void)hipGetLastError();  // not mapped pinned memory: no zero-copy reads of this tensor
    }
    if (c->zero_copy && !r.zcodes)
      return fail(c, ATSI_E_INVALID, "zero-copy mode: the host copy is not mapped pinned memory");
  }
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
  std::vector<bool> old(n), old_cpu(n);
  for (int32_t i = 0; i < n; ++i) {
    old[i] = c->tensors[i].on_host;
    old_cpu[i] = c->tensors[i].on_cpu;
    c->tensors[i].on_host = host_mask[i] != 0;
    c->tensors[i].on_cpu = c->tensors[i].on_cpu && c->tensors[i].on_host;  // HBM tensors run on the GPU
  }
  st = layout_slots(c);
  if (st) {
    for (int32_t i = 0; i < n; ++i) {
      c->tensors[i].on_host = old[i];
      c->tensors[i].on_cpu = old_cpu[i];
    }
    return st;
  }
  ++c->placement_version;
  return ATSI_OK;
}

atsi_status atsi_linear(atsi_ctx* c, atsi_tid w, const void* x, int64_t M, void* y) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, y, "y")) || (st = check_m(c, M)) || (st = check_tid(c, w)))
    return st;
  if ((st = enter(c))) return st;
  const Tensor& t = c->tensors[w];
  QView v{nullptr, nullptr, (int)t.K, (int)t.N};
  LinOp op = plain_op(v, (const __half*)x, (int)M, (__half*)y);
  return run_op(c, op, &w, 1);
}

atsi_status atsi_ffn_swiglu(atsi_ctx* c, atsi_tid gate, atsi_tid up, atsi_tid down, const void* x, int64_t M,
                            void* y) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, y, "y")) || (st = check_m(c, M)) ||
      (st = check_tid(c, gate)) || (st = check_tid(c, up)) || (st = check_tid(c, down)))
    return st;
  const Tensor &tg = c->tensors[gate], &tu = c->tensors[up], &td = c->tensors[down];
  if (tg.K != tu.K || tg.N != tu.N || td.K != tg.N || td.N != tg.K)
    return fail(c, ATSI_E_SHAPE, "SwiGLU shapes: gate/up must be H x I and down I x H");
  if (x == y) return fail(c, ATSI_E_INVALID, "y must not alias x");
  if ((st = enter(c))) return st;
  Scratch sc(c);
  __half* h = sc.take((size_t)M * tg.N);
  if (!h) return fail(c, ATSI_E_WORKSPACE, "scratch too small for the %lld x %lld SwiGLU activation",
                      (long long)M, (long long)tg.N);
  const atsi_tid order[3] = {gate, up, down};
  if ((st = prefetch_call(c, order, 3))) return st;
  // gate/up with the SwiGLU product fused: h = silu(x Wg) * (x Wu)
  LinOp gu = plain_op(QView{nullptr, nullptr, (int)tg.K, (int)tg.N}, (const __half*)x, (int)M, h);
  gu.swiglu = 1;
  if ((st = run_op(c, gu, order, 2))) return st;
  // down: y = h Wd
  LinOp dn = plain_op(QView{nullptr, nullptr, (int)td.K, (int)td.N}, h, (int)M, (__half*)y);
  return run_op(c, dn, &order[2], 1);
}

atsi_status atsi_ffn_swiglu_noalloc(atsi_ctx* c, atsi_tid gate, atsi_tid up, atsi_tid down, const void* x,
                                    int64_t M, void* y) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, y, "y")) || (st = check_m(c, M)) ||
      (st = check_tid(c, gate)) || (st = check_tid(c, up)) || (st = check_tid(c, down)))
    return st;
  const Tensor &tg = c->tensors[gate], &tu = c->tensors[up], &td = c->tensors[down];
  if (tg.K != tu.K || tg.N != tu.N || td.K != tg.N || td.N != tg.K)
    return fail(c, ATSI_E_SHAPE, "SwiGLU shapes: gate/up must be H x I and down I x H");
  if (x == y) return fail(c, ATSI_E_INVALID, "y must not alias x");
  const size_t need = (size_t)M * (size_t)tg.N * 2;
  if (need > kStaticScratchBytes)
    return fail(c, ATSI_E_WORKSPACE, "the %lld x %lld SwiGLU activation (%zu B) exceeds the %zu B static scratch",
                (long long)M, (long long)tg.N, need, kStaticScratchBytes);
  if ((st = enter(c))) return st;
  __half* h = reinterpret_cast<__half*>(c->static_scratch);
  const atsi_tid order[3] = {gate, up, down};
  if ((st = prefetch_call(c, order, 3))) return st;
  LinOp gu = plain_op(QView{nullptr, nullptr, (int)tg.K, (int)tg.N}, (const __half*)x, (int)M, h);
  gu.swiglu = 1;
  if ((st = run_op(c, gu, order, 2, false))) return st;
  LinOp dn = plain_op(QView{nullptr, nullptr, (int)td.K, (int)td.N}, h, (int)M, (__half*)y);
  return run_op(c, dn, &order[2], 1, false);
}

atsi_status atsi_swiglu_gate_up(atsi_ctx* c, atsi_tid gate, atsi_tid up, const void* x, int64_t M, void* h) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, h, "h")) || (st = check_m(c, M)) ||
      (st = check_tid(c, gate)) || (st = check_tid(c, up)))
    return st;
  const Tensor &tg = c->tensors[gate], &tu = c->tensors[up];
  if (tg.K != tu.K || tg.N != tu.N) return fail(c, ATSI_E_SHAPE, "gate and up must have the same shape");
  if (x == h) return fail(c, ATSI_E_INVALID, "h must not alias x");
  if ((st = enter(c))) return st;
  const atsi_tid order[2] = {gate, up};
  if ((st = prefetch_call(c, order, 2))) return st;
  LinOp gu = plain_op(QView{nullptr, nullptr, (int)tg.K, (int)tg.N}, (const __half*)x, (int)M, (__half*)h);
  gu.swiglu = 1;
  return run_op(c, gu, order, 2);
}

atsi_status atsi_decoder_layer(atsi_ctx* c, const atsi_dense_layer* L, void* h, int64_t M, void* q_out,
                               void* k_out, const atsi_layer_debug* dbg) {
  if (!c) return ATSI_E_INVALID;
  if (!L) return fail(c, ATSI_E_INVALID, "layer descriptor is NULL");
  atsi_status st;
  if ((st = check_act(c, h, "h")) || (st = check_m(c, M))) return st;
  if ((q_out && !aligned16(q_out)) || (k_out && !aligned16(k_out)))
    return fail(c, ATSI_E_INVALID, "q_out / k_out must be 16-byte aligned");
  if ((st = check_layer_debug(c, dbg))) return st;
  const atsi_tid ids[7] = {L->q, L->k, L->v, L->o, L->gate, L->up, L->down};
  for (atsi_tid t : ids)
    if ((st = check_tid(c, t))) return st;
  if ((st = check_attention(c, ids, L->n_heads, L->n_kv_heads, L->head_dim, L->eps))) return st;
  const Tensor &tq = c->tensors[L->q];
  const Tensor &tg = c->tensors[L->gate], &tu = c->tensors[L->up], &td = c->tensors[L->down];
  const int64_t H = tq.K;
  const int64_t Hq = (int64_t)L->n_heads * L->head_dim, Hkv = (int64_t)L->n_kv_heads * L->head_dim;
  if (tg.K != H || tu.K != H || tg.N != tu.N || td.K != tg.N || td.N != H)
    return fail(c, ATSI_E_SHAPE, "decoder layer FFN shapes do not match hidden %lld", (long long)H);
  if ((st = enter(c))) return st;
  Scratch sc(c);
  __half* qb = q_out ? (__half*)q_out : sc.take((size_t)M * Hq);
  __half* kb = k_out ? (__half*)k_out : sc.take((size_t)M * Hkv);
  __half* oin = dbg && dbg->attn ? (__half*)dbg->attn : sc.take((size_t)M * Hq);
  __half* hf = dbg && dbg->act ? (__half*)dbg->act : sc.take((size_t)M * tg.N);
  float* y32 = !L->renorm_out ? nullptr : (dbg && dbg->sum32) ? dbg->sum32 : (float*)sc.take((size_t)M * H, 4);
  if (!qb || !kb || !oin || !hf || (L->renorm_out && !y32))
    return fail(c, ATSI_E_WORKSPACE, "scratch too small for a %lld-token layer", (long long)M);
  __half* hh = (__half*)h;
  const int Mi = (int)M;
  const float eps = L->eps;
  bool resident = true;
  for (atsi_tid t : ids) resident = resident && !c->tensors[t].on_host;
  if (c->fused_layer && Mi == 1 && resident && !L->renorm_out && !dbg) {
    // batch-1 decode with every weight in HBM: one fused launch
    LayerArgs la{};
    for (int i = 0; i < kLayerTensors; ++i) {
      const Tensor& t = c->tensors[ids[i]];
      la.w[i] = QView{t.dcodes, t.dscales, (int)t.K, (int)t.N};
    }
    la.h = hh;
    la.q_out = qb;
    la.k_out = kb;
    la.oin = oin;
    la.hf = hf;
    la.H = (int)H;
    la.Hq = (int)Hq;
    la.Hkv = (int)Hkv;
    la.I = (int)tg.N;
    la.head_dim = L->head_dim;
    la.expand = L->n_heads / L->n_kv_heads;
    la.eps = eps;
    la.bar = c->layer_bar;
    if (la.expand <= 64) {
      hipError_t e = launch_decode_layer(la, c->cs);
      if (e == hipSuccess) {
        c->layer_launched = true;
        return ATSI_OK;
      }
      if (e != hipErrorInvalidConfiguration) return hip_fail(c, e, "fused decode layer launch");
      (void)hipGetLastError();  // shape outside the fused kernel: four launches below
    }
  }
  if ((st = prefetch_call(c, ids, 7))) return st;
  if ((st = run_attention(c, ids, L->n_heads, L->n_kv_heads, L->head_dim, eps, hh, Mi, qb, kb, oin))) return st;
  if ((st = copy_h_attn(c, dbg, hh, Mi, H))) return st;
  // 3. f = silu(rms(h) Wg) * (rms(h) Wu)
  LinOp gu = plain_op(QView{nullptr, nullptr, (int)tg.K, (int)tg.N}, hh, Mi, hf);
  gu.swiglu = 1; gu.norm = 1; gu.eps = eps;
  if ((st = run_op(c, gu, &ids[4], 2))) return st;
  // 4. h = h + f Wd (in fp32 and renormalised when asked)
  LinOp dn = plain_op(QView{nullptr, nullptr, (int)td.K, (int)td.N}, hf, Mi, hh);
  dn.res = hh;
  dn.y32 = y32;
  if ((st = run_op(c, dn, &ids[6], 1))) return st;
  if (y32) {
    hipError_t e = launch_rmsnorm32(y32, Mi, (int)H, eps, hh, c->cs);
    if (e != hipSuccess) return hip_fail(c, e, "rmsnorm launch");
  }
  return ATSI_OK;
}

atsi_status atsi_moe_decoder_layer(atsi_ctx* c, const atsi_moe_layer* L, void* h, int64_t M, void* q_out,
                                   void* k_out, const atsi_moe_debug* dbg, const atsi_layer_debug* ldbg) {
  if (!c) return ATSI_E_INVALID;
  if (!L) return fail(c, ATSI_E_INVALID, "layer descriptor is NULL");
  atsi_status st;
  if ((st = check_act(c, h, "h")) || (st = check_m(c, M))) return st;
  if ((q_out && !aligned16(q_out)) || (k_out && !aligned16(k_out)))
    return fail(c, ATSI_E_INVALID, "q_out / k_out must be 16-byte aligned");
  if ((st = check_layer_debug(c, ldbg)) || (st = check_moe_debug(c, dbg))) return st;
  const atsi_tid ids[4] = {L->q, L->k, L->v, L->o};
  if ((st = check_attention(c, ids, L->n_heads, L->n_kv_heads, L->head_dim, L->eps)) || (st = check_moe(c, L->moe)))
    return st;
  const int64_t H = c->tensors[L->q].K, Hq = c->tensors[L->q].N, Hkv = c->tensors[L->k].N;
  if (L->moe->hidden != H) return fail(c, ATSI_E_SHAPE, "MoE hidden %lld != attention hidden %lld",
                                       (long long)L->moe->hidden, (long long)H);
  if ((st = enter(c))) return st;
  Scratch sc(c);
  __half* qb = q_out ? (__half*)q_out : sc.take((size_t)M * Hq);
  __half* kb = k_out ? (__half*)k_out : sc.take((size_t)M * Hkv);
  __half* oin = ldbg && ldbg->attn ? (__half*)ldbg->attn : sc.take((size_t)M * Hq);
  float* inv_r = (float*)sc.take(M, 4);
  if (!qb || !kb || !oin || !inv_r)
    return fail(c, ATSI_E_WORKSPACE, "scratch too small for a %lld-token layer", (long long)M);
  __half* hh = (__half*)h;
  const int Mi = (int)M;
  // expert copies wait for routing; the attention tensors can start now
  if ((st = prefetch_call(c, ids, 4))) return st;
  if ((st = run_attention(c, ids, L->n_heads, L->n_kv_heads, L->head_dim, L->eps, hh, Mi, qb, kb, oin))) return st;
  if ((st = copy_h_attn(c, ldbg, hh, Mi, H))) return st;
  // h = h + MoE(rms(h)): the norm is a per-token factor on the router logits
  // and the expert gate/up products (computed with the routing), the residual
  // is added by the combine
  return run_moe(c, L->moe, hh, Mi, hh, dbg, inv_r, true, L->eps, hh, sc);
}

atsi_status atsi_rmsnorm(atsi_ctx* c, const void* x, int64_t M, int64_t H, float eps, void* y) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, y, "y")) || (st = check_m(c, M))) return st;
  if (H < 8 || H % 8 != 0 || H > (1 << 20) || !(eps >= 0.f))
    return fail(c, ATSI_E_SHAPE, "hidden %lld must be a positive multiple of 8 (eps >= 0)", (long long)H);
  if ((st = enter(c))) return st;
  hipError_t e = launch_rmsnorm((const __half*)x, (int)M, (int)H, eps, (__half*)y, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "rmsnorm launch");
  return ATSI_OK;
}

atsi_status atsi_moe_bucket(atsi_ctx* c, const int32_t* idx, int64_t M, int32_t k, int32_t E, int32_t* counts,
                            int32_t* offsets, int32_t* perm, int32_t* inv_perm) {
  if (!c) return ATSI_E_INVALID;
  if (!idx || !counts || !offsets || !perm || !inv_perm) return fail(c, ATSI_E_INVALID, "NULL buffer");
  if (E < 1 || E > kMaxExperts || k < 1 || k > kMaxTopK || k > E || M < 1 || M > 65536)
    return fail(c, ATSI_E_SHAPE, "bucket: E=%d k=%d M=%lld out of range", E, k, (long long)M);
  atsi_status st = enter(c);
  if (st) return st;
  Scratch sc(c);
  int32_t* order = (int32_t*)sc.take(E, 4);
  int32_t* tiles = (int32_t*)sc.take(2 * ((size_t)M * k + E + 1), 4);
  int32_t* nt = (int32_t*)sc.take(1, 4);
  if (!order || !tiles || !nt) return fail(c, ATSI_E_WORKSPACE, "scratch too small for bucketing");
  hipError_t e = launch_bucket(idx, (int)M, k, E, nullptr, 1, 0, 0, counts, offsets, perm, inv_perm, order, tiles,
                               nt, nullptr, nullptr, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "bucket launch");
  return ATSI_OK;
}

atsi_status atsi_moe_ffn(atsi_ctx* c, const atsi_moe* m, const void* x, int64_t M, void* y,
                         const atsi_moe_debug* dbg) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st;
  if ((st = check_act(c, x, "x")) || (st = check_act(c, y, "y")) || (st = check_m(c, M)) || (st = check_moe(c, m)) ||
      (st = check_moe_debug(c, dbg)))
    return st;
  if (x == y) return fail(c, ATSI_E_INVALID, "y must not alias x");
  if ((st = enter(c))) return st;
  Scratch sc(c);
  return run_moe(c, m, (const __half*)x, (int)M, (__half*)y, dbg, nullptr, false, 0.f, nullptr, sc);
}

atsi_status atsi_set_schedule(atsi_ctx* c, const atsi_tid* order, int32_t n) {
  if (!c) return ATSI_E_INVALID;
  if (n < 0 || (n > 0 && !order)) return fail(c, ATSI_E_INVALID, "schedule of length %d with NULL order", n);
  for (int32_t i = 0; i < n; ++i) {
    atsi_status st = check_tid(c, order[i]);
    if (st) return st;
  }
  c->schedule.assign(order, order + n);
  c->sched_pos = 0;
  c->queue.clear();
  return ATSI_OK;
}

atsi_status atsi_prefetch(atsi_ctx* c, atsi_tid w) {
  if (!c) return ATSI_E_INVALID;
  atsi_status st = check_tid(c, w);
  if (st) return st;
  if ((st = enter(c))) return st;
  if (!c->tensors[w].streamed()) return ATSI_OK;
  c->queue.push_back(w);
  return topup(c);
}

atsi_status atsi_get_stats(atsi_ctx* c, atsi_stats* out, int32_t reset) {
  if (!c || !out) return fail(c, ATSI_E_INVALID, "ctx and out are required");
  *out = c->stats;
  if (reset) c->stats = atsi_stats{};
  return ATSI_OK;
}

atsi_status atsi_set_debug(atsi_ctx* c, uint32_t flags) {
  if (!c) return ATSI_E_INVALID;
  if (flags & ~(uint32_t)(ATSI_DEBUG_POISON | ATSI_DEBUG_SERIALIZE))
    return fail(c, ATSI_E_INVALID, "unknown debug flags 0x%x", flags);
  c->debug = flags;
  return ATSI_OK;
}

atsi_status atsi_set_moe_light_rows(atsi_ctx* c, int32_t rows) {
  if (!c) return ATSI_E_INVALID;
  if (rows < -1 || rows > kMoeLightRowsMax)
    return fail(c, ATSI_E_INVALID, "rows=%d out of range -1..%d", rows, kMoeLightRowsMax);
  atsi_status st = enter(c);
  if (st) return st;
  c->moe_light_rows = rows;
  return ATSI_OK;
}

atsi_status atsi_set_zero_copy(atsi_ctx* c, int32_t enable) {
  if (!c) return ATSI_E_INVALID;
  if (enable != 0 && enable != 1) return fail(c, ATSI_E_INVALID, "enable=%d is not 0 or 1", enable);
  if (enable)
    for (size_t i = 0; i < c->tensors.size(); ++i) {
      const Tensor& t = c->tensors[i];
      if (t.hcodes && !t.zcodes)
        return fail(c, ATSI_E_INVALID, "the host copy of tensor %zu is not mapped pinned memory", i);
    }
  atsi_status st = enter(c);
  if (st) return st;
  if (c->zero_copy != (enable != 0)) {
    c->zero_copy = enable != 0;
    ++c->placement_version;  // expert tables are rewritten with the new entries
  }
  return ATSI_OK;
}

atsi_status atsi_sync(atsi_ctx* c) {
  if (!c) return ATSI_E_INVALID;
  hipError_t e = hipSetDevice(c->device);
  if (e == hipSuccess) e = hipStreamSynchronize(c->ts);
  if (e == hipSuccess && c->ts2) e = hipStreamSynchronize(c->ts2);
  if (e == hipSuccess) e = hipStreamSynchronize(c->cs);
  if (e != hipSuccess) hip_fail(c, e, "stream synchronize");
  if (e == hipSuccess && c->layer_launched) {
    // a grid barrier of the fused decode layer that timed out leaves a flag
    unsigned flag = 0;
    e = hipMemcpy(&flag, c->layer_bar + kLayerBarrierErrWord, sizeof flag, hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
      hip_fail(c, e, "reading the fused-layer barrier flag");
    } else if (flag) {
      (void)hipMemset(c->layer_bar, 0, kLayerBarrierWords * sizeof(unsigned));
      hip_fail(c, hipErrorLaunchTimeOut, "fused decode layer: a grid barrier timed out");
    }
    c->layer_launched = false;
  }
  if (c->latched != ATSI_OK) {
    c->err = c->latched_msg;
    return c->latched;
  }
  return ATSI_OK;
}

atsi_status atsi_set_cpu_backend(atsi_ctx* c, atsi_cpu_pool* pool, void* staging, size_t staging_bytes) {
  if (!c) return ATSI_E_INVALID;
  if (pool && (!staging || ((uintptr_t)staging % kAlign) != 0 || staging_bytes < kAlign))
    return fail(c, ATSI_E_INVALID, "staging must be non-null pinned host memory, 256-byte aligned, >= 256 B");
  if (!pool)
    for (size_t i = 0; i < c->tensors.size(); ++i)
      if (c->tensors[i].on_cpu) return fail(c, ATSI_E_STATE, "tensor %zu is assigned to the CPU backend", i);
  atsi_status st = enter(c);
  if (st) return st;
  HIP_TRY(c, hipStreamSynchronize(c->cs));  // the old staging may still be read by a copy
  c->pool = pool ? &pool->pool : nullptr;
  c->staging = pool ? static_cast<char*>(staging) : nullptr;
  c->staging_bytes = pool ? staging_bytes : 0;
  c->staging_dev = nullptr;
  if (pool) {
    void* d = nullptr;
    if (hipHostGetDevicePointer(&d, staging, 0) == hipSuccess)
      c->staging_dev = static_cast<char*>(d);
    else
      (void)hipGetLastError();  // not mapped: activation transfers go through the DMA engines
  }
  return ATSI_OK;
}

atsi_status atsi_set_backends(atsi_ctx* c, const uint8_t* on_cpu, int32_t n) {
  if (!c) return ATSI_E_INVALID;
  if (!on_cpu) return fail(c, ATSI_E_INVALID, "on_cpu is NULL");
  if (n != (int32_t)c->tensors.size())
    return fail(c, ATSI_E_INVALID, "assignment length %d != %zu registered tensors", n, c->tensors.size());
  bool any = false;
  for (int32_t i = 0; i < n; ++i) {
    if (on_cpu[i] > 1) return fail(c, ATSI_E_INVALID, "on_cpu[%d]=%d is not 0 or 1", i, on_cpu[i]);
    if (on_cpu[i] && !c->tensors[i].on_host)
      return fail(c, ATSI_E_STATE, "tensor %d is placed in HBM; only host-placed tensors run on the CPU", i);
    any = any || on_cpu[i];
  }
  if (any && !c->pool) return fail(c, ATSI_E_STATE, "no CPU backend attached (atsi_set_cpu_backend)");
  atsi_status st = enter(c);
  if (st) return st;
  for (int32_t i = 0; i < n; ++i) c->tensors[i].on_cpu = on_cpu[i] != 0;
  // copies armed or queued for tensors now on the CPU would never be read:
  // free their slots once the copies have landed, and drop them from the queue
  for (Slot& sl : c->slots)
    if (sl.armed && !c->tensors[sl.tid].streamed()) {
      HIP_TRY(c, hipEventSynchronize(sl.ready));
      sl.armed = false;
    }
  c->queue.erase(std::remove_if(c->queue.begin(), c->queue.end(),
                                [&](atsi_tid t) { return !c->tensors[t].streamed(); }),
                 c->queue.end());
  return ATSI_OK;
}

atsi_status atsi_set_timing(atsi_ctx* c, int32_t enable) {
  if (!c) return ATSI_E_INVALID;
  if (enable != 0 && enable != 1) return fail(c, ATSI_E_INVALID, "enable=%d is not 0 or 1", enable);
  atsi_status st = enter(c);
  if (st) return st;
  if ((st = resolve_timing(c))) return st;
  if (enable && c->tev.empty()) {
    c->tev.resize(kTimingEvents, nullptr);
    for (hipEvent_t& e : c->tev) HIP_TRY(c, hipEventCreate(&e));
  }
  const double nan = std::numeric_limits<double>::quiet_NaN();
  if (enable && !c->timing) c->timings.assign(c->tensors.size(), atsi_tensor_timing{nan, nan, nan, nan, nan});
  c->timing = enable != 0;
  return ATSI_OK;
}

atsi_status atsi_get_timings(atsi_ctx* c, int32_t n, atsi_tensor_timing* out) {
  if (!c) return ATSI_E_INVALID;
  if (!out) return fail(c, ATSI_E_INVALID, "out is NULL");
  if (n != (int32_t)c->tensors.size())
    return fail(c, ATSI_E_INVALID, "output length %d != %zu registered tensors", n, c->tensors.size());
  atsi_status st = enter(c);
  if (st) return st;
  if ((st = resolve_timing(c))) return st;
  const double nan = std::numeric_limits<double>::quiet_NaN();
  c->timings.resize(c->tensors.size(), atsi_tensor_timing{nan, nan, nan, nan, nan});
  for (int32_t i = 0; i < n; ++i) out[i] = c->timings[i];
  return ATSI_OK;
}

atsi_status atsi_debug_read_probe(atsi_ctx* c, const void* dev, size_t bytes) {
  if (!c) return ATSI_E_INVALID;
  if (!dev || bytes == 0 || bytes % 16 || (uintptr_t)dev % 16 || bytes >= ((size_t)1 << 31))
    return fail(c, ATSI_E_INVALID,
                "the probe needs a 16-byte aligned device buffer of a positive multiple of 16 bytes below 2 GiB");
  atsi_status st = enter(c);
  if (st) return st;
  hipError_t e = launch_read_probe(dev, bytes, c->layer_bar + kProbeSinkWord, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "read probe launch");
  return ATSI_OK;
}

atsi_status atsi_debug_unpack(atsi_ctx* c, atsi_tid w, int8_t* q_out) {
  if (!c) return ATSI_E_INVALID;
  if (!q_out) return fail(c, ATSI_E_INVALID, "q_out is NULL");
  atsi_status st = check_tid(c, w);
  if (st) return st;
  if ((st = enter(c))) return st;
  QView v;
  std::vector<int> held;
  if ((st = acquire(c, w, &v, held))) return st;
  hipError_t e = launch_unpack(v, q_out, c->cs);
  if (e != hipSuccess) return hip_fail(c, e, "unpack launch");
  return release(c, held);
}

}  // extern "C"
