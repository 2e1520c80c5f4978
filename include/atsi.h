/*
 * atsi.h -- C ABI of the block-int4 quantised-linear hot path with host
 * streaming (tensor-granularity placement, ATSInfer, arxiv 2607.10183).
 *
 * The unit of placement is one weight tensor (Sec. 4.3.2: each tensor i has a
 * size s_i and a backend/placement b_i).  A tensor is read either from HBM
 * (the GPU resident region, Sec. 4.2.1) or from pinned host memory (CPU
 * pinned-memory storage, Sec. 4.2.1); a host tensor is copied into a GPU
 * temporary buffer ("slot") on a transfer stream and consumed on a compute
 * stream, with events ordering the two (Sec. 4.2.2).  By default every host
 * tensor is promoted for each use (the all-GPU runtime assignment of Sec.
 * 4.4.1) and the engine hides the copies behind compute; with a CPU backend
 * attached (atsi_set_cpu_backend), host tensors may instead run on the host
 * CPU (the hybrid execution of Sec. 4.3-4.4), as the runtime assignment of
 * atsi_schedule_transfers decides.
 *
 * Weight format (the paper uses INT4 weights without fixing a layout, Sec. 5.1):
 *   codes  uint8 [N][K/2]  -- row n = output feature n; byte j of a row holds
 *                             input 2j in its low nibble and 2j+1 in its high
 *                             nibble, each as u = q + 8 with q in [-8, 7];
 *   scales uint16[N][K/32] -- IEEE fp16 bit patterns, one per 32 inputs;
 *   weight w[n][k] = scale[n][k/32] * q[n][k].
 * Activations are fp16 row-major [M][K]; outputs fp16 row-major [M][N],
 * accumulated in fp32 and rounded to nearest-even once.  Dequantised weights
 * must be finite in fp16 (|scale| * 8 <= 65504).
 *
 * Ownership: the caller owns every buffer (weights in HBM, pinned host
 * weights, activations, the workspace, the pinned counts buffer) and every
 * stream; the library keeps borrowed pointers until atsi_destroy and itself
 * allocates only host bookkeeping and HIP events.  Device pointers must be
 * 16-byte aligned.
 *
 * Streams: calls only enqueue work on the compute stream (and copies on the
 * transfer stream); they return before the GPU finishes.  Inputs must stay
 * valid until atsi_sync returns.
 *
 * Errors: every call validates its arguments before any HIP call and returns
 * a status; atsi_last_error(ctx) gives a message.  Failures reported by the
 * HIP runtime are latched and returned by the next call and by atsi_sync.
 * No C++ exception crosses this boundary.  A context is not thread-safe.
 */
#ifndef ATSI_H
#define ATSI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATSI_OK = 0,
  ATSI_E_INVALID = 1,        /* null or malformed argument */
  ATSI_E_SHAPE = 2,          /* unsupported shape (K % 32, group != 32, M range) */
  ATSI_E_UNKNOWN_TENSOR = 3, /* tensor id not registered */
  ATSI_E_NO_COPY = 4,        /* placement points at a location with no copy */
  ATSI_E_WORKSPACE = 5,      /* workspace too small for slots or scratch */
  ATSI_E_HIP = 6,            /* HIP runtime error (also: no GPU present) */
  ATSI_E_STATE = 7           /* call not valid in the current state */
} atsi_status;

typedef struct atsi_ctx atsi_ctx;
typedef int32_t atsi_tid;

/* Create a context on `device`.
 * compute_stream, transfer_stream: distinct, non-null hipStream_t handles
 *   (the paper's compute stream and transfer stream, Sec. 4.2.2).
 * transfer_stream2: a second transfer stream (distinct from both), or NULL.
 *   With it, host-to-device copies alternate between the two transfer
 *   streams so that two copies are in flight at once; without it every copy
 *   goes on transfer_stream.
 * workspace: device buffer of workspace_bytes, carved into n_slots temporary
 *   buffers for streamed tensors (Sec. 4.2.1, GPU temporary buffers) and a
 *   scratch region for intermediate activations; 256-byte aligned.
 * host_counts: pinned host memory (hipHostMalloc'd) of at least 128 int32,
 *   where an MoE call with streamed experts reads back its per-expert token
 *   counts (expert transfers wait for routing, Sec. 4.2.2); or NULL, and then
 *   such calls fail with ATSI_E_STATE.
 * n_slots: number of temporary buffers, 2..64.
 * On a machine without a usable GPU this returns ATSI_E_HIP and *out = NULL. */
atsi_status atsi_create(int device, void* compute_stream, void* transfer_stream,
                        void* transfer_stream2, void* workspace, size_t workspace_bytes,
                        int32_t* host_counts, int n_slots, atsi_ctx** out);

/* Drain the context's streams and free what the context itself holds: its
 * slot and routing events (the events that order the compute and transfer
 * streams, Sec. 4.2.2) and host bookkeeping.  Nothing the caller passed in is
 * freed. */
atsi_status atsi_destroy(atsi_ctx* ctx);

/* Message of the last failure on ctx (or of the last failed atsi_create when
 * ctx is NULL).  Valid until the next call on the same context. */
const char* atsi_last_error(const atsi_ctx* ctx);

/* One block-int4 weight tensor: K inputs, N outputs, group must be 32 and
 * K % 32 == 0.  dev_* point at an HBM copy, host_* at a pinned host copy;
 * either pair may be NULL, not both.  The tensor starts HBM-resident when it
 * has an HBM copy, host-resident otherwise. */
typedef struct {
  int64_t K, N;
  int32_t group;
  const uint8_t* dev_codes;
  const uint16_t* dev_scales;
  const uint8_t* host_codes;
  const uint16_t* host_scales;
} atsi_qtensor;

/* Register a tensor (its size s_i and locations, Sec. 4.3.2); ids count from 0. */
atsi_status atsi_tensor_register(atsi_ctx* ctx, const atsi_qtensor* t, atsi_tid* out);

/* Set the placement of tensors 0..n-1 (Sec. 4.3.2, b_i): host_mask[i] = 1
 * reads tensor i from pinned host memory through a temporary buffer, 0 from
 * HBM.  n must equal the number of registered tensors.  Re-lays out the
 * temporary buffers (each sized for the largest host tensor); fails with
 * ATSI_E_WORKSPACE if n_slots of them do not fit.  Drains the streams. */
atsi_status atsi_set_placement(atsi_ctx* ctx, const uint8_t* host_mask, int32_t n);

/* y[M][N] = x[M][K] . W^T for tensor w (fp16 in and out, fp32 accumulation).
 * Decode sizes run kernels that read the codes once per launch: M = 1 a
 * dequantising GEMV, 2 <= M <= 16 a batched-decode kernel on the matrix cores
 * (for K not a multiple of 128, M <= 4 runs GEMV launches instead); larger M
 * runs a dequantise-into-LDS fp16 MFMA GEMM (prefill, Sec. 2.2 and the
 * chunked prefill of Sec. 5.1).  A
 * host-resident w is first copied into a temporary buffer on the transfer
 * stream (Sec. 4.2.2).  1 <= M <= 65536. */
atsi_status atsi_linear(atsi_ctx* ctx, atsi_tid w, const void* x_f16, int64_t M, void* y_f16);

/* Dense SwiGLU feed-forward block (the FFN of a decoder layer of the dense
 * models of Sec. 5.1; every one of its three weight tensors is a unit of
 * placement, Sec. 4.3.2):
 *   y = (silu(x Wg) * (x Wu)) Wd,  silu(z) = z / (1 + exp(-z)),
 * gate and up are H x I tensors, down is I x H.  gate and up run in one
 * launch with the SwiGLU product fused; the intermediate (fp16, M x I) lives
 * in the workspace's scratch region (ATSI_E_WORKSPACE if it does not fit).
 * y must not alias x. */
atsi_status atsi_ffn_swiglu(atsi_ctx* ctx, atsi_tid gate, atsi_tid up, atsi_tid down,
                            const void* x_f16, int64_t M, void* y_f16);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * SwiGLU feed-forward block as atsi_ffn_swiglu, but its M x I fp16
 * intermediate lives in a static device array of the library (16 MiB, one per
 * GPU, held until the process ends) instead of the workspace's scratch
 * region, and no call it makes allocates.  M * I * 2 must not exceed
 * 16 MiB (ATSI_E_WORKSPACE otherwise).  Large prefill chunks whose down
 * projection atsi_ffn_swiglu would split along K (fp32 partial sums in the
 * workspace) run it unsplit here.  Every call on one GPU, from any context,
 * uses that GPU's one array: calls that overlap in time on one GPU race.
 * Host-resident tensors still stream through the context's temporary
 * buffers.  Same arguments, layouts and errors as atsi_ffn_swiglu. */
atsi_status atsi_ffn_swiglu_noalloc(atsi_ctx* ctx, atsi_tid gate, atsi_tid up, atsi_tid down,
                                    const void* x_f16, int64_t M, void* y_f16);

/* RMS normalisation with unit gain (the normalisation between the layers of
 * the pre-norm models of Sec. 5.1; the paper places only weight tensors, so
 * this glue always runs on the GPU): y[t] = x[t] / sqrt(mean_k x[t][k]^2 + eps)
 * for fp16 x, y [M][H] (device, 16-byte aligned, H % 8 == 0), fp32
 * arithmetic and one fp16 rounding; y may alias x.  The glue between the
 * layers of a stack whose hidden state is renormalised after every layer. */
atsi_status atsi_rmsnorm(atsi_ctx* ctx, const void* x_f16, int64_t M, int64_t H, float eps, void* y_f16);

/* The gate/up half of a SwiGLU FFN as one launch:
 *   h[M][I] = silu(x Wg) * (x Wu)   (fp32 accumulation, one fp16 rounding),
 * gate and up H x I, x fp16 [M][H], h fp16 [M][I] (caller-owned device
 * memory, must not alias x).  The kernel atsi_ffn_swiglu and the decoder
 * layers run for their first half, exposed on its own so that it can be
 * checked and timed alone. */
atsi_status atsi_swiglu_gate_up(atsi_ctx* ctx, atsi_tid gate, atsi_tid up, const void* x_f16, int64_t M,
                                void* h_f16);

/* One pre-norm decoder layer whose projections are all quantised tensors. */
typedef struct {
  int32_t n_heads, n_kv_heads, head_dim; /* grouped-query heads; n_heads % n_kv_heads == 0 */
  float eps;                             /* RMS-norm epsilon (unit gain) */
  atsi_tid q, k, v, o, gate, up, down;   /* Q/K/V: H x heads*dim, O: heads*dim x H, FFN as above */
  int32_t renorm_out;                    /* 1: h_out = rms(h + attn + FFN) (see below), 0: plain */
} atsi_dense_layer;

/* Optional device buffers that receive a layer's intermediate activations
 * (each may be NULL; 16-byte aligned), so that every stage can be checked on
 * its own input:
 *   attn    fp16 [M][n_heads*head_dim]: attention output, the input of W_O;
 *   h_attn  fp16 [M][H]: residual stream after the attention block;
 *   act     fp16 [M][I]: SwiGLU activation, the input of W_down (dense layers);
 *   sum32   fp32 [M][H]: h_attn + FFN before the output renormalisation
 *           (dense layers with renorm_out = 1).
 * Buffers not given stay in the workspace's scratch region. */
typedef struct {
  void* attn;
  void* h_attn;
  void* act;
  float* sum32;
} atsi_layer_debug;

/* h <- h + attn(rms(h)) Wo;  h <- h + FFN(rms(h)), in place on h[M][H].
 * With layer->renorm_out = 1 the layer's output is renormalised as well,
 * h <- rms(h + FFN(rms(h))), for stacks whose hidden state is renormalised
 * between layers: the residual sum is kept in fp32 (the FFN output of a
 * layer alone can approach the fp16 range) and only the normalised state is
 * rounded to fp16 (one more launch).
 * Attention is evaluated at context length 1 (each token attends only to
 * itself, so query head i outputs the value of KV head i / (n_heads /
 * n_kv_heads)); the Q and K projections are still computed and written to
 * q_out[M][n_heads*dim] and k_out[M][n_kv_heads*dim] when those are non-NULL
 * (device buffers), else to scratch.  rms(v) = v / sqrt(mean(v^2) + eps).
 * Four launches: fused RMS-norm + Q/K/V, O + residual, fused RMS-norm +
 * gate/up + SwiGLU, down + residual.  Streamed tensors of the layer are
 * queued for copy at entry so their transfers overlap earlier launches.
 * A context created with the environment variable ATSI_FUSED_DECODE_LAYER=1
 * runs a batch-1 layer whose tensors are all HBM-resident, of the 8B shape
 * (hidden 4096, 32 x 128 query and 8 x 128 KV heads, SwiGLU 14336), on a
 * 256-CU device, as one persistent launch with grid barriers instead (the
 * same bits; slower than the four launches on MI355X), unless dbg is given.
 * A barrier of that launch that does not complete is reported by atsi_sync.
 * dbg may be NULL. */
atsi_status atsi_decoder_layer(atsi_ctx* ctx, const atsi_dense_layer* layer, void* h_f16, int64_t M,
                               void* q_out_f16, void* k_out_f16, const atsi_layer_debug* dbg);

/* Execution order of tensors, repeated cyclically (the execution plan of a
 * round, Sec. 4.2.2): the engine copies upcoming host-resident tensors into
 * free temporary buffers as soon as one frees up, up to n_slots - 1 ahead, so
 * weight transfers start as early as dependencies allow.  n = 0 clears it. */
atsi_status atsi_set_schedule(atsi_ctx* ctx, const atsi_tid* order, int32_t n);

/* Queue an early copy of a host-resident tensor (no-op for HBM tensors). */
atsi_status atsi_prefetch(atsi_ctx* ctx, atsi_tid w);

/* A routed mixture-of-experts layer of SwiGLU experts. */
typedef struct {
  int32_t n_experts;          /* E, a multiple of 16, at most 128 */
  int32_t top_k;              /* experts per token, 1..16, <= E */
  int64_t hidden, inter;      /* H and I, multiples of 32 */
  const void* router_w_f16;   /* device fp16 [H][E] (not quantised) */
  const float* router_bias;   /* device fp32 [E], or NULL */
  const atsi_tid* gate;       /* host arrays of E tensor ids: gate/up are H x I, */
  const atsi_tid* up;         /*   down is I x H */
  const atsi_tid* down;
} atsi_moe;

/* Optional device buffers that receive the routing and the expert
 * activations (each may be NULL): logits fp32 [M][E]; idx int32 [M][k] and p
 * fp32 [M][k] (slot j in order of logit descending, expert id ascending);
 * counts int32 [E]; offsets int32 [E+1] (exclusive prefix sum of counts);
 * perm int32 [M*k] (pair ids k*t + j ordered by expert, then token); inv_perm
 * int32 [M*k] (inverse of perm); expert_h fp16 [M*k][I] (SwiGLU activation of
 * pair k*t + j, the input of its expert's W_down) and expert_out fp16
 * [M*k][H] (that expert's output, the term of the combine), both 16-byte
 * aligned, rows in pair order. */
typedef struct {
  float* logits;
  int32_t* idx;
  float* p;
  int32_t* counts;
  int32_t* offsets;
  int32_t* perm;
  int32_t* inv_perm;
  void* expert_h;
  void* expert_out;
} atsi_moe_debug;

/* y[t] = sum_j p[t][j] * FFN_{idx[t][j]}(x[t]) for x, y fp16 [M][H].
 * Router logits l = x W_r + b are accumulated in fp32; each token keeps the
 * top_k experts by (logit descending, expert id ascending) and p is the
 * softmax over the kept logits (the full softmax renormalised over them).
 * Pairs are bucketed by expert; each expert FFN runs on its own tokens only
 * and only routed experts are read.  An expert with any host-resident tensor
 * is streamed after routing resolves (Sec. 4.2.2: expert transfers wait for
 * routing and move only selected experts): the host reads the per-expert
 * counts back (one event wait), copies the active host experts heaviest
 * first into temporary buffers (n_slots >= 3 needed, and the host_counts
 * buffer of atsi_create) while the HBM-resident experts already run.  Expert
 * outputs are kept in fp16 before the fp32 combine.  1 <= M <= 65536.  dbg
 * may be NULL. */
atsi_status atsi_moe_ffn(atsi_ctx* ctx, const atsi_moe* moe, const void* x_f16, int64_t M, void* y_f16,
                         const atsi_moe_debug* dbg);

/* One pre-norm decoder layer whose FFN is the routed MoE above (the layers
 * of the MoE models of Sec. 5, e.g. a 235B-A22B stack):
 *   q, k, v = rms(h) Wq, Wk, Wv;  h += attn Wo   (as atsi_decoder_layer)
 *   h += MoE(rms(h))                              (as atsi_moe_ffn)
 * with rms(v) = v / sqrt(mean(v^2) + eps).  The norm is not materialised:
 * its per-token factor scales the router logits (before the bias) and the
 * expert gate/up products in fp32, and the combine adds the residual, so h
 * (fp16 [M][hidden], device) is updated in place.  q_out / k_out as in
 * atsi_decoder_layer; dbg as in atsi_moe_ffn; ldbg (attn and h_attn; act and
 * sum32 are not used) as in atsi_decoder_layer.  moe->hidden must equal the
 * attention hidden size. */
typedef struct {
  int32_t n_heads, n_kv_heads, head_dim;
  float eps;
  atsi_tid q, k, v, o;
  const atsi_moe* moe;
} atsi_moe_layer;

atsi_status atsi_moe_decoder_layer(atsi_ctx* ctx, const atsi_moe_layer* layer, void* h_f16, int64_t M,
                                   void* q_out_f16, void* k_out_f16, const atsi_moe_debug* dbg,
                                   const atsi_layer_debug* ldbg);

/* Token-to-expert bucketing alone (the same kernel atsi_moe_ffn uses), from
 * device idx int32 [M][k] with ids in [0, n_experts): counts [E], offsets
 * [E+1], perm [M*k], inv_perm [M*k] as in atsi_moe_debug.  Out-of-range ids
 * are skipped (memory-safe, results then unspecified). */
atsi_status atsi_moe_bucket(atsi_ctx* ctx, const int32_t* idx, int64_t M, int32_t k, int32_t n_experts,
                            int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv_perm);

/* Checking modes of the streaming engine (flags may be combined; 0 = off):
 *   ATSI_DEBUG_POISON     every temporary slot is filled with 0xFF bytes
 *                         (codes q = 7, scales fp16 NaN) on the transfer
 *                         stream right before its copy, so a launch that read
 *                         a slot before the copy landed would produce NaN;
 *   ATSI_DEBUG_SERIALIZE  no overlap: each copy waits for every launch already
 *                         enqueued on the compute stream and completes before
 *                         the call goes on (host synchronisation).
 * Outputs must not change with either flag (the engine's ordering is then
 * checked by comparing outputs).  ATSI_E_INVALID for unknown bits. */
#define ATSI_DEBUG_POISON 1u
#define ATSI_DEBUG_SERIALIZE 2u
atsi_status atsi_set_debug(atsi_ctx* ctx, uint32_t flags);

/* Zero-copy expert reads (the paper's copy-kernel path: with host memory
 * mapped and pinned, GPU threads read it directly; background section and
 * Sec. 4.2).  enable = 1: in atsi_moe_ffn and atsi_moe_decoder_layer calls of
 * at most 4 tokens, the expert kernels read the routed host-resident experts
 * in place from their pinned host copies over PCIe, through the same launches
 * as HBM-resident experts: no copy into a temporary slot and no wait on the
 * host for the routing counts.  Larger calls, and every other tensor, keep
 * the copy path.  Outputs are bit-identical to the copy path's.  Requires
 * every registered host copy, and every one registered while enabled, to be
 * mapped pinned host memory (e.g. hipHostMalloc'd): ATSI_E_INVALID names the
 * first that is not.  enable = 0 restores the copy path.  Reads done in place
 * are not counted in atsi_stats. */
atsi_status atsi_set_zero_copy(atsi_ctx* ctx, int32_t enable);

/* Kernel choice for the routed experts of a prefill call (more than 4 tokens;
 * the expert GEMMs of Sec. 2.2's compute-bound phase, only for routed
 * experts, Sec. 3.2). An expert routed at most `rows` pairs in the call runs
 * on the light-expert kernels: tiles that stream each weight through
 * registers once per tile, of 16 rows, or, in calls that route more than 16
 * pairs per expert on average, of 16, 32 or 64 rows (the fewest 16-row blocks
 * that cover its count; at most 32 rows for hidden or intermediate sizes
 * above 2048). 16-row tiles sum each group's exact products and
 * scale them in fp32 (the decode arithmetic); taller tiles round each weight
 * to fp16 once, as the grouped GEMM does. The other experts run on the
 * grouped GEMM (tiles of 64 rows staged through LDS). rows = 0 sends every
 * expert to the grouped GEMM; rows = -1 (the default) every expert to the
 * light kernels, except in calls of more than 16 pairs per expert on shapes
 * that allow only 16-row tiles, which keep the grouped GEMM. The light
 * kernels cover hidden and intermediate sizes that are multiples of 256 up to
 * 4096 (above 2048 only where 16-group slices divide the size evenly); other
 * shapes always take the grouped GEMM. The
 * choice depends only on the call's size and routed counts, so HBM-resident
 * and streamed experts give the same bits; the kernels differ by rounding
 * only.
 * ATSI_E_INVALID for rows < -1 or rows > 2^20. */
atsi_status atsi_set_moe_light_rows(atsi_ctx* ctx, int32_t rows);

/* Wait for the compute and transfer streams (the host-side synchronisation
 * with both streams of Sec. 4.2.2); returns the first latched asynchronous
 * error. */
atsi_status atsi_sync(atsi_ctx* ctx);

/* Transfer counters of the engine (Sec. 4.2.2 moves host tensors into GPU
 * temporary buffers; these count what it moved), cumulative since atsi_create
 * or the last reset.  Counted when the copies are enqueued. */
typedef struct {
  uint64_t h2d_bytes;    /* bytes copied from pinned host memory to the device */
  uint64_t h2d_copies;   /* hipMemcpyAsync calls that moved them */
  uint64_t h2d_tensors;  /* host tensors copied (an expert moved as one copy counts 3) */
  uint64_t host_reads;   /* launches' reads of a host tensor, each served by a copy */
  uint64_t host_read_bytes; /* bytes of those tensors: counted when the reading launch is enqueued, so a
                               copy counts once its consumer is in the stream, never for prefetches alone */
} atsi_stats;

/* *out = the counters; reset != 0 then zeroes them. */
atsi_status atsi_get_stats(atsi_ctx* ctx, atsi_stats* out, int32_t reset);

/* ---- Static tensor placement (Sec. 4.3 problem formulation; Alg. 1) ----
 * Chooses which tensors stay resident in GPU memory.  Host computation only:
 * no GPU call and no context.  Tensor i is the i-th in execution order:
 *   size_bytes[i]  its size (finite, >= 0);
 *   r[i]           latency saved by keeping it on the GPU (t^c - t^g), finite;
 *   c[i]           cost of a backend switch between tensors i-1 and i (c[0] unused), finite;
 *   is_expert      nullable; 1 marks an MoE expert tensor (an operator's experts as one tensor).
 * The result maximises sum_i r[i] [GPU] - sum_{i>=1} c[i] [b_i != b_{i-1}] with
 * the GPU-resident sizes, rounded up to whole granules, within budget_bytes
 * rounded down to whole granules (granularity_bytes > 0; the paper uses MB).
 * With is_expert, Alg. 1's branch applies first: a budget that covers every
 * non-expert tensor puts them all on the GPU and experts are chosen within
 * what remains; otherwise every expert stays on the CPU and the non-expert
 * tensors are chosen within the budget.  Fixed tensors keep their backend
 * while the choice optimises the whole objective, switches included.
 * Outputs: on_gpu_out[n] (caller-owned) = 1 for GPU-resident, 0 otherwise
 * (atsi_set_placement takes the opposite mask: 1 = host); objective_out
 * (nullable) = the objective of that placement from the unrounded inputs.
 * Equal-objective ties go to the placement whose backtrack prefers the CPU
 * predecessor and the fewest units, so results are deterministic.
 * Errors (message from atsi_last_error(NULL)): ATSI_E_INVALID for NULL
 * arrays, non-finite values, a negative size or budget, a non-positive
 * granularity; ATSI_E_SHAPE for n < 1, or when n times the budget units
 * exceeds 2^31 (use a coarser granularity).  Memory: n * units / 4 bytes. */
typedef struct {
  int32_t n;
  const double* size_bytes;
  const double* r;
  const double* c;
  const uint8_t* is_expert;
  double budget_bytes;
  double granularity_bytes;
} atsi_placement_problem;

atsi_status atsi_solve_placement(const atsi_placement_problem* problem, uint8_t* on_gpu_out, double* objective_out);

/* ---- Hybrid CPU-GPU execution: dynamic transfer scheduling (Sec. 4.4) ----
 *
 * A round runs tensors 0..n-1 in execution order.  Tensor i has a default
 * placement b_i (on_gpu[i] = 1: GPU-resident; 0: CPU, i.e. host-placed),
 * GPU and CPU execution times t_gpu[i], t_cpu[i], the activation-transfer
 * (backend switch) cost c[i] at the boundary between tensors i-1 and i
 * (c[0] unused) and the weight-transfer time w[i] (Sec. 4.4.1; for MoE
 * experts in decode, the copy time of the activated experts).  Times are in
 * any one unit (seconds in this library's measurements), finite and >= 0. */
typedef struct {
  int32_t n;
  const uint8_t* on_gpu;
  const double* t_gpu;
  const double* t_cpu;
  const double* c;
  const double* w;
} atsi_transfer_problem;

/* Alg. 2 (Sec. 4.4.2): the runtime backend assignment rb minimising the
 * round latency
 *   T(rb) = sum_i t_i^{rb_i} + sum_{i>=1} c_i [rb_{i-1} != rb_i] + sum_{promoted i} delta_i,
 *   delta_i = max(w_i - seg(j, i), 0),
 * where a promoted tensor (b_i = CPU, rb_i = GPU) has its weights copied from
 * the CPU-side endpoint j: the round start, or the first CPU-run tensor after
 * the previous promotion; seg(j, i) is the default-path time strictly between
 * j and i (execution times on the default backends plus the switches among
 * them).  Two promoted tensors need a CPU-run tensor between them.  GPU-placed
 * tensors always run on the GPU.  Host computation only, no context: O(n^2)
 * time, O(n) memory.
 * Outputs: rb_out[n] (caller-owned) = 1 where tensor i runs on the GPU;
 * latency_out (nullable) = T(rb).  Ties go to the CPU (fewer promotions) and
 * to the earliest endpoint, so results are deterministic.
 * Errors (message from atsi_last_error(NULL)): ATSI_E_INVALID for NULL
 * arrays, on_gpu values other than 0/1, negative or non-finite times;
 * ATSI_E_SHAPE for n outside 1..65536. */
atsi_status atsi_schedule_transfers(const atsi_transfer_problem* problem, uint8_t* rb_out, double* latency_out);

/* T(rb) of Sec. 4.4.1 for a given assignment rb (1 = GPU), under the
 * endpoint reading of atsi_schedule_transfers; *latency_out = +infinity for
 * an assignment that reading cannot reach (two promotions with no CPU-run
 * tensor between).  Errors: those of atsi_schedule_transfers, ATSI_E_INVALID
 * for rb values other than 0/1 or a GPU-placed tensor assigned to the CPU. */
atsi_status atsi_transfer_latency(const atsi_transfer_problem* problem, const uint8_t* rb, double* latency_out);

/* Alg. 3 (Sec. 4.4.3): load-aware re-scheduling.  A rescheduler keeps the
 * measurement snapshot and time of the last scheduling and the assignment it
 * produced.  Each step compares the current snapshot with the kept one: the
 * deviation d is the largest relative change of a measured series' total,
 * max over (t_gpu, t_cpu, c, w) of |sum cur - sum prev| / sum prev (infinite
 * when a series grows from zero; the paper leaves the measure open).  It
 * re-runs atsi_schedule_transfers on the current snapshot when there is no
 * kept snapshot, when the default placement changed, or when d >= eps and
 * now_s - (time of the last scheduling) >= tau_tpot * tpot_s (the paper:
 * eps = 0.15, tau = 5 x the recent TPOT); otherwise it returns the kept
 * assignment.  Applying the assignment (BuildRuntime) is the caller's
 * atsi_set_backends.  Host computation only.
 * create: n tensors per round (1..65536), eps >= 0, tau_tpot >= 0, finite.
 * step: rb_out[n] (caller-owned) = the assignment in force (1 = GPU);
 *   rescheduled_out and deviation_out (nullable) report the decision and d.
 *   Errors: ATSI_E_SHAPE when cur->n differs from the rescheduler's n, and
 *   the errors of atsi_schedule_transfers; the kept state is then unchanged. */
typedef struct atsi_rescheduler atsi_rescheduler;
atsi_status atsi_rescheduler_create(int32_t n, double eps, double tau_tpot, atsi_rescheduler** out);
atsi_status atsi_rescheduler_step(atsi_rescheduler* r, const atsi_transfer_problem* cur, double now_s, double tpot_s,
                                  uint8_t* rb_out, int32_t* rescheduled_out, double* deviation_out);
atsi_status atsi_rescheduler_destroy(atsi_rescheduler* r);

/* The host-CPU backend (the CPU side of the hybrid, Sec. 4.3-4.4): a pool of
 * worker threads (the calling thread takes part as one of them).  A pool
 * runs one product at a time; it may serve several contexts and must outlive
 * every context it is attached to (destroy it after atsi_destroy, or after
 * atsi_set_cpu_backend(ctx, NULL, ...)).  Idle workers spin briefly, then
 * yield, then sleep. */
typedef struct atsi_cpu_pool atsi_cpu_pool;
atsi_status atsi_cpu_pool_create(int32_t threads, atsi_cpu_pool** out);
atsi_status atsi_cpu_pool_destroy(atsi_cpu_pool* pool);

/* y[M][N] = x[M][K] . W^T on the host CPU, all pointers host memory: codes
 * and scales in the layout of this header, x and y fp16 bit patterns
 * (row-major, y must not alias x), fp32 sums, one round-to-nearest-even to
 * fp16.  1 <= M <= 65536, K % 32 == 0.  Errors: ATSI_E_INVALID for NULL
 * pointers, ATSI_E_SHAPE for sizes outside the limits; the message comes
 * from atsi_last_error(NULL).  No GPU is needed. */
atsi_status atsi_cpu_linear(atsi_cpu_pool* pool, const uint8_t* codes, const uint16_t* scales, int64_t N,
                            int64_t K, const uint16_t* x_f16, int64_t M, uint16_t* y_f16);

/* Attach the CPU backend to a context: the pool runs CPU-assigned tensors
 * and staging (pinned host memory, hipHostMalloc'd, 256-byte aligned,
 * staging_bytes long) carries their activations: a CPU-run launch copies its
 * input rows (and residual) to staging on the compute stream, waits for
 * them, computes on the pool and copies its outputs back on the compute
 * stream, so the calling thread blocks for the CPU part (the backend switches
 * are the activation transfers c_i of Sec. 4.4.1).  When staging is mapped
 * pinned memory these copies are done by a small kernel (the paper's copy
 * kernel), so they never queue behind weight copies on the DMA engines;
 * otherwise by hipMemcpy2DAsync.  It needs M*K*2 bytes for
 * the input, M*N*2 per output (4 for an fp32 one, twice for a SwiGLU pair)
 * and M*N*2 for a residual, each rounded up to 256 (ATSI_E_WORKSPACE if
 * staging is too small).  The library uses staging until atsi_destroy or the
 * next atsi_set_cpu_backend, which drains the compute stream first.  pool =
 * NULL detaches the backend (ATSI_E_STATE while a tensor is assigned to the
 * CPU). */
atsi_status atsi_set_cpu_backend(atsi_ctx* ctx, atsi_cpu_pool* pool, void* staging, size_t staging_bytes);

/* Runtime backend assignment (BuildRuntime of Alg. 3): on_cpu[i] = 1 runs
 * tensor i on the CPU backend from its pinned host copy, 0 on the GPU (a
 * host-placed tensor is then promoted: copied through a temporary buffer).
 * n must equal the number of registered tensors; only host-placed tensors
 * may run on the CPU (ATSI_E_STATE otherwise, or without a CPU backend).
 * Within one fused launch the gate and up tensors of a SwiGLU pair must share
 * a backend; the q, k and v projections may differ (the GPU and CPU parts of
 * the launch overlap).  MoE expert tensors run on the GPU only.
 * atsi_set_placement resets every tensor it places in HBM to the GPU. */
atsi_status atsi_set_backends(atsi_ctx* ctx, const uint8_t* on_cpu, int32_t n);

/* Per-tensor measurements for the snapshots of Alg. 3 (Sec. 4.4.3).  With
 * timing on, the context records HIP events around each GPU launch, weight
 * copy and activation transfer, and host clock time around each CPU product.
 * atsi_get_timings drains the streams and reports, per tensor, the latest
 * value since timing was enabled (NaN where none): a fused launch's time is
 * shared among its tensors by their byte sizes. */
typedef struct {
  double t_gpu;  /* GPU execution (s) */
  double t_cpu;  /* CPU execution (s) */
  double d2h;    /* activation transfer into a CPU run of the tensor (s) */
  double h2d;    /* activation transfer out of it (s) */
  double w;      /* weight copy into a temporary buffer (s) */
} atsi_tensor_timing;
atsi_status atsi_set_timing(atsi_ctx* ctx, int32_t enable);
atsi_status atsi_get_timings(atsi_ctx* ctx, int32_t n, atsi_tensor_timing* out);

/* Test export: the CPU backend's fp16 conversions, out[i] = the fp16 bit
 * pattern of in[i] rounded to nearest even, back[i] = that fp16 as fp32
 * (either output nullable).  No GPU is needed. */
atsi_status atsi_debug_cpu_f16(const float* in, int64_t n, uint16_t* out, float* back);

/* Test export: the signed codes q[N][K] (int8, device buffer) of tensor w as
 * the library reads them, from wherever w currently lives. */
atsi_status atsi_debug_unpack(atsi_ctx* ctx, atsi_tid w, int8_t* q_out);

/* Measurement export: one read-only pass over `bytes` of device memory at
 * dev (16-byte aligned, a positive multiple of 16, below 2 GiB), enqueued on
 * the compute stream: non-temporal 16-byte buffer loads, four per thread in
 * flight, workgroups reading contiguous 16 KiB rounds, eight workgroups per
 * CU.  The read ceiling the batch-1 GEMV is compared to (HBM streaming, Sec.
 * 2.2's memory-bound decode); the data is not changed and nothing the caller
 * sees is written.  ATSI_E_INVALID for a bad buffer. */
atsi_status atsi_debug_read_probe(atsi_ctx* ctx, const void* dev, size_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* ATSI_H */
