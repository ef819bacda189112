/*
 * dcp.h -- C ABI of the Data-Centric Parallel (DCP) hot path on one MI355X.
 *
 * Four operations, named after the quantities of the paper's problem
 * statement (Sec. 3.2: n batches with variable sequence lengths s_i, one
 * configuration chosen per batch):
 *
 *   dcp_varlen_attn_fwd  exact softmax attention over packed variable-length
 *                        sequences (block diagonal), returning O and the
 *                        natural-log row log-sum-exp;
 *   dcp_varlen_attn_bwd  its gradients dQ, dK, dV for an upstream dO;
 *   dcp_profile_cost     measured per-length attention cost rows (the
 *                        profiling step of Sec. 3.5);
 *   dcp_plan             per-batch sequence-parallel size, micro-batch,
 *                        gradient accumulation and recomputed layers
 *                        (DCP-intra, Sec. 3.4 / Algorithm 1; DCP-inter,
 *                        Sec. 3.3 / Eq. (3) / Appendix C).
 *
 * Conventions shared by every call
 * --------------------------------
 * - Status: every call returns 0 (DCP_OK) or a negative dcp_status and never
 *   throws across the ABI.  dcp_last_error() returns a thread-local message
 *   for the last failing call on the calling thread.
 * - Ownership: the caller owns every buffer.  The library never allocates
 *   device memory: scratch space comes from a caller-provided workspace whose
 *   size is queried first.  Host arrays are read only during the call.
 *   dcp_varlen_attn_fwd and dcp_varlen_attn_bwd stage the work lists they
 *   build in library-owned pinned host memory (per device, four buffers of
 *   at least 1 MiB, grown by powers of two and kept until the process ends;
 *   a buffer is reused only after the event behind its last copy, so a host
 *   more than four calls ahead of the stream waits there).
 * - Streams: `stream` is a hipStream_t passed as void* (NULL = the null
 *   stream).  Attention calls enqueue work and return without synchronising;
 *   argument errors are detected on the host before anything is enqueued;
 *   a launch failure is reported as DCP_ERR_HIP, while execution faults
 *   surface at the caller's next synchronisation.  dcp_profile_cost
 *   synchronises.  dcp_plan touches no device.
 * - Layout: Q, K, V, O, dO, dQ, dK, dV are bf16 [T, H, D] row-major (token
 *   stride H*D, head stride D, D contiguous), device memory, 16-byte aligned.
 *   LSE is fp32 [H, T].  Rows beyond cu_seqlens[n_seqs] are neither read
 *   for any output nor written.
 */
#ifndef DCP_H
#define DCP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DCP_OK = 0,
  DCP_ERR_INVALID = -1,     /* bad argument (null, inconsistent sizes, overflow) */
  DCP_ERR_UNSUPPORTED = -2, /* valid but not implemented (e.g. head_dim) */
  DCP_ERR_HIP = -3,         /* HIP runtime error, or no usable gfx950 device */
  DCP_ERR_WORKSPACE = -4,   /* workspace null or smaller than queried */
  DCP_ERR_INFEASIBLE = -5,  /* planner: no configuration fits the memory budget */
  DCP_ERR_TABLE = -6        /* planner: bad cost table or length beyond it */
} dcp_status;

/* Message for the last failing call on this thread ("" if none). */
const char* dcp_last_error(void);

/* Library version string. */
const char* dcp_version(void);

/* ------------------------------------------------------------------------ */
/* Packed variable-length attention                                          */
/* ------------------------------------------------------------------------ */

/*
 * Describes one packed batch.  Sequence b owns token rows
 * cu_seqlens_host[b] .. cu_seqlens_host[b+1]-1 and attends only to itself
 * (the "packed parallel" layout of Sec. 1; attention itself is exact softmax
 * attention, Sec. 4.1).
 *   n_seqs          >= 1; empty sequences (equal neighbours) are allowed.
 *   cu_seqlens_host host int32 [n_seqs+1]: cu[0] = 0, non-decreasing,
 *                   cu[n_seqs] <= total_tokens.
 *   total_tokens    T, rows allocated in every [T, H, D] tensor, < 2^31.
 *   n_heads         H in [1, 65535] (all heads share cu_seqlens).
 *   head_dim        D in {64, 72, 128}; anything else is DCP_ERR_UNSUPPORTED.
 *   scale           softmax scale applied to Q K^T, finite and > 0
 *                   (1/sqrt(D) in the usual models).
 *   causal          0: every query sees its whole sequence;
 *                   1: query i sees keys j <= i of its sequence.
 */
typedef struct {
  int32_t n_seqs;
  const int32_t* cu_seqlens_host;
  int64_t total_tokens;
  int32_t n_heads;
  int32_t head_dim;
  float scale;
  int32_t causal;
} dcp_attn_desc;

/* Workspace bytes needed by dcp_varlen_attn_fwd / _bwd for this batch. */
int dcp_varlen_attn_fwd_workspace_size(const dcp_attn_desc* desc, size_t* bytes);
int dcp_varlen_attn_bwd_workspace_size(const dcp_attn_desc* desc, size_t* bytes);

/*
 * Forward: for each sequence and head, O = softmax(scale * Q K^T) V and
 * LSE = ln sum_j exp(scale * q_i . k_j) (fp32, natural log), computed with
 * bf16 matrix-core products, fp32 accumulation and an fp32 online softmax.
 *   q, k, v    bf16 [T, H, D] inputs.
 *   o          bf16 [T, H, D] output (rows of sequences only).
 *   lse        fp32 [H, T] output (rows of sequences only).
 *   workspace  device scratch of at least the queried size.
 */
int dcp_varlen_attn_fwd(const dcp_attn_desc* desc, const void* q, const void* k, const void* v,
                        void* o, float* lse, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward of the forward above for the loss <dO, O>:
 *   dV = P^T dO,  dS = P o (dO V^T - rowsum(dO o O)),
 *   dQ = scale dS K,  dK = scale dS^T Q,  with P = exp(scale Q K^T - LSE).
 *   dout, o, lse  the upstream gradient and the forward's O and LSE.
 *   q, k, v       the forward's inputs.
 *   dq, dk, dv    bf16 [T, H, D] outputs (rows of sequences only).
 *   workspace     device scratch of at least the queried size; it holds the
 *                 work lists, -rowsum(dO o O) and LSE * log2(e) (fp32 [H, T]
 *                 each).  There is no dQ accumulator: dQ is formed by
 *                 query-stationary workgroups (or, for packed windows at head
 *                 widths up to 96, by the window's dK/dV workgroup), so every
 *                 gradient is written once and is bitwise reproducible.
 * The call uses the same desc (scale, causal) as the forward.
 */
int dcp_varlen_attn_bwd(const dcp_attn_desc* desc, const void* dout, const void* o, const float* lse,
                        const void* q, const void* k, const void* v, void* dq, void* dk, void* dv,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * Forward for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * dcp_varlen_attn_fwd without a workspace argument.  Its scratch -- the
 * constant chunks, the tile list and the window masks -- lives in a fixed
 * device array of the library, 8 MiB (8,388,608 bytes) per GPU, held until
 * the process ends; the call allocates no device or pinned memory (no
 * hipMalloc, hipHostMalloc or other allocating HIP or library routine): the
 * tile list is built in ordinary host memory and copied from there, which
 * the runtime stages before the call returns.  The caller still passes q,
 * k, v, o and lse.
 *   Errors: as dcp_varlen_attn_fwd, plus DCP_ERR_WORKSPACE when the batch's
 *   list needs more than 8 MiB (about 520,000 tiles of 256 query rows:
 *   tiles x heads), reported on the host before anything is enqueued.
 *   Sharing: every call on one GPU uses that GPU's single array, and each
 *   call rewrites it (enqueued on `stream`), so calls whose work may overlap
 *   in time -- on different streams, or from different threads without
 *   ordering -- race; order them on one stream or by synchronisation.
 * Outputs equal dcp_varlen_attn_fwd's bit for bit (same kernels, same list).
 */
int dcp_varlen_attn_fwd_noalloc(const dcp_attn_desc* desc, const void* q, const void* k, const void* v, void* o,
                                float* lse, void* stream);

/*
 * Prepared batches.  A training step runs the forward and the backward of
 * the same packed batch, and a profiler or benchmark runs them many times:
 * the tile lists of the three kernel passes (forward, dK/dV, dQ) depend only
 * on cu_seqlens, so they are built once on the host (dcp_batch_create) and
 * copied once into a caller-owned device buffer (dcp_batch_upload); every
 * later dcp_batch_fwd / dcp_batch_bwd on that buffer only launches kernels
 * (no host list building, no host-to-device copy).  Results equal those of
 * dcp_varlen_attn_fwd / _bwd bit for bit (same kernels, same lists).
 *
 *   dcp_batch_create   host only: validates `desc` (as the calls above do),
 *                      copies it and its cu_seqlens, builds the three lists.
 *                      *out is an opaque host handle (NULL on failure).
 *   dcp_batch_workspace_size  bytes of the device buffer: the constant
 *                      chunks, the three lists with their window masks, and
 *                      the backward's fp32 scratch (LSE*log2e and -Delta,
 *                      [H, T] each).
 *   dcp_batch_upload   enqueues the copy of the lists into `workspace`
 *                      (device, 256-byte aligned, at least the size above)
 *                      on `stream` and remembers that buffer and the current
 *                      device; uploading again (to the same or another
 *                      buffer) is allowed.
 *   dcp_batch_fwd/bwd  as dcp_varlen_attn_fwd / _bwd for the batch's
 *                      descriptor; `workspace` must be the buffer of the last
 *                      upload, on the device current at that upload
 *                      (DCP_ERR_INVALID otherwise), and calls are ordered
 *                      after the upload by the stream (or by the caller's
 *                      synchronisation when streams differ).  Calls that
 *                      share one buffer must not overlap in time: the
 *                      backward writes its scratch there.
 *   dcp_batch_destroy  frees the handle (host memory only; NULL is a no-op).
 *                      The device buffer stays the caller's.
 */
typedef struct dcp_batch_s* dcp_batch;
int dcp_batch_create(const dcp_attn_desc* desc, dcp_batch* out);
int dcp_batch_workspace_size(dcp_batch batch, size_t* bytes);
int dcp_batch_upload(dcp_batch batch, void* workspace, size_t workspace_bytes, void* stream);
int dcp_batch_fwd(dcp_batch batch, const void* q, const void* k, const void* v, void* o, float* lse,
                  void* workspace, size_t workspace_bytes, void* stream);
int dcp_batch_bwd(dcp_batch batch, const void* dout, const void* o, const float* lse, const void* q,
                  const void* k, const void* v, void* dq, void* dk, void* dv, void* workspace,
                  size_t workspace_bytes, void* stream);
void dcp_batch_destroy(dcp_batch batch);

/*
 * The work the attention kernels run for `desc` (introspection for
 * schedulers and tests: launches nothing, needs no GPU).  pass 0 is the
 * forward, 1 the dK/dV pass, 2 the dQ pass (at head widths up to 96 the dQ
 * pass launches only its sequence tiles: the dK/dV launch over the same
 * packed windows forms their dQ too).  Each unit is 5 int32
 * {row0, seq0, seqlen, rows, head}: rows [row0, row0 + rows) of head `head`
 * in the sequence occupying rows [seq0, seq0 + seqlen); rows == 0 is
 * padding.  Units [0, *n_tiles) are such sequence tiles (tiles restart at
 * every sequence start, so no block across two sequences is visited).  The
 * rest are packed windows: runs of consecutive sequences, each shorter than
 * the pass's window size (128 rows; 256 for the dK/dV pass at head width
 * 128), sharing one tile of rows
 * [row0, row0 + rows) (row0 == seq0), each
 * row attending only within its own sequence; window w = -seqlen - 1 owns
 * window_starts[4w .. 4w+3], where bit x % 64 of word x / 64 is set when a
 * sequence starts at offset x of the window.  Each part is 8 consecutive
 * per-die lists of equal length.
 *   units          host int32 [cap][5], or NULL to query the counts only.
 *   window_starts  host uint64 [cap_windows][4], or NULL.
 *   n_units, n_tiles, n_windows  outputs (required).
 * Returns DCP_ERR_INVALID for a bad desc or pass, or when a non-null array
 * is too small (nothing is written then).
 */
int dcp_work_list(const dcp_attn_desc* desc, int32_t pass, int32_t* units, size_t cap, size_t* n_units,
                  size_t* n_tiles, uint64_t* window_starts, size_t cap_windows, size_t* n_windows);

/*
 * Instrumentation hook for profilers and benchmarks.  begin/end are
 * hipEvent_t handles (as void*) created by the caller.  While set on the
 * calling thread, every dcp_varlen_attn_fwd call records `begin` right
 * before its attention kernel and `end` right after it (its sequence-tile
 * and packed-window launches), and every dcp_varlen_attn_bwd call does the
 * same around its dK/dV pass, on the call's stream; the Delta and dQ passes
 * and the work-list upload fall outside the pair.  Passing NULL, NULL clears the
 * hook.  Costs two event records per call while set, nothing otherwise.
 */
int dcp_set_kernel_events(void* begin, void* end);

/*
 * The current device as the runtime reports it, for stating the
 * denominators of a measurement: compute units and peak engine clock (kHz).
 * Returns DCP_ERR_HIP when there is no usable gfx950 device.
 */
int dcp_device_info(int32_t* compute_units, int32_t* clock_khz);

/* ------------------------------------------------------------------------ */
/* Per-length cost profile (Sec. 3.5)                                        */
/* ------------------------------------------------------------------------ */

/* One profile row: per-layer costs of one sequence of length seq_len with
 * micro-batch 1 on one device. */
typedef struct {
  int64_t seq_len;
  int64_t t_f_ns;      /* forward time of one layer */
  int64_t t_b_ns;      /* backward time of one layer (no recompute) */
  int64_t m_bytes;     /* activations one layer stashes for backward */
  int64_t m_inp_bytes; /* the layer's input activation */
} dcp_cost_row;

/*
 * Profiling options.  Times are the median over `reps` timed runs after
 * `warmup` untimed ones (the paper times the second of two layers, the
 * first being warm-up).  lin_*_ps_per_token add a caller-supplied linear
 * per-token term (picoseconds/token) for the non-attention part of a layer.
 * Memory is analytic: m = s * act_bytes_per_token, m_inp = s *
 * inp_bytes_per_token.  scale <= 0 selects 1/sqrt(head_dim).
 */
typedef struct {
  int32_t n_heads;
  int32_t head_dim;
  int32_t causal;
  float scale;
  int32_t warmup;
  int32_t reps;
  int64_t lin_f_ps_per_token;
  int64_t lin_b_ps_per_token;
  int64_t act_bytes_per_token;
  int64_t inp_bytes_per_token;
} dcp_profile_opts;

/* Workspace bytes for profiling lengths up to max_len. */
int dcp_profile_workspace_size(int64_t max_len, const dcp_profile_opts* opts, size_t* bytes);

/*
 * Measure one row per length: a single sequence of lengths[i] tokens with
 * the given heads and width, synthetic inputs written into the workspace,
 * forward and backward timed with HIP events on `stream`.  Each length's
 * work lists are built and uploaded before its first run; the warm-up and
 * timed runs are then enqueued back to back with events around every timed
 * forward and backward, so the rows hold device time, not host time.
 * Synchronises.
 *   lengths   host int64 [n], each in [1, max_len used for the workspace].
 *   out_rows  host [n], written only on success.
 */
int dcp_profile_cost(const int64_t* lengths, int32_t n, const dcp_profile_opts* opts, void* workspace,
                     size_t workspace_bytes, void* stream, dcp_cost_row* out_rows);

/* ------------------------------------------------------------------------ */
/* Planner (Secs. 3.2-3.5, Appendix C)                                       */
/* ------------------------------------------------------------------------ */

/* Cost table: rows strictly increasing in seq_len, every value >= 0, plus
 * the model constants of Eqs. (4)-(6): layer count L, constant time T_C and
 * constant memory M_C. */
typedef struct {
  const dcp_cost_row* rows;
  int32_t n_rows;
  int32_t n_layers;
  int64_t T_C_ns;
  int64_t M_C_bytes;
} dcp_cost_table;

enum {
  DCP_PLAN_INTER = 0, /* DCP-inter: full recomputation, balance by accumulation */
  DCP_PLAN_INTRA = 1  /* DCP-intra: fewest recomputed layers that fit memory */
};
enum {
  DCP_PLAN_FLAG_MIN_TIME = 1,      /* rank candidates by raw step time, not Eq. (1) throughput */
  DCP_PLAN_FLAG_NO_HEAD_FILTER = 2 /* allow p that does not divide n_heads */
};

/*
 * Planner options (NULL = defaults from dcp_plan_opts_default):
 *   sp_cands/n_sp       candidate sequence-parallel sizes, strictly increasing
 *                       (default {1,2,4,8}).
 *   b_max               micro-batch sizes 1..b_max are tried (default 64).
 *   n_heads             head count; p must divide it (default 16).
 *   hidden              hidden size moved by each Ulysses all-to-all (1152).
 *   a2a_alpha_ns        per-all-to-all latency (10000).
 *   link_bytes_per_ns   bytes per ns of one point-to-point link (153).
 *   g_min, g_max        accumulation bounds of Appendix C (1, 4).
 *   mode                DCP_PLAN_INTRA (default) or DCP_PLAN_INTER.
 *   flags               DCP_PLAN_FLAG_* bits (0).
 */
typedef struct {
  const int32_t* sp_cands;
  int32_t n_sp;
  int32_t b_max;
  int32_t n_heads;
  int64_t hidden;
  int64_t a2a_alpha_ns;
  int64_t link_bytes_per_ns;
  int32_t g_min;
  int32_t g_max;
  int32_t mode;
  int32_t flags;
} dcp_plan_opts;

void dcp_plan_opts_default(dcp_plan_opts* opts);

/* Caller-sized outputs, one entry per batch; recompute_flags holds
 * n_batches * n_layers bytes, flag [i*L + l] = 1 iff layer l of batch i is
 * recomputed (the first r_i layers).  step_time_ns and mem_bytes may be NULL.
 * idle_ns and makespan_ns describe the whole iteration: makespan =
 * max_i g_i*T_i and idle = sum_i (makespan - g_i*T_i) (Eq. (3) times W). */
typedef struct {
  int32_t* sp_size;
  int32_t* micro_batch;
  int32_t* grad_accum;
  int32_t* recompute_layers;
  uint8_t* recompute_flags;
  int64_t* step_time_ns;
  int64_t* mem_bytes;
  int64_t idle_ns;
  int64_t makespan_ns;
} dcp_plan_out;

/*
 * Plan one iteration.  Every sequence is its own batch when batch_offsets
 * is NULL (then n_batches must equal n_seqs); otherwise batch i packs
 * sequences batch_offsets[i] .. batch_offsets[i+1]-1 (CSR, n_batches+1
 * entries, each batch non-empty).  Each sequence takes the table row with
 * the smallest length >= its own; a pack sums its rows.  All arithmetic is
 * int64 with overflow checks (DCP_ERR_INVALID); the result is bit-exact
 * and deterministic.  Outputs are written only on success.
 * Errors: DCP_ERR_INVALID (arguments), DCP_ERR_TABLE (table or a length
 * beyond it), DCP_ERR_INFEASIBLE (no (p, b, r) fits hbm_budget_bytes; the
 * message names the batch).
 */
int dcp_plan(const int64_t* seq_lens, int32_t n_seqs, const int32_t* batch_offsets, int32_t n_batches,
             const dcp_cost_table* table, int64_t hbm_budget_bytes, const dcp_plan_opts* opts,
             dcp_plan_out* out);

/* ------------------------------------------------------------------------ */
/* Transformer layer around the attention (the unit of Secs. 3.4-3.5)        */
/* ------------------------------------------------------------------------ */

/*
 * One pre-norm transformer layer over a packed batch: the unit whose
 * forward time t_f, backward time t_b and stashed activations m the
 * profiling of Sec. 3.5 measures, and whose forward runs again in the
 * backward when the layer is recomputed (Eqs. (4)-(6)).
 *   y1 = RMSNorm(x; norm1), q = y1 Wq, k = y1 Wk, v = y1 Wv,
 *   o = attention(q, k, v) (dcp_varlen_attn_fwd on `attn`),
 *   h = x + o Wo, y2 = RMSNorm(h; norm2), a = GELU(y2 Wup) (tanh form),
 *   out = h + a Wdown.
 * RMSNorm(z; g) = z * g / sqrt(mean(z^2) + eps) per row.  hidden = H*D of
 * `attn`, at most 4096 (DCP_ERR_UNSUPPORTED beyond); every row of x is a
 * token of some sequence (cu_seqlens[n] must equal total_tokens).  GEMMs run in rocBLAS (bf16 in, fp32 accumulation)
 * with their scratch taken from the caller's workspace; the rocBLAS handle
 * (one per thread and device, kept until the thread ends) is the only
 * device memory the library itself holds.
 */
typedef struct {
  const dcp_attn_desc* attn;
  float eps; /* RMSNorm epsilon, finite and >= 0 */
} dcp_layer_desc;

/* bf16 device weights, row-major [in, out]: wq, wk, wv, wo [hidden, hidden],
 * w_up [hidden, 4*hidden], w_down [4*hidden, hidden]; norm1, norm2 [hidden]. */
typedef struct {
  const void *norm1, *wq, *wk, *wv, *wo, *norm2, *w_up, *w_down;
} dcp_layer_weights;

/* fp32 device gradients of the same shapes; the backward adds into them. */
typedef struct {
  float *norm1, *wq, *wk, *wv, *wo, *norm2, *w_up, *w_down;
} dcp_layer_grads;

/* Bytes of the activation stash (kept from forward to backward when the
 * layer is not recomputed) and of the forward and backward workspaces
 * (256-byte aligned device memory).  Any output may be NULL. */
int dcp_layer_sizes(const dcp_layer_desc* desc, size_t* stash_bytes, size_t* fwd_workspace_bytes,
                    size_t* bwd_workspace_bytes);

/*
 * Forward: out = layer(x), x and out bf16 [T, hidden].  With a stash
 * (device, stash_bytes, 256-byte aligned) every activation the backward
 * needs is kept there; with stash = NULL nothing is kept (the layer will be
 * recomputed).  Enqueued on `stream`.
 */
int dcp_layer_fwd(const dcp_layer_desc* desc, const dcp_layer_weights* w, const void* x, void* out, void* stash,
                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward of <dout, out>: dx (bf16 [T, hidden]) and, added into `grads`,
 * the weight gradients.  `x` is the forward's input.  `stash` is the
 * forward's stash, or NULL when the forward kept none: the forward is then
 * run again first, into the workspace (recomputation).
 */
int dcp_layer_bwd(const dcp_layer_desc* desc, const dcp_layer_weights* w, const void* x, const void* dout, void* dx,
                  const dcp_layer_grads* grads, void* stash, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Schedule replay: DCP against bucket parallelism (Secs. 2.3-2.4, 4.1-4.2)   */
/* ------------------------------------------------------------------------ */

/*
 * Replay options:
 *   n_devices     W, the devices of the data-parallel job (>= 1).
 *   bucket_sp     the fixed sequence-parallel size of the bucket-parallel
 *                 baseline; 0 picks the smallest candidate p (dividing
 *                 n_heads unless DCP_PLAN_FLAG_NO_HEAD_FILTER) at which
 *                 every batch of the stream fits at micro-batch 1.
 *   iter_sync_ns  time of the once-per-iteration gradient synchronisation
 *                 (Sec. 2.4), added to every iteration of both schedules.
 */
typedef struct {
  int32_t n_devices;
  int32_t bucket_sp;
  int64_t iter_sync_ns;
} dcp_sim_opts;

/*
 * Totals over the replayed iterations.  Throughput (Eq. (1), tokens per
 * second) = tokens / time_ns * 1e9; the imbalance ratio of Sec. 4.2 (the
 * share of device time spent waiting for other devices) =
 * 1 - busy_device_ns / (n_devices * makespan_ns).
 *   iterations      iterations formed from the stream.
 *   makespan_ns     sum of the iterations' compute spans, max_i g_i*T_i.
 *   time_ns         makespan_ns + iterations * iter_sync_ns.
 *   busy_device_ns  sum of p_i * g_i * T_i over every batch.
 *   tokens          sum of g_i * b_i * S_i (S_i: tokens of batch i).
 *   bucket_sp       the baseline's sequence-parallel size (0 for DCP).
 */
typedef struct {
  int64_t iterations;
  int64_t makespan_ns;
  int64_t time_ns;
  int64_t busy_device_ns;
  int64_t tokens;
  int32_t bucket_sp;
} dcp_sim_result;

/*
 * Replays a stream of batches (same arguments and validation as dcp_plan)
 * on W devices under two schedules.
 * DCP: each batch takes the planner's (p_i, b_i, r_i, T_i) (opts->mode
 * selects DCP-intra or DCP-inter); batches join the current iteration in
 * stream order while sum_i p_i <= W (the constraint of Eq. (1); devices left
 * over wait out the iteration), and the iteration's accumulation steps g_i
 * follow Eq. (3) within the bounds of Appendix C.
 * Bucket parallelism (the baseline of Sec. 4.1, the static batch sizing of
 * Sec. 2.4): one fixed p, floor(W/p) batches per iteration in stream order,
 * full recomputation, g_i = 1, and per batch the largest b <= b_max whose
 * step time does not exceed the stream's slowest batch at b = 1 and whose
 * memory fits.
 * Integer arithmetic throughout; results are bit-exact.  Errors as for
 * dcp_plan, plus DCP_ERR_INVALID when a batch needs more than W devices.
 */
int dcp_simulate(const int64_t* seq_lens, int32_t n_seqs, const int32_t* batch_offsets, int32_t n_batches,
                 const dcp_cost_table* table, int64_t hbm_budget_bytes, const dcp_plan_opts* opts,
                 const dcp_sim_opts* sim, dcp_sim_result* dcp_out, dcp_sim_result* bucket_out);

#ifdef __cplusplus
}
#endif

#endif /* DCP_H */
