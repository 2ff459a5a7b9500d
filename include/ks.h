/*
 * ks.h — C ABI of the MI355X (gfx950) batched kernel-latency evaluator.
 *
 * The library evaluates the per-kernel latency model of KernelSight-LM
 * (arXiv 2606.28565) for every (hardware spec vector, dispatched-kernel
 * record) pair and aggregates the kernels into per-step latencies:
 *
 *   t      = max(t_roof * eta, t0),                    Eq. 2 (Sec. 5.3)
 *   t_roof = max(F * u / P_peak, Bt / BW_peak),        Eq. 2
 *   u      = ceil(B / N_cu) * N_cu / B,                Sec. 2.2
 *   eta    = 1 / sigma(z) = 1 + exp(-z), z from a per-family MLP head on
 *            dimensionless features,                   Sec. 5.3
 *   t_ar   = alpha0(P) + 2 (P - 1) / P * S / beta,     Eq. 3 (Sec. 5.6)
 *   t_step = max(t_gpu + n c_disp, l) + max(0, c_ovl - t_gpu) + c_tail,
 *                                                      Eq. 4 (Sec. 5.7)
 *
 * Conventions (all entry points):
 *  - Pointers named "device" are device memory owned by the caller; the
 *    library never allocates, frees or keeps them after the call returns.
 *    Structs themselves are read on the host during the call only.
 *  - Work is enqueued asynchronously on the caller's HIP stream; outputs are
 *    valid once that stream has completed the call's work.  Concurrent calls
 *    that share a workspace race.
 *  - Errors are returned as ks_status (never thrown, never abort); the
 *    thread-local message of the last failing call is ks_last_error().
 *  - Host-side checks run before any launch.  Conditions that depend on
 *    device data (ranges, sortedness, offsets) are checked synchronously by
 *    ks_validate(); the evaluation kernels themselves never read or write out
 *    of bounds on bad data: they skip the offending record and raise a flag
 *    that ks_device_status() reports.
 *  - Units: seconds, FLOP/s, bytes, bytes/s.
 */
#ifndef KS_H
#define KS_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KS_OK = 0,
  KS_EINVAL = 1,      /* bad argument: null pointer, bad size, unsorted data */
  KS_ERANGE = 2,      /* a shape or count outside the documented limits      */
  KS_EHIP = 3,        /* a HIP runtime call failed                           */
  KS_EWORKSPACE = 4   /* workspace missing or smaller than required          */
} ks_status;

/* Kernel families (Sec. 5.3 learns eta per family). */
enum {
  KS_GEMM = 0, KS_LM_HEAD, KS_GROUPED_GEMM, KS_ATTN_PREFILL, KS_ATTN_DECODE,
  KS_RMSNORM, KS_ROPE, KS_SILU_MUL, KS_KV_WRITE, KS_EMBED, KS_NFAM
};

/*
 * Dispatched-kernel records (the predictor's per-kernel input, Sec. 4.1),
 * structure of arrays, family-major: records [fam_off[f], fam_off[f+1]) all
 * belong to family f, and within a family their step indices never
 * decrease.  Field meaning per family (unused fields are ignored):
 *
 *   GEMM, LM_HEAD   m = M, n = N, k = K
 *   GROUPED_GEMM    n = N, k = K, a = E experts, b = offset of the E
 *                   per-expert row counts M_e in expert_rows
 *   ATTN_PREFILL,   n = H query heads, k = head dim d, a = Hkv KV heads;
 *   ATTN_DECODE     the queries are the requests of the record's step
 *                   (Sec. 5.8: each decode over its context, a prefill chunk
 *                   over its history plus its causal triangle)
 *   RMSNORM         m = T tokens, n = D
 *   ROPE            m = T, n = rotated heads, k = d
 *   SILU_MUL        m = T rows, n = I output width
 *   KV_WRITE        m = T, n = Hkv, k = d
 *   EMBED           m = T, n = D
 *
 * The batch descriptor of each step (Sec. 4.1) is its request list:
 * requests [req_off[j], req_off[j+1]) with q_r query tokens and h_r cached
 * history tokens.  Limits (KS_ERANGE): n_rows < 2^32; m < 2^24; n, k < 2^18;
 * attention n, k, a < 2^12; q_r, h_r < 2^24; per-step causal pairs < 2^40;
 * sum of a grouped record's M_e < 2^24; E <= 1024; elem_bytes in 1..8.
 */
typedef struct ks_desc {
  int64_t n_rows;
  int64_t fam_off[KS_NFAM + 1];          /* host array, fam_off[0] = 0       */
  const uint32_t *step;                  /* device [n_rows]                  */
  const uint32_t *m, *n, *k, *a, *b;     /* device [n_rows]                  */
  int64_t n_steps;
  const uint32_t *req_off;               /* device [n_steps + 1], req_off[0] = 0 */
  const uint32_t *req_q, *req_h;         /* device [n_req]                   */
  int64_t n_req;
  const uint32_t *expert_rows;           /* device [n_expert_rows] or NULL   */
  int64_t n_expert_rows;
  uint32_t elem_bytes;                   /* dt, bytes per element (2 = bf16) */
  uint32_t reserved;
  /* device [n_rows] or NULL: the number of dispatches each record stands
   * for (Sec. 5.7: decoder layers are homogeneous, so a kernel that is the
   * same in every layer may be one record of multiplicity L).  The step body
   * adds mult * t for the record; per-pair outputs stay per dispatch.  NULL:
   * every record is one dispatch.  Limit: mult < 2^24. */
  const uint32_t *mult;
} ks_desc;

/*
 * One hardware spec vector (Tier A datasheet, Sec. 5.4) and its interconnect
 * (Sec. 5.6).  Passed as a DEVICE array of n_specs records (64 bytes each).
 * alpha0(P) = ar_alpha0 + ar_alpha_log2p * log2(P).
 */
typedef struct ks_spec {
  double peak_flops;       /* P_peak, FLOP/s, > 0                     */
  double hbm_bw;           /* BW_peak, bytes/s, > 0                   */
  double t0;               /* launch floor, s, >= 0                   */
  double l2_bytes;         /* L2 capacity, bytes, >= 0                */
  double ar_alpha0;        /* all-reduce startup, s                   */
  double ar_alpha_log2p;   /* startup growth per doubling of P, s     */
  double ar_beta;          /* effective interconnect bandwidth, B/s   */
  uint32_t n_cu;           /* N_SM, 1 .. 65535                        */
  uint32_t reserved;
} ks_spec;

enum { KS_F32 = 0, KS_BF16 = 1 };
enum { KS_ETA_MLP = 0, KS_ETA_ONE = 1 };

/*
 * Per-family efficiency heads (Sec. 5.3), device arrays, row-major [out][in]:
 *   w1 [KS_NFAM][hidden][in_dim]   (no first-layer bias: feature 15 is 1)
 *   w2 [KS_NFAM][hidden][hidden], b2 [KS_NFAM][hidden]
 *   w3 [KS_NFAM][hidden],         b3 [KS_NFAM]
 * Element type float for KS_F32, bfloat16 bits (uint16) for KS_BF16.
 * z = w3 . relu(W2 relu(W1 x) + b2) + b3;  eta = 1 + exp(-z).
 * Supported: in_dim 16 or 32; hidden 64 or 128 (KS_F32), 64, 128 or 256
 * (KS_BF16).  mode KS_ETA_ONE: eta = 1 (the MLP fields are ignored).
 *
 * Per-family head selection (Sec. 5.3 picks each family's head from a pool):
 * the families whose bit is set in bounded_mask (bit f = family f) take
 * the bounded analytical head of Sec. 5.3 and its efficiency-factor figure
 * instead of the MLP (mode KS_ETA_MLP) or of eta = 1 (mode KS_ETA_ONE):
 *   gamma = sigma(g . x), alpha = gamma sigma(a . x), W' = max(W, 1),
 *   eta = 1 / (gamma - alpha / W'),
 * over the 16 base features x and the record's wave count W.  bounded:
 * device float array [KS_NFAM][2][16], g then a per family (rows of other
 * families are not read); NULL if bounded_mask is 0.  The MLP weights may be
 * NULL when every family is in bounded_mask.  Computed in fp32.
 *
 * Tier B, density-routed measured grids (Sec. 5.5, "Tier B"): for the
 * families whose bit is set in grid_mask, eta comes from a grid of measured
 * values over three of the 16 base features, axis d taking feature
 * grid_axis[d] (0 .. 14) on grid_n[d] >= 2 evenly spaced nodes from
 * grid_lo[d] to grid_hi[d] (finite, lo < hi).  A query is routed to the
 * grid when its coordinates lie in the closed box and the eight corners of
 * its cell are all measured (not NaN); there eta is the trilinear
 * interpolation of the corners.  Other queries of such a family take the
 * family's other head (MLP, bounded head or eta = 1, as above).
 * grid: device float array [KS_NFAM][n0][n1][n2], row-major, NaN for a node
 * never measured (rows of families outside grid_mask are not read); NULL if
 * grid_mask is 0.  n0 n1 n2 <= KS_GRID_MAX_NODES.  Computed in fp32: a query
 * within rounding of a cell face next to an unmeasured node, or of the box,
 * may be routed either way.
 */
enum { KS_GRID_MAX_NODES = 2048 };

typedef struct ks_heads {
  int32_t in_dim, hidden, precision, mode;
  const void *w1, *w2, *b2, *w3, *b3;
  uint32_t bounded_mask;   /* bits 0 .. KS_NFAM-1 */
  uint32_t grid_mask;      /* bits 0 .. KS_NFAM-1 */
  const float *bounded;
  int32_t grid_axis[3];
  int32_t grid_n[3];
  double grid_lo[3], grid_hi[3];
  const float *grid;
} ks_heads;

/* Per-step model record, device arrays [n_steps]. */
typedef struct ks_steps {
  int64_t n_steps;                 /* must equal ks_desc.n_steps               */
  const uint32_t *layers;          /* L                                        */
  const uint32_t *hidden;          /* D (all-reduce message S = T * D * dt)    */
  const uint32_t *tp;              /* P (1: no all-reduce)                     */
  const uint32_t *n_launch;        /* n of Eq. 4: host launches priced c_disp  */
} ks_steps;

/* Host constants of Eq. 4 (host memory, read during the call). */
typedef struct ks_host {
  double c_disp, ell, c_ovl, c_tail, body_scale;
} ks_host;

/* Per-record and per-pair outputs (device; any pointer may be NULL = skip).
 * flops, bytes, blocks: [n_rows]; t_roof, eta, t_kernel: [n_specs][n_rows].
 * source: [n_specs][n_rows], where each pair's eta came from: 0 the head of
 * heads.mode (the MLP, or eta = 1), 1 the bounded analytical head, 2 the
 * measured Tier B grid (density routing, Sec. 5.5). */
typedef struct ks_kernel_out {
  uint64_t *flops, *bytes, *blocks;
  float *t_roof, *eta, *t_kernel;
  uint8_t *source;
} ks_kernel_out;

/* Per-step outputs (device, [n_specs][n_steps], none may be NULL). */
typedef struct ks_step_out {
  double *t_body, *t_gpu, *t_step;
} ks_step_out;

/*
 * Batch expansion (Sec. 4.1: the scheduler's batch descriptor of each step;
 * Sec. 5.7: one embedding and one LM head per step around L homogeneous
 * layers; Sec. 5.8: the dense GEMMs, norms and activations run over the
 * step's T = sum q_r tokens, attention over its requests).  ks_expand writes
 * the records (and the per-step model record) of every kernel the steps of
 * one batch dispatch, on the device, in the layout ks_eval_steps reads.
 *
 * Per layer, in dispatch order (per-GPU shard sizes under TP P: H = Hq/P,
 * Hkv = ceil(Hkv/P), I = ffn/P, I_e = expert_ffn/P, V/P):
 *   GEMM QKV (m T, n (H + 2 Hkv) d, k D); ROPE (T, H + Hkv, d);
 *   KV_WRITE (T, Hkv, d) if kv_write; attention (n H, k d, a Hkv) in
 *   ATTN_PREFILL if the step's prefill flag is set, else ATTN_DECODE;
 *   GEMM O (T, D, H d); RMSNORM (T, D) twice; then dense: GEMM gate/up
 *   (T, 2I, D), SILU_MUL (T, I), GEMM down (T, D, I); or experts > 0: GEMM
 *   router (T, E, D), GROUPED_GEMM gate/up (n 2 I_e, k D, a E,
 *   b (j L + l) E), SILU_MUL (top_k T, I_e), GROUPED_GEMM down (n D, k I_e,
 *   a E, b (j L + l) E).
 * Per step j: EMBED (T, D) and LM_HEAD (m R requests, n V/P, k D).
 * Unused fields are written as 0.  Records are family-major; within a
 * family by step, then layer, then dispatch order.  Grouped records point
 * at the routed row counts M_e of (step j, layer l): the caller passes its
 * [n_steps][L][E] routing array as ks_desc.expert_rows (n_expert_rows =
 * n_steps L E).  Per-step record: layers L, hidden D, tp P, n_launch = L for
 * a step with a prefill chunk (eager, one launch charge per layer) else 0.
 *
 * KS_EXPAND_HOMOGENEOUS: every kernel that is the same in all L layers of
 * a step (all but the grouped GEMMs) is one record of multiplicity L, in
 * dispatch order within its family; the grouped GEMMs stay per layer.
 * KS_EXPAND_PER_LAYER: one record per dispatched kernel (multiplicity 1).
 */
typedef struct ks_model {
  uint32_t hidden;       /* D, >= 1                                       */
  uint32_t layers;       /* L, >= 1                                       */
  uint32_t q_heads;      /* Hq (whole model), divisible by tp             */
  uint32_t kv_heads;     /* Hkv (whole model), >= 1                       */
  uint32_t head_dim;     /* d                                             */
  uint32_t ffn;          /* dense MLP width, divisible by tp (unused for experts > 0) */
  uint32_t vocab;        /* V, divisible by tp                            */
  uint32_t tp;           /* P, >= 1                                       */
  uint32_t experts;      /* E: 0 = dense MLP, else 1 .. 1024 experts      */
  uint32_t top_k;        /* routed copies per token, 1 .. E (experts > 0) */
  uint32_t expert_ffn;   /* per-expert width, divisible by tp (experts > 0) */
  uint32_t kv_write;     /* 1: a KV-cache write kernel per layer, else 0  */
} ks_model;

/* One batch of consecutive steps (device arrays unless noted). */
typedef struct ks_batch {
  int64_t n_steps;
  const uint32_t *req_off;   /* [n_steps + 1], req_off[0] = 0, non-decreasing */
  const uint32_t *req_q;     /* [n_req] query tokens of each request          */
  int64_t n_req;
  const uint8_t *prefill;    /* [n_steps] nonzero: the step has a prefill chunk */
  int64_t n_prefill;         /* host value: how many prefill flags are nonzero */
} ks_batch;

enum { KS_EXPAND_PER_LAYER = 0, KS_EXPAND_HOMOGENEOUS = 1 };

/* Outputs of ks_expand (device, caller-owned).  Record arrays hold
 * fam_off[KS_NFAM] entries (fam_off from ks_expand_layout); mult may be NULL
 * in KS_EXPAND_PER_LAYER mode.  layers, hidden, tp, n_launch: [n_steps],
 * the ks_steps arrays of the batch. */
typedef struct ks_records {
  uint32_t *step, *m, *n, *k, *a, *b, *mult;
  uint32_t *layers, *hidden, *tp, *n_launch;
} ks_records;

/* Host only: the family offsets of the expansion of n_steps steps of which
 * n_prefill carry a prefill chunk (fam_off[0] = 0, fam_off[KS_NFAM] = record
 * count).  Checks the model (KS_EINVAL / KS_ERANGE: sizes not divisible by
 * tp, record fields beyond the ks_desc limits, more than 2^32 - 1 records
 * or routed-row offsets). */
ks_status ks_expand_layout(const ks_model* model, int64_t n_steps, int64_t n_prefill, int32_t mode,
                           int64_t fam_off[KS_NFAM + 1]);

/* Bytes of device workspace ks_expand needs for n_steps steps. */
size_t ks_expand_workspace_bytes(int64_t n_steps);

/* Writes the records of the batch (asynchronous on `stream`).  Host checks
 * as ks_expand_layout plus null pointers and the workspace, and KS_ERANGE
 * for a family with 2^16 or more records per step or 2^31 or more records
 * in all (the record writer's index arithmetic).  Device data
 * that disagrees with the call (request offsets out of order or beyond
 * n_req, a step's T or top_k T at or above 2^24, a prefill flag count other
 * than n_prefill) raises a flag that ks_device_status(ws) reports; the
 * kernels then still write only inside the record arrays. */
ks_status ks_expand(const ks_model* model, const ks_batch* batch, int32_t mode, const ks_records* out,
                    void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Serving simulation with the scheduler in the loop (Sec. 4.1-4.2: the
 * discrete-event simulator asks the predictor for every batch the scheduler
 * forms and advances its clock by the predicted step time; Sec. 5.8: one
 * token-budget loop over computed-token counts gives continuous batching,
 * chunked prefill and prefix-cache-aware FCFS admission, with preemption by
 * recompute under KV pressure; Sec. 2.1: TTFT, TPOT, output throughput).
 * The scheduler runs on the host, one simulation per spec vector, all fed
 * the same requests and run in lockstep: each round every unfinished
 * simulation forms its next step (request r: q_r new tokens over h_r
 * computed ones; prefill flag); the round's steps are expanded on the GPU
 * as one batch in the homogeneous form and priced by one evaluation call
 * against all the spec vectors (A steps x n_specs pairs of steps and specs,
 * of which each step keeps its own simulation's t_step); the host reads one
 * latency per simulation back before the next round.
 *
 * Rules (per step, at the simulation clock):
 *  - requests that have arrived join the waiting queue (FCFS);
 *  - running requests, in admission order, get n = min(target - computed,
 *    budget) tokens, target = prompt + generated; KV blocks of block_tokens
 *    tokens are allocated for computed + n; when they do not fit, cached
 *    prefixes no running request shares are evicted (least recently used
 *    first), then the most recently admitted running request is preempted
 *    (blocks freed, computed reset to 0, back to the front of the queue);
 *  - unless a request was preempted in this step, waiting requests are
 *    admitted FCFS while budget > 0 and fewer than max_num_seqs run: a
 *    cached prefix of c blocks starts computed at min(c, floor((target - 1)
 *    / block_tokens)) blocks; admission stops at the first request whose
 *    blocks do not fit after evicting unused prefixes; a request whose
 *    prompt + output tokens exceed the whole cache is rejected;
 *  - a request whose computed count first covers its group's full prefix
 *    blocks (floor(prefix / block_tokens)) when the group has none cached
 *    turns them into the group's cache entry;
 *  - the step carries a prefill chunk if some scheduled request has more
 *    than one token left to compute; after the step each request's computed
 *    count grows by n; one that reaches its target samples a token (the
 *    first one sets TTFT) and finishes at `output` tokens.
 * TTFT = first token - arrival; TPOT = (last token - first token) /
 * (output - 1), 0 for one output token; E2E = finish - arrival.
 * Dense decoders only (experts = 0).
 */
typedef struct ks_sched {
  int32_t max_num_seqs;        /* running requests per step, >= 1           */
  int32_t max_batched_tokens;  /* token budget per step, >= 1               */
  int32_t block_tokens;        /* tokens per KV block, >= 1                 */
  int32_t prefix_cache;        /* 1: reuse cached prefix blocks, else 0     */
  int64_t kv_blocks;           /* KV-cache capacity in blocks, >= 1         */
} ks_sched;

/* Requests, HOST arrays [n], sorted by arrival (non-decreasing). */
typedef struct ks_requests {
  int64_t n;
  const double *arrival;       /* seconds, finite                           */
  const uint32_t *prompt;      /* prompt tokens, 1 .. 2^24 - 1              */
  const uint32_t *output;      /* output tokens, 1 .. 2^24 - 1              */
  const uint32_t *group;       /* shared-prefix group, 0 = none; NULL: none */
  const uint32_t *prefix;      /* tokens the group shares, <= prompt; NULL if group is NULL */
} ks_requests;

/* Results, HOST arrays owned by the caller (any array may be NULL = skip;
 * the step record stops silently at step_cap steps or entry_cap entries). */
typedef struct ks_sim_out {
  double *ttft, *tpot, *e2e;        /* [n] seconds, 0 for rejected requests  */
  int32_t *state;                   /* [n] 2 finished, 3 rejected            */
  int64_t step_cap, entry_cap;
  double *step_start, *step_latency;   /* [step_cap]                         */
  uint8_t *step_prefill;               /* [step_cap]                         */
  int64_t *step_entry_off;             /* [step_cap + 1] into the entries    */
  uint32_t *entry_req, *entry_q, *entry_h;  /* [entry_cap]: request, q, h   */
  /* written by ks_simulate: */
  int64_t n_steps, n_entries, preemptions;
  double clock;                     /* simulated time when the last request finished */
} ks_sim_out;

/* Bytes of device workspace ks_simulate needs for n_specs simulations (0 on
 * bad arguments). */
size_t ks_simulate_workspace_bytes(const ks_model* model, const ks_sched* sched, int32_t n_specs);

/* Runs n_specs simulations (1 .. 256) to completion (synchronous: it waits
 * for each round's latencies on `stream`).  The one entry point that
 * allocates: two pinned HOST buffers for the rounds' copies (the round's
 * packed batch, 8 max_num_seqs + 9 bytes per simulation plus 4, and its
 * latencies, 8 bytes per simulation), freed before it returns.  specs:
 * DEVICE array of n_specs
 * ks_spec; heads and host as for ks_eval_steps; out: HOST array of n_specs
 * results, out[s] for specs[s] (the same request arrays are read by all).
 * A simulation's results do not depend on the others run beside it, up to
 * the rounding order of its steps' sums (which depends on where a step sits
 * in the round's batch).
 * KS_EINVAL / KS_ERANGE on bad arguments (unsorted arrivals, zero-length
 * prompts or outputs, prefix > prompt, a model with experts, n_specs out of
 * range), KS_EHIP on a failed runtime call, and the evaluation's own
 * statuses; the results are then undefined. */
ks_status ks_simulate(const ks_model* model, const ks_spec* specs, int32_t n_specs, const ks_heads* heads,
                      const ks_host* host, const ks_sched* sched, const ks_requests* requests,
                      ks_sim_out* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Bytes of device workspace ks_eval_kernels / ks_eval_steps / ks_validate
 * need for this record set and spec count (256-byte aligned).  0 on bad
 * arguments. */
size_t ks_workspace_bytes(const ks_desc* desc, int32_t n_specs);

/* Per-pair latencies (Eq. 2) for every spec vector and record.  ws: device
 * workspace of at least ks_workspace_bytes() bytes. */
ks_status ks_eval_kernels(const ks_desc* desc, const ks_spec* specs, int32_t n_specs,
                          const ks_heads* heads, const ks_kernel_out* out,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/* Per-step latencies (Sec. 5.6–5.7, Eq. 3–4) for every spec vector, plus
 * optional per-pair outputs (kout may be NULL).  Every record of a step must
 * be in desc. */
ks_status ks_eval_steps(const ks_desc* desc, const ks_steps* steps,
                        const ks_spec* specs, int32_t n_specs,
                        const ks_heads* heads, const ks_host* host,
                        const ks_step_out* out, const ks_kernel_out* kout,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Allocation-free ks_eval_steps, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, checks and results as ks_eval_steps,
 * without the workspace: the library uses a fixed device array of
 * KS_STATIC_SCRATCH_BYTES on each GPU instead (held from the library's load
 * on that GPU until the process ends).  A call whose ks_workspace_bytes()
 * exceeds it fails with KS_ERANGE before any launch.  Every call on one GPU
 * shares that GPU's array and leaves its contents behind: calls that
 * overlap on one GPU (other streams, other threads) race.  flags: a device
 * uint32 or NULL; if set, the call's bad-data flag word is copied there on
 * the stream after the evaluation (0: no record was skipped; nonzero: the
 * evaluation skipped bad device data, which ks_validate names).  The call
 * issues no hipMalloc, hipFree or hipMemset.
 */
enum { KS_STATIC_SCRATCH_BYTES = 64 << 20 };

ks_status ks_eval_steps_static(const ks_desc* desc, const ks_steps* steps,
                               const ks_spec* specs, int32_t n_specs,
                               const ks_heads* heads, const ks_host* host,
                               const ks_step_out* out, const ks_kernel_out* kout,
                               uint32_t* flags, hipStream_t stream);

/* Synchronous device-side check of the inputs: step order within families,
 * field limits, request and expert offsets, spec sanity.  Synchronizes the
 * stream.  Returns KS_OK, KS_EINVAL or KS_ERANGE with a message. */
ks_status ks_validate(const ks_desc* desc, const ks_steps* steps,
                      const ks_spec* specs, int32_t n_specs,
                      void* ws, size_t ws_bytes, hipStream_t stream);

/* Synchronizes the stream and reports the flag the evaluation (or
 * expansion) kernels raise when they skipped a record on bad data since the
 * workspace's last evaluation (or expansion) call started (KS_OK if none). */
ks_status ks_device_status(const void* ws, size_t ws_bytes, hipStream_t stream);

/* Measurement hook for benchmarks: with both events non-NULL, every later
 * call on this thread of ks_eval_kernels / ks_eval_steps records `before` on
 * its stream right before the evaluation kernel and `after` right after it,
 * and every ks_expand call does the same around its record-writing kernel,
 * so hipEventElapsedTime(before, after) is that one kernel's duration.
 * Calling it with NULLs turns the hook off.  The events are the caller's
 * (created with timing enabled, never destroyed by the library). */
ks_status ks_set_timing_events(hipEvent_t before, hipEvent_t after);

/* Message of the last non-OK status returned on this thread. */
const char* ks_last_error(void);

/* Library version string. */
const char* ks_version(void);

#ifdef __cplusplus
}
#endif
#endif /* KS_H */
