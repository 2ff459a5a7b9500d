// Internal interface between the C-ABI host code (ks_api.cpp) and the HIP
// kernels (ks_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime_api.h>
#include "ks.h"

namespace ks {

constexpr int kWave = 64;
constexpr int kWgWaves = 4;
constexpr int kWgThreads = kWave * kWgWaves;
constexpr int kTileRows = 64;                 // records per wave tile
constexpr int kWgRows = kTileRows * kWgWaves; // records per workgroup tile

// flags raised by the kernels on bad device data (never faults)
enum : uint32_t {
  kErrStep = 1u,      // record step >= n_steps
  kErrReq = 2u,       // request offsets out of order or out of bounds
  kErrExpert = 4u,    // grouped-GEMM expert offsets out of bounds
  kErrRange = 8u,     // a shape or count outside the documented limits
  kErrOrder = 16u,    // steps decrease within a family
  kErrSpec = 32u,     // spec vector not usable
  kErrPrefill = 64u,  // prefill flags disagree with the batch's n_prefill
};

// head kinds compiled into the evaluation kernel
enum HeadKind : int {
  kEtaOne = 0,
  kF32_16_64, kF32_16_128, kF32_32_64, kF32_32_128,
  kBF16_16_64, kBF16_16_128, kBF16_16_256, kBF16_32_64, kBF16_32_128, kBF16_32_256,
  kBoundedOnly,   // no MLP: bounded-head and grid families, eta = 1 for the rest
  kNumKinds
};

// Per-spec constants of the inner loop, computed once per call into the
// workspace (64 bytes each) so the evaluation kernel reads them with scalar
// loads instead of redoing float64 divisions in every wave.
struct alignas(16) SpecC {
  float rcp_p, rcp_bw, bw_over_p, l2, t0, rcp_t0, n_f, rcp_n;
  double rcp_nd;
  uint32_t n;
  float lr;  // log2(BW / P)
  uint32_t pad[4];
};
static_assert(sizeof(SpecC) == 64, "SpecC is one 64-byte record");

struct EvalParams {
  // records
  const uint32_t *step, *m, *n, *k, *a, *b;
  const uint32_t *expert_rows;
  int64_t n_expert_rows;
  const uint32_t *mult;        // [n_rows] dispatches per record, or NULL (1)
  const uint64_t *agg;         // [4][n_steps]: Q, KV, PAIRS, TILES
  int64_t n_steps;
  uint32_t elem_bytes;
  int32_t n_specs;
  const SpecC *spec_c;             // [n_specs], in the workspace
  int64_t fam_off[KS_NFAM + 1];
  int32_t tile_off[KS_NFAM + 1];   // wave-tile offsets per family
  int32_t wgt_off[KS_NFAM + 1];    // workgroup-tile offsets per family
  int32_t n_tiles;
  // work items: every workgroup tile once per spec range of spec_chunk
  // specs (n_chunks ranges; one range of all specs unless the record tiles
  // alone would not fill the GPU)
  int32_t spec_chunk, n_chunks;
  // heads
  const void *w1, *w2, *b2, *w3, *b3;
  uint32_t bounded_mask;       // families that take the bounded analytical head
  const float *bounded;        // [KS_NFAM][2][16]: g then a
  uint32_t grid_mask;          // families with a measured eta grid (Tier B)
  int32_t grid_axis[3], grid_n[3], grid_nodes;
  float grid_lo[3], grid_scale[3];   // node coordinate (c - lo) * scale
  const float *grid;           // [KS_NFAM][grid_nodes]
  // per-record / per-pair outputs (nullable)
  uint64_t *o_flops, *o_bytes, *o_blocks;
  float *o_troof, *o_eta, *o_t;
  // per-step partial sums (nullable: no step sums)
  double *partial;   // [KS_NFAM][n_steps][n_specs] (spec-minor)
  double *carry;     // [n_tiles][n_specs]
  uint32_t *range;   // [KS_NFAM][n_steps][2] record range of each (family, step); nullable
  uint32_t *err;
  uint8_t *o_src;    // per pair: 0 head of the mode, 1 bounded head, 2 grid (nullable)
};

struct FinishParams {
  const uint64_t *agg;                 // [4][n_steps]
  const uint32_t *layers, *hidden, *tp, *n_launch;
  int64_t n_steps;
  int32_t n_specs;
  uint32_t elem_bytes;
  const ks_spec *specs;
  int64_t fam_off[KS_NFAM + 1];
  int32_t tile_off[KS_NFAM + 1];
  const double *partial, *carry;       // [KS_NFAM][n_steps][n_specs], [n_tiles][n_specs]
  int32_t n_tiles;
  const uint32_t *range;               // [KS_NFAM][n_steps][2]
  ks_host host;
  double *t_body, *t_gpu, *t_step;
  // optional: lat[j] = t_step of step j under spec own[j] (both or neither)
  const uint32_t *own;
  double *lat;
};

struct ValidateParams {
  const uint32_t *step, *m, *n, *k, *a, *b;
  const uint32_t *mult;                // nullable
  const uint32_t *expert_rows;
  int64_t n_expert_rows;
  int64_t n_rows;
  int64_t fam_off[KS_NFAM + 1];
  int64_t n_steps;
  const uint32_t *req_off, *req_q, *req_h;
  int64_t n_req;
  const uint64_t *agg;
  const uint32_t *tp;                  // nullable
  const ks_spec *specs;
  int32_t n_specs;
  uint32_t *err;
};

// ---- batch expansion
// m of a record template: 0, the step's tokens T, top_k T, or its requests R
enum : uint32_t { kMZero = 0, kMTok = 1, kMTopk = 2, kMReq = 3 };
struct ExpandTpl {
  uint32_t n, k, a, msrc, grouped;
};
constexpr int kExpandTpl = 4;         // templates per family and layer, at most
constexpr int kExpandBlk = 1024;      // steps per block of the prefill-rank scan

// Item space: family f (KS_ATTN_PREFILL stands for both attention families,
// KS_ATTN_DECODE has no items) owns items [item_off[f], item_off[f+1]),
// per_step[f] per step; item i of the family is step i / per_step[f] and
// slot i % per_step[f], whose template is slot % n_tpl[f] and whose layer is
// slot / n_tpl[f].  The host guarantees per_step[f] < 2^16 and fewer than
// 2^31 items per family (the quotients are then exact in floating point).
struct ExpandParams {
  const uint32_t *req_off, *req_q;
  int64_t n_req;
  const uint8_t *prefill;
  int64_t n_steps, n_prefill;
  uint32_t L, E, top_k, D, P;
  int64_t item_off[KS_NFAM + 1];
  int64_t chunk_off[KS_NFAM + 1];   // 256-item chunks of each family: one per workgroup pass
  double inv_ps[KS_NFAM];           // 1 / per_step[f], for the step index of an item
  float inv_tpl[KS_NFAM];           // 1 / n_tpl[f], for the layer of a slot
  uint32_t per_step[KS_NFAM];
  uint32_t n_tpl[KS_NFAM];
  uint32_t mult[KS_NFAM];
  ExpandTpl tpl[KS_NFAM][kExpandTpl];
  int64_t fam_off[KS_NFAM + 1];
  // workspace
  uint32_t *tok;     // [n_steps] T of each step
  uint32_t *rank;    // [n_steps] prefill steps before it within its block
  uint32_t *blk;     // [n_blk] prefill steps per block, then their exclusive prefix
  int64_t n_blk;
  uint32_t *err;
  // outputs
  uint32_t *o_step, *o_m, *o_n, *o_k, *o_a, *o_b, *o_mult;
  uint32_t *o_layers, *o_hidden, *o_tp, *o_nlaunch;
};

// the flag reset and the expansion; events recorded around the
// record-writing kernel (both null: none)
hipError_t launch_expand(const ExpandParams &p, hipStream_t s, hipEvent_t before, hipEvent_t after);

// ks_eval_steps, and in the same launches lat[j] = t_step of step j under
// spec own[j] (device arrays of n_steps; own[j] < n_specs, the caller's
// guarantee): the serving simulation's per-step latencies
ks_status eval_steps_own(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs, int32_t n_specs,
                         const ks_heads *heads, const ks_host *host, const ks_step_out *out, void *ws,
                         size_t ws_bytes, const uint32_t *own, double *lat, hipStream_t stream);

// workspace bytes of one evaluation call for a record layout (family
// offsets), step count and spec count, without the descriptor's pointers
size_t eval_workspace_bytes(const int64_t fam_off[KS_NFAM + 1], int64_t n_steps, int32_t n_specs);

// the thread-local message ks_last_error() reports; returns st
ks_status set_error(ks_status st, const char *fmt, ...);

hipError_t launch_clear(uint32_t *err, uint32_t *range, int64_t n_range, hipStream_t s);
hipError_t launch_spec_prep(const ks_spec *specs, int32_t n_specs, SpecC *out, uint32_t *err, hipStream_t s);
// launch_clear, then the spec constants of launch_spec_prep (in the same
// launch for a few specs)
hipError_t launch_clear_prep(uint32_t *err, uint32_t *range, int64_t n_range, const ks_spec *specs,
                             int32_t n_specs, SpecC *out, hipStream_t s);
hipError_t launch_attn_agg(const uint32_t *req_off, const uint32_t *q, const uint32_t *h,
                           int64_t n_steps, int64_t n_req, uint64_t *agg, uint32_t *err,
                           hipStream_t s);
hipError_t launch_eval(int kind, const EvalParams &p, hipStream_t s);
hipError_t launch_finish(const FinishParams &p, hipStream_t s);
// per-pair eta source of a call without a grid (p.o_src, families' bounded bit)
hipError_t launch_fill_source(const EvalParams &p, hipStream_t s);
hipError_t launch_validate(const ValidateParams &p, hipStream_t s);

}  // namespace ks
