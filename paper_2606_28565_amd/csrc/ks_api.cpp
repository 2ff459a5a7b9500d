// Host side of the C ABI declared in include/ks.h: argument checks, the
// workspace layout, the launch sequence and error reporting.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "ks.h"
#include "ks_internal.h"

namespace {

thread_local std::string g_err;
// measurement hook (ks_set_timing_events)
thread_local hipEvent_t g_ev_before = nullptr, g_ev_after = nullptr;

// the evaluation kernel, bracketed by the hook's events when they are set
hipError_t timed_eval(int kind, const ks::EvalParams &p, hipStream_t s) {
  const bool timed = g_ev_before && g_ev_after;
  if (timed) {
    const hipError_t e = hipEventRecord(g_ev_before, s);
    if (e != hipSuccess) return e;
  }
  hipError_t e = ks::launch_eval(kind, p, s);
  if (e != hipSuccess) return e;
  if (timed) {
    e = hipEventRecord(g_ev_after, s);
    if (e != hipSuccess) return e;
  }
  // without a grid the evaluation kernel leaves the eta source to this pass
  return p.grid_mask ? hipSuccess : ks::launch_fill_source(p, s);
}

ks_status fail(ks_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

ks_status hip_fail(hipError_t e, const char *what) {
  return fail(KS_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Workspace layout (every region 256-byte aligned):
//   header  : 256 B (uint32 flag word at offset 0)
//   specc   : n_specs * 64 B               per-spec loop constants
//   agg     : 4 * n_steps uint64           per-step attention work
//   range   : KS_NFAM * n_steps * 2 uint32 per (family, step) record range
//   partial : KS_NFAM * n_steps * n_specs double (spec-minor)
//   carry   : n_tiles * n_specs double (spec-minor)
struct Layout {
  size_t specc, agg, range, partial, carry, total;
};

struct Tiles {
  int32_t tile_off[KS_NFAM + 1];
  int32_t wgt_off[KS_NFAM + 1];
};

Tiles tiles_of(const ks_desc *d) {
  Tiles t;
  t.tile_off[0] = t.wgt_off[0] = 0;
  for (int f = 0; f < KS_NFAM; ++f) {
    const int64_t rows = d->fam_off[f + 1] - d->fam_off[f];
    const int64_t nt = (rows + ks::kTileRows - 1) / ks::kTileRows;
    t.tile_off[f + 1] = t.tile_off[f] + (int32_t)nt;
    t.wgt_off[f + 1] = t.wgt_off[f] + (int32_t)((nt + ks::kWgWaves - 1) / ks::kWgWaves);
  }
  return t;
}

Layout layout_of(const ks_desc *d, int32_t n_specs) {
  const Tiles t = tiles_of(d);
  const size_t S = (size_t)d->n_steps;
  Layout L;
  size_t off = 256;
  L.specc = off;
  off += align256((size_t)n_specs * sizeof(ks::SpecC));
  L.agg = off;
  off += align256(4 * S * sizeof(uint64_t));
  L.range = off;
  off += align256((size_t)KS_NFAM * S * 2 * sizeof(uint32_t));
  L.partial = off;
  off += align256((size_t)n_specs * KS_NFAM * S * sizeof(double));
  L.carry = off;
  off += align256((size_t)n_specs * (size_t)t.tile_off[KS_NFAM] * sizeof(double));
  L.total = off;
  return L;
}

ks_status check_desc(const ks_desc *d) {
  if (!d) return fail(KS_EINVAL, "desc is NULL");
  if (d->n_rows < 0 || d->n_rows >= (int64_t(1) << 32) - 1)
    return fail(KS_ERANGE, "n_rows %lld outside [0, 2^32-1)", (long long)d->n_rows);
  if (d->n_steps < 0 || d->n_steps >= (int64_t(1) << 32) - 1)
    return fail(KS_ERANGE, "n_steps %lld outside [0, 2^32-1)", (long long)d->n_steps);
  if (d->n_req < 0 || d->n_req >= (int64_t(1) << 32))
    return fail(KS_ERANGE, "n_req %lld outside [0, 2^32)", (long long)d->n_req);
  if (d->n_expert_rows < 0 || d->n_expert_rows >= (int64_t(1) << 32))
    return fail(KS_ERANGE, "n_expert_rows %lld outside [0, 2^32)", (long long)d->n_expert_rows);
  if (d->fam_off[0] != 0) return fail(KS_EINVAL, "fam_off[0] must be 0");
  for (int f = 0; f < KS_NFAM; ++f)
    if (d->fam_off[f + 1] < d->fam_off[f])
      return fail(KS_EINVAL, "fam_off decreases at family %d", f);
  if (d->fam_off[KS_NFAM] != d->n_rows)
    return fail(KS_EINVAL, "fam_off[KS_NFAM] = %lld != n_rows = %lld", (long long)d->fam_off[KS_NFAM],
                (long long)d->n_rows);
  if (d->n_rows > 0 && (!d->step || !d->m || !d->n || !d->k || !d->a || !d->b))
    return fail(KS_EINVAL, "a record array is NULL");
  if (d->n_rows > 0 && d->n_steps == 0) return fail(KS_EINVAL, "records present but n_steps = 0");
  if (!d->req_off) return fail(KS_EINVAL, "req_off is NULL");
  if (d->n_req > 0 && (!d->req_q || !d->req_h)) return fail(KS_EINVAL, "req_q / req_h is NULL");
  if (d->fam_off[KS_GROUPED_GEMM + 1] > d->fam_off[KS_GROUPED_GEMM] && !d->expert_rows && d->n_expert_rows > 0)
    return fail(KS_EINVAL, "expert_rows is NULL");
  if (d->elem_bytes < 1 || d->elem_bytes > 8) return fail(KS_ERANGE, "elem_bytes %u outside 1..8", d->elem_bytes);
  return KS_OK;
}

ks_status head_kind(const ks_heads *h, int *kind) {
  if (!h) return fail(KS_EINVAL, "heads is NULL");
  const uint32_t all = (1u << KS_NFAM) - 1;
  if (h->bounded_mask & ~all) return fail(KS_EINVAL, "heads.bounded_mask 0x%x has bits beyond the families",
                                          h->bounded_mask);
  if (h->bounded_mask && !h->bounded) return fail(KS_EINVAL, "heads.bounded is NULL with a nonzero mask");
  if (h->mode != KS_ETA_ONE && h->mode != KS_ETA_MLP) return fail(KS_EINVAL, "heads.mode %d unknown", h->mode);
  if (h->grid_mask & ~all) return fail(KS_EINVAL, "heads.grid_mask 0x%x has bits beyond the families", h->grid_mask);
  if (h->grid_mask) {
    if (!h->grid) return fail(KS_EINVAL, "heads.grid is NULL with a nonzero mask");
    int64_t nodes = 1;
    for (int d = 0; d < 3; ++d) {
      if (h->grid_axis[d] < 0 || h->grid_axis[d] > 14)
        return fail(KS_EINVAL, "heads.grid_axis[%d] = %d not a feature 0 .. 14", d, h->grid_axis[d]);
      if (h->grid_n[d] < 2 || h->grid_n[d] > KS_GRID_MAX_NODES)
        return fail(KS_EINVAL, "heads.grid_n[%d] = %d below 2 or above %d", d, h->grid_n[d], (int)KS_GRID_MAX_NODES);
      nodes *= h->grid_n[d];
      const double lo = h->grid_lo[d], hi = h->grid_hi[d];
      const float scale = (float)((h->grid_n[d] - 1) / (hi - lo));
      if (!std::isfinite((float)lo) || !std::isfinite((float)hi) || !(lo < hi) || !std::isfinite(scale))
        return fail(KS_EINVAL, "heads.grid_lo/hi[%d] = %g, %g not finite with lo < hi", d, lo, hi);
    }
    if (nodes > KS_GRID_MAX_NODES)
      return fail(KS_EINVAL, "heads grid of %lld nodes above %d", (long long)nodes, (int)KS_GRID_MAX_NODES);
  }
  // no family left for the MLP: the head-less kernel (bounded and grid
  // families, eta = 1 for the rest)
  if (h->mode == KS_ETA_ONE || h->bounded_mask == all) {
    *kind = (h->bounded_mask | h->grid_mask) ? ks::kBoundedOnly : ks::kEtaOne;
    return KS_OK;
  }
  if (!h->w1 || !h->w2 || !h->b2 || !h->w3 || !h->b3) return fail(KS_EINVAL, "a head parameter pointer is NULL");
  const int in = h->in_dim, hid = h->hidden;
  if (in != 16 && in != 32) return fail(KS_EINVAL, "heads.in_dim %d not 16 or 32", in);
  if (h->precision == KS_F32) {
    if (hid == 64) *kind = in == 16 ? ks::kF32_16_64 : ks::kF32_32_64;
    else if (hid == 128) *kind = in == 16 ? ks::kF32_16_128 : ks::kF32_32_128;
    else return fail(KS_EINVAL, "fp32 heads.hidden %d not 64 or 128", hid);
  } else if (h->precision == KS_BF16) {
    if (hid == 64) *kind = in == 16 ? ks::kBF16_16_64 : ks::kBF16_32_64;
    else if (hid == 128) *kind = in == 16 ? ks::kBF16_16_128 : ks::kBF16_32_128;
    else if (hid == 256) *kind = in == 16 ? ks::kBF16_16_256 : ks::kBF16_32_256;
    else return fail(KS_EINVAL, "bf16 heads.hidden %d not 64, 128 or 256", hid);
  } else {
    return fail(KS_EINVAL, "heads.precision %d unknown", h->precision);
  }
  return KS_OK;
}

ks_status check_common(const ks_desc *d, const ks_spec *specs, int32_t n_specs, void *ws, size_t ws_bytes,
                       Layout *L) {
  ks_status st = check_desc(d);
  if (st != KS_OK) return st;
  if (n_specs < 1 || n_specs > (1 << 20)) return fail(KS_EINVAL, "n_specs %d outside 1..2^20", n_specs);
  if (!specs) return fail(KS_EINVAL, "specs is NULL");
  *L = layout_of(d, n_specs);
  if (!ws) return fail(KS_EWORKSPACE, "workspace is NULL");
  if (ws_bytes < L->total)
    return fail(KS_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, L->total);
  if (reinterpret_cast<uintptr_t>(ws) % 256)
    return fail(KS_EWORKSPACE, "workspace not 256-byte aligned");
  return KS_OK;
}

void fill_eval(ks::EvalParams &p, const ks_desc *d, const ks_spec *specs, int32_t n_specs, const ks_heads *h,
               const ks_kernel_out *out, char *ws, const Layout &L) {
  std::memset(&p, 0, sizeof p);
  p.step = d->step;
  p.m = d->m;
  p.n = d->n;
  p.k = d->k;
  p.a = d->a;
  p.b = d->b;
  p.expert_rows = d->expert_rows;
  p.n_expert_rows = d->expert_rows ? d->n_expert_rows : 0;
  p.mult = d->n_rows > 0 ? d->mult : nullptr;
  p.agg = reinterpret_cast<const uint64_t *>(ws + L.agg);
  p.n_steps = d->n_steps;
  p.elem_bytes = d->elem_bytes;
  p.n_specs = n_specs;
  p.spec_c = reinterpret_cast<const ks::SpecC *>(ws + L.specc);
  const Tiles t = tiles_of(d);
  for (int f = 0; f <= KS_NFAM; ++f) {
    p.fam_off[f] = d->fam_off[f];
    p.tile_off[f] = t.tile_off[f];
    p.wgt_off[f] = t.wgt_off[f];
  }
  p.n_tiles = t.tile_off[KS_NFAM];
  p.spec_chunk = n_specs;
  p.n_chunks = 1;
  p.bounded_mask = h->bounded_mask;
  p.bounded = h->bounded_mask ? h->bounded : nullptr;
  p.grid_mask = h->grid_mask;
  p.grid = h->grid_mask ? h->grid : nullptr;
  p.grid_nodes = 0;
  for (int a = 0; a < 3; ++a) {
    p.grid_axis[a] = h->grid_mask ? h->grid_axis[a] : 0;
    p.grid_n[a] = h->grid_mask ? h->grid_n[a] : 2;
    p.grid_lo[a] = h->grid_mask ? (float)h->grid_lo[a] : 0.0f;
    p.grid_scale[a] = h->grid_mask ? (float)((h->grid_n[a] - 1) / (h->grid_hi[a] - h->grid_lo[a])) : 0.0f;
  }
  if (h->grid_mask) p.grid_nodes = p.grid_n[0] * p.grid_n[1] * p.grid_n[2];
  if (h->mode == KS_ETA_MLP) {
    p.w1 = h->w1;
    p.w2 = h->w2;
    p.b2 = h->b2;
    p.w3 = h->w3;
    p.b3 = h->b3;
  }
  if (out) {
    p.o_flops = out->flops;
    p.o_bytes = out->bytes;
    p.o_blocks = out->blocks;
    p.o_troof = out->t_roof;
    p.o_eta = out->eta;
    p.o_t = out->t_kernel;
    p.o_src = out->source;
  }
  p.err = reinterpret_cast<uint32_t *>(ws);
}

ks_status prologue(const ks_desc *d, const ks_spec *specs, int32_t n_specs, char *ws, const Layout &L,
                   bool with_range, hipStream_t s) {
  hipError_t e = ks::launch_clear_prep(reinterpret_cast<uint32_t *>(ws), reinterpret_cast<uint32_t *>(ws + L.range),
                                       with_range ? 2 * (int64_t)KS_NFAM * d->n_steps : 0, specs, n_specs,
                                       reinterpret_cast<ks::SpecC *>(ws + L.specc), s);
  if (e != hipSuccess) return hip_fail(e, "clear and spec constants launch");
  e = ks::launch_attn_agg(d->req_off, d->req_q, d->req_h, d->n_steps, d->n_req,
                          reinterpret_cast<uint64_t *>(ws + L.agg), reinterpret_cast<uint32_t *>(ws), s);
  if (e != hipSuccess) return hip_fail(e, "attention aggregate launch");
  return KS_OK;
}

// ---- batch expansion: the per-family record templates of a model (the
// per-layer kernel list in dispatch order, and the per-step embedding and
// LM head), the item space and the record counts
struct Plan {
  uint32_t n_tpl[KS_NFAM];          // templates per layer (or per step)
  ks::ExpandTpl tpl[KS_NFAM][ks::kExpandTpl];
  bool per_layer[KS_NFAM];          // dispatched once per layer (else once per step)
  uint32_t per_step[KS_NFAM], mult[KS_NFAM];
  int64_t count[KS_NFAM];
};

ks_status model_plan(const ks_model *md, int64_t n_steps, int64_t n_prefill, int32_t mode, Plan *pl) {
  if (!md) return fail(KS_EINVAL, "model is NULL");
  if (mode != KS_EXPAND_PER_LAYER && mode != KS_EXPAND_HOMOGENEOUS) return fail(KS_EINVAL, "mode %d unknown", mode);
  if (n_steps < 0 || n_steps >= (int64_t(1) << 32) - 1)
    return fail(KS_ERANGE, "n_steps %lld outside [0, 2^32-1)", (long long)n_steps);
  if (n_prefill < 0 || n_prefill > n_steps)
    return fail(KS_EINVAL, "n_prefill %lld outside [0, n_steps]", (long long)n_prefill);
  const uint32_t P = md->tp;
  if (md->layers < 1 || md->hidden < 1 || md->head_dim < 1 || md->kv_heads < 1 || P < 1)
    return fail(KS_EINVAL, "model: layers, hidden, head_dim, kv_heads and tp must be >= 1");
  if (md->q_heads < P || md->q_heads % P) return fail(KS_EINVAL, "model: q_heads %u not a positive multiple of tp %u",
                                                      md->q_heads, P);
  if (md->vocab % P) return fail(KS_EINVAL, "model: vocab %u not divisible by tp %u", md->vocab, P);
  if (md->kv_write > 1) return fail(KS_EINVAL, "model: kv_write %u not 0 or 1", md->kv_write);
  const bool moe = md->experts > 0;
  if (moe) {
    if (md->experts > 1024) return fail(KS_ERANGE, "model: experts %u above 1024", md->experts);
    if (md->top_k < 1 || md->top_k > md->experts)
      return fail(KS_EINVAL, "model: top_k %u outside 1 .. experts", md->top_k);
    if (md->expert_ffn % P) return fail(KS_EINVAL, "model: expert_ffn %u not divisible by tp %u", md->expert_ffn, P);
  } else if (md->ffn % P) {
    return fail(KS_EINVAL, "model: ffn %u not divisible by tp %u", md->ffn, P);
  }
  const uint64_t D = md->hidden, L = md->layers, d = md->head_dim;
  const uint64_t H = md->q_heads / P, Hkv = (md->kv_heads + P - 1) / P;
  const uint64_t I = moe ? 0 : md->ffn / P, Ie = moe ? md->expert_ffn / P : 0, V = md->vocab / P;
  const uint64_t E = md->experts;
  if (H >= 4096 || d >= 4096 || Hkv >= 4096) return fail(KS_ERANGE, "model: attention H, d or Hkv at or above 2^12");
  std::memset(pl, 0, sizeof *pl);
  auto add = [&](int f, uint32_t msrc, uint64_t n, uint64_t k, uint64_t a, bool grouped) {
    pl->tpl[f][pl->n_tpl[f]++] = ks::ExpandTpl{(uint32_t)n, (uint32_t)k, (uint32_t)a, msrc, grouped ? 1u : 0u};
    return n < (1u << 18) && k < (1u << 18);
  };
  bool ok = true;
  // per layer, dispatch order within each family
  ok &= add(KS_GEMM, ks::kMTok, (H + 2 * Hkv) * d, D, 0, false);   // QKV projection
  ok &= add(KS_ROPE, ks::kMTok, H + Hkv, d, 0, false);
  if (md->kv_write) ok &= add(KS_KV_WRITE, ks::kMTok, Hkv, d, 0, false);
  ok &= add(KS_ATTN_PREFILL, ks::kMZero, H, d, Hkv, false);        // either attention family
  ok &= add(KS_GEMM, ks::kMTok, D, H * d, 0, false);                // O projection
  ok &= add(KS_RMSNORM, ks::kMTok, D, 0, 0, false);
  ok &= add(KS_RMSNORM, ks::kMTok, D, 0, 0, false);
  if (!moe) {
    ok &= add(KS_GEMM, ks::kMTok, 2 * I, D, 0, false);              // gate/up
    ok &= add(KS_SILU_MUL, ks::kMTok, I, 0, 0, false);
    ok &= add(KS_GEMM, ks::kMTok, D, I, 0, false);                  // down
  } else {
    ok &= add(KS_GEMM, ks::kMTok, E, D, 0, false);                  // router
    ok &= add(KS_GROUPED_GEMM, ks::kMZero, 2 * Ie, D, E, true);     // gate/up
    ok &= add(KS_SILU_MUL, ks::kMTopk, Ie, 0, 0, false);
    ok &= add(KS_GROUPED_GEMM, ks::kMZero, D, Ie, E, true);         // down
  }
  for (int f = 0; f < KS_NFAM; ++f) pl->per_layer[f] = pl->n_tpl[f] > 0;
  // per step
  ok &= add(KS_EMBED, ks::kMTok, D, 0, 0, false);
  ok &= add(KS_LM_HEAD, ks::kMReq, V, D, 0, false);
  if (!ok) return fail(KS_ERANGE, "model: a record's n or k at or above 2^18");
  int64_t total = 0, items = 0;
  for (int f = 0; f < KS_NFAM; ++f) {
    const bool collapse = mode == KS_EXPAND_HOMOGENEOUS && f != KS_GROUPED_GEMM;
    const uint64_t reps = pl->per_layer[f] && !collapse ? L : 1;
    pl->per_step[f] = (uint32_t)(reps * pl->n_tpl[f]);
    pl->mult[f] = pl->per_layer[f] && collapse ? (uint32_t)L : 1u;
    const int64_t steps = f == KS_ATTN_PREFILL ? n_prefill : (f == KS_ATTN_DECODE ? n_steps - n_prefill : n_steps);
    const int64_t per = f == KS_ATTN_DECODE ? pl->per_step[KS_ATTN_PREFILL] : pl->per_step[f];
    if (per > 0 && steps > ((int64_t(1) << 40) / per)) return fail(KS_ERANGE, "expansion beyond 2^32 records");
    pl->count[f] = per * steps;
    total += pl->count[f];
    items += (int64_t)pl->per_step[f] * n_steps;
  }
  if (total >= (int64_t(1) << 32) - 1 || items >= (int64_t(1) << 32))
    return fail(KS_ERANGE, "expansion of %lld records at or above 2^32 - 1", (long long)total);
  if (moe && (uint64_t)n_steps * L * E >= (uint64_t(1) << 32))
    return fail(KS_ERANGE, "routed-row offsets n_steps L E at or above 2^32");
  if (pl->mult[KS_GEMM] >= (1u << 24)) return fail(KS_ERANGE, "layers at or above 2^24");
  return KS_OK;
}

struct ExpandLayout {
  size_t tok, rank, blk, total;
  int64_t n_blk;
};

ExpandLayout expand_layout_of(int64_t n_steps) {
  ExpandLayout L;
  const size_t S = (size_t)(n_steps < 0 ? 0 : n_steps);
  L.n_blk = (int64_t)((S + ks::kExpandBlk - 1) / ks::kExpandBlk);
  size_t off = 256;
  L.tok = off;
  off += align256(S * sizeof(uint32_t));
  L.rank = off;
  off += align256(S * sizeof(uint32_t));
  L.blk = off;
  off += align256((size_t)L.n_blk * sizeof(uint32_t));
  L.total = off;
  return L;
}

const char *flag_text(uint32_t f) {
  if (f & ks::kErrStep) return "a record's step index is >= n_steps";
  if (f & ks::kErrOrder) return "record steps decrease within a family";
  if (f & ks::kErrReq) return "request offsets out of order or beyond n_req";
  if (f & ks::kErrExpert) return "grouped-GEMM expert offsets beyond n_expert_rows (or E > 1024)";
  if (f & ks::kErrRange) return "a shape or count outside the documented limits";
  if (f & ks::kErrSpec) return "a spec vector is not usable (non-positive peak, bandwidth or n_cu)";
  if (f & ks::kErrPrefill) return "the batch's prefill flags disagree with n_prefill";
  return "unknown";
}

ks_status flag_status(uint32_t f) {
  if (!f) return KS_OK;
  const bool range = (f & (ks::kErrRange | ks::kErrSpec)) &&
                     !(f & (ks::kErrStep | ks::kErrOrder | ks::kErrReq | ks::kErrExpert | ks::kErrPrefill));
  return fail(range ? KS_ERANGE : KS_EINVAL, "device check: %s (flags 0x%x)", flag_text(f), f);
}

}  // namespace

size_t ks::eval_workspace_bytes(const int64_t fam_off[KS_NFAM + 1], int64_t n_steps, int32_t n_specs) {
  ks_desc d;
  std::memset(&d, 0, sizeof d);
  for (int f = 0; f <= KS_NFAM; ++f) d.fam_off[f] = fam_off[f];
  d.n_rows = fam_off[KS_NFAM];
  d.n_steps = n_steps;
  return layout_of(&d, n_specs).total;
}

ks_status ks::set_error(ks_status st, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

extern "C" {

size_t ks_workspace_bytes(const ks_desc *desc, int32_t n_specs) {
  if (check_desc(desc) != KS_OK || n_specs < 1 || n_specs > (1 << 20)) return 0;
  return layout_of(desc, n_specs).total;
}

ks_status ks_eval_kernels(const ks_desc *desc, const ks_spec *specs, int32_t n_specs, const ks_heads *heads,
                          const ks_kernel_out *out, void *ws, size_t ws_bytes, hipStream_t stream) {
  Layout L;
  ks_status st = check_common(desc, specs, n_specs, ws, ws_bytes, &L);
  if (st != KS_OK) return st;
  int kind;
  st = head_kind(heads, &kind);
  if (st != KS_OK) return st;
  if (!out) return fail(KS_EINVAL, "out is NULL");
  char *w = static_cast<char *>(ws);
  st = prologue(desc, specs, n_specs, w, L, false, stream);
  if (st != KS_OK) return st;
  ks::EvalParams p;
  fill_eval(p, desc, specs, n_specs, heads, out, w, L);
  hipError_t e = timed_eval(kind, p, stream);
  if (e != hipSuccess) return hip_fail(e, "evaluation launch");
  return KS_OK;
}

static ks_status eval_steps_impl(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs,
                                 int32_t n_specs, const ks_heads *heads, const ks_host *host,
                                 const ks_step_out *out, const ks_kernel_out *kout, void *ws, size_t ws_bytes,
                                 const uint32_t *own, double *lat, hipStream_t stream) {
  Layout L;
  ks_status st = check_common(desc, specs, n_specs, ws, ws_bytes, &L);
  if (st != KS_OK) return st;
  int kind;
  st = head_kind(heads, &kind);
  if (st != KS_OK) return st;
  if (!steps) return fail(KS_EINVAL, "steps is NULL");
  if (steps->n_steps != desc->n_steps)
    return fail(KS_EINVAL, "steps.n_steps %lld != desc.n_steps %lld", (long long)steps->n_steps,
                (long long)desc->n_steps);
  if (desc->n_steps > 0 && (!steps->layers || !steps->hidden || !steps->tp || !steps->n_launch))
    return fail(KS_EINVAL, "a step array is NULL");
  if (!host) return fail(KS_EINVAL, "host is NULL");
  if (!out || (desc->n_steps > 0 && (!out->t_body || !out->t_gpu || !out->t_step)))
    return fail(KS_EINVAL, "a step output is NULL");
  char *w = static_cast<char *>(ws);
  st = prologue(desc, specs, n_specs, w, L, true, stream);
  if (st != KS_OK) return st;
  ks::EvalParams p;
  fill_eval(p, desc, specs, n_specs, heads, kout, w, L);
  p.partial = reinterpret_cast<double *>(w + L.partial);
  p.carry = reinterpret_cast<double *>(w + L.carry);
  p.range = reinterpret_cast<uint32_t *>(w + L.range);
  hipError_t e = timed_eval(kind, p, stream);
  if (e != hipSuccess) return hip_fail(e, "evaluation launch");

  ks::FinishParams f;
  std::memset(&f, 0, sizeof f);
  f.agg = p.agg;
  f.layers = steps->layers;
  f.hidden = steps->hidden;
  f.tp = steps->tp;
  f.n_launch = steps->n_launch;
  f.n_steps = desc->n_steps;
  f.n_specs = n_specs;
  f.elem_bytes = desc->elem_bytes;
  f.specs = specs;
  for (int i = 0; i <= KS_NFAM; ++i) {
    f.fam_off[i] = p.fam_off[i];
    f.tile_off[i] = p.tile_off[i];
  }
  f.partial = p.partial;
  f.carry = p.carry;
  f.n_tiles = p.n_tiles;
  f.range = p.range;
  f.host = *host;
  f.t_body = out->t_body;
  f.t_gpu = out->t_gpu;
  f.t_step = out->t_step;
  f.own = own;
  f.lat = lat;
  e = ks::launch_finish(f, stream);
  if (e != hipSuccess) return hip_fail(e, "step finish launch");
  return KS_OK;
}

ks_status ks_eval_steps(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs, int32_t n_specs,
                        const ks_heads *heads, const ks_host *host, const ks_step_out *out,
                        const ks_kernel_out *kout, void *ws, size_t ws_bytes, hipStream_t stream) {
  return eval_steps_impl(desc, steps, specs, n_specs, heads, host, out, kout, ws, ws_bytes, nullptr, nullptr,
                         stream);
}

ks_status ks_validate(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs, int32_t n_specs, void *ws,
                      size_t ws_bytes, hipStream_t stream) {
  Layout L;
  ks_status st = check_common(desc, specs, n_specs, ws, ws_bytes, &L);
  if (st != KS_OK) return st;
  if (steps && steps->n_steps != desc->n_steps)
    return fail(KS_EINVAL, "steps.n_steps %lld != desc.n_steps %lld", (long long)steps->n_steps,
                (long long)desc->n_steps);
  char *w = static_cast<char *>(ws);
  st = prologue(desc, specs, n_specs, w, L, false, stream);
  if (st != KS_OK) return st;
  ks::ValidateParams v;
  std::memset(&v, 0, sizeof v);
  v.step = desc->step;
  v.m = desc->m;
  v.n = desc->n;
  v.k = desc->k;
  v.a = desc->a;
  v.b = desc->b;
  v.mult = desc->mult;
  v.expert_rows = desc->expert_rows;
  v.n_expert_rows = desc->expert_rows ? desc->n_expert_rows : 0;
  v.n_rows = desc->n_rows;
  for (int f = 0; f <= KS_NFAM; ++f) v.fam_off[f] = desc->fam_off[f];
  v.n_steps = desc->n_steps;
  v.req_off = desc->req_off;
  v.req_q = desc->req_q;
  v.req_h = desc->req_h;
  v.n_req = desc->n_req;
  v.agg = reinterpret_cast<const uint64_t *>(w + L.agg);
  v.tp = steps ? steps->tp : nullptr;
  v.specs = specs;
  v.n_specs = n_specs;
  v.err = reinterpret_cast<uint32_t *>(w);
  hipError_t e = ks::launch_validate(v, stream);
  if (e != hipSuccess) return hip_fail(e, "validate launch");
  return ks_device_status(ws, ws_bytes, stream);
}

ks_status ks_device_status(const void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!ws || ws_bytes < 256) return fail(KS_EWORKSPACE, "workspace missing or too small");
  uint32_t flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, ws, sizeof flag, hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return hip_fail(e, "flag copy");
  e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "stream synchronize");
  return flag_status(flag);
}

ks_status ks_expand_layout(const ks_model *model, int64_t n_steps, int64_t n_prefill, int32_t mode,
                           int64_t fam_off[KS_NFAM + 1]) {
  if (!fam_off) return fail(KS_EINVAL, "fam_off is NULL");
  Plan pl;
  const ks_status st = model_plan(model, n_steps, n_prefill, mode, &pl);
  if (st != KS_OK) return st;
  fam_off[0] = 0;
  for (int f = 0; f < KS_NFAM; ++f) fam_off[f + 1] = fam_off[f] + pl.count[f];
  return KS_OK;
}

size_t ks_expand_workspace_bytes(int64_t n_steps) {
  if (n_steps < 0 || n_steps >= (int64_t(1) << 32) - 1) return 0;
  return expand_layout_of(n_steps).total;
}

ks_status ks_expand(const ks_model *model, const ks_batch *batch, int32_t mode, const ks_records *out, void *ws,
                    size_t ws_bytes, hipStream_t stream) {
  if (!batch) return fail(KS_EINVAL, "batch is NULL");
  Plan pl;
  ks_status st = model_plan(model, batch->n_steps, batch->n_prefill, mode, &pl);
  if (st != KS_OK) return st;
  const int64_t S = batch->n_steps;
  if (batch->n_req < 0 || batch->n_req >= (int64_t(1) << 32))
    return fail(KS_ERANGE, "n_req %lld outside [0, 2^32)", (long long)batch->n_req);
  if (!batch->req_off) return fail(KS_EINVAL, "batch.req_off is NULL");
  if (batch->n_req > 0 && !batch->req_q) return fail(KS_EINVAL, "batch.req_q is NULL");
  if (S > 0 && !batch->prefill) return fail(KS_EINVAL, "batch.prefill is NULL");
  if (!out) return fail(KS_EINVAL, "out is NULL");
  int64_t total = 0;
  for (int f = 0; f < KS_NFAM; ++f) total += pl.count[f];
  if (total > 0 && (!out->step || !out->m || !out->n || !out->k || !out->a || !out->b))
    return fail(KS_EINVAL, "a record output array is NULL");
  if (mode == KS_EXPAND_HOMOGENEOUS && total > 0 && !out->mult)
    return fail(KS_EINVAL, "out.mult is NULL in the homogeneous mode");
  if (S > 0 && (!out->layers || !out->hidden || !out->tp || !out->n_launch))
    return fail(KS_EINVAL, "a per-step output array is NULL");
  const ExpandLayout L = expand_layout_of(S);
  if (!ws) return fail(KS_EWORKSPACE, "workspace is NULL");
  if (ws_bytes < L.total) return fail(KS_EWORKSPACE, "workspace %zu bytes < %zu required", ws_bytes, L.total);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return fail(KS_EWORKSPACE, "workspace not 256-byte aligned");
  char *w = static_cast<char *>(ws);

  ks::ExpandParams p;
  std::memset(&p, 0, sizeof p);
  p.req_off = batch->req_off;
  p.req_q = batch->req_q;
  p.n_req = batch->n_req;
  p.prefill = batch->prefill;
  p.n_steps = S;
  p.n_prefill = batch->n_prefill;
  p.L = model->layers;
  p.E = model->experts;
  p.top_k = model->experts ? model->top_k : 0;
  p.D = model->hidden;
  p.P = model->tp;
  p.item_off[0] = 0;
  p.fam_off[0] = 0;
  for (int f = 0; f < KS_NFAM; ++f) {
    // the attention items of every step live under ATTN_PREFILL
    p.per_step[f] = f == KS_ATTN_DECODE ? 0 : pl.per_step[f];
    p.n_tpl[f] = pl.n_tpl[f] ? pl.n_tpl[f] : 1;
    p.mult[f] = pl.mult[f];
    for (int t = 0; t < ks::kExpandTpl; ++t) p.tpl[f][t] = pl.tpl[f][t];
    p.item_off[f + 1] = p.item_off[f] + (int64_t)p.per_step[f] * S;
    p.fam_off[f + 1] = p.fam_off[f] + pl.count[f];
    if (p.per_step[f] >= (1u << 16) || p.item_off[f + 1] - p.item_off[f] >= (int64_t(1) << 31))
      return fail(KS_ERANGE, "family %d: %u records per step or %lld items beyond the expansion's limits", f,
                  p.per_step[f], (long long)(p.item_off[f + 1] - p.item_off[f]));
    p.inv_ps[f] = p.per_step[f] ? 1.0 / (double)p.per_step[f] : 0.0;
    p.inv_tpl[f] = 1.0f / (float)p.n_tpl[f];
  }
  p.chunk_off[0] = 0;
  for (int f = 0; f < KS_NFAM; ++f)
    p.chunk_off[f + 1] = p.chunk_off[f] + (p.item_off[f + 1] - p.item_off[f] + 255) / 256;
  p.tok = reinterpret_cast<uint32_t *>(w + L.tok);
  p.rank = reinterpret_cast<uint32_t *>(w + L.rank);
  p.blk = reinterpret_cast<uint32_t *>(w + L.blk);
  p.n_blk = L.n_blk;
  p.err = reinterpret_cast<uint32_t *>(w);
  p.o_step = out->step;
  p.o_m = out->m;
  p.o_n = out->n;
  p.o_k = out->k;
  p.o_a = out->a;
  p.o_b = out->b;
  p.o_mult = out->mult;
  p.o_layers = out->layers;
  p.o_hidden = out->hidden;
  p.o_tp = out->tp;
  p.o_nlaunch = out->n_launch;
  hipError_t e = ks::launch_expand(p, stream, g_ev_before, g_ev_after);
  if (e != hipSuccess) return hip_fail(e, "expansion launch");
  return KS_OK;
}

ks_status ks_set_timing_events(hipEvent_t before, hipEvent_t after) {
  if ((before == nullptr) != (after == nullptr)) return fail(KS_EINVAL, "set both timing events or neither");
  g_ev_before = before;
  g_ev_after = after;
  return KS_OK;
}

const char *ks_last_error(void) { return g_err.c_str(); }

const char *ks_version(void) { return "ks 0.1.0 (gfx950)"; }

}  // extern "C"

ks_status ks::eval_steps_own(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs, int32_t n_specs,
                             const ks_heads *heads, const ks_host *host, const ks_step_out *out, void *ws,
                             size_t ws_bytes, const uint32_t *own, double *lat, hipStream_t stream) {
  if (!own || !lat) return fail(KS_EINVAL, "own or lat is NULL");
  return eval_steps_impl(desc, steps, specs, n_specs, heads, host, out, nullptr, ws, ws_bytes, own, lat, stream);
}
