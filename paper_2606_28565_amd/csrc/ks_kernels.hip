// HIP kernels of the batched kernel-latency evaluator, written for gfx950
// (CDNA4: wave64, MFMA, 160 KB LDS per CU).
//
// Data flow of one evaluation (all on the caller's stream):
//   k_clear      reset the workspace's bad-data flag and step-range table,
//                then form the per-spec constants (k_spec_prep instead for
//                more than 1024 specs)
//   k_attn_agg   per step: Q, KV, PAIRS, TILES of its request list (Sec. 5.8)
//   k_eval<K>    per wave: 64 records of one family x every spec vector:
//                exact counts (Eq. 1-2 operands), waves and u (Sec. 2.2),
//                t_roof (Eq. 2), features and the family's efficiency head
//                on MFMA (Sec. 5.3), t = max(t_roof eta, t0) (Eq. 2), a
//                wavefront segmented sum of t by step, and each (family,
//                step) record range
//   k_stream     instead of k_eval for every call with no MLP family and
//                no measured grid (eta = 1, the bounded head): the same per
//                256 records and wave, four consecutive records per lane
//   k_finish     per (spec, step): body sum, all-reduce (Eq. 3), assembly (Eq. 4)
#include <hip/hip_runtime.h>

#include <atomic>
#include <utility>

#include "ks_internal.h"

namespace ks {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kNoKey = 0xFFFFFFFFu;

// ------------------------------------------------------------------ helpers
__device__ __forceinline__ float rcpf(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ __forceinline__ float log2f_fast(float x) { return __builtin_amdgcn_logf(x); }

// ceil(x / d) for x + d < 2^52, through a float64 reciprocal and one
// correction step each way (the product's error is below one unit there).
__device__ __forceinline__ uint64_t ceil_div(uint64_t x, uint32_t d, double rcp_d) {
  const uint64_t y = x + d - 1;
  uint64_t q = (uint64_t)((double)y * rcp_d);
  if (q * d > y) q -= 1;
  else if ((q + 1) * d <= y) q += 1;
  return q;
}

// two floats -> packed bfloat16 pair, round to nearest even
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// relu on an fp32 value through its bits: a negative float is a negative
// int32 (one integer max, no canonicalization of the input)
__device__ __forceinline__ float relu_f(float x) {
  return __builtin_bit_cast(float, max(__builtin_bit_cast(int, x), 0));
}

// relu on a packed bfloat16 pair: a negative bf16 is a negative int16
__device__ __forceinline__ uint32_t relu_bf16x2(uint32_t v) {
  s16x2 s = __builtin_bit_cast(s16x2, v);
  s16x2 z = {0, 0};
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(s, z));
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// Exchange lanes 32..63 of `lo` with lanes 0..31 of `hi`.
__device__ __forceinline__ void swap32(uint32_t &lo, uint32_t &hi) {
  auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
  lo = r[0];
  hi = r[1];
}

// ------------------------------------------------------------ clear / agg
// Reset the flag word and, when step sums are wanted, the per-(family,
// step) range table (an empty range marks a family without that step).
__device__ void spec_prep_one(const ks_spec *__restrict__ specs, int s, SpecC *__restrict__ out, uint32_t *err);

// With specs (n_specs > 0), the first workgroup also forms their constants
// once the flag word is reset (a bad spec then flags the fresh word).
__global__ void k_clear(uint32_t *err, uint32_t *range, int64_t n_range, const ks_spec *specs, int32_t n_specs,
                        SpecC *specc) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (blockIdx.x == 0) {
    if (threadIdx.x == 0) err[0] = 0;
    if (n_specs > 0) {
      __syncthreads();
      for (int s = threadIdx.x; s < n_specs; s += blockDim.x) spec_prep_one(specs, s, specc, err);
    }
  }
  for (int64_t i = i0; i < n_range; i += (int64_t)gridDim.x * blockDim.x) range[i] = 0;
}

// Per step j: over its requests r, Q = sum q, KV = sum (h + q),
// PAIRS = sum (q h + q (q + 1) / 2), TILES = sum ceil(q / 128).  A group of
// 16 lanes per step strides over its requests, then a butterfly reduction
// within the group.
constexpr int kAggLanes = 16;

__global__ void k_attn_agg(const uint32_t *__restrict__ req_off, const uint32_t *__restrict__ rq,
                           const uint32_t *__restrict__ rh, int64_t n_steps, int64_t n_req,
                           uint64_t *__restrict__ agg, uint32_t *err) {
  const int sub = threadIdx.x & (kAggLanes - 1);
  const int64_t groups = ((int64_t)gridDim.x * blockDim.x) / kAggLanes;
  for (int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kAggLanes; j < n_steps; j += groups) {
    uint32_t r0 = req_off[j], r1 = req_off[j + 1];
    if (r0 > r1 || (int64_t)r1 > n_req) {
      if (sub == 0) atomicOr(err, kErrReq);
      r0 = r1 = 0;
    }
    uint64_t Q = 0, KV = 0, P = 0, T = 0;
    for (uint32_t r = r0 + sub; r < r1; r += kAggLanes) {
      const uint64_t q = rq[r], h = rh[r];
      Q += q;
      KV += h + q;
      P += q * h + ((q * (q + 1)) >> 1);
      T += (q + 127) >> 7;
    }
#pragma unroll
    for (int off = kAggLanes / 2; off > 0; off >>= 1) {
      Q += __shfl_xor(Q, off);
      KV += __shfl_xor(KV, off);
      P += __shfl_xor(P, off);
      T += __shfl_xor(T, off);
    }
    if (sub == 0) {
      agg[j] = Q;
      agg[n_steps + j] = KV;
      agg[2 * n_steps + j] = P;
      agg[3 * n_steps + j] = T;
    }
  }
}

// ------------------------------------------------------------ record counts
struct Cnt {
  uint64_t F, Bt, B, M;
};

// Expert row counts a0 .. a0 + n - 1 of a grouped GEMM (in bounds: the
// caller checks), eight loads issued before any is used, so a record's
// experts cost one memory round trip per eight instead of one each: their
// sum, the experts with rows, and the 128-row tiles, accumulated in T.
template <typename T>
__device__ __forceinline__ void expert_sums(const uint32_t *rows, uint32_t a0, uint32_t n, T &ms, T &act,
                                            T &tiles) {
  ms = act = tiles = 0;
  for (uint32_t e0 = 0; e0 < n; e0 += 8) {
    uint32_t me[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) me[u] = e0 + u < n ? rows[a0 + e0 + u] : 0u;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      ms += (T)me[u];
      act += me[u] > 0 ? 1 : 0;
      tiles += ((T)me[u] + 127) >> 7;
    }
  }
}

// FLOPs F, bytes Bt, thread blocks B and feature row count M of one record.
__device__ __forceinline__ Cnt record_counts(int fam, uint32_t m32, uint32_t n32, uint32_t k32,
                                             uint32_t a32, uint32_t b32, uint32_t step,
                                             const EvalParams &p, uint32_t &bad) {
  const uint64_t dt = p.elem_bytes, M = m32, N = n32, K = k32, A = a32;
  Cnt c{0, 0, 0, M};
  switch (fam) {
    case KS_GEMM:
    case KS_LM_HEAD:
      c.F = 2 * M * N * K;
      c.Bt = dt * (M * K + K * N + M * N);
      c.B = ((M + 127) >> 7) * ((N + 127) >> 7);
      break;
    case KS_GROUPED_GEMM: {
      uint64_t ms = 0, act = 0, tiles = 0;
      if ((uint64_t)b32 + A <= (uint64_t)p.n_expert_rows && A <= 1024) {
        expert_sums(p.expert_rows, b32, a32, ms, act, tiles);
      } else {
        bad |= kErrExpert;
      }
      c.F = 2 * ms * N * K;
      c.Bt = dt * (ms * K + act * K * N + ms * N);
      c.B = tiles * ((N + 127) >> 7);
      c.M = ms;
      break;
    }
    case KS_ATTN_PREFILL:
    case KS_ATTN_DECODE: {
      uint64_t Q = 0, KV = 0, P = 0, T = 0;
      if ((int64_t)step < p.n_steps) {
        Q = p.agg[step];
        KV = p.agg[p.n_steps + step];
        P = p.agg[2 * p.n_steps + step];
        T = p.agg[3 * p.n_steps + step];
      }
      c.F = 4 * N * K * P;
      c.Bt = dt * (2 * N * K * Q + 2 * A * K * KV);
      c.B = N * T;
      c.M = Q;
      break;
    }
    case KS_RMSNORM:
      c.F = 4 * M * N;
      c.Bt = dt * (2 * M * N + N);
      c.B = M;
      break;
    case KS_ROPE:
      c.F = 3 * M * N * K;
      c.Bt = dt * (2 * M * N * K + M * K);
      c.B = M;
      break;
    case KS_SILU_MUL:
      c.F = 5 * M * N;
      c.Bt = 3 * dt * M * N;
      c.B = (M * N + 1023) >> 10;
      break;
    case KS_KV_WRITE:
      c.F = 0;
      c.Bt = 4 * dt * M * N * K;
      c.B = M;
      break;
    default:  // KS_EMBED
      c.F = 0;
      c.Bt = 2 * dt * M * N + 4 * M;
      c.B = M;
      break;
  }
  return c;
}

// The same counts with F and Bt rounded to fp32 as they are formed (each a
// few roundings, within 1e-6 relative of the exact values) and B exact.
// The eta = 1 stream uses it when no per-record count is written: it avoids
// the 64-bit products and 64-bit to float conversions of the exact path.
struct CntF {
  float F, Bt, M;   // M: the row count of feature x10
  uint64_t B;
};

__device__ __forceinline__ float u64_to_f32(uint64_t v) { return (float)v; }

__device__ __forceinline__ CntF record_counts_f(int fam, uint32_t m32, uint32_t n32, uint32_t k32,
                                                uint32_t a32, uint32_t b32, uint32_t step,
                                                const EvalParams &p, uint32_t &bad) {
  const float dt = (float)p.elem_bytes, M = (float)m32, N = (float)n32, K = (float)k32, A = (float)a32;
  CntF c{0.0f, 0.0f, M, 0};
  switch (fam) {
    case KS_GEMM:
    case KS_LM_HEAD:
      c.F = (M * N) * (2.0f * K);
      c.Bt = dt * (M * K + K * N + M * N);
      c.B = (uint64_t)(((m32 + 127u) >> 7) * ((n32 + 127u) >> 7));
      break;
    case KS_GROUPED_GEMM: {
      uint32_t ms = 0, act = 0, tiles = 0;
      if ((uint64_t)b32 + a32 <= (uint64_t)p.n_expert_rows && a32 <= 1024) {
        expert_sums(p.expert_rows, b32, a32, ms, act, tiles);
      } else {
        bad |= kErrExpert;
      }
      const float Ms = (float)ms;
      c.M = Ms;
      c.F = (Ms * N) * (2.0f * K);
      c.Bt = dt * (Ms * K + (float)act * (K * N) + Ms * N);
      c.B = (uint64_t)tiles * ((n32 + 127u) >> 7);
      break;
    }
    case KS_ATTN_PREFILL:
    case KS_ATTN_DECODE: {
      uint64_t Q = 0, KV = 0, P = 0, T = 0;
      if ((int64_t)step < p.n_steps) {
        Q = p.agg[step];
        KV = p.agg[p.n_steps + step];
        P = p.agg[2 * p.n_steps + step];
        T = p.agg[3 * p.n_steps + step];
      }
      const float NK = N * K;   // exact: N, K < 2^12
      c.M = u64_to_f32(Q);
      c.F = (4.0f * NK) * u64_to_f32(P);
      c.Bt = dt * (2.0f * NK * u64_to_f32(Q) + (2.0f * A * K) * u64_to_f32(KV));
      c.B = (uint64_t)n32 * T;
      break;
    }
    case KS_RMSNORM:
      c.F = 4.0f * (M * N);
      c.Bt = dt * (2.0f * (M * N) + N);
      c.B = m32;
      break;
    case KS_ROPE:
      c.F = 3.0f * ((M * N) * K);
      c.Bt = dt * (2.0f * ((M * N) * K) + M * K);
      c.B = m32;
      break;
    case KS_SILU_MUL:
      c.F = 5.0f * (M * N);
      c.Bt = 3.0f * dt * (M * N);
      c.B = ((uint64_t)m32 * n32 + 1023u) >> 10;
      break;
    case KS_KV_WRITE:
      c.F = 0.0f;
      c.Bt = 4.0f * dt * ((M * N) * K);
      c.B = m32;
      break;
    default:  // KS_EMBED
      c.F = 0.0f;
      c.Bt = 2.0f * dt * (M * N) + 4.0f * M;
      c.B = m32;
      break;
  }
  return c;
}

// ------------------------------------------------------------ spec constants
__device__ void spec_prep_one(const ks_spec *__restrict__ specs, int s, SpecC *__restrict__ out, uint32_t *err) {
  const ks_spec sp = specs[s];
  SpecC c = {};
  const double P = sp.peak_flops, BW = sp.hbm_bw;
  // n_cu outside 1 .. 65535 is clamped and flagged (the wave count relies on
  // 24-bit products of it)
  uint32_t n = sp.n_cu;
  if (n < 1u || n > 65535u) {
    atomicOr(err, kErrSpec);
    n = n < 1u ? 1u : 65535u;
  }
  c.n = n;
  c.rcp_p = (float)(1.0 / P);
  c.rcp_bw = (float)(1.0 / BW);
  c.bw_over_p = (float)(BW / P);
  c.lr = (float)log2(BW / P);
  c.l2 = (float)sp.l2_bytes;
  c.t0 = (float)sp.t0;
  c.rcp_t0 = (float)(1.0 / fmax(sp.t0, 1e-9));
  c.n_f = (float)n;
  c.rcp_n = (float)(1.0 / (double)n);
  c.rcp_nd = 1.0 / (double)n;
  out[s] = c;
}

__global__ void k_spec_prep(const ks_spec *__restrict__ specs, int32_t n_specs, SpecC *__restrict__ out,
                            uint32_t *err) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < n_specs) spec_prep_one(specs, s, out, err);
}

// Spec constants through the scalar cache: they are read-only during the
// evaluation kernel and the index is wave-uniform, so the load goes through
// the constant address space.
// (The host pass of this file only parses device functions; it has no
// constant address space.)
__device__ __forceinline__ SpecC spec_at(const SpecC *base, int i) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef const __attribute__((address_space(4))) SpecC *SpecCPtr;
  return ((SpecCPtr)base)[__builtin_amdgcn_readfirstlane(i)];
#else
  return base[i];
#endif
}

// spec-independent per-record quantities
struct RowC {
  uint64_t B;
  float Ff, Btf, Bf, rcp_b, rcp_bt1, la, x0, xs[7];  // la = log2(AI); xs = x8 .. x14
};

__device__ __forceinline__ RowC row_consts(uint64_t B, float Ff, float Btf, float Mf, uint32_t n, uint32_t k) {
  RowC r;
  r.B = B;
  r.Ff = Ff;
  r.Btf = Btf;
  r.Bf = (float)B;
  r.rcp_b = rcpf(fmaxf(r.Bf, 1.0f));
  r.rcp_bt1 = rcpf(fmaxf(r.Btf, 1.0f));
  // log2(0) = -inf for F = 0; every use clamps it from below
  r.la = log2f_fast(r.Ff * r.rcp_bt1);
  r.x0 = fmaxf(r.la, -10.0f) * (1.0f / 16);
  r.xs[0] = log2f_fast(1.0f + r.Ff) * (1.0f / 64);
  r.xs[1] = log2f_fast(1.0f + r.Btf) * (1.0f / 48);
  r.xs[2] = log2f_fast(1.0f + Mf) * (1.0f / 24);
  r.xs[3] = log2f_fast(1.0f + (float)n) * (1.0f / 24);
  r.xs[4] = log2f_fast(1.0f + (float)k) * (1.0f / 24);
  r.xs[5] = log2f_fast(1.0f + r.Ff * r.rcp_b) * (1.0f / 48);
  r.xs[6] = log2f_fast(1.0f + r.Btf * r.rcp_b) * (1.0f / 40);
  return r;
}

// Block counts below 2^23 (every record of the workloads): the wave count
// in fp32 with exact integer-valued products.  With B < 2^23, fl(B fl(1/N)) is
// within 1/N of B/N, so its ceiling is exact unless B/N is an integer k,
// where it may come out k + 1; one test of (W - 1) N >= B corrects that.
// W N <= B + N < 2^24, so the products are exact.
constexpr uint32_t kSmallB = 1u << 23;

struct Roof {
  float t_comp, t_mem, t_roof, u, W;
};

// waves, u and t_roof (Sec. 2.2, Eq. 2)
template <bool kSmall>
__device__ __forceinline__ Roof roofline(const RowC &r, const SpecC &s) {
  Roof o;
  if constexpr (kSmall) {
    // in fp32 with selects: W0 N and (W0 - 1) N are integers below 2^24,
    // exact in fp32; for B = 0, W0 = 0 and the test fails
    const float W0 = ceilf(r.Bf * s.rcp_n);
    const float W = (W0 - 1.0f) * s.n_f >= r.Bf ? W0 - 1.0f : W0;
    o.W = W;
    o.u = r.Bf > 0.0f ? W * s.n_f * r.rcp_b : 1.0f;
  } else if (r.B > 0) {
    const uint64_t W = ceil_div(r.B, s.n, s.rcp_nd);
    o.W = (float)W;
    o.u = (float)(W * s.n) * r.rcp_b;
  } else {
    o.W = 0.0f;
    o.u = 1.0f;
  }
  o.t_comp = r.Ff * o.u * s.rcp_p;
  o.t_mem = r.Btf * s.rcp_bw;
  o.t_roof = fmaxf(o.t_comp, o.t_mem);
  return o;
}

// the 16 dimensionless features (x[16 + i] = x[i]^2 for 32 inputs);
// x1 = log2(AI / ridge) = log2(AI) + log2(BW / P), and the last-wave
// occupancy B / (W N) is 1 / u
template <bool RAW = false>
__device__ __forceinline__ float feature(int i, const RowC &r, const SpecC &s, const Roof &o) {
  // the same rounding wherever the features are formed: no product is fused
  // into a sum (t_comp + t_mem of feature 7 would be, in some schedules)
#pragma clang fp contract(off)
  constexpr float k16 = RAW ? 1.0f : 1.0f / 16;
  switch (i) {
    case 0: return r.x0;
    case 1: return fmaxf(r.la + s.lr, -20.0f) * k16;
    case 2: return log2f_fast(fmaf(r.Bf, s.rcp_n, 1.0f)) * k16;
    case 3: return rcpf(o.u);
    case 4: return log2f_fast(1.0f + o.W) * k16;
    case 5: return fminf(1.0f, s.l2 * r.rcp_bt1);
    case 6: return log2f_fast(fmaxf(o.t_roof * s.rcp_t0, 0x1p-20f)) * k16;
    case 7: {
      const float den = o.t_comp + o.t_mem;
      return den > 0.0f ? o.t_comp * rcpf(den) : 0.0f;
    }
    case 8: return r.xs[0];
    case 9: return r.xs[1];
    case 10: return r.xs[2];
    case 11: return r.xs[3];
    case 12: return r.xs[4];
    case 13: return r.xs[5];
    case 14: return r.xs[6];
    default: return 1.0f;
  }
}

template <int IN, bool RAW = false>
__device__ __forceinline__ void features(const RowC &r, const SpecC &s, const Roof &o, float (&x)[IN]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = feature<RAW>(i, r, s, o);
  if constexpr (IN == 32) {
#pragma unroll
    for (int i = 0; i < 16; ++i) x[16 + i] = x[i] * x[i];
  }
}

// MFMA group schedules of the bf16 heads (gen_sched.py writes them and
// checks their dependencies): {MFMA kind (0 none, 1 layer 1, 2 layer 2),
// block, chunk, VALU kind (0 none, 1 pack, 2 epilogue), block, pack half or
// first epilogue pair, epilogue pairs}.
struct SchedGrp {
  int mk, mb, kc, vk, vb, vj, vn;
};
#include "ks_sched.inc"

// ------------------------------------------------------------ bounded head
// The bounded analytical head (Sec. 5.3 and its efficiency-factor figure):
// eta = 1 / (gamma - alpha / W'), gamma = sigma(g . x), alpha = gamma sigma(a . x),
// W' = max(W, 1).  Written as (1 + e^-zg) W' (1 + E) / ((W' - 1) + W' E),
// E = e^-za: every term is positive, so nothing cancels when alpha nears
// gamma.  prm: g (16) then a (16), in LDS.
__device__ __forceinline__ float bounded_eta(const float (&x)[16], float W, const float *prm) {
  float zg = 0.0f, za = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    zg = fmaf(prm[i], x[i], zg);
    za = fmaf(prm[16 + i], x[i], za);
  }
  const float w = fmaxf(W, 1.0f);
  const float eg = __expf(-zg), ea = __expf(-za);
  return (1.0f + eg) * (w * (1.0f + ea)) * rcpf((w - 1.0f) + w * ea);
}

// ------------------------------------------------------------ Tier B grid
// The measured efficiency grid of Sec. 5.5 (Tier B), density-routed: the
// query's three coordinates (features grid_axis[d]) are mapped to node
// units t_d = (c_d - lo_d) (n_d - 1) / (hi_d - lo_d); inside the closed box,
// with all eight corners of the cell measured (not NaN), eta is their
// trilinear interpolation and `routed` is set; elsewhere the caller keeps
// the family's other head.  g: the family's nodes, row-major [n0][n1][n2],
// in LDS.  Every read stays in the family's nodes: the cell index is clamped
// to 0 .. n_d - 2 (a NaN coordinate clamps to 0 and is never routed).
__device__ __forceinline__ float grid_eta(const RowC &r, const SpecC &s, const Roof &o, const EvalParams &p,
                                          const float *g, bool &routed) {
  float fr[3];
  int idx[3];
  bool in = true;
#pragma unroll
  for (int d = 0; d < 3; ++d) {
    const float t = (feature(p.grid_axis[d], r, s, o) - p.grid_lo[d]) * p.grid_scale[d];
    const float top = (float)(p.grid_n[d] - 1);
    in = in && t >= 0.0f && t <= top;
    const float tc = fminf(fmaxf(t, 0.0f), top);
    idx[d] = min((int)tc, p.grid_n[d] - 2);
    fr[d] = tc - (float)idx[d];
  }
  const int s2 = p.grid_n[2], s1 = p.grid_n[1] * s2;
  const float *c = g + (idx[0] * s1 + idx[1] * s2 + idx[2]);
  const float v000 = c[0], v001 = c[1], v010 = c[s2], v011 = c[s2 + 1];
  const float v100 = c[s1], v101 = c[s1 + 1], v110 = c[s1 + s2], v111 = c[s1 + s2 + 1];
  const bool known = !__builtin_isnan(v000) && !__builtin_isnan(v001) && !__builtin_isnan(v010) &&
                     !__builtin_isnan(v011) && !__builtin_isnan(v100) && !__builtin_isnan(v101) &&
                     !__builtin_isnan(v110) && !__builtin_isnan(v111);
  routed = in && known;
  const float a00 = fmaf(fr[2], v001 - v000, v000), a01 = fmaf(fr[2], v011 - v010, v010);
  const float a10 = fmaf(fr[2], v101 - v100, v100), a11 = fmaf(fr[2], v111 - v110, v110);
  const float b0 = fmaf(fr[1], a01 - a00, a00), b1 = fmaf(fr[1], a11 - a10, a10);
  return fmaf(fr[0], b1 - b0, b0);
}

// ------------------------------------------------------------ bf16 MFMA head
// Orientation: hidden units are the MFMA rows (A = weights), the 64 records
// of a wave are the columns (B = activations, two 32-column blocks), so the
// C tile of one layer is already the B operand of the next one once the
// hidden units are renumbered; the renumbering is folded into the order in
// which W2's columns are staged in LDS.
//
// v_mfma_f32_32x32x16_bf16 lane layout (l = lane, g = l / 32):
//   A[i][k]: lane l holds row l % 32, k = 8 g .. 8 g + 7
//   B[k][j]: lane l holds col l % 32, k = 8 g .. 8 g + 7
//   C[i][j]: lane l holds col l % 32, rows 8 jj + 4 g + ii, register 4 jj + ii
template <int IN, int HID>
struct HeadBF16 {
  static constexpr int MB = HID / 32;   // 32-row blocks of every layer
  static constexpr int KC1 = IN / 16;   // K chunks of layer 1
  static constexpr int KC2 = HID / 16;  // K chunks of layer 2
  static constexpr int W1_DW = MB * KC1 * 64 * 4;
  static constexpr int W2_DW = MB * KC2 * 64 * 4;
  static constexpr int B2_DW = MB * 2 * 16;
  static constexpr int W3_DW = MB * 2 * 16;
  static constexpr int OFF_W2 = W1_DW;
  static constexpr int OFF_B2 = OFF_W2 + W2_DW;
  static constexpr int OFF_W3 = OFF_B2 + B2_DW;
  static constexpr int OFF_B3 = OFF_W3 + W3_DW;
  static constexpr int LDS_DW = OFF_B3 + 4;
  static constexpr bool kMlp = true;

  // layer-2 K slot s (0..15) of chunk kc -> hidden unit of layer 1's C tile
  __device__ static __forceinline__ int hid_of(int kc, int s) {
    const int g = s >> 3, t = s & 7;
    return (kc >> 1) * 32 + 8 * (2 * (kc & 1) + (t >> 2)) + 4 * g + (t & 3);
  }
  // C-tile register r of row-block mb, lane group g -> output unit
  __device__ static __forceinline__ int out_of(int mb, int g, int r) {
    return mb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
  }

  // The head takes the raw features (x1, x2, x4 and x6 without their 1/16,
  // the squares of 32-input heads without 1/256) and W1's columns carry the
  // scale instead.  Both are powers of two: bf16 rounding commutes with
  // them and the MFMA's products are exact, so every product and sum is the
  // same bit for bit, and the spec loop saves four multiplies per record.
  static constexpr bool kRaw = true;
  // W1 column k times the scale its feature drops in the raw form
  __device__ static __forceinline__ uint32_t raw_scaled(uint16_t w, int k) {
    const int b = k & 15;
    if (b != 1 && b != 2 && b != 4 && b != 6) return w;
    const float f = bf16_to_f32(w) * (k < 16 ? 1.0f / 16 : 1.0f / 256);
    return __builtin_bit_cast(uint32_t, f) >> 16;
  }
  __device__ static void stage(uint32_t *lds, int fam, const EvalParams &p) {
    // The two-wave heads (hidden 64 and 128, 256 registers) take the thread
    // index through an opaque copy, so that the per-thread addresses of
    // these loops are formed here, when a family is staged, rather than
    // hoisted out of the work loop and kept live across it (the 16-128 head
    // spilled them to scratch); the one-wave heads keep the hoisted form
    // (the opaque copy there made their scalar spills to VGPR lanes grow).
    int tid = (int)threadIdx.x;
    if constexpr (HID <= 128) asm volatile("" : "+v"(tid));
    const uint16_t *w1 = (const uint16_t *)p.w1 + (size_t)fam * HID * IN;
    const uint16_t *w2 = (const uint16_t *)p.w2 + (size_t)fam * HID * HID;
    const uint16_t *b2 = (const uint16_t *)p.b2 + (size_t)fam * HID;
    const uint16_t *w3 = (const uint16_t *)p.w3 + (size_t)fam * HID;
    const uint16_t *b3 = (const uint16_t *)p.b3 + fam;
    for (int d = tid; d < W1_DW; d += kWgThreads) {
      const int q = d & 3, lane = (d >> 2) & 63, frag = d >> 8;
      const int kc = frag % KC1, mb = frag / KC1;
      const int row = mb * 32 + (lane & 31);
      const int k0 = kc * 16 + (lane >> 5) * 8 + 2 * q;
      lds[d] = raw_scaled(w1[row * IN + k0], k0) | (raw_scaled(w1[row * IN + k0 + 1], k0 + 1) << 16);
    }
    if ((reinterpret_cast<uintptr_t>(w2) & 15) == 0) {
      // W2 by 16-byte row chunks: hidden units 8 c8 .. 8 c8 + 7 of a row are,
      // by hid_of, slots 0-3 of lane (row mod 32) and of lane (row mod 32) +
      // 32 of one K chunk's fragment, at dwords 0-1 (first 8 of the chunk's
      // 16 units) or 2-3 (last 8): each load feeds two 8-byte LDS writes
      // (one 2-byte load per unit, scattered, took several times longer)
      for (int c = tid; c < HID * HID / 8; c += kWgThreads) {
        const int row = c / (HID / 8), col = (c % (HID / 8)) * 8;
        const u32x4 v = *reinterpret_cast<const u32x4 *>(w2 + (size_t)row * HID + col);
        const int kc = 2 * (col >> 5) + ((col >> 4) & 1);
        const int frag = (row >> 5) * KC2 + kc;
        const int d0 = (frag * 64 + (row & 31)) * 4 + ((col & 8) ? 2 : 0);
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<u32x2 *>(lds + OFF_W2 + d0) = u32x2{v[0], v[1]};
        *reinterpret_cast<u32x2 *>(lds + OFF_W2 + d0 + 32 * 4) = u32x2{v[2], v[3]};
      }
    } else {
      for (int d = tid; d < W2_DW; d += kWgThreads) {
        const int q = d & 3, lane = (d >> 2) & 63, frag = d >> 8;
        const int kc = frag % KC2, mb = frag / KC2;
        const int row = mb * 32 + (lane & 31);
        const int s0 = (lane >> 5) * 8 + 2 * q;
        lds[OFF_W2 + d] = (uint32_t)w2[row * HID + hid_of(kc, s0)] |
                          ((uint32_t)w2[row * HID + hid_of(kc, s0 + 1)] << 16);
      }
    }
    for (int d = tid; d < B2_DW; d += kWgThreads) {
      const int r = d & 15, g = (d >> 4) & 1, mb = d >> 5;
      lds[OFF_B2 + d] = __builtin_bit_cast(uint32_t, bf16_to_f32(b2[out_of(mb, g, r)]));
    }
    for (int d = tid; d < W3_DW; d += kWgThreads) {
      const int r = d & 15, g = (d >> 4) & 1, mb = d >> 5;
      lds[OFF_W3 + d] = __builtin_bit_cast(uint32_t, bf16_to_f32(w3[out_of(mb, g, r)]));
    }
    if (tid == 0) lds[OFF_B3] = __builtin_bit_cast(uint32_t, bf16_to_f32(b3[0]));
  }

  // layer 3 over one 32-unit block of layer 2, in fp32: z += w3 . relu(h2)
  template <typename W3>
  __device__ static __forceinline__ void epilogue(const f32x16 &c0, const f32x16 &c1, const W3 &w3,
                                                  float &z0, float &z1) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      z0 = fmaf(w3[r], relu_f(c0[r]), z0);
      z1 = fmaf(w3[r], relu_f(c1[r]), z1);
    }
  }

  __device__ static __forceinline__ f32x16 mfma(const u32x4 &a, const u32x4 &b, const f32x16 &c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                   c, 0, 0, 0);
  }

  __device__ static __forceinline__ void fence() { __builtin_amdgcn_sched_barrier(0); }

  __device__ static __forceinline__ u32x4 frag_w1(const uint32_t *lds, int mb, int kc, int lane) {
    return *(const u32x4 *)(lds + ((mb * KC1 + kc) * 64 + lane) * 4);
  }
  __device__ static __forceinline__ u32x4 frag_w2(const uint32_t *lds, int mb, int kc, int lane) {
    return *(const u32x4 *)(lds + OFF_W2 + ((mb * KC2 + kc) * 64 + lane) * 4);
  }

  // relu + bf16 rounding of register pairs [2 q0, 2 q1) of one layer-1 block
  // (every conversion before the first relu: no op waits on the one just
  // before it)
  __device__ static __forceinline__ void pack_part(const f32x16 &c0, const f32x16 &c1, u32x4 (&h0)[2],
                                                   u32x4 (&h1)[2], int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      h0[q >> 2][q & 3] = pack_bf16(c0[2 * q], c0[2 * q + 1]);
      h1[q >> 2][q & 3] = pack_bf16(c1[2 * q], c1[2 * q + 1]);
    }
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      h0[q >> 2][q & 3] = relu_bf16x2(h0[q >> 2][q & 3]);
      h1[q >> 2][q & 3] = relu_bf16x2(h1[q >> 2][q & 3]);
    }
  }

  // ---- a fixed schedule of MFMA groups (hidden 128 and 256)
  // A group is one weight fragment times the two 32-record column blocks
  // (two MFMAs, 64 cycles of the matrix core), followed by a slice of VALU
  // work of another stage.  The table interleaves layer-1 blocks with the
  // first layer-2 chunks so that each layer-1 block is packed (relu, bf16)
  // in the groups right after it and before the chunk that consumes it,
  // and starts each layer-2 block's epilogue one group after that block's
  // last MFMA (and finishes it within the next block), so no VALU op waits
  // on an MFMA that is still in flight behind it and the matrix core never
  // drains.
  using Grp = SchedGrp;
  static constexpr int kNoV = 0, kPackV = 1, kEpiV = 2;
  __device__ static constexpr Grp sched(int i) {
    if constexpr (MB == 4) return KC1 == 1 ? kSched_4_1[i] : kSched_4_2[i];
    else return KC1 == 1 ? kSched_8_1[i] : kSched_8_2[i];
  }
  static constexpr int kNG = MB == 4 ? (KC1 == 1 ? sizeof(kSched_4_1) : sizeof(kSched_4_2)) / sizeof(Grp)
                                     : (KC1 == 1 ? sizeof(kSched_8_1) : sizeof(kSched_8_2)) / sizeof(Grp);

  struct S4 {
    u32x4 XB[2][KC1];
    u32x4 frag[3];
    f32x16 a1[2][2];
    u32x4 H0[MB][2], H1[MB][2];
    f32x16 c0, c1, p0, p1, bias;
    float w3r[2][16];
    float zacc[4];
    uint32_t lo[3];   // the lane's fragment offset (dwords) from LDS 0, 64 KB and 128 KB
    int lane, g;
  };

  // weight fragment of group I, from the lane's base address in LDS plus a
  // constant offset
  // (ds_read offsets are 16-bit byte offsets: fragments beyond 64 KB use a
  // second or third lane base, 64 KB and 128 KB further on)
  template <int I>
  __device__ static __forceinline__ u32x4 frag_of(const uint32_t *lds, const uint32_t (&lo)[3]) {
    constexpr Grp q = sched(I);
    constexpr int off = q.mk == 1 ? (q.mb * KC1 + q.kc) * 256 : OFF_W2 + (q.mb * KC2 + q.kc) * 256;
    return *(const u32x4 *)(lds + lo[off >> 14] + (off & 16383));
  }

  struct NoHook {
    template <class IC>
    __device__ __forceinline__ void operator()(IC) const {}
  };

  template <int I, class F = NoHook>
  __device__ static __forceinline__ void group(S4 &st, const uint32_t *lds, F &&hook = F{}) {
    constexpr Grp q = sched(I);
    // weight fragment of the group two ahead
    if constexpr (I + 2 < kNG && sched(I + 2).mk != 0) st.frag[(I + 2) % 3] = frag_of<I + 2>(lds, st.lo);
    const u32x4 a = st.frag[I % 3];
    if constexpr (q.mk == 1) {
      f32x16 &x0 = st.a1[q.mb & 1][0], &x1 = st.a1[q.mb & 1][1];
      if constexpr (q.kc == 0) {
        x0 = mfma(a, st.XB[0][0], f32x16{});
        x1 = mfma(a, st.XB[1][0], f32x16{});
      } else {
        x0 = mfma(a, st.XB[0][q.kc], x0);
        x1 = mfma(a, st.XB[1][q.kc], x1);
      }
    } else if constexpr (q.mk == 2) {
      if constexpr (q.kc == 0) {
        if constexpr (q.mb > 0) {
          // block mb-1 is complete: its accumulators feed the epilogue, and
          // its layer-3 weights are fetched a group before they are used
          st.p0 = st.c0;
          st.p1 = st.c1;
#pragma unroll
          for (int j = 0; j < 16; ++j)
            st.w3r[(q.mb - 1) & 1][j] = __builtin_bit_cast(float, lds[OFF_W3 + ((q.mb - 1) * 2 + st.g) * 16 + j]);
        }
        st.c1 = mfma(a, st.H1[0][0], st.bias);
        st.c0 = mfma(a, st.H0[0][0], st.bias);
      } else {
        st.c0 = mfma(a, st.H0[q.kc >> 1][q.kc & 1], st.c0);
        st.c1 = mfma(a, st.H1[q.kc >> 1][q.kc & 1], st.c1);
      }
      if constexpr (q.kc == KC2 / 2 && q.mb + 1 < MB)
        st.bias = *(const f32x16 *)(lds + OFF_B2 + ((q.mb + 1) * 2 + st.g) * 16);
      if constexpr (q.kc == KC2 - 1 && q.mb == MB - 1) {
#pragma unroll
        for (int j = 0; j < 16; ++j)
          st.w3r[q.mb & 1][j] = __builtin_bit_cast(float, lds[OFF_W3 + (q.mb * 2 + st.g) * 16 + j]);
      }
    }
    fence();
    if constexpr (q.vk == kPackV) {
      pack_part(st.a1[q.vb & 1][0], st.a1[q.vb & 1][1], st.H0[q.vb], st.H1[q.vb], 4 * q.vj, 4 * q.vj + 4);
    } else if constexpr (q.vk == kEpiV) {
      // layer 3 in fp32: relu through the sign bit, one FMA per hidden
      // unit with w3 staged as fp32 (a v_dot2c on bf16 pairs issues
      // alongside the MFMAs far worse than plain VALU ops: measured 1.7%
      // slower on the capacity grid)
#pragma unroll
      for (int j = q.vj; j < q.vj + q.vn; ++j) {
        const float *w = st.w3r[q.vb & 1];
        st.zacc[j & 1] = fmaf(w[2 * j], relu_f(st.p0[2 * j]), st.zacc[j & 1]);
        st.zacc[2 + (j & 1)] = fmaf(w[2 * j], relu_f(st.p1[2 * j]), st.zacc[2 + (j & 1)]);
        st.zacc[j & 1] = fmaf(w[2 * j + 1], relu_f(st.p0[2 * j + 1]), st.zacc[j & 1]);
        st.zacc[2 + (j & 1)] = fmaf(w[2 * j + 1], relu_f(st.p1[2 * j + 1]), st.zacc[2 + (j & 1)]);
      }
      // an empty use pins the slice here; otherwise the dot chain, whose
      // result is only needed at the end, is sunk below every MFMA
      asm volatile("" ::"v"(st.zacc[0]), "v"(st.zacc[1]), "v"(st.zacc[2]), "v"(st.zacc[3]));
    }
    hook(std::integral_constant<int, I>{});
    fence();
  }

  template <class F, int... I>
  __device__ static __forceinline__ void groups_h(S4 &st, const uint32_t *lds, F &hook,
                                                  std::integer_sequence<int, I...>) {
    (group<I>(st, lds, hook), ...);
  }

  // ---- the pieces of one spec's head (mlp4 runs them in order; the
  // software-pipelined spec loop of k_eval spreads the last block's
  // epilogue over the next spec's groups).  kPipe: the heads whose group
  // schedule that loop knows.  hook_at(I): what the loop does after group
  // I: the previous spec's last-block epilogue pairs [tp0, tp1), its eta,
  // its tail; the next spec's roofline, the features in the mask feat, the
  // squares [sq0, sq1) of a 32-input head, and the packing of layer-1 K
  // chunks [pk0, pk1).  The epilogue pairs come before the first group that
  // overwrites the last block's accumulators; the other pieces sit mostly
  // in groups with no VALU work of their own.
  struct Hook {
    int tp0, tp1;
    bool eta, tail, roof;
    uint32_t feat;
    int sq0, sq1, pk0, pk1;
  };
  static constexpr bool kPipe = (MB == 4 && KC1 == 1) || (MB == 8 && KC1 == 2);
  // the first group that overwrites the last block's accumulators (p0, p1)
  __device__ static constexpr int first_p_write() {
    for (int i = 0; i < kNG; ++i)
      if (sched(i).mk == 2 && sched(i).kc == 0 && sched(i).mb > 0) return i;
    return kNG;
  }
  __device__ static constexpr Hook hook_at(int I) {
    Hook h{0, 0, false, false, false, 0u, 0, 0, 0, 0};
    if constexpr (MB == 4) {
      // two waves per SIMD: the other wave's MFMAs cover larger slices
      if (I == 0) h.tp0 = 0, h.tp1 = 2;
      if (I == 5) h.tp0 = 2, h.tp1 = 4;
      if (I == 6) h.tp0 = 4, h.tp1 = 6;
      if (I == 11) h.tp0 = 6, h.tp1 = 8;
      if (I == 12) h.eta = true;
      if (I == 14) h.tail = true;
      if (I == 20) h.roof = true;
      if (I == 22) h.feat = 0xeu;
      if (I == 24) h.feat = 0xf0u;
      if (I == 28) h.feat = 0xff01u, h.pk0 = 0, h.pk1 = KC1;
    } else {
      // one wave per SIMD: slices small enough to issue in the shadow of
      // one group's MFMA pair, in groups without VALU work of their own
      constexpr int tp[8] = {0, 1, 4, 5, 8, 9, 12, 13};
      for (int j = 0; j < 8; ++j)
        if (I == tp[j]) h.tp0 = j, h.tp1 = j + 1;
      if (I == 16) h.eta = true;
      if (I == 20) h.tail = true;
      if (I == 35) h.roof = true;
      constexpr int ft[8] = {37, 39, 41, 43, 45, 47, 51, 53};   // features 1 .. 7, then 0 and 8 .. 15
      for (int f = 1; f < 8; ++f)
        if (I == ft[f - 1]) h.feat = 1u << f;
      if (I == ft[7]) h.feat = 0xff01u;
      if (I == 55) h.pk0 = 0, h.pk1 = 1;
      if (I == 57) h.sq0 = 0, h.sq1 = 8;
      if (I == 59) h.sq0 = 8, h.sq1 = 16;
      if (I == 61) h.pk0 = 1, h.pk1 = 2;
    }
    return h;
  }
  // every epilogue pair once, before the accumulators are overwritten;
  // every feature, square and chunk once, in order
  __device__ static constexpr bool hooks_ok() {
    int pairs = 0, last_tp = -1, eta = -1, tail = -1, roof = -1, pk = 0, sq = 0;
    uint32_t feats = 0;
    for (int i = 0; i < kNG; ++i) {
      const Hook h = hook_at(i);
      if (h.tp1 > h.tp0) {
        if (h.tp0 != pairs || i >= first_p_write()) return false;
        pairs = h.tp1, last_tp = i;
      }
      if (h.eta) eta = i;
      if (h.tail) tail = i;
      if (h.roof) roof = i;
      if (h.feat && (roof < 0 || (feats & h.feat))) return false;
      feats |= h.feat;
      if (h.sq1 > h.sq0) {
        if (h.sq0 != sq || feats != 0xffffu) return false;
        sq = h.sq1;
      }
      if (h.pk1 > h.pk0) {
        if (h.pk0 != pk) return false;
        for (int kc = h.pk0; kc < h.pk1; ++kc)
          if (kc == 0 ? feats != 0xffffu : sq < 16) return false;
        pk = h.pk1;
      }
    }
    return pairs == 8 && last_tp < eta && eta < tail && tail < roof && feats == 0xffffu && pk == KC1 &&
           (KC1 == 1 || sq == 16);
  }
  static_assert(!kPipe || hooks_ok(), "every hook once, in order, the epilogue before its accumulators go");
  __device__ static __forceinline__ void init_state(S4 &st) {
    st.lane = threadIdx.x & 63;
    st.g = st.lane >> 5;
    st.lo[0] = st.lane * 4;
    st.lo[1] = st.lo[0] + 16384;
    st.lo[2] = st.lo[0] + 32768;
    // opaque to the compiler, so it keeps the bases rather than forming
    // each address beyond 64 KB anew
    asm volatile("" : "+v"(st.lo[1]), "+v"(st.lo[2]));
#pragma unroll
    for (int j = 0; j < 4; ++j) st.zacc[j] = 0.0f;
  }
  // before a spec's groups: its features, the first fragments and b2; the
  // previous spec's partial layer-3 sums move to zp
  __device__ static __forceinline__ void begin_spec(S4 &st, const u32x4 (&XB)[2][KC1], const uint32_t *lds,
                                                    float (&zp)[4]) {
#pragma unroll
    for (int kc = 0; kc < KC1; ++kc) {
      st.XB[0][kc] = XB[0][kc];
      st.XB[1][kc] = XB[1][kc];
    }
    st.frag[0] = frag_of<0>(lds, st.lo);
    st.frag[1] = frag_of<1>(lds, st.lo);
    st.bias = *(const f32x16 *)(lds + OFF_B2 + st.g * 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      zp[j] = st.zacc[j];
      st.zacc[j] = 0.0f;
    }
    fence();
  }
  template <class F>
  __device__ static __forceinline__ void run_groups(S4 &st, const uint32_t *lds, F &hook) {
    groups_h(st, lds, hook, std::make_integer_sequence<int, kNG>{});
    // the last block's accumulators feed its epilogue in the next spec's groups
    st.p0 = st.c0;
    st.p1 = st.c1;
  }
  // register pairs [j0, j1) of the last block's epilogue into zp
  __device__ static __forceinline__ void tail_pairs(const S4 &st, float (&zp)[4], int j0, int j1) {
#pragma unroll
    for (int j = j0; j < j1; ++j) {
      const float *w = st.w3r[(MB - 1) & 1];
      zp[j & 1] = fmaf(w[2 * j], relu_f(st.p0[2 * j]), zp[j & 1]);
      zp[2 + (j & 1)] = fmaf(w[2 * j], relu_f(st.p1[2 * j]), zp[2 + (j & 1)]);
      zp[j & 1] = fmaf(w[2 * j + 1], relu_f(st.p0[2 * j + 1]), zp[j & 1]);
      zp[2 + (j & 1)] = fmaf(w[2 * j + 1], relu_f(st.p1[2 * j + 1]), zp[2 + (j & 1)]);
    }
  }
  // z: lanes l and l ^ 32 hold the two halves of the same record's dot
  // product; after the swap lane l < 32 adds block 0's halves of record l
  // and lane l >= 32 block 1's halves of record l.
  __device__ static __forceinline__ float tail_reduce(const float (&zp)[4], const uint32_t *lds) {
    uint32_t u0 = __builtin_bit_cast(uint32_t, zp[0] + zp[1]);
    uint32_t u1 = __builtin_bit_cast(uint32_t, zp[2] + zp[3]);
    swap32(u0, u1);
    return __builtin_bit_cast(float, u0) + __builtin_bit_cast(float, u1) +
           __builtin_bit_cast(float, lds[OFF_B3]);
  }

  // x -> bf16 pairs; the swap turns "own record" into the B layout of the
  // two 32-record column blocks
  __device__ static __forceinline__ void pack_x(const float (&x)[IN], u32x4 (&XB)[2][KC1], int kc0 = 0,
                                                int kc1 = KC1) {
    uint32_t P[IN / 2];
#pragma unroll
    for (int c = 8 * kc0; c < 8 * kc1; ++c) P[c] = pack_bf16(x[2 * c], x[2 * c + 1]);
#pragma unroll
    for (int kc = kc0; kc < kc1; ++kc) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t lo = P[8 * kc + q], hi = P[8 * kc + 4 + q];
        swap32(lo, hi);
        XB[0][kc][q] = lo;
        XB[1][kc][q] = hi;
      }
    }
  }

  // one spec's head on the features XB: the groups, then the last block's
  // epilogue and the reduction
  __device__ static __forceinline__ float mlp4(const u32x4 (&XB)[2][KC1], const uint32_t *lds) {
    S4 st;
    init_state(st);
    float unused[4];
    begin_spec(st, XB, lds, unused);
    NoHook none;
    run_groups(st, lds, none);
    tail_pairs(st, st.zacc, 0, 8);
    return tail_reduce(st.zacc, lds);
  }

  // z of the lane's own record; x: that record's features (fp32).
  //
  // A SIMD's VALU and matrix core only overlap when VALU work is issued in
  // the shadow of in-flight MFMAs of the same wave, and the compiler does not
  // interleave on its own.  So the body is scheduled by hand: straight-line
  // groups fenced by sched_barrier, each holding the LDS prefetch of a later
  // weight fragment, one MFMA pair, and a few VALU ops of another stage:
  //   layer 1, block mb      | relu/bf16 packing of layer-1 block mb-1
  //   layer 2, block 0       | packing of the last layer-1 block
  //   layer 2, block mb >= 1 | epilogue of layer-2 block mb-1 (relu, bf16,
  //                            dot with w3)
  // Only the features, the last epilogue and the tail stay exposed.
  __device__ static __forceinline__ float mlp(const float (&x)[IN], const uint32_t *lds) {
    static_assert(MB == 2 || MB == 4 || MB == 8, "hidden 64, 128 or 256");
    if constexpr (MB == 4 || MB == 8) {
      u32x4 XB[2][KC1];
      pack_x(x, XB);
      return mlp4(XB, lds);
    } else {
      const int lane = threadIdx.x & 63, g = lane >> 5;
      // features -> bf16 pairs; the swap turns "own record" into the B
      // layout of the two 32-record column blocks
      uint32_t P[IN / 2];
#pragma unroll
      for (int c = 0; c < IN / 2; ++c) P[c] = pack_bf16(x[2 * c], x[2 * c + 1]);
      u32x4 XB[2][KC1];
#pragma unroll
      for (int kc = 0; kc < KC1; ++kc) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t lo = P[8 * kc + q], hi = P[8 * kc + 4 + q];
          swap32(lo, hi);
          XB[0][kc][q] = lo;
          XB[1][kc][q] = hi;
        }
      }
      // ---- layer 1 | packing of the previous layer-1 block
      u32x4 H0[MB][2], H1[MB][2];
      f32x16 a1[2][2];
      u32x4 w1f[KC1];
#pragma unroll
      for (int kc = 0; kc < KC1; ++kc) w1f[kc] = frag_w1(lds, 0, kc, lane);
      fence();
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        u32x4 cur[KC1];
#pragma unroll
        for (int kc = 0; kc < KC1; ++kc) {
          cur[kc] = w1f[kc];
          if (mb + 1 < MB) w1f[kc] = frag_w1(lds, mb + 1, kc, lane);
        }
        a1[mb & 1][0] = f32x16{};
        a1[mb & 1][1] = f32x16{};
#pragma unroll
        for (int kc = 0; kc < KC1; ++kc) {
          a1[mb & 1][0] = mfma(cur[kc], XB[0][kc], a1[mb & 1][0]);
          a1[mb & 1][1] = mfma(cur[kc], XB[1][kc], a1[mb & 1][1]);
        }
        if (mb > 0) pack_part(a1[(mb - 1) & 1][0], a1[(mb - 1) & 1][1], H0[mb - 1], H1[mb - 1], 0, 8);
        fence();
      }
      // ---- layer 2: weight fragments prefetched two chunks ahead
      constexpr int NCH = MB * KC2;   // (block, chunk) pairs in order
      u32x4 wf[3];
      wf[0] = frag_w2(lds, 0, 0, lane);
      wf[1] = frag_w2(lds, 0, 1, lane);
      f32x16 bias = *(const f32x16 *)(lds + OFF_B2 + g * 16);
      f32x16 c0 = {}, c1 = {}, p0 = {}, p1 = {};
      float w3r[16];
      float z0 = 0.0f, z1 = 0.0f;
      fence();
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int mb = i / KC2, kc = i % KC2;
        if (i + 2 < NCH) wf[(i + 2) % 3] = frag_w2(lds, (i + 2) / KC2, (i + 2) % KC2, lane);
        if (kc == 0 && mb > 0) {
          // block mb-1's accumulators become the epilogue's inputs
          p0 = c0;
          p1 = c1;
#pragma unroll
          for (int q = 0; q < 16; ++q) w3r[q] = __builtin_bit_cast(float, lds[OFF_W3 + ((mb - 1) * 2 + g) * 16 + q]);
        }
        const u32x4 a = wf[i % 3];
        if (kc == 0) {
          c1 = mfma(a, H1[0][0], bias);
          c0 = mfma(a, H0[0][0], bias);
        } else {
          c0 = mfma(a, H0[kc >> 1][kc & 1], c0);
          c1 = mfma(a, H1[kc >> 1][kc & 1], c1);
        }
        if (kc == KC2 / 2 && mb + 1 < MB) bias = *(const f32x16 *)(lds + OFF_B2 + ((mb + 1) * 2 + g) * 16);
        if (mb == 0) {
          // pack the last layer-1 block over the first PG groups, all of
          // which come before chunk 2 (MB - 1), its first consumer
          constexpr int PG = 2 * (MB - 1) < 4 ? 2 * (MB - 1) : 4;
          if (kc < PG) pack_part(a1[(MB - 1) & 1][0], a1[(MB - 1) & 1][1], H0[MB - 1], H1[MB - 1],
                                 kc * 8 / PG, (kc + 1) * 8 / PG);
        } else {
          // chunk kc's share of block mb-1's epilogue: register pairs
          // [8 kc / KC2, 8 (kc + 1) / KC2) of the 8
#pragma unroll
          for (int q = kc * 8 / KC2; q < (kc + 1) * 8 / KC2; ++q) {
            z0 = fmaf(w3r[2 * q], relu_f(p0[2 * q]), z0);
            z1 = fmaf(w3r[2 * q], relu_f(p1[2 * q]), z1);
            z0 = fmaf(w3r[2 * q + 1], relu_f(p0[2 * q + 1]), z0);
            z1 = fmaf(w3r[2 * q + 1], relu_f(p1[2 * q + 1]), z1);
          }
          // an empty use pins this part here; otherwise the dot chain, whose
          // result is only needed at the end, is sunk below every MFMA
          asm volatile("" ::"v"(z0), "v"(z1));
        }
        fence();
      }
#pragma unroll
      for (int q = 0; q < 16; ++q) w3r[q] = __builtin_bit_cast(float, lds[OFF_W3 + ((MB - 1) * 2 + g) * 16 + q]);
      epilogue(c0, c1, w3r, z0, z1);
      // lanes l and l ^ 32 hold the two halves of the same record's dot
      // product; after the swap lane l < 32 adds block 0's halves of record
      // l and lane l >= 32 block 1's halves of record l.
      uint32_t u0 = __builtin_bit_cast(uint32_t, z0), u1 = __builtin_bit_cast(uint32_t, z1);
      swap32(u0, u1);
      return __builtin_bit_cast(float, u0) + __builtin_bit_cast(float, u1) +
             __builtin_bit_cast(float, lds[OFF_B3]);
    }
  }
};

// ------------------------------------------------------------ fp32 MFMA head
// Same orientation with v_mfma_f32_32x32x2_f32 (K = 2 per instruction):
//   A[i][k]: lane l holds row l % 32, k = g;  B[k][j]: col l % 32, k = g;
//   C as for the bf16 instruction.
template <int IN, int HID>
struct HeadF32 {
  static constexpr bool kRaw = false;
  static constexpr int MB = HID / 32;
  static constexpr int C1 = IN / 2;
  static constexpr int W1_DW = MB * C1 * 64;
  static constexpr int W2_DW = MB * MB * 64 * 16;
  static constexpr int B2_DW = MB * 2 * 16;
  static constexpr int W3_DW = MB * 2 * 16;
  static constexpr int OFF_W2 = W1_DW;
  static constexpr int OFF_B2 = OFF_W2 + W2_DW;
  static constexpr int OFF_W3 = OFF_B2 + B2_DW;
  static constexpr int OFF_B3 = OFF_W3 + W3_DW;
  static constexpr int LDS_DW = OFF_B3 + 4;
  static constexpr bool kMlp = true;

  __device__ static __forceinline__ int out_of(int mb, int g, int r) {
    return mb * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
  }

  __device__ static void stage(uint32_t *lds, int fam, const EvalParams &p) {
    const float *w1 = (const float *)p.w1 + (size_t)fam * HID * IN;
    const float *w2 = (const float *)p.w2 + (size_t)fam * HID * HID;
    const float *b2 = (const float *)p.b2 + (size_t)fam * HID;
    const float *w3 = (const float *)p.w3 + (size_t)fam * HID;
    float *f = (float *)lds;
    for (int d = threadIdx.x; d < W1_DW; d += kWgThreads) {
      const int lane = d & 63, c = (d >> 6) % C1, mb = (d >> 6) / C1;
      f[d] = w1[(mb * 32 + (lane & 31)) * IN + 2 * c + (lane >> 5)];
    }
    // [mb2][mb][lane][r]: W2[out = mb2 32 + l % 32][in = out_of(mb, g, r)]
    for (int d = threadIdx.x; d < W2_DW; d += kWgThreads) {
      const int r = d & 15, lane = (d >> 4) & 63, blk = d >> 10;
      const int mb = blk % MB, mb2 = blk / MB;
      f[OFF_W2 + d] = w2[(mb2 * 32 + (lane & 31)) * HID + out_of(mb, lane >> 5, r)];
    }
    for (int d = threadIdx.x; d < B2_DW; d += kWgThreads) {
      const int r = d & 15, g = (d >> 4) & 1, mb = d >> 5;
      f[OFF_B2 + d] = b2[out_of(mb, g, r)];
      f[OFF_W3 + d] = w3[out_of(mb, g, r)];
    }
    if (threadIdx.x == 0) f[OFF_B3] = ((const float *)p.b3)[fam];
  }

  __device__ static __forceinline__ float mlp(const float (&x)[IN], const uint32_t *lds) {
    const int lane = threadIdx.x & 63, g = lane >> 5;
    const float *f = (const float *)lds;
    float XB[2][C1];
#pragma unroll
    for (int c = 0; c < C1; ++c) {
      uint32_t lo = __builtin_bit_cast(uint32_t, x[2 * c]);
      uint32_t hi = __builtin_bit_cast(uint32_t, x[2 * c + 1]);
      swap32(lo, hi);
      XB[0][c] = __builtin_bit_cast(float, lo);
      XB[1][c] = __builtin_bit_cast(float, hi);
    }
    f32x16 H1[2][MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      f32x16 c0 = {}, c1 = {};
#pragma unroll
      for (int c = 0; c < C1; ++c) {
        const float a = f[(mb * C1 + c) * 64 + lane];
        c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, XB[0][c], c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a, XB[1][c], c1, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        c0[r] = fmaxf(c0[r], 0.0f);
        c1[r] = fmaxf(c1[r], 0.0f);
      }
      H1[0][mb] = c0;
      H1[1][mb] = c1;
    }
    float z0 = 0.0f, z1 = 0.0f;
#pragma unroll 1
    for (int mb2 = 0; mb2 < MB; ++mb2) {
      const f32x16 bias = *(const f32x16 *)(f + OFF_B2 + (mb2 * 2 + g) * 16);
      f32x16 c0 = bias, c1 = bias;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const float *a = f + OFF_W2 + ((mb2 * MB + mb) * 64 + lane) * 16;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          c0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[r], H1[0][mb][r], c0, 0, 0, 0);
          c1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a[r], H1[1][mb][r], c1, 0, 0, 0);
        }
      }
      const float *w3 = f + OFF_W3 + (mb2 * 2 + g) * 16;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        z0 = fmaf(w3[r], fmaxf(c0[r], 0.0f), z0);
        z1 = fmaf(w3[r], fmaxf(c1[r], 0.0f), z1);
      }
    }
    uint32_t a0 = __builtin_bit_cast(uint32_t, z0), a1 = __builtin_bit_cast(uint32_t, z1);
    swap32(a0, a1);
    return __builtin_bit_cast(float, a0) + __builtin_bit_cast(float, a1) + f[OFF_B3];
  }
};

struct HeadOne {
  static constexpr int LDS_DW = 1;
  static constexpr bool kMlp = false;
  __device__ static void stage(uint32_t *, int, const EvalParams &) {}
  template <int IN>
  __device__ static float mlp(const float (&)[IN], const uint32_t *) { return 0.0f; }
};

// kMinWg: workgroups per CU the register allocator must fit (2 = two waves
// per SIMD, at most 256 registers per lane).
template <int KIND> struct KindOf;
template <> struct KindOf<kEtaOne> { using H = HeadOne; static constexpr int IN = 16; };
template <> struct KindOf<kBoundedOnly> { using H = HeadOne; static constexpr int IN = 16; };
template <> struct KindOf<kF32_16_64> { using H = HeadF32<16, 64>; static constexpr int IN = 16; };
template <> struct KindOf<kF32_16_128> { using H = HeadF32<16, 128>; static constexpr int IN = 16; };
template <> struct KindOf<kF32_32_64> { using H = HeadF32<32, 64>; static constexpr int IN = 32; };
template <> struct KindOf<kF32_32_128> { using H = HeadF32<32, 128>; static constexpr int IN = 32; };
template <> struct KindOf<kBF16_16_64> { using H = HeadBF16<16, 64>; static constexpr int IN = 16; };
template <> struct KindOf<kBF16_16_128> { using H = HeadBF16<16, 128>; static constexpr int IN = 16; };
template <> struct KindOf<kBF16_16_256> { using H = HeadBF16<16, 256>; static constexpr int IN = 16; };
template <> struct KindOf<kBF16_32_64> { using H = HeadBF16<32, 64>; static constexpr int IN = 32; };
template <> struct KindOf<kBF16_32_128> { using H = HeadBF16<32, 128>; static constexpr int IN = 32; };
template <> struct KindOf<kBF16_32_256> { using H = HeadBF16<32, 256>; static constexpr int IN = 32; };

// ------------------------------------------------------------ segmented scan
// Inclusive scan of a wave's 64 values, segmented by sorted keys, with DPP
// lane moves (no LDS round trips), in Hillis-Steele form: within each row
// of 16 lanes every lane adds the partial of the lane 1, 2, 4 and 8 below
// it (the last two only for lanes 4..15 and 8..15), then lane 15 of each
// row is added into rows 1 and 3 and lane 31 into rows 2 and 3.  A step's
// factor is 1 where its source lane holds the same key, so, the keys being
// sorted, the source's partial covers only lanes of the same segment; 0
// otherwise.  Sums are built in at most 6 levels of adds of non-negative
// terms, so the fp32 result errs by at most 6 * 2^-24 relative; tiles and
// families are then summed in fp64.

// key of the DPP source lane, or a value unequal to key where the pattern
// has no source (bound_ctrl off: such lanes keep `old`)
template <int CTRL, int ROW, int BANK>
__device__ __forceinline__ uint32_t dpp_key(uint32_t key) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)(key ^ 1u), (int)key, CTRL, ROW, BANK, false);
}

// Factor of each seg_scan step (row_shr:1, 2, 4, 8, row_bcast:15, 31).
__device__ __forceinline__ void seg_factors(uint32_t key, float (&f)[6]) {
  f[0] = dpp_key<0x111, 0xf, 0xf>(key) == key ? 1.0f : 0.0f;
  f[1] = dpp_key<0x112, 0xf, 0xf>(key) == key ? 1.0f : 0.0f;
  f[2] = dpp_key<0x114, 0xf, 0xe>(key) == key ? 1.0f : 0.0f;
  f[3] = dpp_key<0x118, 0xf, 0xc>(key) == key ? 1.0f : 0.0f;
  f[4] = dpp_key<0x142, 0xa, 0xf>(key) == key ? 1.0f : 0.0f;
  f[5] = dpp_key<0x143, 0xc, 0xf>(key) == key ? 1.0f : 0.0f;
}

// Each step is one v_fmac_f32 with its first source read through DPP
// (v += f * v[source lane]); lanes a step's bank or row mask leaves out keep
// v, and lanes whose source lies outside the row read 0 (bound_ctrl).  A DPP
// read of a VGPR written by the VALU op just before needs two wait states,
// hence the s_nop 1 before every step (the compiler does not see into the
// block, so the waits are explicit).
__device__ __forceinline__ float seg_scan(float v, const float (&f)[6]) {
  asm volatile(
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %2 row_shr:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %3 row_shr:4 row_mask:0xf bank_mask:0xe\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %4 row_shr:8 row_mask:0xf bank_mask:0xc\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %5 row_bcast:15 row_mask:0xa bank_mask:0xf\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %6 row_bcast:31 row_mask:0xc bank_mask:0xf\n"
      : "+v"(v)
      : "v"(f[0]), "v"(f[1]), "v"(f[2]), "v"(f[3]), "v"(f[4]), "v"(f[5]));
  return v;
}

// ------------------------------------------------------------ evaluation
// Workgroup = 4 waves; a workgroup tile is 4 consecutive 64-record wave
// tiles of one family, so the family's head is staged in LDS once and
// shared.  Workgroups stride over workgroup tiles and restage only when the
// family changes (records are family-major).
template <int KIND> struct MinWg { static constexpr int value = 1; };
template <> struct MinWg<kBF16_16_64> { static constexpr int value = 2; };
template <> struct MinWg<kBF16_16_128> { static constexpr int value = 2; };
template <> struct MinWg<kBF16_32_64> { static constexpr int value = 2; };
template <> struct MinWg<kBF16_32_128> { static constexpr int value = 2; };

// One wave's tile: 64 consecutive records of one family (nvalid = 0 for an
// idle wave of a family's last workgroup tile).
struct Tile {
  int fam, tile_in_fam, nvalid;
  int64_t row0, fam_lo, fam_hi;
};

// fam0: a family at or before the tile's (workgroups walk tiles in order)
__device__ __forceinline__ Tile locate(const EvalParams &p, int wt, int wave, int fam0) {
  Tile t;
  int fam = fam0;
  while (wt >= p.wgt_off[fam + 1]) ++fam;
  t.fam = fam;
  t.tile_in_fam = (wt - p.wgt_off[fam]) * kWgWaves + wave;
  t.fam_lo = p.fam_off[fam];
  t.fam_hi = p.fam_off[fam + 1];
  t.row0 = t.fam_lo + (int64_t)t.tile_in_fam * kTileRows;
  const int64_t left = t.fam_hi - t.row0;
  t.nvalid = left <= 0 ? 0 : (left < kTileRows ? (int)left : kTileRows);
  return t;
}

// The record fields a lane's family uses (the others are never read), plus
// the steps just before and after the tile within its family: prev and next
// by scalar loads, or (VEC) pn by one vector load, the one before in lane 0
// and the one after in the other lanes (see tile_edges).
struct Fields {
  uint32_t st, m, n, k, a, b, prev, next, pn;
  float mult;   // dispatches the record stands for (1 without a multiplicity array)
};

template <bool MULT, bool VEC>
__device__ __forceinline__ Fields load_fields(const EvalParams &p, const Tile &t, int lane) {
  Fields f = {0, 0, 0, 0, 0, 0, kNoKey, kNoKey, kNoKey, 1.0f};
  if (t.nvalid == 0) return f;
  // wave-uniform bases plus a 32-bit lane offset (no per-lane 64-bit
  // address arithmetic)
  const uint32_t off = (uint32_t)(lane < t.nvalid ? lane : 0);
  const int64_t r0 = t.row0;
  const int fam = t.fam;
  const bool grouped = fam == KS_GROUPED_GEMM;
  const bool attn = fam == KS_ATTN_PREFILL || fam == KS_ATTN_DECODE;
  f.st = (p.step + r0)[off];
  f.n = (p.n + r0)[off];
  if (!grouped && !attn) f.m = (p.m + r0)[off];
  if (fam != KS_RMSNORM && fam != KS_SILU_MUL && fam != KS_EMBED) f.k = (p.k + r0)[off];
  if (grouped || attn) f.a = (p.a + r0)[off];
  if (grouped) f.b = (p.b + r0)[off];
  if constexpr (MULT) f.mult = (float)(p.mult + r0)[off];   // exact below 2^24
  const bool hp = t.row0 > t.fam_lo, hn = t.row0 + kTileRows < t.fam_hi;
  if constexpr (VEC) {
    // one vector load for both neighbours (each lane's address stays inside
    // the family: the tile's first row where a neighbour does not exist).
    // In a short loop a scalar load here costs its whole latency: the next
    // scalar load of the spec loop waits for it (scalar loads complete out
    // of order, so waits are for all of them).
    const int pn_off = lane == 0 ? (hp ? -1 : 0) : (hn ? kTileRows : 0);
    f.pn = (p.step + r0)[pn_off];
  } else {
    if (hp) f.prev = p.step[t.row0 - 1];
    if (hn) f.next = p.step[t.row0 + kTileRows];
  }
  return f;
}

// the steps just before and after tile t (kNoKey where the family ends)
template <bool VEC>
__device__ __forceinline__ void tile_edges(const Tile &t, const Fields &f, uint32_t &prev, uint32_t &next) {
  if constexpr (VEC) {
    prev = t.row0 > t.fam_lo ? __builtin_amdgcn_readlane(f.pn, 0) : kNoKey;
    next = t.row0 + kTileRows < t.fam_hi ? __builtin_amdgcn_readlane(f.pn, 1) : kNoKey;
  } else {
    prev = f.prev;
    next = f.next;
  }
}

// Variants, each a separate instantiation so that the kernels without them
// keep their registers and schedule: kVarGrid compiles Tier B routing in,
// kVarMult weights each record's step-sum term by its multiplicity.
enum : int { kVarGrid = 1, kVarMult = 2, kNumVars = 4 };

// heads that take the software-pipelined spec loop
template <class H, class = void> struct PipeOK : std::false_type {};
template <class H> struct PipeOK<H, std::enable_if_t<H::kPipe>> : std::true_type {};

// Spec s's per-pair outputs of the lane's record and its segmented step sum:
// a tail lane stores its segment's sum to dst[s] (dst: the tile's carry
// slots or the (family, step) partials, one per spec, contiguous), a record
// of multiplicity m adding m t (one fp32 rounding).
template <bool MULT>
__device__ __forceinline__ void spec_tail(const EvalParams &p, int s, float t_roof, float eta, float t, bool valid,
                                          bool live, int64_t row, float tfac, const float (&fac)[6], double *dst) {
  // (the per-pair test first: a call without per-pair outputs forms no
  // address)
  if ((p.o_troof || p.o_eta || p.o_t) && valid) {
    const size_t i = (size_t)s * (size_t)p.fam_off[KS_NFAM] + (size_t)row;
    if (p.o_troof) p.o_troof[i] = t_roof;
    if (p.o_eta) p.o_eta[i] = eta;
    if (p.o_t) p.o_t[i] = t;
  }
  if (p.partial) {
    const float v = seg_scan(MULT ? t * tfac : (live ? t : 0.0f), fac);
    if (dst) dst[s] = (double)v;
  }
}

// work items per workgroup below which the heads take contiguous ranges
constexpr int kBlockedItems = 32;

// the workgroup tile and the spec range of work item w: w / n and w % n,
// with no integer division in the usual case of one range of all specs
__device__ __forceinline__ int item_tile(int w, int n) {
  if (n == 1) return w;
  return w / n;
}
__device__ __forceinline__ int item_range(int w, int n) {
  if (n == 1) return 0;
  return w % n;
}

template <int KIND, int VAR>
__global__ __launch_bounds__(kWgThreads, MinWg<KIND>::value) void k_eval(EvalParams p) {
  constexpr bool GRID = (VAR & kVarGrid) != 0;
  constexpr bool MULT = (VAR & kVarMult) != 0;
  using H = typename KindOf<KIND>::H;
  constexpr int IN = KindOf<KIND>::IN;
  __shared__ __align__(16) uint32_t lds[H::LDS_DW];   // 16-byte fragment reads, 8-byte staging writes
  __shared__ float bnd_lds[32];   // the bounded head of the staged family: g then a
  __shared__ float grid_lds[KS_GRID_MAX_NODES];   // the staged family's measured grid
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // work item w: workgroup tile w / n_chunks, specs [s0, s1) of range w % n_chunks
  const int n_chunks = p.n_chunks;
  const int n_work = p.wgt_off[KS_NFAM] * n_chunks;
  int staged = -1;
  // the next tile's fields are loaded while the current one is evaluated
  Tile tn = {};
  Fields fn = {0, 0, 0, 0, 0, 0, kNoKey, kNoKey, kNoKey, 1.0f};
  // tiles without a head, and the heads that run one wave per SIMD, take
  // their neighbour steps by a vector load (the scalar loads' round trip is
  // waited for by the next scalar or LDS wait, which one wave per SIMD
  // cannot cover; with two waves per SIMD the vector load measured no
  // better overall)
  constexpr bool VEC = !H::kMlp || MinWg<KIND>::value == 1;
  // With few work items per workgroup the heads take a contiguous range of
  // them, so that a workgroup meets one or two families and stages their
  // weights into LDS once or twice (striding over the grid it restaged them
  // at nearly every item); with many, striding balances the families'
  // different per-tile costs better, and so it does for calls where some
  // families take the bounded head or a grid (far cheaper tiles than the
  // MLP's); the HBM-bound kinds always stride, which keeps the chip's loads
  // in one window.  (The bounds are wave-uniform: readfirstlane keeps them
  // in scalar registers.)
  const int G = (int)gridDim.x, b = (int)blockIdx.x;
  const bool blocked = H::kMlp && !GRID && p.bounded_mask == 0u && n_work < kBlockedItems * G;
  const int w_begin = blocked ? __builtin_amdgcn_readfirstlane(b * (n_work / G) + min(b, n_work % G)) : b;
  const int w_end =
      blocked ? __builtin_amdgcn_readfirstlane(w_begin + n_work / G + (b < n_work % G ? 1 : 0)) : n_work;
  const int w_step = blocked ? 1 : G;
  if (w_begin < w_end) {
    tn = locate(p, item_tile(w_begin, n_chunks), wave, 0);
    fn = load_fields<MULT, VEC>(p, tn, lane);
  }
  for (int w = w_begin; w < w_end; w += w_step) {
    const Tile tc = tn;
    const Fields fc = fn;
    if (w + w_step < w_end) {
      tn = locate(p, item_tile(w + w_step, n_chunks), wave, tc.fam);
      fn = load_fields<MULT, VEC>(p, tn, lane);
    }
    const int s_lo = item_range(w, n_chunks) * p.spec_chunk;
    const int s_hi = min(s_lo + p.spec_chunk, p.n_specs);
    const int fam = tc.fam;
    // this family takes the bounded head (the plain eta = 1 stream has none)
    const bool bnd = KIND != kEtaOne && ((p.bounded_mask >> fam) & 1u);
    // ... and a measured grid that routes some of its records
    const bool grd = GRID && ((p.grid_mask >> fam) & 1u);
    if (H::kMlp || (KIND != kEtaOne && (p.bounded_mask || GRID))) {
      if (fam != staged) {
        __syncthreads();
        if (bnd) {
          if (threadIdx.x < 32) bnd_lds[threadIdx.x] = p.bounded[fam * 32 + threadIdx.x];
        } else {
          if constexpr (H::kMlp) H::stage(lds, fam, p);
        }
        if (grd) {
          const float *src = p.grid + (size_t)fam * p.grid_nodes;
          for (int i = threadIdx.x; i < p.grid_nodes; i += kWgThreads) grid_lds[i] = src[i];
        }
        __syncthreads();
        staged = fam;
      }
    }
    if (tc.nvalid == 0) continue;
    const int nvalid = tc.nvalid;
    const bool valid = lane < nvalid;
    const int64_t row = tc.row0 + (valid ? lane : 0);

    uint32_t bad = 0;
    if ((int64_t)fc.st >= p.n_steps) bad |= kErrStep;
    RowC rc;
    // F, Bt and the feature row count in fp32 as they are formed (a few
    // roundings, within 1e-6 relative of the exact counts) when no count is
    // written: no 64-bit products or 64-bit to float conversions.  Calls
    // with a measured grid keep the exact path, so that a record's cell is
    // the one the exact features give.
    if (!GRID && !p.o_flops && !p.o_bytes && !p.o_blocks) {
      const CntF cf = record_counts_f(fam, fc.m, fc.n, fc.k, fc.a, fc.b, fc.st, p, bad);
      rc = row_consts(cf.B, cf.F, cf.Bt, cf.M, fc.n, fc.k);
    } else {
      const Cnt c = record_counts(fam, fc.m, fc.n, fc.k, fc.a, fc.b, fc.st, p, bad);
      if (valid) {
        if (p.o_flops) p.o_flops[row] = c.F;
        if (p.o_bytes) p.o_bytes[row] = c.Bt;
        if (p.o_blocks) p.o_blocks[row] = c.B;
      }
      rc = row_consts(c.B, (float)c.F, (float)c.Bt, (float)c.M, fc.n, fc.k);
    }
    if (valid && bad) atomicOr(p.err, bad);
    const bool live = valid && !(bad & kErrStep);
    const bool small = __ballot(rc.B >= kSmallB) == 0;   // wave-uniform

    // segment structure of this tile (spec-independent): keys are sorted
    const uint32_t key = live ? fc.st : kNoKey;
    const uint32_t key_dn = dpp_key<0x130, 0xf, 0xf>(key);   // wave_shl:1, lane 63: unequal
    const bool is_tail = live && key_dn != key;
    const uint32_t key0 = __builtin_amdgcn_readfirstlane(key);
    uint32_t prev, next;
    tile_edges<VEC>(tc, fc, prev, next);
    const bool to_carry = is_tail && key == key0 && prev == key0;
    const int tile_id = p.tile_off[fam] + tc.tile_in_fam;
    if (p.range) {
      // the (family, step) record range, written where its global first
      // and last records are
      const uint32_t key_up = dpp_key<0x138, 0xf, 0xf>(key);   // wave_shr:1
      const bool head = live && (lane == 0 ? prev != key : key_up != key);
      const bool tail = live && (lane == nvalid - 1 ? next != key : key_dn != key);
      if (head) p.range[2 * ((size_t)fam * p.n_steps + key)] = (uint32_t)row;
      if (tail) p.range[2 * ((size_t)fam * p.n_steps + key) + 1] = (uint32_t)(row + 1);
    }
    // A tail lane stores its segment's sum (seg_scan): into the tile's carry
    // slot if the segment continues from the previous tile, else into the
    // (spec, family, step) partial.
    float fac[6];
    seg_factors(key, fac);
    // the scan input is m t for a live record of multiplicity m (1 without
    // a multiplicity array) and 0 otherwise: one product per spec instead
    // of a select.  A lane that is not live either repeats lane 0's record
    // (a tail lane past nvalid, whose t is finite whenever lane 0's is) or
    // is flagged bad data; both sit at or after the wave's last live lane or
    // carry a flagged record, so the scan of every live segment is unchanged.
    const float tfac = MULT ? (live ? fc.mult : 0.0f) : 0.0f;
    // (spec-minor layout: a tail lane's sums for all specs are one
    // contiguous run, so its stores fill whole cache lines)
    double *dst = nullptr;
    if (p.partial && is_tail) {
      if (to_carry)
        dst = p.carry + (size_t)tile_id * (size_t)p.n_specs;
      else
        dst = p.partial + ((size_t)fam * (size_t)p.n_steps + key) * (size_t)p.n_specs;
    }

    if constexpr (PipeOK<H>::value && !GRID) {
      if (!bnd) {
        // Software-pipelined spec loop: spec s's MFMA groups carry, in their
        // VALU slots, the last block's epilogue and the tail of spec s - 1
        // (early groups) and the roofline and features of spec s + 1 (late
        // groups), so that no VALU work of a spec stands outside the MFMA
        // stream.  Spec s - 1's last-block accumulators and layer-3 partial
        // sums live on in the head state (p0/p1, zp) until its epilogue
        // has read them.
        using S4 = typename H::S4;
        S4 st;
        H::init_state(st);
        // specs s_lo + s, s = 0 .. S - 1
        const int S = s_hi - s_lo;
        SpecC sc = spec_at(p.spec_c, s_lo);
        Roof o = small ? roofline<true>(rc, sc) : roofline<false>(rc, sc);
        constexpr int KC1 = H::KC1;
        u32x4 XB[2][KC1];
        {
          float x[IN];
          features<IN, H::kRaw>(rc, sc, o, x);
          H::pack_x(x, XB);
        }
        float zp[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        float tr_prev = 0.0f, t0_prev = 0.0f;
        // one spec's groups; NEXT: whether a next spec exists (the last
        // spec's groups are a second copy without the next spec's work)
        auto spec_iter = [&](int s, auto next_c) {
          constexpr bool NEXT = decltype(next_c)::value;
          const SpecC sn = spec_at(p.spec_c, s_lo + (NEXT ? s + 1 : s));
          Roof on;
          u32x4 XBn[2][KC1];
          float xn[IN];
          float eta_prev = 1.0f;
          const float tr_cur = o.t_roof, t0_cur = sc.t0;
          H::begin_spec(st, XB, lds, zp);
          // after each group, its share of the neighbouring specs' work
          // (hook_at)
          auto hook = [&](auto ic) {
            constexpr int I = decltype(ic)::value;
            constexpr typename H::Hook a = H::hook_at(I);
            if constexpr (a.tp1 > a.tp0) H::tail_pairs(st, zp, a.tp0, a.tp1);
            if constexpr (a.eta) eta_prev = 1.0f + __expf(-H::tail_reduce(zp, lds));
            if constexpr (a.tail) {
              if (s > 0)
                spec_tail<MULT>(p, s_lo + s - 1, tr_prev, eta_prev, fmaxf(tr_prev * eta_prev, t0_prev), valid, live,
                                row, tfac, fac, dst);
            }
            if constexpr (NEXT && a.roof) on = small ? roofline<true>(rc, sn) : roofline<false>(rc, sn);
            if constexpr (NEXT && a.feat != 0u) {
#pragma unroll
              for (int i = 0; i < 16; ++i)
                if ((a.feat >> i) & 1u) xn[i] = feature<H::kRaw>(i, rc, sn, on);
            }
            if constexpr (NEXT && a.sq1 > a.sq0) {
#pragma unroll
              for (int i = a.sq0; i < a.sq1; ++i) xn[16 + i] = xn[i] * xn[i];
            }
            if constexpr (NEXT && a.pk1 > a.pk0) H::pack_x(xn, XBn, a.pk0, a.pk1);
          };
          H::run_groups(st, lds, hook);
          tr_prev = tr_cur;
          t0_prev = t0_cur;
          if constexpr (NEXT) {
            o = on;
            sc = sn;
#pragma unroll
            for (int kc = 0; kc < KC1; ++kc) {
              XB[0][kc] = XBn[0][kc];
              XB[1][kc] = XBn[1][kc];
            }
          }
        };
        for (int s = 0; s + 1 < S; ++s) spec_iter(s, std::true_type{});
        spec_iter(S - 1, std::false_type{});
        // the last spec's epilogue and tail
        float zl[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) zl[j] = st.zacc[j];
        H::tail_pairs(st, zl, 0, 4);
        H::tail_pairs(st, zl, 4, 8);
        const float eta = 1.0f + __expf(-H::tail_reduce(zl, lds));
        spec_tail<MULT>(p, s_lo + S - 1, tr_prev, eta, fmaxf(tr_prev * eta, t0_prev), valid, live, row, tfac, fac,
                        dst);
        continue;
      }
    }
    for (int s = s_lo; s < s_hi; ++s) {
      const SpecC sc = spec_at(p.spec_c, s);
      const Roof o = small ? roofline<true>(rc, sc) : roofline<false>(rc, sc);
      float eta = 1.0f;
      // Tier B first: the family's other head runs only if some record of
      // the wave is not routed to the grid
      bool routed = false;
      float eta_g = 0.0f;
      if (grd) eta_g = grid_eta(rc, sc, o, p, grid_lds, routed);
      const bool other = !grd || __ballot(valid && !routed) != 0;
      if (bnd) {
        if (other) {
          float x[16];
          features<16>(rc, sc, o, x);
          eta = bounded_eta(x, o.W, bnd_lds);
        }
      } else {
        if constexpr (H::kMlp) {
          if (other) {
            float x[IN];
            features<IN, H::kRaw>(rc, sc, o, x);
            const float z = H::mlp(x, lds);
            eta = 1.0f + __expf(-z);
          }
        }
      }
      if (routed) eta = eta_g;
      const float t = fmaxf(o.t_roof * eta, sc.t0);
      // (without a grid the source is a per-family constant, written by
      // k_fill_source instead, so the plain kernels keep their registers)
      if constexpr (GRID) {
        if (valid && p.o_src) p.o_src[(size_t)s * (size_t)p.fam_off[KS_NFAM] + (size_t)row] = routed ? 2 : (bnd ? 1 : 0);
      }
      spec_tail<MULT>(p, s, o.t_roof, eta, t, valid, live, row, tfac, fac, dst);
    }
  }
}

// ------------------------------------------------------------ eta = 1 stream
// The pure roofline (eta = 1, Eq. 2), or the bounded head on its families,
// for every (spec, record) pair: its per-pair outputs and/or the step sums
// (Sec. 5.7).  A wave takes a workgroup tile on its own (256 consecutive
// records of one family: four 64-record tiles) and each lane four
// consecutive records of it, so that each 16-lane DPP row holds exactly one
// 64-record tile.  A lane loads its four records of a field with one
// 16-byte load, so the wave's load of a field covers the tile's 1 KB
// contiguously.  Per spec a lane writes its four records' per-pair outputs
// as one vector store each, and sums their t in runs of equal step (one FMA
// each); one
// segmented scan per row then joins the lanes' last runs, and each run's
// tail record adds the carry-in of the lanes before it.  The cross-lane
// work is thus per four records instead of per record.  Runs are split at
// the 64-record tile boundaries as in k_eval, and the partial sums, carries
// and record ranges are the ones k_eval writes, so k_finish reads either
// alike.
constexpr int kStreamR = 4;                       // records per lane
static_assert(kWave * kStreamR == kWgRows, "a wave of the stream takes one workgroup tile");
static_assert(kTileRows == 16 * kStreamR, "a 64-record tile is one 16-lane row");

// what a launch of the stream computes: step sums, per-pair outputs, and
// whether records carry multiplicities (step sums only)
enum : int { kStrSums = 1, kStrPair = 2, kStrMult = 4, kStrBnd = 8 };

// The bounded analytical head in the stream (families with their bounded
// bit; the others keep eta = 1).  Its two logits g . x and a . x are split
// into the spec-independent features (x0, x8 .. x15: one partial sum per
// record and logit, formed once per tile) and the spec-dependent ones (x1 ..
// x7, per spec); the parameters are read through the scalar cache.
struct SBnd {
  float zg[kStreamR], za[kStreamR];   // g . x and a . x over x0, x8 .. x15
  float la[kStreamR];                 // log2(F / max(Bt, 1))
  float bf[kStreamR];                 // B
  float rb[kStreamR];                 // 1 / max(B, 1)
  float rbt[kStreamR];                // 1 / max(Bt, 1)
};

__device__ __forceinline__ float bnd_param(const float *base, int i) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef const __attribute__((address_space(4))) float *CPtr;
  return ((CPtr)base)[i];
#else
  return base[i];
#endif
}

// fields a family's counts read besides step and n
constexpr bool uses_m(int fam) {
  return fam != KS_GROUPED_GEMM && fam != KS_ATTN_PREFILL && fam != KS_ATTN_DECODE;
}
constexpr bool uses_k(int fam) { return fam != KS_RMSNORM && fam != KS_SILU_MUL && fam != KS_EMBED; }
constexpr bool uses_a(int fam) {
  return fam == KS_GROUPED_GEMM || fam == KS_ATTN_PREFILL || fam == KS_ATTN_DECODE;
}
constexpr bool uses_b(int fam) { return fam == KS_GROUPED_GEMM; }
constexpr bool uses_field(int fam, int f) {
  return f == 0 || f == 2 || (f == 1 && uses_m(fam)) || (f == 3 && uses_k(fam)) || (f == 4 && uses_a(fam)) ||
         (f == 5 && uses_b(fam));
}
// a workgroup tile of the stream: family, first row, valid rows, first tile id
struct STile {
  int fam, nvalid, tile0;
  int64_t row0;
  bool hp, hn;   // a record of the family exists just before / after it
};

// workgroup tile wt, one of family fam's
__device__ __forceinline__ STile stream_locate(const EvalParams &p, int wt, int fam) {
  STile t;
  const int in_fam = wt - p.wgt_off[fam];
  const int64_t lo = p.fam_off[fam], hi = p.fam_off[fam + 1];
  t.fam = fam;
  t.row0 = lo + (int64_t)in_fam * kWgRows;
  const int64_t left = hi - t.row0;
  t.nvalid = left < kWgRows ? (int)left : kWgRows;
  t.tile0 = p.tile_off[fam] + in_fam * kWgWaves;
  t.hp = in_fam > 0;
  t.hn = left > kWgRows;
  return t;
}

// Inclusive segmented scan within each 16-lane row (row_shr 1, 2, 4, 8):
// v += g[i] * v[lane - 2^i], g[i] = 1 where that lane's key is this lane's
// (keys sorted, so the lanes between share it too).  Lanes without a source
// in the row read 0 (bound_ctrl) or are left out by the bank mask.
__device__ __forceinline__ float row_scan(float v, const float (&g)[4]) {
  asm volatile(
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %2 row_shr:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %3 row_shr:4 row_mask:0xf bank_mask:0xe\n"
      "s_nop 1\n"
      "v_fmac_f32_dpp %0, %0, %4 row_shr:8 row_mask:0xf bank_mask:0xc\n"
      : "+v"(v)
      : "v"(g[0]), "v"(g[1]), "v"(g[2]), "v"(g[3]));
  return v;
}

// Block counts below 2^22: the wave count W = ceil(B / N) in fp32 as the
// ceiling of (B - 1/2) fl(1/N).  B - 1/2 is exact, and the two roundings
// move the quotient by at most (B/N) (2^-23 + 2^-48) < 1/(2N), while
// (B - 1/2)/N lies at least 1/(2N) away from every integer (B and N are
// integers), so the ceiling is exact.
constexpr uint32_t kStreamSmallB = 1u << 22;

// What the spec loop needs of a lane's four records besides their roofline
// operands.  Runs never mix live and other records (those carry key
// kNoKey), so the t of a record that is not live never reaches a stored
// sum and needs no masking.  Per-record flags are bits of one word (bit j:
// record j) so that they take one register rather than a lane mask each.
struct SRec {
  uint32_t key[kStreamR];
  float fj[kStreamR];      // 1: record j continues the run of record j - 1
  float mf[kStreamR];      // the record's multiplicity (step sums with multiplicities)
  uint32_t off[kStreamR];  // with 32-bit offsets: byte offset of record j's sum slot from the spec-0 partial
  uint32_t ptail;          // bit j: record j ends a run within its 64-record tile
  uint32_t to_carry;       // bit j: ... and that run continues from the previous tile
  uint32_t first;          // bit j: record j is in the lane's first run
  float g[4], fc;          // row-scan factors; the lane's first run continues the lane before
  int tile;
};

// a lane's four consecutive records (4 lane .. 4 lane + 3 of the tile) of
// one field array, base: the tile's first record: one 16-byte load when the
// four are valid and the address is 16-byte aligned, else one load per
// record with its index clamped to the tile's valid rows (nvalid >= 1).
// The 16-byte loads are non-temporal: every record is read once per call.
__device__ __forceinline__ u32x4 load_quad(const uint32_t *base, int lane, int nvalid) {
  const uint32_t *q = reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(base) +
                                                         (uint32_t)(16 * lane));
  if (kStreamR * lane + kStreamR - 1 < nvalid && (reinterpret_cast<uintptr_t>(q) & 15) == 0)
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(q));
  u32x4 r;
#pragma unroll
  for (int j = 0; j < kStreamR; ++j) {
    const int i = kStreamR * lane + j;
    r[j] = base[i < nvalid ? i : nvalid - 1];
  }
  return r;
}

// four consecutive per-pair values of a lane (records 4 lane .. 4 lane + 3
// of the tile) at base + 4 lane (base: the tile's first record, the same
// for the whole wave, so the lane's part is a 32-bit offset): one 16-byte
// store (non-temporal: nothing here reads it back) when all four are valid
// and the address is 16-byte aligned, else one store per valid record
__device__ __forceinline__ void store_quad(float *base, int lane, int nvalid, const float (&v)[kStreamR]) {
  typedef float f32x4 __attribute__((ext_vector_type(4)));
  float *q = reinterpret_cast<float *>(reinterpret_cast<char *>(base) + (uint32_t)(16 * lane));
  if (kStreamR * lane + kStreamR - 1 < nvalid && (reinterpret_cast<uintptr_t>(q) & 15) == 0) {
    __builtin_nontemporal_store(f32x4{v[0], v[1], v[2], v[3]}, reinterpret_cast<f32x4 *>(q));
  } else {
#pragma unroll
    for (int j = 0; j < kStreamR; ++j)
      if (kStreamR * lane + j < nvalid) q[j] = v[j];
  }
}

// Spec loop.  W = ceil(B / N) as the ceiling of (B - 1/2) / N: in fp32 for
// block counts below 2^22 (as above), else in fp64, exact by the same
// argument below 2^51 (the exact path of k_eval assumes B < 2^52); then
// F u / P = W (F / B) (N / P), the first factor per record and the second
// per spec.  BH: B - 1/2 per record, as float or double; frb, btf: F / B
// and Bt per record.  part: the partials of the tile's family ([step][spec]).
// The sum slots are addressed as the spec's uniform base plus the records'
// 32-bit byte offsets r.off (the launcher takes this kernel for step sums
// only when the partial and carry regions span less than 4 GiB), so a spec
// costs no per-lane address arithmetic.  With one or two specs (BUF) a
// tail's sums are stored after the loop, both specs' in one 16-byte store
// (its slots are adjacent and 16-byte aligned); with more, each spec's as
// it is formed.
template <int VAR, bool BND, bool BUF, class BH>
__device__ __forceinline__ void stream_specs(const EvalParams &p, const STile &tc, int lane, const SRec &r,
                                             const BH (&bh)[kStreamR], const float (&frb)[kStreamR],
                                             const float (&btf)[kStreamR], double *part, bool any_tail,
                                             const SBnd &q, const float *prm) {
  constexpr bool SUMS = (VAR & kStrSums) != 0, PAIR = (VAR & kStrPair) != 0, MULT = (VAR & kStrMult) != 0;
  const size_t n_rows = (size_t)p.fam_off[KS_NFAM];
  // spec s: per-pair outputs, and (SUMS) each record's run sum so far in
  // v: a tail record's v is its stored sum
  auto spec = [&](int s, float (&v)[kStreamR]) {
    const SpecC sc = spec_at(p.spec_c, s);
    const float np = sc.n_f * sc.rcp_p;
    float t[kStreamR], tr[kStreamR], eta[kStreamR];
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) {
      float W;
      if constexpr (sizeof(BH) == sizeof(float))
        W = ceilf(bh[j] * sc.rcp_n);
      else
        W = (float)ceil(bh[j] * sc.rcp_nd);
      const float tc_ = W * (frb[j] * np), tm = btf[j] * sc.rcp_bw;
      tr[j] = fmaxf(tc_, tm);
      if constexpr (BND) {
        // x1 .. x7 of this spec (Sec. 5.3 feature list; u = W N / B, and
        // a record without blocks has u = 1), then the bounded head
#pragma clang fp contract(off)
        const float u = q.bf[j] > 0.0f ? W * sc.n_f * q.rb[j] : 1.0f;   // (1 / B for B >= 1)
        float x[8];
        x[1] = fmaxf(q.la[j] + sc.lr, -20.0f) * (1.0f / 16);
        x[2] = log2f_fast(fmaf(q.bf[j], sc.rcp_n, 1.0f)) * (1.0f / 16);
        x[3] = rcpf(u);
        x[4] = log2f_fast(1.0f + W) * (1.0f / 16);
        x[5] = fminf(1.0f, sc.l2 * q.rbt[j]);
        x[6] = log2f_fast(fmaxf(tr[j] * sc.rcp_t0, 0x1p-20f)) * (1.0f / 16);
        const float den = tc_ + tm;
        x[7] = den > 0.0f ? tc_ * rcpf(den) : 0.0f;
        float zg = q.zg[j], za = q.za[j];
#pragma unroll
        for (int i = 1; i < 8; ++i) {
          zg = fmaf(bnd_param(prm, i), x[i], zg);
          za = fmaf(bnd_param(prm, 16 + i), x[i], za);
        }
        const float w = fmaxf(W, 1.0f);
        const float eg = __expf(-zg), ea = __expf(-za);
        eta[j] = (1.0f + eg) * (w * (1.0f + ea)) * rcpf((w - 1.0f) + w * ea);
        t[j] = fmaxf(tr[j] * eta[j], sc.t0);
      } else {
        eta[j] = 1.0f;
        t[j] = fmaxf(tr[j], sc.t0);
      }
    }
    if constexpr (PAIR) {
      const size_t i0 = (size_t)s * n_rows + (size_t)tc.row0;
      if (p.o_troof) store_quad(p.o_troof + i0, lane, tc.nvalid, tr);
      if (p.o_eta) store_quad(p.o_eta + i0, lane, tc.nvalid, eta);
      if (p.o_t) store_quad(p.o_t + i0, lane, tc.nvalid, t);
    }
    if constexpr (SUMS) {
      float acc[kStreamR];
#pragma unroll
      for (int j = 0; j < kStreamR; ++j) {
        const float x = MULT ? t[j] * r.mf[j] : t[j];
        acc[j] = j == 0 ? x : fmaf(r.fj[j], acc[j - 1], x);
      }
      // the run ending at this lane's last record, over the row's lanes so far
      const float x = row_scan(acc[kStreamR - 1], r.g);
      // what the lanes before add to this lane's first run (0 at a row start)
      const float cin = r.fc * __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                                           0, __builtin_bit_cast(int, x), 0x111, 0xf, 0xf, true));
#pragma unroll
      for (int j = 0; j < kStreamR; ++j) v[j] = ((r.first >> j) & 1u) ? acc[j] + cin : acc[j];
    }
  };
  if constexpr (BUF && SUMS) {
    float v0[kStreamR], v1[kStreamR];
    spec(0, v0);
    const bool two = p.n_specs == 2;
    if (two) spec(1, v1);
    if (any_tail) {
      if (two) {
        typedef double f64x2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int j = 0; j < kStreamR; ++j)
          if ((r.ptail >> j) & 1u)
            *reinterpret_cast<f64x2 *>(reinterpret_cast<char *>(part) + r.off[j]) = f64x2{(double)v0[j], (double)v1[j]};
      } else {
#pragma unroll
        for (int j = 0; j < kStreamR; ++j)
          if ((r.ptail >> j) & 1u) *reinterpret_cast<double *>(reinterpret_cast<char *>(part) + r.off[j]) = (double)v0[j];
      }
    }
  } else {
    for (int s = 0; s < p.n_specs; ++s) {
      float v[kStreamR];
      spec(s, v);
      if constexpr (SUMS) {
        if (any_tail) {
#pragma unroll
          for (int j = 0; j < kStreamR; ++j)
            if ((r.ptail >> j) & 1u) *reinterpret_cast<double *>(reinterpret_cast<char *>(part + s) + r.off[j]) = (double)v[j];
        }
      }
    }
  }
}

// the spec loop's instance: bounded head or not, one or two specs (whose
// sums are stored after the loop) or more
template <int VAR, class BH>
__device__ __forceinline__ void stream_dispatch(const EvalParams &p, const STile &tc, int lane, const SRec &r,
                                                const BH (&bh)[kStreamR], const float (&frb)[kStreamR],
                                                const float (&btf)[kStreamR], double *part, bool any_tail,
                                                const SBnd &q, const float *prm, bool bnd) {
  constexpr bool B = (VAR & kStrBnd) != 0;
  if (p.n_specs <= 2) {
    if (bnd)
      stream_specs<VAR, B, true>(p, tc, lane, r, bh, frb, btf, part, any_tail, q, prm);
    else
      stream_specs<VAR, false, true>(p, tc, lane, r, bh, frb, btf, part, any_tail, q, prm);
  } else {
    if (bnd)
      stream_specs<VAR, B, false>(p, tc, lane, r, bh, frb, btf, part, any_tail, q, prm);
    else
      stream_specs<VAR, false, false>(p, tc, lane, r, bh, frb, btf, part, any_tail, q, prm);
  }
}

// A tile's loads: the lane's four records of each field its family uses
// (16 bytes per lane and field, so the wave's load of a field covers the
// tile contiguously; zero for the unused fields), the multiplicities, and
// the steps just before and after the tile (lane 0 and lane 1 of one load;
// each address inside the family: the tile's first row where a neighbour
// does not exist).
struct SLoad {
  u32x4 f[6];
  u32x4 mult;
  uint32_t pn;
};

template <int FAM, int VAR>
__device__ __forceinline__ void stream_load(const EvalParams &p, const STile &t, int lane, SLoad &o) {
  const uint32_t *src[6] = {p.step, p.m, p.n, p.k, p.a, p.b};
#pragma unroll
  for (int f = 0; f < 6; ++f) {
    o.f[f] = u32x4{0, 0, 0, 0};
    if (uses_field(FAM, f)) o.f[f] = load_quad(src[f] + t.row0, lane, t.nvalid);
  }
  if constexpr ((VAR & kStrMult) != 0) o.mult = load_quad(p.mult + t.row0, lane, t.nvalid);
  o.pn = 0;
  if constexpr ((VAR & kStrSums) != 0) {
    const int pn_off = lane == 0 ? (t.hp ? -1 : 0) : (t.hn ? kWgRows : 0);
    o.pn = (p.step + t.row0)[pn_off];
  }
}

// One workgroup tile of family FAM, its loads in `in`; rng and part: the
// family's range table and partials.
template <int FAM, int VAR>
__device__ __forceinline__ void stream_tile(const EvalParams &p, const STile &tc, int lane, uint32_t *rng,
                                            double *part, const SLoad &in) {
  constexpr bool SUMS = (VAR & kStrSums) != 0, PAIR = (VAR & kStrPair) != 0, MULT = (VAR & kStrMult) != 0;
  uint32_t v[6][kStreamR];
#pragma unroll
  for (int f = 0; f < 6; ++f) {
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) v[f][j] = uses_field(FAM, f) ? in.f[f][j] : 0u;
  }
  SRec r;
  if constexpr (MULT) {
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) r.mf[j] = (float)in.mult[j];   // exact below 2^24
  }
  const uint32_t pn = in.pn;

  // per record: counts and the spec-independent roofline operands; exact
  // (u64) when the per-record counts are written, else in fp32
  uint32_t bad = 0;
  bool live[kStreamR];
  bool big = false;
  uint64_t B[kStreamR];
  float Ff[kStreamR], Btf[kStreamR], Mf[kStreamR];
  // a step at or past n_steps (none can be when n_steps >= 2^32)
  const bool lim = p.n_steps <= (int64_t)UINT32_MAX;
  const uint32_t n_steps32 = (uint32_t)p.n_steps;
  const bool exact = PAIR && (p.o_flops || p.o_bytes || p.o_blocks);   // wave-uniform
#pragma unroll
  for (int j = 0; j < kStreamR; ++j) {
    const bool valid = kStreamR * lane + j < tc.nvalid;
    uint32_t b = 0;
    if (lim && v[0][j] >= n_steps32) b |= kErrStep;
    if (PAIR && exact) {
      const Cnt c = record_counts(FAM, v[1][j], v[2][j], v[3][j], v[4][j], v[5][j], v[0][j], p, b);
      if (valid) {
        const size_t row = (size_t)tc.row0 + (size_t)(kStreamR * lane + j);
        if (p.o_flops) p.o_flops[row] = c.F;
        if (p.o_bytes) p.o_bytes[row] = c.Bt;
        if (p.o_blocks) p.o_blocks[row] = c.B;
      }
      B[j] = c.B;
      Ff[j] = (float)c.F;
      Btf[j] = (float)c.Bt;
      Mf[j] = (float)c.M;
    } else {
      const CntF cf = record_counts_f(FAM, v[1][j], v[2][j], v[3][j], v[4][j], v[5][j], v[0][j], p, b);
      B[j] = cf.B;
      Ff[j] = cf.F;
      Btf[j] = cf.Bt;
      Mf[j] = cf.M;
    }
    if (valid) bad |= b;
    live[j] = valid && !(b & kErrStep);
    r.key[j] = live[j] ? v[0][j] : kNoKey;
    big |= B[j] >= kStreamSmallB;
  }
  if (bad) atomicOr(p.err, bad);
  const bool small = __ballot(big) == 0;   // wave-uniform

  bool any_tail = false;
  if constexpr (SUMS) {
    const uint32_t prev = tc.hp ? __builtin_amdgcn_readlane(pn, 0) : kNoKey;
    const uint32_t next = tc.hn ? __builtin_amdgcn_readlane(pn, 1) : kNoKey;
    // neighbours: the record before this lane's first (lane 0: the tile
    // edge) and after its last (lane 63: the tile edge)
    const uint32_t kp =
        (uint32_t)__builtin_amdgcn_update_dpp((int)prev, (int)r.key[kStreamR - 1], 0x138, 0xf, 0xf, false);
    const uint32_t kn = (uint32_t)__builtin_amdgcn_update_dpp((int)next, (int)r.key[0], 0x130, 0xf, 0xf, false);
    const int row_lane = lane & 15;
    r.tile = tc.tile0 + (lane >> 4);
    // the key of the row's first record and of the record before the row
    // (row_newbcast:0 gives each row its lane 0)
    const uint32_t rk0 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)r.key[0], 0x150, 0xf, 0xf, false);
    const uint32_t rkp = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)kp, 0x150, 0xf, 0xf, false);
    r.ptail = r.to_carry = r.first = 0;
    uint32_t heads = 0, ends = 0;   // bit j: record j starts / ends its (family, step) range
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) {
      const uint32_t key = r.key[j];
      const uint32_t before = j == 0 ? kp : r.key[j - 1];
      const uint32_t after = j == kStreamR - 1 ? kn : r.key[j + 1];
      r.fj[j] = j > 0 && key == before ? 1.0f : 0.0f;
      heads |= (live[j] && before != key ? 1u : 0u) << j;
      ends |= (live[j] && after != key ? 1u : 0u) << j;
      // a run's last record within its 64-record tile
      const bool pt = live[j] && (after != key || (j == kStreamR - 1 && row_lane == 15));
      r.ptail |= (pt ? 1u : 0u) << j;
      r.to_carry |= (key == rk0 && rkp == rk0 ? 1u : 0u) << j;
      r.first |= (key == r.key[0] ? 1u : 0u) << j;
    }
    // the (family, step) record range, written where its global first and
    // last records are
    const uint32_t row_l = (uint32_t)tc.row0 + (uint32_t)(kStreamR * lane);
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) {
      if ((heads >> j) & 1u) rng[2 * (size_t)r.key[j]] = row_l + j;
      if ((ends >> j) & 1u) rng[2 * (size_t)r.key[j] + 1] = row_l + j + 1;
    }
    any_tail = __ballot(r.ptail != 0) != 0;
    {
      // carries lie after the partials: their offset from this family's
      // partials is (carry - part) + tile S 8
      const uint32_t S8 = (uint32_t)p.n_specs * 8u;
      const uint32_t cbase = (uint32_t)((const char *)p.carry - (const char *)part) + (uint32_t)r.tile * S8;
#pragma unroll
      for (int j = 0; j < kStreamR; ++j) r.off[j] = ((r.to_carry >> j) & 1u) ? cbase : r.key[j] * S8;
    }
    r.fc = row_lane != 0 && kp == r.key[0] ? 1.0f : 0.0f;
    // row-scan factors on the lanes' last keys
    const uint32_t kl = r.key[kStreamR - 1];
    r.g[0] = dpp_key<0x111, 0xf, 0xf>(kl) == kl ? 1.0f : 0.0f;
    r.g[1] = dpp_key<0x112, 0xf, 0xf>(kl) == kl ? 1.0f : 0.0f;
    r.g[2] = dpp_key<0x114, 0xf, 0xe>(kl) == kl ? 1.0f : 0.0f;
    r.g[3] = dpp_key<0x118, 0xf, 0xc>(kl) == kl ? 1.0f : 0.0f;
  }
  // the bounded head's spec-independent part (families with their bit set)
  SBnd q;
  const float *prm = nullptr;
  const bool bnd = (VAR & kStrBnd) != 0 && ((p.bounded_mask >> FAM) & 1u);   // wave-uniform
  if constexpr ((VAR & kStrBnd) != 0) {
    if (bnd) {
      prm = p.bounded + FAM * 32;
      // read the parameters again in each tile rather than hold them in
      // scalar registers across the family's tiles
      asm volatile("" : "+s"(prm));
#pragma unroll
      for (int j = 0; j < kStreamR; ++j) {
#pragma clang fp contract(off)
        const float bf = (float)B[j];
        const float rb = rcpf(fmaxf(bf, 1.0f));
        q.bf[j] = bf;
        q.rb[j] = rb;
        q.rbt[j] = rcpf(fmaxf(Btf[j], 1.0f));
        // log2(0) = -inf for F = 0; the clamps of x0 and x1 take it
        q.la[j] = log2f_fast(Ff[j] * q.rbt[j]);
        float xi[9];
        xi[0] = fmaxf(q.la[j], -10.0f) * (1.0f / 16);
        xi[1] = log2f_fast(1.0f + Ff[j]) * (1.0f / 64);
        xi[2] = log2f_fast(1.0f + Btf[j]) * (1.0f / 48);
        xi[3] = log2f_fast(1.0f + Mf[j]) * (1.0f / 24);
        xi[4] = log2f_fast(1.0f + (float)v[2][j]) * (1.0f / 24);
        xi[5] = log2f_fast(1.0f + (float)v[3][j]) * (1.0f / 24);   // 0 for the families without K
        xi[6] = log2f_fast(1.0f + Ff[j] * rb) * (1.0f / 48);
        xi[7] = log2f_fast(1.0f + Btf[j] * rb) * (1.0f / 40);
        xi[8] = 1.0f;
        // x0, x8 .. x15 of the feature list: parameter indices 0, 8 .. 15
        float zg = bnd_param(prm, 0) * xi[0], za = bnd_param(prm, 16) * xi[0];
#pragma unroll
        for (int i = 1; i < 9; ++i) {
          zg = fmaf(bnd_param(prm, 7 + i), xi[i], zg);
          za = fmaf(bnd_param(prm, 23 + i), xi[i], za);
        }
        q.zg[j] = zg;
        q.za[j] = za;
      }
    }
  }
  float frb[kStreamR];
  if (small) {
    float bh[kStreamR];
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) {
      const float Bf = (float)(uint32_t)B[j];
      bh[j] = Bf - 0.5f;
      frb[j] = Ff[j] * rcpf(fmaxf(Bf, 1.0f));
    }
    stream_dispatch<VAR>(p, tc, lane, r, bh, frb, Btf, part, any_tail, q, prm, bnd);
  } else {
    double bh[kStreamR];
#pragma unroll
    for (int j = 0; j < kStreamR; ++j) {
      bh[j] = (double)B[j] - 0.5;
      frb[j] = Ff[j] * rcpf(fmaxf((float)B[j], 1.0f));
    }
    stream_dispatch<VAR>(p, tc, lane, r, bh, frb, Btf, part, any_tail, q, prm, bnd);
  }
}

// Waves per SIMD the register allocator must fit, at least: six for the
// plain step sums (seven spills and measured slower); the other variants
// take what their registers allow.
template <int VAR> struct StreamOcc {
  static constexpr int value =
      VAR == kStrSums ? 6 : ((VAR & kStrBnd) && (VAR & kStrSums) && (VAR & kStrPair) ? 3 : 4);
};

// The wave's tiles of family FAM, from tile wt on in steps of stride (wt
// advances past them).  Looping over one family at a time keeps the
// family's constants and code out of the other families' loops (fewer live
// registers than dispatching on the family per tile); issuing a tile's
// loads a tile ahead measured no faster.
template <int FAM, int VAR>
__device__ __forceinline__ void stream_family(const EvalParams &p, int &wt, int stride, int lane) {
  const int end = p.wgt_off[FAM + 1];
  if (wt >= end) return;
  uint32_t *rng = nullptr;
  double *part = nullptr;
  if constexpr ((VAR & kStrSums) != 0) {
    rng = p.range + 2 * (size_t)FAM * (size_t)p.n_steps;
    part = p.partial + (size_t)FAM * (size_t)p.n_steps * (size_t)p.n_specs;
  }
  for (; wt < end; wt += stride) {
    const STile t = stream_locate(p, wt, FAM);
    SLoad in;
    stream_load<FAM, VAR>(p, t, lane, in);
    stream_tile<FAM, VAR>(p, t, lane, rng, part, in);
  }
}

template <int VAR>
__global__ __launch_bounds__(kWgThreads) __attribute__((amdgpu_waves_per_eu(StreamOcc<VAR>::value)))
void k_stream(EvalParams p) {
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int stride = (int)gridDim.x * kWgWaves;
  // Workgroups go to the eight XCDs round-robin (workgroup b to XCD b mod
  // 8).  With step sums they are renumbered so that each XCD takes one
  // contiguous eighth of the tiles of every pass over the grid: the partial
  // sums and record ranges of consecutive steps (several to a cache line)
  // are then written from one XCD's L2 instead of up to eight, each holding
  // a partial line (per-pair outputs alone measured faster without it).
  int b = (int)blockIdx.x;
  if ((VAR & kStrSums) != 0 && (gridDim.x & 7u) == 0u) b = (b & 7) * (int)(gridDim.x >> 3) + (b >> 3);
  int wt = b * kWgWaves + wave;
  stream_family<KS_GEMM, VAR>(p, wt, stride, lane);
  stream_family<KS_LM_HEAD, VAR>(p, wt, stride, lane);
  stream_family<KS_GROUPED_GEMM, VAR>(p, wt, stride, lane);
  stream_family<KS_ATTN_PREFILL, VAR>(p, wt, stride, lane);
  stream_family<KS_ATTN_DECODE, VAR>(p, wt, stride, lane);
  stream_family<KS_RMSNORM, VAR>(p, wt, stride, lane);
  stream_family<KS_ROPE, VAR>(p, wt, stride, lane);
  stream_family<KS_SILU_MUL, VAR>(p, wt, stride, lane);
  stream_family<KS_KV_WRITE, VAR>(p, wt, stride, lane);
  stream_family<KS_EMBED, VAR>(p, wt, stride, lane);
  static_assert(KS_EMBED == KS_NFAM - 1, "every family has its loop");
}

// ------------------------------------------------------------ eta source
// Per pair, where eta came from when no grid routes any pair: 1 for the
// families on the bounded head, 0 (the head of the mode) for the others.
__global__ void k_fill_source(uint8_t *src, EvalParams p) {
  const int64_t n_rows = p.fam_off[KS_NFAM];
  const int64_t total = (int64_t)p.n_specs * n_rows;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t row = i % n_rows;
    int f = 0;
    while (row >= p.fam_off[f + 1]) ++f;
    src[i] = (uint8_t)((p.bounded_mask >> f) & 1u);
  }
}

// ------------------------------------------------------------ step finish
// per (spec, step): t_body, t_comm (Eq. 3, two all-reduces per layer),
// t_gpu and t_step (Eq. 4).  The partial sums are spec-minor and the
// outputs step-minor, so a workgroup takes a tile of kFinSteps steps x
// kFinSpecs specs (kFinSpecs a power of two, at least the spec count or
// 16): it reads with the spec fastest, passes the three results through
// LDS, and writes with the step fastest.
constexpr int kFinThreads = 256;

__global__ __launch_bounds__(kFinThreads) void k_finish(FinishParams p, int spec_bits) {
  __shared__ double res[3][kFinThreads];
  const int tps = 1 << spec_bits;                 // specs per tile
  const int tst = kFinThreads >> spec_bits;        // steps per tile
  const int64_t n_st = (p.n_steps + tst - 1) / tst;
  const int64_t n_sp = (p.n_specs + tps - 1) / tps;
  const int tid = threadIdx.x;
  for (int64_t tile = blockIdx.x; tile < n_st * n_sp; tile += gridDim.x) {
    const int64_t j0 = (tile % n_st) * tst;
    const int s0 = (int)(tile / n_st) * tps;
    // phase 1: thread (step jj, spec ss), spec fastest
    {
      const int ss = tid & (tps - 1), jj = tid >> spec_bits;
      const int s = s0 + ss;
      const int64_t j = j0 + jj;
      if (s < p.n_specs && j < p.n_steps) {
        const size_t S = (size_t)p.n_specs;
        // every family's range, then its partial and first carry, are
        // loaded before any is summed (independent loads in flight together
        // instead of a chain of ten); the sum keeps family order: partial,
        // then the carries of its later tiles
        uint32_t r0[KS_NFAM], r1[KS_NFAM];
#pragma unroll
        for (int f = 0; f < KS_NFAM; ++f) {
          r0[f] = p.range[2 * (f * p.n_steps + j)];
          r1[f] = p.range[2 * (f * p.n_steps + j) + 1];
        }
        bool any[KS_NFAM];
        int t_first[KS_NFAM], t_last[KS_NFAM];
        double part[KS_NFAM], car1[KS_NFAM];
#pragma unroll
        for (int f = 0; f < KS_NFAM; ++f) {
          // clamped to the family's rows: a range left half-written by
          // unsorted input (reported by ks_validate) still indexes only this
          // family's tiles
          const int64_t base = p.fam_off[f], top = p.fam_off[f + 1];
          int64_t a = r0[f], b = r1[f];
          a = a < base ? base : (a > top ? top : a);
          b = b < base ? base : (b > top ? top : b);
          any[f] = a < b;
          t_first[f] = any[f] ? p.tile_off[f] + (int)((a - base) / kTileRows) : 0;
          t_last[f] = any[f] ? p.tile_off[f] + (int)((b - 1 - base) / kTileRows) : 0;
          part[f] = any[f] ? p.partial[((size_t)f * (size_t)p.n_steps + (size_t)j) * S + s] : 0.0;
          car1[f] = t_last[f] > t_first[f] ? p.carry[(size_t)(t_first[f] + 1) * S + s] : 0.0;
        }
        double body = 0.0;
#pragma unroll
        for (int f = 0; f < KS_NFAM; ++f) {
          if (!any[f]) continue;
          body += part[f];
          if (t_last[f] > t_first[f]) body += car1[f];
          for (int t = t_first[f] + 2; t <= t_last[f]; ++t) body += p.carry[(size_t)t * S + s];
        }
        const ks_spec sp = p.specs[s];
        const double P = (double)p.tp[j];
        const double Sb = (double)p.agg[j] * (double)p.hidden[j] * (double)p.elem_bytes;
        double t_ar = 0.0;
        if (P > 1.0)
          t_ar = sp.ar_alpha0 + sp.ar_alpha_log2p * log2(P) + 2.0 * (P - 1.0) / P * Sb / sp.ar_beta;
        const double comm = 2.0 * (double)p.layers[j] * t_ar;
        const double gpu = p.host.body_scale * body + comm;
        const double step = fmax(gpu + (double)p.n_launch[j] * p.host.c_disp, p.host.ell) +
                            fmax(0.0, p.host.c_ovl - gpu) + p.host.c_tail;
        res[0][ss * tst + jj] = body;
        res[1][ss * tst + jj] = gpu;
        res[2][ss * tst + jj] = step;
      }
    }
    __syncthreads();
    // phase 2: thread (spec ss, step jj), step fastest
    {
      const int jj = tid % tst, ss = tid / tst;
      const int s = s0 + ss;
      const int64_t j = j0 + jj;
      if (s < p.n_specs && j < p.n_steps) {
        const size_t o = (size_t)s * (size_t)p.n_steps + (size_t)j;
        p.t_body[o] = res[0][ss * tst + jj];
        p.t_gpu[o] = res[1][ss * tst + jj];
        p.t_step[o] = res[2][ss * tst + jj];
        if (p.own && p.own[j] == (uint32_t)s) p.lat[j] = res[2][ss * tst + jj];
      }
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------ validation
__global__ void k_validate(ValidateParams p) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t t0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  uint32_t bad = 0;
  for (int64_t i = t0; i < p.n_rows; i += stride) {
    int f = 0;
    while (i >= p.fam_off[f + 1]) ++f;
    const uint32_t st = p.step[i];
    if ((int64_t)st >= p.n_steps) bad |= kErrStep;
    if (i > p.fam_off[f] && p.step[i - 1] > st) bad |= kErrOrder;
    const uint32_t m = p.m[i], n = p.n[i], k = p.k[i], a = p.a[i], b = p.b[i];
    if (m >= (1u << 24) || n >= (1u << 18) || k >= (1u << 18)) bad |= kErrRange;
    if (p.mult && p.mult[i] >= (1u << 24)) bad |= kErrRange;
    if ((f == KS_ATTN_PREFILL || f == KS_ATTN_DECODE) && (n >= 4096u || k >= 4096u || a >= 4096u))
      bad |= kErrRange;
    if (f == KS_GROUPED_GEMM) {
      if (a > 1024u || (uint64_t)b + a > (uint64_t)p.n_expert_rows) {
        bad |= kErrExpert;
      } else {
        uint64_t ms, act, tiles;
        expert_sums(p.expert_rows, b, a, ms, act, tiles);
        if (ms >= (1ull << 24)) bad |= kErrRange;
      }
    }
  }
  for (int64_t j = t0; j < p.n_steps; j += stride) {
    if (p.req_off[j] > p.req_off[j + 1] || (int64_t)p.req_off[j + 1] > p.n_req) bad |= kErrReq;
    if (p.agg[2 * p.n_steps + j] >= (1ull << 40)) bad |= kErrRange;
    if (p.tp && p.tp[j] < 1u) bad |= kErrRange;
  }
  if (t0 == 0 && p.n_steps > 0 && p.req_off[0] != 0) bad |= kErrReq;
  for (int64_t r = t0; r < p.n_req; r += stride)
    if (p.req_q[r] >= (1u << 24) || p.req_h[r] >= (1u << 24)) bad |= kErrRange;
  for (int64_t s = t0; s < p.n_specs; s += stride) {
    const ks_spec sp = p.specs[s];
    const bool ok = sp.peak_flops > 0.0 && sp.peak_flops < 1e30 && sp.hbm_bw > 0.0 && sp.hbm_bw < 1e30 &&
                    sp.t0 >= 0.0 && sp.t0 < 1e3 && sp.l2_bytes >= 0.0 && sp.l2_bytes < 1e30 &&
                    sp.ar_beta > 0.0 && sp.ar_beta < 1e30 && sp.ar_alpha0 >= 0.0 && sp.ar_alpha0 < 1e3 &&
                    sp.ar_alpha_log2p >= 0.0 && sp.ar_alpha_log2p < 1e3 && sp.n_cu >= 1u && sp.n_cu <= 65535u;
    if (!ok) bad |= kErrSpec;
  }
  if (bad) atomicOr(p.err, bad);
}

// ------------------------------------------------------------ launchers
static int grid_for(int64_t n, int block, int cap) {
  int64_t g = (n + block - 1) / block;
  if (g < 1) g = 1;
  return (int)(g < cap ? g : cap);
}

hipError_t launch_clear(uint32_t *err, uint32_t *range, int64_t n_range, hipStream_t s) {
  hipLaunchKernelGGL(k_clear, dim3(grid_for(n_range, 256, 2048)), dim3(256), 0, s, err, range, n_range,
                     (const ks_spec *)nullptr, 0, (SpecC *)nullptr);
  return hipGetLastError();
}

hipError_t launch_attn_agg(const uint32_t *req_off, const uint32_t *q, const uint32_t *h, int64_t n_steps,
                           int64_t n_req, uint64_t *agg, uint32_t *err, hipStream_t s) {
  if (n_steps == 0) return hipSuccess;
  hipLaunchKernelGGL(k_attn_agg, dim3(grid_for(n_steps, 256 / kAggLanes, 8192)), dim3(256), 0, s, req_off, q, h,
                     n_steps, n_req, agg, err);
  return hipGetLastError();
}

hipError_t launch_spec_prep(const ks_spec *specs, int32_t n_specs, SpecC *out, uint32_t *err, hipStream_t s) {
  hipLaunchKernelGGL(k_spec_prep, dim3(grid_for(n_specs, 256, 4096)), dim3(256), 0, s, specs, n_specs, out, err);
  return hipGetLastError();
}

// up to this many specs the clear kernel's first workgroup forms the spec
// constants (one launch less); more take their own grid
constexpr int32_t kFusedSpecs = 1024;

hipError_t launch_clear_prep(uint32_t *err, uint32_t *range, int64_t n_range, const ks_spec *specs,
                             int32_t n_specs, SpecC *out, hipStream_t s) {
  const bool fused = n_specs <= kFusedSpecs;
  hipLaunchKernelGGL(k_clear, dim3(grid_for(n_range, 256, 2048)), dim3(256), 0, s, err, range, n_range, specs,
                     fused ? n_specs : 0, out);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || fused) return e;
  return launch_spec_prep(specs, n_specs, out, err, s);
}

// The persistent grid: as many workgroups as are resident at once (the
// occupancy the compiled kernel's registers and LDS allow, times the CU
// count), so no workgroup of the head kinds waits for another to finish.
// Cached per device and kernel.
constexpr int kMaxDevices = 64;
static std::atomic<int> g_resident[kMaxDevices][kNumKinds][kNumVars];

template <int KIND, int VAR>
static hipError_t resident_wgs(int *out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::atomic<int> *slot = dev < kMaxDevices ? &g_resident[dev][KIND][VAR] : nullptr;
  int r = slot ? slot->load(std::memory_order_relaxed) : 0;
  if (r == 0) {
    int per_cu = 0, n_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_eval<KIND, VAR>, kWgThreads, 0);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    r = (per_cu < 1 ? 1 : per_cu) * (n_cu < 1 ? 1 : n_cu);
    if (slot) slot->store(r, std::memory_order_relaxed);
  }
  *out = r;
  return hipSuccess;
}

template <int KIND, int VAR>
static hipError_t launch_grid(const EvalParams &p, hipStream_t s) {
  int cap = 0;
  const hipError_t e = resident_wgs<KIND, VAR>(&cap);
  if (e != hipSuccess) return e;
  const int n_wgt = p.wgt_off[KS_NFAM];
  // Too few record tiles to fill the GPU (e.g. one serving round of many
  // spec vectors): split the spec loop into ranges, each a work item of its
  // own, so that ranges of the same tile run on different CUs.  The sums
  // and outputs of different specs are disjoint; the record ranges are
  // written alike by every range.
  EvalParams q = p;
  q.spec_chunk = p.n_specs;
  q.n_chunks = 1;
  if (n_wgt < cap && p.n_specs > 1) {
    const int want = (cap + n_wgt - 1) / n_wgt;
    const int chunks = want < p.n_specs ? want : p.n_specs;
    q.spec_chunk = (p.n_specs + chunks - 1) / chunks;
    q.n_chunks = (p.n_specs + q.spec_chunk - 1) / q.spec_chunk;
  }
  const int64_t work = (int64_t)n_wgt * q.n_chunks;
  const int grid = work < cap ? (int)work : cap;
  hipLaunchKernelGGL((k_eval<KIND, VAR>), dim3(grid), dim3(kWgThreads), 0, s, q);
  return hipGetLastError();
}

// k_stream: every eta = 1 evaluation (per-pair outputs and/or step sums,
// with or without multiplicities); grid-stride over workgroup tiles, one
// per wave.  As many workgroups as are resident, cached per device and
// variant.
constexpr int kNumStreamVars = 16;
// Workgroups per CU of a variant, at most (0: as many as are resident):
// the per-pair outputs alone fit seven waves per SIMD in registers and
// measured faster at five.
template <int VAR> struct StreamWgCap {
  static constexpr int value = VAR == kStrPair ? 5 : 0;
};
static std::atomic<int> g_stream_resident[kMaxDevices][kNumStreamVars];

template <int VAR>
static hipError_t launch_stream(const EvalParams &p, hipStream_t s) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::atomic<int> *slot = dev < kMaxDevices ? &g_stream_resident[dev][VAR] : nullptr;
  int cap = slot ? slot->load(std::memory_order_relaxed) : 0;
  if (cap == 0) {
    int per_cu = 0, n_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_stream<VAR>, kWgThreads, 0);
    if (e != hipSuccess) return e;
    e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    if (StreamWgCap<VAR>::value > 0 && per_cu > StreamWgCap<VAR>::value) per_cu = StreamWgCap<VAR>::value;
    cap = (per_cu < 1 ? 1 : per_cu) * (n_cu < 1 ? 1 : n_cu);
    if (slot) slot->store(cap, std::memory_order_relaxed);
  }
  const int n_wgt = p.wgt_off[KS_NFAM];
  const int need = (n_wgt + kWgWaves - 1) / kWgWaves;
  hipLaunchKernelGGL((k_stream<VAR>), dim3(need < cap ? need : cap), dim3(kWgThreads), 0, s, p);
  return hipGetLastError();
}

// eta = 1 (no bounded or grid family: those select the head-less kind)
template <int KIND>
static hipError_t launch_kind(const EvalParams &p, hipStream_t s);

static hipError_t launch_eta_one(const EvalParams &p, hipStream_t s) {
  if (p.grid_mask || p.bounded_mask) return hipErrorInvalidValue;
  // the stream addresses the sum slots by 32-bit offsets from the partials:
  // step sums whose partial and carry regions (carries after partials) span
  // 4 GiB or more take the one-record-per-lane kernel instead (its
  // head-less kind without bounded or grid families is eta = 1)
  if (p.partial) {
    const bool after = p.carry > p.partial;
    const uint64_t span = after ? (uint64_t)((const char *)p.carry - (const char *)p.partial) +
                                      (uint64_t)p.n_tiles * (uint64_t)p.n_specs * sizeof(double)
                                : ~0ull;
    if (span >= (1ull << 32)) return launch_kind<kBoundedOnly>(p, s);
  }
  const bool sums = p.partial && p.range;
  const bool pair = p.o_flops || p.o_bytes || p.o_blocks || p.o_troof || p.o_eta || p.o_t;
  // multiplicities matter only for the step sums
  const bool mult = sums && p.mult;
  if (!sums) return launch_stream<kStrPair>(p, s);
  if (mult) return pair ? launch_stream<kStrSums | kStrPair | kStrMult>(p, s) : launch_stream<kStrSums | kStrMult>(p, s);
  return pair ? launch_stream<kStrSums | kStrPair>(p, s) : launch_stream<kStrSums>(p, s);
}

// no MLP family and no grid: the bounded families and eta = 1 for the rest,
// on the stream (same 4 GiB condition for the sum slots)
static hipError_t launch_bounded_stream(const EvalParams &p, hipStream_t s) {
  if (p.partial) {
    const bool after = p.carry > p.partial;
    const uint64_t span = after ? (uint64_t)((const char *)p.carry - (const char *)p.partial) +
                                      (uint64_t)p.n_tiles * (uint64_t)p.n_specs * sizeof(double)
                                : ~0ull;
    if (span >= (1ull << 32)) return launch_kind<kBoundedOnly>(p, s);
  }
  const bool sums = p.partial && p.range;
  const bool pair = p.o_flops || p.o_bytes || p.o_blocks || p.o_troof || p.o_eta || p.o_t;
  const bool mult = sums && p.mult;
  constexpr int B = kStrBnd;
  if (!sums) return launch_stream<B | kStrPair>(p, s);
  if (mult)
    return pair ? launch_stream<B | kStrSums | kStrPair | kStrMult>(p, s) : launch_stream<B | kStrSums | kStrMult>(p, s);
  return pair ? launch_stream<B | kStrSums | kStrPair>(p, s) : launch_stream<B | kStrSums>(p, s);
}

template <int KIND>
static hipError_t launch_kind(const EvalParams &p, hipStream_t s) {
  // multiplicities matter only for the step sums
  const bool mult = p.mult && p.partial;
  if (p.grid_mask)
    return mult ? launch_grid<KIND, kVarGrid | kVarMult>(p, s) : launch_grid<KIND, kVarGrid>(p, s);
  return mult ? launch_grid<KIND, kVarMult>(p, s) : launch_grid<KIND, 0>(p, s);
}

hipError_t launch_eval(int kind, const EvalParams &p, hipStream_t s) {
  if (p.wgt_off[KS_NFAM] == 0) return hipSuccess;
  switch (kind) {
    case kEtaOne: return launch_eta_one(p, s);
    case kBoundedOnly: return p.grid_mask ? launch_kind<kBoundedOnly>(p, s) : launch_bounded_stream(p, s);
    case kF32_16_64: return launch_kind<kF32_16_64>(p, s);
    case kF32_16_128: return launch_kind<kF32_16_128>(p, s);
    case kF32_32_64: return launch_kind<kF32_32_64>(p, s);
    case kF32_32_128: return launch_kind<kF32_32_128>(p, s);
    case kBF16_16_64: return launch_kind<kBF16_16_64>(p, s);
    case kBF16_16_128: return launch_kind<kBF16_16_128>(p, s);
    case kBF16_16_256: return launch_kind<kBF16_16_256>(p, s);
    case kBF16_32_64: return launch_kind<kBF16_32_64>(p, s);
    case kBF16_32_128: return launch_kind<kBF16_32_128>(p, s);
    case kBF16_32_256: return launch_kind<kBF16_32_256>(p, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_fill_source(const EvalParams &p, hipStream_t s) {
  const int64_t total = (int64_t)p.n_specs * p.fam_off[KS_NFAM];
  if (!p.o_src || total == 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_source, dim3(grid_for(total, 256, 8192)), dim3(256), 0, s, p.o_src, p);
  return hipGetLastError();
}

hipError_t launch_finish(const FinishParams &p, hipStream_t s) {
  if (p.n_steps == 0) return hipSuccess;
  int bits = 0;   // specs per tile: the spec count rounded up to a power of two, at most 16
  while (bits < 4 && (1 << bits) < p.n_specs) ++bits;
  const int64_t tiles = ((p.n_steps + (kFinThreads >> bits) - 1) / (kFinThreads >> bits)) *
                        (((int64_t)p.n_specs + (1 << bits) - 1) >> bits);
  hipLaunchKernelGGL(k_finish, dim3(grid_for(tiles, 1, 8192)), dim3(kFinThreads), 0, s, p, bits);
  return hipGetLastError();
}

hipError_t launch_validate(const ValidateParams &p, hipStream_t s) {
  hipLaunchKernelGGL(k_validate, dim3(1024), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace ks
