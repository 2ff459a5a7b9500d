// Batch expansion on gfx950: the batch descriptors of consecutive steps
// (request lists, prefill flags) -> the records of every kernel each step
// dispatches, family-major, in the layout the evaluation kernel streams
// (Sec. 4.1: the scheduler's batch descriptor; Sec. 5.7: one embedding and
// one LM head per step around L homogeneous layers; Sec. 5.8: GEMMs, norms
// and activations over the step's T tokens, attention over its requests).
//
//   k_expand_steps    per step: T = sum q_r (16 lanes per step), the
//                     per-step model record (L, D, P, launches)
//   k_expand_rank     per block of 1024 steps: each step's count of earlier
//                     prefill steps in the block, and the block's total
//   k_expand_scan     one workgroup: exclusive prefix of the block totals
//                     (and their sum checked against n_prefill)
//   k_expand_records  one thread per record: step and slot from the item
//                     index, fields from the family's templates, stores to
//                     the record arrays (HBM write stream)
//   k_expand_small    all of the above (and the flag reset) in one
//                     workgroup, for batches of at most 1024 steps and 16k
//                     records (a serving round): one launch instead of five
#include <hip/hip_runtime.h>

#include "ks_internal.h"

namespace ks {

constexpr int kTokLanes = 16;

// steps g0, g0 + groups, ... (one group of kTokLanes lanes, lane sub)
__device__ __forceinline__ void expand_steps(const ExpandParams &p, int64_t g0, int64_t groups, int sub) {
  uint32_t bad = 0;
  for (int64_t j = g0; j < p.n_steps; j += groups) {
    uint32_t r0 = p.req_off[j], r1 = p.req_off[j + 1];
    if (r0 > r1 || (int64_t)r1 > p.n_req || (j == 0 && r0 != 0)) {
      bad |= kErrReq;
      r0 = r1 = 0;
    }
    uint64_t T = 0;
    for (uint32_t r = r0 + sub; r < r1; r += kTokLanes) T += p.req_q[r];
#pragma unroll
    for (int off = kTokLanes / 2; off > 0; off >>= 1) T += __shfl_xor(T, off);
    if (sub == 0) {
      // T and top_k T feed record m fields (limit 2^24)
      const uint64_t k = p.top_k > 1 ? p.top_k : 1;
      if (T * k >= (1ull << 24)) bad |= kErrRange;
      p.tok[j] = T >= (1ull << 32) ? 0xFFFFFFFFu : (uint32_t)T;
      const bool pre = p.prefill[j] != 0;
      p.o_layers[j] = p.L;
      p.o_hidden[j] = p.D;
      p.o_tp[j] = p.P;
      p.o_nlaunch[j] = pre ? p.L : 0u;
    }
  }
  if (bad) atomicOr(p.err, bad);
}

__global__ __launch_bounds__(256) void k_expand_steps(ExpandParams p) {
  expand_steps(p, ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / kTokLanes,
               ((int64_t)gridDim.x * blockDim.x) / kTokLanes, threadIdx.x & (kTokLanes - 1));
}

// In-block exclusive prefix of the prefill flags: thread t of block b owns
// steps b 1024 + 4 t .. + 3.
__device__ __forceinline__ void expand_rank(const ExpandParams &p, int64_t blk) {
  __shared__ uint32_t wsum[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t j0 = blk * kExpandBlk + 4 * tid;
  uint32_t fl[4], cnt = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    fl[i] = (j0 + i < p.n_steps && p.prefill[j0 + i] != 0) ? 1u : 0u;
    cnt += fl[i];
  }
  uint32_t incl = cnt;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t v = __shfl_up(incl, off);
    if (lane >= off) incl += v;
  }
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  uint32_t base = 0;
  for (int w = 0; w < wave; ++w) base += wsum[w];
  uint32_t excl = base + incl - cnt;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (j0 + i < p.n_steps) p.rank[j0 + i] = excl;
    excl += fl[i];
  }
  if (tid == 255) p.blk[blk] = excl;
}

__global__ __launch_bounds__(256) void k_expand_rank(ExpandParams p) { expand_rank(p, blockIdx.x); }

// Exclusive prefix of the block totals in place, 256 at a time; the grand
// total must equal the batch's n_prefill.
__device__ __forceinline__ void expand_scan(const ExpandParams &p) {
  __shared__ uint32_t wsum[4];
  __shared__ uint64_t carry_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  uint64_t carry = 0;
  for (int64_t c0 = 0; c0 < p.n_blk; c0 += 256) {
    const int64_t i = c0 + tid;
    const uint32_t v = i < p.n_blk ? p.blk[i] : 0u;
    uint32_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t u = __shfl_up(incl, off);
      if (lane >= off) incl += u;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t base = 0;
    for (int w = 0; w < wave; ++w) base += wsum[w];
    if (i < p.n_blk) p.blk[i] = (uint32_t)(carry + base + incl - v);
    if (tid == 255) carry_s = carry + base + incl;
    __syncthreads();
    carry = carry_s;
    __syncthreads();
  }
  if (tid == 0 && (int64_t)carry != p.n_prefill) atomicOr(p.err, kErrPrefill);
}

__global__ __launch_bounds__(256) void k_expand_scan(ExpandParams p) { expand_scan(p); }

// One record per item.  Attention items are the (step, layer) pairs of all
// steps: a prefill step's go to ATTN_PREFILL at its rank among prefill
// steps, the others to ATTN_DECODE at their rank among the rest (an item
// whose rank is beyond the family's records, when the flags disagree with
// n_prefill, is not written).
//
// A workgroup pass covers one 256-item chunk of one family, so the family,
// its templates and its divisors are wave-uniform: the step index comes from
// one fp64 FMA (i / per_step: exact below 2^31 items with per_step < 2^16,
// the 2^-20 lift keeps whole quotients whole), the layer from one fp32 FMA
// (slot / n_tpl with slot < 2^16), the template from selects among the
// family's at most four, and the record index is 32-bit.
__device__ __forceinline__ void expand_records(const ExpandParams &p, int64_t c0, int64_t cstep) {
  const int64_t n_chunks = p.chunk_off[KS_NFAM];
  const int64_t n_pre = p.n_prefill, n_dec = p.n_steps - p.n_prefill;
  uint32_t bad = 0;
  int f = 0;
  for (int64_t c = c0; c < n_chunks; c += cstep) {
    while (c >= p.chunk_off[f + 1]) ++f;
    const int64_t i64 = (c - p.chunk_off[f]) * 256 + threadIdx.x;
    if (i64 >= p.item_off[f + 1] - p.item_off[f]) continue;
    const uint32_t idx = (uint32_t)i64;
    const uint32_t ps = p.per_step[f];
    const uint32_t j = (uint32_t)__builtin_fma((double)idx, p.inv_ps[f], 0x1p-20);
    const uint32_t slot = idx - j * ps;
    const uint32_t layer = (uint32_t)fmaf((float)slot, p.inv_tpl[f], 0x1p-6f);
    const uint32_t ti = slot - layer * p.n_tpl[f];
    const ExpandTpl t0 = p.tpl[f][0], t1 = p.tpl[f][1], t2 = p.tpl[f][2], t3 = p.tpl[f][3];
    const uint32_t tn = ti == 0 ? t0.n : ti == 1 ? t1.n : ti == 2 ? t2.n : t3.n;
    const uint32_t tk = ti == 0 ? t0.k : ti == 1 ? t1.k : ti == 2 ? t2.k : t3.k;
    const uint32_t ta = ti == 0 ? t0.a : ti == 1 ? t1.a : ti == 2 ? t2.a : t3.a;
    const uint32_t tm = ti == 0 ? t0.msrc : ti == 1 ? t1.msrc : ti == 2 ? t2.msrc : t3.msrc;
    const uint32_t tg = ti == 0 ? t0.grouped : ti == 1 ? t1.grouped : ti == 2 ? t2.grouped : t3.grouped;
    uint32_t dst;
    if (f == KS_ATTN_PREFILL) {
      const int64_t r = (int64_t)p.blk[j / kExpandBlk] + p.rank[j];
      int64_t d;
      if (p.prefill[j] != 0) {
        d = r < n_pre ? p.fam_off[KS_ATTN_PREFILL] + r * ps + slot : -1;
      } else {
        const int64_t rd = (int64_t)j - r;
        d = (rd >= 0 && rd < n_dec) ? p.fam_off[KS_ATTN_DECODE] + rd * ps + slot : -1;
      }
      if (d < 0) {
        bad |= kErrPrefill;
        continue;
      }
      dst = (uint32_t)d;
    } else {
      dst = (uint32_t)p.fam_off[f] + idx;
    }
    uint32_t m = 0;
    if (tm == kMTok) {
      m = p.tok[j];
    } else if (tm == kMTopk) {
      m = p.tok[j] * p.top_k;
    } else if (tm == kMReq) {
      const uint32_t r0 = p.req_off[j], r1 = p.req_off[j + 1];
      m = r1 >= r0 ? r1 - r0 : 0u;
    }
    // written once and read by a later kernel: stream past the caches
    __builtin_nontemporal_store(j, p.o_step + dst);
    __builtin_nontemporal_store(m, p.o_m + dst);
    __builtin_nontemporal_store(tn, p.o_n + dst);
    __builtin_nontemporal_store(tk, p.o_k + dst);
    __builtin_nontemporal_store(ta, p.o_a + dst);
    __builtin_nontemporal_store(tg ? (j * p.L + layer) * p.E : 0u, p.o_b + dst);
    if (p.o_mult) __builtin_nontemporal_store(p.mult[f], p.o_mult + dst);
  }
  if (bad) atomicOr(p.err, bad);
}

__global__ __launch_bounds__(256) void k_expand_records(ExpandParams p) { expand_records(p, blockIdx.x, gridDim.x); }

// One workgroup: the flag reset, then each stage in turn, separated by
// barriers (the per-step T, ranks and block prefix reach the later stages
// through global memory within the workgroup).
__global__ __launch_bounds__(256) void k_expand_small(ExpandParams p) {
  if (threadIdx.x == 0) p.err[0] = 0;
  __syncthreads();
  expand_steps(p, threadIdx.x / kTokLanes, 256 / kTokLanes, threadIdx.x & (kTokLanes - 1));
  __syncthreads();
  expand_rank(p, 0);
  __syncthreads();
  expand_scan(p);
  __syncthreads();
  expand_records(p, 0, 1);
}

// batches the one-workgroup path takes: one rank block, at most 64 chunks
constexpr int64_t kSmallChunks = 64;

static int grid_cap(int64_t n, int block, int cap) {
  int64_t g = (n + block - 1) / block;
  if (g < 1) g = 1;
  return (int)(g < cap ? g : cap);
}

hipError_t launch_expand(const ExpandParams &p, hipStream_t s, hipEvent_t before, hipEvent_t after) {
  if (p.n_steps > 0 && p.n_blk == 1 && p.chunk_off[KS_NFAM] <= kSmallChunks) {
    if (before && after) {
      const hipError_t e = hipEventRecord(before, s);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_expand_small, dim3(1), dim3(256), 0, s, p);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return before && after ? hipEventRecord(after, s) : hipSuccess;
  }
  hipError_t e = launch_clear(p.err, nullptr, 0, s);
  if (e != hipSuccess || p.n_steps == 0) return e;
  hipLaunchKernelGGL(k_expand_steps, dim3(grid_cap(p.n_steps * kTokLanes, 256, 16384)), dim3(256), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_expand_rank, dim3((unsigned)p.n_blk), dim3(256), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_expand_scan, dim3(1), dim3(256), 0, s, p);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (before && after) {
    e = hipEventRecord(before, s);
    if (e != hipSuccess) return e;
  }
  if (p.item_off[KS_NFAM] > 0) {
    hipLaunchKernelGGL(k_expand_records, dim3(grid_cap(p.chunk_off[KS_NFAM] * 256, 256, 8192)), dim3(256), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return before && after ? hipEventRecord(after, s) : hipSuccess;
}

}  // namespace ks
