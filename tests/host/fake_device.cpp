// Host stand-ins for the HIP runtime calls and the kernel launches of the
// library, so that its host code (argument checks, workspace layouts, the
// expansion plan, the serving simulator) builds with g++ alone and runs
// under AddressSanitizer and UndefinedBehaviorSanitizer on a machine without
// a GPU.  TEST INFRASTRUCTURE ONLY: it is linked into the CPU test driver,
// never into the library.
//
// "Device" pointers are host memory here.  The launches do only what the
// host code and the test driver need:
//   launch_attn_agg   the per-step request sums (Q, KV, PAIRS, TILES)
//   launch_expand     the per-step arrays (layers, hidden, tp, n_launch)
//   launch_finish     a stand-in step latency,
//                     t_step = 1e-3 + 2e-7 Q + 1e-4 s + 5e-4 [n_launch > 0]
//                     (s: the spec index), and t_body = t_gpu = t_step
//                     and, with own, each step's latency under its own spec
// and the others do nothing.  The stand-in latency is not the model: the
// driver prices schedules with it so that the oracle's scheduler, given the
// same function, must form the same batches.
#include <hip/hip_runtime_api.h>

#include <cstdlib>
#include <cstring>

#include "ks_internal.h"

extern "C" {
hipError_t hipHostMalloc(void **ptr, size_t size, unsigned int) {
  *ptr = std::malloc(size);
  return *ptr ? hipSuccess : hipErrorOutOfMemory;
}
hipError_t hipHostFree(void *ptr) {
  std::free(ptr);
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void *dst, const void *src, size_t n, hipMemcpyKind, hipStream_t) {
  if (n) std::memcpy(dst, src, n);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
const char *hipGetErrorString(hipError_t) { return "host stand-in"; }
}

namespace ks {

hipError_t launch_clear(uint32_t *err, uint32_t *range, int64_t n_range, hipStream_t) {
  err[0] = 0;
  for (int64_t i = 0; i < n_range; ++i) range[i] = 0;
  return hipSuccess;
}

hipError_t launch_spec_prep(const ks_spec *, int32_t, SpecC *, uint32_t *, hipStream_t) { return hipSuccess; }

hipError_t launch_clear_prep(uint32_t *err, uint32_t *range, int64_t n_range, const ks_spec *specs, int32_t n_specs,
                             SpecC *out, hipStream_t st) {
  const hipError_t e = launch_clear(err, range, n_range, st);
  return e != hipSuccess ? e : launch_spec_prep(specs, n_specs, out, err, st);
}

hipError_t launch_attn_agg(const uint32_t *req_off, const uint32_t *q, const uint32_t *h, int64_t n_steps,
                           int64_t n_req, uint64_t *agg, uint32_t *err, hipStream_t) {
  for (int64_t j = 0; j < n_steps; ++j) {
    uint64_t Q = 0, KV = 0, P = 0, T = 0;
    uint32_t r0 = req_off[j], r1 = req_off[j + 1];
    if (r0 > r1 || (int64_t)r1 > n_req) {
      err[0] |= kErrReq;
      r0 = r1 = 0;
    }
    for (uint32_t r = r0; r < r1; ++r) {
      const uint64_t qq = q[r], hh = h[r];
      Q += qq;
      KV += hh + qq;
      P += qq * hh + qq * (qq + 1) / 2;
      T += (qq + 127) / 128;
    }
    agg[j] = Q;
    agg[n_steps + j] = KV;
    agg[2 * n_steps + j] = P;
    agg[3 * n_steps + j] = T;
  }
  return hipSuccess;
}

hipError_t launch_eval(int, const EvalParams &, hipStream_t) { return hipSuccess; }

hipError_t launch_finish(const FinishParams &p, hipStream_t) {
  for (int32_t s = 0; s < p.n_specs; ++s)
    for (int64_t j = 0; j < p.n_steps; ++j) {
      double t = 1e-3 + 2e-7 * (double)p.agg[j];
      t += 1e-4 * (double)s;
      t += 5e-4 * (p.n_launch[j] > 0 ? 1.0 : 0.0);
      const size_t i = (size_t)s * (size_t)p.n_steps + (size_t)j;
      p.t_body[i] = t;
      p.t_gpu[i] = t;
      p.t_step[i] = t;
      if (p.own && p.own[j] == (uint32_t)s) p.lat[j] = t;
    }
  return hipSuccess;
}

hipError_t launch_fill_source(const EvalParams &, hipStream_t) { return hipSuccess; }
hipError_t launch_validate(const ValidateParams &, hipStream_t) { return hipSuccess; }

hipError_t launch_expand(const ExpandParams &p, hipStream_t, hipEvent_t, hipEvent_t) {
  p.err[0] = 0;
  for (int64_t j = 0; j < p.n_steps; ++j) {
    p.o_layers[j] = p.L;
    p.o_hidden[j] = p.D;
    p.o_tp[j] = p.P;
    p.o_nlaunch[j] = p.prefill[j] ? p.L : 0;
  }
  return hipSuccess;
}

}  // namespace ks
