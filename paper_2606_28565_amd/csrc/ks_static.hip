// Allocation-free variant of ks_eval_steps for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid hipMalloc): the evaluation's workspace is a
// file-scope device array of fixed size instead of a caller-provided buffer.
//
// In host code the array's name is only a host-side stand-in; its device
// address is looked up once per device with hipGetSymbolAddress (with that
// device current) and only that address is ever handed to the evaluation.
// Every call on a device shares that device's array, so calls that overlap
// on one GPU race; the evaluation clears what must start at zero (the flag
// word and the step-range table) with its own kernel on every call.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ks.h"
#include "ks_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[KS_STATIC_SCRATCH_BYTES];

constexpr int kMaxStaticDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxStaticDevices];   // device address of `scratch`, per device

// The device address of this device's copy of `scratch` (looked up on the
// first call on the device, with the device current).
ks_status scratch_ptr(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return ks::set_error(KS_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxStaticDevices)
    return ks::set_error(KS_EINVAL, "device %d beyond the %d devices the static scratch supports", dev,
                         kMaxStaticDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return ks::set_error(KS_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    if (reinterpret_cast<uintptr_t>(p) % 256)
      return ks::set_error(KS_EHIP, "static scratch at %p not 256-byte aligned", p);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return KS_OK;
}

}  // namespace

extern "C" ks_status ks_eval_steps_static(const ks_desc *desc, const ks_steps *steps, const ks_spec *specs,
                                          int32_t n_specs, const ks_heads *heads, const ks_host *host,
                                          const ks_step_out *out, const ks_kernel_out *kout, uint32_t *flags,
                                          hipStream_t stream) {
  // size check before any runtime call: bad arguments get the evaluation's
  // own message (its checks run before its first launch)
  const size_t need = ks_workspace_bytes(desc, n_specs);
  if (need == 0) return ks_eval_steps(desc, steps, specs, n_specs, heads, host, out, kout, nullptr, 0, stream);
  if (need > (size_t)KS_STATIC_SCRATCH_BYTES)
    return ks::set_error(KS_ERANGE,
                         "this call needs %zu bytes of workspace, above the %d-byte static scratch; "
                         "use ks_eval_steps with a caller-provided workspace",
                         need, (int)KS_STATIC_SCRATCH_BYTES);
  void *ws = nullptr;
  ks_status st = scratch_ptr(&ws);
  if (st != KS_OK) return st;
  st = ks_eval_steps(desc, steps, specs, n_specs, heads, host, out, kout, ws, (size_t)KS_STATIC_SCRATCH_BYTES,
                     stream);
  if (st != KS_OK || !flags) return st;
  // the bad-data flag word (offset 0 of the workspace) for the caller
  const hipError_t e = hipMemcpyAsync(flags, ws, sizeof(uint32_t), hipMemcpyDeviceToDevice, stream);
  if (e != hipSuccess) return ks::set_error(KS_EHIP, "flag copy: %s", hipGetErrorString(e));
  return KS_OK;
}
