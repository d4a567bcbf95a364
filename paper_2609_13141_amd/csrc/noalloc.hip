// The SAS decode step (Alg. 2) for callers that cannot allocate device
// memory: its scratch lives in a file-scope device array instead of a
// caller-provided workspace.  The kernels are those of sas_decode_step.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/sas.h"
#include "kernels.h"

namespace {

// One copy per GPU, resident from the library's first use of that GPU until
// the process ends.  Host code must never pass `scratch` itself to a kernel
// or a copy: in host code the name is a stand-in, not a device address; the
// per-device address comes from hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[SAS_DECODE_NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// The current device's copy of the scratch array, looked up once per device
// with that device current.
sas_status scratch_of_current_device(void** out) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (sas_status)sas::set_error(SAS_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= MAX_DEVICES)
    return (sas_status)sas::set_error(SAS_ERR_UNSUPPORTED, "device %d (supported: 0..%d)", dev, MAX_DEVICES - 1);
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t g = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (g != hipSuccess || !p)
      return (sas_status)sas::set_error(SAS_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                                        hipGetErrorString(g));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SAS_OK;
}

}  // namespace

extern "C" sas_status sas_decode_step_noalloc(const sas_config* cfg, int32_t batch, const void* x,
                                              const int32_t* pos, const sas_layer_weights* w, sas_paged_kv* cache,
                                              void* y, int32_t* sel_idx, void* stream) {
  if (!cfg) return (sas_status)sas::set_error(SAS_ERR_INVALID_ARGUMENT, "config is NULL");
  if (!cache) return (sas_status)sas::set_error(SAS_ERR_INVALID_ARGUMENT, "cache is NULL");
  if (batch <= 0) return (sas_status)sas::set_error(SAS_ERR_INVALID_ARGUMENT, "batch %d must be positive", batch);
  const long long context = (long long)cache->max_blocks * cfg->block_size;
  if (cache->max_blocks <= 0 || context > INT32_MAX)
    return (sas_status)sas::set_error(SAS_ERR_INVALID_ARGUMENT, "cache max_blocks %d is out of range",
                                      cache->max_blocks);
  // the size check needs no device: oversized calls fail before the GPU is touched
  const size_t need = sas_workspace_size(cfg, SAS_OP_DECODE, batch, (int32_t)context);
  if (need == 0) {  // invalid configuration: let the full validation name the problem
    return sas_decode_step(cfg, batch, x, pos, w, cache, y, sel_idx, nullptr, nullptr, 0, stream);
  }
  if (need > SAS_DECODE_NOALLOC_SCRATCH_BYTES)
    return (sas_status)sas::set_error(
        SAS_ERR_WORKSPACE,
        "sas_decode_step_noalloc: batch %d over a cache of %d blocks needs %zu bytes of scratch; its static "
        "scratch holds %zu (use sas_decode_step with a workspace)",
        batch, cache->max_blocks, need, (size_t)SAS_DECODE_NOALLOC_SCRATCH_BYTES);
  void* ptr = nullptr;
  const sas_status st = scratch_of_current_device(&ptr);
  if (st != SAS_OK) return st;
  return sas_decode_step(cfg, batch, x, pos, w, cache, y, sel_idx, nullptr, ptr, SAS_DECODE_NOALLOC_SCRATCH_BYTES,
                         stream);
}
