// Accept-and-rollback without a caller-provided workspace: the workspace is a
// fixed array in device memory owned by the library, for callers that cannot
// allocate (code under HIP graph capture, serving loops, harnesses that forbid
// allocation). The kernels are those of specrouter_accept_and_rollback.

#include <mutex>
#include <stdint.h>

#include "sr_internal.h"

// One array per device, resident from the library's load until the process
// ends. Its name is a host-side stand-in: host code only ever uses the device
// address looked up for the current device.
static __device__ __align__(256) unsigned char scratch[SPECROUTER_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;

struct DeviceScratch {
  void* ptr = nullptr;  // device address of `scratch` on this device
  bool clean = false;   // the array is known to be zero (the accept kernels leave it so)
};

std::mutex g_mutex;
DeviceScratch g_dev[kMaxDevices];

__global__ void __launch_bounds__(256) clear_kernel(sr::u32x4* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = sr::u32x4{0u, 0u, 0u, 0u};
}

// The current device's scratch address, looked up once per device, and the
// array cleared on `stream` when it is not known to be zero. NULL on error.
void* device_scratch(hipStream_t stream, int* rc) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *rc = SR_ELAUNCH;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mutex);
  DeviceScratch& d = g_dev[dev];
  if (!d.ptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *rc = SR_ELAUNCH;
      return nullptr;
    }
    d.ptr = p;
  }
  if (!d.clean) {
    constexpr size_t n = SPECROUTER_NOALLOC_SCRATCH_BYTES / 16;
    hipLaunchKernelGGL(clear_kernel, dim3(1024), dim3(256), 0, stream, (sr::u32x4*)d.ptr, n);
    if (hipGetLastError() != hipSuccess) {
      *rc = SR_ELAUNCH;
      return nullptr;
    }
    d.clean = true;
  }
  *rc = SR_OK;
  return d.ptr;
}

// After a call that may have stopped between its launches, clear again
// before the next use.
void mark_dirty() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return;
  std::lock_guard<std::mutex> lock(g_mutex);
  g_dev[dev].clean = false;
}

}  // namespace

extern "C" int specrouter_accept_and_rollback_noalloc(
    const void* p_logits, int64_t p_batch_stride, const void* q_logits, int64_t q_batch_stride, int logits_dtype,
    const int32_t* draft_tokens, const int32_t* gamma, const float* u_accept, const float* u_resample,
    const int32_t* kv_len, int32_t* accept_len, int32_t* out_tokens, int32_t* new_len, float* accept_prob,
    float* p_tok, float* q_tok, float* kl, float* tv, int B, int gamma_max, int V,
    const specrouter_sampling* sampling, int32_t* cache_kv_len, uint8_t* cache_mask, int32_t* phys_len,
    int L_cap, int32_t* status, void* stream) {
  // Size first, from the shape alone: a problem whose workspace exceeds the
  // fixed array is refused before anything touches the device.
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA || V <= 0) return SR_EINVAL;
  if (logits_dtype != SR_F32 && logits_dtype != SR_BF16) return SR_EUNSUPPORTED;
  const size_t need = sr::accept_workspace_bytes(B, gamma_max, V, logits_dtype);
  if (need == 0) return SR_EUNSUPPORTED;
  if (need > SPECROUTER_NOALLOC_SCRATCH_BYTES) return SR_ESCRATCH;
  int rc = SR_OK;
  void* ws = device_scratch((hipStream_t)stream, &rc);
  if (!ws) return rc;
  rc = specrouter_accept_and_rollback(p_logits, p_batch_stride, q_logits, q_batch_stride, logits_dtype, draft_tokens,
                                      gamma, u_accept, u_resample, kv_len, accept_len, out_tokens, new_len,
                                      accept_prob, p_tok, q_tok, kl, tv, B, gamma_max, V, sampling, cache_kv_len,
                                      cache_mask, phys_len, L_cap, ws, SPECROUTER_NOALLOC_SCRATCH_BYTES, status,
                                      stream);
  if (rc == SR_ELAUNCH) mark_dirty();
  return rc;
}
