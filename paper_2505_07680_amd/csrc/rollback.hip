// Logical KV rollback (Section 4.4, rollback mechanism; Eq. 9).
//
// Per sequence: n = min(kv_len, new_len); the validity bits of cache entries
// [n, kv_len) are cleared and kv_len becomes n. No K/V data is touched. The
// common physical length (max over sequences) is reduced in the same pass.
// One workgroup handles the whole batch (a verify step rolls back at most
// gamma_max + 1 entries per sequence), so the reduction needs no atomics and
// the call is a single short launch.

#include <limits.h>

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kThreads = 256;

__global__ void __launch_bounds__(kThreads)
rollback_kernel(int32_t* __restrict__ kv_len, uint8_t* __restrict__ mask,
                const int32_t* __restrict__ new_len, int32_t* __restrict__ phys_len, int B,
                int L_cap, int32_t* __restrict__ status) {
  __shared__ int red_max[kThreads / 64];
  __shared__ int red_st[kThreads / 64];
  int mx = INT_MIN;
  int st = 0;
  for (int b = threadIdx.x; b < B; b += kThreads) {
    const int old = kv_len[b];
    const int want = new_len[b];
    if (old < 0 || old > L_cap || want < 0) {
      st |= SR_ST_KVLEN;
      mx = max(mx, old);
      continue;
    }
    if (want > old) st |= SR_ST_ROLLBACK_GROW;
    const int n = min(old, want);
    if (mask) {
      uint8_t* m = mask + (size_t)b * L_cap;
      for (int x = n; x < old; ++x) m[x] = 0;
    }
    kv_len[b] = n;
    mx = max(mx, n);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    mx = max(mx, __shfl_xor(mx, off, 64));
    st |= __shfl_xor(st, off, 64);
  }
  const int w = wave_id();
  if ((threadIdx.x & 63) == 0) {
    red_max[w] = mx;
    red_st[w] = st;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < kThreads / 64; ++i) {
      mx = max(mx, red_max[i]);
      st |= red_st[i];
    }
    if (phys_len) *phys_len = mx;
    if (st && status) atomicOr(status, st);
  }
}

}  // namespace

int launch_rollback(int32_t* kv_len, uint8_t* cache_mask, const int32_t* new_len,
                    int32_t* phys_len, int B, int L_cap, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(rollback_kernel, dim3(1), dim3(kThreads), 0, stream, kv_len, cache_mask,
                     new_len, phys_len, B, L_cap, status);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

}  // namespace sr
