// Glue between the verifier levels of a multi-level chain (multi-level
// verification, Section 3.1; VerifyProcessor and RollbackProcessor, Section
// 4.3), on the device so a chain step needs no host round trip:
//
//   chain_window:    the next level verifies the first min(k_b + 1, cap)
//                    tokens the level below emitted (its accepted drafts and
//                    its correction or bonus token); their draft
//                    distribution is the level below's own verifier rows;
//   chain_consensus: after the upper level, the rows every level keeps (upper
//                    ctx + 1 + k_u, lower ctx + 1 + min(k_l, k_u)) and the
//                    tokens the lower levels have emitted but not cached.
//
// One thread per sequence; both are a few scalar loads and stores.

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kChainThreads = 256;

__global__ void __launch_bounds__(kChainThreads)
chain_window_kernel(const int32_t* __restrict__ accept_len, const int32_t* __restrict__ out_tokens, int B,
                    int gmax, int cap, const int32_t* __restrict__ ctx_len, int32_t* __restrict__ gamma_next,
                    int32_t* __restrict__ drafts_next, int32_t* __restrict__ kv_len_next) {
  const int b = blockIdx.x * kChainThreads + threadIdx.x;
  if (b >= B) return;
  const int k = accept_len[b];
  const int g = (k >= 0 && k <= gmax) ? min(k + 1, cap) : -1;  // -1: flagged by the level below
  gamma_next[b] = g;
  const int32_t* src = out_tokens + (size_t)b * (gmax + 1);
  int32_t* dst = drafts_next + (size_t)b * cap;
  for (int j = 0; j < cap; ++j) dst[j] = j < g ? src[j] : 0;
  if (kv_len_next) kv_len_next[b] = ctx_len[b] + 1 + max(g, 0);
}

__global__ void __launch_bounds__(kChainThreads)
chain_consensus_kernel(const int32_t* __restrict__ ctx_len, const int32_t* __restrict__ k_lower,
                       const int32_t* __restrict__ out_lower, int gmax_lower,
                       const int32_t* __restrict__ k_upper, const int32_t* __restrict__ out_upper,
                       int gmax_upper, int B, int32_t* __restrict__ len_upper, int32_t* __restrict__ len_lower,
                       int32_t* __restrict__ pending, int32_t* __restrict__ n_pending,
                       int32_t* __restrict__ status) {
  const int b = blockIdx.x * kChainThreads + threadIdx.x;
  if (b >= B) return;
  const int ctx = ctx_len[b];
  const int kl = k_lower[b], ku = k_upper[b];
  int up = ctx, lo = ctx, p0 = -1, p1 = -1, n = 0;
  if (kl >= 0 && ku >= 0) {
    if (ku > kl + 1 || kl > gmax_lower || ku > gmax_upper) {
      if (status) atomicOr(status, (int32_t)SR_ST_CHAIN);
    } else {
      up = ctx + 1 + ku;
      lo = ctx + 1 + min(kl, ku);
      const int last = out_upper[(size_t)b * (gmax_upper + 1) + ku];
      if (ku == kl + 1) {  // the upper level accepted the lower level's own token
        p0 = out_lower[(size_t)b * (gmax_lower + 1) + kl];
        p1 = last;
        n = 2;
      } else {
        p0 = last;
        n = 1;
      }
    }
  }
  len_upper[b] = up;
  len_lower[b] = lo;
  pending[(size_t)b * 2] = p0;
  pending[(size_t)b * 2 + 1] = p1;
  n_pending[b] = n;
}

}  // namespace

int launch_chain_window(const int32_t* accept_len, const int32_t* out_tokens, int B, int gmax, int cap,
                        const int32_t* ctx_len, int32_t* gamma_next, int32_t* drafts_next,
                        int32_t* kv_len_next, hipStream_t stream) {
  hipLaunchKernelGGL(chain_window_kernel, dim3((B + kChainThreads - 1) / kChainThreads), dim3(kChainThreads), 0,
                     stream, accept_len, out_tokens, B, gmax, cap, ctx_len, gamma_next, drafts_next, kv_len_next);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

int launch_chain_consensus(const int32_t* ctx_len, const int32_t* k_lower, const int32_t* out_lower,
                           int gmax_lower, const int32_t* k_upper, const int32_t* out_upper, int gmax_upper,
                           int B, int32_t* len_upper, int32_t* len_lower, int32_t* pending,
                           int32_t* n_pending, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(chain_consensus_kernel, dim3((B + kChainThreads - 1) / kChainThreads), dim3(kChainThreads),
                     0, stream, ctx_len, k_lower, out_lower, gmax_lower, k_upper, out_upper, gmax_upper, B,
                     len_upper, len_lower, pending, n_pending, status);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

}  // namespace sr
