// Internal declarations and device helpers shared by the verify-step kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "specrouter.h"

namespace sr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();

// Hardware 2^x (one instruction; results below 2^-126 flush to zero).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
// The wave's index in its workgroup, as a wave-uniform (scalar) value, so that
// branches on it are scalar branches rather than exec-mask regions.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// Buffer resource for raw buffer loads/stores over [base, base + bytes):
// offsets are 32-bit and accesses past the end read zero / are dropped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// Widen the two bf16 halves of a 32-bit word to fp32 (exact).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Cross-lane moves without LDS: DPP within each row of 16 lanes, and the
// gfx950 row swaps across 16- and 32-lane halves.
namespace dpp {
constexpr int kXor1 = 0xB1;         // quad_perm [1,0,3,2]: lane i reads lane i^1
constexpr int kXor2 = 0x4E;         // quad_perm [2,3,0,1]: lane i reads lane i^2
constexpr int kHalfMirror = 0x141;  // lane i reads lane 7-i within its group of 8
constexpr int kMirror = 0x140;      // lane i reads lane 15-i within its row of 16
}  // namespace dpp

template <int C>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, C, 0xf, 0xf, false);
}
template <int C>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint64_t lo = dpp_u32<C>((uint32_t)u), hi = dpp_u32<C>((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(lo | (hi << 32)));
}
// The same for the permutation patterns above (every lane has a source lane,
// so no fill value is needed, and the compiler can fold the move into the
// operation that reads it).
template <int C>
__device__ __forceinline__ uint32_t perm_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)x, C, 0xf, 0xf, false);
}
template <int C>
__device__ __forceinline__ float perm_f32(float x) {
  return __uint_as_float(perm_u32<C>(__float_as_uint(x)));
}
template <int C>
__device__ __forceinline__ double perm_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint64_t lo = perm_u32<C>((uint32_t)u), hi = perm_u32<C>((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(lo | (hi << 32)));
}

// max(a, b) for non-NaN operands as the median of (a, b, +inf): one
// instruction, without the quieting of the operands that fmaxf needs (the
// +inf comes from an opaque scalar move, so that the compiler keeps the
// median instead of turning it back into fmaxf).
__device__ __forceinline__ float opaque_inf() {
  float r;
  asm("s_mov_b32 %0, 0x7f800000" : "=s"(r));
  return r;
}
__device__ __forceinline__ float max_nn(float a, float b) { return __builtin_amdgcn_fmed3f(a, b, opaque_inf()); }

// (value of the even row, value of the odd row) of each pair of 16-lane rows,
// in every lane; with kHalf32 the same for the two 32-lane halves.
template <bool kHalf32>
__device__ __forceinline__ void swap_halves(uint32_t x, uint32_t& even, uint32_t& odd) {
  const auto r = kHalf32 ? __builtin_amdgcn_permlane32_swap(x, x, false, false)
                         : __builtin_amdgcn_permlane16_swap(x, x, false, false);
  even = r[0];
  odd = r[1];
}
template <bool kHalf32>
__device__ __forceinline__ void swap_halves_f32(float x, float& even, float& odd) {
  uint32_t e, o;
  swap_halves<kHalf32>(__float_as_uint(x), e, o);
  even = __uint_as_float(e);
  odd = __uint_as_float(o);
}
template <bool kHalf32>
__device__ __forceinline__ void swap_halves_f64(double x, double& even, double& odd) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  uint32_t el, ol, eh, oh;
  swap_halves<kHalf32>((uint32_t)u, el, ol);
  swap_halves<kHalf32>((uint32_t)(u >> 32), eh, oh);
  even = __longlong_as_double((long long)((uint64_t)el | ((uint64_t)eh << 32)));
  odd = __longlong_as_double((long long)((uint64_t)ol | ((uint64_t)oh << 32)));
}

// Wave-wide reductions over the 64 lanes, bit-identical in every lane: a fixed
// tree (pairs, quads, groups of 8, rows of 16, then the row pairs and halves,
// the lower part always on the left).
__device__ __forceinline__ float wave_max(float x) {
  x = max_nn(x, perm_f32<dpp::kXor1>(x));
  x = max_nn(x, perm_f32<dpp::kXor2>(x));
  x = max_nn(x, perm_f32<dpp::kHalfMirror>(x));
  x = max_nn(x, perm_f32<dpp::kMirror>(x));
  float e, o;
  swap_halves_f32<false>(x, e, o);
  x = max_nn(e, o);
  swap_halves_f32<true>(x, e, o);
  return max_nn(e, o);
}
__device__ __forceinline__ float wave_sum(float x) {
  x = x + perm_f32<dpp::kXor1>(x);
  x = x + perm_f32<dpp::kXor2>(x);
  x = x + perm_f32<dpp::kHalfMirror>(x);
  x = x + perm_f32<dpp::kMirror>(x);
  float e, o;
  swap_halves_f32<false>(x, e, o);
  x = e + o;
  swap_halves_f32<true>(x, e, o);
  return e + o;
}
__device__ __forceinline__ double wave_sum_d(double x) {
  x = x + perm_f64<dpp::kXor1>(x);
  x = x + perm_f64<dpp::kXor2>(x);
  x = x + perm_f64<dpp::kHalfMirror>(x);
  x = x + perm_f64<dpp::kMirror>(x);
  double e, o;
  swap_halves_f64<false>(x, e, o);
  x = e + o;
  swap_halves_f64<true>(x, e, o);
  return e + o;
}
__device__ __forceinline__ int wave_max_i(int x) {
  x = max(x, (int)perm_u32<dpp::kXor1>((uint32_t)x));
  x = max(x, (int)perm_u32<dpp::kXor2>((uint32_t)x));
  x = max(x, (int)perm_u32<dpp::kHalfMirror>((uint32_t)x));
  x = max(x, (int)perm_u32<dpp::kMirror>((uint32_t)x));
  uint32_t e, o;
  swap_halves<false>((uint32_t)x, e, o);
  x = max((int)e, (int)o);
  swap_halves<true>((uint32_t)x, e, o);
  return max((int)e, (int)o);
}

// Reductions over the four 16-lane rows only (lanes i, i^16, i^32, i^48),
// as ((row 0, row 1), (row 2, row 3)) in every lane.
__device__ __forceinline__ float max_across_rows(float x) {
  float e, o;
  swap_halves_f32<false>(x, e, o);
  x = fmaxf(e, o);
  swap_halves_f32<true>(x, e, o);
  return fmaxf(e, o);
}
__device__ __forceinline__ float sum_across_rows(float x) {
  float e, o;
  swap_halves_f32<false>(x, e, o);
  x = e + o;
  swap_halves_f32<true>(x, e, o);
  return e + o;
}

__device__ __forceinline__ int wave_min_i(int x) {
  x = min(x, (int)perm_u32<dpp::kXor1>((uint32_t)x));
  x = min(x, (int)perm_u32<dpp::kXor2>((uint32_t)x));
  x = min(x, (int)perm_u32<dpp::kHalfMirror>((uint32_t)x));
  x = min(x, (int)perm_u32<dpp::kMirror>((uint32_t)x));
  uint32_t e, o;
  swap_halves<false>((uint32_t)x, e, o);
  x = min((int)e, (int)o);
  swap_halves<true>((uint32_t)x, e, o);
  return min((int)e, (int)o);
}

// Wave-wide inclusive prefix sum of an int in ascending lane order: DPP row
// shifts inside each 16-lane row (lanes without a source read 0), then the
// totals of the earlier rows.
__device__ __forceinline__ int wave_incl_scan_i(int x) {
  x += (int)dpp_u32<0x111>((uint32_t)x);  // row_shr:1
  x += (int)dpp_u32<0x112>((uint32_t)x);  // row_shr:2
  x += (int)dpp_u32<0x114>((uint32_t)x);  // row_shr:4
  x += (int)dpp_u32<0x118>((uint32_t)x);  // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31);
  const int r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  return x + (row == 0 ? 0 : row == 1 ? r0 : row == 2 ? r0 + r1 : r0 + r1 + r2);
}

// The value of lane `src` (wave-uniform) in every lane.
__device__ __forceinline__ int lane_value(int x, int src) { return __builtin_amdgcn_readlane(x, src); }
__device__ __forceinline__ double lane_value(double x, int src) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, src);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), src);
  return __longlong_as_double((long long)((uint64_t)lo | ((uint64_t)hi << 32)));
}

// Merge two (max, sum-of-exp2(x*log2e - max*log2e)) partials.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float M = fmaxf(m, m2);
  if (M == kNegInf) {
    m = M;
    s = 0.f;
    return;
  }
  s = s * exp2f((m - M) * kLog2e) + s2 * exp2f((m2 - M) * kLog2e);
  m = M;
}

// Device-scope (agent) synchronisation primitives.
__device__ __forceinline__ uint32_t atomic_load_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t atomic_add_release(uint32_t* p, uint32_t v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void fence_acquire_agent() {
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Values handed between workgroups of one launch (possibly on different XCDs,
// whose L2 caches are not coherent with each other) are written and read with
// relaxed device-scope atomics, which are served at the device coherence
// point; no cache-wide write-back or invalidate is needed.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this wave's earlier stores have completed (they are then visible
// to device-coherent loads anywhere on the device).
__device__ __forceinline__ void stores_done() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// ---------------------------------------------------------------------------
// Host-side launchers (one per translation unit). Arguments are already
// validated by the C ABI layer.

struct AttentionPlan {
  int nq;          // 16-row query blocks per wave
  int qg;          // query groups (of four waves) per workgroup
  int q_chunks;    // workgroups along the query rows of one (sequence, kv head)
  int split_keys;  // keys per split (multiple of 32)
  int n_splits;    // splits along the cache
  size_t part_offset;  // byte offset of the split partials in the workspace
  int ordered;         // more workgroups than fit at once: dispatched longest job first
  size_t order_offset;  // byte offset of the dispatch order in the workspace
  size_t workspace_bytes;
};

int attention_plan(int B, int gamma_max, int Hq, int Hkv, int D, int L_cap, AttentionPlan* plan);

int launch_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                            const uint8_t* cache_mask, const int32_t* kv_len,
                            const int32_t* gamma, float* out, int B, int gamma_max, int Hq,
                            int Hkv, int D, int L_cap, float scale, void* workspace,
                            const AttentionPlan& plan, int32_t* status, hipStream_t stream);

struct AcceptPlan {
  int chunk;          // vocabulary entries per workgroup task
  int n_chunks;       // chunks per row
  size_t workspace_bytes;
};

int accept_plan(int B, int gamma_max, int V, int dtype, AcceptPlan* plan);
// The workspace bytes an accept call of this shape needs (0: unsupported
// shape); host arithmetic only, no device query.
size_t accept_workspace_bytes(int B, int gamma_max, int V, int dtype);

// Rollback applied by the accept call itself (after each sequence's outcome):
// the same update as launch_rollback with new_len = the accept's new length.
struct AcceptRollback {
  int32_t* kv_len;    // [B] cache lengths, in/out
  uint8_t* mask;      // [B][L_cap] validity mask, or NULL
  int32_t* phys_len;  // max over sequences of the new lengths, or NULL
  int L_cap;
};

int launch_accept(const void* p_logits, int64_t p_stride, const void* q_logits, int64_t q_stride,
                  int dtype, const int32_t* drafts, const int32_t* gamma, const float* u_acc,
                  const float* u_res, const int32_t* kv_len, int32_t* accept_len,
                  int32_t* out_tokens, int32_t* new_len, float* accept_prob, float* p_tok,
                  float* q_tok, float* kl, float* tv, int B, int gamma_max, int V, float temperature,
                  int top_k, float top_p, const AcceptRollback* rollback, void* workspace,
                  const AcceptPlan& plan, int32_t* status, hipStream_t stream);

int launch_chain_window(const int32_t* accept_len, const int32_t* out_tokens, int B, int gmax, int cap,
                        const int32_t* ctx_len, int32_t* gamma_next, int32_t* drafts_next,
                        int32_t* kv_len_next, hipStream_t stream);
int launch_chain_consensus(const int32_t* ctx_len, const int32_t* k_lower, const int32_t* out_lower,
                           int gmax_lower, const int32_t* k_upper, const int32_t* out_upper, int gmax_upper,
                           int B, int32_t* len_upper, int32_t* len_lower, int32_t* pending,
                           int32_t* n_pending, int32_t* status, hipStream_t stream);

int launch_kv_append(const void* k_new, const void* v_new, const int32_t* gamma, void* k_cache, void* v_cache,
                     uint8_t* cache_mask, int32_t* kv_len, const int32_t* shared_len, int B, int gamma_max,
                     int Hkv, int D, int L_cap, int32_t* status, hipStream_t stream);
int launch_kv_compact(void* k_cache, void* v_cache, uint8_t* cache_mask, int32_t* kv_len, int B, int Hkv, int D,
                      int L_cap, int32_t* status, hipStream_t stream);

int launch_rollback(int32_t* kv_len, uint8_t* cache_mask, const int32_t* new_len,
                    int32_t* phys_len, int B, int L_cap, int32_t* status, hipStream_t stream);

// Cached per-device properties.
int device_cu_count();

}  // namespace sr
