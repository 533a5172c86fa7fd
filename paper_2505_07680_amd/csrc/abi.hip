// C ABI of the verify step: host-side argument checks, workspace queries and
// dispatch to the kernels. Every check here happens before anything is
// enqueued; data that lives on the device is checked by the kernels.

#include <atomic>
#include <stdint.h>

#include "sr_internal.h"

namespace sr {

int device_cu_count() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (dev >= 0 && dev < 64) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -1;
  if (dev >= 0 && dev < 64) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

}  // namespace sr

namespace {

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool attention_shape_ok(int B, int gamma_max, int Hq, int Hkv, int L_cap) {
  return B > 0 && gamma_max >= 0 && gamma_max <= SPECROUTER_MAX_GAMMA && Hq > 0 && Hkv > 0 &&
         Hq % Hkv == 0 && L_cap >= gamma_max + 1 && L_cap <= SPECROUTER_MAX_CACHE_ROWS && B <= 65535;
}

// Checks and launch shared by the accept entry points (rollback NULL: none).
int accept_impl(const void* p_logits, int64_t p_batch_stride, const void* q_logits, int64_t q_batch_stride,
                int logits_dtype, const int32_t* draft_tokens, const int32_t* gamma, const float* u_accept,
                const float* u_resample, const int32_t* kv_len, int32_t* accept_len, int32_t* out_tokens,
                int32_t* new_len, float* accept_prob, float* p_tok, float* q_tok, float* kl, float* tv, int B,
                int gamma_max, int V, const specrouter_sampling* sampling, const sr::AcceptRollback* rollback,
                void* workspace, size_t workspace_bytes, int32_t* status, void* stream) {
  const float temperature = sampling ? sampling->temperature : 1.f;
  const int top_k = sampling ? sampling->top_k : 0;
  const float top_p = sampling ? sampling->top_p : 1.f;
  if (!(temperature >= 0.f && temperature < __builtin_inff())) return SR_EINVAL;
  if (top_k < 0 || !(top_p > 0.f && top_p <= 1.f)) return SR_EINVAL;
  const bool greedy = temperature == 0.f;
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA || V <= 0) return SR_EINVAL;
  if (logits_dtype != SR_F32 && logits_dtype != SR_BF16) return SR_EUNSUPPORTED;
  if (!p_logits || !gamma || !accept_len || !out_tokens) return SR_EINVAL;
  if (!greedy && !u_resample) return SR_EINVAL;
  if (gamma_max > 0 && (!q_logits || !draft_tokens || (!greedy && !u_accept))) return SR_EINVAL;
  if (new_len && !kv_len) return SR_EINVAL;
  if (p_batch_stride < (int64_t)(gamma_max + 1) * V) return SR_EINVAL;
  if (gamma_max > 0 && q_batch_stride < (int64_t)gamma_max * V) return SR_EINVAL;
  const int esz = logits_dtype == SR_BF16 ? 2 : 4;
  if ((p_batch_stride * esz) % 16 != 0 || !aligned16(p_logits)) return SR_EUNSUPPORTED;
  if (gamma_max > 0 && ((q_batch_stride * esz) % 16 != 0 || !aligned16(q_logits)))
    return SR_EUNSUPPORTED;
  sr::AcceptPlan plan;
  const int rc = sr::accept_plan(B, gamma_max, V, logits_dtype, &plan);
  if (rc != SR_OK) return rc;
  if (!workspace || workspace_bytes < plan.workspace_bytes || !aligned16(workspace))
    return SR_EWORKSPACE;
  return sr::launch_accept(p_logits, p_batch_stride, q_logits, q_batch_stride, logits_dtype,
                           draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len,
                           out_tokens, new_len, accept_prob, p_tok, q_tok, kl, tv, B, gamma_max,
                           V, temperature, top_k, top_p, rollback, workspace, plan, status,
                           (hipStream_t)stream);
}

}  // namespace

extern "C" {

int specrouter_abi_version(void) { return SPECROUTER_ABI_VERSION; }

const char* specrouter_status_string(int code) {
  switch (code) {
    case SR_OK: return "ok";
    case SR_EINVAL: return "invalid argument (size, NULL or misaligned pointer)";
    case SR_EUNSUPPORTED: return "unsupported configuration (head dim, dtype or vocabulary alignment)";
    case SR_EWORKSPACE: return "workspace missing or too small";
    case SR_ELAUNCH: return "HIP launch or device query failed";
    case SR_ESCRATCH: return "workspace needed exceeds the library's fixed no-allocation array";
    case SR_ST_GAMMA: return "device data: gamma outside [0, gamma_max]";
    case SR_ST_KVLEN: return "device data: kv_len or new_len out of range";
    case SR_ST_TOKEN: return "device data: draft token outside [0, V)";
    case SR_ST_UNIFORM: return "device data: uniform outside [0, 1)";
    case SR_ST_ROLLBACK_GROW: return "device data: rollback would grow a sequence (ignored)";
    case SR_ST_TIMEOUT: return "device: inter-workgroup wait timed out";
    case SR_ST_CHAIN: return "device data: accept lengths one chain step cannot produce";
    default: return "unknown code";
  }
}

size_t specrouter_verify_attention_workspace_size(int B, int gamma_max, int Hq, int Hkv, int D,
                                                  int L_cap) {
  if (!attention_shape_ok(B, gamma_max, Hq, Hkv, L_cap) || (D != 64 && D != 128)) return 0;
  sr::AttentionPlan plan;
  if (sr::attention_plan(B, gamma_max, Hq, Hkv, D, L_cap, &plan) != SR_OK) return 0;
  return plan.workspace_bytes;
}

int specrouter_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                                const uint8_t* cache_mask, const int32_t* kv_len,
                                const int32_t* gamma, float* out, int B, int gamma_max, int Hq,
                                int Hkv, int D, int L_cap, float scale, void* workspace,
                                size_t workspace_bytes, int32_t* status, void* stream) {
  if (!q || !k_cache || !v_cache || !kv_len || !gamma || !out) return SR_EINVAL;
  if (!attention_shape_ok(B, gamma_max, Hq, Hkv, L_cap)) return SR_EINVAL;
  if (D != 64 && D != 128) return SR_EUNSUPPORTED;
  if (!(scale > 0.f && scale < __builtin_inff())) return SR_EINVAL;  // a positive, finite score scale
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return SR_EINVAL;
  sr::AttentionPlan plan;
  const int rc = sr::attention_plan(B, gamma_max, Hq, Hkv, D, L_cap, &plan);
  if (rc != SR_OK) return rc;
  if (plan.workspace_bytes > 0 &&
      (!workspace || workspace_bytes < plan.workspace_bytes || !aligned16(workspace)))
    return SR_EWORKSPACE;
  return sr::launch_verify_attention(q, k_cache, v_cache, cache_mask, kv_len, gamma, out, B,
                                     gamma_max, Hq, Hkv, D, L_cap, scale, workspace, plan, status,
                                     (hipStream_t)stream);
}

size_t specrouter_accept_workspace_size(int B, int gamma_max, int V, int logits_dtype) {
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA || V <= 0) return 0;
  if (logits_dtype != SR_F32 && logits_dtype != SR_BF16) return 0;
  sr::AcceptPlan plan;
  if (sr::accept_plan(B, gamma_max, V, logits_dtype, &plan) != SR_OK) return 0;
  return plan.workspace_bytes;
}

int specrouter_accept_and_diverge_sampled(const void* p_logits, int64_t p_batch_stride,
                                          const void* q_logits, int64_t q_batch_stride, int logits_dtype,
                                          const int32_t* draft_tokens, const int32_t* gamma,
                                          const float* u_accept, const float* u_resample,
                                          const int32_t* kv_len, int32_t* accept_len,
                                          int32_t* out_tokens, int32_t* new_len, float* accept_prob,
                                          float* p_tok, float* q_tok, float* kl, float* tv, int B,
                                          int gamma_max, int V, const specrouter_sampling* sampling,
                                          void* workspace, size_t workspace_bytes, int32_t* status,
                                          void* stream) {
  return accept_impl(p_logits, p_batch_stride, q_logits, q_batch_stride, logits_dtype, draft_tokens, gamma,
                     u_accept, u_resample, kv_len, accept_len, out_tokens, new_len, accept_prob, p_tok, q_tok, kl,
                     tv, B, gamma_max, V, sampling, nullptr, workspace, workspace_bytes, status, stream);
}

int specrouter_accept_and_rollback(const void* p_logits, int64_t p_batch_stride, const void* q_logits,
                                   int64_t q_batch_stride, int logits_dtype, const int32_t* draft_tokens,
                                   const int32_t* gamma, const float* u_accept, const float* u_resample,
                                   const int32_t* kv_len, int32_t* accept_len, int32_t* out_tokens,
                                   int32_t* new_len, float* accept_prob, float* p_tok, float* q_tok, float* kl,
                                   float* tv, int B, int gamma_max, int V, const specrouter_sampling* sampling,
                                   int32_t* cache_kv_len, uint8_t* cache_mask, int32_t* phys_len, int L_cap,
                                   void* workspace, size_t workspace_bytes, int32_t* status, void* stream) {
  if (!kv_len || !cache_kv_len || L_cap <= 0) return SR_EINVAL;
  const sr::AcceptRollback rb{cache_kv_len, cache_mask, phys_len, L_cap};
  return accept_impl(p_logits, p_batch_stride, q_logits, q_batch_stride, logits_dtype, draft_tokens, gamma,
                     u_accept, u_resample, kv_len, accept_len, out_tokens, new_len, accept_prob, p_tok, q_tok, kl,
                     tv, B, gamma_max, V, sampling, &rb, workspace, workspace_bytes, status, stream);
}

int specrouter_accept_and_diverge(const void* p_logits, int64_t p_batch_stride,
                                  const void* q_logits, int64_t q_batch_stride, int logits_dtype,
                                  const int32_t* draft_tokens, const int32_t* gamma,
                                  const float* u_accept, const float* u_resample,
                                  const int32_t* kv_len, int32_t* accept_len,
                                  int32_t* out_tokens, int32_t* new_len, float* accept_prob,
                                  float* p_tok, float* q_tok, float* kl, float* tv, int B,
                                  int gamma_max, int V, void* workspace, size_t workspace_bytes,
                                  int32_t* status, void* stream) {
  return specrouter_accept_and_diverge_sampled(p_logits, p_batch_stride, q_logits, q_batch_stride,
                                               logits_dtype, draft_tokens, gamma, u_accept, u_resample,
                                               kv_len, accept_len, out_tokens, new_len, accept_prob, p_tok,
                                               q_tok, kl, tv, B, gamma_max, V, nullptr, workspace,
                                               workspace_bytes, status, stream);
}

int specrouter_chain_window(const int32_t* accept_len, const int32_t* out_tokens, int B, int gamma_max,
                            int gamma_cap, const int32_t* ctx_len, int32_t* gamma_next, int32_t* drafts_next,
                            int32_t* kv_len_next, void* stream) {
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (gamma_cap < 1 || gamma_cap > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (!accept_len || !out_tokens || !gamma_next || !drafts_next) return SR_EINVAL;
  if ((ctx_len == nullptr) != (kv_len_next == nullptr)) return SR_EINVAL;
  return sr::launch_chain_window(accept_len, out_tokens, B, gamma_max, gamma_cap, ctx_len, gamma_next, drafts_next,
                                 kv_len_next, (hipStream_t)stream);
}

int specrouter_chain_consensus(const int32_t* ctx_len, const int32_t* k_lower, const int32_t* out_lower,
                               int gamma_max_lower, const int32_t* k_upper, const int32_t* out_upper,
                               int gamma_max_upper, int B, int32_t* len_upper, int32_t* len_lower,
                               int32_t* pending, int32_t* n_pending, int32_t* status, void* stream) {
  if (B <= 0 || gamma_max_lower < 0 || gamma_max_lower > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (gamma_max_upper < 0 || gamma_max_upper > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (!ctx_len || !k_lower || !out_lower || !k_upper || !out_upper) return SR_EINVAL;
  if (!len_upper || !len_lower || !pending || !n_pending) return SR_EINVAL;
  return sr::launch_chain_consensus(ctx_len, k_lower, out_lower, gamma_max_lower, k_upper, out_upper,
                                    gamma_max_upper, B, len_upper, len_lower, pending, n_pending, status,
                                    (hipStream_t)stream);
}

int specrouter_kv_append(const void* k_new, const void* v_new, const int32_t* gamma, void* k_cache, void* v_cache,
                         uint8_t* cache_mask, int32_t* kv_len, const int32_t* shared_len, int B, int gamma_max,
                         int Hkv, int D, int L_cap, int32_t* status, void* stream) {
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA || Hkv <= 0 || L_cap <= 0) return SR_EINVAL;
  if (D != 64 && D != 128) return SR_EUNSUPPORTED;
  if (!k_new || !v_new || !gamma || !k_cache || !v_cache || !kv_len) return SR_EINVAL;
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) || !aligned16(v_cache)) return SR_EINVAL;
  return sr::launch_kv_append(k_new, v_new, gamma, k_cache, v_cache, cache_mask, kv_len, shared_len, B, gamma_max,
                              Hkv, D, L_cap, status, (hipStream_t)stream);
}

int specrouter_kv_compact(void* k_cache, void* v_cache, uint8_t* cache_mask, int32_t* kv_len, int B, int Hkv, int D,
                          int L_cap, int32_t* status, void* stream) {
  if (B <= 0 || Hkv <= 0 || L_cap <= 0) return SR_EINVAL;
  if (D != 64 && D != 128) return SR_EUNSUPPORTED;
  if (!k_cache || !v_cache || !cache_mask || !kv_len) return SR_EINVAL;
  if (!aligned16(k_cache) || !aligned16(v_cache)) return SR_EINVAL;
  return sr::launch_kv_compact(k_cache, v_cache, cache_mask, kv_len, B, Hkv, D, L_cap, status, (hipStream_t)stream);
}

int specrouter_rollback(int32_t* kv_len, uint8_t* cache_mask, const int32_t* new_len,
                        int32_t* phys_len, int B, int L_cap, int32_t* status, void* stream) {
  if (!kv_len || !new_len || B <= 0 || L_cap <= 0) return SR_EINVAL;
  return sr::launch_rollback(kv_len, cache_mask, new_len, phys_len, B, L_cap, status,
                             (hipStream_t)stream);
}

}  // extern "C"
