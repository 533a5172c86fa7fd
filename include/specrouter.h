/*
 * specrouter.h -- C ABI of the speculative-decoding verify step on MI355X (gfx950).
 *
 * One verify step at one verifier level of a multi-level speculative-decoding
 * chain (SpecRouter, arXiv 2505.07680) is three calls, enqueued in this order
 * on one stream:
 *
 *   specrouter_verify_attention    attention of the gamma_b + 1 new query rows of
 *                                  every sequence against that sequence's own KV
 *                                  cache, under the logical validity mask
 *                                  (Section 2.2 step 2; Section 4.4, Eq. 8);
 *   specrouter_accept_and_diverge  speculative accept/reject of the drafts with
 *                                  residual resampling and the bonus token
 *                                  (Section 2.2 steps 3-4), plus per-position
 *                                  total variation distance (Eq. 5) and KL
 *                                  divergence that feed the chain scheduler's
 *                                  similarity estimate (Section 4.2, Eq. 6);
 *   specrouter_rollback            logical rollback of every sequence's cache to
 *                                  its accepted prefix, no KV data moved
 *                                  (Section 4.4, rollback mechanism, Eq. 9).
 *
 * Conventions shared by every call
 *   - Pointers named in a signature are DEVICE (HBM) pointers owned by the
 *     caller unless stated otherwise. The library never allocates, frees or
 *     keeps a pointer after a call returns, and never synchronizes: each call
 *     only enqueues kernels on `stream` (a hipStream_t passed as void*; NULL =
 *     the default stream) and returns.
 *   - Return value: SR_OK, or a negative SR_E* code for an error detected on the
 *     host before anything was enqueued (bad sizes, NULL or misaligned
 *     pointers, a workspace that is too small) or a failed launch.
 *   - Values that live on the device (lengths, gamma, tokens, uniforms) cannot
 *     be checked on the host without a synchronization; they are checked by the
 *     kernels, which OR SR_ST_* bits into *status (if status is non-NULL; the
 *     caller clears it) and give the affected sequence defined "invalid"
 *     outputs instead of computing on bad data.
 *   - Calls that share a workspace, or whose outputs alias, must not overlap
 *     in time (put them on one stream). Different calls on different streams
 *     with separate buffers are independent. The library holds no global state
 *     beyond cached device properties and the fixed per-device array of
 *     specrouter_accept_and_rollback_noalloc (whose calls share it), so every
 *     other entry point is reentrant and thread-safe.
 *
 * Shapes: B sequences; gamma_max >= max_b gamma_b (0..16); Hq query heads and
 * Hkv kv heads with Hq % Hkv == 0 (query head h reads kv head h / (Hq/Hkv));
 * head dimension D in {64, 128}; L_cap cache rows per (sequence, kv head),
 * at most SPECROUTER_MAX_CACHE_ROWS for the attention call (its slabs are
 * addressed with 32-bit byte offsets); vocabulary size V.
 */
#ifndef SPECROUTER_H
#define SPECROUTER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPECROUTER_ABI_VERSION 5
#define SPECROUTER_MAX_GAMMA 16
#define SPECROUTER_MAX_CACHE_ROWS (1 << 22)
/* Size of the library's own device array behind specrouter_accept_and_rollback_noalloc. */
#define SPECROUTER_NOALLOC_SCRATCH_BYTES (16u << 20)

/* Host-side return codes. */
enum {
  SR_OK = 0,
  SR_EINVAL = -1,       /* bad size, NULL required pointer, misaligned pointer */
  SR_EUNSUPPORTED = -2, /* D not in {64,128}, unknown logits dtype */
  SR_EWORKSPACE = -3,   /* workspace NULL or smaller than the *_workspace_size query */
  SR_ELAUNCH = -4,      /* the HIP runtime refused a launch or a device query */
  SR_ESCRATCH = -5,     /* the problem needs more workspace than the library's fixed array holds */
};

/* Logits element types. */
enum { SR_F32 = 0, SR_BF16 = 1 };

/* Device-side data-error bits OR-ed into *status. */
enum {
  SR_ST_GAMMA = 1,          /* gamma_b outside [0, gamma_max] */
  SR_ST_KVLEN = 2,          /* kv_len_b outside its valid range, or a negative new_len_b */
  SR_ST_TOKEN = 4,          /* a draft token outside [0, V) */
  SR_ST_UNIFORM = 8,        /* a needed uniform outside [0, 1) (NaN included) */
  SR_ST_ROLLBACK_GROW = 16, /* rollback asked to grow a sequence (treated as a no-op) */
  SR_ST_TIMEOUT = 32,       /* not set since ABI version 4 (accept waits are bounded and recover) */
  SR_ST_CHAIN = 64,         /* accept lengths that one chain step cannot produce */
};

/* SPECROUTER_ABI_VERSION of the loaded library. */
int specrouter_abi_version(void);

/* Static English text for an SR_E* return code or a single SR_ST_* bit. Never NULL. */
const char* specrouter_status_string(int code);

/* ------------------------------------------------------------------------ */
/* Verification attention (Section 2.2 step 2; Section 4.4, Eq. 8).
 *
 * For sequence b, query head h (kv head g = h / (Hq/Hkv)) and new row
 * i in [0, gamma_b], at cache position pos = kv_len_b - (gamma_b + 1) + i:
 *
 *   out[b][i][h][:] = softmax_j(scale * q[b][i][h] . k[b][g][j]) v[b][g][j]
 *
 * over the keys j <= pos with cache_mask[b][j] != 0 (all j < kv_len_b when
 * cache_mask is NULL). Entries under mask 0 or at j >= kv_len_b are ignored
 * whatever they hold (even NaN/Inf). A row with no visible key, and every row
 * i > gamma_b, is written as 0. The caller has already written this step's
 * gamma_b + 1 new K/V rows at [kv_len_b - gamma_b - 1, kv_len_b).
 *
 * q          bf16 [B][gamma_max+1][Hq][D]          (16-byte aligned)
 * k_cache    bf16 [B][Hkv][L_cap][D]               (16-byte aligned)
 * v_cache    bf16 [B][Hkv][L_cap][D]               (16-byte aligned)
 * cache_mask u8   [B][L_cap] in {0,1}, or NULL
 * kv_len     i32  [B]  valid physical length incl. the new rows; must lie in
 *                      [gamma_b + 1, L_cap], else SR_ST_KVLEN and zero output
 * gamma      i32  [B]  in [0, gamma_max] (0 = plain decode), else SR_ST_GAMMA
 * out        fp32 [B][gamma_max+1][Hq][D]          (16-byte aligned)
 * scale      score scale, normally 1/sqrt(D); must be positive and finite (else SR_EINVAL)
 * workspace  device scratch of specrouter_verify_attention_workspace_size()
 *            bytes (may be NULL when that size is 0). Zero-fill it once before
 *            its first use; every call leaves its counters zero again (it holds
 *            per-(sequence, kv head, query chunk) arrival counters of the cache
 *            splits, their partial results, and, when the call has more
 *            workgroups than fit on the device at once, their dispatch order,
 *            rewritten by every call)
 * Precision: bf16 products, fp32 accumulation and softmax, in a fixed order
 * (repeated calls give identical bits).
 */
size_t specrouter_verify_attention_workspace_size(int B, int gamma_max, int Hq, int Hkv, int D,
                                                  int L_cap);
int specrouter_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                                const uint8_t* cache_mask, const int32_t* kv_len,
                                const int32_t* gamma, float* out, int B, int gamma_max, int Hq,
                                int Hkv, int D, int L_cap, float scale, void* workspace,
                                size_t workspace_bytes, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* Accept and diverge (Section 2.2 steps 3-4, probabilistic acceptance; Eq. 2;
 * Eq. 5), one sweep over the logits.
 *
 * With p_j = softmax(p_logits[b][j]) (j = 0..gamma_b) and
 * q_j = softmax(q_logits[b][j]) (j < gamma_b), for each sequence b:
 *   a_j  = min(1, p_j(x_j) / q_j(x_j)), x_j = draft_tokens[b][j];
 *   k_b  = first j < gamma_b with NOT (u_accept[b][j] < a_j), else gamma_b;
 *   t_b  = one token drawn by CDF inversion (ascending vocabulary order,
 *          smallest x with C(x) > u_resample[b][k_b] * C(V-1)) from
 *          max(0, p_k - q_k) if k_b < gamma_b (p_k if that residual is all
 *          zero), else from p_gamma;
 *   TV_j = 1/2 sum_v |p_j - q_j|,  KL_j = KL(p_j || q_j) in nats, j < gamma_b.
 *
 * p_logits      [B][gamma_max+1][V], rows contiguous, batch stride
 *               p_batch_stride ELEMENTS; rows j > gamma_b are never read
 * q_logits      [B][gamma_max][V], batch stride q_batch_stride elements (may be
 *               a view into another level's p_logits); rows j >= gamma_b never read
 * logits_dtype  SR_F32 or SR_BF16 (both tensors; bf16 is widened in-kernel)
 * draft_tokens  i32 [B][gamma_max];  gamma i32 [B]
 * u_accept      fp32 [B][gamma_max] in [0,1);  u_resample fp32 [B][gamma_max+1] in [0,1)
 * kv_len        i32 [B] or NULL; when given, new_len[b] = kv_len[b] - gamma_b + k_b
 *               (the accepted prefix, ready for specrouter_rollback)
 * accept_len    i32 [B]: k_b, or -1 for a sequence with bad data
 * out_tokens    i32 [B][gamma_max+1]: x_0..x_{k-1}, t_b, then -1
 * new_len       i32 [B] or NULL (must be NULL when kv_len is NULL); -> kv_len[b]
 *               unchanged for a sequence with bad data
 * accept_prob, p_tok, q_tok, kl, tv: fp32 [B][gamma_max] or NULL each; entries
 *               j >= gamma_b (and all entries of a bad sequence) are NaN
 * workspace     device scratch of specrouter_accept_workspace_size() bytes; it
 *               must be zero-filled before its FIRST use and every call leaves
 *               it zero-filled again, whatever shape the next call has (each
 *               call clears every word it wrote)
 * Logits must be finite or -inf, with |logit| / T < 2^23; a row that is
 * entirely -inf is not supported. Any V from 1 to 524281: rows need no
 * alignment, but the logits pointers and the batch strides (in bytes) must be
 * multiples of 16, else SR_EUNSUPPORTED (with V * element size not a multiple
 * of 16, allocate each sequence's rows with a padded batch stride).
 * The kernels need no co-residency of their workgroups: no workgroup waits
 * without bound (a bounded wait for the other chunks of a row falls back to
 * recomputing that chunk's sum later), so other work on the device slows the
 * call down but never stalls it; repeated calls give identical bits.
 */
size_t specrouter_accept_workspace_size(int B, int gamma_max, int V, int logits_dtype);
int specrouter_accept_and_diverge(const void* p_logits, int64_t p_batch_stride,
                                  const void* q_logits, int64_t q_batch_stride, int logits_dtype,
                                  const int32_t* draft_tokens, const int32_t* gamma,
                                  const float* u_accept, const float* u_resample,
                                  const int32_t* kv_len, int32_t* accept_len,
                                  int32_t* out_tokens, int32_t* new_len, float* accept_prob,
                                  float* p_tok, float* q_tok, float* kl, float* tv, int B,
                                  int gamma_max, int V, void* workspace, size_t workspace_bytes,
                                  int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* Accept and diverge under a sampling rule (Section 2.2 step 3: the chosen
 * sampling rule, greedy or probabilistic acceptance; the sampling parameters
 * of the logits processors, Section 4.1).
 *
 * temperature T > 0: every distribution of specrouter_accept_and_diverge
 *   becomes softmax(logits / T) -- p and q, the acceptance test, the residual
 *   and bonus draws, TV and KL alike (T = 1 is specrouter_accept_and_diverge).
 *   The drafts are assumed drawn from the draft model's softmax(logits / T).
 * temperature 0: greedy decoding. p_j and q_j are one-hot at their argmax
 *   (the lowest vocabulary index among equal maxima); draft x_j is accepted
 *   iff x_j == argmax p_j, and the extra token is argmax p_k. u_accept and
 *   u_resample are not read (may be NULL); accept_prob, p_tok and q_tok are 1
 *   or 0, TV_j is 0 when argmax p_j == argmax q_j and 1 otherwise, KL_j is 0
 *   or +infinity likewise. No SR_ST_UNIFORM check is made.
 * top_k, top_p (T > 0 only; greedy decoding keeps the argmax anyway): the
 *   logits processors after the temperature, applied to every verifier row
 *   and every draft row alike (the drafts are assumed drawn from the filtered
 *   draft distribution); every output is then computed on the filtered
 *   distributions. top_k in [1, V) keeps the logits that are at least the
 *   k-th largest (ties with it all kept); 0 or >= V is off. top_p in (0, 1)
 *   keeps a logit iff the mass, under softmax of what top-k kept, of the
 *   strictly larger logits is below top_p (ties kept or dropped together;
 *   the largest logit always stays); 1 is off. top_k < 0 or top_p outside
 *   (0, 1] is SR_EINVAL. With a filter on, one extra kernel finds each row's
 *   threshold first (a radix select over the row); top-p decides on fp32
 *   masses, so a logit whose larger mass is within ~1e-7 of top_p may fall
 *   either way.
 * A NULL sampling pointer means temperature 1. The sampling struct is a host
 * pointer, read before the call returns. temperature must be finite and >= 0
 * (else SR_EINVAL). All other arguments, the workspace and the outputs are as
 * for specrouter_accept_and_diverge.
 */
typedef struct specrouter_sampling {
  float temperature;
  int top_k;
  float top_p;
} specrouter_sampling;

int specrouter_accept_and_diverge_sampled(const void* p_logits, int64_t p_batch_stride,
                                          const void* q_logits, int64_t q_batch_stride,
                                          int logits_dtype, const int32_t* draft_tokens,
                                          const int32_t* gamma, const float* u_accept,
                                          const float* u_resample, const int32_t* kv_len,
                                          int32_t* accept_len, int32_t* out_tokens,
                                          int32_t* new_len, float* accept_prob, float* p_tok,
                                          float* q_tok, float* kl, float* tv, int B,
                                          int gamma_max, int V,
                                          const specrouter_sampling* sampling, void* workspace,
                                          size_t workspace_bytes, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* Rollback (Section 4.4, logical rollback and Eq. 9).
 *
 * For every sequence: n = min(kv_len[b], new_len[b]); cache_mask[b][n:kv_len[b]) = 0;
 * kv_len[b] = n. Idempotent (new_len holds absolute lengths L'_b). No K/V byte
 * is read or written. phys_len = max_b kv_len[b] afterwards, which is Eq. 9's
 * L - r_min when every sequence started at the common length L.
 *
 * kv_len      i32 [B] in/out; entries outside [0, L_cap] set SR_ST_KVLEN and are
 *             left unchanged
 * cache_mask  u8 [B][L_cap] in/out, or NULL
 * new_len     i32 [B]; negative -> SR_ST_KVLEN (unchanged), > kv_len ->
 *             SR_ST_ROLLBACK_GROW (unchanged)
 * phys_len    i32 [1] out, or NULL
 */
int specrouter_rollback(int32_t* kv_len, uint8_t* cache_mask, const int32_t* new_len,
                        int32_t* phys_len, int B, int L_cap, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* Accept-and-diverge followed by the rollback, in one call (Section 2.2
 * steps 3-4 and Section 4.4): the same results as
 * specrouter_accept_and_diverge_sampled(...) with these arguments, then
 * specrouter_rollback(cache_kv_len, cache_mask, <its new_len>, phys_len, B,
 * L_cap, status), bit for bit -- outputs, lengths, mask, phys_len and status
 * bits. The rollback of each sequence is done by the accept's own finishing
 * step as soon as that sequence's outcome is known, so the verify step needs
 * one launch fewer.
 *
 * kv_len        required here (the accept's new length is kv_len - gamma_b + k_b)
 * new_len       may be NULL (the rollback uses the value internally)
 * cache_kv_len  i32 [B] in/out, the lengths rolled back (may be kv_len itself)
 * cache_mask    u8 [B][L_cap] in/out, or NULL
 * phys_len      i32 [1] out (max over sequences of the new lengths), or NULL
 * L_cap         > 0, the cache rows per sequence
 * The workspace is the accept's (specrouter_accept_workspace_size); a call of
 * either accept entry point leaves it ready for the other.
 */
int specrouter_accept_and_rollback(const void* p_logits, int64_t p_batch_stride, const void* q_logits,
                                   int64_t q_batch_stride, int logits_dtype, const int32_t* draft_tokens,
                                   const int32_t* gamma, const float* u_accept, const float* u_resample,
                                   const int32_t* kv_len, int32_t* accept_len, int32_t* out_tokens,
                                   int32_t* new_len, float* accept_prob, float* p_tok, float* q_tok, float* kl,
                                   float* tv, int B, int gamma_max, int V, const specrouter_sampling* sampling,
                                   int32_t* cache_kv_len, uint8_t* cache_mask, int32_t* phys_len, int L_cap,
                                   void* workspace, size_t workspace_bytes, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* specrouter_accept_and_rollback without a workspace argument, for callers
 * that cannot allocate device memory: code under HIP graph capture, serving
 * loops that must not allocate, harnesses that forbid it.
 *
 * Same arguments, results and kernels as specrouter_accept_and_rollback minus
 * (workspace, workspace_bytes): the workspace is a fixed array of
 * SPECROUTER_NOALLOC_SCRATCH_BYTES in device memory that the library owns,
 * one per device, resident until the process ends. The call allocates
 * nothing. It returns SR_ESCRATCH, before touching the device, when the
 * workspace this shape needs (specrouter_accept_workspace_size) exceeds the
 * array. The first call on a device also enqueues one clearing kernel on
 * `stream` (and so does the first call after a call that failed with
 * SR_ELAUNCH); every call leaves the array ready for the next.
 * Calls on one device share its array: calls that overlap in time on one
 * device (different streams, threads or processes' graphs) race and give
 * wrong results; serialise them, e.g. on one stream.
 */
int specrouter_accept_and_rollback_noalloc(
    const void* p_logits, int64_t p_batch_stride, const void* q_logits, int64_t q_batch_stride, int logits_dtype,
    const int32_t* draft_tokens, const int32_t* gamma, const float* u_accept, const float* u_resample,
    const int32_t* kv_len, int32_t* accept_len, int32_t* out_tokens, int32_t* new_len, float* accept_prob,
    float* p_tok, float* q_tok, float* kl, float* tv, int B, int gamma_max, int V,
    const specrouter_sampling* sampling, int32_t* cache_kv_len, uint8_t* cache_mask, int32_t* phys_len,
    int L_cap, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* KV-cache state (Section 4.4, StateManager: logical validity mask, Eq. 8;
 * rollback and physical truncation, Eq. 9). Device pointers; cache layout as
 * for specrouter_verify_attention; D in {64, 128}; K/V bytes are moved
 * verbatim.
 *
 * specrouter_kv_append: write a step's new rows -- the pending token and the
 * drafts, gamma_b + 1 rows of k_new/v_new bf16 [B][gamma_max+1][Hkv][D]
 * (16-byte aligned) -- at the sequence's cursor, mark them valid in
 * cache_mask (if not NULL) and set kv_len[b] = cursor + gamma_b + 1. The
 * cursor is kv_len[b] when shared_len is NULL (per-sequence layout), else
 * *shared_len, one physical length for the whole batch (the paper's layout:
 * a sequence that rolled back further than the others keeps masked holes
 * between its last valid row and the shared length; rows are never shifted).
 * A sequence with gamma_b outside [0, gamma_max] (SR_ST_GAMMA), kv_len[b]
 * outside [0, L_cap] or cursor + gamma_b + 1 > L_cap (SR_ST_KVLEN) is left
 * untouched. *shared_len is not changed: after a rollback it is the
 * rollback's phys_len (Eq. 9's L - r_min); after an append it is the largest
 * new kv_len.
 *
 * specrouter_kv_compact: reclaim the holes. For every sequence the rows j <
 * kv_len[b] with cache_mask[b][j] != 0 move, in order and in place, to the
 * front; the mask becomes 1 on [0, n) and 0 on [n, old kv_len[b]); kv_len[b]
 * = n. Rows past n keep stale bytes (masked). Attention over the compacted
 * cache equals attention over the holed one. Two kernels; reads and writes
 * every K/V row from the first hole on.
 */
int specrouter_kv_append(const void* k_new, const void* v_new, const int32_t* gamma,
                         void* k_cache, void* v_cache, uint8_t* cache_mask, int32_t* kv_len,
                         const int32_t* shared_len, int B, int gamma_max, int Hkv, int D,
                         int L_cap, int32_t* status, void* stream);
int specrouter_kv_compact(void* k_cache, void* v_cache, uint8_t* cache_mask, int32_t* kv_len,
                          int B, int Hkv, int D, int L_cap, int32_t* status, void* stream);

/* ------------------------------------------------------------------------ */
/* Multi-level chains (Section 3.1, multi-level verification; Section 4.3,
 * VerifyProcessor repeated per level and RollbackProcessor's consensus).
 *
 * A chain step with drafter M1, an intermediate verifier and an upper
 * verifier is: the intermediate level's verify step (attention, accept),
 * specrouter_chain_window, the upper level's verify step with q_logits set to
 * the intermediate level's p_logits rows (a strided view), then
 * specrouter_chain_consensus and one specrouter_rollback per level. The
 * tokens the upper level verifies are exact samples of the intermediate
 * level's distribution and the window length is fixed before each of them is
 * drawn, so the step emits tokens of the upper level's distribution. Longer
 * chains repeat the pair of calls level by level.
 */

/* Window of the next verifier level (device pointers; stream as above).
 * accept_len  i32 [B]: k_b of the level below (-1 for a flagged sequence)
 * out_tokens  i32 [B][gamma_max+1]: its emitted tokens
 * gamma_cap   the next level's window limit (1..SPECROUTER_MAX_GAMMA)
 * ctx_len     i32 [B] or NULL: committed context length (without the pending
 *             token) of the next level's cache
 * gamma_next  i32 [B] out: min(k_b + 1, gamma_cap), or -1 when k_b < 0 or
 *             k_b > gamma_max (the next level then flags SR_ST_GAMMA)
 * drafts_next i32 [B][gamma_cap] out: the first gamma_next_b emitted tokens,
 *             then 0
 * kv_len_next i32 [B] out or NULL (NULL exactly when ctx_len is NULL):
 *             ctx_len_b + 1 + max(gamma_next_b, 0), the next level's length
 *             once its K/V rows for the pending token and the drafts are
 *             written */
int specrouter_chain_window(const int32_t* accept_len, const int32_t* out_tokens, int B,
                            int gamma_max, int gamma_cap, const int32_t* ctx_len,
                            int32_t* gamma_next, int32_t* drafts_next, int32_t* kv_len_next,
                            void* stream);

/* Consensus after the upper level (device pointers).
 * ctx_len    i32 [B]: committed context length before the step (every level
 *            then holds one row for the previous step's pending token)
 * k_lower, out_lower [B], [B][gamma_max_lower+1]: the intermediate level's
 *            accept lengths and emitted tokens
 * k_upper, out_upper [B], [B][gamma_max_upper+1]: the upper level's
 * len_upper  i32 [B] out: ctx + 1 + k_upper (rows the upper level keeps)
 * len_lower  i32 [B] out: ctx + 1 + min(k_lower, k_upper) (rows the
 *            intermediate and draft levels keep)
 * pending    i32 [B][2] out: the tokens the lower levels must run first in
 *            the next step -- out_lower[k_lower] when k_upper == k_lower + 1,
 *            then out_upper[k_upper] -- padded with -1; the upper level's only
 *            pending token is the last of them
 * n_pending  i32 [B] out: 1 or 2 (0 for a sequence a level flagged)
 * A flagged sequence (k < 0) keeps ctx rows and gets no pending token; so does
 * one whose lengths one chain step cannot produce (k_upper > k_lower + 1 or a
 * length past its window), which also sets SR_ST_CHAIN in *status. */
int specrouter_chain_consensus(const int32_t* ctx_len, const int32_t* k_lower,
                               const int32_t* out_lower, int gamma_max_lower,
                               const int32_t* k_upper, const int32_t* out_upper,
                               int gamma_max_upper, int B, int32_t* len_upper,
                               int32_t* len_lower, int32_t* pending, int32_t* n_pending,
                               int32_t* status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPECROUTER_H */
