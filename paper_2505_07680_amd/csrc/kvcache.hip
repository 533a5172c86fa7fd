// KV-cache state updates around the verify step (Section 4.4, StateManager):
//
//   kv_append:  a step's gamma_b + 1 new K/V rows (the pending token and the
//               drafts) written at the sequence's cursor and marked valid.
//               The cursor is the sequence's own length, or one physical
//               length shared by the batch (the paper's layout: a sequence
//               that rolled back further keeps masked holes below it).
//   kv_compact: optional reclamation of the holes: each sequence's valid
//               rows moved to the front in order (in place), then the mask
//               and length rewritten.
//
// K/V bytes move verbatim (16-byte vector loads and stores).

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kKvThreads = 256;

// One workgroup per sequence: the cursor is read once, every row chunk is
// copied, then the length is advanced (the only writer of kv_len[b]).
__global__ void __launch_bounds__(kKvThreads)
kv_append_kernel(const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new,
                 const int32_t* __restrict__ gamma, u32x4* __restrict__ k_cache, u32x4* __restrict__ v_cache,
                 uint8_t* __restrict__ mask, int32_t* __restrict__ kv_len, const int32_t* __restrict__ shared_len,
                 int gmax, int Hkv, int D, int L_cap, int32_t* __restrict__ status) {
  __shared__ int s_cur, s_n;
  const int b = blockIdx.x;
  if (threadIdx.x == 0) {
    const int g = gamma[b];
    const int L = kv_len[b];
    const int cur = shared_len ? *shared_len : L;
    int n = g + 1;
    uint32_t bad = 0;
    if (g < 0 || g > gmax) bad |= SR_ST_GAMMA;
    else if (L < 0 || L > L_cap || cur < 0 || cur + n > L_cap) bad |= SR_ST_KVLEN;
    if (bad) {
      n = 0;
      if (status) atomicOr(status, (int32_t)bad);
    }
    s_cur = cur;
    s_n = n;
  }
  __syncthreads();
  const int cur = s_cur, n = s_n;
  const int cpr = D / 8;  // 16-byte chunks per row
  const int total = n * Hkv * cpr;
  for (int idx = threadIdx.x; idx < total; idx += kKvThreads) {
    const int c = idx % cpr;
    const int h = (idx / cpr) % Hkv;
    const int i = idx / (cpr * Hkv);
    const size_t src = (((size_t)b * (gmax + 1) + i) * Hkv + h) * cpr + c;
    const size_t dst = (((size_t)b * Hkv + h) * L_cap + cur + i) * cpr + c;
    k_cache[dst] = k_new[src];
    v_cache[dst] = v_new[src];
  }
  if (mask)
    for (int i = threadIdx.x; i < n; i += kKvThreads) mask[(size_t)b * L_cap + cur + i] = 1;
  if (threadIdx.x == 0 && n > 0) kv_len[b] = cur + n;
}

// Compaction of one (sequence, kv head) slab, in place, 64 positions per
// block: the valid rows' destinations come from a wave prefix sum of the mask;
// a block's rows are all loaded (and the loads completed) before any of them
// is stored, and a row only moves to a lower position, so no row is
// overwritten before it has been read.
__global__ void __launch_bounds__(kKvThreads)
kv_compact_kernel(u32x4* __restrict__ k_cache, u32x4* __restrict__ v_cache, const uint8_t* __restrict__ mask,
                  const int32_t* __restrict__ kv_len, int Hkv, int D, int L_cap) {
  __shared__ int s_dst[64];
  __shared__ int s_cnt;
  const int b = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  const int L = kv_len[b];
  if (L < 0 || L > L_cap) return;  // reported by the mask kernel
  const int cpr = D / 8;
  const int per = cpr / 4;  // chunks of a row per thread (four threads per row)
  const int tid = threadIdx.x;
  const int p_local = tid / 4, quarter = tid % 4;
  u32x4* kslab = k_cache + ((size_t)b * Hkv + h) * L_cap * cpr;
  u32x4* vslab = v_cache + ((size_t)b * Hkv + h) * L_cap * cpr;
  int offset = 0;  // valid rows before this block
  for (int base = 0; base < L; base += 64) {
    if (tid < 64) {
      const int p = base + tid;
      const int valid = p < L && mask[(size_t)b * L_cap + p] != 0;
      const int incl = wave_incl_scan_i(valid);
      s_dst[tid] = valid ? offset + incl - 1 : -1;
      if (tid == 63) s_cnt = incl;
    }
    __syncthreads();
    const int cnt = s_cnt;
    const bool in_place = cnt == min(64, L - base) && offset == base;  // block-uniform: nothing moves
    const int p = base + p_local;
    const int dst = s_dst[p_local];
    u32x4 kr[4], vr[4];
    const bool move = !in_place && dst >= 0 && dst != p;
    if (move) {
      for (int c = 0; c < per; ++c) {
        kr[c] = kslab[(size_t)p * cpr + quarter * per + c];
        vr[c] = vslab[(size_t)p * cpr + quarter * per + c];
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // every load of this block has returned before any store
    __syncthreads();
    if (move) {
      for (int c = 0; c < per; ++c) {
        kslab[(size_t)dst * cpr + quarter * per + c] = kr[c];
        vslab[(size_t)dst * cpr + quarter * per + c] = vr[c];
      }
    }
    offset += cnt;
    __syncthreads();  // s_dst and s_cnt are rewritten by the next block
  }
}

// After every slab of a sequence moved: mask = 1 on the new prefix, 0 up to
// the old length; kv_len = the count of valid rows.
__global__ void __launch_bounds__(kKvThreads)
kv_compact_mask_kernel(uint8_t* __restrict__ mask, int32_t* __restrict__ kv_len, int L_cap,
                       int32_t* __restrict__ status) {
  __shared__ int s_part[kKvThreads / 64];
  const int b = blockIdx.x;
  const int L = kv_len[b];
  if (L < 0 || L > L_cap) {
    if (threadIdx.x == 0 && status) atomicOr(status, (int32_t)SR_ST_KVLEN);
    return;
  }
  int cnt = 0;
  for (int p = threadIdx.x; p < L; p += kKvThreads) cnt += mask[(size_t)b * L_cap + p] != 0;
  const int w = wave_id();
  const int tot = wave_incl_scan_i(cnt);
  if ((threadIdx.x & 63) == 63) s_part[w] = tot;
  __syncthreads();
  int n = 0;
  for (int i = 0; i < kKvThreads / 64; ++i) n += s_part[i];
  __syncthreads();  // every count is read before the mask changes
  for (int p = threadIdx.x; p < L; p += kKvThreads) mask[(size_t)b * L_cap + p] = p < n ? 1 : 0;
  if (threadIdx.x == 0) kv_len[b] = n;
}

}  // namespace

int launch_kv_append(const void* k_new, const void* v_new, const int32_t* gamma, void* k_cache, void* v_cache,
                     uint8_t* cache_mask, int32_t* kv_len, const int32_t* shared_len, int B, int gamma_max,
                     int Hkv, int D, int L_cap, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(kv_append_kernel, dim3(B), dim3(kKvThreads), 0, stream, (const u32x4*)k_new,
                     (const u32x4*)v_new, gamma, (u32x4*)k_cache, (u32x4*)v_cache, cache_mask, kv_len, shared_len,
                     gamma_max, Hkv, D, L_cap, status);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

int launch_kv_compact(void* k_cache, void* v_cache, uint8_t* cache_mask, int32_t* kv_len, int B, int Hkv, int D,
                      int L_cap, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(kv_compact_kernel, dim3((unsigned)(B * Hkv)), dim3(kKvThreads), 0, stream,
                     (u32x4*)k_cache, (u32x4*)v_cache, (const uint8_t*)cache_mask, (const int32_t*)kv_len, Hkv, D,
                     L_cap);
  if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  hipLaunchKernelGGL(kv_compact_mask_kernel, dim3(B), dim3(kKvThreads), 0, stream, cache_mask, kv_len, L_cap,
                     status);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

}  // namespace sr
