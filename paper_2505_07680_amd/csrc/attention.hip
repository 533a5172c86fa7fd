// Verification attention for gfx950 (Section 2.2 step 2; Section 4.4, Eq. 8).
//
// Work decomposition. One workgroup (4 waves) handles one (sequence b, kv head
// g, query chunk, key split). All G*(gamma_b+1) query rows that read kv head g
// (the GQA group times the new positions) are processed together, so every K/V
// byte of the split is read from HBM exactly once. Each wave owns 16 of every
// 64 keys and keeps its own online-softmax state (no workgroup barrier inside
// the key loop); the four states are merged through LDS at the end. Splits of
// one (b, g) are merged by a small combine kernel (skipped when one split
// covers the cache).
//
// Per 16-key wave tile:
//   * K and V rows are fetched with coalesced 16-byte loads into a two-deep
//     register ring, so two tiles are in flight while one is computed, and
//     staged in a wave-private LDS slot; V rows that are invalid (past the
//     split/kv_len, or mask 0) are zeroed while staging, so whatever those
//     rows hold never reaches the output;
//   * S^T = K Q^T on MFMA (v_mfma_f32_16x16x32_bf16: 16 keys x 16 queries per
//     block, K=32 over the head dimension); each lane then holds 4 scores of
//     ONE query, so the softmax max/sum need only two cross-lane steps;
//   * P is rounded to bf16 in place: its accumulator layout is exactly the B
//     operand of O^T += V^T P^T (v_mfma_f32_16x16x16_bf16, K=16 over the keys);
//     the V^T operand is gathered from LDS with 16-bit reads.
// Scores are kept in log2 units (scale * log2(e) folded in) and exponentiated
// with exp2.

#include "sr_internal.h"

namespace sr {
namespace {

typedef short shortx4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kWaveKeys = 16;
constexpr int kTileKeys = kWaves * kWaveKeys;
constexpr int kMaxNQ = 5;

template <int D>
struct Geo {
  static constexpr int kKStride = D * 2 + 16;  // LDS bytes per staged K (and Q) row
  static constexpr int kVStride = D * 2 + 8;   // LDS bytes per staged V row
  static constexpr int kChunksPerRow = D / 8;  // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 64 / kChunksPerRow;
  static constexpr int kLoads = kWaveKeys / kRowsPerLoad;  // 16-byte loads per lane per tensor per tile
  static constexpr int kSlotK = kWaveKeys * kKStride;
  static constexpr int kWaveBytes = kSlotK + kWaveKeys * kVStride;
};

template <int D, int NQ>
struct Lds {
  static constexpr int MQ = 16 * NQ;
  static constexpr int kStage = kWaves * Geo<D>::kWaveBytes + MQ * Geo<D>::kKStride;
  static constexpr int kComb = 2 * MQ * (D + 2) * 4;
  static constexpr int kBytes = kStage > kComb ? kStage : kComb;
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo;
  const __bf16 b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Order LDS accesses of one wave around a point (compiler barrier; the LDS
// unit serves one wave's requests in order).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int D>
struct Stage {  // one 16-key wave tile in flight
  u32x4 k[Geo<D>::kLoads], v[Geo<D>::kLoads];
  uint32_t mbyte;  // validity byte of key (lane mod 16), evaluated when consumed
};

// 2 waves per SIMD for up to 3 query groups (all fits in 256 registers).
template <int NQ>
struct Occ {
  static constexpr int kMinWaves = NQ <= 3 ? 2 : 1;
};

template <int D, int NQ>
__global__ void __launch_bounds__(kThreads, Occ<NQ>::kMinWaves)
attn_split_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
                  const uint16_t* __restrict__ vc, const uint8_t* __restrict__ mask,
                  const int32_t* __restrict__ kv_len, const int32_t* __restrict__ gamma,
                  float* __restrict__ out, float* __restrict__ part_o,
                  float* __restrict__ part_ml, int gmax, int Hq, int Hkv, int L_cap,
                  float scale_log2, int split_keys, int n_splits, int32_t* __restrict__ status) {
  using GG = Geo<D>;
  constexpr int MQ = 16 * NQ;
  constexpr int DB = D / 16;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Lds<D, NQ>::kBytes];

  const int split = blockIdx.x;
  const int g = blockIdx.y % Hkv;
  const int qc = blockIdx.y / Hkv;
  const int b = blockIdx.z;
  const int G = Hq / Hkv;
  const int R = G * (gmax + 1);
  const int gam = gamma[b];
  const int L = kv_len[b];
  const bool valid = gam >= 0 && gam <= gmax && L >= gam + 1 && L <= L_cap;
  if (!valid && split == 0 && qc == 0 && g == 0 && threadIdx.x == 0 && status) {
    atomicOr(status, (gam < 0 || gam > gmax) ? SR_ST_GAMMA : SR_ST_KVLEN);
  }
  const int row0 = qc * MQ;
  const int row_end = min(R, row0 + MQ);
  const int Mb = valid ? G * (gam + 1) : 0;
  const int key_begin = split * split_keys;
  const int key_end = valid ? min(key_begin + split_keys, L) : 0;
  const bool work = row0 < Mb && key_begin < key_end;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int l16 = lane & 15;
  const int lg = lane >> 4;

  if (!work) {
    // Nothing to compute here. With a single split this workgroup owns the
    // output rows and writes them as zero; otherwise the combine kernel does.
    if (n_splits == 1) {
      for (int idx = tid; idx < (row_end - row0) * (D / 4); idx += kThreads) {
        const int r = row0 + idx / (D / 4);
        const int d4 = idx % (D / 4);
        const int i = r / G, h = g * G + r % G;
        *(float4*)(out + ((size_t)(b * (gmax + 1) + i) * Hq + h) * D + d4 * 4) = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    return;
  }

  // ---- stage this workgroup's query rows (bf16, zero beyond the live rows)
  unsigned char* qst = lds + kWaves * GG::kWaveBytes;
  for (int idx = tid; idx < MQ * GG::kChunksPerRow; idx += kThreads) {
    const int rl = idx / GG::kChunksPerRow;
    const int c = idx % GG::kChunksPerRow;
    const int r = row0 + rl;
    u32x4 val = u32x4{0u, 0u, 0u, 0u};
    if (r < Mb) {
      const int i = r / G, h = g * G + r % G;
      val = *(const u32x4*)(q + ((size_t)(b * (gmax + 1) + i) * Hq + h) * D + c * 8);
    }
    *(u32x4*)(qst + rl * GG::kKStride + c * 16) = val;
  }
  __syncthreads();

  unsigned char* kst = lds + w * GG::kWaveBytes;
  unsigned char* vst = kst + GG::kSlotK;
  const size_t slab = ((size_t)b * Hkv + g) * (size_t)L_cap;
  const uint16_t* kslab = kc + slab * D;
  const uint16_t* vslab = vc + slab * D;
  const uint8_t* mrow = mask ? mask + (size_t)b * L_cap : nullptr;
  const int causal0 = L - gam - 1;  // cache position of new row 0

  floatx4 o[DB][NQ];
  float m_run[NQ], l_run[NQ];
#pragma unroll
  for (int qg = 0; qg < NQ; ++qg) {
    m_run[qg] = kNegInf;
    l_run[qg] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][qg] = floatx4{0.f, 0.f, 0.f, 0.f};
  }

  const int n_tiles = (key_end - key_begin + kTileKeys - 1) / kTileKeys;

  // Loads are unconditional (rows clamped to the split's last valid key), so
  // the loop body issues a fixed number of loads per tile and each stage
  // waits only for its own loads; refetches past the end hit the same line.
  const uint8_t* mload = mrow ? mrow : (const uint8_t*)kslab;
  auto fetch = [&](int t, Stage<D>& st) __attribute__((always_inline)) {
    const int kb0 = key_begin + t * kTileKeys + w * kWaveKeys;
#pragma unroll
    for (int u = 0; u < GG::kLoads; ++u) {
      const int row = min(kb0 + u * GG::kRowsPerLoad + lane / GG::kChunksPerRow, key_end - 1);
      const size_t off = (size_t)row * D + (lane % GG::kChunksPerRow) * 8;
      st.k[u] = *(const u32x4*)(kslab + off);
      st.v[u] = *(const u32x4*)(vslab + off);
    }
    st.mbyte = mload[min(kb0 + (lane & (kWaveKeys - 1)), key_end - 1)];
  };

  auto consume = [&](int t, Stage<D>& st) __attribute__((always_inline)) {
    const int kb0 = key_begin + t * kTileKeys + w * kWaveKeys;
    const bool key_ok = lane < kWaveKeys && kb0 + lane < key_end && (mrow == nullptr || st.mbyte != 0u);
    const uint32_t vbits = (uint32_t)__ballot(key_ok) & 0xffffu;
#pragma unroll
    for (int u = 0; u < GG::kLoads; ++u) {
      const int rl = u * GG::kRowsPerLoad + lane / GG::kChunksPerRow;
      const int c = lane % GG::kChunksPerRow;
      *(u32x4*)(kst + rl * GG::kKStride + c * 16) = st.k[u];
      const u32x4 vv = ((vbits >> rl) & 1u) ? st.v[u] : u32x4{0u, 0u, 0u, 0u};
      uint32_t* dst = (uint32_t*)(vst + rl * GG::kVStride + c * 16);
      *(uint2*)dst = make_uint2(vv.x, vv.y);
      *(uint2*)(dst + 2) = make_uint2(vv.z, vv.w);
    }
    wave_lds_sync();
    fetch(t + 2, st);  // refill this ring entry: two tiles in flight during the compute below
    if (t >= n_tiles || kb0 >= key_end) return;  // wave-uniform: nothing of this tile to compute
    // ---- S^T = K Q^T (16 keys x 16 queries per group)
    floatx4 sacc[NQ];
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) sacc[qg] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const int col = (ks * 32 + lg * 8) * 2;
      const bf16x8 ka = *(const bf16x8*)(kst + l16 * GG::kKStride + col);
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) {
        if (row0 + qg * 16 < Mb) {
          const bf16x8 qb = *(const bf16x8*)(qst + (qg * 16 + l16) * GG::kKStride + col);
          sacc[qg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb, sacc[qg], 0, 0, 0);
        }
      }
    }
    // ---- mask, online softmax, P in bf16 (lane: keys lg*4 + e of query l16)
    shortx4 pb[NQ];
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) {
      if (row0 + qg * 16 < Mb) {
        const int r = row0 + qg * 16 + l16;
        const int lim = r < Mb ? causal0 + r / G : -1;  // last key this query row sees
        float s[4];
        float mt = kNegInf;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int kl = lg * 4 + e;
          const bool vis = ((vbits >> kl) & 1u) && (kb0 + kl <= lim);
          s[e] = vis ? sacc[qg][e] * scale_log2 : kNegInf;
          mt = fmaxf(mt, s[e]);
        }
        mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
        mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
        const float mn = fmaxf(m_run[qg], mt);
        const bool none = (mn == kNegInf);
        const float alpha = none ? 1.f : exp2f(m_run[qg] - mn);
        float pk[4];
        float ls = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pk[e] = none ? 0.f : exp2f(s[e] - mn);
          ls += pk[e];
        }
        ls += __shfl_xor(ls, 16, 64);
        ls += __shfl_xor(ls, 32, 64);
        l_run[qg] = l_run[qg] * alpha + ls;
        m_run[qg] = mn;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db][qg] *= alpha;
        const uint32_t w0 = pack_bf16x2(pk[0], pk[1]);
        const uint32_t w1 = pack_bf16x2(pk[2], pk[3]);
        pb[qg] = __builtin_bit_cast(shortx4, make_uint2(w0, w1));
      }
    }
    // ---- O^T += V^T P^T (K = 16 keys)
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const unsigned char* vcol = vst + (lg * 4) * GG::kVStride + (db * 16 + l16) * 2;
      const uint32_t v0 = *(const uint16_t*)(vcol);
      const uint32_t v1 = *(const uint16_t*)(vcol + GG::kVStride);
      const uint32_t v2 = *(const uint16_t*)(vcol + 2 * GG::kVStride);
      const uint32_t v3 = *(const uint16_t*)(vcol + 3 * GG::kVStride);
      const shortx4 va = __builtin_bit_cast(shortx4, make_uint2(v0 | (v1 << 16), v2 | (v3 << 16)));
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) {
        if (row0 + qg * 16 < Mb) o[db][qg] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb[qg], o[db][qg], 0, 0, 0);
      }
    }
    wave_lds_sync();  // this tile's LDS reads are issued before the slot is rewritten
  };

  Stage<D> sa, sb;
  fetch(0, sa);
  fetch(1, sb);
  for (int t = 0; t < n_tiles; t += 2) {
    consume(t, sa);
    consume(t + 1, sb);
  }
  __syncthreads();

  // ---- merge the four waves' states: (2,3) -> (0,1), then 1 -> 0
  float* cm = (float*)lds;  // 2 slots of [MQ] m, [MQ] l, [MQ][D] o
  constexpr int kSlot = MQ * (D + 2);
#pragma unroll
  for (int step = 0; step < 2; ++step) {
    const int half = step == 0 ? 2 : 1;
    if (w >= half && w < 2 * half) {
      float* sl = cm + (w - half) * kSlot;
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) {
        const int rl = qg * 16 + l16;
        if (lg == 0) {
          sl[rl] = m_run[qg];
          sl[MQ + rl] = l_run[qg];
        }
#pragma unroll
        for (int db = 0; db < DB; ++db)
          *(floatx4*)(sl + 2 * MQ + rl * D + db * 16 + lg * 4) = o[db][qg];
      }
    }
    __syncthreads();
    if (w < half) {
      const float* sl = cm + w * kSlot;
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) {
        const int rl = qg * 16 + l16;
        const float m2 = sl[rl];
        const float l2 = sl[MQ + rl];
        const float M = fmaxf(m_run[qg], m2);
        const float ca = M == kNegInf ? 0.f : exp2f(m_run[qg] - M);
        const float cb = M == kNegInf ? 0.f : exp2f(m2 - M);
        l_run[qg] = l_run[qg] * ca + l2 * cb;
        m_run[qg] = M;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const floatx4 o2 = *(const floatx4*)(sl + 2 * MQ + rl * D + db * 16 + lg * 4);
          o[db][qg] = o[db][qg] * ca + o2 * cb;
        }
      }
    }
    __syncthreads();
  }

  if (w == 0) {
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) {
      const int r = row0 + qg * 16 + l16;
      if (r >= row_end) continue;
      if (n_splits == 1) {
        const int i = r / G, h = g * G + r % G;
        const float inv = l_run[qg] > 0.f ? 1.f / l_run[qg] : 0.f;
        float* dst = out + ((size_t)(b * (gmax + 1) + i) * Hq + h) * D + lg * 4;
#pragma unroll
        for (int db = 0; db < DB; ++db) *(floatx4*)(dst + db * 16) = o[db][qg] * inv;
      } else {
        const size_t rec = ((size_t)(b * Hkv + g) * n_splits + split) * R + r;
        float* dst = part_o + rec * D + lg * 4;
#pragma unroll
        for (int db = 0; db < DB; ++db) *(floatx4*)(dst + db * 16) = o[db][qg];
        if (lg == 0) {
          part_ml[rec * 2] = m_run[qg];
          part_ml[rec * 2 + 1] = l_run[qg];
        }
      }
    }
  }
}

// Merge the split partials of one (sequence, kv head) for 16 query rows.
template <int D>
__global__ void __launch_bounds__(256)
attn_combine_kernel(const float* __restrict__ part_o, const float* __restrict__ part_ml,
                    const int32_t* __restrict__ kv_len, const int32_t* __restrict__ gamma,
                    float* __restrict__ out, int gmax, int Hq, int Hkv, int L_cap,
                    int split_keys, int n_splits) {
  const int row_blocks = gridDim.x / Hkv;
  const int g = blockIdx.x / row_blocks;
  const int rb = blockIdx.x % row_blocks;
  const int b = blockIdx.y;
  const int G = Hq / Hkv;
  const int R = G * (gmax + 1);
  const int gam = gamma[b];
  const int L = kv_len[b];
  const bool valid = gam >= 0 && gam <= gmax && L >= gam + 1 && L <= L_cap;
  const int Mb = valid ? G * (gam + 1) : 0;
  const int ns = valid ? min(n_splits, (L + split_keys - 1) / split_keys) : 0;
  for (int idx = threadIdx.x; idx < 16 * (D / 4); idx += blockDim.x) {
    const int r = rb * 16 + idx / (D / 4);
    const int d4 = idx % (D / 4);
    if (r >= R) continue;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < Mb) {
      const size_t base = (size_t)(b * Hkv + g) * n_splits;
      float M = kNegInf;
      for (int s = 0; s < ns; ++s) M = fmaxf(M, part_ml[((base + s) * R + r) * 2]);
      if (M != kNegInf) {
        float den = 0.f;
        for (int s = 0; s < ns; ++s) {
          const size_t rec = (base + s) * R + r;
          const float c = exp2f(part_ml[rec * 2] - M);
          den += c * part_ml[rec * 2 + 1];
          const float4 v = *(const float4*)(part_o + rec * D + d4 * 4);
          acc.x += c * v.x;
          acc.y += c * v.y;
          acc.z += c * v.z;
          acc.w += c * v.w;
        }
        const float inv = den > 0.f ? 1.f / den : 0.f;
        acc.x *= inv;
        acc.y *= inv;
        acc.z *= inv;
        acc.w *= inv;
      }
    }
    const int i = r / G, h = g * G + r % G;
    *(float4*)(out + ((size_t)(b * (gmax + 1) + i) * Hq + h) * D + d4 * 4) = acc;
  }
}

typedef void (*SplitKernel)(const uint16_t*, const uint16_t*, const uint16_t*, const uint8_t*,
                            const int32_t*, const int32_t*, float*, float*, float*, int, int, int,
                            int, float, int, int, int32_t*);

template <int D>
SplitKernel pick_split(int nq) {
  switch (nq) {
    case 1: return attn_split_kernel<D, 1>;
    case 2: return attn_split_kernel<D, 2>;
    case 3: return attn_split_kernel<D, 3>;
    case 4: return attn_split_kernel<D, 4>;
    default: return attn_split_kernel<D, 5>;
  }
}

SplitKernel pick_split(int D, int nq) { return D == 64 ? pick_split<64>(nq) : pick_split<128>(nq); }

}  // namespace

int attention_plan(int B, int gamma_max, int Hq, int Hkv, int D, int L_cap, AttentionPlan* plan) {
  const int G = Hq / Hkv;
  const int R = G * (gamma_max + 1);
  plan->nq = R <= 16 * kMaxNQ ? (R + 15) / 16 : kMaxNQ;
  plan->q_chunks = (R + 16 * plan->nq - 1) / (16 * plan->nq);
  const int cus = device_cu_count();
  if (cus <= 0) return SR_ELAUNCH;
  int per_cu = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)pick_split(D, plan->nq),
                                                   kThreads, 0) != hipSuccess || per_cu < 1)
    per_cu = 1;
  const long pairs = (long)B * Hkv * plan->q_chunks;
  const long target = (long)cus * per_cu;
  long splits = (target + pairs - 1) / pairs;
  const long max_splits = (L_cap + kWaveKeys - 1) / kWaveKeys;
  if (splits < 1) splits = 1;
  if (splits > max_splits) splits = max_splits;
  int sk = (int)((L_cap + splits - 1) / splits);
  sk = (sk + kWaveKeys - 1) / kWaveKeys * kWaveKeys;
  plan->split_keys = sk;
  plan->n_splits = (L_cap + sk - 1) / sk;
  plan->workspace_bytes =
      plan->n_splits > 1 ? (size_t)B * Hkv * plan->n_splits * R * (D + 2) * sizeof(float) : 0;
  return SR_OK;
}

int launch_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                            const uint8_t* cache_mask, const int32_t* kv_len,
                            const int32_t* gamma, float* out, int B, int gamma_max, int Hq,
                            int Hkv, int D, int L_cap, float scale, void* workspace,
                            const AttentionPlan& plan, int32_t* status, hipStream_t stream) {
  const int G = Hq / Hkv;
  const int R = G * (gamma_max + 1);
  float* part_o = (float*)workspace;
  float* part_ml = part_o ? part_o + (size_t)B * Hkv * plan.n_splits * R * D : nullptr;
  dim3 grid(plan.n_splits, Hkv * plan.q_chunks, B);
  hipLaunchKernelGGL(pick_split(D, plan.nq), grid, dim3(kThreads), 0, stream,
                     (const uint16_t*)q, (const uint16_t*)k_cache, (const uint16_t*)v_cache,
                     cache_mask, kv_len, gamma, out, part_o, part_ml, gamma_max, Hq, Hkv, L_cap,
                     scale * kLog2e, plan.split_keys, plan.n_splits, status);
  if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  if (plan.n_splits > 1) {
    dim3 cgrid(Hkv * ((R + 15) / 16), B);
    if (D == 64)
      hipLaunchKernelGGL(attn_combine_kernel<64>, cgrid, dim3(256), 0, stream, part_o, part_ml,
                         kv_len, gamma, out, gamma_max, Hq, Hkv, L_cap, plan.split_keys,
                         plan.n_splits);
    else
      hipLaunchKernelGGL(attn_combine_kernel<128>, cgrid, dim3(256), 0, stream, part_o, part_ml,
                         kv_len, gamma, out, gamma_max, Hq, Hkv, L_cap, plan.split_keys,
                         plan.n_splits);
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  }
  return SR_OK;
}

}  // namespace sr
