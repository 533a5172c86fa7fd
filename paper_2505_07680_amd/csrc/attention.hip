// Verification attention for gfx950 (Section 2.2 step 2; Section 4.4, Eq. 8).
//
// Work decomposition. One workgroup handles one (sequence b, kv head g, query
// chunk, key split). All G*(gamma_b+1) query rows that read kv head g (the GQA
// group times the new positions) are processed together, so every K/V byte of
// the split is read from HBM exactly once. Four key streams: stream s owns 16
// of every 64 keys and keeps its own online-softmax state; the four states
// are merged through LDS at the end. Up to 48 query rows, a workgroup is four
// waves, one per stream, with no workgroup barrier inside the key loop. Up
// to 96 rows it is eight waves in two query groups: the two waves of a
// stream each fetch half of every K/V tile into a shared LDS slot (double
// buffered, one workgroup barrier per tile) and each computes its own group's
// rows over the whole tile, so the tile is still read once. When the
// cache is split, each split publishes its (max, sum, unnormalised output)
// partial and bumps a per-(b, g, query chunk) arrival counter; the last
// workgroup to arrive merges all partials in split order and writes the
// output, then resets the counter, so the workspace is left ready for the
// next call. The summation order is fixed, so results are reproducible.
// When the workgroups outnumber what the device holds at once, a small
// kernel first sorts the jobs by key count and the workgroups take them
// longest first, so that the device does not idle behind a few long
// workgroups at the end of a ragged batch.
//
// Per 16-key tile of a stream:
//   * K and V rows are fetched with coalesced 16-byte loads into a register
//     ring (two tiles deep, or four half tiles with two query groups), so
//     loads stay in flight while a tile is computed, and staged in the
//     stream's LDS slot; rows at or past kv_len are fetched
//     out of the buffer range (they read as zero, with no memory traffic) and
//     V rows under mask 0 are zeroed while staging, so whatever those rows
//     hold never reaches the output;
//   * S^T = K Q^T on MFMA (v_mfma_f32_16x16x32_bf16: 16 keys x 16 queries per
//     block, K=32 over the head dimension); each lane then holds 4 scores of
//     ONE query, so the softmax max/sum need only two cross-lane steps;
//   * the softmax reference maximum of a row is raised only when a tile exceeds
//     it by more than 2^8, so the output accumulators are rarely rescaled;
//   * P is rounded to bf16 in place: its accumulator layout is exactly the B
//     operand of O^T += V^T P^T (v_mfma_f32_16x16x16_bf16, K=16 over the keys);
//     the V^T operand is gathered from LDS with 16-bit reads.
// Scores are kept in log2 units (scale * log2(e) folded in) and exponentiated
// with exp2.

#include "sr_internal.h"

namespace sr {
namespace {

typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = 4;  // key streams
constexpr int kWaveKeys = 16;
// At most three 16-row query blocks per wave (the accumulators stay in 256
// registers at two waves per SIMD) and two query groups per workgroup: more
// than 96 rows go to further query chunks, which read the same K/V again.
constexpr int kMaxNQ = 3;
constexpr int kMaxQG = 2;
constexpr float kLazy = 8.f;  // log2 headroom of the lazily rescaled softmax reference
// Arrival counters sit one per 128-byte line: the splits of different
// (sequence, kv head, query chunk) jobs then never contend for one line.
constexpr int kCounterStride = 32;
constexpr int kMaxSplitKeys = 8448;  // keys per split at most (about 4 MB of K/V at D = 128)
// Byte offset past the end of any K/V slab (slabs are below 2^31 bytes): a
// buffer load there returns zero without touching memory.
constexpr uint32_t kOutOfRange = 0x7ffffff0u;
// Cache-policy operand of the K/V loads when one workgroup is the only
// reader of its K/V tiles (a single query chunk): non-temporal. With several
// query chunks the others re-read the same tiles, which then should stay in
// the caches (plain loads).
constexpr int kStreamLoad = 2;

template <int D>
struct Geo {
  static constexpr int kKStride = D * 2 + 16;  // LDS bytes per staged K (and Q) row
  // LDS bytes per staged V row: four consecutive rows' 32-byte column blocks
  // fall on different banks for the transposing reads of the V^T operand
  static constexpr int kVStride = D * 2 + 32;
  static constexpr int kChunksPerRow = D / 8;  // 16-byte chunks per row
  static constexpr int kRowsPerLoad = 64 / kChunksPerRow;
  static constexpr int kLoads = kWaveKeys / kRowsPerLoad;  // 16-byte loads per lane per tensor per tile
  static constexpr int kSlotK = kWaveKeys * kKStride;
  static constexpr int kWaveBytes = kSlotK + kWaveKeys * kVStride;
};

// Threads, ring depth and LDS buffers per slot of a workgroup with QG query
// groups: with two groups each wave fetches half of a tile, so a four-deep
// ring of half tiles holds the registers of a two-deep ring of whole ones.
template <int QG>
struct Shape {
  static constexpr int kThreads = 64 * kWaves * QG;
  static constexpr int kRing = QG == 1 ? 2 : 4;
  static constexpr int kBufs = QG == 1 ? 1 : 2;
};

template <int D, int NQ, int QG>
struct Lds {
  static constexpr int MQ = 16 * NQ;
  static constexpr int kStage = kWaves * Shape<QG>::kBufs * Geo<D>::kWaveBytes + QG * MQ * Geo<D>::kKStride;
  // Merge of the four stream states of each query group: the columns are
  // reduced in kPasses passes so that a group's four fp32 slices fit in 72 KB
  // (two four-wave workgroups per CU, or one of eight, fit in its 160 KB).
  static constexpr int kPasses = (kWaves * MQ * D * 4 <= 73728) ? 1 : (kWaves * MQ * D * 2 <= 73728) ? 2 : 4;
  static constexpr int kDp = D / kPasses;                 // columns per pass
  static constexpr int kRowStride = kDp + 4;              // floats; padded against bank conflicts
  static constexpr int kSlot = MQ * kRowStride;           // floats per wave slice
  static constexpr int kMl = QG * kWaves * kSlot * 4;     // byte offset of the (m, l) exchange
  static constexpr int kComb = kMl + QG * (kWaves + 1) * 2 * MQ * 4;
  static constexpr int kBytes = kStage > kComb ? kStage : kComb;
};

// 16-byte device-coherent (sc1) buffer access to the split partials; the
// descriptor's range check turns an out-of-range offset into a dropped store
// or a zero load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t partial_rsrc(const float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), 0, (int)bytes, 0x00020000);
}
constexpr int kDeviceCoherent = 16;  // cache-policy operand: sc1

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

template <int D, int QG>
struct Stage {  // one wave's part of a 16-key tile in flight
  u32x4 k[Geo<D>::kLoads / QG], v[Geo<D>::kLoads / QG];
  uint32_t mbyte;  // validity byte of key (lane mod 16), evaluated when consumed
};

// Waves per SIMD the register allocation must allow: three for one row block
// (168 registers), else two (256).
template <int D, int NQ, int QG, bool NT>
__global__ void __launch_bounds__(Shape<QG>::kThreads, NQ == 1 && QG == 1 ? 3 : 2)
attn_split_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
                  const uint16_t* __restrict__ vc, const uint8_t* __restrict__ mask,
                  const int32_t* __restrict__ kv_len, const int32_t* __restrict__ gamma,
                  float* __restrict__ out, float* __restrict__ part_o,
                  float* __restrict__ part_ml, uint32_t* __restrict__ counters,
                  const int32_t* __restrict__ order, int B, int gmax, int Hq, int Hkv, int L_cap,
                  float scale_log2, int split_keys, int n_splits, int q_chunks,
                  int32_t* __restrict__ status) {
  using GG = Geo<D>;
  constexpr int MQ = 16 * NQ;
  constexpr int DB = D / 16;
  constexpr int kT = Shape<QG>::kThreads;
  constexpr int kRing = Shape<QG>::kRing;
  constexpr int kBufs = Shape<QG>::kBufs;
  constexpr int kLd = GG::kLoads / QG;  // 16-byte loads per lane per tensor per tile
  __shared__ __attribute__((aligned(16))) unsigned char lds[Lds<D, NQ, QG>::kBytes];

  // Workgroup order: with an order table (more workgroups than fit on the
  // device at once), the table's: jobs by decreasing key count, so that the
  // last workgroups to start are the shortest. Otherwise (sequence, kv head)
  // pair fastest, then key split in descending order, then query chunk.
  // Workgroups are dealt to the XCDs round-robin, so each XCD gets every
  // split of an even share of the pairs (and the query chunks of one pair and
  // split share an XCD and its L2).
  const int P = B * Hkv;
  const int rest = (int)(blockIdx.x / (unsigned)P);
  const int code = order ? __builtin_amdgcn_readfirstlane(order[blockIdx.x])
                         : ((int)(blockIdx.x % (unsigned)P) * q_chunks + rest / n_splits) * n_splits +
                               (n_splits - 1 - rest % n_splits);
  const int split = code % n_splits;
  const int job = code / n_splits;
  const int qc = job % q_chunks;
  const int pair_id = job / q_chunks;
  const int g = pair_id % Hkv;
  const int b = pair_id / Hkv;
  const int G = Hq / Hkv;
  const int R = G * (gmax + 1);
  const int gam = gamma[b];
  const int L = kv_len[b];
  const bool valid = gam >= 0 && gam <= gmax && L >= gam + 1 && L <= L_cap;
  if (!valid && split == 0 && qc == 0 && g == 0 && threadIdx.x == 0 && status) {
    atomicOr(status, (gam < 0 || gam > gmax) ? SR_ST_GAMMA : SR_ST_KVLEN);
  }
  const int row0 = qc * QG * MQ;
  const int row_end = min(R, row0 + QG * MQ);
  const int Mb = valid ? G * (gam + 1) : 0;
  const int ns = valid ? (L + split_keys - 1) / split_keys : 0;  // splits that hold keys
  const bool work = row0 < Mb && split < ns;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = wave_id();
  const int ws = w % kWaves;  // key stream
  const int h = w / kWaves;   // query group: rows rbase .. rbase + MQ - 1
  const int rbase = row0 + h * MQ;
  const int l16 = lane & 15;
  const int lg = lane >> 4;

  if (!work) {
    // Nothing to compute. Split 0 of a query chunk without live rows (or of an
    // invalid sequence) owns those output rows and writes them as zero.
    if (split == 0) {
      for (int idx = tid; idx < (row_end - row0) * (D / 4); idx += kT) {
        const int r = row0 + idx / (D / 4);
        const int d4 = idx % (D / 4);
        const int i = r / G, hh = g * G + r % G;
        *(float4*)(out + ((size_t)(b * (gmax + 1) + i) * Hq + hh) * D + d4 * 4) = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
    return;
  }

  unsigned char* qst = lds + kWaves * kBufs * GG::kWaveBytes;
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

  // Tile j holds keys [16 j, 16 j + 16). Split s owns the keys
  // [s split_keys, (s + 1) split_keys), dealt round-robin to the four
  // streams, so a stream's tiles are first, first + 4, first + 8, ... below
  // j_end.
  const int first0 = split * (split_keys / kWaveKeys);
  const int first = first0 + ws;
  const int j_end = min((L + kWaveKeys - 1) / kWaveKeys, (split + 1) * (split_keys / kWaveKeys));
  const int row_lim = min(L, j_end * kWaveKeys);  // a refill past the stream's last tile reads nothing

  // Every fetch issues the same loads (rows at or past kv_len, and tiles past
  // the stream's last, read out of range, as zero, with no traffic), so each
  // wait covers exactly the loads it needs, in the first iteration as in
  // every later one.
  const uint8_t* mload = mrow ? mrow : (const uint8_t*)kslab;
  // K/V slabs of (b, g) as buffer resources: 32-bit row offsets
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kslab, (size_t)L_cap * D * 2);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vslab, (size_t)L_cap * D * 2);
  const int lane_row = lane / GG::kChunksPerRow;
  const int lane_chunk = lane % GG::kChunksPerRow;
  const uint32_t lane_col = (uint32_t)lane_chunk * 16;
  // this wave's rows of a tile: load u covers rows (h kLd + u) kRowsPerLoad + lane_row
  auto fetch = [&](int j, Stage<D, QG>& st) __attribute__((always_inline)) {
    const int kb0 = j * kWaveKeys;
#pragma unroll
    for (int u = 0; u < kLd; ++u) {
      const int row = kb0 + (h * kLd + u) * GG::kRowsPerLoad + lane_row;
      const uint32_t off = row < row_lim ? (uint32_t)row * (D * 2) + lane_col : kOutOfRange;
      st.k[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, NT ? kStreamLoad : 0));
      st.v[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rv, off, 0, NT ? kStreamLoad : 0));
    }
    st.mbyte = mload[min(kb0 + (lane & (kWaveKeys - 1)), L - 1)];
  };
  // Ring entry st holds tile j: stage it in LDS buffer buf of the stream's
  // slot, refill it with the stream's tile kRing further on, compute tile j,
  // and leave the refilled tile's number in j.
  auto step = [&](int& j, Stage<D, QG>& st, int buf) __attribute__((always_inline)) {
    unsigned char* kst = lds + (ws * kBufs + buf) * GG::kWaveBytes;
    unsigned char* vst = kst + GG::kSlotK;
    const int kb0 = j * kWaveKeys;
    const bool key_ok = lane < kWaveKeys && kb0 + lane < L && (mrow == nullptr || st.mbyte != 0u);
    const uint32_t vbits = (uint32_t)__ballot(key_ok) & 0xffffu;
    const bool all_rows = vbits == 0xffffu;  // wave-uniform
#pragma unroll
    for (int u = 0; u < kLd; ++u) {
      const int rl = (h * kLd + u) * GG::kRowsPerLoad + lane_row;
      *(u32x4*)(kst + rl * GG::kKStride + lane_chunk * 16) = st.k[u];
      const u32x4 vv = (all_rows || ((vbits >> rl) & 1u)) ? st.v[u] : u32x4{0u, 0u, 0u, 0u};
      uint32_t* dst = (uint32_t*)(vst + rl * GG::kVStride + lane_chunk * 16);
      *(uint2*)dst = make_uint2(vv.x, vv.y);
      *(uint2*)(dst + 2) = make_uint2(vv.z, vv.w);
    }
    if constexpr (QG == 1)
      wave_lds_sync();
    else
      __syncthreads();  // both halves of the tile are in the slot
    const int nx = j + kRing * kWaves;
    __builtin_amdgcn_sched_barrier(0);
    fetch(nx, st);  // the ring's other tiles and this refill stay in flight during the compute below
    __builtin_amdgcn_sched_barrier(0);
    const int jc = j;
    j = nx;
    if (jc >= j_end || rbase >= Mb) return;  // wave-uniform: past the stream's last tile, or no live rows
    const bool full = vbits == 0xffffu && kb0 + kWaveKeys - 1 <= causal0;  // wave-uniform
    // ---- S^T = K Q^T (16 keys x 16 queries per block)
    floatx4 sacc[NQ];
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) sacc[qg] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) {
      const int col = (ks * 32 + lg * 8) * 2;
      const bf16x8 ka = *(const bf16x8*)(kst + l16 * GG::kKStride + col);
      bf16x8 qb[NQ];
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) qb[qg] = *(const bf16x8*)(qst + (h * MQ + qg * 16 + l16) * GG::kKStride + col);
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) sacc[qg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qb[qg], sacc[qg], 0, 0, 0);
    }
    // ---- mask, online softmax, P in bf16 (lane: keys lg*4 + e of query l16)
    // Row blocks without live rows go through both products too (on zero
    // query rows and zero P): a branch around each MFMA costs more than the
    // MFMA. Only the softmax is skipped for them.
    shortx4 pb[NQ];
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) pb[qg] = shortx4{0, 0, 0, 0};
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) {
      if (rbase + qg * 16 < Mb) {
        const int r = rbase + qg * 16 + l16;
        float s[4];
        float mt = kNegInf;
        if (full) {
          // every row of the wave sees all 16 keys (rows past Mb are dropped
          // at the end); the scale is positive, so the maximum is taken on the
          // raw products and each probability below is one fma and one exp2
          mt = fmaxf(fmaxf(sacc[qg][0], sacc[qg][1]), fmaxf(sacc[qg][2], sacc[qg][3])) * scale_log2;
#pragma unroll
          for (int e = 0; e < 4; ++e) s[e] = sacc[qg][e];
        } else {
          const int lim = r < Mb ? causal0 + r / G : -1;  // last key this query row sees
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int kl = lg * 4 + e;
            const bool vis = ((vbits >> kl) & 1u) && (kb0 + kl <= lim);
            s[e] = vis ? sacc[qg][e] * scale_log2 : kNegInf;
            mt = fmaxf(mt, s[e]);
          }
        }
        mt = max_across_rows(mt);
        // Lazy rescaling: a row keeps its reference maximum until a tile
        // exceeds it by more than kLazy (log2 units), so P stays below
        // 2^kLazy and the output accumulators are rescaled only then
        // (skipped by the whole wave when no row needs it).
        // (straight-line: every exponential is computed and selected, no
        // per-entry branches)
        const bool grow = mt > m_run[qg] + kLazy;
        const float mref = grow ? mt : m_run[qg];
        // exp2(-inf) = 0 covers a first reference (the old one -inf); equal
        // references, -inf ones included, give 1
        const float alpha = m_run[qg] == mref ? 1.f : exp2_hw(m_run[qg] - mref);
        const float mr = mref == kNegInf ? 0.f : mref;  // (-inf: every score of the row so far is -inf)
        float pk[4];
        float ls = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pk[e] = exp2_hw(full ? fmaf(s[e], scale_log2, -mr) : s[e] - mr);
          ls += pk[e];
        }
        ls = sum_across_rows(ls);
        l_run[qg] = l_run[qg] * alpha + ls;
        m_run[qg] = mref;
        if (__ballot(grow) != 0ull) {
#pragma unroll
          for (int db = 0; db < DB; ++db) o[db][qg] *= alpha;
        }
        const uint32_t w0 = pack_bf16x2(pk[0], pk[1]);
        const uint32_t w1 = pack_bf16x2(pk[2], pk[3]);
        pb[qg] = __builtin_bit_cast(shortx4, make_uint2(w0, w1));
      }
    }
    // ---- O^T += V^T P^T (K = 16 keys)
    // The V^T operand (lane: column l16 of the block, keys lg*4 .. lg*4+3) by
    // the LDS transposing read: in each 16-lane group, lane j names the four
    // columns 4 (j mod 4) .. +3 of key row lg*4 + j/4, and lane i receives
    // column i of the group's four key rows.
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const unsigned char* vrow = vst + (lg * 4 + (l16 >> 2)) * GG::kVStride + (db * 16 + (l16 & 3) * 4) * 2;
      const shortx4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) shortx4*)vrow);
#pragma unroll
      for (int qg = 0; qg < NQ; ++qg) {
        o[db][qg] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, pb[qg], o[db][qg], 0, 0, 0);
      }
    }
    // One query group: this tile's LDS reads are issued before the slot is
    // rewritten. Two: the slot's other buffer takes the next tile, and the
    // barrier of the step after it orders every read of this one first.
    if constexpr (QG == 1) wave_lds_sync();
  };

  // Issue order: this workgroup's query rows, then the ring; the query rows
  // are staged in LDS while the K/V tiles are still in flight. Each group is
  // kept together (no interleaving by the scheduler), so every wait covers
  // exactly what it needs: a step waits for its own tile only.
  constexpr int kQChunks = QG * MQ * GG::kChunksPerRow;
  constexpr int kQLoads = (kQChunks + kT - 1) / kT;
  u32x4 qv[kQLoads];
#pragma unroll
  for (int u = 0; u < kQLoads; ++u) {
    const int idx = min(tid + u * kT, kQChunks - 1);
    const int r = min(row0 + idx / GG::kChunksPerRow, Mb - 1);  // rows past Mb are zeroed below
    const int i = r / G, hh = g * G + r % G;
    qv[u] = *(const u32x4*)(q + ((size_t)(b * (gmax + 1) + i) * Hq + hh) * D + (idx % GG::kChunksPerRow) * 8);
  }
  __builtin_amdgcn_sched_barrier(0);
  Stage<D, QG> ring[kRing];
  int jr[kRing];
#pragma unroll
  for (int r = 0; r < kRing; ++r) {
    jr[r] = first + r * kWaves;
    fetch(jr[r], ring[r]);
    __builtin_amdgcn_sched_barrier(0);
  }
  // (unconditional: a thread past the last chunk rewrites that chunk with
  // the same value, and no load is moved into a branch after the K/V loads)
#pragma unroll
  for (int u = 0; u < kQLoads; ++u) {
    const int idx = min(tid + u * kT, kQChunks - 1);
    const int rl = idx / GG::kChunksPerRow;
    const u32x4 val = row0 + rl < Mb ? qv[u] : u32x4{0u, 0u, 0u, 0u};
    *(u32x4*)(qst + rl * GG::kKStride + (idx % GG::kChunksPerRow) * 16) = val;
  }
  __syncthreads();

  // The ring holds the stream's next kRing tiles (ascending). With two query
  // groups every wave runs the same number of rounds (counted on stream 0,
  // whose tiles come first), so the barriers inside the steps pair up; a step
  // past a stream's last tile still stages (zeros) and meets the barrier.
  if constexpr (QG == 1) {
    while (jr[0] < j_end) {
#pragma unroll
      for (int r = 0; r < kRing; ++r) step(jr[r], ring[r], 0);
    }
  } else {
    const int rounds = (j_end - first0 + kRing * kWaves - 1) / (kRing * kWaves);
    for (int it = 0; it < rounds; ++it) {
#pragma unroll
      for (int r = 0; r < kRing; ++r) step(jr[r], ring[r], r % kBufs);
    }
  }
  __syncthreads();

  // ---- merge the four stream states of each query group (every wave and lane takes part)
  using LL = Lds<D, NQ, QG>;
  const int tg = tid - h * 64 * kWaves;                               // thread index in the group
  float* slots = (float*)lds + h * kWaves * LL::kSlot;                  // [kWaves][MQ][kRowStride]
  float* mlx = (float*)(lds + LL::kMl) + h * (kWaves + 1) * 2 * MQ;     // [kWaves][2][MQ]: each stream's (m, l)
  float* mlf = mlx + kWaves * 2 * MQ;                                   // [2][MQ]: merged (M, L)
  if (lg == 0) {
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) {
      mlx[(ws * 2) * MQ + qg * 16 + l16] = m_run[qg];
      mlx[(ws * 2 + 1) * MQ + qg * 16 + l16] = l_run[qg];
    }
  }
  __syncthreads();
  float cw[NQ];  // this stream's weight exp2(m_w - M) per row block
#pragma unroll
  for (int qg = 0; qg < NQ; ++qg) {
    const int rl = qg * 16 + l16;
    float M = kNegInf;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) M = fmaxf(M, mlx[(v * 2) * MQ + rl]);
    float Lsum = 0.f;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
      const float c = M == kNegInf ? 0.f : exp2f(mlx[(v * 2) * MQ + rl] - M);
      Lsum += c * mlx[(v * 2 + 1) * MQ + rl];
    }
    cw[qg] = M == kNegInf ? 0.f : exp2f(m_run[qg] - M);
    if (ws == 0 && lg == 0) {
      mlf[rl] = M;
      mlf[MQ + rl] = Lsum;
    }
  }

  // With a single split holding keys the result is final here, otherwise it
  // is published as the split's partial.
  const size_t pair = (size_t)(b * Hkv + g);
  const int n_rec = (int)((size_t)n_splits * P) * R;  // records in the partial arrays
  const __amdgpu_buffer_rsrc_t rs_o = partial_rsrc(part_o, (uint32_t)((size_t)n_rec * D * 4));
  const __amdgpu_buffer_rsrc_t rs_ml = partial_rsrc(part_ml, (uint32_t)((size_t)n_rec * 8));
  constexpr int kItemsP = (MQ * (LL::kDp / 4) + 64 * kWaves - 1) / (64 * kWaves);
#pragma unroll
  for (int pass = 0; pass < LL::kPasses; ++pass) {
    __syncthreads();  // (m, l) exchange read / previous pass's slices consumed
#pragma unroll
    for (int qg = 0; qg < NQ; ++qg) {
      const int rl = qg * 16 + l16;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int col = db * 16 + lg * 4 - pass * LL::kDp;
        if (col >= 0 && col < LL::kDp) *(floatx4*)(slots + (ws * MQ + rl) * LL::kRowStride + col) = o[db][qg] * cw[qg];
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kItemsP; ++k) {
      const int idx = tg + k * 64 * kWaves;
      if (idx >= MQ * (LL::kDp / 4)) continue;
      const int rl = idx / (LL::kDp / 4);
      const int c4 = idx % (LL::kDp / 4);
      const int r = rbase + rl;
      if (r >= row_end) continue;
      floatx4 sum = *(const floatx4*)(slots + rl * LL::kRowStride + c4 * 4);
#pragma unroll
      for (int v = 1; v < kWaves; ++v) sum += *(const floatx4*)(slots + (v * MQ + rl) * LL::kRowStride + c4 * 4);
      const int col = pass * LL::kDp + c4 * 4;
      if (ns == 1) {
        const float Lr = mlf[MQ + rl];
        const int i = r / G, hh = g * G + r % G;
        *(floatx4*)(out + ((size_t)(b * (gmax + 1) + i) * Hq + hh) * D + col) =
            (r < Mb && Lr > 0.f) ? sum * (1.f / Lr) : floatx4{0.f, 0.f, 0.f, 0.f};
      } else if (r < Mb) {
        const uint32_t rec = (uint32_t)((pair * n_splits + split) * R + r);
        __builtin_amdgcn_raw_buffer_store_b128(sum, rs_o, (rec * D + col) * 4, 0, kDeviceCoherent);
        if (pass == 0 && c4 == 0)
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, floatx2{mlf[rl], mlf[MQ + rl]}), rs_ml, rec * 8, 0, kDeviceCoherent);
      }
    }
  }
  if (ns == 1) return;

  // ---- arrive: the last split of this job to finish merges all partials
  stores_done();
  __syncthreads();
  __shared__ uint32_t last_flag;
  if (tid == 0) {
    uint32_t* cnt = counters + (size_t)job * kCounterStride;
    const uint32_t before = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = before == (uint32_t)(ns - 1);
    if (last) st_dev(cnt, 0u);  // every split of this job has arrived: reset for the next call
    last_flag = last ? 1u : 0u;
  }
  __syncthreads();
  if (last_flag == 0u) return;
  __atomic_signal_fence(__ATOMIC_SEQ_CST);

  // Each thread owns kItems (row, 4 columns) items and folds the splits in
  // with a running max, kGroup splits per round of loads.
  constexpr int kItems = (QG * MQ * (D / 4) + kT - 1) / kT;
  constexpr int kGroup = kItems >= 16 ? 1 : (16 / kItems > 8 ? 8 : 16 / kItems);
  const int n_items = (row_end - row0) * (D / 4);
  float mx[kItems], den[kItems];
  floatx4 acc[kItems];
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    mx[k] = kNegInf;
    den[k] = 0.f;
    acc[k] = floatx4{0.f, 0.f, 0.f, 0.f};
  }
  for (int sp0 = 0; sp0 < ns; sp0 += kGroup) {
    floatx2 ml2[kGroup][kItems];
    floatx4 o2[kGroup][kItems];
#pragma unroll
    for (int j = 0; j < kGroup; ++j)
#pragma unroll
      for (int k = 0; k < kItems; ++k) {
        const int sp = min(sp0 + j, ns - 1);  // repeats of the last split are discarded below
        const int idx = min(tid + k * kT, n_items - 1);
        const int r = min(row0 + idx / (D / 4), Mb - 1);  // rows past Mb hold no partial; their result is discarded
        const uint32_t rec = (uint32_t)((pair * n_splits + sp) * R + r);
        ml2[j][k] = __builtin_bit_cast(floatx2, __builtin_amdgcn_raw_buffer_load_b64(rs_ml, rec * 8, 0, kDeviceCoherent));
        o2[j][k] = __builtin_amdgcn_raw_buffer_load_b128(rs_o, (rec * D + (idx % (D / 4)) * 4) * 4, 0, kDeviceCoherent);
      }
#pragma unroll
    for (int j = 0; j < kGroup; ++j) {
      if (sp0 + j >= ns) break;
#pragma unroll
      for (int k = 0; k < kItems; ++k) {
        const float M = fmaxf(mx[k], ml2[j][k].x);
        if (M == kNegInf) continue;
        const float ca = exp2f(mx[k] - M);
        const float cb = exp2f(ml2[j][k].x - M);
        den[k] = den[k] * ca + ml2[j][k].y * cb;
        acc[k] = acc[k] * ca + o2[j][k] * cb;
        mx[k] = M;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kItems; ++k) {
    const int idx = tid + k * kT;
    if (idx >= n_items) continue;
    const int r = row0 + idx / (D / 4);
    const bool live = r < Mb && den[k] > 0.f;
    const floatx4 res = live ? acc[k] * (1.f / den[k]) : floatx4{0.f, 0.f, 0.f, 0.f};
    const int i = r / G, hh = g * G + r % G;
    *(floatx4*)(out + ((size_t)(b * (gmax + 1) + i) * Hq + hh) * D + (idx % (D / 4)) * 4) = res;
  }
}

typedef void (*SplitKernel)(const uint16_t*, const uint16_t*, const uint16_t*, const uint8_t*,
                            const int32_t*, const int32_t*, float*, float*, float*, uint32_t*,
                            const int32_t*, int, int, int, int, int, float, int, int, int, int32_t*);

// The dispatch order of the split workgroups when there are more than fit on
// the device at once (one workgroup of kOrderThreads): every job (sequence,
// kv head, query chunk, split) by decreasing key count (in 16-key tiles, a
// counting sort), empty jobs last, so that the workgroups that start last
// are the shortest and the device does not idle behind a few long ones.
// Jobs of equal count take any order among themselves (the results do not
// depend on the order). Entry: ((b Hkv + g) q_chunks + qc) n_splits + split;
// the jobs of one (sequence, split) are consecutive, kv head fastest.
constexpr int kOrderThreads = 1024;
constexpr int kOrderBuckets = 1024;  // 0: empty; t: t tiles (the last bucket also takes longer jobs)
constexpr int kOrderKept = 4;        // buckets a thread keeps between the two passes
static_assert(kOrderThreads == kOrderBuckets, "one scan element per thread");
__global__ void __launch_bounds__(kOrderThreads)
attn_order_kernel(const int32_t* __restrict__ kv_len, const int32_t* __restrict__ gamma, int B, int gmax,
                  int Hkv, int q_chunks, int L_cap, int split_keys, int n_splits, int32_t* __restrict__ order) {
  __shared__ int cnt[kOrderBuckets];
  __shared__ int wsum[kOrderThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per_item = Hkv * q_chunks;  // jobs of one (sequence, split)
  const int n_items = B * n_splits;
  auto bucket = [&](int item) __attribute__((always_inline)) {
    const int b = item / n_splits, sp = item % n_splits;
    const int gam = gamma[b], L = kv_len[b];
    const bool valid = gam >= 0 && gam <= gmax && L >= gam + 1 && L <= L_cap;
    const int len = valid ? min(L, (sp + 1) * split_keys) - sp * split_keys : 0;
    return len <= 0 ? 0 : min((len + kWaveKeys - 1) / kWaveKeys, kOrderBuckets - 1);
  };
  cnt[tid] = 0;
  __syncthreads();
  // the first kOrderKept items of a thread keep their bucket for the second pass
  int kept[kOrderKept];
#pragma unroll
  for (int u = 0; u < kOrderKept; ++u) {
    const int item = tid + u * kOrderThreads;
    kept[u] = item < n_items ? bucket(item) : 0;
    if (item < n_items) atomicAdd(&cnt[kept[u]], per_item);
  }
  for (int item = tid + kOrderKept * kOrderThreads; item < n_items; item += kOrderThreads)
    atomicAdd(&cnt[bucket(item)], per_item);
  __syncthreads();
  // start of bucket t: the jobs of every longer bucket (thread t holds
  // bucket kOrderBuckets - 1 - t, an inclusive scan in thread order)
  const int t_b = kOrderBuckets - 1 - tid;
  const int c = cnt[t_b];
  int incl = c;
  for (int d = 1; d < 64; d <<= 1) {
    const int o = __shfl_up(incl, d, 64);
    if (lane >= d) incl += o;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  for (int i = 0; i < w; ++i) incl += wsum[i];
  cnt[t_b] = incl - c;  // now each bucket's next free position (each thread rewrites only its own)
  __syncthreads();
  auto place = [&](int item, int bk) __attribute__((always_inline)) {
    const int pos = atomicAdd(&cnt[bk], per_item);
    const int b = item / n_splits, sp = item % n_splits;
    for (int j = 0; j < per_item; ++j) {
      // kv head fastest: with a multiple of 8 heads the query chunks of one
      // (pair, split) fall on one XCD and share its L2
      const int qc = j / Hkv, g = j % Hkv;
      order[pos + j] = ((b * Hkv + g) * q_chunks + qc) * n_splits + sp;
    }
  };
#pragma unroll
  for (int u = 0; u < kOrderKept; ++u) {
    const int item = tid + u * kOrderThreads;
    if (item < n_items) place(item, kept[u]);
  }
  for (int item = tid + kOrderKept * kOrderThreads; item < n_items; item += kOrderThreads) place(item, bucket(item));
}

template <int D>
SplitKernel pick_split(int nq, int qg, int q_chunks) {
  if (qg == 1) {
    switch (nq) {
      case 1: return attn_split_kernel<D, 1, 1, true>;
      case 2: return attn_split_kernel<D, 2, 1, true>;
      default: return attn_split_kernel<D, 3, 1, true>;
    }
  }
  if (nq == 2) return attn_split_kernel<D, 2, 2, true>;
  return q_chunks == 1 ? attn_split_kernel<D, 3, 2, true> : attn_split_kernel<D, 3, 2, false>;
}

SplitKernel pick_split(int D, int nq, int qg, int q_chunks) {
  return D == 64 ? pick_split<64>(nq, qg, q_chunks) : pick_split<128>(nq, qg, q_chunks);
}

}  // namespace

int attention_plan(int B, int gamma_max, int Hq, int Hkv, int D, int L_cap, AttentionPlan* plan) {
  const int G = Hq / Hkv;
  const int R = G * (gamma_max + 1);
  // Up to 48 rows: one four-wave group of ceil(R / 16) row blocks. Beyond:
  // two groups of two (up to 64 rows) or three blocks, in as many query
  // chunks of 96 rows as needed.
  if (R <= 16 * kMaxNQ) {
    plan->qg = 1;
    plan->nq = (R + 15) / 16;
  } else {
    plan->qg = kMaxQG;
    plan->nq = R <= 2 * 32 ? 2 : kMaxNQ;
  }
  const int rows_per_chunk = 16 * plan->nq * plan->qg;
  plan->q_chunks = (R + rows_per_chunk - 1) / rows_per_chunk;
  const int cus = device_cu_count();
  if (cus <= 0) return SR_ELAUNCH;
  int per_cu = 1;
  const int threads = plan->qg == 1 ? Shape<1>::kThreads : Shape<kMaxQG>::kThreads;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
          &per_cu, (const void*)pick_split(D, plan->nq, plan->qg, plan->q_chunks), threads, 0) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  const long pairs = (long)B * Hkv * plan->q_chunks;
  const long target = (long)cus * per_cu;
  // Splits enough for one workgroup per CU: a four-wave workgroup keeps
  // enough K/V loads in flight to stream at the device's rate, and fewer
  // splits mean fewer partials to merge (at 16 sequences of 2054 keys, two
  // splits per (sequence, kv head) measured 30.5 us against 32.7 with four).
  long splits = ((long)cus + pairs - 1) / pairs;
  // Bound a workgroup's keys, so the last workgroups of a ragged batch do not
  // run long after the rest have finished.
  const long by_length = (L_cap + kMaxSplitKeys - 1) / kMaxSplitKeys;
  if (splits < by_length) splits = by_length;
  const long max_splits = (L_cap + kWaveKeys - 1) / kWaveKeys;
  if (splits < 1) splits = 1;
  if (splits > max_splits) splits = max_splits;
  // Offsets into the partial arrays are 32-bit (buffer addressing): keep
  // them below 2^31 bytes.
  const long rec_per_split = (long)B * Hkv * R;
  const long max_by_offset = (long)(0x7fffffffL / ((long)D * 4 * (rec_per_split > 0 ? rec_per_split : 1)));
  if (splits > max_by_offset) splits = max_by_offset > 1 ? max_by_offset : 1;
  int sk = (int)((L_cap + splits - 1) / splits);
  sk = (sk + kWaveKeys - 1) / kWaveKeys * kWaveKeys;
  plan->split_keys = sk;
  plan->n_splits = (L_cap + sk - 1) / sk;
  // [arrival counters: B*Hkv*q_chunks, one per 128-byte line][partial o][partial (m, l)][order]
  const size_t counters = (size_t)B * Hkv * plan->q_chunks * kCounterStride * sizeof(uint32_t);
  plan->part_offset = counters;
  size_t bytes = plan->n_splits > 1 ? counters + (size_t)B * Hkv * plan->n_splits * R * (D + 2) * sizeof(float) : 0;
  const long n_jobs = (long)plan->n_splits * pairs;
  plan->ordered = n_jobs > target ? 1 : 0;
  plan->order_offset = (bytes + 15) / 16 * 16;
  if (plan->ordered) bytes = plan->order_offset + (size_t)n_jobs * sizeof(int32_t);
  plan->workspace_bytes = bytes;
  return SR_OK;
}

int launch_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                            const uint8_t* cache_mask, const int32_t* kv_len,
                            const int32_t* gamma, float* out, int B, int gamma_max, int Hq,
                            int Hkv, int D, int L_cap, float scale, void* workspace,
                            const AttentionPlan& plan, int32_t* status, hipStream_t stream) {
  const int G = Hq / Hkv;
  const int R = G * (gamma_max + 1);
  uint32_t* counters = (uint32_t*)workspace;
  float* part_o = workspace ? (float*)((char*)workspace + plan.part_offset) : nullptr;
  float* part_ml = part_o ? part_o + (size_t)B * Hkv * plan.n_splits * R * D : nullptr;
  dim3 grid((unsigned)((long)plan.n_splits * plan.q_chunks * B * Hkv));
  const int threads = plan.qg == 1 ? Shape<1>::kThreads : Shape<kMaxQG>::kThreads;
  int32_t* order = plan.ordered ? (int32_t*)((char*)workspace + plan.order_offset) : nullptr;
  if (order) {
    hipLaunchKernelGGL(attn_order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, kv_len, gamma, B, gamma_max,
                       Hkv, plan.q_chunks, L_cap, plan.split_keys, plan.n_splits, order);
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  }
  hipLaunchKernelGGL(pick_split(D, plan.nq, plan.qg, plan.q_chunks), grid, dim3(threads), 0, stream,
                     (const uint16_t*)q, (const uint16_t*)k_cache, (const uint16_t*)v_cache,
                     cache_mask, kv_len, gamma, out, part_o, part_ml, counters, order, B, gamma_max, Hq,
                     Hkv, L_cap, scale * kLog2e, plan.split_keys, plan.n_splits, plan.q_chunks, status);
  if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  return SR_OK;
}

}  // namespace sr
