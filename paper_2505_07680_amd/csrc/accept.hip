// Accept-and-diverge for gfx950: speculative accept/reject with residual
// resampling and the bonus token (Section 2.2 steps 3-4, probabilistic
// acceptance; Eq. 2), plus per-position total variation distance (Eq. 5) and
// KL divergence, in one pass over the verifier and draft logits.
//
// Rows and chunks. A live row is one (sequence b, position j <= gamma_b): for
// j < gamma_b the verifier row p_j together with the draft row q_j (a "pair
// row"), for j = gamma_b the verifier row alone (it feeds the bonus token).
// Each row is cut into chunks of 256*E vocabulary entries; a workgroup task is
// one (row, chunk), each lane holding E entries of p and q in registers.
//
// Sweep kernel (persistent; the single pass over HBM). The grid is sized to be
// resident at once. Workgroup w takes tasks w, w + G, w + 2G, ... over the live
// rows only (a row table built from gamma in LDS), with G a multiple of the
// chunks per row, so the chunks of one row are processed at the same time by
// neighbouring workgroups. Per task:
//   1. chunk maxima of p and q, then the sums of exp(z - max) and the KL
//      numerator sum exp(p - max_p) ((p - max_p) - (q - max_q)), merged over
//      the four waves in a fixed order and published as one record with
//      device-coherent stores;
//   2. pair rows only: one wave re-loads the row's records until all of them
//      are present, merges them into the two log-normalisers (fp64, fixed
//      order; the finish kernel merges identically, so both get bit-identical
//      values), and every lane finishes sum |P - Q| over the entries still in
//      its registers. The chunk's sum is stored for the finish kernel.
// A record is four 8-byte words stored bit-inverted: a word that reads as all
// zeros has not been written yet (the inverted pattern would be a NaN, which
// no record holds), and naturally aligned 8-byte accesses are single-copy
// atomic, so a waiting wave needs no counter, no atomics and no wait for its
// own stores to complete. The finish kernel zeroes the records after use.
// Only sum |P - Q| is needed: with d = P - Q, a chunk's residual mass
// sum max(0, d) is (sum |d| + sum d) / 2 and sum d is the difference of the
// chunk's P and Q masses, which the records already hold.
//
// Finish kernel (one workgroup per sequence, one wave per row): merges the
// records into TV, KL, p(x), q(x) and a_j, runs the accept chain, and draws the
// token: a prefix scan over the stopping row's chunk masses finds the chunk
// that holds u*W, and that chunk alone is re-read and scanned in ascending
// vocabulary order with its element weights computed exactly as in the sweep.
// It also zeroes the sequence's records for the next call.
//
// Precision: exponentials in fp32 (relative error ~1e-7; weights below 2^-126
// of their chunk's largest flush to zero), every sum in fp64
// beyond a lane's own entries; TV and KL carry ~1e-7 relative error, and a
// draw can differ from exact arithmetic only when u*W lies within ~1e-7 W of
// a CDF breakpoint.

#include <limits.h>
#include <math.h>

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kThreads = 256;  // sweep workgroup: four waves, one chunk per task
constexpr int kWaves = kThreads / 64;

// Fixed-order merges of the per-wave partials.
__device__ __forceinline__ float max_waves(const float* v) {
  float m = v[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) m = fmaxf(m, v[i]);
  return m;
}
__device__ __forceinline__ double sum_waves(const double* v) {
  double a = v[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) a += v[i];
  return a;
}
constexpr int kSlots = 2;                // chunk records per lane in the row merges
constexpr int kMaxChunks = 64 * kSlots;  // chunks per row
constexpr int kMaxRows = SPECROUTER_MAX_GAMMA + 1;
constexpr int kMaxSeqs = 4096;           // sequences per sweep launch (row table in LDS)
constexpr uint32_t kSpinLimit = 1u << 22;
constexpr int kDeviceCoherent = 16;      // buffer cache-policy operand: sc1

// Per-(row, chunk) record of the first pass, as values.
struct StatRec {
  float mp, mq;  // chunk maxima of the p and q logits (-inf: none)
  double sp;     // sum exp(p - mp)
  double sq;     // sum exp(q - mq)
  double kl;     // sum exp(p - mp) ((p - mp) - (q - mq))
};
// In memory: four 8-byte words {mp | mq << 32, sp, sq, kl}, each inverted.
constexpr int kRecBytes = 32;

__device__ __forceinline__ void pack_rec(const StatRec& r, u32x4& w0, u32x4& w1) {
  const uint64_t a = ~((uint64_t)__float_as_uint(r.mp) | ((uint64_t)__float_as_uint(r.mq) << 32));
  const uint64_t b = ~__builtin_bit_cast(uint64_t, r.sp);
  const uint64_t c = ~__builtin_bit_cast(uint64_t, r.sq);
  const uint64_t d = ~__builtin_bit_cast(uint64_t, r.kl);
  w0 = u32x4{(uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32)};
  w1 = u32x4{(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)d, (uint32_t)(d >> 32)};
}
// True when all four words have been written.
__device__ __forceinline__ bool rec_present(const u32x4& w0, const u32x4& w1) {
  return (w0[0] | w0[1]) != 0u && (w0[2] | w0[3]) != 0u && (w1[0] | w1[1]) != 0u && (w1[2] | w1[3]) != 0u;
}
__device__ __forceinline__ StatRec unpack_rec(const u32x4& w0, const u32x4& w1) {
  StatRec r;
  r.mp = __uint_as_float(~w0[0]);
  r.mq = __uint_as_float(~w0[1]);
  r.sp = __builtin_bit_cast(double, ~((uint64_t)w0[2] | ((uint64_t)w0[3] << 32)));
  r.sq = __builtin_bit_cast(double, ~((uint64_t)w1[0] | ((uint64_t)w1[1] << 32)));
  r.kl = __builtin_bit_cast(double, ~((uint64_t)w1[2] | ((uint64_t)w1[3] << 32)));
  return r;
}

template <bool BF16>
struct Elt;

template <>
struct Elt<false> {
  static constexpr int VEC = 4;  // entries per 16-byte load
  __device__ static void load(const void* row, int x, float* out) {
    const floatx4 v = *(const floatx4*)((const float*)row + x);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[i] = v[i];
  }
  __device__ static float one(const void* row, int x) { return ((const float*)row)[x]; }
};

template <>
struct Elt<true> {
  static constexpr int VEC = 8;
  __device__ static void load(const void* row, int x, float* out) {
    const u32x4 u = *(const u32x4*)((const uint16_t*)row + x);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      out[2 * i] = bf16_lo(u[i]);
      out[2 * i + 1] = bf16_hi(u[i]);
    }
  }
  __device__ static float one(const void* row, int x) {
    return __uint_as_float((uint32_t)((const uint16_t*)row)[x] << 16);
  }
};

struct Args {
  const void* p;
  int64_t p_stride;
  const void* q;
  int64_t q_stride;
  const int32_t* drafts;
  const int32_t* gamma;
  const float* u_acc;
  const float* u_res;
  const int32_t* kv_len;
  int32_t* accept_len;
  int32_t* out_tokens;
  int32_t* new_len;
  float* accept_prob;
  float* p_tok;
  float* q_tok;
  float* kl;
  float* tv;
  int B, gmax, V, nc;
  float lg;       // log2(e) / T: softmax(z / T) entries are 2^((z - m) lg)
  double inv_t;   // 1 / T
  u32x4* stats;     // [B][gmax+1][nc] records, two 16-byte halves each
  double* tvabs;    // [B][gmax+1][nc] sum |P - Q| per chunk (pair rows)
  float* xlogit;    // [B][gmax+1][2] the draft token's p and q logits (pair rows)
  float* thr;       // [B][gmax+1][2] top-k / top-p thresholds of the p and q rows, or NULL (no filtering)
  int32_t* status;
  // rollback applied by the finish kernel (rb_kv NULL: none)
  int32_t* rb_kv;     // [B] cache lengths, in/out
  uint8_t* rb_mask;   // [B][L_cap] validity mask, or NULL
  int32_t* rb_phys;   // max over all sequences of the new lengths, or NULL
  int rb_lcap;
  int rb_reset;       // this launch's sweep sets *rb_phys to INT_MIN first (the call's first launch)
};

// exp2_hw drops weights under 2^-126 of their chunk's largest. The sweep and
// the finish kernel both use it, so a draw sees the same weights the chunk
// sums were built from.

// Pairwise sum of a lane's entries (a fixed tree, log2(N) roundings deep).
template <int N>
__device__ __forceinline__ float tree_sum(float (&v)[N]) {
#pragma unroll
  for (int s = N / 2; s > 0; s /= 2)
#pragma unroll
    for (int i = 0; i < s; ++i) v[i] += v[i + s];
  return v[0];
}

// Normaliser of a row: its maximum M and S = sum over chunks of
// s_c 2^((m_c - M) log2 e), so that softmax(z) = e^(z - M) / S. A chunk's
// entries e^(z - m_c) (as the chunk sums hold them) turn into probabilities
// by the factor f_c = 2^((m_c - M) log2 e) / S. The chunk records are held
// lane-wise (chunk lane*nslot + i in slot i) and merged in a fixed order, so
// the sweep and the finish kernel get bit-identical M, S and f_c.
struct RowNorm {
  float M;     // row maximum (-inf: none)
  double S;    // sum of the chunks' rescaled sums (>= 1 when M is finite)
  float invS;  // 1/S rounded to fp32
  float lg;    // log2(e) / T
  __device__ float factor(float m) const {  // f_c for a chunk whose maximum is m
    return m == kNegInf ? 0.f : exp2_hw((m - M) * lg) * invS;
  }
  __device__ double log_norm(double inv_t) const { return (double)M * inv_t + log(S); }  // ln sum e^(z/T)
};

__device__ __forceinline__ RowNorm row_norm(const float (&m)[kSlots], const double (&s)[kSlots], float lg) {
  RowNorm r;
  r.lg = lg;
  float ml = kNegInf;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) ml = fmaxf(ml, m[i]);
  r.M = wave_max(ml);
  double acc = 0.0;
  if (r.M != kNegInf) {
#pragma unroll
    for (int i = 0; i < kSlots; ++i)
      if (m[i] != kNegInf) acc += s[i] * (double)exp2_hw((m[i] - r.M) * lg);
  }
  r.S = wave_sum_d(acc);
  r.invS = r.S > 0.0 ? (float)(1.0 / r.S) : 0.f;
  return r;
}


// Inclusive prefix over sequences of their live-row counts (gamma_b + 1, or 0
// for an invalid gamma), in LDS. Each thread scans a contiguous segment; the
// segment totals are scanned across the workgroup in parallel.
__device__ void build_row_table(const int32_t* gamma, int gmax, int B, int* rows) {
  __shared__ int wsum[kThreads / 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63, w = tid >> 6;
  const int per = (B + kThreads - 1) / kThreads;
  const int b0 = min(tid * per, B), b1 = min(b0 + per, B);
  int run = 0;
  for (int b = b0; b < b1; ++b) {
    const int g = gamma[b];
    run += (g >= 0 && g <= gmax) ? g + 1 : 0;
    rows[b] = run;
  }
  const int incl = wave_incl_scan_i(run);
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int off = incl - run;
  for (int i = 0; i < w; ++i) off += wsum[i];
  for (int b = b0; b < b1; ++b) rows[b] += off;
  __syncthreads();
}

// ============================================================================
// Sweep kernel

// One task's entries as loaded: fp32 entries are replaced by their
// exponentials in the first pass and kept for the second; bf16 entries stay
// packed and the second pass recomputes the exponentials (the registers then
// hold twice as many entries per byte of HBM read).
template <bool BF16, int E>
struct Raw;
template <int E>
struct Raw<false, E> {
  float p[E], q[E];  // exponentials after the first pass
  __device__ float gp(int e) const { return p[e]; }
  __device__ float gq(int e) const { return q[e]; }
};
// An opaque copy: each phase unpacks bf16 entries afresh instead of the
// compiler keeping every unpacked value live from the first use to the last.
__device__ __forceinline__ uint32_t fresh(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}
template <int E>
struct Raw<true, E> {
  u32x4 pk[E / 8], qk[E / 8];  // as loaded
  __device__ float gp(int e) const {
    const uint32_t w = fresh(pk[e / 8][(e % 8) / 2]);
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  }
  __device__ float gq(int e) const {
    const uint32_t w = fresh(qk[e / 8][(e % 8) / 2]);
    return (e & 1) ? bf16_hi(w) : bf16_lo(w);
  }
};

// Set the entries below a threshold to -inf (the top-k / top-p filter).
template <int E>
__device__ __forceinline__ void mask_below(Raw<false, E>& r, float tp, float tq) {
#pragma unroll
  for (int e = 0; e < E; ++e) {
    r.p[e] = r.p[e] >= tp ? r.p[e] : kNegInf;
    r.q[e] = r.q[e] >= tq ? r.q[e] : kNegInf;
  }
}
__device__ __forceinline__ uint32_t mask_pair(uint32_t w, float t) {
  constexpr uint32_t kNegInfBf16 = 0xff80u;
  const uint32_t lo = bf16_lo(w) >= t ? (w & 0xffffu) : kNegInfBf16;
  const uint32_t hi = bf16_hi(w) >= t ? (w >> 16) : kNegInfBf16;
  return lo | (hi << 16);
}
template <int E>
__device__ __forceinline__ void mask_below(Raw<true, E>& r, float tp, float tq) {
#pragma unroll
  for (int v = 0; v < E / 8; ++v)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r.pk[v][i] = mask_pair(r.pk[v][i], tp);
      r.qk[v][i] = mask_pair(r.qk[v][i], tq);
    }
}

struct TaskInfo {
  int b, j, c, row;
  int x;  // the row's draft token (pair rows; -1 for a bonus row)
  bool pair;
  const char* prow;
  const char* qrow;  // the draft row (a pair row), or the p row for a bonus row (never read)
};

template <bool BF16>
__device__ __forceinline__ TaskInfo decode_task(const Args& A, const int* rows, long task) {
  TaskInfo t;
  const int rank = (int)(task / A.nc);
  t.c = (int)(task % A.nc);
  int lo = 0, hi = A.B - 1;  // first sequence whose prefix exceeds rank
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (rows[mid] > rank) hi = mid;
    else lo = mid + 1;
  }
  t.b = lo;
  const int first = lo ? rows[lo - 1] : 0;
  t.j = rank - first;
  t.pair = t.j < rows[lo] - first - 1;
  t.row = t.b * (A.gmax + 1) + t.j;
  const size_t esz = BF16 ? 2 : 4;
  t.prow = (const char*)A.p + ((size_t)t.b * A.p_stride + (size_t)t.j * A.V) * esz;
  t.qrow = t.pair ? (const char*)A.q + ((size_t)t.b * A.q_stride + (size_t)t.j * A.V) * esz : t.prow;
  t.x = t.pair ? A.drafts[(size_t)t.b * A.gmax + t.j] : -1;  // uniform: a scalar load
  return t;
}

// Issue the loads of one task (always the same count, so the waits of the
// task before it stay exact). Offsets past V are clamped into the row.
template <bool BF16, int E>
__device__ __forceinline__ void issue_loads(const Args& A, const TaskInfo& t, Raw<BF16, E>& r) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int NV = E / VEC;
  const int lane = threadIdx.x & 63;
  const int base = t.c * (kThreads * E) + (threadIdx.x >> 6) * (64 * E);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int x = min(base + (v * 64 + lane) * VEC, A.V - VEC);
    if constexpr (BF16) {
      r.pk[v] = *(const u32x4*)((const uint16_t*)t.prow + x);
    } else {
      const floatx4 f = *(const floatx4*)((const float*)t.prow + x);
#pragma unroll
      for (int i = 0; i < 4; ++i) r.p[v * 4 + i] = f[i];
    }
  }
  // The draft row through a buffer resource: a bonus row has none, so its
  // resource is empty and the same loads return zeros with no memory traffic.
  constexpr uint32_t kEsz = BF16 ? 2u : 4u;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(t.qrow, t.pair ? (size_t)A.V * kEsz : 0);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int x = min(base + (v * 64 + lane) * VEC, A.V - VEC);
    const u32x4 u = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rq, (uint32_t)x * kEsz, 0, 0));
    if constexpr (BF16) {
      r.qk[v] = u;
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) r.q[v * 4 + i] = __uint_as_float(u[i]);
    }
  }
}

// Workgroup state of the sweep and its two passes over a task.
struct SweepShared {
  float m[2][kWaves];
  double s[3][kWaves];
  float f[2];        // this chunk's factors f_c for p and q
  int ix[2][kWaves];  // greedy: the waves' argmax indices of p and q
};

template <bool BF16, int E>
struct Sweep {
  static constexpr int VEC = Elt<BF16>::VEC;
  static constexpr int kChunk = kThreads * E;
  const Args& A;
  SweepShared& sh;
  const int tid, lane, w, nc, nslot;
  const __amdgpu_buffer_rsrc_t rs_stats;

  __device__ Sweep(const Args& a, SweepShared& s)
      : A(a), sh(s), tid(threadIdx.x), lane(threadIdx.x & 63), w(threadIdx.x >> 6), nc(a.nc),
        nslot((a.nc + 63) / 64),
        rs_stats(make_rsrc(a.stats, (size_t)a.B * (a.gmax + 1) * a.nc * kRecBytes)) {}

  // First pass over a task's entries: chunk maxima, exponentials, sums, KL
  // numerator, and the published record. Leaves the chunk maxima in cmp/cmq
  // (and, for fp32, the exponentials in r).
  __device__ __forceinline__ void first_pass(const TaskInfo& t, Raw<BF16, E>& r, float& cmp, float& cmq) {
    const int base = t.c * kChunk + w * (64 * E);
    if (A.thr) {  // top-k / top-p: entries below the row's threshold become -inf (workgroup-uniform branch)
      const float tp = A.thr[(size_t)t.row * 2];
      const float tq = t.pair ? A.thr[(size_t)t.row * 2 + 1] : kNegInf;
      mask_below(r, tp, tq);
    }
    // The draft token's two logits, for the finish kernel's acceptance test:
    // the lane that holds entry x stores them (once per row).
    const int xo = t.x - base;  // offset of x in this wave's entries
    if (xo >= 0 && xo < 64 * E && lane == (xo % (64 * VEC)) / VEC) {
      const int ex = (xo / (64 * VEC)) * VEC + xo % VEC;
      float zp = 0.f, zq = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e)
        if (e == ex) {
          zp = r.gp(e);
          zq = r.gq(e);
        }
      A.xlogit[(size_t)t.row * 2] = zp;
      A.xlogit[(size_t)t.row * 2 + 1] = zq;
    }
    auto in_v = [&](int e) __attribute__((always_inline)) {  // entry e lies below V
      return base + ((e / VEC) * 64 + lane) * VEC < A.V;
    };
    float mp = kNegInf, mq = kNegInf;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const bool in = in_v(e);
      const float zp = r.gp(e), zq = r.gq(e);  // unconditional: then a select
      mp = fmaxf(mp, in ? zp : kNegInf);
      mq = fmaxf(mq, in && t.pair ? zq : kNegInf);
      if (e % 8 == 7) __builtin_amdgcn_sched_barrier(0);  // unpack eight entries at a time
    }
    mp = wave_max(mp);
    if (t.pair) mq = wave_max(mq);
    if (lane == 0) {
      sh.m[0][w] = mp;
      sh.m[1][w] = mq;
    }
    __syncthreads();
    cmp = max_waves(sh.m[0]);
    cmq = max_waves(sh.m[1]);

    // exponentials, sums, KL numerator; groups of four are summed as
    // (a0 + a1) + (a2 + a3), then a tree over groups
    const float lg = A.lg;
    const float rp = cmp == kNegInf ? 0.f : cmp * lg;
    const float rq = cmq == kNegInf ? 0.f : cmq * lg;
    // the KL numerator on logits relative to the chunk maxima, so that the
    // row-level merge subtracts no large terms (two rows whose filtered
    // distributions coincide give exactly zero)
    const float op = cmp == kNegInf ? 0.f : cmp;
    const float oq = cmq == kNegInf ? 0.f : cmq;
    double dsp, dsq = 0.0, dkl = 0.0;
    if (t.pair) {
      float gp[E / 4], gq[E / 4], gk[E / 4];
#pragma unroll
      for (int g = 0; g < E / 4; ++g) {
        float ep[4], eq[4], kt[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int e = g * 4 + i;
          const bool in = in_v(e);
          const float zp = r.gp(e), zq = r.gq(e);
          ep[i] = in ? exp2_hw(fmaf(zp, lg, -rp)) : 0.f;
          eq[i] = in ? exp2_hw(fmaf(zq, lg, -rq)) : 0.f;
          kt[i] = ep[i] > 0.f ? ep[i] * ((zp - op) - (zq - oq)) : 0.f;
          if constexpr (!BF16) {
            r.p[e] = ep[i];
            r.q[e] = eq[i];
          }
        }
        gp[g] = (ep[0] + ep[1]) + (ep[2] + ep[3]);
        gq[g] = (eq[0] + eq[1]) + (eq[2] + eq[3]);
        gk[g] = (kt[0] + kt[1]) + (kt[2] + kt[3]);
        __builtin_amdgcn_sched_barrier(0);  // bounds live ranges: one group at a time
      }
      dsp = wave_sum_d((double)tree_sum(gp));
      dsq = wave_sum_d((double)tree_sum(gq));
      dkl = wave_sum_d((double)tree_sum(gk));
    } else {
      float gp[E / 4];
#pragma unroll
      for (int g = 0; g < E / 4; ++g) {
        float ep[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float zp = r.gp(g * 4 + i);
          ep[i] = in_v(g * 4 + i) ? exp2_hw(fmaf(zp, lg, -rp)) : 0.f;
        }
        gp[g] = (ep[0] + ep[1]) + (ep[2] + ep[3]);
      }
      dsp = wave_sum_d((double)tree_sum(gp));
    }
    if (lane == 0) {
      sh.s[0][w] = dsp;
      sh.s[1][w] = dsq;
      sh.s[2][w] = dkl;
    }
    __syncthreads();
    if (tid == 0) {
      const size_t rec = (size_t)t.row * nc + t.c;
      StatRec sr;
      sr.mp = cmp;
      sr.mq = cmq;
      sr.sp = sum_waves(sh.s[0]);
      sr.sq = sum_waves(sh.s[1]);
      sr.kl = sum_waves(sh.s[2]);
      u32x4 w0, w1;
      pack_rec(sr, w0, w1);
      __builtin_amdgcn_raw_buffer_store_b128(w0, rs_stats, (uint32_t)(rec * kRecBytes), 0, kDeviceCoherent);
      __builtin_amdgcn_raw_buffer_store_b128(w1, rs_stats, (uint32_t)(rec * kRecBytes + 16), 0, kDeviceCoherent);
    }
  }

  // Greedy decoding: the chunk's maxima of p and q and the lowest index
  // holding each, published as the chunk's record (indices in the sum fields).
  __device__ __forceinline__ void argmax_pass(const TaskInfo& t, const Raw<BF16, E>& r) {
    const int base = t.c * kChunk + w * (64 * E);
    float bp = kNegInf, bq = kNegInf;
    int ip = -1, iq = -1;
#pragma unroll
    for (int e = 0; e < E; ++e) {  // a lane's entries in ascending index order
      const int idx = base + ((e / VEC) * 64 + lane) * VEC + e % VEC;
      const bool in = idx < A.V;
      const float zp = r.gp(e), zq = r.gq(e);
      if (in && (ip < 0 || zp > bp)) {
        bp = zp;
        ip = idx;
      }
      if (in && (iq < 0 || zq > bq)) {
        bq = zq;
        iq = idx;
      }
    }
    const float mp = wave_max(bp);
    const int jp = wave_min_i(ip >= 0 && bp == mp ? ip : INT_MAX);
    float mq = kNegInf;
    int jq = INT_MAX;
    if (t.pair) {
      mq = wave_max(bq);
      jq = wave_min_i(iq >= 0 && bq == mq ? iq : INT_MAX);
    }
    if (lane == 0) {
      sh.m[0][w] = mp;
      sh.m[1][w] = mq;
      sh.ix[0][w] = jp;
      sh.ix[1][w] = jq;
    }
    __syncthreads();
    if (tid == 0) {
      StatRec sr;
      sr.mp = max_waves(sh.m[0]);
      sr.mq = max_waves(sh.m[1]);
      int ap = INT_MAX, aq = INT_MAX;
      for (int i = 0; i < kWaves; ++i) {
        if (sh.m[0][i] == sr.mp) ap = min(ap, sh.ix[0][i]);
        if (sh.m[1][i] == sr.mq) aq = min(aq, sh.ix[1][i]);
      }
      sr.sp = (double)ap;
      sr.sq = (double)aq;
      sr.kl = 0.0;
      u32x4 w0, w1;
      pack_rec(sr, w0, w1);
      const size_t rec = (size_t)t.row * nc + t.c;
      __builtin_amdgcn_raw_buffer_store_b128(w0, rs_stats, (uint32_t)(rec * kRecBytes), 0, kDeviceCoherent);
      __builtin_amdgcn_raw_buffer_store_b128(w1, rs_stats, (uint32_t)(rec * kRecBytes + 16), 0, kDeviceCoherent);
    }
    __syncthreads();  // the next task rewrites sh.m and sh.ix
  }

  // One wave: re-load the records of a pair row until all of them are
  // present, merge them into the row's normalisers and leave the chunk's
  // factors in sh.f (lane 0 writes them).
  __device__ __forceinline__ void row_factors(const TaskInfo& t, float cmp, float cmq) {
    float m1[kSlots], m2[kSlots];
    double s1[kSlots], s2[kSlots];
    for (uint32_t it = 0;; ++it) {
      bool ok = true;
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        const int cc = lane * nslot + i;
        const bool in = i < nslot && cc < nc;
        const uint32_t off = (uint32_t)(((size_t)t.row * nc + (in ? cc : 0)) * kRecBytes);
        const u32x4 w0 = __builtin_amdgcn_raw_buffer_load_b128(rs_stats, off, 0, kDeviceCoherent);
        const u32x4 w1 = __builtin_amdgcn_raw_buffer_load_b128(rs_stats, off + 16, 0, kDeviceCoherent);
        ok = ok && (!in || rec_present(w0, w1));
        const StatRec sr = unpack_rec(w0, w1);
        m1[i] = in ? sr.mp : kNegInf;
        m2[i] = in ? sr.mq : kNegInf;
        s1[i] = in ? sr.sp : 0.0;
        s2[i] = in ? sr.sq : 0.0;
      }
      if (__ballot(!ok) == 0ull) break;
      if (it == kSpinLimit) {
        if (lane == 0 && A.status) atomicOr(A.status, SR_ST_TIMEOUT);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    const RowNorm np = row_norm(m1, s1, A.lg);
    const RowNorm nq = row_norm(m2, s2, A.lg);
    if (lane == 0) {
      sh.f[0] = np.factor(cmp);
      sh.f[1] = nq.factor(cmq);
    }
  }

  // Every wave, after a barrier that follows row_factors: sum |P - Q| over the
  // entries kept from the first pass; the chunk's sum is stored for the finish
  // kernel.
  __device__ __forceinline__ void tv_pass(const TaskInfo& t, const Raw<BF16, E>& r, float cmp, float cmq) {
    const float fp = sh.f[0], fq = sh.f[1];
    const float lg = A.lg;
    const float rp = cmp == kNegInf ? 0.f : cmp * lg;
    const float rq = cmq == kNegInf ? 0.f : cmq * lg;
    const int base = t.c * kChunk + w * (64 * E);
    float ga[E / 4];
#pragma unroll
    for (int g = 0; g < E / 4; ++g) {
      float a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = g * 4 + i;
        float ep, eq;
        if constexpr (BF16) {
          const bool in = base + ((e / VEC) * 64 + lane) * VEC < A.V;
          const float zp = r.gp(e), zq = r.gq(e);
          ep = in ? exp2_hw(fmaf(zp, lg, -rp)) : 0.f;
          eq = in ? exp2_hw(fmaf(zq, lg, -rq)) : 0.f;
        } else {
          ep = r.p[e];
          eq = r.q[e];
        }
        {
          // separately rounded products: identical p and q rows give exactly zero
#pragma clang fp contract(off)
          a[i] = fabsf(ep * fp - eq * fq);
        }
      }
      ga[g] = (a[0] + a[1]) + (a[2] + a[3]);
      __builtin_amdgcn_sched_barrier(0);
    }
    const double dtv = wave_sum_d((double)tree_sum(ga));
    if (lane == 0) sh.s[0][w] = dtv;
    __syncthreads();
    if (tid == 0) A.tvabs[(size_t)t.row * nc + t.c] = sum_waves(sh.s[0]);
  }
};

// Persistent sweep: workgroup w takes tasks w, w + G, w + 2G, ... two deep.
template <bool BF16, int E>
__global__ void __launch_bounds__(kThreads)
accept_sweep_kernel(Args A) {
  extern __shared__ int s_rows[];  // [B] inclusive prefix of live rows
  __shared__ SweepShared sh;
  Sweep<BF16, E> S(A, sh);
  const int w = S.w;
  if (A.rb_reset && A.rb_phys && blockIdx.x == 0 && threadIdx.x == 0) *A.rb_phys = INT_MIN;  // see finish_rollback

  build_row_table(A.gamma, A.gmax, A.B, s_rows);
  const long n_tasks = (long)s_rows[A.B - 1] * S.nc;

  // Pipeline: the second pass of task i runs after the loads of task i+1 are
  // issued and before its first pass, so the other chunks of task i's row have
  // had a whole first pass to publish. Every LDS slot is rewritten only after a
  // barrier that follows its last read.
  long task = blockIdx.x;
  if (task >= n_tasks) return;
  TaskInfo t = decode_task<BF16>(A, s_rows, task);
  Raw<BF16, E> cur;
  issue_loads<BF16, E>(A, t, cur);
  float cmp, cmq;
  S.first_pass(t, cur, cmp, cmq);
  for (;;) {
    const long task_n = task + gridDim.x;
    const bool more = task_n < n_tasks;
    const TaskInfo tn = decode_task<BF16>(A, s_rows, more ? task_n : task);  // past the end: reload (cached)
    Raw<BF16, E> nxt;
    // Waves 1-3 prefetch first. Wave 0 polls the row's records first (a wave's
    // loads complete in issue order, so its poll would otherwise also wait for
    // its prefetch) and prefetches after.
    __builtin_amdgcn_sched_barrier(0);
    if (w != 0 || !t.pair) issue_loads<BF16, E>(A, tn, nxt);
    __builtin_amdgcn_sched_barrier(0);
    if (t.pair) {  // workgroup-uniform
      if (w == 0) {
        S.row_factors(t, cmp, cmq);
        __builtin_amdgcn_sched_barrier(0);
        issue_loads<BF16, E>(A, tn, nxt);
        __builtin_amdgcn_sched_barrier(0);
      }
      __syncthreads();
      S.tv_pass(t, cur, cmp, cmq);
    }
    if (!more) break;
    float cmp_n, cmq_n;
    S.first_pass(tn, nxt, cmp_n, cmq_n);
    task = task_n;
    t = tn;
    cur = nxt;
    cmp = cmp_n;
    cmq = cmq_n;
  }
}

// Greedy decoding: one pass of chunk argmaxes, no second pass and no waiting
// (workgroup w takes tasks w, w + G, ..., loading one task ahead).
template <bool BF16, int E>
__global__ void __launch_bounds__(kThreads)
accept_argmax_kernel(Args A) {
  extern __shared__ int s_rows[];
  __shared__ SweepShared sh;
  Sweep<BF16, E> S(A, sh);
  if (A.rb_reset && A.rb_phys && blockIdx.x == 0 && threadIdx.x == 0) *A.rb_phys = INT_MIN;  // see finish_rollback
  build_row_table(A.gamma, A.gmax, A.B, s_rows);
  const long n_tasks = (long)s_rows[A.B - 1] * S.nc;
  long task = blockIdx.x;
  if (task >= n_tasks) return;
  TaskInfo t = decode_task<BF16>(A, s_rows, task);
  Raw<BF16, E> cur;
  issue_loads<BF16, E>(A, t, cur);
  for (;;) {
    const long task_n = task + gridDim.x;
    const bool more = task_n < n_tasks;
    const TaskInfo tn = decode_task<BF16>(A, s_rows, more ? task_n : task);
    Raw<BF16, E> nxt;
    __builtin_amdgcn_sched_barrier(0);
    issue_loads<BF16, E>(A, tn, nxt);
    __builtin_amdgcn_sched_barrier(0);
    S.argmax_pass(t, cur);
    if (!more) break;
    task = task_n;
    t = tn;
    cur = nxt;
  }
}

// ============================================================================
// Finish kernel

__device__ void write_invalid(const Args& A, int b, uint32_t bits) {
  const int lane = threadIdx.x & 63;
  if (lane == 0) {
    A.accept_len[b] = -1;
    if (A.new_len) A.new_len[b] = A.kv_len[b];
    if (A.status) atomicOr(A.status, (int32_t)bits);
  }
  for (int j = lane; j <= A.gmax; j += 64) A.out_tokens[(size_t)b * (A.gmax + 1) + j] = -1;
  const float nan = __builtin_nanf("");
  for (int j = lane; j < A.gmax; j += 64) {
    const size_t o = (size_t)b * A.gmax + j;
    if (A.accept_prob) A.accept_prob[o] = nan;
    if (A.p_tok) A.p_tok[o] = nan;
    if (A.q_tok) A.q_tok[o] = nan;
    if (A.kl) A.kl[o] = nan;
    if (A.tv) A.tv[o] = nan;
  }
}

// Rollback of sequence b from `old` to `want` rows (Section 4.4, Eq. 9),
// exactly as the rollback call does it: a length outside [0, L_cap] or a
// negative target is flagged and left alone, a target above the length is
// flagged and ignored; otherwise the mask entries [n, old) are cleared and
// the length becomes n = min(old, want). The physical length is the maximum
// of the resulting lengths over all sequences: the call's first sweep launch
// sets it to INT_MIN and every sequence folds its length in with an atomic
// maximum (no result is waited for). `old` is read at the start of the
// finish kernel, so the rollback adds no round trip. Called by one whole
// wave.
__device__ void finish_rollback(const Args& A, int b, int old, int want) {
  if (!A.rb_kv) return;
  const int lane = threadIdx.x & 63;
  int n = old;
  int32_t st = 0;
  if (old < 0 || old > A.rb_lcap || want < 0) {
    st = SR_ST_KVLEN;
  } else {
    if (want > old) st = SR_ST_ROLLBACK_GROW;
    n = min(old, want);
    if (A.rb_mask)
      for (int x = n + lane; x < old; x += 64) A.rb_mask[(size_t)b * A.rb_lcap + x] = 0;
  }
  if (lane == 0) {
    A.rb_kv[b] = n;
    if (st && A.status) atomicOr(A.status, st);
    if (A.rb_phys) atomicMax(A.rb_phys, n);
  }
}

// Zero the records of sequence b's live rows (the "not yet written" state the
// next call's sweep waits on). Called by one whole wave.
__device__ void clear_records(const Args& A, int b, int gam) {
  const size_t first = (size_t)b * (A.gmax + 1) * A.nc * 2;
  const size_t n = (size_t)(gam + 1) * A.nc * 2;
  for (size_t i = threadIdx.x & 63; i < n; i += 64) A.stats[first + i] = u32x4{0u, 0u, 0u, 0u};
}

// Wave-wide inclusive prefix sum (fp64) in ascending lane order: DPP row
// shifts inside each 16-lane row, then the totals of the earlier rows.
__device__ __forceinline__ double wave_incl_scan(double x) {
  x = x + dpp_f64<0x111>(x);  // row_shr:1 (lanes without a source read 0)
  x = x + dpp_f64<0x112>(x);  // row_shr:2
  x = x + dpp_f64<0x114>(x);  // row_shr:4
  x = x + dpp_f64<0x118>(x);  // row_shr:8
  const double r0 = lane_value(x, 15), r1 = lane_value(x, 31), r2 = lane_value(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  const double r01 = r0 + r1;
  return x + (row == 0 ? 0.0 : row == 1 ? r0 : row == 2 ? r01 : r01 + r2);
}

struct RowRes {
  double a;
  float p_tok, q_tok, kl, tv;
};

// A row's chunk records, lane-wise (chunk lane*nslot + i in slot i).
struct RowRecs {
  float mp[kSlots], mq[kSlots];
  double sp[kSlots], sq[kSlots], kl[kSlots], ta[kSlots];
};

__device__ __forceinline__ void load_row(const Args& A, int row, bool pair, RowRecs& R) {
  const int lane = threadIdx.x & 63;
  const int nslot = (A.nc + 63) / 64;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int cc = lane * nslot + i;
    const bool in = i < nslot && cc < A.nc;
    const StatRec r = in ? unpack_rec(A.stats[((size_t)row * A.nc + cc) * 2], A.stats[((size_t)row * A.nc + cc) * 2 + 1])
                         : StatRec{kNegInf, kNegInf, 0.0, 0.0, 0.0};
    R.mp[i] = r.mp;
    R.sp[i] = r.sp;
    R.mq[i] = pair ? r.mq : kNegInf;
    R.sq[i] = pair ? r.sq : 0.0;
    R.kl[i] = pair ? r.kl : 0.0;
    R.ta[i] = in && pair ? A.tvabs[(size_t)row * A.nc + cc] : 0.0;
  }
}

// What the accept chain and the draw need of one row, kept in LDS by the
// wave that merged the row: the chunks' masses (p, and the residual
// max(0, p - q) for a pair row) and maxima, and the row's normalisers.
struct FinishShared {
  double mass[kMaxRows][2][kMaxChunks];  // [row][p, residual][chunk]
  float cmax[kMaxRows][2][kMaxChunks];   // [row][p, q][chunk] chunk maxima
  float norm[kMaxRows][4];               // M_p, 1/S_p, M_q, 1/S_q
  int resid[kMaxRows];                   // the residual has positive mass
  RowRes rr[kMaxRows];
  int x[kMaxRows];
  float uacc[kMaxRows], ures[kMaxRows];
};

// Finish kernel: one workgroup per sequence with at least four waves.
//   load:  every thread loads its position's draft and uniforms together
//          with gamma (one round trip);
//   rows:  one wave per live row j <= gamma merges the row's records (the
//          draft token's two logits are loaded alongside) into a_j, p(x),
//          q(x), TV_j and KL_j, and leaves the row's chunk masses, maxima
//          and normalisers in LDS;
//   chain: wave 0 finds the stopping row k and, from k's chunk masses, the
//          chunk that holds u*W and the offset of u*W inside it;
//   draw:  waves 0-3 re-read that chunk (each thread a contiguous run of
//          entries), weigh it exactly as the sweep did, and a block-wide
//          prefix scan in ascending vocabulary order finds the token.
template <bool BF16, int E>
__global__ void __launch_bounds__(1024)
accept_finish_kernel(Args A) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int kChunk = kThreads * E;
  __shared__ FinishShared F;
  __shared__ uint32_t s_bad;
  __shared__ int s_k, s_cs, s_resid, s_hit[4], s_last[4], s_tok;
  __shared__ double s_rem, s_wt[4];
  __shared__ float s_fac[4];  // rp, rq, fp, fq of the draw chunk
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int nw = blockDim.x >> 6;
  const int G1 = A.gmax + 1;
  const int nslot = (A.nc + 63) / 64;
  // ---- load: gamma and the per-position inputs in one round trip
  const int gam = A.gamma[b];
  if (tid == 0) s_bad = 0;
  if (tid < G1) {
    const int j = tid;
    const int x = j < A.gmax ? A.drafts[(size_t)b * A.gmax + j] : -1;
    const float ua = j < A.gmax ? A.u_acc[(size_t)b * A.gmax + j] : 0.f;
    const float ur = A.u_res[(size_t)b * G1 + j];
    F.x[j] = x;
    F.uacc[j] = ua;
    F.ures[j] = ur;
  }
  const int kvl = A.kv_len ? A.kv_len[b] : 0;
  const int rb_old = A.rb_kv ? A.rb_kv[b] : 0;
  // row w's records and draft logits, in the same round trip (pair or bonus
  // row is decided once gamma has arrived)
  RowRecs R0;
  float zx0[2] = {0.f, 0.f};
  if (w <= A.gmax) {
    load_row(A, b * G1 + w, true, R0);
    if (w < A.gmax) {
      zx0[0] = A.xlogit[((size_t)b * G1 + w) * 2];
      zx0[1] = A.xlogit[((size_t)b * G1 + w) * 2 + 1];
    }
  }
  if (gam < 0 || gam > A.gmax) {
    if (w == 0) {
      write_invalid(A, b, SR_ST_GAMMA);
      finish_rollback(A, b, rb_old, kvl);
    }
    return;  // the sweep touched no row of this sequence
  }
  __syncthreads();
  // ---- data checks
  if (tid <= gam) {
    uint32_t bad = 0;
    const int j = tid;
    if (j < gam) {
      const int x = F.x[j];
      if (x < 0 || x >= A.V) bad |= SR_ST_TOKEN;
      const float u = F.uacc[j];
      if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
    }
    const float u = F.ures[j];
    if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
    if (j == 0 && A.kv_len && kvl < gam + 1) bad |= SR_ST_KVLEN;
    if (bad) atomicOr(&s_bad, bad);
  }
  // ---- rows (one wave per live row)
  const size_t esz = BF16 ? 2 : 4;
  for (int j = w; j <= gam; j += nw) {
    const bool pair = j < gam;
    const int x = pair ? F.x[j] : -1;
    const bool xin = x >= 0 && x < A.V;
    RowRecs R;
    float zpx, zqx;
    if (j == w) {
      R = R0;
      zpx = zx0[0];
      zqx = zx0[1];
    } else {  // a second row for this wave (gamma_max + 1 > waves)
      load_row(A, b * G1 + j, true, R);
      zpx = A.xlogit[((size_t)b * G1 + j) * 2];
      zqx = A.xlogit[((size_t)b * G1 + j) * 2 + 1];
    }
    if (!pair) {  // the bonus row: p only
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        R.mq[i] = kNegInf;
        R.sq[i] = 0.0;
        R.kl[i] = 0.0;
        R.ta[i] = 0.0;
      }
    }
    const RowNorm np = row_norm(R.mp, R.sp, A.lg);
    const RowNorm nq = row_norm(R.mq, R.sq, A.lg);
    // chunk masses with the same factors the sweep's sum |P - Q| used
    double my_res = 0.0;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      const int cc = lane * nslot + i;
      const double pm = R.sp[i] * (double)np.factor(R.mp[i]);
      const double qm = R.sq[i] * (double)nq.factor(R.mq[i]);
      const double rm = pair ? fmax(0.0, 0.5 * (R.ta[i] + pm - qm)) : 0.0;
      my_res += rm;
      if (i < nslot && cc < A.nc) {
        F.mass[j][0][cc] = pm;
        F.mass[j][1][cc] = rm;
        F.cmax[j][0][cc] = R.mp[i];
        F.cmax[j][1][cc] = R.mq[i];
      }
    }
    const bool residual = pair && wave_sum_d(my_res) > 0.0;
    if (lane == 0) {
      F.norm[j][0] = np.M;
      F.norm[j][1] = np.invS;
      F.norm[j][2] = nq.M;
      F.norm[j][3] = nq.invS;
      F.resid[j] = residual ? 1 : 0;
    }
    if (!pair) continue;  // the bonus row needs no divergences
    const double Lp = np.log_norm(A.inv_t), Lq = nq.log_norm(A.inv_t);
    // KL = (1/T) sum_c f_c (kl_c + s_c ((m_c - M_p) - (m'_c - M_q))) - (ln S_p - ln S_q),
    // kl_c being the chunk's numerator relative to its maxima m_c (p) and m'_c (q)
    double tvd = 0.0, kld = 0.0;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      tvd += R.ta[i];
      if (R.mp[i] != kNegInf) {
        const double dm = ((double)R.mp[i] - (double)np.M) - ((double)R.mq[i] - (double)nq.M);
        kld += (double)np.factor(R.mp[i]) * (R.kl[i] + R.sp[i] * dm);
      }
    }
    tvd = 0.5 * wave_sum_d(tvd);
    kld = A.inv_t * wave_sum_d(kld) - (log(np.S) - log(nq.S));
    // p(x), q(x) and a = min(1, p(x)/q(x)): one exponential per lane (0-2)
    const double lpx = (double)zpx * A.inv_t - Lp;
    const double lqx = (double)zqx * A.inv_t - Lq;
    const double arg = lane == 0 ? lpx : (lane == 1 ? lqx : lpx - lqx);
    const double ex = exp(arg);
    const double pt = lane_value(ex, 0), qt = lane_value(ex, 1), rt = lane_value(ex, 2);
    if (lane == 0) {
      double a = __builtin_nan("");
      if (xin) a = (lqx == -INFINITY || lpx >= lqx) ? 1.0 : rt;
      F.rr[j] = RowRes{a, xin ? (float)pt : __builtin_nanf(""), xin ? (float)qt : __builtin_nanf(""), (float)kld,
                       (float)tvd};
    }
  }
  __syncthreads();
  if (s_bad) {
    if (w == 0) {
      clear_records(A, b, gam);  // every wave has finished reading them
      write_invalid(A, b, s_bad);
      finish_rollback(A, b, rb_old, kvl);
    }
    return;
  }
  // ---- accept chain and the chunk of the draw (wave 0)
  if (w == 0) {
    bool rej = false;
    if (lane < gam) rej = !((double)F.uacc[lane] < F.rr[lane].a);
    const unsigned long long rmask = __ballot(rej);
    const int k = rmask ? (__ffsll((long long)rmask) - 1) : gam;
    const bool residual = F.resid[k] != 0;
    double mass[kSlots];
    double my = 0.0;
    int my_last = -1;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      const int cc = lane * nslot + i;
      const bool in = i < nslot && cc < A.nc;
      mass[i] = in ? F.mass[k][residual ? 1 : 0][cc] : 0.0;
      my += mass[i];
      if (mass[i] > 0.0) my_last = cc;
    }
    const double incl = wave_incl_scan(my);
    const double W = lane_value(incl, 63);
    const double target = (double)F.ures[k] * W;
    // the first chunk with positive mass whose end exceeds the target
    int cs = -1;
    double pre = 0.0;
    const unsigned long long hit = __ballot(incl > target && my > 0.0);
    if (hit) {
      const int hl = __ffsll((long long)hit) - 1;
      double run = incl - my;
      int found = -1;
      double fpre = 0.0;
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        if (found < 0 && mass[i] > 0.0 && run + mass[i] > target) {
          found = lane * nslot + i;
          fpre = run;
        }
        run += mass[i];
      }
      cs = lane_value(found, hl);
      pre = lane_value(fpre, hl);
    }
    if (cs < 0) {  // rounding put the target at the very end: the last chunk with mass
      cs = max(wave_max_i(my_last), 0);
      double before = 0.0;
#pragma unroll
      for (int i = 0; i < kSlots; ++i)
        if (lane * nslot + i < cs) before += mass[i];
      pre = wave_sum_d(before);
    }
    if (lane == 0) {
      // the chunk's maxima and factors, as the sweep used them
      const bool pair = k < gam;
      const float cmp = F.cmax[k][0][cs];
      const float cmq = pair ? F.cmax[k][1][cs] : kNegInf;
      RowNorm np, nq;
      np.M = F.norm[k][0];
      np.invS = F.norm[k][1];
      np.lg = A.lg;
      nq.M = pair ? F.norm[k][2] : kNegInf;
      nq.invS = pair ? F.norm[k][3] : 0.f;
      nq.lg = A.lg;
      s_k = k;
      s_cs = cs;
      s_resid = residual ? 1 : 0;
      s_rem = target - pre;
      s_fac[0] = cmp == kNegInf ? 0.f : cmp * A.lg;
      s_fac[1] = cmq == kNegInf ? 0.f : cmq * A.lg;
      s_fac[2] = np.factor(cmp);
      s_fac[3] = nq.factor(cmq);
    }
  }
  __syncthreads();
  // ---- the draw: waves 0-3 scan chunk cs in ascending vocabulary order, in
  // passes of 4096 entries (thread t of a pass holds 16 consecutive entries);
  // every wave reaches every barrier, only waves 0-3 work between them
  const int k = s_k;
  {
    constexpr int kPerT = 16;
    constexpr int kPass = 256 * kPerT;
    const bool residual = s_resid != 0;
    const float rp = s_fac[0], rq = s_fac[1], fp = s_fac[2], fq = s_fac[3];
    const bool filt = A.thr != nullptr;
    const float thr_p = filt ? A.thr[((size_t)b * G1 + k) * 2] : kNegInf;
    const float thr_q = filt && k < gam ? A.thr[((size_t)b * G1 + k) * 2 + 1] : kNegInf;
    const char* prow = (const char*)A.p + ((size_t)b * A.p_stride + (size_t)k * A.V) * esz;
    const char* qrow = (const char*)A.q + ((size_t)b * A.q_stride + (size_t)k * A.V) * esz;
    const double rem0 = s_rem;
    double carry = 0.0;  // mass of the earlier passes
    int last_tok = -1;
    if (tid == 0) s_tok = -1;
    for (int pass = 0; pass < kChunk / kPass; ++pass) {
      float wt[kPerT];
      double sum = 0.0, incl = 0.0;
      int mine = -1;
      const int x0 = s_cs * kChunk + pass * kPass + tid * kPerT;
      if (w < 4) {
        float zp[kPerT], zq[kPerT];
#pragma unroll
        for (int v = 0; v < kPerT / VEC; ++v) Elt<BF16>::load(prow, min(x0 + v * VEC, A.V - VEC), zp + v * VEC);
        if (residual) {
#pragma unroll
          for (int v = 0; v < kPerT / VEC; ++v) Elt<BF16>::load(qrow, min(x0 + v * VEC, A.V - VEC), zq + v * VEC);
        }
        if (filt) {  // the same top-k / top-p filter the sweep applied
#pragma unroll
          for (int e = 0; e < kPerT; ++e) {
            zp[e] = zp[e] >= thr_p ? zp[e] : kNegInf;
            zq[e] = zq[e] >= thr_q ? zq[e] : kNegInf;
          }
        }
#pragma unroll
        for (int e = 0; e < kPerT; ++e) {
          float wv = 0.f;
          if (x0 + e < A.V) {
#pragma clang fp contract(off)
            const float ep = exp2_hw(fmaf(zp[e], A.lg, -rp));
            if (residual) {
              const float eq = exp2_hw(fmaf(zq[e], A.lg, -rq));
              wv = fmaxf(ep * fp - eq * fq, 0.f);
            } else {
              wv = ep * fp;
            }
          }
          wt[e] = wv;
          sum += (double)wv;
          if (wv > 0.f) mine = x0 + e;
        }
        incl = wave_incl_scan(sum);
        const int lmax = wave_max_i(mine);
        if (lane == 63) s_wt[w] = incl;
        if (lane == 0) s_last[w] = lmax;
      }
      __syncthreads();
      const double total = ((s_wt[0] + s_wt[1]) + s_wt[2]) + s_wt[3];
      const double rem = rem0 - carry;
      for (int i = 0; i < 4; ++i) last_tok = max(last_tok, s_last[i]);
      const bool here = rem < total;  // workgroup-uniform
      if (here && w < 4) {
        double excl_w = 0.0;
        for (int i = 0; i < w; ++i) excl_w += s_wt[i];
        incl += excl_w;
        const unsigned long long h = __ballot(incl > rem && sum > 0.0);
        if (lane == 0) s_hit[w] = h ? __ffsll((long long)h) - 1 : -1;
      }
      __syncthreads();
      if (here) {
        if (w < 4) {
          int hw = -1;
          for (int i = 0; i < 4; ++i)
            if (hw < 0 && s_hit[i] >= 0) hw = i;
          if (hw == w && lane == s_hit[w]) {
            double run = incl - sum;
            int found = -1;
#pragma unroll
            for (int e = 0; e < kPerT; ++e) {
              run += (double)wt[e];
              if (found < 0 && wt[e] > 0.f && run > rem) found = x0 + e;
            }
            s_tok = found >= 0 ? found : mine;
          }
          if (hw < 0 && tid == 0) s_tok = last_tok < 0 ? 0 : last_tok;  // rounding: the pass's last positive entry
        }
        break;  // workgroup-uniform
      }
      carry += total;
    }
    __syncthreads();
    if (tid == 0 && s_tok < 0) s_tok = last_tok < 0 ? 0 : last_tok;  // the target lies past the chunk's total
  }
  __syncthreads();
  if (w != 0) return;
  const int tok = s_tok;
  clear_records(A, b, gam);  // every read of them is done
  // ---- outputs
  int32_t* ot = A.out_tokens + (size_t)b * G1;
  for (int j = lane; j <= A.gmax; j += 64) ot[j] = j < k ? F.x[j] : (j == k ? tok : -1);
  const float nan = __builtin_nanf("");
  for (int j = lane; j < A.gmax; j += 64) {
    const size_t o = (size_t)b * A.gmax + j;
    const bool live = j < gam;
    if (A.accept_prob) A.accept_prob[o] = live ? (float)F.rr[j].a : nan;
    if (A.p_tok) A.p_tok[o] = live ? F.rr[j].p_tok : nan;
    if (A.q_tok) A.q_tok[o] = live ? F.rr[j].q_tok : nan;
    if (A.kl) A.kl[o] = live ? F.rr[j].kl : nan;
    if (A.tv) A.tv[o] = live ? F.rr[j].tv : nan;
  }
  if (lane == 0) {
    A.accept_len[b] = k;
    if (A.new_len) A.new_len[b] = kvl - gam + k;
  }
  finish_rollback(A, b, rb_old, kvl - gam + k);
}

// ============================================================================
// Top-k / top-p thresholds (the logits processors after the temperature)
//
// One workgroup of 1024 threads per live row (verifier rows p_0..p_gamma,
// draft rows q_0..q_{gamma-1}). Logits are compared through an
// order-preserving 32-bit key (-0 counted as +0), and the threshold is found
// by a most-significant-digit radix select: a 12-bit first digit (sign,
// exponent and three mantissa bits, so that logits of one row spread over
// many bins), then 10 + 10 bits for fp32 keys or 4 bits for bf16 keys (whose
// low 16 bits are fixed by the sign). Each level histograms the digit of the
// keys that still match the selected prefix into one LDS histogram shared by
// the waves:
//   top-k: counts; the bin holding the k-th largest key is the one where the
//     count of larger keys first reaches k;
//   top-p: masses 2^((z - M) log2(e)/T) (fp32 terms, fp64 sums) over the keys
//     top-k kept; the bin of the smallest kept logit is the lowest non-empty
//     bin whose mass above (the larger bins plus the mass above the prefix)
//     is below p times the total.
// The first level reads the row from memory. When the selected bin (or, with
// top-p to follow, the bin and every key above it) holds at most kFiltCap
// keys, one more read gathers those keys into LDS and the remaining levels
// (and the whole of top-p after top-k) run on them there; otherwise every
// level reads the row again. Under top-p alone one read before the first
// level finds the row maximum M. The threshold t (a logit value; entries
// below it are removed) goes to thr[b][j][p or q]. Keys are exact, so top-k
// matches the exact rule; top-p decides on fp32 masses, so it may differ from
// exact arithmetic only when the mass above a logit is within ~1e-7 of p.

constexpr int kFiltThreads = 1024;
constexpr int kFiltWaves = kFiltThreads / 64;
constexpr int kFiltBins = 4096;  // the widest digit: 12 bits
constexpr int kFiltCap = 8064;   // candidate keys held in LDS (two workgroups fit a CU's 160 KB)
constexpr int kFiltUnroll = 4;   // row loads in flight per thread

__device__ __forceinline__ uint32_t order_key(float z) {
  const uint32_t u = __float_as_uint(z + 0.f);  // -0 -> +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

struct FiltShared {
  uint32_t cnt[kFiltBins];
  double mass[kFiltBins];
  uint32_t cand[kFiltCap];
  uint32_t wtot_u[kFiltWaves];
  double wtot_d[kFiltWaves];
  uint32_t wmax[kFiltWaves];
  uint32_t n;      // candidates gathered so far
  uint32_t pick;   // selected bin
  uint32_t need;   // top-k: keys still to count inside the selected bin
  uint32_t nge;    // top-k: keys in the selected bin and the bins above it
  uint32_t cpick;  // top-p: keys in the selected bin
  int lowest;      // top-p: the lowest qualifying bin
  double above;    // top-p: mass above the selected prefix
  double total;    // top-p: mass of the keys top-k kept
};

// Digit layout of level l: bits [shift, shift + bits) of the key.
template <bool BF16>
__device__ __forceinline__ int filt_shift(int l) {
  return l == 0 ? 20 : BF16 ? 16 : l == 1 ? 10 : 0;
}
template <bool BF16>
__device__ __forceinline__ int filt_bits(int l) {
  return l == 0 ? 12 : BF16 ? 4 : 10;
}

// Block-wide exclusive prefix sums in thread order (a fixed order).
__device__ __forceinline__ uint32_t filt_excl_scan(FiltShared& F, uint32_t s) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint32_t incl = (uint32_t)wave_incl_scan_i((int)s);
  if (lane == 63) F.wtot_u[w] = incl;
  __syncthreads();
  uint32_t base = 0u;
  for (int i = 0; i < w; ++i) base += F.wtot_u[i];
  return base + incl - s;
}
__device__ __forceinline__ double filt_excl_scan(FiltShared& F, double s, double& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const double incl = wave_incl_scan(s);
  if (lane == 63) F.wtot_d[w] = incl;
  __syncthreads();
  double base = 0.0;
  total = 0.0;
  for (int i = 0; i < kFiltWaves; ++i) {
    if (i == w) base = total;
    total += F.wtot_d[i];
  }
  return base + incl - s;
}

// Histogram pass over the row in memory: digit (key >> shift) & dmask of the
// keys with (key & pmask) == prefix and key >= lo; kmax collects every key.
template <bool BF16, bool MASS>
__device__ void filt_hist_row(FiltShared& F, const char* row, int V, uint32_t prefix, uint32_t pmask, int shift,
                              uint32_t dmask, uint32_t lo, float M, float lg, uint32_t& kmax) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int STEP = kFiltThreads * VEC;
  for (int x0 = (int)threadIdx.x * VEC; x0 < V; x0 += STEP * kFiltUnroll) {
    float z[kFiltUnroll][VEC];
#pragma unroll
    for (int u = 0; u < kFiltUnroll; ++u)
      if (x0 + u * STEP < V) Elt<BF16>::load(row, x0 + u * STEP, z[u]);
#pragma unroll
    for (int u = 0; u < kFiltUnroll; ++u) {
      if (x0 + u * STEP >= V) break;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t key = order_key(z[u][i]);
        kmax = max(kmax, key);
        if ((key & pmask) == prefix && key >= lo) {
          const uint32_t d = (key >> shift) & dmask;
          atomicAdd(&F.cnt[d], 1u);
          if (MASS) atomicAdd(&F.mass[d], (double)exp2_hw((z[u][i] - M) * lg));
        }
      }
    }
  }
}

// The same over the n candidate keys in LDS.
template <bool MASS>
__device__ void filt_hist_cand(FiltShared& F, int n, uint32_t prefix, uint32_t pmask, int shift, uint32_t dmask,
                               uint32_t lo, float M, float lg) {
  for (int i = threadIdx.x; i < n; i += kFiltThreads) {
    const uint32_t key = F.cand[i];
    if ((key & pmask) == prefix && key >= lo) {
      const uint32_t d = (key >> shift) & dmask;
      atomicAdd(&F.cnt[d], 1u);
      if (MASS) atomicAdd(&F.mass[d], (double)exp2_hw((key_value(key) - M) * lg));
    }
  }
}

// Gathers the row's keys in [klo, khi] into F.cand (F.n counts them; the
// caller has checked that they fit).
template <bool BF16>
__device__ void filt_gather_row(FiltShared& F, const char* row, int V, uint32_t klo, uint32_t khi) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int STEP = kFiltThreads * VEC;
  for (int x0 = (int)threadIdx.x * VEC; x0 < V; x0 += STEP * kFiltUnroll) {
    float z[kFiltUnroll][VEC];
#pragma unroll
    for (int u = 0; u < kFiltUnroll; ++u)
      if (x0 + u * STEP < V) Elt<BF16>::load(row, x0 + u * STEP, z[u]);
#pragma unroll
    for (int u = 0; u < kFiltUnroll; ++u) {
      if (x0 + u * STEP >= V) break;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        const uint32_t key = order_key(z[u][i]);
        if (key >= klo && key <= khi) {
          const uint32_t slot = atomicAdd(&F.n, 1u);
          if (slot < (uint32_t)kFiltCap) F.cand[slot] = key;
        }
      }
    }
  }
}

// Thread t owns bins nb-1-t*per down to nb-t*per-per (descending order).
struct FiltOwn {
  int per, own, hi;
  __device__ explicit FiltOwn(int nb) {
    per = nb > kFiltThreads ? nb / kFiltThreads : 1;
    own = (int)threadIdx.x * per < nb ? per : 0;
    hi = nb - 1 - (int)threadIdx.x * per;
  }
};

// top-k: the bin holding the need-th largest key of the histogram.
__device__ void filt_select_count(FiltShared& F, int nb, uint32_t need) {
  const FiltOwn o(nb);
  uint32_t c[4], s = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    c[i] = i < o.own ? F.cnt[o.hi - i] : 0u;
    s += c[i];
  }
  uint32_t run = filt_excl_scan(F, s);  // keys in the higher bins
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (i < o.own && run < need && need <= run + c[i]) {
      F.pick = (uint32_t)(o.hi - i);
      F.need = need - run;
      F.nge = run + c[i];
    }
    run += c[i];
  }
  __syncthreads();
}

// top-p: the lowest non-empty bin whose mass above is below p times the
// total (the total is this histogram's at the first level).
__device__ void filt_select_mass(FiltShared& F, int nb, float top_p, bool first) {
  const FiltOwn o(nb);
  const double above = F.above;
  uint32_t c[4];
  double ms[4], s = 0.0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    c[i] = i < o.own ? F.cnt[o.hi - i] : 0u;
    ms[i] = i < o.own ? F.mass[o.hi - i] : 0.0;
    s += ms[i];
  }
  double all;
  double run = above + filt_excl_scan(F, s, all);  // mass above this thread's first bin
  const double total = first ? all : F.total;
  const double bar = (double)top_p * total;
  int low = -1;
  double low_above = 0.0;
  uint32_t low_cnt = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (i < o.own && c[i] > 0u && run < bar) {
      low = o.hi - i;
      low_above = run;
      low_cnt = c[i];
    }
    run += ms[i];
  }
  if (low >= 0) atomicMin(&F.lowest, low);
  __syncthreads();
  if (low >= 0 && low == F.lowest) {
    F.pick = (uint32_t)low;
    F.above = low_above;
    F.cpick = low_cnt;
  }
  if (first && threadIdx.x == 0) F.total = total;
  __syncthreads();
}

template <bool BF16>
__global__ void __launch_bounds__(kFiltThreads)
accept_filter_kernel(Args A, int top_k, float top_p) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int kLevels = BF16 ? 2 : 3;
  __shared__ FiltShared F;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per_seq = 2 * A.gmax + 1;  // p rows 0..gmax, then q rows 0..gmax-1
  const int b = (int)blockIdx.x / per_seq, r = (int)blockIdx.x % per_seq;
  const bool is_q = r > A.gmax;
  const int j = is_q ? r - (A.gmax + 1) : r;
  const int gam = A.gamma[b];
  if (gam < 0 || gam > A.gmax || (is_q ? j >= gam : j > gam)) return;  // not a live row
  const size_t esz = BF16 ? 2 : 4;
  const char* row = is_q ? (const char*)A.q + ((size_t)b * A.q_stride + (size_t)j * A.V) * esz
                         : (const char*)A.p + ((size_t)b * A.p_stride + (size_t)j * A.V) * esz;
  const int V = A.V;

  auto clear = [&](int nb) {
    __syncthreads();  // every thread is done with the previous level's histogram and picks
    for (int i = tid; i < nb; i += kFiltThreads) {
      F.cnt[i] = 0u;
      F.mass[i] = 0.0;
    }
    if (tid == 0) {
      F.pick = 0u;
      F.need = 1u;
      F.nge = 0u;
      F.cpick = 0u;
      F.lowest = INT_MAX;
    }
    __syncthreads();
  };
  // Gathers the keys in [klo, khi] into F.cand; returns their count.
  auto gather = [&](uint32_t klo, uint32_t khi) {
    __syncthreads();  // every thread has read the picks (and is done with F.cand)
    if (tid == 0) F.n = 0u;
    __syncthreads();
    filt_gather_row<BF16>(F, row, V, klo, khi);
    __syncthreads();
    return (int)min(F.n, (uint32_t)kFiltCap);
  };
  int ncand = 0;        // keys in F.cand
  bool cand_ge = false;  // F.cand holds every key >= lo

  // ---- top-k: radix select of the k-th largest key
  uint32_t kmax = 0u;
  uint32_t lo = 0u;  // keys below lo are removed
  bool have_max = false;
  if (top_k > 0) {
    uint32_t prefix = 0u, pmask = 0u, need = (uint32_t)top_k;
    bool in_lds = false;
    for (int l = 0; l < kLevels; ++l) {
      const int sh = filt_shift<BF16>(l), nb = 1 << filt_bits<BF16>(l);
      clear(nb);
      if (in_lds)
        filt_hist_cand<false>(F, ncand, prefix, pmask, sh, (uint32_t)nb - 1u, 0u, 0.f, 0.f);
      else
        filt_hist_row<BF16, false>(F, row, V, prefix, pmask, sh, (uint32_t)nb - 1u, 0u, 0.f, 0.f, kmax);
      __syncthreads();
      filt_select_count(F, nb, need);
      const uint32_t pick = F.pick;
      need = F.need;
      // with top-p to follow, keep every key from this bin up (top-p's input)
      const uint32_t want = top_p < 1.f ? F.nge : F.cnt[pick];
      const uint32_t pbase = prefix | (pick << sh);
      const uint32_t pspan = (1u << sh) - 1u;  // the bits below this digit
      prefix = pbase;
      pmask |= ((uint32_t)nb - 1u) << sh;
      if (l == 0 && want <= (uint32_t)kFiltCap) {
        ncand = gather(pbase, top_p < 1.f ? 0xffffffffu : (pbase | pspan));
        in_lds = true;
        cand_ge = top_p < 1.f;
      }
    }
    if (BF16) prefix |= (prefix & 0x80000000u) ? 0u : 0xffffu;  // the fixed low half of bf16 keys
    lo = prefix;
    have_max = true;
  }

  // ---- top-p over the keys top-k kept
  uint32_t thr_key = lo;
  if (top_p < 1.f) {
    if (!have_max) {  // the row maximum M first
      constexpr int STEP = kFiltThreads * VEC;
      for (int x0 = tid * VEC; x0 < V; x0 += STEP * kFiltUnroll) {
        float z[kFiltUnroll][VEC];
#pragma unroll
        for (int u = 0; u < kFiltUnroll; ++u)
          if (x0 + u * STEP < V) Elt<BF16>::load(row, x0 + u * STEP, z[u]);
#pragma unroll
        for (int u = 0; u < kFiltUnroll; ++u) {
          if (x0 + u * STEP >= V) break;
#pragma unroll
          for (int i = 0; i < VEC; ++i) kmax = max(kmax, order_key(z[u][i]));
        }
      }
    }
    const uint32_t wm = (uint32_t)wave_max_i((int)(kmax ^ 0x80000000u)) ^ 0x80000000u;  // unsigned max
    if (lane == 0) F.wmax[w] = wm;
    if (tid == 0) F.above = 0.0;
    __syncthreads();
    uint32_t m = 0u;
    for (int i = 0; i < kFiltWaves; ++i) m = max(m, F.wmax[i]);
    const float M = key_value(m);
    uint32_t prefix = 0u, pmask = 0u;
    bool in_lds = cand_ge;
    for (int l = 0; l < kLevels; ++l) {
      const int sh = filt_shift<BF16>(l), nb = 1 << filt_bits<BF16>(l);
      clear(nb);
      uint32_t dummy = 0u;
      if (in_lds)
        filt_hist_cand<true>(F, ncand, prefix, pmask, sh, (uint32_t)nb - 1u, lo, M, A.lg);
      else
        filt_hist_row<BF16, true>(F, row, V, prefix, pmask, sh, (uint32_t)nb - 1u, lo, M, A.lg, dummy);
      __syncthreads();
      filt_select_mass(F, nb, top_p, l == 0);
      const uint32_t pick = F.pick, cpick = F.cpick;
      const uint32_t pbase = prefix | (pick << sh);
      const uint32_t pspan = (1u << sh) - 1u;
      prefix = pbase;
      pmask |= ((uint32_t)nb - 1u) << sh;
      if (l == 0 && !in_lds && cpick <= (uint32_t)kFiltCap) {
        ncand = gather(max(pbase, lo), pbase | pspan);
        in_lds = true;
      }
    }
    if (BF16) prefix |= (prefix & 0x80000000u) ? 0u : 0xffffu;
    thr_key = prefix;
  }
  if (tid == 0) A.thr[((size_t)b * (A.gmax + 1) + j) * 2 + (is_q ? 1 : 0)] = key_value(thr_key);
}

// Greedy finish kernel: one workgroup per sequence, one wave per live row.
// A row's argmax is the lowest index holding the largest of its chunk maxima;
// draft x_j is accepted iff it is argmax p_j, the extra token is argmax p_k,
// and the outputs are the one-hot values (a_j, p(x), q(x) in {0, 1}; TV_j 0
// or 1 and KL_j 0 or +infinity as the two argmaxes agree or not).
__global__ void __launch_bounds__(1024)
accept_finish_greedy_kernel(Args A) {
  __shared__ int s_x[kMaxRows], s_ap[kMaxRows];
  __shared__ RowRes s_rr[kMaxRows];
  __shared__ uint32_t s_bad;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int nw = blockDim.x >> 6;
  const int G1 = A.gmax + 1;
  const int nslot = (A.nc + 63) / 64;
  const int gam = A.gamma[b];
  if (tid == 0) s_bad = 0;
  if (tid < A.gmax) s_x[tid] = A.drafts[(size_t)b * A.gmax + tid];
  const int kvl = A.kv_len ? A.kv_len[b] : 0;
  const int rb_old = A.rb_kv ? A.rb_kv[b] : 0;
  if (gam < 0 || gam > A.gmax) {
    if (w == 0) {
      write_invalid(A, b, SR_ST_GAMMA);
      finish_rollback(A, b, rb_old, kvl);
    }
    return;  // the sweep touched no row of this sequence
  }
  __syncthreads();
  if (tid <= gam) {
    uint32_t bad = 0;
    if (tid < gam && (s_x[tid] < 0 || s_x[tid] >= A.V)) bad |= SR_ST_TOKEN;
    if (tid == 0 && A.kv_len && kvl < gam + 1) bad |= SR_ST_KVLEN;
    if (bad) atomicOr(&s_bad, bad);
  }
  for (int j = w; j <= gam; j += nw) {
    const bool pair = j < gam;
    RowRecs R;
    load_row(A, b * G1 + j, pair, R);
    float mp = kNegInf, mq = kNegInf;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      mp = fmaxf(mp, R.mp[i]);
      mq = fmaxf(mq, R.mq[i]);
    }
    mp = wave_max(mp);
    int ap = INT_MAX, aq = INT_MAX;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      const int cc = lane * nslot + i;
      if (i < nslot && cc < A.nc && R.mp[i] == mp) ap = min(ap, (int)R.sp[i]);
    }
    ap = wave_min_i(ap);
    if (pair) {
      mq = wave_max(mq);
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        const int cc = lane * nslot + i;
        if (i < nslot && cc < A.nc && R.mq[i] == mq) aq = min(aq, (int)R.sq[i]);
      }
      aq = wave_min_i(aq);
    }
    if (lane == 0) {
      s_ap[j] = ap;
      if (pair) {
        const int x = s_x[j];
        const float hit_p = x == ap ? 1.f : 0.f, hit_q = x == aq ? 1.f : 0.f;
        s_rr[j] = RowRes{(double)hit_p, hit_p, hit_q, ap == aq ? 0.f : __builtin_inff(), ap == aq ? 0.f : 1.f};
      }
    }
  }
  __syncthreads();
  if (w != 0) return;
  if (s_bad) {
    clear_records(A, b, gam);
    write_invalid(A, b, s_bad);
    finish_rollback(A, b, rb_old, kvl);
    return;
  }
  const unsigned long long rmask = __ballot(lane < gam && s_x[lane < gam ? lane : 0] != s_ap[lane < gam ? lane : 0]);
  const int k = rmask ? (__ffsll((long long)rmask) - 1) : gam;
  const int tok = s_ap[k];
  clear_records(A, b, gam);
  int32_t* ot = A.out_tokens + (size_t)b * G1;
  for (int j = lane; j <= A.gmax; j += 64) ot[j] = j < k ? s_x[j] : (j == k ? tok : -1);
  const float nan = __builtin_nanf("");
  for (int j = lane; j < A.gmax; j += 64) {
    const size_t o = (size_t)b * A.gmax + j;
    const bool live = j < gam;
    if (A.accept_prob) A.accept_prob[o] = live ? (float)s_rr[j].a : nan;
    if (A.p_tok) A.p_tok[o] = live ? s_rr[j].p_tok : nan;
    if (A.q_tok) A.q_tok[o] = live ? s_rr[j].q_tok : nan;
    if (A.kl) A.kl[o] = live ? s_rr[j].kl : nan;
    if (A.tv) A.tv[o] = live ? s_rr[j].tv : nan;
  }
  if (lane == 0) {
    A.accept_len[b] = k;
    if (A.new_len) A.new_len[b] = kvl - gam + k;
  }
  finish_rollback(A, b, rb_old, kvl - gam + k);
}

// Entries per lane per chunk.
constexpr int kEf32 = 16;
constexpr int kEbf16 = 32;

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct Layout {
  size_t stats, tvabs, xlogit, thr, total;
};

Layout layout(int B, int gamma_max, int n_chunks) {
  const size_t rows = (size_t)B * (gamma_max + 1);
  Layout L;
  L.stats = 0;
  L.tvabs = align256(rows * n_chunks * kRecBytes);
  L.xlogit = L.tvabs + align256(rows * n_chunks * sizeof(double));
  L.thr = L.xlogit + align256(rows * 2 * sizeof(float));
  L.total = L.thr + align256(rows * 2 * sizeof(float));
  return L;
}

template <bool BF16>
const void* sweep_fn() {
  return (const void*)accept_sweep_kernel<BF16, BF16 ? kEbf16 : kEf32>;
}

int resident_per_cu(const void* fn, size_t lds) {
  int per_cu = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, lds) != hipSuccess || per_cu < 1)
    per_cu = 1;
  return per_cu;
}

}  // namespace

int accept_plan(int B, int gamma_max, int V, int dtype, AcceptPlan* plan) {
  const bool bf16 = dtype == SR_BF16;
  plan->chunk = kThreads * (bf16 ? kEbf16 : kEf32);
  plan->n_chunks = (V + plan->chunk - 1) / plan->chunk;
  if (plan->n_chunks > kMaxChunks) return SR_EUNSUPPORTED;
  const int Bl = B < kMaxSeqs ? B : kMaxSeqs;
  if ((size_t)Bl * (gamma_max + 1) * plan->n_chunks * kRecBytes >= 0x7fffffffu) return SR_EUNSUPPORTED;
  plan->workspace_bytes = layout(B, gamma_max, plan->n_chunks).total;
  const int cus = device_cu_count();
  if (cus <= 0) return SR_ELAUNCH;
  const long max_tasks = (long)Bl * (gamma_max + 1) * plan->n_chunks;
  // persistent grid: every workgroup resident at once, a multiple of the
  // chunks per row, and no more than the largest possible task count
  const long cap = (long)cus * resident_per_cu(bf16 ? sweep_fn<true>() : sweep_fn<false>(), Bl * sizeof(int));
  long grid = cap / plan->n_chunks * plan->n_chunks;
  if (grid == 0) grid = cap;
  if (grid > max_tasks) grid = max_tasks;
  plan->grid = (int)grid;
  return SR_OK;
}

int launch_accept(const void* p_logits, int64_t p_stride, const void* q_logits, int64_t q_stride,
                  int dtype, const int32_t* drafts, const int32_t* gamma, const float* u_acc,
                  const float* u_res, const int32_t* kv_len, int32_t* accept_len,
                  int32_t* out_tokens, int32_t* new_len, float* accept_prob, float* p_tok,
                  float* q_tok, float* kl, float* tv, int B, int gamma_max, int V, float temperature,
                  int top_k, float top_p, const AcceptRollback* rollback, void* workspace,
                  const AcceptPlan& plan, int32_t* status, hipStream_t stream) {
  const Layout L = layout(B, gamma_max, plan.n_chunks);
  const bool greedy = temperature == 0.f;
  const int G1 = gamma_max + 1;
  const size_t esz = dtype == SR_BF16 ? 2 : 4;
  char* ws = (char*)workspace;
  const int nw = G1 < 4 ? 4 : (G1 < 16 ? G1 : 16);  // the draw uses waves 0-3
  // sequences in launches of at most kMaxSeqs (the sweep's row table)
  for (int b0 = 0; b0 < B; b0 += kMaxSeqs) {
    const int Bl = B - b0 < kMaxSeqs ? B - b0 : kMaxSeqs;
    Args A;
    A.p = (const char*)p_logits + (size_t)b0 * p_stride * esz;
    A.p_stride = p_stride;
    A.q = q_logits ? (const char*)q_logits + (size_t)b0 * q_stride * esz : nullptr;
    A.q_stride = q_stride;
    A.drafts = drafts ? drafts + (size_t)b0 * gamma_max : nullptr;
    A.gamma = gamma + b0;
    A.u_acc = u_acc ? u_acc + (size_t)b0 * gamma_max : nullptr;
    A.u_res = u_res ? u_res + (size_t)b0 * G1 : nullptr;
    A.kv_len = kv_len ? kv_len + b0 : nullptr;
    A.accept_len = accept_len + b0;
    A.out_tokens = out_tokens + (size_t)b0 * G1;
    A.new_len = new_len ? new_len + b0 : nullptr;
    A.accept_prob = accept_prob ? accept_prob + (size_t)b0 * gamma_max : nullptr;
    A.p_tok = p_tok ? p_tok + (size_t)b0 * gamma_max : nullptr;
    A.q_tok = q_tok ? q_tok + (size_t)b0 * gamma_max : nullptr;
    A.kl = kl ? kl + (size_t)b0 * gamma_max : nullptr;
    A.tv = tv ? tv + (size_t)b0 * gamma_max : nullptr;
    A.B = Bl;
    A.gmax = gamma_max;
    A.V = V;
    A.nc = plan.n_chunks;
    A.stats = (u32x4*)(ws + L.stats) + (size_t)b0 * G1 * plan.n_chunks * 2;
    A.tvabs = (double*)(ws + L.tvabs) + (size_t)b0 * G1 * plan.n_chunks;
    A.xlogit = (float*)(ws + L.xlogit) + (size_t)b0 * G1 * 2;
    A.status = status;
    // top-k / top-p only under sampling (greedy keeps the argmax anyway)
    const int k_eff = top_k > 0 && top_k < V ? top_k : 0;
    const float p_eff = top_p < 1.f ? top_p : 1.f;
    const bool filt = !greedy && (k_eff > 0 || p_eff < 1.f);
    A.thr = filt ? (float*)(ws + L.thr) + (size_t)b0 * G1 * 2 : nullptr;
    A.rb_kv = rollback ? rollback->kv_len + b0 : nullptr;
    A.rb_mask = rollback && rollback->mask ? rollback->mask + (size_t)b0 * rollback->L_cap : nullptr;
    A.rb_phys = rollback ? rollback->phys_len : nullptr;
    A.rb_lcap = rollback ? rollback->L_cap : 0;
    A.rb_reset = b0 == 0 ? 1 : 0;
    A.lg = greedy ? 0.f : (float)(1.4426950408889634 / (double)temperature);
    A.inv_t = greedy ? 0.0 : 1.0 / (double)temperature;
    const size_t lds = Bl * sizeof(int);
    if (greedy) {
      if (dtype == SR_BF16)
        hipLaunchKernelGGL((accept_argmax_kernel<true, kEbf16>), dim3(plan.grid), dim3(kThreads), lds, stream, A);
      else
        hipLaunchKernelGGL((accept_argmax_kernel<false, kEf32>), dim3(plan.grid), dim3(kThreads), lds, stream, A);
      if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
      hipLaunchKernelGGL(accept_finish_greedy_kernel, dim3(Bl), dim3(64 * nw), 0, stream, A);
      if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
      continue;
    }
    if (filt) {  // the rows' top-k / top-p thresholds first
      const dim3 grid_f((unsigned)(Bl * (2 * G1 - 1)));
      if (dtype == SR_BF16)
        hipLaunchKernelGGL(accept_filter_kernel<true>, grid_f, dim3(kFiltThreads), 0, stream, A, k_eff, p_eff);
      else
        hipLaunchKernelGGL(accept_filter_kernel<false>, grid_f, dim3(kFiltThreads), 0, stream, A, k_eff, p_eff);
      if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
    }
    if (dtype == SR_BF16)
      hipLaunchKernelGGL((accept_sweep_kernel<true, kEbf16>), dim3(plan.grid), dim3(kThreads), lds, stream, A);
    else
      hipLaunchKernelGGL((accept_sweep_kernel<false, kEf32>), dim3(plan.grid), dim3(kThreads), lds, stream, A);
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
    if (dtype == SR_BF16)
      hipLaunchKernelGGL((accept_finish_kernel<true, kEbf16>), dim3(Bl), dim3(64 * nw), 0, stream, A);
    else
      hipLaunchKernelGGL((accept_finish_kernel<false, kEf32>), dim3(Bl), dim3(64 * nw), 0, stream, A);
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  }
  return SR_OK;
}

}  // namespace sr
