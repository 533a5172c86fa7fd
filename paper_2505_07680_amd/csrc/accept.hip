// Accept-and-diverge for gfx950: speculative accept/reject with residual
// resampling and the bonus token (Section 2.2 steps 3-4, probabilistic
// acceptance), plus per-position total variation distance (Eq. 5) and KL
// divergence, in one sweep over the verifier and draft logits.
//
// Decomposition. A "row" is one (sequence b, position j) pair: for j < gamma_b
// the verifier row p_j together with the draft row q_j, for j = gamma_b the
// verifier row alone (it feeds the bonus token). Each row is cut into chunks
// of 8192 vocabulary entries, one chunk per workgroup, and each of the
// workgroup's four waves owns 2048 contiguous entries (32 per lane, loaded
// with coalesced 16-byte loads and kept in registers).
//
// Single sweep. TV and the residual max(0, p - q) need both rows' log-
// normalisers, which depend on the whole row. Every wave therefore
//   1. computes its span's (max, sum of exp) for p and q and its share of
//      sum p (z_p - z_q) (the KL numerator), publishes them, and waits at a
//      per-row counter until every wave of the row has published;
//   2. merges all partials of the row (in a fixed order, in fp64, so every wave
//      gets bit-identical log-normalisers) and finishes TV and the residual mass
//      of its span from the values still in registers.
// The last wave to finish a row computes the row's TV, KL, p(x), q(x) and
// acceptance probability; the last row of a sequence to finish runs the
// sequence epilogue: the accept chain, and one token drawn by CDF inversion.
// The inversion locates the 2048-entry span that holds the target from the
// per-span residual (or p) masses and re-reads only that span, scanning it in
// fp64 in ascending vocabulary order.
//
// The grid is persistent and launched cooperatively, so all workgroups are
// co-resident and the per-row wait always completes; a wait is still bounded
// (SR_ST_TIMEOUT) so the kernel always drains. Counters live in the caller's
// workspace and are reset by the kernel that used them.

#include <math.h>

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kE = 32;                  // entries per lane per row
constexpr int kChunk = kThreads * kE;   // entries per workgroup task
constexpr int kSpan = 64 * kE;          // contiguous entries per wave
constexpr uint32_t kSpinLimit = 1u << 22;

struct WavePart {
  float mp, sp, mq, sq, kl, tv, res, pad;
};

struct RowRes {
  double lp, lq, a;
  int32_t ok;
  int32_t pad;
};

template <bool BF16>
struct Elt;

template <>
struct Elt<false> {
  static constexpr int VEC = 4;
  __device__ static void load(const void* row, int idx, float* o) {
    const float4 v = *(const float4*)((const float*)row + idx);
    o[0] = v.x;
    o[1] = v.y;
    o[2] = v.z;
    o[3] = v.w;
  }
  __device__ static float one(const void* row, int idx) { return ((const float*)row)[idx]; }
};

template <>
struct Elt<true> {
  static constexpr int VEC = 8;
  __device__ static void load(const void* row, int idx, float* o) {
    const uint4 u = *(const uint4*)((const uint16_t*)row + idx);
    o[0] = bf16_lo(u.x);
    o[1] = bf16_hi(u.x);
    o[2] = bf16_lo(u.y);
    o[3] = bf16_hi(u.y);
    o[4] = bf16_lo(u.z);
    o[5] = bf16_hi(u.z);
    o[6] = bf16_lo(u.w);
    o[7] = bf16_hi(u.w);
  }
  __device__ static float one(const void* row, int idx) {
    return __uint_as_float((uint32_t)((const uint16_t*)row)[idx] << 16);
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
  int B, gmax, V, n_chunks;
  WavePart* parts;   // [rows][n_chunks * kWaves]
  RowRes* rowres;    // [rows]
  uint32_t* cnt1;    // [rows] waves past pass 1
  uint32_t* cnt2;    // [rows] waves done with the row
  uint32_t* cnt_seq; // [B] rows done
  int32_t* status;
};

__device__ __forceinline__ bool wait_count(const uint32_t* c, uint32_t target) {
  uint32_t it = 0;
  while (atomic_load_agent(c) < target) {
    __builtin_amdgcn_s_sleep(2);
    if (++it > kSpinLimit) return false;
  }
  return true;
}

// (max, sum) merge in fp64 of the partials of one row, identical in every wave.
template <int FIELD_M, int FIELD_S>
__device__ double row_lse(const WavePart* parts, int n) {
  const int lane = threadIdx.x & 63;
  double m = -INFINITY, s = 0.0;
  for (int i = lane; i < n; i += 64) {
    const float* f = (const float*)&parts[i];
    const double m2 = f[FIELD_M], s2 = f[FIELD_S];
    const double M = fmax(m, m2);
    if (M != -INFINITY) {
      s = s * exp(m - M) + s2 * exp(m2 - M);
      m = M;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const double m2 = __shfl_xor(m, off, 64);
    const double s2 = __shfl_xor(s, off, 64);
    const double M = fmax(m, m2);
    if (M != -INFINITY) {
      s = s * exp(m - M) + s2 * exp(m2 - M);
      m = M;
    }
  }
  return m + log(s);
}

template <bool BF16>
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

// Weight of vocabulary entry x of the sampling row, in fp64.
template <bool BF16>
__device__ __forceinline__ double sample_weight(const void* prow, const void* qrow, int x,
                                                double lp, double lq, bool residual) {
  const double pz = exp((double)Elt<BF16>::one(prow, x) - lp);
  if (!residual) return pz;
  const double qz = exp((double)Elt<BF16>::one(qrow, x) - lq);
  return fmax(0.0, pz - qz);
}

// Sequence epilogue: accept chain, token draw, outputs. Run by one wave.
template <bool BF16>
__device__ void sequence_epilogue(const Args& A, int b) {
  const int lane = threadIdx.x & 63;
  const int gam = A.gamma[b];
  const int rows_per_seq = A.gmax + 1;
  // ---- data checks
  uint32_t bad = 0;
  for (int j = lane; j <= gam; j += 64) {
    if (j < gam) {
      const int x = A.drafts[(size_t)b * A.gmax + j];
      if (x < 0 || x >= A.V) bad |= SR_ST_TOKEN;
      const float u = A.u_acc[(size_t)b * A.gmax + j];
      if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
    }
    const float u = A.u_res[(size_t)b * rows_per_seq + j];
    if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
  }
  if (A.kv_len && lane == 0 && A.kv_len[b] < gam + 1) bad |= SR_ST_KVLEN;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) bad |= __shfl_xor(bad, off, 64);
  if (bad) {
    write_invalid<BF16>(A, b, bad);
    return;
  }
  // ---- accept chain
  const RowRes* rr = A.rowres + (size_t)b * rows_per_seq;
  int k = gam;
  for (int j = 0; j < gam; ++j) {
    const double u = (double)A.u_acc[(size_t)b * A.gmax + j];
    if (!(u < rr[j].a)) {
      k = j;
      break;
    }
  }
  // ---- span masses of the sampling row
  const int row = b * rows_per_seq + k;
  const WavePart* parts = A.parts + (size_t)row * A.n_chunks * kWaves;
  const int n_spans = A.n_chunks * kWaves;
  const double lp = rr[k].lp, lq = rr[k].lq;
  bool residual = k < gam;
  double W = 0.0;
  if (residual) {
    for (int s = 0; s < n_spans; ++s) W += (double)parts[s].res;
    if (!(W > 0.0)) residual = false;
  }
  if (!residual) {
    W = 0.0;
    for (int s = 0; s < n_spans; ++s)
      if (parts[s].mp != -INFINITY) W += (double)parts[s].sp * exp((double)parts[s].mp - lp);
  }
  const double target = (double)A.u_res[(size_t)b * rows_per_seq + k] * W;
  // locate the span
  int s0 = 0;
  double prefix = 0.0;
  int last_pos = -1;
  for (int s = 0; s < n_spans; ++s) {
    const double ws = residual ? (double)parts[s].res
                               : (parts[s].mp == -INFINITY ? 0.0 : (double)parts[s].sp * exp((double)parts[s].mp - lp));
    if (ws > 0.0) last_pos = s;
    if (ws > 0.0 && prefix + ws > target) {
      s0 = s;
      break;
    }
    prefix += ws;
    s0 = s + 1;
  }
  if (s0 >= n_spans) {  // rounding left the target past the last mass: take the last span with mass
    s0 = last_pos < 0 ? 0 : last_pos;
    prefix = 0.0;
    for (int s = 0; s < s0; ++s)
      prefix += residual ? (double)parts[s].res
                         : (parts[s].mp == -INFINITY ? 0.0 : (double)parts[s].sp * exp((double)parts[s].mp - lp));
  }
  // ---- scan spans s0.. in fp64, ascending vocabulary order
  const void* prow = (const char*)A.p + ((size_t)b * A.p_stride + (size_t)k * A.V) * (BF16 ? 2 : 4);
  const void* qrow = residual ? (const char*)A.q + ((size_t)b * A.q_stride + (size_t)k * A.V) * (BF16 ? 2 : 4) : nullptr;
  constexpr int VEC = Elt<BF16>::VEC;
  double rem = target - prefix;
  int tok = -1;
  int last_tok = -1;
  for (int s = s0; s < n_spans && tok < 0; ++s) {
    const int base = (s / kWaves) * kChunk + (s % kWaves) * kSpan;
    for (int v = 0; v < kE / VEC && tok < 0; ++v) {
      const int x0 = base + (v * 64 + lane) * VEC;
      double wl[VEC];
      double sum = 0.0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        wl[e] = (x0 + e < A.V) ? sample_weight<BF16>(prow, qrow, x0 + e, lp, lq, residual) : 0.0;
        sum += wl[e];
      }
      // inclusive scan over lanes
      double incl = sum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const double y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
      }
      const double total = __shfl(incl, 63, 64);
      // last entry with positive weight so far (fallback)
      int my_last = -1;
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if (wl[e] > 0.0) my_last = x0 + e;
      int lmax = my_last;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) lmax = max(lmax, __shfl_xor(lmax, off, 64));
      if (lmax >= 0) last_tok = lmax;
      if (rem < total) {
        const unsigned long long hit = __ballot(incl > rem);
        const int hl = __ffsll((long long)hit) - 1;
        int found = -1;
        if (lane == hl) {
          double c = incl - sum;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            c += wl[e];
            if (found < 0 && wl[e] > 0.0 && c > rem) found = x0 + e;
          }
          if (found < 0) found = my_last;
        }
        tok = __shfl(found, hl, 64);
      } else {
        rem -= total;
      }
    }
  }
  if (tok < 0) tok = last_tok < 0 ? 0 : last_tok;
  // ---- outputs
  int32_t* ot = A.out_tokens + (size_t)b * rows_per_seq;
  for (int j = lane; j <= A.gmax; j += 64) {
    int v = -1;
    if (j < k) v = A.drafts[(size_t)b * A.gmax + j];
    else if (j == k) v = tok;
    ot[j] = v;
  }
  const float nan = __builtin_nanf("");
  for (int j = gam + lane; j < A.gmax; j += 64) {
    const size_t o = (size_t)b * A.gmax + j;
    if (A.accept_prob) A.accept_prob[o] = nan;
    if (A.p_tok) A.p_tok[o] = nan;
    if (A.q_tok) A.q_tok[o] = nan;
    if (A.kl) A.kl[o] = nan;
    if (A.tv) A.tv[o] = nan;
  }
  if (lane == 0) {
    A.accept_len[b] = k;
    if (A.new_len) A.new_len[b] = A.kv_len[b] - gam + k;
  }
}

template <bool BF16>
__global__ void __launch_bounds__(kThreads)
accept_kernel(Args A) {
  constexpr int VEC = Elt<BF16>::VEC;
  constexpr int NV = kE / VEC;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int rows_per_seq = A.gmax + 1;
  const long total_tasks = (long)A.B * rows_per_seq * A.n_chunks;
  const int n_spans = A.n_chunks * kWaves;

  for (long task = blockIdx.x; task < total_tasks; task += gridDim.x) {
    const int row = (int)(task / A.n_chunks);
    const int c = (int)(task % A.n_chunks);
    const int b = row / rows_per_seq;
    const int j = row % rows_per_seq;
    const int gam = A.gamma[b];
    if (gam < 0 || gam > A.gmax) {
      if (j == 0 && c == 0 && w == 0) write_invalid<BF16>(A, b, SR_ST_GAMMA);
      continue;
    }
    if (j > gam) continue;
    const bool pair = j < gam;
    const int span = c * kWaves + w;
    const int base = c * kChunk + w * kSpan;
    WavePart* rparts = A.parts + (size_t)row * n_spans;
    const void* prow = (const char*)A.p + ((size_t)b * A.p_stride + (size_t)j * A.V) * (BF16 ? 2 : 4);
    const void* qrow = (const char*)A.q + ((size_t)b * A.q_stride + (size_t)j * A.V) * (BF16 ? 2 : 4);

    // ---- load this wave's span (kept in registers through pass 2)
    float zp[kE], zq[kE];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const int x = base + (v * 64 + lane) * VEC;
      if (x < A.V) {
        Elt<BF16>::load(prow, x, zp + v * VEC);
        if (pair) Elt<BF16>::load(qrow, x, zq + v * VEC);
      } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) zp[v * VEC + e] = kNegInf;
      }
      if (!pair || x >= A.V) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) zq[v * VEC + e] = kNegInf;
      }
    }
    // ---- pass 1: span maxima, exp sums, KL numerator
    float mp = kNegInf, mq = kNegInf;
#pragma unroll
    for (int e = 0; e < kE; ++e) {
      mp = fmaxf(mp, zp[e]);
      mq = fmaxf(mq, zq[e]);
    }
    mp = wave_max(mp);
    mq = wave_max(mq);
    const float rp = mp == kNegInf ? 0.f : mp * kLog2e;
    const float rq = mq == kNegInf ? 0.f : mq * kLog2e;
    float sp = 0.f, sq = 0.f, klp = 0.f;
#pragma unroll
    for (int e = 0; e < kE; ++e) {
      const float ep = exp2f(fmaf(zp[e], kLog2e, -rp));
      const float eq = exp2f(fmaf(zq[e], kLog2e, -rq));
      sp += ep;
      sq += eq;
      klp += ep > 0.f ? ep * (zp[e] - zq[e]) : 0.f;
      zp[e] = ep;  // keep the exponentials for pass 2
      zq[e] = eq;
    }
    sp = wave_sum(sp);
    if (pair) {
      sq = wave_sum(sq);
      klp = wave_sum(klp);
    }
    if (lane == 0) {
      WavePart& wp = rparts[span];
      wp.mp = mp;
      wp.sp = sp;
      wp.mq = mq;
      wp.sq = sq;
      wp.kl = klp;
      wp.tv = 0.f;
      wp.res = 0.f;
    }
    bool ok = true;
    if (pair) {
      // ---- barrier: all waves of the row have published pass 1
      if (lane == 0) atomic_add_release(A.cnt1 + row, 1u);
      ok = wait_count(A.cnt1 + row, (uint32_t)n_spans);
      fence_acquire_agent();
      const double Lp = row_lse<0, 1>(rparts, n_spans);
      const double Lq = row_lse<2, 3>(rparts, n_spans);
      // ---- pass 2: TV and residual mass of this span
      const float fp = mp == kNegInf ? 0.f : (float)exp((double)mp - Lp);
      const float fq = mq == kNegInf ? 0.f : (float)exp((double)mq - Lq);
      float tvs = 0.f, res = 0.f;
#pragma unroll
      for (int e = 0; e < kE; ++e) {
        const float d = zp[e] * fp - zq[e] * fq;
        tvs += fabsf(d);
        res += fmaxf(d, 0.f);
      }
      tvs = wave_sum(tvs);
      res = wave_sum(res);
      if (lane == 0) {
        rparts[span].tv = tvs;
        rparts[span].res = res;
      }
    }
    if (!ok && lane == 0 && A.status) atomicOr(A.status, SR_ST_TIMEOUT);
    // ---- last wave of the row finalises it
    uint32_t prev = 0;
    if (lane == 0) prev = atomic_add_release(A.cnt2 + row, 1u);
    prev = __shfl(prev, 0, 64);
    if (prev != (uint32_t)n_spans - 1) continue;
    fence_acquire_agent();
    {
      const double Lp = row_lse<0, 1>(rparts, n_spans);
      double Lq = 0.0, tvd = 0.0, kld = 0.0;
      if (pair) {
        Lq = row_lse<2, 3>(rparts, n_spans);
        for (int i = lane; i < n_spans; i += 64) {
          tvd += (double)rparts[i].tv;
          if (rparts[i].mp != -INFINITY) kld += (double)rparts[i].kl * exp((double)rparts[i].mp - Lp);
        }
        tvd = 0.5 * wave_sum_d(tvd);
        kld = wave_sum_d(kld) - (Lp - Lq);
      }
      if (lane == 0) {
        RowRes& r = A.rowres[row];
        r.lp = Lp;
        r.lq = Lq;
        r.a = 1.0;
        if (pair) {
          const int x = A.drafts[(size_t)b * A.gmax + j];
          const size_t o = (size_t)b * A.gmax + j;
          double pt = __builtin_nan(""), qt = __builtin_nan(""), a = __builtin_nan("");
          if (x >= 0 && x < A.V) {
            const double lpx = (double)Elt<BF16>::one(prow, x) - Lp;
            const double lqx = (double)Elt<BF16>::one(qrow, x) - Lq;
            pt = exp(lpx);
            qt = exp(lqx);
            a = (lqx == -INFINITY || lpx >= lqx) ? 1.0 : exp(lpx - lqx);
          }
          r.a = a;
          if (A.accept_prob) A.accept_prob[o] = (float)a;
          if (A.p_tok) A.p_tok[o] = (float)pt;
          if (A.q_tok) A.q_tok[o] = (float)qt;
          if (A.kl) A.kl[o] = (float)kld;
          if (A.tv) A.tv[o] = (float)tvd;
        }
        __hip_atomic_store(A.cnt1 + row, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(A.cnt2 + row, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    // ---- last row of the sequence runs the epilogue
    if (lane == 0) prev = atomic_add_release(A.cnt_seq + b, 1u);
    prev = __shfl(prev, 0, 64);
    if (prev != (uint32_t)gam) continue;
    fence_acquire_agent();
    sequence_epilogue<BF16>(A, b);
    if (lane == 0) __hip_atomic_store(A.cnt_seq + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct Layout {
  size_t parts, rowres, cnt1, cnt2, cnt_seq, total;
};

Layout layout(int B, int gamma_max, int n_chunks) {
  const size_t rows = (size_t)B * (gamma_max + 1);
  Layout L;
  L.parts = 0;
  L.rowres = L.parts + align256(rows * n_chunks * kWaves * sizeof(WavePart));
  L.cnt1 = L.rowres + align256(rows * sizeof(RowRes));
  L.cnt2 = L.cnt1 + align256(rows * sizeof(uint32_t));
  L.cnt_seq = L.cnt2 + align256(rows * sizeof(uint32_t));
  L.total = L.cnt_seq + align256((size_t)B * sizeof(uint32_t));
  return L;
}

}  // namespace

int accept_plan(int B, int gamma_max, int V, int dtype, AcceptPlan* plan) {
  plan->chunk = kChunk;
  plan->n_chunks = (V + kChunk - 1) / kChunk;
  plan->workspace_bytes = layout(B, gamma_max, plan->n_chunks).total;
  const int cus = device_cu_count();
  if (cus <= 0) return SR_ELAUNCH;
  int per_cu = 0;
  const void* fn = dtype == SR_BF16 ? (const void*)accept_kernel<true> : (const void*)accept_kernel<false>;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, 0) != hipSuccess || per_cu < 1)
    return SR_ELAUNCH;
  const long tasks = (long)B * (gamma_max + 1) * plan->n_chunks;
  long grid = (long)cus * per_cu;
  if (grid > tasks) grid = tasks;
  grid = grid / plan->n_chunks * plan->n_chunks;
  if (grid < plan->n_chunks) return SR_EUNSUPPORTED;  // a row would not fit on the device at once
  plan->grid = (int)grid;
  return SR_OK;
}

int launch_accept(const void* p_logits, int64_t p_stride, const void* q_logits, int64_t q_stride,
                  int dtype, const int32_t* drafts, const int32_t* gamma, const float* u_acc,
                  const float* u_res, const int32_t* kv_len, int32_t* accept_len,
                  int32_t* out_tokens, int32_t* new_len, float* accept_prob, float* p_tok,
                  float* q_tok, float* kl, float* tv, int B, int gamma_max, int V,
                  void* workspace, const AcceptPlan& plan, int32_t* status, hipStream_t stream) {
  const Layout L = layout(B, gamma_max, plan.n_chunks);
  char* ws = (char*)workspace;
  Args A;
  A.p = p_logits;
  A.p_stride = p_stride;
  A.q = q_logits;
  A.q_stride = q_stride;
  A.drafts = drafts;
  A.gamma = gamma;
  A.u_acc = u_acc;
  A.u_res = u_res;
  A.kv_len = kv_len;
  A.accept_len = accept_len;
  A.out_tokens = out_tokens;
  A.new_len = new_len;
  A.accept_prob = accept_prob;
  A.p_tok = p_tok;
  A.q_tok = q_tok;
  A.kl = kl;
  A.tv = tv;
  A.B = B;
  A.gmax = gamma_max;
  A.V = V;
  A.n_chunks = plan.n_chunks;
  A.parts = (WavePart*)(ws + L.parts);
  A.rowres = (RowRes*)(ws + L.rowres);
  A.cnt1 = (uint32_t*)(ws + L.cnt1);
  A.cnt2 = (uint32_t*)(ws + L.cnt2);
  A.cnt_seq = (uint32_t*)(ws + L.cnt_seq);
  A.status = status;
  void* args[] = {&A};
  const void* fn = dtype == SR_BF16 ? (const void*)accept_kernel<true> : (const void*)accept_kernel<false>;
  const hipError_t e = hipLaunchCooperativeKernel(fn, dim3(plan.grid), dim3(kThreads), args, 0, stream);
  return e == hipSuccess ? SR_OK : SR_ELAUNCH;
}

}  // namespace sr
