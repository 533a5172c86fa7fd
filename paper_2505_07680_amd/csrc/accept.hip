// Accept-and-diverge for gfx950: speculative accept/reject with residual
// resampling and the bonus token (Section 2.2 steps 3-4, probabilistic
// acceptance), plus per-position total variation distance (Eq. 5) and KL
// divergence, with one sweep over the verifier and draft logits.
//
// Decomposition. A "row" is one (sequence b, position j) pair: for j < gamma_b
// the verifier row p_j together with the draft row q_j, for j = gamma_b the
// verifier row alone (it feeds the bonus token). Each row is cut into chunks
// of 256*E vocabulary entries, one chunk per workgroup task, and each of the
// workgroup's four waves owns 64*E contiguous entries (E per lane, loaded with
// coalesced 16-byte loads and kept in registers): a "span".
//
// Sweep kernel (the single pass over HBM). TV and the residual max(0, p - q)
// need both rows' log-normalisers, which depend on the whole row, so every
// wave
//   1. computes its span's (max, sum of exp) for p and q and its share of
//      sum p (z_p - z_q) (the KL numerator) and publishes them;
//   2. once every span of the row has published, merges the partials (fixed
//      order, fp64 sums, so every wave gets bit-identical log-normalisers)
//      and finishes TV and the residual mass of its span from the values still
//      in registers.
// Partials are written with device-coherent stores; once a workgroup's
// stores have completed it bumps the row's counter (one atomic per
// workgroup), and a single lane polls that counter, so waiting costs no
// memory traffic beyond one word and no cache maintenance is needed. The
// sweep launches one workgroup per (row, chunk) task, in row-major order.
//
// Finish kernel (one workgroup per sequence, one wave per row). With every
// partial in memory it computes each row's TV, KL, p(x), q(x) and acceptance
// probability, runs the accept chain, and draws one token by CDF inversion:
// the wave holding the sampling row finds the span that contains the target
// from its per-span residual (or p) masses with a prefix scan, re-reads only
// that span and scans it in fp64 in ascending vocabulary order. It also
// resets the sweep's row counters for the next call.
//
// A workgroup waits only for the other workgroups of its own row, which have
// neighbouring indices: workgroups are dispatched in index order, so the
// earlier rows never wait on later ones and the rows complete in order as
// slots free up (a row needs only its own chunks resident at once). Waits are
// still bounded (SR_ST_TIMEOUT) so the kernel always drains.

#include <math.h>

#include "sr_internal.h"

namespace sr {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxSpans = 256;  // spans per row handled by the wave-parallel merges
constexpr int kMaxRows = SPECROUTER_MAX_GAMMA + 1;
constexpr int kSpanSlots = kMaxSpans / 64;
constexpr uint32_t kSpinLimit = 1u << 22;

// Per-span partial record.
struct SpanRec {
  float mp, sp, mq, sq, kl, tv, res, pad;
};

struct RowLogits {  // p and q logits of the row's draft token
  float zp, zq;
};

typedef float floatx8 __attribute__((ext_vector_type(8)));

template <bool BF16>
struct Elt;

template <>
struct Elt<false> {
  static constexpr int VEC = 4;
  typedef floatx4 Vec;
  __device__ static Vec load(const void* row, int idx) { return *(const floatx4*)((const float*)row + idx); }
  __device__ static float one(const void* row, int idx) { return ((const float*)row)[idx]; }
};

template <>
struct Elt<true> {
  static constexpr int VEC = 8;
  typedef floatx8 Vec;
  __device__ static Vec load(const void* row, int idx) {
    const u32x4 u = *(const u32x4*)((const uint16_t*)row + idx);
    Vec o;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = bf16_lo(u[i]);
      o[2 * i + 1] = bf16_hi(u[i]);
    }
    return o;
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
  int B, gmax, V, n_chunks, chunk, span;
  SpanRec* recs;      // [rows][spans]
  RowLogits* rowx;    // [rows]
  uint32_t* cnt;      // [rows] workgroups whose pass-1 partials are complete
  int32_t* status;
};

// Merge (max, sum) pairs held lane-wise (up to kSpanSlots per lane) into the
// row's natural-log normaliser; fixed order, fp64 sum.
__device__ __forceinline__ double merge_lse(const float (&m)[kSpanSlots], const float (&s)[kSpanSlots], int nslot) {
  float ml = kNegInf;
#pragma unroll
  for (int i = 0; i < kSpanSlots; ++i)
    if (i < nslot) ml = fmaxf(ml, m[i]);
  const float M = wave_max(ml);
  double acc = 0.0;
#pragma unroll
  for (int i = 0; i < kSpanSlots; ++i)
    if (i < nslot && m[i] != kNegInf) acc += (double)s[i] * exp((double)m[i] - (double)M);
  return (double)M + log(wave_sum_d(acc));
}

// ============================================================================
// Sweep kernel

struct Task {
  int row, span, base, j;
  bool exists, live, pair;
  const void* prow;
  const void* qrow;
};

template <bool BF16>
__device__ __forceinline__ Task make_task(const Args& A, long task, long total, int w) {
  Task t;
  t.exists = task < total;
  t.live = false;
  t.pair = false;
  if (!t.exists) return t;
  const int G1 = A.gmax + 1;
  t.row = (int)(task / A.n_chunks);
  const int c = (int)(task % A.n_chunks);
  const int b = t.row / G1;
  t.j = t.row % G1;
  const int gam = A.gamma[b];
  t.live = gam >= 0 && gam <= A.gmax && t.j <= gam;
  t.pair = t.live && t.j < gam;
  t.span = c * kWaves + w;
  t.base = c * A.chunk + w * A.span;
  const size_t esz = BF16 ? 2 : 4;
  t.prow = (const char*)A.p + ((size_t)b * A.p_stride + (size_t)t.j * A.V) * esz;
  t.qrow = (const char*)A.q + ((size_t)b * A.q_stride + (size_t)t.j * A.V) * esz;
  return t;
}

template <bool BF16, int E>
__device__ __forceinline__ void load_span(const Args& A, const Task& t, float (&zp)[E], float (&zq)[E]) {
  typedef Elt<BF16> L;
  constexpr int VEC = L::VEC;
  const int lane = threadIdx.x & 63;
  if (!t.live) return;
#pragma unroll
  for (int v = 0; v < E / VEC; ++v) {
    const int x = t.base + (v * 64 + lane) * VEC;
    const bool in = x < A.V;
    typename L::Vec pv, qv;
    pv = kNegInf;
    qv = kNegInf;
    if (in) pv = L::load(t.prow, x);
    if (in && t.pair) qv = L::load(t.qrow, x);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      zp[v * VEC + e] = pv[e];
      zq[v * VEC + e] = qv[e];
    }
  }
}

// Pass 1: span maxima, exponentials (in place), sums and KL numerator; publish.
template <bool BF16, int E>
__device__ __forceinline__ void pass1(const Args& A, const Task& t, float (&zp)[E], float (&zq)[E], float& mp,
                                      float& mq) {
  const int lane = threadIdx.x & 63;
  if (!t.live) return;
  mp = kNegInf;
  mq = kNegInf;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    mp = fmaxf(mp, zp[e]);
    mq = fmaxf(mq, zq[e]);
  }
  mp = wave_max(mp);
  if (t.pair) mq = wave_max(mq);
  const float rp = mp == kNegInf ? 0.f : mp * kLog2e;
  const float rq = mq == kNegInf ? 0.f : mq * kLog2e;
  float sp = 0.f, sq = 0.f, klp = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const float ep = exp2f(fmaf(zp[e], kLog2e, -rp));
    sp += ep;
    if (t.pair) {
      const float eq = exp2f(fmaf(zq[e], kLog2e, -rq));
      sq += eq;
      klp += ep > 0.f ? ep * (zp[e] - zq[e]) : 0.f;
      zq[e] = eq;
    }
    zp[e] = ep;
  }
  sp = wave_sum(sp);
  if (t.pair) {
    sq = wave_sum(sq);
    klp = wave_sum(klp);
  }
  SpanRec* rec = A.recs + (size_t)t.row * A.n_chunks * kWaves + t.span;
  if (lane < 5) {
    const float val = lane == 0 ? mp : lane == 1 ? sp : lane == 2 ? mq : lane == 3 ? sq : klp;
    st_dev(&rec->mp + lane, val);
  }
  if (t.pair && t.span == 0 && lane == 0) {
    // the draft token's logits, for the acceptance probability
    const int b = t.row / (A.gmax + 1);
    const int x = A.drafts[(size_t)b * A.gmax + t.j];
    if (x >= 0 && x < A.V) A.rowx[t.row] = RowLogits{Elt<BF16>::one(t.prow, x), Elt<BF16>::one(t.qrow, x)};
  }
}

// Pass 2 (pair rows, after the row's counter is complete): merge, TV and
// residual mass of this span.
template <int E>
__device__ __forceinline__ void pass2(const Args& A, const Task& t, const float (&zp)[E], const float (&zq)[E],
                                      float mp, float mq) {
  const int lane = threadIdx.x & 63;
  const int n_spans = A.n_chunks * kWaves;
  const int nslot = (n_spans + 63) / 64;
  const SpanRec* rr = A.recs + (size_t)t.row * n_spans;
  float m1[kSpanSlots], s1[kSpanSlots], m2[kSpanSlots], s2[kSpanSlots];
#pragma unroll
  for (int i = 0; i < kSpanSlots; ++i) {
    const int s = lane * nslot + i;  // lane-major blocks: same merge order as the finish kernel
    const bool in = i < nslot && s < n_spans;
    m1[i] = in ? ld_dev(&rr[s].mp) : kNegInf;
    s1[i] = in ? ld_dev(&rr[s].sp) : 0.f;
    m2[i] = in ? ld_dev(&rr[s].mq) : kNegInf;
    s2[i] = in ? ld_dev(&rr[s].sq) : 0.f;
  }
  const double Lp = merge_lse(m1, s1, nslot);
  const double Lq = merge_lse(m2, s2, nslot);
  const float fp = mp == kNegInf ? 0.f : (float)exp((double)mp - Lp);
  const float fq = mq == kNegInf ? 0.f : (float)exp((double)mq - Lq);
  float tvs = 0.f, res = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    // separately rounded products (no fused multiply-add), so identical p and
    // q rows give exactly zero
#pragma clang fp contract(off)
    const float d = zp[e] * fp - zq[e] * fq;
    tvs += fabsf(d);
    res += fmaxf(d, 0.f);
  }
  tvs = wave_sum(tvs);
  res = wave_sum(res);
  SpanRec* rec = A.recs + (size_t)t.row * n_spans + t.span;
  if (lane < 2) (&rec->tv)[lane] = lane == 0 ? tvs : res;  // read only after the sweep
}

template <bool BF16, int E>
__global__ void __launch_bounds__(kThreads)
accept_sweep_kernel(Args A) {
  __shared__ uint32_t s_ok;
  const int w = threadIdx.x >> 6;
  const long total = (long)A.B * (A.gmax + 1) * A.n_chunks;
  const Task t = make_task<BF16>(A, blockIdx.x, total, w);
  if (!t.live) return;  // workgroup-uniform
  float zp[E], zq[E];
  float mp = kNegInf, mq = kNegInf;
  load_span<BF16, E>(A, t, zp, zq);
  pass1<BF16, E>(A, t, zp, zq, mp, mq);
  if (!t.pair) return;
  // ---- wait until every chunk of the row has published pass 1
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t* c = A.cnt + t.row;
    __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t ok = 0;
    for (uint32_t it = 0; it <= kSpinLimit; ++it) {
      if (ld_dev(c) >= (uint32_t)A.n_chunks) {
        ok = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    if (!ok && A.status) atomicOr(A.status, SR_ST_TIMEOUT);
    s_ok = ok;
  }
  __syncthreads();
  pass2<E>(A, t, zp, zq, mp, mq);
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

// Wave-wide inclusive prefix sum (fp64).
__device__ __forceinline__ double wave_incl_scan(double x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const double y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  return x;
}

struct RowRes {
  double a;
  float p_tok, q_tok, kl, tv;
};

// Draw one token from the row the wave holds. mass[i] is the mass of span
// lane*nslot + i (spans in lane-major blocks so the prefix is a lane scan).
template <bool BF16>
__device__ int draw_token(const Args& A, int b, int k, bool residual, double lp, double lq,
                          const double (&mass)[kSpanSlots], int n_spans) {
  constexpr int VEC = Elt<BF16>::VEC;
  const int lane = threadIdx.x & 63;
  const int nslot = (n_spans + 63) / 64;
  const int G1 = A.gmax + 1;
  double my = 0.0;
  int my_last = -1;
#pragma unroll
  for (int i = 0; i < kSpanSlots; ++i) {
    if (i < nslot) {
      my += mass[i];
      if (mass[i] > 0.0) my_last = lane * nslot + i;
    }
  }
  const double incl = wave_incl_scan(my);
  const double W = __shfl(incl, 63, 64);
  const double target = (double)A.u_res[(size_t)b * G1 + k] * W;
  int last_span = my_last;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) last_span = max(last_span, __shfl_xor(last_span, off, 64));
  int s0 = -1;
  double prefix = 0.0;
  const unsigned long long hit = __ballot(incl > target && my > 0.0);
  if (hit) {
    const int hl = __ffsll((long long)hit) - 1;
    double c = incl - my;
    int found = -1;
    double pre = 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i) {
      if (i < nslot && found < 0 && mass[i] > 0.0 && c + mass[i] > target) {
        found = lane * nslot + i;
        pre = c;
      }
      if (i < nslot) c += mass[i];
    }
    s0 = __shfl(found, hl, 64);
    prefix = __shfl(pre, hl, 64);
  }
  if (s0 < 0) {  // rounding put the target past the total: the last span with mass
    s0 = max(last_span, 0);
    double pre = 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i)
      if (i < nslot && lane * nslot + i < s0) pre += mass[i];
    prefix = wave_sum_d(pre);
  }
  // scan spans s0.. in fp64, ascending vocabulary order
  const size_t esz = BF16 ? 2 : 4;
  const void* prow = (const char*)A.p + ((size_t)b * A.p_stride + (size_t)k * A.V) * esz;
  const void* qrow = residual ? (const char*)A.q + ((size_t)b * A.q_stride + (size_t)k * A.V) * esz : nullptr;
  const int E = A.span / 64;
  double rem = target - prefix;
  int tok = -1;
  int last_tok = -1;
  for (int s = s0; s < n_spans && tok < 0; ++s) {
    const int base = (s / kWaves) * A.chunk + (s % kWaves) * A.span;
    for (int v = 0; v < E / VEC && tok < 0; ++v) {
      const int x0 = base + (v * 64 + lane) * VEC;
      double wl[VEC];
      double sum = 0.0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        double wt = 0.0;
        if (x0 + e < A.V) {
          wt = exp((double)Elt<BF16>::one(prow, x0 + e) - lp);
          if (residual) wt = fmax(0.0, wt - exp((double)Elt<BF16>::one(qrow, x0 + e) - lq));
        }
        wl[e] = wt;
        sum += wt;
      }
      const double inc = wave_incl_scan(sum);
      const double total = __shfl(inc, 63, 64);
      int mine = -1;
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if (wl[e] > 0.0) mine = x0 + e;
      int lmax = mine;
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) lmax = max(lmax, __shfl_xor(lmax, off, 64));
      if (lmax >= 0) last_tok = lmax;
      if (rem < total) {
        const unsigned long long h = __ballot(inc > rem);
        const int hl = __ffsll((long long)h) - 1;
        int found = -1;
        if (lane == hl) {
          double c = inc - sum;
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            c += wl[e];
            if (found < 0 && wl[e] > 0.0 && c > rem) found = x0 + e;
          }
          if (found < 0) found = mine;
        }
        tok = __shfl(found, hl, 64);
      } else {
        rem -= total;
      }
    }
  }
  if (tok < 0) tok = last_tok < 0 ? 0 : last_tok;
  return tok;
}

template <bool BF16>
__global__ void __launch_bounds__(1024)
accept_finish_kernel(Args A) {
  __shared__ RowRes rr[kMaxRows];
  __shared__ uint32_t s_bad;
  const int b = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int nw = blockDim.x >> 6;
  const int G1 = A.gmax + 1;
  const int n_spans = A.n_chunks * kWaves;
  const int nslot = (n_spans + 63) / 64;
  const int gam = A.gamma[b];
  if (gam < 0 || gam > A.gmax) {
    if (w == 0) write_invalid(A, b, SR_ST_GAMMA);
    return;  // the sweep touched no row of this sequence
  }
  if (threadIdx.x == 0) s_bad = 0;
  __syncthreads();
  // ---- data checks
  uint32_t bad = 0;
  for (int j = threadIdx.x; j <= gam; j += blockDim.x) {
    if (j < gam) {
      const int x = A.drafts[(size_t)b * A.gmax + j];
      if (x < 0 || x >= A.V) bad |= SR_ST_TOKEN;
      const float u = A.u_acc[(size_t)b * A.gmax + j];
      if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
    }
    const float u = A.u_res[(size_t)b * G1 + j];
    if (!(u >= 0.f && u < 1.f)) bad |= SR_ST_UNIFORM;
  }
  if (threadIdx.x == 0 && A.kv_len && A.kv_len[b] < gam + 1) bad |= SR_ST_KVLEN;
  if (bad) atomicOr(&s_bad, bad);
  // ---- reset the sweep's row counters for the next call
  for (int j = threadIdx.x; j < gam; j += blockDim.x) A.cnt[b * G1 + j] = 0u;
  // ---- finalise rows (one wave per row); spans in lane-major blocks of nslot
  double lp_k = 0.0, lq_k = 0.0;
  double mass[kSpanSlots];
  int my_row = -1;
  for (int j = w; j <= gam; j += nw) {
    const SpanRec* rp = A.recs + (size_t)(b * G1 + j) * n_spans;
    const bool pair = j < gam;
    float mp[kSpanSlots], sp[kSpanSlots], mq[kSpanSlots], sq[kSpanSlots], klv[kSpanSlots], tvv[kSpanSlots],
        rsv[kSpanSlots];
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i) {
      const int s = lane * nslot + i;
      const bool in = i < nslot && s < n_spans;
      mp[i] = in ? rp[s].mp : kNegInf;
      sp[i] = in ? rp[s].sp : 0.f;
      mq[i] = in && pair ? rp[s].mq : kNegInf;
      sq[i] = in && pair ? rp[s].sq : 0.f;
      klv[i] = in && pair ? rp[s].kl : 0.f;
      tvv[i] = in && pair ? rp[s].tv : 0.f;
      rsv[i] = in && pair ? rp[s].res : 0.f;
    }
    const double Lp = merge_lse(mp, sp, nslot);
    double Lq = 0.0, tvd = 0.0, kld = 0.0;
    if (pair) {
      Lq = merge_lse(mq, sq, nslot);
#pragma unroll
      for (int i = 0; i < kSpanSlots; ++i) {
        tvd += (double)tvv[i];
        if (mp[i] != kNegInf) kld += (double)klv[i] * exp((double)mp[i] - Lp);
      }
      tvd = 0.5 * wave_sum_d(tvd);
      kld = wave_sum_d(kld) - (Lp - Lq);
    }
    // span masses for a possible draw from this row: residual (pair rows) and p
    double res_tot = 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i) res_tot += (double)rsv[i];
    const bool residual = pair && wave_sum_d(res_tot) > 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i)
      mass[i] = residual ? (double)rsv[i] : (mp[i] == kNegInf ? 0.0 : (double)sp[i] * exp((double)mp[i] - Lp));
    my_row = j;
    lp_k = Lp;
    lq_k = Lq;
    if (lane == 0) {
      double a = 1.0, pt = __builtin_nan(""), qt = __builtin_nan("");
      if (pair) {
        const int x = A.drafts[(size_t)b * A.gmax + j];
        a = __builtin_nan("");
        if (x >= 0 && x < A.V) {
          const RowLogits rl = A.rowx[b * G1 + j];
          const double lpx = (double)rl.zp - Lp;
          const double lqx = (double)rl.zq - Lq;
          pt = exp(lpx);
          qt = exp(lqx);
          a = (lqx == -INFINITY || lpx >= lqx) ? 1.0 : exp(lpx - lqx);
        }
      }
      rr[j] = RowRes{a, (float)pt, (float)qt, (float)kld, (float)tvd};
    }
    // a wave keeps the masses of its last row only; more rows than waves
    // (gamma_max = 16) are re-derived below by the owning wave if needed
    if (j + nw <= gam) my_row = -1;
  }
  __syncthreads();
  if (s_bad) {
    if (w == 0) write_invalid(A, b, s_bad);
    return;
  }
  // ---- accept chain: first j with NOT (u_acc < a_j) (every wave computes it)
  bool rej = false;
  if (lane < gam) rej = !((double)A.u_acc[(size_t)b * A.gmax + lane] < rr[lane].a);
  const unsigned long long rmask = __ballot(rej);
  const int k = rmask ? (__ffsll((long long)rmask) - 1) : gam;
  const int owner = k % nw;
  if (w != owner) return;
  if (my_row != k) {
    // the owning wave processed row k before its last row: rebuild its masses
    const SpanRec* rp = A.recs + (size_t)(b * G1 + k) * n_spans;
    const bool pair = k < gam;
    float mp[kSpanSlots], sp[kSpanSlots], mq[kSpanSlots], sq[kSpanSlots], rsv[kSpanSlots];
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i) {
      const int s = lane * nslot + i;
      const bool in = i < nslot && s < n_spans;
      mp[i] = in ? rp[s].mp : kNegInf;
      sp[i] = in ? rp[s].sp : 0.f;
      mq[i] = in && pair ? rp[s].mq : kNegInf;
      sq[i] = in && pair ? rp[s].sq : 0.f;
      rsv[i] = in && pair ? rp[s].res : 0.f;
    }
    lp_k = merge_lse(mp, sp, nslot);
    lq_k = pair ? merge_lse(mq, sq, nslot) : 0.0;
    double res_tot = 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i) res_tot += (double)rsv[i];
    const bool residual = pair && wave_sum_d(res_tot) > 0.0;
#pragma unroll
    for (int i = 0; i < kSpanSlots; ++i)
      mass[i] = residual ? (double)rsv[i] : (mp[i] == kNegInf ? 0.0 : (double)sp[i] * exp((double)mp[i] - lp_k));
  }
  bool residual = false;
  if (k < gam) {
    double tot = 0.0;
    const SpanRec* rp = A.recs + (size_t)(b * G1 + k) * n_spans;
    for (int s = lane; s < n_spans; s += 64) tot += (double)rp[s].res;
    residual = wave_sum_d(tot) > 0.0;
  }
  const int tok = draw_token<BF16>(A, b, k, residual, lp_k, lq_k, mass, n_spans);
  // ---- outputs
  int32_t* ot = A.out_tokens + (size_t)b * G1;
  for (int j = lane; j <= A.gmax; j += 64) ot[j] = j < k ? A.drafts[(size_t)b * A.gmax + j] : (j == k ? tok : -1);
  const float nan = __builtin_nanf("");
  for (int j = lane; j < A.gmax; j += 64) {
    const size_t o = (size_t)b * A.gmax + j;
    const bool live = j < gam;
    if (A.accept_prob) A.accept_prob[o] = live ? (float)rr[j].a : nan;
    if (A.p_tok) A.p_tok[o] = live ? rr[j].p_tok : nan;
    if (A.q_tok) A.q_tok[o] = live ? rr[j].q_tok : nan;
    if (A.kl) A.kl[o] = live ? rr[j].kl : nan;
    if (A.tv) A.tv[o] = live ? rr[j].tv : nan;
  }
  if (lane == 0) {
    A.accept_len[b] = k;
    if (A.new_len) A.new_len[b] = A.kv_len[b] - gam + k;
  }
}

// Entries per lane per row: the sweep's register tile.
constexpr int kE = 16;

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct Layout {
  size_t recs, rowx, cnt, total;
};

Layout layout(int B, int gamma_max, int n_chunks) {
  const size_t rows = (size_t)B * (gamma_max + 1);
  const size_t spans = rows * n_chunks * kWaves;
  Layout L;
  L.recs = 0;
  L.rowx = L.recs + align256(spans * sizeof(SpanRec));
  L.cnt = L.rowx + align256(rows * sizeof(RowLogits));
  L.total = L.cnt + align256(rows * sizeof(uint32_t));
  return L;
}

}  // namespace

int accept_plan(int B, int gamma_max, int V, int dtype, AcceptPlan* plan) {
  plan->chunk = kThreads * kE;
  plan->n_chunks = (V + plan->chunk - 1) / plan->chunk;
  if (plan->n_chunks * kWaves > kMaxSpans) return SR_EUNSUPPORTED;
  plan->workspace_bytes = layout(B, gamma_max, plan->n_chunks).total;
  const long tasks = (long)B * (gamma_max + 1) * plan->n_chunks;
  if (tasks > 0x7fffffffL) return SR_EINVAL;
  const long grid = tasks;
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
  A.chunk = plan.chunk;
  A.span = plan.chunk / kWaves;
  A.recs = (SpanRec*)(ws + L.recs);
  A.rowx = (RowLogits*)(ws + L.rowx);
  A.cnt = (uint32_t*)(ws + L.cnt);
  A.status = status;
  const long tasks = (long)B * (gamma_max + 1) * plan.n_chunks;
  if (dtype == SR_BF16)
    hipLaunchKernelGGL((accept_sweep_kernel<true, kE>), dim3((unsigned)tasks), dim3(kThreads), 0, stream, A);
  else
    hipLaunchKernelGGL((accept_sweep_kernel<false, kE>), dim3((unsigned)tasks), dim3(kThreads), 0, stream, A);
  if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  const int nw = gamma_max + 1 < 16 ? gamma_max + 1 : 16;
  if (dtype == SR_BF16)
    hipLaunchKernelGGL(accept_finish_kernel<true>, dim3(B), dim3(64 * nw), 0, stream, A);
  else
    hipLaunchKernelGGL(accept_finish_kernel<false>, dim3(B), dim3(64 * nw), 0, stream, A);
  return hipGetLastError() == hipSuccess ? SR_OK : SR_ELAUNCH;
}

}  // namespace sr
