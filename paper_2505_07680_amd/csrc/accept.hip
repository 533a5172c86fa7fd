// Accept-and-diverge for gfx950: speculative accept/reject with residual
// resampling and the bonus token (Section 2.2 steps 3-4, probabilistic
// acceptance; Eq. 2), plus per-position total variation distance (Eq. 5) and
// KL divergence, in one launch and one pass over the verifier and draft
// logits.
//
// Rows, chunks, tasks. A live row is one (sequence b, position j <= gamma_b):
// for j < gamma_b the verifier row p_j together with the draft row q_j (a
// "pair row"), for j = gamma_b the verifier row alone (the bonus row). A row
// is cut into chunks of 4096 vocabulary entries; a task is one (row, chunk),
// each of the workgroup's four waves holding 1024 entries of it, 16 entries
// of p (and q) per lane. Workgroup w takes tasks w, w + G, w + 2G, ... over
// the live rows only (a row table built from gamma in LDS).
//
// Row alignment. Loads are 16-byte vectors at 16-byte-aligned addresses. Row j
// starts j*V entries after its sequence's (16-byte-aligned) first row, so it
// sits phi_j = (j*V) mod (entries per 16 bytes) entries past an aligned
// address, the same for p_j and q_j; a row is read from that aligned address
// on, and the entries before its start and past its end are masked out (they
// act as -inf logits). Any V is handled this way.
//
// Sweep launch (one HBM read of every live logit). Workgroup g takes tasks
// g, g + G, g + 2G, ... (G the persistent grid size, what fits on the device
// at once) from an LDS table decoded a window at a time; task k+1's loads are
// issued before task k's first pass, and pair task k's TV sum is formed during
// step k+1:
//  1. first pass: each wave's maxima m over its 1024 entries, integer
//     exponent shifts r = ceil(m log2(e)/T), the exponentials 2^x with
//     x = z log2(e)/T - r (kept in registers until the TV sum; the largest
//     lies in (1/2, 1]), their sums and the KL numerator sum e_p (x_p - x_q);
//     after one barrier a builder wave folds the four waves into the chunk's
//     shifts (the largest; powers of two) and one 32-byte record per chunk,
//     published with device-coherent stores, bit-inverted so that
//     an all-zero word means "not yet written" (naturally aligned 8-byte
//     accesses are single-copy atomic);
//  2. one step later, one wave (rotating over the four) has loaded the row's
//     records (issued before the step's prefetch, so that they return during
//     its first pass) and re-loads them until all are present (for at most
//     about 200 us, then the task gives up, see below); it merges them into
//     the row's normalisers in a fixed order (fp64); each wave forms its own
//     factors f_p = 2^(r_w - r_max)/S_p, f_q likewise, from its own shifts
//     r_w (integers, so 2^(r_w - r_max) is exact; 1/S from the hardware
//     reciprocal estimate and two Newton steps); the lanes then sum |P - Q|
//     over their entries, scaled so that one of the two factors is 1
//     (fma(a, rho, -b) with rho = min/max of the factors), and each wave
//     publishes its part.
// Waiting is bounded: a task whose row is not complete after the time limit
// publishes a "skipped" mark instead of its sum, and the row's finaliser
// recomputes that chunk's sum from memory with the same arithmetic. No
// workgroup ever waits without bound, so the launch needs no co-residency of
// its workgroups, and results do not depend on which workgroup computed what
// (every merge is in a fixed order, every recomputation bit-identical).
//
// Finish launch (one workgroup per sequence): its waves finalise the rows,
// TV_j = 1/2 sum |P - Q|, KL_j, p(x_j), q(x_j) and a_j from the records, the
// sums and the draft token's logits, into LDS; wave 0 then runs the accept
// chain, the draw (chunk masses of the stopping row rebuilt from its records,
// the chunk holding u*W re-read and scanned in ascending vocabulary order with
// its weights computed exactly as in the sweep), the outputs, the rollback,
// and zeroes every workspace word the sequence's rows used, so the workspace
// is all zero again when the call ends. The physical length is written by the
// launch's last finished sequence.
//
// Greedy decoding (T = 0) runs the same launches with chunk argmaxes in place
// of the first pass and no TV step or waiting.
//
// Precision: exponentials in fp32 (relative error ~1e-7; weights below 2^-126
// of their chunk's largest flush to zero), sums in fp32 over a wave's 1024
// entries (a fixed tree: relative error at most ~6e-7 of the sum of
// magnitudes) and in fp64 beyond; the log-normalisers are r_max ln 2 + ln S
// in fp64 and log-probabilities are formed from the exponent arguments
// actually used, so rows with the same filtered distribution give KL = 0 and
// p(x) = q(x) to fp64 rounding. A draw can differ from exact arithmetic only when u*W lies
// within ~1e-7 W of a CDF breakpoint. Logits must satisfy |z|/T < 2^23 (the
// shifts are exact fp32 integers).

#include <limits.h>
#include <math.h>

#include "sr_internal.h"

// v_mul_legacy_f32: 0 * x = 0 for every x (infinities and NaN included).
extern "C" __device__ float sr_fmul_legacy(float, float) __asm("llvm.amdgcn.fmul.legacy");

namespace sr {
namespace {

constexpr int kThreads = 256;  // four waves, one task
constexpr int kWaves = kThreads / 64;
constexpr int kFinWaves = 8;  // waves of a finish workgroup
constexpr int kSlots = 2;               // chunk records per lane in a row merge
constexpr int kMaxChunks = 64 * kSlots; // per row
constexpr int kMaxRows = SPECROUTER_MAX_GAMMA + 1;
constexpr int kMaxSeqs = 4096;               // sequences per launch (row table in LDS)
constexpr int kDeviceCoherent = 16;          // buffer cache-policy operand: sc1
constexpr int kStreamLoad = 2;               // buffer cache-policy operand: non-temporal (the sweep reads each logit once)
constexpr uint64_t kWaitTicks = 20000;       // 200 us of the 100 MHz real-time counter
constexpr double kLn2 = 0.6931471805599453;
constexpr double kSkipped = -1.0;            // a chunk sum left to the finaliser

// ---------------------------------------------------------------------------
// Records

// Per-(row, chunk) record of the first pass.
//   sampling: rp, rq  integer exponent shifts (-inf: the chunk holds no live entry)
//             sp, sq  sums of 2^(z lg - r), kl  sum e_p (x_p - x_q)
//   greedy:   rp, rq  maxima of p and q; sp, sq  the lowest index holding them
//             (INT_MAX: none), kl = 0
struct StatRec {
  float rp, rq;
  double sp, sq, kl;
};
constexpr int kRecBytes = 32;

__device__ __forceinline__ void pack_rec(const StatRec& r, u32x4& w0, u32x4& w1) {
  const uint64_t a = ~((uint64_t)__float_as_uint(r.rp) | ((uint64_t)__float_as_uint(r.rq) << 32));
  const uint64_t b = ~__builtin_bit_cast(uint64_t, r.sp);
  const uint64_t c = ~__builtin_bit_cast(uint64_t, r.sq);
  const uint64_t d = ~__builtin_bit_cast(uint64_t, r.kl);
  w0 = u32x4{(uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32)};
  w1 = u32x4{(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)d, (uint32_t)(d >> 32)};
}
__device__ __forceinline__ bool rec_present(const u32x4& w0, const u32x4& w1) {
  return (w0[0] | w0[1]) != 0u && (w0[2] | w0[3]) != 0u && (w1[0] | w1[1]) != 0u && (w1[2] | w1[3]) != 0u;
}
__device__ __forceinline__ StatRec unpack_rec(const u32x4& w0, const u32x4& w1) {
  StatRec r;
  r.rp = __uint_as_float(~w0[0]);
  r.rq = __uint_as_float(~w0[1]);
  r.sp = __builtin_bit_cast(double, ~((uint64_t)w0[2] | ((uint64_t)w0[3] << 32)));
  r.sq = __builtin_bit_cast(double, ~((uint64_t)w1[0] | ((uint64_t)w1[1] << 32)));
  r.kl = __builtin_bit_cast(double, ~((uint64_t)w1[2] | ((uint64_t)w1[3] << 32)));
  return r;
}

// What a row's finaliser hands to its sequence's finisher.
struct RowOut {
  double a;                    // min(1, p(x)/q(x)); greedy: 1 or 0
  float p_tok, q_tok, kl, tv;
  int argp;                    // greedy: argmax of p
  int pad;
};
static_assert(sizeof(RowOut) == 32, "RowOut is two 16-byte words");

// ---------------------------------------------------------------------------
// Arguments

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
  int B, gmax, V, nc;       // sequences, gamma_max, vocabulary, chunks per row
  float lg;                 // log2(e) / T: softmax(z / T) entries are 2^(z lg - r)
  // workspace
  u32x4* recs;       // [B][gmax+1][nc] records, two 16-byte words each
  double* tva;       // [B][gmax+1][nc][4] each wave's sum |fma(a, rho, -b)| (pair rows), or kSkipped
  float* xlogit;     // [B][gmax+1][4] the draft token's exponent arguments and shifts, p then q (pair rows)
  float* thr;        // [B][gmax+1][2] top-k / top-p thresholds of the p and q rows, or NULL
  uint32_t* fincnt;  // sequences of this launch finished
  int32_t* status;
  // rollback applied as each sequence finishes (rb_kv NULL: none)
  int32_t* rb_kv;            // [B] cache lengths, in/out (this launch's sequences)
  uint8_t* rb_mask;          // [B][L_cap] validity mask, or NULL
  int32_t* rb_phys;          // max over all sequences of the new lengths, or NULL
  const int32_t* rb_kv_all;  // the whole batch's cache lengths (rb_kv - n_before)
  int rb_lcap;
  int n_before;              // sequences of the call handled by earlier launches
};

// Task geometry: each lane holds 16 entries of p (and of q), 32 bytes of
// bf16 or 64 of fp32; a task (chunk) is 4096 entries. (With 32 bf16 entries
// per lane the exponentials kept for the deferred TV sum need more registers
// than three workgroups per CU allow.)
template <bool BF16>
struct Vec {
  static constexpr int N = BF16 ? 8 : 4;  // entries per 16-byte vector
  static constexpr int esz = BF16 ? 2 : 4;
  static constexpr int E = 16;                  // entries per lane per task
  static constexpr int kWaveSpan = 64 * E;      // entries of one wave in a task
  static constexpr int kChunk = kThreads * E;   // entries of a task
};

// A lane's E entries as loaded (E/N 16-byte vectors).
template <bool BF16>
struct Loaded {
  u32x4 v[Vec<BF16>::E / Vec<BF16>::N];
};

template <bool BF16>
__device__ __forceinline__ void widen(const Loaded<BF16>& L, float (&z)[Vec<BF16>::E]) {
  constexpr int kE = Vec<BF16>::E;
  if constexpr (BF16) {
#pragma unroll
    for (int i = 0; i < kE / 8; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        z[i * 8 + 2 * k] = bf16_lo(L.v[i][k]);
        z[i * 8 + 2 * k + 1] = bf16_hi(L.v[i][k]);
      }
  } else {
#pragma unroll
    for (int i = 0; i < kE / 4; ++i)
#pragma unroll
      for (int k = 0; k < 4; ++k) z[i * 4 + k] = __uint_as_float(L.v[i][k]);
  }
}

// Aligned position (entries from the row's aligned start) of a lane's entry e
// in the first-pass layout: vector e / N of the wave, lanes side by side.
template <bool BF16>
__device__ __forceinline__ int lane_pos(int wbase, int lane, int e) {
  constexpr int N = Vec<BF16>::N;
  return wbase + ((e / N) * 64 + lane) * N + e % N;
}

// Entries between row j's aligned start and its first entry.
template <bool BF16>
__device__ __forceinline__ int row_phase(const Args& A, int j) {
  return (int)(((int64_t)j * A.V) % Vec<BF16>::N);
}

// One row of p (and q) as buffer resources over its aligned span.
struct RowSpan {
  __amdgpu_buffer_rsrc_t rp, rq;
  int phi;
};

template <bool BF16>
__device__ __forceinline__ RowSpan row_span(const Args& A, int b, int j, bool with_q) {
  constexpr int N = Vec<BF16>::N, esz = Vec<BF16>::esz;
  RowSpan s;
  s.phi = row_phase<BF16>(A, j);
  // bytes up to the 16-byte boundary after the row's last entry: the last
  // vector is read whole (it never leaves the 16-byte block holding the row's
  // last byte), vectors wholly past it read zero
  const size_t span = (size_t)((s.phi + A.V + N - 1) / N) * 16;
  const char* pr = (const char*)A.p + ((int64_t)b * A.p_stride + (int64_t)j * A.V - s.phi) * esz;
  s.rp = make_rsrc(pr, span);
  const char* qr = with_q ? (const char*)A.q + ((int64_t)b * A.q_stride + (int64_t)j * A.V - s.phi) * esz : pr;
  s.rq = make_rsrc(qr, with_q ? span : 0);
  return s;
}

// Inclusive prefix over sequences of their live-row counts (gamma_b + 1, or 0
// for an invalid gamma), in LDS.
__device__ void build_row_table(const int32_t* gamma, int gmax, int B, int* rows) {
  __shared__ int wsum[kWaves];
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

struct TaskInfo {
  int b, j, c, row, x, gam, phi;
  float thp, thq;  // the row's top-k / top-p thresholds (read only when A.thr is set)
  bool pair, full;
};

// A workgroup's tasks, decoded a window at a time into LDS, one per thread:
// sequence (12 bits), position (5), live-row count (5) and chunk (7) packed in
// one word, the draft token and the row's thresholds. The task loop then
// reads its next task with no division, search or global load.
constexpr int kTab = kThreads;
struct TaskTable {
  int pack[kTab];
  int x[kTab];
  float thp[kTab], thq[kTab];
};

// Tasks k0 .. k0 + kTab - 1 of this workgroup (task blockIdx.x + k * gridDim.x).
__device__ void fill_tasks(const Args& A, const int* rows, long n_tasks, int k0, TaskTable& tab) {
  const int tid = threadIdx.x;
  const long task = blockIdx.x + (long)(k0 + tid) * gridDim.x;
  if (task < n_tasks) {
    const int rank = (int)(task / A.nc), c = (int)(task % A.nc);
    int lo = 0, hi = A.B - 1;  // first sequence whose prefix exceeds rank
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (rows[mid] > rank) hi = mid;
      else lo = mid + 1;
    }
    const int first = lo ? rows[lo - 1] : 0;
    const int j = rank - first, gam = rows[lo] - first - 1;
    const int row = lo * (A.gmax + 1) + j;
    tab.pack[tid] = lo | (j << 12) | (gam << 17) | (c << 22);
    tab.x[tid] = j < gam ? A.drafts[(size_t)lo * A.gmax + j] : -1;
    tab.thp[tid] = A.thr ? A.thr[(size_t)row * 2] : kNegInf;
    tab.thq[tid] = A.thr && j < gam ? A.thr[(size_t)row * 2 + 1] : kNegInf;
  }
  __syncthreads();
}

template <bool BF16>
__device__ __forceinline__ TaskInfo decode_task(const Args& A, const TaskTable& tab, int k) {
  TaskInfo t;
  const int i = k % kTab;
  const int pk = __builtin_amdgcn_readfirstlane(tab.pack[i]);
  t.b = pk & 0xfff;
  t.j = (pk >> 12) & 31;
  t.gam = (pk >> 17) & 31;
  t.c = pk >> 22;
  t.pair = t.j < t.gam;
  t.row = t.b * (A.gmax + 1) + t.j;
  t.phi = row_phase<BF16>(A, t.j);
  constexpr int kChunk = Vec<BF16>::kChunk;
  t.full = t.c * kChunk >= t.phi && (t.c + 1) * kChunk <= t.phi + A.V;
  t.x = __builtin_amdgcn_readfirstlane(tab.x[i]);
  t.thp = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(tab.thp[i])));
  t.thq = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(tab.thq[i])));
  return t;
}

// One task's loads (always the same count). A bonus row's draft resource is
// empty: its loads return zeros without memory traffic.
// With live false the resources are empty too (a prefetch past the last task).
template <bool BF16>
__device__ __forceinline__ void issue_loads(const Args& A, const TaskInfo& t, Loaded<BF16>& lp, Loaded<BF16>& lq,
                                            bool live = true) {
  constexpr int N = Vec<BF16>::N, esz = Vec<BF16>::esz, kE = Vec<BF16>::E;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wbase = t.c * Vec<BF16>::kChunk + w * Vec<BF16>::kWaveSpan;
  RowSpan s = row_span<BF16>(A, t.b, t.j, t.pair);
  if (!live) s.rp = s.rq = make_rsrc(A.p, 0);
#pragma unroll
  for (int i = 0; i < kE / N; ++i)
    lp.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            s.rp, (uint32_t)((wbase + (i * 64 + lane) * N) * esz), 0, kStreamLoad));
#pragma unroll
  for (int i = 0; i < kE / N; ++i)
    lq.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                            s.rq, (uint32_t)((wbase + (i * 64 + lane) * N) * esz), 0, kStreamLoad));
}

// Entries outside the row (before its start or past its end) become -inf.
template <bool BF16>
__device__ __forceinline__ void mask_range(float (&z)[Vec<BF16>::E], int wbase, int phi, int V) {
  constexpr int kE = Vec<BF16>::E;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int e = 0; e < kE; ++e) {
    const int i = lane_pos<BF16>(wbase, lane, e) - phi;
    z[e] = (i >= 0 && i < V) ? z[e] : kNegInf;
  }
}
template <int kE>
__device__ __forceinline__ void mask_below(float (&z)[kE], float t) {
#pragma unroll
  for (int e = 0; e < kE; ++e) z[e] = z[e] >= t ? z[e] : kNegInf;
}

// Pairwise sum of a lane's entries (a fixed tree).
template <int kE>
__device__ __forceinline__ float tree_sum(const float (&v)[kE]) {
  float a[kE];
#pragma unroll
  for (int i = 0; i < kE; ++i) a[i] = v[i];
#pragma unroll
  for (int s = kE / 2; s > 0; s /= 2)
#pragma unroll
    for (int i = 0; i < s; ++i) a[i] += a[i + s];
  return a[0];
}

__device__ __forceinline__ uint32_t rec_off(int row, int nc, int c) {
  return (uint32_t)(((size_t)row * nc + c) * kRecBytes);
}

// ---------------------------------------------------------------------------
// First pass (the workgroup: one task)

// Per-task workgroup state.
// The waves' results of a task's first pass, read by the record's builder
// after one barrier. Two sets, used by alternate tasks: a wave may start the
// next task's first pass (and write its results) while the builder still
// reads this task's, but not the one after (that waits for the next task's
// barrier, which the builder reaches only after its reads).
struct WaveSlots {
  float m[2][kWaves];      // the waves' shifts of p and q (-inf: no entry); greedy: their maxima
  double s[3][kWaves];     // the waves' sums (p, q, KL numerator; greedy: argmax indices in s[0..1])
};

struct TaskShared {
  WaveSlots x[2];          // by task parity
  float rM_p, rM_q;        // the TV step's row normalisers (largest chunk shift, sum)
  double S_p, S_q;
  int ok;                  // the row's records were all present in time
};

// A wave's exponent shifts for p and q (-inf where the wave has no entry).
struct WaveShift {
  float rp, rq;
};

// The draft token's exponent arguments x_p, x_q and its chunk's shifts, for
// the acceptance test (p(x) = 2^x_p 2^(r_c - r_max) / S_p, the kernel's own
// distribution): the lane that holds the token stores them (once per row).
template <bool BF16>
__device__ __forceinline__ void store_xlogit(const Args& A, const TaskInfo& t, int wbase,
                                             const float (&zp)[Vec<BF16>::E], const float (&zq)[Vec<BF16>::E],
                                             float rp, float rq) {
  constexpr int N = Vec<BF16>::N, kE = Vec<BF16>::E, kWaveSpan = Vec<BF16>::kWaveSpan;
  const int lane = threadIdx.x & 63;
  const int xo = t.x + t.phi - wbase;  // aligned offset of x in this wave's entries
  if (t.x < 0 || t.x >= A.V || xo < 0 || xo >= kWaveSpan) return;
  if (lane != (xo % (64 * N)) / N) return;
  const int ex = (xo / (64 * N)) * N + xo % N;
  float vp = 0.f, vq = 0.f;
#pragma unroll
  for (int e = 0; e < kE; ++e)
    if (e == ex) {
      vp = zp[e];
      vq = zq[e];
    }
  float* o = A.xlogit + (size_t)t.row * 4;
  st_dev(o, fmaf(vp, A.lg, -rp));
  st_dev(o + 1, rp);
  st_dev(o + 2, fmaf(vq, A.lg, -rq));
  st_dev(o + 3, rq);
}

__device__ __forceinline__ void store_rec(const __amdgpu_buffer_rsrc_t& rs, uint32_t off, const StatRec& r) {
  u32x4 w0, w1;
  pack_rec(r, w0, w1);
  __builtin_amdgcn_raw_buffer_store_b128(w0, rs, off, 0, kDeviceCoherent);
  __builtin_amdgcn_raw_buffer_store_b128(w1, rs, off + 16, 0, kDeviceCoherent);
}

// Raw logits of one wave's entries, masked: entries outside the row and below
// the row's top-k / top-p threshold become -inf.
template <bool BF16>
__device__ __forceinline__ void masked_logits(const Args& A, const TaskInfo& t, int wbase, const Loaded<BF16>& Lp,
                                              const Loaded<BF16>& Lq, float (&zp)[Vec<BF16>::E],
                                              float (&zq)[Vec<BF16>::E]) {
  widen<BF16>(Lp, zp);
  widen<BF16>(Lq, zq);
  if (!t.full) {
    mask_range<BF16>(zp, wbase, t.phi, A.V);
    mask_range<BF16>(zq, wbase, t.phi, A.V);
  }
  if (A.thr) {  // workgroup-uniform
    mask_below(zp, t.thp);
    if (t.pair) mask_below(zq, t.thq);
  }
}

// Integer exponent shift of a maximum (0 for an empty chunk, whose entries
// are all -inf and give 0 anyway).
__device__ __forceinline__ float shift_of(float m, float lg) { return m == kNegInf ? 0.f : ceilf(m * lg); }

// The exponentials of one wave's entries under shifts rp, rq, their sums and
// the KL numerator (groups of four entries summed as (a0 + a1) + (a2 + a3),
// then a tree over the groups).
template <int kE>
__device__ __forceinline__ void wave_exps(const float (&zp)[kE], const float (&zq)[kE], float lg, float rp, float rq,
                                          bool pair, float (&ep)[kE], float (&eq)[kE], double& sp, double& sq,
                                          double& kl) {
  float gp[kE / 4];
  if (pair) {  // workgroup-uniform
    float gq[kE / 4], gk[kE / 4];
#pragma unroll
    for (int g = 0; g < kE / 4; ++g) {
      float kt[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int e = g * 4 + i;
        const float xp = fmaf(zp[e], lg, -rp);
        const float xq = fmaf(zq[e], lg, -rq);
        ep[e] = exp2_hw(xp);
        eq[e] = exp2_hw(xq);
        kt[i] = sr_fmul_legacy(ep[e], xp - xq);  // 0 where p is -inf, +inf where only q is
      }
      gp[g] = (ep[g * 4] + ep[g * 4 + 1]) + (ep[g * 4 + 2] + ep[g * 4 + 3]);
      gq[g] = (eq[g * 4] + eq[g * 4 + 1]) + (eq[g * 4 + 2] + eq[g * 4 + 3]);
      gk[g] = (kt[0] + kt[1]) + (kt[2] + kt[3]);
    }
    sq = (double)wave_sum(tree_sum(gq));
    kl = (double)wave_sum(tree_sum(gk));
  } else {  // a bonus row: p alone (eq is not read)
#pragma unroll
    for (int g = 0; g < kE / 4; ++g) {
#pragma unroll
      for (int i = 0; i < 4; ++i) ep[g * 4 + i] = exp2_hw(fmaf(zp[g * 4 + i], lg, -rp));
      gp[g] = (ep[g * 4] + ep[g * 4 + 1]) + (ep[g * 4 + 2] + ep[g * 4 + 3]);
    }
    sq = 0.0;
    kl = 0.0;
  }
  sp = (double)wave_sum(tree_sum(gp));
}

// Sampling: each wave's maxima and shifts (its own: no exchange between the
// waves before the exponentials), exponentials (left in ep/eq), sums and KL
// numerator; lane 0 of wave `builder` folds the four waves into the chunk's
// record, in the chunk's shifts (the largest of the waves'; the rescaling
// factors are powers of two). Returns the wave's shifts, which its TV step
// needs.
template <bool BF16>
__device__ __forceinline__ WaveShift first_pass(const Args& A, const TaskInfo& t, const Loaded<BF16>& Lp,
                                                const Loaded<BF16>& Lq, float (&ep)[Vec<BF16>::E],
                                                float (&eq)[Vec<BF16>::E], WaveSlots& sh,
                                                const __amdgpu_buffer_rsrc_t& rs_recs, int builder) {
  constexpr int kE = Vec<BF16>::E;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wbase = t.c * Vec<BF16>::kChunk + w * Vec<BF16>::kWaveSpan;
  float zp[kE], zq[kE];
  masked_logits<BF16>(A, t, wbase, Lp, Lq, zp, zq);
  float mp = kNegInf, mq = kNegInf;
#pragma unroll
  for (int e = 0; e < kE; ++e) {
    mp = fmaxf(mp, zp[e]);
    mq = fmaxf(mq, zq[e]);
  }
  mp = wave_max(mp);
  mq = t.pair ? wave_max(mq) : kNegInf;
  const float rp = shift_of(mp, A.lg), rq = shift_of(mq, A.lg);
  if (t.pair) store_xlogit<BF16>(A, t, wbase, zp, zq, rp, rq);
  double sp, sq, kl;
  wave_exps(zp, zq, A.lg, rp, rq, t.pair, ep, eq, sp, sq, kl);
  WaveShift ws;
  ws.rp = mp == kNegInf ? kNegInf : rp;
  ws.rq = mq == kNegInf ? kNegInf : rq;
  if (lane == 0) {
    sh.m[0][w] = ws.rp;
    sh.m[1][w] = ws.rq;
    sh.s[0][w] = sp;
    sh.s[1][w] = sq;
    sh.s[2][w] = kl;
  }
  __syncthreads();
  if (w == builder && lane == 0) {
    float rpc = kNegInf, rqc = kNegInf;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      rpc = fmaxf(rpc, sh.m[0][i]);
      rqc = fmaxf(rqc, sh.m[1][i]);
    }
    // e in the chunk's shifts = e_w 2^(r_w - r_c); the KL terms' exponent
    // difference gains (r_p,w - r_p,c) - (r_q,w - r_q,c) (0 where q has no
    // entry: those terms are 0 or +inf already)
    StatRec r;
    r.rp = rpc;
    r.rq = rqc;
    r.sp = 0.0;
    r.sq = 0.0;
    r.kl = 0.0;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      const float rpw = sh.m[0][i], rqw = sh.m[1][i];
      if (rpw != kNegInf) {
        const double f = ldexp(1.0, (int)(rpw - rpc));
        const double d = rqw == kNegInf ? 0.0 : (double)(rpw - rpc) - (double)(rqw - rqc);
        r.sp += f * sh.s[0][i];
        r.kl += f * (sh.s[2][i] + d * sh.s[0][i]);
      }
      if (rqw != kNegInf) r.sq += ldexp(1.0, (int)(rqw - rqc)) * sh.s[1][i];
    }
    store_rec(rs_recs, rec_off(t.row, A.nc, t.c), r);
  }
  return ws;
}

// Greedy decoding: the chunk's maxima of p and q and the lowest index holding
// each (lanes scan their entries in ascending index order).
template <bool BF16>
__device__ __forceinline__ void argmax_pass(const Args& A, const TaskInfo& t, const Loaded<BF16>& Lp,
                                            const Loaded<BF16>& Lq, WaveSlots& sh,
                                            const __amdgpu_buffer_rsrc_t& rs_recs) {
  constexpr int kE = Vec<BF16>::E;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wbase = t.c * Vec<BF16>::kChunk + w * Vec<BF16>::kWaveSpan;
  float zp[kE], zq[kE];
  widen<BF16>(Lp, zp);
  widen<BF16>(Lq, zq);
  float bp = kNegInf, bq = kNegInf;
  int ip = INT_MAX, iq = INT_MAX;
#pragma unroll
  for (int e = 0; e < kE; ++e) {
    const int i = lane_pos<BF16>(wbase, lane, e) - t.phi;
    const bool in = t.full || (i >= 0 && i < A.V);
    if (in && (ip == INT_MAX || zp[e] > bp)) {
      bp = zp[e];
      ip = i;
    }
    if (in && (iq == INT_MAX || zq[e] > bq)) {
      bq = zq[e];
      iq = i;
    }
  }
  const float mp = wave_max(bp);
  const int jp = wave_min_i(ip != INT_MAX && bp == mp ? ip : INT_MAX);
  float mq = kNegInf;
  int jq = INT_MAX;
  if (t.pair) {
    mq = wave_max(bq);
    jq = wave_min_i(iq != INT_MAX && bq == mq ? iq : INT_MAX);
  }
  if (lane == 0) {
    sh.m[0][w] = mp;
    sh.m[1][w] = mq;
    sh.s[0][w] = (double)jp;
    sh.s[1][w] = (double)jq;
  }
  __syncthreads();
  if (tid == 0) {
    StatRec r;
    r.rp = kNegInf;
    r.rq = kNegInf;
    int ap = INT_MAX, aq = INT_MAX;
    for (int i = 0; i < kWaves; ++i) {
      r.rp = fmaxf(r.rp, sh.m[0][i]);
      r.rq = fmaxf(r.rq, sh.m[1][i]);
    }
    for (int i = 0; i < kWaves; ++i) {
      if (sh.m[0][i] == r.rp) ap = min(ap, (int)sh.s[0][i]);
      if (sh.m[1][i] == r.rq) aq = min(aq, (int)sh.s[1][i]);
    }
    r.sp = (double)ap;
    r.sq = (double)aq;
    r.kl = 0.0;
    store_rec(rs_recs, rec_off(t.row, A.nc, t.c), r);
  }
}

// ---------------------------------------------------------------------------
// Row merges (one wave; the same code wherever a row is merged, so every
// merge of a row gives the same bits)

// A row's chunk records, lane-wise: chunk lane * kSlots + i in slot i.
struct RowRecs {
  float rp[kSlots], rq[kSlots];
  double sp[kSlots], sq[kSlots], kl[kSlots];
};

// A row's record words as loaded (device-coherent loads), lane-wise.
struct RecWords {
  u32x4 w[kSlots][2];
};

__device__ __forceinline__ void issue_recs(const Args& A, const __amdgpu_buffer_rsrc_t& rs, int row, RecWords& W) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int c = lane * kSlots + i;
    const uint32_t off = rec_off(row, A.nc, c < A.nc ? c : 0);
    W.w[i][0] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, kDeviceCoherent);
    W.w[i][1] = __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16, 0, kDeviceCoherent);
  }
}

// The records from their words; true (wave-uniform) when all are present.
__device__ __forceinline__ bool decode_recs(const Args& A, const RecWords& W, RowRecs& R) {
  const int lane = threadIdx.x & 63;
  bool ok = true;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int c = lane * kSlots + i;
    const bool in = c < A.nc;
    const u32x4 w0 = W.w[i][0], w1 = W.w[i][1];
    ok = ok && (!in || rec_present(w0, w1));
    const StatRec r = unpack_rec(w0, w1);
    R.rp[i] = in ? r.rp : kNegInf;
    R.rq[i] = in ? r.rq : kNegInf;
    R.sp[i] = in ? r.sp : 0.0;
    R.sq[i] = in ? r.sq : 0.0;
    R.kl[i] = in ? r.kl : 0.0;
  }
  return __ballot(!ok) == 0ull;
}

// Loads the records; true (wave-uniform) when all are present.
__device__ __forceinline__ bool load_recs(const Args& A, const __amdgpu_buffer_rsrc_t& rs, int row, RowRecs& R) {
  RecWords W;
  issue_recs(A, rs, row, W);
  return decode_recs(A, W, R);
}

// A distribution's normaliser: the largest shift r_max and
// S = sum_c s_c 2^(r_c - r_max), so that its entries are 2^x 2^(r_c - r_max) / S
// (shifts are integers: 2^(r_c - r_max) is exact).
struct Norm {
  float rM;
  double S;
};

__device__ __forceinline__ double pow2(float r, float rM) {
  return r == kNegInf ? 0.0 : ldexp(1.0, (int)(r - rM));
}

__device__ __forceinline__ Norm merge_norm(const float (&r)[kSlots], const double (&s)[kSlots]) {
  float m = kNegInf;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) m = fmaxf(m, r[i]);
  Norm n;
  n.rM = wave_max(m);
  double acc = 0.0;
  if (n.rM != kNegInf) {
#pragma unroll
    for (int i = 0; i < kSlots; ++i) acc += s[i] * pow2(r[i], n.rM);
  }
  n.S = wave_sum_d(acc);
  return n;
}

// Factor turning a chunk's exponentials into probabilities.
__device__ __forceinline__ double factor(float r, const Norm& n) {
  return (r == kNegInf || !(n.S > 0.0)) ? 0.0 : pow2(r, n.rM) / n.S;
}

// The TV sum of a chunk with factors fp, fq is scale * sum |fma(e_p, rho_p,
// -e_q rho_q)|: the larger factor is scale, and of the two ratios rho = f/scale
// the larger side's is exactly 1 (so rows with equal factors subtract
// exactly, and the product on that side is exact).
struct TvPar {
  double scale;
  float rho_p, rho_q;
};
// 1/s (s > 0) from the hardware estimate and two Newton steps.
__device__ __forceinline__ double recip(double s) {
  double r = __builtin_amdgcn_rcp(s);
  r = fma(r, fma(-s, r, 1.0), r);
  return fma(r, fma(-s, r, 1.0), r);
}
// The factors of a wave with shifts ws against the row normalisers, without a
// division: f = 2^(r_w - r_max)/S, and the smaller side's ratio is
// 2^(k) S_big/S_small with k the difference of the shift offsets.
__device__ __forceinline__ TvPar tv_par(const WaveShift& ws, const Norm& np, const Norm& nq) {
  const bool hp = ws.rp != kNegInf && np.S > 0.0, hq = ws.rq != kNegInf && nq.S > 0.0;
  const double ip = recip(hp ? np.S : 1.0), iq = recip(hq ? nq.S : 1.0);
  const int a = hp ? (int)(ws.rp - np.rM) : 0, b = hq ? (int)(ws.rq - nq.rM) : 0;
  const double fp = hp ? ldexp(ip, a) : 0.0, fq = hq ? ldexp(iq, b) : 0.0;
  const bool both = hp && hq;
  const float rq = both ? (float)ldexp(np.S * iq, b - a) : 0.f;  // f_q/f_p
  const float rp = both ? (float)ldexp(nq.S * ip, a - b) : 0.f;  // f_p/f_q
  const bool pbig = fp >= fq;
  TvPar t;
  t.scale = pbig ? fp : fq;
  t.rho_p = pbig ? (hp ? 1.f : 0.f) : rp;
  t.rho_q = pbig ? rq : 1.f;
  return t;
}
// One entry's scaled difference e_p rho_p - e_q rho_q.
__device__ __forceinline__ float tv_diff(float ep, float eq, float rho_p, float rho_q) {
  return fmaf(ep, rho_p, -(eq * rho_q));
}

// One wave's part of a chunk's TV sum.
template <int kE>
__device__ __forceinline__ double tv_wave(const float (&ep)[kE], const float (&eq)[kE], float rho_p, float rho_q) {
  float g[kE / 4];
#pragma unroll
  for (int k = 0; k < kE / 4; ++k) {
    float d[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) d[i] = fabsf(tv_diff(ep[k * 4 + i], eq[k * 4 + i], rho_p, rho_q));
    g[k] = (d[0] + d[1]) + (d[2] + d[3]);
  }
  return (double)wave_sum(tree_sum(g));
}
// A chunk's TV sum from its waves' parts, in a fixed order.
__device__ __forceinline__ double tv_chunk(const double (&part)[kWaves]) {
  return ((part[0] + part[1]) + part[2]) + part[3];
}

__device__ __forceinline__ float lane_float(float x, int src) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), src));
}

// The polling wave: the row's records from the words of a first attempt (W,
// issued earlier), else re-loaded until all are present (for a bounded
// time); merge them and leave the row's normalisers in LDS.
__device__ __forceinline__ void poll_row(const Args& A, const __amdgpu_buffer_rsrc_t& rs, const TaskInfo& t,
                                         const RecWords& W, TaskShared& sh) {
  const int lane = threadIdx.x & 63;
  RowRecs R;
  bool ok = decode_recs(A, W, R);
  if (!ok) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    for (;;) {
      __builtin_amdgcn_s_sleep(2);
      ok = load_recs(A, rs, t.row, R);
      if (ok || __builtin_amdgcn_s_memrealtime() - t0 > kWaitTicks) break;
    }
  }
  if (ok) {
    const Norm np = merge_norm(R.rp, R.sp);
    const Norm nq = merge_norm(R.rq, R.sq);
    if (lane == 0) {
      sh.rM_p = np.rM;
      sh.S_p = np.S;
      sh.rM_q = nq.rM;
      sh.S_q = nq.S;
    }
  }
  if (lane == 0) sh.ok = ok ? 1 : 0;
}

// A wave's share of a chunk's TV sum, scaled: scale * sum |e_p rho_p - e_q rho_q|
// with the wave's own factors against the row normalisers.
template <int kE>
__device__ __forceinline__ double tv_wave_scaled(const float (&ep)[kE], const float (&eq)[kE], const WaveShift& ws,
                                                 const Norm& np, const Norm& nq) {
  const TvPar par = tv_par(ws, np, nq);
  return par.scale * tv_wave(ep, eq, par.rho_p, par.rho_q);
}

// ---------------------------------------------------------------------------
// Sequence outputs (one wave)

__device__ void write_invalid(const Args& A, int b, uint32_t bits) {
  const int lane = threadIdx.x & 63;
  if (lane == 0) {
    A.accept_len[b] = -1;
    if (A.new_len) A.new_len[b] = A.kv_len[b];
    if (A.status && bits) atomicOr(A.status, (int32_t)bits);
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
// flagged and ignored; otherwise the mask entries [n, old) are cleared and the
// length becomes n = min(old, want). `old` is read when the sequence finishes.
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
    st_dev((uint32_t*)A.rb_kv + b, (uint32_t)n);
    if (st && A.status) atomicOr(A.status, st);
  }
}

// One wave, after its sequences' rollbacks have completed: count them; the
// launch's last finished sequence writes the physical length, the maximum of
// the rolled-back lengths of the whole batch so far (Eq. 9), and resets the
// counter.
__device__ void count_finished(const Args& A, uint32_t n) {
  if (!A.rb_kv || !A.rb_phys || n == 0) return;
  const int lane = threadIdx.x & 63;
  stores_done();
  uint32_t old = 0;
  if (lane == 0) old = __hip_atomic_fetch_add(A.fincnt, n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  old = (uint32_t)__builtin_amdgcn_readfirstlane((int)old);
  if (old + n != (uint32_t)A.B) return;
  int m = INT_MIN;
  for (int b = lane; b < A.n_before + A.B; b += 64) m = max(m, (int)ld_dev((const uint32_t*)A.rb_kv_all + b));
  m = wave_max_i(m);
  if (lane == 0) {
    *A.rb_phys = m;
    st_dev(A.fincnt, 0u);
  }
}

// Zero every workspace word sequence b's rows used, so the workspace is all
// zero again when the call ends: the next call, whatever its shape, lays its
// regions over these bytes, and its polls take any non-zero record word for a
// published one.
__device__ void clear_sequence(const Args& A, int b, int gam) {
  const int lane = threadIdx.x & 63;
  const size_t r0 = (size_t)b * (A.gmax + 1);
  const u32x4 z4 = u32x4{0u, 0u, 0u, 0u};
  // the records with device-coherent stores
  const uint32_t nrec = (uint32_t)((gam + 1) * A.nc * 2);  // 16-byte words
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(A.recs + r0 * A.nc * 2, (size_t)nrec * 16);
  for (uint32_t i = lane; i < nrec; i += 64) __builtin_amdgcn_raw_buffer_store_b128(z4, rs, i * 16u, 0, kDeviceCoherent);
  for (size_t i = lane; i < (size_t)gam * A.nc * kWaves; i += 64) A.tva[r0 * A.nc * kWaves + i] = 0.0;
  for (int i = lane; i < 2 * (gam + 1); i += 64)
    if (A.thr) A.thr[r0 * 2 + i] = 0.f;
  for (int i = lane; i < 4 * gam; i += 64) A.xlogit[r0 * 4 + i] = 0.f;
}

// ---------------------------------------------------------------------------
// The draw (one wave)

// Wave-wide inclusive prefix sum (fp64) in ascending lane order.
__device__ __forceinline__ double wave_incl_scan_d(double x) {
  x = x + dpp_f64<0x111>(x);  // row_shr:1 (lanes without a source read 0)
  x = x + dpp_f64<0x112>(x);  // row_shr:2
  x = x + dpp_f64<0x114>(x);  // row_shr:4
  x = x + dpp_f64<0x118>(x);  // row_shr:8
  const double r0 = lane_value(x, 15), r1 = lane_value(x, 31), r2 = lane_value(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  const double r01 = r0 + r1;
  return x + (row == 0 ? 0.0 : row == 1 ? r0 : row == 2 ? r01 : r01 + r2);
}

// The draw at row k of sequence b: from the residual max(0, p_k - q_k) if
// k < gamma and it has mass, else from p_k; the smallest x with C(x) > u W in
// ascending vocabulary order (the last entry with weight if rounding leaves
// none). Two steps: the row's finaliser finds the chunk holding u W from the
// chunk masses (its records R, normalisers np, nq and chunk TV sums tva) and
// leaves a plan; once the stopping row is known, four waves scan that chunk,
// one pass of 1024 entries each (16 consecutive entries per lane), with its
// weights computed exactly as in the sweep, and combine their sums in pass
// order.
struct DrawPlan {
  double rem;       // the target's offset into the chunk's mass
  double S_p, S_q;  // the row normalisers: each pass's factors come from them
  float rM_p, rM_q, tp, tq;
  int c, resid;
};

template <bool BF16>
__device__ DrawPlan draw_plan(const Args& A, int b, int k, int gam, float u, const RowRecs& R, const Norm& np,
                              const Norm& nq, const double (&tva)[kSlots]) {
  const int lane = threadIdx.x & 63;
  const int row = b * (A.gmax + 1) + k;
  const bool pair = k < gam;
  double mres[kSlots], mp[kSlots];
  double my_res = 0.0;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    const int c = lane * kSlots + i;
    const double fp = factor(R.rp[i], np);
    mp[i] = fp * R.sp[i];
    mres[i] = 0.0;
    if (pair && c < A.nc) {
      const double fq = factor(R.rq[i], nq);
      mres[i] = fmax(0.0, 0.5 * (tva[i] + mp[i] - fq * R.sq[i]));
    }
    my_res += mres[i];
  }
  const bool resid = pair && wave_sum_d(my_res) > 0.0;
  double m[kSlots], my = 0.0;
  int my_last = -1;
#pragma unroll
  for (int i = 0; i < kSlots; ++i) {
    m[i] = resid ? mres[i] : mp[i];
    my += m[i];
    if (m[i] > 0.0) my_last = lane * kSlots + i;
  }
  const double incl = wave_incl_scan_d(my);
  const double W = lane_value(incl, 63);
  const double target = (double)u * W;
  // the first chunk with weight whose end exceeds the target
  int c = -1;
  double pre = 0.0;
  const unsigned long long hit = __ballot(incl > target && my > 0.0);
  if (hit) {
    const int hl = __ffsll((long long)hit) - 1;
    double run = incl - my;
    int found = -1;
    double fpre = 0.0;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      if (found < 0 && m[i] > 0.0 && run + m[i] > target) {
        found = lane * kSlots + i;
        fpre = run;
      }
      run += m[i];
    }
    c = lane_value(found, hl);
    pre = lane_value(fpre, hl);
  } else {  // rounding put the target at the very end: the last chunk with weight
    c = max(wave_max_i(my_last), 0);
    double before = 0.0;
#pragma unroll
    for (int i = 0; i < kSlots; ++i)
      if (lane * kSlots + i < c) before += m[i];
    pre = wave_sum_d(before);
  }
  const double rem = target - pre;
  DrawPlan d;
  d.rem = rem;
  d.rM_p = np.rM;
  d.S_p = np.S;
  d.rM_q = nq.rM;
  d.S_q = nq.S;
  d.resid = resid ? 1 : 0;
  d.c = c;
  d.tp = A.thr ? A.thr[(size_t)row * 2] : kNegInf;
  d.tq = A.thr && resid ? A.thr[(size_t)row * 2 + 1] : kNegInf;
  return d;
}

// One pass of the scan (this wave's quarter of the chunk, which one sweep
// wave held): a lane's weights and the last index among them with weight;
// returns the factor turning the pass's weights into probabilities. The
// pass's shifts are the sweep wave's own (its maxima over the same entries),
// so the weights are the sweep's exponentials.
template <bool BF16>
__device__ __forceinline__ double draw_weights(const Args& A, int b, int k, const DrawPlan& d, int pass,
                                               float (&wt)[Vec<BF16>::E], int& mine) {
  constexpr int N = Vec<BF16>::N, esz = Vec<BF16>::esz, kE = Vec<BF16>::E;
  const int lane = threadIdx.x & 63;
  const RowSpan s = row_span<BF16>(A, b, k, d.resid != 0);
  const int pos0 = d.c * Vec<BF16>::kChunk + pass * Vec<BF16>::kWaveSpan + lane * kE;
  Loaded<BF16> lp, lq;
#pragma unroll
  for (int i = 0; i < kE / N; ++i) {
    const uint32_t off = (uint32_t)((pos0 + i * N) * esz);
    lp.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(s.rp, off, 0, 0));
    lq.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(s.rq, off, 0, 0));
  }
  float zp[kE], zq[kE];
  widen<BF16>(lp, zp);
  widen<BF16>(lq, zq);
  float mp = kNegInf, mq = kNegInf;
#pragma unroll
  for (int e = 0; e < kE; ++e) {
    const int i = pos0 + e - s.phi;
    const bool in = i >= 0 && i < A.V;
    zp[e] = in && zp[e] >= d.tp ? zp[e] : kNegInf;
    zq[e] = in && zq[e] >= d.tq ? zq[e] : kNegInf;
    mp = fmaxf(mp, zp[e]);
    mq = fmaxf(mq, zq[e]);
  }
  mp = wave_max(mp);
  mq = d.resid ? wave_max(mq) : kNegInf;
  const float rp = shift_of(mp, A.lg), rq = shift_of(mq, A.lg);
  const WaveShift ws{mp == kNegInf ? kNegInf : rp, mq == kNegInf ? kNegInf : rq};
  const Norm np{d.rM_p, d.S_p}, nq{d.rM_q, d.S_q};
  const double fp = factor(ws.rp, np);
  const TvPar par = d.resid ? tv_par(ws, np, nq) : TvPar{fp, 1.f, 0.f};
  mine = -1;
#pragma unroll
  for (int e = 0; e < kE; ++e) {
    const int i = pos0 + e - s.phi;
    const float ep = exp2_hw(fmaf(zp[e], A.lg, -rp));
    float wv;
    if (d.resid) {
      const float eq = exp2_hw(fmaf(zq[e], A.lg, -rq));
      wv = fmaxf(tv_diff(ep, eq, par.rho_p, par.rho_q), 0.f);
    } else {
      wv = ep;
    }
    wt[e] = wv;
    if (wv > 0.f) mine = i;
  }
  return d.resid ? par.scale : fp;
}

// Shared state of the scan.
struct DrawShared {
  double tot[kWaves];   // each pass's total (its prefix at lane 63)
  int hit[kWaves];      // the pass holds the target
  int last[kWaves];     // the pass's last index with weight
  int tok;
};

// The four waves (w < 4) scan the chunk of plan d; returns the token (valid in
// waves 0-3 after the call; every wave of the workgroup must call it).
template <bool BF16>
__device__ int draw_scan(const Args& A, int b, int k, const DrawPlan& d, DrawShared& ds) {
  constexpr int kE = Vec<BF16>::E;
  const int lane = threadIdx.x & 63, w = wave_id();
  float wt[kE];
  int mine = -1;
  double lsum = 0.0, pincl = 0.0, scale = 0.0;
  if (w < kWaves) {
    scale = draw_weights<BF16>(A, b, k, d, w, wt, mine);
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < kE; ++e) acc += (double)wt[e];
    lsum = acc * scale;
    pincl = wave_incl_scan_d(lsum);
    const int last = wave_max_i(mine);
    if (lane == 63) ds.tot[w] = pincl;
    if (lane == 0) ds.last[w] = last;
  }
  __syncthreads();
  if (w < kWaves) {
    double carry = 0.0;  // the previous passes' totals, in pass order
    for (int i = 0; i < w; ++i) carry += ds.tot[i];
    const double sincl = carry + pincl;
    const unsigned long long h = __ballot(sincl > d.rem && lsum > 0.0);
    if (lane == 0) ds.hit[w] = h ? 1 : 0;
    if (h) {
      const int pos0 = d.c * Vec<BF16>::kChunk + w * Vec<BF16>::kWaveSpan + lane * kE;
      const int phi = row_phase<BF16>(A, k);
      const int hl = __ffsll((long long)h) - 1;
      double run = sincl - lsum;
      int found = -1;
#pragma unroll
      for (int e = 0; e < kE; ++e) {
        run += (double)wt[e] * scale;
        if (found < 0 && wt[e] > 0.f && run > d.rem) found = pos0 + e - phi;
      }
      const int t = __builtin_amdgcn_readlane(found >= 0 ? found : mine, hl);
      if (lane == 0) ds.last[w] = ~t;  // a hit: its token (bit-inverted), read below
    }
  }
  __syncthreads();
  int tok = -1, last = -1;
  for (int i = 0; i < kWaves; ++i) {
    if (tok < 0 && ds.hit[i]) tok = ~ds.last[i];
    if (!ds.hit[i]) last = max(last, ds.last[i]);
  }
  if (tok < 0) tok = last < 0 ? 0 : last;  // the target lies past the chunk's total (rounding)
  return tok;
}

// ---------------------------------------------------------------------------
// Row finaliser (wave 0 of the workgroup whose task completed the row)

// Recompute the sums of the chunks whose owners gave up waiting, from memory,
// with the owners' arithmetic and layout (one wave takes the four waves'
// entries in turn and combines their parts in the same order: same bits).
template <bool BF16>
__device__ void redo_skipped(const Args& A, int b, int j, const RowRecs& R, const Norm& np, const Norm& nq,
                             double (&tva)[kSlots]) {
  constexpr int N = Vec<BF16>::N, esz = Vec<BF16>::esz, kE = Vec<BF16>::E;
  constexpr int kChunk = Vec<BF16>::kChunk, kWaveSpan = Vec<BF16>::kWaveSpan;
  const int lane = threadIdx.x & 63;
  const RowSpan s = row_span<BF16>(A, b, j, true);
  const int row = b * (A.gmax + 1) + j;
  for (;;) {
    int cl = -1;
#pragma unroll
    for (int i = kSlots - 1; i >= 0; --i)
      if (tva[i] == kSkipped) cl = lane * kSlots + i;
    const unsigned long long pend = __ballot(cl >= 0);
    if (!pend) break;
    const int src = __ffsll((long long)pend) - 1;
    const int c = __builtin_amdgcn_readlane(cl, src);  // the lowest skipped chunk of that lane
    TaskInfo t;
    t.c = c;
    t.row = row;
    t.pair = true;
    t.phi = s.phi;
    t.full = c * kChunk >= s.phi && (c + 1) * kChunk <= s.phi + A.V;
    t.thp = A.thr ? A.thr[(size_t)row * 2] : kNegInf;
    t.thq = A.thr ? A.thr[(size_t)row * 2 + 1] : kNegInf;
    double part[kWaves];
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) {
      const int wbase = c * kChunk + ww * kWaveSpan;
      Loaded<BF16> lp, lq;
#pragma unroll
      for (int i = 0; i < kE / N; ++i) {
        const uint32_t off = (uint32_t)((wbase + (i * 64 + lane) * N) * esz);
        lp.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(s.rp, off, 0, 0));
        lq.v[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(s.rq, off, 0, 0));
      }
      float zp[kE], zq[kE], ep[kE], eq[kE];
      masked_logits<BF16>(A, t, wbase, lp, lq, zp, zq);
      // the owner wave's shifts: its maxima over these entries
      float mp = kNegInf, mq = kNegInf;
#pragma unroll
      for (int e = 0; e < kE; ++e) {
        mp = fmaxf(mp, zp[e]);
        mq = fmaxf(mq, zq[e]);
      }
      mp = wave_max(mp);
      mq = wave_max(mq);
      const float rp = shift_of(mp, A.lg), rq = shift_of(mq, A.lg);
#pragma unroll
      for (int e = 0; e < kE; ++e) {
        ep[e] = exp2_hw(fmaf(zp[e], A.lg, -rp));
        eq[e] = exp2_hw(fmaf(zq[e], A.lg, -rq));
      }
      const WaveShift ws{mp == kNegInf ? kNegInf : rp, mq == kNegInf ? kNegInf : rq};
      part[ww] = tv_wave_scaled(ep, eq, ws, np, nq);
    }
    const double sum = tv_chunk(part);  // the owners' parts, combined as the finaliser combines them
    if (lane == src) {
#pragma unroll
      for (int i = 0; i < kSlots; ++i)
        if (lane * kSlots + i == c) tva[i] = sum;
    }
  }
}

// Row j of sequence b (one wave): its row results, and (sampling) the plan of
// the draw the sequence would make if it stopped at row j, from u_res[j]; the
// finisher uses one of those once the accept chain is known. Every load the
// row needs is issued first, then consumed.
template <bool BF16, bool GREEDY>
__device__ RowOut finalize_row(const Args& A, int b, int j, int gam, const __amdgpu_buffer_rsrc_t& rs_recs,
                               DrawPlan& plan) {
  const int lane = threadIdx.x & 63;
  const int row = b * (A.gmax + 1) + j;
  const bool pair = j < gam;
  RecWords W;
  issue_recs(A, rs_recs, row, W);  // all present: the sweep launch has completed
  double part[kSlots][kWaves];
  float xs[4] = {0.f, 0.f, 0.f, 0.f};
  float u = 0.f;
  if (!GREEDY) {
    if (pair) {
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        const int c = lane * kSlots + i;
        const double* tp = A.tva + ((size_t)row * A.nc + (c < A.nc ? c : 0)) * kWaves;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) part[i][w] = tp[w];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) xs[i] = A.xlogit[(size_t)row * 4 + i];
    }
    u = A.u_res[row];
  }
  const int x = pair ? A.drafts[(size_t)b * A.gmax + j] : -1;
  RowRecs R;
  decode_recs(A, W, R);
  RowOut o;
  o.pad = 0;
  o.argp = -1;
  const bool xin = x >= 0 && x < A.V;
  const float nan = __builtin_nanf("");
  if constexpr (GREEDY) {
    float mp = kNegInf, mq = kNegInf;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      mp = fmaxf(mp, R.rp[i]);
      mq = fmaxf(mq, R.rq[i]);
    }
    mp = wave_max(mp);
    mq = wave_max(mq);
    int ap = INT_MAX, aq = INT_MAX;
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      const bool in = lane * kSlots + i < A.nc;
      if (in && R.rp[i] == mp) ap = min(ap, (int)R.sp[i]);
      if (in && R.rq[i] == mq) aq = min(aq, (int)R.sq[i]);
    }
    ap = wave_min_i(ap);
    aq = wave_min_i(aq);
    o.argp = ap;
    const float hp = x == ap ? 1.f : 0.f, hq = x == aq ? 1.f : 0.f;
    o.a = pair ? (double)hp : 0.0;
    o.p_tok = pair ? hp : nan;
    o.q_tok = pair ? hq : nan;
    o.kl = pair ? (ap == aq ? 0.f : __builtin_inff()) : nan;
    o.tv = pair ? (ap == aq ? 0.f : 1.f) : nan;
  } else {
    const Norm np = merge_norm(R.rp, R.sp);
    Norm nq = Norm{kNegInf, 0.0};
    double tva[kSlots];
#pragma unroll
    for (int i = 0; i < kSlots; ++i) {
      // a chunk's TV sum: its four waves' parts in a fixed order; kSkipped if
      // any part was left to the finaliser; 0 past the row
      bool skipped = false;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) skipped = skipped || part[i][w] == kSkipped;
      tva[i] = lane * kSlots + i >= A.nc ? 0.0 : skipped ? kSkipped : tv_chunk(part[i]);
    }
    o.a = 0.0;
    o.p_tok = o.q_tok = o.kl = o.tv = nan;
    if (pair) {
      nq = merge_norm(R.rq, R.sq);
      redo_skipped<BF16>(A, b, j, R, np, nq, tva);
      // TV = 1/2 sum_c tva_c (the waves' parts come scaled);
      // KL = sum_c f_c (ln2 kl_c + ln2 s_c d_c) - ln(S_p / S_q) sum_c f_c s_c with
      // d_c = (r_c - r_max) - (r'_c - r'_max) (integers): the log-ratio of an
      // entry is ln2 (x_p - x_q) + ln2 d_c - ln(S_p / S_q)
      double tvs = 0.0, klt = 0.0, mass = 0.0;
#pragma unroll
      for (int i = 0; i < kSlots; ++i) {
        const double fp = factor(R.rp[i], np);
        tvs += tva[i];
        if (fp > 0.0) {
          const double d = ((double)R.rp[i] - (double)np.rM) - ((double)R.rq[i] - (double)nq.rM);
          klt += fp * (kLn2 * R.kl[i] + kLn2 * d * R.sp[i]);
          mass += fp * R.sp[i];
        }
      }
      const double tv = 0.5 * wave_sum_d(tvs);
      const double kl = wave_sum_d(klt) - log(np.S / nq.S) * wave_sum_d(mass);
      // p(x), q(x) as the kernel's own entries 2^x 2^(r_c - r_max) / S (the
      // exponentials the sums were built from), a = min(1, p(x)/q(x))
      double px = __builtin_nan(""), qx = __builtin_nan("");
      if (xin) {
        px = (double)exp2_hw(xs[0]) * pow2(xs[1], np.rM) / np.S;
        qx = (double)exp2_hw(xs[2]) * pow2(xs[3], nq.rM) / nq.S;
      }
      o.a = !xin ? __builtin_nan("") : (qx == 0.0 || px >= qx) ? 1.0 : px / qx;
      o.p_tok = xin ? (float)px : nan;
      o.q_tok = xin ? (float)qx : nan;
      o.kl = (float)kl;
      o.tv = (float)tv;
    }
    plan = draw_plan<BF16>(A, b, j, gam, u, R, np, nq, tva);
  }
  return o;
}

// ---------------------------------------------------------------------------
// Sequence finisher (one wave)

// A sequence's per-position inputs as wave 0 holds them (lane j: position j),
// loaded when the finish kernel starts so that they are in registers when
// the accept chain needs them.
struct SeqIn {
  int x;         // draft token x_j (lane < gamma), else -1
  float ua, ur;  // u_acc[j], u_res[j]
  int kvl, rb_old;
};

template <bool GREEDY>
__device__ __forceinline__ SeqIn load_seq_inputs(const Args& A, int b, int gam) {
  const int lane = threadIdx.x & 63;
  const int G1 = A.gmax + 1;
  SeqIn in;
  in.x = -1;
  in.ua = 0.f;
  in.ur = 0.f;
  if (lane <= gam) {
    if (lane < gam) in.x = A.drafts[(size_t)b * A.gmax + lane];
    if (!GREEDY) {
      if (lane < gam) in.ua = A.u_acc[(size_t)b * A.gmax + lane];
      in.ur = A.u_res[(size_t)b * G1 + lane];
    }
  }
  in.kvl = A.kv_len ? A.kv_len[b] : 0;
  in.rb_old = A.rb_kv ? A.rb_kv[b] : 0;
  return in;
}

// What the finisher's waves share.
struct FinShared {
  DrawShared ds;
  uint32_t bits;
  int k;
};

// The sequence's outcome (every wave of the workgroup calls it): wave 0 reads
// the per-position inputs, checks them and runs the accept chain; the first
// four waves scan the stopping row's chunk for the drawn token (greedy: the
// row's argmax); wave 0 writes the outputs and the rollback while the last
// wave zeroes the sequence's workspace words.
template <bool BF16, bool GREEDY>
__device__ void finish_sequence(const Args& A, int b, int gam, const RowOut* rows, const DrawPlan* plans,
                                const SeqIn& in, FinShared& fs) {
  const int lane = threadIdx.x & 63, w = wave_id();
  const int G1 = A.gmax + 1;
  int x = -1;
  double a = 0.0;
  float o_p = 0.f, o_q = 0.f, o_kl = 0.f, o_tv = 0.f;
  int kvl = 0, rb_old = 0;
  if (w == 0) {
    const float ua = in.ua, ur = in.ur;
    x = in.x;
    int argp = -1;
    if (lane <= gam) {
      const RowOut& ro = rows[lane];
      a = ro.a;
      o_p = ro.p_tok;
      o_q = ro.q_tok;
      o_kl = ro.kl;
      o_tv = ro.tv;
      argp = ro.argp;
    }
    kvl = in.kvl;
    rb_old = in.rb_old;
    // data checks
    uint32_t bad = 0;
    if (lane < gam) {
      if (x < 0 || x >= A.V) bad |= SR_ST_TOKEN;
      if (!GREEDY && !(ua >= 0.f && ua < 1.f)) bad |= SR_ST_UNIFORM;
    }
    if (!GREEDY && lane <= gam && !(ur >= 0.f && ur < 1.f)) bad |= SR_ST_UNIFORM;
    if (lane == 0 && A.kv_len && kvl < gam + 1) bad |= SR_ST_KVLEN;
    uint32_t bits = 0;
    if (__ballot(bad & SR_ST_TOKEN)) bits |= SR_ST_TOKEN;
    if (__ballot(bad & SR_ST_UNIFORM)) bits |= SR_ST_UNIFORM;
    if (__ballot(bad & SR_ST_KVLEN)) bits |= SR_ST_KVLEN;
    // the accept chain
    const bool rej = lane < gam && (GREEDY ? x != argp : !((double)ua < a));
    const unsigned long long rmask = __ballot(rej);
    if (lane == 0) {
      fs.bits = bits;
      fs.k = rmask ? (__ffsll((long long)rmask) - 1) : gam;
    }
  }
  __syncthreads();
  const uint32_t bits = fs.bits;
  const int k = fs.k;
  int tok = 0;
  if (!bits) {  // workgroup-uniform
    if constexpr (GREEDY) tok = rows[k].argp;
    else tok = draw_scan<BF16>(A, b, k, plans[k], fs.ds);
  }
  if (w == kFinWaves - 1) clear_sequence(A, b, gam);
  if (w != 0) return;
  if (bits) {
    write_invalid(A, b, bits);
    finish_rollback(A, b, rb_old, kvl);
    count_finished(A, 1);
    return;
  }
  // outputs
  int32_t* ot = A.out_tokens + (size_t)b * G1;
  if (lane <= A.gmax) ot[lane] = lane < k ? x : (lane == k ? tok : -1);
  const float nan = __builtin_nanf("");
  if (lane < A.gmax) {
    const size_t o = (size_t)b * A.gmax + lane;
    const bool live = lane < gam;
    if (A.accept_prob) A.accept_prob[o] = live ? (float)a : nan;
    if (A.p_tok) A.p_tok[o] = live ? o_p : nan;
    if (A.q_tok) A.q_tok[o] = live ? o_q : nan;
    if (A.kl) A.kl[o] = live ? o_kl : nan;
    if (A.tv) A.tv[o] = live ? o_tv : nan;
  }
  if (lane == 0) {
    A.accept_len[b] = k;
    if (A.new_len) A.new_len[b] = kvl - gam + k;
  }
  finish_rollback(A, b, rb_old, kvl - gam + k);
  count_finished(A, 1);
}

// Sequences whose gamma is out of range have no rows: workgroup 0 writes
// their invalid outputs and rollbacks first (all its threads, one sequence
// per wave at a time).
// ---------------------------------------------------------------------------
// The launches

// One step of the sweep, task k (cur): wave 0 issues the loads of the previous
// task's row records (they are ahead of the prefetch in its queue, so they
// return during this task's first pass); every wave issues the next task's
// loads; the first pass of task k; then the previous task's TV sum, with its
// exponentials kept in registers. Returns whether a next task exists.
template <bool BF16, bool GREEDY>
__device__ __forceinline__ bool sweep_step(const Args& A, const int* s_rows, long n_tasks, int n_my, int k,
                                           TaskTable& tab, TaskShared& sh, const __amdgpu_buffer_rsrc_t& rs_recs,
                                           const TaskInfo& cur, const Loaded<BF16>& lp, const Loaded<BF16>& lq,
                                           float (&ep)[Vec<BF16>::E], float (&eq)[Vec<BF16>::E], WaveShift& ws,
                                           TaskInfo prev, bool has_prev, const float (&pp)[Vec<BF16>::E],
                                           const float (&pq)[Vec<BF16>::E], const WaveShift& pws, TaskInfo& nxt,
                                           Loaded<BF16>& np_, Loaded<BF16>& nq_) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const bool tv = !GREEDY && has_prev && prev.pair;  // workgroup-uniform
  // The poll and the merge of the records go to wave k mod 4, so that every
  // SIMD gets its share of that work.
  const bool poller = w == (k & (kWaves - 1));
  RecWords W;
  if (tv && poller) issue_recs(A, rs_recs, prev.row, W);
  // The table is refilled when the next task starts a new window (every read
  // of the old window came before the previous task's barriers); past the
  // end the prefetch reads through an empty resource.
  const bool more = k + 1 < n_my;
  if (more && (k + 1) % kTab == 0) fill_tasks(A, s_rows, n_tasks, k + 1, tab);
  nxt = decode_task<BF16>(A, tab, more ? k + 1 : k);
  issue_loads<BF16>(A, nxt, np_, nq_, more);
  if constexpr (GREEDY) argmax_pass<BF16>(A, cur, lp, lq, sh.x[k & 1], rs_recs);
  else ws = first_pass<BF16>(A, cur, lp, lq, ep, eq, sh.x[k & 1], rs_recs, (k + 2) & (kWaves - 1));
  if (tv) {
    if (poller) poll_row(A, rs_recs, prev, W, sh);
    __syncthreads();
    const double part = sh.ok ? tv_wave_scaled(pp, pq, pws, Norm{sh.rM_p, sh.S_p}, Norm{sh.rM_q, sh.S_q}) : kSkipped;
    if (lane == 0)
      __hip_atomic_store(A.tva + ((size_t)prev.row * A.nc + prev.c) * kWaves + w, part, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  return more;
}

// The TV sum of the last task (nothing left to overlap its poll with).
template <bool BF16>
__device__ __forceinline__ void sweep_last_tv(const Args& A, TaskShared& sh, const __amdgpu_buffer_rsrc_t& rs_recs,
                                              const TaskInfo& prev, const float (&pp)[Vec<BF16>::E],
                                              const float (&pq)[Vec<BF16>::E], const WaveShift& pws) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (!prev.pair) return;
  if (w == 0) {
    RecWords W;
    issue_recs(A, rs_recs, prev.row, W);
    poll_row(A, rs_recs, prev, W, sh);
  }
  __syncthreads();
  const double part = sh.ok ? tv_wave_scaled(pp, pq, pws, Norm{sh.rM_p, sh.S_p}, Norm{sh.rM_q, sh.S_q}) : kSkipped;
  if (lane == 0)
    __hip_atomic_store(A.tva + ((size_t)prev.row * A.nc + prev.c) * kWaves + w, part, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

// Sweep: workgroup g takes tasks g, g + G, g + 2G, ... (G the grid size),
// loading one task ahead and finishing each pair task's TV sum during the next
// task. The loop body is unrolled twice so that the two sets of loaded vectors
// and of exponentials swap roles without copies.
template <bool BF16, bool GREEDY>
__global__ void __launch_bounds__(kThreads, 2) accept_kernel(Args A) {
  constexpr int E = Vec<BF16>::E;
  extern __shared__ int s_rows[];  // [B] inclusive prefix of live rows
  __shared__ TaskShared sh;
  __shared__ TaskTable tab;
  build_row_table(A.gamma, A.gmax, A.B, s_rows);
  const long n_tasks = (long)s_rows[A.B - 1] * A.nc;
  if (blockIdx.x >= n_tasks) return;
  const int n_my = (int)((n_tasks - blockIdx.x + gridDim.x - 1) / gridDim.x);  // this workgroup's tasks
  const __amdgpu_buffer_rsrc_t rs_recs = make_rsrc(A.recs, (size_t)A.B * (A.gmax + 1) * A.nc * kRecBytes);
  fill_tasks(A, s_rows, n_tasks, 0, tab);
  TaskInfo ta = decode_task<BF16>(A, tab, 0), tb = ta;
  Loaded<BF16> pa, qa, pb, qb;
  issue_loads<BF16>(A, ta, pa, qa);
  float epa[E], eqa[E], epb[E], eqb[E];
  WaveShift wsa{kNegInf, kNegInf}, wsb{kNegInf, kNegInf};
  bool has_prev = false;
  for (int k = 0;; k += 2) {
    if (!sweep_step<BF16, GREEDY>(A, s_rows, n_tasks, n_my, k, tab, sh, rs_recs, ta, pa, qa, epa, eqa, wsa, tb,
                                  has_prev, epb, eqb, wsb, tb, pb, qb)) {
      if (!GREEDY) sweep_last_tv<BF16>(A, sh, rs_recs, ta, epa, eqa, wsa);
      break;
    }
    has_prev = true;
    if (!sweep_step<BF16, GREEDY>(A, s_rows, n_tasks, n_my, k + 1, tab, sh, rs_recs, tb, pb, qb, epb, eqb, wsb, ta,
                                  true, epa, eqa, wsa, ta, pa, qa)) {
      if (!GREEDY) sweep_last_tv<BF16>(A, sh, rs_recs, tb, epb, eqb, wsb);
      break;
    }
  }
}

// Finish: one workgroup per sequence, after the sweep. Its eight waves
// finalise the sequence's rows (wave w takes rows w, w + 8, ...) into LDS,
// each with the plan of the draw the sequence would make if it stopped there;
// then the sequence's outcome (finish_sequence). A sequence with gamma
// outside [0, gamma_max] gets the invalid outputs.

template <bool BF16, bool GREEDY>
__global__ void __launch_bounds__(64 * kFinWaves) accept_finish_kernel(Args A) {
  __shared__ RowOut s_out[kMaxRows];
  __shared__ DrawPlan s_plan[kMaxRows];
  __shared__ FinShared fs;
  const int b = blockIdx.x, lane = threadIdx.x & 63, w = wave_id();
  const int gam = A.gamma[b];
  if (!(gam >= 0 && gam <= A.gmax)) {
    if (w == 0) {
      write_invalid(A, b, SR_ST_GAMMA);
      finish_rollback(A, b, A.rb_kv ? A.rb_kv[b] : 0, A.kv_len ? A.kv_len[b] : 0);
      count_finished(A, 1);
    }
    return;
  }
  SeqIn in;
  if (w == 0) in = load_seq_inputs<GREEDY>(A, b, gam);
  const __amdgpu_buffer_rsrc_t rs_recs = make_rsrc(A.recs, (size_t)A.B * (A.gmax + 1) * A.nc * kRecBytes);
  for (int j = w; j <= gam; j += kFinWaves) {
    DrawPlan plan;
    const RowOut o = finalize_row<BF16, GREEDY>(A, b, j, gam, rs_recs, plan);
    if (lane == 0) {
      s_out[j] = o;
      if (!GREEDY) s_plan[j] = plan;
    }
  }
  __syncthreads();
  finish_sequence<BF16, GREEDY>(A, b, gam, s_out, s_plan, in, fs);
}

// ============================================================================
// Top-k / top-p thresholds in two workgroup widths (filter.inc): 512 threads
// when the rows fill at least two workgroups per CU (two then fit a CU, by
// registers and LDS, so one row's selection overlaps the other's streaming),
// else 1024 (fewer rows than that: each row gets more of the device).
namespace filt512 {
constexpr int kFiltThreads = 512;
#include "filter.inc"
}  // namespace filt512
namespace filt1024 {
constexpr int kFiltThreads = 1024;
#include "filter.inc"
}  // namespace filt1024

// ============================================================================
// Plan and launch

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

struct Layout {
  size_t recs, tva, xlogit, thr, fincnt, total;
};

Layout layout(int B, int gamma_max, int nc) {
  const size_t rows = (size_t)B * (gamma_max + 1);
  Layout L;
  L.recs = 0;
  L.tva = L.recs + align256(rows * nc * kRecBytes);
  L.xlogit = L.tva + align256(rows * nc * kWaves * sizeof(double));
  L.thr = L.xlogit + align256(rows * 4 * sizeof(float));
  L.fincnt = L.thr + align256(rows * 2 * sizeof(float));
  L.total = L.fincnt + 256;
  return L;
}

// Chunks per row: the row's aligned span is at most V + N - 1 entries.
int chunks_per_row(int V, int dtype) {
  const int N = dtype == SR_BF16 ? 8 : 4;
  const int chunk = dtype == SR_BF16 ? Vec<true>::kChunk : Vec<false>::kChunk;
  const int span = V % N == 0 ? V : V + N - 1;
  return (span + chunk - 1) / chunk;
}

int resident_per_cu(const void* fn, size_t lds) {
  int per_cu = 1;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kThreads, lds) != hipSuccess || per_cu < 1)
    per_cu = 1;
  return per_cu;
}

// The persistent grid of a launch: what fits on the device at once, a
// multiple of the chunks per row (the chunks of a row are then taken up
// together), and no more than the task count. 0: no device.
int persistent_grid(const void* fn, long max_tasks, int Bl, int nc) {
  const int cus = device_cu_count();
  if (cus <= 0) return 0;
  const long cap = (long)cus * resident_per_cu(fn, Bl * sizeof(int));
  long grid = cap / nc * nc;
  if (grid == 0) grid = cap;
  if (grid > max_tasks) grid = max_tasks;
  return grid < 1 ? 1 : (int)grid;
}

}  // namespace

size_t accept_workspace_bytes(int B, int gamma_max, int V, int dtype) {
  if (B <= 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA || V <= 0) return 0;
  if (dtype != SR_F32 && dtype != SR_BF16) return 0;
  const int nc = chunks_per_row(V, dtype);
  if (nc > kMaxChunks) return 0;
  const int Bl = B < kMaxSeqs ? B : kMaxSeqs;
  if ((size_t)Bl * (gamma_max + 1) * nc * kRecBytes >= 0x7fffffffu) return 0;
  return layout(B, gamma_max, nc).total;
}

int accept_plan(int B, int gamma_max, int V, int dtype, AcceptPlan* plan) {
  plan->chunk = dtype == SR_BF16 ? Vec<true>::kChunk : Vec<false>::kChunk;
  plan->n_chunks = chunks_per_row(V, dtype);
  plan->workspace_bytes = accept_workspace_bytes(B, gamma_max, V, dtype);
  return plan->workspace_bytes == 0 ? SR_EUNSUPPORTED : SR_OK;
}

int launch_accept(const void* p_logits, int64_t p_stride, const void* q_logits, int64_t q_stride,
                  int dtype, const int32_t* drafts, const int32_t* gamma, const float* u_acc,
                  const float* u_res, const int32_t* kv_len, int32_t* accept_len,
                  int32_t* out_tokens, int32_t* new_len, float* accept_prob, float* p_tok,
                  float* q_tok, float* kl, float* tv, int B, int gamma_max, int V, float temperature,
                  int top_k, float top_p, const AcceptRollback* rollback, void* workspace,
                  const AcceptPlan& plan, int32_t* status, hipStream_t stream) {
  const int nc = plan.n_chunks;
  const Layout L = layout(B, gamma_max, nc);
  const bool greedy = temperature == 0.f;
  const int G1 = gamma_max + 1;
  const size_t esz = dtype == SR_BF16 ? 2 : 4;
  char* ws = (char*)workspace;
  // top-k / top-p only under sampling (greedy keeps the argmax anyway)
  const int k_eff = top_k > 0 && top_k < V ? top_k : 0;
  const float p_eff = top_p < 1.f ? top_p : 1.f;
  const bool filt = !greedy && (k_eff > 0 || p_eff < 1.f);
  // sequences in launches of at most kMaxSeqs (the row table)
  for (int b0 = 0; b0 < B; b0 += kMaxSeqs) {
    const int Bl = B - b0 < kMaxSeqs ? B - b0 : kMaxSeqs;
    const size_t r0 = (size_t)b0 * G1;
    Args A;
    A.p = (const char*)p_logits + (size_t)b0 * p_stride * esz;
    A.p_stride = p_stride;
    A.q = q_logits ? (const char*)q_logits + (size_t)b0 * q_stride * esz : nullptr;
    A.q_stride = q_stride;
    A.drafts = drafts ? drafts + (size_t)b0 * gamma_max : nullptr;
    A.gamma = gamma + b0;
    A.u_acc = u_acc ? u_acc + (size_t)b0 * gamma_max : nullptr;
    A.u_res = u_res ? u_res + r0 : nullptr;
    A.kv_len = kv_len ? kv_len + b0 : nullptr;
    A.accept_len = accept_len + b0;
    A.out_tokens = out_tokens + r0;
    A.new_len = new_len ? new_len + b0 : nullptr;
    A.accept_prob = accept_prob ? accept_prob + (size_t)b0 * gamma_max : nullptr;
    A.p_tok = p_tok ? p_tok + (size_t)b0 * gamma_max : nullptr;
    A.q_tok = q_tok ? q_tok + (size_t)b0 * gamma_max : nullptr;
    A.kl = kl ? kl + (size_t)b0 * gamma_max : nullptr;
    A.tv = tv ? tv + (size_t)b0 * gamma_max : nullptr;
    A.B = Bl;
    A.gmax = gamma_max;
    A.V = V;
    A.nc = nc;
    A.lg = greedy ? 0.f : (float)(1.4426950408889634 / (double)temperature);
    A.recs = (u32x4*)(ws + L.recs) + r0 * nc * 2;
    A.tva = (double*)(ws + L.tva) + r0 * nc * kWaves;
    A.xlogit = (float*)(ws + L.xlogit) + r0 * 4;
    A.thr = filt ? (float*)(ws + L.thr) + r0 * 2 : nullptr;
    A.fincnt = (uint32_t*)(ws + L.fincnt);
    A.status = status;
    A.rb_kv = rollback ? rollback->kv_len + b0 : nullptr;
    A.rb_mask = rollback && rollback->mask ? rollback->mask + (size_t)b0 * rollback->L_cap : nullptr;
    A.rb_phys = rollback ? rollback->phys_len : nullptr;
    A.rb_kv_all = rollback ? rollback->kv_len : nullptr;
    A.rb_lcap = rollback ? rollback->L_cap : 0;
    A.n_before = b0;
    const long max_tasks = (long)Bl * G1 * nc;
    const void* fn = dtype == SR_BF16 ? (greedy ? (const void*)accept_kernel<true, true> : (const void*)accept_kernel<true, false>)
                                      : (greedy ? (const void*)accept_kernel<false, true> : (const void*)accept_kernel<false, false>);
    const int n_wg = persistent_grid(fn, max_tasks, Bl, nc);
    if (n_wg == 0) return SR_ELAUNCH;
    const size_t lds = Bl * sizeof(int);  // the row table
    if (filt) {  // the rows' top-k / top-p thresholds first
      const dim3 grid_f((unsigned)(Bl * (2 * G1 - 1)));
      if ((long)grid_f.x >= 2L * device_cu_count()) {
        const dim3 blk(filt512::kFiltThreads);
        if (dtype == SR_BF16)
          hipLaunchKernelGGL(filt512::accept_filter_kernel<true>, grid_f, blk, 0, stream, A, k_eff, p_eff);
        else
          hipLaunchKernelGGL(filt512::accept_filter_kernel<false>, grid_f, blk, 0, stream, A, k_eff, p_eff);
      } else {
        const dim3 blk(filt1024::kFiltThreads);
        if (dtype == SR_BF16)
          hipLaunchKernelGGL(filt1024::accept_filter_kernel<true>, grid_f, blk, 0, stream, A, k_eff, p_eff);
        else
          hipLaunchKernelGGL(filt1024::accept_filter_kernel<false>, grid_f, blk, 0, stream, A, k_eff, p_eff);
      }
      if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
    }
    const dim3 grid((unsigned)n_wg), block(kThreads);
    if (dtype == SR_BF16) {
      if (greedy) hipLaunchKernelGGL((accept_kernel<true, true>), grid, block, lds, stream, A);
      else hipLaunchKernelGGL((accept_kernel<true, false>), grid, block, lds, stream, A);
    } else {
      if (greedy) hipLaunchKernelGGL((accept_kernel<false, true>), grid, block, lds, stream, A);
      else hipLaunchKernelGGL((accept_kernel<false, false>), grid, block, lds, stream, A);
    }
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
    const dim3 grid_s((unsigned)Bl), block_s(64 * kFinWaves);
    if (dtype == SR_BF16) {
      if (greedy) hipLaunchKernelGGL((accept_finish_kernel<true, true>), grid_s, block_s, 0, stream, A);
      else hipLaunchKernelGGL((accept_finish_kernel<true, false>), grid_s, block_s, 0, stream, A);
    } else {
      if (greedy) hipLaunchKernelGGL((accept_finish_kernel<false, true>), grid_s, block_s, 0, stream, A);
      else hipLaunchKernelGGL((accept_finish_kernel<false, false>), grid_s, block_s, 0, stream, A);
    }
    if (hipGetLastError() != hipSuccess) return SR_ELAUNCH;
  }
  return SR_OK;
}

}  // namespace sr
