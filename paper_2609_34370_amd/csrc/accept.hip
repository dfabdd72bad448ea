// Speculative-sampling acceptance (the rule of [sd] the paper builds on, Related Work; its use
// in verification, Sec. 4 and Fig. 3): ratio tests on the drafts, then one inverse-CDF sample
// from the residual max(0, p - q) at the first rejection, or from p_k when every draft passes.
//
// Every decision is taken in exact arithmetic, so any reduction order gives the same integers:
//   test      (double)u * (double)q(x) < (double)p(x)   (a product of two fp32 is exact)
//   weights   W_v = floor(w_v * 2^(40-e)), e = floor(log2 max p)   (integer bit shifts; the scale
//             is the target row's, so with logits it is known from the row statistics)
//   threshold t = floor(u * sum W) from a 128-bit product
//   token     the smallest m whose inclusive prefix of W exceeds t
//
// Partial results are kept per sub-chunk of 4096 vocab entries, one workgroup per sub-chunk:
// its four waves take 1024 entries each and combine in LDS in a fixed order, so every consumer
// reads the same partials.  Kernels, in order on the caller's stream (kernel boundaries are
// the only synchronisation):
//   rounds    (logit inputs) the tests run in rounds of doubling width, positions {0,1},
//             {2..5}, {6..13}, ... (or {0}, {1,2}, {3..6}, ... when a first round over {0,1}
//             would read a lot; one round for short rows), a round from the third on taking
//             every remaining position when they are at most twice its width; a round takes
//             only the sequences that passed every test before it (a device-side list), so rows
//             past a rejection are rarely read.
//     stats   round 0: the statistics (max, sum of 2^(y - max)) of its target and draft rows,
//             per (row, sub-chunk), and the inputs of its tests.  The tests of a round are
//             independent of each other, so nothing here waits for a decision.
//     tests   round r, one workgroup per sequence of the round's list: the round's tests from
//             those statistics, the first failure a, and the sequence's job in the stream
//             launch: the residual of row a (or the bonus row) to sum, or, for a sequence that
//             passed every test of the round, round r+1's statistics (it joins that list).
//     stream  round r, one work item per (sequence of the list, sub-chunk): the job, after one
//             load of its record.  So the sampled rows of finished sequences stream together
//             with the next round's rows.
//   init      (probability inputs) one thread per sequence: geometry, draft-id check, tests.
//   max pass  (probability inputs) per sub-chunk: max of p, bad flag.
//   sum pass  (probability inputs) per sub-chunk: the sums of W_v.
//   search    one workgroup per sequence: total, exact threshold, the sub-chunk holding it,
//             the token inside that sub-chunk (its four waves split the entries), outputs.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "spexis.h"

namespace spexis {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kWaveSub = kAcceptSub / kWaves;   // entries of a sub-chunk one wave takes (1024)
constexpr int kF4 = kWaveSub / (kWave * 4);      // float4 loads per lane (4)
constexpr int kPerLane = 4 * kF4;                // vocab entries per lane (16)
constexpr int kRoundGrid = 65536;                // workgroups of a later round's stream (256 per CU)
constexpr int kTestsGrid = 4096;                 // workgroups of a later round's tests
constexpr int64_t kOneRoundBytes = 192ll << 20;  // target rows that one test round reads whole
constexpr int64_t kRoundRowBytes = 256ll << 10;  // rows this long pay for the launches of a round
constexpr int64_t kNarrowFirstBytes = 256ll << 20;  // a first round over {0,1} reading more starts with {0}
constexpr int64_t kStatPairItems = 16384;        // statistics passes of more (row, sub-chunk) items pair them

enum Mode { kResidual = 1, kBonus = 2, kDone = 3 };
// the job of a listed sequence in a round's stream launch
enum Job { kJobNone = 0, kJobResidual = 1, kJobBonus = 2, kJobNext = 3 };

struct Geom {
  int t0, d0, k, valid;
};

__device__ __forceinline__ Geom load_geom(const AcceptParams& p, int b) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p.geo + 4 * (int64_t)b);
  return Geom{(int)v[0], (int)v[1], (int)v[2], (int)v[3]};
}

// Rows of sequence b: first target row t0, first draft row d0, draft count k (clamped so that
// every row index stays inside its buffer); n = its query tokens (the sequence is valid iff n >= 1).
__device__ __forceinline__ Geom seq_geom(const AcceptParams& p, int b, int& n) {
  const int a0 = p.qsl ? clampi(p.qsl[b], 0, p.T) : b;
  const int a1 = p.qsl ? clampi(p.qsl[b + 1], a0, p.T) : b + 1;
  n = a1 - a0;
  const int nd = p.T - p.B > 0 ? p.T - p.B : 0;
  int k = n - 1;
  if (k < 0) k = 0;
  if (k > p.max_k) k = p.max_k;
  if (k > nd) k = nd;   // only reachable with an inconsistent qsl: stay inside the draft rows
  return Geom{a0, clampi(a0 - b, 0, nd - k), k, n >= 1 ? 1 : 0};
}

// p = 2^(x*c - M) * (1/Z): the probability of a logit, the same expression in every pass
// (R = 1/Z is rounded once per row).  x*c - M is one explicit fused multiply-add, so no site
// can contract it differently from another: every pass sees the same probabilities.
__device__ __forceinline__ float logit_prob(float x, float c, float M, float R) {
  return fast_exp2(__builtin_fmaf(x, c, -M)) * R;
}

__device__ __forceinline__ bool bad_value(float x) { return !(x >= 0.f) || isinf(x); }

// floor(w * 2^s) for a finite w >= 0 and a shift s with w * 2^s < 2^41, by integer shifts.
__device__ __forceinline__ uint64_t fixed_weight(float w, int s) {
  const uint32_t bits = __float_as_uint(w);
  const uint32_t ef = (bits >> 23) & 0xFF;
  const uint64_t mant = ef ? ((bits & 0x7FFFFFu) | 0x800000u) : (bits & 0x7FFFFFu);
  const int sh = (ef ? (int)ef - 150 : -149) + s;
  if (sh >= 0) return mant << sh;
  return -sh >= 32 ? 0ull : (mant >> (-sh));
}

// floor(log2 M) for a finite M > 0.
__device__ __forceinline__ int floor_log2(float M) {
  const uint32_t bits = __float_as_uint(M);
  const uint32_t ef = (bits >> 23) & 0xFF;
  if (ef) return (int)ef - 127;
  return (31 - __clz(bits & 0x7FFFFFu)) - 149;
}

// floor(u * S) exactly for an fp32 u, clamped to [0, S-1].
__device__ __forceinline__ uint64_t exact_threshold(float u, uint64_t S) {
  if (!(u > 0.f)) return 0;
  if (u >= 1.f) return S - 1;
  const uint32_t bits = __float_as_uint(u);
  const uint32_t ef = (bits >> 23) & 0xFF;
  const uint64_t mu = ef ? ((bits & 0x7FFFFFu) | 0x800000u) : (bits & 0x7FFFFFu);
  const int shift = -(ef ? (int)ef - 150 : -149);   // u = mu * 2^-shift, shift >= 24
  const uint64_t lo = mu * S;
  const uint64_t hi = __umul64hi(mu, S);
  uint64_t t;
  if (shift >= 128) t = 0;
  else if (shift >= 64) t = hi >> (shift - 64);
  else t = (lo >> shift) | (hi << (64 - shift));
  return t < S ? t : S - 1;
}

// Four consecutive vocab entries starting at e (e % 4 == 0); entries >= V read as `fill`.
__device__ __forceinline__ f32x4 load4(const float* row, int e, int V, bool vec, float fill) {
  if (vec && e + 3 < V) return *reinterpret_cast<const f32x4*>(row + e);
  f32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = e + i < V ? row[e + i] : fill;
  return r;
}

// Wave `wave`'s coalesced part of sub-chunk `sub`: lane l holds entries
// sub*4096 + 1024 wave + 256 j + 4 l + i.  A part inside the row takes the straight-line path,
// so all its loads are in flight together.
// kNT: non-temporal loads, for rows read once (the statistics pass).
template <bool kNT = false>
__device__ __forceinline__ void load_sub(const float* row, int sub, int wave, int V, bool vec, float fill, int lane,
                                         float (&v)[kPerLane]) {
  const int base = sub * kAcceptSub + wave * kWaveSub;
  if (vec && base + kWaveSub <= V) {
    const f32x4* src = reinterpret_cast<const f32x4*>(row + base) + lane;
#pragma unroll
    for (int j = 0; j < kF4; ++j) {
      const f32x4 x = kNT ? __builtin_nontemporal_load(src + j * kWave) : src[j * kWave];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kF4; ++j) {
    const f32x4 x = load4(row, base + j * 4 * kWave + 4 * lane, V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
  }
}

// The (max, sum) partial of lane l's first sub-chunk (x = l), loaded ahead of its reduction so
// that a consumer can have all of its partial loads in flight at once.
struct Part2 {
  float a, b;
};
__device__ __forceinline__ Part2 part_first(const float* part, int nsub, int lane, float fa, float fb) {
  if (lane >= nsub) return Part2{fa, fb};
  const f32x2 v = *reinterpret_cast<const f32x2*>(part + 2 * lane);
  return Part2{v[0], v[1]};
}

// Statistics of one logit row from its sub-chunk partials, combined in a fixed order by one
// full wave (every consumer calls exactly this, so all of them get identical M and 1/Z, the
// latter returned in Z).  A row without a finite maximum or with a bad sum gives Z = NaN.
// `f` is part_first(part, ...) with fill (-inf, 0).
__device__ __forceinline__ void row_stats(const float* part, int nsub, int lane, Part2 f, float& M, float& Z) {
  float mm = f.a;
  for (int x = lane + kWave; x < nsub; x += kWave) mm = fmaxf(mm, part[2 * x]);
  mm = wave_max(mm);
  float zz = 0.f;
  int nan = 0;
  if (lane < nsub) {
    nan |= f.b != f.b;
    if (f.a != -INFINITY) zz += f.b * fast_exp2(f.a - mm);
  }
  for (int x = lane + kWave; x < nsub; x += kWave) {
    const float z = part[2 * x + 1];
    nan |= z != z;
    if (part[2 * x] != -INFINITY) zz += z * fast_exp2(part[2 * x] - mm);
  }
  zz = wave_sum(zz);
  nan = wave_or(nan);
  M = mm;
  Z = (nan || !(mm > -INFINITY) || !(mm < INFINITY)) ? NAN : 1.0f / zz;   // reciprocal of the sum
}

// Sub-chunk statistics of row i of sequence b (which = 0 target, 1 draft).
__device__ __forceinline__ float* lse_slot(const AcceptParams& p, int b, int i, int which) {
  return p.lse_part + ((((int64_t)b * (p.max_k + 1) + i) * 2 + which) * p.nsub) * 2;
}

// Final outputs of sequence b (called by exactly one thread).
__device__ void write_outputs(const AcceptParams& p, int b, const Geom& g, int a, int token, int status) {
  int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
  for (int i = 0; i <= p.max_k; ++i) row[i] = i < a ? p.ids[g.d0 + i] : (i == a ? token : -1);
  if (p.tok_prob && token < 0) p.tok_prob[b] = 0.f;
  p.accepted_len[b] = a;
  p.row_status[b] = status;
  if (p.seq_lens_inout) p.seq_lens_inout[b] -= g.k - a;
}

// Outputs of a sequence that samples nothing (called by exactly one thread).
__device__ void write_invalid(const AcceptParams& p, int b, int n) {
  int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
  for (int i = 0; i <= p.max_k; ++i) row[i] = -1;
  if (p.tok_prob) p.tok_prob[b] = 0.f;
  p.accepted_len[b] = 0;
  p.row_status[b] = n >= 1 ? SPEXIS_ROW_BAD_TOKEN : SPEXIS_ROW_BAD_VALUE;
  p.st_mode[b] = kDone;
  p.st_a[b] = 0;
  reinterpret_cast<u32x4*>(p.srec)[3 * (int64_t)b + 1] = u32x4{(uint32_t)kDone, 0u, 0u, 0u};
}

// Row context of a tested or sampled position a: target row a (P) and, for a residual, draft
// row a (Q), with their statistics in logits mode.
struct RowCtx {
  const float* P;
  const float* Q;        // nullptr for the bonus row
  float Mp, Rp, Mq, Rq;  // row maxima (scaled) and reciprocal sums (logits mode)
  bool logits;
};

__device__ __forceinline__ float prob_of(const RowCtx& r, float raw, float c, bool draft) {
  if (!r.logits) return raw;
  return draft ? logit_prob(raw, c, r.Mq, r.Rq) : logit_prob(raw, c, r.Mp, r.Rp);
}

// Context of position a of sequence b (computed identically everywhere); `with_q` also takes
// draft row a.  In logits mode both rows' partials are loaded before either is reduced.
__device__ __forceinline__ RowCtx row_ctx(const AcceptParams& p, int b, const Geom& g, int a, bool with_q, int lane) {
  RowCtx r;
  r.P = p.target + (int64_t)(g.t0 + a) * p.V;
  r.Q = with_q ? p.draft + (int64_t)(g.d0 + a) * p.V : nullptr;
  r.logits = p.kind == 1;
  r.Mp = r.Rp = r.Mq = r.Rq = 1.f;
  if (r.logits) {
    // partials computed here (per 4096-entry sub-chunk) or given by the caller (per column tile)
    const bool ext = p.ext_tstats != nullptr;
    const int np = ext ? p.ext_parts : p.nsub;
    const float* lp = ext ? p.ext_tstats + (int64_t)(g.t0 + a) * np * 2 : lse_slot(p, b, a, 0);
    const float* lq = ext ? p.ext_dstats + (int64_t)(g.d0 + a) * np * 2 : lse_slot(p, b, a, 1);
    const Part2 fp = part_first(lp, np, lane, -INFINITY, 0.f);
    const Part2 fq = with_q ? part_first(lq, np, lane, -INFINITY, 0.f) : Part2{-INFINITY, 0.f};
    row_stats(lp, np, lane, fp, r.Mp, r.Rp);
    if (with_q) row_stats(lq, np, lane, fq, r.Mq, r.Rq);
  }
  return r;
}

// Combines a value of each of the four waves in wave order through LDS; every thread gets the
// result.  (All four waves must call it.)
template <typename T, typename F>
__device__ __forceinline__ T wg_combine(T v, int wave, int lane, F op) {
  __shared__ T sm[kWaves];
  if (lane == 0) sm[wave] = v;
  __syncthreads();
  T r = sm[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) r = op(r, sm[w]);
  __syncthreads();   // sm may be reused by the next call
  return r;
}

// Probability inputs: the largest target probability over sub-chunk `sub` of the sampled row,
// and whether the sampled row(s) hold a NaN, an infinity or a negative value there, written to
// max_part / bad_part by one workgroup.
__device__ void sub_maxima(const AcceptParams& p, const RowCtx& r, bool residual, int b, int sub, int wave, int lane) {
  const bool vec = (p.V & 3) == 0;
  float pv[kPerLane], qv[kPerLane];
  load_sub(r.P, sub, wave, p.V, vec, 0.f, lane, pv);
  if (residual) load_sub(r.Q, sub, wave, p.V, vec, 0.f, lane, qv);
  float mp = 0.f;
  int bad = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    bad |= bad_value(pv[e]) || (residual && bad_value(qv[e]));
    mp = pv[e] > mp ? pv[e] : mp;
  }
  mp = wg_combine(wave_max(mp), wave, lane, [](float x, float y) { return fmaxf(x, y); });
  bad = wg_combine(wave_or(bad), wave, lane, [](int x, int y) { return x | y; });
  if (threadIdx.x == 0) {
    p.max_part[(int64_t)b * p.nsub + sub] = mp;
    p.bad_part[(int64_t)b * p.nsub + sub] = bad;
  }
}

// The scale of the sampled row, M = the largest probability of target row a (with logits
// 2^0 * (1/Z), from its statistics), and whether a row the sampling reads holds a NaN, an
// infinity or a negative value (with logits: a row whose statistics are not finite).  One
// full wave; every consumer gets the same values.
__device__ __forceinline__ void sampled_scale(const AcceptParams& p, const RowCtx& r, int b, bool residual, int lane,
                                              float& M, int& bad) {
  if (r.logits) {
    M = r.Rp;
    bad = !(r.Rp > 0.f) || isinf(r.Rp) || (residual && (!(r.Rq > 0.f) || isinf(r.Rq)));
    return;
  }
  M = 0.f;
  bad = 0;
  for (int x = lane; x < p.nsub; x += kWave) {
    M = fmaxf(M, p.max_part[(int64_t)b * p.nsub + x]);
    bad |= p.bad_part[(int64_t)b * p.nsub + x];
  }
  M = wave_max(M);
  bad = wave_or(bad);
}

// Fixed-point weight of one entry: of p (use_p) or of the residual max(0, p - q).  The sums and
// the search evaluate exactly this expression.
__device__ __forceinline__ uint64_t entry_weight(const RowCtx& r, float c, float pv_raw, float qv_raw, bool use_p,
                                                 int s) {
  const float P = prob_of(r, pv_raw, c, false);
  float w;
  if (use_p) {
    w = P;
  } else {
    const float d = P - prob_of(r, qv_raw, c, true);
    w = d > 0.f ? d : 0.f;
  }
  return fixed_weight(w, s);
}

// Fixed-point sums over sub-chunk `sub` of the sampled row at shift s, by one workgroup: the
// residual weights (0 for a bonus row) and the weights of p (the fallback of an empty
// residual), written to sum_part[b][sub][0..1].  pv / qv hold the sub-chunk's entries.
__device__ void sub_sums(const AcceptParams& p, const RowCtx& r, bool residual, int b, int sub, int s, int wave,
                         int lane, const float (&pv)[kPerLane], const float (&qv)[kPerLane]) {
  uint64_t sr = 0, sp = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    sp += entry_weight(r, p.c, pv[e], 0.f, true, s);
    if (residual) sr += entry_weight(r, p.c, pv[e], qv[e], false, s);
  }
  const auto add = [](uint64_t x, uint64_t y) { return x + y; };
  sr = wg_combine(wave_sum_u64(sr), wave, lane, add);
  sp = wg_combine(wave_sum_u64(sp), wave, lane, add);
  if (threadIdx.x == 0) {
    uint64_t* dst = p.sum_part + ((int64_t)b * p.nsub + sub) * 2;
    dst[0] = sr;
    dst[1] = sp;
  }
}

// The sampled row(s) of sequence b at position a over sub-chunk `sub`: entries, statistics,
// scale, then the fixed-point sums (a bad or empty row writes none; the search reports it).
__device__ void sample_sums(const AcceptParams& p, int b, const Geom& g, int a, bool residual, int sub, int wave,
                            int lane) {
  const bool vec = (p.V & 3) == 0;
  const float fill = p.kind == 1 ? -INFINITY : 0.f;
  // the entries first: their loads overlap the reductions of the row statistics and maxima
  float pv[kPerLane], qv[kPerLane];
  // non-temporal: the search reads back one sub-chunk of these rows at most (measured: the
  // acceptance of 512 sequences of 152064-entry rows 6 us faster, a whole verification step
  // about 2 us, and no slower at 64 sequences of 128256)
  load_sub<true>(p.target + (int64_t)(g.t0 + a) * p.V, sub, wave, p.V, vec, fill, lane, pv);
  if (residual) {
    load_sub<true>(p.draft + (int64_t)(g.d0 + a) * p.V, sub, wave, p.V, vec, fill, lane, qv);
  } else {
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) qv[e] = 0.f;
  }
  const RowCtx r = row_ctx(p, b, g, a, residual, lane);
  float M;
  int bad;
  sampled_scale(p, r, b, residual, lane, M, bad);
  if (sub == 0 && threadIdx.x == 0) {
    // the search's record: geometry, position and mode, bad flag and scale, row statistics
    u32x4* rec = reinterpret_cast<u32x4*>(p.srec) + 3 * (int64_t)b;
    rec[0] = u32x4{(uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k, (uint32_t)a};
    rec[1] = u32x4{(uint32_t)(residual ? kResidual : kBonus), (uint32_t)bad, __float_as_uint(M), 0u};
    rec[2] = u32x4{__float_as_uint(r.Mp), __float_as_uint(r.Rp), __float_as_uint(r.Mq), __float_as_uint(r.Rq)};
  }
  if (bad || !(M > 0.f)) return;   // the same decision in every wave
  sub_sums(p, r, residual, b, sub, 40 - floor_log2(M), wave, lane, pv, qv);
}

// ---------------------------------------------------------------------------------- init

__global__ __launch_bounds__(kThreads) void accept_init_kernel(AcceptParams p) {
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b >= p.B) return;
  int n;
  const Geom g = seq_geom(p, b, n);
  bool ok = n >= 1;
  for (int i = 0; ok && i < g.k; ++i) {
    const int x = p.ids[g.d0 + i];
    ok = x >= 0 && x < p.V;
  }
  *reinterpret_cast<u32x4*>(p.geo + 4 * (int64_t)b) = u32x4{(uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k, ok ? 1u : 0u};
  if (!ok) return write_invalid(p, b, n);
  int a = 0;
  while (a < g.k) {
    const int x = p.ids[g.d0 + a];
    const double pp = (double)p.target[(int64_t)(g.t0 + a) * p.V + x];
    const double qq = (double)p.draft[(int64_t)(g.d0 + a) * p.V + x];
    const double u = (double)p.u_accept[g.d0 + a];
    if (u * qq < pp) ++a; else break;
  }
  p.st_a[b] = a;
  p.st_mode[b] = a < g.k ? kResidual : kBonus;
}

// ------------------------------------------------------------------- logits: statistics

// (max, sum of 2^(y - max)) of one wave's entries; NaN sum if a logit is NaN/+inf.
__device__ __forceinline__ void wave_stats(float (&v)[kPerLane], float c, float& m, float& z) {
  m = -INFINITY;
  int bad = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    bad |= !(v[e] < INFINITY);   // NaN or +inf: the row's probabilities are undefined
    v[e] *= c;
    m = fmaxf(m, v[e]);
  }
  m = wave_max(m);
  bad = wave_or(bad);
  z = 0.f;
  if (m != -INFINITY) {
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) z += fast_exp2(v[e] - m);
  }
  z = wave_sum(z);
  if (bad) z = NAN;
}

// Sequence b's rows and state for the tests launches (valid: 1 valid, 0 no query token, -1 a
// draft id outside [0, V)), written once per sequence by the pass before the first tests launch
// (the statistics or the gather pass).  That launch then reads one record per sequence instead
// of query_start_loc and every draft id: a dependent round trip less.
__device__ __forceinline__ void store_geom_state(const AcceptParams& p, int b, const Geom& g, int bad_id) {
  const int state = !g.valid ? 0 : bad_id ? -1 : 1;
  *reinterpret_cast<u32x4*>(p.geo + 4 * (int64_t)b) = u32x4{(uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k, (uint32_t)state};
}

// Sequence li of round r's list: all sequences in round 0 (their stored record; with no drafts
// at all there are no ids to check, and no pass before writes one), the ones still accepting
// after.
__device__ __forceinline__ void round_seq(const AcceptParams& p, int r, int li, int& b, Geom& g) {
  if (r == 0) {
    b = li;
    if (p.max_k == 0) {
      int n;
      g = seq_geom(p, b, n);
    } else {
      g = load_geom(p, b);
    }
    return;
  }
  const u32x4 e = *reinterpret_cast<const u32x4*>(p.lists + ((int64_t)(r - 1) * p.B + li) * 4);
  b = (int)e[0];
  g = Geom{(int)e[1], (int)e[2], (int)e[3], 1};
}

__device__ __forceinline__ int round_count(const AcceptParams& p, int r) { return r == 0 ? p.B : p.counts[r]; }

// The inputs of test pos of sequence b: target and draft entries of draft x_pos, u_pos, and
// whether x_pos is a valid id (called by one thread).
__device__ __forceinline__ void gather_test(const AcceptParams& p, int b, const Geom& g, int pos) {
  const int x = p.ids[g.d0 + pos];
  const bool ok = x >= 0 && x < p.V;
  f32x4 t;
  if (p.tg_given) {   // gathered by the LM head (the same fp32 values)
    t[0] = ok ? p.tg_given[g.t0 + pos] : 0.f;
    t[1] = ok ? p.dg_given[g.d0 + pos] : 0.f;
  } else {
    t[0] = ok ? p.target[(int64_t)(g.t0 + pos) * p.V + x] : 0.f;
    t[1] = ok ? p.draft[(int64_t)(g.d0 + pos) * p.V + x] : 0.f;
  }
  t[2] = p.u_accept[g.d0 + pos];
  t[3] = ok ? 1.f : 0.f;
  *reinterpret_cast<f32x4*>(p.tin + ((int64_t)b * p.max_k + pos) * 4) = t;
}

// Statistics of one row over sub-chunk `sub` from its entries v (overwritten): the four waves'
// (max, sum) combined in wave order (common maximum, rescaled sums; NaN stays NaN), written by
// thread 0 to the row's slot.  (All four waves must call it.)
__device__ __forceinline__ void store_sub_stats(const AcceptParams& p, float (&v)[kPerLane], float* slot, int sub,
                                                int wave, int lane) {
  __shared__ float sm_m[kWaves], sm_z[kWaves];
  float m, z;
  wave_stats(v, p.c, m, z);
  if (lane == 0) {
    sm_m[wave] = m;
    sm_z[wave] = z;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sm_m[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sm_m[w]);
    float Z = 0.f;
    bool nan = false;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      nan |= sm_z[w] != sm_z[w];
      if (sm_m[w] != -INFINITY) Z += sm_z[w] * fast_exp2(sm_m[w] - M);
    }
    *reinterpret_cast<f32x2*>(slot + 2 * sub) = f32x2{M, nan ? NAN : Z};
  }
  __syncthreads();
}

// A round's positions [lo, hi) of sequence b over sub-chunk `sub`: statistics of target rows
// lo..min(hi-1, k) and draft rows lo..min(hi, k)-1 (target rows first), each row's loads issued
// before the previous row reduces.
__device__ void next_round_stats(const AcceptParams& p, int b, const Geom& g, int lo, int hi, int sub, int wave,
                                 int lane) {
  const int nt = min(hi - 1, g.k) - lo + 1;   // >= 1: lo <= k
  const int nd = max(0, min(hi, g.k) - lo);
  const int rows = nt + nd;
  const bool vec = (p.V & 3) == 0;
  auto row = [&](int j) {
    return j < nt ? p.target + (int64_t)(g.t0 + lo + j) * p.V : p.draft + (int64_t)(g.d0 + lo + j - nt) * p.V;
  };
  auto slot = [&](int j) { return j < nt ? lse_slot(p, b, lo + j, 0) : lse_slot(p, b, lo + j - nt, 1); };
  float va[kPerLane], vb[kPerLane];
  load_sub<true>(row(0), sub, wave, p.V, vec, -INFINITY, lane, va);
  for (int j = 0; j < rows; j += 2) {
    if (j + 1 < rows) load_sub<true>(row(j + 1), sub, wave, p.V, vec, -INFINITY, lane, vb);
    store_sub_stats(p, va, slot(j), sub, wave, lane);
    if (j + 1 < rows) {
      if (j + 2 < rows) load_sub<true>(row(j + 2), sub, wave, p.V, vec, -INFINITY, lane, va);
      store_sub_stats(p, vb, slot(j + 1), sub, wave, lane);
    }
  }
}

// Round 0, positions [0, hi): statistics of target rows 0..min(hi-1, k) and draft rows
// 0..min(hi, k)-1 of every sequence, one work item per (row, SUBS consecutive sub-chunks), and
// the inputs of the tests at those positions.  An item issues the loads of all its sub-chunks
// before it reduces the first.  (Items of one row each keep more loads in flight than items
// that stream a sequence's rows one after another.)
template <int SUBS>
__global__ __launch_bounds__(kThreads) void accept_stats_kernel(AcceptParams p, int hi) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  if (blockIdx.x == 0 && threadIdx.x <= kAcceptMaxRounds) p.counts[threadIdx.x] = 0;
  const int rows = 2 * hi;
  const int ngrp = (p.nsub + SUBS - 1) / SUBS;
  const int64_t total = (int64_t)p.B * rows * ngrp;
  for (int64_t item = blockIdx.x; item < total; item += gridDim.x) {
    const int grp = (int)(item % ngrp);
    const int64_t rest = item / ngrp;
    const int rr = (int)(rest % rows), b = (int)(rest / rows);
    const int pos = rr >> 1, which = rr & 1;
    int n;
    const Geom g = seq_geom(p, b, n);
    const bool skip = !g.valid || pos > g.k || (which == 1 && pos == g.k);
    const int sub0 = grp * SUBS, nsubs = min(SUBS, p.nsub - sub0);
    float v[SUBS][kPerLane];
    if (!skip) {
      const float* row = which ? p.draft + (int64_t)(g.d0 + pos) * p.V : p.target + (int64_t)(g.t0 + pos) * p.V;
#pragma unroll
      for (int u = 0; u < SUBS; ++u)
        if (u < nsubs) load_sub<true>(row, sub0 + u, wave, p.V, (p.V & 3) == 0, -INFINITY, lane, v[u]);
    }
    // the first item of each sequence records it for the tests launches (its id loads follow the
    // row's, so they add no round trip)
    if (rr == 0 && grp == 0 && wave == 0) {
      int bad = 0;
      for (int i = lane; i < g.k; i += kWave) {
        const int x = p.ids[g.d0 + i];
        bad |= x < 0 || x >= p.V;
      }
      bad = wave_or(bad);
      if (lane == 0) store_geom_state(p, b, g, bad);
    }
    if (skip) continue;
    // the inputs of test pos, gathered here so that the decision needs no dependent gather
    if (which == 0 && pos < g.k && grp == 0 && threadIdx.x == 0) gather_test(p, b, g, pos);
#pragma unroll
    for (int u = 0; u < SUBS; ++u)   // nsubs is the same for the whole workgroup
      if (u < nsubs) store_sub_stats(p, v[u], lse_slot(p, b, pos, which), sub0 + u, wave, lane);
  }
}

// Given per-tile statistics of `rows` rows reduced to one (max, sum) per row, one wave per row:
// M = max over the tiles, then Z = sum of z * 2^(m - M) (lane-strided partial sums, combined
// across the wave in a fixed order; every consumer reads the reduced pair).  Each lane's tiles
// are loaded 8 at a time, the loads of a group issued together.
__global__ __launch_bounds__(kThreads) void accept_combine_kernel(const float* src, int parts, int rows,
                                                                  float* dst) {
  constexpr int kG = 8;
  const int lane = threadIdx.x % kWave;
  const int row = blockIdx.x * kWaves + threadIdx.x / kWave;
  if (row >= rows) return;
  const f32x2* part = reinterpret_cast<const f32x2*>(src + (int64_t)row * parts * 2);
  float mm = -INFINITY;
  for (int x0 = lane; x0 < parts; x0 += kG * kWave) {
    f32x2 v[kG];
#pragma unroll
    for (int u = 0; u < kG; ++u) v[u] = part[min(x0 + u * kWave, parts - 1)];
#pragma unroll
    for (int u = 0; u < kG; ++u)
      if (x0 + u * kWave < parts) mm = fmaxf(mm, v[u][0]);
  }
  mm = wave_max(mm);
  float zz = 0.f;
  int nan = 0;
  for (int x0 = lane; x0 < parts; x0 += kG * kWave) {
    f32x2 v[kG];
#pragma unroll
    for (int u = 0; u < kG; ++u) v[u] = part[min(x0 + u * kWave, parts - 1)];
#pragma unroll
    for (int u = 0; u < kG; ++u) {
      if (x0 + u * kWave >= parts) continue;
      nan |= v[u][1] != v[u][1];
      if (v[u][0] != -INFINITY) zz += v[u][1] * fast_exp2(v[u][0] - mm);
    }
  }
  zz = wave_sum(zz);
  nan = wave_or(nan);
  if (lane == 0) *reinterpret_cast<f32x2*>(dst + (int64_t)row * 2) = f32x2{mm, nan ? NAN : zz};
}

// The inputs of every test, when the statistics are given and no stats pass gathers them.
__global__ __launch_bounds__(kThreads) void accept_gather_kernel(AcceptParams p) {
  // one thread per (sequence, draft position); max_k >= 1 (with no drafts there is nothing to
  // gather or check)
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)p.B * p.max_k) return;
  const int b = (int)(idx / p.max_k), i = (int)(idx % p.max_k);
  int n;
  const Geom g = seq_geom(p, b, n);
  if (i == 0) {
    int bad = 0;
    for (int j = 0; j < g.k; ++j) {
      const int x = p.ids[g.d0 + j];
      bad |= x < 0 || x >= p.V;
    }
    store_geom_state(p, b, g, bad);
  }
  if (!g.valid || i >= g.k) return;
  gather_test(p, b, g, i);
}

// Round r, positions [lo, hi), step 1 of 2: one workgroup per sequence of the round's list runs
// the tests at those positions from the statistics (its waves split the positions) and finds
// the first failure.  A failure at a: the sequence is done testing, and the residual of row a
// will be sampled.  No failure: the bonus row k will be sampled if the round reached position
// k, else the sequence joins round r+1 (positions [hi, hi2)), whose test inputs it gathers.
// It leaves the stream launch of the round one record per list entry (the job: the fixed-point
// sums of the sampled row at its scale, or round r+1's statistics) and the search its record.
// So the stream launch's items start streaming after one load, instead of each repeating the
// tests.
__global__ __launch_bounds__(kThreads) void accept_tests_kernel(AcceptParams p, int r, int lo, int hi, int hi2) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int count = round_count(p, r);
  __shared__ int sm_fail[kWaves];
  __shared__ f32x4 sm_rc[kWaves];   // row statistics (Mp, Rp, Mq, Rq) a wave computed
  for (int li = blockIdx.x; li < count; li += gridDim.x) {
    int b;
    Geom g;
    round_seq(p, r, li, b, g);
    u32x4* rec = reinterpret_cast<u32x4*>(p.strec) + 3 * (int64_t)li;
    if (r == 0 && g.valid != 1) {   // no query token, or a draft id out of range
      if (threadIdx.x == 0) {
        write_invalid(p, b, g.valid == 0 ? 0 : 1);
        rec[1] = u32x4{(uint32_t)kJobNone, 0u, 0u, 0u};
      }
      continue;
    }
    // position i fails when !(u_i q_i(x_i) < p_i(x_i)) (NaN statistics fail)
    const float* tin = p.tin + (int64_t)b * p.max_k * 4;
    const int end = min(hi, g.k);
    // a wave the round's tests leave idle computes the bonus row's statistics meanwhile, in case
    // every test passes
    const int wbonus = hi > g.k && end - lo < kWaves ? max(end - lo, 0) : -1;
    int fail = g.k + 1;   // none
    for (int i = lo + wave; i < end; i += kWaves) {
      const f32x2 t = *reinterpret_cast<const f32x2*>(tin + 4 * i);
      const float u = tin[4 * i + 2];
      const RowCtx rc = row_ctx(p, b, g, i, true, lane);
      const float pp = logit_prob(t[0], p.c, rc.Mp, rc.Rp);
      const float qq = logit_prob(t[1], p.c, rc.Mq, rc.Rq);
      if (!((double)u * (double)qq < (double)pp)) {
        fail = i;
        if (lane == 0) sm_rc[wave] = f32x4{rc.Mp, rc.Rp, rc.Mq, rc.Rq};   // the sampled row's, if first
        break;
      }
    }
    if (wave == wbonus) {
      const RowCtx rc = row_ctx(p, b, g, g.k, false, lane);
      if (lane == 0) sm_rc[wave] = f32x4{rc.Mp, rc.Rp, rc.Mq, rc.Rq};
    }
    if (lane == 0) sm_fail[wave] = fail;
    __syncthreads();
    const int a = min(min(sm_fail[0], sm_fail[1]), min(sm_fail[2], sm_fail[3]));
    __syncthreads();
    if (wave != 0) continue;
    const u32x4 q0 = u32x4{(uint32_t)b, (uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k};
    if (a < g.k || hi > g.k) {
      // a failure at a: the residual of row a; every test passed and the round reached k: the
      // bonus row k.  Either way the scale is known from row a's statistics, which the wave that
      // tested position a (or the one that took the bonus row) computed: the same values row_ctx
      // gives here.
      const bool residual = a < g.k;
      const int pos = residual ? a : g.k;
      const int from = residual ? (a - lo) % kWaves : wbonus;
      RowCtx rc;
      if (from >= 0) {
        const f32x4 st = sm_rc[from];
        rc.P = p.target + (int64_t)(g.t0 + pos) * p.V;
        rc.Q = residual ? p.draft + (int64_t)(g.d0 + pos) * p.V : nullptr;
        rc.logits = true;
        rc.Mp = st[0];
        rc.Rp = st[1];
        rc.Mq = residual ? st[2] : 1.f;
        rc.Rq = residual ? st[3] : 1.f;
      } else {
        rc = row_ctx(p, b, g, pos, residual, lane);
      }
      float M;
      int bad;
      sampled_scale(p, rc, b, residual, lane, M, bad);
      if (lane == 0) {
        const u32x4 stats{__float_as_uint(rc.Mp), __float_as_uint(rc.Rp), __float_as_uint(rc.Mq),
                          __float_as_uint(rc.Rq)};
        u32x4* srec = reinterpret_cast<u32x4*>(p.srec) + 3 * (int64_t)b;
        srec[0] = u32x4{(uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k, (uint32_t)pos};
        srec[1] = u32x4{(uint32_t)(residual ? kResidual : kBonus), (uint32_t)bad, __float_as_uint(M), 0u};
        srec[2] = stats;
        // a bad or empty row has no sums to compute (the search reports it)
        const bool go = !bad && M > 0.f;
        rec[0] = q0;
        rec[1] = u32x4{(uint32_t)(go ? (residual ? kJobResidual : kJobBonus) : kJobNone), (uint32_t)pos, 0u,
                       (uint32_t)(go ? 40 - floor_log2(M) : 0)};
        rec[2] = stats;
      }
    } else {
      // hi <= k <= max_k: round r+1 exists (the host passes hi2 > hi)
      if (lane == 0) {
        const int at = __hip_atomic_fetch_add(p.counts + r + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *reinterpret_cast<u32x4*>(p.lists + ((int64_t)r * p.B + at) * 4) = q0;
        rec[0] = q0;
        rec[1] = u32x4{(uint32_t)kJobNext, (uint32_t)hi, (uint32_t)hi2, 0u};
      }
      for (int pos = hi + lane; pos < min(hi2, g.k); pos += kWave) gather_test(p, b, g, pos);
    }
  }
}

// Round r, step 2 of 2: one work item per (sequence of the list, sub-chunk) does the job the
// tests launch recorded for the sequence: the fixed-point sums of the sampled row(s) over its
// sub-chunk, or the statistics of round r+1's rows over its sub-chunk.  So the sampled rows of
// finished sequences stream together with the next round's rows.
__global__ __launch_bounds__(kThreads) void accept_stream_kernel(AcceptParams p, int r) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int64_t total = (int64_t)round_count(p, r) * p.nsub;
  const bool vec = (p.V & 3) == 0;
  for (int64_t item = blockIdx.x; item < total; item += gridDim.x) {
    const int sub = (int)(item % p.nsub), li = (int)(item / p.nsub);
    const u32x4* rec = reinterpret_cast<const u32x4*>(p.strec) + 3 * (int64_t)li;
    const u32x4 q0 = rec[0], q1 = rec[1], q2 = rec[2];
    const int job = (int)q1[0];
    if (job != kJobResidual && job != kJobBonus && job != kJobNext) continue;
    const int b = (int)q0[0];
    const Geom g{(int)q0[1], (int)q0[2], (int)q0[3], 1};
    if (job == kJobNext) {
      next_round_stats(p, b, g, (int)q1[1], (int)q1[2], sub, wave, lane);
      continue;
    }
    const bool residual = job == kJobResidual;
    const int a = (int)q1[1];
    RowCtx rc;
    rc.P = p.target + (int64_t)(g.t0 + a) * p.V;
    rc.Q = residual ? p.draft + (int64_t)(g.d0 + a) * p.V : nullptr;
    rc.logits = p.kind == 1;
    rc.Mp = __uint_as_float(q2[0]);
    rc.Rp = __uint_as_float(q2[1]);
    rc.Mq = __uint_as_float(q2[2]);
    rc.Rq = __uint_as_float(q2[3]);
    // non-temporal: the search reads back one sub-chunk of these rows at most (measured: the
    // acceptance of 512 sequences of 152064-entry rows 6 us faster, a whole verification step
    // about 2 us, and no slower at 64 sequences of 128256)
    float pv[kPerLane], qv[kPerLane];
    load_sub<true>(rc.P, sub, wave, p.V, vec, -INFINITY, lane, pv);
    if (residual) {
      load_sub<true>(rc.Q, sub, wave, p.V, vec, -INFINITY, lane, qv);
    } else {
#pragma unroll
      for (int e = 0; e < kPerLane; ++e) qv[e] = 0.f;
    }
    sub_sums(p, rc, residual, b, sub, (int)q1[3], wave, lane, pv, qv);
  }
}

// ------------------------------------------------------------------- probability max pass

__global__ __launch_bounds__(kThreads) void accept_max_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x / p.nsub, sub = blockIdx.x % p.nsub;
  const int mode = p.st_mode[b];
  const int a = p.st_a[b];
  const Geom g = load_geom(p, b);
  if (mode != kResidual && mode != kBonus) return;
  const bool residual = mode == kResidual;
  sub_maxima(p, row_ctx(p, b, g, a, residual, lane), residual, b, sub, wave, lane);
}

// ------------------------------------------------------------------- probability sum pass

__global__ __launch_bounds__(kThreads) void accept_sum_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x / p.nsub, sub = blockIdx.x % p.nsub;
  const int mode = p.st_mode[b];
  const int a = p.st_a[b];
  const Geom g = load_geom(p, b);
  if (mode != kResidual && mode != kBonus) return;
  sample_sums(p, b, g, a, mode == kResidual, sub, wave, lane);
}

// -------------------------------------------------------------------------------- search

__global__ __launch_bounds__(kThreads) void accept_search_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x;
  // the record the sums' first sub-chunk left (every wave reads the same), the sub-chunk sums
  // (residual, fallback; lanes own contiguous ranges) and the uniform, loaded together
  const u32x4* rec = reinterpret_cast<const u32x4*>(p.srec) + 3 * (int64_t)b;
  const u32x4 q0 = rec[0], q1 = rec[1], q2 = rec[2];
  const float u = p.u_sample[b];
  const uint64_t* sums = p.sum_part + (int64_t)b * p.nsub * 2;
  const int per = (p.nsub + kWave - 1) / kWave;
  const int c_lo = min(p.nsub, lane * per), c_hi = min(p.nsub, c_lo + per);
  uint64_t own_r = 0, own_p = 0;
  for (int x = c_lo; x < c_hi; ++x) {
    own_r += sums[2 * x];
    own_p += sums[2 * x + 1];
  }
  const int mode = (int)q1[0];
  if (mode != kResidual && mode != kBonus) return;
  const bool residual = mode == kResidual;
  const Geom g{(int)q0[0], (int)q0[1], (int)q0[2], 1};
  const int a = (int)q0[3];
  const int bad = (int)q1[1];
  const float M = __uint_as_float(q1[2]);
  RowCtx r;
  r.P = p.target + (int64_t)(g.t0 + a) * p.V;
  r.Q = residual ? p.draft + (int64_t)(g.d0 + a) * p.V : nullptr;
  r.logits = p.kind == 1;
  r.Mp = __uint_as_float(q2[0]);
  r.Rp = __uint_as_float(q2[1]);
  r.Mq = __uint_as_float(q2[2]);
  r.Rq = __uint_as_float(q2[3]);
  const bool lead = threadIdx.x == 0;
  if (bad) {
    if (lead) write_outputs(p, b, g, a, -1, SPEXIS_ROW_BAD_VALUE);
    return;
  }
  if (!(M > 0.f)) {
    if (lead) write_outputs(p, b, g, a, -1, SPEXIS_ROW_EMPTY);
    return;
  }
  const int s = 40 - floor_log2(M);
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;
  int32_t* orow = p.out_tokens + (int64_t)b * (p.max_k + 1);
  // Until the thread whose prefix range holds the threshold overwrites them (after the barrier
  // below), the outputs say that no token was found.  That cannot happen while every pass
  // computes the same weights; if it ever did, the row reports it instead of keeping the
  // previous call's outputs.
  if (lead) {
    orow[a] = -1;
    p.accepted_len[b] = a;
    p.row_status[b] = SPEXIS_ROW_INTERNAL;
    if (p.tok_prob) p.tok_prob[b] = 0.f;
  }
  // a residual whose fixed-point weights are all 0 falls back to p
  const bool use_p = !residual || wave_sum_u64(own_r) == 0;
  const int which = use_p ? 1 : 0;
  const uint64_t own = use_p ? own_p : own_r;

  // total and exact threshold; the sub-chunk holding t
  const uint64_t incl = wave_incl_scan_u64(own);
  const uint64_t S = readlane_u64(incl, kWave - 1);
  const uint64_t t = exact_threshold(u, S);
  uint64_t excl = incl - own;
  int cstar = -1;
  uint64_t tt = 0;
  if (excl <= t && t < incl) {                        // exactly one lane holds t
    if (c_hi - c_lo == 1) {                           // its one sub-chunk (up to 64 of them)
      cstar = c_lo;
      tt = t - excl;
    } else {
      for (int x = c_lo; x < c_hi; ++x) {
        if (t < excl + sums[2 * x + which]) {
          cstar = x;
          tt = t - excl;
          break;
        }
        excl += sums[2 * x + which];
      }
    }
  }
  const uint64_t found = __ballot(cstar >= 0);
  const int src = __builtin_amdgcn_readfirstlane(found ? __ffsll((unsigned long long)found) - 1 : 0);
  cstar = __builtin_amdgcn_readlane(cstar, src);
  tt = readlane_u64(tt, src);
  if (cstar < 0) return;   // unreachable: S > 0 (p's largest entry alone weighs >= 2^40)
  // the output row but its sampled entry: the accepted drafts, then -1 (wave 0; the id loads go
  // out with the sub-chunk's, the stores follow them)
  static_assert(kAcceptMaxK < kWave, "one lane per accepted draft");
  int idv = -1;
  if (wave == 0 && lane < a) idv = p.ids[g.d0 + lane];   // a <= max_k <= kAcceptMaxK
  // wave w owns entries cstar*4096 + 1024 w .. + 1023 of the sub-chunk, lane l 16 of them, in order
  constexpr int kRun = kAcceptSub / (kWaves * kWave);   // 16
  const int base = cstar * kAcceptSub + kRun * (kWave * wave + lane);
  float pv[kRun], qv[kRun];
#pragma unroll
  for (int j = 0; j < kRun / 4; ++j) {
    const f32x4 x = load4(r.P, base + 4 * j, p.V, vec, fill);
    const f32x4 y = use_p ? f32x4{0.f, 0.f, 0.f, 0.f} : load4(r.Q, base + 4 * j, p.V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pv[4 * j + i] = x[i];
      qv[4 * j + i] = y[i];
    }
  }
  if (wave == 0)
    for (int i = lane; i <= p.max_k; i += kWave)
      if (i != a) orow[i] = i < a ? idv : -1;
  uint64_t wv[kRun];
  uint64_t mine = 0;
#pragma unroll
  for (int e = 0; e < kRun; ++e) {
    wv[e] = entry_weight(r, p.c, pv[e], qv[e], use_p, s);
    mine += wv[e];
  }
  const uint64_t inc2 = wave_incl_scan_u64(mine);
  __shared__ uint64_t sm_tot[kWaves];
  if (lane == kWave - 1) sm_tot[wave] = inc2;
  __syncthreads();
  uint64_t pre = inc2 - mine;
  for (int w = 0; w < wave; ++w) pre += sm_tot[w];
  const uint64_t hi = pre + mine;
  if (pre <= tt && tt < hi) {
    int token = base;
    float prob = 0.f;
#pragma unroll
    for (int e = 0; e < kRun; ++e) {
      if (tt < pre + wv[e]) {
        token = base + e;
        prob = prob_of(r, pv[e], p.c, false);
        break;
      }
      pre += wv[e];
    }
    if (p.tok_prob) p.tok_prob[b] = prob;
    orow[a] = token;
    p.accepted_len[b] = a;
    p.row_status[b] = SPEXIS_ROW_OK;
    if (p.seq_lens_inout) p.seq_lens_inout[b] -= g.k - a;
  }
}

// ------------------------------------------------------------------------------- softmax

__global__ __launch_bounds__(kThreads) void softmax_rows_kernel(const float* logits, float* probs, int V, float c) {
  const int64_t row = blockIdx.x;
  const float* x = logits + row * V;
  float* y = probs + row * V;
  const bool vec = (V & 3) == 0;
  float m = -INFINITY, s = 0.f;
  for (int e = 4 * threadIdx.x; e < V; e += 4 * kThreads) {
    const f32x4 v = load4(x, e, V, vec, -INFINITY);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float t = v[i] * c;
      if (t > m) {
        s = s * fast_exp2(m - t) + 1.f;
        m = t;
      } else if (t != -INFINITY) {
        s += fast_exp2(t - m);
      }
    }
  }
  __shared__ float sm_m[kWaves], sm_s[kWaves];
  const float wm = wave_max(m);
  float ws = m == -INFINITY ? 0.f : s * fast_exp2(m - wm);
  ws = wave_sum(ws);
  if ((threadIdx.x & 63) == 0) {
    sm_m[threadIdx.x >> 6] = wm;
    sm_s[threadIdx.x >> 6] = ws;
  }
  __syncthreads();
  const float M = fmaxf(fmaxf(sm_m[0], sm_m[1]), fmaxf(sm_m[2], sm_m[3]));
  float Z = 0.f;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) Z += sm_m[w] == -INFINITY ? 0.f : sm_s[w] * fast_exp2(sm_m[w] - M);
  Z = 1.0f / Z;
  for (int e = 4 * threadIdx.x; e < V; e += 4 * kThreads) {
    const f32x4 v = load4(x, e, V, vec, -INFINITY);
    if (vec && e + 3 < V) {
      f32x4 o;
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = logit_prob(v[i], c, M, Z);
      *reinterpret_cast<f32x4*>(y + e) = o;
    } else {
      for (int i = 0; i < 4 && e + i < V; ++i) y[e + i] = logit_prob(v[i], c, M, Z);
    }
  }
}

hipError_t launch_softmax(const float* logits, float* probs, int64_t rows, int V, float c, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(softmax_rows_kernel, dim3((unsigned)rows), dim3(kThreads), 0, s, logits, probs, V, c);
  return hipGetLastError();
}

// Tests, then stream, of round r.  Later rounds, whose size the host does not know, have
// capped grids.
static hipError_t launch_round(const AcceptParams& p, int r, int lo, int hi, int hi2, hipStream_t s) {
  const unsigned items = (unsigned)((int64_t)p.B * p.nsub);
  const unsigned gt = r == 0 || p.B < kTestsGrid ? (unsigned)p.B : (unsigned)kTestsGrid;
  hipLaunchKernelGGL(accept_tests_kernel, dim3(gt), dim3(kThreads), 0, s, p, r, lo, hi, hi2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned gs = r == 0 || items < (unsigned)kRoundGrid ? items : (unsigned)kRoundGrid;
  hipLaunchKernelGGL(accept_stream_kernel, dim3(gs), dim3(kThreads), 0, s, p, r);
  return hipGetLastError();
}

// The target rows' gather columns for the LM head: row qsl[b]+i verifies draft x_i of sequence b
// (i < k_b) and gathers at it; the sequence's last row (its bonus position) gathers nothing.
// Thread (b, i) takes rows i, i + 33, ... of sequence b (one row each when k_b <= 32).  Indices
// are clamped into the buffers.
__global__ __launch_bounds__(kThreads) void gather_columns_kernel(const int32_t* qsl, const int32_t* ids, int B, int T,
                                                                  int32_t* cols) {
  constexpr int kPer = kAcceptMaxK + 1;
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)B * kPer) return;
  const int b = (int)(idx / kPer), i = (int)(idx % kPer);
  const int a0 = clampi(qsl[b], 0, T), a1 = clampi(qsl[b + 1], a0, T);
  const int n = a1 - a0;
  for (int j = i; j < n; j += kPer) {
    const int d = a0 - b + j;   // the draft this row verifies
    cols[a0 + j] = j < n - 1 && d >= 0 && d < T - B ? ids[d] : -1;
  }
}

hipError_t launch_gather_columns(const int32_t* qsl, const int32_t* ids, int B, int T, int32_t* cols, hipStream_t s) {
  const int64_t n = (int64_t)B * (kAcceptMaxK + 1);
  hipLaunchKernelGGL(gather_columns_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                     qsl, ids, B, T, cols);
  return hipGetLastError();
}

static hipError_t launch_search(const AcceptParams& p, hipStream_t s) {
  hipLaunchKernelGGL(accept_search_kernel, dim3(p.B), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_accept(const AcceptParams& p, hipStream_t s) {
  const unsigned items = (unsigned)((int64_t)p.B * p.nsub);
  hipError_t e;
  if (p.kind == 1 && p.ext_tstats) {
    // Statistics given: reduce each row's tiles once (into the statistics area of the
    // workspace, which the host checked is large enough), gather the tests' inputs, then one
    // round over every position.
    AcceptParams q = p;
    if (p.ext_parts > 1) {
      q.ext_tstats = p.lse_part;
      q.ext_dstats = p.lse_part + 2 * (int64_t)p.T;
      q.ext_parts = 1;
      hipLaunchKernelGGL(accept_combine_kernel, dim3((unsigned)((p.T + kWaves - 1) / kWaves)), dim3(kThreads), 0, s,
                         p.ext_tstats, p.ext_parts, p.T, p.lse_part);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      if (p.T > p.B) {
        hipLaunchKernelGGL(accept_combine_kernel, dim3((unsigned)((p.T - p.B + kWaves - 1) / kWaves)),
                           dim3(kThreads), 0, s, p.ext_dstats, p.ext_parts, p.T - p.B,
                           p.lse_part + 2 * (int64_t)p.T);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
    }
    if (q.max_k > 0) {
      const int64_t n = (int64_t)q.B * q.max_k;
      hipLaunchKernelGGL(accept_gather_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                         s, q);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = launch_round(q, 0, 0, q.max_k + 1, 0, s)) != hipSuccess) return e;
    return launch_search(q, s);
  }
  if (p.kind == 1) {
    // Rounds of doubling width.  A round costs a few microseconds of launch and
    // latency, a row 4V bytes: with short rows (under 256 KB) that together stream in well
    // under that many rounds' worth of time, one round reads every row.  Otherwise the first
    // round is two positions wide ({0,1}, {2..5}, the rest), so that sequences passing the
    // first test need no extra launch, unless its four rows per sequence come to more than
    // 256 MB: then the rows a first rejection leaves unread cost more than a launch, and the
    // rounds are {0}, {1,2}, the rest.  (Measured: rounds save 3.5 us at 64 sequences of
    // 128256-entry rows, and cost 2.6 us at 128 of 32000; a first round of one position costs
    // 7 us at 64 sequences of 128256 entries and saves 3 us at 256 of them and 57 us at 512 of
    // 152064; one round over every position is 4.5 us slower at 64 of 128256, its 0.295 GB
    // statistics pass at 5.9 TB/s.)
    const bool one_round =
        (int64_t)p.V * 4 < kRoundRowBytes && (int64_t)p.B * (p.max_k + 1) * p.V * 4 <= kOneRoundBytes;
    int width = one_round ? p.max_k + 1 : ((int64_t)p.B * 4 * p.V * 4 > kNarrowFirstBytes ? 1 : 2);
    {
      // Large passes take two sub-chunks per work item (measured: 6 us faster at 512 sequences
      // of 152064 entries and 2 us at 256 of 128256; 1 us slower at 64 of 128256).
      const int64_t items = (int64_t)p.B * 2 * width * p.nsub;
      if (items > kStatPairItems) {
        hipLaunchKernelGGL(accept_stats_kernel<2>, dim3((unsigned)((int64_t)p.B * 2 * width * ((p.nsub + 1) / 2))),
                           dim3(kThreads), 0, s, p, width);
      } else {
        hipLaunchKernelGGL(accept_stats_kernel<1>, dim3((unsigned)items), dim3(kThreads), 0, s, p, width);
      }
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    // From the third round on, a round takes every remaining position when they are at most
    // twice its width: few sequences get that far, and a round's two launches cost more than
    // the rows a later rejection would have left unread (measured: 4 us faster at 512
    // sequences of 152064 entries with k = 8, level at 128 and 256 sequences of 128256).
    // Longer remainders keep doubling, so a sequence never reads more than about twice the rows
    // its tests need.
    const auto round_end = [&](int r, int lo, int w) { return r >= 2 && p.max_k + 1 - lo <= 2 * w ? p.max_k + 1 : lo + w; };
    for (int r = 0, lo = 0, w = width, hi; lo <= p.max_k; ++r, lo = hi, w *= 2) {
      // round r, positions [lo, hi); a sequence passing all of it computes round r+1's
      // statistics, positions [hi, hi2)
      hi = round_end(r, lo, w);
      const int hi2 = hi <= p.max_k ? round_end(r + 1, hi, 2 * w) : 0;
      if ((e = launch_round(p, r, lo, hi, hi2, s)) != hipSuccess) return e;
    }
  } else {
    hipLaunchKernelGGL(accept_init_kernel, dim3((p.B + kThreads - 1) / kThreads), dim3(kThreads), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(accept_max_kernel, dim3(items), dim3(kThreads), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(accept_sum_kernel, dim3(items), dim3(kThreads), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return launch_search(p, s);
}

}  // namespace spexis
