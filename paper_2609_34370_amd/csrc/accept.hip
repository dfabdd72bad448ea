// Speculative-sampling acceptance (the rule of [sd] the paper builds on, Related Work; its use
// in verification, Sec. 4 and Fig. 3): ratio tests on the drafts, then one inverse-CDF sample
// from the residual max(0, p - q) at the first rejection, or from p_k when every draft passes.
//
// Every decision is taken in exact arithmetic, so any reduction order gives the same integers:
//   test      (double)u * (double)q(x) < (double)p(x)   (a product of two fp32 is exact)
//   weights   W_v = floor(w_v * 2^(40-e)), e = floor(log2 max w)   (integer bit shifts)
//   threshold t = floor(u * sum W) from a 128-bit product
//   token     the smallest m whose inclusive prefix of W exceeds t
//
// Kernels, in order on the caller's stream (kernel boundaries are the only synchronisation;
// the one atomic appends a sequence to the next round's list):
//   init      one thread per sequence: geometry, draft-id check; with probability inputs
//             also the ratio tests.
//   round i   (logit inputs, i = 0..max_k) one work item per (sequence still testing, 8
//             sub-chunks of 4096 entries), one wave per sub-chunk.  An item first re-derives
//             test i-1 from the row statistics round i-1 left (every item of a sequence
//             reaches the same decision).  Accepted: it computes the statistics
//             (max, sum of 2^(y - max)) of target row i and draft row i over its entries, and
//             the sequence moves to round i+1 (or, at i = k, is done with the bonus row k).
//             Rejected: it computes the residual maxima of row i-1 over its entries instead.
//             Only rows a sequence reaches are read.  Statistics alternate between two
//             buffers by round parity, so a round never overwrites what it reads.
//   max pass  (probability inputs) per sub-chunk: max of the weights, max of p, bad flag.
//   sum pass  per sub-chunk: sum of W_v.
//   search    one wave per sequence: total, exact threshold, the sub-chunk holding it, the
//             token inside that sub-chunk, outputs.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "spexis.h"

namespace spexis {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kF4 = kAcceptSub / (kWave * 4);   // float4 loads per lane per sub-chunk (16)
constexpr int kPerLane = 4 * kF4;                // vocab entries per lane per sub-chunk (64)

enum Mode { kTesting = 0, kResidual = 1, kBonus = 2, kDone = 3 };

struct Geom {
  int t0, d0, k, valid;
};

__device__ __forceinline__ Geom load_geom(const AcceptParams& p, int b) {
  const u32x4 v = *reinterpret_cast<const u32x4*>(p.geo + 4 * (int64_t)b);
  return Geom{(int)v[0], (int)v[1], (int)v[2], (int)v[3]};
}

// p = 2^(x*c - M) * (1/Z): the probability of a logit, the same expression in every pass
// (R = 1/Z is rounded once per row).
__device__ __forceinline__ float logit_prob(float x, float c, float M, float R) {
  return fast_exp2(x * c - M) * R;
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

// One wave's coalesced view of sub-chunk `sub`: lane l holds entries sub*4096 + 256 j + 4 l + i.
// A sub-chunk inside the row (all but the last of a row whose length is a multiple of 4) takes
// the straight-line path, so all 16 loads are in flight together.
__device__ __forceinline__ void load_sub(const float* row, int sub, int V, bool vec, float fill, int lane,
                                         float (&v)[kPerLane]) {
  if (vec && (sub + 1) * kAcceptSub <= V) {
    const f32x4* src = reinterpret_cast<const f32x4*>(row + sub * kAcceptSub) + lane;
#pragma unroll
    for (int j = 0; j < kF4; ++j) {
      const f32x4 x = src[j * kWave];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kF4; ++j) {
    const f32x4 x = load4(row, sub * kAcceptSub + j * 4 * kWave + 4 * lane, V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
  }
}

// The 64 consecutive entries base .. base+63 of one lane (base % 4 == 0), same fast path.
__device__ __forceinline__ void load_run(const float* row, int base, int V, bool vec, float fill,
                                         float (&v)[kPerLane]) {
  if (vec && base + kPerLane <= V) {
    const f32x4* src = reinterpret_cast<const f32x4*>(row + base);
#pragma unroll
    for (int j = 0; j < kF4; ++j) {
      const f32x4 x = src[j];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kF4; ++j) {
    const f32x4 x = load4(row, base + 4 * j, V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
  }
}

// Statistics of one logit row from its sub-chunk partials, combined in a fixed order by one
// full wave (every consumer calls exactly this, so all of them get identical M and 1/Z, the
// latter returned in Z).  A row without a finite maximum or with a bad sum gives Z = NaN.
__device__ __forceinline__ void row_stats(const float* part, int nsub, int lane, float& M, float& Z) {
  float mm = -INFINITY;
  for (int x = lane; x < nsub; x += kWave) mm = fmaxf(mm, part[2 * x]);
  mm = wave_max(mm);
  float zz = 0.f;
  int nan = 0;
  for (int x = lane; x < nsub; x += kWave) {
    const float z = part[2 * x + 1];
    nan |= z != z;
    if (part[2 * x] != -INFINITY) zz += z * fast_exp2(part[2 * x] - mm);
  }
  zz = wave_sum(zz);
  nan = wave_or(nan);
  M = mm;
  Z = (nan || !(mm > -INFINITY) || !(mm < INFINITY)) ? NAN : 1.0f / zz;   // reciprocal of the sum
}

__device__ __forceinline__ float* lse_slot(const AcceptParams& p, int parity, int which, int b) {
  return p.lse_part + ((((int64_t)parity * 2 + which) * p.B + b) * p.nsub) * 2;
}

// Final outputs of sequence b (called by exactly one thread).
__device__ void write_outputs(const AcceptParams& p, int b, const Geom& g, int a, int token, int status) {
  int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
  for (int i = 0; i <= p.max_k; ++i) row[i] = i < a ? p.ids[g.d0 + i] : (i == a ? token : -1);
  p.accepted_len[b] = a;
  p.row_status[b] = status;
  if (p.seq_lens_inout) p.seq_lens_inout[b] -= g.k - a;
}

// Row context of the sampled row(s): target row a (P) and, for a residual, draft row a (Q).
struct RowCtx {
  const float* P;
  const float* Q;     // nullptr for the bonus row
  float Mp, Rp, Mq, Rq;  // row maxima (scaled) and reciprocal sums (logits mode)
  bool logits;
};

__device__ __forceinline__ float prob_of(const RowCtx& r, float raw, float c, bool draft) {
  if (!r.logits) return raw;
  return draft ? logit_prob(raw, c, r.Mq, r.Rq) : logit_prob(raw, c, r.Mp, r.Rp);
}

// Residual / bonus maxima of one sub-chunk by one wave, written to max_part / bad_part.
__device__ void sub_maxima(const AcceptParams& p, const RowCtx& r, bool residual, int b, int sub, int lane) {
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;
  float pv[kPerLane], qv[kPerLane];
  load_sub(r.P, sub, p.V, vec, fill, lane, pv);
  if (residual) load_sub(r.Q, sub, p.V, vec, fill, lane, qv);
  float mw = 0.f, mp = 0.f;
  int bad = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    const float P = prob_of(r, pv[e], p.c, false);
    const float Q = residual ? prob_of(r, qv[e], p.c, true) : 0.f;
    bad |= bad_value(P) || (residual && bad_value(Q));
    const float d = P - Q;
    const float w = residual ? (d > 0.f ? d : 0.f) : P;
    mw = w > mw ? w : mw;
    mp = P > mp ? P : mp;
  }
  mw = wave_max(mw);
  mp = wave_max(mp);
  bad = wave_or(bad);
  if (lane == 0) {
    p.max_part[((int64_t)b * p.nsub + sub) * 2] = mw;
    p.max_part[((int64_t)b * p.nsub + sub) * 2 + 1] = mp;
    p.bad_part[(int64_t)b * p.nsub + sub] = bad;
  }
}

// ---------------------------------------------------------------------------------- init

__global__ __launch_bounds__(kThreads) void accept_init_kernel(AcceptParams p) {
  if (blockIdx.x == 0 && threadIdx.x < p.max_k + 2) p.counts[threadIdx.x] = 0;
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b >= p.B) return;
  const int a0 = clampi(p.qsl[b], 0, p.T);
  const int a1 = clampi(p.qsl[b + 1], a0, p.T);
  const int n = a1 - a0;
  int nd = p.T - p.B;
  if (nd < 0) nd = 0;
  int k = n - 1;
  if (k < 0) k = 0;
  if (k > p.max_k) k = p.max_k;
  if (k > nd) k = nd;   // only reachable with an inconsistent qsl: stay inside the draft rows
  const Geom g{a0, clampi(a0 - b, 0, nd - k), k, 0};
  bool ok = n >= 1;
  for (int i = 0; ok && i < g.k; ++i) {
    const int x = p.ids[g.d0 + i];
    ok = x >= 0 && x < p.V;
  }
  *reinterpret_cast<u32x4*>(p.geo + 4 * (int64_t)b) = u32x4{(uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k, ok ? 1u : 0u};
  if (!ok) {
    int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
    for (int i = 0; i <= p.max_k; ++i) row[i] = -1;
    p.accepted_len[b] = 0;
    p.row_status[b] = n >= 1 ? SPEXIS_ROW_BAD_TOKEN : SPEXIS_ROW_BAD_VALUE;
    p.st_mode[b] = kDone;
    p.st_a[b] = 0;
    return;
  }
  if (p.kind == 0) {
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
  } else {
    // the inputs of every test, gathered now so that a round needs no dependent gather
    for (int i = 0; i < g.k; ++i) {
      const int x = p.ids[g.d0 + i];
      f32x4 t;
      t[0] = p.target[(int64_t)(g.t0 + i) * p.V + x];
      t[1] = p.draft[(int64_t)(g.d0 + i) * p.V + x];
      t[2] = p.u_accept[g.d0 + i];
      t[3] = 0.f;
      *reinterpret_cast<f32x4*>(p.tin + ((int64_t)b * p.max_k + i) * 4) = t;
    }
    p.st_a[b] = 0;
    p.st_mode[b] = kTesting;
  }
}

// ---------------------------------------------------------------- logits: one test round

// (max, sum of 2^(y - max)) of one wave's 64 entries per lane; NaN sum if a logit is NaN/+inf.
__device__ __forceinline__ void sub_stats(float (&v)[kPerLane], float c, float& m, float& z) {
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

__global__ __launch_bounds__(kThreads) void accept_round_kernel(AcceptParams p, int i) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nseq = i == 0 ? p.B : p.counts[i];
  const int64_t total = (int64_t)nseq * p.ipr;
  const bool vec = (p.V & 3) == 0;
  for (int64_t item = blockIdx.x; item < total; item += gridDim.x) {
    const int sidx = (int)(item / p.ipr);
    const int part = (int)(item % p.ipr);
    const int sub = part * kSubPerItem + wave;   // this wave's sub-chunk
    const bool has = sub < p.nsub;
    int b;
    Geom g;
    if (i == 0) {
      b = sidx;
      g = load_geom(p, b);
      if (!g.valid) continue;
    } else {
      const u32x4 e = *reinterpret_cast<const u32x4*>(p.lists + ((int64_t)i * p.B + sidx) * 4);
      b = (int)e[0];
      g = Geom{(int)e[1], (int)e[2], (int)e[3], 1};
    }
    bool reject = false;
    RowCtx r;
    if (i >= 1) {
      // test i-1 from the statistics round i-1 left (same decision in every wave of every item)
      const f32x4 t = *reinterpret_cast<const f32x4*>(p.tin + ((int64_t)b * p.max_k + i - 1) * 4);
      r.P = p.target + (int64_t)(g.t0 + i - 1) * p.V;
      r.Q = p.draft + (int64_t)(g.d0 + i - 1) * p.V;
      r.logits = true;
      row_stats(lse_slot(p, (i - 1) & 1, 0, b), p.nsub, lane, r.Mp, r.Rp);
      row_stats(lse_slot(p, (i - 1) & 1, 1, b), p.nsub, lane, r.Mq, r.Rq);
      const float pp = logit_prob(t[0], p.c, r.Mp, r.Rp);
      const float qq = logit_prob(t[1], p.c, r.Mq, r.Rq);
      reject = !((double)t[2] * (double)qq < (double)pp);
    }
    if (reject) {
      // the sequence stops at a = i-1: residual maxima of row i-1 over this item's entries
      if (has) sub_maxima(p, r, true, b, sub, lane);
      if (part == 0 && threadIdx.x == 0) {
        p.st_a[b] = i - 1;
        p.st_mode[b] = kResidual;
      }
      continue;
    }
    // accepted (or i = 0): statistics of target row i, and of draft row i while i < k
    const bool two = i < g.k;
    if (has) {
      float vt[kPerLane], vd[kPerLane];
      load_sub(p.target + (int64_t)(g.t0 + i) * p.V, sub, p.V, vec, -INFINITY, lane, vt);
      if (two) load_sub(p.draft + (int64_t)(g.d0 + i) * p.V, sub, p.V, vec, -INFINITY, lane, vd);
      float m, z;
      sub_stats(vt, p.c, m, z);
      if (lane == 0) {
        float* dst = lse_slot(p, i & 1, 0, b) + 2 * sub;
        dst[0] = m;
        dst[1] = z;
      }
      if (two) {
        sub_stats(vd, p.c, m, z);
        if (lane == 0) {
          float* dst = lse_slot(p, i & 1, 1, b) + 2 * sub;
          dst[0] = m;
          dst[1] = z;
        }
      }
    }
    if (part == 0 && threadIdx.x == 0) {
      if (two) {
        const int pos = __hip_atomic_fetch_add(p.counts + i + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *reinterpret_cast<u32x4*>(p.lists + ((int64_t)(i + 1) * p.B + pos) * 4) =
            u32x4{(uint32_t)b, (uint32_t)g.t0, (uint32_t)g.d0, (uint32_t)g.k};
      } else {
        p.st_a[b] = g.k;
        p.st_mode[b] = kBonus;
      }
    }
  }
}

// Context of the sampled row of sequence b after the tests (computed identically everywhere).
__device__ __forceinline__ RowCtx sampled_row(const AcceptParams& p, int b, const Geom& g, int a, bool residual,
                                              int lane) {
  RowCtx r;
  r.P = p.target + (int64_t)(g.t0 + a) * p.V;
  r.Q = residual ? p.draft + (int64_t)(g.d0 + a) * p.V : nullptr;
  r.logits = p.kind == 1;
  r.Mp = r.Rp = r.Mq = r.Rq = 1.f;
  if (r.logits) {
    row_stats(lse_slot(p, a & 1, 0, b), p.nsub, lane, r.Mp, r.Rp);
    if (residual) row_stats(lse_slot(p, a & 1, 1, b), p.nsub, lane, r.Mq, r.Rq);
  }
  return r;
}

// Row maxima and bad flag of the sampled row (one wave; any reduction order gives the same).
// Logit bonus rows have no max pass: their largest probability is 2^0 * (1/Z).
__device__ __forceinline__ void sampled_maxima(const AcceptParams& p, const RowCtx& r, int b, bool residual, int lane,
                                               float& MW, float& MP, int& bad) {
  if (r.logits && !residual) {
    MP = MW = r.Rp;   // 2^0 * (1/Z)
    bad = !(MP > 0.f) || isinf(MP);
    return;
  }
  MW = 0.f;
  MP = 0.f;
  bad = 0;
  for (int x = lane; x < p.nsub; x += kWave) {
    MW = fmaxf(MW, p.max_part[((int64_t)b * p.nsub + x) * 2]);
    MP = fmaxf(MP, p.max_part[((int64_t)b * p.nsub + x) * 2 + 1]);
    bad |= p.bad_part[(int64_t)b * p.nsub + x];
  }
  MW = wave_max(MW);
  MP = wave_max(MP);
  bad = wave_or(bad);
}

// ------------------------------------------------------------------- probability max pass

__global__ __launch_bounds__(kThreads) void accept_max_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x / p.ipr;
  const int sub = (blockIdx.x % p.ipr) * kSubPerItem + wave;
  const int mode = p.st_mode[b];
  const int a = p.st_a[b];
  const Geom g = load_geom(p, b);
  if ((mode != kResidual && mode != kBonus) || sub >= p.nsub) return;
  const bool residual = mode == kResidual;
  const RowCtx r = sampled_row(p, b, g, a, residual, lane);
  sub_maxima(p, r, residual, b, sub, lane);
}

// ------------------------------------------------------------------------------ sum pass

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

__global__ __launch_bounds__(kThreads) void accept_sum_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x / p.ipr;
  const int sub = (blockIdx.x % p.ipr) * kSubPerItem + wave;
  const int mode = p.st_mode[b];
  const int a = p.st_a[b];
  const Geom g = load_geom(p, b);
  if ((mode != kResidual && mode != kBonus) || sub >= p.nsub) return;
  const bool residual = mode == kResidual;
  const RowCtx r = sampled_row(p, b, g, a, residual, lane);
  float MW, MP;
  int bad;
  sampled_maxima(p, r, b, residual, lane, MW, MP, bad);
  const bool use_p = !residual || MW == 0.f;   // empty residual: fall back to p_a
  const float M = use_p ? MP : MW;
  if (bad || !(M > 0.f)) return;                // the search kernel writes these outputs
  const int s = 40 - floor_log2(M);
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;
  float pv[kPerLane], qv[kPerLane];
  load_sub(r.P, sub, p.V, vec, fill, lane, pv);
  if (!use_p) load_sub(r.Q, sub, p.V, vec, fill, lane, qv);
  uint64_t sum = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) sum += entry_weight(r, p.c, pv[e], use_p ? 0.f : qv[e], use_p, s);
  sum = wave_sum_u64(sum);
  if (lane == 0) p.sum_part[(int64_t)b * p.nsub + sub] = sum;
}

// -------------------------------------------------------------------------------- search

__global__ __launch_bounds__(kThreads) void accept_search_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x * kWaves + wave;
  if (b >= p.B) return;
  const int mode = p.st_mode[b];
  const int a = p.st_a[b];
  const Geom g = load_geom(p, b);
  if (mode != kResidual && mode != kBonus) return;
  const bool residual = mode == kResidual;
  const RowCtx r = sampled_row(p, b, g, a, residual, lane);
  float MW, MP;
  int bad;
  sampled_maxima(p, r, b, residual, lane, MW, MP, bad);
  // the sub-chunk sums, prefetched while the maxima reduce (lanes own contiguous ranges)
  const uint64_t* sums = p.sum_part + (int64_t)b * p.nsub;
  const int per = (p.nsub + kWave - 1) / kWave;
  const int c_lo = min(p.nsub, lane * per), c_hi = min(p.nsub, c_lo + per);
  uint64_t own = 0;
  for (int x = c_lo; x < c_hi; ++x) own += sums[x];
  if (bad) {
    if (lane == 0) write_outputs(p, b, g, a, -1, SPEXIS_ROW_BAD_VALUE);
    return;
  }
  const bool use_p = !residual || MW == 0.f;
  const float M = use_p ? MP : MW;
  if (!(M > 0.f)) {
    if (lane == 0) write_outputs(p, b, g, a, -1, SPEXIS_ROW_EMPTY);
    return;
  }
  const int s = 40 - floor_log2(M);
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;

  // total and exact threshold; the sub-chunk holding t
  uint64_t incl = own;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint64_t y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  const uint64_t S = __shfl(incl, kWave - 1, kWave);
  const uint64_t t = exact_threshold(p.u_sample[b], S);
  uint64_t excl = incl - own;
  int cstar = -1;
  uint64_t tt = 0;
  if (excl <= t && t < incl) {                        // exactly one lane holds t
    for (int x = c_lo; x < c_hi; ++x) {
      if (t < excl + sums[x]) {
        cstar = x;
        tt = t - excl;
        break;
      }
      excl += sums[x];
    }
  }
  const uint64_t found = __ballot(cstar >= 0);
  const int src = found ? __ffsll((unsigned long long)found) - 1 : 0;
  cstar = __shfl(cstar, src, kWave);
  tt = __shfl(tt, src, kWave);
  if (cstar < 0) return;   // unreachable: S > 0 because M > 0 gives a weight >= 2^40
  // lane l owns entries cstar*4096 + 64 l .. + 63 of the sub-chunk, in order
  const int base = cstar * kAcceptSub + kPerLane * lane;
  float pv[kPerLane], qv[kPerLane];
  load_run(r.P, base, p.V, vec, fill, pv);
  if (!use_p) load_run(r.Q, base, p.V, vec, fill, qv);
  uint64_t wv[kPerLane];
  uint64_t mine = 0;
#pragma unroll
  for (int e = 0; e < kPerLane; ++e) {
    wv[e] = entry_weight(r, p.c, pv[e], use_p ? 0.f : qv[e], use_p, s);
    mine += wv[e];
  }
  uint64_t inc2 = mine;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint64_t y = __shfl_up(inc2, o, kWave);
    if (lane >= o) inc2 += y;
  }
  uint64_t pre = inc2 - mine;
  if (pre <= tt && tt < inc2) {
    int token = base;
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) {
      if (tt < pre + wv[e]) {
        token = base + e;
        break;
      }
      pre += wv[e];
    }
    write_outputs(p, b, g, a, token, SPEXIS_ROW_OK);
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

hipError_t launch_accept(const AcceptParams& p, hipStream_t s) {
  hipLaunchKernelGGL(accept_init_kernel, dim3((p.B + kThreads - 1) / kThreads), dim3(kThreads), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned items = (unsigned)((int64_t)p.B * p.ipr);
  if (p.kind == 1) {
    // bounded grid: the work items of the sequences still testing are strided over it
    const unsigned grid = items < 2048 ? items : 2048;
    for (int i = 0; i <= p.max_k; ++i) {
      hipLaunchKernelGGL(accept_round_kernel, dim3(grid), dim3(kThreads), 0, s, p, i);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  } else {
    hipLaunchKernelGGL(accept_max_kernel, dim3(items), dim3(kThreads), 0, s, p);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(accept_sum_kernel, dim3(items), dim3(kThreads), 0, s, p);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(accept_search_kernel, dim3((p.B + kWaves - 1) / kWaves), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace spexis
