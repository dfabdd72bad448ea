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
// Kernels, all on the caller's stream:
//   init        one thread per sequence: draft-id check, and in probability mode the tests
//   lse round i (logits mode, i = 0..max_k) over the sequences still testing: the statistics
//               (max, sum of 2^(y - max)) of target row i and draft row i, one wave per
//               4096-entry sub-chunk; the last work item of a sequence to finish combines the
//               sub-chunks in a fixed order and runs test i.  Only rows a sequence reaches are
//               read: a rejected or finished sequence leaves the next round's list.
//   max pass    per sub-chunk: max of the weights, max of p, bad-value flag
//   sum pass    per sub-chunk: sum of W_v; the last work item of a sequence scans the sub-chunk
//               sums, takes the exact threshold and finds the token inside one sub-chunk.
// Work items of one sequence communicate through the workspace: each producer issues a
// device-scope release fence before it counts itself in; only the last arrival acquires.
// Nothing ever waits on another workgroup.
#include <math.h>

#include "common.h"
#include "kernels.h"
#include "spexis.h"

namespace spexis {

constexpr int kThreads = 256;
constexpr int kF4 = kAcceptSub / (kWave * 4);   // float4 loads per lane per sub-chunk (16)
constexpr int kPerLane = 4 * kF4;                // vocab entries per lane per sub-chunk (64)

enum Mode { kTesting = 0, kResidual = 1, kBonus = 2, kDone = 3 };

struct Geom {
  int t0, d0, k, n;
};

__device__ __forceinline__ Geom seq_geom(const AcceptParams& p, int b) {
  Geom g;
  const int a0 = clampi(p.qsl[b], 0, p.T);
  const int a1 = clampi(p.qsl[b + 1], a0, p.T);
  g.n = a1 - a0;
  g.k = g.n - 1;
  if (g.k < 0) g.k = 0;
  if (g.k > p.max_k) g.k = p.max_k;
  g.t0 = a0;
  int nd = p.T - p.B;
  if (nd < 0) nd = 0;
  if (g.k > nd) g.k = nd;   // only reachable with an inconsistent qsl: stay inside the draft rows
  g.d0 = clampi(a0 - b, 0, nd - g.k);
  return g;
}

// p = 2^(x*c - M) / Z: the probability of a logit, the same expression in every pass.
__device__ __forceinline__ float logit_prob(float x, float c, float M, float Z) {
  return fast_exp2(x * c - M) / Z;
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
__device__ __forceinline__ void load_sub(const float* row, int sub, int V, bool vec, float fill, int lane,
                                         float (&v)[kPerLane]) {
#pragma unroll
  for (int j = 0; j < kF4; ++j) {
    const f32x4 x = load4(row, sub * kAcceptSub + j * 4 * kWave + 4 * lane, V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[4 * j + i] = x[i];
  }
}

// Count this work item in on the sequence's counter; true in the last of `expected` items.
// Producers: the partials written by any thread of the workgroup reach memory (barrier, then a
// device-scope release fence) before the count.  The last arrival acquires once.
__device__ __forceinline__ bool arrive_last(int32_t* ctr, int expected, int* sm_flag) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    const int prev = __hip_atomic_fetch_add(ctr, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const bool last = prev == expected - 1;
    if (last) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    *sm_flag = last;
  }
  __syncthreads();
  return *sm_flag != 0;
}

// Final outputs of sequence b (called by exactly one thread).
__device__ void write_outputs(const AcceptParams& p, int b, const Geom& g, int a, int token, int status) {
  int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
  for (int i = 0; i <= p.max_k; ++i) row[i] = i < a ? p.ids[g.d0 + i] : (i == a ? token : -1);
  p.accepted_len[b] = a;
  p.row_status[b] = status;
  if (p.seq_lens_inout) p.seq_lens_inout[b] -= g.k - a;
}

// ---------------------------------------------------------------------------------- init

__global__ __launch_bounds__(kThreads) void accept_init_kernel(AcceptParams p) {
  if (blockIdx.x == 0 && threadIdx.x < p.max_k + 2) p.counts[threadIdx.x] = 0;
  const int b = blockIdx.x * kThreads + threadIdx.x;
  if (b >= p.B) return;
  const Geom g = seq_geom(p, b);
  p.ctr[b] = 0;
  bool ok = g.n >= 1;
  for (int i = 0; ok && i < g.k; ++i) {
    const int x = p.ids[g.d0 + i];
    ok = x >= 0 && x < p.V;
  }
  if (!ok) {
    int32_t* row = p.out_tokens + (int64_t)b * (p.max_k + 1);
    for (int i = 0; i <= p.max_k; ++i) row[i] = -1;
    p.accepted_len[b] = 0;
    p.row_status[b] = g.n >= 1 ? SPEXIS_ROW_BAD_TOKEN : SPEXIS_ROW_BAD_VALUE;
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
    p.st_a[b] = 0;
    p.st_mode[b] = kTesting;
  }
}

// ---------------------------------------------------------------- logits: row statistics

// Combine the sub-chunk statistics of one row in a fixed order (one wave).
__device__ __forceinline__ void combine_lse(const float* part, int nsub, int lane, float& M, float& Z) {
  float mm = -INFINITY;
  for (int x = lane; x < nsub; x += kWave) mm = fmaxf(mm, part[2 * x]);
  mm = wave_max(mm);
  float zz = 0.f;
  if (mm != -INFINITY)
    for (int x = lane; x < nsub; x += kWave) zz += part[2 * x + 1] * fast_exp2(part[2 * x] - mm);
  M = mm;
  Z = wave_sum(zz);
}

__global__ __launch_bounds__(kThreads) void accept_lse_kernel(AcceptParams p, int i) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int nseq = i == 0 ? p.B : p.counts[i];
  const int64_t total = (int64_t)nseq * 2 * p.ipr;
  const bool vec = (p.V & 3) == 0;
  __shared__ int sm_flag;
  for (int64_t item = blockIdx.x; item < total; item += gridDim.x) {
    const int sidx = (int)(item / (2 * p.ipr));
    const int which = (int)((item / p.ipr) & 1);   // 0 target row i, 1 draft row i
    const int part = (int)(item % p.ipr);
    const int b = i == 0 ? sidx : p.lists[(int64_t)i * p.B + sidx];
    if (p.st_mode[b] != kTesting) continue;
    const Geom g = seq_geom(p, b);
    if (i > g.k || (which == 1 && i >= g.k)) continue;
    const float* row = which == 0 ? p.target + (int64_t)(g.t0 + i) * p.V : p.draft + (int64_t)(g.d0 + i) * p.V;
    for (int s = wave; s < kSubPerItem; s += kThreads / kWave) {
      const int sub = part * kSubPerItem + s;
      if (sub >= p.nsub) break;
      float v[kPerLane];
      load_sub(row, sub, p.V, vec, -INFINITY, lane, v);
      float m = -INFINITY;
#pragma unroll
      for (int e = 0; e < kPerLane; ++e) {
        v[e] *= p.c;
        m = fmaxf(m, v[e]);
      }
      m = wave_max(m);
      float z = 0.f;
      if (m != -INFINITY) {
#pragma unroll
        for (int e = 0; e < kPerLane; ++e) z += fast_exp2(v[e] - m);
      }
      z = wave_sum(z);
      if (lane == 0) {
        float* dst = p.lse_part + (((int64_t)which * p.B + b) * p.nsub + sub) * 2;
        dst[0] = m;
        dst[1] = z;
      }
    }
    const int expected = p.ipr * (i < g.k ? 2 : 1);
    if (!arrive_last(p.ctr + b, expected, &sm_flag)) continue;
    if (wave == 0) {
      float Mt, Zt, Md = 0.f, Zd = 1.f;
      combine_lse(p.lse_part + (int64_t)b * p.nsub * 2, p.nsub, lane, Mt, Zt);
      if (i < g.k) combine_lse(p.lse_part + ((int64_t)p.B + b) * p.nsub * 2, p.nsub, lane, Md, Zd);
      if (lane == 0) {
        float* rs = p.row_stats + ((int64_t)b * (p.max_k + 1) + i) * 4;
        rs[0] = Mt;
        rs[1] = Zt;
        rs[2] = Md;
        rs[3] = Zd;
        if (i < g.k) {
          const int x = p.ids[g.d0 + i];
          const float pp = logit_prob(p.target[(int64_t)(g.t0 + i) * p.V + x], p.c, Mt, Zt);
          const float qq = logit_prob(p.draft[(int64_t)(g.d0 + i) * p.V + x], p.c, Md, Zd);
          const double u = (double)p.u_accept[g.d0 + i];
          if (u * (double)qq < (double)pp) {
            p.st_a[b] = i + 1;   // still testing: the next round reads row i+1
            const int pos = __hip_atomic_fetch_add(p.counts + i + 1, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            p.lists[(int64_t)(i + 1) * p.B + pos] = b;
          } else {
            p.st_a[b] = i;
            p.st_mode[b] = kResidual;
          }
        } else {
          p.st_a[b] = g.k;
          p.st_mode[b] = kBonus;
        }
        p.ctr[b] = 0;
      }
    }
  }
}

// ------------------------------------------------------------------- weights of a vocab entry

struct RowCtx {
  const float* P;
  const float* Q;     // nullptr for the bonus row
  float Mp, Zp, Mq, Zq;
  bool logits;
};

__device__ __forceinline__ RowCtx row_ctx(const AcceptParams& p, int b, const Geom& g, int a, bool residual) {
  RowCtx r;
  r.P = p.target + (int64_t)(g.t0 + a) * p.V;
  r.Q = residual ? p.draft + (int64_t)(g.d0 + a) * p.V : nullptr;
  r.logits = p.kind == 1;
  r.Mp = r.Zp = r.Mq = r.Zq = 1.f;
  if (r.logits) {
    const float* rs = p.row_stats + ((int64_t)b * (p.max_k + 1) + a) * 4;
    r.Mp = rs[0];
    r.Zp = rs[1];
    r.Mq = rs[2];
    r.Zq = rs[3];
  }
  return r;
}

__device__ __forceinline__ float prob_of(const RowCtx& r, float raw, float c, bool draft) {
  if (!r.logits) return raw;
  return draft ? logit_prob(raw, c, r.Mq, r.Zq) : logit_prob(raw, c, r.Mp, r.Zp);
}

// ------------------------------------------------------------------------------ max pass

__global__ __launch_bounds__(kThreads) void accept_max_kernel(AcceptParams p) {
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int b = blockIdx.x / p.ipr;
  const int part = blockIdx.x % p.ipr;
  const int mode = p.st_mode[b];
  if (mode != kResidual && mode != kBonus) return;
  const Geom g = seq_geom(p, b);
  const bool residual = mode == kResidual;
  const RowCtx r = row_ctx(p, b, g, p.st_a[b], residual);
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;
  for (int s = wave; s < kSubPerItem; s += kThreads / kWave) {
    const int sub = part * kSubPerItem + s;
    if (sub >= p.nsub) break;
    float pv[kPerLane], qv[kPerLane];
    load_sub(r.P, sub, p.V, vec, fill, lane, pv);
    if (residual) load_sub(r.Q, sub, p.V, vec, fill, lane, qv);
    float mw = 0.f, mp = 0.f;
    int bad = 0;
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) {
      const float P = prob_of(r, pv[e], p.c, false);
      const float Q = residual ? prob_of(r, qv[e], p.c, true) : 0.f;
      bad |= bad_value(P) | (residual && bad_value(Q));
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
  const int part = blockIdx.x % p.ipr;
  const int mode = p.st_mode[b];
  if (mode != kResidual && mode != kBonus) return;
  const Geom g = seq_geom(p, b);
  const int a = p.st_a[b];
  const bool residual = mode == kResidual;
  __shared__ float sm_f[2][kThreads / kWave];
  __shared__ int sm_i[kThreads / kWave];
  __shared__ int sm_flag;

  // the max pass of the whole row (every work item of the sequence combines it the same way)
  float MW = 0.f, MP = 0.f;
  int bad = 0;
  for (int x = threadIdx.x; x < p.nsub; x += kThreads) {
    MW = fmaxf(MW, p.max_part[((int64_t)b * p.nsub + x) * 2]);
    MP = fmaxf(MP, p.max_part[((int64_t)b * p.nsub + x) * 2 + 1]);
    bad |= p.bad_part[(int64_t)b * p.nsub + x];
  }
  MW = wave_max(MW);
  MP = wave_max(MP);
  bad = wave_or(bad);
  if (lane == 0) {
    sm_f[0][wave] = MW;
    sm_f[1][wave] = MP;
    sm_i[wave] = bad;
  }
  __syncthreads();
  MW = fmaxf(fmaxf(sm_f[0][0], sm_f[0][1]), fmaxf(sm_f[0][2], sm_f[0][3]));
  MP = fmaxf(fmaxf(sm_f[1][0], sm_f[1][1]), fmaxf(sm_f[1][2], sm_f[1][3]));
  bad = sm_i[0] | sm_i[1] | sm_i[2] | sm_i[3];
  if (bad) {
    if (part == 0 && threadIdx.x == 0) write_outputs(p, b, g, a, -1, SPEXIS_ROW_BAD_VALUE);
    return;
  }
  const bool use_p = !residual || MW == 0.f;   // empty residual: fall back to p_a
  const float M = use_p ? MP : MW;
  if (!(M > 0.f)) {
    if (part == 0 && threadIdx.x == 0) write_outputs(p, b, g, a, -1, SPEXIS_ROW_EMPTY);
    return;
  }
  const int s = 40 - floor_log2(M);
  const RowCtx r = row_ctx(p, b, g, a, residual);
  const bool vec = (p.V & 3) == 0;
  const float fill = r.logits ? -INFINITY : 0.f;
  for (int sc = wave; sc < kSubPerItem; sc += kThreads / kWave) {
    const int sub = part * kSubPerItem + sc;
    if (sub >= p.nsub) break;
    float pv[kPerLane], qv[kPerLane];
    load_sub(r.P, sub, p.V, vec, fill, lane, pv);
    if (!use_p) load_sub(r.Q, sub, p.V, vec, fill, lane, qv);
    uint64_t sum = 0;
#pragma unroll
    for (int e = 0; e < kPerLane; ++e) sum += entry_weight(r, p.c, pv[e], use_p ? 0.f : qv[e], use_p, s);
    sum = wave_sum_u64(sum);
    if (lane == 0) p.sum_part[(int64_t)b * p.nsub + sub] = sum;
  }
  if (!arrive_last(p.ctr + b, p.ipr, &sm_flag)) return;
  if (wave != 0) return;

  // ---- last work item of sequence b, one wave: total, exact threshold, sub-chunk, token
  const uint64_t* sums = p.sum_part + (int64_t)b * p.nsub;
  const int per = (p.nsub + kWave - 1) / kWave;       // contiguous sub-chunk range of this lane
  const int c_lo = min(p.nsub, lane * per), c_hi = min(p.nsub, c_lo + per);
  uint64_t own = 0;
  for (int x = c_lo; x < c_hi; ++x) own += sums[x];
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
  // broadcast (cstar, tt) from the lane that found them
  const uint64_t found = __ballot(cstar >= 0);
  const int src = found ? __ffsll((unsigned long long)found) - 1 : 0;
  cstar = __shfl(cstar, src, kWave);
  tt = __shfl(tt, src, kWave);
  if (cstar < 0) return;   // unreachable: S > 0 because M > 0 gives a weight >= 2^40
  // lane l owns entries cstar*4096 + 64 l .. + 63 of the sub-chunk, in order
  const int base = cstar * kAcceptSub + kPerLane * lane;
  uint64_t wv[kPerLane];
  uint64_t mine = 0;
#pragma unroll
  for (int j = 0; j < kF4; ++j) {
    const f32x4 pv4 = load4(r.P, base + 4 * j, p.V, vec, fill);
    f32x4 qv4 = {0.f, 0.f, 0.f, 0.f};
    if (!use_p) qv4 = load4(r.Q, base + 4 * j, p.V, vec, fill);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      wv[4 * j + i] = entry_weight(r, p.c, pv4[i], qv4[i], use_p, s);
      mine += wv[4 * j + i];
    }
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
  if (lane == 0) p.ctr[b] = 0;
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
  __shared__ float sm_m[4], sm_s[4];
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
  for (int w = 0; w < 4; ++w) Z += sm_m[w] == -INFINITY ? 0.f : sm_s[w] * fast_exp2(sm_m[w] - M);
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
  if (p.kind == 1) {
    // bounded grid: work items of the sequences still testing are strided over it
    const int64_t items = (int64_t)p.B * 2 * p.ipr;
    const unsigned grid = (unsigned)(items < 1024 ? items : 1024);
    for (int i = 0; i <= p.max_k; ++i) {
      hipLaunchKernelGGL(accept_lse_kernel, dim3(grid), dim3(kThreads), 0, s, p, i);
      if ((e = hipGetLastError()) != hipSuccess) return e;
    }
  }
  const unsigned grid = (unsigned)((int64_t)p.B * p.ipr);
  hipLaunchKernelGGL(accept_max_kernel, dim3(grid), dim3(kThreads), 0, s, p);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(accept_sum_kernel, dim3(grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace spexis
