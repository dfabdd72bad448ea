// Look-ahead KV-memory estimate (Sec. 5, Remaining-Length-Aware Scheduling; Algorithm 1).
//
// For look-ahead iteration i of a pipeline of depth pp whose speculation is accepted with
// probability theta, a request with w rejections has accepted t = i - pp*w tokens and generated
// k = t + w, with probability p(i, w) = C(k, t) theta^t (1 - theta)^w, w = 0 .. floor(i/pp).
// From those terms:
//   E_gen  = sum_w k p(i, w)
//   Pfin_r = prec_r * sum_w [k >= remaining_r] p(i, w)
//   mem_i  = L_total + (n - sum_r Pfin_r) E_gen - sum_r cur_len_r Pfin_r.
//
// One workgroup per iteration i (fp64 throughout).  Wave 0 computes the w terms 64 at a time
// and stores their running sums S(w) = p(i, 0) + .. + p(i, w) in LDS (DPP scans), while every
// thread's first requests are already loading.  k = i - (pp - 1) w never rises with w, so the w
// with k >= remaining_r are a prefix 0 .. w*_r of the terms and Pfin_r = prec_r S(w*_r): each
// request costs O(1).  Requests are taken eight per thread per pass, loads issued together; the
// sums over requests reduce in a fixed order (lanes by DPP, then waves).
#include "common.h"
#include "kernels.h"

namespace spexis {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kUnroll = 8;

// x^e for e >= 0 by repeated squaring (0^0 = 1).
__device__ __forceinline__ double powi(double x, int e) {
  double r = 1.0;
  while (e > 0) {
    if (e & 1) r *= x;
    x *= x;
    e >>= 1;
  }
  return r;
}

// The DPP lane moves of the integer wave scan, on an fp64 value (both halves move together;
// lanes not written get +0).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double update_dpp_f64(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, kRowMask, 0xF, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, kRowMask, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ double readlane_f64(double v, int lane) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), lane);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Inclusive prefix sum of fp64 values over the lanes of a wave, in the order of the integer scan.
__device__ __forceinline__ double wave_incl_scan_f64(double v) {
  v += update_dpp_f64<kDppRowShr + 1, 0xF>(v);
  v += update_dpp_f64<kDppRowShr + 2, 0xF>(v);
  v += update_dpp_f64<kDppRowShr + 4, 0xF>(v);
  v += update_dpp_f64<kDppRowShr + 8, 0xF>(v);
  v += update_dpp_f64<kDppRowBcast15, 0xA>(v);
  v += update_dpp_f64<kDppRowBcast31, 0xC>(v);
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
  return readlane_f64(wave_incl_scan_f64(v), kWave - 1);
}

}  // namespace

__global__ __launch_bounds__(kThreads) void lookahead_kernel(LookaheadParams p) {
  __shared__ double S[kLookaheadMaxIters + 1];   // running sums of p(i, w) over w
  __shared__ double red[3][kWaves];
  __shared__ double gen_sm;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int i = blockIdx.x + 1;
  const int w_max = i / p.pp;
  const int n = p.n;

  // this thread's first kUnroll requests, in flight during the table build
  int64_t len[kUnroll] = {};
  int32_t tau[kUnroll] = {};
  double prec[kUnroll] = {};
  auto load = [&](int base) {   // indices clamped into [0, n): n > 0 here
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = min(base + (int)threadIdx.x + kThreads * u, n - 1);
      len[u] = p.cur_len[r];
      tau[u] = p.remaining[r];
      prec[u] = p.prec[r];
    }
  };
  if (n > 0) load(0);

  if (wave == 0) {
    const double th = p.theta, nth = 1.0 - p.theta;
    double carry = 0.0, gen = 0.0;
    for (int base = 0; base <= w_max; base += kWave) {
      const int w = base + lane;
      double term = 0.0;
      if (w <= w_max) {
        const int t = i - p.pp * w, k = t + w;
        const int lo = min(t, w);   // C(k, t) = C(k, w) = prod_{j=1..lo} (k - lo + j) / j
        double c = 1.0;
        for (int j = 1; j <= lo; ++j) c = c * (double)(k - lo + j) / (double)j;
        term = c * powi(th, t) * powi(nth, w);
        gen += (double)k * term;
      }
      const double run = carry + wave_incl_scan_f64(term);
      if (w <= w_max) S[w] = run;
      carry = readlane_f64(run, kWave - 1);
    }
    gen = wave_sum_f64(gen);
    if (lane == 0) gen_sm = gen;
  }
  __syncthreads();

  double nfin = 0.0, lfin = 0.0, ltot = 0.0;
  for (int base = 0; base < n; base += kThreads * kUnroll) {
    if (base > 0) load(base);
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (base + (int)threadIdx.x + kThreads * u >= n) continue;
      ltot += (double)len[u];
      if (tau[u] > i) continue;   // k <= i for every w
      const int64_t ws = p.pp == 1 ? w_max : min((int64_t)w_max, ((int64_t)i - tau[u]) / (p.pp - 1));
      const double pf = prec[u] * S[ws];
      nfin += pf;
      lfin += (double)len[u] * pf;
    }
  }
  nfin = wave_sum_f64(nfin);
  lfin = wave_sum_f64(lfin);
  ltot = wave_sum_f64(ltot);
  if (lane == 0) {
    red[0][wave] = nfin;
    red[1][wave] = lfin;
    red[2][wave] = ltot;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double a = 0.0, b = 0.0, c = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      a += red[0][w];
      b += red[1][w];
      c += red[2][w];
    }
    const double gen = gen_sm;
    p.mem[i - 1] = c + ((double)n - a) * gen - b;
    if (p.e_gen) p.e_gen[i - 1] = gen;
    if (p.e_nfin) p.e_nfin[i - 1] = a;
    if (p.e_lfin) p.e_lfin[i - 1] = b;
  }
}

hipError_t launch_lookahead(const LookaheadParams& p, hipStream_t s) {
  hipLaunchKernelGGL(lookahead_kernel, dim3(p.iters), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace spexis
