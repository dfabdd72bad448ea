// Linear layers of the drafting adapter (Implementation: a linear layer and an attention layer,
// then the LM head): y = x W^T (+ R) for bf16 x [M][K], W [N][K], optional bf16 residual R
// [M][N], bf16 output y [M][N], fp32 accumulation.
//
// The adapter runs once per drafted token on the batch's exit hidden states: M is the batch (tens
// to hundreds of rows) and W, read once, is the whole cost.  The work decomposition is built to
// keep enough of W in flight:
//   * a workgroup computes 32 output columns for up to 128 rows (1, 2 or 4 row tiles of 32);
//     its four waves split the K range and add their accumulators through LDS in a fixed order;
//   * when the columns and row groups give too few workgroups to fill the chip, the K range is
//     also split over workgroups (S = 2, 4 or 8): each writes an fp32 partial, and a second
//     kernel adds the partials in order, adds the residual and rounds to bf16;
//   * both MFMA operands (v_mfma_f32_32x32x16_bf16) are loaded straight into registers, 64 K
//     values per chunk: lane half h takes K = 32h + 8s .. +7 at MFMA step s for its row of x and
//     its column of W alike (the contraction order is free when both sides use it).  W is
//     packed (pack.hip), so a wave's operand load reads 1 KB of contiguous memory;
//   * workgroups of one (column tile, K split) and consecutive row groups go to one XCD in turn,
//     so a W tile read for one row group is an L2 hit for the next.
#include "common.h"
#include "kernels.h"

namespace spexis {

namespace {

constexpr int kThreads = 256;
constexpr int kCh = 64;   // K values per chunk

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;   // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

}  // namespace

template <int NRT, int DEPTH>
__global__ __launch_bounds__(kThreads) void linear_kernel(LinearParams p) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
  const int mg = local % p.mgroups;
  const int ts = (local / p.mgroups) * 8 + xcd;
  if (ts >= p.ntiles * p.S) return;
  const int tile = ts % p.ntiles, split = ts / p.ntiles;
  const int n0 = tile * 32, m0 = mg * 32 * NRT;
  const int kbase = split * (p.K / p.S) + wave * p.kw + 32 * half;
  const int nch = p.kw / kCh;

  // W is packed (pack.hip): the wave's columns are tile row `tile`, its K range starts at chunk
  // kbase / 64, and lane l reads 16 contiguous bytes at s * 512 + 8 l of each 4 KB tile
  const int kchunks = p.K / kCh;
  const uint16_t* wp = reinterpret_cast<const uint16_t*>(p.w) +
                       ((int64_t)tile * kchunks + (split * (p.K / p.S) + wave * p.kw) / kCh) * kPackTile + 8 * lane;
  const uint16_t* xp[NRT];
#pragma unroll
  for (int t = 0; t < NRT; ++t)
    xp[t] = reinterpret_cast<const uint16_t*>(p.x) + (int64_t)min(m0 + 32 * t + col, p.M - 1) * p.K + kbase;

  u32x4 wb[DEPTH][4], xa[DEPTH][NRT][4];
  auto load = [&](int d, int j) {   // chunk j into buffer d (past the end: the last chunk again)
    const int jc = min(j, nch - 1);
    const int off = jc * kCh;
#pragma unroll
    for (int s = 0; s < 4; ++s) wb[d][s] = *reinterpret_cast<const u32x4*>(wp + (int64_t)jc * kPackTile + 512 * s);
#pragma unroll
    for (int t = 0; t < NRT; ++t)
#pragma unroll
      for (int s = 0; s < 4; ++s) xa[d][t][s] = *reinterpret_cast<const u32x4*>(xp[t] + off + 8 * s);
  };

  f32x16 acc[NRT];
#pragma unroll
  for (int t = 0; t < NRT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[t][e] = 0.f;

#pragma unroll
  for (int d = 0; d < DEPTH; ++d) load(d, d);
  for (int j = 0; j < nch; j += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      if (j + d < nch) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
          for (int t = 0; t < NRT; ++t)
            acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(xa[d][t][s]), as_bf16x8(wb[d][s]), acc[t], 0,
                                                              0, 0);
      }
      load(d, j + d + DEPTH);
    }
  }

  // the four waves' accumulators, added in wave order
  constexpr int kRows = 32 * NRT;
  __shared__ float red[4][kRows][33];
#pragma unroll
  for (int t = 0; t < NRT; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) red[wave][32 * t + 8 * (i >> 2) + 4 * half + (i & 3)][col] = acc[t][i];
  __syncthreads();
  for (int e = threadIdx.x; e < kRows * 32; e += kThreads) {
    const int r = e >> 5, c = e & 31;
    const int m = m0 + r, n = n0 + c;
    if (m >= p.M || n >= p.N) continue;
    const float v = ((red[0][r][c] + red[1][r][c]) + red[2][r][c]) + red[3][r][c];
    if (p.S > 1) {
      p.part[((int64_t)split * p.M + m) * p.N + n] = v;
    } else {
      const float y = p.res ? v + bf16_f(reinterpret_cast<const uint16_t*>(p.res)[(int64_t)m * p.N + n]) : v;
      reinterpret_cast<uint16_t*>(p.y)[(int64_t)m * p.N + n] = bf16_rne(y);
    }
  }
}

// y = bf16(sum_s part[s] (in order) + R): 4 consecutive outputs per thread.
__global__ __launch_bounds__(kThreads) void linear_reduce_kernel(LinearParams p) {
  const int64_t total = (int64_t)p.M * p.N;
  const int64_t e0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  if (e0 >= total) return;
  const int cnt = (int)min((int64_t)4, total - e0);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < p.S; ++s) {
    const float* src = p.part + (int64_t)s * total + e0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i < cnt) v[i] += src[i];
  }
  uint16_t* y = reinterpret_cast<uint16_t*>(p.y) + e0;
  const uint16_t* r = p.res ? reinterpret_cast<const uint16_t*>(p.res) + e0 : nullptr;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (i < cnt) y[i] = bf16_rne(r ? v[i] + bf16_f(r[i]) : v[i]);
}

// Row tiles, K split and grid for a problem (the same choice in the workspace query and the launch).
void linear_plan(int M, int N, int K, LinearParams& p) {
  const int need = (M + 31) / 32;
  const int nrt = need <= 1 ? 1 : (need <= 2 ? 2 : 4);
  p.M = M;
  p.N = N;
  p.K = K;
  p.nrt = nrt;
  p.ntiles = (N + 31) / 32;
  p.mgroups = (M + 32 * nrt - 1) / (32 * nrt);
  int S = 1;
  while (S < 8 && (int64_t)p.ntiles * p.mgroups * S < 512 && K % (4 * kCh * 2 * S) == 0) S *= 2;
  p.S = S;
  p.kw = K / (4 * S);
}

template <int NRT, int DEPTH>
static hipError_t launch_linear_nrt(const LinearParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)((p.ntiles * p.S + 7) / 8) * 8 * p.mgroups;
  hipLaunchKernelGGL((linear_kernel<NRT, DEPTH>), dim3((unsigned)grid), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_linear(const LinearParams& p, hipStream_t s) {
  hipError_t e = p.nrt == 1 ? launch_linear_nrt<1, 6>(p, s)
                            : (p.nrt == 2 ? launch_linear_nrt<2, 3>(p, s) : launch_linear_nrt<4, 2>(p, s));
  if (e != hipSuccess || p.S == 1) return e;
  const int64_t quads = ((int64_t)p.M * p.N + 3) / 4;
  hipLaunchKernelGGL(linear_reduce_kernel, dim3((unsigned)((quads + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                     p);
  return hipGetLastError();
}

}  // namespace spexis
