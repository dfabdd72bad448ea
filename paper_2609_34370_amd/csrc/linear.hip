// Linear layers of the drafting adapter (Implementation: a linear layer and an attention layer,
// then the LM head): y = x W^T (+ R) for bf16 x [M][K], a packed W [N][K], an optional bf16
// residual R [M][N], bf16 output y [M][N], fp32 accumulation.
//
// The adapter runs once per drafted token on the batch's exit hidden states: M is the batch (tens
// to hundreds of rows), and W, read once, is the cost.  The layer runs on the projection kernel
// of the LM head (lm_head.hip: 128 output columns per workgroup, x shared through LDS, W streamed
// from its packed layout).  An adapter matrix has few column tiles, so the K range is split over
// workgroups until the chip is covered -- as long as the fp32 partials cost no more traffic than
// the weight; then a second kernel adds the partials in order, adds the residual and rounds
// to bf16.  Without a split the projection writes bf16 (with the residual) itself.  Several
// layers of one input (the attention layer's q, k, v) run as one projection of their stacked
// weights, the second kernel routing each layer's columns to its own output.
#include "common.h"
#include "kernels.h"

namespace spexis {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;   // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float from_bf16(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

}  // namespace

// y = bf16(sum_s part[s] (in order) + R): 4 consecutive outputs per thread; with split outputs,
// each group of four goes to the output that owns its columns.
__global__ __launch_bounds__(kThreads) void linear_reduce_kernel(LinearParams p) {
  const int64_t total = (int64_t)p.M * p.N;
  const int64_t e0 = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  if (e0 >= total) return;
  const int cnt = (int)min((int64_t)4, total - e0);
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  if (cnt == 4 && (total & 3) == 0) {   // 16-byte aligned in every partial
    // the partials in groups of 8, every load of a group issued together, added in order
    for (int s0 = 0; s0 < p.S; s0 += 8) {
      f32x4 x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        x[u] = *reinterpret_cast<const f32x4*>(p.part + (int64_t)min(s0 + u, p.S - 1) * total + e0);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < p.S)
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] += x[u][i];
    }
  } else {
    for (int s = 0; s < p.S; ++s)
      for (int i = 0; i < cnt; ++i) v[i] += p.part[(int64_t)s * total + e0 + i];
  }
  uint16_t* y = reinterpret_cast<uint16_t*>(p.y) + e0;
  if (p.nout > 0) {
    // split outputs: the four columns lie in one output (its bounds are multiples of 4)
    const int64_t row = e0 / p.N;
    const int c = (int)(e0 - row * p.N);
    void* base = p.ys[0];
    int lo = 0, hi = p.off[1];
#pragma unroll
    for (int j = 1; j < kLinearMaxOutputs; ++j)
      if (j < p.nout && c >= p.off[j]) {
        base = p.ys[j];
        lo = p.off[j];
        hi = p.off[j + 1];
      }
    y = reinterpret_cast<uint16_t*>(base) + row * (hi - lo) + (c - lo);
  }
  const uint16_t* r = p.res ? reinterpret_cast<const uint16_t*>(p.res) + e0 : nullptr;
  for (int i = 0; i < cnt; ++i) y[i] = to_bf16(r ? v[i] + from_bf16(r[i]) : v[i]);
}

// K split for a problem (the same choice in the workspace query and the launch): the smallest
// power of two up to 8 that gives at least 256 workgroups, while K / S stays a multiple of 64 and the
// partials (S M N fp32, written once and read once) stay within the weight's own traffic
// (2 S M N 4 <= 2 N K 2, i.e. 2 S M <= K).
int linear_split(int M, int N, int K) {
  const int64_t wgs = projection_workgroups(M, N);
  int S = 1;
  while (S < 8 && wgs * S < 256 && K % (kLmK * 2 * S) == 0 && (int64_t)2 * (2 * S) * M <= K) S *= 2;
  return S;
}

hipError_t launch_linear(const LinearParams& p, hipStream_t s) {
  hipError_t e = launch_projection(p.proj, s);
  if (e != hipSuccess || (p.S == 1 && p.nout == 0)) return e;
  const int64_t quads = ((int64_t)p.M * p.N + 3) / 4;
  hipLaunchKernelGGL(linear_reduce_kernel, dim3((unsigned)((quads + kThreads - 1) / kThreads)), dim3(kThreads), 0, s,
                     p);
  return hipGetLastError();
}

}  // namespace spexis
