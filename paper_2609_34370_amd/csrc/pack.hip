// Weight packing for the matrix-core projections (LM head and adapter linear layers).
//
// A weight W [N][K] (bf16, row-major, K % 64 == 0) is stored as tiles of 32 rows x 64 K values,
// tile (n, c) = rows 32n .. 32n+31, K 64c .. 64c+63, each tile 4 KB, tiles in (n, c) order.
// Inside a tile, row r, K value 64c + 32h + 8s + e sits at ((s * 2 + h) * 32 + r) * 8 + e.
// That is the B-operand order of v_mfma_f32_32x32x16_bf16 as the kernels use it (lane
// l = 32h + r holds row r, K values 32h + 8s .. +7 at step s): one operand load of a wave reads
// 1 KB of contiguous memory, 8 full cache lines, instead of 16 bytes from each of 32 rows.
// Rows past N are zero.
#include "common.h"
#include "kernels.h"

namespace spexis {

__global__ __launch_bounds__(256) void pack_weight_kernel(const uint16_t* w, int N, int K, uint16_t* out) {
  const int64_t unit = (int64_t)blockIdx.x * 256 + threadIdx.x;   // 16-byte unit of the output
  const int64_t chunks = K / 64;
  const int64_t total = (int64_t)((N + 31) / 32) * chunks * 256;
  if (unit >= total) return;
  const int64_t tile = unit >> 8;
  const int within = (int)(unit & 255);
  const int s = within >> 6, h = (within >> 5) & 1, r = within & 31;
  const int64_t n = tile / chunks, c = tile % chunks;
  const int64_t row = 32 * n + r;
  u32x4 v = {0u, 0u, 0u, 0u};
  if (row < N) v = *reinterpret_cast<const u32x4*>(w + row * K + 64 * c + 32 * h + 8 * s);
  *reinterpret_cast<u32x4*>(out + unit * 8) = v;
}

hipError_t launch_pack_weight(const void* w, int N, int K, void* out, hipStream_t s) {
  const int64_t total = (int64_t)((N + 31) / 32) * (K / 64) * 256;
  hipLaunchKernelGGL(pack_weight_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(w), N, K, static_cast<uint16_t*>(out));
  return hipGetLastError();
}

}  // namespace spexis
