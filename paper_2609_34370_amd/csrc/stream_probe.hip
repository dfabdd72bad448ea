// HBM read-rate probes for the benchmark's roofline fractions: how fast this GPU streams a large
// buffer into the compute units with coalesced 16-byte loads, in two access patterns.  Not part
// of libspexis (its own small library, loaded only by the benchmark).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kUnroll = 8;   // independent 16-byte loads in flight per thread

// Workgroup g reads 16-byte elements g*256 + t + j*grid*256 (j = 0, 1, ...): every wave covers
// 1 KB contiguous per load, consecutive workgroups neighbouring KBs.  Each thread folds what
// it read into one word (so no load is dead) and writes it to out[g*256 + t].
__global__ __launch_bounds__(kThreads) void stream_read_kernel(const u32x4* __restrict__ buf, int64_t n,
                                                               uint32_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + (kUnroll - 1) * stride < n; i += kUnroll * stride) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int j = 0; j < kUnroll; ++j) v[j] = __builtin_nontemporal_load(buf + i + j * stride);
#pragma unroll
    for (int j = 0; j < kUnroll; ++j) acc ^= v[j];
  }
  for (; i < n; i += stride) acc ^= buf[i];
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

// Workgroup g reads whole chunks of `chunk` elements, chunks g, g + grid, ...: each workgroup
// streams a contiguous range (measured on MI355X: about 6.9 TB/s for chunks of 64 KB and more,
// against about 6.4 TB/s for the strided pattern above, whose waves jump by grid KB).
__global__ __launch_bounds__(kThreads) void chunk_read_kernel(const u32x4* __restrict__ buf, int64_t n, int64_t chunk,
                                                              uint32_t* __restrict__ out) {
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int64_t c0 = (int64_t)blockIdx.x * chunk; c0 < n; c0 += (int64_t)gridDim.x * chunk) {
    const int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
    int64_t i = c0 + threadIdx.x;
    for (; i + (kUnroll - 1) * kThreads < c1; i += kUnroll * kThreads) {
      u32x4 v[kUnroll];
#pragma unroll
      for (int j = 0; j < kUnroll; ++j) v[j] = __builtin_nontemporal_load(buf + i + j * kThreads);
#pragma unroll
      for (int j = 0; j < kUnroll; ++j) acc ^= v[j];
    }
    for (; i < c1; i += kThreads) acc ^= buf[i];
  }
  out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = acc.x ^ acc.y ^ acc.z ^ acc.w;
}

}  // namespace

extern "C" {

// Reads `bytes` (a multiple of 16, 16-byte aligned) of device memory at `buf` with `grid`
// workgroups of 256 threads; `out` receives grid * 256 uint32 words.  Returns a hipError_t.
int spexis_probe_stream_read(const void* buf, int64_t bytes, int grid, void* out, void* stream) {
  if (!buf || !out || bytes <= 0 || bytes % 16 != 0 || grid <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(stream_read_kernel, dim3(grid), dim3(kThreads), 0, (hipStream_t)stream,
                     static_cast<const u32x4*>(buf), bytes / 16, static_cast<uint32_t*>(out));
  return (int)hipGetLastError();
}

// The same read in whole chunks of `chunk_bytes` (a multiple of 16) per workgroup.
int spexis_probe_chunk_read(const void* buf, int64_t bytes, int grid, int64_t chunk_bytes, void* out, void* stream) {
  if (!buf || !out || bytes <= 0 || bytes % 16 != 0 || grid <= 0 || chunk_bytes <= 0 || chunk_bytes % 16 != 0)
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(chunk_read_kernel, dim3(grid), dim3(kThreads), 0, (hipStream_t)stream,
                     static_cast<const u32x4*>(buf), bytes / 16, chunk_bytes / 16, static_cast<uint32_t*>(out));
  return (int)hipGetLastError();
}

}  // extern "C"
