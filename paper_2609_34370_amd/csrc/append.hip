// KV-cache append: the n_b = k_b + 1 new rows of each sequence go to positions
// L_b .. S_b-1 of the shared paged cache (speculative-parallel execution, Sec. 4: speculative
// and normal execution share one cache, so rows of rejected drafts are simply overwritten).
#include "common.h"
#include "kernels.h"

namespace spexis {

// One workgroup per (sequence, KV head); its four waves take the sequence's tokens in turn.
// K rows: D/8 lanes each move one 16-byte chunk (eight head-dim values) of a token.
// V rows: 2-byte stores, head-dim index d at slot position swap23(slot).
template <int D, int BS>
__global__ __launch_bounds__(256) void append_kv_kernel(AppendParams p) {
  const int b = blockIdx.x / p.hkv;
  const int h = blockIdx.x % p.hkv;
  const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int q0 = clampi(p.qsl[b], 0, p.total_tokens);
  const int q1 = clampi(p.qsl[b + 1], q0, p.total_tokens);
  const int cap = p.max_blocks * BS;
  const int n = q1 - q0 < cap ? q1 - q0 : cap;
  const int S = clampi(p.seq_lens[b], n, cap);
  const int L = S - n;
  const uint16_t* nk = reinterpret_cast<const uint16_t*>(p.new_k);
  const uint16_t* nv = reinterpret_cast<const uint16_t*>(p.new_v);
  uint16_t* kc = reinterpret_cast<uint16_t*>(p.k_cache);
  uint16_t* vc = reinterpret_cast<uint16_t*>(p.v_cache);
  for (int j = wave; j < n; j += 4) {
    const int pos = L + j;
    const int blk = clampi(p.block_tables[(int64_t)b * p.max_blocks + pos / BS], 0, p.num_blocks - 1);
    const int slot = pos % BS;
    const int64_t src = ((int64_t)(q0 + j) * p.hkv + h) * D;
    const int64_t head = (int64_t)blk * p.hkv + h;
    if (lane < D / 8) {
      u32x4 v = ld16(nk + src + lane * 8);
      st16(kc + ((head * (D / 8) + lane) * BS + slot) * 8, v);
    }
    const int vslot = (slot & ~12) | (((slot >> 2) & 1) << 3) | (((slot >> 3) & 1) << 2);
#pragma unroll
    for (int d = lane; d < D; d += kWave) vc[(head * D + d) * BS + vslot] = nv[src + d];
  }
}

template <int D, int BS>
static hipError_t launch_append_t(const AppendParams& p, hipStream_t s) {
  hipLaunchKernelGGL((append_kv_kernel<D, BS>), dim3(p.num_seqs * p.hkv), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_append(const AppendParams& p, hipStream_t s) {
  if (p.head_dim == 128) return p.block_size == 16 ? launch_append_t<128, 16>(p, s) : launch_append_t<128, 32>(p, s);
  return p.block_size == 16 ? launch_append_t<64, 16>(p, s) : launch_append_t<64, 32>(p, s);
}

}  // namespace spexis
