// KV-cache append: the n_b = k_b + 1 new rows of each sequence go to positions
// L_b .. S_b-1 of the shared paged cache (speculative-parallel execution, Sec. 4: speculative
// and normal execution share one cache, so rows of rejected drafts are simply overwritten).
#include "common.h"
#include "kernels.h"

namespace spexis {

// One workgroup per (sequence, KV head).  Its threads take (token, 16-byte chunk) pairs of the
// sequence's new K and V rows -- n * D/8 chunks of each -- so that the workgroup's loads are
// issued together (five rows of D = 128: 160 chunks, one per thread), not one token per wave
// in turn.  K chunks keep their 16 bytes together (the K layout holds 8 head-dim values of a
// slot contiguously); V values go to slot position swap23(slot) of each head-dim row.
template <int D, int BS>
__global__ __launch_bounds__(256) void append_kv_kernel(AppendParams p) {
  constexpr int kCh = D / 8;
  const int b = blockIdx.x / p.hkv;
  const int h = blockIdx.x % p.hkv;
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
  for (int c = threadIdx.x; c < 2 * n * kCh; c += 256) {
    const int which = c / (n * kCh), rc = c % (n * kCh), j = rc / kCh, ch = rc % kCh;
    const int pos = L + j;
    const u32x4 v = ld16((which ? nv : nk) + ((int64_t)(q0 + j) * p.hkv + h) * D + 8 * ch);
    const int blk = clampi(p.block_tables[(int64_t)b * p.max_blocks + pos / BS], 0, p.num_blocks - 1);
    const int slot = pos % BS;
    const int64_t head = (int64_t)blk * p.hkv + h;
    if (which == 0) {
      st16(kc + ((head * kCh + ch) * BS + slot) * 8, v);
    } else {
      const int vslot = (slot & ~12) | (((slot >> 2) & 1) << 3) | (((slot >> 3) & 1) << 2);
#pragma unroll
      for (int e = 0; e < 8; ++e) vc[(head * D + 8 * ch + e) * BS + vslot] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
    }
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
