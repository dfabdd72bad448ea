// KV-cache append: the n_b = k_b + 1 new rows of each sequence go to positions
// L_b .. S_b-1 of the shared paged cache (speculative-parallel execution, Sec. 4: speculative
// and normal execution share one cache, so rows of rejected drafts are simply overwritten).
#include "common.h"
#include "kernels.h"

namespace spexis {

// One workgroup per (sequence, KV head), for the sequence's n = S - L new rows (64 at a time).
// K: threads take (token, 16-byte chunk) pairs, one 16-byte load and store each (the K layout
// holds 8 head-dim values of a slot together).
// V: the chunk's new rows go through LDS; then a thread takes one (16-slot unit, head-dim row)
// that the positions touch: it loads the unit's 32 bytes, puts the new values at their slots
// (slot positions swap23(slot) inside the unit) and stores the 32 bytes back -- two 16-byte
// stores instead of one 2-byte store per new value.  The unit's other slots are rewritten
// unchanged: a sequence's blocks are its own, and this workgroup is the only one writing head h
// of them.
// Every pool access is non-temporal: the attention launched next would otherwise write back the
// lines these stores leave dirty in the caches.  Against plain 2-byte V stores, append plus the
// attention after it went from 144.9 to 141.5 us at 64 sequences of 5 new rows (block size 16),
// from 499.5 to 487.8 us at 256 of 6 and from 411.0 to 399.7 us at 128 of 0-8, and stayed level
// at 512 of 9 new rows in blocks of 32 (328.1 against 328.9 us).
template <int D, int BS>
__global__ __launch_bounds__(256) void append_kv_kernel(AppendParams p) {
  constexpr int kCh = D / 8;
  constexpr int kChunk = 64;   // new V rows staged in LDS at a time
  __shared__ uint16_t sv[kChunk][D];
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
  const int32_t* table = p.block_tables + (int64_t)b * p.max_blocks;
  for (int j0 = 0; j0 < n; j0 += kChunk) {
    const int cn = min(kChunk, n - j0);
    for (int c = threadIdx.x; c < 2 * cn * kCh; c += 256) {
      const int which = c / (cn * kCh), rc = c % (cn * kCh), j = rc / kCh, ch = rc % kCh;
      const u32x4 v = ld16((which ? nv : nk) + ((int64_t)(q0 + j0 + j) * p.hkv + h) * D + 8 * ch);
      if (which == 0) {
        const int pos = L + j0 + j;
        const int blk = clampi(table[pos / BS], 0, p.num_blocks - 1);
        __builtin_nontemporal_store(
            v, reinterpret_cast<u32x4*>(kc + ((((int64_t)blk * p.hkv + h) * kCh + ch) * BS + pos % BS) * 8));
      } else {
        *reinterpret_cast<u32x4*>(&sv[j][8 * ch]) = v;
      }
    }
    __syncthreads();
    // the 16-slot units that positions lo .. hi-1 touch (a unit never spans two blocks)
    const int lo = L + j0, hi = lo + cn;
    const int u0 = lo >> 4, nu = ((hi - 1) >> 4) - u0 + 1;
    for (int c = threadIdx.x; c < nu * D; c += 256) {
      const int u = u0 + c / D, d = c % D;
      const int pos0 = u * 16;
      const int blk = clampi(table[pos0 / BS], 0, p.num_blocks - 1);
      uint16_t* row = vc + (((int64_t)blk * p.hkv + h) * D + d) * BS + pos0 % BS;
      const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row)),
                  c8 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row + 8));
      uint32_t w[8] = {a[0], a[1], a[2], a[3], c8[0], c8[1], c8[2], c8[3]};
#pragma unroll
      for (int ls = 0; ls < 16; ++ls) {
        const int pos = pos0 + ls;
        if (pos < lo || pos >= hi) continue;
        const int ps = (ls & ~12) | (((ls >> 2) & 1) << 3) | (((ls >> 3) & 1) << 2);   // swap23
        const uint32_t val = sv[pos - lo][d];
        w[ps >> 1] = (ps & 1) ? ((w[ps >> 1] & 0x0000FFFFu) | (val << 16)) : ((w[ps >> 1] & 0xFFFF0000u) | val);
      }
      __builtin_nontemporal_store(u32x4{w[0], w[1], w[2], w[3]}, reinterpret_cast<u32x4*>(row));
      __builtin_nontemporal_store(u32x4{w[4], w[5], w[6], w[7]}, reinterpret_cast<u32x4*>(row + 8));
    }
    // the next chunk reuses the staging rows and may rewrite a unit this one wrote (a workgroup
    // barrier orders the two: same workgroup, same CU)
    __syncthreads();
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
