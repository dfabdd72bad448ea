// Verification attention: the k+1 query tokens of each sequence (its last accepted token and
// the k drafts, Sec. 4) attend causally over that sequence's paged KV cache, all query heads
// of one KV head (GQA group) together.
//
// Work decomposition: one workgroup per (KV chunk, sequence, KV head).  The G*(k+1) query rows
// of a (sequence, KV head) pair -- at most 64 -- form one or two 32-row tiles.  Each of the
// four waves streams its own 32-key tiles of the chunk (tiles w, w+4, ...) from HBM straight
// into matrix-core operand registers, keeps its own online-softmax state, and the waves merge
// through LDS at the end.  Chunks of one sequence merge in a second kernel (split-KV).
//
// Per 32-key tile and 32-row tile, with v_mfma_f32_32x32x16_bf16 (operand A: lane l holds row
// l%32, k-slice 8*(l/32)..+7; B: column l%32, same k-slice; C: lane l, value i holds row
// 8*(i/4) + 4*(l/32) + i%4, column l%32):
//   S^T[key][row] = K[key][:] . Q[row][:]   A = K tile (one 16-byte load per lane per k-step:
//                                           the K layout keeps 8 head-dim values of a slot
//                                           together), B = Q (registers, loaded once)
//   lane l then owns query row l%32 and keys (i/4)*8 + 4*(l/32) + i%4: the row maximum is a
//   max over 16 values plus one exchange with lane l^32.
//   O^T[d][row] += V^T[d][key] . P^T[key][row]   A = V^T tile: the V layout stores slots with
//                                           bits 2 and 3 swapped, so the 8 keys a lane needs
//                                           for k-step s are 16 contiguous bytes; B = P^T is
//                                           exactly the lane's score values 8s..8s+7.
#include "common.h"
#include "kernels.h"

namespace spexis {

constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" of the running maxima
constexpr float kLazy = 8.0f;         // base-2 headroom before the running maximum moves
constexpr int kMaxChunkBlocks = 512;  // block ids of one chunk staged in LDS (chunk <= 8192 tokens)

template <int D, int BS, int NT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(NT == 1 ? 2 : 1)))
void verify_attn_kernel(AttnParams p) {
  constexpr int KS = D / 16;   // k-steps of the score product
  constexpr int MT = D / 32;   // 32-wide head-dim tiles of the output
  const int item = blockIdx.x;
  const int kvh = item % p.hkv;
  const int rest = item / p.hkv;
  const int b = rest % p.num_seqs;
  const int c = rest / p.num_seqs;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 31, half = lane >> 5;

  // Block ids this chunk may use, loaded together with the sequence geometry (the chunk start
  // does not depend on the sequence length).
  const int32_t* bt = p.block_tables + (int64_t)b * p.max_blocks;
  const int blk0 = (c * p.chunk) / BS;
  int bt_pre[kMaxChunkBlocks / 256];
#pragma unroll
  for (int u = 0; u < kMaxChunkBlocks / 256; ++u) {
    const int x = blk0 + threadIdx.x + 256 * u;
    bt_pre[u] = bt[x < p.max_blocks ? x : p.max_blocks - 1];
  }

  // ---- sequence geometry (clamped so that every address stays inside its buffer)
  const int cap = p.max_blocks * BS;
  const int q0 = clampi(p.qsl[b], 0, p.total_tokens);
  const int q1 = clampi(p.qsl[b + 1], q0, p.total_tokens);
  int n = q1 - q0;
  if (n > p.rmax / p.group) n = p.rmax / p.group;
  if (n < 1) return;
  const int S = clampi(p.seq_lens[b], n, cap);
  const int L = S - n;
  const int R = p.group * n;
  int nch = (S + p.chunk - 1) / p.chunk;
  if (nch > p.nch_max) nch = p.nch_max;
  if (c >= nch) return;
  const int t_begin = c * p.chunk;
  const int t_end = (c == nch - 1) ? S : t_begin + p.chunk;   // the last chunk takes the rest
  const int ntiles = (t_end - t_begin + 31) >> 5;

  // Block ids of the chunk, staged in LDS: tile addresses then never wait on a global load
  // (which, counted in order with the K/V loads, would drain the prefetch pipeline).
  __shared__ int sm_blk[kMaxChunkBlocks];
#pragma unroll
  for (int u = 0; u < kMaxChunkBlocks / 256; ++u)
    sm_blk[threadIdx.x + 256 * u] = clampi(bt_pre[u], 0, p.num_blocks - 1);
  auto block_of = [&](int token) {
    const int x = token / BS - blk0;
    return x < kMaxChunkBlocks ? sm_blk[x] : clampi(bt[token / BS], 0, p.num_blocks - 1);
  };
  const uint16_t* kc = reinterpret_cast<const uint16_t*>(p.k_cache);
  const uint16_t* vc = reinterpret_cast<const uint16_t*>(p.v_cache);
  const int64_t head_stride = (int64_t)BS * D;   // elements of one (block, head) chunk

  // ---- query rows of this lane: row r = nt*32 + col is (token j, head g) with r = j*G + g.
  // The score product's B operand (Q) is the same for the four waves: wave 0 stages it in LDS
  // in operand order, every wave reads it back per tile.
  __shared__ u32x4 sm_q[NT][KS][kWave];
  int lim[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = nt * 32 + col;
    const int j = r < R ? r / p.group : n - 1;    // padding rows repeat a real row
    const int g = r < R ? r % p.group : 0;
    lim[nt] = L + j;                              // keys 0..L+j are visible
    if (wave == 0) {
      const uint16_t* qrow = reinterpret_cast<const uint16_t*>(p.q) +
                             ((int64_t)(q0 + j) * p.hq + kvh * p.group + g) * D + 8 * half;
#pragma unroll
      for (int s = 0; s < KS; ++s) sm_q[nt][s][lane] = ld16(qrow + 16 * s);
    }
  }

  __syncthreads();   // block ids and Q staged

  float m[NT], l[NT];
  f32x16 acc[NT][MT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m[nt] = kNegBig;
    l[nt] = 0.f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[nt][mt][i] = 0.f;
  }

  // Operand buffers.  Tile i of this wave is chunk tile wave + 4 i; DEPTH buffers rotate so
  // that DEPTH-1 tiles are in flight while one is computed.  Loads are issued unconditionally:
  // an index past the wave's last tile re-reads that tile (an L2 hit), which keeps the number of
  // outstanding loads the same on every path and lets the waits stay partial.
  constexpr int DEPTH = 2;
  struct Buf {
    u32x4 k[KS];
    u32x4 v[MT][2];
  };
  Buf buf[DEPTH];
  const int cnt = ntiles > wave ? (ntiles - wave + 3) / 4 : 0;   // tiles of this wave

  auto load_tile = [&](Buf& B, int i) {
    const int t0 = t_begin + (wave + 4 * (i < cnt ? i : cnt - 1)) * 32;
    int tk = t0 + col;
    if (tk > S - 1) tk = S - 1;                   // past the end: any valid slot, masked later
    const int kb = block_of(tk);
    const uint16_t* kp = kc + ((int64_t)kb * p.hkv + kvh) * head_stride + (tk % BS) * 8 + half * BS * 8;
#pragma unroll
    for (int s = 0; s < KS; ++s) B.k[s] = ld16(kp + s * (2 * BS * 8));
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      int tv = t0 + 16 * s2;
      if (tv > S - 1) tv = S - 1;
      const int vb = block_of(tv);
      const uint16_t* vp = vc + ((int64_t)vb * p.hkv + kvh) * head_stride + (BS == 32 ? 16 * s2 : 0) +
                           8 * half + (int64_t)col * BS;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) B.v[mt][s2] = ld16(vp + (int64_t)(32 * mt) * BS);
    }
  };

  auto process = [&](Buf& B, int i) {
    const int t0 = t_begin + (wave + 4 * i) * 32;
    if (t0 + 32 > S) {
      // the tile runs past the sequence: zero V rows of keys >= S (they may hold anything)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          // 32-bit word w holds positions 2w, 2w+1 of the lane's 8 keys
          const int kbase = t0 + 16 * s2 + 8 * ((2 * w) >> 2) + 4 * half + ((2 * w) & 3);
          const uint32_t keep = (kbase < S ? 0x0000FFFFu : 0u) | (kbase + 1 < S ? 0xFFFF0000u : 0u);
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) B.v[mt][s2][w] &= keep;
        }
      }
    }
    const bool need_mask = t0 + 31 > L;

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(B.k[s]), as_bf16x8(sm_q[nt][s][lane]), sc, 0, 0, 0);
      float x[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) x[e] = sc[e] * p.scale_log2e;
      if (need_mask) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = t0 + (e >> 2) * 8 + 4 * half + (e & 3);
          if (key > lim[nt]) x[e] = -INFINITY;
        }
      }
      float mx = x[0];
#pragma unroll
      for (int e = 1; e < 16; ++e) mx = fmaxf(mx, x[e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      // Lazy rescaling: the reference maximum moves only when a score exceeds it by more than
      // 2^kLazy, so 2^(x - m) stays <= 2^kLazy and the accumulators are rescaled rarely.
      if (__builtin_amdgcn_ballot_w64(mx > m[nt] + kLazy) != 0) {
        const float mnew = fmaxf(m[nt], mx);
        const float alpha = fast_exp2(m[nt] - mnew);
        m[nt] = mnew;
        l[nt] *= alpha;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[nt][mt][e] *= alpha;
      }
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        x[e] = fast_exp2(x[e] - m[nt]);
        ps += x[e];
      }
      l[nt] += ps;
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        u32x4 pw;
#pragma unroll
        for (int w = 0; w < 4; ++w) pw[w] = pack_bf16x2(x[8 * s2 + 2 * w], x[8 * s2 + 2 * w + 1]);
        const bf16x8 pb = as_bf16x8(pw);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[nt][mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(B.v[mt][s2]), pb, acc[nt][mt], 0, 0, 0);
      }
    }
  };

  if (cnt > 0) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) load_tile(buf[d], d);
    for (int i = 0; i < cnt; i += DEPTH) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        if (i + d >= cnt) break;
        process(buf[d], i + d);
        load_tile(buf[d], i + d + DEPTH);
      }
    }
  }

  // ---- merge the four waves: common maximum per row, then a two-level sum through LDS
  __shared__ float sm_m[4][NT * 32];
  __shared__ float sm_l[4][NT * 32];
  __shared__ float sm_acc[2][NT * MT * 16 * 64];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    l[nt] += __shfl_xor(l[nt], 32, kWave);
    if (half == 0) sm_m[wave][nt * 32 + col] = m[nt];
  }
  __syncthreads();
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = nt * 32 + col;
    const float M = fmaxf(fmaxf(sm_m[0][r], sm_m[1][r]), fmaxf(sm_m[2][r], sm_m[3][r]));
    const float f = fast_exp2(m[nt] - M);
    m[nt] = M;
    l[nt] *= f;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[nt][mt][i] *= f;
    if (half == 0) sm_l[wave][r] = l[nt];
  }
  if (wave >= 2) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sm_acc[wave - 2][((nt * MT + mt) * 16 + i) * 64 + lane] = acc[nt][mt][i];
  }
  __syncthreads();
  if (wave < 2) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[nt][mt][i] += sm_acc[wave][((nt * MT + mt) * 16 + i) * 64 + lane];
  }
  __syncthreads();
  if (wave == 1) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) sm_acc[0][((nt * MT + mt) * 16 + i) * 64 + lane] = acc[nt][mt][i];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int r = nt * 32 + col;
    const float lt = sm_l[0][r] + sm_l[1][r] + sm_l[2][r] + sm_l[3][r];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[nt][mt][i] += sm_acc[0][((nt * MT + mt) * 16 + i) * 64 + lane];
    if (r >= R) continue;
    const int j = r / p.group, g = r % p.group;
    if (nch == 1) {
      const float inv = 1.0f / lt;
      uint16_t* orow = reinterpret_cast<uint16_t*>(p.out) + ((int64_t)(q0 + j) * p.hq + kvh * p.group + g) * D;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          u32x2 w;
          w[0] = pack_bf16x2(acc[nt][mt][4 * a] * inv, acc[nt][mt][4 * a + 1] * inv);
          w[1] = pack_bf16x2(acc[nt][mt][4 * a + 2] * inv, acc[nt][mt][4 * a + 3] * inv);
          *reinterpret_cast<u32x2*>(orow + 32 * mt + 8 * a + 4 * half) = w;
        }
    } else {
      float* slot = p.ws + ((int64_t)(b * p.hkv + kvh) * p.nch_max + c) * attn_slot_floats(p.rmax, D);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          f32x4 v = {acc[nt][mt][4 * a], acc[nt][mt][4 * a + 1], acc[nt][mt][4 * a + 2], acc[nt][mt][4 * a + 3]};
          *reinterpret_cast<f32x4*>(slot + (int64_t)r * D + 32 * mt + 8 * a + 4 * half) = v;
        }
      if (half == 0) {
        slot[(int64_t)p.rmax * D + r] = m[nt];
        slot[(int64_t)p.rmax * D + p.rmax + r] = lt;
      }
    }
  }
}

// Split-KV merge: o = sum_c acc_c * 2^(m_c - M) / sum_c l_c * 2^(m_c - M), M = max_c m_c.
template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnParams p) {
  const int kvh = blockIdx.x % p.hkv;
  const int b = blockIdx.x / p.hkv;
  const int cap = p.max_blocks * p.block_size;
  const int q0 = clampi(p.qsl[b], 0, p.total_tokens);
  const int q1 = clampi(p.qsl[b + 1], q0, p.total_tokens);
  int n = q1 - q0;
  if (n > p.rmax / p.group) n = p.rmax / p.group;
  if (n < 1) return;
  const int S = clampi(p.seq_lens[b], n, cap);
  int nch = (S + p.chunk - 1) / p.chunk;
  if (nch > p.nch_max) nch = p.nch_max;
  if (nch <= 1) return;
  const int R = p.group * n;
  const int64_t slot_f = attn_slot_floats(p.rmax, D);
  const float* base = p.ws + (int64_t)(b * p.hkv + kvh) * p.nch_max * slot_f;
  __shared__ float w[64][64];   // [chunk][row] normalised weights (nch_max <= 64, rmax <= 64)
  for (int r = threadIdx.x; r < R; r += blockDim.x) {
    float M = kNegBig;
    for (int c = 0; c < nch; ++c) M = fmaxf(M, base[c * slot_f + (int64_t)p.rmax * D + r]);
    float den = 0.f;
    for (int c = 0; c < nch; ++c) {
      const float e = fast_exp2(base[c * slot_f + (int64_t)p.rmax * D + r] - M);
      w[c][r] = e;
      den += e * base[c * slot_f + (int64_t)p.rmax * D + p.rmax + r];
    }
    const float inv = 1.0f / den;
    for (int c = 0; c < nch; ++c) w[c][r] *= inv;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < R * (D / 4); idx += blockDim.x) {
    const int r = idx / (D / 4), d = (idx % (D / 4)) * 4;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int c = 0; c < nch; ++c) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(base + c * slot_f + (int64_t)r * D + d);
      o += a * w[c][r];
    }
    const int j = r / p.group, g = r % p.group;
    uint16_t* orow = reinterpret_cast<uint16_t*>(p.out) + ((int64_t)(q0 + j) * p.hq + kvh * p.group + g) * D;
    u32x2 v;
    v[0] = pack_bf16x2(o[0], o[1]);
    v[1] = pack_bf16x2(o[2], o[3]);
    *reinterpret_cast<u32x2*>(orow + d) = v;
  }
}

template <int D, int BS, int NT>
static hipError_t launch_attn_t(const AttnParams& p, hipStream_t s) {
  const int64_t grid = (int64_t)p.nch_max * p.num_seqs * p.hkv;
  hipLaunchKernelGGL((verify_attn_kernel<D, BS, NT>), dim3((unsigned)grid), dim3(256), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.nch_max <= 1) return e;
  hipLaunchKernelGGL((attn_merge_kernel<D>), dim3(p.num_seqs * p.hkv), dim3(256), 0, s, p);
  return hipGetLastError();
}

template <int D, int BS>
static hipError_t launch_attn_nt(const AttnParams& p, hipStream_t s) {
  return p.rmax <= 32 ? launch_attn_t<D, BS, 1>(p, s) : launch_attn_t<D, BS, 2>(p, s);
}

hipError_t launch_attention(const AttnParams& p, hipStream_t s) {
  if (p.head_dim == 128) return p.block_size == 16 ? launch_attn_nt<128, 16>(p, s) : launch_attn_nt<128, 32>(p, s);
  return p.block_size == 16 ? launch_attn_nt<64, 16>(p, s) : launch_attn_nt<64, 32>(p, s);
}

}  // namespace spexis
