// Verification attention: the k+1 query tokens of each sequence (its last accepted token and
// the k drafts, Sec. 4) attend causally over that sequence's paged KV cache, all query heads
// of one KV head (GQA group) together.
//
// Work decomposition.  An item is one (sequence, KV head) pair: its G*(k+1) query rows -- at
// most 64, one or two 32-row tiles -- against the sequence's keys.  For each KV head the keys
// of all sequences form one stream of 32-key tiles (sequence, then position), cut into equal
// contiguous shares; wave (share s, head h) is wave s*Hkv + h, so the waves of a workgroup
// walk the same tiles of neighbouring heads at about the same time and read neighbouring
// memory (the cache stores a block's heads together).  A wave walks its share alone: no
// barrier, no merge, a prefetch pipeline of DEPTH tiles that runs on across sequence
// boundaries, and block ids fetched one tile ahead with scalar loads (their wait counter is
// not the one the tile loads use).  An item a wave covers whole is normalised and written as
// bf16; an item cut between shares leaves fp32 partials (reference maximum, sum,
// unnormalised output) that a second kernel combines -- the partial of a share's first item
// held in LDS until the wave ends.  Balance is exact to one tile, whatever the mix of sequence
// lengths.
//
// Per 32-key tile and 32-row tile, with v_mfma_f32_32x32x16_bf16 (operand A: lane l holds row
// l%32, k-slice 8*(l/32)..+7; B: column l%32, same k-slice; C: lane l, value i holds row
// 8*(i/4) + 4*(l/32) + i%4, column l%32):
//   S^T[key][row] = K[key][:] . Q[row][:]   A = K tile (one 16-byte load per lane per k-step:
//                                           the K layout keeps 8 head-dim values of a slot
//                                           together), B = Q (registers, loaded per item)
//   lane l then owns query row l%32 and keys (i/4)*8 + 4*(l/32) + i%4: the row maximum is a
//   max over 16 values plus one exchange with lane l^32.
//   O^T[d][row] += V^T[d][key] . P^T[key][row]   A = V^T tile: the V layout stores slots with
//                                           bits 2 and 3 swapped, so the 8 keys a lane needs
//                                           for k-step s are 16 contiguous bytes; B = P^T is
//                                           exactly the lane's score values 8s..8s+7.
#include "common.h"
#include "kernels.h"

namespace spexis {

// Lane l and lane l ^ 32 combined, in one cross-half lane swap (v_permlane32_swap): the swap of a
// value with itself leaves the lower half's value in the first result and the upper half's in the
// second, in every lane.
__device__ __forceinline__ float halves_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" of the running maxima

// acc[mt] *= alpha (alpha per lane: the lane's query row), in place on the registers that hold the
// accumulators.  Written out because otherwise the compiler keeps a second copy of every
// accumulator in vector registers, refreshed by one v_accvgpr_read per accumulator on every tile,
// for the rare tiles that take this path.  The hazard checks do not look inside inline assembly:
// the leading s_nops give an accumulator's last MFMA its 18+ wait states before the first read
// (this is its own basic block, so no MFMA is scheduled in between), the trailing one covers the
// last write before the next MFMA reads it as its C operand.
template <int MT>
__device__ __forceinline__ void scale_acc(f32x16 (&acc)[MT], float alpha) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      float v = acc[mt][e], t;
      asm volatile("v_accvgpr_read_b32 %1, %0\n\tv_mul_f32 %1, %1, %2\n\tv_accvgpr_write_b32 %0, %1"
                   : "+a"(v), "=&v"(t)
                   : "v"(alpha));
      acc[mt][e] = v;
    }
  asm volatile("s_nop 4");
}
constexpr float kLazy = 8.0f;         // base-2 headroom before the running maximum moves
constexpr int kWaitVmcnt0 = 0x0F70;   // s_waitcnt operand: vmcnt(0), expcnt and lgkmcnt not waited

// Read-only view of an int32 array: loads through it at wave-uniform addresses become scalar
// loads, counted apart from the vector loads of the tiles.
typedef const __attribute__((address_space(4))) int32_t sint32;

struct SeqGeo {
  int q0, n, S, nt;   // first query token, query tokens, keys, 32-key tiles (0: no query)
};

// Geometry of sequence b, clamped so that every address derived from it stays in its buffer.
template <typename Ptr>
__device__ __forceinline__ SeqGeo seq_geo(const AttnParams& p, Ptr qsl, Ptr seq_lens, int b) {
  SeqGeo g;
  g.q0 = clampi(qsl[b], 0, p.total_tokens);
  const int q1 = clampi(qsl[b + 1], g.q0, p.total_tokens);
  g.n = min(q1 - g.q0, p.rmax / p.group);
  g.S = clampi(seq_lens[b], max(g.n, 1), p.max_blocks * p.block_size);
  g.nt = g.n >= 1 ? (g.S + 31) >> 5 : 0;
  return g;
}

// Position in a head's tile stream: sequence, tile of the sequence, and the sequence's size.
struct Cursor {
  int b, t, nt, S;
};

__device__ __forceinline__ void advance(const AttnParams& p, Cursor& c) {
  if (++c.t < c.nt) return;
  c.t = 0;
  SeqGeo g;
  do {
    if (c.b + 1 >= p.num_seqs) return;   // never past the stream's end; stay on a valid item
    ++c.b;
    g = seq_geo(p, (sint32*)p.qsl, (sint32*)p.seq_lens, c.b);
  } while (g.nt == 0);
  c.nt = g.nt;
  c.S = g.S;
}

// Share geometry of a head's tile stream: shares pair up, shares 2j and 2j+1 covering tiles
// [2jP, 2(j+1)P), the first (the wave on an even XCD) P + dlt of them and the second P - dlt.
// dlt = 0 gives equal shares of P.
__device__ __forceinline__ int share_delta(int P, int skew) { return (int)(((int64_t)P * skew) >> 10); }
__device__ __forceinline__ int64_t share_first(int s, int P, int dlt) {
  return (int64_t)(s >> 1) * 2 * P + (s & 1) * (P + dlt);
}
__device__ __forceinline__ int share_size(int s, int P, int dlt) { return (s & 1) ? P - dlt : P + dlt; }
__device__ __forceinline__ int share_of(int g, int P, int dlt) {
  const int j = g / (2 * P);
  return 2 * j + (g - 2 * P * j >= P + dlt ? 1 : 0);
}

template <int D, int BS, int NT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1)))
void verify_attn_kernel(AttnParams p) {
  constexpr int KS = D / 16;   // k-steps of the score product
  constexpr int MT = D / 32;   // 32-wide head-dim tiles of the output
  // Tiles in flight: the register file of one wave per SIMD holds DEPTH operand buffers.
  constexpr int DEPTH = NT == 1 ? 3 : 2;
  const int lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  // Physical wave qw -> (share s, head h); wid = s * hkv + h names its partial slots and header.
  // Paired shares (skew > 0): workgroups alternate between the XCDs of even and odd index, and
  // wave qw = 8m + 4 par + r takes u = 4m + r: share 2 (u / hkv) + par of head u % hkv.  So the
  // two shares of each pair run on XCDs of opposite parity, and the four waves of a workgroup
  // take neighbouring heads of one share.  The host makes nwaves a multiple of 8 and of 2 hkv,
  // which makes the map a bijection of [0, nwaves).
  const int qw = __builtin_amdgcn_readfirstlane((int)blockIdx.x * 4 + (int)(threadIdx.x >> 6));
  int s_, h_;
  if (p.skew > 0) {
    const int u = ((qw >> 3) << 2) | (qw & 3);
    s_ = 2 * (u / p.hkv) + ((qw >> 2) & 1);
    h_ = u % p.hkv;
  } else {
    s_ = qw / p.hkv;
    h_ = qw % p.hkv;
  }
  const int wid = s_ * p.hkv + h_;
  const int64_t slot_f = attn_slot_floats(p.rmax, D);
  float* slots = p.ws + (int64_t)wid * 2 * slot_f;
  int32_t* hdr = reinterpret_cast<int32_t*>(p.ws + (int64_t)p.nwaves * 2 * slot_f) + (int64_t)wid * kAttnHdrInts;

  auto no_share = [&]() {
    if (lane == 0) *reinterpret_cast<u32x4*>(hdr) = u32x4{0u, 0u, 0u, 0u};
  };
  const int h = h_, share = s_;
  if (share >= p.nshares) return no_share();

  // ---- this wave's share [g0, g0 + cnt) of head h's tile stream
  int total, b0 = 0, f0 = 0;
  Cursor start;
  if (p.num_seqs <= kWave) {
    // one pass: lane b holds sequence b's geometry; the share start is read from the lanes
    const SeqGeo gl = lane < p.num_seqs ? seq_geo(p, p.qsl, p.seq_lens, lane) : SeqGeo{0, 0, 0, 0};
    const int incl = wave_incl_scan_i32(gl.nt, lane);
    total = __builtin_amdgcn_readlane(incl, kWave - 1);   // < 2^31 (host)
    const int even = (total + p.nshares - 1) / p.nshares;
    const int P = max(p.tiles_per_wave > 0 ? p.tiles_per_wave : kAttnMinTilesPerWave, even);
    if (share_first(share, P, share_delta(P, p.skew)) >= total) return no_share();
    const int g0 = (int)share_first(share, P, share_delta(P, p.skew));
    const uint64_t hit = __builtin_amdgcn_ballot_w64(incl > g0);
    if (hit == 0) return no_share();
    const int l0 = __builtin_ctzll(hit);
    b0 = l0;
    f0 = __builtin_amdgcn_readlane(incl - gl.nt, l0);
    start.b = b0;
    start.nt = __builtin_amdgcn_readlane(gl.nt, l0);
    start.S = __builtin_amdgcn_readlane(gl.S, l0);
    start.t = g0 - f0;
  } else {
    int per_lane = 0;
    for (int base = 0; base < p.num_seqs; base += kWave)
      if (base + lane < p.num_seqs) per_lane += seq_geo(p, p.qsl, p.seq_lens, base + lane).nt;
    total = __builtin_amdgcn_readfirstlane(wave_sum_i32(per_lane));   // < 2^31 (host)
    const int even = (total + p.nshares - 1) / p.nshares;
    const int P = max(p.tiles_per_wave > 0 ? p.tiles_per_wave : kAttnMinTilesPerWave, even);
    if (share_first(share, P, share_delta(P, p.skew)) >= total) return no_share();
    const int g0 = (int)share_first(share, P, share_delta(P, p.skew));
    // the sequence holding tile g0, and the stream index of its first tile
    int before = 0;
    for (int base = 0; base < p.num_seqs; base += kWave) {
      const int b = base + lane;
      const int v = b < p.num_seqs ? seq_geo(p, p.qsl, p.seq_lens, b).nt : 0;
      const int incl = wave_incl_scan_i32(v, lane);
      const uint64_t hit = __builtin_amdgcn_ballot_w64(before + incl > g0);
      if (hit != 0) {
        const int l0 = __builtin_ctzll(hit);
        b0 = base + l0;
        f0 = before + __builtin_amdgcn_readlane(incl - v, l0);
        break;
      }
      before += __builtin_amdgcn_readlane(incl, kWave - 1);
    }
    b0 = __builtin_amdgcn_readfirstlane(b0);
    f0 = __builtin_amdgcn_readfirstlane(f0);
    const SeqGeo g = seq_geo(p, (sint32*)p.qsl, (sint32*)p.seq_lens, b0);
    if (g.nt == 0 || g0 < f0 || g0 - f0 >= g.nt) return no_share();   // inputs changed under us
    start.b = b0;
    start.nt = g.nt;
    start.S = g.S;
    start.t = g0 - f0;
  }
  const int P = max(p.tiles_per_wave > 0 ? p.tiles_per_wave : kAttnMinTilesPerWave,
                    (total + p.nshares - 1) / p.nshares);
  const int dlt = share_delta(P, p.skew);
  const int g0 = (int)share_first(share, P, dlt);
  const int cnt = min(share_size(share, P, dlt), total - g0);

  const uint16_t* kc = reinterpret_cast<const uint16_t*>(p.k_cache);
  const uint16_t* vc = reinterpret_cast<const uint16_t*>(p.v_cache);
  const int64_t head_stride = (int64_t)BS * D;   // elements of one (block, head) chunk
  // Physical blocks of a tile: keys 0..15 and 16..31 (one block when BS = 32).  The second id
  // repeats the first past the sequence end; those keys are masked.
  auto tile_blocks = [&](const Cursor& c, int& ka, int& kb) {
    sint32* row = (sint32*)p.block_tables + (int64_t)c.b * p.max_blocks;
    if (BS == 16) {
      ka = clampi(row[2 * c.t], 0, p.num_blocks - 1);
      kb = clampi(row[min(2 * c.t + 1, (c.S - 1) >> 4)], 0, p.num_blocks - 1);
    } else {
      ka = kb = clampi(row[c.t], 0, p.num_blocks - 1);
    }
  };

  // load side: the tile being issued (lc, its block ids) and the next one (nc), one step ahead
  Cursor lc = start, nc = start;
  int lidx = 0, la, lb, na = 0, nb = 0;
  // both tiles' block ids fetched together (with one tile, the next cursor is the same one)
  if (cnt > 1) advance(p, nc);
  tile_blocks(lc, la, lb);
  tile_blocks(nc, na, nb);

  // Operand buffers; DEPTH rotate so that DEPTH-1 tiles are in flight while one is computed.
  // Loads are issued unconditionally -- past the share's end they re-read its last tile (an L2
  // hit) -- so the count of outstanding loads is the same on every path and waits stay partial.
  struct Buf {
    u32x4 k[KS];
    u32x4 v[MT][2];
  };
  Buf buf[DEPTH];

  auto load_tile = [&](Buf& B, int i) {
    if (i < cnt && i > lidx) {
      lc = nc;
      la = na;
      lb = nb;
      lidx = i;
      if (i + 1 < cnt) {
        advance(p, nc);
        tile_blocks(nc, na, nb);
      }
    }
    const int t0 = lc.t * 32;
    const int tk = min(t0 + col, lc.S - 1);   // past the end: any valid slot, masked later
    const int kblk = (BS == 16 && (tk >> 4) != 2 * lc.t) ? lb : la;
    const uint16_t* kp = kc + ((int64_t)kblk * p.hkv + h) * head_stride + (tk % BS) * 8 + half * BS * 8;
    // K tiles are read once: non-temporal loads (measured faster than plain loads of K on every
    // workload, the call alone timed)
#pragma unroll
    for (int s = 0; s < KS; ++s) B.k[s] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kp + s * (2 * BS * 8)));
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const int vblk = (BS == 16 && s2 == 1) ? lb : la;
      const uint16_t* vp = vc + ((int64_t)vblk * p.hkv + h) * head_stride + (BS == 32 ? 16 * s2 : 0) +
                           8 * half + (int64_t)col * BS;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        // V is read once too: non-temporal at block size 16 (the call as fast or faster, and
        // the acceptance launched after it 2-4 us faster: workload 2 2.7 us faster per step,
        // workload 3 8.3 us, workload 4 3.1 us); plain at block size 32, where a lane's 16
        // bytes are half of a 64-byte head-dim row (non-temporal: the call 8 us slower at 512
        // sequences)
        const u32x4* a = reinterpret_cast<const u32x4*>(vp + (int64_t)(32 * mt) * BS);
        B.v[mt][s2] = BS == 16 ? __builtin_nontemporal_load(a) : *a;
      }
    }
  };

  // process side: the item being computed and its online-softmax state
  Cursor pc = start;
  int q0 = 0, n = 1, L = 0, R = 0;
  bool starts_before = false;
  int head_b = 0, head_f = 0, head_nt = 0, head_q0 = 0, head_n = 0, head_flag = 0;
  int lim[NT];
  // Q, the score product's B operand, in operand order: with two row tiles, row tile 0 in this
  // wave's part of LDS and row tile 1 in registers (both in registers would not fit next to two
  // tiles' accumulators); one row tile in registers.
  constexpr bool kQinLds = NT == 2;
  u32x4 qr[kQinLds ? 1 : NT][KS];
  const int wave = threadIdx.x >> 6;
  // Each wave's KS KB of LDS: Q's row tile 0 while an item runs (two row tiles), and the scratch
  // through which an item's outputs are transposed at its end.
  __shared__ u32x4 sm_q[4][KS][kWave];
  u32x4* const scr = &sm_q[wave][0][0];
  // The partial of the share's first item (its later part, which ends inside the share) waits in
  // this wave's LDS, its maxima and sums in registers, and goes to memory when the wave ends:
  // stores issued in the middle of a share cost far more than their bytes (a timing-only copy
  // without them ran 9% faster at 20 and at 63 rows per item).  With two row tiles of 128-wide
  // heads the four waves' stashes and row tile 0 of Q fill the 160 KB of LDS exactly.
  __shared__ f32x4 sm_stash[4][NT * 32 * D / 4];
  float st_m[NT], st_l[NT];
  bool stashed = false;
  int stash_rows = 0;
  float m[NT], l[NT];
  f32x16 acc[NT][MT];

  auto begin_item = [&](int i) {
    const SeqGeo g = seq_geo(p, (sint32*)p.qsl, (sint32*)p.seq_lens, pc.b);
    q0 = g.q0;
    n = g.n;
    L = pc.S - n;
    R = p.group * n;
    starts_before = i == 0 && pc.t != 0;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      // row r = nt*32 + col is (token j, head g) with r = j*G + g; padding rows repeat a real row
      const int r = nt * 32 + col;
      const int j = r < R ? r / p.group : n - 1;
      const int gq = r < R ? r % p.group : 0;
      lim[nt] = L + j;   // keys 0..L+j are visible
      const uint16_t* qrow = reinterpret_cast<const uint16_t*>(p.q) +
                             ((int64_t)(q0 + j) * p.hq + h * p.group + gq) * D + 8 * half;
      if (kQinLds && nt == 0) {
        u32x4 t[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) t[s] = ld16(qrow + 16 * s);
#pragma unroll
        for (int s = 0; s < KS; ++s) sm_q[wave][s][lane] = t[s];
      } else {
#pragma unroll
        for (int s = 0; s < KS; ++s) qr[kQinLds ? 0 : nt][s] = ld16(qrow + 16 * s);
      }
      m[nt] = kNegBig;
      l[nt] = 0.f;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[nt][mt][e] = 0.f;
    }
    // Wait for Q here, explicitly (this drains the tiles in flight, once per item): the wait
    // counter then knows Q complete on every path, and the tile loop's waits stay partial.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  };

  auto end_item = [&](int i) {
    const bool ends_after = pc.t < pc.nt - 1;
    const bool whole = !starts_before && !ends_after;
    if (!whole && !starts_before) {   // this wave holds the item's first tiles
      head_flag = 1;
      head_b = pc.b;
      head_f = g0 + i - pc.t;
      head_nt = pc.nt;
      head_q0 = q0;
      head_n = n;
    }
    // Outputs leave through the wave's LDS scratch, transposed, so that each store writes whole
    // 16-byte chunks of consecutive rows: stored straight from the accumulators, an instruction
    // writes 8 bytes into each of 32 rows, and a timing-only copy without the output stores ran
    // 29 us (10%) faster at 63 rows per item.  The scratch holds Q's row tile 0 during the item,
    // no longer needed here; a wave's LDS operations run in order.
    constexpr int kOc = D / 8;   // 16-byte chunks of a bf16 output row
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const float lt = halves_sum(l[nt]);
      const int lr = nt * 32 + col;   // row of the item (and of the partial slot)
      if (whole) {
        // bf16 rows, chunk c of row col at chunk c ^ (col mod kOc) of the scratch row
        const float inv = 1.0f / lt;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            u32x2 w;
            w[0] = pack_bf16x2(acc[nt][mt][4 * a] * inv, acc[nt][mt][4 * a + 1] * inv);
            w[1] = pack_bf16x2(acc[nt][mt][4 * a + 2] * inv, acc[nt][mt][4 * a + 3] * inv);
            const int c = 4 * mt + a;
            reinterpret_cast<u32x2*>(scr)[(col * kOc + (c ^ (col & (kOc - 1)))) * 2 + half] = w;
            __builtin_amdgcn_sched_barrier(0);   // one chunk at a time: few registers live
          }
#pragma unroll 1
        for (int q = lane; q < 32 * kOc; q += kWave) {
          const int row = q / kOc, c = q % kOc, r = nt * 32 + row;
          const u32x4 v = scr[row * kOc + (c ^ (row & (kOc - 1)))];
          if (r < R) {
            const int j = r / p.group, gq = r % p.group;
            // written once, read by a later kernel: non-temporal (1-4 us faster at workloads 2-5)
            __builtin_nontemporal_store(
                v, reinterpret_cast<u32x4*>(reinterpret_cast<uint16_t*>(p.out) +
                                            ((int64_t)(q0 + j) * p.hq + h * p.group + gq) * D + 8 * c));
          }
        }
      } else if (starts_before) {
        if (lr < R) {
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int a = 0; a < 4; ++a)
              sm_stash[wave][(lr * D + 32 * mt + 8 * a + 4 * half) / 4] =
                  f32x4{acc[nt][mt][4 * a], acc[nt][mt][4 * a + 1], acc[nt][mt][4 * a + 2], acc[nt][mt][4 * a + 3]};
        }
        st_m[nt] = m[nt];
        st_l[nt] = lt;
      }
      // (an item this wave starts and a later share finishes is the share's last: its partial
      // is stored after the tile loop, from the accumulators it leaves behind)
    }
    if (starts_before) {
      stashed = true;
      stash_rows = R;
    }
  };

  auto process = [&](Buf& B, int i) {
    if (i >= cnt) return;   // padding past the share's end
    if (i == 0 || pc.t == 0) begin_item(i);
    const int t0 = pc.t * 32;
    const int S = pc.S;
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
    const bool need_mask = t0 + 31 > L;   // causal edge (keys >= S are past every row's limit)

#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      f32x16 sc;
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
#pragma unroll
      for (int s = 0; s < KS; ++s)
        sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            as_bf16x8(B.k[s]),
            as_bf16x8(kQinLds && nt == 0 ? sm_q[wave][s][lane] : qr[kQinLds ? 0 : nt][s]),
            sc, 0, 0, 0);
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
      mx = halves_max(mx);
      // Lazy rescaling: the reference maximum moves only when a score exceeds it by more than
      // 2^kLazy, so 2^(x - m) stays <= 2^kLazy and the accumulators are rescaled rarely.
      if (__builtin_amdgcn_ballot_w64(mx > m[nt] + kLazy) != 0) {
        const float mold = m[nt];
        const float mnew = fmaxf(mold, mx);
        const float alpha = fast_exp2(mold - mnew);
        m[nt] = mnew;
        l[nt] *= alpha;
        // a row still at kNegBig has added nothing yet (its accumulators are zero): the first tile
        // of an item moves every row's maximum and scales nothing
        if (__builtin_amdgcn_ballot_w64(mold > kNegBig) != 0) scale_acc<MT>(acc[nt], alpha);
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
    if (pc.t == pc.nt - 1 || i == cnt - 1) end_item(i);
    if (i + 1 < cnt) advance(p, pc);
  };

  // Wait counts retire in issue order, so the loop is shaped for them: every pass runs a whole
  // group of DEPTH tiles with no exit inside it (an exit edge back to the loop head would make
  // one buffer look younger than the next, and each wait for it would drain the prefetched
  // tiles); the share is padded to a multiple of DEPTH with tiles that are loaded but skipped.
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) load_tile(buf[d], d);
  for (int i = 0; i < cnt; i += DEPTH) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) {
      process(buf[d], i + d);
      load_tile(buf[d], i + d + DEPTH);
    }
  }

  // The share's last item, if a later share finishes it: its partial to slot 1, through the LDS
  // scratch in two halves of the head dimension (32 rows x D/2 columns each), so that each store
  // writes 16-byte chunks of consecutive rows.  Here, past the tile loop, the transpose costs no
  // registers the loop needs (inside it, it spilled).
  // Partials are written once and read by the merge launch.  With two row tiles (33 to 64 rows:
  // large partials) they are stored non-temporally, like the outputs, so that the end of this
  // launch does not wait for them to be written back from the caches (the call 11.6 us faster at
  // 63 rows per item, 99 MB of partials); with one row tile plain stores leave the merge's reads
  // to the caches (at 20 rows per item the merge ran 6.0 against 7.6 us, the call 1 us faster).
  auto put4 = [](float* a, u32x4 v) {
    if (NT == 2) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(a));
    else *reinterpret_cast<u32x4*>(a) = v;
  };
  auto put1 = [](float* a, float v) {
    if (NT == 2) __builtin_nontemporal_store(v, a);
    else *a = v;
  };
  if (head_flag) {
    constexpr int kHc = D / 8;   // 16-byte chunks of half an fp32 row
    float* slot1 = slots + slot_f;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const float lt = halves_sum(l[nt]);
      const int lr = nt * 32 + col;
#pragma unroll
      for (int hm = 0; hm < 2; ++hm) {
#pragma unroll
        for (int mt = hm * MT / 2; mt < (hm + 1) * MT / 2; ++mt)
#pragma unroll
          for (int a = 0; a < 4; ++a) {
            const int c = 8 * (mt - hm * MT / 2) + 2 * a + half;
            scr[col * kHc + (c ^ (col & (kHc - 1)))] =
                u32x4{__float_as_uint(acc[nt][mt][4 * a]), __float_as_uint(acc[nt][mt][4 * a + 1]),
                      __float_as_uint(acc[nt][mt][4 * a + 2]), __float_as_uint(acc[nt][mt][4 * a + 3])};
          }
        for (int q = lane; q < 32 * kHc; q += kWave) {
          const int row = q / kHc, c = q % kHc, r = nt * 32 + row;
          const u32x4 v = scr[row * kHc + (c ^ (row & (kHc - 1)))];
          if (r < R) put4(slot1 + (int64_t)r * D + hm * (D / 2) + 4 * c, v);
        }
      }
      if (half == 0 && lr < R) {
        put1(slot1 + (int64_t)p.rmax * D + lr, m[nt]);
        put1(slot1 + (int64_t)p.rmax * D + p.rmax + lr, lt);
      }
    }
  }

  // the stashed partial to slot 0, 16 bytes per lane and step, stored as above (the wave's own
  // LDS writes are complete before its reads).  (Issued instead right after the share's last tile load, so that
  // the stores drain under the last tiles' compute, it needed the loop split in two, and the
  // kernel ran slower.)
  if (stashed) {
    for (int idx = lane; idx < stash_rows * D / 4; idx += kWave)
      put4(slots + 4 * (int64_t)idx, __builtin_bit_cast(u32x4, sm_stash[wave][idx]));
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int r = nt * 32 + col;
      if (half == 0 && r < stash_rows) {
        put1(slots + (int64_t)p.rmax * D + r, st_m[nt]);
        put1(slots + (int64_t)p.rmax * D + p.rmax + r, st_l[nt]);
      }
    }
  }

  // header of the slot-1 partial: the item this wave starts and a later share finishes
  if (lane == 0) {
    *reinterpret_cast<u32x4*>(hdr) = u32x4{(uint32_t)head_flag, (uint32_t)head_b, (uint32_t)head_f, (uint32_t)head_nt};
    *reinterpret_cast<u32x4*>(hdr + 4) = u32x4{(uint32_t)P, (uint32_t)head_q0, (uint32_t)head_n, (uint32_t)dlt};
  }
}

// Combines the partials of every item cut between shares: workgroup w handles the item whose
// first tiles wave w (share s, head h) holds, in its slot 1; shares s+1 .. s_last of head h
// hold the rest, in their slot 0, where s_last holds the item's last tile.
//   o = sum_c acc_c 2^(m_c - M) / sum_c l_c 2^(m_c - M),   M = max_c m_c
// Contributors are read four at a time, every load of a group issued together.
// U: output values per thread (4 or 8); the launcher takes 8 when one pass of the workgroup's
// threads then covers an item's rows (up to 32), 4 for taller items.
template <int D, int U>
__global__ __launch_bounds__(512) void attn_merge_kernel(AttnParams p) {
  const int w = blockIdx.x;
  const int64_t slot_f = attn_slot_floats(p.rmax, D);
  const int32_t* hdr = reinterpret_cast<const int32_t*>(p.ws + (int64_t)p.nwaves * 2 * slot_f) +
                       (int64_t)w * kAttnHdrInts;
  const u32x4 h0 = *reinterpret_cast<const u32x4*>(hdr);
  const u32x4 h1 = *reinterpret_cast<const u32x4*>(hdr + 4);   // loaded with h0: one round trip
  if (h0[0] != 1u) return;
  const int f = (int)h0[2], nt = (int)h0[3], P = (int)h1[0], q0 = (int)h1[1], n = (int)h1[2], dlt = (int)h1[3];
  const int h = w % p.hkv, s0 = w / p.hkv;
  const int C = min(share_of(f + nt - 1, P, dlt), p.nshares - 1) - s0 + 1;   // contributing shares
  const int R = p.group * n;
  const int64_t mo = (int64_t)p.rmax * D, lo = mo + p.rmax;
  auto slot = [&](int c) -> const float* {
    return p.ws + ((int64_t)((s0 + c) * p.hkv + h) * 2 + (c == 0 ? 1 : 0)) * slot_f;
  };
  constexpr int NQ = U / 4;   // f32x4 per contributor and thread
  for (int idx = threadIdx.x; idx < R * (D / U); idx += blockDim.x) {
    const int r = idx / (D / U), d = (idx % (D / U)) * U;
    float M = kNegBig, den = 0.f;
    f32x4 o[NQ];
#pragma unroll
    for (int v = 0; v < NQ; ++v) o[v] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < C; c0 += 4) {
      float mv[4], lv[4];
      f32x4 av[4][NQ];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float* sp = slot(min(c0 + k, C - 1));
        mv[k] = sp[mo + r];
        lv[k] = sp[lo + r];
#pragma unroll
        for (int v = 0; v < NQ; ++v) {
          // read once: non-temporal for items of up to 32 rows (whose partials the caches
          // hold; the call 0.5 us faster and the acceptance after it 0.9 us at 20 rows), plain
          // for taller ones (their partials come from memory; non-temporal loads were 2.4 us
          // slower at 63 rows)
          const f32x4* a = reinterpret_cast<const f32x4*>(sp + (int64_t)r * D + d + 4 * v);
          av[k][v] = U == 8 ? __builtin_nontemporal_load(a) : *a;
        }
      }
      float mc = M;
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (c0 + k < C) mc = fmaxf(mc, mv[k]);
      const float a = fast_exp2(M - mc);
      den *= a;
#pragma unroll
      for (int v = 0; v < NQ; ++v) o[v] *= a;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (c0 + k >= C) continue;
        const float e = fast_exp2(mv[k] - mc);
        den += e * lv[k];
#pragma unroll
        for (int v = 0; v < NQ; ++v) o[v] += av[k][v] * e;
      }
      M = mc;
    }
    const float inv = 1.0f / den;
    const int j = r / p.group, gq = r % p.group;
    uint16_t* orow = reinterpret_cast<uint16_t*>(p.out) + ((int64_t)(q0 + j) * p.hq + h * p.group + gq) * D;
#pragma unroll
    for (int v = 0; v < NQ; ++v) {
      u32x2 v2;
      v2[0] = pack_bf16x2(o[v][0] * inv, o[v][1] * inv);
      v2[1] = pack_bf16x2(o[v][2] * inv, o[v][3] * inv);
      // final outputs, read only by a later kernel: non-temporal, so that it does not write
      // them back out of the caches (2.9 us per step at workload 2, 9.8 us at workload 5)
      __builtin_nontemporal_store(v2, reinterpret_cast<u32x2*>(orow + d + 4 * v));
    }
  }
}

template <int D, int BS, int NT>
static hipError_t launch_attn_t(const AttnParams& p, hipStream_t s) {
  hipLaunchKernelGGL((verify_attn_kernel<D, BS, NT>), dim3((unsigned)(p.nwaves / 4)), dim3(256), 0, s, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // 512 threads: fewer items per thread
  if (p.rmax <= 32)
    hipLaunchKernelGGL((attn_merge_kernel<D, 8>), dim3((unsigned)p.nwaves), dim3(512), 0, s, p);
  else
    hipLaunchKernelGGL((attn_merge_kernel<D, 4>), dim3((unsigned)p.nwaves), dim3(512), 0, s, p);
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
