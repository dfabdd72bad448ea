// LM-head projection in front of acceptance, with the softmax statistics fused into its
// epilogue.  The verifying stage owns an LM head (Implementation); its logits are the target
// rows acceptance reads (Sec. 4, Related Work [sd]).  For bf16 h [M][d] and W [V][d]:
//   logits[m][v] = sum_j h[m][j] W[v][j]   (fp32 accumulation, fp32 output)
// and for every row and 128-column tile, at temperature T (c = log2(e)/T):
//   stats = (max_v x*c, sum_v 2^(x*c - max))   over the tile's columns v < V.
// Acceptance combines the tiles of a row into its normaliser without reading the row again.
//
// Work decomposition: one workgroup per (vocabulary tile of 256 columns, or 128 for narrow
// outputs; group of up to 192 rows of h, or all of up to 128 rows); its four waves split the
// tile in a grid of waves (below), each holding 32x32 accumulator tiles of
// v_mfma_f32_32x32x16_bf16 (A operand: h rows, B operand: W rows).
//   * W, the stream that matters (V*d*2 bytes, read once), goes straight from HBM into each
//     wave's registers, DEPTH K-steps of 64 ahead.  It is packed (pack.hip) so that each operand
//     load of a wave reads 1 KB of contiguous memory; lane half h takes K = 32h + 8s .. +7 of
//     its column at MFMA step s (the contraction order over K is free as long as h uses the
//     same).
//   * h is shared by the four waves: it goes through LDS, one step per stage, fetched into
//     registers NA steps ahead (NA register sets).  Wait counts retire in issue order: the wait
//     for h step i+1 leaves the NA steps of W loaded after it in flight, and W runs DEPTH >=
//     NA + 2 steps ahead, so the compute of step i+1 never waits for its W.  Few row tiles leave
//     registers for NA = 4, DEPTH = 8 (one column tile per wave); two column tiles per wave and
//     the larger row groups use NA = 2, DEPTH = 4.
//   * Each XCD takes blocks of its vocabulary tiles x row groups (tile_of), so its resident
//     workgroups share the K-slices of h and W they read through its L2.
#include "common.h"
#include "kernels.h"

namespace spexis {

namespace {

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;   // NaN
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_float(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }


// Waits until at most N LDS reads (or scalar loads) of the wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_lgkm() {
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// One 16-byte LDS read, written as an instruction (byte address addr).
__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  u32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr) : "memory");
  return v;
}
// Ties a register to the wait before it: no use of v moves above that wait.
__device__ __forceinline__ void tie(u32x4& v) { asm volatile("" : "+v"(v)); }
// A 16-byte-per-lane buffer load into LDS (lane l's bytes at lds + 16 l).  Kept out of the
// kernel templates: the host side of a template kernel cannot instantiate this builtin.
__device__ __forceinline__ void buffer_load_lds16(__amdgpu_buffer_rsrc_t rs, __attribute__((address_space(3))) void* lds,
                                                  int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds, 16, voff, soff, 0, 0);
}

// W rows are read once: non-temporal loads keep them from evicting h out of L2.
template <bool kStream>
__device__ __forceinline__ u32x4 ldw(const uint16_t* p) {
  if (kStream) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return *reinterpret_cast<const u32x4*>(p);
}

// Workgroup -> (vocabulary tile nt, row group mg).  Workgroup i runs on XCD i % 8, which takes
// the vocabulary tiles nt = 8 j + XCD; the XCD's workgroups, in launch order, walk blocks of
// kTileBlock of its tiles, and within a block the row groups in blocks of kGroupBlock, each
// (tiles x groups) block in tile-major order.  The XCD's resident workgroups (one per CU) then
// cover a few row groups of a few tiles at a time, so each K-step's slice of h and of W is
// fetched into the XCD's L2 once for several workgroups.
constexpr int kTileBlock = 8, kGroupBlock = 4;
__device__ __forceinline__ void tile_of(int bid, int ntiles, int groups, int& nt, int& mg) {
  const int xcd = bid & 7, local = bid >> 3;
  const int per_xcd = (ntiles + 7) / 8;                     // tiles of an XCD (the last may be absent)
  const int tb = local / (kTileBlock * groups), rem = local % (kTileBlock * groups);
  const int ctb = min(kTileBlock, per_xcd - tb * kTileBlock);   // tiles in this block
  const int full = groups / kGroupBlock * kGroupBlock;      // groups in whole group blocks
  int t, g;
  if (rem < ctb * full) {
    const int gb = rem / (ctb * kGroupBlock), r2 = rem % (ctb * kGroupBlock);
    t = r2 / kGroupBlock;
    g = gb * kGroupBlock + r2 % kGroupBlock;
  } else {
    const int r2 = rem - ctb * full, tail = groups - full;
    t = r2 / tail;
    g = full + r2 % tail;
  }
  nt = 8 * (tb * kTileBlock + t) + xcd;
  mg = g;
}

}  // namespace

// Waves form a WR x WC grid over the workgroup's (32 * WR * RT) rows x (32 * WC * CT) columns:
// wave (wr, wc) computes RT row tiles x CT column tiles.  The launched shapes put the four waves
// side by side (WR = 1) with two column tiles each (256 columns per workgroup): against one tile
// each, that halves the h fragments each wave reads from LDS per MFMA and the h rows staged per
// column.  (A 2 x 2 grid over 128 columns does the former but loads each W tile twice.)
// Statistics stay per 128-column tile: a 256-column workgroup writes two.
template <bool kStream, int RT, int CT, int WR, int NA, int DEPTH, int WPE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE)))
void lm_head_kernel(LmParams p) {
  static_assert(DEPTH >= NA + 2 && DEPTH % NA == 0 && DEPTH % 2 == 0, "pipeline shape");
  constexpr int WC = 4 / WR;
  constexpr int kCols = 32 * WC * CT;           // columns of the workgroup
  constexpr int kStatTiles = kCols / kLmCols;   // its 128-column statistics tiles
  static_assert(WR * WC == 4 && (kCols == 128 || kCols == 256), "wave grid");
  constexpr int NRT = WR * RT;   // row tiles of the workgroup
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  const int wr = wave / WC, wc = wave % WC;
  const int wgcols = (p.V + kCols - 1) / kCols;
  int nt, mg;
  tile_of(blockIdx.x, wgcols, p.mgroups, nt, mg);
  if (nt >= wgcols) return;
  const int m0 = mg * 32 * NRT, n0 = nt * kCols;
  const int rows = min(32 * NRT, p.M - m0);
  // K split: workgroup row ks takes K values ks * klen .. +klen-1 (nsteps steps of 64)
  const int ks = blockIdx.y;
  const int klen = p.d / p.ksplit, nsteps = klen / kLmK;
  // column tile c of this wave is packed tile row n0 / 32 + CT wc + c (clamped for the columns
  // past V, whose results are dropped); lane l reads 16 contiguous bytes at s * 512 + 8 l of each
  // tile
  const uint16_t* wrow[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) {
    const int wtile = min(n0 / 32 + CT * wc + c, (p.V + 31) / 32 - 1);
    wrow[c] = reinterpret_cast<const uint16_t*>(p.w) +
              ((int64_t)wtile * (p.d / kLmK) + (int64_t)ks * nsteps) * kPackTile + 8 * lane;
  }
  const uint16_t* hbase = reinterpret_cast<const uint16_t*>(p.h) + (int64_t)m0 * p.d + (int64_t)ks * klen;

  // h in LDS: stage x, row r, 16-byte chunk kc of the step stored at position kc ^ ((r >> 1) & 7),
  // so that the 16 rows one ds_read_b128 pass serves hit 16 distinct 16-byte bank groups.  Only
  // the workgroup's NRT row tiles are staged: 32 * NRT rows * 8 chunks = NRT chunks per thread.
  // (At least 72 rows: the epilogue transposes 4 x 32 x 36 floats through this space.)
  constexpr int kAChunks = NRT;
  constexpr int kStage = (32 * NRT > 72 ? 32 * NRT : 72) * 8;
  __shared__ u32x4 sm_a[2][kStage];
  u32x4 areg[NA][kAChunks];   // h chunks of the next NA steps, in flight
  auto load_a = [&](u32x4 (&dst)[kAChunks], int j) {
    j = min(j, nsteps - 1);   // past the end: re-read the last step (kept unconditional)
#pragma unroll
    for (int u = 0; u < kAChunks; ++u) {
      const int q = threadIdx.x + 256 * u;
      const int r = min(q >> 3, rows - 1), kc = q & 7;
      dst[u] = *reinterpret_cast<const u32x4*>(hbase + (int64_t)r * p.d + j * kLmK + 8 * kc);
    }
  };
  auto store_a = [&](const u32x4 (&src)[kAChunks], int stage) {
#pragma unroll
    for (int u = 0; u < kAChunks; ++u) {
      const int q = threadIdx.x + 256 * u;
      const int r = q >> 3, kc = q & 7;
      sm_a[stage][r * 8 + (kc ^ ((r >> 1) & 7))] = src[u];
    }
  };
  u32x4 wb[DEPTH][CT][4];
  auto load_w = [&](u32x4 (&dst)[CT][4], int j) {
    const int64_t off = (int64_t)min(j, nsteps - 1) * kPackTile;
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int s = 0; s < 4; ++s) dst[c][s] = ldw<kStream>(wrow[c] + off + 512 * s);
  };

  f32x16 acc[RT][CT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[t][c][e] = 0.f;

  // prologue: h step 0 into stage 0, W steps 0 .. DEPTH-1, h steps 1 .. NA into registers
  load_a(areg[0], 0);
#pragma unroll
  for (int b = 0; b < DEPTH; ++b) load_w(wb[b], b);
  store_a(areg[0], 0);
#pragma unroll
  for (int a = 1; a <= NA; ++a) load_a(areg[a % NA], a);
  __syncthreads();

  // The A fragments of k-step s+1 are read from LDS while the MFMAs of k-step s run.
  auto frag = [&](int stage, int t, int s) {
    const int m = 32 * (wr * RT + t) + col;
    return sm_a[stage][m * 8 + ((4 * half + s) ^ ((m >> 1) & 7))];
  };
  auto compute = [&](const u32x4 (&w)[CT][4], int stage) {
    u32x4 fa[2][RT];
#pragma unroll
    for (int t = 0; t < RT; ++t) fa[0][t] = frag(stage, t, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s + 1 < 4) {
#pragma unroll
        for (int t = 0; t < RT; ++t) fa[(s + 1) & 1][t] = frag(stage, t, s + 1);
      }
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const bf16x8 bop = as_bf16x8(w[c][s]);
#pragma unroll
        for (int t = 0; t < RT; ++t)
          acc[t][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(fa[s & 1][t]), bop, acc[t][c], 0, 0, 0);
      }
    }
  };

  // step i: compute from stage i%2 and W buffer i%DEPTH; move h step i+1 (fetched NA steps ago)
  // into the other stage and fetch h step i+1+NA into the same registers; refill the W buffer
  // with step i+DEPTH
  for (int j = 0; j < nsteps; j += DEPTH) {
#pragma unroll
    for (int jj = 0; jj < DEPTH; ++jj) {
      if (j + jj < nsteps) compute(wb[jj], jj & 1);
      store_a(areg[(jj + 1) % NA], (jj + 1) & 1);
      load_a(areg[(jj + 1) % NA], j + jj + 1 + NA);
      load_w(wb[jj], j + jj + DEPTH);
      __syncthreads();
    }
  }

  // ---- epilogue: logits (or partials, or bf16 outputs), and each row's statistics over each
  // of this workgroup's 128-column statistics tiles.  Accumulator value i of lane l in tile (t, c): row
  // 32 (wr RT + t) + 8 (i / 4) + 4 (l / 32) + i % 4, column 32 (CT wc + c) + l % 32.
  auto out_row = [&](int t, int i) { return 32 * (wr * RT + t) + 8 * (i >> 2) + 4 * half + (i & 3); };
  auto out_col = [&](int c) { return n0 + 32 * (CT * wc + c) + col; };
  // Logits (or K-split partials) are written once and read by a later kernel: non-temporal
  // stores keep them from evicting the h and W lines the other workgroups still read through L2
  // (measured at 320 x 4096 @ 128256: 469 against 480 us; at 4608 x 3584 @ 152064: 5332 against
  // 5684 us).
  // the gather columns of the rows lanes below 32 reduce in the statistics (loaded first: their
  // latency passes under the logits stores)
  int gcol[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int grow = 32 * (wr * RT + t) + lane;
    gcol[t] = p.gout && p.stats && lane < 32 && grow < rows ? p.gcols[m0 + grow] : -1;
  }
  if (p.logits) {
    float* out = p.logits + (int64_t)ks * p.M * p.V;
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int v = out_col(c);
      if (v >= p.V) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = out_row(t, i);
          if (r < rows) __builtin_nontemporal_store(acc[t][c][i], out + (int64_t)(m0 + r) * p.V + v);
        }
    }
  }
  if (p.y) {
    const uint16_t* res = reinterpret_cast<const uint16_t*>(p.res);
    uint16_t* y = reinterpret_cast<uint16_t*>(p.y);
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int v = out_col(c);
      if (v >= p.V) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = out_row(t, i);
          if (r < rows) {
            const int64_t at = (int64_t)(m0 + r) * p.V + v;
            y[at] = bf16_rne(res ? acc[t][c][i] + bf16_float(res[at]) : acc[t][c][i]);
          }
        }
    }
  }
  if (!p.stats) return;
  // Row statistics: each wave transposes one 32x32 tile at a time through its part of the (now
  // free) h stages; lane r < 32 reduces row r over the tile's 32 columns, then over the wave's
  // CT tiles in order; the waves of a row and 128-column statistics tile are combined in order
  // at the end.
  __shared__ float sm_m[WC][32 * NRT], sm_z[WC][32 * NRT];
  constexpr int kTS = 36;   // floats per transposed row (16-byte aligned, padded)
  float* tile = reinterpret_cast<float*>(&sm_a[0][0]) + wave * 32 * kTS;
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    float wm = -INFINITY, wz = 0.f;
    const int grow = 32 * (wr * RT + t) + lane;
    const int gc = gcol[t];
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const bool live = out_col(c) < p.V;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        tile[(8 * (i >> 2) + 4 * half + (i & 3)) * kTS + col] = live ? acc[t][c][i] : -INFINITY;
      if (lane < 32) {
        // x c rounded once, then x c - max: no contraction into one fused operation
#pragma clang fp contract(off)
        f32x4 x[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) x[q] = *reinterpret_cast<const f32x4*>(tile + lane * kTS + 4 * q) * p.c;
        const int cb = out_col(c) - col;   // the tile's first column
        if (gc >= cb && gc < cb + 32 && gc < p.V) p.gout[m0 + grow] = tile[lane * kTS + (gc - cb)];
        float mx = -INFINITY;
#pragma unroll
        for (int q = 0; q < 8; ++q) mx = fmaxf(fmaxf(mx, fmaxf(x[q][0], x[q][1])), fmaxf(x[q][2], x[q][3]));
        float e = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
          for (int q = 0; q < 8; ++q)
#pragma unroll
            for (int u = 0; u < 4; ++u) e += fast_exp2(x[q][u] - mx);
        }
        if (c == 0) {
          wm = mx;
          wz = e;
        } else {
          const float M = fmaxf(wm, mx);
          wz = (wm != -INFINITY ? wz * fast_exp2(wm - M) : 0.f) + (mx != -INFINITY ? e * fast_exp2(mx - M) : 0.f);
          wm = M;
        }
      }
    }
    if (lane < 32) {
      sm_m[wc][32 * (wr * RT + t) + lane] = wm;
      sm_z[wc][32 * (wr * RT + t) + lane] = wz;
    }
  }
  __syncthreads();
  constexpr int kWavesPerStat = WC / kStatTiles;   // waves of a row within one statistics tile
  for (int q = threadIdx.x; q < rows * kStatTiles; q += 256) {
    const int r = q % rows, st = q / rows, w0 = st * kWavesPerStat;
    const int tile = nt * kStatTiles + st;
    if (tile >= p.ntiles) continue;
    float M = sm_m[w0][r];
#pragma unroll
    for (int w = 1; w < kWavesPerStat; ++w) M = fmaxf(M, sm_m[w0 + w][r]);
    float Z = 0.f;
#pragma unroll
    for (int w = 0; w < kWavesPerStat; ++w)
      if (sm_m[w0 + w][r] != -INFINITY) Z += sm_z[w0 + w][r] * fast_exp2(sm_m[w0 + w][r] - M);
    *reinterpret_cast<f32x2*>(p.stats + ((int64_t)(m0 + r) * p.ntiles + tile) * 2) = f32x2{M, Z};
  }
}

// More than 160 rows of a wide projection (an LM head's vocabulary): one workgroup of eight waves
// (two per SIMD) per (256-column tile, group of 320 rows), so that each K-slice of W crosses L2
// once per 320 rows.  Both operands go through LDS: every K-step of 64 the
// workgroup copies h (320 rows, 40 KB) and W (eight packed 32-column tiles, 32 KB) from memory
// straight into one of two stages, a step ahead, and the waves read their fragments from the
// stage, those of the next MFMA step while the current step's MFMAs run.  Wave (wr, wc) of a
// 2 x 4 grid computes rows 160 wr .. +160 (five row tiles)
// by columns 64 wc .. +64 (two column tiles): 160 accumulators, within the 256 registers a wave
// has at two waves per SIMD.  Against four waves per 160-row x 256-column workgroup (two row
// groups, each reading W), the L2 serves about 2.35 GB instead of 3.4 GB at 320 x 4096 @ 128256.
// Epilogue as lm_head_kernel's: logits or bf16 outputs, then each row's statistics per
// 128-column tile.
template <int RT, int CT, int WR, int WC>
__global__ __launch_bounds__(64 * WR * WC) __attribute__((amdgpu_waves_per_eu(WR * WC / 4)))
void lm_head_wide_kernel(LmParams p) {
  constexpr int NRT = WR * RT;        // row tiles of the workgroup
  constexpr int kRows = 32 * NRT;     // rows of the group
  constexpr int kCols = 32 * WC * CT; // columns of the workgroup
  constexpr int kStatTiles = kCols / kLmCols;
  static_assert(kCols == 256 && WC % kStatTiles == 0, "two 128-column statistics tiles, whole waves each");
  // the wave index wave-uniform (scalar), so the copies' LDS destinations are scalar sums
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63, col = lane & 31, half = lane >> 5;
  const int wr = wave / WC, wc = wave % WC;
  const int wgcols = (p.V + kCols - 1) / kCols;
  int nt, mg;
  tile_of(blockIdx.x, wgcols, p.mgroups, nt, mg);
  if (nt >= wgcols) return;
  const int n0 = nt * kCols, m0 = mg * kRows;
  const int rows = min(kRows, p.M - m0);
  const int nsteps = p.d / kLmK;
  const int wtiles = (p.V + 31) / 32;
  const uint16_t* hbase = reinterpret_cast<const uint16_t*>(p.h) + (int64_t)m0 * p.d;
  const uint16_t* wbase = reinterpret_cast<const uint16_t*>(p.w);

  // stage x of h: row r, chunk kc (8 K values) at r * 8 + (kc ^ ((r >> 1) & 7)) (the 16 rows of
  // one ds_read_b128 pass hit distinct bank groups); stage x of W: packed tile c (columns
  // n0 + 32 c ..), its 256 chunks in packed order.  One array: h stages 0 and 1, then W stages
  // 0 and 1.
  constexpr int kHStage = kRows * 8, kWStage = kCols / 32 * 256;
  __shared__ u32x4 sm[2 * kHStage + 2 * kWStage];
  // Copies go from memory straight into a stage (buffer loads to LDS, 1 KB per wave and
  // instruction, lane l's 16 bytes at slot 64 u + l): no staging registers, which leaves room
  // for two sets of operand fragments.  Buffer resources span the group's rows of h and the
  // workgroup's packed W tiles: loads past them (rows past M, columns past V) return zeros,
  // whose results are dropped.
  constexpr int kWaves = WR * WC;
  constexpr int kHCopies = kHStage / 64 / kWaves;   // copy instructions per wave and step
  constexpr int kWCopies = kWStage / 64 / kWaves;
  static_assert(kHStage % (64 * kWaves) == 0 && kWStage % (64 * kWaves) == 0, "copy split");
  const int wt0 = n0 / 32, wtn = min(kCols / 32, wtiles - wt0);
  const __amdgpu_buffer_rsrc_t hrs =
      __builtin_amdgcn_make_buffer_rsrc((void*)hbase, (short)0, rows * p.d * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(wbase + (int64_t)wt0 * (p.d / kLmK) * kPackTile), (short)0, wtn * (p.d / kLmK) * kPackTile * 2,
      0x00020000);
  int hoff[kHCopies], woff[kWCopies];   // byte offsets of the lane's chunks at step 0
#pragma unroll
  for (int u = 0; u < kHCopies; ++u) {
    const int q = (wave * kHCopies + u) * 64 + lane;
    const int r = q >> 3, kc = (q & 7) ^ ((r >> 1) & 7);
    hoff[u] = (r * p.d + 8 * kc) * 2;
  }
#pragma unroll
  for (int u = 0; u < kWCopies; ++u) {
    const int q = (wave * kWCopies + u) * 64 + lane;
    woff[u] = ((q >> 8) * (p.d / kLmK) * kPackTile + 8 * (q & 255)) * 2;
  }
  auto copy_step = [&](int j, int stage) {
#pragma unroll
    for (int u = 0; u < kHCopies; ++u)
      buffer_load_lds16(hrs, (__attribute__((address_space(3))) void*)(sm + stage * kHStage + (wave * kHCopies + u) * 64),
                        hoff[u], j * kLmK * 2);
#pragma unroll
    for (int u = 0; u < kWCopies; ++u)
      buffer_load_lds16(
          wrs, (__attribute__((address_space(3))) void*)(sm + 2 * kHStage + stage * kWStage + (wave * kWCopies + u) * 64),
          woff[u], j * kPackTile * 2);
  };

  f32x16 acc[RT][CT];
#pragma unroll
  for (int t = 0; t < RT; ++t)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[t][c][e] = 0.f;

  // Fragment reads are written as instructions: the compiler would make every LDS read wait for
  // all copies to LDS in flight (into either stage), which cancels the copies' prefetch.  The
  // reads of MFMA step s + 1 go out before step s's MFMAs, and each step waits for its own
  // fragments by count (LDS reads return in order).  Byte addresses: A fragment of row tile t at
  // step s, h stage + (32 (wr RT + t) + col) * 128 + ((4 half + s) ^ ((col >> 1) & 7)) * 16 (row
  // m's swizzle (m >> 1) & 7 is col's, 32 (wr RT + t) being a multiple of 16); B fragment of
  // column tile c, W stage + ((CT wc + c) * 256 + 64 s + lane) * 16.
  static_assert(RT + CT <= 15, "one lgkmcnt covers a step's fragment reads");
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) u32x4*)sm;   // LDS byte address
  uint32_t aaddr[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    aaddr[s] = lds0 + (32 * wr * RT + col) * 128 + (((4 * half + s) ^ ((col >> 1) & 7)) << 4);
  const uint32_t baddr = lds0 + 2 * kHStage * 16 + (CT * wc * 256 + lane) * 16;
  auto lds_read = [](uint32_t addr) { return lds_read_b128(addr); };
  auto compute = [&](int stage) {
    u32x4 a[2][RT], b[2][CT];
    auto frags = [&](int s, int x) {
#pragma unroll
      for (int t = 0; t < RT; ++t) a[x][t] = lds_read(aaddr[s] + stage * kHStage * 16 + t * 4096);
#pragma unroll
      for (int c = 0; c < CT; ++c) b[x][c] = lds_read(baddr + stage * kWStage * 16 + c * 4096 + s * 1024);
    };
    frags(0, 0);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int x = s & 1;
      if (s < 3) {
        frags(s + 1, x ^ 1);
        wait_lgkm<RT + CT>();   // this step's reads done; the next step's stay in flight
      } else {
        wait_lgkm<0>();
      }
      // tie the fragments to the wait, so that no use of them moves above it
#pragma unroll
      for (int t = 0; t < RT; ++t) tie(a[x][t]);
#pragma unroll
      for (int c = 0; c < CT; ++c) tie(b[x][c]);
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int c = 0; c < CT; ++c)
          acc[t][c] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a[x][t]), as_bf16x8(b[x][c]), acc[t][c], 0, 0, 0);
    }
  };

  // step j: wait for this wave's copies of step j, then the barrier makes every wave's copies
  // visible and tells that all have finished step j - 1, whose stage step j + 1 now fills while
  // step j is computed
  copy_step(0, 0);
  for (int j = 0; j < nsteps; ++j) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (j + 1 < nsteps) copy_step(j + 1, (j + 1) & 1);
    compute(j & 1);
  }
  __syncthreads();   // the epilogue's transposes reuse h stage 0

  // ---- epilogue (accumulator value i of lane l in tile (t, c): row 32 (wr RT + t) + 8 (i / 4)
  // + 4 (l / 32) + i % 4, column 32 (CT wc + c) + l % 32)
  auto out_row = [&](int t, int i) { return 32 * (wr * RT + t) + 8 * (i >> 2) + 4 * half + (i & 3); };
  auto out_col = [&](int c) { return n0 + 32 * (CT * wc + c) + col; };
  // the gather columns of the rows lanes below 32 reduce in the statistics (loaded first: their
  // latency passes under the logits stores)
  int gcol[RT];
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    const int grow = 32 * (wr * RT + t) + lane;
    gcol[t] = p.gout && p.stats && lane < 32 && grow < rows ? p.gcols[m0 + grow] : -1;
  }
  if (p.logits) {
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int v = out_col(c);
      if (v >= p.V) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = out_row(t, i);
          if (r < rows) __builtin_nontemporal_store(acc[t][c][i], p.logits + (int64_t)(m0 + r) * p.V + v);
        }
    }
  }
  if (p.y) {
    const uint16_t* res = reinterpret_cast<const uint16_t*>(p.res);
    uint16_t* y = reinterpret_cast<uint16_t*>(p.y);
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const int v = out_col(c);
      if (v >= p.V) continue;
#pragma unroll
      for (int t = 0; t < RT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int r = out_row(t, i);
          if (r < rows) {
            const int64_t at = (int64_t)(m0 + r) * p.V + v;
            y[at] = bf16_rne(res ? acc[t][c][i] + bf16_float(res[at]) : acc[t][c][i]);
          }
        }
    }
  }
  if (!p.stats) return;
  // Row statistics: each wave transposes one 32x32 tile at a time through its part of the (now
  // free) h stages; lane r < 32 reduces row r over the tile's 32 columns, then over the wave's CT
  // tiles in order; the two waves of a row and 128-column statistics tile combine in order.
  __shared__ float sm_m[WC][kRows], sm_z[WC][kRows];
  constexpr int kTS = 36;   // floats per transposed row (16-byte aligned, padded)
  float* tile = reinterpret_cast<float*>(&sm[0]) + wave * 32 * kTS;
#pragma unroll
  for (int t = 0; t < RT; ++t) {
    float wm = -INFINITY, wz = 0.f;
    const int grow = 32 * (wr * RT + t) + lane;
    const int gc = gcol[t];
#pragma unroll
    for (int c = 0; c < CT; ++c) {
      const bool live = out_col(c) < p.V;
#pragma unroll
      for (int i = 0; i < 16; ++i)
        tile[(8 * (i >> 2) + 4 * half + (i & 3)) * kTS + col] = live ? acc[t][c][i] : -INFINITY;
      if (lane < 32) {
        // x c rounded once, then x c - max: no contraction into one fused operation
#pragma clang fp contract(off)
        f32x4 x[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) x[q] = *reinterpret_cast<const f32x4*>(tile + lane * kTS + 4 * q) * p.c;
        const int cb = out_col(c) - col;   // the tile's first column
        if (gc >= cb && gc < cb + 32 && gc < p.V) p.gout[m0 + grow] = tile[lane * kTS + (gc - cb)];
        float mx = -INFINITY;
#pragma unroll
        for (int q = 0; q < 8; ++q) mx = fmaxf(fmaxf(mx, fmaxf(x[q][0], x[q][1])), fmaxf(x[q][2], x[q][3]));
        float e = 0.f;
        if (mx != -INFINITY) {
#pragma unroll
          for (int q = 0; q < 8; ++q)
#pragma unroll
            for (int u = 0; u < 4; ++u) e += fast_exp2(x[q][u] - mx);
        }
        if (c == 0) {
          wm = mx;
          wz = e;
        } else {
          const float M = fmaxf(wm, mx);
          wz = (wm != -INFINITY ? wz * fast_exp2(wm - M) : 0.f) + (mx != -INFINITY ? e * fast_exp2(mx - M) : 0.f);
          wm = M;
        }
      }
    }
    if (lane < 32) {
      sm_m[wc][32 * (wr * RT + t) + lane] = wm;
      sm_z[wc][32 * (wr * RT + t) + lane] = wz;
    }
  }
  __syncthreads();
  constexpr int kWavesPerStat = WC / kStatTiles;
  for (int q = threadIdx.x; q < rows * kStatTiles; q += 64 * kWaves) {
    const int r = q % rows, st = q / rows, w0 = st * kWavesPerStat;
    const int stile = nt * kStatTiles + st;
    if (stile >= p.ntiles) continue;
    float M = sm_m[w0][r];
#pragma unroll
    for (int w = 1; w < kWavesPerStat; ++w) M = fmaxf(M, sm_m[w0 + w][r]);
    float Z = 0.f;
#pragma unroll
    for (int w = 0; w < kWavesPerStat; ++w)
      if (sm_m[w0 + w][r] != -INFINITY) Z += sm_z[w0 + w][r] * fast_exp2(sm_m[w0 + w][r] - M);
    *reinterpret_cast<f32x2*>(p.stats + ((int64_t)(m0 + r) * p.ntiles + stile) * 2) = f32x2{M, Z};
  }
}

template <int RT, int CT, int WR, int NA, int DEPTH, int WPE>
static hipError_t launch_lm_nrt(const LmParams& q, hipStream_t s) {
  // grid: tiles of 8 vocabulary tiles (one per XCD) x row groups of 32 WR RT rows, row groups
  // innermost; y: K split
  LmParams p = q;
  p.mgroups = (p.M + 32 * WR * RT - 1) / (32 * WR * RT);
  const int wgcols = (p.V + 32 * (4 / WR) * CT - 1) / (32 * (4 / WR) * CT);
  const int64_t grid = (int64_t)((wgcols + 7) / 8) * 8 * p.mgroups;
  const dim3 g((unsigned)grid, (unsigned)p.ksplit);
  if (p.mgroups == 1)
    hipLaunchKernelGGL((lm_head_kernel<true, RT, CT, WR, NA, DEPTH, WPE>), g, dim3(256), 0, s, p);
  else
    hipLaunchKernelGGL((lm_head_kernel<false, RT, CT, WR, NA, DEPTH, WPE>), g, dim3(256), 0, s, p);
  return hipGetLastError();
}

// Row groups of the many-row shape: 192 rows (six tiles) when that pads M to at most 5% more rows
// than groups of 160 (five tiles), else 160.  The larger group makes about 10% fewer L2 requests
// per output (measured 4.73 against 4.98 ms at 4608 x 3584 @ 152064); 320 rows keep two groups
// of 160 rather than two of 192.
static int64_t group_rows(int64_t M) {
  const int64_t p160 = (M + 159) / 160 * 160, p192 = (M + 191) / 192 * 192;
  return p192 * 20 <= p160 * 21 ? 192 : 160;
}

// The eight-wave kernel takes 161 to 320 rows (one group), and more rows in groups of 320 when
// those pad M by no more than its speed per row makes up for: it ran 12% faster than the
// four-wave groups of 192 at 4608 x 3584 @ 152064 (4273 against 4885 us without logits), so it
// is taken while its padded rows stay within 1.12 times theirs.
static bool wide_rows(int64_t M) {
  const int64_t g = group_rows(M);
  return M <= 320 || (M + 319) / 320 * 320 * 100 <= (M + g - 1) / g * g * 112;
}

// Up to 128 rows, 256-column workgroups when the columns alone give at least one workgroup per
// CU (an LM head's vocabulary); narrower outputs (hidden-size projections) keep 128 columns, whose
// twice as many workgroups the K split then fills the chip with.
static bool wide_columns(int64_t M, int64_t N) { return M > 128 || (N + 255) / 256 >= 256; }

int64_t projection_workgroups(int64_t M, int64_t N) {
  // the shapes launch_projection picks: one row group up to 128 rows, groups of 160 or 192 rows
  // beyond
  const int64_t cols = wide_columns(M, N) ? (N + 255) / 256 : (N + kLmCols - 1) / kLmCols;
  if (M <= 128) return cols;
  if (M > 160 && wide_rows(M)) return cols * ((M + 319) / 320);
  return cols * ((M + group_rows(M) - 1) / group_rows(M));
}

hipError_t launch_projection(const LmParams& p, hipStream_t s) {
  // row tiles computed per workgroup: the smallest instantiated count covering the rows (a
  // group of fewer rows repeats its last row in the padding tiles, whose results are dropped).
  // Wide shapes are 256 columns: four waves across, each two column tiles of 32 (wide_columns).
  // Up to 64 rows, a hint of two waves per SIMD; more rows take more accumulators and one.
  // Beyond 128 rows, groups of 160 or 192 rows (group_rows).  Every load -- h from L2, W from
  // HBM -- is an L1 miss, and each CU's capacity for pending misses bounds the streams, so wider
  // tiles' fewer requests per MFMA pay: at 4096 @ 128256, 180 against 188 us for 128-column
  // workgroups at 32 rows, 190 against 205 at 64, 215 against 265 at 128, and at 320 rows 437
  // against 460 us for 320 x 128 workgroups on a 2 x 2 wave grid.  Narrow outputs: 128 columns,
  // one column tile per wave.
  const int need = (p.M + 31) / 32;
  if (!wide_columns(p.M, p.V)) {
    if (need <= 1) return launch_lm_nrt<1, 1, 1, 4, 8, 2>(p, s);
    if (need <= 2) return launch_lm_nrt<2, 1, 1, 4, 8, 2>(p, s);
    return launch_lm_nrt<4, 1, 1, 4, 8, 1>(p, s);
  }
  if (need <= 1) return launch_lm_nrt<1, 2, 1, 2, 4, 2>(p, s);
  if (need <= 2) return launch_lm_nrt<2, 2, 1, 2, 4, 2>(p, s);
  if (need <= 4) return launch_lm_nrt<4, 2, 1, 2, 4, 1>(p, s);
  if (need >= 6 && p.ksplit == 1 && wide_rows(p.M)) {
    // groups of 320 rows, one eight-wave workgroup per (256-column tile, group): lm_head_wide_kernel
    LmParams q = p;
    q.mgroups = (p.M + 319) / 320;
    const int wgcols = (p.V + 255) / 256;
    hipLaunchKernelGGL((lm_head_wide_kernel<5, 2, 2, 4>), dim3((unsigned)((wgcols + 7) / 8 * 8 * q.mgroups)),
                       dim3(512), 0, s, q);
    return hipGetLastError();
  }
  if (group_rows(p.M) == 192) return launch_lm_nrt<6, 2, 1, 2, 4, 1>(p, s);
  return launch_lm_nrt<5, 2, 1, 2, 4, 1>(p, s);
}

}  // namespace spexis
