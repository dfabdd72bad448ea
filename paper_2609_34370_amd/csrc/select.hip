// Acceptance-guided selective speculation (Sec. 5): the draft tokens of a batch are ranked by
// confidence and the lowest-ranked fraction alpha is dropped before verification.  A draft's
// score is the confidence of its whole prefix -- the fp32 product of the draft probabilities
// along its sequence, in order -- since a draft can only be verified after every earlier one.
// Drafts are ordered by score, higher first, equal scores by lower index; the last m of that
// order are dropped, and each sequence keeps its drafts before its first dropped one.
//
// One workgroup does it all in LDS (at most 16384 drafts):
//   1. confidences into LDS (clamped), then each sequence's prefix products in place;
//   2. the score of rank R = N - m (the last kept one) by a radix select on the fp32 bits --
//      scores are non-negative, so their bit patterns order as integers -- four passes of 8
//      bits, MSB first.  Each pass counts the digits of the keys that match the digits chosen
//      so far into 32 copies of a 256-bin histogram (lane l adds to copy l % 32, so lanes with
//      equal digits hit distinct banks), sums the copies, and every wave finds the next digit;
//   3. a draft ranks in the first R if its score is above that threshold, or equal to it and
//      among the first `rem` such drafts by index (ordinals of ties from wave ballots, only
//      when the tie at the threshold is split);
//   4. each sequence keeps its prefix before the first draft outside the first R; a block scan
//      of kept_k + 1 gives the reduced batch's query_start_loc.
// Draft j lives with thread j % 1024 in every flat pass, so LDS accesses are unit-stride.
#include "common.h"
#include "kernels.h"

namespace spexis {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kPer = kSelectMaxDrafts / kThreads;   // drafts per thread in the flat passes (16)
constexpr int kCopies = 32;                          // histogram copies

// Draft range of a sequence whose query rows are a0 .. a1-1 (its qsl entries) in a batch of T
// tokens: first draft index d0 and count k, clamped so that every index stays inside the N
// drafts.
__device__ __forceinline__ void draft_range(const SelectParams& p, int b, int a0, int a1, int& d0, int& k) {
  a0 = clampi(a0, 0, p.T);
  a1 = clampi(a1, a0, p.T);
  k = min(max(a1 - a0 - 1, 0), p.N);
  d0 = clampi(a0 - b, 0, p.N - k);
}

// Exclusive scan of v over the workgroup; *total receives the sum.  Uses sm[kWaves].
__device__ __forceinline__ int block_excl_scan(int v, int* sm, int* total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int incl = wave_incl_scan_i32(v, lane);
  if (lane == kWave - 1) sm[wave] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int s = sm[w];
    before += w < wave ? s : 0;
    all += s;
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

}  // namespace

__global__ __launch_bounds__(kThreads) void select_kernel(SelectParams p) {
  __shared__ float sc[kSelectMaxDrafts];            // confidence, then prefix score, per draft
  __shared__ uint8_t fl[kSelectMaxDrafts];          // 1 if the draft ranks in the first R
  __shared__ u32x4 hist[2][256 * kCopies / 4];      // two histogram buffers, bin-major copies
  __shared__ int tot[256];
  __shared__ int rowcnt[kPer * kWaves];
  __shared__ int scan_sm[kWaves];
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int N = p.N, B = p.B, R = p.N - p.m;

  // query rows of this thread's first sequence (b = tid), fetched with the confidences
  const int q0 = p.qsl[min(tid, B)], q1 = p.qsl[min(tid + 1, B)];

  if (N > 0) {
    // 1. clamped confidences (NaN, negatives and -0 become +0), loads issued back to back
    float c[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) c[u] = p.conf[min(tid + kThreads * u, N - 1)];
#pragma unroll
    for (int u = 0; u < 2 * 256 * kCopies / 4 / kThreads; ++u)
      (&hist[0][0])[tid + kThreads * u] = u32x4{0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int j = tid + kThreads * u;
      if (j < N) sc[j] = c[u] > 0.f ? fminf(c[u], 1.f) : 0.f;
    }
    __syncthreads();
    for (int b = tid; b < B; b += kThreads) {
      int d0, k;
      draft_range(p, b, b == tid ? q0 : p.qsl[b], b == tid ? q1 : p.qsl[b + 1], d0, k);
      float s = 1.f;
      for (int i = 0; i < k; i += 4) {
        float x[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) x[v] = sc[min(d0 + i + v, N - 1)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          if (i + v < k) {
            s = s * x[v];   // fp32 product, round to nearest, in draft order
            sc[d0 + i + v] = s;
          }
        }
      }
    }
    __syncthreads();

    // 2. radix select of the R-th largest score (skipped when nothing is dropped)
    uint32_t thr = 0;
    int rem = 0, eq = 0;
    if (p.m > 0) {
      uint32_t prefix = 0;
      rem = R;
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        int* h = reinterpret_cast<int*>(&hist[pass & 1][0]);
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
          const int j = tid + kThreads * u;
          if (j < N) {
            const uint32_t x = __float_as_uint(sc[j]);
            if (pass == 0 || (x >> (shift + 8)) == prefix)
              atomicAdd(&h[((x >> shift) & 255) * kCopies + (lane & (kCopies - 1))], 1);
          }
        }
        __syncthreads();
        // bin totals: thread t sums copies 8(t%4) .. +7 of bin t/4 and clears them for the pass
        // after next (the next pass uses the other buffer)
        {
          u32x4* hv = &hist[pass & 1][0];
          const u32x4 a = hv[2 * tid], e = hv[2 * tid + 1];
          hv[2 * tid] = u32x4{0, 0, 0, 0};
          hv[2 * tid + 1] = u32x4{0, 0, 0, 0};
          int s = (int)(a[0] + a[1] + a[2] + a[3] + e[0] + e[1] + e[2] + e[3]);
          s += __builtin_amdgcn_mov_dpp(s, kDppQuadXor1, 0xF, 0xF, false);
          s += __builtin_amdgcn_mov_dpp(s, kDppQuadXor2, 0xF, 0xF, false);
          if ((tid & 3) == 0) tot[tid >> 2] = s;
        }
        __syncthreads();
        // every wave finds the digit: lane l holds digits 255-4l .. 252-4l, so a lane scan runs
        // from the top digit down
        int hh[4], t = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          hh[q] = tot[255 - 4 * lane - q];
          t += hh[q];
        }
        int cum = wave_incl_scan_i32(t, lane) - t;   // keys with a higher digit
        int dig = -1, r2 = 0, e2 = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if (cum < rem && cum + hh[q] >= rem) {
            dig = 255 - 4 * lane - q;
            r2 = rem - cum;
            e2 = hh[q];
          }
          cum += hh[q];
        }
        // exactly one lane finds it: rem <= the count of keys matching the digits so far
        const int src = __builtin_amdgcn_readfirstlane(__ffsll((unsigned long long)__ballot(dig >= 0)) - 1) & 63;
        prefix = (prefix << 8) | (uint32_t)__builtin_amdgcn_readlane(dig, src);
        rem = __builtin_amdgcn_readlane(r2, src);
        eq = __builtin_amdgcn_readlane(e2, src);
      }
      thr = prefix;   // the R-th largest score; `rem` of the `eq` drafts scoring exactly thr are kept
    }

    // 3. rank flags: above the threshold, or tied with it and among the first `rem` by index
    const bool split = p.m > 0 && eq > rem;
    int rank_in_wave[kPer];
    if (split) {
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int j = tid + kThreads * u;
        const bool tie = j < N && __float_as_uint(sc[j]) == thr;
        const unsigned long long bal = __ballot(tie);
        rank_in_wave[u] = __popcll(bal & ((1ull << lane) - 1));
        if (lane == 0) rowcnt[u * kWaves + wave] = __popcll(bal);
      }
      __syncthreads();
      if (wave == 0) {   // exclusive scan of the (row, wave) tie counts, in index order
        int v[4], t = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = rowcnt[4 * lane + q];
          t += v[q];
        }
        int ex = wave_incl_scan_i32(t, lane) - t;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          rowcnt[4 * lane + q] = ex;
          ex += v[q];
        }
      }
      __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int j = tid + kThreads * u;
      if (j < N) {
        const uint32_t x = __float_as_uint(sc[j]);
        bool in = true;
        if (p.m > 0) {
          in = x > thr;
          if (x == thr) in = !split || rowcnt[u * kWaves + wave] + rank_in_wave[u] < rem;
        }
        fl[j] = in ? 1 : 0;
      }
    }
    __syncthreads();
  }

  // 4. kept prefix per sequence, its flags, and the reduced query_start_loc
  int offset = 0;
  if (tid == 0) p.kept_qsl[0] = 0;
  for (int base = 0; base < B; base += kThreads) {
    const int b = base + tid;
    int kk = 0;
    if (b < B) {
      int d0, k;
      draft_range(p, b, base == 0 ? q0 : p.qsl[b], base == 0 ? q1 : p.qsl[b + 1], d0, k);
      bool more = true;
      for (int i = 0; i < k && more; i += 4) {
        uint8_t f[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) f[v] = fl[min(d0 + i + v, N - 1)];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          more = more && i + v < k && f[v];
          kk += more ? 1 : 0;
        }
      }
      for (int i = kk; i < k; ++i) fl[d0 + i] = 0;
      p.kept_k[b] = kk;
    }
    int total;
    const int before = block_excl_scan(b < B ? kk + 1 : 0, scan_sm, &total);
    if (b < B) p.kept_qsl[b + 1] = offset + before + kk + 1;
    offset += total;
  }
  __syncthreads();
  for (int j = tid; j < N; j += kThreads) p.keep[j] = fl[j];
}

hipError_t launch_select(const SelectParams& p, hipStream_t s) {
  hipLaunchKernelGGL(select_kernel, dim3(1), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace spexis
