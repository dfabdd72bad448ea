// Launch parameters and host-side launchers of the libspexis kernels (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spexis {

struct AppendParams {
  void* k_cache;
  void* v_cache;
  const int32_t* qsl;
  const int32_t* seq_lens;
  const int32_t* block_tables;
  const void* new_k;
  const void* new_v;
  int num_blocks, hkv, block_size, head_dim, num_seqs, max_blocks, total_tokens;
};

struct AttnParams {
  const void* k_cache;
  const void* v_cache;
  const int32_t* qsl;
  const int32_t* seq_lens;
  const int32_t* block_tables;
  const void* q;
  void* out;
  float* ws;             // per-wave partial slots [nwaves][2][slot], then headers [nwaves][kAttnHdrInts]
  int num_blocks, hkv, block_size, head_dim, num_seqs, max_blocks, total_tokens;
  int hq, group;         // Hq, G = Hq / Hkv
  int rmax;              // G * max_query_len (rows per (sequence, KV head)), <= 64
  int tiles_per_wave;    // 32-key tiles per share; 0: the even split of each head's tiles
  int nshares;           // shares per KV head; wave s*hkv + h takes share s of head h
  int nwaves;            // waves of the attention grid (4 per workgroup, >= nshares * hkv)
  int skew;              // 0: equal shares; else paired shares, the even-XCD one skew/1024 longer
  float scale_log2e;     // scale * log2(e): scores live in the base-2 domain
};

constexpr int kAttnHdrInts = 8;           // per-wave header of the partial an item's first wave leaves
constexpr int kAttnMinTilesPerWave = 2;   // floor of the even split (short batches)
constexpr int kAttnMaxWaves = 1024;       // waves of the even split: one per SIMD of 256 CUs
// Tiles moved, per 1024, from the share of each pair on an odd XCD to the one on an even XCD:
// waves on odd XCDs stream the cache a few per cent slower.
constexpr int kAttnXcdSkew = 28;

// One partial slot: [rmax][D] unnormalised output, then rmax reference maxima and rmax sums.
// Rounded up to 16 floats so that every slot starts 64-byte aligned.
__host__ __device__ inline int64_t attn_slot_floats(int rmax, int D) { return ((int64_t)rmax * (D + 2) + 15) / 16 * 16; }
__host__ __device__ inline int64_t attn_ws_bytes(int nwaves, int rmax, int D) {
  return (int64_t)nwaves * (2 * attn_slot_floats(rmax, D) * 4 + kAttnHdrInts * 4);
}

// LM-head projection logits = h W^T with the row statistics of its 128-column tiles.
// The projection out = h W^T shared by the LM head and the adapter's linear layers.
struct LmParams {
  const void* h;         // [M][d] bf16
  const void* w;         // [V][d] bf16, packed (launch_pack_weight)
  float* logits;         // [M][V] fp32 (null: not written); with ksplit > 1, [ksplit][M][V] partials
  float* stats;          // [M][ntiles][2]: max of x*c and sum of 2^(x*c - max) over each tile (or null)
  void* y;               // [M][V] bf16 output, bf16(acc + res), instead of logits (ksplit == 1)
  const void* res;       // [M][V] bf16 residual for y, or null
  int M, V, d, ntiles, mgroups;   // ntiles: 128-column statistics tiles; mgroups: set by the launcher
  int ksplit;            // K split over workgroups (grid y); each takes d / ksplit
  float c;               // log2(e) / temperature
  // Fused gathers (gout null: none; needs stats): gout[m] = logits[m][gcols[m]] for every row
  // whose gcols[m] lies in [0, V).
  const int32_t* gcols;
  float* gout;
};

constexpr int kLmCols = 128;   // columns of a statistics tile, and of a narrow projection's workgroup
constexpr int kLmK = 64;       // K per pipeline step (four MFMA k-steps)

// Selective speculation over a batch of B sequences, T query tokens, N = T - B drafts.
struct SelectParams {
  const int32_t* qsl;
  const float* conf;     // [N] draft confidences
  int B, T, N, m;        // m = floor(alpha * N) drafts dropped
  int32_t* kept_k;       // [B]
  int32_t* kept_qsl;     // [B+1]
  int32_t* keep;         // [N]
};

constexpr int kSelectMaxDrafts = 16384;

// spexis_linear: the projection kernel, then (K split) the reduce of its partials.
constexpr int kLinearMaxOutputs = 4;   // outputs of one split linear call

struct LinearParams {
  LmParams proj;
  float* part;       // fp32 [S][M][N] when S > 1 or nout > 0
  const void* res;   // bf16 [M][N] or null
  void* y;           // bf16 [M][N] (nout == 0)
  int M, N, S;
  int nout;                          // 0: y alone; else outputs 0 .. nout-1 take columns
  int off[kLinearMaxOutputs + 1];    // off[i] .. off[i+1]-1 (multiples of 4, off[nout] = N)
  void* ys[kLinearMaxOutputs];       // bf16 [M][off[i+1] - off[i]]
};

struct LookaheadParams {
  const int64_t* cur_len;    // [n] current length of each running request
  const int32_t* remaining;  // [n] predicted remaining length
  const double* prec;        // [n] precision of that prediction
  int n, pp, iters;
  double theta;
  double* mem;               // [iters]
  double* e_gen;             // [iters] or null
  double* e_nfin;            // [iters] or null
  double* e_lfin;            // [iters] or null
};

constexpr int kLookaheadMaxIters = 1024;

struct AcceptParams {
  int kind;              // 0 probs, 1 logits
  int B, V, max_k, T;
  int nsub;              // ceil(V / kAcceptSub): partial results are kept per sub-chunk
  float c;               // log2(e) / temperature (logits mode)
  const int32_t* qsl;    // null: sequence b is row b alone (no drafts; plain sampling)
  const float* target;
  const float* draft;
  const int32_t* ids;
  const float* u_accept;
  const float* u_sample;
  int32_t* accepted_len;
  int32_t* out_tokens;
  int32_t* row_status;
  int32_t* seq_lens_inout;
  float* tok_prob;       // [B] or null: probability of the emitted token under p at its position
  // workspace views
  int32_t* geo;          // [B][4] first target row, first draft row, k, state (1 valid; logits
                         // mode: 0 no query token, -1 a draft id out of range; probabilities: 0 invalid)
  int32_t* st_a;         // [B] final a_b
  int32_t* st_mode;      // [B] 1 residual, 2 bonus, 3 done (outputs written)
  float* lse_part;       // [B][max_k+1][2 target/draft][nsub][2] (max, sum of 2^(y-max)) (logits mode)
  int32_t* counts;       // [kAcceptMaxRounds+1] sequences entering round r (r >= 1; logits mode)
  int32_t* lists;        // [kAcceptMaxRounds][B][4] those sequences: b, first target row, first draft row, k
  const float* ext_tstats;   // logits mode with given statistics: [T][ext_parts][2] for the target
  const float* ext_dstats;   // rows, [T-B][ext_parts][2] for the draft rows (max of y*c, sum of
  int ext_parts;             // 2^(y*c - max) per column tile); null / 0: computed here
  float* tin;            // [B][max_k][4] test inputs of position i: target and draft logit of x_i,
                         // u_i, and 1 if x_i is a valid id (logits mode; gathered by the stats pass)
  float* max_part;       // [B][nsub] max of the sampled target row (probability inputs)
  int32_t* bad_part;     // [B][nsub] the sampled row(s) hold a bad value (probability inputs)
  uint64_t* sum_part;    // [B][nsub][2] fixed-point sums of the residual and of p
  int32_t* srec;         // [B][12] the search's record of b: t0, d0, k, a | mode, bad, scale, 0 |
                         // Mp, Rp, Mq, Rq (written by the tests launch that ends its testing, or
                         // by write_invalid)
  int32_t* strec;        // [B][12] a round's job per list entry (logits mode): b, t0, d0, k | job,
                         // position or next round's lo, next round's hi, shift | Mp, Rp, Mq, Rq
  const float* tg_given; // with given statistics, optionally the logits at the drafts: target row
  const float* dg_given; // t0+i at x_i ([T]) and draft row d0+i at x_i ([T-B]); null: read them
};

constexpr int kAcceptMaxK = 32;      // drafts per sequence the boundary takes (below one wave's lanes)
constexpr int kAcceptMaxRounds = 8;  // test rounds: widths 2, 4, 8, ... cover max_k <= 509
constexpr int kAcceptSub = 4096;     // vocab entries per partial result (one workgroup's share)

hipError_t launch_append(const AppendParams& p, hipStream_t s);
hipError_t launch_attention(const AttnParams& p, hipStream_t s);

hipError_t launch_select(const SelectParams& p, hipStream_t s);
hipError_t launch_lookahead(const LookaheadParams& p, hipStream_t s);
int linear_split(int M, int N, int K);
hipError_t launch_pack_weight(const void* w, int N, int K, void* out, hipStream_t s);
// packed weight tile (32 rows x 64 K values, 2048 elements) holding rows 32n.., K values 64c..
constexpr int kPackTile = 2048;
hipError_t launch_linear(const LinearParams& p, hipStream_t s);
hipError_t launch_projection(const LmParams& p, hipStream_t s);
// Workgroups launch_projection runs for M rows and N columns (without a K split; at most 8 more
// are launched to round the column workgroups up to a multiple of 8 per row group).
int64_t projection_workgroups(int64_t M, int64_t N);
hipError_t launch_softmax(const float* logits, float* probs, int64_t rows, int V, float c, hipStream_t s);
hipError_t launch_accept(const AcceptParams& p, hipStream_t s);
hipError_t launch_gather_columns(const int32_t* qsl, const int32_t* ids, int B, int T, int32_t* cols, hipStream_t s);

}  // namespace spexis
