// extern "C" entry points of libspexis: host-side validation of scalar arguments, workspace
// carving and kernel launches on the caller's stream.  No entry point allocates, frees or
// synchronises.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <numeric>
#include <string>

#include "kernels.h"
#include "spexis.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int ok() {
  g_last_error.clear();
  return SPEXIS_OK;
}

int hip_result(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SPEXIS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

constexpr int kMaxRows = 64;       // query rows per (sequence, KV head)
constexpr int kMaxK = spexis::kAcceptMaxK;
constexpr int kMaxVocab = 1 << 22; // keeps sum W_v < 2^63 (W_v < 2^41)

bool bad_cache_shape(int32_t bs, int32_t d) { return !((bs == 16 || bs == 32) && (d == 64 || d == 128)); }

// Shares per KV head, grid waves and the 32-key tiles of a share.  kv_chunk_tokens = 0: about
// kAttnMaxWaves waves split each head's tiles evenly (at least kAttnMinTilesPerWave each), in
// pairs of shares whose waves run on XCDs of opposite parity, the even one kAttnXcdSkew / 1024
// longer (skew); otherwise every share takes ceil(kv_chunk_tokens / 32) tiles and there are
// enough shares for the most tiles that max_seq_len allows.  (The kernel widens the shares if the
// sequences hold more.)
bool attn_waves(int32_t num_seqs, int32_t num_kv_heads, int32_t max_seq_len, int32_t req, int* tpw,
                int* nshares, int* nwaves, int* skew) {
  const int64_t max_tiles = (int64_t)num_seqs * ((max_seq_len + 31) / 32);   // per KV head
  const int64_t per = req > 0 ? ((int64_t)req + 31) / 32 : spexis::kAttnMinTilesPerWave;
  int64_t sh = std::max<int64_t>((max_tiles + per - 1) / per, 1);
  int64_t w;
  *skew = 0;
  if (req == 0) {
    sh = std::min<int64_t>(sh, std::max(1, spexis::kAttnMaxWaves / num_kv_heads));
    if (sh >= 2 && spexis::kAttnXcdSkew > 0) {
      // paired shares: an even count per head, and a grid whose waves map one to one onto
      // (share, head) (a multiple of 8 waves and of 2 hkv), kept within one wave per SIMD
      const int64_t L = std::lcm<int64_t>(8, 2 * (int64_t)num_kv_heads);
      int64_t s2 = sh & ~(int64_t)1;
      while (s2 > 2 && round_up(s2 * num_kv_heads, L) > spexis::kAttnMaxWaves) s2 -= 2;
      if (round_up(s2 * num_kv_heads, L) <= spexis::kAttnMaxWaves) {
        sh = s2;
        w = round_up(sh * num_kv_heads, L);
        *skew = spexis::kAttnXcdSkew;
      } else {
        w = round_up(sh * num_kv_heads, 4);
      }
    } else {
      w = round_up(sh * num_kv_heads, 4);
    }
  } else {
    w = round_up(sh * num_kv_heads, 4);
  }
  *tpw = req > 0 ? (int)per : 0;
  *nshares = (int)std::min<int64_t>(sh, 1 << 30);
  *nwaves = (int)std::min<int64_t>(w, 1 << 30);
  return w <= (1 << 24);
}

struct AcceptLayout {
  size_t geo, st_a, st_mode, counts, lists, lse, tin, max_part, bad_part, sum_part, srec, strec, total;
};

int64_t accept_nsub(int64_t V) { return (V + spexis::kAcceptSub - 1) / spexis::kAcceptSub; }

AcceptLayout accept_layout(int64_t B, int64_t V, int64_t max_k) {
  const int64_t ns = accept_nsub(V);
  AcceptLayout l{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t at = off;
    off += (size_t)round_up((int64_t)bytes, 256);
    return at;
  };
  l.geo = take(B * 16);
  l.st_a = take(B * 4);
  l.st_mode = take(B * 4);
  l.counts = take((spexis::kAcceptMaxRounds + 1) * 4);
  l.lists = take(spexis::kAcceptMaxRounds * B * 4 * 4);
  l.lse = take(B * (max_k + 1) * 2 * ns * 2 * 4);
  l.tin = take(B * (max_k > 0 ? max_k : 1) * 4 * 4);
  l.max_part = take(B * ns * 4);
  l.bad_part = take(B * ns * 4);
  l.sum_part = take(B * ns * 2 * 8);
  l.srec = take(B * 48);
  l.strec = take(B * 48);
  l.total = off;
  return l;
}

}  // namespace

extern "C" {

int spexis_version(void) { return SPEXIS_VERSION; }

const char* spexis_last_error(void) { return g_last_error.c_str(); }

int spexis_append_kv(void* k_cache, void* v_cache, int32_t num_blocks, int32_t num_kv_heads,
                     int32_t block_size, int32_t head_dim, int32_t num_seqs,
                     const int32_t* query_start_loc, const int32_t* seq_lens,
                     const int32_t* block_tables, int32_t max_blocks_per_seq,
                     int32_t total_tokens, int32_t max_query_len, const void* new_k,
                     const void* new_v, void* stream) {
  if (num_blocks <= 0 || num_kv_heads <= 0 || num_seqs < 0 || max_blocks_per_seq <= 0 || total_tokens < 0 ||
      max_query_len <= 0)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_append_kv: non-positive size");
  if (bad_cache_shape(block_size, head_dim))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_append_kv: block_size %d / head_dim %d not in {16,32} x {64,128}",
                block_size, head_dim);
  if (num_seqs == 0 || total_tokens == 0) return ok();
  if (!k_cache || !v_cache || !query_start_loc || !seq_lens || !block_tables || !new_k || !new_v)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_append_kv: null pointer");
  spexis::AppendParams p{k_cache, v_cache, query_start_loc, seq_lens, block_tables, new_k, new_v,
                         num_blocks, num_kv_heads, block_size, head_dim, num_seqs, max_blocks_per_seq,
                         total_tokens};
  return hip_result(spexis::launch_append(p, (hipStream_t)stream), "spexis_append_kv");
}

size_t spexis_verify_attention_workspace_size(int32_t num_seqs, int32_t num_q_heads, int32_t num_kv_heads,
                                              int32_t head_dim, int32_t max_query_len, int32_t max_seq_len,
                                              int32_t kv_chunk_tokens) {
  if (num_seqs <= 0 || num_kv_heads <= 0 || num_q_heads <= 0 || max_query_len <= 0 || max_seq_len <= 0)
    return 0;
  int tpw, nshares, nwaves, skew;
  if (!attn_waves(num_seqs, num_kv_heads, max_seq_len, kv_chunk_tokens, &tpw, &nshares, &nwaves, &skew)) return 0;
  const int rmax = (num_q_heads / num_kv_heads) * max_query_len;
  return (size_t)spexis::attn_ws_bytes(nwaves, rmax, head_dim);
}

int spexis_verify_attention(const void* k_cache, const void* v_cache, int32_t num_blocks,
                            int32_t num_kv_heads, int32_t block_size, int32_t head_dim,
                            int32_t num_seqs, const int32_t* query_start_loc,
                            const int32_t* seq_lens, const int32_t* block_tables,
                            int32_t max_blocks_per_seq, int32_t total_tokens,
                            int32_t max_query_len, int32_t max_seq_len, const void* q,
                            int32_t num_q_heads, float scale, void* out,
                            int32_t kv_chunk_tokens, void* workspace, size_t workspace_bytes,
                            void* stream) {
  if (num_blocks <= 0 || num_kv_heads <= 0 || num_q_heads <= 0 || num_seqs < 0 || max_blocks_per_seq <= 0 ||
      total_tokens < 0 || max_query_len <= 0 || max_seq_len <= 0 || kv_chunk_tokens < 0)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: non-positive size");
  if (num_q_heads % num_kv_heads != 0)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: %d query heads not a multiple of %d KV heads",
                num_q_heads, num_kv_heads);
  if (!std::isfinite(scale)) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: scale not finite");
  if (bad_cache_shape(block_size, head_dim))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_verify_attention: block_size %d / head_dim %d not in {16,32} x {64,128}",
                block_size, head_dim);
  const int group = num_q_heads / num_kv_heads;
  if ((int64_t)group * max_query_len > kMaxRows)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_verify_attention: (Hq/Hkv)*max_query_len = %d > %d",
                group * max_query_len, kMaxRows);
  if ((int64_t)max_blocks_per_seq * block_size < max_query_len)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: block tables hold fewer slots than a query");
  // every tile index of the stream fits in 32 bits
  if ((int64_t)num_seqs * (((int64_t)max_blocks_per_seq * block_size + 31) / 32) >= (1ll << 31))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_verify_attention: more than 2^31 key tiles");
  if (num_seqs == 0 || total_tokens == 0) return ok();
  if (!k_cache || !v_cache || !query_start_loc || !seq_lens || !block_tables || !q || !out)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: null pointer");
  if (q == out) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_attention: out aliases q");
  int tpw, nshares, nwaves, skew;
  if (!attn_waves(num_seqs, num_kv_heads, max_seq_len, kv_chunk_tokens, &tpw, &nshares, &nwaves, &skew))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_verify_attention: kv_chunk_tokens %d asks for too many waves",
                kv_chunk_tokens);
  const size_t need = spexis_verify_attention_workspace_size(num_seqs, num_q_heads, num_kv_heads, head_dim,
                                                             max_query_len, max_seq_len, kv_chunk_tokens);
  if (!workspace || workspace_bytes < need)
    return fail(SPEXIS_ERR_WORKSPACE_TOO_SMALL, "spexis_verify_attention: workspace %zu bytes < %zu needed",
                workspace_bytes, need);
  spexis::AttnParams p{};
  p.k_cache = k_cache;
  p.v_cache = v_cache;
  p.qsl = query_start_loc;
  p.seq_lens = seq_lens;
  p.block_tables = block_tables;
  p.q = q;
  p.out = out;
  p.ws = static_cast<float*>(workspace);
  p.num_blocks = num_blocks;
  p.hkv = num_kv_heads;
  p.block_size = block_size;
  p.head_dim = head_dim;
  p.num_seqs = num_seqs;
  p.max_blocks = max_blocks_per_seq;
  p.total_tokens = total_tokens;
  p.hq = num_q_heads;
  p.group = group;
  p.rmax = group * max_query_len;
  p.tiles_per_wave = tpw;
  p.nshares = nshares;
  p.nwaves = nwaves;
  p.skew = skew;
  p.scale_log2e = (float)((double)scale * 1.4426950408889634);
  return hip_result(spexis::launch_attention(p, (hipStream_t)stream), "spexis_verify_attention");
}

int spexis_softmax_rows(const float* logits, float* probs, int64_t rows, int32_t vocab, float temperature,
                        void* stream) {
  if (rows < 0 || vocab <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_softmax_rows: bad size");
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_softmax_rows: temperature must be finite and > 0");
  if (rows >= (1ll << 31)) return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_softmax_rows: too many rows");
  if (rows == 0) return ok();
  if (!logits || !probs) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_softmax_rows: null pointer");
  const float c = (float)(1.4426950408889634 / (double)temperature);
  return hip_result(spexis::launch_softmax(logits, probs, rows, vocab, c, (hipStream_t)stream),
                    "spexis_softmax_rows");
}

size_t spexis_accept_workspace_size(int32_t num_seqs, int32_t vocab, int32_t max_k) {
  if (num_seqs <= 0 || vocab <= 0 || max_k < 0) return 0;
  return accept_layout(num_seqs, vocab, max_k).total;
}

}  // extern "C"

namespace {

// Scratch of spexis_accept_noalloc: one copy of this array per GPU, resident until the process
// ends.  In host code its name stands for no device address; kernels get the address that
// hipGetSymbolAddress returns for the current device, looked up once per device.
static __device__ __align__(256) unsigned char scratch[SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int static_scratch_of_current_device(const char* who, void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SPEXIS_ERR_HIP, "%s: hipGetDevice: %s", who, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(SPEXIS_ERR_UNSUPPORTED, "%s: device %d >= %d", who, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SPEXIS_ERR_HIP, "%s: hipGetSymbolAddress of the scratch array: %s", who, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return SPEXIS_OK;
}

int accept_impl(const char* who, int32_t kind, int32_t num_seqs, int32_t vocab, int32_t max_k, float temperature,
                int32_t total_tokens, const int32_t* query_start_loc, const float* target, const float* draft,
                const float* target_stats, const float* draft_stats, int32_t stats_parts,
                const int32_t* draft_ids, const float* u_accept, const float* u_sample, int32_t* accepted_len,
                int32_t* out_tokens, int32_t* row_status, int32_t* seq_lens_inout, void* workspace,
                size_t workspace_bytes, void* stream, float* tok_prob = nullptr, bool static_scratch = false,
                const float* target_gathered = nullptr, const float* draft_gathered = nullptr) {
  // query_start_loc == nullptr (internal callers only): every sequence is one row, no drafts
  if (kind != SPEXIS_INPUT_PROBS && kind != SPEXIS_INPUT_LOGITS)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: kind %d is neither PROBS nor LOGITS", who, kind);
  if (num_seqs < 0 || vocab <= 0 || max_k < 0 || total_tokens < num_seqs)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: bad size", who);
  if (kind == SPEXIS_INPUT_LOGITS && (!(temperature > 0.f) || !std::isfinite(temperature)))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: temperature must be finite and > 0 for logits", who);
  if (max_k > kMaxK) return fail(SPEXIS_ERR_UNSUPPORTED, "%s: max_k %d > %d", who, max_k, kMaxK);
  if (vocab > kMaxVocab) return fail(SPEXIS_ERR_UNSUPPORTED, "%s: vocab %d > %d", who, vocab, kMaxVocab);
  if (num_seqs == 0) return ok();
  const bool has_drafts = total_tokens > num_seqs;
  if ((!query_start_loc && total_tokens != num_seqs) || !target || !u_sample || !accepted_len || !out_tokens ||
      !row_status ||
      (has_drafts && (!draft || !draft_ids || !u_accept)))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: null pointer", who);
  const AcceptLayout lay = accept_layout(num_seqs, vocab, max_k);
  if (static_scratch) {
    if (lay.total > (size_t)SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES)
      return fail(SPEXIS_ERR_UNSUPPORTED, "%s: needs %zu bytes of scratch, more than the %d of the static array", who,
                  lay.total, SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES);
    const int rc = static_scratch_of_current_device(who, &workspace);
    if (rc != SPEXIS_OK) return rc;
    workspace_bytes = SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES;
  }
  if (!workspace || workspace_bytes < lay.total)
    return fail(SPEXIS_ERR_WORKSPACE_TOO_SMALL, "%s: workspace %zu bytes < %zu needed", who, workspace_bytes,
                lay.total);
  const int64_t nsub = accept_nsub(vocab);
  if ((int64_t)num_seqs * (max_k + 1) * 2 * nsub >= (1ll << 31))
    return fail(SPEXIS_ERR_UNSUPPORTED, "%s: grid too large", who);
  char* ws = static_cast<char*>(workspace);
  spexis::AcceptParams p{};
  p.kind = kind;
  p.B = num_seqs;
  p.V = vocab;
  p.max_k = max_k;
  p.T = total_tokens;
  p.nsub = (int)nsub;
  p.c = kind == SPEXIS_INPUT_LOGITS ? (float)(1.4426950408889634 / (double)temperature) : 1.f;
  p.qsl = query_start_loc;
  p.target = target;
  p.draft = draft;
  p.ids = draft_ids;
  p.u_accept = u_accept;
  p.u_sample = u_sample;
  p.accepted_len = accepted_len;
  p.out_tokens = out_tokens;
  p.row_status = row_status;
  p.seq_lens_inout = seq_lens_inout;
  p.tok_prob = tok_prob;
  p.geo = reinterpret_cast<int32_t*>(ws + lay.geo);
  p.st_a = reinterpret_cast<int32_t*>(ws + lay.st_a);
  p.st_mode = reinterpret_cast<int32_t*>(ws + lay.st_mode);
  p.counts = reinterpret_cast<int32_t*>(ws + lay.counts);
  p.lists = reinterpret_cast<int32_t*>(ws + lay.lists);
  p.lse_part = reinterpret_cast<float*>(ws + lay.lse);
  p.tin = reinterpret_cast<float*>(ws + lay.tin);
  p.max_part = reinterpret_cast<float*>(ws + lay.max_part);
  p.bad_part = reinterpret_cast<int32_t*>(ws + lay.bad_part);
  p.sum_part = reinterpret_cast<uint64_t*>(ws + lay.sum_part);
  p.srec = reinterpret_cast<int32_t*>(ws + lay.srec);
  p.strec = reinterpret_cast<int32_t*>(ws + lay.strec);
  p.ext_tstats = target_stats;
  p.ext_dstats = draft_stats;
  p.ext_parts = stats_parts;
  p.tg_given = target_gathered;
  p.dg_given = draft_gathered;
  return hip_result(spexis::launch_accept(p, (hipStream_t)stream), who);
}

}  // namespace

extern "C" {

int spexis_accept(int32_t kind, int32_t num_seqs, int32_t vocab, int32_t max_k, float temperature,
                  int32_t total_tokens, const int32_t* query_start_loc, const float* target, const float* draft,
                  const int32_t* draft_ids, const float* u_accept, const float* u_sample, int32_t* accepted_len,
                  int32_t* out_tokens, int32_t* row_status, int32_t* seq_lens_inout, void* workspace,
                  size_t workspace_bytes, void* stream) {
  return accept_impl("spexis_accept", kind, num_seqs, vocab, max_k, temperature, total_tokens, query_start_loc,
                     target, draft, nullptr, nullptr, 0, draft_ids, u_accept, u_sample, accepted_len, out_tokens,
                     row_status, seq_lens_inout, workspace, workspace_bytes, stream);
}

int spexis_accept_noalloc(int32_t kind, int32_t num_seqs, int32_t vocab, int32_t max_k, float temperature,
                          int32_t total_tokens, const int32_t* query_start_loc, const float* target,
                          const float* draft, const int32_t* draft_ids, const float* u_accept, const float* u_sample,
                          int32_t* accepted_len, int32_t* out_tokens, int32_t* row_status, int32_t* seq_lens_inout,
                          void* stream) {
  return accept_impl("spexis_accept_noalloc", kind, num_seqs, vocab, max_k, temperature, total_tokens,
                     query_start_loc, target, draft, nullptr, nullptr, 0, draft_ids, u_accept, u_sample, accepted_len,
                     out_tokens, row_status, seq_lens_inout, nullptr, 0, stream, nullptr, true);
}

int32_t spexis_lm_head_tiles(int32_t vocab) { return vocab > 0 ? (vocab + spexis::kLmCols - 1) / spexis::kLmCols : 0; }

int spexis_accept_with_stats(int32_t num_seqs, int32_t vocab, int32_t max_k, float temperature,
                             int32_t total_tokens, const int32_t* query_start_loc, const float* target_logits,
                             const float* draft_logits, const float* target_stats, const float* draft_stats,
                             int32_t stats_tiles, const int32_t* draft_ids, const float* u_accept,
                             const float* u_sample, const float* target_gathered, const float* draft_gathered,
                             int32_t* accepted_len, int32_t* out_tokens, int32_t* row_status,
                             int32_t* seq_lens_inout, void* workspace, size_t workspace_bytes, void* stream) {
  const bool has_drafts = total_tokens > num_seqs;
  if (num_seqs > 0 && (!target_stats || (has_drafts && !draft_stats)))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_accept_with_stats: null statistics");
  if ((target_gathered == nullptr) != (draft_gathered == nullptr))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_accept_with_stats: give both gathered arrays or neither");
  if (stats_tiles <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_accept_with_stats: stats_tiles <= 0");
  // the per-row reductions of the statistics live in the workspace's statistics area
  if (num_seqs > 0 && max_k >= 0 && total_tokens > (int64_t)num_seqs * (max_k + 1))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT,
                "spexis_accept_with_stats: total_tokens %d > num_seqs * (max_k + 1)", total_tokens);
  return accept_impl("spexis_accept_with_stats", SPEXIS_INPUT_LOGITS, num_seqs, vocab, max_k, temperature,
                     total_tokens, query_start_loc, target_logits, draft_logits, target_stats,
                     has_drafts ? draft_stats : target_stats, stats_tiles, draft_ids, u_accept, u_sample,
                     accepted_len, out_tokens, row_status, seq_lens_inout, workspace, workspace_bytes, stream,
                     nullptr, false, has_drafts ? target_gathered : nullptr, has_drafts ? draft_gathered : nullptr);
}

size_t spexis_sample_workspace_size(int32_t rows, int32_t vocab) {
  if (rows <= 0 || vocab <= 0) return 0;
  return accept_layout(rows, vocab, 0).total + (size_t)round_up((int64_t)rows * 4, 256);
}

int spexis_sample_tokens(int32_t kind, int32_t rows, int32_t vocab, float temperature, const float* input,
                         const float* stats, int32_t stats_tiles, const float* u, int32_t* tokens, float* token_prob,
                         int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream) {
  if (rows < 0 || vocab <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_sample_tokens: bad size");
  if (stats && kind != SPEXIS_INPUT_LOGITS)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_sample_tokens: statistics need logits");
  if (stats && stats_tiles <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_sample_tokens: stats_tiles <= 0");
  if (rows == 0) return ok();
  if (!input || !u || !tokens || !row_status)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_sample_tokens: null pointer");
  const size_t need = spexis_sample_workspace_size(rows, vocab);
  if (!workspace || workspace_bytes < need)
    return fail(SPEXIS_ERR_WORKSPACE_TOO_SMALL, "spexis_sample_tokens: workspace %zu bytes < %zu needed",
                workspace_bytes, need);
  const size_t acc_bytes = accept_layout(rows, vocab, 0).total;
  int32_t* accepted = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + acc_bytes);
  return accept_impl("spexis_sample_tokens", kind, rows, vocab, 0, temperature, rows, nullptr, input, nullptr,
                     stats, stats, stats ? stats_tiles : 0, nullptr, nullptr, u, accepted, tokens, row_status,
                     nullptr, workspace, acc_bytes, stream, token_prob);
}

int spexis_select_drafts(int32_t num_seqs, int32_t total_tokens, const int32_t* query_start_loc,
                         const float* draft_conf, float alpha, int32_t* kept_k, int32_t* kept_query_start_loc,
                         int32_t* keep, void* stream) {
  if (num_seqs < 0 || total_tokens < num_seqs)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_select_drafts: bad size");
  if (!(alpha >= 0.f) || !(alpha < 1.f))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_select_drafts: alpha must be in [0, 1)");
  const int32_t N = total_tokens - num_seqs;
  if (N > spexis::kSelectMaxDrafts)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_select_drafts: %d drafts > %d", N, spexis::kSelectMaxDrafts);
  if (num_seqs == 0) return ok();
  if (!query_start_loc || !kept_k || !kept_query_start_loc || (N > 0 && (!draft_conf || !keep)))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_select_drafts: null pointer");
  spexis::SelectParams p{};
  p.qsl = query_start_loc;
  p.conf = draft_conf;
  p.B = num_seqs;
  p.T = total_tokens;
  p.N = N;
  p.m = (int)std::floor((double)alpha * (double)N);
  p.kept_k = kept_k;
  p.kept_qsl = kept_query_start_loc;
  p.keep = keep;
  return hip_result(spexis::launch_select(p, (hipStream_t)stream), "spexis_select_drafts");
}

size_t spexis_packed_weight_size(int32_t rows, int32_t cols) {
  if (rows <= 0 || cols <= 0 || cols % 64 != 0) return 0;
  return (size_t)((rows + 31) / 32) * 32 * (size_t)cols * 2;
}

int spexis_pack_weight(const void* weight, int32_t rows, int32_t cols, void* packed, void* stream) {
  if (!weight || !packed) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_pack_weight: null pointer");
  if (rows <= 0 || cols <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_pack_weight: bad size");
  if (cols % 64 != 0)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_pack_weight: cols %d is not a multiple of 64", cols);
  if ((int64_t)((rows + 31) / 32) * (cols / 64) * 256 >= (1ll << 40))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_pack_weight: too large");
  return hip_result(spexis::launch_pack_weight(weight, rows, cols, packed, (hipStream_t)stream), "spexis_pack_weight");
}

size_t spexis_linear_workspace_size(int32_t rows, int32_t out_features, int32_t in_features) {
  if (rows <= 0 || out_features <= 0 || in_features <= 0 || in_features % 256 != 0) return 0;
  const int S = spexis::linear_split(rows, out_features, in_features);
  return S > 1 ? (size_t)S * rows * out_features * sizeof(float) : 0;
}

int spexis_linear(const void* x, const void* weight, const void* residual, int32_t rows, int32_t out_features,
                  int32_t in_features, void* y, void* workspace, size_t workspace_bytes, void* stream) {
  if (rows < 0 || out_features <= 0 || in_features <= 0)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear: bad size");
  if (in_features % 256 != 0)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear: in_features %d is not a multiple of 256", in_features);
  if (rows == 0) return ok();
  if (!x || !weight || !y) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear: null pointer");
  const int64_t tiles = (out_features + spexis::kLmCols - 1) / spexis::kLmCols;
  if (spexis::projection_workgroups(rows, out_features) + 8 * rows >= (1ll << 31) ||
      (int64_t)rows * out_features >= (1ll << 36) ||
      (int64_t)rows * in_features >= (1ll << 40))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear: problem too large");
  const int S = spexis::linear_split(rows, out_features, in_features);
  const size_t need = spexis_linear_workspace_size(rows, out_features, in_features);
  if (need > 0 && (!workspace || workspace_bytes < need))
    return fail(SPEXIS_ERR_WORKSPACE_TOO_SMALL, "spexis_linear: workspace %zu bytes < %zu needed", workspace_bytes,
                need);
  spexis::LinearParams p{};
  p.proj.h = x;
  p.proj.w = weight;
  p.proj.M = rows;
  p.proj.V = out_features;
  p.proj.d = in_features;
  p.proj.ntiles = (int)tiles;
  p.proj.ksplit = S;
  if (S > 1) {
    p.proj.logits = static_cast<float*>(workspace);   // [S][rows][out] partials
  } else {
    p.proj.y = y;
    p.proj.res = residual;
  }
  p.part = static_cast<float*>(workspace);
  p.res = residual;
  p.y = y;
  p.M = rows;
  p.N = out_features;
  p.S = S;
  return hip_result(spexis::launch_linear(p, (hipStream_t)stream), "spexis_linear");
}

size_t spexis_linear_split_workspace_size(int32_t rows, int32_t total_out_features, int32_t in_features) {
  if (rows <= 0 || total_out_features <= 0 || in_features <= 0 || in_features % 256 != 0) return 0;
  const int S = spexis::linear_split(rows, total_out_features, in_features);
  return (size_t)S * rows * total_out_features * sizeof(float);
}

int spexis_linear_split(const void* x, const void* weight, int32_t rows, int32_t in_features, int32_t num_outputs,
                        const int32_t* out_features, void* const* outputs, void* workspace, size_t workspace_bytes,
                        void* stream) {
  if (rows < 0 || in_features <= 0 || num_outputs < 1 || num_outputs > spexis::kLinearMaxOutputs || !out_features)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear_split: bad size or output count");
  int64_t N = 0;
  for (int i = 0; i < num_outputs; ++i) {
    if (out_features[i] <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear_split: bad output width");
    if (out_features[i] % 4 != 0)
      return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear_split: output width %d is not a multiple of 4",
                  out_features[i]);
    N += out_features[i];
  }
  if (in_features % 256 != 0)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear_split: in_features %d is not a multiple of 256",
                in_features);
  if (N >= (1ll << 30)) return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear_split: problem too large");
  if (rows == 0) return ok();
  if (!x || !weight || !outputs) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear_split: null pointer");
  for (int i = 0; i < num_outputs; ++i)
    if (!outputs[i]) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_linear_split: null output %d", i);
  if (spexis::projection_workgroups(rows, N) + 8 * rows >= (1ll << 31) || (int64_t)rows * N >= (1ll << 36) ||
      (int64_t)rows * in_features >= (1ll << 40))
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_linear_split: problem too large");
  const int S = spexis::linear_split(rows, (int)N, in_features);
  const size_t need = spexis_linear_split_workspace_size(rows, (int)N, in_features);
  if (!workspace || workspace_bytes < need)
    return fail(SPEXIS_ERR_WORKSPACE_TOO_SMALL, "spexis_linear_split: workspace %zu bytes < %zu needed",
                workspace_bytes, need);
  spexis::LinearParams p{};
  p.proj.h = x;
  p.proj.w = weight;
  p.proj.M = rows;
  p.proj.V = (int)N;
  p.proj.d = in_features;
  p.proj.ntiles = (int)((N + spexis::kLmCols - 1) / spexis::kLmCols);
  p.proj.ksplit = S;
  p.proj.logits = static_cast<float*>(workspace);   // [S][rows][N] fp32 products, S >= 1
  p.part = static_cast<float*>(workspace);
  p.M = rows;
  p.N = (int)N;
  p.S = S;
  p.nout = num_outputs;
  p.off[0] = 0;
  for (int i = 0; i < num_outputs; ++i) {
    p.off[i + 1] = p.off[i] + out_features[i];
    p.ys[i] = outputs[i];
  }
  for (int i = num_outputs + 1; i <= spexis::kLinearMaxOutputs; ++i) p.off[i] = (int)N;
  return hip_result(spexis::launch_linear(p, (hipStream_t)stream), "spexis_linear_split");
}

int spexis_lookahead_memory(int32_t num_requests, const int64_t* cur_len, const int32_t* remaining,
                            const double* precision, int32_t pp, double theta, int32_t iters, double* mem,
                            double* e_gen, double* e_nfin, double* e_lfin, void* stream) {
  if (!mem) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_lookahead_memory: null pointer");
  if (num_requests < 0 || pp < 1 || iters < 1)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_lookahead_memory: bad size");
  if (!(theta >= 0.0 && theta <= 1.0))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_lookahead_memory: theta must be in [0, 1]");
  if (iters > spexis::kLookaheadMaxIters)
    return fail(SPEXIS_ERR_UNSUPPORTED, "spexis_lookahead_memory: %d iterations > %d", iters,
                spexis::kLookaheadMaxIters);
  if (num_requests > 0 && (!cur_len || !remaining || !precision))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_lookahead_memory: null pointer");
  spexis::LookaheadParams p{};
  p.cur_len = cur_len;
  p.remaining = remaining;
  p.prec = precision;
  p.n = num_requests;
  p.pp = pp;
  p.iters = iters;
  p.theta = theta;
  p.mem = mem;
  p.e_gen = e_gen;
  p.e_nfin = e_nfin;
  p.e_lfin = e_lfin;
  return hip_result(spexis::launch_lookahead(p, (hipStream_t)stream), "spexis_lookahead_memory");
}

size_t spexis_lm_head_stats_size(int32_t rows, int32_t vocab) {
  if (rows <= 0 || vocab <= 0) return 0;
  return (size_t)rows * spexis_lm_head_tiles(vocab) * 2 * sizeof(float);
}

}  // extern "C"

namespace {

int lm_head_impl(const char* who, const void* hidden, const void* weight, int32_t rows, int32_t vocab,
                 int32_t hidden_dim, float temperature, float* logits, float* stats, const int32_t* gather_cols,
                 float* gathered, void* stream) {
  if (rows < 0 || vocab <= 0 || hidden_dim <= 0) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: bad size", who);
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: temperature must be finite and > 0", who);
  if (hidden_dim % 256 != 0)
    return fail(SPEXIS_ERR_UNSUPPORTED, "%s: hidden_dim %d is not a multiple of 256", who, hidden_dim);
  if (rows == 0) return ok();
  if (!hidden || !weight || !stats) return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: null pointer", who);
  if ((gather_cols == nullptr) != (gathered == nullptr))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "%s: give gather_cols and gathered together", who);
  const int64_t tiles = spexis_lm_head_tiles(vocab);
  if (spexis::projection_workgroups(rows, vocab) + 8 * rows >= (1ll << 31) || (int64_t)rows * vocab >= (1ll << 40))
    return fail(SPEXIS_ERR_UNSUPPORTED, "%s: problem too large", who);
  spexis::LmParams p{};
  p.h = hidden;
  p.w = weight;
  p.logits = logits;
  p.stats = stats;
  p.M = rows;
  p.V = vocab;
  p.d = hidden_dim;
  p.ntiles = (int)tiles;
  p.ksplit = 1;
  p.c = (float)(1.4426950408889634 / (double)temperature);
  p.gcols = gather_cols;
  p.gout = gathered;
  return hip_result(spexis::launch_projection(p, (hipStream_t)stream), who);
}

}  // namespace

extern "C" {

int spexis_lm_head(const void* hidden, const void* weight, int32_t rows, int32_t vocab, int32_t hidden_dim,
                   float temperature, float* logits, float* stats, void* stream) {
  return lm_head_impl("spexis_lm_head", hidden, weight, rows, vocab, hidden_dim, temperature, logits, stats,
                      nullptr, nullptr, stream);
}

int spexis_lm_head_gather(const void* hidden, const void* weight, int32_t rows, int32_t vocab, int32_t hidden_dim,
                          float temperature, float* logits, float* stats, const int32_t* gather_cols,
                          float* gathered, void* stream) {
  if (rows > 0 && (!gather_cols || !gathered))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_lm_head_gather: null gather_cols or gathered");
  return lm_head_impl("spexis_lm_head_gather", hidden, weight, rows, vocab, hidden_dim, temperature, logits, stats,
                      gather_cols, gathered, stream);
}

int spexis_verify_gather_columns(int32_t num_seqs, int32_t total_tokens, const int32_t* query_start_loc,
                                 const int32_t* draft_ids, int32_t* cols, void* stream) {
  if (num_seqs < 0 || total_tokens < num_seqs)
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_gather_columns: bad size");
  if (num_seqs == 0) return ok();
  if (!query_start_loc || !cols || (total_tokens > num_seqs && !draft_ids))
    return fail(SPEXIS_ERR_INVALID_ARGUMENT, "spexis_verify_gather_columns: null pointer");
  return hip_result(spexis::launch_gather_columns(query_start_loc, draft_ids, num_seqs, total_tokens, cols,
                                                  (hipStream_t)stream),
                    "spexis_verify_gather_columns");
}

}  // extern "C"
