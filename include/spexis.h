/*
 * spexis.h -- C ABI of the speculative-verification hot path on one MI355X (gfx950).
 *
 * Spexis (speculative-parallel execution, Sec. 4) verifies the k tokens a self-speculative
 * draft proposes with one pass of the full model: the k+1 query tokens of a sequence (its
 * last accepted token and the k drafts) are appended to the paged KV cache that speculative
 * and normal execution share, attend causally over that cache, and the speculative-sampling
 * rule the paper adopts from [sd] (Related Work) decides how many drafts survive.  This
 * library computes exactly that step:
 *
 *   spexis_append_kv         write the k+1 new K/V rows of every sequence into the cache
 *   spexis_verify_attention  causal grouped-query attention of those rows over the cache
 *   spexis_accept            ratio tests, residual / bonus sampling, outputs
 *   spexis_lm_head           logits = h W^T with fused softmax statistics (next to accept)
 *   spexis_lm_head_gather    the same, also gathering each row's logit at a given column
 *   spexis_verify_gather_columns  those columns for the target rows: the drafts they verify
 *   spexis_accept_with_stats acceptance from logits whose statistics are known
 *   spexis_accept_noalloc    spexis_accept in a static scratch array (callers that cannot allocate)
 *   spexis_select_drafts     selective speculation: drop the least confident drafts first
 *   spexis_lookahead_memory  look-ahead KV-memory estimate of the running requests (Algorithm 1)
 *   spexis_linear            a linear layer of the drafting adapter (bf16, fp32 accumulation)
 *   spexis_linear_split      several linear layers of one input (q, k, v) in one projection
 *   spexis_pack_weight       weight layout of the projections above (done once per weight)
 *   spexis_sample_tokens     one token per row of logits or probabilities, with its probability
 *   spexis_softmax_rows      temperature softmax of logit rows (probability inputs)
 *
 * Conventions shared by every entry point
 *   - Pointers are DEVICE pointers unless a parameter says "host".  Every call is
 *     asynchronous on `stream` (a hipStream_t passed as void*; NULL = the null stream);
 *     the library never synchronises and never reads device data on the host.
 *   - The caller owns all memory: cache pools, block tables, outputs and workspaces.  The
 *     library allocates nothing and holds no device state between calls, apart from the
 *     static scratch array of spexis_accept_noalloc (whose contents no call depends on).
 *   - Scalars are validated on the host before any launch.  Device data (block ids, lengths,
 *     token ids) is trusted for correctness but clamped for memory safety: an inconsistent
 *     value gives an unspecified result, never an access outside the buffers described here.
 *   - Return codes: SPEXIS_OK, or a negative code with a message in spexis_last_error().
 *   - A call with no work (no sequences, no query tokens, or no rows) validates its scalar
 *     arguments and returns SPEXIS_OK without reading or writing any buffer; its buffer
 *     pointers may then be NULL (as a zero-element tensor's are).
 *   - Calls on one stream run in order; calls that share a workspace or an output and run
 *     concurrently on different streams race.
 *
 * Batch description (append, attention)
 *   num_seqs        B, sequences in the step
 *   query_start_loc [B+1] int32: sequence b owns query rows qsl[b] .. qsl[b+1]-1;
 *                   n_b = qsl[b+1]-qsl[b] = k_b + 1 >= 1, qsl[0] = 0, qsl[B] = total_tokens
 *   seq_lens        [B] int32: S_b, tokens of sequence b in the cache AFTER the append;
 *                   L_b = S_b - n_b are the tokens cached before this step
 *   block_tables    [B][max_blocks_per_seq] int32 physical block ids; token t of sequence b
 *                   lives in block block_tables[b][t / block_size], slot t % block_size
 *   total_tokens    host: T = qsl[B], rows of q / out / new_k / new_v
 *   max_query_len   host: >= max_b n_b
 *
 * Paged cache layout (bf16, one pool for K and one for V, num_blocks blocks each)
 *   K pool  [num_blocks][Hkv][D/8][block_size][8]
 *           element (blk, h, slot, d) at ((((blk*Hkv + h)*(D/8) + d/8)*bs + slot)*8 + d%8)
 *   V pool  [num_blocks][Hkv][D][block_size], slot index stored with bits 2 and 3 swapped
 *           element (blk, h, slot, d) at (((blk*Hkv + h)*D + d)*bs + swap23(slot)),
 *           swap23(s) = (s & ~12) | ((s >> 2 & 1) << 3) | ((s >> 3 & 1) << 2)
 *   Each (block, head) is one contiguous 4 KB (bs 16) or 8 KB (bs 32) chunk of each pool.
 *   The layout lets the attention kernel load both matrix-core operands straight from HBM
 *   with fully coalesced 16-byte loads (K: eight head-dim values of one slot; V: eight
 *   slots of one head-dim index, in the order the score tile produces them).
 */
#ifndef SPEXIS_H
#define SPEXIS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEXIS_VERSION 100

#define SPEXIS_OK 0
#define SPEXIS_ERR_INVALID_ARGUMENT (-1)  /* null pointer, non-positive size, Hq % Hkv != 0 ... */
#define SPEXIS_ERR_UNSUPPORTED (-2)       /* a shape outside the supported set (see each call) */
#define SPEXIS_ERR_WORKSPACE_TOO_SMALL (-3)
#define SPEXIS_ERR_HIP (-4)               /* a HIP launch failed; message has hipGetErrorString */

/* row_status codes written by spexis_accept */
#define SPEXIS_ROW_OK 0
#define SPEXIS_ROW_EMPTY 1      /* the sampled target row had no positive entry */
#define SPEXIS_ROW_BAD_VALUE 2  /* the sampled row held a NaN, an infinity or a negative value */
#define SPEXIS_ROW_BAD_TOKEN 3  /* a draft token id outside [0, vocab) */
#define SPEXIS_ROW_INTERNAL 4   /* the sampling search found no token (a library fault, never
                                   expected): token -1, seq_lens_inout unchanged */

/* input kinds of spexis_accept */
#define SPEXIS_INPUT_PROBS 0
#define SPEXIS_INPUT_LOGITS 1

/* Library version (SPEXIS_VERSION). */
int spexis_version(void);

/* Message of the last failed call on this host thread ("" if none).  Host memory owned by
 * the library, valid until the next call on the same thread. */
const char* spexis_last_error(void);

/*
 * spexis_append_kv -- write the n_b = k_b + 1 new K/V rows of every sequence into the cache.
 *
 * Defined by the shared-cache design of speculative-parallel execution (Sec. 4): verified
 * and speculative tokens live in one paged cache, so a step's rows go to positions
 * L_b .. S_b-1 of their sequence, overwriting whatever a rejected speculation left there.
 * For every b, j < n_b and KV head h: token position L_b + j receives
 * new_k[qsl[b]+j][h][:] and new_v[qsl[b]+j][h][:].  Nothing else in the pools changes.
 *
 *   k_cache, v_cache   bf16 pools in the layout above (written)
 *   num_blocks         blocks per pool; num_kv_heads Hkv >= 1; block_size in {16, 32};
 *                      head_dim in {64, 128}
 *   new_k, new_v       [total_tokens][Hkv][head_dim] bf16, row-major (read)
 * Errors: INVALID_ARGUMENT for null pointers or non-positive sizes; UNSUPPORTED for other
 * block sizes or head dims.
 */
int spexis_append_kv(void* k_cache, void* v_cache, int32_t num_blocks, int32_t num_kv_heads,
                     int32_t block_size, int32_t head_dim, int32_t num_seqs,
                     const int32_t* query_start_loc, const int32_t* seq_lens,
                     const int32_t* block_tables, int32_t max_blocks_per_seq,
                     int32_t total_tokens, int32_t max_query_len, const void* new_k,
                     const void* new_v, void* stream);

/*
 * Bytes of workspace spexis_verify_attention needs for these host-side bounds (> 0 whenever
 * the sizes are valid; 0 for invalid sizes).  kv_chunk_tokens as in spexis_verify_attention.
 * With kv_chunk_tokens = 0 it is at most 1024 * (2 * (Hq/Hkv) * max_query_len * (head_dim + 2)
 * + 40) * 4 bytes (about 68 MB at 64 rows, head_dim 128), whatever the sequence lengths.
 */
size_t spexis_verify_attention_workspace_size(int32_t num_seqs, int32_t num_q_heads,
                                              int32_t num_kv_heads, int32_t head_dim,
                                              int32_t max_query_len, int32_t max_seq_len,
                                              int32_t kv_chunk_tokens);

/*
 * spexis_verify_attention -- the target model's joint verification pass over the drafts
 * (Sec. 4: drafts are verified together by the full model; Related Work: the base model
 * verifies the draft model's tokens in parallel).
 *
 * For every b, query token j < n_b and query head h, with G = Hq/Hkv and g = h / G:
 *   out[qsl[b]+j][h][:] = sum_{t <= L_b + j} softmax_t(scale * <q[qsl[b]+j][h], k[b,t,g]>)
 *                         * v[b,t,g][:]
 * i.e. a query token sees the cached prefix and itself but not later drafts.  bf16 inputs,
 * fp32 accumulation, bf16 output.
 *
 *   q       [total_tokens][Hq][head_dim] bf16 (read);  out: same shape, bf16 (written;
 *           must not alias q)
 *   scale   softmax scale, usually 1/sqrt(head_dim)
 *   max_seq_len      host: >= max_b S_b, and S_b <= max_blocks_per_seq * block_size
 *   kv_chunk_tokens  host: the keys of all (sequence, KV head) pairs are cut into 32-key
 *                    tiles and split into equal shares, one per wave; 0 = an even split
 *                    over at most 1024 waves, otherwise shares of ceil(kv_chunk_tokens/32)
 *                    tiles (widened if the sequences hold more than max_seq_len allows)
 *   workspace        fp32 partials of pairs cut between shares, plus one header per share;
 *                    >= spexis_verify_attention_workspace_size(...) bytes, device memory
 * Supported: head_dim in {64, 128}, block_size in {16, 32}, (Hq/Hkv) * max_query_len <= 64,
 * num_seqs * Hkv * ceil(max_blocks_per_seq * block_size / 32) < 2^31.
 * Errors: INVALID_ARGUMENT, UNSUPPORTED, WORKSPACE_TOO_SMALL, HIP.
 */
int spexis_verify_attention(const void* k_cache, const void* v_cache, int32_t num_blocks,
                            int32_t num_kv_heads, int32_t block_size, int32_t head_dim,
                            int32_t num_seqs, const int32_t* query_start_loc,
                            const int32_t* seq_lens, const int32_t* block_tables,
                            int32_t max_blocks_per_seq, int32_t total_tokens,
                            int32_t max_query_len, int32_t max_seq_len, const void* q,
                            int32_t num_q_heads, float scale, void* out,
                            int32_t kv_chunk_tokens, void* workspace, size_t workspace_bytes,
                            void* stream);

/*
 * spexis_softmax_rows -- the probabilities p = softmax(logits / T) and q that the acceptance
 * rule of [sd] (Related Work) compares, for callers that pass probabilities to spexis_accept
 * (Sec. 4: the verifying model's outputs are turned into per-token probabilities):
 * probs[r][v] = exp((logits[r][v] - max_u logits[r][u]) / T) / sum_u exp(...), fp32, for rows
 * r < rows (the temperature divides the logits of target and draft rows alike).  Computed as
 * 2^(x c - M) / Z with c = log2(e) / T, the expression spexis_accept uses with logits.  logits
 * and probs are [rows][vocab] fp32 and may alias.
 * Errors: INVALID_ARGUMENT (null, rows < 0, vocab <= 0, temperature <= 0 or not finite).
 */
int spexis_softmax_rows(const float* logits, float* probs, int64_t rows, int32_t vocab,
                        float temperature, void* stream);

/* Bytes of workspace spexis_accept needs. */
size_t spexis_accept_workspace_size(int32_t num_seqs, int32_t vocab, int32_t max_k);

/*
 * spexis_accept -- speculative-sampling acceptance, the rule of [sd] (Related Work) that
 * decides how many drafts survive verification (Sec. 4, Fig. 3: accepted tokens continue,
 * rejected ones are re-executed).
 *
 * Sequence b has k_b = qsl[b+1]-qsl[b]-1 drafts x_i = draft_ids[qsl[b]-b+i].  Its target
 * rows are target[qsl[b]+i] (i = 0..k_b), its draft rows draft[qsl[b]-b+i] (i < k_b).
 * kind = SPEXIS_INPUT_PROBS: rows are fp32 probabilities p_i, q_i.
 * kind = SPEXIS_INPUT_LOGITS: rows are fp32 logits; p_i = softmax(target_i / T) and
 *        q_i = softmax(draft_i / T) are formed on the fly (temperature > 0).
 * For every b:
 *   1. any x_i outside [0, vocab): row_status = BAD_TOKEN, accepted_len = 0, tokens -1.
 *   2. draft i is accepted iff (double)u_accept[qsl[b]-b+i] * (double)q_i(x_i)
 *      < (double)p_i(x_i), an exact comparison equal to u < min(1, p/q) for u in [0,1);
 *      a_b = number of leading accepts.
 *   3. a_b < k_b: weights w = max(0, fp32(p_a - q_a)); a_b = k_b: w = p_k (bonus).  Rows
 *      read here must be finite and >= 0, else row_status = BAD_VALUE and the token at
 *      position a_b is -1.  (row_status = INTERNAL flags a library fault, never expected.)
 *   4. the token at position a_b is the inverse-CDF sample of w with u_sample[b], taken in
 *      exact fixed point at the scale of the target row: M = max p_a in [2^e, 2^(e+1)),
 *      W_v = floor(w_v * 2^(40-e)), S = sum W_v (if S = 0 for a residual, the weights are
 *      p_a's instead), t = floor(u_sample[b] * S) (exact), token = smallest m with
 *      W_0 + ... + W_m > t.  p_a without a positive entry: row_status = EMPTY, token -1.
 * Outputs: accepted_len[b] = a_b; out_tokens[b][0..a_b) = x_0..x_{a_b-1};
 *   out_tokens[b][a_b] = the sampled token; out_tokens[b][i > a_b] = -1 (out_tokens is
 *   [B][max_k+1] int32); row_status[b]; if seq_lens_inout != NULL,
 *   seq_lens_inout[b] -= k_b - a_b (rows of rejected drafts become stale), except for
 *   BAD_TOKEN rows.
 *
 *   total_tokens  host: T = qsl[B]; target has T rows, draft T - B rows of `vocab` fp32
 *   max_k         host: >= max_b k_b, <= 32
 *   u_accept      [T-B] fp32, u_sample [B] fp32, in [0,1)
 *   workspace     >= spexis_accept_workspace_size(num_seqs, vocab, max_k) bytes
 * Supported: vocab <= 4194304.  Errors: INVALID_ARGUMENT, UNSUPPORTED,
 * WORKSPACE_TOO_SMALL, HIP.
 */
int spexis_accept(int32_t kind, int32_t num_seqs, int32_t vocab, int32_t max_k,
                  float temperature, int32_t total_tokens, const int32_t* query_start_loc,
                  const float* target, const float* draft, const int32_t* draft_ids,
                  const float* u_accept, const float* u_sample, int32_t* accepted_len,
                  int32_t* out_tokens, int32_t* row_status, int32_t* seq_lens_inout,
                  void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of the static scratch array spexis_accept_noalloc works in (16 MiB per GPU). */
#define SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES (16 << 20)

/*
 * spexis_accept_noalloc -- spexis_accept without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Arguments, outputs and errors as spexis_accept; the kernels' scratch is a
 * static device array of SPEXIS_ACCEPT_NOALLOC_SCRATCH_BYTES that every GPU the library runs on
 * holds until the process ends.  Its address is looked up on the first call on each device (with
 * that device current; `stream` must belong to it).  The call allocates nothing and calls no
 * allocating routine.
 *   - A problem whose workspace (spexis_accept_workspace_size) exceeds the array is rejected with
 *     SPEXIS_ERR_UNSUPPORTED before any launch: 16 MiB holds e.g. 1024 sequences of 8 drafts over a
 *     152064-entry vocabulary.
 *   - Every call on one GPU shares that GPU's array, and the array keeps the last call's
 *     contents.  No kernel reads scratch it has not written in the same call (the round
 *     counters are cleared by the first kernel), so the contents left by an earlier call never
 *     matter.  Calls that overlap on one GPU (different streams, or host threads) race on the
 *     array and give undefined results; serialise them.
 */
int spexis_accept_noalloc(int32_t kind, int32_t num_seqs, int32_t vocab, int32_t max_k,
                          float temperature, int32_t total_tokens, const int32_t* query_start_loc,
                          const float* target, const float* draft, const int32_t* draft_ids,
                          const float* u_accept, const float* u_sample, int32_t* accepted_len,
                          int32_t* out_tokens, int32_t* row_status, int32_t* seq_lens_inout,
                          void* stream);

/*
 * spexis_lm_head -- the output projection in front of acceptance (the verifying stage owns an
 * LM head, Implementation), with the softmax statistics acceptance needs fused into it:
 *   logits[m][v] = sum_j hidden[m][j] * weight[v][j]        (fp32 accumulation)
 *   stats[m][t] = (max x*c, sum 2^(x*c - max)) over columns v of tile t = v / 128, v < vocab,
 *                 x = logits[m][v], c = log2(e) / temperature
 *
 *   hidden   [rows][hidden_dim] bf16 (read);  weight [vocab][hidden_dim] bf16 packed by
 *            spexis_pack_weight (read)
 *   logits   [rows][vocab] fp32 (written), or NULL to write only the statistics
 *   stats    [rows][spexis_lm_head_tiles(vocab)][2] fp32 (written)
 * Supported: hidden_dim a multiple of 256.  Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
int spexis_lm_head(const void* hidden, const void* weight, int32_t rows, int32_t vocab,
                   int32_t hidden_dim, float temperature, float* logits, float* stats,
                   void* stream);

/*
 * spexis_lm_head_gather -- spexis_lm_head that also gathers, in its epilogue, the logit each row
 * contributes to an acceptance test: the target and draft logits at the drafted token x_i (the
 * gathers at x_i fused into the LM head of the verifying stage, Implementation; the tests of
 * [sd], Related Work).  Arguments as spexis_lm_head (stats must not be NULL), plus
 *   gather_cols  [rows] int32: the column row m gathers, or -1 (any value outside [0, vocab)
 *                gathers nothing).  For draft rows these are the draft ids themselves; for target
 *                rows spexis_verify_gather_columns builds them.
 *   gathered     [rows] fp32 output: gathered[m] = logits[m][gather_cols[m]], the same fp32 value
 *                the logits output holds; rows that gather nothing are not written
 * Errors: as spexis_lm_head; INVALID_ARGUMENT for a NULL gather_cols or gathered.
 */
int spexis_lm_head_gather(const void* hidden, const void* weight, int32_t rows, int32_t vocab,
                          int32_t hidden_dim, float temperature, float* logits, float* stats,
                          const int32_t* gather_cols, float* gathered, void* stream);

/*
 * spexis_verify_gather_columns -- the target rows' gather columns of a verification batch: row
 * qsl[b]+i verifies draft x_i = draft_ids[qsl[b]-b+i] (i < k_b) and gathers at it; each
 * sequence's last row (its bonus position) gets -1.
 *   total_tokens  host: T = qsl[B];  draft_ids [T-B] int32;  cols [T] int32 output
 * Errors: INVALID_ARGUMENT (bad sizes, NULL pointers), HIP.
 */
int spexis_verify_gather_columns(int32_t num_seqs, int32_t total_tokens, const int32_t* query_start_loc,
                                 const int32_t* draft_ids, int32_t* cols, void* stream);

/* Column tiles per row of spexis_lm_head's statistics: ceil(vocab / 128). */
int32_t spexis_lm_head_tiles(int32_t vocab);

/* Bytes of spexis_lm_head's statistics for `rows` rows. */
size_t spexis_lm_head_stats_size(int32_t rows, int32_t vocab);

/*
 * spexis_accept_with_stats -- spexis_accept for logits whose softmax statistics are already
 * known, e.g. from spexis_lm_head (same temperature): the acceptance then reads a logit row
 * only where it samples, never to normalise it.  Arguments and outputs as spexis_accept with
 * kind = SPEXIS_INPUT_LOGITS, plus
 *   target_stats  [T][stats_tiles][2] fp32, draft_stats [T-B][stats_tiles][2] fp32: for
 *                 every row, (max y*c, sum 2^(y*c - max)) over each of stats_tiles disjoint
 *                 column ranges that together cover the row, c = log2(e) / temperature
 *   target_gathered, draft_gathered  both NULL, or [T] and [T-B] fp32: the logits at the drafts,
 *                 target row qsl[b]+i and draft row qsl[b]-b+i at x_i (i < k_b), as
 *                 spexis_lm_head_gather writes them; then the tests read no logit row
 * Errors: as spexis_accept; INVALID_ARGUMENT if only one gathered array is given.
 */
int spexis_accept_with_stats(int32_t num_seqs, int32_t vocab, int32_t max_k, float temperature,
                             int32_t total_tokens, const int32_t* query_start_loc,
                             const float* target_logits, const float* draft_logits,
                             const float* target_stats, const float* draft_stats,
                             int32_t stats_tiles, const int32_t* draft_ids,
                             const float* u_accept, const float* u_sample,
                             const float* target_gathered, const float* draft_gathered,
                             int32_t* accepted_len, int32_t* out_tokens, int32_t* row_status,
                             int32_t* seq_lens_inout, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * spexis_select_drafts -- acceptance-guided selective speculation (Sec. 5): rank the batch's
 * draft tokens by confidence and drop the lowest-ranked fraction alpha before verification.
 *   - draft i of sequence b (index qsl[b]-b+i, i < k_b = qsl[b+1]-qsl[b]-1) has confidence
 *     draft_conf[...], typically the draft model's probability of the token it drafted; NaN
 *     counts as 0 and values are clamped into [0, 1];
 *   - its score is the confidence of its prefix, the fp32 product of the confidences of drafts
 *     0..i of its sequence taken in order (a draft is verified only after every earlier one);
 *   - the N = T - B drafts are ordered by score, higher first, equal scores lower index first;
 *     the last m = floor(alpha * N) are dropped, and every sequence keeps the drafts before its
 *     first dropped one.
 * Outputs: kept_k [B] (drafts kept per sequence), kept_query_start_loc [B+1] (the
 * query_start_loc of the reduced batch, kept_k[b] + 1 tokens per sequence), keep [N] (1 for a
 * kept draft, else 0).
 *   total_tokens  host: T = qsl[B];  alpha: host, in [0, 1)
 * No workspace: one workgroup holds the scores in LDS.  draft_conf and keep may be NULL when
 * T == B.  Supported: T - B <= 16384.  Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
int spexis_select_drafts(int32_t num_seqs, int32_t total_tokens, const int32_t* query_start_loc,
                         const float* draft_conf, float alpha, int32_t* kept_k,
                         int32_t* kept_query_start_loc, int32_t* keep, void* stream);

/*
 * spexis_pack_weight -- lays out a bf16 weight W [rows][cols] (row-major) for spexis_lm_head and
 * spexis_linear, once per weight: tiles of 32 rows x 64 columns, 4 KB each, in (row tile, column
 * tile) order; inside a tile the element (r, 64c + 32h + 8s + e) sits at ((s*2 + h)*32 + r)*8 + e,
 * the operand order of the matrix-core instruction, so that the projections read W as
 * contiguous 1 KB runs.  Rows past `rows` are zero.
 *   weight  [rows][cols] bf16, device;  packed: spexis_packed_weight_size(rows, cols) bytes,
 *           device, written; may not alias weight
 * Supported: cols % 64 == 0.  Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
int spexis_pack_weight(const void* weight, int32_t rows, int32_t cols, void* packed, void* stream);

/* Bytes of a packed weight: ceil(rows / 32) * 32 * cols * 2 (0 for unsupported sizes). */
size_t spexis_packed_weight_size(int32_t rows, int32_t cols);

/*
 * spexis_linear -- a linear layer of the drafting adapter (Implementation: the adapter is a
 * linear layer and an attention layer followed by the LM head), also its attention layer's
 * input and output projections:
 *   y[r][o] = bf16( sum_j x[r][j] * W[o][j]  (+ residual[r][o]) )
 * with fp32 accumulation (the order over j is the library's) and one round to nearest even.
 *   x         [rows][in_features] bf16;  weight: [out_features][in_features] bf16 packed by
 *             spexis_pack_weight
 *   residual  [rows][out_features] bf16 or NULL;  y: [rows][out_features] bf16 output (may not
 *             alias x or weight; may alias residual)
 *   workspace >= spexis_linear_workspace_size(rows, out_features, in_features) bytes (0 when
 *             the problem fills the chip without splitting K; then it may be NULL)
 * Supported: in_features % 256 == 0.  Errors: INVALID_ARGUMENT, UNSUPPORTED,
 * WORKSPACE_TOO_SMALL, HIP.
 */
int spexis_linear(const void* x, const void* weight, const void* residual, int32_t rows, int32_t out_features,
                  int32_t in_features, void* y, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spexis_linear needs for this problem (0 if none). */
size_t spexis_linear_workspace_size(int32_t rows, int32_t out_features, int32_t in_features);

/*
 * spexis_linear_split -- several linear layers of one input in one call: the drafting adapter's
 * attention-layer q, k and v projections of x (Implementation).  weight is the packed stack of
 * the layers' weights, W = [W_0; W_1; ...] with W_i [out_features[i]][in_features] in output
 * order (spexis_pack_weight of the stacked rows), and output i receives its columns of x W^T:
 *   y_i[r][o] = bf16( sum_j x[r][j] * W[c_i + o][j] ),   c_i = out_features[0] + ... + [i-1]
 * with fp32 accumulation (the order over j is the library's) and one round to nearest even; no
 * residual.  One projection launch and one launch that adds the K-split partials and routes each
 * layer's columns: at few rows, where each launch is latency-bound, fewer launches than one
 * spexis_linear per layer.
 *   x            [rows][in_features] bf16
 *   num_outputs  1 .. 4;  out_features: host [num_outputs], each > 0 and a multiple of 4
 *   outputs      host [num_outputs] of device pointers: output i is [rows][out_features[i]]
 *                bf16 (may not alias x, weight or one another)
 *   workspace    >= spexis_linear_split_workspace_size(rows, sum of out_features, in_features)
 *                bytes (the fp32 products pass through it: never 0 when rows > 0)
 * Supported: in_features % 256 == 0.  Errors: INVALID_ARGUMENT (bad sizes or count, NULL
 * pointers), UNSUPPORTED (widths, in_features, size), WORKSPACE_TOO_SMALL, HIP.
 */
int spexis_linear_split(const void* x, const void* weight, int32_t rows, int32_t in_features, int32_t num_outputs,
                        const int32_t* out_features, void* const* outputs, void* workspace, size_t workspace_bytes,
                        void* stream);

/* Bytes of workspace spexis_linear_split needs (0 for an empty or unsupported problem). */
size_t spexis_linear_split_workspace_size(int32_t rows, int32_t total_out_features, int32_t in_features);

/*
 * spexis_sample_tokens -- draws one token per row from softmax(logits / T) (kind LOGITS) or from
 * the given fp32 probabilities (kind PROBS), and returns the token's probability.  Drafting uses
 * it on the adapter's LM-head rows (Implementation): the token is the draft x, its probability
 * q(x) the draft's confidence that selective speculation ranks (Sec. 5).  The draw is the bonus
 * sampling of spexis_accept with no drafts: the exact fixed-point inverse CDF with the row's
 * uniform, so PROBS input gives the same token as any exact implementation of that rule.
 *   rows, vocab     R >= 0 rows of V entries;  input [R][V] fp32
 *   stats           optional (LOGITS only): [R][stats_tiles][2] from spexis_lm_head at the same
 *                   temperature; then no pass over the rows computes their normalisers
 *   u               [R] fp32 uniforms in [0, 1)
 *   tokens          [R] int32 output (-1 for a row that cannot be sampled)
 *   token_prob      [R] fp32 output or NULL: the probability of the token (0 when none); in
 *                   LOGITS mode computed as in spexis_accept (2^(x c - M) / Z, c = log2(e) / T)
 *   row_status      [R] int32 output, SPEXIS_ROW_* as in spexis_accept
 *   workspace       >= spexis_sample_workspace_size(R, V) bytes
 * Errors: INVALID_ARGUMENT, UNSUPPORTED (V > 2^22), WORKSPACE_TOO_SMALL, HIP.
 */
int spexis_sample_tokens(int32_t kind, int32_t rows, int32_t vocab, float temperature, const float* input,
                         const float* stats, int32_t stats_tiles, const float* u, int32_t* tokens, float* token_prob,
                         int32_t* row_status, void* workspace, size_t workspace_bytes, void* stream);

/* Bytes of workspace spexis_sample_tokens needs. */
size_t spexis_sample_workspace_size(int32_t rows, int32_t vocab);

/*
 * spexis_lookahead_memory -- the look-ahead memory estimate of Algorithm 1 (Sec. 5,
 * Remaining-Length-Aware Scheduling): the expected KV-cache tokens the running requests hold
 * in each of the next `iters` decoding iterations, which the scheduler compares with the cache
 * size before admitting a new request.
 *   For iteration i = 1 .. iters and w = 0 .. floor(i / pp) rejections, t = i - pp*w accepted
 *   and k = t + w generated tokens have probability p(i, w) = C(k, t) theta^t (1 - theta)^w;
 *   E_gen(i) = sum_w k p(i, w);  Pfin_r(i) = precision[r] * sum_{w : k >= remaining[r]} p(i, w);
 *   mem[i-1] = sum_r cur_len[r] + (n - sum_r Pfin_r) E_gen - sum_r cur_len[r] Pfin_r.
 *   num_requests   n >= 0, the running requests
 *   cur_len        [n] int64, current length of each request (tokens in the cache)
 *   remaining      [n] int32, predicted remaining length (the ordinal thresholds 4, 8, .., 64,
 *                  or a large value for "more than 64")
 *   precision      [n] fp64, the precision of that prediction, the paper's E(tau)
 *   pp, theta      host: pipeline depth >= 1 and speculation accuracy in [0, 1]
 *   iters          host: look-ahead iterations, 1 .. 1024 (the paper uses 64)
 *   mem            [iters] fp64 output; e_gen, e_nfin, e_lfin: optional [iters] fp64 outputs of
 *                  E_gen, sum_r Pfin_r and sum_r cur_len[r] Pfin_r (NULL to skip)
 * All fp64.  No workspace.  Errors: INVALID_ARGUMENT, UNSUPPORTED, HIP.
 */
int spexis_lookahead_memory(int32_t num_requests, const int64_t* cur_len, const int32_t* remaining,
                            const double* precision, int32_t pp, double theta, int32_t iters,
                            double* mem, double* e_gen, double* e_nfin, double* e_lfin, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPEXIS_H */
