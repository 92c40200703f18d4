/*
 * agentspec_verify.h -- C ABI of the batched speculative-verification step.
 *
 * Speculative decoding proposes several draft tokens per request and verifies
 * them with the target model in a single pass; the output is the same as
 * plain decoding (paper, Sec. 2.2).  In a batch, every request i carries its
 * own draft length k_i >= 0 (the per-request draft length L_i that the
 * redundancy-aware allocator hands out, Sec. 4.2 / Alg. 2; k_i = 0 for a
 * request that does not speculate), so the target scores n_i = k_i + 1
 * positions of request i, and the step's cost grows with the number of drafts
 * D(b) it verifies (Sec. 3.1).  The library implements that verify pass on one
 * AMD Instinct MI355X (gfx950):
 *
 *   verify_attention -- the attention of all sum_i n_i query rows of one layer
 *                       against each request's paged KV cache;
 *   verify_accept    -- the vocabulary argmax of every scored position and
 *                       greedy acceptance: the longest draft prefix that agrees
 *                       with the target, plus one bonus token.  The rejection
 *                       rate of Sec. 3.1 is (k_i - accept_len_i) / k_i.
 *   verify_budget    -- the step upstream of both: the redundancy-aware draft
 *                       lengths k_i = L_i of Sec. 4.2 / Alg. 2, and the verify
 *                       step's q_start / tokens / seq_lens built from them.
 *   verify_kv_append -- the n_i new tokens' K/V written into their cache slots
 *                       before verify_attention reads them.
 *   verify_attention_append -- both in one launch sequence: the attention
 *                       reads the new tokens from the caller's arrays while it
 *                       stores them into the cache.
 *   verify_accept_sampled -- verify_accept at a temperature T > 0: each row
 *                       draws its token from softmax(logits / T) instead of
 *                       taking the argmax (speculative sampling with drafts
 *                       that are single tokens).
 *   verify_lmhead_accept -- verify_accept fed by the LM head itself: the
 *                       logits of every scored position are computed from the
 *                       final hidden states and reduced to the argmax on the
 *                       fly, never stored.
 *   verify_check_batch -- the batch descriptor's preconditions, checked on the
 *                       device.
 *
 * Conventions shared by the calls
 * --------------------------------
 *  - Requests are packed: query rows q_start[i] .. q_start[i+1]-1 (int32,
 *    num_seqs+1 entries, q_start[0] = 0, non-decreasing) belong to request i;
 *    total_q = q_start[num_seqs].  Row j of request i is the model input at
 *    absolute position S_i - n_i + j, where S_i = seq_lens[i] counts the
 *    request's cached keys including the n_i new ones (their K/V are in the
 *    cache before verify_attention runs: the caller writes them, or calls
 *    verify_kv_append first on the same stream).
 *  - All array pointers are device pointers owned by the caller.  The library
 *    allocates nothing, keeps no state between calls, never reads device data
 *    on the host, and is safe to call from several host threads on different
 *    streams (each call with its own workspace).
 *  - Calls are asynchronous: they validate host-side arguments, enqueue their
 *    kernels on `stream` and return.  Device-side errors surface at the next
 *    synchronising HIP call.
 *  - Return value: VERIFY_OK (0) or a negative status; on a negative status
 *    nothing was enqueued.  verify_status_string() names a status.
 *  - Storage dtypes: VERIFY_F32 (IEEE binary32) or VERIFY_BF16 (bfloat16).
 *    Arithmetic is fp32 (bf16 products accumulate in fp32); outputs are
 *    rounded to the storage dtype with round-to-nearest-even.
 */
#ifndef AGENTSPEC_VERIFY_H
#define AGENTSPEC_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum verify_status {
    VERIFY_OK = 0,
    VERIFY_EINVAL = -1,       /* null pointer, negative size, inconsistent arguments   */
    VERIFY_EUNSUPPORTED = -2, /* head_dim, block_size or dtype this library does not handle,
                                 or sizes beyond a launch grid's limits                 */
    VERIFY_EWORKSPACE = -3,   /* workspace smaller than the size query returned        */
    VERIFY_EHIP = -4          /* a kernel launch failed (hipGetLastError)               */
};

enum verify_dtype { VERIFY_F32 = 0, VERIFY_BF16 = 1 };

/* Shape and layout of one attention layer. */
typedef struct verify_attn_params {
    int32_t num_seqs;           /* requests in the batch (>= 0)                         */
    int32_t num_q_heads;        /* Hq                                                   */
    int32_t num_kv_heads;       /* Hkv; Hq % Hkv == 0; q-head h reads KV head h/(Hq/Hkv) */
    int32_t head_dim;           /* D: 64 or 128                                         */
    int32_t block_size;         /* tokens per KV block: must be 16                       */
    int32_t max_blocks_per_seq; /* row stride of block_tables                           */
    int32_t num_blocks;         /* physical blocks in k_cache / v_cache                 */
    int32_t sliding_window;     /* W > 0: row at position p sees keys p-W < t <= p;
                                   0: full causal (keys t <= p)                         */
    float scale;                /* softmax scale; 0 selects 1/sqrt(D)                   */
    int32_t dtype;              /* verify_dtype of q, k_cache, v_cache and out          */
    int32_t kv_split_blocks;    /* KV blocks per split-K work item; 0 = automatic.
                                   Results agree across splits up to fp32 rounding.     */
} verify_attn_params;

/*
 * verify_attention -- softmax attention of every packed query row against its
 * request's paged KV cache (the target-model scoring of Sec. 2.2, for one
 * layer).
 *
 * For request i, row j (0 <= j < n_i), query head h, with p = S_i - n_i + j,
 * g = h / (Hq/Hkv) and the visible keys t in [max(0, p-W+1), p] (W > 0) or
 * [0, p] (W = 0):
 *     out[row][h] = sum_t softmax_t(scale * <q[row][h], K_g[t]>) * V_g[t]
 * where K_g[t], V_g[t] are read through block_tables[i][t / 16].  With sinks,
 * head h's sink logit sinks[h] joins each of its rows' softmax as one more
 * logit whose value is zero (it only enlarges the denominator): the attention
 * sinks of GPT-OSS models, which the paper serves but does not describe.
 *
 *   q            [total_q][Hq][D]                     (dtype)
 *   k_cache      [num_blocks][Hkv][D/x][16][x]        x = 16 bytes / element
 *                (token t, dim d of a block at [d/x][t][d%x])
 *   v_cache      [num_blocks][Hkv][D][16]             (token t, dim d at [d][t])
 *   block_tables [num_seqs][max_blocks_per_seq] int32 physical block ids; the
 *                first ceil(S_i/16) entries of row i are read, ids outside
 *                [0, num_blocks) are skipped (their keys contribute nothing)
 *   seq_lens     [num_seqs] int32 S_i, with n_i <= S_i <= max_seq_len and
 *                S_i <= 16 * max_blocks_per_seq (larger values are clamped)
 *   q_start      [num_seqs + 1] int32
 *   sinks        [Hq] float sink logits in the units of the scaled scores
 *                (scale * <q, k>), or NULL for none
 *   out          [total_q][Hq][D]                     (dtype); a row with no
 *                visible key (S_i < n_i) is written as zeros
 *   max_q_len    host upper bound on n_i; max_seq_len host upper bound on S_i
 *                (they size the launch; tighter bounds launch less idle work).
 *                Rows of a request with n_i > max_q_len that the launch does
 *                not reach (verify_attention_plan gives the reach: rows j with
 *                j * (Hq/Hkv) + h % (Hq/Hkv) below the row groups times the
 *                rows per group of the request's row class) are not
 *                computed: their outputs are written as quiet NaN.
 *   workspace    device scratch of at least the size returned by
 *                verify_attention_workspace_size() for the same (params,
 *                total_q, max_q_len, max_seq_len); may be NULL if that size is
 *                0.  Its contents on entry are ignored.
 */
int verify_attention_workspace_size(const verify_attn_params *params, int32_t total_q,
                                    int32_t max_q_len, int32_t max_seq_len, size_t *bytes);

int verify_attention(const verify_attn_params *params, int32_t total_q, int32_t max_q_len,
                     int32_t max_seq_len, const void *q, const void *k_cache,
                     const void *v_cache, const int32_t *block_tables,
                     const int32_t *seq_lens, const int32_t *q_start, const float *sinks,
                     void *out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * verify_attention_append -- verify_kv_append and verify_attention in one
 * launch sequence: the n_i new tokens' K/V of every request (the scored
 * positions of Sec. 2.2 are the new tokens, positions S_i - n_i .. S_i - 1)
 * are written into their cache slots, and the attention reads them from
 * k_new / v_new while it walks the cache, so it never waits for the writes.
 *
 *   k_new, v_new [total_q][Hkv][D] (dtype): row j of request i holds the K
 *                and V of position S_i - n_i + j (the layout of
 *                verify_kv_append); required when total_q > 0
 *   k_cache, v_cache: read as by verify_attention and written in place: every
 *                new token whose position lies in [0, min(S_i, max_seq_len,
 *                16 * max_blocks_per_seq)) and whose block id lies in
 *                [0, num_blocks) is stored to its slot, element bits
 *                unchanged; other new tokens are neither stored nor read.
 *   all other arguments and the workspace as for verify_attention (the size
 *   that verify_attention_workspace_size returns covers both calls).
 * Under verify_attention's bounds (S_i <= max_seq_len <= 16 *
 * max_blocks_per_seq), out and the cache equal, bit for bit, what
 * verify_kv_append followed by verify_attention on the same stream writes.
 * k_new / v_new must not overlap the caches.
 */
int verify_attention_append(const verify_attn_params *params, int32_t total_q, int32_t max_q_len,
                            int32_t max_seq_len, const void *q, const void *k_new,
                            const void *v_new, void *k_cache, void *v_cache,
                            const int32_t *block_tables, const int32_t *seq_lens,
                            const int32_t *q_start, const float *sinks, void *out,
                            void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * verify_attention_plan -- the work decomposition verify_attention would use
 * for the same arguments, for tests and tools (nothing is launched).
 * verify_attention_append may launch fewer persistent workgroups where its
 * kernel fits fewer per compute unit; it is not described here.
 *
 *   info     int32[VERIFY_ATTN_PLAN_INFO], written in full (unused entries 0)
 *   info[0]  1: bf16 persistent MFMA schedule, 0: fp32 split-K VALU kernel
 *   bf16:    info[5] row classes (1 or 2), one persistent launch each; a
 *            request whose Hq/Hkv * n_i is at most info[10] is in class 0,
 *            the others in class 1.  Class 0 in info[1..4], class 1 in
 *            info[6..9]: workgroups, query rows per row group, row groups
 *            per (request, KV head) at most, fixed units per workgroup (0:
 *            equal shares).  A unit is one 16-token block of one (request, KV
 *            head, row group) pair of the class's requests; units are
 *            numbered request by request, then KV head, then row group, then
 *            block, and workgroup w owns units [U w / N, U (w + 1) / N) of the
 *            class's U units (N = min(workgroups, U)).
 *   fp32:    info[1] splits per request at most, info[2] query rows per work
 *            item, info[3] row groups, info[4] KV blocks per split.
 * Same argument checks as verify_attention_workspace_size.
 */
#define VERIFY_ATTN_PLAN_INFO 11
int verify_attention_plan(const verify_attn_params *params, int32_t total_q, int32_t max_q_len,
                          int32_t max_seq_len, int32_t *info);

/*
 * verify_kv_append -- the verify step's new tokens' K and V into the paged
 * cache (the K/V that verify_attention reads for positions S_i - n_i .. S_i - 1).
 *
 * Row j of request i (the token at position p = S_i - n_i + j) is written to
 * slot p % 16 of block block_tables[i][p / 16], for every KV head, in the
 * layouts of verify_attention.  params supplies num_seqs, num_kv_heads,
 * head_dim, block_size, max_blocks_per_seq, num_blocks and dtype (the other
 * fields are validated as for verify_attention and otherwise unused).
 *
 *   k_new, v_new [total_q][Hkv][D] (dtype): the new tokens' keys and values
 *   k_cache, v_cache: written in place; rows with a negative position or a
 *                block id outside [0, num_blocks) are skipped
 * No workspace.  Element bits are copied unchanged.
 */
int verify_kv_append(const verify_attn_params *params, int32_t total_q, const void *k_new,
                     const void *v_new, const int32_t *block_tables, const int32_t *seq_lens,
                     const int32_t *q_start, void *k_cache, void *v_cache, hipStream_t stream);

/*
 * verify_accept -- vocabulary argmax of each scored position and greedy
 * acceptance of the drafts (Sec. 2.2 verification; Sec. 3.1 rejection rate).
 *
 *   logits      [total_q][row_stride] (logits_dtype), vocab entries per row used;
 *               row_stride = 0 means vocab
 *   tokens      [total_q] int32: tokens[q_start[i]] is request i's last committed
 *               token, tokens[q_start[i] + j] (1 <= j <= k_i) is its draft j
 *   argmax_out  [total_q] int32 or NULL: argmax_out[r] = the lowest index v with
 *               logits[r][v] equal to the row maximum (-0.0 equals +0.0; if the
 *               row holds a NaN, the index of its first NaN)
 *   accept_len  [num_seqs] int32: m_i = number of leading drafts j = 1..k_i with
 *               tokens[q_start[i] + j] == argmax[q_start[i] + j - 1]
 *   num_emitted [num_seqs] int32: m_i + 1 (0 for a request with no rows)
 *   emitted     [total_q] int32: request i's drafts 1..m_i, then the bonus token
 *               argmax[q_start[i] + m_i], starting at emitted[q_start[i]]; the
 *               request's remaining rows are set to -1
 *   workspace   device scratch of at least verify_accept_workspace_size() bytes
 *               (may be NULL if that is 0); its contents on entry are ignored.
 * Requires vocab >= 1 and vocab < 2^31.
 */
int verify_accept_workspace_size(int32_t num_seqs, int32_t total_q, int64_t vocab,
                                 int32_t logits_dtype, size_t *bytes);

int verify_accept(int32_t num_seqs, int32_t total_q, int64_t vocab, int64_t row_stride,
                  int32_t logits_dtype, const void *logits, const int32_t *tokens,
                  const int32_t *q_start, int32_t *argmax_out, int32_t *accept_len,
                  int32_t *num_emitted, int32_t *emitted, void *workspace,
                  size_t workspace_bytes, hipStream_t stream);

/*
 * verify_accept_noalloc -- verify_accept for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  It takes no workspace; its scratch (the
 * per-(row, chunk) maxima and, when argmax_out is NULL, the argmax) lives in
 * a device array of VERIFY_NOALLOC_SCRATCH_BYTES that the library holds on
 * each GPU it runs on until the process ends.  The call itself allocates
 * nothing.
 *
 * Arguments, outputs and results are verify_accept's (bit-identical).
 * VERIFY_EWORKSPACE (nothing enqueued) if verify_accept_workspace_size() for
 * the same (num_seqs, total_q, vocab, logits_dtype) exceeds
 * VERIFY_NOALLOC_SCRATCH_BYTES; with bf16 logits that holds up to about
 * 340 000 rows.  VERIFY_EHIP if the scratch's device address cannot be
 * obtained.
 * All calls on one GPU share its scratch: calls that overlap on one GPU (on
 * different streams, or from different host threads without ordering) race
 * and may return wrong results.  Calls on one stream are ordered and safe.
 */
#define VERIFY_NOALLOC_SCRATCH_BYTES (4u << 20)

int verify_accept_noalloc(int32_t num_seqs, int32_t total_q, int64_t vocab, int64_t row_stride,
                          int32_t logits_dtype, const void *logits, const int32_t *tokens,
                          const int32_t *q_start, int32_t *argmax_out, int32_t *accept_len,
                          int32_t *num_emitted, int32_t *emitted, hipStream_t stream);

/*
 * verify_accept_sampled -- stochastic verification at temperature T > 0
 * (Sec. 2.2: the speculative output follows the target's distribution).
 *
 * The drafts are single tokens, i.e. proposals with all their probability on
 * one token.  Speculative rejection sampling then accepts draft d at row r
 * with probability p_r(d), p_r = softmax(logits[r] / T), and on rejection
 * emits a token from p_r with d removed.  Drawing y_r ~ p_r and accepting
 * iff y_r == d is the same rule, so the call draws one y_r per row and runs
 * verify_accept's acceptance with y in place of the argmax.
 *
 * y_r = argmax_v (x_v * inv_T + g_v) (the Gumbel-max rule), where
 *   inv_T = (float)(1.0 / (double)temperature);
 *   g_v   = -log(-log u_v), u_v = ((w >> 9) + 0.5) * 2^-23 (exact in fp32);
 *   w     = word (v mod 4) of Philox4x32-10 (Salmon et al., SC 2011) with key
 *           (seed mod 2^32, seed >> 32) and counter (v / 4, r, offset, 0);
 *   log   = an fp32 atanh-series log: x = m 2^e with m in [sqrt(2)/2, sqrt(2)),
 *           z = (m - 1) / (m + 1), log x = e ln2 + 2 z (1 + z^2 (1/3 + z^2 (1/5
 *           + z^2 (1/7 + z^2 / 9)))), every step one fp32 operation (the
 *           products with fused multiply-add as written).
 * The draw is therefore a pure function of (logits, temperature, seed, offset,
 * row index) and is reproduced bit for bit by any implementation of those
 * steps.  NaN logits and ties follow verify_accept: the first NaN wins, equal
 * scores go to the lower index.  Rows are independent draws as long as
 * (seed, offset) is not reused; use offset for the decoding step.
 *
 *   temperature  finite, > 0 (VERIFY_EINVAL otherwise)
 *   sampled_out  [total_q] int32 or NULL: the drawn y_r
 * All other arguments, the workspace size and the outputs are verify_accept's,
 * with y in place of the argmax.
 */
int verify_accept_sampled(int32_t num_seqs, int32_t total_q, int64_t vocab, int64_t row_stride,
                          int32_t logits_dtype, const void *logits, const int32_t *tokens,
                          const int32_t *q_start, float temperature, uint64_t seed,
                          uint32_t offset, int32_t *sampled_out, int32_t *accept_len,
                          int32_t *num_emitted, int32_t *emitted, void *workspace,
                          size_t workspace_bytes, hipStream_t stream);

/*
 * verify_lmhead_accept -- the verify pass's LM head fused with greedy
 * acceptance (Sec. 2.2: the target scores every proposed position in one pass
 * and keeps the drafts that agree with its own greedy choice).
 *
 * For every scored row r and vocabulary entry v the logit is
 *     z[r][v] = <hidden[r], weight[v]>        (bf16 products, fp32 sums)
 * and argmax[r] is the lowest v attaining the row maximum (a NaN logit counts
 * as the maximum: the first NaN wins; -0.0 equals +0.0).  The logits are
 * reduced as they are produced and never written to memory.  Acceptance then
 * follows verify_accept exactly.  The fp32 sums are taken in a fixed order
 * inside the kernel but not in ascending h, so two logits closer than the
 * rounding of a hidden_size-term fp32 dot product may compare either way;
 * the plain definition in exact arithmetic fixes the order otherwise.
 *
 *   hidden      [total_q][hidden_size] bf16: the final hidden states (after
 *               the last normalisation) of the scored rows
 *   weight      [vocab][hidden_size] bf16: the LM-head (output embedding)
 *               weight, row v = token v
 *   hidden_size multiple of 32; vocab >= 1 and < 2^31; both pointers 16-byte
 *               aligned (VERIFY_EINVAL otherwise)
 *   dtype       VERIFY_BF16 (VERIFY_F32 returns VERIFY_EUNSUPPORTED)
 * tokens, q_start, argmax_out, accept_len, num_emitted and emitted are
 * verify_accept's.  workspace: at least
 * verify_lmhead_accept_workspace_size() bytes (may be NULL if that is 0); its
 * contents on entry are ignored.
 */
int verify_lmhead_accept_workspace_size(int32_t num_seqs, int32_t total_q, int32_t hidden_size,
                                        int64_t vocab, int32_t dtype, size_t *bytes);

int verify_lmhead_accept(int32_t num_seqs, int32_t total_q, int32_t hidden_size, int64_t vocab,
                         int32_t dtype, const void *hidden, const void *weight,
                         const int32_t *tokens, const int32_t *q_start, int32_t *argmax_out,
                         int32_t *accept_len, int32_t *num_emitted, int32_t *emitted,
                         void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * verify_budget -- redundancy-aware draft budget (Sec. 4.2, Alg. 2).
 *
 * Request i owns the candidate continuations retrieved for it (rows
 * cand_start[i] .. cand_start[i+1]-1; the paper retrieves them from the
 * request's generation history under the same semantic block and query).
 * The call scores each request's consensus and hands out the batch budget:
 *
 *   n_i   = number of candidates of request i (empty ones included)
 *   CT_i* = the non-empty prefix that the most candidates start with (the
 *           longest, then the lexicographically smallest, among equally
 *           frequent ones); c_i = the number of candidates starting with it
 *   p(n)  = g_min + (1 - g_min) (1 - e^(1-n))
 *   g_i   = (c_i / n_i) p(n_i)            (0 if request i has no non-empty one)
 *   B_t   = floor(alpha / num_seqs),  G = sum_i g_i (ascending i, double)
 *   L_i   = max(|CT_i*|, floor(B_t g_i / G)) (share 0 if G = 0), at most the
 *           length of the longest candidate starting with CT_i* (the lowest row
 *           among equals), whose first L_i tokens become request i's drafts.
 *
 *   cand_start  [num_seqs + 1] int32, non-decreasing, cand_start[num_seqs] <= num_cands
 *               (device values outside [0, num_cands] are clamped)
 *   cand_len    [num_cands] int32, tokens per candidate, clamped to [0, max_cand_len]
 *   cand_tokens [num_cands][max_cand_len] int32, row-major
 *   last_token  [num_seqs] int32: request i's last committed token
 *   ctx_len     [num_seqs] int32 or NULL: cached context length L_ctx of request i
 *   alpha >= 0, 0 <= g_min <= 1 (host doubles)
 * Outputs (device, caller-owned):
 *   score [num_seqs] double g_i; agree, prefix_len, source, draft_len
 *   [num_seqs] int32 (c_i, |CT_i*|, candidate row or -1, L_i);
 *   q_start [num_seqs + 1] int32: exclusive prefix sum of L_i + 1;
 *   tokens  [tokens_capacity] int32, capacity >= num_seqs * (max_cand_len + 1):
 *           tokens[q_start[i]] = last_token[i], then the L_i drafts;
 *   seq_lens [num_seqs] int32, given iff ctx_len is: ctx_len[i] + L_i + 1.
 * q_start, tokens and seq_lens are the verify_attention / verify_accept
 * descriptor of the next step (max_q_len <= max_cand_len + 1 bounds it).
 * No workspace; VERIFY_EINVAL on null or inconsistent arguments,
 * VERIFY_EUNSUPPORTED if num_seqs * (max_cand_len + 1) >= 2^31.
 */
int verify_budget(int32_t num_seqs, int32_t num_cands, int32_t max_cand_len,
                  const int32_t *cand_start, const int32_t *cand_len, const int32_t *cand_tokens,
                  const int32_t *last_token, const int32_t *ctx_len, double alpha, double g_min,
                  double *score, int32_t *agree, int32_t *prefix_len, int32_t *source,
                  int32_t *draft_len, int32_t *q_start, int32_t *tokens, int64_t tokens_capacity,
                  int32_t *seq_lens, hipStream_t stream);

/*
 * verify_check_batch -- validation of a verify batch's descriptor on the
 * device, for callers that want bad data reported rather than given the
 * defined behaviour of the calls above (which skip block ids outside the
 * cache, write zeros for rows without visible keys and NaN for rows a launch
 * does not reach, and may read out of bounds if q_start does not describe
 * total_q rows).  It checks the preconditions of the packed-request
 * convention (Sec. 2.2 scoring of n_i = k_i + 1 positions per request) and of
 * verify_attention / verify_kv_append.  Nothing else is read or written.
 *
 *   num_seqs, total_q, q_start   as for verify_attention and verify_accept
 *   max_q_len    > 0: the host bound on n_i to check; 0: not checked
 *   params       NULL: only q_start (and max_q_len) are checked, as the
 *                acceptance calls use it.  Otherwise the attention layer's
 *                shape (num_seqs must agree; block_size 16), and:
 *   max_seq_len  host bound on S_i
 *   seq_lens     [num_seqs] int32, required with params
 *   block_tables [num_seqs][max_blocks_per_seq] int32 or NULL (ids unchecked)
 *   counts       int32[VERIFY_CHECK_COUNTS] on the device, reset and written
 *                by the call (asynchronously, on `stream`):
 *     [VERIFY_CHECK_ROWS]     requests i whose q_start[i] < 0,
 *                             q_start[i + 1] < q_start[i] or > total_q, with
 *                             q_start[0] != 0 or q_start[num_seqs] != total_q
 *                             counted against the first or last request
 *     [VERIFY_CHECK_QLEN]     requests with n_i > max_q_len
 *     [VERIFY_CHECK_SHORT]    requests with S_i < n_i (rows without keys)
 *     [VERIFY_CHECK_LONG]     requests with S_i > max_seq_len or
 *                             S_i > 16 * max_blocks_per_seq
 *     [VERIFY_CHECK_BLOCK_ID] requests with a block id outside
 *                             [0, num_blocks) among the blocks their rows can
 *                             read: positions [lo, min(S_i, 16 *
 *                             max_blocks_per_seq)), lo = 0 without a window,
 *                             else max(0, S_i - n_i - W + 1)
 *     [VERIFY_CHECK_FIRST]    the lowest offending request, INT32_MAX if none
 * VERIFY_EINVAL (nothing enqueued) on negative sizes, a NULL counts, a NULL
 * q_start with num_seqs > 0, seq_lens or block_tables without params, or
 * params that disagree with num_seqs.  The index arrays are read only within
 * their stated sizes, whatever they hold.
 */
#define VERIFY_CHECK_ROWS 0
#define VERIFY_CHECK_QLEN 1
#define VERIFY_CHECK_SHORT 2
#define VERIFY_CHECK_LONG 3
#define VERIFY_CHECK_BLOCK_ID 4
#define VERIFY_CHECK_FIRST 5
#define VERIFY_CHECK_COUNTS 6
int verify_check_batch(int32_t num_seqs, int32_t total_q, int32_t max_q_len,
                       const int32_t *q_start, const verify_attn_params *params,
                       int32_t max_seq_len, const int32_t *seq_lens,
                       const int32_t *block_tables, int32_t *counts, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char *verify_status_string(int status);

/* Library ABI version (major * 10000 + minor * 100 + patch). */
int verify_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* AGENTSPEC_VERIFY_H */
