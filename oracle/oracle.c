/*
 * oracle.c -- CPU oracle for the batched speculative-verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark load it.  It shares no code, header, table or helper with the
 * HIP library: the paged-cache layout, the bf16 decoding, the masks and the
 * acceptance rule are all written out again here from their definitions.
 *
 * What it computes (paper: Sec. 2.2 states that speculative decoding proposes
 * several tokens and verifies them with the target model in one pass, and that
 * the result is identical to plain decoding; Sec. 3.1 defines the rejection
 * rate as rejected over proposed drafts per request):
 *
 *   oracle_attention  -- for each requested (query row, query head) pair, the
 *                        plain definition of causal softmax attention of that
 *                        row against its request's paged KV cache, in double
 *                        precision, keys visited in ascending position order.
 *   oracle_kv_append  -- the new tokens' K/V written into their cache slots.
 *   oracle_argmax     -- per logits row, the lowest index attaining the maximum
 *                        (plus the gap to the runner-up, for near-tie flags).
 *   oracle_lmhead_argmax -- the logits of selected rows from the final hidden
 *                        states and the LM-head weight (a plain dot product
 *                        per vocabulary entry), then oracle_argmax's rule.
 *   oracle_sample     -- each row's token drawn from softmax(logits / T) by the
 *                        Gumbel-max rule (Philox4x32-10 noise), the stochastic
 *                        verification's replacement for the argmax.
 *   oracle_accept     -- greedy acceptance: the longest prefix of drafts equal
 *                        to the target's argmax, followed by one bonus token.
 *   oracle_budget     -- redundancy-aware draft budget (Sec. 4.2, Alg. 2): the
 *                        per-request draft lengths and the verify step's
 *                        batch descriptor built from them.
 *
 * Readings of the paper that this file encodes (the paper relies on its
 * serving engine for verification and does not spell these out):
 *   - acceptance is greedy (argmax); ties in the argmax go to the lowest index;
 *     a NaN anywhere in a row makes the first NaN the argmax; -0.0 == +0.0;
 *   - query row j of a request with n scored positions and S cached keys sits
 *     at absolute position p = S - n + j and sees keys t <= p (bottom-right
 *     aligned causal mask inside the draft);
 *   - a sliding window W > 0 keeps keys with p - W < t <= p;
 *   - query head h reads KV head floor(h / (Hq / Hkv)) (grouped-query);
 *   - scale defaults to 1/sqrt(head_dim); no soft-cap, no bias; attention
 *     sinks only when given (see oracle_attention);
 *   - a row with no visible key (only possible when S < n) yields zeros;
 *   - a key whose block id lies outside [0, num_blocks) is not a key at all:
 *     it takes no part in the softmax (the library's convention for unmapped
 *     block-table entries), and a row left without keys yields zeros.
 *
 * Paged KV layout read here (element index, x = 16 bytes / element size):
 *   K: [num_blocks][Hkv][D/x][16][x]   -> K[t][d] of physical block b, head g
 *      is k_cache[(((b*Hkv + g)*(D/x) + d/x)*16 + t%16)*x + d%x]
 *   V: [num_blocks][Hkv][D][16]        -> V[t][d] = v_cache[((b*Hkv + g)*D + d)*16 + t%16]
 *   b = block_tables[i*max_blocks_per_seq + t/16].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_F32 0
#define ORACLE_BF16 1

static double elem_to_double(const void *base, int dtype, int64_t idx)
{
    if (dtype == ORACLE_F32) {
        return (double)((const float *)base)[idx];
    }
    /* bfloat16 is the upper half of an IEEE binary32 word. */
    uint32_t bits = (uint32_t)((const uint16_t *)base)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int elem_size(int dtype) { return dtype == ORACLE_F32 ? 4 : 2; }

/* Request owning global query row `row` (q_start is an exclusive prefix sum). */
static int find_request(int num_seqs, const int32_t *q_start, int32_t row)
{
    for (int i = 0; i < num_seqs; ++i)
        if (row >= q_start[i] && row < q_start[i + 1]) return i;
    return -1;
}

/*
 * out[pair][d] = sum_t w_t V_t[d] / sum_t w_t,  w_t = exp(s_t - max_u s_u),
 * s_t = scale * <q_row_head, K_t>,  t over the visible keys of the row.
 * With sinks (one logit per query head, in the units of s_t; NULL for none)
 * the head's sink joins the softmax as a logit whose value is zero: it adds
 * exp(sink - max) to the denominator only (the attention sinks of the
 * GPT-OSS models the paper serves; the paper itself does not describe them).
 * Returns 0, or -1 on an argument that cannot be interpreted.
 */
int oracle_attention(int32_t num_seqs, int32_t num_q_heads, int32_t num_kv_heads,
                     int32_t head_dim, int32_t max_blocks_per_seq, int32_t num_blocks,
                     int32_t sliding_window,
                     double scale, int32_t dtype, const void *q, const void *k_cache,
                     const void *v_cache, const int32_t *block_tables,
                     const int32_t *seq_lens, const int32_t *q_start, int64_t n_pairs,
                     const int32_t *pair_row, const int32_t *pair_head, const double *sinks,
                     double *out)
{
    const int D = head_dim;
    if (num_q_heads % num_kv_heads != 0) return -1;
    const int group = num_q_heads / num_kv_heads;
    const int x = 16 / elem_size(dtype);
    if (D % x != 0) return -1;
    if (scale == 0.0) scale = 1.0 / sqrt((double)D);
    int bad = 0;

#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
    for (int64_t pr = 0; pr < n_pairs; ++pr) {
        const int32_t row = pair_row[pr];
        const int32_t h = pair_head[pr];
        double *o = out + pr * D;
        for (int d = 0; d < D; ++d) o[d] = 0.0;
        const int i = find_request(num_seqs, q_start, row);
        if (i < 0 || h < 0 || h >= num_q_heads) { bad = 1; continue; }
        const int64_t n = q_start[i + 1] - q_start[i];
        const int64_t S = seq_lens[i];
        const int64_t j = row - q_start[i];
        const int64_t p = S - n + j; /* absolute position of this query row */
        int64_t lo = 0;
        if (sliding_window > 0 && p - sliding_window + 1 > lo) lo = p - sliding_window + 1;
        if (p < lo || p < 0) continue; /* nothing visible: output stays zero */
        const int g = h / group;

        const int64_t nkeys = p - lo + 1;
        double *s = (double *)malloc(sizeof(double) * nkeys);
        if (!s) { bad = 1; continue; }
        double smax = -INFINITY;
        for (int64_t t = lo; t <= p; ++t) {
            const int64_t b = block_tables[(int64_t)i * max_blocks_per_seq + t / 16];
            if (b < 0 || b >= num_blocks) { s[t - lo] = -INFINITY; continue; } /* no key */
            double acc = 0.0;
            for (int d = 0; d < D; ++d) {
                const double qd = elem_to_double(q, dtype, ((int64_t)row * num_q_heads + h) * D + d);
                const int64_t kidx =
                    ((((int64_t)b * num_kv_heads + g) * (D / x) + d / x) * 16 + t % 16) * x + d % x;
                acc += qd * elem_to_double(k_cache, dtype, kidx);
            }
            s[t - lo] = scale * acc;
            if (s[t - lo] > smax) smax = s[t - lo];
        }
        /* an attention sink is one more logit in the softmax, with no value */
        const double sink = sinks ? sinks[h] : -INFINITY;
        if (sink > smax) smax = sink;
        double denom = sinks ? exp(sink - smax) : 0.0;
        if (smax == -INFINITY) { free(s); continue; } /* no key and no sink: zeros */
        for (int64_t t = lo; t <= p; ++t) {
            const int64_t b = block_tables[(int64_t)i * max_blocks_per_seq + t / 16];
            if (b < 0 || b >= num_blocks) continue;
            const double w = exp(s[t - lo] - smax);
            denom += w;
            for (int d = 0; d < D; ++d) {
                const int64_t vidx = (((int64_t)b * num_kv_heads + g) * D + d) * 16 + t % 16;
                o[d] += w * elem_to_double(v_cache, dtype, vidx);
            }
        }
        for (int d = 0; d < D; ++d) o[d] /= denom;
        free(s);
    }
    return bad ? -1 : 0;
}

/*
 * argmax[r] = min { v : x[r][v] = max_u x[r][u] }  (first NaN if the row has
 * one).  gap[r] = x[r][argmax] - max_{v != argmax} x[r][v]  (+inf for vocab 1,
 * NaN if the row holds a NaN).  gap may be NULL.
 */
int oracle_argmax(int64_t rows, int64_t vocab, int64_t row_stride, int32_t dtype,
                  const void *logits, int32_t *argmax, double *gap)
{
    if (vocab <= 0) return -1;
    if (row_stride == 0) row_stride = vocab;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t base = r * row_stride;
        int64_t best = 0;
        double bestv = elem_to_double(logits, dtype, base);
        int has_nan = isnan(bestv);
        for (int64_t v = 1; v < vocab && !has_nan; ++v) {
            const double x = elem_to_double(logits, dtype, base + v);
            if (isnan(x)) { best = v; bestv = x; has_nan = 1; break; }
            if (x > bestv) { best = v; bestv = x; }
        }
        argmax[r] = (int32_t)best;
        if (gap) {
            if (has_nan) { gap[r] = NAN; continue; }
            double second = -INFINITY;
            for (int64_t v = 0; v < vocab; ++v) {
                if (v == best) continue;
                const double x = elem_to_double(logits, dtype, base + v);
                if (x > second) second = x;
            }
            gap[r] = vocab == 1 ? INFINITY : bestv - second;
        }
    }
    return 0;
}

/*
 * The verify pass ends with the LM head: logits[r][v] = <hidden[r], weight[v]>,
 * hidden [rows][H] and weight [vocab][H] (the usual lm_head layout), both in
 * `dtype`.  The products of the exact inputs are summed in double, h
 * ascending, and the row's argmax follows oracle_argmax (lowest index among
 * equal maxima, the first NaN if any, -0.0 == +0.0), with the gap to the
 * runner-up (NaN for a NaN row, +inf when vocab = 1).  Only the n_sel rows
 * listed in sel_rows are computed; argmax, gap and (if not NULL) logits
 * [n_sel][vocab] receive them in that order.  Returns 0, or -1 on bad sizes.
 */
int oracle_lmhead_argmax(int64_t n_sel, const int32_t *sel_rows, int32_t hidden, int64_t vocab,
                         int32_t dtype, const void *hid, const void *weight, int32_t *argmax,
                         double *gap, double *logits)
{
    if (vocab <= 0 || hidden <= 0) return -1;
    double *row = (double *)malloc(sizeof(double) * vocab);
    if (!row) return -1;
    for (int64_t s = 0; s < n_sel; ++s) {
        const int64_t r = sel_rows[s];
#pragma omp parallel for schedule(static)
        for (int64_t v = 0; v < vocab; ++v) {
            double acc = 0.0;
            for (int32_t h = 0; h < hidden; ++h)
                acc += elem_to_double(hid, dtype, r * hidden + h) *
                       elem_to_double(weight, dtype, v * hidden + h);
            row[v] = acc;
        }
        int64_t best = 0;
        int has_nan = isnan(row[0]);
        for (int64_t v = 1; v < vocab && !has_nan; ++v) {
            if (isnan(row[v])) { best = v; has_nan = 1; }
            else if (row[v] > row[best]) best = v;
        }
        argmax[s] = (int32_t)best;
        if (gap) {
            double second = -INFINITY;
            for (int64_t v = 0; v < vocab; ++v)
                if (v != best && row[v] > second) second = row[v];
            gap[s] = has_nan ? NAN : (vocab == 1 ? INFINITY : row[best] - second);
        }
        if (logits) memcpy(logits + s * vocab, row, sizeof(double) * vocab);
    }
    free(row);
    return 0;
}

/*
 * Stochastic verification (temperature T > 0).  With drafts that put all of
 * their probability on one token (the suffix / n-gram style drafts of Sec. 2.2
 * and 4.1), speculative rejection sampling accepts draft d with probability
 * p(d) and, on a rejection, draws from p with d's mass removed; sampling
 * y ~ p = softmax(logits / T) and accepting iff y == d (emitting y otherwise)
 * does exactly that.  So the stochastic step is the greedy one with each row's
 * argmax replaced by a sample, drawn by the Gumbel-max rule
 *     y = argmax_v ( x_v / T + g_v ),   g_v = -log(-log(u_v)),  u_v ~ U(0, 1),
 * ties to the lowest index, a NaN logit maximal (as in oracle_argmax).
 *
 * u_v comes from Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): key
 * (seed low word, seed high word), counter (v / 4, row, offset, 0), output word
 * v % 4, mapped to u = ((w >> 9) + 0.5) * 2^-23 = (2 (w >> 9) + 1) * 2^-24: the top
 * 23 bits, so that u is an odd multiple of 2^-24 that fp32 holds exactly, in
 * [2^-24, 1 - 2^-24].  (With 24 bits the sum (w >> 8) + 0.5 needs 25
 * significant bits and rounds, and the top code would give u = 1 and an
 * unbounded noise term.)  The score is computed in fp32
 * as fmaf(x, inv_temperature, g) with g from sample_log below, so that an
 * implementation making the same fp32 operations draws the same tokens.
 */
static void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        c0 = hi1 ^ c1 ^ k0;
        c1 = lo1;
        c2 = hi0 ^ c3 ^ k1;
        c3 = lo0;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Natural log in fp32 for x > 0 normal: x = m 2^e with m in [sqrt(1/2), sqrt(2)),
 * log x = e ln 2 + 2 atanh(z), z = (m - 1) / (m + 1), the atanh series to z^9
 * (|z| <= 0.1716, truncation below 1e-9). */
static float sample_log(float x)
{
    uint32_t bits;
    memcpy(&bits, &x, 4);
    int e = (int)((bits >> 23) & 0xFF) - 127;
    uint32_t mb = (bits & 0x7FFFFFu) | 0x3F800000u;
    float m;
    memcpy(&m, &mb, 4);
    if (m > 1.41421354f) { m = m * 0.5f; e += 1; }
    const float z = (m - 1.0f) / (m + 1.0f);
    const float z2 = z * z;
    float poly = fmaf(z2, 0.111111112f, 0.142857149f);
    poly = fmaf(z2, poly, 0.200000003f);
    poly = fmaf(z2, poly, 0.333333343f);
    poly = fmaf(z2, poly, 1.0f);
    const float r = 2.0f * z * poly;
    return fmaf((float)e, 0.693147182f, r);
}

static float sample_uniform(uint32_t w) { return ((float)(w >> 9) + 0.5f) * 0x1p-23f; }

static float gumbel_noise(uint64_t seed, uint32_t offset, int64_t row, int64_t v)
{
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    const uint32_t ctr[4] = {(uint32_t)(v >> 2), (uint32_t)row, offset, 0u};
    uint32_t out[4];
    philox4x32_10(ctr, key, out);
    const float u = sample_uniform(out[v & 3]);
    return -sample_log(-sample_log(u));
}

/* Test hooks for the generator and the log: the raw Philox block, sample_log
 * applied elementwise, and the noise term g of a raw Philox output word. */
void oracle_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out)
{
    philox4x32_10(ctr, key, out);
}

void oracle_sample_log(int64_t n, const float *x, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = sample_log(x[i]);
}

void oracle_gumbel_of_word(int64_t n, const uint32_t *w, float *u, float *g)
{
    for (int64_t i = 0; i < n; ++i) {
        u[i] = sample_uniform(w[i]);
        g[i] = -sample_log(-sample_log(u[i]));
    }
}

int oracle_sample(int64_t rows, int64_t vocab, int64_t row_stride, int32_t dtype,
                  const void *logits, float inv_temperature, uint64_t seed, uint32_t offset,
                  int32_t *sampled)
{
    if (vocab <= 0 || vocab > 0x7fffffff || !(inv_temperature > 0.0f)) return -1;
    if (row_stride == 0) row_stride = vocab;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t base = r * row_stride;
        int64_t best = 0;
        float bestv = 0.0f;
        for (int64_t v = 0; v < vocab; ++v) {
            const float x = (float)elem_to_double(logits, dtype, base + v);
            if (isnan(x)) { best = v; break; }
            const float sc = fmaf(x, inv_temperature, gumbel_noise(seed, offset, r, v));
            if (v == 0 || sc > bestv) { best = v; bestv = sc; }
        }
        sampled[r] = (int32_t)best;
    }
    return 0;
}

/*
 * Greedy acceptance.  Request i owns rows q_start[i] .. q_start[i+1]-1
 * (n_i = k_i + 1 rows).  tokens[q_start[i]] is the last committed token and
 * tokens[q_start[i] + j] (1 <= j <= k_i) is draft j.  Row j's argmax is the
 * target's prediction for the token after row j's input, so draft j+1 is
 * accepted while argmax[q_start[i] + j] == tokens[q_start[i] + j + 1].
 *   accept_len[i]  = m_i, the number of leading accepted drafts (0..k_i);
 *   num_emitted[i] = m_i + 1 (accepted drafts plus the bonus token), or 0 for
 *                    a request with no rows;
 *   emitted[q_start[i] + j] = draft j+1 for j < m_i, argmax of row m_i for
 *                    j = m_i, and -1 for the remaining rows of the request.
 */
int oracle_accept(int32_t num_seqs, const int32_t *q_start, const int32_t *tokens,
                  const int32_t *argmax, int32_t *accept_len, int32_t *num_emitted,
                  int32_t *emitted)
{
    for (int i = 0; i < num_seqs; ++i) {
        const int32_t q0 = q_start[i];
        const int32_t n = q_start[i + 1] - q0;
        if (n <= 0) { accept_len[i] = 0; num_emitted[i] = 0; continue; }
        const int32_t k = n - 1;
        int32_t m = 0;
        while (m < k && argmax[q0 + m] == tokens[q0 + m + 1]) ++m;
        for (int32_t j = 0; j < n; ++j)
            emitted[q0 + j] = j < m ? tokens[q0 + j + 1] : (j == m ? argmax[q0 + m] : -1);
        accept_len[i] = m;
        num_emitted[i] = m + 1;
    }
    return 0;
}

/*
 * KV append: the K and V of the verify step's new tokens go into the paged
 * cache before attention reads them.  Row j of request i is the token at
 * position p = S_i - n_i + j; its K/V for KV head g land in slot p % 16 of
 * physical block block_tables[i][p / 16] (layouts as in oracle_attention).
 * k_new, v_new: [total_q][num_kv_heads][head_dim] in the cache's dtype.  Rows
 * whose position is negative or whose block id lies outside [0, num_blocks)
 * are skipped.  Element bits are copied unchanged.
 */
int oracle_kv_append(int32_t num_seqs, int32_t num_kv_heads, int32_t head_dim,
                     int32_t max_blocks_per_seq, int32_t num_blocks, int32_t dtype,
                     const void *k_new, const void *v_new, const int32_t *block_tables,
                     const int32_t *seq_lens, const int32_t *q_start, void *k_cache,
                     void *v_cache)
{
    const int D = head_dim, e = elem_size(dtype), x = 16 / e;
    if (D % x != 0) return -1;
    for (int i = 0; i < num_seqs; ++i) {
        const int64_t n = q_start[i + 1] - q_start[i];
        for (int64_t j = 0; j < n; ++j) {
            const int64_t row = q_start[i] + j;
            const int64_t p = (int64_t)seq_lens[i] - n + j;
            if (p < 0 || p / 16 >= max_blocks_per_seq) continue;
            const int64_t b = block_tables[(int64_t)i * max_blocks_per_seq + p / 16];
            if (b < 0 || b >= num_blocks) continue;
            for (int g = 0; g < num_kv_heads; ++g)
                for (int d = 0; d < D; ++d) {
                    const int64_t src = (row * num_kv_heads + g) * D + d;
                    const int64_t kidx = (((b * num_kv_heads + g) * (D / x) + d / x) * 16 + p % 16) * x + d % x;
                    const int64_t vidx = ((b * num_kv_heads + g) * D + d) * 16 + p % 16;
                    memcpy((char *)k_cache + kidx * e, (const char *)k_new + src * e, e);
                    memcpy((char *)v_cache + vidx * e, (const char *)v_new + src * e, e);
                }
        }
    }
    return 0;
}

/*
 * Redundancy-aware budget allocation (Sec. 4.2 and its pseudocode, Alg. 2):
 * the per-request draft lengths L_i of the next verify step, and the verify
 * step's batch descriptor built from them.
 *
 * Inputs.  Request i owns candidate continuations cand_start[i] ..
 * cand_start[i+1]-1, rows of cand_tokens [C][max_len] with cand_len[r] valid
 * tokens each; last_token[i] is its last committed token; ctx_len (nullable)
 * its cached context length.  alpha and g_min are the method's two
 * hyperparameters.
 *
 * Readings of the paper (it leaves these open):
 *   - n_i counts every candidate of the request, empty ones included;
 *   - the most frequent continuation prefix CT_i* is the non-empty prefix that
 *     the most candidates start with; among equally frequent ones the longest,
 *     then the lexicographically smallest; c_i is the number of candidates
 *     starting with it (0, and g_i = 0, when every candidate is empty);
 *   - p(n) = g_min + (1 - g_min)(1 - e^(1-n)): the equation's form, the one
 *     that gives p(1) = g_min, the minimum confidence under the least support
 *     (the pseudocode's exponent -n does not);
 *   - B_t = floor(alpha / bz) with bz = num_seqs; G = sum_i g_i in ascending i;
 *   - L_i = max(|CT_i*|, floor((B_t * g_i) / G)), the share being 0 when G = 0,
 *     and at most the length of the longest candidate starting with CT_i*
 *     (the lowest row among equals): its first L_i tokens are the drafts.
 *
 * Outputs: score g_i, agree c_i, prefix_len |CT_i*|, source (that candidate's
 * row, -1 if none), draft_len L_i; q_start[num_seqs+1] (exclusive prefix sum
 * of L_i + 1), tokens (per request: last_token, then the L_i drafts) and, if
 * ctx_len is given, seq_lens = ctx_len + L_i + 1.
 */
static int common_prefix(const int32_t *a, int32_t la, const int32_t *b, int32_t lb)
{
    int32_t m = la < lb ? la : lb, k = 0;
    while (k < m && a[k] == b[k]) ++k;
    return k;
}

int oracle_budget(int32_t num_seqs, int32_t max_len, const int32_t *cand_start,
                  const int32_t *cand_len, const int32_t *cand_tokens,
                  const int32_t *last_token, const int32_t *ctx_len, double alpha,
                  double g_min, double *score, int32_t *agree, int32_t *prefix_len,
                  int32_t *source, int32_t *draft_len, int32_t *q_start, int32_t *tokens,
                  int32_t *seq_lens)
{
    if (num_seqs < 0 || max_len < 0 || !(alpha >= 0.0) || !(g_min >= 0.0 && g_min <= 1.0))
        return -1;
    q_start[0] = 0;
    if (num_seqs == 0) return 0;
    const double bt = floor(alpha / (double)num_seqs);
    double G = 0.0;
    for (int i = 0; i < num_seqs; ++i) {
        const int32_t r0 = cand_start[i], n = cand_start[i + 1] - r0;
        score[i] = 0.0; agree[i] = 0; prefix_len[i] = 0; source[i] = -1;
        /* Every non-empty prefix of every candidate, counted by its definition:
         * prefix (a, l) -- the first l tokens of candidate a -- is shared by
         * the candidates b whose common prefix with a is at least l tokens.
         * The most frequent prefix wins; equally frequent ones go to the
         * longer, then to the lexicographically smaller token sequence. */
        int32_t best_c = 0, best_l = 0, best_row = -1;
        for (int32_t a = 0; a < n; ++a) {
            const int32_t ra = r0 + a, la = cand_len[ra];
            if (la <= 0) continue;
            const int32_t *ta = cand_tokens + (int64_t)ra * max_len;
            for (int32_t l = 1; l <= la; ++l) {
                int32_t c = 0;
                for (int32_t b = 0; b < n; ++b) {
                    const int32_t rb = r0 + b;
                    if (cand_len[rb] < l) continue;
                    if (common_prefix(ta, l, cand_tokens + (int64_t)rb * max_len, l) == l) ++c;
                }
                int better = c > best_c || (c == best_c && l > best_l);
                if (!better && c == best_c && l == best_l && best_row >= 0) {
                    const int32_t *tb = cand_tokens + (int64_t)best_row * max_len;
                    int32_t k = 0;
                    while (k < l && ta[k] == tb[k]) ++k;
                    better = k < l && ta[k] < tb[k];
                }
                if (better) { best_c = c; best_l = l; best_row = ra; }
            }
        }
        if (best_c == 0) continue;
        /* drafts come from the longest candidate starting with the prefix
         * (lowest row on ties) */
        const int32_t *pref = cand_tokens + (int64_t)best_row * max_len;
        int32_t src = -1;
        for (int32_t b = 0; b < n; ++b) {
            const int32_t rb = r0 + b;
            if (cand_len[rb] < best_l) continue;
            if (common_prefix(pref, best_l, cand_tokens + (int64_t)rb * max_len, best_l) != best_l)
                continue;
            if (src < 0 || cand_len[rb] > cand_len[src]) src = rb;
        }
        const double p = g_min + (1.0 - g_min) * (1.0 - exp(1.0 - (double)n));
        score[i] = ((double)best_c / (double)n) * p;
        agree[i] = best_c;
        prefix_len[i] = best_l;
        source[i] = src;
    }
    for (int i = 0; i < num_seqs; ++i) G += score[i];
    for (int i = 0; i < num_seqs; ++i) {
        int64_t L = 0;
        if (source[i] >= 0) {
            const double share = G > 0.0 ? floor((bt * score[i]) / G) : 0.0;
            L = prefix_len[i];
            if (share > (double)L) L = (int64_t)share;
            if (L > cand_len[source[i]]) L = cand_len[source[i]];
        }
        draft_len[i] = (int32_t)L;
        q_start[i + 1] = q_start[i] + (int32_t)L + 1;
        tokens[q_start[i]] = last_token[i];
        for (int64_t j = 0; j < L; ++j)
            tokens[q_start[i] + 1 + j] = cand_tokens[(int64_t)source[i] * max_len + j];
        if (ctx_len) seq_lens[i] = ctx_len[i] + (int32_t)L + 1;
    }
    return 0;
}

int oracle_num_threads(void)
{
    int n = 1;
#ifdef _OPENMP
#pragma omp parallel
    {
#pragma omp master
        n = omp_get_num_threads();
    }
#endif
    return n;
}
