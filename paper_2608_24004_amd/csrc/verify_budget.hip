// verify_budget.hip -- redundancy-aware draft budget (paper Sec. 4.2 and its
// pseudocode, Alg. 2): per-request draft lengths for the next verify step,
// and the verify step's batch descriptor built from them.
//
// Batches of at most 8 requests whose candidates fit 64 KiB run as one
// workgroup (budget_fused, one launch: the candidates staged in LDS, then both
// steps below); larger ones as two kernels on one stream, which spreads the
// scoring over one compute unit per request:
//   budget_score   one wavefront per request: groups the request's candidate
//                  continuations by first token, picks the most frequent
//                  prefix (largest group; longest common prefix, then smallest
//                  first token on ties), the candidate its drafts are copied
//                  from (the group's longest, lowest row on ties) and the
//                  consensus score g_i = (c_i / n_i) p(n_i), in double;
//   budget_assign  one workgroup for the batch: G = sum_i g_i in ascending i
//                  (the order fixes the rounding of every share), the draft
//                  lengths L_i = max(|CT_i*|, floor(B_t g_i / G)) capped at the
//                  source candidate, q_start by a prefix scan, then tokens and
//                  seq_lens.
#include "common.h"

namespace averify {
namespace {

constexpr int kAssignThreads = 1024;

__device__ __forceinline__ int wave_max_i32(int v) {
    for (int o = 1; o < kWave; o <<= 1) v = max(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ int wave_min_i32(int v) {
    for (int o = 1; o < kWave; o <<= 1) v = min(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ int clamp_len(int len, int max_len) { return min(max(len, 0), max_len); }

// Score of request i (one wavefront): candidate rows r0 .. r0 + n - 1, whose
// lengths and tokens come from len_of(r) and tok_at(r, k) (LDS or global).
// Writes score, agree, prefix_len and source of request i from lane 0.
//
// The candidates that share a first token form a group; the group's common
// prefix is the longest prefix all of its members start with, i.e. the
// minimum over members of each member's common prefix with any one fixed
// member.  With at most one candidate per lane (n <= 64), every lane compares
// its candidate with its group's lowest row only, four tokens at a time, and
// the group sizes and minima are gathered across lanes; larger candidate sets
// take each candidate against every member of its group in turn.
template <typename LenF, typename TokF>
__device__ __forceinline__ void score_request(int i, int r0, int n, LenF len_of, TokF tok_at,
                                              double g_min, int lane, double* score,
                                              int32_t* agree, int32_t* prefix_len,
                                              int32_t* source) {
    // Per candidate a: size c of its first-token group and l, the group's
    // common prefix; then the wavefront's choice below.
    int best_c = 0, best_l = 0, best_tok = INT32_MAX;
    if (n <= kWave) {
        const int a = lane;
        const bool in = a < n;
        const int la = in ? len_of(r0 + a) : 0;
        const bool valid = la > 0;
        const int t0 = valid ? tok_at(r0 + a, 0) : 0;
        // group size and lowest member (rows ascend with the lane)
        int c = 0, rep = a;
        for (int b = 0; b < n; ++b) {
            const int vb = __builtin_amdgcn_readlane((int)valid, b);
            const int tb = __builtin_amdgcn_readlane(t0, b);
            if (valid && vb && tb == t0) {
                ++c;
                rep = min(rep, b);
            }
        }
        // common prefix with the lowest member (at least the first token)
        const int lrep = __shfl(la, rep);
        const int m = min(la, lrep);
        int k = 1;
        if (valid) {
            const int ra = r0 + a, rr = r0 + rep;
            bool same = true;
            while (same && k < m) {
                int x[4], y[4];
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const int kk = min(k + d, m - 1);
                    x[d] = tok_at(ra, kk);
                    y[d] = tok_at(rr, kk);
                }
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    if (same && k < m && x[d] == y[d]) ++k;
                    else same = false;
                }
            }
        }
        const int lcp = valid ? k : 0;
        // the group's common prefix: the minimum over its members
        int l = la;
        for (int b = 0; b < n; ++b) {
            const int vb = __builtin_amdgcn_readlane((int)valid, b);
            const int tb = __builtin_amdgcn_readlane(t0, b);
            const int lb = __builtin_amdgcn_readlane(lcp, b);
            if (valid && vb && tb == t0) l = min(l, lb);
        }
        if (valid) {
            best_c = c;
            best_l = l;
            best_tok = t0;
        }
    } else {
        for (int a = lane; a < n; a += kWave) {
            const int ra = r0 + a;
            const int la = len_of(ra);
            if (la == 0) continue;
            const int t0 = tok_at(ra, 0);
            int c = 0, l = la;
            for (int b = 0; b < n; ++b) {
                const int rb = r0 + b;
                const int lb = len_of(rb);
                if (lb == 0 || tok_at(rb, 0) != t0) continue;
                ++c;
                const int m = min(l, lb);
                int k = 1;
                while (k < m && tok_at(ra, k) == tok_at(rb, k)) ++k;
                l = min(l, k);
            }
            if (c > best_c || (c == best_c && (l > best_l || (l == best_l && t0 < best_tok)))) {
                best_c = c;
                best_l = l;
                best_tok = t0;
            }
        }
    }
    // Wavefront choice: largest group, then longest prefix, then smallest token.
    const int c_max = wave_max_i32(best_c);
    const int l_max = wave_max_i32(best_c == c_max ? best_l : -1);
    const int tok = wave_min_i32(best_c == c_max && best_l == l_max ? best_tok : INT32_MAX);

    // Source: the group's longest candidate, the lowest row among equals.
    int src_len = -1, src_row = INT32_MAX;
    if (c_max > 0) {
        for (int b = lane; b < n; b += kWave) {
            const int rb = r0 + b;
            const int lb = len_of(rb);
            if (lb == 0 || tok_at(rb, 0) != tok) continue;
            if (lb > src_len) {  // rows ascend within a lane: the first of a length wins
                src_len = lb;
                src_row = rb;
            }
        }
    }
    const int len_max = wave_max_i32(src_len);
    const int row = wave_min_i32(src_len == len_max && len_max >= 0 ? src_row : INT32_MAX);

    if (lane == 0) {
        if (c_max == 0) {
            score[i] = 0.0;
            agree[i] = 0;
            prefix_len[i] = 0;
            source[i] = -1;
        } else {
            const double p = g_min + (1.0 - g_min) * (1.0 - exp(1.0 - (double)n));
            score[i] = ((double)c_max / (double)n) * p;
            agree[i] = c_max;
            prefix_len[i] = l_max;
            source[i] = row;
        }
    }
}

// Candidate rows of request i, clamped to the candidate array.
__device__ __forceinline__ void request_rows(const int32_t* __restrict__ cand_start, int num_cands,
                                             int i, int& r0, int& n) {
    r0 = min(max(cand_start[i], 0), num_cands);
    n = min(max(cand_start[i + 1], r0), num_cands) - r0;
}

__global__ __launch_bounds__(kWave) void budget_score(
    int num_cands, int max_len, const int32_t* __restrict__ cand_start,
    const int32_t* __restrict__ cand_len, const int32_t* __restrict__ cand_tokens, double g_min,
    double* __restrict__ score, int32_t* __restrict__ agree, int32_t* __restrict__ prefix_len,
    int32_t* __restrict__ source) {
    const int i = blockIdx.x;
    int r0, n;
    request_rows(cand_start, num_cands, i, r0, n);
    score_request(
        i, r0, n, [&](int r) { return clamp_len(cand_len[r], max_len); },
        [&](int r, int k) { return cand_tokens[(int64_t)r * max_len + k]; }, g_min, threadIdx.x,
        score, agree, prefix_len, source);
}

// Draft lengths, q_start, tokens and seq_lens of the batch (one workgroup of
// kAssignThreads; every thread calls it).  G = sum_i g_i in ascending i fixes
// the rounding of every share.  Candidate tokens come from tok_at(row, k)
// (LDS or global); the drafts of each round of requests are copied by the
// whole workgroup, one (request, position) per thread.
template <typename TokF>
__device__ __forceinline__ void assign_batch(
    int num_seqs, int max_len, const int32_t* __restrict__ cand_len, TokF tok_at,
    const int32_t* __restrict__ last_token,
    const int32_t* __restrict__ ctx_len, double alpha, const double* score,
    const int32_t* prefix_len, const int32_t* source, int32_t* __restrict__ draft_len,
    int32_t* __restrict__ q_start, int32_t* __restrict__ tokens, int32_t* __restrict__ seq_lens) {
    __shared__ double G_s;
    __shared__ int wsum[kAssignThreads / kWave];
    __shared__ int carry_s;
    __shared__ int r_q0[kAssignThreads], r_len[kAssignThreads], r_src[kAssignThreads];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
    if (wv == 0) {
        // G in ascending i, as one sequential sum: wavefront 0 loads 64 scores
        // at a time and adds them in order from its registers
        double G = 0.0;
        for (int base = 0; base < num_seqs; base += kWave) {
            const double v = base + lane < num_seqs ? score[base + lane] : 0.0;
            const uint64_t bits = __double_as_longlong(v);
            const int cnt = min(kWave, num_seqs - base);
            for (int j = 0; j < cnt; ++j) {
                const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)bits, j);
                const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(bits >> 32), j);
                G += __longlong_as_double(((long long)hi << 32) | lo);
            }
        }
        if (lane == 0) {
            G_s = G;
            carry_s = 0;
            q_start[0] = 0;
        }
    }
    __syncthreads();
    const double G = G_s;
    const double bt = num_seqs > 0 ? floor(alpha / (double)num_seqs) : 0.0;
    for (int base = 0; base < num_seqs; base += kAssignThreads) {
        const int i = base + tid;
        int L = 0, src = -1;
        if (i < num_seqs) {
            src = source[i];
            if (src >= 0) {
                const double share = G > 0.0 ? floor((bt * score[i]) / G) : 0.0;
                const int cap = clamp_len(cand_len[src], max_len);
                L = prefix_len[i];
                if (share > (double)L) L = share >= (double)cap ? cap : (int)share;
                L = min(L, cap);
            }
            draft_len[i] = L;
        }
        // exclusive prefix of L + 1 over the chunk, continued from the carry
        const int u = i < num_seqs ? L + 1 : 0;
        int x = u;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane == kWave - 1) wsum[wv] = x;
        __syncthreads();
        if (wv == 0) {
            int s = lane < kAssignThreads / kWave ? wsum[lane] : 0;
#pragma unroll
            for (int o = 1; o < kAssignThreads / kWave; o <<= 1) {
                const int y = __shfl_up(s, o);
                if (lane >= o) s += y;
            }
            if (lane < kAssignThreads / kWave) wsum[lane] = s;
        }
        __syncthreads();
        const int q0 = carry_s + (wv > 0 ? wsum[wv - 1] : 0) + x - u;
        r_q0[tid] = q0;
        r_len[tid] = L;
        r_src[tid] = max(src, 0);
        if (i < num_seqs) {
            q_start[i + 1] = q0 + L + 1;
            tokens[q0] = last_token[i];
            if (ctx_len) seq_lens[i] = ctx_len[i] + L + 1;
        }
        __syncthreads();
        // the round's drafts: position j of request base + t
        const int nr = min(kAssignThreads, num_seqs - base);
        for (int e = tid; e < nr * max_len; e += kAssignThreads) {
            const int t = e / max_len, j = e - t * max_len;
            if (j < r_len[t]) tokens[r_q0[t] + 1 + j] = tok_at(r_src[t], j);
        }
        if (tid == kAssignThreads - 1) carry_s = q0 + u;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kAssignThreads) void budget_assign(
    int num_seqs, int max_len, const int32_t* __restrict__ cand_len,
    const int32_t* __restrict__ cand_tokens, const int32_t* __restrict__ last_token,
    const int32_t* __restrict__ ctx_len, double alpha, const double* __restrict__ score,
    const int32_t* __restrict__ prefix_len, const int32_t* __restrict__ source,
    int32_t* __restrict__ draft_len, int32_t* __restrict__ q_start, int32_t* __restrict__ tokens,
    int32_t* __restrict__ seq_lens) {
    assign_batch(num_seqs, max_len, cand_len,
                 [&](int r, int k) { return cand_tokens[(int64_t)r * max_len + k]; }, last_token,
                 ctx_len, alpha, score, prefix_len, source, draft_len, q_start, tokens, seq_lens);
}

// Batches whose candidates fit kFusedLdsBytes of LDS run as one workgroup:
// the candidates (lengths and tokens) are staged in LDS, each wavefront scores
// requests in turn, and the same workgroup assigns the budget, all in one
// launch (the call is latency-bound: the prefix comparisons are chains of
// dependent reads, which LDS answers far sooner than global memory).
constexpr size_t kFusedLdsBytes = 64 * 1024;
constexpr int kFusedMaxSeqs = 8;

size_t fused_lds_bytes(int num_cands, int max_len) {
    return (size_t)num_cands * ((size_t)max_len + 1) * sizeof(int32_t);
}

__global__ __launch_bounds__(kAssignThreads) void budget_fused(
    int num_seqs, int num_cands, int max_len, const int32_t* __restrict__ cand_start,
    const int32_t* __restrict__ cand_len, const int32_t* __restrict__ cand_tokens,
    const int32_t* __restrict__ last_token, const int32_t* __restrict__ ctx_len, double alpha,
    double g_min, double* __restrict__ score, int32_t* __restrict__ agree,
    int32_t* __restrict__ prefix_len, int32_t* __restrict__ source, int32_t* __restrict__ draft_len,
    int32_t* __restrict__ q_start, int32_t* __restrict__ tokens, int32_t* __restrict__ seq_lens) {
    extern __shared__ int32_t s_cands[];  // [num_cands] lengths, then [num_cands][max_len] tokens
    int32_t* s_len = s_cands;
    int32_t* s_tok = s_cands + num_cands;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
    for (int r = tid; r < num_cands; r += kAssignThreads) s_len[r] = clamp_len(cand_len[r], max_len);
    for (int e = tid; e < num_cands * max_len; e += kAssignThreads) s_tok[e] = cand_tokens[e];
    __syncthreads();
    for (int i = wv; i < num_seqs; i += kAssignThreads / kWave) {
        int r0, n;
        request_rows(cand_start, num_cands, i, r0, n);
        score_request(
            i, r0, n, [&](int r) { return s_len[r]; }, [&](int r, int k) { return s_tok[r * max_len + k]; },
            g_min, lane, score, agree, prefix_len, source);
    }
    __syncthreads();
    assign_batch(num_seqs, max_len, cand_len, [&](int r, int k) { return s_tok[r * max_len + k]; },
                 last_token, ctx_len, alpha, score, prefix_len, source, draft_len, q_start, tokens,
                 seq_lens);
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_budget(int32_t num_seqs, int32_t num_cands, int32_t max_cand_len,
                             const int32_t* cand_start, const int32_t* cand_len,
                             const int32_t* cand_tokens, const int32_t* last_token,
                             const int32_t* ctx_len, double alpha, double g_min, double* score,
                             int32_t* agree, int32_t* prefix_len, int32_t* source,
                             int32_t* draft_len, int32_t* q_start, int32_t* tokens,
                             int64_t tokens_capacity, int32_t* seq_lens, hipStream_t stream) {
    if (num_seqs < 0 || num_cands < 0 || max_cand_len < 0) return VERIFY_EINVAL;
    if (!(alpha >= 0.0) || !(alpha < 1e300) || !(g_min >= 0.0 && g_min <= 1.0)) return VERIFY_EINVAL;
    if (num_seqs > 0 && max_cand_len < 1) return VERIFY_EINVAL;
    if (tokens_capacity < (int64_t)num_seqs * ((int64_t)max_cand_len + 1)) return VERIFY_EINVAL;
    if ((int64_t)num_seqs * ((int64_t)max_cand_len + 1) >= ((int64_t)1 << 31)) return VERIFY_EUNSUPPORTED;
    if (!q_start) return VERIFY_EINVAL;
    if (num_seqs > 0 && (!cand_start || !last_token || !score || !agree || !prefix_len || !source ||
                         !draft_len || !tokens))
        return VERIFY_EINVAL;
    if (num_cands > 0 && (!cand_len || !cand_tokens)) return VERIFY_EINVAL;
    if ((ctx_len == nullptr) != (seq_lens == nullptr)) return VERIFY_EINVAL;
    const size_t lds = fused_lds_bytes(num_cands, max_cand_len);
    // One workgroup scores every request on one compute unit; beyond a few
    // requests, one workgroup per request on as many compute units (plus a
    // second launch) is faster: 10.1 vs 16.5 us at 32 requests.
    if (lds <= kFusedLdsBytes && num_seqs <= kFusedMaxSeqs) {
        hipLaunchKernelGGL(budget_fused, dim3(1), dim3(kAssignThreads), lds, stream, num_seqs,
                           num_cands, max_cand_len, cand_start, cand_len, cand_tokens, last_token,
                           ctx_len, alpha, g_min, score, agree, prefix_len, source, draft_len,
                           q_start, tokens, seq_lens);
        return check_launch();
    }
    // an empty batch still gets its descriptor, q_start[0] = 0, from budget_assign
    if (num_seqs > 0)
        hipLaunchKernelGGL(budget_score, dim3((unsigned)num_seqs), dim3(kWave), 0, stream, num_cands,
                           max_cand_len, cand_start, cand_len, cand_tokens, g_min, score, agree,
                           prefix_len, source);
    hipLaunchKernelGGL(budget_assign, dim3(1), dim3(kAssignThreads), 0, stream, num_seqs,
                       max_cand_len, cand_len, cand_tokens, last_token, ctx_len, alpha, score,
                       prefix_len, source, draft_len, q_start, tokens, seq_lens);
    return check_launch();
}
