// verify_check.hip -- device-side validation of a verify batch's descriptor
// (q_start, seq_lens, block_tables) against the preconditions the other
// calls state.  Those calls never read device data on the host and define
// what they do with ids outside the cache (skip them); this call reports such
// data instead, for callers that want to catch a bad batch before it runs.
//
// One workgroup per request (grid-strided): thread 0 tests the request's
// scalars, all threads test the block ids the request's rows can read, and a
// workgroup-wide OR joins them.  Offending requests are counted with global
// atomics into the caller's counts array, which a one-wave kernel resets
// first on the same stream.
#include <climits>

#include "common.h"

namespace averify {
namespace {

constexpr int kCheckThreads = 256;
constexpr int kCheckMaxWorkgroups = 4096;

struct CArgs {
    int num_seqs, total_q, max_q_len, max_seq_len, max_blocks, num_blocks, window;
};

__global__ __launch_bounds__(kWave) void check_reset(int32_t* __restrict__ counts) {
    const int t = threadIdx.x;
    if (t < VERIFY_CHECK_COUNTS) counts[t] = t == VERIFY_CHECK_FIRST ? INT32_MAX : 0;
}

__global__ __launch_bounds__(kCheckThreads) void check_batch(CArgs a, const int32_t* __restrict__ q_start,
                                                             const int32_t* __restrict__ seq_lens,
                                                             const int32_t* __restrict__ block_tables,
                                                             int32_t* __restrict__ counts) {
    for (int i = blockIdx.x; i < a.num_seqs; i += gridDim.x) {
        const int q0 = q_start[i], q1 = q_start[i + 1];
        const bool bad_rows = q0 < 0 || q1 < q0 || q1 > a.total_q || (i == 0 && q0 != 0) ||
                              (i == a.num_seqs - 1 && q1 != a.total_q);
        const int64_t n = q1 >= q0 ? (int64_t)q1 - q0 : 0;
        const bool bad_qlen = a.max_q_len > 0 && n > a.max_q_len;
        bool short_seq = false, long_seq = false;
        int bad_id = 0;
        if (seq_lens) {
            const int S = seq_lens[i];
            const int64_t cap = (int64_t)kBlockTokens * a.max_blocks;
            short_seq = S < n;
            long_seq = S > a.max_seq_len || S > cap;
            if (block_tables) {
                // keys the request's rows can see: up to position S - 1, from
                // the first row's window start (0 without a window)
                const int64_t hi = std::min<int64_t>(std::max(S, 0), cap);
                const int64_t lo = a.window > 0 ? std::max<int64_t>(0, hi - n - a.window + 1) : 0;
                const int32_t* row = block_tables + (int64_t)i * a.max_blocks;
                for (int64_t b = lo / kBlockTokens + threadIdx.x; b < (hi + kBlockTokens - 1) / kBlockTokens;
                     b += kCheckThreads) {
                    const int id = row[b];
                    bad_id |= id < 0 || id >= a.num_blocks;
                }
            }
        }
        const bool any_bad_id = __syncthreads_or(bad_id) != 0;
        if (threadIdx.x == 0) {
            const bool flag[VERIFY_CHECK_FIRST] = {bad_rows, bad_qlen, short_seq, long_seq, any_bad_id};
            bool any = false;
            for (int k = 0; k < VERIFY_CHECK_FIRST; ++k)
                if (flag[k]) {
                    atomicAdd(&counts[k], 1);
                    any = true;
                }
            if (any) atomicMin(&counts[VERIFY_CHECK_FIRST], i);
        }
    }
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_check_batch(int32_t num_seqs, int32_t total_q, int32_t max_q_len,
                                  const int32_t* q_start, const verify_attn_params* params,
                                  int32_t max_seq_len, const int32_t* seq_lens,
                                  const int32_t* block_tables, int32_t* counts, hipStream_t stream) {
    if (num_seqs < 0 || total_q < 0 || max_q_len < 0 || !counts) return VERIFY_EINVAL;
    if (num_seqs > 0 && !q_start) return VERIFY_EINVAL;
    if (params) {
        if (params->num_seqs != num_seqs || params->block_size != kBlockTokens ||
            params->max_blocks_per_seq <= 0 || params->num_blocks < 0 || params->sliding_window < 0 ||
            max_seq_len < 0 || (num_seqs > 0 && !seq_lens))
            return VERIFY_EINVAL;
    } else if (seq_lens || block_tables) {
        return VERIFY_EINVAL;  // the cache's shape is needed to check them
    }
    CArgs a{};
    a.num_seqs = num_seqs;
    a.total_q = total_q;
    a.max_q_len = max_q_len;
    if (params) {
        a.max_seq_len = max_seq_len;
        a.max_blocks = params->max_blocks_per_seq;
        a.num_blocks = params->num_blocks;
        a.window = params->sliding_window;
    }
    hipLaunchKernelGGL(check_reset, dim3(1), dim3(kWave), 0, stream, counts);
    if (num_seqs > 0)
        hipLaunchKernelGGL(check_batch, dim3((unsigned)std::min(num_seqs, kCheckMaxWorkgroups)),
                           dim3(kCheckThreads), 0, stream, a, q_start, params ? seq_lens : nullptr,
                           params ? block_tables : nullptr, counts);
    return check_launch();
}
