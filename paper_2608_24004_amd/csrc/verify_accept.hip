// verify_accept.hip -- vocabulary argmax of every scored position and greedy
// acceptance of the drafts (paper Sec. 2.2: the target verifies all proposed
// tokens in one pass and the output equals plain greedy decoding; Sec. 3.1:
// rejection rate = rejected / proposed drafts per request).
//
// Two kernels on one stream:
//   argmax_chunks  grid (chunks, rows): each workgroup streams one contiguous
//                  chunk of one logits row with 16-byte coalesced loads and
//                  reduces it to a packed (order key, ~index) 64-bit maximum,
//                  which is the lowest index among equal maxima;
//   accept_scan    one wavefront per request: reduces its rows' chunk
//                  partials to the row argmax, then finds the first draft
//                  that disagrees (wavefront ballot) and writes the accepted
//                  drafts and the bonus token.
#include "common.h"

namespace averify {
namespace {

constexpr int kArgmaxThreads = 256;
constexpr int kArgmaxUnroll = 4;  // 16-byte vectors in flight per thread

// Monotone map from a float to an unsigned key: a > b  <=>  key(a) > key(b)
// for non-NaN values, -0.0 and +0.0 share a key, and NaN maps above +inf.
__device__ __forceinline__ uint32_t order_key(uint32_t bits) {
    const uint32_t mag = bits & 0x7fffffffu;
    if (mag > 0x7f800000u) return 0xffffffffu;
    if (mag == 0) bits = 0;
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

__device__ __forceinline__ uint64_t pack(uint32_t key, uint32_t idx) {
    return ((uint64_t)key << 32) | (uint32_t)(0xffffffffu - idx);
}

// True if any bf16 half of the four words is a NaN (|h| > 0x7f80).
__device__ __forceinline__ bool any_nan_bf16x8(const uint4& v) {
    const uint32_t m = 0x7fff7fffu, c = 0x007f007fu, s = 0x80008000u;
    return (((v.x & m) + c) | ((v.y & m) + c) | ((v.z & m) + c) | ((v.w & m) + c)) & s;
}
__device__ __forceinline__ bool any_nan_f32x4(const uint4& v) {
    const uint32_t m = 0x7fffffffu, inf = 0x7f800000u;
    return ((v.x & m) > inf) | ((v.y & m) > inf) | ((v.z & m) > inf) | ((v.w & m) > inf);
}

constexpr uint32_t kNone = 0xffffffffu;  // no element recorded

// Scan one 16-byte vector of E elements starting at element index `base`.
// Keeps the first strict maximum in ascending index order (float compare:
// -0.0 == +0.0), so ties inside a thread go to the lower index.  A vector with
// a NaN only records the index of its first NaN (a thread scans ascending
// indices, so the first NaN it records is its lowest); finite maxima are then
// irrelevant for the row.
template <typename T>
__device__ __forceinline__ void scan_vec(const uint4& v, uint32_t base, float& best,
                                         uint32_t& best_idx, uint32_t& nan_idx) {
    constexpr int E = Storage<T>::kPer16B;
    float x[E];
    unpack16(v, x, T());
    const bool nan = (E == 8) ? any_nan_bf16x8(v) : any_nan_f32x4(v);
    if (!nan) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const bool gt = x[e] > best;
            best = gt ? x[e] : best;
            best_idx = gt ? base + e : best_idx;
        }
    } else if (nan_idx == kNone) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (x[e] != x[e]) { nan_idx = base + e; break; }
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kArgmaxThreads) void argmax_chunks(
    const T* __restrict__ logits, int64_t row_stride, int64_t vocab, int64_t chunk_elems,
    int nchunks, uint64_t* __restrict__ partial) {
    constexpr int E = Storage<T>::kPer16B;
    const int64_t row = blockIdx.y;
    const int c = blockIdx.x;
    const T* rowp = logits + row * row_stride;
    const int64_t lo = (int64_t)c * chunk_elems;
    const int64_t hi = min(vocab, lo + chunk_elems);
    const int tid = threadIdx.x;

    float best = -INFINITY;
    uint32_t best_idx = kNone;  // first strict finite/inf maximum seen
    uint32_t nan_idx = kNone;   // first NaN seen

    if ((reinterpret_cast<uintptr_t>(rowp + lo) & 15u) == 0) {
        const uint4* vp = reinterpret_cast<const uint4*>(rowp + lo);
        const int64_t nvec = (hi - lo) / E;
        // Batches of kArgmaxUnroll vectors per thread, the next batch loaded
        // before the current one is scanned so that loads stay in flight
        // while the wavefront compares.
        constexpr int64_t kStep = (int64_t)kArgmaxUnroll * kArgmaxThreads;
        int64_t vi = tid;
        if (vi + (kArgmaxUnroll - 1) * kArgmaxThreads < nvec) {
            uint4 cur[kArgmaxUnroll];
#pragma unroll
            for (int u = 0; u < kArgmaxUnroll; ++u) cur[u] = ld16_stream(vp + vi + u * kArgmaxThreads);
            for (; vi + kStep + (kArgmaxUnroll - 1) * kArgmaxThreads < nvec; vi += kStep) {
                uint4 nxt[kArgmaxUnroll];
#pragma unroll
                for (int u = 0; u < kArgmaxUnroll; ++u) nxt[u] = ld16_stream(vp + vi + kStep + u * kArgmaxThreads);
#pragma unroll
                for (int u = 0; u < kArgmaxUnroll; ++u)
                    scan_vec<T>(cur[u], (uint32_t)(lo + (vi + u * kArgmaxThreads) * E), best, best_idx, nan_idx);
#pragma unroll
                for (int u = 0; u < kArgmaxUnroll; ++u) cur[u] = nxt[u];
            }
#pragma unroll
            for (int u = 0; u < kArgmaxUnroll; ++u)
                scan_vec<T>(cur[u], (uint32_t)(lo + (vi + u * kArgmaxThreads) * E), best, best_idx, nan_idx);
            vi += kStep;
        }
        for (; vi < nvec; vi += kArgmaxThreads) {
            uint4 v = ld16_stream(vp + vi);
            scan_vec<T>(v, (uint32_t)(lo + vi * E), best, best_idx, nan_idx);
        }
        for (int64_t e = lo + nvec * E + tid; e < hi; e += kArgmaxThreads) {
            const float x = Storage<T>::load(rowp, e);
            if (x != x) {
                if (nan_idx == kNone) nan_idx = (uint32_t)e;
            } else if (x > best) { best = x; best_idx = (uint32_t)e; }
        }
    } else {
        for (int64_t e = lo + tid; e < hi; e += kArgmaxThreads) {
            const float x = Storage<T>::load(rowp, e);
            if (x != x) {
                if (nan_idx == kNone) nan_idx = (uint32_t)e;
            } else if (x > best) { best = x; best_idx = (uint32_t)e; }
        }
    }

    // Threads that saw only -inf report nothing, except thread 0, which owns
    // the chunk's first element: an all -inf chunk reports its lowest index.
    uint64_t packed = 0;
    if (nan_idx != kNone) {
        packed = pack(0xffffffffu, nan_idx);
    } else if (best_idx != kNone) {
        packed = pack(order_key(__float_as_uint(best)), best_idx);
    } else if (tid == 0 && lo < hi) {
        packed = pack(order_key(__float_as_uint(-INFINITY)), (uint32_t)lo);
    }
    packed = wave_max_u64(packed);

    __shared__ uint64_t red[kArgmaxThreads / kWave];
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    if (lane == 0) red[wid] = packed;
    __syncthreads();
    if (tid == 0) {
        uint64_t m = red[0];
#pragma unroll
        for (int w = 1; w < kArgmaxThreads / kWave; ++w) m = red[w] > m ? red[w] : m;
        partial[row * nchunks + c] = m;
    }
}

__global__ __launch_bounds__(kWave) void accept_scan(
    int num_seqs, const int32_t* __restrict__ q_start, const int32_t* __restrict__ tokens,
    const uint64_t* __restrict__ partial, int nchunks, int32_t* __restrict__ argmax_out,
    int32_t* __restrict__ accept_len, int32_t* __restrict__ num_emitted,
    int32_t* __restrict__ emitted) {
    const int i = blockIdx.x;
    if (i >= num_seqs) return;
    const int lane = threadIdx.x;
    const int q0 = q_start[i];
    const int n = q_start[i + 1] - q0;
    if (n <= 0) {
        if (lane == 0) { accept_len[i] = 0; num_emitted[i] = 0; }
        return;
    }
    const int k = n - 1;   // drafts; draft j+1 sits at tokens[q0 + j + 1]
    int m = -1;            // accepted drafts, once known
    int32_t bonus = 0;
    for (int j0 = 0; j0 < n; j0 += kWave) {
        // each lane reduces the chunk partials of one row to its argmax
        const int j = j0 + lane;
        int32_t am = 0;
        if (j < n) {
            const uint64_t* pr = partial + (int64_t)(q0 + j) * nchunks;
            uint64_t best = 0;
            for (int c = 0; c < nchunks; ++c) best = pr[c] > best ? pr[c] : best;
            am = (int32_t)(0xffffffffu - (uint32_t)best);
            argmax_out[q0 + j] = am;
        }
        if (m < 0) {
            // stop at the first row whose argmax disagrees with the next
            // draft, or at row k, which has no draft after it
            const bool stop = (j < n) && (j == k || am != tokens[q0 + j + 1]);
            const uint64_t ballot = __ballot(stop);
            if (ballot) {
                const int first = (int)__builtin_ctzll(ballot);
                m = j0 + first;
                bonus = __shfl(am, first);
            }
        }
    }
    for (int j = lane; j < n; j += kWave) {
        int32_t v = -1;
        if (j < m) v = tokens[q0 + j + 1];
        else if (j == m) v = bonus;
        emitted[q0 + j] = v;
    }
    if (lane == 0) { accept_len[i] = m; num_emitted[i] = m + 1; }
}

struct AcceptPlan {
    int64_t chunk_elems;
    int nchunks;
    size_t partial_bytes;
    size_t argmax_bytes;  // scratch argmax when the caller passes none
};

// Rows are cut into chunks so that the whole grid is about one round of
// resident workgroups (eight 256-thread workgroups on each of MI355X's 256
// compute units): a second, partly filled round would leave most of the chip
// idle for its duration.  Chunks are whole 16-byte vectors per thread.
constexpr int64_t kArgmaxTargetWgs = 2048;

AcceptPlan plan_accept(int32_t total_q, int64_t vocab, int32_t dtype) {
    AcceptPlan p{};
    const int per16 = dtype == VERIFY_BF16 ? 8 : 4;
    const int64_t quantum = (int64_t)kArgmaxThreads * per16;
    const int64_t want = std::max<int64_t>(1, kArgmaxTargetWgs / std::max<int64_t>(1, total_q));
    const int64_t per_chunk = (vocab + want - 1) / want;
    p.chunk_elems = (per_chunk + quantum - 1) / quantum * quantum;
    p.nchunks = (int)((vocab + p.chunk_elems - 1) / p.chunk_elems);
    p.partial_bytes = align_up((size_t)total_q * p.nchunks * sizeof(uint64_t), 256);
    p.argmax_bytes = align_up((size_t)total_q * sizeof(int32_t), 256);
    return p;
}

bool accept_args_ok(int32_t num_seqs, int32_t total_q, int64_t vocab, int32_t dtype) {
    return num_seqs >= 0 && total_q >= 0 && vocab >= 1 && vocab < (int64_t)0x7fffffff &&
           (dtype == VERIFY_F32 || dtype == VERIFY_BF16);
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_accept_workspace_size(int32_t num_seqs, int32_t total_q, int64_t vocab,
                                            int32_t logits_dtype, size_t* bytes) {
    if (!bytes) return VERIFY_EINVAL;
    if (!accept_args_ok(num_seqs, total_q, vocab, logits_dtype)) {
        return (logits_dtype == VERIFY_F32 || logits_dtype == VERIFY_BF16) ? VERIFY_EINVAL
                                                                            : VERIFY_EUNSUPPORTED;
    }
    const AcceptPlan p = plan_accept(total_q, vocab, logits_dtype);
    *bytes = p.partial_bytes + p.argmax_bytes;
    return VERIFY_OK;
}

extern "C" int verify_accept(int32_t num_seqs, int32_t total_q, int64_t vocab, int64_t row_stride,
                             int32_t logits_dtype, const void* logits, const int32_t* tokens,
                             const int32_t* q_start, int32_t* argmax_out, int32_t* accept_len,
                             int32_t* num_emitted, int32_t* emitted, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
    if (logits_dtype != VERIFY_F32 && logits_dtype != VERIFY_BF16) return VERIFY_EUNSUPPORTED;
    if (!accept_args_ok(num_seqs, total_q, vocab, logits_dtype)) return VERIFY_EINVAL;
    if (row_stride == 0) row_stride = vocab;
    if (row_stride < vocab) return VERIFY_EINVAL;
    if (num_seqs > 0 && (!q_start || !accept_len || !num_emitted)) return VERIFY_EINVAL;
    if (total_q > 0 && (!logits || !tokens || !emitted)) return VERIFY_EINVAL;
    const AcceptPlan p = plan_accept(total_q, vocab, logits_dtype);
    const size_t need = p.partial_bytes + p.argmax_bytes;
    if (workspace_bytes < need || (need > 0 && !workspace)) return VERIFY_EWORKSPACE;
    if (num_seqs == 0) return VERIFY_OK;

    uint64_t* partial = static_cast<uint64_t*>(workspace);
    int32_t* am = argmax_out ? argmax_out
                             : reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + p.partial_bytes);
    if (total_q > 0) {
        dim3 grid(p.nchunks, total_q);
        if (logits_dtype == VERIFY_BF16) {
            hipLaunchKernelGGL(argmax_chunks<uint16_t>, grid, dim3(kArgmaxThreads), 0, stream,
                               static_cast<const uint16_t*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial);
        } else {
            hipLaunchKernelGGL(argmax_chunks<float>, grid, dim3(kArgmaxThreads), 0, stream,
                               static_cast<const float*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial);
        }
        if (check_launch() != VERIFY_OK) return VERIFY_EHIP;
    }
    hipLaunchKernelGGL(accept_scan, dim3(num_seqs), dim3(kWave), 0, stream, num_seqs, q_start,
                       tokens, partial, p.nchunks, am, accept_len, num_emitted, emitted);
    return check_launch();
}
