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
//   sample_chunks  the same for stochastic verification: the maximum of the
//                  logits over T plus Gumbel noise (a sample of the row's
//                  softmax);
//   accept_scan    one wavefront per request: reduces its rows' chunk
//                  partials to the row argmax, then finds the first draft
//                  that disagrees (wavefront ballot) and writes the accepted
//                  drafts and the bonus token.
#include <atomic>
#include <mutex>

#include "common.h"

// Scratch of verify_accept_noalloc (the per-(row, chunk) maxima, then the
// argmax when the caller passes none): one copy per GPU, held until the
// process ends.  In host code this name is not a device address; the
// address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[VERIFY_NOALLOC_SCRATCH_BYTES];

namespace averify {
namespace {

constexpr int kArgmaxThreads = 256;
constexpr int kArgmaxUnroll = 2;  // 16-byte vectors in flight per thread

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
    int nchunks, uint64_t* __restrict__ partial, int64_t row0) {
    constexpr int E = Storage<T>::kPer16B;
    const int64_t row = row0 + blockIdx.y;
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

// ---------------------------------------------------------------- sampling (T > 0)
//
// With drafts that put all their probability on one token, speculative
// rejection sampling at temperature T accepts draft d with probability p(d)
// and otherwise draws from p without d; drawing y ~ p = softmax(logits / T)
// per row and accepting iff y == d is that same rule.  y is drawn by the
// Gumbel-max rule y = argmax_v (x_v / T + g_v), g_v = -log(-log u_v), with u_v
// from Philox4x32-10 (Salmon et al., SC 2011; key = seed, counter =
// (v / 4, row, offset, 0), output word v % 4) and the log written below from
// the atanh series, every step an fp32 operation with fixed rounding, so the
// draw is reproducible bit for bit.  u = ((w >> 9) + 0.5) 2^-23 takes the top
// 23 bits: an odd multiple of 2^-24 that fp32 holds exactly, inside
// [2^-24, 1 - 2^-24], so g stays below 16.7 (24 bits would round the top code
// to u = 1).
//
// sample_chunks has argmax_chunks' grid and output, but its cost is
// arithmetic (the generator and two logs per logit), so it skips the logs of
// logits that cannot win.  -log(-log u) <= -log(1 - u), and 1 - u = n 2^-24
// with n = 2^24 - 2k - 1 (k = w >> 9), so g <= (clz(n) - 7) ln 2: a bound
// from one integer instruction.  A logit whose score under that bound stays
// below a score already reached in the chunk can be neither the row's maximum
// nor tied with it.  The others are queued per wavefront in LDS and evaluated
// 64 at a time, one per lane, so the logs run on full wavefronts.  The
// threshold is the wavefront's best evaluated score, raised after every
// batch; after the first batches almost no logit is queued.
struct SampleParams {
    uint32_t k0, k1;   // seed: key words
    uint32_t offset;   // counter word 2 (e.g. the decoding step)
    float inv_t;       // 1 / T, rounded to fp32 on the host
};

__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                              uint32_t k0, uint32_t k1, uint32_t out[4]) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        // one 32 x 32 -> 64-bit product gives both halves of each multiply
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        c0 = n0;
        c1 = (uint32_t)p1;
        c2 = n2;
        c3 = (uint32_t)p0;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

// log x for normal x > 0: x = m 2^e, m in [sqrt(1/2), sqrt(2)), z = (m-1)/(m+1),
// log x = e ln 2 + 2 (z + z^3/3 + z^5/5 + z^7/7 + z^9/9).
__device__ __forceinline__ float series_log(float x) {
    const uint32_t bits = __float_as_uint(x);
    int e = (int)((bits >> 23) & 0xFFu) - 127;
    float m = __uint_as_float((bits & 0x7FFFFFu) | 0x3F800000u);
    if (m > 1.41421354f) {
        m = m * 0.5f;
        e += 1;
    }
    const float z = (m - 1.0f) / (m + 1.0f);
    const float z2 = z * z;
    float poly = fmaf(z2, 0.111111112f, 0.142857149f);
    poly = fmaf(z2, poly, 0.200000003f);
    poly = fmaf(z2, poly, 0.333333343f);
    poly = fmaf(z2, poly, 1.0f);
    const float r = 2.0f * z * poly;
    return fmaf((float)e, 0.693147182f, r);
}

// Gumbel noise of the 23-bit code k = w >> 9.
__device__ __forceinline__ float gumbel_of_code(uint32_t k) {
    const float u = ((float)k + 0.5f) * 0x1p-23f;
    return -series_log(-series_log(u));
}

// An upper bound of gumbel_of_code(k): (clz(n) - 7) ln 2 >= -log(1 - u) >= g,
// with ln 2 rounded up and 1e-3 added, far above the few 1e-6 by which the
// fp32 evaluation of g can exceed its exact value.
__device__ __forceinline__ float gumbel_bound(uint32_t k) {
    const uint32_t n = 0xFFFFFFu - 2u * k;  // >= 1
    return fmaf((float)(__clz(n) - 7), 0.69315f, 1.0e-3f);
}
constexpr float kGumbelMax = 16.64f;  // >= gumbel_bound(k) for every k (n = 1: 24 ln 2)

constexpr int kSampleQueue = 2 * kWave;  // entries per wavefront queue
constexpr int kSampleUnroll = 2;         // 16-byte vectors per lane per iteration

template <typename T>
__global__ __launch_bounds__(kArgmaxThreads) void sample_chunks(
    const T* __restrict__ logits, int64_t row_stride, int64_t vocab, int64_t chunk_elems,
    int nchunks, uint64_t* __restrict__ partial, SampleParams sp, int64_t row0) {
    constexpr int E = Storage<T>::kPer16B;
    // queued logit: (x bits, code k, index, unused)
    __shared__ uint4 queue[kArgmaxThreads / kWave][kSampleQueue];
    __shared__ uint64_t red[kArgmaxThreads / kWave];
    const int64_t row = row0 + blockIdx.y;
    const uint32_t urow = (uint32_t)row;
    const int c = blockIdx.x;
    const T* rowp = logits + row * row_stride;
    const int64_t lo = (int64_t)c * chunk_elems;
    const int64_t hi = min(vocab, lo + chunk_elems);
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wid = tid / kWave;
    uint4* q = queue[wid];

    float best = -INFINITY;     // best evaluated score of this lane ...
    uint32_t best_idx = kNone;  // ... and its index (lowest among equal scores)
    uint32_t nan_idx = kNone;   // first NaN seen
    float thr = -INFINITY;      // wavefront-uniform: a score reached in this chunk
    int qn = 0;                 // wavefront-uniform queue fill

    auto take = [&](float x, uint32_t k, uint32_t idx) {
        const float s = fmaf(x, sp.inv_t, gumbel_of_code(k));
        if (s > best || (s == best && idx < best_idx)) {
            best = s;
            best_idx = idx;
        }
    };
    // Evaluate queue entries 0..63 (one per lane) and move the rest down.  One
    // wavefront's LDS accesses are served in program order, and the moved
    // entries [64, qn) never overlap their targets [0, qn - 64).
    auto flush = [&]() {
        const uint4 e = q[lane];
        const int rest = qn - kWave;
        uint4 m = make_uint4(0u, 0u, 0u, 0u);
        if (lane < rest) m = q[kWave + lane];
        asm volatile("" ::: "memory");
        if (lane < rest) q[lane] = m;
        asm volatile("" ::: "memory");
        take(__uint_as_float(e.x), e.y, e.z);
        qn = rest;
        const float wm = wave_max_xor(best, kWave);
        thr = fmaxf(thr, __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(wm))));
    };
    // One 16-byte vector of E logits at element `base`; `have` is false for
    // lanes past the chunk's last vector, which still take part in the ballots.
    auto scan = [&](const uint4& v, uint32_t base, bool have) {
        float x[E];
        unpack16(v, x, T());
        const bool nan = have && ((E == 8) ? any_nan_bf16x8(v) : any_nan_f32x4(v));
        if (nan && nan_idx == kNone) {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (x[e] != x[e]) { nan_idx = base + e; break; }
            }
        }
        // a lane that holds a NaN reports it; its other logits drop out
        const bool live = have && nan_idx == kNone;
#pragma unroll
        for (int b = 0; b < E / 4; ++b) {
            const float xm = fmaxf(fmaxf(x[4 * b], x[4 * b + 1]), fmaxf(x[4 * b + 2], x[4 * b + 3]));
            const bool any = live && fmaf(xm, sp.inv_t, kGumbelMax) >= thr;
            if (__ballot(any) == 0) continue;
            uint32_t w[4];
            philox4x32_10((base >> 2) + b, urow, sp.offset, 0u, sp.k0, sp.k1, w);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t k = w[e] >> 9;
                const float xe = x[4 * b + e];
                const bool cand = any && fmaf(xe, sp.inv_t, gumbel_bound(k)) >= thr;
                const uint64_t bal = __ballot(cand);
                if (bal == 0) continue;
                if (cand) {
                    const uint32_t below = __builtin_amdgcn_mbcnt_hi(
                        (uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
                    q[qn + (int)below] = make_uint4(__float_as_uint(xe), k, base + 4 * b + e, 0u);
                }
                qn += (int)__popcll(bal);
                if (qn >= kWave) flush();
            }
        }
    };
    // A logit outside the 16-byte vectors, evaluated directly (ascending per lane).
    auto one = [&](int64_t e) {
        const float x = Storage<T>::load(rowp, e);
        if (x != x) {
            if (nan_idx == kNone) nan_idx = (uint32_t)e;
        } else if (nan_idx == kNone) {
            uint32_t w[4];
            philox4x32_10((uint32_t)(e >> 2), urow, sp.offset, 0u, sp.k0, sp.k1, w);
            take(x, w[e & 3] >> 9, (uint32_t)e);
        }
    };

    if ((reinterpret_cast<uintptr_t>(rowp + lo) & 15u) == 0) {
        const uint4* vp = reinterpret_cast<const uint4*>(rowp + lo);
        const int64_t nvec = (hi - lo) / E;
        // Loop bounds are per wavefront (every lane reaches every ballot);
        // the next iteration's vectors load while this one's are scanned.
        constexpr int64_t kStep = (int64_t)kSampleUnroll * kArgmaxThreads;
        const int64_t wave_first = tid - lane;
        uint4 cur[kSampleUnroll], nxt[kSampleUnroll];
        auto load = [&](int64_t v0, uint4 (&dst)[kSampleUnroll]) {
#pragma unroll
            for (int u = 0; u < kSampleUnroll; ++u) {
                const int64_t vi = v0 + u * kArgmaxThreads + tid;
                dst[u] = vi < nvec ? ld16_stream(vp + vi) : make_uint4(0u, 0u, 0u, 0u);
            }
        };
        if (wave_first < nvec) load(0, cur);
        for (int64_t v0 = 0; v0 + wave_first < nvec; v0 += kStep) {
            if (v0 + kStep + wave_first < nvec) load(v0 + kStep, nxt);
#pragma unroll
            for (int u = 0; u < kSampleUnroll; ++u) {
                const int64_t vi = v0 + u * kArgmaxThreads + tid;
                scan(cur[u], (uint32_t)(lo + vi * E), vi < nvec);
            }
#pragma unroll
            for (int u = 0; u < kSampleUnroll; ++u) cur[u] = nxt[u];
        }
        for (int64_t e = lo + nvec * E + tid; e < hi; e += kArgmaxThreads) one(e);
    } else {
        for (int64_t e = lo + tid; e < hi; e += kArgmaxThreads) one(e);
    }
    if (qn > 0 && lane < qn) {
        const uint4 e = q[lane];
        take(__uint_as_float(e.x), e.y, e.z);
    }

    uint64_t packed = 0;
    if (nan_idx != kNone) {
        packed = pack(0xffffffffu, nan_idx);
    } else if (best_idx != kNone) {
        packed = pack(order_key(__float_as_uint(best)), best_idx);
    }
    packed = wave_max_u64(packed);
    if (lane == 0) red[wid] = packed;
    __syncthreads();
    if (tid == 0) {
        uint64_t m = red[0];
#pragma unroll
        for (int w = 1; w < kArgmaxThreads / kWave; ++w) m = red[w] > m ? red[w] : m;
        partial[row * nchunks + c] = m;
    }
}

// Partials a lane of accept_scan reduces at most: rows with more chunks
// (the fused LM head leaves one per workgroup) share a row among lanes.
constexpr int kScanChunksPerLane = 16;

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
    // L lanes share a row (a power of two; each lane reads at most
    // kScanChunksPerLane of the row's partials), R = 64 / L rows per round
    int L = 1;
    while (L < kWave && L * kScanChunksPerLane < nchunks) L <<= 1;
    const int R = kWave / L;
    const int sub = lane & (L - 1);
    for (int j0 = 0; j0 < n; j0 += R) {
        const int j = j0 + lane / L;
        uint64_t best = 0;
        if (j < n) {
            // all of a lane's loads of a pass are issued before any is
            // compared, so a pass costs one memory latency, not sixteen
            const uint64_t* pr = partial + (int64_t)(q0 + j) * nchunks;
            for (int c0 = sub; c0 < nchunks; c0 += L * kScanChunksPerLane) {
                uint64_t v[kScanChunksPerLane];
#pragma unroll
                for (int t = 0; t < kScanChunksPerLane; ++t) {
                    const int c = c0 + t * L;
                    v[t] = c < nchunks ? pr[c] : 0;
                }
#pragma unroll
                for (int t = 0; t < kScanChunksPerLane; ++t) best = v[t] > best ? v[t] : best;
            }
        }
        for (int o = 1; o < L; o <<= 1) {  // within the row's aligned group of L lanes
            const uint64_t other = shfl_xor_u64(best, o);
            best = other > best ? other : best;
        }
        const int32_t am = (int32_t)(0xffffffffu - (uint32_t)best);
        const bool lead = sub == 0 && j < n;
        if (lead) argmax_out[q0 + j] = am;
        if (m < 0) {
            // stop at the first row whose argmax disagrees with the next
            // draft, or at row k, which has no draft after it
            const bool stop = lead && (j == k || am != tokens[q0 + j + 1]);
            const uint64_t ballot = __ballot(stop);
            if (ballot) {
                const int first = (int)__builtin_ctzll(ballot);
                m = j0 + first / L;
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

// Rows are cut into chunks so that the whole grid is about two rounds of
// resident workgroups (eight 256-thread workgroups on each of MI355X's 256
// compute units), each thread keeping two 16-byte vectors in flight.
// Measured on the Qwen-shaped logits (288 x 151936 bf16): 17.2 us, against
// 18.1-19.3 us for one round with four vectors in flight and 18.3-22 us for
// the other combinations of one, two or four rounds and one to eight
// vectors tried.  Chunks are whole 16-byte vectors per thread.
constexpr int64_t kArgmaxTargetWgs = 4096;

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

// Launch the per-chunk scan (argmax, or the sampler when sp is given) and the
// acceptance scan after argument checks shared by both entry points.
int accept_launch(int32_t num_seqs, int32_t total_q, int64_t vocab, int64_t row_stride,
                  int32_t logits_dtype, const void* logits, const int32_t* tokens,
                  const int32_t* q_start, int32_t* argmax_out, int32_t* accept_len,
                  int32_t* num_emitted, int32_t* emitted, void* workspace, size_t workspace_bytes,
                  const SampleParams* sp, hipStream_t stream) {
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
    // rows go on grid y, at most 65535 per launch
    constexpr int kRowsPerLaunch = 65535;
    for (int64_t r0 = 0; r0 < total_q; r0 += kRowsPerLaunch) {
        const dim3 grid(p.nchunks, (unsigned)std::min<int64_t>(kRowsPerLaunch, total_q - r0));
        const dim3 block(kArgmaxThreads);
        const bool bf16 = logits_dtype == VERIFY_BF16;
        if (sp && bf16) {
            hipLaunchKernelGGL(sample_chunks<uint16_t>, grid, block, 0, stream,
                               static_cast<const uint16_t*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial, *sp, r0);
        } else if (sp) {
            hipLaunchKernelGGL(sample_chunks<float>, grid, block, 0, stream,
                               static_cast<const float*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial, *sp, r0);
        } else if (bf16) {
            hipLaunchKernelGGL(argmax_chunks<uint16_t>, grid, block, 0, stream,
                               static_cast<const uint16_t*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial, r0);
        } else {
            hipLaunchKernelGGL(argmax_chunks<float>, grid, block, 0, stream,
                               static_cast<const float*>(logits), row_stride, vocab,
                               p.chunk_elems, p.nchunks, partial, r0);
        }
        if (check_launch() != VERIFY_OK) return VERIFY_EHIP;
    }
    return launch_accept_scan(num_seqs, q_start, tokens, partial, p.nchunks, am, accept_len,
                              num_emitted, emitted, stream);
}

}  // namespace

int launch_accept_scan(int num_seqs, const int32_t* q_start, const int32_t* tokens,
                       const uint64_t* partial, int nchunks, int32_t* argmax_out,
                       int32_t* accept_len, int32_t* num_emitted, int32_t* emitted,
                       hipStream_t stream) {
    if (num_seqs <= 0) return VERIFY_OK;
    hipLaunchKernelGGL(accept_scan, dim3(num_seqs), dim3(kWave), 0, stream, num_seqs, q_start,
                       tokens, partial, nchunks, argmax_out, accept_len, num_emitted, emitted);
    return check_launch();
}

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
    return accept_launch(num_seqs, total_q, vocab, row_stride, logits_dtype, logits, tokens, q_start,
                         argmax_out, accept_len, num_emitted, emitted, workspace, workspace_bytes,
                         nullptr, stream);
}

extern "C" int verify_accept_sampled(int32_t num_seqs, int32_t total_q, int64_t vocab,
                                     int64_t row_stride, int32_t logits_dtype, const void* logits,
                                     const int32_t* tokens, const int32_t* q_start,
                                     float temperature, uint64_t seed, uint32_t offset,
                                     int32_t* sampled_out, int32_t* accept_len, int32_t* num_emitted,
                                     int32_t* emitted, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream) {
    if (!(temperature > 0.0f) || !(temperature < 3.0e38f)) return VERIFY_EINVAL;
    SampleParams sp;
    sp.k0 = (uint32_t)seed;
    sp.k1 = (uint32_t)(seed >> 32);
    sp.offset = offset;
    sp.inv_t = (float)(1.0 / (double)temperature);
    if (!(sp.inv_t > 0.0f) || !(sp.inv_t < 3.0e38f)) return VERIFY_EINVAL;
    return accept_launch(num_seqs, total_q, vocab, row_stride, logits_dtype, logits, tokens, q_start,
                         sampled_out, accept_len, num_emitted, emitted, workspace, workspace_bytes,
                         &sp, stream);
}

// Device address of `scratch` on the current device, looked up on the first
// call per device (with that device current) and kept.
static int noalloc_scratch(void** out) {
    static std::atomic<void*> ptrs[64];
    static std::mutex mu;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return VERIFY_EHIP;
    }
    if (dev < 0 || dev >= 64) return VERIFY_EUNSUPPORTED;
    void* p = ptrs[dev].load(std::memory_order_acquire);
    if (!p) {
        std::lock_guard<std::mutex> lock(mu);
        p = ptrs[dev].load(std::memory_order_relaxed);
        if (!p) {
            if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
                (void)hipGetLastError();
                return VERIFY_EHIP;
            }
            ptrs[dev].store(p, std::memory_order_release);
        }
    }
    *out = p;
    return VERIFY_OK;
}

extern "C" int verify_accept_noalloc(int32_t num_seqs, int32_t total_q, int64_t vocab,
                                     int64_t row_stride, int32_t logits_dtype, const void* logits,
                                     const int32_t* tokens, const int32_t* q_start,
                                     int32_t* argmax_out, int32_t* accept_len,
                                     int32_t* num_emitted, int32_t* emitted, hipStream_t stream) {
    // sizes first: a call the scratch cannot hold fails before any HIP call
    if (logits_dtype != VERIFY_F32 && logits_dtype != VERIFY_BF16) return VERIFY_EUNSUPPORTED;
    if (!accept_args_ok(num_seqs, total_q, vocab, logits_dtype)) return VERIFY_EINVAL;
    const AcceptPlan p = plan_accept(total_q, vocab, logits_dtype);
    const size_t need = p.partial_bytes + p.argmax_bytes;
    if (need > (size_t)VERIFY_NOALLOC_SCRATCH_BYTES) return VERIFY_EWORKSPACE;
    void* ws = nullptr;
    const int rc = noalloc_scratch(&ws);
    if (rc != VERIFY_OK) return rc;
    // every partial the scan reads is written by the argmax pass of the same
    // call, so nothing of the previous call's contents needs clearing
    return accept_launch(num_seqs, total_q, vocab, row_stride, logits_dtype, logits, tokens, q_start,
                         argmax_out, accept_len, num_emitted, emitted, ws,
                         (size_t)VERIFY_NOALLOC_SCRATCH_BYTES, nullptr, stream);
}
