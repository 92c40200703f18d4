// verify_lmhead.hip -- the LM head of the verify pass fused with greedy
// acceptance: logits[r][v] = <hidden[r], weight[v]> for every scored position
// r and vocabulary entry v, reduced to each row's argmax on the fly, so the
// [total_q][vocab] logits never reach HBM; then the longest accepted draft
// prefix plus the bonus token (paper Sec. 2.2: the target scores all proposed
// tokens in one pass and the result equals plain greedy decoding).
//
// The contraction is dense (every weight row meets every scored row), so it
// runs on MFMA: v_mfma_f32_32x32x16_bf16 with the vocabulary on the M side
// (A = 32 weight rows x 16 hidden dims) and the scored rows on the N side
// (B = 16 hidden dims x 32 rows).  A lane of the 32 x 32 result holds one
// scored row (column l % 32) and 16 vocabulary entries, so most of the argmax
// is a running compare inside the lane.
//
// Work split.  lmhead_argmax launches one 12-wavefront workgroup per compute
// unit (three wavefronts per SIMD).  Workgroup w owns the vocabulary range
// [V w / N, V (w+1) / N); wavefront (q, g) takes vocabulary quarter q of it and
// scored-row group g (of three) of the current row chunk, and walks its
// quarter in passes of two 32-entry tiles (the last pass may hold one).  Per
// pass, the hidden dimension is walked in steps of 32: each step's weight rows
// (256 = 4 quarters x 64) and scored rows (up to 288 = 3 groups x 3 tiles of
// 32) are copied once, 16 bytes per lane, from global memory into a ring of
// four LDS stages (three steps in flight), read from there as MFMA operands by
// every wavefront that needs them, and accumulated in registers (2 x 3 tiles
// of 16 floats per lane).  At the end of a pass the lane folds its logits
// into a running (maximum, first index, first NaN) per scored row.  Every
// weight byte is read from HBM once per row chunk; the hidden states (a few
// MB) come from L2.  More than 288 scored rows are cut into row chunks, each
// walking the weights again.
//
// After the last pass the wavefronts' maxima are merged into one packed
// (order key, ~index) word per (scored row, workgroup), the format of
// verify_accept's per-chunk partials, and the same acceptance scan finishes
// the step.
#include <type_traits>

#include "common.h"

namespace averify {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kLmRowGroups = 3;                    // scored-row groups per workgroup
constexpr int kLmWaves = 4 * kLmRowGroups;         // 4 vocabulary quarters x the row groups
constexpr int kLmQuarters = 4;
constexpr int kLmThreads = kLmWaves * kWave;
constexpr int kLmStep = 32;                        // hidden dims per LDS stage
constexpr int kLmStages = 4;                       // LDS ring stages
constexpr int kLmDepth = kLmStages - 1;            // stages in flight
constexpr int kLmWaveRows = 64;                    // weight rows per wavefront and pass
constexpr int kLmWRows = kLmQuarters * kLmWaveRows;  // weight rows per stage (256)
constexpr int kLmMaxTiles = 3;                     // scored-row tiles of 32 per wavefront
constexpr int kLmRowBytes = kLmStep * 2;           // one row of a stage: 32 bf16 = 64 bytes
constexpr uint32_t kLmNone = 0xffffffffu;

struct LArgs {
    int T;           // scored rows
    int H;           // hidden size (multiple of kLmStep)
    int V;           // vocabulary
    int nwg;         // workgroups (vocabulary ranges)
    int chunk_rows;  // scored rows per row chunk (<= kLmRowGroups * 32 * MT)
    int nchunks;     // row chunks
    int passes;      // passes of two tiles per wavefront over its vocabulary quarter
    int nk;          // hidden steps per pass (H / kLmStep)
};

// A stage holds kLmRowGroups * MT * 32 scored rows, then 256 weight rows, each 32 bf16 = four
// 16-byte chunks.  Chunk c of row r is stored at position c ^ f(r), f(r) =
// 2 ((r >> 2) & 1) + ((r >> 3) & 1).  A ds_read_b128 of 32 rows at one logical
// chunk (two chunks per row, one per half-wave) then takes gfx950's minimum of
// four LDS cycles; measured with the LDS bank-conflict counter, the unswizzled
// layout takes sixteen and an XOR of bits 1-3 eight.
__device__ __forceinline__ int swz(int r, int c) {
    return c ^ (((r >> 2) & 1) << 1) ^ ((r >> 3) & 1);
}

// f(std::integral_constant<int, v>) for a runtime v in [0, M].
template <int M, typename F>
__device__ __forceinline__ void with_count(int v, F&& f) {
    if constexpr (M == 0) {
        f(std::integral_constant<int, 0>{});
    } else {
        if (v >= M) f(std::integral_constant<int, M>{});
        else with_count<M - 1>(v, f);
    }
}

// Vocabulary quarter q [lo, hi) of workgroup w.
__device__ __forceinline__ void wave_range(const LArgs& a, int w, int q, int& lo, int& hi) {
    const int64_t v0 = (int64_t)a.V * w / a.nwg, v1 = (int64_t)a.V * (w + 1) / a.nwg;
    const int64_t len = v1 - v0;
    lo = (int)(v0 + len * q / kLmQuarters);
    hi = (int)(v0 + len * (q + 1) / kLmQuarters);
}

// Fold one logit into a running (maximum, first index, first NaN): logits
// arrive in ascending vocabulary order, so a strict compare keeps the lowest
// index among equal maxima (-0.0 == +0.0).
__device__ __forceinline__ void fold(float x, uint32_t v, bool ok, float& best, uint32_t& bidx,
                                     uint32_t& nidx) {
    const bool nan = ok && x != x;
    nidx = (nan && nidx == kLmNone) ? v : nidx;
    const bool gt = ok && x > best;
    best = gt ? x : best;
    bidx = gt ? v : bidx;
}

template <int MT>
__global__ __launch_bounds__(kLmThreads)
__attribute__((amdgpu_waves_per_eu(kLmRowGroups, kLmRowGroups)))
void lmhead_argmax(LArgs a, const uint16_t* __restrict__ hid, const uint16_t* __restrict__ wt,
                   uint64_t* __restrict__ partial) {
    constexpr int HROWS = kLmRowGroups * MT * 32;        // scored rows per stage
    constexpr int STAGE = (HROWS + kLmWRows) * kLmRowBytes;
    constexpr int NI = (HROWS + kLmWRows) * 4 / kWave;   // 1 KiB global->LDS loads per stage
    constexpr int CPT_HI = (NI + kLmWaves - 1) / kLmWaves;
    constexpr int CPT_LO = NI / kLmWaves;
    static_assert(NI * kWave == (HROWS + kLmWRows) * 4, "whole 1 KiB loads per stage");
    static_assert(CPT_HI * (kLmDepth - 1) < 64, "vmcnt range");

    __shared__ __attribute__((aligned(16))) uint8_t stage[kLmStages][STAGE];
    __shared__ uint64_t red[kLmQuarters][HROWS];

    const int w = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);  // wavefront-uniform
    const int c32 = lane & 31, h = lane >> 5;
    const int cpt = wv < NI % kLmWaves || NI % kLmWaves == 0 ? CPT_HI : CPT_LO;
    const int wq = wv % kLmQuarters;  // vocabulary quarter
    const int wg = wv / kLmQuarters;  // row group: rows [32 MT wg, 32 MT (wg + 1)) of a chunk

    // this wavefront's vocabulary quarter and the workgroup's range
    int vlo, vhi;
    wave_range(a, w, wq, vlo, vhi);
    const int wg_lo = (int)((int64_t)a.V * w / a.nwg);
    const int wg_hi = (int)((int64_t)a.V * (w + 1) / a.nwg);
    const int wtiles = (vhi - vlo + 31) / 32;  // this wavefront's 32-entry tiles

    const uint32_t stage_lds =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)&stage[0][0];
    const int units = a.nchunks * a.passes * a.nk;

    // ---- loader: unit u = (row chunk, pass, hidden step); one unit fills one
    // stage.  Load c2 of this wavefront is stage load i = 12 c2 + wv, covering
    // stage chunks [64 i, 64 i + 64); lane l moves chunk 64 i + l.
    const uint16_t* src[CPT_HI];
    int l_u = 0, l_ks = 0;
    auto set_sources = [&](int u) {
        const int mc = u / (a.passes * a.nk);
        const int p = (u / a.nk) % a.passes;
        const int r0 = mc * a.chunk_rows;
        const int r1 = min(a.T, r0 + a.chunk_rows);
#pragma unroll
        for (int c2 = 0; c2 < CPT_HI; ++c2) {
            const int i = c2 * kLmWaves + wv;
            if (i >= NI) {  // this wavefront has one load fewer
                src[c2] = hid;
                continue;
            }
            const int pos = i * kWave + lane;        // stage chunk
            const int row = pos >> 2, cs = pos & 3;  // stage row, stored chunk
            const int c = swz(row, cs);              // logical chunk: dims 8c .. 8c+7
            const uint16_t* sp;
            if (row < HROWS) {
                const int r = min(r0 + row, r1 - 1);  // rows past the chunk repeat its last
                sp = hid + (int64_t)r * a.H + c * 8;
            } else {
                const int wr = row - HROWS;           // weight row of the stage
                const int q = wr / kLmWaveRows, t = wr % kLmWaveRows;
                int qlo, qhi;
                wave_range(a, w, q, qlo, qhi);
                int v = qlo + p * kLmWaveRows + t;
                // rows past the quarter read the workgroup's first row again
                // (served from cache; their results are never used)
                if (v >= qhi) v = min(wg_lo, a.V - 1);
                sp = wt + (int64_t)v * a.H + c * 8;
            }
            src[c2] = sp;
        }
    };
    auto dma_unit = [&](int st) {
        const uint32_t base = stage_lds + st * STAGE;
        const int koff = l_ks * kLmStep;
#pragma unroll
        for (int c2 = 0; c2 < CPT_HI; ++c2) {
            const int i = c2 * kLmWaves + wv;
            if (i < NI) dma16(base + i * (kWave * 16), src[c2] + koff);
        }
    };
    // issue the loads of the loader's unit into stage st, then step the loader
    // (it stays on the last unit, loading it again, so that every iteration
    // issues the same number of loads)
    auto dma_next = [&](int st) {
        dma_unit(st);
        if (l_u + 1 < units) {
            ++l_u;
            if (++l_ks == a.nk) {
                l_ks = 0;
                set_sources(l_u);
            }
        }
    };

    // ---- running maxima per scored-row tile
    float best[MT];
    uint32_t bidx[MT], nidx[MT];
#pragma unroll
    for (int n = 0; n < MT; ++n) {
        best[n] = -INFINITY;
        bidx[n] = kLmNone;
        nidx[n] = kLmNone;
    }

    // row tiles of this wavefront's group that hold rows of the current chunk
    int mtv = MT;
    // One hidden step of a pass: NT = weight tiles of this wavefront (1 or 2),
    // MV = row tiles holding rows of the chunk (a compile-time count, so that
    // the step is straight-line code: every fragment of a 16-dim half is
    // read before its products, one LDS round trip per half instead of one
    // per row tile).
    auto compute = [&](int st, auto& acc, auto mv) {
        constexpr int NT = sizeof(acc) / sizeof(acc[0]);
        constexpr int MV = decltype(mv)::value;
        if constexpr (MV > 0) {
            const uint8_t* hs = stage[st];
            const uint8_t* ws = stage[st] + HROWS * kLmRowBytes;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int cs = swz(c32, 2 * j + h) * 16;  // same swizzle for every tile row
                bf16x8_t wf[NT], hf[MV];
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    wf[t] = __builtin_bit_cast(
                        bf16x8_t, *reinterpret_cast<const uint4*>(
                                      ws + (wq * kLmWaveRows + t * 32 + c32) * kLmRowBytes + cs));
#pragma unroll
                for (int n = 0; n < MV; ++n)
                    hf[n] = __builtin_bit_cast(
                        bf16x8_t, *reinterpret_cast<const uint4*>(
                                      hs + ((wg * MT + n) * 32 + c32) * kLmRowBytes + cs));
#pragma unroll
                for (int n = 0; n < MV; ++n)
#pragma unroll
                    for (int t = 0; t < NT; ++t)
                        acc[t][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[t], hf[n], acc[t][n], 0, 0, 0);
            }
        }
    };

    // fold a pass's logits into the running maxima: lane (h, c32) holds entry
    // 8 (e / 4) + 4 h + e % 4 of each weight tile
    auto end_pass = [&](int p, auto& acc) {
        constexpr int NT = sizeof(acc) / sizeof(acc[0]);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int v0 = vlo + p * kLmWaveRows + t * 32 + 4 * h;
#pragma unroll
            for (int n = 0; n < MT; ++n) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int v = v0 + 8 * (e >> 2) + (e & 3);
                    fold(acc[t][n][e], (uint32_t)v, v < vhi, best[n], bidx[n], nidx[n]);
                }
                // one tile at a time: keeps the scheduler from moving every
                // accumulator into vector registers at once
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    // merge the four wavefronts' maxima of a row chunk and store one packed
    // word per scored row
    auto end_chunk = [&](int mc) {
        const int r0 = mc * a.chunk_rows;
        const int nrows = min(a.T, r0 + a.chunk_rows) - r0;
#pragma unroll
        for (int n = 0; n < MT; ++n) {
            uint64_t pk = 0;
            if (nidx[n] != kLmNone) pk = pack(0xffffffffu, nidx[n]);
            else if (bidx[n] != kLmNone) pk = pack(order_key(__float_as_uint(best[n])), bidx[n]);
            const uint64_t other = shfl_xor_u64(pk, 32);
            pk = other > pk ? other : pk;
            if (h == 0) red[wq][(wg * MT + n) * 32 + c32] = pk;
            best[n] = -INFINITY;
            bidx[n] = kLmNone;
            nidx[n] = kLmNone;
        }
        lds_barrier();
        for (int r = tid; r < nrows; r += kLmThreads) {
            uint64_t m = red[0][r];
#pragma unroll
            for (int q = 1; q < kLmQuarters; ++q) m = red[q][r] > m ? red[q][r] : m;
            // a range whose logits are all -inf reports its first entry
            if (m == 0 && wg_lo < wg_hi) m = pack(order_key(__float_as_uint(-INFINITY)), (uint32_t)wg_lo);
            partial[(int64_t)(r0 + r) * a.nwg + w] = m;
        }
        lds_barrier();
    };

    set_sources(0);
#pragma unroll
    for (int r = 0; r < kLmDepth; ++r) dma_next(r);

    // Ring pipeline per hidden step: wait for this wavefront's loads of the
    // step's stage, barrier (everyone's loads landed, everyone is done with
    // the previous stage), refill the previous stage kLmDepth steps ahead,
    // compute.  One pass walks the hidden dimension with the accumulators in
    // registers; its tile count is fixed for the pass, so the inner loop has
    // no branch around the products.
    int st = 0;
    auto step = [&]() {
        if (cpt == CPT_HI) wait_vmcnt<CPT_HI * (kLmDepth - 1)>();
        else wait_vmcnt<CPT_LO * (kLmDepth - 1)>();
        lds_barrier();
        dma_next(st == 0 ? kLmStages - 1 : st - 1);
    };
    auto pass = [&](int p, auto ntiles) {
        constexpr int NT = decltype(ntiles)::value;
        if constexpr (NT == 0) {
            // no vocabulary left for this wavefront: keep the pipeline's pace
            for (int ks = 0; ks < a.nk; ++ks) {
                step();
                st = st == kLmStages - 1 ? 0 : st + 1;
            }
        } else {
            f32x16_t acc[NT][MT];
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int n = 0; n < MT; ++n) acc[t][n] = f32x16_t{};
            auto walk = [&](auto mv) {
                int ks = 0;
                do {  // nk >= 1
                    step();
                    compute(st, acc, mv);
                    st = st == kLmStages - 1 ? 0 : st + 1;
                } while (++ks < a.nk);
            };
            with_count<MT>(mtv, walk);
            end_pass(p, acc);
        }
    };
    for (int mc = 0; mc < a.nchunks; ++mc) {
        {
            const int r0 = mc * a.chunk_rows;
            const int left = min(a.T, r0 + a.chunk_rows) - r0 - wg * MT * 32;
            mtv = __builtin_amdgcn_readfirstlane(min(MT, max(0, (left + 31) / 32)));
        }
        for (int p = 0; p < a.passes; ++p) {
            const int nt = min(2, max(0, wtiles - 2 * p));
            if (nt == 2) pass(p, std::integral_constant<int, 2>{});
            else if (nt == 1) pass(p, std::integral_constant<int, 1>{});
            else pass(p, std::integral_constant<int, 0>{});
        }
        end_chunk(mc);
    }
    // no global->LDS load may still be writing when the workgroup's LDS is freed
    wait_vmcnt<0>();
}

template <int MT>
void launch_lmhead(const LArgs& a, const uint16_t* hid, const uint16_t* wt, uint64_t* partial,
                   hipStream_t stream) {
    hipLaunchKernelGGL(lmhead_argmax<MT>, dim3(a.nwg), dim3(kLmThreads), 0, stream, a, hid, wt,
                       partial);
}

struct LmPlan {
    LArgs a;
    int mt;
    size_t partial_bytes, argmax_bytes;
};

int lm_cus() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) {
        (void)hipGetLastError();
        v = 256;
    }
    return v;
}

bool lm_args_ok(int32_t num_seqs, int32_t total_q, int32_t hidden_size, int64_t vocab) {
    return num_seqs >= 0 && total_q >= 0 && hidden_size >= kLmStep && hidden_size % kLmStep == 0 &&
           vocab >= 1 && vocab < (int64_t)0x7fffffff;
}

LmPlan plan_lmhead(int32_t total_q, int32_t hidden_size, int64_t vocab) {
    LmPlan pl{};
    LArgs& a = pl.a;
    a.T = total_q;
    a.H = hidden_size;
    a.V = (int)vocab;
    a.nwg = (int)std::min<int64_t>(lm_cus(), vocab);
    constexpr int max_rows = kLmRowGroups * kLmMaxTiles * 32;
    a.nchunks = std::max(1, (total_q + max_rows - 1) / max_rows);
    a.chunk_rows = std::max(1, (total_q + a.nchunks - 1) / a.nchunks);
    pl.mt = (a.chunk_rows + kLmRowGroups * 32 - 1) / (kLmRowGroups * 32);
    const int64_t wg_len = (vocab + a.nwg - 1) / a.nwg;
    const int64_t q_len = (wg_len + kLmQuarters - 1) / kLmQuarters;
    const int64_t tiles = (q_len + 31) / 32;
    a.passes = (int)std::max<int64_t>(1, (tiles + 1) / 2);
    a.nk = hidden_size / kLmStep;
    pl.partial_bytes = align_up((size_t)total_q * a.nwg * sizeof(uint64_t), 256);
    pl.argmax_bytes = align_up((size_t)total_q * sizeof(int32_t), 256);
    return pl;
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_lmhead_accept_workspace_size(int32_t num_seqs, int32_t total_q,
                                                   int32_t hidden_size, int64_t vocab,
                                                   int32_t dtype, size_t* bytes) {
    if (!bytes) return VERIFY_EINVAL;
    if (dtype != VERIFY_BF16) return dtype == VERIFY_F32 ? VERIFY_EUNSUPPORTED : VERIFY_EINVAL;
    if (!lm_args_ok(num_seqs, total_q, hidden_size, vocab)) return VERIFY_EINVAL;
    const LmPlan pl = plan_lmhead(total_q, hidden_size, vocab);
    *bytes = pl.partial_bytes + pl.argmax_bytes;
    return VERIFY_OK;
}

extern "C" int verify_lmhead_accept(int32_t num_seqs, int32_t total_q, int32_t hidden_size,
                                    int64_t vocab, int32_t dtype, const void* hidden,
                                    const void* weight, const int32_t* tokens,
                                    const int32_t* q_start, int32_t* argmax_out,
                                    int32_t* accept_len, int32_t* num_emitted, int32_t* emitted,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (dtype != VERIFY_BF16) return dtype == VERIFY_F32 ? VERIFY_EUNSUPPORTED : VERIFY_EINVAL;
    if (!lm_args_ok(num_seqs, total_q, hidden_size, vocab)) return VERIFY_EINVAL;
    if (num_seqs > 0 && (!q_start || !accept_len || !num_emitted)) return VERIFY_EINVAL;
    if (total_q > 0 && (!hidden || !weight || !tokens || !emitted)) return VERIFY_EINVAL;
    // rows are copied in 16-byte pieces
    if (((uintptr_t)hidden | (uintptr_t)weight) & 15u) return VERIFY_EINVAL;
    const LmPlan pl = plan_lmhead(total_q, hidden_size, vocab);
    const size_t need = pl.partial_bytes + pl.argmax_bytes;
    if (workspace_bytes < need || (need > 0 && !workspace)) return VERIFY_EWORKSPACE;
    if (num_seqs == 0) return VERIFY_OK;
    uint64_t* partial = static_cast<uint64_t*>(workspace);
    int32_t* am = argmax_out ? argmax_out
                             : reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + pl.partial_bytes);
    if (total_q > 0) {
        const uint16_t* hs = static_cast<const uint16_t*>(hidden);
        const uint16_t* ws = static_cast<const uint16_t*>(weight);
        switch (pl.mt) {
            case 1: launch_lmhead<1>(pl.a, hs, ws, partial, stream); break;
            case 2: launch_lmhead<2>(pl.a, hs, ws, partial, stream); break;
            case 3: launch_lmhead<3>(pl.a, hs, ws, partial, stream); break;
            default: return VERIFY_EUNSUPPORTED;
        }
        if (check_launch() != VERIFY_OK) return VERIFY_EHIP;
    }
    return launch_accept_scan(num_seqs, q_start, tokens, partial, pl.a.nwg, am, accept_len,
                              num_emitted, emitted, stream);
}
