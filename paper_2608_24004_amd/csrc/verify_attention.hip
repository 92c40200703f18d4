// verify_attention.hip -- multi-query paged GQA attention of the speculative
// verify pass (paper Sec. 2.2: the target model scores every proposed token
// of every request in one pass; Sec. 3.1: the per-step verification cost is
// what decides whether speculation pays off at large batch).
//
// Work decomposition.  A work item is (request i, KV head g, row group, split
// s): the rows are the G * n_i query rows (G = Hq/Hkv q-heads sharing KV head
// g, times the n_i = k_i + 1 positions of the request), the split is a run of
// consecutive 16-token KV blocks.  One workgroup of four wavefronts handles a
// work item; its wavefronts take the split's blocks round-robin, each keeps an
// online-softmax state (running max, running sum, unnormalised output) per row,
// and the four states are merged through LDS at the end.  A request whose keys
// fit one split writes its output directly; otherwise every split writes a
// normalised partial output and its log-sum-exp, and attn_combine merges them.
//
// Masks.  Row j of request i sits at position p = S_i - n_i + j and sees keys
// t <= p, and with a sliding window W only t > p - W; the walk covers the
// union of the rows' visible blocks only.
#include "common.h"

namespace averify {
namespace {

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kValuRows = 8;  // query rows per VALU work item
constexpr float kLog2e = 1.4426950408889634f;

struct AttnArgs {
    const void* q;
    const void* kc;
    const void* vc;
    const int32_t* block_tables;
    const int32_t* seq_lens;
    const int32_t* q_start;
    void* out;
    float* part_o;    // [total_q][Hq][max_splits][D]   normalised partial outputs
    float* part_lse;  // [total_q][Hq][max_splits]      log2-sum-exp of each split
    int num_seqs, hq, hkv, group, max_blocks, num_blocks, window, max_seq_len;
    float scale_log2;  // softmax scale * log2(e): scores live in the log2 domain
    int split_blocks, max_splits, row_groups;
};

// Per-request geometry, recomputed identically by every kernel.
struct SeqGeom {
    int q0, n, S, b_lo, b_hi, nsplit;
};

__device__ __forceinline__ SeqGeom seq_geom(const AttnArgs& a, int i) {
    SeqGeom g;
    g.q0 = a.q_start[i];
    g.n = a.q_start[i + 1] - g.q0;
    int S = a.seq_lens[i];
    S = max(0, min(S, min(a.max_seq_len, a.max_blocks * kBlockTokens)));
    g.S = S;
    const int key_lo = a.window > 0 ? max(0, S - g.n - a.window + 1) : 0;
    g.b_lo = key_lo / kBlockTokens;
    g.b_hi = (S + kBlockTokens - 1) / kBlockTokens;
    const int nb = max(0, g.b_hi - g.b_lo);
    g.nsplit = min(a.max_splits, (nb + a.split_blocks - 1) / a.split_blocks);
    return g;
}

// ------------------------------------------------------------------ VALU path
//
// Lane layout inside a wavefront, per 16-token block:
//   scores  lane = t + 16*dq: key t, dimension quarter dq; the partial dot
//           products of the four quarters are summed with two xor-shuffles;
//   output  lane owns D/64 consecutive output dimensions, reading V^T rows
//           (16 keys of one dimension are contiguous in the V layout) and the
//           16 probabilities of the block broadcast through readlane.
template <typename T, int D>
__global__ __launch_bounds__(kAttnThreads) void attn_valu(AttnArgs a) {
    constexpr int X = Storage<T>::kPer16B;  // elements per 16 bytes
    constexpr int NC = D / X;               // 16-byte chunks per key
    constexpr int CPL = NC / 4;             // chunks per lane
    constexpr int DPL = D / kWave;          // output dimensions per lane
    constexpr int RB = kValuRows;
    constexpr int VCH = kBlockTokens / X;   // 16-byte chunks per V^T row
    static_assert(NC % 4 == 0 && D % kWave == 0, "head_dim");

    const int i = blockIdx.z;
    const int kvh = blockIdx.y / a.row_groups;
    const int rg = blockIdx.y - kvh * a.row_groups;
    const int s = blockIdx.x;
    const SeqGeom sg = seq_geom(a, i);
    const int rows_total = a.group * sg.n;
    const int r0 = rg * RB;
    if (r0 >= rows_total || s >= sg.nsplit) return;
    const int sb = sg.b_lo + s * a.split_blocks;
    const int se = min(sg.b_hi, sb + a.split_blocks);
    const int nrows = min(RB, rows_total - r0);

    __shared__ float q_s[RB][D];
    __shared__ float merge_o[kAttnWaves][RB][D];
    __shared__ float merge_m[kAttnWaves][RB];
    __shared__ float merge_l[kAttnWaves][RB];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = tid / kWave;
    const T* qp = static_cast<const T*>(a.q);
    for (int e = tid; e < RB * D; e += kAttnThreads) {
        const int r = e / D, d = e - r * D;
        float v = 0.f;
        if (r < nrows) {
            const int rr = r0 + r;
            const int j = rr / a.group, gh = rr - j * a.group;
            const int64_t qrow = sg.q0 + j;
            v = Storage<T>::load(qp, (qrow * a.hq + kvh * a.group + gh) * D + d) * a.scale_log2;
        }
        q_s[r][d] = v;
    }
    __syncthreads();

    float m_r[RB], l_r[RB], o[RB][DPL];
    int pos_r[RB], lo_r[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        m_r[r] = -INFINITY;
        l_r[r] = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[r][e] = 0.f;
        const int j = (r0 + r) / a.group;
        pos_r[r] = sg.S - sg.n + j;
        lo_r[r] = a.window > 0 ? pos_r[r] - a.window + 1 : 0;
    }

    const int t = lane & 15, dq = lane >> 4;
    const T* kc = static_cast<const T*>(a.kc);
    const T* vc = static_cast<const T*>(a.vc);
    const int64_t tile = (int64_t)kBlockTokens * D;
    const int32_t* btab = a.block_tables + (int64_t)i * a.max_blocks;

    for (int b = sb + w; b < se; b += kAttnWaves) {
        const int phys = btab[b];
        if (phys < 0 || phys >= a.num_blocks) continue;
        const T* ktile = kc + ((int64_t)phys * a.hkv + kvh) * tile;
        const T* vtile = vc + ((int64_t)phys * a.hkv + kvh) * tile;
        float kf[CPL * X];
#pragma unroll
        for (int u = 0; u < CPL; ++u)
            unpack16(ld16(ktile + ((dq * CPL + u) * kBlockTokens + t) * X), &kf[u * X], T());
        float vf[DPL][kBlockTokens];
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            const T* vrow = vtile + (lane * DPL + e) * kBlockTokens;
#pragma unroll
            for (int c = 0; c < VCH; ++c) unpack16(ld16(vrow + c * X), &vf[e][c * X], T());
        }
        const int tk = b * kBlockTokens + t;

#pragma unroll
        for (int r = 0; r < RB; ++r) {
            if (r >= nrows) break;
            float sc = 0.f;
#pragma unroll
            for (int u = 0; u < CPL; ++u) {
                const float* qv = &q_s[r][(dq * CPL + u) * X];
#pragma unroll
                for (int e = 0; e < X; ++e) sc = fmaf(qv[e], kf[u * X + e], sc);
            }
            sc += __shfl_xor(sc, 16);
            sc += __shfl_xor(sc, 32);
            const bool vis = tk <= pos_r[r] && tk >= lo_r[r];
            sc = vis ? sc : -INFINITY;
            const float mx = wave_max_xor(sc, 16);
            const float mnew = fmaxf(m_r[r], mx);
            const float muse = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = exp2f(m_r[r] - muse);
            const float pt = exp2f(sc - muse);
            l_r[r] = l_r[r] * alpha + wave_sum_xor(pt, 16);
            m_r[r] = mnew;
            float acc[DPL];
#pragma unroll
            for (int e = 0; e < DPL; ++e) acc[e] = o[r][e] * alpha;
#pragma unroll
            for (int tt = 0; tt < kBlockTokens; ++tt) {
                const float ptt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pt), tt));
#pragma unroll
                for (int e = 0; e < DPL; ++e) acc[e] = fmaf(ptt, vf[e][tt], acc[e]);
            }
#pragma unroll
            for (int e = 0; e < DPL; ++e) o[r][e] = acc[e];
        }
    }

    // merge the four wavefronts' states
#pragma unroll
    for (int r = 0; r < RB; ++r) {
        if (lane == 0) {
            merge_m[w][r] = m_r[r];
            merge_l[w][r] = l_r[r];
        }
#pragma unroll
        for (int e = 0; e < DPL; ++e) merge_o[w][r][lane * DPL + e] = o[r][e];
    }
    __syncthreads();
    T* outp = static_cast<T*>(a.out);
    for (int e = tid; e < nrows * D; e += kAttnThreads) {
        const int r = e / D, d = e - r * D;
        float M = -INFINITY;
#pragma unroll
        for (int ww = 0; ww < kAttnWaves; ++ww) M = fmaxf(M, merge_m[ww][r]);
        float L = 0.f, O = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int ww = 0; ww < kAttnWaves; ++ww) {
                const float f = exp2f(merge_m[ww][r] - M);
                L = fmaf(f, merge_l[ww][r], L);
                O = fmaf(f, merge_o[ww][r][d], O);
            }
        }
        const int rr = r0 + r;
        const int j = rr / a.group, gh = rr - j * a.group;
        const int64_t hrow = (int64_t)(sg.q0 + j) * a.hq + kvh * a.group + gh;
        const float val = L > 0.f ? O / L : 0.f;
        if (sg.nsplit == 1) {
            Storage<T>::store(outp, hrow * D + d, val);
        } else {
            const int64_t pi = hrow * a.max_splits + s;
            a.part_o[pi * D + d] = val;
            if (d == 0) a.part_lse[pi] = L > 0.f ? M + log2f(L) : -INFINITY;
        }
    }
}

// ------------------------------------------------------------------ MFMA path (bf16)
//
// Work item as for the VALU path, with up to NW*TPW*16 rows.  The workgroup's
// NW wavefronts split the query rows (TPW tiles of 16 rows each) and share the
// KV blocks: every block's K and V tiles (16 tokens x D, contiguous in the
// paged layout) are loaded once per workgroup with 16-byte coalesced loads,
// staged through a double-buffered LDS ring, and read by every wavefront as
// MFMA operands.  Two blocks are in flight in registers while the current one
// is consumed.
//
// Per block and 16-row tile, with lane = 16*lg + l16:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, A = K (16 keys x 32 dims, lane
//                 holds 8 consecutive dims of key l16: one 16-byte LDS read
//                 of the x-packed K tile), B = Q^T (8 dims of row l16);
//                 result lane holds keys 4lg..4lg+3 of row l16;
//   O^T += V^T P^T v_mfma_f32_16x16x16_bf16, A = V^T (dims x 16 keys, lane
//                 holds 4 keys of dim l16: one 8-byte read of the V^T tile),
//                 B = P^T (the same 4 keys of row l16, straight from the S
//                 registers after the online-softmax update).
// The output tile is O^T: lane holds dims 4lg..4lg+3 of row l16, so a row's
// state (running max, rescale factor) lives in the lanes that own its scores.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8_t, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

template <int D, int NW, int TPW>
__global__ __launch_bounds__(NW * kWave) void attn_mfma(AttnArgs a) {
    constexpr int NT = NW * kWave;
    constexpr int TILE_BYTES = kBlockTokens * D * 2;  // one (block, head) K or V tile
    constexpr int CH = 2 * TILE_BYTES / 16;           // 16-byte chunks per block (K then V)
    constexpr int CPT = (CH + NT - 1) / NT;           // chunks per thread per block
    constexpr int KC = D / 32;                        // QK^T steps of 32 dims
    constexpr int DT = D / 16;                        // PV output tiles of 16 dims
    constexpr int ROWS = NW * TPW * 16;

    __shared__ __attribute__((aligned(16))) uint8_t stage[2][2 * TILE_BYTES];

    const int i = blockIdx.z;
    const int kvh = blockIdx.y / a.row_groups;
    const int rg = blockIdx.y - kvh * a.row_groups;
    const int s = blockIdx.x;
    const SeqGeom sg = seq_geom(a, i);
    const int rows_total = a.group * sg.n;
    const int r0 = rg * ROWS;
    if (r0 >= rows_total || s >= sg.nsplit) return;
    const int sb = sg.b_lo + s * a.split_blocks;
    const int se = min(sg.b_hi, sb + a.split_blocks);

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int w = tid / kWave;
    const int l16 = lane & 15, lg = lane >> 4;
    const int wrow0 = r0 + w * TPW * 16;          // first row of this wavefront
    const bool active = wrow0 < rows_total;       // wavefront-uniform

    // Q operands of this lane's rows (zeros for padding rows)
    bf16x8_t qop[TPW][KC];
    int row_j[TPW];
    const uint16_t* qp = static_cast<const uint16_t*>(a.q);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        const int rr = wrow0 + t * 16 + l16;
        const bool valid = rr < rows_total;
        const int j = rr / a.group, gh = rr - j * a.group;
        row_j[t] = valid ? j : -1;
        const int64_t base = ((int64_t)(sg.q0 + j) * a.hq + kvh * a.group + gh) * D;
#pragma unroll
        for (int cc = 0; cc < KC; ++cc) {
            uint4 v = make_uint4(0, 0, 0, 0);
            if (valid) v = ld16(qp + base + (cc * 4 + lg) * 8);
            qop[t][cc] = as_bf16x8(v);
        }
    }

    f32x4_t o[TPW][DT];
    float m_r[TPW], l_r[TPW];
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        m_r[t] = -INFINITY;
        l_r[t] = 0.f;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[t][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }

    const uint8_t* kbase = static_cast<const uint8_t*>(a.kc);
    const uint8_t* vbase = static_cast<const uint8_t*>(a.vc);
    const int32_t* btab = a.block_tables + (int64_t)i * a.max_blocks;
    const int p_first = sg.S - sg.n;   // position of the request's first query row

    auto load_block = [&](int b, uint4* regs) {
        const int phys = btab[b];
        if (phys < 0 || phys >= a.num_blocks) return;
        const int64_t off = ((int64_t)phys * a.hkv + kvh) * TILE_BYTES;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            const int idx = tid + c * NT;
            if (CH % NT == 0 || idx < CH) {
                const uint8_t* src = idx < CH / 2 ? kbase + off + idx * 16 : vbase + off + (idx - CH / 2) * 16;
                regs[c] = ld16(src);
            }
        }
    };
    auto store_block = [&](int st, const uint4* regs) {
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            const int idx = tid + c * NT;
            if (CH % NT == 0 || idx < CH) *reinterpret_cast<uint4*>(&stage[st][idx * 16]) = regs[c];
        }
    };
    auto compute = [&](int st, int b) {
        const int phys = btab[b];
        if (!active || phys < 0 || phys >= a.num_blocks) return;
        const uint8_t* ks = stage[st];
        const uint8_t* vs = stage[st] + TILE_BYTES;
        f32x4_t sacc[TPW];
#pragma unroll
        for (int t = 0; t < TPW; ++t) sacc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int cc = 0; cc < KC; ++cc) {
            const bf16x8_t kop = as_bf16x8(*reinterpret_cast<const uint4*>(ks + ((cc * 4 + lg) * 16 + l16) * 16));
#pragma unroll
            for (int t = 0; t < TPW; ++t)
                sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[t][cc], sacc[t], 0, 0, 0);
        }
        const int key0 = b * kBlockTokens + 4 * lg;
        // blocks entirely below the first row's position and inside the last
        // row's window need no mask
        const bool need_mask = (b * kBlockTokens + kBlockTokens - 1 > p_first) ||
                               (a.window > 0 && b * kBlockTokens < sg.S - a.window);
        i16x4_t pop[TPW];
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            float sv[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) sv[r] = sacc[t][r] * a.scale_log2;
            if (need_mask) {
                const int p = p_first + row_j[t];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int key = key0 + r;
                    const bool vis = row_j[t] >= 0 && key <= p && (a.window == 0 || key > p - a.window);
                    sv[r] = vis ? sv[r] : -INFINITY;
                }
            }
            float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
            mx = fmaxf(mx, __shfl_xor(mx, 16));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mnew = fmaxf(m_r[t], mx);
            const float muse = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = exp2f(m_r[t] - muse);
            float pr[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) pr[r] = exp2f(sv[r] - muse);
            l_r[t] = l_r[t] * alpha + ((pr[0] + pr[1]) + (pr[2] + pr[3]));
            m_r[t] = mnew;
            const uint32_t lo = pack_bf16x2(pr[0], pr[1]), hi = pack_bf16x2(pr[2], pr[3]);
            pop[t] = __builtin_bit_cast(i16x4_t, make_uint2(lo, hi));
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[t][dt] *= alpha;
        }
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const uint2 vv = *reinterpret_cast<const uint2*>(vs + (dt * 16 + l16) * 32 + lg * 8);
            const i16x4_t vop = __builtin_bit_cast(i16x4_t, vv);
#pragma unroll
            for (int t = 0; t < TPW; ++t)
                o[t][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, pop[t], o[t][dt], 0, 0, 0);
        }
    };

    // double-buffered LDS ring fed by two register sets
    uint4 pa[CPT], pb[CPT];
    if (sb < se) load_block(sb, pa);
    if (sb + 1 < se) load_block(sb + 1, pb);
    if (sb < se) store_block(0, pa);
    if (sb + 2 < se) load_block(sb + 2, pa);
    __syncthreads();
    for (int b = sb; b < se; b += 2) {
        compute(0, b);
        if (b + 1 < se) store_block(1, pb);
        if (b + 3 < se) load_block(b + 3, pb);
        __syncthreads();
        if (b + 1 >= se) break;
        compute(1, b + 1);
        if (b + 2 < se) store_block(0, pa);
        if (b + 4 < se) load_block(b + 4, pa);
        __syncthreads();
    }

    if (!active) return;
    uint16_t* outp = static_cast<uint16_t*>(a.out);
#pragma unroll
    for (int t = 0; t < TPW; ++t) {
        float L = l_r[t];
        L += __shfl_xor(L, 16);
        L += __shfl_xor(L, 32);
        const int rr = wrow0 + t * 16 + l16;
        if (rr >= rows_total) continue;
        const int j = rr / a.group, gh = rr - j * a.group;
        const int64_t hrow = (int64_t)(sg.q0 + j) * a.hq + kvh * a.group + gh;
        const float inv = L > 0.f ? 1.f / L : 0.f;
        if (sg.nsplit == 1) {
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const int d0 = dt * 16 + 4 * lg;
                const uint2 v = make_uint2(pack_bf16x2(o[t][dt][0] * inv, o[t][dt][1] * inv),
                                           pack_bf16x2(o[t][dt][2] * inv, o[t][dt][3] * inv));
                *reinterpret_cast<uint2*>(outp + hrow * D + d0) = v;
            }
        } else {
            const int64_t pi = hrow * a.max_splits + s;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const int d0 = dt * 16 + 4 * lg;
                *reinterpret_cast<f32x4_t*>(a.part_o + pi * D + d0) = o[t][dt] * inv;
            }
            if (lg == 0) a.part_lse[pi] = L > 0.f ? m_r[t] + log2f(L) : -INFINITY;
        }
    }
}

// ------------------------------------------------------------------ combine
//
// One wavefront per (query row, q-head): log-sum-exp merge of the split
// partials, O = sum_s 2^(lse_s - M) o_s / sum_s 2^(lse_s - M).  Also writes
// the zero output of rows whose request has no key at all.
template <typename T, int D>
__global__ __launch_bounds__(kAttnThreads) void attn_combine(AttnArgs a, int total_q) {
    constexpr int DPL = D / kWave;
    const int64_t item = (int64_t)blockIdx.x * kAttnWaves + threadIdx.x / kWave;
    if (item >= (int64_t)total_q * a.hq) return;
    const int lane = threadIdx.x & (kWave - 1);
    const int row = (int)(item / a.hq);
    // request owning `row`: the largest i with q_start[i] <= row
    int lo = 0, hi = a.num_seqs - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.q_start[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const SeqGeom sg = seq_geom(a, lo);
    if (sg.nsplit == 1) return;
    T* outp = static_cast<T*>(a.out);
    float acc[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
    float L = 0.f;
    if (sg.nsplit > 1) {
        const int64_t pi0 = item * a.max_splits;
        float M = -INFINITY;
        for (int s = 0; s < sg.nsplit; ++s) M = fmaxf(M, a.part_lse[pi0 + s]);
        if (M != -INFINITY) {
            for (int s = 0; s < sg.nsplit; ++s) {
                const float lse = a.part_lse[pi0 + s];
                if (lse == -INFINITY) continue;
                const float f = exp2f(lse - M);
                L += f;
                const float* po = a.part_o + (pi0 + s) * D + lane * DPL;
#pragma unroll
                for (int e = 0; e < DPL; ++e) acc[e] = fmaf(f, po[e], acc[e]);
            }
        }
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e)
        Storage<T>::store(outp, item * D + lane * DPL + e, L > 0.f ? acc[e] / L : 0.f);
}

// ------------------------------------------------------------------ host side

struct AttnPlan {
    bool mfma;        // bf16 storage: MFMA kernel; fp32 storage: VALU kernel
    int nw, tpw;      // MFMA: wavefronts per workgroup, 16-row tiles per wavefront
    int split_blocks;
    int max_splits;
    int row_groups;
    size_t part_o_bytes;
    size_t part_lse_bytes;
};

int validate(const verify_attn_params* p, int32_t total_q, int32_t max_q_len,
             int32_t max_seq_len) {
    if (!p) return VERIFY_EINVAL;
    if (p->dtype != VERIFY_F32 && p->dtype != VERIFY_BF16) return VERIFY_EUNSUPPORTED;
    if (p->head_dim != 64 && p->head_dim != 128) return VERIFY_EUNSUPPORTED;
    if (p->block_size != kBlockTokens) return VERIFY_EUNSUPPORTED;
    if (p->num_seqs < 0 || p->num_q_heads <= 0 || p->num_kv_heads <= 0) return VERIFY_EINVAL;
    if (p->num_q_heads % p->num_kv_heads != 0) return VERIFY_EINVAL;
    if (p->max_blocks_per_seq <= 0 || p->num_blocks < 0 || p->sliding_window < 0) return VERIFY_EINVAL;
    if (p->kv_split_blocks < 0 || !(p->scale >= 0.f) || p->scale > 3.0e38f) return VERIFY_EINVAL;
    if (total_q < 0 || max_q_len < 0 || max_seq_len < 0) return VERIFY_EINVAL;
    if (p->num_seqs > 65535) return VERIFY_EUNSUPPORTED;
    return VERIFY_OK;
}

AttnPlan make_plan(const verify_attn_params* p, int32_t total_q, int32_t max_q_len,
                   int32_t max_seq_len) {
    AttnPlan pl{};
    const int G = p->num_q_heads / p->num_kv_heads;
    int64_t nb_max = ((int64_t)max_seq_len + kBlockTokens - 1) / kBlockTokens;
    if (p->sliding_window > 0) {
        const int64_t span = (int64_t)p->sliding_window + max_q_len - 1;
        nb_max = std::min<int64_t>(nb_max, (span + kBlockTokens - 1) / kBlockTokens + 1);
    }
    nb_max = std::max<int64_t>(nb_max, 1);
    int sb = p->kv_split_blocks;
    if (sb == 0) {
        // aim for about 8192 work items over the batch, at least 32 blocks per split
        const int64_t total = (int64_t)std::max(1, p->num_seqs) * p->num_kv_heads * nb_max;
        int64_t want = (total + 8191) / 8192;
        want = std::max<int64_t>(32, (want + 3) / 4 * 4);
        sb = (int)std::min<int64_t>(want, nb_max);
    }
    pl.split_blocks = std::max(1, sb);
    pl.max_splits = (int)((nb_max + pl.split_blocks - 1) / pl.split_blocks);
    const int64_t rows = (int64_t)G * std::max(1, max_q_len);
    pl.mfma = p->dtype == VERIFY_BF16;
    if (pl.mfma) {
        const int64_t tiles = (rows + 15) / 16;
        if (tiles <= 8) { pl.tpw = 1; pl.nw = (int)std::max<int64_t>(2, tiles); }
        else if (tiles <= 16) { pl.tpw = 2; pl.nw = (int)((tiles + 1) / 2); }
        else { pl.tpw = 2; pl.nw = 8; }
        const int64_t per = (int64_t)pl.nw * pl.tpw * 16;
        pl.row_groups = (int)((rows + per - 1) / per);
    } else {
        pl.row_groups = (int)((rows + kValuRows - 1) / kValuRows);
    }
    if (pl.max_splits > 1) {
        const size_t items = (size_t)total_q * p->num_q_heads * pl.max_splits;
        pl.part_o_bytes = align_up(items * p->head_dim * sizeof(float), 256);
        pl.part_lse_bytes = align_up(items * sizeof(float), 256);
    }
    return pl;
}

template <int D, int NW, int TPW>
void launch_mfma_k(const AttnArgs& a, const AttnPlan& pl, hipStream_t stream) {
    dim3 grid(pl.max_splits, a.hkv * pl.row_groups, a.num_seqs);
    hipLaunchKernelGGL((attn_mfma<D, NW, TPW>), grid, dim3(NW * kWave), 0, stream, a);
}

template <int D>
void launch_mfma(const AttnArgs& a, const AttnPlan& pl, hipStream_t stream) {
    if (pl.tpw == 1) {
        switch (pl.nw) {
            case 2: launch_mfma_k<D, 2, 1>(a, pl, stream); break;
            case 3: launch_mfma_k<D, 3, 1>(a, pl, stream); break;
            case 4: launch_mfma_k<D, 4, 1>(a, pl, stream); break;
            case 5: launch_mfma_k<D, 5, 1>(a, pl, stream); break;
            case 6: launch_mfma_k<D, 6, 1>(a, pl, stream); break;
            case 7: launch_mfma_k<D, 7, 1>(a, pl, stream); break;
            default: launch_mfma_k<D, 8, 1>(a, pl, stream); break;
        }
    } else {
        switch (pl.nw) {
            case 5: launch_mfma_k<D, 5, 2>(a, pl, stream); break;
            case 6: launch_mfma_k<D, 6, 2>(a, pl, stream); break;
            case 7: launch_mfma_k<D, 7, 2>(a, pl, stream); break;
            default: launch_mfma_k<D, 8, 2>(a, pl, stream); break;
        }
    }
}

template <typename T, int D>
void launch_combine(const AttnArgs& a, int total_q, hipStream_t stream) {
    const int64_t items = (int64_t)total_q * a.hq;
    if (items > 0) {
        dim3 cgrid((unsigned)((items + kAttnWaves - 1) / kAttnWaves));
        hipLaunchKernelGGL((attn_combine<T, D>), cgrid, dim3(kAttnThreads), 0, stream, a, total_q);
    }
}

template <typename T, int D>
void launch(const AttnArgs& a, const AttnPlan& pl, int total_q, hipStream_t stream) {
    if constexpr (sizeof(T) == 2) {
        launch_mfma<D>(a, pl, stream);
    } else {
        dim3 grid(pl.max_splits, a.hkv * pl.row_groups, a.num_seqs);
        hipLaunchKernelGGL((attn_valu<T, D>), grid, dim3(kAttnThreads), 0, stream, a);
    }
    launch_combine<T, D>(a, total_q, stream);
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_attention_workspace_size(const verify_attn_params* params, int32_t total_q,
                                               int32_t max_q_len, int32_t max_seq_len,
                                               size_t* bytes) {
    if (!bytes) return VERIFY_EINVAL;
    const int rc = validate(params, total_q, max_q_len, max_seq_len);
    if (rc != VERIFY_OK) return rc;
    const AttnPlan pl = make_plan(params, total_q, max_q_len, max_seq_len);
    *bytes = pl.part_o_bytes + pl.part_lse_bytes;
    return VERIFY_OK;
}

extern "C" int verify_attention(const verify_attn_params* params, int32_t total_q,
                                int32_t max_q_len, int32_t max_seq_len, const void* q,
                                const void* k_cache, const void* v_cache,
                                const int32_t* block_tables, const int32_t* seq_lens,
                                const int32_t* q_start, void* out, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
    const int rc = validate(params, total_q, max_q_len, max_seq_len);
    if (rc != VERIFY_OK) return rc;
    const verify_attn_params& p = *params;
    if (p.num_seqs > 0 && (!seq_lens || !q_start || !block_tables)) return VERIFY_EINVAL;
    if (total_q > 0 && (!q || !k_cache || !v_cache || !out)) return VERIFY_EINVAL;
    const AttnPlan pl = make_plan(params, total_q, max_q_len, max_seq_len);
    const size_t need = pl.part_o_bytes + pl.part_lse_bytes;
    if (workspace_bytes < need || (need > 0 && !workspace)) return VERIFY_EWORKSPACE;
    if ((int64_t)p.num_kv_heads * pl.row_groups > 65535) return VERIFY_EUNSUPPORTED;
    if (p.num_seqs == 0 || total_q == 0) return VERIFY_OK;

    AttnArgs a{};
    a.q = q;
    a.kc = k_cache;
    a.vc = v_cache;
    a.block_tables = block_tables;
    a.seq_lens = seq_lens;
    a.q_start = q_start;
    a.out = out;
    a.part_o = need ? static_cast<float*>(workspace) : nullptr;
    a.part_lse = need ? reinterpret_cast<float*>(static_cast<char*>(workspace) + pl.part_o_bytes)
                      : nullptr;
    a.num_seqs = p.num_seqs;
    a.hq = p.num_q_heads;
    a.hkv = p.num_kv_heads;
    a.group = p.num_q_heads / p.num_kv_heads;
    a.max_blocks = p.max_blocks_per_seq;
    a.num_blocks = p.num_blocks;
    a.window = p.sliding_window;
    a.max_seq_len = max_seq_len;
    const float scale = p.scale > 0.f ? p.scale : 1.0f / sqrtf((float)p.head_dim);
    a.scale_log2 = scale * kLog2e;
    a.split_blocks = pl.split_blocks;
    a.max_splits = pl.max_splits;
    a.row_groups = pl.row_groups;

    if (p.dtype == VERIFY_BF16) {
        if (p.head_dim == 128) launch<uint16_t, 128>(a, pl, total_q, stream);
        else launch<uint16_t, 64>(a, pl, total_q, stream);
    } else {
        if (p.head_dim == 128) launch<float, 128>(a, pl, total_q, stream);
        else launch<float, 64>(a, pl, total_q, stream);
    }
    return check_launch();
}

extern "C" const char* verify_status_string(int status) {
    switch (status) {
        case VERIFY_OK: return "ok";
        case VERIFY_EINVAL: return "invalid argument";
        case VERIFY_EUNSUPPORTED: return "unsupported shape or dtype";
        case VERIFY_EWORKSPACE: return "workspace too small";
        case VERIFY_EHIP: return "HIP launch failure";
        default: return "unknown status";
    }
}

extern "C" int verify_abi_version(void) { return 10000; }
