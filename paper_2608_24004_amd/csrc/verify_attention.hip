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
#include <atomic>

#include "common.h"

// m0 is set inside the global->LDS load sequence (see dma16); the compiler
// reloads m0 before each of its own uses, so clobbering it there is safe.
#pragma clang diagnostic ignored "-Winline-asm"

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
    const float* sinks;  // [Hq] sink logits (natural-log units) or null
    const void* k_new;   // fused append: [total_q][Hkv][D] new keys and values, or null
    const void* v_new;
    int num_seqs, hq, hkv, group, max_blocks, num_blocks, window, max_seq_len;
    float scale_log2;  // softmax scale * log2(e): scores live in the log2 domain
    int split_blocks, max_splits, row_groups;
};

// A head's attention sink is one more logit in each row's softmax with a zero
// value: it adds 2^(sink log2(e) - m) to the row's denominator, with m the
// maximum the row's sums are relative to (0 without sinks; for a row with no
// key, m = -inf makes it infinite and the output 0).
__device__ __forceinline__ float sink_term(const float* sinks, int h, float m) {
    return sinks ? exp2f(sinks[h] * kLog2e - m) : 0.f;
}

// Per-request geometry, recomputed identically by every kernel.
struct SeqGeom {
    int q0, n, S, b_lo, b_hi, nsplit;
    int s_raw;  // seq_lens[i] before clamping: the new tokens sit at s_raw - n .. s_raw - 1
};

__device__ __forceinline__ SeqGeom seq_geom(const AttnArgs& a, int i) {
    SeqGeom g;
    g.q0 = a.q_start[i];
    g.n = a.q_start[i + 1] - g.q0;
    int S = a.seq_lens[i];
    g.s_raw = S;
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
// APPEND: the fused KV append (verify_attention_append).  Keys and values of
// the request's new tokens are read from k_new / v_new instead of the cache,
// and the work items of row group 0 (splits cover disjoint blocks) store them
// into the cache as well.
template <typename T, int D, bool APPEND>
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
    // APPEND: new-token positions the walk reaches, and the first row's position
    const int p0 = sg.s_raw - sg.n;
    const int nlo = max(p0, 0), nhi = min(sg.s_raw, sg.S);
    const T* knew = static_cast<const T*>(a.k_new);
    const T* vnew = static_cast<const T*>(a.v_new);

    for (int b = sb + w; b < se; b += kAttnWaves) {
        const int phys = btab[b];
        if (phys < 0 || phys >= a.num_blocks) continue;
        const T* ktile = kc + ((int64_t)phys * a.hkv + kvh) * tile;
        const T* vtile = vc + ((int64_t)phys * a.hkv + kvh) * tile;
        const int tk = b * kBlockTokens + t;
        // APPEND: a new token's key comes from k_new (its row's 16-byte chunks)
        const bool knew_t = APPEND && tk >= nlo && tk < nhi;
        const int64_t nrow = (int64_t)sg.q0 + (tk - p0);
        float kf[CPL * X];
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
            const int c16 = dq * CPL + u;
            const T* kp = knew_t ? knew + (nrow * a.hkv + kvh) * D + c16 * X
                                 : ktile + (c16 * kBlockTokens + t) * X;
            const uint4 kraw = ld16(kp);
            if (APPEND && knew_t && rg == 0)
                *reinterpret_cast<uint4*>(const_cast<T*>(ktile) + (c16 * kBlockTokens + t) * X) = kraw;
            unpack16(kraw, &kf[u * X], T());
        }
        float vf[DPL][kBlockTokens];
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            const T* vrow = vtile + (lane * DPL + e) * kBlockTokens;
#pragma unroll
            for (int c = 0; c < VCH; ++c) unpack16(ld16(vrow + c * X), &vf[e][c * X], T());
        }
        if (APPEND && b * kBlockTokens < nhi && (b + 1) * kBlockTokens > nlo) {
            // the new tokens' values: dimension lane * DPL + e of row
            // q0 + (position - p0), for the block's new positions
#pragma unroll
            for (int tt = 0; tt < kBlockTokens; ++tt) {
                const int pos = b * kBlockTokens + tt;
                if (pos < nlo || pos >= nhi) continue;
                const int64_t vrow_new = ((int64_t)sg.q0 + (pos - p0)) * a.hkv + kvh;
#pragma unroll
                for (int e = 0; e < DPL; ++e) {
                    const int d = lane * DPL + e;
                    const T v = vnew[vrow_new * D + d];
                    vf[e][tt] = Storage<T>::load(&v, 0);
                    if (rg == 0) const_cast<T*>(vtile)[d * kBlockTokens + tt] = v;
                }
            }
        }

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
        if (sg.nsplit == 1) {
            const float den = L + sink_term(a.sinks, kvh * a.group + gh, M);
            Storage<T>::store(outp, hrow * D + d, den > 0.f ? O / den : 0.f);
        } else {
            const float val = L > 0.f ? O / L : 0.f;
            const int64_t pi = hrow * a.max_splits + s;
            a.part_o[pi * D + d] = val;
            if (d == 0) a.part_lse[pi] = L > 0.f ? M + log2f(L) : -INFINITY;
        }
    }
}

// ------------------------------------------------------------------ MFMA path (bf16)
//
// Persistent, load-balanced schedule.  A unit is one 16-token KV block of one
// (request i, KV head g, row group) pair; units are numbered request by
// request, then head, then row group, then block.  attn_schedule writes the
// per-request unit offsets (a prefix sum over the batch), then attn_persist
// launches a fixed number of workgroups (all resident at once) and gives
// workgroup w the contiguous unit range [U*w/N, U*(w+1)/N), N = min(NWG, U): every
// workgroup streams the same number of KV bytes whatever the context lengths,
// so no workgroup is left running alone at the end.  A pair whose units all
// fall in one range is finished in place; a pair cut by a range boundary
// leaves one partial (normalised output + log-sum-exp) per workgroup in slot
// P + w (P = pair index), and attn_combine_slots merges them.
//
// Inside a workgroup the NW wavefronts split the pair's query rows (TPW tiles
// of 16 rows each) and share the KV blocks: each block's K and V tiles (16
// tokens x D, contiguous in the paged layout) are copied once, 16 bytes per
// lane, straight from global memory into a ring of PD + 1 LDS stages (PD
// blocks in flight), and read from there by every wavefront as MFMA operands.
// The load stream runs straight across pair boundaries; the block id of each
// block it loads is a scalar load issued one block earlier.
//
// Per block and 16-row tile, with lane = 16*lg + l16:
//   S^T = K Q^T   v_mfma_f32_16x16x32_bf16, A = K (16 keys x 32 dims, lane
//                 holds 8 consecutive dims of key l16: one 16-byte LDS read
//                 of the x-packed K tile), B = Q^T (8 dims of row l16);
//                 the result lane holds keys 4lg..4lg+3 of row l16;
//   O^T += V^T P^T v_mfma_f32_16x16x16_bf16, A = V^T (16 dims x 16 keys, lane
//                 holds 4 keys of dim l16: one 8-byte read of the V^T tile),
//                 B = P^T (the same 4 keys of row l16, straight from the S
//                 registers after the online-softmax update).
// The output tile is O^T: lane holds dims 4lg..4lg+3 of row l16, so a row's
// running max and rescale factor live in the lanes that own its scores.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

// Maximum of v over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four lanes that hold
// one row of an MFMA result tile).  Each permlane swap exchanges half of the
// wavefront between its two operands; with both operands equal to v, the two
// results of lane l are v of l and of l ^ 32 (l ^ 16), in some order.
__device__ __forceinline__ float row_max_4lanes(float v) {
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Softmax weights may exceed 1 by up to this factor (log2) before the stored
// row maximum is raised.
constexpr float kSlackLog2 = 8.f;

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8_t as_bf16x8(const uint4& v) { return __builtin_bit_cast(bf16x8_t, v); }


// Scalars of the persistent launch.  The pointers travel as separate
// __restrict__ kernel arguments (MPtrs) so that the compiler can prove the
// metadata arrays are never written by the kernel and read them with scalar
// loads: a vector load there would make every wait on it drain the KV
// prefetch queue.
struct PArgs {
    int num_seqs, hq, hkv, group, max_blocks, num_blocks, window, max_seq_len;
    float scale_log2;
    float inv_scale_log2;  // 1 / scale_log2 (0 when the scale is 0)
    int rows_per_group;   // NW * TPW * 16
    int rg_max;           // row groups per (request, KV head) at most
    int nwg;              // workgroups of the persistent launch
    int spb;              // > 0: fixed number of units per workgroup
    int inline_sched;     // 1: attn_persist computes the unit offsets itself
    int rows_lo, rows_hi; // the launch's row class: requests whose group * n_i lies in
                          // [rows_lo, rows_hi]; the others belong to another launch
    const float* sinks;   // [Hq] sink logits (natural-log units) or null
};

struct MPtrs {
    const uint16_t* q;
    const uint8_t* kc;
    const uint8_t* vc;
    const int32_t* block_tables;
    const int32_t* seq_lens;
    const int32_t* q_start;
    uint16_t* out;
    int32_t* unit_start;  // [num_seqs + 1] first unit of each request (schedule pass)
    uint16_t* slot_o;     // [slots][rows_per_group][D] normalised partial outputs, bf16
                          // (slot_o_index)
    float* slot_lse;      // [slots][rows_per_group]    their log2-sum-exp
    const uint16_t* k_new;  // fused append: [total_q][Hkv][D] new keys, or null
    const uint16_t* v_new;  //               and values
};

struct ReqGeom {
    int q0, n, S, b_lo, nb, rg;
};

// Offset in slot_o of row lr (within the row group), dims d .. d+3 (d % 4 ==
// 0), of slot `slot`.  Each 16-row tile of a slot is stored in the order the
// MFMA output registers hold it: 16-dim column block dt, then lane
// 16 (d / 4 % 4) + lr % 16, then the four dims.  The partial outputs are
// stored in bf16 (the log2-sum-exp in fp32), as a split-K merge usually keeps
// them in the output's type: they are normalised, so rounding them adds at most
// 2^-9 relative error to the merged row, and it halves the bytes written at
// the end of every range and read back by the merge.
template <int D>
__device__ __forceinline__ int64_t slot_o_index(int64_t slot, int rows_per_group, int lr, int d) {
    const int lane = ((d >> 2) & 3) * 16 + (lr & 15);
    return (slot * rows_per_group + (lr & ~15)) * D + ((d >> 4) * kWave + lane) * 4;
}

__device__ __forceinline__ ReqGeom req_geom(const PArgs& a, const int32_t* __restrict__ q_start,
                                            const int32_t* __restrict__ seq_lens, int i) {
    ReqGeom r;
    r.q0 = q_start[i];
    r.n = q_start[i + 1] - r.q0;
    int S = seq_lens[i];
    S = max(0, min(S, min(a.max_seq_len, a.max_blocks * kBlockTokens)));
    r.S = S;
    const int key_lo = a.window > 0 ? max(0, S - r.n - a.window + 1) : 0;
    r.b_lo = key_lo / kBlockTokens;
    const int b_hi = (S + kBlockTokens - 1) / kBlockTokens;
    r.nb = max(0, b_hi - r.b_lo);
    const int rows = a.group * max(0, r.n);
    r.rg = min(a.rg_max, (rows + a.rows_per_group - 1) / a.rows_per_group);
    if (rows < a.rows_lo || rows > a.rows_hi) r.rg = 0;  // another launch's request
    return r;
}

// Rows past the launch's reach: a request with more than max_q_len rows can
// need more row groups than the launch provides (rg_max); those rows are not
// computed, and their outputs are written as a quiet NaN instead of being
// left stale.  Threads t = t0, t0 + nt, ... cover the batch's requests.
template <int D>
__device__ void mark_unreached_rows(const PArgs& a, const int32_t* __restrict__ q_start,
                                    uint16_t* __restrict__ out, int t0, int nt) {
    const int reach = a.rg_max * a.rows_per_group;  // local rows of one (request, KV head)
    for (int i = t0; i < a.num_seqs; i += nt) {
        const int q0 = q_start[i];
        const int rows = a.group * (q_start[i + 1] - q0);
        if (rows < a.rows_lo || rows > a.rows_hi) continue;
        for (int rr = reach; rr < rows; ++rr)
            for (int g = 0; g < a.hkv; ++g) {
                const int64_t hrow = (int64_t)(q0 + rr / a.group) * a.hq + g * a.group + rr % a.group;
                for (int d = 0; d < D; ++d) out[hrow * D + d] = 0x7fc0;  // bf16 quiet NaN
            }
    }
}

// Workgroups that share the U units in equal-share mode: at most one per unit,
// so that every participating workgroup owns at least one unit.
__device__ __forceinline__ int sharing_wgs(const PArgs& a, int U) { return min(a.nwg, max(U, 1)); }

// Workgroup that owns unit u (inverse of the range split).
__device__ __forceinline__ int owner_of(const PArgs& a, int u, int U) {
    if (a.spb > 0) return u / a.spb;
    return (int)(((int64_t)(u + 1) * sharing_wgs(a, U) - 1) / U);
}

// One workgroup: exclusive prefix sum of Hkv * row_groups * blocks over the batch.
template <int D>
__global__ __launch_bounds__(1024) void attn_schedule(PArgs a, const int32_t* __restrict__ q_start,
                                                     const int32_t* __restrict__ seq_lens,
                                                     int32_t* __restrict__ unit_start,
                                                     uint16_t* __restrict__ out) {
    mark_unreached_rows<D>(a, q_start, out, threadIdx.x, blockDim.x);
    __shared__ int wsum[16];
    __shared__ int carry_s;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wv = tid / kWave;
    if (tid == 0) carry_s = 0;
    __syncthreads();
    for (int base = 0; base < a.num_seqs; base += 1024) {
        const int i = base + tid;
        int u = 0;
        if (i < a.num_seqs) {
            const ReqGeom r = req_geom(a, q_start, seq_lens, i);
            u = a.hkv * r.rg * r.nb;
        }
        int x = u;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane == kWave - 1) wsum[wv] = x;
        __syncthreads();
        if (wv == 0) {
            int sv = lane < 16 ? wsum[lane] : 0;
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) {
                const int y = __shfl_up(sv, o);
                if (lane >= o) sv += y;
            }
            if (lane < 16) wsum[lane] = sv;
        }
        __syncthreads();
        const int excl = carry_s + (wv > 0 ? wsum[wv - 1] : 0) + x - u;
        if (i < a.num_seqs) unit_start[i] = excl;
        __syncthreads();
        if (tid == 1023) carry_s = excl + u;
        __syncthreads();
    }
    if (tid == 0) unit_start[a.num_seqs] = carry_s;
}

struct Cursor {
    int i, g, r, b;  // request, KV head, row group, block
    ReqGeom rq;
};

__device__ __forceinline__ void advance(const PArgs& a, const int32_t* __restrict__ q_start,
                                        const int32_t* __restrict__ seq_lens, Cursor& c) {
    if (++c.b < c.rq.b_lo + c.rq.nb) return;
    c.b = c.rq.b_lo;
    if (++c.r < c.rq.rg) return;
    c.r = 0;
    if (++c.g < a.hkv) return;
    c.g = 0;
    while (++c.i < a.num_seqs) {
        c.rq = req_geom(a, q_start, seq_lens, c.i);
        if (c.rq.rg > 0 && c.rq.nb > 0) break;
    }
    c.b = c.rq.b_lo;
}

// Batches of at most this many requests are scheduled inside attn_persist:
// every workgroup computes the per-request unit offsets itself (a scan over
// the batch's metadata, cheaper than a separate launch), and workgroup 0
// also stores them for the merge pass.
constexpr int kInlineSchedSeqs = 256;

// Exclusive prefix over the batch of each request's units (Hkv * row groups *
// blocks) into sched[0 .. num_seqs], sched[num_seqs] = total; one wavefront.
__device__ __forceinline__ void sched_prefix(const PArgs& a, const int32_t* __restrict__ q_start,
                                             const int32_t* __restrict__ seq_lens, int32_t* sched,
                                             int lane) {
    int carry = 0;
    for (int base = 0; base < a.num_seqs; base += kWave) {
        const int i = base + lane;
        int u = 0;
        if (i < a.num_seqs) {
            const ReqGeom r = req_geom(a, q_start, seq_lens, i);
            u = a.hkv * r.rg * r.nb;
        }
        int x = u;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (i < a.num_seqs) sched[i] = carry + x - u;
        carry += __shfl(x, kWave - 1);
    }
    if (lane == 0) sched[a.num_seqs] = carry;
}

// Unit range [us, ue) of workgroup w (empty when w has none).
__device__ __forceinline__ void unit_range(const PArgs& a, int U, int w, int& us, int& ue) {
    if (a.spb > 0) {
        us = (int)min((int64_t)U, (int64_t)w * a.spb);
        ue = (int)min((int64_t)U, (int64_t)us + a.spb);
    } else {
        const int n = sharing_wgs(a, U);
        us = w < n ? (int)((int64_t)U * w / n) : U;
        ue = w < n ? (int)((int64_t)U * (w + 1) / n) : U;
    }
}

// Value of a wavefront-uniform load, marked uniform for the compiler (a load
// through LDS or a pointer the kernel also writes is otherwise taken as
// divergent, and so is everything computed from it).
__device__ __forceinline__ int uniform_load(const int32_t* p) { return __builtin_amdgcn_readfirstlane(*p); }

// Cursor of unit u: its request is the largest i with unit_start[i] <= u.
__device__ __forceinline__ Cursor locate_unit(const PArgs& a, const int32_t* __restrict__ q_start,
                                              const int32_t* __restrict__ seq_lens,
                                              const int32_t* unit_start, int u) {
    int lo = 0, hi = a.num_seqs - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (uniform_load(unit_start + mid) <= u) lo = mid; else hi = mid - 1;
    }
    Cursor c;
    c.i = lo;
    c.rq = req_geom(a, q_start, seq_lens, lo);
    const int off = u - uniform_load(unit_start + lo);
    const int pq = off / c.rq.nb;  // pair within the request: head * rg + row group
    c.g = pq / c.rq.rg;
    c.r = pq - c.g * c.rq.rg;
    c.b = c.rq.b_lo + (off - pq * c.rq.nb);
    return c;
}

// One online-softmax step of a 16-row tile over one 16-key block.  sacc holds
// raw scores <q, k> in the MFMA result layout (lane 16 lg + l16: keys
// key0 .. key0 + 3 of the tile's row l16, key0 = 16 b + 4 lg); row_j is the
// row's draft position (-1: no row) and p_first the position of the request's
// first row.  The exponentials are taken against the stored maximum m as long
// as no score exceeds it by more than 2^kSlackLog2; only then (on a row's
// first keys, and rarely after) does the wavefront reduce the new row maximum
// over the row's four lanes and rescale l and o.  The weights stay below
// 2^kSlackLog2, and bf16 rounds them with the same relative error at any
// magnitude.  Returns the weights as the bf16 B operand of the PV product.
template <int DT>
__device__ __forceinline__ i16x4_t softmax_step(const f32x4_t& sacc, bool need_mask, int row_j,
                                                int p_first, int key0, int window, float c,
                                                float inv_c, float& m, float& l, float& thr,
                                                float& neg_m, f32x4_t (&o)[DT]) {
    float sv[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = sacc[r];
    if (need_mask) {
        const int p = p_first + row_j;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int key = key0 + r;
            const bool vis = row_j >= 0 && key <= p && (window == 0 || key > p - window);
            sv[r] = vis ? sv[r] : -INFINITY;
        }
    }
    const float mx = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    if (__builtin_amdgcn_ballot_w64(!(mx <= thr))) {
        const float rmax = row_max_4lanes(mx) * c;
        if (rmax > m) {
            // m = -inf: nothing accumulated yet, alpha = 0 keeps it 0
            const float alpha = __builtin_amdgcn_exp2f(m - rmax);
            l *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
            m = rmax;
            neg_m = -rmax;
            thr = (rmax + kSlackLog2) * inv_c;
        }
    }
    // exponent arguments are <= kSlackLog2: the raw v_exp_f32 is exact enough
    // and results below 2^-126 only flush to zero
    float pr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[r], c, neg_m));
    l += (pr[0] + pr[1]) + (pr[2] + pr[3]);
    return __builtin_bit_cast(i16x4_t, make_uint2(pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3])));
}

// Whether every row of the request sees every key of block b: the block lies
// below the first row's position and, with a window, inside the last row's
// window.
__device__ __forceinline__ bool block_needs_mask(int b, int p_first, int S, int window) {
    return (b * kBlockTokens + kBlockTokens - 1 > p_first) ||
           (window > 0 && b * kBlockTokens < S - window);
}

// Global->LDS loads need about sixteen wavefronts per compute unit to reach
// full HBM bandwidth, so one-tile configurations are held to four waves per
// SIMD (at most 128 registers each).
// Waves per SIMD the persistent kernel is built for.  The fused append's
// four-wavefront kernel is held to three, the residency of the plain one: its
// patch would otherwise take it to 192 registers and two workgroups per
// compute unit (long-context fused call 9.27 -> 8.66 ms); the few values it
// then keeps in scratch are reloaded only on pair switches and patched blocks.
template <int TPW, int NW = 1, bool APPEND = false>
constexpr int persist_waves_per_eu() { return TPW == 1 ? 4 : (APPEND && NW == 4 && TPW == 2 ? 3 : 2); }

// APPEND: the fused KV append (verify_attention_append).  The request's new
// tokens, positions S_i - n_i .. S_i - 1 of rows q_start[i] .. q_start[i+1]-1,
// are taken from k_new / v_new: after a block holding some of them has landed
// in LDS, the workgroup overwrites their K and V there (one extra barrier, on
// those blocks only), and the workgroup of the pair's first row group also
// stores them into the cache.  Readers never depend on that store, so no
// ordering between workgroups is needed.
template <int D, int NW, int TPW, int PD, bool APPEND>
__global__ __launch_bounds__(NW * kWave)
__attribute__((amdgpu_waves_per_eu(persist_waves_per_eu<TPW, NW, APPEND>()))) void attn_persist(
    PArgs a, const uint16_t* __restrict__ qg, const uint8_t* __restrict__ kcg,
    const uint8_t* __restrict__ vcg, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ q_start,
    int32_t* __restrict__ unit_start, uint16_t* __restrict__ out,
    uint16_t* __restrict__ slot_o, float* __restrict__ slot_lse,
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new) {
    constexpr int NT = NW * kWave;
    constexpr int TILE_BYTES = kBlockTokens * D * 2;  // one (block, head) K or V tile
    constexpr int CH = 2 * TILE_BYTES / 16;           // 16-byte chunks per block (K then V)
    constexpr int CPT = CH / NT;                      // chunks per thread per block
    constexpr int KC = D / 32;                        // QK^T steps of 32 dims
    constexpr int DT = D / 16;                        // PV output tiles of 16 dims
    constexpr int ROWS = NW * TPW * 16;
    constexpr int NS = PD + 1;                        // LDS stages: PD blocks in flight
    static_assert(CH % NT == 0, "every thread loads the same number of chunks");
    static_assert(CPT * (NS - 2) < 64, "vmcnt range");

    __shared__ __attribute__((aligned(16))) uint8_t stage[NS][2 * TILE_BYTES];
    __shared__ int32_t sched[kInlineSchedSeqs + 1];

    const int w = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wv = tid / kWave;
    const int l16 = lane & 15, lg = lane >> 4;

    const int32_t* ustart = unit_start;
    if (a.inline_sched) {
        if (wv == 0) {
            sched_prefix(a, q_start, seq_lens, sched, lane);
            if (w == 0) {
                for (int i = lane; i <= a.num_seqs; i += kWave) unit_start[i] = sched[i];
                mark_unreached_rows<D>(a, q_start, out, lane, kWave);
            }
        }
        __syncthreads();
        ustart = sched;
    }
    const int U = uniform_load(ustart + a.num_seqs);
    int us, ue;
    unit_range(a, U, w, us, ue);
    if (us >= ue) return;
    const Cursor c0 = locate_unit(a, q_start, seq_lens, ustart, us);

    const uint32_t stage_lds =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)&stage[0][0];
    // One unit = one block's K and V tiles, copied into an LDS stage with CPT
    // global->LDS loads per thread (wavefront w's c-th load fills the 1 KiB
    // at chunk c*NT + 64w).  Every call issues exactly CPT loads, invalid
    // block ids reading block 0 (compute skips them through ok_mask), so the
    // explicit vmcnt waits below count exactly.
    // Bit s: stage s holds a valid block.  Every wavefront runs the same
    // loader steps, so each keeps its own copy in a scalar register.
    uint32_t ok_mask = 0;
    auto dma_unit = [&](const Cursor& c, int st, int phys) {
        const int g = c.g;
        const bool ok = phys >= 0 && phys < a.num_blocks;
        ok_mask = ok ? (ok_mask | (1u << st)) : (ok_mask & ~(1u << st));
        phys = ok ? phys : 0;
        const int64_t off = ((int64_t)phys * a.hkv + g) * TILE_BYTES;
        const uint32_t base = stage_lds + st * (2 * TILE_BYTES);
#pragma unroll
        for (int c2 = 0; c2 < CPT; ++c2) {
            const int wchunk = c2 * NT + wv * kWave;  // first chunk of this wavefront's load
            const int idx = wchunk + lane;
            const uint8_t* srcp = idx < CH / 2 ? kcg + off + idx * 16 : vcg + off + (idx - CH / 2) * 16;
            dma16(base + wchunk * 16, srcp);
        }
    };

    // ---- state of the pair being computed
    int st_i = -1, st_g = -1, st_rg = -1;
    int st_ps = 0;  // first unit of the pair
    ReqGeom srq{};
    bool active = false;
    bf16x8_t qop[TPW][KC];
    int row_j[TPW];
    f32x4_t o[TPW][DT];
    // Online softmax state per tile, in the log2 domain: m_r is the maximum
    // the row's exponentials are taken against (identical in the four lanes
    // that hold the row), thr the raw score above which a lane needs a new
    // maximum, neg_m = -m_r (0 while the row has seen no key).
    float m_r[TPW], l_r[TPW], thr[TPW], neg_m[TPW];
    float sink_l2[TPW];  // the row's head's sink logit in the log2 domain (-inf: none)
    // APPEND: the pair's new-token positions [st_nlo, st_nhi) (those the walk
    // reaches) and the position of its first row, S_i - n_i
    int st_nlo = 0, st_nhi = 0, st_p0 = 0;

    // Pair of cursor c, reached at unit u.
    auto init_pair = [&](const Cursor& c, int u) {
        st_i = c.i;
        st_ps = u - (c.b - c.rq.b_lo);
        srq = c.rq;
        st_g = c.g;
        st_rg = c.r;
        if constexpr (APPEND) {
            const int s_raw = uniform_load(seq_lens + c.i);
            st_p0 = s_raw - srq.n;
            st_nlo = max(st_p0, 0);
            st_nhi = min(s_raw, srq.S);
        }
        const int rows = a.group * srq.n;
        const int wrow0 = st_rg * ROWS + wv * TPW * 16;
        active = wrow0 < rows;
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            const int rr = wrow0 + t * 16 + l16;
            const bool valid = rr < rows;
            const int j = rr / a.group, gh = rr - j * a.group;
            row_j[t] = valid ? j : -1;
            const int64_t base = ((int64_t)(srq.q0 + j) * a.hq + st_g * a.group + gh) * D;
#pragma unroll
            for (int cc = 0; cc < KC; ++cc) {
                uint4 v = make_uint4(0, 0, 0, 0);
                if (valid) v = ld16(qg + base + (cc * 4 + lg) * 8);
                qop[t][cc] = as_bf16x8(v);
            }
            m_r[t] = -INFINITY;
            l_r[t] = 0.f;
            thr[t] = -INFINITY;
            neg_m[t] = 0.f;
            sink_l2[t] = a.sinks && valid ? a.sinks[st_g * a.group + gh] * kLog2e : -INFINITY;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[t][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        }
        // Settle the Q loads here, on the (rare) pair-switch path.  Otherwise
        // the compiler cannot tell whether they are still in flight when the
        // next block's MFMA reads the operands, and waits for the whole load
        // queue, prefetched KV blocks included, before every block.
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    };

    auto flush_pair = [&]() {
        if (!active) return;
        const bool whole = st_ps >= us && st_ps + srq.nb <= ue;
        const int rows = a.group * srq.n;
        const int64_t slot = (int64_t)(st_i * a.hkv + st_g) * a.rg_max + st_rg + w;
#pragma unroll
        for (int t = 0; t < TPW; ++t) {
            float L = l_r[t];
            L += __shfl_xor(L, 16);
            L += __shfl_xor(L, 32);
            const int lr = (wv * TPW + t) * 16 + l16;
            const int rr = st_rg * ROWS + lr;
            if (rr >= rows) continue;
            if (whole) {
                const float den = L + (a.sinks ? exp2f(sink_l2[t] - m_r[t]) : 0.f);
                const float inv = den > 0.f ? 1.f / den : 0.f;
                const int j = rr / a.group, gh = rr - j * a.group;
                const int64_t hrow = (int64_t)(srq.q0 + j) * a.hq + st_g * a.group + gh;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const int d0 = dt * 16 + 4 * lg;
                    const uint2 v = make_uint2(pack_bf16x2(o[t][dt][0] * inv, o[t][dt][1] * inv),
                                               pack_bf16x2(o[t][dt][2] * inv, o[t][dt][3] * inv));
                    *reinterpret_cast<uint2*>(out + hrow * D + d0) = v;
                }
            } else {
                // the tile's 16 rows x D values in register order (see
                // slot_o_index): each store writes 512 bytes contiguous
                const float inv = L > 0.f ? 1.f / L : 0.f;
                const int64_t srow = slot * ROWS + lr;
                uint16_t* tb = slot_o + (slot * ROWS + (wv * TPW + t) * 16) * D + lane * 4;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt)
                    *reinterpret_cast<uint2*>(tb + dt * (kWave * 4)) =
                        make_uint2(pack_bf16x2(o[t][dt][0] * inv, o[t][dt][1] * inv),
                                   pack_bf16x2(o[t][dt][2] * inv, o[t][dt][3] * inv));
                if (lg == 0) slot_lse[srow] = L > 0.f ? m_r[t] + log2f(L) : -INFINITY;
            }
        }
    };

    auto compute = [&](int st, int b) {
        if (!active || !((ok_mask >> st) & 1u)) return;
        const uint8_t* ks = stage[st];
        const uint8_t* vs = stage[st] + TILE_BYTES;
        f32x4_t sacc[TPW];
#pragma unroll
        for (int t = 0; t < TPW; ++t) sacc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int cc = 0; cc < KC; ++cc) {
            const bf16x8_t kop =
                as_bf16x8(*reinterpret_cast<const uint4*>(ks + ((cc * 4 + lg) * 16 + l16) * 16));
#pragma unroll
            for (int t = 0; t < TPW; ++t)
                sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop, qop[t][cc], sacc[t], 0, 0, 0);
        }
        const int p_first = srq.S - srq.n;  // position of the request's first query row
        const bool need_mask = block_needs_mask(b, p_first, srq.S, a.window);
        i16x4_t pop[TPW];
#pragma unroll
        for (int t = 0; t < TPW; ++t)
            pop[t] = softmax_step<DT>(sacc[t], need_mask, row_j[t], p_first, b * kBlockTokens + 4 * lg,
                                      a.window, a.scale_log2, a.inv_scale_log2, m_r[t], l_r[t],
                                      thr[t], neg_m[t], o[t]);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const uint2 vv = *reinterpret_cast<const uint2*>(vs + (dt * 16 + l16) * 32 + lg * 8);
            const i16x4_t vop = __builtin_bit_cast(i16x4_t, vv);
#pragma unroll
            for (int t = 0; t < TPW; ++t)
                o[t][dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vop, pop[t], o[t][dt], 0, 0, 0);
        }
    };

    // APPEND: overwrite the new tokens of block b in stage st with their K and
    // V from k_new / v_new (16 bytes = 8 dims of one token per step), and, in
    // the pair's first row group, store them into the cache block as well.
    auto patch_new = [&](int st, int b) {
        constexpr int DC = D / 8;  // 16-byte chunks per key
        const int pos0 = b * kBlockTokens;
        const int t_lo = max(st_nlo - pos0, 0), t_hi = min(st_nhi - pos0, kBlockTokens);
        uint8_t* ks = stage[st];
        uint16_t* vs = reinterpret_cast<uint16_t*>(stage[st] + TILE_BYTES);
        const bool writer = st_rg == 0;
        const int phys = uniform_load(block_tables + (int64_t)st_i * a.max_blocks + b);
        const int64_t toff = ((int64_t)phys * a.hkv + st_g) * TILE_BYTES;
        uint8_t* kw = const_cast<uint8_t*>(kcg) + toff;
        uint16_t* vw = reinterpret_cast<uint16_t*>(const_cast<uint8_t*>(vcg) + toff);
        // K and V of one token's 8 dims per step, both loads in flight together
        for (int e = tid; e < (t_hi - t_lo) * DC; e += NT) {
            const int t = t_lo + e / DC, dc = e % DC;
            const int64_t row = srq.q0 + (pos0 + t - st_p0);
            const int64_t src = (row * a.hkv + st_g) * D + dc * 8;
            const uint4 kv = ld16(k_new + src);
            const uint4 vv = ld16(v_new + src);
            const int kchunk = dc * kBlockTokens + t;
            *reinterpret_cast<uint4*>(ks + kchunk * 16) = kv;
            const uint32_t vh[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
            for (int k = 0; k < 8; ++k)
                vs[(dc * 8 + k) * kBlockTokens + t] = (uint16_t)(vh[k >> 1] >> (16 * (k & 1)));
            if (writer) {
                *reinterpret_cast<uint4*>(kw + kchunk * 16) = kv;
#pragma unroll
                for (int k = 0; k < 8; ++k)
                    vw[(dc * 8 + k) * kBlockTokens + t] = (uint16_t)(vh[k >> 1] >> (16 * (k & 1)));
            }
        }
    };

    // ---- pipeline: a ring of NS = PD + 1 LDS stages, PD blocks in flight.
    // At unit uu: wait for this thread's loads of uu (the PD - 1 younger units
    // may stay in flight), barrier (everyone's loads of uu have landed and
    // everyone is done with uu - 1), refill the stage of uu - 1 with unit
    // uu + PD, compute uu.  The loader cursor stops at the last unit and loads
    // it again instead of issuing nothing, keeping the count fixed.
    Cursor lc = c0;
    int lu = us;
    // Block id of the loader's unit: a scalar load, issued once the previous
    // unit's compute has read its LDS operands (so that no LDS wait there
    // also waits for it) and consumed after the next barrier.
    auto fetch_phys = [&]() { return block_tables[(int64_t)lc.i * a.max_blocks + lc.b]; };
    auto dma_next = [&](int st, int phys) {
        dma_unit(lc, st, phys);
        if (lu + 1 < ue) {
            advance(a, q_start, seq_lens, lc);
            ++lu;
        }
    };
#pragma unroll
    for (int r = 0; r < PD; ++r) dma_next(r, fetch_phys());
    int phys_next = fetch_phys();

    Cursor cc = c0;
    init_pair(cc, us);
    int st = 0;
    for (int uu = us; uu < ue; ++uu) {
        wait_vmcnt<CPT * (PD - 1)>();
        lds_barrier();
        dma_next(st == 0 ? NS - 1 : st - 1, phys_next);
        if (cc.i != st_i || cc.g != st_g || cc.r != st_rg) {
            flush_pair();
            init_pair(cc, uu);
        }
        if constexpr (APPEND) {
            // block-uniform: every wavefront takes the same branch
            const int pos0 = cc.b * kBlockTokens;
            if (((ok_mask >> st) & 1u) && pos0 < st_nhi && pos0 + kBlockTokens > st_nlo) {
                patch_new(st, cc.b);
                lds_barrier();
            }
        }
        compute(st, cc.b);
        asm volatile("" ::: "memory");
        phys_next = fetch_phys();
        advance(a, q_start, seq_lens, cc);
        st = st == NS - 1 ? 0 : st + 1;
    }
    // no global->LDS load may still be writing when the workgroup's LDS is freed
    wait_vmcnt<0>();
    flush_pair();
}

// Merges the partial slots of pairs cut by workgroup range boundaries, and
// writes the zero output of rows whose request has no key.  Grid (pairs, row
// chunks); a thread owns one row and four consecutive output dimensions.  The
// slots of a row are read kCombineSlots at a time, every load of a round
// issued before any is used (a pair is cut into a handful of slots, so one
// round usually covers it), and merged with a running maximum.
constexpr int kCombineThreads = 256;
constexpr int kCombineSlots = 8;

template <int D>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_slots(
    PArgs a, const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ q_start,
    const int32_t* __restrict__ unit_start, const uint16_t* __restrict__ slot_o,
    const float* __restrict__ slot_lse, uint16_t* __restrict__ out) {
    constexpr int QUADS = D / 4;                       // 4-dim vectors per row
    constexpr int RPB = kCombineThreads / QUADS;       // rows per workgroup
    const int P = blockIdx.x;
    const int per_req = a.hkv * a.rg_max;
    const int i = P / per_req;
    const int rem = P - i * per_req;
    const int g = rem / a.rg_max, rg = rem - g * a.rg_max;
    // the request's metadata and unit offsets are read together, before any
    // test, so that they cost one memory latency instead of one each
    const int U = unit_start[a.num_seqs];
    const int ustart_i = unit_start[i];
    const ReqGeom rq = req_geom(a, q_start, seq_lens, i);
    if (rg >= rq.rg) return;
    const int ROWS = a.rows_per_group;
    const int rows = a.group * rq.n;
    const int lr = blockIdx.y * RPB + threadIdx.x / QUADS;  // row within the group
    const int rr = rg * ROWS + lr;
    if (lr >= ROWS || rr >= rows) return;
    const bool empty = rq.nb == 0;
    int wf = 0, wl = 0;
    if (!empty) {
        const int ps = ustart_i + (g * rq.rg + rg) * rq.nb;
        wf = owner_of(a, ps, U);
        wl = owner_of(a, ps + rq.nb - 1, U);
        if (wf == wl) return;  // finished in place by its only workgroup
    }
    const int d0 = (threadIdx.x % QUADS) * 4;
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    if (!empty) {
        // slots of the pair: one per workgroup wf .. wl; a slot holding
        // log-sum-exp -inf (no visible key in its range) adds nothing
        const int64_t slot0 = (int64_t)P + wf;
        const int ns = wl - wf + 1;
        float M = -INFINITY, L = 0.f;
        for (int s0 = 0; s0 < ns; s0 += kCombineSlots) {
            float lse[kCombineSlots];
            f32x4_t o[kCombineSlots];
            // every load is issued unconditionally (slots past the pair's last
            // re-read the last one and are masked afterwards), so that the
            // round's loads leave back to back; conditional loads compiled to a
            // branch and a wait per slot, one memory latency each
            uint2 v[kCombineSlots];
#pragma unroll
            for (int k = 0; k < kCombineSlots; ++k) {
                const int64_t sl = slot0 + min(s0 + k, ns - 1);
                lse[k] = slot_lse[sl * ROWS + lr];
                v[k] = *reinterpret_cast<const uint2*>(slot_o + slot_o_index<D>(sl, ROWS, lr, d0));
            }
#pragma unroll
            for (int k = 0; k < kCombineSlots; ++k) {
                const bool in = s0 + k < ns;
                lse[k] = in ? lse[k] : -INFINITY;
                o[k] = in ? f32x4_t{bf16_lo(v[k].x), bf16_hi(v[k].x), bf16_lo(v[k].y), bf16_hi(v[k].y)}
                          : f32x4_t{0.f, 0.f, 0.f, 0.f};
            }
            float m = M;
#pragma unroll
            for (int k = 0; k < kCombineSlots; ++k) m = fmaxf(m, lse[k]);
            if (m == -INFINITY) continue;
            // rescale what earlier rounds summed (nothing yet: M = -inf gives 0)
            const float r = __builtin_amdgcn_exp2f(M - m);
            L *= r;
            acc *= r;
#pragma unroll
            for (int k = 0; k < kCombineSlots; ++k) {
                const float f = lse[k] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(lse[k] - m);
                L += f;
                acc += f * o[k];
            }
            M = m;
        }
        if (M != -INFINITY) {
            L += sink_term(a.sinks, g * a.group + rr % a.group, M);
            acc *= 1.f / L;
        }
    }
    const int j = rr / a.group, gh = rr - j * a.group;
    const int64_t hrow = (int64_t)(rq.q0 + j) * a.hq + g * a.group + gh;
    *reinterpret_cast<uint2*>(out + hrow * D + d0) =
        make_uint2(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]));
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
    T* outp = static_cast<T*>(a.out);
    {
        // rows past the launch's reach (a request with more than max_q_len
        // rows) are not computed: quiet NaN instead of stale memory
        const int h = (int)(item - (int64_t)row * a.hq);
        const int rr = (row - sg.q0) * a.group + h % a.group;
        if (rr >= a.row_groups * kValuRows) {
#pragma unroll
            for (int e = 0; e < DPL; ++e) Storage<T>::store(outp, item * D + lane * DPL + e, __builtin_nanf(""));
            return;
        }
    }
    if (sg.nsplit == 1) return;
    float acc[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
    float L = 0.f;
    if (sg.nsplit > 1) {
        const int64_t pi0 = item * a.max_splits;
        float M = -INFINITY;
        const int h = (int)(item - (int64_t)row * a.hq);
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
            L += sink_term(a.sinks, h, M);
        }
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e)
        Storage<T>::store(outp, item * D + lane * DPL + e, L > 0.f ? acc[e] / L : 0.f);
}

// ------------------------------------------------------------------ KV append
//
// The verify step's new tokens (row j of request i sits at position
// p = S_i - n_i + j) get their K and V written into slot p % 16 of block
// block_tables[i][p / 16]: K x-packed ([D/x][16][x] per block and head), V
// transposed ([D][16]).  One workgroup per (request, KV head) writes all of
// the request's new tokens of that head, so the tokens that share a 32-byte
// V sector (consecutive slots of one dimension) are written by one compute
// unit and leave its L2 as one sector.  K moves in 16-byte chunks, thread
// items ordered (chunk, token) so that consecutive threads write consecutive
// slots; V moves element by element, items ordered (dimension, token).
// Tokens with a negative position or a block id outside [0, num_blocks) are
// skipped.
constexpr int kAppendThreads = 256;

template <typename T, int D>
__global__ __launch_bounds__(kAppendThreads) void attn_kv_append(
    int num_seqs, int hkv, int max_blocks, int num_blocks, const T* __restrict__ k_new,
    const T* __restrict__ v_new, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ q_start, T* __restrict__ kc,
    T* __restrict__ vc) {
    constexpr int X = Storage<T>::kPer16B;
    constexpr int NC = D / X;  // 16-byte chunks per key
    const int i = blockIdx.x, g = blockIdx.y;
    const int q0 = q_start[i];
    const int n = q_start[i + 1] - q0;
    if (n <= 0) return;
    const int64_t p0 = (int64_t)seq_lens[i] - n;  // position of the request's row 0
    const int32_t* bt = block_tables + (int64_t)i * max_blocks;
    // physical block of token j, or -1 when the token is skipped
    auto block_of = [&](int j) {
        const int64_t p = p0 + j;
        if (p < 0 || p / kBlockTokens >= max_blocks) return -1;
        const int b = bt[p / kBlockTokens];
        return (b < 0 || b >= num_blocks) ? -1 : b;
    };
    for (int it = threadIdx.x; it < n * NC; it += kAppendThreads) {
        const int c = it / n, j = it - c * n;
        const int b = block_of(j);
        if (b < 0) continue;
        const int t = (int)((p0 + j) % kBlockTokens);
        const uint4 v = ld16(k_new + ((int64_t)(q0 + j) * hkv + g) * D + c * X);
        *reinterpret_cast<uint4*>(kc + ((((int64_t)b * hkv + g) * NC + c) * kBlockTokens + t) * X) = v;
    }
    for (int it = threadIdx.x; it < n * D; it += kAppendThreads) {
        const int d = it / n, j = it - d * n;
        const int b = block_of(j);
        if (b < 0) continue;
        const int t = (int)((p0 + j) % kBlockTokens);
        vc[(((int64_t)b * hkv + g) * D + d) * kBlockTokens + t] = v_new[((int64_t)(q0 + j) * hkv + g) * D + d];
    }
}

// ------------------------------------------------------------------ host side

struct AttnPlan {
    bool mfma;        // bf16 storage: persistent MFMA kernel; fp32 storage: VALU kernel
    // VALU path
    int split_blocks;
    int max_splits;
    int row_groups;
    size_t part_o_bytes;
    size_t part_lse_bytes;
    // MFMA path: one persistent launch per row class
    struct Class {
        int nw, tpw;          // wavefronts per workgroup, 16-row tiles per wavefront
        int rg_max;           // row groups per (request, KV head)
        int nwg;              // persistent workgroups
        int spb;              // fixed units per workgroup (0: equal shares)
        int rows_lo, rows_hi; // requests with Hq/Hkv * n_i in [rows_lo, rows_hi]
        int64_t slots;        // partial slots
        size_t off;           // workspace offset of the class's arrays
        size_t unit_bytes, slot_o_bytes, slot_lse_bytes;
    };
    int nclass;
    Class cls[2];
    size_t total_bytes;
};

// Batches whose requests carry up to this many query rows per KV head (three
// 16-row tiles) and more than that run in two launches, each with its own
// kernel shape (see make_plan).
constexpr int kShortClassRows = 48;

// A launch whose workgroups would each own more than this many units (each
// unit a 16-token block of 8 KiB at head dim 128, so about 3 ms of streaming)
// launches up to eight times the resident workgroups: the hardware hands the
// next workgroup to whichever compute unit frees a slot first, so faster
// compute units take more of the work (long-context batch: 10.06 -> 9.10 ms at
// eight times; at the short Qwen and DSK calls the extra start-ups cost more
// than the balance gains).
constexpr int64_t kOversubUnits = 4096;

// KV blocks in flight per workgroup.  Three (a 32 KiB ring at D = 128) lets
// four workgroups share a compute unit's 160 KiB of LDS; the four-wavefront
// two-tile shape runs two workgroups per compute unit (its registers allow no
// more) and takes five.  More workgroups per compute unit beat deeper rings:
// each workgroup advances one block per barrier, so the per-block latency of
// one workgroup is what more workgroups hide.
constexpr int prefetch_depth(int d, int nw, int tpw) { return d == 128 && nw == 4 && tpw == 2 ? 5 : 3; }

// The kernel shapes a plan may choose: head dim, wavefronts per workgroup,
// 16-row tiles per wavefront.  with_shape calls f(Shape<...>{}) for the
// matching entry and returns false if there is none.
template <int D_, int NW_, int TPW_>
struct Shape {
    static constexpr int D = D_, NW = NW_, TPW = TPW_, PD = prefetch_depth(D_, NW_, TPW_);
};

template <typename F>
bool with_shape(int d, int nw, int tpw, F&& f) {
#define AVERIFY_SHAPE(D_, NW_, TPW_)                       \
    if (d == D_ && nw == NW_ && tpw == TPW_) {             \
        f(Shape<D_, NW_, TPW_>{});                         \
        return true;                                       \
    }
    AVERIFY_SHAPE(128, 1, 1)
    AVERIFY_SHAPE(128, 1, 3)
    AVERIFY_SHAPE(128, 2, 1)
    AVERIFY_SHAPE(128, 2, 2)
    AVERIFY_SHAPE(128, 4, 2)
    AVERIFY_SHAPE(64, 1, 1)
    AVERIFY_SHAPE(64, 1, 5)
    AVERIFY_SHAPE(64, 2, 1)
    AVERIFY_SHAPE(64, 4, 1)
    AVERIFY_SHAPE(64, 4, 2)
    AVERIFY_SHAPE(64, 4, 3)
    AVERIFY_SHAPE(64, 4, 4)
#undef AVERIFY_SHAPE
    return false;
}

template <typename S, bool APPEND = false>
constexpr auto persist_kernel() {
    return attn_persist<S::D, S::NW, S::TPW, S::PD, APPEND>;
}

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

// Compute units of the current device and resident workgroups per compute
// unit of a kernel (cached per device; fallbacks when no device is visible).
int device_cus() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) { (void)hipGetLastError(); return 256; }
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) {
        (void)hipGetLastError();
        v = 256;
    }
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

template <typename S, bool APPEND = false>
int resident_wgs() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) { (void)hipGetLastError(); return 2; }
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&v, persist_kernel<S, APPEND>(), S::NW * kWave, 0) !=
            hipSuccess ||
        v <= 0) {
        (void)hipGetLastError();
        v = 1;
    }
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

// Kernel shape (wavefronts per workgroup, tiles per wavefront) for row groups
// of up to `tiles` 16-row tiles.  A single tile goes to single-wavefront
// workgroups: every wavefront is an independent worker with its own LDS ring
// and no barrier.  More rows use NW wavefronts sharing one ring (NW divides
// the 16-byte chunks of a block, 512 at D = 128 and 256 at D = 64, so every
// thread loads alike).  At D = 128 a wavefront takes two tiles once there are
// three or more: fewer wavefronts per block mean fewer barriers and more
// workgroups per compute unit, which is what hides the per-block latency of
// the online softmax.  Rows beyond the shape's reach are split into row
// groups, each walking the request's KV again.
void pick_shape(int head_dim, int64_t tiles, int64_t nb_max, int& nw, int& tpw) {
    if (tiles <= 1) {
        nw = 1;
        tpw = 1;
    } else if (head_dim == 128) {
        nw = tiles <= 4 ? 2 : 4;
        tpw = tiles == 2 ? 1 : 2;
        if (tiles == 3 && nb_max >= 64) { nw = 1; tpw = 3; }
    } else {
        nw = tiles <= 2 ? 2 : 4;
        tpw = (int)std::min<int64_t>(4, (tiles + nw - 1) / nw);
        if (tiles == 5 && nb_max >= 64) { nw = 1; tpw = 5; }
    }
}

// The persistent launch of one row class: requests with rows_lo <= Hq/Hkv *
// n_i <= rows_hi, of which no request has more than `rows` rows.
int plan_class(const verify_attn_params* p, int64_t rows, int64_t nb_max, int rows_lo, int rows_hi,
               bool append, AttnPlan::Class& c) {
    c = AttnPlan::Class{};
    pick_shape(p->head_dim, (rows + 15) / 16, nb_max, c.nw, c.tpw);
    c.rows_lo = rows_lo;
    c.rows_hi = rows_hi;
    const int64_t per = (int64_t)c.nw * c.tpw * 16;
    c.rg_max = (int)((rows + per - 1) / per);
    const int64_t pairs = (int64_t)std::max(1, p->num_seqs) * p->num_kv_heads * c.rg_max;
    const int64_t units_max = pairs * nb_max;
    if (units_max >= (int64_t)1 << 31) return VERIFY_EUNSUPPORTED;
    c.spb = p->kv_split_blocks;
    if (c.spb > 0) {
        c.nwg = (int)std::min<int64_t>((units_max + c.spb - 1) / c.spb, (int64_t)1 << 30);
    } else {
        int res = 0;
        // the fused-append kernel holds more registers, and may fit fewer
        // workgroups per compute unit
        if (!with_shape(p->head_dim, c.nw, c.tpw, [&](auto sh) {
                res = append ? resident_wgs<decltype(sh), true>() : resident_wgs<decltype(sh)>();
            }))
            return VERIFY_EUNSUPPORTED;
        const int64_t resident = (int64_t)device_cus() * res;
        const int64_t mult = std::min<int64_t>(8, std::max<int64_t>(1, units_max / resident / kOversubUnits));
        c.nwg = (int)(resident * mult);
    }
    c.slots = pairs + c.nwg;
    c.unit_bytes = align_up(sizeof(int32_t) * ((size_t)std::max(1, p->num_seqs) + 1), 256);
    c.slot_o_bytes = align_up((size_t)c.slots * per * p->head_dim * sizeof(uint16_t), 256);
    c.slot_lse_bytes = align_up((size_t)c.slots * per * sizeof(float), 256);
    return VERIFY_OK;
}

int make_plan(const verify_attn_params* p, int32_t total_q, int32_t max_q_len,
              int32_t max_seq_len, AttnPlan* out, bool append = false) {
    AttnPlan pl{};
    const int G = p->num_q_heads / p->num_kv_heads;
    int64_t nb_max = ((int64_t)max_seq_len + kBlockTokens - 1) / kBlockTokens;
    if (p->sliding_window > 0) {
        const int64_t span = (int64_t)p->sliding_window + max_q_len - 1;
        nb_max = std::min<int64_t>(nb_max, (span + kBlockTokens - 1) / kBlockTokens + 1);
    }
    nb_max = std::max<int64_t>(nb_max, 1);
    const int64_t rows = (int64_t)G * std::max(1, max_q_len);
    pl.mfma = p->dtype == VERIFY_BF16;
    if (pl.mfma) {
        // One launch sized by the largest request.  At head dim 128, when that
        // takes the four-wavefront shape (five tiles or more), the requests
        // of up to three tiles get a launch of their own with the shape of
        // three tiles: the four-wavefront shape streams 5.4 TB/s on pairs of
        // one tile but 4.2 TB/s on pairs of eight, and 5.9-6.0 TB/s on pairs
        // of three in the three-tile shape (long contexts), so mixing draft
        // lengths in one launch runs every pair at about the slow rate.
        int rc;
        if (p->head_dim == 128 && (rows + 15) / 16 >= 5) {
            pl.nclass = 2;
            rc = plan_class(p, kShortClassRows, nb_max, 0, kShortClassRows, append, pl.cls[0]);
            if (rc == VERIFY_OK)
                rc = plan_class(p, rows, nb_max, kShortClassRows + 1, INT32_MAX, append, pl.cls[1]);
        } else {
            pl.nclass = 1;
            rc = plan_class(p, rows, nb_max, 0, INT32_MAX, append, pl.cls[0]);
        }
        if (rc != VERIFY_OK) return rc;
        size_t off = 0;
        for (int k = 0; k < pl.nclass; ++k) {
            AttnPlan::Class& c = pl.cls[k];
            c.off = off;
            off += c.unit_bytes + c.slot_o_bytes + c.slot_lse_bytes;
        }
        pl.total_bytes = off;
    } else {
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
        pl.row_groups = (int)((rows + kValuRows - 1) / kValuRows);
        // grid (splits, KV heads x row groups, requests): y is a 16-bit dimension
        if ((int64_t)p->num_kv_heads * pl.row_groups > 65535) return VERIFY_EUNSUPPORTED;
        if (pl.max_splits > 1) {
            const size_t items = (size_t)total_q * p->num_q_heads * pl.max_splits;
            pl.part_o_bytes = align_up(items * p->head_dim * sizeof(float), 256);
            pl.part_lse_bytes = align_up(items * sizeof(float), 256);
        }
        pl.total_bytes = pl.part_o_bytes + pl.part_lse_bytes;
    }
    *out = pl;
    return VERIFY_OK;
}

// Schedule pass, then the persistent kernel of the plan's shape, then the
// merge of partial slots.  Returns false if the plan names no known shape.
bool launch_persist(const PArgs& a, const MPtrs& m, const AttnPlan::Class& pl, int head_dim,
                    int max_rows, hipStream_t stream) {
    return with_shape(head_dim, pl.nw, pl.tpw, [&](auto sh) {
        using S = decltype(sh);
        if (!a.inline_sched)
            hipLaunchKernelGGL((attn_schedule<S::D>), dim3(1), dim3(1024), 0, stream, a, m.q_start,
                               m.seq_lens, m.unit_start, m.out);
        if (m.k_new)
            hipLaunchKernelGGL((persist_kernel<S, true>()), dim3(a.nwg), dim3(S::NW * kWave), 0, stream,
                               a, m.q, m.kc, m.vc, m.block_tables, m.seq_lens, m.q_start, m.unit_start,
                               m.out, m.slot_o, m.slot_lse, m.k_new, m.v_new);
        else
            hipLaunchKernelGGL(persist_kernel<S>(), dim3(a.nwg), dim3(S::NW * kWave), 0, stream, a,
                               m.q, m.kc, m.vc, m.block_tables, m.seq_lens, m.q_start, m.unit_start,
                               m.out, m.slot_o, m.slot_lse, nullptr, nullptr);
        const int64_t pairs = (int64_t)a.num_seqs * a.hkv * a.rg_max;
        constexpr int RPB = kCombineThreads / (S::D / 4);
        // rows of a row group: at most rows_per_group, at most G * max_q_len
        const int group_rows = std::max(1, std::min(a.rows_per_group, max_rows));
        const unsigned chunks = (unsigned)((group_rows + RPB - 1) / RPB);
        if (pairs > 0)
            hipLaunchKernelGGL((attn_combine_slots<S::D>), dim3((unsigned)pairs, chunks),
                               dim3(kCombineThreads), 0, stream, a, m.seq_lens, m.q_start,
                               m.unit_start, m.slot_o, m.slot_lse, m.out);
    });
}

template <typename T, int D>
void launch_valu(const AttnArgs& a, const AttnPlan& pl, int total_q, hipStream_t stream) {
    dim3 grid(pl.max_splits, a.hkv * pl.row_groups, a.num_seqs);
    if (a.k_new)
        hipLaunchKernelGGL((attn_valu<T, D, true>), grid, dim3(kAttnThreads), 0, stream, a);
    else
        hipLaunchKernelGGL((attn_valu<T, D, false>), grid, dim3(kAttnThreads), 0, stream, a);
    const int64_t items = (int64_t)total_q * a.hq;
    if (items > 0) {
        dim3 cgrid((unsigned)((items + kAttnWaves - 1) / kAttnWaves));
        hipLaunchKernelGGL((attn_combine<T, D>), cgrid, dim3(kAttnThreads), 0, stream, a, total_q);
    }
}

}  // namespace
}  // namespace averify

using namespace averify;

extern "C" int verify_attention_workspace_size(const verify_attn_params* params, int32_t total_q,
                                               int32_t max_q_len, int32_t max_seq_len,
                                               size_t* bytes) {
    if (!bytes) return VERIFY_EINVAL;
    int rc = validate(params, total_q, max_q_len, max_seq_len);
    if (rc != VERIFY_OK) return rc;
    // enough for verify_attention and verify_attention_append alike
    AttnPlan pl, pla;
    rc = make_plan(params, total_q, max_q_len, max_seq_len, &pl);
    if (rc == VERIFY_OK) rc = make_plan(params, total_q, max_q_len, max_seq_len, &pla, true);
    if (rc != VERIFY_OK) return rc;
    *bytes = std::max(pl.total_bytes, pla.total_bytes);
    return VERIFY_OK;
}

namespace {

// verify_attention, and with k_new / v_new non-null verify_attention_append
int attention_call(const verify_attn_params* params, int32_t total_q, int32_t max_q_len,
                   int32_t max_seq_len, const void* q, const void* k_cache, const void* v_cache,
                   const int32_t* block_tables, const int32_t* seq_lens, const int32_t* q_start,
                   const float* sinks, void* out, void* workspace, size_t workspace_bytes,
                   const void* k_new, const void* v_new, hipStream_t stream) {
    int rc = validate(params, total_q, max_q_len, max_seq_len);
    if (rc != VERIFY_OK) return rc;
    const verify_attn_params& p = *params;
    if (p.num_seqs > 0 && (!seq_lens || !q_start || !block_tables)) return VERIFY_EINVAL;
    if (total_q > 0 && (!q || !k_cache || !v_cache || !out)) return VERIFY_EINVAL;
    // a query row sits at a position of its own request, so its cache holds
    // at least one block
    if (total_q > 0 && p.num_blocks < 1) return VERIFY_EINVAL;
    AttnPlan pl;
    rc = make_plan(params, total_q, max_q_len, max_seq_len, &pl, k_new != nullptr);
    if (rc != VERIFY_OK) return rc;
    if (workspace_bytes < pl.total_bytes || (pl.total_bytes > 0 && !workspace)) return VERIFY_EWORKSPACE;
    if (p.num_seqs == 0 || total_q == 0) return VERIFY_OK;
    const float scale = p.scale > 0.f ? p.scale : 1.0f / sqrtf((float)p.head_dim);

    if (pl.mfma) {
        MPtrs m{};
        m.q = static_cast<const uint16_t*>(q);
        m.kc = static_cast<const uint8_t*>(k_cache);
        m.vc = static_cast<const uint8_t*>(v_cache);
        m.block_tables = block_tables;
        m.seq_lens = seq_lens;
        m.q_start = q_start;
        m.out = static_cast<uint16_t*>(out);
        m.k_new = static_cast<const uint16_t*>(k_new);
        m.v_new = static_cast<const uint16_t*>(v_new);
        PArgs a{};
        a.num_seqs = p.num_seqs;
        a.hq = p.num_q_heads;
        a.hkv = p.num_kv_heads;
        a.group = p.num_q_heads / p.num_kv_heads;
        a.max_blocks = p.max_blocks_per_seq;
        a.num_blocks = p.num_blocks;
        a.window = p.sliding_window;
        a.max_seq_len = max_seq_len;
        a.scale_log2 = scale * kLog2e;
        a.inv_scale_log2 = a.scale_log2 > 0.f ? 1.f / a.scale_log2 : 0.f;
        a.inline_sched = p.num_seqs <= kInlineSchedSeqs;
        a.sinks = sinks;
        const int64_t max_rows = (int64_t)a.group * std::max(1, max_q_len);
        // one launch per row class, one after another on the stream; each
        // writes only its own requests' outputs
        for (int k = 0; k < pl.nclass; ++k) {
            const AttnPlan::Class& c = pl.cls[k];
            char* ws = static_cast<char*>(workspace) + c.off;
            m.unit_start = reinterpret_cast<int32_t*>(ws);
            m.slot_o = reinterpret_cast<uint16_t*>(ws + c.unit_bytes);
            m.slot_lse = reinterpret_cast<float*>(ws + c.unit_bytes + c.slot_o_bytes);
            a.rows_per_group = c.nw * c.tpw * 16;
            a.rg_max = c.rg_max;
            a.nwg = c.nwg;
            a.spb = c.spb;
            a.rows_lo = c.rows_lo;
            a.rows_hi = c.rows_hi;
            const int64_t class_rows = std::min<int64_t>(max_rows, c.rows_hi);
            if (!launch_persist(a, m, c, p.head_dim, (int)std::min<int64_t>(class_rows, 1 << 30), stream))
                return VERIFY_EUNSUPPORTED;
        }
        return check_launch();
    }

    AttnArgs a{};
    a.q = q;
    a.kc = k_cache;
    a.vc = v_cache;
    a.block_tables = block_tables;
    a.seq_lens = seq_lens;
    a.q_start = q_start;
    a.out = out;
    a.part_o = pl.part_o_bytes ? static_cast<float*>(workspace) : nullptr;
    a.part_lse = pl.part_o_bytes
                     ? reinterpret_cast<float*>(static_cast<char*>(workspace) + pl.part_o_bytes)
                     : nullptr;
    a.num_seqs = p.num_seqs;
    a.hq = p.num_q_heads;
    a.hkv = p.num_kv_heads;
    a.group = p.num_q_heads / p.num_kv_heads;
    a.max_blocks = p.max_blocks_per_seq;
    a.num_blocks = p.num_blocks;
    a.window = p.sliding_window;
    a.max_seq_len = max_seq_len;
    a.scale_log2 = scale * kLog2e;
    a.split_blocks = pl.split_blocks;
    a.max_splits = pl.max_splits;
    a.row_groups = pl.row_groups;
    a.sinks = sinks;
    a.k_new = k_new;
    a.v_new = v_new;
    if (p.head_dim == 128) launch_valu<float, 128>(a, pl, total_q, stream);
    else launch_valu<float, 64>(a, pl, total_q, stream);
    return check_launch();
}

}  // namespace

extern "C" int verify_attention(const verify_attn_params* params, int32_t total_q,
                                int32_t max_q_len, int32_t max_seq_len, const void* q,
                                const void* k_cache, const void* v_cache,
                                const int32_t* block_tables, const int32_t* seq_lens,
                                const int32_t* q_start, const float* sinks, void* out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return attention_call(params, total_q, max_q_len, max_seq_len, q, k_cache, v_cache,
                          block_tables, seq_lens, q_start, sinks, out, workspace, workspace_bytes,
                          nullptr, nullptr, stream);
}

extern "C" int verify_attention_append(const verify_attn_params* params, int32_t total_q,
                                       int32_t max_q_len, int32_t max_seq_len, const void* q,
                                       const void* k_new, const void* v_new, void* k_cache,
                                       void* v_cache, const int32_t* block_tables,
                                       const int32_t* seq_lens, const int32_t* q_start,
                                       const float* sinks, void* out, void* workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
    if (total_q > 0 && (!k_new || !v_new)) return VERIFY_EINVAL;
    return attention_call(params, total_q, max_q_len, max_seq_len, q, k_cache, v_cache,
                          block_tables, seq_lens, q_start, sinks, out, workspace, workspace_bytes,
                          total_q > 0 ? k_new : nullptr, total_q > 0 ? v_new : nullptr, stream);
}

extern "C" int verify_attention_plan(const verify_attn_params* params, int32_t total_q,
                                     int32_t max_q_len, int32_t max_seq_len, int32_t* info) {
    if (!info) return VERIFY_EINVAL;
    int rc = validate(params, total_q, max_q_len, max_seq_len);
    if (rc != VERIFY_OK) return rc;
    AttnPlan pl;
    rc = make_plan(params, total_q, max_q_len, max_seq_len, &pl);
    if (rc != VERIFY_OK) return rc;
    for (int k = 0; k < VERIFY_ATTN_PLAN_INFO; ++k) info[k] = 0;
    if (pl.mfma) {
        info[0] = 1;
        info[5] = pl.nclass;
        for (int k = 0; k < pl.nclass; ++k) {
            const AttnPlan::Class& c = pl.cls[k];
            int32_t* d = k == 0 ? info + 1 : info + 6;
            d[0] = c.nwg;
            d[1] = c.nw * c.tpw * 16;
            d[2] = c.rg_max;
            d[3] = c.spb;
        }
        info[10] = pl.nclass > 1 ? pl.cls[0].rows_hi : INT32_MAX;
    } else {
        info[0] = 0;
        info[1] = pl.max_splits;
        info[2] = kValuRows;
        info[3] = pl.row_groups;
        info[4] = pl.split_blocks;
    }
    return VERIFY_OK;
}

extern "C" int verify_kv_append(const verify_attn_params* params, int32_t total_q,
                                const void* k_new, const void* v_new, const int32_t* block_tables,
                                const int32_t* seq_lens, const int32_t* q_start, void* k_cache,
                                void* v_cache, hipStream_t stream) {
    int rc = validate(params, total_q, 0, 0);
    if (rc != VERIFY_OK) return rc;
    const verify_attn_params& p = *params;
    if (total_q == 0 || p.num_seqs == 0) return VERIFY_OK;
    if (!k_new || !v_new || !block_tables || !seq_lens || !q_start || !k_cache || !v_cache)
        return VERIFY_EINVAL;
    if (p.num_kv_heads > 65535) return VERIFY_EUNSUPPORTED;  // grid y
    const dim3 grid((unsigned)p.num_seqs, (unsigned)p.num_kv_heads);
#define AVERIFY_APPEND(T, D)                                                                       \
    hipLaunchKernelGGL((attn_kv_append<T, D>), grid, dim3(kAppendThreads), 0, stream, p.num_seqs,    \
                       p.num_kv_heads,                                                             \
                       p.max_blocks_per_seq, p.num_blocks, static_cast<const T*>(k_new),          \
                       static_cast<const T*>(v_new), block_tables, seq_lens, q_start,             \
                       static_cast<T*>(k_cache), static_cast<T*>(v_cache))
    if (p.dtype == VERIFY_BF16) {
        if (p.head_dim == 128) AVERIFY_APPEND(uint16_t, 128);
        else AVERIFY_APPEND(uint16_t, 64);
    } else {
        if (p.head_dim == 128) AVERIFY_APPEND(float, 128);
        else AVERIFY_APPEND(float, 64);
    }
#undef AVERIFY_APPEND
    return check_launch();
}
