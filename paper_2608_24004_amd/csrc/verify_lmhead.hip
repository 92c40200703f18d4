// verify_lmhead.hip -- the LM head of the verify pass fused with greedy
// acceptance: logits[r][v] = <hidden[r], weight[v]> for every scored position
// r and vocabulary entry v, reduced to each row's argmax on the fly, so the
// [total_q][vocab] logits never reach HBM; then the longest accepted draft
// prefix plus the bonus token (paper Sec. 2.2: the target scores all proposed
// tokens in one pass and the result equals plain greedy decoding).
//
// The contraction is dense (every weight row meets every scored row), so it
// runs on MFMA: v_mfma_f32_16x16x32_bf16 with the vocabulary on the M side
// (A = 16 weight rows x 32 hidden dims) and the scored rows on the N side
// (B = 32 hidden dims x 16 rows).  A lane of a 16 x 16 result holds one
// scored row (column l % 16) and four consecutive vocabulary entries, so most
// of the argmax is a running compare inside the lane.
//
// Work split.  lmhead_argmax launches one 8-wavefront workgroup per compute
// unit (two wavefronts per SIMD).  The vocabulary is cut into 16-row tiles.
// Workgroups form groups, one per XCD (workgroup w runs on XCD w % 8), and
// each group owns one eighth of the tiles.  Up to 288 scored rows, a group's
// 32 workgroups split its tiles evenly.  Beyond that the rows are cut into
// row chunks of at most 288: the group's workgroups are dealt out over the
// chunks, and the workgroups of different chunks split the group's tiles the
// same way, so the workgroups that share a vocabulary range run side by side
// on one XCD and the weight they read comes from HBM once, then from that
// XCD's L2 (Qwen shapes at 2152 rows: eight chunks of 269 rows, 3.55 ms ->
// 2.35 ms against eight workgroup-private passes over the weight).  Rows
// beyond 288 per workgroup of a group are walked in rounds, one after
// another.  Where workgroups land on XCDs decides only the speed.
//
// A workgroup walks its tiles in passes: the register file holds the pass's
// block of fp32 logits, so every pass sees all of its chunk's scored rows at
// once.  Wavefront (g, q) takes scored-row group g (of two: MT tiles, up to 9)
// and vocabulary group q (of four: NT tiles of the pass) and holds NT x MT
// result tiles of 4 floats per lane; NT is 5, or 6 where that packs the
// workgroup's tiles into fewer slots (kLmNT).
// Qwen shapes: MT 9, NT 5, passes of 20 tiles (320 x 288 logits), 37 or 38
// tiles per workgroup, two passes, the hidden states staged twice.
//
// Per pass the hidden dimension is walked in steps of 64.  A step's weight
// tiles and scored-row tiles (128 contiguous bytes per row: the HBM stream
// runs at about 5.7 TB/s with rows of this length against 3.5 TB/s with
// 64-byte rows) are copied once, 16 bytes per lane, from global memory into
// one of two LDS stages; every wavefront reads its MFMA operands from there.
// While a step's products run, the next step's copies are issued between
// them.  Only rows that exist are staged: a pass holds exactly its tiles, with
// no padding rows.  At the end of a pass each lane folds its logits into a
// (maximum, first index) per scored row, merged across the workgroup with a
// 64-bit LDS max.
//
// After the last pass of a row chunk the workgroup stores one packed (order
// key, ~index) word per scored row in its column of the row's partials (the
// format of verify_accept's per-chunk partials; a column no workgroup owns
// holds 0, which loses every comparison), and the same acceptance scan
// finishes the step.
#include <type_traits>

#include "common.h"

// m0 is set inside the global->LDS load sequence (see dma16_if_lt); the
// compiler reloads m0 before each of its own uses, so clobbering it there is
// safe.
#pragma clang diagnostic ignored "-Winline-asm"

namespace averify {
namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

constexpr int kLmRowGroups = 2;                         // scored-row groups per workgroup
constexpr int kLmVocGroups = 4;                         // vocabulary groups per workgroup
constexpr int kLmWaves = kLmRowGroups * kLmVocGroups;   // 8
constexpr int kLmThreads = kLmWaves * kWave;
constexpr int kLmTile = 16;                             // rows per tile (MFMA M and N)
constexpr int kLmStageTiles = 38;                       // 2 KiB tiles per LDS stage at most
constexpr int kLmMaxRT = 18 / kLmRowGroups;             // scored-row tiles per group
constexpr int kLmChunkRows = kLmRowGroups * kLmMaxRT * kLmTile;  // 288

// Vocabulary tiles per wavefront and pass (NT): 5, or 6 for 5 to 7 scored-row
// tiles per wavefront (MT), where the two LDS stages (2 MT + 4 NT tiles of 2 KiB
// each, 38 at most) and the accumulators (4 NT MT registers, 180 at most) hold
// it.  Every pass runs NT tiles per wavefront whether or not the workgroup has
// that many left, so the launch takes the NT with the fewest tile slots
// (passes x NT; plan_lmhead).  DSK shapes (192-row chunks, 62.6 tiles per
// workgroup): NT 6 in three passes against NT 5 in four, 478 -> 410 us.
constexpr int kLmNT = 5;
constexpr bool lm_wide_ok(int mt) { return mt >= 5 && mt <= 7; }
constexpr int kLmMinStep = 32;                          // hidden_size granularity
constexpr int kLmStep = 64;                             // hidden dims per LDS stage
constexpr int kLmXcds = 8;                              // MI355X: 8 XCDs, each with its own L2

struct LArgs {
    int T;           // scored rows
    int H;           // hidden size (multiple of kLmMinStep)
    int V;           // vocabulary
    int tiles;       // vocabulary tiles of 16 rows
    int nwg;         // workgroups
    int xg;          // workgroup groups, one vocabulary slice each (workgroup w is in group w % xg)
    int kg;          // workgroups per group (nwg / xg)
    int nc;          // row chunks per round; a group's workgroups are dealt out over them
    int rounds;      // rounds of row chunks, walked one after another
    int round_rows;  // scored rows per round (the last round may hold fewer)
    int ncols;       // partial words per scored row: xg * ceil(kg / nc)
    int nk;          // hidden steps per pass: ceil(H / kLmStep)
    int tail;        // 1 if the last step holds only 32 dims (H % 64 == 32)
};

// A staged row holds CH 16-byte chunks.  Chunk c of tile row r (0..15) is
// stored at position c ^ ((r >> 1) mod CH).  An operand read (lane l: row
// l % 16, logical chunk l / 16 of the 32-dim half) then takes gfx950's minimum
// of four LDS cycles per ds_read_b128, measured for 64- and 128-byte rows;
// the plain layout takes twice (64-byte rows) or four times (128-byte rows) as
// long, and so does an XOR with (r >> 2).
template <int CH>
__device__ __forceinline__ int swz(int r, int c) {
    return c ^ ((r >> 1) & (CH - 1));
}

// f(std::integral_constant<int, i>) for i = 0 .. N-1
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I < N) {
        f(std::integral_constant<int, I>{});
        static_for<N, I + 1>(f);
    }
}

// A pointer every lane holds the same value of, in scalar registers.
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
    const uint64_t u = (uint64_t)(uintptr_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)u);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(u >> 32));
    return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// If C < n: 16 bytes per lane from global memory at sbase + voff (a
// wavefront-uniform base and a per-lane 32-bit byte offset, the
// global_load_lds_dwordx4 saddr form) into LDS bytes [lds + 16 l, lds + 16 l +
// 16) of lane l.  The test is made inside the statement, so a skipped load
// leaves no branch in the compiler's view of the surrounding products.
template <int C>
__device__ __forceinline__ void dma16_if_lt(int n, uint32_t lds_wave_base, const void* sbase,
                                            uint32_t voff) {
    asm volatile("s_cmp_le_i32 %3, %4\n\ts_cbranch_scc1 1f\n\t"
                 "s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2\n1:"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds_wave_base)), "v"(voff),
                   "s"(uniform_ptr(sbase)), "s"(n), "n"(C)
                 : "memory", "m0", "scc");
}

// Whether logit x replaces the running maximum best: logits arrive in
// ascending vocabulary order, so a strict compare keeps the lowest index among
// equal maxima (-0.0 == +0.0), and the first NaN replaces any number and is
// then kept (a NaN counts as the maximum).  !(x <= best) is x > best or x a
// NaN; once best is a NaN nothing replaces it.  Bitwise operators keep it
// free of branches.
__device__ __forceinline__ bool fold_take(float x, float best) {
    return !(x <= best) & (best == best);
}

// Largest of v over lanes l, l ^ 16, l ^ 32 and l ^ 48 (the four lanes that
// hold one scored row of a 16 x 16 result tile).  Each permlane swap exchanges
// half of the wavefront between its two operands; with both operands equal,
// lane l gets the values of l and l ^ 32 (l ^ 16), in an order that is the
// same for both halves of the word.
__device__ __forceinline__ uint64_t max4_u64(uint64_t v) {
    auto both = [](uint64_t x, auto swap) {
        const auto lo = swap((uint32_t)x);
        const auto hi = swap((uint32_t)(x >> 32));
        const uint64_t c0 = ((uint64_t)hi[0] << 32) | lo[0];
        const uint64_t c1 = ((uint64_t)hi[1] << 32) | lo[1];
        return c0 > c1 ? c0 : c1;
    };
    v = both(v, [](uint32_t u) { return __builtin_amdgcn_permlane32_swap(u, u, false, false); });
    return both(v, [](uint32_t u) { return __builtin_amdgcn_permlane16_swap(u, u, false, false); });
}

// MT = scored-row tiles per row group (the row chunk holds at most 2 MT
// tiles), NT = vocabulary tiles per wavefront and pass
template <int MT, int NT>
__global__ __launch_bounds__(kLmThreads)
__attribute__((amdgpu_waves_per_eu(kLmRowGroups, kLmRowGroups)))
void lmhead_argmax(LArgs a, const uint16_t* __restrict__ hid, const uint16_t* __restrict__ wt,
                   uint64_t* __restrict__ partial) {
    constexpr int KS = kLmStep;
    constexpr int CH = KS / 8;                            // 16-byte chunks per staged row
    constexpr int TB = kLmTile * KS * 2;                  // bytes per staged tile (2 KiB)
    constexpr int LPT = TB / 1024;                        // 1 KiB loads per tile
    constexpr int KSUB = KS / 32;                         // 32-dim products per stage
    constexpr int HT = kLmRowGroups * MT;                 // scored-row tile slots per stage
    constexpr int PT = kLmVocGroups * NT;                 // vocabulary tiles per pass
    constexpr int STAGE = (HT + PT) * TB;
    constexpr int CPT = ((HT + PT) * LPT + kLmWaves - 1) / kLmWaves;  // loads per wave
    static_assert(HT + PT <= kLmStageTiles && 4 * NT * MT <= 180, "stages and accumulators");
    constexpr int SLOTS = KSUB * MT;                      // product groups per step
    // load c2 is issued before product group slot_of(c2) = h MT + n: the
    // loads are spread over the first two thirds of the step, so that they
    // queue while the matrix cores run instead of all after the barrier
    // (measured 459 -> 392 us on the Qwen-shaped call)
    constexpr int SPREAD = SLOTS * 2 / 3 > 0 ? SLOTS * 2 / 3 : 1;
    constexpr auto slot_of = [](int c2) { return c2 * SPREAD / CPT; };
    static_assert(kLmWaves % LPT == 0, "a wavefront loads the same part of every tile");
    static_assert(CPT < 64, "vmcnt range");

    __shared__ __attribute__((aligned(1024))) uint8_t stage[2][STAGE];

    const int w = blockIdx.x;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);  // wavefront-uniform
    const int r16 = lane & 15, kq = lane >> 4;
    const int vq = wv % kLmVocGroups;  // vocabulary group
    const int rg = wv / kLmVocGroups;  // scored-row group: tiles [MT rg, MT (rg + 1)) of a chunk

    // This workgroup's place: group x (one per XCD when the launch fills
    // them: consecutive workgroups go to consecutive XCDs), row chunk c of
    // every round, and j-th of the group's nc_w workgroups on that chunk.  The
    // group's vocabulary slice is cut into nc_w ranges; the workgroups of
    // different chunks that share a range run side by side on one XCD, so the
    // weight they read is fetched from HBM once and served from that XCD's L2
    // to the others.  Chunk c holds a share of a round's rows proportional to
    // nc_w, which gives every workgroup the same work.
    const int x = w % a.xg, k = w / a.xg;
    const int c_w = k % a.nc, j_w = k / a.nc;
    const int full = a.kg / a.nc, rem = a.kg % a.nc;
    const int nc_w = full + (c_w < rem ? 1 : 0);            // workgroups of chunk c_w in the group
    const int s_w = c_w * full + min(c_w, rem);             // of chunks before it
    const int nmax = full + (rem ? 1 : 0);
    const int x0 = (int)((int64_t)a.tiles * x / a.xg), x1 = (int)((int64_t)a.tiles * (x + 1) / a.xg);
    const int t0 = x0 + (int)((int64_t)(x1 - x0) * j_w / nc_w);
    const int t1 = x0 + (int)((int64_t)(x1 - x0) * (j_w + 1) / nc_w);
    const int ntw = t1 - t0;
    const int col = x * nmax + j_w;  // this workgroup's partial word of a row
    const int passes = max(1, (ntw + PT - 1) / PT);
    auto pass_tiles = [&](int p, int& pt0, int& pt) {
        pt0 = t0 + ntw * p / passes;
        pt = t0 + ntw * (p + 1) / passes - pt0;
    };
    auto chunk_tiles = [&](int rnd, int& r0, int& rows) {
        const int base = rnd * a.round_rows;
        const int64_t tr = min(a.T - base, a.round_rows);
        r0 = base + (int)(tr * s_w / a.kg);
        rows = base + (int)(tr * (s_w + nc_w) / a.kg) - r0;
    };

    const uint32_t stage_lds =
        (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)&stage[0][0];
    const int units = a.rounds * passes * a.nk;

    // ---- loader.  Unit u = (row chunk, pass, hidden step) fills one stage:
    // its scored-row tiles into slots [0, HT) and its vocabulary tiles into
    // slots [HT, HT + PT), two 1 KiB global->LDS loads per tile.  Stage load
    // L (tile L / 2, part L % 2) is issued by wavefront L % 8, so a wavefront
    // always loads the same part of its tiles: lane l moves tile row
    // (64 part + l) / 8, stored chunk (64 part + l) % 8.  Each load reads from
    // a wavefront-uniform base (the tile's first row at the unit's step) plus a
    // per-lane offset; rows past the scored rows or the vocabulary repeat the
    // last one.  In a 32-dim last step the upper four chunks repeat the lower.
    const int jpart = wv % LPT;
    const int lrow = (jpart * kWave + lane) / CH;
    const int lc16 = swz<CH>(lrow, (jpart * kWave + lane) % CH) * 16;
    const int i0 = wv / LPT;  // first tile of this wavefront; its c-th load is tile i0 + 4 c
    constexpr int TSTEP = kLmWaves / LPT;  // tiles between a wavefront's consecutive loads
    // the loader's unit: index, hidden step, and per (chunk, pass) the global
    // base of this wavefront's first scored-row tile (h) and vocabulary tile
    // (v), their LDS slots, the last row a load may read relative to each
    // base (rows past it repeat it), and the load counts: loads c < hc are
    // scored-row tiles, c < vc exist at all (0 once every unit is loaded)
    int l_u = 0, l_ks = 0, l_tail = 0, l_hslot = 0, l_vslot = 0, l_hc = 0, l_vc = 0;
    int l_hlim = 0, l_vlim = 0;
    const uint16_t* l_hbase = hid;
    const uint16_t* l_vbase = wt;
    auto loader_set = [&](int u) {  // the loader's unit becomes u (< units)
        l_u = u;
        const int cp = u / a.nk;
        const int ks = u - cp * a.nk;
        l_ks = ks;
        l_tail = a.tail && ks == a.nk - 1;
        if (ks != 0 && u != 0) return;  // same (chunk, pass) as the previous unit
        const int c = cp / passes, p = cp - (cp / passes) * passes;
        int r0, rows, pt0, pt;
        chunk_tiles(c, r0, rows);
        pass_tiles(p, pt0, pt);
        const int htc = (rows + kLmTile - 1) / kLmTile;
        const int hrow = r0 + i0 * kLmTile, vrow = (pt0 - htc + i0) * kLmTile;
        l_hbase = hid + (int64_t)hrow * a.H;
        l_vbase = wt + (int64_t)vrow * a.H;
        l_hslot = i0;
        l_vslot = HT - htc + i0;
        l_hlim = a.T - 1 - hrow;
        l_vlim = a.V - 1 - vrow;
        l_hc = max(0, (htc - i0 + TSTEP - 1) / TSTEP);
        l_vc = max(0, (htc + pt - i0 + TSTEP - 1) / TSTEP);
    };
    // per step: the loader's bases at its hidden step, the LDS addresses of
    // its first tiles in stage st, and the lane's chunk offset
    const uint16_t* d_hb = hid;
    const uint16_t* d_vb = wt;
    uint32_t d_hl = 0, d_vl = 0, d_c16 = 0;
    int d_n = 0;
    auto dma_prepare = [&](int st) {
        d_hb = l_hbase + l_ks * KS;
        d_vb = l_vbase + l_ks * KS;
        const uint32_t sbase = stage_lds + st * STAGE + jpart * 1024;
        d_hl = sbase + l_hslot * TB;
        d_vl = sbase + l_vslot * TB;
        d_c16 = (uint32_t)(l_tail ? (lc16 & 63) : lc16);
        d_n = l_u < units ? l_vc : 0;
    };
    // load c2 of this wavefront for the prepared unit
    auto dma_one = [&](auto c2c) {
        constexpr int c2 = decltype(c2c)::value;
        constexpr int tr = c2 * TSTEP * kLmTile;  // row of the load's tile from its base
        const bool is_h = c2 < l_hc;
        const uint32_t voff = (uint32_t)(min(tr + lrow, is_h ? l_hlim : l_vlim) * (a.H * 2)) + d_c16;
        dma16_if_lt<c2>(d_n, (is_h ? d_hl : d_vl) + c2 * TSTEP * TB, is_h ? d_hb : d_vb, voff);
    };
    auto dma_all = [&](int st) {
        dma_prepare(st);
        static_for<CPT>([&](auto c2) { dma_one(c2); });
    };
    auto loader_next = [&]() {
        if (l_u + 1 < units) loader_set(l_u + 1);
        else l_u = units;
    };

    // ---- running maxima of the row chunk, one packed (order key, ~index)
    // word per scored row, merged with a 64-bit LDS max at the end of every
    // pass (so that no register holds them while the products run)
    __shared__ uint64_t row_max[kLmChunkRows];
    for (int r = tid; r < kLmChunkRows; r += kLmThreads) row_max[r] = 0;

    // One hidden step on stage st: NT vocabulary tiles (first tile vt0 of the
    // pass) x MT scored-row tiles, KSUB products of 32 dims each.  The weight
    // fragments of a 32-dim half are read once and kept; each scored-row
    // fragment feeds NT products.  The loads of the loader's unit into the
    // other stage are issued between the product groups.
    auto compute = [&](int st, auto& acc, int vt0, int nt) {
        constexpr int G = KSUB * MT;  // product groups of the step
        const int tmax = max(nt - 1, 0);
        const uint8_t* sb = stage[st];
        dma_prepare(st ^ 1);
        const int off0 = r16 * (CH * 16);
        auto woff = [&](int h) { return off0 + swz<CH>(r16, 4 * h + kq) * 16; };
        // scored-row fragment of group g (32-dim half g / MT, tile g % MT),
        // read by an LDS load the compiler does not see
        const uint32_t hrow = (uint32_t)(uintptr_t)(
            __attribute__((address_space(3))) const uint8_t*)(sb + rg * MT * TB + off0);
        auto hread = [&](auto gc) {
            constexpr int g = decltype(gc)::value;
            constexpr int h = g / MT, n = g % MT;
            const uint32_t addr = hrow + (uint32_t)(swz<CH>(r16, 4 * h + kq) * 16);
            u32x4 v;
            asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "n"(n * TB) : "memory");
            return v;
        };
        auto wread = [&](int h, int t) {
            return __builtin_bit_cast(
                bf16x8_t, *reinterpret_cast<const uint4*>(sb + (HT + vt0 + min(t, tmax)) * TB + woff(h)));
        };
        bf16x8_t wf[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) wf[t] = wread(0, t);
        // three scored-row fragments in flight: the fragment of group g + 2 is
        // requested before group g's products, and an explicit wait (every
        // LDS load but the two newest has landed) makes group g's ready.  The
        // fragment passes through the wait as an operand, so the products
        // that use it cannot be placed before the wait.
        u32x4 hf[4];
        hf[0] = hread(std::integral_constant<int, 0>{});
        if constexpr (G > 1) hf[1] = hread(std::integral_constant<int, 1>{});
        if constexpr (G > 2) hf[2] = hread(std::integral_constant<int, 2>{});
        static_for<G>([&](auto gc) {
            constexpr int g = decltype(gc)::value;
            constexpr int h = g / MT, n = g % MT;
            static_for<CPT>([&](auto c2) {
                if constexpr (slot_of(decltype(c2)::value) == g) dma_one(c2);
            });
            if constexpr (g + 3 < G) {
                hf[(g + 3) % 4] = hread(std::integral_constant<int, g + 3>{});
                asm volatile("s_waitcnt lgkmcnt(3)" : "+v"(hf[g % 4]) : : "memory");
            } else if constexpr (g + 2 < G) {
                asm volatile("s_waitcnt lgkmcnt(2)" : "+v"(hf[g % 4]) : : "memory");
            } else if constexpr (g + 1 < G) {
                asm volatile("s_waitcnt lgkmcnt(1)" : "+v"(hf[g % 4]) : : "memory");
            } else {
                asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(hf[g % 4]) : : "memory");
            }
            const bf16x8_t hv = __builtin_bit_cast(bf16x8_t, hf[g % 4]);
            if constexpr (n == MT - 1 && h + 1 < KSUB) {
                // the half's last group: each weight fragment is reloaded for
                // the next half right after its last product
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    acc[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t], hv, acc[t][n], 0, 0, 0);
                    wf[t] = wread(h + 1, t);
                }
            } else {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    acc[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[t], hv, acc[t][n], 0, 0, 0);
            }
        });
    };

    // fold a pass's logits into the chunk's maxima: lane (kq, r16) holds
    // vocabulary entries 4 kq .. 4 kq + 3 of each tile for scored row r16
    auto end_pass = [&](auto& acc, int vbase, int nt) {
#pragma unroll
        for (int n = 0; n < MT; ++n) {
            float best = -INFINITY;
            int bloc = -1;  // t * 16 + e of the maximum
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                // entries past the pass's tiles or the vocabulary count as -inf,
                // which replaces nothing
                const bool full = t < nt && vbase + (t + 1) * kLmTile <= a.V;  // wavefront-uniform
                const int lim = t < nt ? a.V - (vbase + t * kLmTile + 4 * kq) : 0;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    float x = acc[t][n][e];
                    if (!full) x = e < lim ? x : -INFINITY;
                    const bool take = fold_take(x, best);
                    best = take ? x : best;
                    bloc = take ? t * kLmTile + e : bloc;
                }
            }
            uint64_t pk = bloc >= 0 ? pack(order_key(__float_as_uint(best)), (uint32_t)(vbase + 4 * kq + bloc)) : 0;
            pk = max4_u64(pk);
            if (kq == 0 && pk != 0) atomicMax(reinterpret_cast<unsigned long long*>(&row_max[(rg * MT + n) * kLmTile + r16]),
                                                (unsigned long long)pk);
        }
    };

    // store the chunk's maxima, one packed word per scored row, and clear
    // them for the next chunk
    auto end_chunk = [&](int c) {
        int r0, rows;
        chunk_tiles(c, r0, rows);
        lds_barrier();  // every wavefront's last pass is merged
        const int v_first = t0 * kLmTile;
        for (int r = tid; r < kLmChunkRows; r += kLmThreads) {
            uint64_t m = row_max[r];
            row_max[r] = 0;
            // a range whose logits are all -inf reports its first entry
            if (m == 0 && ntw > 0) m = pack(order_key(__float_as_uint(-INFINITY)), (uint32_t)v_first);
            if (r < rows) {
                uint64_t* pr = partial + (int64_t)(r0 + r) * a.ncols;
                pr[col] = m;
                // a chunk with fewer workgroups than nmax leaves the group's
                // last word of its rows to its last workgroup: the neutral 0
                if (nc_w < nmax && j_w == nc_w - 1) pr[col + 1] = 0;
            }
        }
    };

    // Double-buffered pipeline per hidden step: wait for this wavefront's
    // loads of the step's stage, barrier (everyone's loads landed, everyone is
    // done with the other stage), then compute on this stage while the next
    // unit's loads go into the other one.
    loader_set(0);
    dma_all(0);
    loader_next();
    int st = 0;
    for (int rnd = 0; rnd < a.rounds; ++rnd) {
        for (int p = 0; p < passes; ++p) {
            int pt0, pt;
            pass_tiles(p, pt0, pt);
            const int vt0 = pt * vq / kLmVocGroups;
            const int nt = pt * (vq + 1) / kLmVocGroups - vt0;
            // every wavefront runs NT vocabulary tiles; a group with
            // fewer repeats its last one (or the pass's first) and folds only
            // its own
            f32x4_t acc[NT][MT];
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int n = 0; n < MT; ++n) acc[t][n] = f32x4_t{};
            int ks = 0;
            do {  // nk >= 1
                wait_vmcnt<0>();
                lds_barrier();
                if (a.tail && ks == a.nk - 1) {
                    // a 32-dim last step: clear dims 32..63 of every staged row
                    // (they repeat dims 0..31), so the upper half adds exact zeros
                    for (int e = tid; e < (HT + PT) * kLmTile * 4; e += kLmThreads) {
                        const int row = e >> 2;
                        *reinterpret_cast<uint4*>(stage[st] + row * (CH * 16) +
                                                  swz<CH>(row & 15, 4 + (e & 3)) * 16) = make_uint4(0, 0, 0, 0);
                    }
                    lds_barrier();
                }
                compute(st, acc, vt0, nt);
                loader_next();
                st ^= 1;
            } while (++ks < a.nk);
            end_pass(acc, (pt0 + vt0) * kLmTile, nt);
        }
        end_chunk(rnd);
    }
    // no global->LDS load may still be writing when the workgroup's LDS is freed
    wait_vmcnt<0>();
}

template <int MT, int NT>
void launch_lmhead(const LArgs& a, const uint16_t* hid, const uint16_t* wt, uint64_t* partial,
                   hipStream_t stream) {
    hipLaunchKernelGGL((lmhead_argmax<MT, NT>), dim3(a.nwg), dim3(kLmThreads), 0, stream, a, hid,
                       wt, partial);
}

// launch lmhead_argmax<mt, nt> (1 <= mt <= kLmMaxRT; nt kLmNT, or kLmNT + 1
// where lm_wide_ok(mt))
template <int M = 1>
bool launch_lmhead_mt(int mt, int nt, const LArgs& a, const uint16_t* hid, const uint16_t* wt,
                      uint64_t* partial, hipStream_t stream) {
    if constexpr (M > kLmMaxRT) {
        return false;
    } else {
        if (mt == M) {
            if (nt == kLmNT) {
                launch_lmhead<M, kLmNT>(a, hid, wt, partial, stream);
                return true;
            }
            if constexpr (lm_wide_ok(M)) {
                if (nt == kLmNT + 1) {
                    launch_lmhead<M, kLmNT + 1>(a, hid, wt, partial, stream);
                    return true;
                }
            }
            return false;
        }
        return launch_lmhead_mt<M + 1>(mt, nt, a, hid, wt, partial, stream);
    }
}

struct LmPlan {
    LArgs a;
    int mt, nt;
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
    return num_seqs >= 0 && total_q >= 0 && hidden_size >= kLmMinStep && hidden_size % kLmMinStep == 0 &&
           vocab >= 1 && vocab < (int64_t)0x7fffffff;
}

LmPlan plan_lmhead(int32_t total_q, int32_t hidden_size, int64_t vocab) {
    LmPlan pl{};
    LArgs& a = pl.a;
    a.T = total_q;
    a.H = hidden_size;
    a.V = (int)vocab;
    a.tiles = (int)((vocab + kLmTile - 1) / kLmTile);
    a.nwg = std::min(lm_cus(), a.tiles);
    a.xg = a.nwg % kLmXcds == 0 ? kLmXcds : 1;
    a.kg = a.nwg / a.xg;
    // rounds: as few as hold the rows (a round's chunks hold at most 288 rows
    // each, one chunk per workgroup of a group at most)
    const int64_t per_round = (int64_t)kLmChunkRows * a.kg;
    a.rounds = (int)std::max<int64_t>(1, (total_q + per_round - 1) / per_round);
    a.round_rows = std::max(1, (int)(((int64_t)total_q + a.rounds - 1) / a.rounds));
    // chunks per round: the fewest whose largest chunk (the workgroups of a
    // group dealt out over them, rows in proportion) fits 288 rows
    int rows_max = a.round_rows;
    for (a.nc = 1; a.nc <= a.kg; ++a.nc) {
        const int nmax = (a.kg + a.nc - 1) / a.nc;
        rows_max = (int)(((int64_t)a.round_rows * nmax + a.kg - 1) / a.kg);
        if (rows_max <= kLmChunkRows) break;
    }
    a.ncols = a.xg * ((a.kg + a.nc - 1) / a.nc);
    const int htc = (rows_max + kLmTile - 1) / kLmTile;
    pl.mt = std::max(1, (htc + kLmRowGroups - 1) / kLmRowGroups);
    // vocabulary tiles per wavefront and pass: the fewest tile slots for the
    // largest workgroup's tiles (ties to the narrower)
    const int64_t per_group = (a.tiles + a.xg - 1) / a.xg;
    const int64_t ntw = (per_group + a.kg / a.nc - 1) / (a.kg / a.nc);
    auto slots = [&](int nt) { return (ntw + kLmVocGroups * nt - 1) / (kLmVocGroups * nt) * nt; };
    pl.nt = lm_wide_ok(pl.mt) && slots(kLmNT + 1) < slots(kLmNT) ? kLmNT + 1 : kLmNT;
    a.nk = (hidden_size + kLmStep - 1) / kLmStep;
    a.tail = hidden_size % kLmStep != 0;
    pl.partial_bytes = align_up((size_t)total_q * a.ncols * sizeof(uint64_t), 256);
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
        if (!launch_lmhead_mt(pl.mt, pl.nt, pl.a, hs, ws, partial, stream)) return VERIFY_EUNSUPPORTED;
        if (check_launch() != VERIFY_OK) return VERIFY_EHIP;
    }
    return launch_accept_scan(num_seqs, q_start, tokens, partial, pl.a.ncols, am, accept_len,
                              num_emitted, emitted, stream);
}
