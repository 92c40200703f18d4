// common.h -- helpers shared by the HIP sources of the verify library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "agentspec_verify.h"

namespace averify {

constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kBlockTokens = 16; // tokens per paged KV block

// ---------------------------------------------------------------- conversions

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> bf16 with round-to-nearest-even (gfx950 v_cvt_pk_bf16_f32; a NaN
// stays a quiet NaN).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

template <typename T> struct Storage;
template <> struct Storage<float> {
    static constexpr int kPer16B = 4;
    __device__ static float load(const float* p, int64_t i) { return p[i]; }
    __device__ static void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Storage<uint16_t> {
    static constexpr int kPer16B = 8;
    __device__ static float load(const uint16_t* p, int64_t i) { return bf16_to_f32(p[i]); }
    __device__ static void store(uint16_t* p, int64_t i, float v) { p[i] = f32_to_bf16(v); }
};

// 16-byte loads.  The streaming variant marks the access non-temporal: data
// read exactly once should not displace cache lines that are reused.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ uint4 ld16_stream(const void* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Unpack one 16-byte vector of storage elements into fp32.
__device__ __forceinline__ void unpack16(const uint4& v, float* out, float) {
    out[0] = __uint_as_float(v.x);
    out[1] = __uint_as_float(v.y);
    out[2] = __uint_as_float(v.z);
    out[3] = __uint_as_float(v.w);
}
__device__ __forceinline__ void unpack16(const uint4& v, float* out, uint16_t) {
    out[0] = bf16_lo(v.x); out[1] = bf16_hi(v.x);
    out[2] = bf16_lo(v.y); out[3] = bf16_hi(v.y);
    out[4] = bf16_lo(v.z); out[5] = bf16_hi(v.z);
    out[6] = bf16_lo(v.w); out[7] = bf16_hi(v.w);
}

// ---------------------------------------------------------------- wave reductions

__device__ __forceinline__ float wave_max_xor(float v, int width) {
    for (int o = 1; o < width; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}
__device__ __forceinline__ float wave_sum_xor(float v, int width) {
    for (int o = 1; o < width; o <<= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = __shfl_xor(lo, o);
    hi = __shfl_xor(hi, o);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    for (int o = 1; o < kWave; o <<= 1) {
        uint64_t w = shfl_xor_u64(v, o);
        v = w > v ? w : v;
    }
    return v;
}

// ---------------------------------------------------------------- argmax keys

// Monotone map from a float to an unsigned key: a > b  <=>  key(a) > key(b)
// for non-NaN values, -0.0 and +0.0 share a key, and NaN maps above +inf.
__device__ __forceinline__ uint32_t order_key(uint32_t bits) {
    const uint32_t mag = bits & 0x7fffffffu;
    if (mag > 0x7f800000u) return 0xffffffffu;
    if (mag == 0) bits = 0;
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

// (order key, ~index) in one word: the larger word has the larger key and,
// among equal keys, the lower index, so a max-reduction keeps the first maximum.
__device__ __forceinline__ uint64_t pack(uint32_t key, uint32_t idx) {
    return ((uint64_t)key << 32) | (uint32_t)(0xffffffffu - idx);
}

// ---------------------------------------------------------------- global->LDS pipelines

// s_waitcnt immediate (gfx9 encoding) that waits for vmcnt == 0 and leaves
// expcnt (bits 6:4) and lgkmcnt (bits 11:8) at their no-wait maxima.
constexpr int kWaitVmcnt0 = 0x0F70;

// Workgroup barrier that orders LDS only: the staging rings live in LDS and
// global memory needs no ordering between the waves of a workgroup.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// 16 bytes per lane from global memory straight into LDS (gfx950
// global_load_lds_dwordx4): lane l of the wavefront writes LDS bytes
// [lds + 16 l, lds + 16 l + 16).  The load is issued from inline assembly so
// that its completion is tracked by the pipeline's explicit waits alone; the
// compiler does not see it and adds no waits of its own.  m0 (the LDS base of
// the copy) is set inside the same statement and listed as clobbered; nothing
// else in these kernels uses m0 (no LDS-direct, movrel or message
// instructions), so no value of the compiler's lives in it across the copy.
__device__ __forceinline__ void dma16(uint32_t lds_wave_base, const void* src) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(__builtin_amdgcn_readfirstlane(lds_wave_base)), "v"(src)
                 : "memory", "m0");
}

// Wait until at most N vector-memory operations of this wavefront are in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt is a 6-bit counter");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// ---------------------------------------------------------------- host helpers

// Greedy acceptance from per-(row, chunk) packed maxima (verify_accept.hip):
// reduces partial[row * nchunks + c] over c to each row's argmax, then writes
// the accepted drafts and the bonus token of every request.  Returns a status.
int launch_accept_scan(int num_seqs, const int32_t* q_start, const int32_t* tokens,
                       const uint64_t* partial, int nchunks, int32_t* argmax_out,
                       int32_t* accept_len, int32_t* num_emitted, int32_t* emitted,
                       hipStream_t stream);

inline int check_launch() {
    return hipGetLastError() == hipSuccess ? VERIFY_OK : VERIFY_EHIP;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace averify
