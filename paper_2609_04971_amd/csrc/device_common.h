// Device helpers shared by the gfx950 kernels: scoped atomics, a bounded
// wait, wave shuffles and DPP reductions, and bf16 rounding.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "internal.h"

namespace bkv {
namespace dev {

// 16 bytes as a native vector: loads and stores of it are single 128-bit
// memory instructions and it always stays in registers (a struct copy of
// uint4 goes through memcpy and can end up in scratch).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Hand-offs between work items of one launch.  The MI355X's eight XCDs
// have separate L2 caches.  Agent-scope *atomic* loads and stores are
// coherent across them by themselves (they carry the sc1 cache policy);
// agent-scope acquire/release fences would instead write back and
// invalidate whole L2 caches, which is far too slow to do per work item.
// So data passed between work items is written and read only with these
// atomic accesses, and ordering comes from waiting for the wave's memory
// operations to complete before the store that publishes them.
__device__ inline float ld_coherent(const float* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_coherent(float* p, float v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline int ld_flag(const int* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_flag(int* p, int v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline int fetch_add_relaxed(int* p, int v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void raise_error(int* hdr, int bits) {
    __hip_atomic_fetch_or(hdr + kHdrErr, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until every load and store this wave has issued has completed
// (s_waitcnt with all counters at zero).  Called by every thread before
// the workgroup barrier that precedes a publishing store.
__device__ inline void wait_all_memory() { __builtin_amdgcn_s_waitcnt(0); }

// Bounded wait for a flag to become non-zero.  Every wait in this library
// is on work with a lower ticket, which has already started and publishes
// before it waits on anything, so it ends; the bound only turns a broken
// invariant into an error instead of a hang.  About 2^22 polls with a short
// sleep between them.
constexpr int kSpinLimit = 1 << 22;
__device__ inline bool wait_flag(const int* p) {
    for (int i = 0; i < kSpinLimit; ++i) {
        if (ld_flag(p) != 0) return true;
        __builtin_amdgcn_s_sleep(1);
    }
    return false;
}

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0..N-1.
// Keeps register arrays indexed by constants from the start, so they are
// never demoted to scratch memory.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Workspace stamp check (one thread).
__device__ inline bool stamp_ok(const int* hdr, int P, int budget) {
    return (uint32_t)hdr[kHdrMagic] == kWsMagic && hdr[kHdrP] == P && hdr[kHdrBudget] == budget;
}

__device__ inline float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, 64); }
__device__ inline int shfl_xor_i(int v, int m) { return __shfl_xor(v, m, 64); }

// Wave reductions over all 64 lanes without an LDS round trip: DPP swaps
// within quads (quad_perm [1,0,3,2], then [2,3,0,1]), the half-row mirror
// and the row mirror leave every lane of a 16-lane row holding the row's
// result; the four row results are then combined as scalars (readlane), so
// the answer is wave-uniform.  All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ unsigned dpp_min_u32(unsigned v) {
    const unsigned w = (unsigned)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xf, 0xf, false);
    return w < v ? w : v;
}

__device__ __forceinline__ unsigned wave_min_u32(unsigned v) {
    v = dpp_min_u32<0xb1>(v);
    v = dpp_min_u32<0x4e>(v);
    v = dpp_min_u32<0x141>(v);
    v = dpp_min_u32<0x140>(v);
    const unsigned a = (unsigned)__builtin_amdgcn_readlane((int)v, 0), b = (unsigned)__builtin_amdgcn_readlane((int)v, 16);
    const unsigned c = (unsigned)__builtin_amdgcn_readlane((int)v, 32), d = (unsigned)__builtin_amdgcn_readlane((int)v, 48);
    return min(min(a, b), min(c, d));
}

// Lexicographic minimum of 64-bit keys over the wave: the high words first,
// then the low words of the lanes that hold it.
__device__ __forceinline__ unsigned long long wave_min_u64(unsigned long long v) {
    const unsigned hi = wave_min_u32((unsigned)(v >> 32));
    const unsigned lo = wave_min_u32((unsigned)(v >> 32) == hi ? (unsigned)v : 0xffffffffu);
    return ((unsigned long long)hi << 32) | lo;
}

// Order-preserving map of a float to an unsigned key (-0 counts as +0).
__device__ __forceinline__ unsigned ord_key(float f) {
    unsigned u = __float_as_uint(f == 0.f ? 0.f : f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf, false));
}

// Sum within each quad of lanes (all four lanes hold it).
__device__ __forceinline__ float quad_sum(float v) { return dpp_add<0x4e>(dpp_add<0xb1>(v)); }

// Sum within each row of 16 lanes (every lane of the row holds it).
__device__ __forceinline__ float row16_sum(float v) { return dpp_add<0x140>(dpp_add<0x141>(quad_sum(v))); }

// Sum over the wave, the same in every lane.
__device__ __forceinline__ float wave_sum(float v) {
    v = dpp_add<0x140>(dpp_add<0x141>(quad_sum(v)));
    const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (a + b) + (c + d);
}

// bf16 <-> fp32.  bf16 is the top half of binary32; rounding is to
// nearest, ties to even, and NaN stays NaN.
__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

}  // namespace dev
}  // namespace bkv
