// (a1) Beacon maintenance for gfx950.
//
// Beacons stand for clusters of pre-RoPE queries under cosine similarity
// (Section 3.2 "Beacon queries"; Section 4.2; the nearest-representative
// similarity of Appendix D.1, Algorithm 1).  Online rule: each new query
// fills the lowest empty slot if there is one; otherwise it joins the slot
// of largest cosine similarity (ties -> lowest slot, cosine 0 when a norm is
// 0) and that slot moves to the running mean of its members.
//
// Heads of up to 16 slots take one wave (a 64-thread workgroup) each: the
// queries of a head are taken strictly in order, each seeing the previous
// update, so a head's work is one sequential chain, and small workgroups let
// many heads' chains run side by side on a compute unit (a layer-stacked
// call has thousands of heads).  Lanes 4c .. 4c+3 each take a quarter of
// slot c's dot product and a quad sum completes it.  Heads of more slots
// take four waves: all four bring the beacons in and compute their norms in
// one pass, the first takes the queries with one lane per slot, and the
// others wait for it at the barrier before the write-back.  The head's
// beacons live in LDS (rows padded to D + 4 floats) together with their
// squared norms, which are kept up to date as slots change; every 16-byte
// beacon load of a chunk is issued before the first wait.  Per query an
// argmax over the lanes (DPP, no LDS round trip) picks the slot and the
// lanes update that slot's D coordinates and its norm in parallel.  Finally
// the changed slots are written back (at most T*G of the C rows; the others
// still hold what was read).  The LDS is sized by C.
#include <math.h>

#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

// Query elements are loaded raw and widened only where they are used, so
// that a prefetch is not waited on right after it is issued.
__device__ __forceinline__ float widen(uint16_t v) { return dev::bf16_to_f32(v); }
__device__ __forceinline__ float widen(float v) { return v; }

// Dot product of two LEN-float rows in LDS (16-byte aligned), with four
// independent partial sums so that the FMAs do not wait on each other.
template <int LEN>
__device__ __forceinline__ float row_dot(const float* a, const float* b) {
    const float4* ar = reinterpret_cast<const float4*>(a);
    const float4* br = reinterpret_cast<const float4*>(b);
    float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll 8
    for (int d4 = 0; d4 < LEN / 4; ++d4) {
        const float4 u = ar[d4], v = br[d4];
        p0 = fmaf(u.x, v.x, p0);
        p1 = fmaf(u.y, v.y, p1);
        p2 = fmaf(u.z, v.z, p2);
        p3 = fmaf(u.w, v.w, p3);
    }
    return (p0 + p1) + (p2 + p3);
}

// Orders the wave's LDS accesses for the compiler: one lane's write before
// the fence is seen by another lane's read after it.  A wave's LDS
// instructions execute in order, so a wavefront-scope fence needs no wait
// instruction; in particular it does not wait for the next query's global
// loads in flight (a workgroup-scope fence or barrier would).
__device__ __forceinline__ void wave_lds_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

constexpr int kMaxSlots = 64;   // the boundary rejects C > 64: one bit per slot in a 64-bit mask
constexpr int kLoadChunk = 8;   // 16-byte beacon loads in flight per thread
constexpr int kQuadSlots = 16;  // C up to this: one wave per head, four lanes per slot's dot product
static_assert(kMaxSlots <= 64, "one lane of the query wave per slot holds its count and its dirty bit");

// LDS bytes of one head: C padded beacon rows, the current query, C norms,
// C counts, the mask of changed slots.
template <int D>
constexpr size_t smem_bytes(int C) {
    return ((size_t)C * (D + 4) + D + C) * sizeof(float) + (size_t)C * sizeof(int) + sizeof(unsigned long long);
}

// NW waves per workgroup: 1 for C <= kQuadSlots (the query wave alone, four
// lanes per slot's dot product), 4 for more slots (all four waves load the
// beacons and compute their norms in one pass, the first wave takes the
// queries with one lane per slot, the others wait at the barrier before the
// write-back).
template <typename T, int D, int NW>
__global__ __launch_bounds__(64 * NW) void beacon_update_kernel(const T* __restrict__ q_new, int T_steps,
                                                                float* beacons, int32_t* counts, int32_t* assign,
                                                                int Hq, int Hkv, int C) {
    constexpr int NT = 64 * NW;    // threads
    constexpr int LD = D + 4;      // padded row
    constexpr int PER = D / 64;    // coordinates per lane in lane-parallel loops
    constexpr int QD = D / 4;      // coordinates per lane of a slot's dot product (four lanes per slot)
    extern __shared__ __attribute__((aligned(16))) float smem[];
    float* bl = smem;                            // [C][LD]
    float* xs = bl + C * LD;                     // [D], 16-byte aligned: C * LD and D are multiples of 4
    float* bn2 = xs + D;                         // [C] squared norm of each slot
    int* cnt = reinterpret_cast<int*>(bn2 + C);  // [C]
    unsigned long long* dirty_out = reinterpret_cast<unsigned long long*>(cnt + C);  // 8-byte aligned
    auto sync = [] {
        if constexpr (NW > 1)
            __syncthreads();
        else
            wave_lds_fence();
    };
    const int tid = threadIdx.x, lane = tid & 63;
    const int h = blockIdx.x, b = h / Hkv, kh = h % Hkv;
    const int G = Hq / Hkv;
    float* bh = beacons + (size_t)h * C * D;
    const int nq = T_steps * G;
    auto query_ptr = [&](int qq) {
        const int t = qq / G, g = qq - t * G;
        return q_new + (((size_t)b * Hq + (size_t)kh * G + g) * T_steps + t) * D;
    };
    // The first query, the counts and a chunk of beacon vectors are loaded
    // unconditionally (threads past the end re-read the last element) and
    // pinned by an empty asm before the first store uses them, so the
    // compiler neither sinks a load into the guarded store nor waits
    // between loads: a chunk's loads all issue before the first wait (the
    // beacons of 16 slots, or of 64 with four waves, are one chunk).
    T xnext[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) xnext[k] = query_ptr(0)[lane + 64 * k];
    int cv = counts[(size_t)h * C + min(tid, C - 1)];
    asm volatile("" : "+v"(cv));
    const int n4 = C * D / 4;
    for (int base = 0; base < n4; base += NT * kLoadChunk) {
        dev::u32x4 v[kLoadChunk];
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k)
            v[k] = reinterpret_cast<const dev::u32x4*>(bh)[min(base + tid + NT * k, n4 - 1)];
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k) asm volatile("" : "+v"(v[k]));
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k) {
            const int i = base + tid + NT * k;
            if (i < n4) *reinterpret_cast<dev::u32x4*>(&bl[(4 * i) / D * LD + (4 * i) % D]) = v[k];
        }
    }
    if (tid < C) cnt[tid] = cv;
    sync();
    // squared norms: four threads per slot
    for (int c0 = 0; c0 < C; c0 += NT / 4) {
        const int c = c0 + (tid >> 2), part = tid & 3;
        float p = 0.f;
        if (c < C) {
            const float4* r = reinterpret_cast<const float4*>(&bl[c * LD + part * QD]);
#pragma unroll
            for (int d4 = 0; d4 < QD / 4; ++d4) {
                const float4 u = r[d4];
                p = fmaf(u.x, u.x, p);
                p = fmaf(u.y, u.y, p);
                p = fmaf(u.z, u.z, p);
                p = fmaf(u.w, u.w, p);
            }
        }
        p = dev::quad_sum(p);
        if (c < C && part == 0) bn2[c] = p;
    }
    sync();

    if (tid < 64) {
        unsigned long long dirty = 0;  // slots changed (wave-uniform)
        for (int q = 0; q < nq; ++q) {
            float xn = 0.f;
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                const float x = widen(xnext[k]);
                xs[lane + 64 * k] = x;
                xn = fmaf(x, x, xn);
            }
            // the next query (the last one again at the end: no branch to
            // join, so nothing waits for it before its use)
#pragma unroll
            for (int k = 0; k < PER; ++k) xnext[k] = query_ptr(min(q + 1, nq - 1))[lane + 64 * k];
            xn = dev::wave_sum(xn);
            wave_lds_fence();
            // lowest empty slot, if any
            const unsigned long long empty = __ballot(lane < C && cnt[lane] == 0);
            int chosen;
            if (empty) {
                chosen = __ffsll(empty) - 1;
#pragma unroll
                for (int k = 0; k < PER; ++k) bl[chosen * LD + lane + 64 * k] = xs[lane + 64 * k];
                if (lane == 0) {
                    cnt[chosen] = 1;
                    bn2[chosen] = xn;
                }
            } else {
                // argmax over the slots, ties -> lowest slot: the smallest
                // inverted order key of the cosine over the wave, then the
                // lowest lane that holds it.  The cosine takes hardware
                // reciprocal square roots (about 1 ulp each), so the choice can
                // differ from exact arithmetic only where the two best cosines
                // lie within a few 1e-7 of each other.
                const float rx = __builtin_amdgcn_rsqf(xn);
                auto cosine = [&](float dot, float bn) {
                    return (xn == 0.f || bn == 0.f) ? 0.f : dot * rx * __builtin_amdgcn_rsqf(bn);
                };
                unsigned key = ~0u;
                bool holds;  // this lane speaks for a slot
                int shift;   // lane -> slot
                if constexpr (NW == 1) {
                    // C <= 16: lanes 4c .. 4c+3 each take a quarter of slot c
                    const int c = lane >> 2, part = lane & 3;
                    const float dot = dev::quad_sum(c < C ? row_dot<QD>(&bl[c * LD + part * QD], &xs[part * QD]) : 0.f);
                    holds = c < C && part == 0;
                    if (holds) key = ~dev::ord_key(cosine(dot, bn2[c]));
                    shift = 2;
                } else {
                    // lane c takes slot c
                    const float dot = (lane < C) ? row_dot<D>(&bl[lane * LD], xs) : 0.f;
                    holds = lane < C;
                    if (holds) key = ~dev::ord_key(cosine(dot, bn2[lane]));
                    shift = 0;
                }
                const unsigned kmin = dev::wave_min_u32(key);
                chosen = (__ffsll(__ballot(holds && key == kmin)) - 1) >> shift;
                const int n = cnt[chosen] + 1;
                const float inv = 1.0f / (float)n;
                float p = 0.f;
#pragma unroll
                for (int k = 0; k < PER; ++k) {
                    const int d = lane + 64 * k;
                    const float bv = bl[chosen * LD + d];
                    const float nv = bv + (xs[d] - bv) * inv;
                    bl[chosen * LD + d] = nv;
                    p = fmaf(nv, nv, p);
                }
                p = dev::wave_sum(p);
                if (lane == 0) {
                    cnt[chosen] = n;
                    bn2[chosen] = p;
                }
            }
            dirty |= 1ull << chosen;
            if (assign && lane == 0) assign[(size_t)h * T_steps * G + q] = chosen;
            wave_lds_fence();
        }
        if (lane == 0) *dirty_out = dirty;
    }
    sync();
    // write back the changed slots only: the others still hold what was read
    const unsigned long long dirty = *dirty_out;
    for (int i = tid; i < n4; i += NT) {
        const int c = (4 * i) / D, d = (4 * i) % D;
        if ((dirty >> c) & 1ull) reinterpret_cast<float4*>(bh)[i] = *reinterpret_cast<const float4*>(&bl[c * LD + d]);
    }
    if (tid < C && ((dirty >> tid) & 1ull)) counts[(size_t)h * C + tid] = cnt[tid];
}

}  // namespace

hipError_t launch_beacon_update(const bkv_dims& d, const void* q_new, int T, float* beacons, int32_t* counts,
                                int32_t* assign, hipStream_t s) {
    const int P = d.B * d.Hkv;
    if (P == 0 || T == 0) return hipSuccess;
    const bool bf = d.dtype == BKV_BF16;
#define BKV_LAUNCH_BU(TY, DD)                                                                                   \
    if (d.C <= kQuadSlots)                                                                                  \
        hipLaunchKernelGGL((beacon_update_kernel<TY, DD, 1>), dim3(P), dim3(64), smem_bytes<DD>(d.C), s,            \
                           static_cast<const TY*>(q_new), T, beacons, counts, assign, d.Hq, d.Hkv, d.C);           \
    else                                                                                                    \
        hipLaunchKernelGGL((beacon_update_kernel<TY, DD, 4>), dim3(P), dim3(256), smem_bytes<DD>(d.C), s,           \
                           static_cast<const TY*>(q_new), T, beacons, counts, assign, d.Hq, d.Hkv, d.C)
    if (bf && d.D == 128) {
        BKV_LAUNCH_BU(uint16_t, 128);
    } else if (bf) {
        BKV_LAUNCH_BU(uint16_t, 64);
    } else if (d.D == 128) {
        BKV_LAUNCH_BU(float, 128);
    } else {
        BKV_LAUNCH_BU(float, 64);
    }
#undef BKV_LAUNCH_BU
    return hipGetLastError();
}

}  // namespace bkv
