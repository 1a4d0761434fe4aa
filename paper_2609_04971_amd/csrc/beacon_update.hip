// (a1) Beacon maintenance for gfx950.
//
// Beacons stand for clusters of pre-RoPE queries under cosine similarity
// (Section 3.2 "Beacon queries"; Section 4.2; the nearest-representative
// similarity of Appendix D.1, Algorithm 1).  Online rule: each new query
// fills the lowest empty slot if there is one; otherwise it joins the slot
// of largest cosine similarity (ties -> lowest slot, cosine 0 when a norm is
// 0) and that slot moves to the running mean of its members.
//
// One wave (a 64-thread workgroup) per (batch, kv-head): the queries of a
// head are taken strictly in order, each seeing the previous update, so a
// head's work is one sequential chain, and small workgroups let many heads'
// chains run side by side on a compute unit (a layer-stacked call has
// thousands of heads).  The head's beacons live in LDS (rows padded to
// D + 4 floats) together with their squared norms, which are kept up to
// date as slots change.  The wave brings the beacons in with up to eight
// 16-byte loads per lane in flight, then computes the norms, four lanes per
// slot.  Per query: lanes 4c .. 4c+3 each take a quarter of slot c's dot
// product (16-byte LDS reads) and a quad sum completes it; an argmax over
// the lanes (DPP, no LDS round trip) picks the slot; the lanes update that
// slot's D coordinates and its norm in parallel.  Finally the wave writes
// back the slots that changed (at most T*G of the C rows; the others still
// hold what was read).  The LDS is sized by C.
#include <math.h>

#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

// Query elements are loaded raw and widened only where they are used, so
// that a prefetch is not waited on right after it is issued.
__device__ __forceinline__ float widen(uint16_t v) { return dev::bf16_to_f32(v); }
__device__ __forceinline__ float widen(float v) { return v; }

// Orders the wave's LDS accesses for the compiler: one lane's write before
// the fence is seen by another lane's read after it.  A wave's LDS
// instructions execute in order, so a wavefront-scope fence needs no wait
// instruction; in particular it does not wait for the next query's global
// loads in flight (a workgroup-scope fence or barrier would).
__device__ __forceinline__ void wave_lds_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

constexpr int kThreads = 64;    // one wave per head
constexpr int kMaxSlots = 64;   // the boundary rejects C > 64: one bit per slot in a 64-bit mask
constexpr int kLoadChunk = 8;   // 16-byte beacon loads in flight per lane
static_assert(kMaxSlots <= kThreads, "one lane per slot holds its count and its dirty bit");

// LDS bytes of one head: C padded beacon rows, the current query, C norms,
// C counts.
template <int D>
constexpr size_t smem_bytes(int C) {
    return ((size_t)C * (D + 4) + D + C) * sizeof(float) + (size_t)C * sizeof(int);
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void beacon_update_kernel(const T* __restrict__ q_new, int T_steps,
                                                                 float* beacons, int32_t* counts, int32_t* assign,
                                                                 int Hq, int Hkv, int C) {
    constexpr int LD = D + 4;      // padded row
    constexpr int PER = D / 64;    // coordinates per lane in lane-parallel loops
    constexpr int QD = D / 4;      // coordinates per lane of a slot's dot product (four lanes per slot)
    extern __shared__ __attribute__((aligned(16))) float smem[];
    float* bl = smem;                            // [C][LD]
    float* xs = bl + C * LD;                     // [D], 16-byte aligned: C * LD and D are multiples of 4
    float* bn2 = xs + D;                         // [C] squared norm of each slot
    int* cnt = reinterpret_cast<int*>(bn2 + C);  // [C]
    const int lane = threadIdx.x;
    const int h = blockIdx.x, b = h / Hkv, kh = h % Hkv;
    const int G = Hq / Hkv;
    float* bh = beacons + (size_t)h * C * D;
    const int nq = T_steps * G;
    auto query_ptr = [&](int qq) {
        const int t = qq / G, g = qq - t * G;
        return q_new + (((size_t)b * Hq + (size_t)kh * G + g) * T_steps + t) * D;
    };
    // The first query, the counts and a chunk of beacon vectors are loaded
    // unconditionally (lanes past the end re-read the last element) and
    // pinned by an empty asm before the first store uses them, so the
    // compiler neither sinks a load into the guarded store nor waits
    // between loads: a chunk's loads all issue before the first wait.
    T xnext[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) xnext[k] = query_ptr(0)[lane + 64 * k];
    int cv = counts[(size_t)h * C + min(lane, C - 1)];
    asm volatile("" : "+v"(cv));
    const int n4 = C * D / 4;
    for (int base = 0; base < n4; base += kThreads * kLoadChunk) {
        dev::u32x4 v[kLoadChunk];
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k)
            v[k] = reinterpret_cast<const dev::u32x4*>(bh)[min(base + lane + kThreads * k, n4 - 1)];
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k) asm volatile("" : "+v"(v[k]));
#pragma unroll
        for (int k = 0; k < kLoadChunk; ++k) {
            const int i = base + lane + kThreads * k;
            if (i < n4) *reinterpret_cast<dev::u32x4*>(&bl[(4 * i) / D * LD + (4 * i) % D]) = v[k];
        }
    }
    if (lane < C) cnt[lane] = cv;
    wave_lds_fence();
    // squared norms: four lanes per slot, sixteen slots at a time
    for (int c0 = 0; c0 < C; c0 += kThreads / 4) {
        const int c = c0 + (lane >> 2), part = lane & 3;
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
    wave_lds_fence();

    unsigned long long dirty = 0;  // slots changed (wave-uniform)
    for (int q = 0; q < nq; ++q) {
        float xn = 0.f;
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const float x = widen(xnext[k]);
            xs[lane + 64 * k] = x;
            xn = fmaf(x, x, xn);
        }
        // the next query (the last one again at the end: no branch to join,
        // so nothing waits for it before its use)
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
            // argmax over the slots, ties -> lowest slot: the minimum of
            // (inverted order key of the cosine, slot)
            unsigned long long best = ~0ull;
            for (int c0 = 0; c0 < C; c0 += kThreads / 4) {
                const int c = c0 + (lane >> 2), part = lane & 3;
                float dot = 0.f;
                if (c < C) {
                    const float4* ar = reinterpret_cast<const float4*>(&bl[c * LD + part * QD]);
                    const float4* xr = reinterpret_cast<const float4*>(&xs[part * QD]);
                    float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll
                    for (int d4 = 0; d4 < QD / 4; ++d4) {
                        const float4 u = ar[d4], v = xr[d4];
                        p0 = fmaf(u.x, v.x, p0);
                        p1 = fmaf(u.y, v.y, p1);
                        p2 = fmaf(u.z, v.z, p2);
                        p3 = fmaf(u.w, v.w, p3);
                    }
                    dot = (p0 + p1) + (p2 + p3);
                }
                dot = dev::quad_sum(dot);
                const float bn = (c < C) ? bn2[c] : 0.f;
                const float cs = (xn == 0.f || bn == 0.f) ? 0.f : dot / (sqrtf(xn) * sqrtf(bn));
                const unsigned long long key =
                    (c < C && part == 0) ? ((unsigned long long)(~dev::ord_key(cs)) << 32) | (unsigned)c : ~0ull;
                best = key < best ? key : best;
            }
            chosen = (int)(unsigned)dev::wave_min_u64(best);
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
    // write back the changed slots only: the others still hold what was read
    for (int i = lane; i < n4; i += kThreads) {
        const int c = (4 * i) / D, d = (4 * i) % D;
        if ((dirty >> c) & 1ull) reinterpret_cast<float4*>(bh)[i] = *reinterpret_cast<const float4*>(&bl[c * LD + d]);
    }
    if (lane < C && ((dirty >> lane) & 1ull)) counts[(size_t)h * C + lane] = cnt[lane];
}

}  // namespace

hipError_t launch_beacon_update(const bkv_dims& d, const void* q_new, int T, float* beacons, int32_t* counts,
                                int32_t* assign, hipStream_t s) {
    const int P = d.B * d.Hkv;
    if (P == 0 || T == 0) return hipSuccess;
    const bool bf = d.dtype == BKV_BF16;
#define BKV_LAUNCH_BU(TY, DD)                                                                                   \
    hipLaunchKernelGGL((beacon_update_kernel<TY, DD>), dim3(P), dim3(kThreads), smem_bytes<DD>(d.C), s,                   \
                       static_cast<const TY*>(q_new), T, beacons, counts, assign, d.Hq, d.Hkv, d.C)
    if (bf && d.D == 128)
        BKV_LAUNCH_BU(uint16_t, 128);
    else if (bf)
        BKV_LAUNCH_BU(uint16_t, 64);
    else if (d.D == 128)
        BKV_LAUNCH_BU(float, 128);
    else
        BKV_LAUNCH_BU(float, 64);
#undef BKV_LAUNCH_BU
    return hipGetLastError();
}

}  // namespace bkv
