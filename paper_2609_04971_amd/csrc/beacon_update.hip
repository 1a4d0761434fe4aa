// (a1) Beacon maintenance for gfx950.
//
// Beacons stand for clusters of pre-RoPE queries under cosine similarity
// (Section 3.2 "Beacon queries"; Section 4.2; the nearest-representative
// similarity of Appendix D.1, Algorithm 1).  Online rule: each new query
// fills the lowest empty slot if there is one; otherwise it joins the slot
// of largest cosine similarity (ties -> lowest slot, cosine 0 when a norm is
// 0) and that slot moves to the running mean of its members.
//
// One wave per (batch, kv-head); the T*G queries of the head's group are
// processed strictly in order (t-major, then g), each seeing the previous
// update.  The head's beacons live in LDS (rows padded to D + 4 floats so
// that sixteen lanes reading 16-byte vectors of sixteen different slots hit
// distinct banks) together with their squared norms, which are kept up to
// date as slots change.  Per query, lane c accumulates slot c's dot product
// over D with 16-byte LDS reads; all lanes share the query's squared norm;
// an argmax over lanes picks the slot, and the lanes update that slot's D
// coordinates and its norm in parallel.  The step is latency-bound.
#include <math.h>

#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr int kMaxC = 64;

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, size_t i);
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, size_t i) { return dev::bf16_to_f32(p[i]); }
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, size_t i) { return p[i]; }

// Dot product of two D-float rows in LDS (16-byte aligned), with four
// independent partial sums so that the FMAs do not wait on each other.
template <int D>
__device__ __forceinline__ float row_dot_impl(const float* a, const float* b) {
    const float4* ar = reinterpret_cast<const float4*>(a);
    const float4* br = reinterpret_cast<const float4*>(b);
    float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll 8
    for (int d4 = 0; d4 < D / 4; ++d4) {
        const float4 u = ar[d4], v = br[d4];
        p0 = fmaf(u.x, v.x, p0);
        p1 = fmaf(u.y, v.y, p1);
        p2 = fmaf(u.z, v.z, p2);
        p3 = fmaf(u.w, v.w, p3);
    }
    return (p0 + p1) + (p2 + p3);
}

// Sum over the wave (all 64 lanes hold the result).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += dev::shfl_xor_f(v, o);
    return v;
}

template <typename T, int D>
__global__ __launch_bounds__(64) void beacon_update_kernel(const T* __restrict__ q_new, int T_steps, float* beacons,
                                                           int32_t* counts, int32_t* assign, int Hq, int Hkv, int C) {
    constexpr int LD = D + 4;        // padded row: 16-byte reads of 16 slots hit distinct banks
    constexpr int PER = D / 64;      // coordinates per lane in lane-parallel loops
    __shared__ __attribute__((aligned(16))) float bl[kMaxC * LD];
    __shared__ __attribute__((aligned(16))) float xs[D];
    __shared__ float bn2[kMaxC];     // squared norm of each slot
    __shared__ int cnt[kMaxC];
    auto row_dot = [](const float* a, const float* b) { return row_dot_impl<D>(a, b); };
    const int lane = threadIdx.x;
    const int h = blockIdx.x, b = h / Hkv, kh = h % Hkv;
    const int G = Hq / Hkv;
    float* bh = beacons + (size_t)h * C * D;
    // query q = t * G + g; its coordinates are loaded one query ahead (the
    // first one before the beacons)
    const int nq = T_steps * G;
    auto query_ptr = [&](int qq) {
        const int t = qq / G, g = qq - t * G;
        return q_new + (((size_t)b * Hq + (size_t)kh * G + g) * T_steps + t) * D;
    };
    float xnext[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) xnext[k] = load_elem<T>(query_ptr(0), lane + 64 * k);
    // beacons in with 16-byte loads (D is a multiple of 4 and rows are 16-byte aligned)
    for (int i = lane; i < C * D / 4; i += 64) {
        const float4 v = reinterpret_cast<const float4*>(bh)[i];
        const int c = (4 * i) / D, d = (4 * i) % D;
        *reinterpret_cast<float4*>(&bl[c * LD + d]) = v;
    }
    if (lane < C) cnt[lane] = counts[(size_t)h * C + lane];
    __syncthreads();
    if (lane < C) bn2[lane] = row_dot(&bl[lane * LD], &bl[lane * LD]);  // squared norms
    __syncthreads();

    for (int q = 0; q < nq; ++q) {
        {
            float xn = 0.f;
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                const float v = xnext[k];
                xs[lane + 64 * k] = v;
                xn = fmaf(v, v, xn);
            }
            if (q + 1 < nq) {
#pragma unroll
                for (int k = 0; k < PER; ++k) xnext[k] = load_elem<T>(query_ptr(q + 1), lane + 64 * k);
            }
            xn = wave_sum(xn);
            __syncthreads();
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
                const float dot = (lane < C) ? row_dot(&bl[lane * LD], xs) : 0.f;
                const float bn = (lane < C) ? bn2[lane] : 0.f;
                float cs = (xn == 0.f || bn == 0.f) ? 0.f : dot / (sqrtf(xn) * sqrtf(bn));
                if (lane >= C) cs = -INFINITY;
                int idx = lane;
                // argmax over lanes, ties -> lowest slot
#pragma unroll
                for (int o = 32; o > 0; o >>= 1) {
                    const float oc = dev::shfl_xor_f(cs, o);
                    const int oi = dev::shfl_xor_i(idx, o);
                    if (oc > cs || (oc == cs && oi < idx)) {
                        cs = oc;
                        idx = oi;
                    }
                }
                chosen = idx;
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
                p = wave_sum(p);
                if (lane == 0) {
                    cnt[chosen] = n;
                    bn2[chosen] = p;
                }
            }
            if (assign && lane == 0) assign[(size_t)h * T_steps * G + q] = chosen;
            __syncthreads();
        }
    }
    for (int i = lane; i < C * D / 4; i += 64) {
        const int c = (4 * i) / D, d = (4 * i) % D;
        reinterpret_cast<float4*>(bh)[i] = *reinterpret_cast<const float4*>(&bl[c * LD + d]);
    }
    if (lane < C) counts[(size_t)h * C + lane] = cnt[lane];
}

}  // namespace

hipError_t launch_beacon_update(const bkv_dims& d, const void* q_new, int T, float* beacons, int32_t* counts,
                                int32_t* assign, hipStream_t s) {
    const int P = d.B * d.Hkv;
    if (P == 0 || T == 0) return hipSuccess;
    const bool bf = d.dtype == BKV_BF16;
#define BKV_LAUNCH_BU(TY, DD)                                                                                   \
    hipLaunchKernelGGL((beacon_update_kernel<TY, DD>), dim3(P), dim3(64), 0, s, static_cast<const TY*>(q_new), T, \
                       beacons, counts, assign, d.Hq, d.Hkv, d.C)
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
