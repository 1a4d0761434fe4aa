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
// update.  The head's beacons live in LDS; lane c computes slot c's dot
// product and squared norm over D, an argmax over lanes picks the slot, and
// the lanes then update that slot's D coordinates in parallel.  The step is
// latency-bound (a few thousand FMAs per query).
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

template <typename T, int D>
__global__ __launch_bounds__(64) void beacon_update_kernel(const T* __restrict__ q_new, int T_steps, float* beacons,
                                                           int32_t* counts, int32_t* assign, int Hq, int Hkv, int C) {
    __shared__ float bl[kMaxC][D + 1];
    __shared__ float xs[D];
    __shared__ int cnt[kMaxC];
    const int lane = threadIdx.x;
    const int h = blockIdx.x, b = h / Hkv, kh = h % Hkv;
    const int G = Hq / Hkv;
    float* bh = beacons + (size_t)h * C * D;
    for (int i = lane; i < C * D; i += 64) bl[i / D][i % D] = bh[i];
    if (lane < C) cnt[lane] = counts[(size_t)h * C + lane];
    __syncthreads();

    int q = 0;
    for (int t = 0; t < T_steps; ++t) {
        for (int g = 0; g < G; ++g, ++q) {
            const T* x = q_new + (((size_t)b * Hq + (size_t)kh * G + g) * T_steps + t) * D;
            for (int d = lane; d < D; d += 64) xs[d] = load_elem<T>(x, d);
            __syncthreads();
            // lowest empty slot, if any
            const unsigned long long empty = __ballot(lane < C && cnt[lane] == 0);
            int chosen;
            if (empty) {
                chosen = __ffsll(empty) - 1;
                for (int d = lane; d < D; d += 64) bl[chosen][d] = xs[d];
                if (lane == 0) cnt[chosen] = 1;
            } else {
                float dot = 0.f, bn = 0.f, xn = 0.f;
                if (lane < C) {
                    for (int d = 0; d < D; ++d) {
                        const float bv = bl[lane][d], xv = xs[d];
                        dot = fmaf(xv, bv, dot);
                        bn = fmaf(bv, bv, bn);
                        xn = fmaf(xv, xv, xn);
                    }
                }
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
                for (int d = lane; d < D; d += 64) {
                    const float bv = bl[chosen][d];
                    bl[chosen][d] = bv + (xs[d] - bv) * inv;
                }
                __syncthreads();
                if (lane == 0) cnt[chosen] = n;
            }
            if (assign && lane == 0) assign[(size_t)h * T_steps * G + q] = chosen;
            __syncthreads();
        }
    }
    for (int i = lane; i < C * D; i += 64) bh[i] = bl[i / D][i % D];
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
