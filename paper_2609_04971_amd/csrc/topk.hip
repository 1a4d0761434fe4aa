// (a4) Per-head selection for gfx950.
//
// The first n_prefix and the last W tokens are always kept; the remaining
// k_sel = budget - n_prefix - W places go to the other tokens of highest
// score, ties to the lower index, and the kept indices come out ascending
// (Section 2.2 TopK; Algorithm 2, I_keep / k_sel / TopK / Sort).  If
// N <= budget every token is kept.
//
// One 1024-thread workgroup per head.  Scores map to a monotone uint32 key
// (-0 first canonicalised to +0), and an exact radix select with 8-bit
// digits (4 passes, LDS histograms per wave) finds the k_sel-th largest
// candidate key theta and how many candidates equal to theta are taken.
// The emit pass needs no sort: each thread owns a contiguous run of indices,
// and two block-wide exclusive scans (ties taken so far, kept so far) give
// every kept index its output position in ascending order.
#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ uint32_t order_key(float s) {
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0u;  // -0 ranks with +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Block-wide exclusive scan of one int per thread; returns the prefix and
// sets *total.  `buf` holds kWaves + 1 ints.
__device__ __forceinline__ int block_excl_scan(int v, int* buf, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) buf[wave] = x;
    __syncthreads();
    if (wave == 0) {
        int w = (lane < kWaves) ? buf[lane] : 0;
#pragma unroll
        for (int o = 1; o < kWaves; o <<= 1) {
            int y = __shfl_up(w, o, 64);
            if (lane >= o) w += y;
        }
        if (lane < kWaves) buf[lane] = w;  // inclusive totals per wave
    }
    __syncthreads();
    const int before = (wave > 0 ? buf[wave - 1] : 0) + x - v;
    *total = buf[kWaves - 1];
    __syncthreads();
    return before;
}

__global__ __launch_bounds__(kThreads) void topk_kernel(const float* __restrict__ scores, int32_t* __restrict__ kept,
                                                         int N, int budget, int W, int n_prefix, int n_keep) {
    __shared__ int hist[kWaves][256];
    __shared__ int tot[256];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ int s_digit, s_above;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = blockIdx.x;
    const float* s = scores + (size_t)h * N;
    int32_t* out = kept + (size_t)h * n_keep;

    if (N <= budget) {
        for (int i = tid; i < N; i += kThreads) out[i] = i;
        return;
    }
    const int lo = n_prefix, hi = N - W;  // candidates [lo, hi)
    const int ksel = budget - n_prefix - W;

    uint32_t prefix = 0, pmask = 0;
    int remaining = ksel;  // how many still to take at or below the current prefix
    if (ksel > 0) {
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            for (int i = tid; i < kWaves * 256; i += kThreads) (&hist[0][0])[i] = 0;
            __syncthreads();
            for (int j = lo + tid; j < hi; j += kThreads) {
                const uint32_t u = order_key(s[j]);
                if ((u & pmask) == prefix) atomicAdd(&hist[wave][(u >> shift) & 255u], 1);
            }
            __syncthreads();
            if (tid < 256) {
                int c = 0;
#pragma unroll
                for (int w = 0; w < kWaves; ++w) c += hist[w][tid];
                tot[tid] = c;
            }
            __syncthreads();
            // suffix sums over digits 255..0 by wave 0: lane l owns digits 4l..4l+3
            if (wave == 0) {
                const int d0 = 4 * lane;
                const int c0 = tot[d0], c1 = tot[d0 + 1], c2 = tot[d0 + 2], c3 = tot[d0 + 3];
                const int mine = c0 + c1 + c2 + c3;
                // sum over lanes > lane (inclusive-from-the-top scan)
                int x = mine;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    int y = __shfl_down(x, o, 64);
                    if (lane + o < 64) x += y;
                }
                const int above_lane = x - mine;  // digits >= 4(lane+1)
                // S(d) = number of matching candidates with digit >= d
                const int S3 = above_lane + c3, S2 = S3 + c2, S1 = S2 + c1, S0 = S1 + c0;
                const int r = remaining;
                if (S3 >= r && above_lane < r) { s_digit = d0 + 3; s_above = above_lane; }
                if (S2 >= r && S3 < r) { s_digit = d0 + 2; s_above = S3; }
                if (S1 >= r && S2 < r) { s_digit = d0 + 1; s_above = S2; }
                if (S0 >= r && S1 < r) { s_digit = d0; s_above = S1; }
            }
            __syncthreads();
            prefix |= (uint32_t)s_digit << shift;
            pmask |= 255u << shift;
            remaining -= s_above;
            __syncthreads();
        }
    }
    const uint32_t theta = prefix;
    const int need_eq = (ksel > 0) ? remaining : 0;  // ties at theta to take, lowest index first

    // Emit: thread t owns indices [t*per, min((t+1)*per, N)).
    const int per = (N + kThreads - 1) / kThreads;
    const int j0 = min(tid * per, N), j1 = min(j0 + per, N);
    int n_sure = 0, n_eq = 0;
    for (int j = j0; j < j1; ++j) {
        if (j < lo || j >= hi) {
            ++n_sure;
        } else if (ksel > 0) {
            const uint32_t u = order_key(s[j]);
            n_sure += (u > theta);
            n_eq += (u == theta);
        }
    }
    int total;
    const int eq_before = block_excl_scan(n_eq, scan_buf, &total);
    const int eq_take = max(0, min(n_eq, need_eq - eq_before));
    int pos = block_excl_scan(n_sure + eq_take, scan_buf, &total);
    int eq_seen = eq_before;
    for (int j = j0; j < j1; ++j) {
        bool keep;
        if (j < lo || j >= hi) {
            keep = true;
        } else if (ksel > 0) {
            const uint32_t u = order_key(s[j]);
            if (u > theta) {
                keep = true;
            } else if (u == theta) {
                keep = eq_seen < need_eq;
                ++eq_seen;
            } else {
                keep = false;
            }
        } else {
            keep = false;
        }
        if (keep && pos < n_keep) out[pos++] = j;
    }
    (void)lane;
}

}  // namespace

hipError_t launch_topk(const bkv_dims& d, const float* scores, int32_t* kept, hipStream_t s) {
    const int P = d.B * d.Hkv;
    const int n_keep = d.N < d.budget ? d.N : d.budget;
    hipLaunchKernelGGL(topk_kernel, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W, d.n_prefix,
                       n_keep);
    return hipGetLastError();
}

}  // namespace bkv
