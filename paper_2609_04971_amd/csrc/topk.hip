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
//
// Up to 32768 tokens the head's keys are read from HBM once, coalesced, and
// held in registers (32 per thread, token tid + 1024 i) through the radix
// passes.  Digit counts use four histogram copies per wave, and the wave's
// most common digit is added once by one lane, since same-address LDS
// atomics serialise.  The emit pass ranks kept tokens with ballots: a
// wave's 64 consecutive tokens are ranked by mbcnt, and one block scan over
// the per-wave counts in token order gives each run its base.  Longer heads
// stream the scores from memory on every pass and emit from contiguous
// per-thread runs.
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

constexpr int kRegKeys = 32768;  // longest head whose keys stay in registers

// Order keys of one head, read from global memory on every access.
struct GlobalKeys {
    const float* s;
    __device__ void init(const float* row, int) { s = row; }
    __device__ uint32_t operator[](int j) const { return order_key(s[j]); }
};

template <class Keys>
__device__ void topk_head(const float* __restrict__ scores, int32_t* __restrict__ kept, int N, int budget, int W,
                          int n_prefix, int n_keep, Keys& keys) {
    __shared__ int hist[kWaves][256];
    __shared__ int tot[256];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ int s_digit, s_above;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int h = blockIdx.x;
    int32_t* out = kept + (size_t)h * n_keep;

    if (N <= budget) {
        for (int i = tid; i < N; i += kThreads) out[i] = i;
        return;
    }
    keys.init(scores + (size_t)h * N, N);
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
                const uint32_t u = keys[j];
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
            const uint32_t u = keys[j];
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
            const uint32_t u = keys[j];
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

__global__ __launch_bounds__(kThreads) void topk_kernel(const float* __restrict__ scores, int32_t* __restrict__ kept,
                                                         int N, int budget, int W, int n_prefix, int n_keep) {
    GlobalKeys keys;
    topk_head(scores, kept, N, budget, W, n_prefix, n_keep, keys);
}

// Suffix scan over the 256 digit counts tot[] by wave 0: the digit d at
// which the running count from the top reaches `remaining`, and how many
// matching keys lie strictly above it.
__device__ __forceinline__ void find_digit(const int* tot, int remaining, int* s_digit, int* s_above) {
    const int lane = threadIdx.x & 63;
    const int d0 = 4 * lane;
    const int c0 = tot[d0], c1 = tot[d0 + 1], c2 = tot[d0 + 2], c3 = tot[d0 + 3];
    const int mine = c0 + c1 + c2 + c3;
    int x = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int y = __shfl_down(x, o, 64);
        if (lane + o < 64) x += y;
    }
    const int above_lane = x - mine;  // digits >= 4(lane+1)
    const int S3 = above_lane + c3, S2 = S3 + c2, S1 = S2 + c1, S0 = S1 + c0;
    const int r = remaining;
    if (S3 >= r && above_lane < r) { *s_digit = d0 + 3; *s_above = above_lane; }
    if (S2 >= r && S3 < r) { *s_digit = d0 + 2; *s_above = S3; }
    if (S1 >= r && S2 < r) { *s_digit = d0 + 1; *s_above = S2; }
    if (S0 >= r && S1 < r) { *s_digit = d0; *s_above = S1; }
}

constexpr int kPer = kRegKeys / kThreads;  // keys per thread
constexpr int kSub = 4;                      // histogram copies per wave
constexpr int kRows = kPer * kWaves;         // (row i, wave) runs of 64 tokens

// Add one to digit d of this lane's histogram copy.  The most common digit
// among the wave's active lanes is counted with one atomic by its first lane
// (digits are often concentrated, and same-address LDS atomics serialise);
// the other lanes add their own.
__device__ __forceinline__ void count_digit(int* hw, uint32_t d, bool active) {
    const uint64_t act = __builtin_amdgcn_ballot_w64(active);
    if (act == 0) return;
    const int leader = __builtin_ctzll(act);
    const uint32_t dl = __builtin_amdgcn_readlane(d, leader);
    const uint64_t same = __builtin_amdgcn_ballot_w64(active && d == dl);
    const int lane = threadIdx.x & 63;
    if (lane == leader) atomicAdd(&hw[dl], (int)__builtin_popcountll(same));
    else if (active && d != dl) atomicAdd(&hw[d], 1);
}

// Lanes below this one whose bit is set in mask.
__device__ __forceinline__ int rank_in_wave(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

// Exclusive scan, in place, of the kRows per-run counts c[i][wave] in
// token order (run (i, w) covers tokens i*1024 + 64 w ... + 63).
__device__ __forceinline__ void scan_runs(int* c, int* buf) {
    const int t = threadIdx.x;
    const int v = (t < kRows) ? c[t] : 0;
    int total;
    const int before = block_excl_scan(v, buf, &total);
    if (t < kRows) c[t] = before;
    __syncthreads();
}

__global__ __launch_bounds__(kThreads) void topk_reg_kernel(const float* __restrict__ scores,
                                                             int32_t* __restrict__ kept, int N, int budget, int W,
                                                             int n_prefix, int n_keep) {
    __shared__ int hist[kWaves][kSub][256];
    __shared__ int part[kThreads / 256][256];
    __shared__ int tot[256];
    __shared__ int runs[kRows];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ uint32_t red_min[kWaves], red_max[kWaves];
    __shared__ int s_digit, s_above;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int sub = lane >> 4;
    uint32_t key_lo = 0;
    int vbits = 0;
    const int h = blockIdx.x;
    const float* srow = scores + (size_t)h * N;
    int32_t* out = kept + (size_t)h * n_keep;
    if (N <= budget) {
        for (int i = tid; i < N; i += kThreads) out[i] = i;
        return;
    }
    const int lo = n_prefix, hi = N - W;  // candidates [lo, hi)
    const int ksel = budget - n_prefix - W;
    // key i of this thread is token tid + i * kThreads (coalesced loads, all
    // in flight at once; tokens past N read token N - 1 and are no candidates)
    uint32_t u[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) u[i] = order_key(srow[min(tid + i * kThreads, N - 1)]);
    uint32_t cand = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int j = tid + i * kThreads;
        if (j >= lo && j < hi) cand |= 1u << i;
    }
    // Radix select on v = key - (smallest candidate key) over only the bits
    // that vary: the first digit then spreads over the occupied range
    // instead of a few exponent values.
    {
        uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
        for (int i = 0; i < kPer; ++i)
            if ((cand >> i) & 1u) {
                kmin = min(kmin, u[i]);
                kmax = max(kmax, u[i]);
            }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, o, 64));
            kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, o, 64));
        }
        if (lane == 0) {
            red_min[wave] = kmin;
            red_max[wave] = kmax;
        }
        __syncthreads();
        kmin = red_min[0];
        kmax = red_max[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) {
            kmin = min(kmin, red_min[w]);
            kmax = max(kmax, red_max[w]);
        }
        key_lo = kmin;
        vbits = (kmax > kmin) ? 32 - __builtin_clz(kmax - kmin) : 0;
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) u[i] -= key_lo;  // candidates only are compared from here on
    uint32_t prefix = 0, pmask = 0;
    int remaining = ksel;
    if (ksel > 0) {
        const int npass = (vbits + 7) / 8;
        for (int pass = 0; pass < npass; ++pass) {
            const int shift = max(0, vbits - 8 * (pass + 1));
            int* hz = &hist[0][0][0];
            for (int i = tid; i < kWaves * kSub * 256; i += kThreads) hz[i] = 0;
            __syncthreads();
            int* hw = &hist[wave][sub][0];
#pragma unroll
            for (int i = 0; i < kPer; ++i)
                count_digit(hw, (u[i] >> shift) & 255u, ((cand >> i) & 1u) && (u[i] & pmask) == prefix);
            __syncthreads();
            {   // digit d's count: thread (d, q) sums the copies of waves 4q..4q+3
                const int d = tid & 255, q = tid >> 8;
                int c = 0;
#pragma unroll
                for (int w = 4 * q; w < 4 * q + 4; ++w)
#pragma unroll
                    for (int b = 0; b < kSub; ++b) c += hist[w][b][d];
                part[q][d] = c;
            }
            __syncthreads();
            if (tid < 256) tot[tid] = part[0][tid] + part[1][tid] + part[2][tid] + part[3][tid];
            __syncthreads();
            if (wave == 0) find_digit(tot, remaining, &s_digit, &s_above);
            __syncthreads();
            prefix |= (uint32_t)s_digit << shift;
            pmask |= 255u << shift;
            remaining -= s_above;
            __syncthreads();
        }
    }
    const uint32_t theta = prefix;
    const int need_eq = (ksel > 0) ? remaining : 0;  // ties at theta to take, lowest index first
    // Ties: rank of each tied candidate among the tied ones, in token order.
    uint64_t eqb[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        eqb[i] = __builtin_amdgcn_ballot_w64(ksel > 0 && ((cand >> i) & 1u) && u[i] == theta);
        if (lane == 0) runs[i * kWaves + wave] = (int)__builtin_popcountll(eqb[i]);
    }
    __syncthreads();
    scan_runs(runs, scan_buf);
    uint32_t keep = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const bool c = (cand >> i) & 1u;
        const int j = tid + i * kThreads;
        bool k;
        if (j >= N)
            k = false;
        else if (!c)
            k = true;  // forced prefix / recent window
        else if (ksel <= 0)
            k = false;
        else if (u[i] > theta)
            k = true;
        else
            k = u[i] == theta && runs[i * kWaves + wave] + rank_in_wave(eqb[i]) < need_eq;
        if (k) keep |= 1u << i;
    }
    __syncthreads();  // tie ranks read before the counts are reused
    uint64_t kb[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        kb[i] = __builtin_amdgcn_ballot_w64((keep >> i) & 1u);
        if (lane == 0) runs[i * kWaves + wave] = (int)__builtin_popcountll(kb[i]);
    }
    __syncthreads();
    scan_runs(runs, scan_buf);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        if ((keep >> i) & 1u) {
            const int pos = runs[i * kWaves + wave] + rank_in_wave(kb[i]);
            if (pos < n_keep) out[pos] = tid + i * kThreads;
        }
    }
}

}  // namespace

hipError_t launch_topk(const bkv_dims& d, const float* scores, int32_t* kept, hipStream_t s) {
    const int P = d.B * d.Hkv;
    const int n_keep = d.N < d.budget ? d.N : d.budget;
    if (d.N <= kRegKeys)
        hipLaunchKernelGGL(topk_reg_kernel, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W,
                           d.n_prefix, n_keep);
    else
        hipLaunchKernelGGL(topk_kernel, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W,
                           d.n_prefix, n_keep);
    return hipGetLastError();
}

}  // namespace bkv
