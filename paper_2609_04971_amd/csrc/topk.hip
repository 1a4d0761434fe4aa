// (a4) Per-head selection for gfx950.
//
// The first n_prefix and the last W tokens are always kept; the remaining
// k_sel = budget - n_prefix - W places go to the other tokens of highest
// score, ties to the lower index, and the kept indices come out ascending
// (Section 2.2 TopK; Algorithm 2, I_keep / k_sel / TopK / Sort).  If
// N <= budget every token is kept.
//
// One 1024-thread workgroup per head.  Scores map to a monotone uint32 key
// (-0 first canonicalised to +0); the selection finds the k_sel-th largest
// candidate key theta and how many candidates equal to theta are taken.
// The emit needs no sort: block-wide exclusive scans (ties taken so far,
// kept so far) give every kept index its output position in ascending
// order.
//
// Up to 32768 tokens the head's keys are read from HBM once, coalesced, and
// held in registers (32 per thread, token tid + 1024 i).  A first stage
// bins the candidates by value, linearly over [min, max] of their scores
// into 4096 bins (the map is monotone under rounding, so a higher bin beats
// a lower one).  Bits of the float key would follow its exponent and put a
// whole head in a handful of bins; value bins spread a head's keys over
// many, and the bin holding the threshold usually has a few dozen.  Up to
// 512 of them are ranked directly by (key descending, token ascending),
// which gives theta and the ties to take; more (many equal or nearly equal
// scores), or NaN / +inf candidates, go through an exact radix select with
// 8-bit digits over the bits that vary, whose counts use four histogram
// copies per wave and add the wave's most common digit once, by one lane,
// since same-address LDS atomics serialise.  Ties at theta are
// ranked in token order only when some of them must be left out.  The emit
// ranks kept tokens with ballots: a wave's 64 consecutive tokens are ranked
// by mbcnt, and one block scan over the per-wave counts in token order
// gives each run its base.  Longer heads stream the scores from memory on
// every pass (8-bit radix digits from the top) and emit from contiguous
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

// Block-wide suffix scan of the kBins first-stage counts (thread t owns the
// bins of its reversed index rt = kThreads - 1 - t, 4 rt .. 4 rt + 3, so the
// exclusive prefix in thread order counts every higher bin): the bin at
// which the running count from the top reaches `remaining`, and how many
// candidates lie strictly above it.
__device__ __forceinline__ void find_wide_digit(const int* cnt, int remaining, int* buf, int* s_digit,
                                                int* s_above) {
    const int rt = kThreads - 1 - (int)threadIdx.x;
    const int d0 = 4 * rt;
    const int c0 = cnt[d0], c1 = cnt[d0 + 1], c2 = cnt[d0 + 2], c3 = cnt[d0 + 3];
    int total;
    const int above = block_excl_scan(c0 + c1 + c2 + c3, buf, &total);  // bins >= 4 (rt + 1)
    const int S3 = above + c3, S2 = S3 + c2, S1 = S2 + c1, S0 = S1 + c0;
    const int r = remaining;
    if (S3 >= r && above < r) { *s_digit = d0 + 3; *s_above = above; }
    if (S2 >= r && S3 < r) { *s_digit = d0 + 2; *s_above = S3; }
    if (S1 >= r && S2 < r) { *s_digit = d0 + 1; *s_above = S2; }
    if (S0 >= r && S1 < r) { *s_digit = d0; *s_above = S1; }
}

// Float min / max over the block through order keys (DPP within waves, LDS
// across them); `slot` holds kWaves words.  Every thread gets the result.
__device__ __forceinline__ uint32_t block_min_u32(uint32_t v, uint32_t* slot) {
    v = dev::wave_min_u32(v);
    if ((threadIdx.x & 63) == 0) slot[threadIdx.x >> 6] = v;
    __syncthreads();
    uint32_t m = slot[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = min(m, slot[w]);
    __syncthreads();
    return m;
}
__device__ __forceinline__ float key_to_float(uint32_t k) {  // inverse of order_key (on keys it produces)
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// OR over the wave (DPP within rows, then the four rows), wave-uniform.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_or(uint32_t v) {
    return v | (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xf, 0xf, false);
}
__device__ __forceinline__ uint32_t wave_or_u32(uint32_t v) {
    v = dpp_or<0x140>(dpp_or<0x141>(dpp_or<0x4e>(dpp_or<0xb1>(v))));
    return (uint32_t)(__builtin_amdgcn_readlane((int)v, 0) | __builtin_amdgcn_readlane((int)v, 16) |
                      __builtin_amdgcn_readlane((int)v, 32) | __builtin_amdgcn_readlane((int)v, 48));
}

constexpr int kBins = 4096;    // value bins of the first stage
constexpr int kMaxRank = 512;  // candidates ranked directly at most

// Value bin of score v: monotone non-decreasing in v (each step is a
// correctly rounded operation or a clamp), so every key in a higher bin
// beats every key in a lower one.  -inf lands in bin 0.
__device__ __forceinline__ int value_bin(float v, float vmin, float scale) {
    const float t = (v - vmin) * scale;
    return (int)fminf(fmaxf(floorf(t), 0.f), (float)(kBins - 1));
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
                          int n_prefix, int n_keep, Keys& keys, int h) {
    __shared__ int hist[kWaves][256];  // also the kBins value histogram
    static_assert(kWaves * 256 == kBins, "LDS reuse");
    __shared__ int tot[256];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ uint32_t red[kWaves];
    __shared__ uint32_t ck[kMaxRank];
    __shared__ int ci[kMaxRank];
    __shared__ int s_digit, s_above, s_ncand, s_need;
    __shared__ uint32_t s_theta;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t* out = kept + (size_t)h * n_keep;

    if (N <= budget) {
        for (int i = tid; i < N; i += kThreads) out[i] = i;
        return;
    }
    keys.init(scores + (size_t)h * N, N);
    const int lo = n_prefix, hi = N - W;  // candidates [lo, hi)
    const int ksel = budget - n_prefix - W;
    if (tid == 0) {
        s_ncand = 0;
        s_need = 0;
    }

    // First, as in the register kernel: value bins over [min, max] of the
    // candidates' scores, then a direct rank of the threshold bin's keys;
    // keys in higher bins are larger than theta, keys in lower ones smaller,
    // so the emit below needs only theta and the number of ties to take.
    bool decided = false;
    uint32_t theta_v = 0;
    int need_v = 0;
    if (ksel > 0) {
        constexpr uint32_t kNegInf = 0x007fffffu, kPosInf = 0xff800000u;
        uint32_t kall = 0xffffffffu, kfin = 0xffffffffu, kmx = 0u;
        for (int j = lo + tid; j < hi; j += kThreads) {
            const uint32_t u = keys[j];
            kall = min(kall, u);
            kfin = min(kfin, u > kNegInf ? u : 0xffffffffu);
            kmx = max(kmx, u);
        }
        kall = block_min_u32(kall, red);
        kfin = block_min_u32(kfin, red);
        kmx = ~block_min_u32(~kmx, red);
        const float vmin = key_to_float(kfin), vmax = key_to_float(kmx);
        const float width = vmax - vmin, scale = (float)kBins / width;
        if (kall >= kNegInf && kmx < kPosInf && kfin < kPosInf && vmax > vmin && width < INFINITY &&
            scale < INFINITY) {
            int* h1 = &hist[0][0];
            for (int i = tid; i < kBins; i += kThreads) h1[i] = 0;
            __syncthreads();
            for (int j = lo + tid; j < hi; j += kThreads) atomicAdd(&h1[value_bin(key_to_float(keys[j]), vmin, scale)], 1);
            __syncthreads();
            find_wide_digit(h1, ksel, scan_buf, &s_digit, &s_above);
            __syncthreads();
            const int bstar = s_digit, rem = ksel - s_above, ncand = h1[bstar];
            if (ncand <= kMaxRank) {
                for (int j = lo + tid; j < hi; j += kThreads) {
                    const uint32_t u = keys[j];
                    if (value_bin(key_to_float(u), vmin, scale) == bstar) {
                        const int slot = atomicAdd(&s_ncand, 1);
                        ck[slot] = u;
                        ci[slot] = j;
                    }
                }
                __syncthreads();
                int rank = kMaxRank;
                uint32_t mk = 0;
                if (tid < ncand) {
                    mk = ck[tid];
                    const int mi = ci[tid];
                    rank = 0;
                    for (int c = 0; c < ncand; ++c) rank += (ck[c] > mk) || (ck[c] == mk && ci[c] < mi);
                    if (rank == rem - 1) s_theta = mk;
                }
                __syncthreads();
                if (tid < ncand && mk == s_theta && rank < rem) atomicAdd(&s_need, 1);
                __syncthreads();
                theta_v = s_theta;
                need_v = s_need;
                decided = true;
            }
        }
    }

    uint32_t prefix = 0, pmask = 0;
    int remaining = ksel;  // how many still to take at or below the current prefix
    if (ksel > 0 && !decided) {
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
    const uint32_t theta = decided ? theta_v : prefix;
    // ties at theta to take, lowest index first
    const int need_eq = (ksel > 0) ? (decided ? need_v : remaining) : 0;

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
    topk_head(scores, kept, N, budget, W, n_prefix, n_keep, keys, blockIdx.x);
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

constexpr int kPerMax = kRegKeys / kThreads;  // keys per thread at most
constexpr int kSub = 4;                         // histogram copies per wave

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

// Exclusive scan, in place, of the ROWS per-run counts c[i][wave] in
// token order (run (i, w) covers tokens i*1024 + 64 w ... + 63).
template <int ROWS>
__device__ __forceinline__ void scan_runs(int* c, int* buf) {
    const int t = threadIdx.x;
    const int v = (t < ROWS) ? c[t] : 0;
    int total;
    const int before = block_excl_scan(v, buf, &total);
    if (t < ROWS) c[t] = before;
    __syncthreads();
}

// PER keys per thread (8 or 32): heads of up to 1024 PER tokens.
template <int PER>
__global__ __launch_bounds__(kThreads) void topk_reg_kernel(const float* __restrict__ scores,
                                                             int32_t* __restrict__ kept, int N, int budget, int W,
                                                             int n_prefix, int n_keep) {
    // per-wave 8-bit histograms; the value histogram and the candidate list
    // of the first stage reuse the same memory before them
    __shared__ int hist[kWaves][kSub][256];
    static_assert(kWaves * kSub * 256 >= kBins + 2 * kMaxRank, "LDS reuse");
    __shared__ int part[kThreads / 256][256];
    __shared__ int tot[256];
    __shared__ int runs[PER * kWaves];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ uint32_t red[kWaves];
    __shared__ uint32_t red3[3][kWaves];
    __shared__ int s_digit, s_above, s_ncand, s_need, s_eqtot;
    __shared__ uint32_t s_theta;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int sub = lane >> 4;
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
    uint32_t u[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) u[i] = order_key(srow[min(tid + i * kThreads, N - 1)]);
    uint32_t pos_cand = 0;  // candidate positions (the rest are forced keeps or past N)
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        const int j = tid + i * kThreads;
        if (j >= lo && j < hi) pos_cand |= 1u << i;
    }
    uint32_t comp = pos_cand;  // candidates still competing for the remaining places
    uint32_t sure = 0;         // candidates kept whatever the threshold
    int remaining = ksel;
    bool decided = false;      // theta and need_eq known
    uint32_t theta = 0;
    int need_eq = 0;
    int eq_total = -1;         // candidates equal to theta, when known
    if (tid == 0) {
        s_ncand = 0;
        s_need = 0;
        s_eqtot = 0;
    }
    __syncthreads();  // the counters are clear before any wave adds to them
    if (ksel > 0) {
        // ---- stage 1: value bins over [vmin, vmax] of the candidates -----------
        // In key order -inf is kNegInf and the finite scores lie strictly
        // between it and kPosInf; NaN or +inf candidates take the radix path,
        // and vmin is the smallest finite score.
        constexpr uint32_t kNegInf = 0x007fffffu, kPosInf = 0xff800000u;
        uint32_t kall = 0xffffffffu, kfin = 0xffffffffu, kmx = 0u;
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const bool c = (pos_cand >> i) & 1u;
            kall = min(kall, c ? u[i] : 0xffffffffu);
            kfin = min(kfin, (c && u[i] > kNegInf) ? u[i] : 0xffffffffu);
            kmx = max(kmx, c ? u[i] : 0u);
        }
        {   // the three minima over the block in one exchange
            const uint32_t a = dev::wave_min_u32(kall), b = dev::wave_min_u32(kfin), c = dev::wave_min_u32(~kmx);
            if (lane == 0) {
                red3[0][wave] = a;
                red3[1][wave] = b;
                red3[2][wave] = c;
            }
            __syncthreads();
            kall = red3[0][0];
            kfin = red3[1][0];
            uint32_t nmx = red3[2][0];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) {
                kall = min(kall, red3[0][w]);
                kfin = min(kfin, red3[1][w]);
                nmx = min(nmx, red3[2][w]);
            }
            kmx = ~nmx;
        }
        const bool finite_or_neg_inf = kall >= kNegInf && kmx < kPosInf;
        const float vmin = key_to_float(kfin), vmax = key_to_float(kmx);
        const float width = vmax - vmin;
        const float scale = (float)kBins / width;
        const bool use_bins = finite_or_neg_inf && kfin < kPosInf && vmax > vmin && width < INFINITY &&
                              scale < INFINITY;
        if (use_bins) {
            int* h1 = &hist[0][0][0];
            for (int i = tid; i < kBins; i += kThreads) h1[i] = 0;
            __syncthreads();
            // value bins are spread, so plain atomics rarely collide
#pragma unroll
            for (int i = 0; i < PER; ++i)
                if ((pos_cand >> i) & 1u) atomicAdd(&h1[value_bin(key_to_float(u[i]), vmin, scale)], 1);
            __syncthreads();
            find_wide_digit(h1, remaining, scan_buf, &s_digit, &s_above);
            __syncthreads();
            const int bstar = s_digit;
            remaining -= s_above;
            const int ncand = h1[bstar];
            comp = 0;
#pragma unroll
            for (int i = 0; i < PER; ++i) {
                const int b = value_bin(key_to_float(u[i]), vmin, scale);
                sure |= (b > bstar ? 1u : 0u) << i;
                comp |= (b == bstar ? 1u : 0u) << i;
            }
            sure &= pos_cand;
            comp &= pos_cand;
            if (ncand <= kMaxRank) {
                // ---- stage 2a: rank the threshold bin's keys by (key descending,
                // token ascending); rank remaining - 1 is theta
                uint32_t* ck = reinterpret_cast<uint32_t*>(h1 + kBins);
                int* ci = h1 + kBins + kMaxRank;
                const uint32_t wcomp = wave_or_u32(comp);  // positions where some lane competes
#pragma unroll
                for (int i = 0; i < PER; ++i) {
                    if (!((wcomp >> i) & 1u)) continue;  // wave-uniform: usually skipped
                    if ((comp >> i) & 1u) {
                        const int slot = atomicAdd(&s_ncand, 1);
                        ck[slot] = u[i];
                        ci[slot] = tid + i * kThreads;
                    }
                }
                __syncthreads();
                int rank = kMaxRank;
                uint32_t mk = 0;
                if (tid < ncand) {
                    mk = ck[tid];
                    const int mi = ci[tid];
                    rank = 0;
                    for (int c = 0; c < ncand; ++c) {
                        const uint32_t k = ck[c];
                        rank += (k > mk) || (k == mk && ci[c] < mi);
                    }
                    if (rank == remaining - 1) s_theta = mk;
                }
                __syncthreads();
                theta = s_theta;
                if (tid < ncand && mk == theta) {
                    atomicAdd(&s_eqtot, 1);
                    if (rank < remaining) atomicAdd(&s_need, 1);
                }
                __syncthreads();
                need_eq = s_need;
                eq_total = s_eqtot;
                decided = true;
            }
        }
    }
    if (ksel > 0 && !decided) {
        // ---- stage 2b: exact radix select among the competing keys ----------
        // on v = key - (smallest competing key), over only the bits that vary
        uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
        for (int i = 0; i < PER; ++i)
            if ((comp >> i) & 1u) {
                kmin = min(kmin, u[i]);
                kmax = max(kmax, u[i]);
            }
        kmin = block_min_u32(kmin, red);
        kmax = ~block_min_u32(~kmax, red);
        const uint32_t key_lo = kmin;
        const int vbits = (kmax > kmin) ? 32 - __builtin_clz(kmax - kmin) : 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) u[i] -= key_lo;  // compared only where competing from here on
        uint32_t prefix = 0, pmask = 0;
        const int npass = (vbits + 7) / 8;
        for (int pass = 0; pass < npass; ++pass) {
            const int shift = max(0, vbits - 8 * (pass + 1));
            int* hz = &hist[0][0][0];
            for (int i = tid; i < kWaves * kSub * 256; i += kThreads) hz[i] = 0;
            __syncthreads();
            int* hw = &hist[wave][sub][0];
#pragma unroll
            for (int i = 0; i < PER; ++i)
                count_digit(hw, (u[i] >> shift) & 255u, ((comp >> i) & 1u) && (u[i] & pmask) == prefix);
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
            if (pass == npass - 1) eq_total = tot[s_digit];  // every bit decided: the keys equal to theta
            __syncthreads();
        }
        theta = prefix;
        need_eq = remaining;
    }
    // ---- emit ------------------------------------------------------------------
    // Ties at theta are ranked in token order only when some must be left out.
    const bool rank_ties = ksel > 0 && eq_total != need_eq;
    uint64_t eqb[PER];
    if (rank_ties) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            eqb[i] = __builtin_amdgcn_ballot_w64(((comp >> i) & 1u) && u[i] == theta);
            if (lane == 0) runs[i * kWaves + wave] = (int)__builtin_popcountll(eqb[i]);
        }
        __syncthreads();
        scan_runs<PER * kWaves>(runs, scan_buf);
    }
    // forced tokens (prefix, recent window) below N, the sure candidates, and
    // the competing ones at or above theta (ties only as far as need_eq)
    uint32_t valid = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) valid |= (tid + i * kThreads < N ? 1u : 0u) << i;
    uint32_t keep = valid & ~pos_cand;
    if (ksel > 0) {
        keep |= sure;
        const uint32_t wcomp = wave_or_u32(comp);
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            if (!((wcomp >> i) & 1u)) continue;  // wave-uniform
            bool k = u[i] > theta;
            if (u[i] == theta) k = !rank_ties || runs[i * kWaves + wave] + rank_in_wave(eqb[i]) < need_eq;
            if (((comp >> i) & 1u) && k) keep |= 1u << i;
        }
    }
    if (rank_ties) __syncthreads();  // tie ranks read before the counts are reused
    uint64_t kb[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        kb[i] = __builtin_amdgcn_ballot_w64((keep >> i) & 1u);
        if (lane == 0) runs[i * kWaves + wave] = (int)__builtin_popcountll(kb[i]);
    }
    __syncthreads();
    scan_runs<PER * kWaves>(runs, scan_buf);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        if ((keep >> i) & 1u) {
            const int pos = runs[i * kWaves + wave] + rank_in_wave(kb[i]);
            if (pos < n_keep) out[pos] = tid + i * kThreads;
        }
    }
}


// ---- heads split over several workgroups ------------------------------------
//
// A layer of fewer heads than twice the compute units leaves most of the
// machine idle with one workgroup per head, so each head's tokens are cut
// into M slices of at most kSliceMax, one workgroup each, over three
// launches (the kernel boundaries are the only synchronisation):
//   hist: each slice bins its candidates' scores over the fixed range
//         [-32, 0) nats (kBins bins; scores at or above 0 and NaN go to the
//         top bin, scores below -32 to the bottom one) and adds its counts
//         to the head's histogram in the workspace;
//   cut:  every slice finds the threshold bin T of the head from the full
//         histogram, counts its candidates above T, and lists those in T
//         (order key, token) in the workspace;
//   emit: every slice ranks the threshold bin's list by (key descending,
//         token ascending), which decides each listed token exactly; its
//         output position is the number of kept tokens in lower slices (the
//         forced ones, the counts above T and the listed kept tokens below
//         it) plus its rank within the slice.
// Scores returned by bkv_score are log-weights at or below 0, so the
// threshold bin rarely holds more than a few dozen tokens.  A head whose
// threshold bin lists more than kMaxRank tokens (ties in bulk, or a
// threshold far outside the range), or a workspace without the library's
// stamp, is selected whole by one workgroup of the emit launch with the
// one-workgroup algorithm above.
constexpr int kSliceMax = 16384;
constexpr int kSlicePer = kSliceMax / kThreads;  // tokens per thread at most
constexpr float kFixLo = -32.f;
constexpr float kFixScale = kBins / 32.f;  // bins per nat

// Bin of order key u over the fixed range: monotone non-decreasing in the key.
__device__ __forceinline__ int fixed_bin(uint32_t u) {
    if (u >= 0x80000000u) return kBins - 1;  // +0, positive scores, +inf, NaN
    const float v = key_to_float(u);          // negative scores and -inf (-NaN: NaN, to bin 0)
    return (int)fminf(fmaxf(floorf((v - kFixLo) * kFixScale), 0.f), (float)(kBins - 1));
}

struct SplitArgs {
    const float* scores;
    int32_t* kept;
    int N, budget, W, n_prefix, n_keep, P, M, slice;
    const int* hdr;  // workspace header (stamp)
    int* hist;       // [P][kBins] counts of the candidates' bins (left zero by the emit)
    int* head;       // [P][kTkHeadWords]: listed tokens, threshold bin, count above it
    uint32_t* cand;  // [P][kMaxRank][2]: the threshold bin's (order key, token)
    int* acnt;       // [P][kTkMaxSlices]: candidates above the threshold bin per slice
};

__device__ __forceinline__ int tk_ksel(const SplitArgs& a) { return a.budget - a.n_prefix - a.W; }

__global__ __launch_bounds__(kThreads) void topk_hist_kernel(SplitArgs a) {
    __shared__ int lh[kBins];
    const int h = blockIdx.x / a.M, sl = blockIdx.x % a.M, tid = threadIdx.x;
    if (sl == 0 && tid == 0) a.head[h * kTkHeadWords] = 0;  // the list of the cut launch starts empty
    if (tk_ksel(a) <= 0) return;
    const int lo = max(a.n_prefix, sl * a.slice), hi = min(a.N - a.W, (sl + 1) * a.slice);
    for (int i = tid; i < kBins; i += kThreads) lh[i] = 0;
    __syncthreads();
    const float* row = a.scores + (size_t)h * a.N;
    float v[kSlicePer];
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        const int j = lo + tid + i * kThreads;
        v[i] = j < hi ? row[j] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i)
        if (lo + tid + i * kThreads < hi) atomicAdd(&lh[fixed_bin(order_key(v[i]))], 1);
    __syncthreads();
    int* gh = a.hist + (size_t)h * kBins;
    for (int i = tid; i < kBins; i += kThreads) {
        const int c = lh[i];
        if (c) atomicAdd(&gh[i], c);
    }
}

__global__ __launch_bounds__(kThreads) void topk_cut_kernel(SplitArgs a) {
    __shared__ int scan_buf[kWaves + 1];
    __shared__ int s_digit, s_above;
    const int h = blockIdx.x / a.M, sl = blockIdx.x % a.M, tid = threadIdx.x;
    const int ksel = tk_ksel(a);
    if (ksel <= 0) return;
    // this slice's candidates in flight while the histogram is read
    const int lo = max(a.n_prefix, sl * a.slice), hi = min(a.N - a.W, (sl + 1) * a.slice);
    const float* row = a.scores + (size_t)h * a.N;
    float v[kSlicePer];
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        const int j = lo + tid + i * kThreads;
        v[i] = j < hi ? row[j] : 0.f;
    }
    // the bin holding the ksel-th candidate from the top (every slice finds
    // the same one; the candidates outnumber ksel since N > budget)
    if (tid == 0) {
        s_digit = 0;
        s_above = 0;
    }
    __syncthreads();
    find_wide_digit(a.hist + (size_t)h * kBins, ksel, scan_buf, &s_digit, &s_above);
    __syncthreads();
    const int T = s_digit;
    int* hw = a.head + h * kTkHeadWords;
    if (sl == 0 && tid == 0) {
        hw[1] = T;
        hw[2] = s_above;
    }
    uint32_t* ch = a.cand + (size_t)h * kMaxRank * 2;
    int above = 0;
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        const int j = lo + tid + i * kThreads;
        if (j >= hi) break;
        const uint32_t u = order_key(v[i]);
        const int b = fixed_bin(u);
        above += b > T;
        if (b == T) {
            const int p = atomicAdd(&hw[0], 1);
            if (p < kMaxRank) {
                ch[2 * p] = u;
                ch[2 * p + 1] = (uint32_t)j;
            }
        }
    }
    int total;
    block_excl_scan(above, scan_buf, &total);
    if (tid == 0) a.acnt[h * kTkMaxSlices + sl] = total;
}

__global__ __launch_bounds__(kThreads) void topk_emit_kernel(SplitArgs a) {
    __shared__ uint32_t ck[kMaxRank];
    __shared__ int ci[kMaxRank];
    __shared__ uint32_t tbits[kSliceMax / 32];  // listed tokens of this slice that are kept
    __shared__ int runs[kSlicePer * kWaves];
    __shared__ int scan_buf[kWaves + 1];
    __shared__ int s_below, s_lower;
    const int h = blockIdx.x / a.M, sl = blockIdx.x % a.M, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int N = a.N, ksel = tk_ksel(a);
    const int* hw = a.head + h * kTkHeadWords;
    // every independent load in flight at once: the head's words, the stamp,
    // the counts of lower slices and this slice's scores
    const int j0 = sl * a.slice, j1 = min(N, j0 + a.slice);
    const float* row = a.scores + (size_t)h * N;
    float v[kSlicePer];
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        const int j = j0 + tid + i * kThreads;
        v[i] = j < j1 ? row[j] : 0.f;
    }
    const int hw0 = hw[0], hw1 = hw[1], hw2 = hw[2];
    const int lower = (ksel > 0 && tid < sl) ? a.acnt[h * kTkMaxSlices + tid] : 0;  // sl < 64
    const int n = ksel > 0 ? hw0 : 0;
    const bool stamped = (uint32_t)a.hdr[kHdrMagic] == kWsMagic && a.hdr[kHdrP] == a.P;
    {   // this slice's share of the head's histogram is cleared for the next call
        int* gh = a.hist + (size_t)h * kBins;
        for (int i = sl * kBins / a.M + tid; i < (sl + 1) * kBins / a.M; i += kThreads) gh[i] = 0;
    }
    if (!stamped || n > kMaxRank) {
        if (sl == 0) {
            GlobalKeys keys;
            topk_head(a.scores, a.kept, N, a.budget, a.W, a.n_prefix, a.n_keep, keys, h);
        }
        return;
    }
    const int T = ksel > 0 ? hw1 : kBins;
    const int rem = ksel > 0 ? ksel - hw2 : 0;  // listed tokens to keep
    const uint32_t* ch = a.cand + (size_t)h * kMaxRank * 2;
    for (int i = tid; i < n; i += kThreads) {
        ck[i] = ch[2 * i];
        ci[i] = (int)ch[2 * i + 1];
    }
    for (int i = tid; i < kSliceMax / 32; i += kThreads) tbits[i] = 0u;
    if (tid == 0) s_below = 0;
    int lower_sum = lower;  // wave 0 holds the lower slices' counts (sl < 64)
    if (tid < 64) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) lower_sum += __shfl_xor(lower_sum, o, 64);
        if (tid == 0) s_lower = lower_sum;
    }
    __syncthreads();
    if (tid < n) {
        const uint32_t mk = ck[tid];
        const int mi = ci[tid];
        int rank = 0;
        for (int c = 0; c < n; ++c) rank += (ck[c] > mk) || (ck[c] == mk && ci[c] < mi);
        if (rank < rem) {
            if (mi < j0)
                atomicAdd(&s_below, 1);
            else if (mi < j1)
                atomicOr(&tbits[(mi - j0) >> 5], 1u << ((mi - j0) & 31));
        }
    }
    __syncthreads();
    // kept tokens before this slice: forced ones, those above T, listed ones
    const int lo = a.n_prefix, hi = N - a.W;  // candidates [lo, hi)
    const int base = min(j0, lo) + max(0, j0 - hi) + s_below + s_lower;
    // token j0 + tid + i * kThreads (coalesced); runs of 64 tokens in order
    const int per = (j1 - j0 + kThreads - 1) / kThreads;
    uint32_t keep = 0;
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        if (i >= per) break;
        const int j = j0 + tid + i * kThreads;
        bool k = false;
        if (j < j1) {
            if (j < lo || j >= hi) {
                k = true;
            } else if (ksel > 0) {
                const int b = fixed_bin(order_key(v[i]));
                k = b > T || (b == T && ((tbits[(j - j0) >> 5] >> ((j - j0) & 31)) & 1u));
            }
        }
        keep |= (k ? 1u : 0u) << i;
        const uint64_t kb = __builtin_amdgcn_ballot_w64(k);
        if (lane == 0) runs[i * kWaves + wave] = (int)__builtin_popcountll(kb);
    }
    __syncthreads();
    {
        const int nr = per * kWaves;
        const int v = tid < nr ? runs[tid] : 0;
        int total;
        const int before = block_excl_scan(v, scan_buf, &total);
        if (tid < nr) runs[tid] = before;
        __syncthreads();
    }
    int32_t* out = a.kept + (size_t)h * a.n_keep;
#pragma unroll
    for (int i = 0; i < kSlicePer; ++i) {
        if (i >= per) break;
        const bool k = (keep >> i) & 1u;
        const uint64_t kb = __builtin_amdgcn_ballot_w64(k);
        if (k) {
            const int pos = base + runs[i * kWaves + wave] + rank_in_wave(kb);
            if (pos < a.n_keep) out[pos] = j0 + tid + i * kThreads;
        }
    }
}

}  // namespace

// Slices per head of the split selection for this layer on this device;
// 1: one workgroup per head.
int topk_slices(const bkv_dims& d, int* slice) {
    const int P = d.B * d.Hkv;
    if (d.N <= d.budget || d.N <= kTkMinN || P < 1) return 1;
    int dev_id = 0, cus = 256;
    if (hipGetDevice(&dev_id) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id) != hipSuccess)
        cus = 256;
    // about two workgroups per compute unit; split only where a head would
    // otherwise leave seven of eight compute units idle (measured: 32 heads
    // of 64K tokens 109 -> 33 us, of 16K 20 -> 19 us; 128 heads of 32K
    // 23 us with one workgroup each, 32 us split)
    const int m0 = (2 * cus + P - 1) / P;
    if (m0 < 8) return 1;
    int sl = (d.N + m0 - 1) / m0;
    sl = (sl + 63) / 64 * 64;
    if (sl < 2048) sl = 2048;
    if (sl > kSliceMax) sl = kSliceMax;
    const int M = (d.N + sl - 1) / sl;
    if (M < 2 || M > kTkMaxSlices) return 1;
    *slice = sl;
    return M;
}

hipError_t launch_topk(const bkv_dims& d, const WsLayout& L, const float* scores, int32_t* kept, void* ws,
                       hipStream_t s) {
    const int P = d.B * d.Hkv;
    const int n_keep = d.N < d.budget ? d.N : d.budget;
    int slice = 0;
    const int M = (ws && L.tk_hist && P <= kTkMaxHeads) ? topk_slices(d, &slice) : 1;
    if (M > 1) {
        char* w = static_cast<char*>(ws);
        SplitArgs a;
        a.scores = scores;
        a.kept = kept;
        a.N = d.N;
        a.budget = d.budget;
        a.W = d.W;
        a.n_prefix = d.n_prefix;
        a.n_keep = n_keep;
        a.P = P;
        a.M = M;
        a.slice = slice;
        a.hdr = reinterpret_cast<const int*>(w);
        a.hist = reinterpret_cast<int*>(w + L.tk_hist);
        a.head = reinterpret_cast<int*>(w + L.tk_head);
        a.cand = reinterpret_cast<uint32_t*>(w + L.tk_cand);
        a.acnt = reinterpret_cast<int*>(w + L.tk_cnt);
        hipLaunchKernelGGL(topk_hist_kernel, dim3(P * M), dim3(kThreads), 0, s, a);
        hipLaunchKernelGGL(topk_cut_kernel, dim3(P * M), dim3(kThreads), 0, s, a);
        hipLaunchKernelGGL(topk_emit_kernel, dim3(P * M), dim3(kThreads), 0, s, a);
        return hipGetLastError();
    }
    if (d.N <= 8 * kThreads)
        hipLaunchKernelGGL(topk_reg_kernel<8>, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W,
                           d.n_prefix, n_keep);
    else if (d.N <= kRegKeys)
        hipLaunchKernelGGL(topk_reg_kernel<kPerMax>, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W,
                           d.n_prefix, n_keep);
    else
        hipLaunchKernelGGL(topk_kernel, dim3(P), dim3(kThreads), 0, s, scores, kept, d.N, d.budget, d.W,
                           d.n_prefix, n_keep);
    return hipGetLastError();
}

}  // namespace bkv
