// The selection and compaction work items of the fused eviction launch
// (evict_kernel in score.hip), for a 256-thread workgroup.  They run on
// data other work items of the same launch produced on other XCDs, so they
// read it with agent-coherent loads, and what they publish they write with
// agent-coherent stores (the MI355X's per-XCD L2 caches are not coherent
// with each other for ordinary accesses).
//
//   select_item   (a4) one head's kept set: the first n_prefix and the last
//                 W tokens, plus the k_sel other tokens of highest score,
//                 ties to the lower index, ascending (Section 2.2 TopK;
//                 Algorithm 2, I_keep / k_sel / TopK / Sort);
//   compact_item  (a5) one segment of one head's order-preserving in-place
//                 compaction (Eq. 8; Algorithm 2, Gather after Sort).
#pragma once

#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace roles {

constexpr int kNT = 256;  // threads per workgroup
constexpr int kNW = kNT / 64;

__device__ __forceinline__ uint32_t order_key(float s) {
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0u;  // -0 ranks with +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(uint32_t k) {  // inverse of order_key on the keys it makes
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Block-wide exclusive scan of one int per thread; *total gets the sum.
// buf holds kNW ints.  Ends with a barrier, so buf can be reused at once.
__device__ __forceinline__ int block_scan(int v, int* buf, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) buf[wave] = x;
    __syncthreads();
    int before = x - v, sum = 0;
#pragma unroll
    for (int w = 0; w < kNW; ++w) {
        const int t = buf[w];
        if (w < wave) before += t;
        sum += t;
    }
    *total = sum;
    __syncthreads();
    return before;
}

// Minimum of an unsigned over the block (every thread gets it); buf holds kNW.
__device__ __forceinline__ uint32_t block_min(uint32_t v, uint32_t* buf) {
    v = dev::wave_min_u32(v);
    if ((threadIdx.x & 63) == 0) buf[threadIdx.x >> 6] = v;
    __syncthreads();
    uint32_t m = buf[0];
#pragma unroll
    for (int w = 1; w < kNW; ++w) m = min(m, buf[w]);
    __syncthreads();
    return m;
}

constexpr int kSelRank = 512;  // candidates ranked directly at most

// BINS value bins of the first stage (a multiple of kNT, at least 1024)
template <int BINS>
struct SelLds {
    int hist[BINS + 4];  // one spare bin
    uint32_t ck[kSelRank];
    int ci[kSelRank + kNT];  // candidate tokens, then per-thread counts
    uint32_t red[kNW];
    int scan[kNW];
    int digit, above, ncand, need, eqtot;
    uint32_t theta;
};

// Value bin of score v over [vmin, vmin + BINS / scale]: monotone
// non-decreasing in v, so a key in a higher bin beats any in a lower one.
template <int BINS>
__device__ __forceinline__ int value_bin(float v, float vmin, float scale) {
    const float t = (v - vmin) * scale;
    return (int)fminf(fmaxf(floorf(t), 0.f), (float)(BINS - 1));
}

// Suffix search over 256-digit or value-bin counts: thread t owns the
// B = n / kNT bins of reversed index rt = kNT-1-t, so the exclusive scan in
// thread order counts every higher bin.  Sets sl.digit to the bin at which
// the count from the top reaches r and sl.above to the count strictly above.
template <int B, class L>
__device__ __forceinline__ void find_from_top(const int* cnt, int r, L& sl) {
    const int rt = kNT - 1 - (int)threadIdx.x;
    int c[B], sum = 0;
#pragma unroll
    for (int i = 0; i < B; ++i) {
        c[i] = cnt[B * rt + i];
        sum += c[i];
    }
    int total;
    int above = block_scan(sum, sl.scan, &total);  // candidates in bins >= B (rt + 1)
#pragma unroll
    for (int i = B - 1; i >= 0; --i) {
        const int incl = above + c[i];
        if (incl >= r && above < r) {
            sl.digit = B * rt + i;
            sl.above = above;
        }
        above = incl;
    }
    __syncthreads();
}

// One head's selection.  srow: its N scores (written by other work items:
// read coherently); out: its n_keep = min(budget, N) kept indices (read by
// other work items: written coherently).  Candidates are [lo, hi) with
// lo = n_prefix, hi = N - W; ksel = budget - n_prefix - W of them are kept.
// Scores of one head for plain loads that are coherent across the XCDs'
// L2 caches (the sc1 cache policy, as agent-scope atomic loads use) but,
// unlike atomic loads, may be issued back to back by the compiler.
struct ScoreRow {
#if defined(__HIP_DEVICE_COMPILE__)
    __amdgpu_buffer_rsrc_t r;
    __device__ ScoreRow(const float* p, int n) : r(make(p, n)) {}
    // the descriptor from wave-uniform values (else every load is a loop)
    __device__ static __amdgpu_buffer_rsrc_t make(const float* p, int n) {
        const uintptr_t a = reinterpret_cast<uintptr_t>(p);
        const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
        void* q = reinterpret_cast<void*>(((uintptr_t)hi << 32) | lo);
        return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, __builtin_amdgcn_readfirstlane(n * 4), 0x00020000);
    }
    // offsets past the row read 0 (the buffer's range check)
    __device__ uint32_t key(int j) const {
        return order_key(__uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, j * 4, 0, kSc1)));
    }
#else
    __device__ ScoreRow(const float*, int) {}
    __device__ uint32_t key(int) const { return 0; }
#endif
    static constexpr int kSc1 = 16;  // cache policy bits: sc1
};

template <int BINS>
__device__ void select_stream(const float* srow, int32_t* out, int N, int budget, int W, int n_prefix,
                              SelLds<BINS>& sl) {
    const int tid = threadIdx.x;
    const int lo = n_prefix, hi = N - W, ksel = budget - n_prefix - W;
    const int n_keep = budget;
    const ScoreRow row(srow, N);
    auto key = [&](int j) { return row.key(j); };
    uint32_t theta = 0;
    int need = 0;
    bool decided = ksel <= 0;
    if (!decided) {
        // ---- value bins over [min, max] of the finite candidate scores -------
        constexpr uint32_t kNegInf = 0x007fffffu, kPosInf = 0xff800000u;
        uint32_t kall = 0xffffffffu, kfin = 0xffffffffu, nkmx = 0xffffffffu;
#pragma unroll 16
        for (int j = lo + tid; j < hi; j += kNT) {
            const uint32_t u = key(j);
            kall = min(kall, u);
            kfin = min(kfin, u > kNegInf ? u : 0xffffffffu);
            nkmx = min(nkmx, ~u);
        }
        kall = block_min(kall, sl.red);
        kfin = block_min(kfin, sl.red);
        const uint32_t kmx = ~block_min(nkmx, sl.red);
        const float vmin = key_float(kfin), vmax = key_float(kmx);
        const float width = vmax - vmin, scale = (float)BINS / width;
        if (kall >= kNegInf && kmx < kPosInf && kfin < kPosInf && vmax > vmin && width < INFINITY &&
            scale < INFINITY) {
            for (int i = tid; i < BINS; i += kNT) sl.hist[i] = 0;
            if (tid == 0) {
                sl.ncand = 0;
                sl.need = 0;
            }
            __syncthreads();
#pragma unroll 16
            for (int j = lo + tid; j < hi; j += kNT) atomicAdd(&sl.hist[value_bin<BINS>(key_float(key(j)), vmin, scale)], 1);
            __syncthreads();
            find_from_top<BINS / kNT>(sl.hist, ksel, sl);
            const int bstar = sl.digit, rem = ksel - sl.above, ncand = sl.hist[bstar];
            if (ncand <= kSelRank) {
                // rank the threshold bin's keys by (key descending, index ascending)
#pragma unroll 8
                for (int j = lo + tid; j < hi; j += kNT) {
                    const uint32_t u = key(j);
                    if (value_bin<BINS>(key_float(u), vmin, scale) == bstar) {
                        const int slot = atomicAdd(&sl.ncand, 1);
                        sl.ck[slot] = u;
                        sl.ci[slot] = j;
                    }
                }
                __syncthreads();
                for (int c0 = tid; c0 < ncand; c0 += kNT) {
                    const uint32_t mk = sl.ck[c0];
                    const int mi = sl.ci[c0];
                    int rank = 0;
                    for (int c = 0; c < ncand; ++c) rank += (sl.ck[c] > mk) || (sl.ck[c] == mk && sl.ci[c] < mi);
                    if (rank == rem - 1) sl.theta = mk;
                }
                __syncthreads();
                for (int c0 = tid; c0 < ncand; c0 += kNT) {
                    const uint32_t mk = sl.ck[c0];
                    const int mi = sl.ci[c0];
                    if (mk != sl.theta) continue;
                    int rank = 0;
                    for (int c = 0; c < ncand; ++c) rank += (sl.ck[c] > mk) || (sl.ck[c] == mk && sl.ci[c] < mi);
                    if (rank < rem) atomicAdd(&sl.need, 1);
                }
                __syncthreads();
                theta = sl.theta;
                need = sl.need;
                decided = true;
            }
        }
    }
    if (!decided) {
        // ---- exact radix select: 8-bit digits of the key from the top --------
        uint32_t prefix = 0, pmask = 0;
        int remaining = ksel;
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            for (int i = tid; i < 256; i += kNT) sl.hist[i] = 0;
            __syncthreads();
#pragma unroll 8
            for (int j = lo + tid; j < hi; j += kNT) {
                const uint32_t u = key(j);
                if ((u & pmask) == prefix) atomicAdd(&sl.hist[(u >> shift) & 255u], 1);
            }
            __syncthreads();
            find_from_top<1>(sl.hist, remaining, sl);
            prefix |= (uint32_t)sl.digit << shift;
            pmask |= 255u << shift;
            remaining -= sl.above;
            __syncthreads();
        }
        theta = prefix;
        need = remaining;
    }
    // ---- emit: thread t owns tokens [t per, (t + 1) per), ascending ------------
    const int per = (N + kNT - 1) / kNT;
    const int j0 = min(tid * per, N), j1 = min(j0 + per, N);
    int n_sure = 0, n_eq = 0;
    for (int j = j0; j < j1; ++j) {
        if (j < lo || j >= hi) {
            ++n_sure;
        } else if (ksel > 0) {
            const uint32_t u = key(j);
            n_sure += (u > theta);
            n_eq += (u == theta);
        }
    }
    int total;
    const int eq_before = block_scan(n_eq, sl.scan, &total);
    const int eq_take = max(0, min(n_eq, need - eq_before));
    int pos = block_scan(n_sure + eq_take, sl.scan, &total);
    int eq_seen = eq_before;
    for (int j = j0; j < j1; ++j) {
        bool keep = true;
        if (j >= lo && j < hi) {
            if (ksel <= 0) {
                keep = false;
            } else {
                const uint32_t u = key(j);
                if (u == theta) {
                    keep = eq_seen < need;
                    ++eq_seen;
                } else {
                    keep = u > theta;
                }
            }
        }
        if (keep && pos < n_keep) dev::st_flag(out + pos++, j);
    }
}

// Lanes below this one whose bit is set in mask.
__device__ __forceinline__ int rank_in_wave(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
}

// Exclusive scan, in place, of 2 kNT per-run counts in run order.
__device__ __forceinline__ void scan_runs(int* c, int* buf) {
    const int t = threadIdx.x;
    const int a0 = c[2 * t], a1 = c[2 * t + 1];
    int total;
    const int before = block_scan(a0 + a1, buf, &total);
    c[2 * t] = before;
    c[2 * t + 1] = before + a0;
    __syncthreads();
}

// The selection with the head's scores in registers, thread t holding the
// PER consecutive tokens PER t ... PER t + PER - 1 (heads of up to kNT * PER
// tokens), so that the kept tokens come out in order with one block scan.
// The candidates' scores are binned linearly over [-32, 0] in BINS bins
// (log-probabilities; lower scores share the first bin), a monotone map, so
// every key in a higher bin beats every key in a lower one.  The bin that
// holds the k_sel-th largest candidate has a few dozen keys on the
// workloads' scores; they are ranked directly by (key descending, token
// ascending), which decides theta and the ties.  Returns false, having
// written nothing, if that bin holds more than kSelRank candidates (many
// equal or nearly equal scores): the caller then takes the exact radix
// select.
template <int BINS, int PER>
__device__ bool select_bins(const float* srow, int32_t* out, int N, int budget, int W, int n_prefix,
                            SelLds<BINS>& sl) {
    static_assert(PER % 32 == 0 && kNT * PER / 32 <= BINS, "the kept-member bitmap fits the histogram");
    constexpr float kBS = BINS / 32.0f;  // bins per nat
    const int tid = threadIdx.x;
    const int lo = n_prefix, hi = N - W, ksel = budget - n_prefix - W;
    const int j0 = PER * tid;
    // this thread's candidates are i in [ilo, ihi), its forced tokens the
    // other i below iend (tokens from N on are neither)
    const int ilo = min(max(lo - j0, 0), PER), ihi = min(max(hi - j0, 0), PER), iend = min(max(N - j0, 0), PER);
    float v[PER];
#if defined(__HIP_DEVICE_COMPILE__)
    const __amdgpu_buffer_rsrc_t r = ScoreRow::make(srow, N);
    if ((reinterpret_cast<uintptr_t>(srow) & 15) == 0) {  // every load in flight at once
        dev::static_for<PER / 4>([&](auto qc) {
            constexpr int q = decltype(qc)::value;
            const auto x = __builtin_amdgcn_raw_buffer_load_b128(r, (j0 + 4 * q) * 4, 0, ScoreRow::kSc1);
            v[4 * q] = __uint_as_float(x[0]);
            v[4 * q + 1] = __uint_as_float(x[1]);
            v[4 * q + 2] = __uint_as_float(x[2]);
            v[4 * q + 3] = __uint_as_float(x[3]);
        });
    } else {
        dev::static_for<PER>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            v[i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (j0 + i) * 4, 0, ScoreRow::kSc1));
        });
    }
#endif
    // each key's bin, computed once (the scores themselves are not needed
    // again: the threshold bin's members are re-read)
    int bn[PER];
    dev::static_for<PER>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        bn[i] = (int)fminf(fmaxf(floorf((v[i] + 32.0f) * kBS), 0.f), (float)(BINS - 1));
    });
    // per-key flags as bits of masks built once, and integer arithmetic in the
    // per-key loops (comparisons there would become branches and masks)
    auto range_mask = [](int q, int a, int b) {  // bits i - 32 q of i in [a, b)
        const int x = min(max(a - 32 * q, 0), 32), y = min(max(b - 32 * q, 0), 32);
        const uint32_t below_y = y >= 32 ? 0xffffffffu : (1u << y) - 1u;
        const uint32_t below_x = x >= 32 ? 0xffffffffu : (1u << x) - 1u;
        return below_y & ~below_x;
    };
    uint32_t cm[PER / 32], fm[PER / 32];  // candidates; forced tokens
#pragma unroll
    for (int q = 0; q < PER / 32; ++q) {
        cm[q] = range_mask(q, ilo, ihi);
        fm[q] = range_mask(q, 0, iend) & ~cm[q];
    }
    auto bit = [&](const uint32_t* m, int i) { return (m[i / 32] >> (i % 32)) & 1u; };
    auto gt = [](int b, int t) { return (uint32_t)(t - b) >> 31; };             // b > t
    auto eq = [](int b, int t) { return ((uint32_t)(b ^ t) - 1u) >> 31; };      // b == t (small values)
    int* extra = sl.ci + kSelRank;  // kNT per-thread counts of kept threshold-bin members
    int bstar = BINS, nmem = 0;     // no candidate is kept by default
    if (ksel > 0) {
        for (int i = tid; i < BINS + 1; i += kNT) sl.hist[i] = 0;
        if (tid == 0) sl.ncand = 0;
        extra[tid] = 0;
        __syncthreads();
        dev::static_for<PER>([&](auto ic) {  // non-candidates count in the spare bin BINS
            constexpr int i = decltype(ic)::value;
            atomicAdd(&sl.hist[BINS + (bn[i] - BINS) * (int)bit(cm, i)], 1);
        });
        __syncthreads();
        find_from_top<BINS / kNT>(sl.hist, ksel, sl);
        bstar = sl.digit;
        const int rem = ksel - sl.above, ncand = sl.hist[bstar];
        if (ncand > kSelRank) return false;  // uniform: every thread read the same count
        // the threshold bin's members: a mask, then their scores re-read
        uint32_t mm[PER / 32];
#pragma unroll
        for (int q = 0; q < PER / 32; ++q) mm[q] = 0;
        dev::static_for<PER>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            mm[i / 32] |= (bit(cm, i) & eq(bn[i], bstar)) << (i % 32);
        });
        const ScoreRow row(srow, N);
#pragma unroll
        for (int q = 0; q < PER / 32; ++q) {
            for (uint32_t m = mm[q]; m; m &= m - 1) {
                const int j = j0 + 32 * q + __builtin_ctz(m);
                const int slot = atomicAdd(&sl.ncand, 1);
                sl.ck[slot] = row.key(j);
                sl.ci[slot] = j;
            }
        }
        __syncthreads();  // also: the histogram is read; it becomes the bitmap
        int* bits = sl.hist;  // kept members, one bit per token
        for (int i = tid; i < (N + 31) / 32; i += kNT) bits[i] = 0;
        __syncthreads();
        for (int c0 = tid; c0 < ncand; c0 += kNT) {
            const uint32_t mk = sl.ck[c0];
            const int mi = sl.ci[c0];
            int rank = 0;
            for (int c = 0; c < ncand; ++c) rank += (sl.ck[c] > mk) || (sl.ck[c] == mk && sl.ci[c] < mi);
            if (rank < rem) {
                atomicOr(&bits[mi >> 5], 1u << (mi & 31));
                atomicAdd(&extra[mi / PER], 1);
            }
        }
        __syncthreads();
        nmem = extra[tid];
    }
    // emit: this thread's kept tokens in order, after those of lower threads.
    // Keep masks first (forced tokens, and candidates above the threshold
    // bin), then the kept members of the threshold bin from the bitmap.
    uint32_t km[PER / 32];
#pragma unroll
    for (int q = 0; q < PER / 32; ++q) km[q] = 0;
    int n = nmem;
    dev::static_for<PER>([&](auto ic) {
        constexpr int i = decltype(ic)::value;
        const uint32_t k = bit(fm, i) | (bit(cm, i) & gt(bn[i], bstar));
        km[i / 32] |= k << (i % 32);
        n += (int)k;
    });
    if (ksel > 0) {
        const uint32_t* bits = reinterpret_cast<const uint32_t*>(sl.hist);
#pragma unroll
        for (int q = 0; q < PER / 32; ++q) {
            const int w0 = j0 + 32 * q;  // a multiple of 32: one bitmap word
            if (w0 < N) km[q] |= bits[w0 >> 5];
        }
    }
    int total;
    int pos = block_scan(n, sl.scan, &total);  // ends with a barrier: the bitmap is read
    if (budget <= BINS) {
        // the kept tokens in output order in LDS, then stored coalesced
        int* stage = sl.hist;
#pragma unroll
        for (int q = 0; q < PER / 32; ++q) {
            for (uint32_t m = km[q]; m; m &= m - 1) {
                if (pos < budget) stage[pos] = j0 + 32 * q + __builtin_ctz(m);
                ++pos;
            }
        }
        __syncthreads();
        for (int i = tid; i < min(total, budget); i += kNT) dev::st_flag(out + i, stage[i]);
        return true;
    }
#pragma unroll
    for (int q = 0; q < PER / 32; ++q) {
        for (uint32_t m = km[q]; m; m &= m - 1) {
            if (pos < budget) dev::st_flag(out + pos, j0 + 32 * q + __builtin_ctz(m));
            ++pos;
        }
    }
    return true;
}

// One head's selection; see select_bins and select_stream.
template <int BINS>
__device__ __forceinline__ void select_item(const float* srow, int32_t* out, int N, int budget, int W, int n_prefix,
                            SelLds<BINS>& sl) {
    if (N <= budget) {
        for (int i = threadIdx.x; i < N; i += kNT) dev::st_flag(out + i, i);
        return;
    }
    constexpr int PER = 128;  // scores per thread in registers
    if (N <= kNT * PER && select_bins<BINS, PER>(srow, out, N, budget, W, n_prefix, sl)) return;
    __syncthreads();  // the fast path's LDS is reused
    select_stream<BINS>(srow, out, N, budget, W, n_prefix, sl);
}

constexpr int kSegF = 256;  // compaction rows per fused work item

// One segment (rows [seg kSegF, ...)) of head h's in-place compaction.
// kh: the head's kept indices (read coherently); flags: the head's
// per-segment read-done flags.  A segment loads every source row of K and V
// it moves into registers, raises its flag, waits for every lower segment
// whose source rows [first, last] meet its destination rows (those still
// have to read rows it overwrites; they hold lower tickets), then stores.
// Returns false if the kept indices are not strictly ascending within
// [0, N) (the segment then moves nothing).  s_src holds kSegF ints.
template <int RB>
__device__ __forceinline__ bool compact_item(char* Kh, char* Vh, const int32_t* kh, int* flags, int seg, int n_keep, int N,
                             int* s_src, int* s_bits, int* hdr) {
    constexpr int VPR = RB / 16;
    constexpr int NV = 2 * kSegF * VPR / kNT;  // 16-byte vectors per thread (K and V)
    const int tid = threadIdx.x;
    const int i0 = seg * kSegF;
    const int rows = min(kSegF, n_keep - i0);
    if (tid == 0) s_bits[0] = s_bits[1] = 0;
    __syncthreads();
    if (tid < rows) {
        const int src = dev::ld_flag(kh + i0 + tid);
        s_src[tid] = src;
        if (src != i0 + tid) s_bits[0] = 1;  // something moves
        if (src < i0 + tid || src >= N || (i0 + tid > 0 && src <= dev::ld_flag(kh + i0 + tid - 1))) s_bits[1] = 1;
    }
    __syncthreads();
    const bool bad = s_bits[1] != 0;
    const bool move = s_bits[0] != 0 && !bad;
    dev::u32x4 buf[NV];
    if (move) {
        dev::static_for<NV>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int e = tid + k * kNT;
            const int which = e / (kSegF * VPR);  // 0 = K, 1 = V
            const int r = (e / VPR) % kSegF, v = e % VPR;
            if (r < rows && s_src[r] != i0 + r) {
                const char* base = which ? Vh : Kh;
                buf[k] = __builtin_nontemporal_load(reinterpret_cast<const dev::u32x4*>(base + (size_t)s_src[r] * RB) + v);
            }
        });
    }
    dev::wait_all_memory();  // every read has returned before the flag goes up
    __syncthreads();
    if (tid == 0) dev::st_flag(flags + seg, 1);
    if (move) {
        if (tid < 64) {
            for (int sp = tid; sp < seg; sp += 64) {
                const int first = dev::ld_flag(kh + sp * kSegF);
                const int last = dev::ld_flag(kh + min((sp + 1) * kSegF, n_keep) - 1);
                if (last >= i0 && first < i0 + rows && !dev::wait_flag(flags + sp)) {
                    s_bits[0] = 0;
                    dev::raise_error(hdr, kErrCompactWait);
                }
            }
        }
        __syncthreads();
        if (s_bits[0]) {
            dev::static_for<NV>([&](auto kc) {
                constexpr int k = decltype(kc)::value;
                const int e = tid + k * kNT;
                const int which = e / (kSegF * VPR);
                const int r = (e / VPR) % kSegF, v = e % VPR;
                if (r < rows && s_src[r] != i0 + r) {
                    char* base = which ? Vh : Kh;
                    __builtin_nontemporal_store(buf[k], reinterpret_cast<dev::u32x4*>(base + (size_t)(i0 + r) * RB) + v);
                }
            });
        }
    }
    return !bad;
}

}  // namespace roles
}  // namespace bkv
