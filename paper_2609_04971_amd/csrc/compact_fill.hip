// Hole-filling compaction for gfx950: rows [0, n) of each head end up
// holding the kept set, but only the kept rows at or above n move.  A kept
// row below n stays where it is; the m-th evicted position below n
// (ascending) takes the m-th kept row at or above n (ascending).  The
// order-preserving compaction of Algorithm 2 (Gather after Sort) shifts
// every row after the first evicted one; this layout moves at most the
// kept rows that lie past n, which after a periodic eviction of B_max -> 7/8
// B_max (Section 5.1) is at most 1/8 of the cache.
//
// Sources lie at or above n and destinations below it, so no move can read
// a row another move writes: the copy needs no ordering at all.  One
// workgroup per head first writes src_of (the old position of the row each
// position ends up with), then a grid of items of 1024 positions copies the
// rows whose src_of differs from their position.
//
// src_of: a bitmap of the kept positions below n goes to LDS; position p
// is a hole of rank m = p - (kept positions below p), counted from a block
// scan of the bitmap words' popcounts and the popcount of p's word below p,
// and takes kept[c + m], c being the number of kept rows below n.
#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr int kMapThreads = 256;  // small workgroups: many heads in flight per compute unit
constexpr int kMapWaves = kMapThreads / 64;
constexpr int kCopyThreads = 256;
constexpr int kCopyItem = 1024;  // positions per copy work item
constexpr int kCopyRows = 64;    // rows copied per pass

// Exclusive scan of one int per thread over the block; buf holds kMapWaves ints.
__device__ __forceinline__ int block_excl_scan(int v, int* buf) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(x, o, 64);
        if (lane >= o) x += y;
    }
    if (lane == 63) buf[wave] = x;
    __syncthreads();
    int before = x - v;
    for (int w = 0; w < wave; ++w) before += buf[w];
    __syncthreads();
    return before;
}

__global__ __launch_bounds__(kMapThreads) void fill_map_kernel(const int32_t* __restrict__ kept,
                                                               int32_t* __restrict__ src_of, int N, int n_keep,
                                                               int P, int budget, int* hdr) {
    __shared__ uint32_t bits[kMaxFillKeep / 32];
    __shared__ int wpre[kMaxFillKeep / 32];  // kept positions below each word
    __shared__ int scan_buf[kMapWaves];
    __shared__ int s_c, s_bad, s_ok;
    const int h = blockIdx.x, tid = threadIdx.x;
    const int32_t* kh = kept + (size_t)h * n_keep;
    int32_t* so = src_of + (size_t)h * n_keep;
    const int nw = (n_keep + 31) / 32;
    for (int w = tid; w < nw; w += kMapThreads) bits[w] = 0u;
    if (tid == 0) {
        s_c = 0;
        s_bad = 0;
        const dev::u32x4 hd = *reinterpret_cast<const dev::u32x4*>(hdr);
        s_ok = hd[kHdrMagic] == kWsMagic && (int)hd[kHdrP] == P && (int)hd[kHdrBudget] == budget;
        if (!s_ok) dev::raise_error(hdr, kErrStamp);
    }
    __syncthreads();
    int below = 0;  // kept positions below n seen by this thread
#pragma unroll 4
    for (int i = tid; i < n_keep; i += kMapThreads) {
        const int k = kh[i];
        if (k < 0 || k >= N || (i > 0 && k <= kh[i - 1])) s_bad = 1;  // benign race: any writer stores 1
        if (k >= 0 && k < n_keep) {
            atomicOr(&bits[k >> 5], 1u << (k & 31));
            ++below;
        }
    }
    if (below) atomicAdd(&s_c, below);
    __syncthreads();
    if (s_bad && tid == 0) dev::raise_error(hdr, kErrBadIndex);
    if (s_bad || !s_ok) {  // move nothing
        for (int p = tid; p < n_keep; p += kMapThreads) so[p] = p;
        return;
    }
    const int c = s_c;
    // kept positions below each bitmap word: thread t takes the words
    // [w0, w1), a block scan gives the count below w0
    const int wpt = (nw + kMapThreads - 1) / kMapThreads;
    const int w0 = min(tid * wpt, nw), w1 = min(w0 + wpt, nw);
    int mine = 0;
    for (int w = w0; w < w1; ++w) mine += __builtin_popcount(bits[w]);
    int below_w = block_excl_scan(mine, scan_buf);
    for (int w = w0; w < w1; ++w) {
        wpre[w] = below_w;
        below_w += __builtin_popcount(bits[w]);
    }
    __syncthreads();
    // one position per thread and pass: coalesced stores, and loads that
    // do not wait on one another (a kept position loads kept[0], unused)
#pragma unroll 4
    for (int p = tid; p < n_keep; p += kMapThreads) {
        const uint32_t b = bits[p >> 5];
        const int i = p & 31;
        const bool stays = (b >> i) & 1u;
        const int kept_below = wpre[p >> 5] + __builtin_popcount(b & ((1u << i) - 1u));
        const int from = kh[stays ? 0 : c + (p - kept_below)];  // hole of rank p - kept_below
        so[p] = stays ? p : from;
    }
}

// RB = row bytes; VPR = 16-byte vectors per row.  Item (head, chunk) lists
// the moves among positions [kCopyItem chunk, + kCopyItem) (those whose
// src_of differs from the position) in LDS, in any order, then copies them
// kCopyRows rows per pass.  Items sized by positions rather than by moves
// keep the grid small where few rows move (the steady state of a periodic
// eviction moves a few per cent of them).
template <int RB>
__global__ __launch_bounds__(kCopyThreads) void fill_copy_kernel(char* K, char* V, const int32_t* __restrict__ src_of,
                                                                 int n_keep, int nchunk, size_t head_stride) {
    constexpr int VPR = RB / 16;
    constexpr int NV = 2 * kCopyRows * VPR / kCopyThreads;  // 16-byte vectors per thread and pass (K and V)
    static_assert(2 * kCopyRows * VPR % kCopyThreads == 0, "whole vectors per thread");
    __shared__ int s_src[kCopyItem], s_dst[kCopyItem];
    __shared__ int s_n;
    const int h = blockIdx.x / nchunk, ch = blockIdx.x - h * nchunk;
    const int j0 = ch * kCopyItem, rows = min(kCopyItem, n_keep - j0);
    const int tid = threadIdx.x;
    if (tid == 0) s_n = 0;
    __syncthreads();
    for (int r = tid; r < rows; r += kCopyThreads) {
        const int src = src_of[(size_t)h * n_keep + j0 + r];
        if (src != j0 + r) {
            const int slot = atomicAdd(&s_n, 1);  // at most rows slots
            s_src[slot] = src;
            s_dst[slot] = j0 + r;
        }
    }
    __syncthreads();
    const int nm = s_n;
    char* Kh = K + (size_t)h * head_stride;
    char* Vh = V + (size_t)h * head_stride;
    for (int m0 = 0; m0 < nm; m0 += kCopyRows) {
        const int mr = min(kCopyRows, nm - m0);
        dev::u32x4 buf[NV];
        dev::static_for<NV>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int e = tid + k * kCopyThreads;
            const int which = e / (kCopyRows * VPR);
            const int r = (e / VPR) % kCopyRows, v = e % VPR;
            if (r < mr)
                buf[k] = __builtin_nontemporal_load(
                    reinterpret_cast<const dev::u32x4*>((which ? Vh : Kh) + (size_t)s_src[m0 + r] * RB) + v);
        });
        dev::static_for<NV>([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            const int e = tid + k * kCopyThreads;
            const int which = e / (kCopyRows * VPR);
            const int r = (e / VPR) % kCopyRows, v = e % VPR;
            if (r < mr)
                __builtin_nontemporal_store(
                    buf[k], reinterpret_cast<dev::u32x4*>((which ? Vh : Kh) + (size_t)s_dst[m0 + r] * RB) + v);
        });
    }
}

}  // namespace

hipError_t launch_compact_fill(const bkv_dims& d, void* K, void* V, const int32_t* kept, int32_t* src_of, void* ws,
                               hipStream_t s) {
    const int P = d.B * d.Hkv;
    const int n_keep = d.N < d.budget ? d.N : d.budget;
    if (P == 0 || n_keep == 0) return hipSuccess;
    hipLaunchKernelGGL(fill_map_kernel, dim3(P), dim3(kMapThreads), 0, s, kept, src_of, d.N, n_keep, P, d.budget,
                       static_cast<int*>(ws));
    const int nchunk = (n_keep + kCopyItem - 1) / kCopyItem;
    const int es = d.dtype == BKV_BF16 ? 2 : 4;
    const int rb = d.D * es;
    const size_t hs = (size_t)d.N_cap * rb;
    char* k = static_cast<char*>(K);
    char* v = static_cast<char*>(V);
    switch (rb) {
        case 128: hipLaunchKernelGGL(fill_copy_kernel<128>, dim3(P * nchunk), dim3(kCopyThreads), 0, s, k, v, src_of, n_keep, nchunk, hs); break;
        case 256: hipLaunchKernelGGL(fill_copy_kernel<256>, dim3(P * nchunk), dim3(kCopyThreads), 0, s, k, v, src_of, n_keep, nchunk, hs); break;
        default: hipLaunchKernelGGL(fill_copy_kernel<512>, dim3(P * nchunk), dim3(kCopyThreads), 0, s, k, v, src_of, n_keep, nchunk, hs); break;
    }
    return hipGetLastError();
}

}  // namespace bkv
