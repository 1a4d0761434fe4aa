// Continual FPS for gfx950: farthest point sampling of pre-RoPE queries
// under cosine similarity (Appendix D.1, Algorithm 1), and the gather that
// replaces a query buffer by its selection (Section 4.2, Eq. fps_q; the
// FPS steps of Algorithm 2).
//
// One head per workgroup, three kernels by set size:
//
//  - fps_gram_kernel, n <= 64, one wave.  These are the buffers of the
//    continual path (B_Q^max = n_beacon + n_recent rows).  The whole Gram
//    matrix Q Q^T of the head comes from MFMA (exact bf16 products, fp32
//    sums; fp32 input uses the fp32 MFMA) and its diagonal gives the norms.
//    avg_i is then a column sum, and each pick costs one LDS read per lane
//    and a wave argmin on DPP and scalar instructions.
//  - fps_reg_kernel, bf16 and 64 < n <= 1024, 512 threads.  Prefill-sized
//    sets held in MFMA operand registers: each pick is one MFMA pass over
//    the head's rows against the picked row, and one barrier.
//  - fps_stream_kernel, fp32 sets and bf16 sets past 1024 rows, n up to
//    32768, 512 threads.  Thread t owns rows j = t + 512 i and keeps their
//    S_j and 1/|q_j| in registers; each pick re-reads every row once to
//    form cos(q_j, q_r), so the kernel moves about (m + 3) n D elements.
//
// The two larger kernels use the regrouped average
//     sum_j cos(q_i, q_j) = (q_i / |q_i|) . sum_j (q_j / |q_j|),
// which is O(n D) instead of O(n^2 D).  All three take the lowest index among equal values at every argmin, treat a
// zero vector as having cosine 0 with everything, and emit the picks in
// selection order.  The 1/n of avg_i is left out: it does not move the
// argmin.
#include <math.h>

#include "device_common.h"
#include "internal.h"

namespace bkv {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
using dev::u32x4;

constexpr int kGramMaxN = 64;
constexpr int kLdg = kGramMaxN + 1;  // LDS row stride of the cosine matrix: mirrored writes hit distinct banks
constexpr int kStreamThreads = 512;
constexpr int kStreamWaves = kStreamThreads / 64;
constexpr int kStreamMaxRpt = 64;  // rows per thread: n <= 32768
constexpr int kMaxGather = 128;    // rows a gather may write per head

// Elements per 16-byte chunk and their conversion to fp32.
template <typename T>
struct Elt;
template <>
struct Elt<uint16_t> {
    static constexpr int EV = 8;
    __device__ static void unpack(const u32x4& c, float* f) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            f[2 * i] = __uint_as_float(c[i] << 16);
            f[2 * i + 1] = __uint_as_float(c[i] & 0xffff0000u);
        }
    }
};
template <>
struct Elt<float> {
    static constexpr int EV = 4;
    __device__ static void unpack(const u32x4& c, float* f) {
#pragma unroll
        for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(c[i]);
    }
};

__device__ __forceinline__ u32x4 load16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void store16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

__device__ __forceinline__ float inv_norm(float sumsq) { return sumsq > 0.f ? 1.0f / sqrtf(sumsq) : 0.f; }

// Write chunk `piece` (16 source bytes) of a gathered row: copied bit for
// bit when the type is kept, widened to fp32 otherwise.
template <typename T, int D>
__device__ __forceinline__ void store_chunk(void* dst_row, int piece, const u32x4& c, bool widen) {
    constexpr int EV = Elt<T>::EV;
    if (sizeof(T) == 2 && widen) {
        float f[EV];
        Elt<T>::unpack(c, f);
        float* o = static_cast<float*>(dst_row) + piece * EV;
#pragma unroll
        for (int q = 0; q < EV / 4; ++q) {
            u32x4 w;
#pragma unroll
            for (int e = 0; e < 4; ++e) w[e] = __float_as_uint(f[4 * q + e]);
            store16(o + 4 * q, w);
        }
    } else {
        store16(static_cast<T*>(dst_row) + piece * EV, c);
    }
}

__device__ __forceinline__ void write_counts(int32_t* counts, int h, int dst_rows, int k, int tid, int nthreads) {
    if (!counts) return;
    int32_t* c = counts + (size_t)h * dst_rows;
    for (int i = tid; i < dst_rows; i += nthreads) c[i] = i < k ? 1 : 0;
}

// ---- n <= 64: Gram matrix on MFMA, one wave per head ---------------------------

// A lane's share of a 16-row block in MFMA operand order: lane group
// g = lane >> 4 holds bytes [64 v + 16 g, 64 v + 16 g + 16) of row
// (lane & 15), for v < NV.  The same registers serve as A (rows of the
// tile) and as B (columns), since both come from Q.
template <typename T, int D>
struct Blk {
    static constexpr int NV = D * (int)sizeof(T) / 64;
    u32x4 v[NV];
};

template <typename T, int D>
__device__ __forceinline__ void load_blk(Blk<T, D>& b, const T* head, int row0, int n, int lane) {
    constexpr int EV = Elt<T>::EV;
    const int r = row0 + (lane & 15);
    const T* p = head + (size_t)r * D + (lane >> 4) * EV;
#pragma unroll
    for (int v = 0; v < Blk<T, D>::NV; ++v) b.v[v] = (r < n) ? load16(p + v * 4 * EV) : u32x4{0u, 0u, 0u, 0u};
}

template <int D>
__device__ __forceinline__ void gram_mma(f32x4& acc, const Blk<uint16_t, D>& a, const Blk<uint16_t, D>& b) {
#pragma unroll
    for (int v = 0; v < Blk<uint16_t, D>::NV; ++v)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v[v]),
                                                      __builtin_bit_cast(bf16x8_t, b.v[v]), acc, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ void gram_mma(f32x4& acc, const Blk<float, D>& a, const Blk<float, D>& b) {
#pragma unroll
    for (int v = 0; v < Blk<float, D>::NV; ++v)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v[v][e]), __uint_as_float(b.v[v][e]), acc, 0,
                                                       0, 0);
}

// min(v, v of the lane that DPP control CTRL names); all 64 lanes active.
template <int CTRL>
__device__ __forceinline__ float dpp_min(float v) {
    const int w = __builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, 0xf, 0xf, false);
    return fminf(v, __int_as_float(w));
}

__device__ __forceinline__ float lane_value(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Minimum over the wave, the same in every lane: swaps within quads, then
// the half-row and row mirrors give each 16-lane row its minimum (DPP, no
// LDS round trip), and the four row minima are combined as scalars.
__device__ __forceinline__ float wave_min(float v) {
    v = dpp_min<0xb1>(v);   // quad_perm [1, 0, 3, 2]
    v = dpp_min<0x4e>(v);   // quad_perm [2, 3, 0, 1]
    v = dpp_min<0x141>(v);  // row_half_mirror
    v = dpp_min<0x140>(v);  // row_mirror
    return fminf(fminf(lane_value(v, 0), lane_value(v, 16)), fminf(lane_value(v, 32), lane_value(v, 48)));
}

// NB = ceil(n / 16) row blocks.  src is not restrict: dst may be src.
template <typename T, int D, int NB>
__global__ __launch_bounds__(64) void fps_gram_kernel(const T* src, int src_rows, int n, int kmax, int32_t* picks,
                                                      void* dst, int widen, int dst_rows, int32_t* counts) {
    __shared__ float G[16 * NB * kLdg];
    const int lane = threadIdx.x, g = lane >> 4, c16 = lane & 15;
    const int h = blockIdx.x;
    const T* qh = src + (size_t)h * src_rows * D;

    Blk<T, D> blk[NB];
    dev::static_for<NB>([&](auto I) { load_blk<T, D>(blk[I], qh, I * 16, n, lane); });
    // Gram tiles I <= J; each value also goes to its mirror, so the matrix
    // is exactly symmetric.  Lane (g, c16), register v of tile (I, J) holds
    // row 16 I + 4 g + v, column 16 J + c16.
    dev::static_for<NB>([&](auto I) {
        dev::static_for<NB>([&](auto J) {
            if constexpr (I <= J) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                gram_mma<D>(acc, blk[I], blk[J]);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int row = 16 * I + 4 * g + v, col = 16 * J + c16;
                    if (I != J || row <= col) {
                        G[row * kLdg + col] = acc[v];
                        G[col * kLdg + row] = acc[v];
                    }
                }
            }
        });
    });
    __syncthreads();
    // Lane i keeps 1/|q_i| (from the diagonal); cos(q_i, q_j) is formed as
    // G[j][i] * inv_i * inv_j when it is needed, with inv_j read from lane j.
    const bool live = lane < n;
    const float inv = live ? inv_norm(G[lane * kLdg + lane]) : 0.f;

    // first pick: argmin of the summed cosines of row `lane` (avg times n)
    // (a compile-time bound with a wave-uniform test: the cross-lane read
    // keeps a loop with a run-time trip count from being unrolled)
    float S = 0.f;
#pragma unroll
    for (int j = 0; j < 16 * NB; ++j)
        if (j < n) S = fmaf(G[j * kLdg + lane], lane_value(inv, j), S);
    S *= inv;
    bool done = !live;
    int mypick = 0;  // lane k keeps pick k
    for (int k = 0; k < kmax; ++k) {
        const float key = done ? INFINITY : S;
        const float mn = wave_min(key);
        // lowest undone lane at the minimum (never empty: an undone lane
        // exists while k < min(m, n), and a NaN key counts as a candidate)
        const unsigned long long bal = __ballot(!done && !(key > mn));
        const int r = __ffsll(bal) - 1;
        if (lane == k) mypick = r;
        if (lane == r) done = true;
        const float c = G[r * kLdg + lane] * inv * lane_value(inv, r);
        if (!done) S = (k == 0) ? c : fmaxf(S, c);
    }
    if (picks && lane < kmax) picks[(size_t)h * kmax + lane] = mypick;

    if (dst) {
        // The picked rows are still in the operand registers: lane (g, c)
        // writes bytes [64 v + 16 g, +16) of destination rows c, c + 16, ...,
        // which sit in the same lane group g of the source row's block, so
        // a cross-lane read (one per block and dword) fetches them.  Nothing
        // is re-read from memory, and every store follows all of the loads,
        // so dst may be src.
        constexpr int NV = Blk<T, D>::NV;
        const size_t drow_bytes = (size_t)D * ((sizeof(T) == 2 && widen) ? 4 : sizeof(T));
        char* dh = static_cast<char*>(dst) + (size_t)h * dst_rows * drow_bytes;
        for (int i0 = 0; i0 < kmax; i0 += 16) {
            const int i = i0 + c16;
            const int src_row = __shfl(mypick, i < kmax ? i : kmax - 1, 64);
            const int src_lane = (g << 4) | (src_row & 15), src_blk = src_row >> 4;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                u32x4 x = {0u, 0u, 0u, 0u};
                dev::static_for<NB>([&](auto I) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const unsigned y = (unsigned)__shfl((int)blk[I].v[v][e], src_lane, 64);
                        x[e] = (src_blk == I) ? y : x[e];
                    }
                });
                if (i < kmax) store_chunk<T, D>(dh + (size_t)i * drow_bytes, 4 * v + g, x, widen);
            }
        }
    }
    write_counts(counts, h, dst_rows, kmax, lane, 64);
}

// ---- n up to 32768: rows streamed per pick, 1024 threads per head -----------------

// Row loads are issued eight 16-byte chunks at a time, so that at most 32
// registers hold loads in flight next to the per-row state.
constexpr int kChunkGroup = 8;

// <row, x> for a row of D elements in global memory and D floats in LDS.
// x is re-read for every row (through an offset the compiler cannot see
// through): kept in registers across rows it would take D of them.
template <typename T, int D>
__device__ __forceinline__ float row_dot(const T* row, const float* x_lds) {
    constexpr int EV = Elt<T>::EV, CPR = D * (int)sizeof(T) / 16;
    int off = 0;
    asm volatile("" : "+v"(off));
    const float* x = x_lds + off;
    float p[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c0 = 0; c0 < CPR; c0 += kChunkGroup) {
#pragma unroll
        for (int c = c0; c < c0 + kChunkGroup; ++c) {
            float f[EV];
            Elt<T>::unpack(load16(row + c * EV), f);
#pragma unroll
            for (int e = 0; e < EV; ++e) p[e & 3] = fmaf(f[e], x[c * EV + e], p[e & 3]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    return (p[0] + p[1]) + (p[2] + p[3]);
}

template <typename T, int D>
__device__ __forceinline__ float row_sumsq(const T* row) {
    constexpr int EV = Elt<T>::EV, CPR = D * (int)sizeof(T) / 16;
    float p[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c0 = 0; c0 < CPR; c0 += kChunkGroup) {
#pragma unroll
        for (int c = c0; c < c0 + kChunkGroup; ++c) {
            float f[EV];
            Elt<T>::unpack(load16(row + c * EV), f);
#pragma unroll
            for (int e = 0; e < EV; ++e) p[e & 3] = fmaf(f[e], f[e], p[e & 3]);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    return (p[0] + p[1]) + (p[2] + p[3]);
}

template <typename T, int D, int RPT>
__global__ __launch_bounds__(kStreamThreads) void fps_stream_kernel(const T* src, int src_rows, int n, int kmax,
                                                                    int32_t* picks, void* dst, int widen, int dst_rows,
                                                                    int32_t* counts) {
    constexpr int NT = kStreamThreads;
    constexpr int EV = Elt<T>::EV, CPR = D * (int)sizeof(T) / 16;
    constexpr int NRG = NT / CPR;  // row groups of the column pass
    __shared__ __attribute__((aligned(16))) float red[NRG * D];
    __shared__ __attribute__((aligned(16))) float vec[D];  // mean direction, then the current pick
    __shared__ float tinv[NT];
    __shared__ unsigned long long wkey[kStreamWaves];
    __shared__ float winv[kStreamWaves];
    __shared__ int spick[kMaxGather];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int h = blockIdx.x;
    const T* qh = src + (size_t)h * src_rows * D;

    // norms of the owned rows
    float inv[RPT], S[RPT];
    unsigned long long done = 0;  // bit i: row t + NT i picked (or absent)
    dev::static_for<RPT>([&](auto i) {
        const int j = t + NT * i;
        inv[i] = (j < n) ? inv_norm(row_sumsq<T, D>(qh + (size_t)j * D)) : 0.f;
        S[i] = 0.f;
        if (j >= n) done |= 1ull << i;
        __builtin_amdgcn_sched_barrier(0);  // one row's loads in flight at a time: no spills
    });

    // sum of the unit vectors, NT rows at a time: thread (rg, cp) adds chunk
    // cp of rows rg, rg + NRG, ... of the tile, scaled by their inverse norms
    {
        const int cp = t % CPR, rg = t / CPR;
        float acc[EV];
#pragma unroll
        for (int e = 0; e < EV; ++e) acc[e] = 0.f;
        dev::static_for<RPT>([&](auto i) {
            if (NT * i < n) {  // uniform
                tinv[t] = inv[i];
                __syncthreads();
                for (int s = rg; s < NT && NT * i + s < n; s += NRG) {
                    float f[EV];
                    Elt<T>::unpack(load16(qh + (size_t)(NT * i + s) * D + cp * EV), f);
                    const float w = tinv[s];
#pragma unroll
                    for (int e = 0; e < EV; ++e) acc[e] = fmaf(f[e], w, acc[e]);
                }
                __syncthreads();
            }
        });
#pragma unroll
        for (int e = 0; e < EV; ++e) red[rg * D + cp * EV + e] = acc[e];
        __syncthreads();
        if (t < D) {
            float s = 0.f;
            for (int r = 0; r < NRG; ++r) s += red[r * D + t];
            vec[t] = s;
        }
        __syncthreads();
    }
    // avg_i times n
    dev::static_for<RPT>([&](auto i) {
        const int j = t + NT * i;
        if (j < n) S[i] = row_dot<T, D>(qh + (size_t)j * D, vec) * inv[i];
        __builtin_amdgcn_sched_barrier(0);
    });
    __syncthreads();  // every thread is done with vec before it holds the first pick

    for (int k = 0; k < kmax; ++k) {
        // (S, j) lexicographic minimum over the unpicked rows
        unsigned long long best = ~0ull;
        float binv = 0.f;
        dev::static_for<RPT>([&](auto i) {
            if (!((done >> i) & 1ull)) {
                const unsigned long long key = ((unsigned long long)dev::ord_key(S[i]) << 32) | (unsigned)(t + NT * i);
                if (key < best) {
                    best = key;
                    binv = inv[i];
                }
            }
        });
        const unsigned long long wbest = dev::wave_min_u64(best);
        if (wbest == ~0ull) {
            if (lane == 0) wkey[wave] = wbest;
        } else if (best == wbest) {  // keys are unique: exactly one lane
            wkey[wave] = wbest;
            winv[wave] = binv;
        }
        __syncthreads();
        unsigned long long gb = ~0ull;
        float rinv = 0.f;
#pragma unroll
        for (int w = 0; w < kStreamWaves; ++w) {
            const unsigned long long x = wkey[w];
            if (x < gb) {
                gb = x;
                rinv = winv[w];
            }
        }
        const int r = (int)(unsigned)gb;  // an unpicked row exists while k < min(m, n)
        if (t < CPR) {
            float f[EV];
            Elt<T>::unpack(load16(qh + (size_t)r * D + t * EV), f);
#pragma unroll
            for (int e = 0; e < EV; ++e) vec[t * EV + e] = f[e];
        }
        if (t == 0) {
            if (picks) picks[(size_t)h * kmax + k] = r;
            if (k < kMaxGather) spick[k] = r;
        }
        if (r % NT == t) done |= 1ull << (r / NT);
        __syncthreads();
        dev::static_for<RPT>([&](auto i) {
            if (!((done >> i) & 1ull)) {
                // the row address is formed here on every pick: hoisted out
                // of the pick loop, RPT 64-bit addresses would stay live
                int j = t + NT * i;
                asm volatile("" : "+v"(j));
                const float c = row_dot<T, D>(qh + (size_t)j * D, vec) * inv[i] * rinv;
                S[i] = (k == 0) ? c : fmaxf(S[i], c);
            }
            __builtin_amdgcn_sched_barrier(0);
        });
    }

    if (dst) {
        // all chunks of all picked rows are in registers on every wave
        // before any wave stores, so dst may be src
        constexpr int IT = (kMaxGather * CPR + NT - 1) / NT;
        u32x4 buf[IT];
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int c = t + NT * it, i = c / CPR, piece = c % CPR;
            buf[it] = (i < kmax) ? load16(qh + (size_t)spick[i] * D + piece * EV) : u32x4{0u, 0u, 0u, 0u};
        }
        dev::wait_all_memory();
        __syncthreads();
        const size_t drow_bytes = (size_t)D * ((sizeof(T) == 2 && widen) ? 4 : sizeof(T));
        char* dh = static_cast<char*>(dst) + (size_t)h * dst_rows * drow_bytes;
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int c = t + NT * it, i = c / CPR, piece = c % CPR;
            if (i < kmax) store_chunk<T, D>(dh + (size_t)i * drow_bytes, piece, buf[it], widen);
        }
    }
    write_counts(counts, h, dst_rows, kmax, t, NT);
}

// ---- 64 < n <= 1024, bf16: rows resident in MFMA operand registers ------------

constexpr int kRegThreads = 512;
constexpr int kRegWaves = kRegThreads / 64;
constexpr int kRegMaxNB = 8;                           // 16-row blocks per wave
constexpr int kRegMaxN = kRegWaves * 16 * kRegMaxNB;  // 1024

// Wave w holds rows 16 NB w .. 16 NB (w + 1) - 1 as NB blocks in the Gram
// kernel's operand layout (lane (g, c16), vector v: bytes [64 v + 16 g, +16)
// of row 16 b + c16 of the wave's block b), loaded once.  The norms, the
// sum of unit vectors and avg_i (C21's regrouped form) come from those
// registers.  Each pick then costs one MFMA pass per block with the picked
// row in every column of B, so lane (g, c16) receives <q_j, q_r> for rows
// 16 b + 4 g + v, where it keeps their S_j and 1/|q_j|.  Every wave posts
// its best (S, j) key and the candidate row itself (operand order) to LDS,
// so a single barrier per pick settles the argmin and hands every wave the
// picked row.  Nothing is re-read from memory until the gather.
template <int D, int NB>
__global__ __launch_bounds__(kRegThreads) void fps_reg_kernel(const uint16_t* src, int src_rows, int n, int kmax,
                                                             int32_t* picks, void* dst, int widen, int dst_rows,
                                                             int32_t* counts) {
    constexpr int NV = Blk<uint16_t, D>::NV;
    constexpr int RW = 16 * NB;  // rows per wave
    constexpr int CPR = D * 2 / 16;
    __shared__ __attribute__((aligned(16))) float rinv_s[kRegWaves * RW];  // 1/|q_j| of every row
    __shared__ __attribute__((aligned(16))) float rs0_s[kRegWaves * RW];   // avg_j times n
    __shared__ __attribute__((aligned(16))) float part[kRegWaves][D];      // per-wave sums of unit vectors
    __shared__ __attribute__((aligned(16))) float uvec[D];
    __shared__ u32x4 cand[2][kRegWaves][NV * 4];                            // each wave's candidate row
    __shared__ unsigned long long wkey[2][kRegWaves];
    __shared__ int spick[kMaxGather];
    const int t = threadIdx.x, lane = t & 63, g = lane >> 4, c16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(t >> 6);
    const int h = blockIdx.x;
    const uint16_t* qh = src + (size_t)h * src_rows * D;
    const int row0 = w * RW;

    Blk<uint16_t, D> q[NB];
    dev::static_for<NB>([&](auto b) { load_blk<uint16_t, D>(q[b], qh, row0 + 16 * b, n, lane); });

    // norms (rows past n are zero: inverse norm 0) and the wave's sum of
    // unit vectors, lane (g, c16) adding elements 32 v + 8 g + e of its rows
    float usum[NV][8];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) usum[v][e] = 0.f;
    dev::static_for<NB>([&](auto b) {
        float p = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            float f[8];
            Elt<uint16_t>::unpack(q[b].v[v], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) p = fmaf(f[e], f[e], p);
        }
        p += dev::shfl_xor_f(p, 16);
        p += dev::shfl_xor_f(p, 32);
        const float inv = inv_norm(p);
        if (g == 0) rinv_s[row0 + 16 * b + c16] = inv;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            float f[8];
            Elt<uint16_t>::unpack(q[b].v[v], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) usum[v][e] = fmaf(f[e], inv, usum[v][e]);
        }
    });
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float s = dev::row16_sum(usum[v][e]);  // over the 16 lanes of group g
            if (c16 == 0) part[w][32 * v + 8 * g + e] = s;
        }
    __syncthreads();
    if (t < D) {
        float s = 0.f;
#pragma unroll
        for (int x = 0; x < kRegWaves; ++x) s += part[x][t];
        uvec[t] = s;
    }
    __syncthreads();
    // avg_j times n = (q_j . sum of unit vectors) / |q_j|
    dev::static_for<NB>([&](auto b) {
        float p = 0.f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
            float f[8];
            Elt<uint16_t>::unpack(q[b].v[v], f);
#pragma unroll
            for (int e = 0; e < 8; ++e) p = fmaf(f[e], uvec[32 * v + 8 * g + e], p);
        }
        p += dev::shfl_xor_f(p, 16);
        p += dev::shfl_xor_f(p, 32);
        if (g == 0) rs0_s[row0 + 16 * b + c16] = p * rinv_s[row0 + 16 * b + c16];
    });
    __syncthreads();
    // The 16 lanes of lane group g all receive the MFMA results for rows
    // 16 b + 4 g + v (b < NB, v < 4); lane c16 tracks CPL of them, number
    // cg = CPL c16 + c: block cg / 4, v = cg % 4.  Its S_j and 1/|q_j| stay
    // in registers.
    constexpr int CPL = NB >= 4 ? NB / 4 : 1;
    float S[CPL], cinv[CPL];
    unsigned done = 0;  // bit c: candidate c picked, past n, or absent
    auto cand_row = [&](int c) {
        const int cg = c16 * CPL + c;
        return row0 + 16 * (cg >> 2) + 4 * g + (cg & 3);
    };
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int row = cand_row(c);
        const bool live = c16 * CPL + c < 4 * NB && row < n;
        S[c] = live ? rs0_s[row] : 0.f;
        cinv[c] = live ? rinv_s[row] : 0.f;
        if (!live) done |= 1u << c;
    }

    for (int k = 0; k < kmax; ++k) {
        const int buf = k & 1;
        // (S, j) lexicographic minimum over the wave's unpicked rows
        unsigned long long best = ~0ull;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const unsigned long long key = ((unsigned long long)dev::ord_key(S[c]) << 32) | (unsigned)cand_row(c);
            if (!((done >> c) & 1u) && key < best) best = key;
        }
        const unsigned long long wb = dev::wave_min_u64(best);
        const unsigned wlo = __builtin_amdgcn_readfirstlane((unsigned)wb);
        const unsigned whi = __builtin_amdgcn_readfirstlane((unsigned)(wb >> 32));
        if (whi != ~0u || wlo != ~0u) {
            // the wave's candidate row, from the operand registers of the
            // four lanes that hold it
            const int jl = (int)wlo - row0, bb = jl >> 4;
            if (c16 == (jl & 15)) {
                dev::static_for<NB>([&](auto b) {
                    if (b == bb) {
#pragma unroll
                        for (int v = 0; v < NV; ++v) cand[buf][w][4 * v + g] = q[b].v[v];
                    }
                });
            }
        }
        if (lane == 0) wkey[buf][w] = ((unsigned long long)whi << 32) | wlo;
        __syncthreads();
        // the double-buffered posts let the next pick write without a second
        // barrier: every wave has read these before it passes the next one
        unsigned long long gb = ~0ull;
        int ws = 0;
#pragma unroll
        for (int x = 0; x < kRegWaves; ++x) {
            const unsigned long long y = wkey[buf][x];
            if (y < gb) {
                gb = y;
                ws = x;
            }
        }
        // an unpicked row exists while k < min(m, n); the clamp only keeps
        // the reads below in bounds whatever the keys hold
        const int r = min(max(__builtin_amdgcn_readfirstlane((int)(unsigned)gb), 0), n - 1);
        ws = __builtin_amdgcn_readfirstlane(ws);
        const float rinv = rinv_s[r];
        Blk<uint16_t, D> pr;
#pragma unroll
        for (int v = 0; v < NV; ++v) pr.v[v] = cand[buf][ws][4 * v + g];
        if (t == 0) {
            if (picks) picks[(size_t)h * kmax + k] = r;
            if (k < kMaxGather) spick[k] = r;
        }
#pragma unroll
        for (int c = 0; c < CPL; ++c)
            if (cand_row(c) == r) done |= 1u << c;
        // <q_j, q_r> for every row of the wave; each lane keeps its own
        float dot[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) dot[c] = 0.f;
        dev::static_for<NB>([&](auto b) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            gram_mma<D>(acc, q[b], pr);
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const int cg = c16 * CPL + c;
                if ((cg >> 2) == b) {
                    const int v = cg & 3;
                    dot[c] = v == 0 ? acc[0] : v == 1 ? acc[1] : v == 2 ? acc[2] : acc[3];
                }
            }
        });
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const float cs = dot[c] * cinv[c] * rinv;
            S[c] = (k == 0) ? cs : fmaxf(S[c], cs);
        }
    }
    __syncthreads();  // spick complete

    if (dst) {
        // every chunk of every picked row is in registers on every wave
        // before any wave stores, so dst may be src
        constexpr int IT = (kMaxGather * CPR + kRegThreads - 1) / kRegThreads;
        u32x4 bufr[IT];
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int c = t + kRegThreads * it, i = c / CPR, piece = c % CPR;
            bufr[it] = (i < kmax) ? load16(qh + (size_t)spick[i] * D + piece * 8) : u32x4{0u, 0u, 0u, 0u};
        }
        dev::wait_all_memory();
        __syncthreads();
        const size_t drow_bytes = (size_t)D * (widen ? 4 : 2);
        char* dh = static_cast<char*>(dst) + (size_t)h * dst_rows * drow_bytes;
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            const int c = t + kRegThreads * it, i = c / CPR, piece = c % CPR;
            if (i < kmax) store_chunk<uint16_t, D>(dh + (size_t)i * drow_bytes, piece, bufr[it], widen);
        }
    }
    write_counts(counts, h, dst_rows, kmax, t, kRegThreads);
}

template <typename T, int D>
hipError_t launch_typed(int H, int n, int kmax, const void* src, int src_rows, int32_t* picks, void* dst, int widen,
                        int dst_rows, int32_t* counts, hipStream_t s) {
    const T* q = static_cast<const T*>(src);
    if (n <= kGramMaxN) {
        const dim3 grid(H), block(64);
        switch ((n + 15) / 16) {
            case 1: hipLaunchKernelGGL((fps_gram_kernel<T, D, 1>), grid, block, 0, s, q, src_rows, n, kmax, picks, dst, widen, dst_rows, counts); break;
            case 2: hipLaunchKernelGGL((fps_gram_kernel<T, D, 2>), grid, block, 0, s, q, src_rows, n, kmax, picks, dst, widen, dst_rows, counts); break;
            case 3: hipLaunchKernelGGL((fps_gram_kernel<T, D, 3>), grid, block, 0, s, q, src_rows, n, kmax, picks, dst, widen, dst_rows, counts); break;
            default: hipLaunchKernelGGL((fps_gram_kernel<T, D, 4>), grid, block, 0, s, q, src_rows, n, kmax, picks, dst, widen, dst_rows, counts); break;
        }
        return hipGetLastError();
    }
    if (sizeof(T) == 2 && n <= kRegMaxN) {
        const uint16_t* qb = reinterpret_cast<const uint16_t*>(src);
        const dim3 grid(H), block(kRegThreads);
#define BKV_FPS_REG(NB) \
    hipLaunchKernelGGL((fps_reg_kernel<D, NB>), grid, block, 0, s, qb, src_rows, n, kmax, picks, dst, widen, dst_rows, counts)
        const int nb = (n + 16 * kRegWaves - 1) / (16 * kRegWaves);
        if (nb <= 1) BKV_FPS_REG(1);
        else if (nb <= 2) BKV_FPS_REG(2);
        else if (nb <= 4) BKV_FPS_REG(4);
        else BKV_FPS_REG(kRegMaxNB);
#undef BKV_FPS_REG
        return hipGetLastError();
    }
    const int rows_per_thread = (n + kStreamThreads - 1) / kStreamThreads;
    const dim3 grid(H), block(kStreamThreads);
#define BKV_FPS_STREAM(R) \
    hipLaunchKernelGGL((fps_stream_kernel<T, D, R>), grid, block, 0, s, q, src_rows, n, kmax, picks, dst, widen, dst_rows, counts)
    if (rows_per_thread <= 1) BKV_FPS_STREAM(1);
    else if (rows_per_thread <= 2) BKV_FPS_STREAM(2);
    else if (rows_per_thread <= 4) BKV_FPS_STREAM(4);
    else if (rows_per_thread <= 8) BKV_FPS_STREAM(8);
    else if (rows_per_thread <= 16) BKV_FPS_STREAM(16);
    else if (rows_per_thread <= 32) BKV_FPS_STREAM(32);
    else BKV_FPS_STREAM(kStreamMaxRpt);
#undef BKV_FPS_STREAM
    return hipGetLastError();
}

}  // namespace

hipError_t launch_fps(int H, int n, int kmax, int D, int dtype, const void* src, int src_rows, int32_t* picks,
                      void* dst, int dst_dtype, int dst_rows, int32_t* counts, hipStream_t s) {
    const int widen = (dst && dtype == BKV_BF16 && dst_dtype == BKV_F32) ? 1 : 0;
    if (dtype == BKV_BF16)
        return D == 64 ? launch_typed<uint16_t, 64>(H, n, kmax, src, src_rows, picks, dst, widen, dst_rows, counts, s)
                       : launch_typed<uint16_t, 128>(H, n, kmax, src, src_rows, picks, dst, widen, dst_rows, counts, s);
    return D == 64 ? launch_typed<float, 64>(H, n, kmax, src, src_rows, picks, dst, widen, dst_rows, counts, s)
                   : launch_typed<float, 128>(H, n, kmax, src, src_rows, picks, dst, widen, dst_rows, counts, s);
}

}  // namespace bkv
