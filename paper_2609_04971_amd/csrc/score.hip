// (a2)+(a3) Observation rows and key scores for gfx950.
//
// For every (batch, kv-head) the observation rows y_r are the occupied
// beacons rotated to the current step plus the recent queries of the GQA
// group (Section 4.3; Algorithm 2).  With l_rj = scale * <y_r, k_j>, the
// key score is  s_j = max_r (l_rj - lse_r),  lse_r = log sum_j exp(l_rj):
// softmax attention normalised over all N keys (Eq. 4), aggregated by max
// over every query and head of the group (Eq. 6, max form).
//
// One launch scores a layer.  Each head gets 2 * nch workgroups, which
// take a per-head ticket when they start: the first nch tickets are
//   S(h, c)  row statistics (max m, sum z) of l over key chunk c; the last
//            S item of a head folds them into lse_r;
// and the next nch are
//   F(h, c)  recompute l for chunk c and write s_j = max_r (l_rj - lse_r).
// An F item waits only for the S items of its head, which hold lower
// tickets, have started, and never wait, so the schedule cannot deadlock
// whatever the residency.  The grid lists a head's F workgroups `lag`
// heads after its S workgroups, so the second read of a head's keys follows
// the first closely (it tends to hit the MI355X's memory-side cache rather
// than HBM).  The fused eviction (evict_kernel, below) adds a selection and
// compaction items per head under the same tickets.
//
// The only data passed between work items are the per-chunk statistics and
// lse, a few KB per head.  Those go through agent-scope atomic loads and
// stores, which are coherent across the MI355X's per-XCD L2 caches by
// themselves; a producer waits for its stores to complete (s_waitcnt)
// before the counter or flag that publishes them, so no L2 write-back or
// invalidation is needed.
//
// Logits come from v_mfma_f32_16x16x32_bf16 (fp32 accumulation of exact
// bf16 products; fp32 caches use v_mfma_f32_16x16x4_f32).  Statistics are
// kept in log2 units (v_exp_f32 computes 2^x): s2 = scale * log2(e).  In F
// items the accumulator starts at -lse2_r / s2, so the MFMA yields
// l_rj - lse_r (up to the factor s2) directly and the epilogue is one max
// per element.  Two paths:
//   fast (bf16, R <= 1152): a rows kernel first writes each head's
//     observation rows to the workspace in MFMA operand order; work items
//     hold a group of up to 144 rows in registers and stage 32-key groups
//     of K through LDS (direct-to-LDS loads, double-buffered per wave).
//     Heads of four row groups give each wave one group and share one key
//     stream among the four waves (row split); see the sections below.
//   generic (fp32, or more rows): every item builds its rows in LDS from
//     the read-only inputs (RoPE, then rounding to the cache dtype) and
//     reads key tiles straight from HBM into MFMA operand registers with
//     16-byte loads, each load instruction covering 64 contiguous bytes of
//     each of 16 rows.
#include <math.h>
#include <string.h>

#include "device_common.h"
#include "evict_roles.h"
#include "internal.h"

namespace bkv {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;  // 4 waves
constexpr int kWaves = 4;
constexpr int kMaxC = 64;

template <typename T>
struct Tr;
template <>
struct Tr<uint16_t> {  // bf16 storage
    static constexpr int ES = 2;
    static constexpr int PAD = 8;   // LDS row padding, elements (16 bytes)
    static constexpr int RG = 144;  // observation rows resident in LDS at a time
};
template <>
struct Tr<float> {
    static constexpr int ES = 4;
    static constexpr int PAD = 4;
    static constexpr int RG = 64;
};

struct Args {
    const void* K;
    const void* qwin;
    const float* beacons;
    const int32_t* counts;
    const float* rope_cos;
    const float* rope_sin;
    float* scores;
    float* row_lse;
    int* hdr;
    int* hctl;      // [P][kHcWords] per-head control lines
    float* part_m;  // [P][nch][R_pad_max] chunk row maxima (log2 units)
    float* part_z;  // [P][nch][R_pad_max] chunk row sums relative to part_m
    float* lse2;    // [P][R_pad_max] row log2-normalisers
    uint16_t* rows; // [P][R_pad_max / 16][NV][64] observation rows, one MFMA operand vector per lane
    int* rmeta;     // [P][kMetaWords] occupied beacon slots of each head
    int B, Hq, Hkv, G, N, N_cap, W, C, P, budget;
    int R_pad_max, nch, key_chunk, lag, total;
    float s2;     // scale * log2(e)
    float s2ln2;  // s2 * ln(2): log2-units-of-raw-dot -> natural log
    int mean;     // aggregate by the mean over rows (else the max)
    int causal;   // recent row w sees keys up to N - W + w only
    int tickets;  // work items per head (the ticket limit)
    // the fused eviction launch (evict_kernel): after each head's score items
    // one selection item and nsegF compaction items of roles::kSegF rows
    int fused;
    char* Kc;       // K and V, compacted in place
    char* Vc;
    int32_t* kept;  // [P][n_keep]
    int* cflags;    // [P][nseg_cap] compaction read-done flags
    int n_prefix, n_keep, nsegF, nseg_cap, lag2, lag3;
    // grid regions of the fused launch: slots [rs[i], rs[i+1]) hold rper[i]
    // workgroups each, starting at workgroup rb[i]
    int nreg;
    int rs[8], rb[8], rper[8];
};

// Which (key, row) pairs enter the scores: keys at or past N never do, and
// with the causal option recent row w of a query head (rows nact..R-1 of
// the head, w = (row - nact) % W, oldest first) sees keys up to its own
// position N - W + w only.  Beacon rows and padding rows see every key.
struct KeyMask {
    int N, W, nact, R, causal;
    __device__ __forceinline__ int limit(int row) const {  // last key the row sees
        return (causal && row >= nact && row < R) ? N - W + (row - nact) % W : N - 1;
    }
    // keys below this are seen by every row
    __device__ __forceinline__ int all_see_below() const { return causal ? min(N, N - W + 1) : N; }
};

__device__ __forceinline__ KeyMask key_mask(const Args& a, int nact) {
    return KeyMask{a.N, a.W, nact, nact + a.G * a.W, a.causal};
}

// Per-lane operand: NV 16-byte vectors of one row.  Vector v of lane group
// g (lane >> 4) holds bytes [64 v + 16 g, 64 v + 16 g + 16) of the row, so
// the four lane groups of a load instruction read 64 contiguous bytes of
// each row and two consecutive instructions complete a 128-byte line.  For
// bf16 vector v is one MFMA step (k = 32 elements); for fp32 it is four.
template <typename T, int D>
struct Op {
    static constexpr int NV = D * Tr<T>::ES / 64;
    static constexpr int EV = 16 / Tr<T>::ES;  // elements per vector
    dev::u32x4 v[NV];
};

template <typename T, int D>
__device__ __forceinline__ void load_key_tile(Op<T, D>& op, const T* Khead, int key, int g) {
    const T* row = Khead + (size_t)key * D + g * Op<T, D>::EV;
#pragma unroll
    for (int v = 0; v < Op<T, D>::NV; ++v)
        op.v[v] = *reinterpret_cast<const dev::u32x4*>(row + v * 4 * Op<T, D>::EV);
}

template <typename T, int D>
__device__ __forceinline__ void load_row_tile(Op<T, D>& op, const T* lds_row, int g) {
    const T* row = lds_row + g * Op<T, D>::EV;
#pragma unroll
    for (int v = 0; v < Op<T, D>::NV; ++v)
        op.v[v] = *reinterpret_cast<const dev::u32x4*>(row + v * 4 * Op<T, D>::EV);
}

// acc += A * B over the whole head dimension; A supplies the output rows
// (lane & 15 = row within the tile), B the output columns.
__device__ __forceinline__ void mma(f32x4& acc, const Op<uint16_t, 128>& a, const Op<uint16_t, 128>& b) {
#pragma unroll
    for (int v = 0; v < 4; ++v)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v[v]),
                                                      __builtin_bit_cast(bf16x8_t, b.v[v]), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma(f32x4& acc, const Op<uint16_t, 64>& a, const Op<uint16_t, 64>& b) {
#pragma unroll
    for (int v = 0; v < 2; ++v)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v[v]),
                                                      __builtin_bit_cast(bf16x8_t, b.v[v]), acc, 0, 0, 0);
}
template <int D>
__device__ __forceinline__ void mma(f32x4& acc, const Op<float, D>& a, const Op<float, D>& b) {
#pragma unroll
    for (int v = 0; v < Op<float, D>::NV; ++v) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.v[v][e]), __uint_as_float(b.v[v][e]), acc,
                                                       0, 0, 0);
    }
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// (m, z) <- merge of two partial log2-sum-exp statistics.
__device__ __forceinline__ void merge_mz(float& m, float& z, float m2, float z2) {
    float M = fmaxf(m, m2);
    if (M == -INFINITY) return;
    float a = (m == -INFINITY) ? 0.f : z * fast_exp2(m - M);
    float b = (m2 == -INFINITY) ? 0.f : z2 * fast_exp2(m2 - M);
    z = a + b;
    m = M;
}

// Mean form: fold four log2 weights y (one key, four rows) into the key's
// running (max m, sum z of exp2(y - m)), so that no weight underflows the
// fp32 range however small all of them are; z >= 1 once m is finite.
__device__ __forceinline__ void add_weights(float& m, float& z, f32x4 y) {
    const float mnew = fmaxf(m, fmaxf(fmaxf(y[0], y[1]), fmaxf(y[2], y[3])));
    const float ms = (mnew == -INFINITY) ? 0.f : mnew;  // no row sees the key yet: z stays 0
    z = z * fast_exp2(m - ms) + ((fast_exp2(y[0] - ms) + fast_exp2(y[1] - ms)) +
                                 (fast_exp2(y[2] - ms) + fast_exp2(y[3] - ms)));
    m = mnew;
}

template <typename T>
__device__ __forceinline__ T to_elem(float f);
template <>
__device__ __forceinline__ uint16_t to_elem<uint16_t>(float f) { return dev::f32_to_bf16_rne(f); }
template <>
__device__ __forceinline__ float to_elem<float>(float f) { return f; }

// Rotate-half RoPE of one beacon pair (x, y) -> (x c - y s, y c + x s),
// each product and the sum rounded to fp32 separately: the pragma keeps
// these operations out of fused multiply-adds even after inlining.
__device__ __forceinline__ float2 rope_pair(float x, float y, float c, float s) {
#pragma clang fp contract(off)
    const float a = x * c;
    const float b = y * s;
    const float e = y * c;
    const float f = x * s;
    return make_float2(a - b, e + f);
}

// The four 16-key tiles of one 64-key group (keys past N read key N-1).
template <typename T, int D>
__device__ __forceinline__ void load_group(Op<T, D>* kop, const T* Kh, int kb, int N, int c16, int g) {
#pragma unroll
    for (int t = 0; t < 4; ++t) load_key_tile<T, D>(kop[t], Kh, min(kb + t * 16 + c16, N - 1), g);
}

template <typename T, int D>
struct alignas(16) Smem {
    T y[Tr<T>::RG * (D + Tr<T>::PAD)];
    float red_m[kWaves][Tr<T>::RG];
    float red_z[kWaves][Tr<T>::RG];
    float nlse[Tr<T>::RG];
    float best[kWaves * 64 * 4];   // F items: per-key maxima of the chunk (up to 1024 keys)
    float bests[kWaves * 64 * 4];  // F items, mean form: per-key weight sums relative to best
    int act[kMaxC];
    int nact;
};

// Occupied beacon slots of head h, ascending, into act / *nact.
__device__ __forceinline__ void active_slots(const Args& a, int h, int* act, int* nact) {
    if (threadIdx.x == 0) {
        const int32_t* cnt = a.counts + (size_t)h * a.C;  // not read when C == 0
        int n = 0;
        for (int c = 0; c < a.C; ++c)
            if (cnt[c] > 0) act[n++] = c;
        *nact = n;
    }
    __syncthreads();
}

// Observation rows [r0, r0 + nr) of head h into LDS rows of stride LD: rows
// below nact are the occupied beacons rotated to the step and rounded to the
// cache dtype, then the G*W recent queries (contiguous in q_win), then zero
// padding.
template <typename T, int D, int LD>
__device__ void build_rows(const Args& a, int h, int r0, int nr, const int* act, int nact, T* y) {
    constexpr int VPR = D * Tr<T>::ES / 16;
    const int tid = threadIdx.x;
    const int b = h / a.Hkv, kh = h % a.Hkv;
    const int R = nact + a.G * a.W;
    // beacon rows in this group
    const int bl = max(0, min(nact, r0 + nr) - r0);
    for (int idx = tid; idx < bl * (D / 2); idx += kThreads) {
        const int r = idx / (D / 2), i = idx % (D / 2);
        const float* beta = a.beacons + ((size_t)h * a.C + act[r0 + r]) * D;
        float2 p = make_float2(beta[i], beta[i + D / 2]);
        if (a.rope_cos) p = rope_pair(p.x, p.y, a.rope_cos[i], a.rope_sin[i]);
        y[r * LD + i] = to_elem<T>(p.x);
        y[r * LD + i + D / 2] = to_elem<T>(p.y);
    }
    // recent rows and padding, 16 bytes at a time
    const T* q = reinterpret_cast<const T*>(a.qwin) + ((size_t)b * a.Hq + (size_t)kh * a.G) * a.W * D;
    for (int i = tid; i < (nr - bl) * VPR; i += kThreads) {
        const int r = bl + i / VPR, v = i % VPR;
        const int gr = r0 + r;  // row index within the head
        dev::u32x4 val = {0u, 0u, 0u, 0u};
        if (gr < R) val = reinterpret_cast<const dev::u32x4*>(q + (size_t)(gr - nact) * D)[v];
        *reinterpret_cast<dev::u32x4*>(y + r * LD + v * (16 / Tr<T>::ES)) = val;
    }
}

// Fold a head's chunk statistics into lse (called by the head's last S item)
// and publish it.
__device__ void fold_and_publish(const Args& a, int h, const int* act, int nact, int* hc) {
    const int tid = threadIdx.x;
    const int R = nact + a.G * a.W;
    const size_t hb = (size_t)h * a.nch * a.R_pad_max;
    for (int r = tid; r < a.R_pad_max; r += kThreads) {
        float mm = -INFINITY, zz = 0.f;
        if (r < R) {
            // 32 chunks' statistics in flight at once (all of a 32K head):
            // these are memory round trips on the head's critical path
            for (int c0 = 0; c0 < a.nch; c0 += 32) {
                float pm[32], pz[32];
#pragma unroll
                for (int u = 0; u < 32; ++u) {
                    const size_t i = hb + (size_t)min(c0 + u, a.nch - 1) * a.R_pad_max + r;
                    pm[u] = dev::ld_coherent(a.part_m + i);
                    pz[u] = dev::ld_coherent(a.part_z + i);
                }
#pragma unroll
                for (int u = 0; u < 32; ++u)
                    if (c0 + u < a.nch) merge_mz(mm, zz, pm[u], pz[u]);
            }
        }
        // padding rows, and rows that see no key, never contribute: +inf
        // seeds their final pass at -inf
        const float l2 = (r < R && zz > 0.f) ? mm + log2f(zz) : INFINITY;
        dev::st_coherent(a.lse2 + (size_t)h * a.R_pad_max + r, l2);
        if (a.row_lse && r < R) {
            const int slot = (r < nact) ? act[r] : a.C + (r - nact);
            a.row_lse[(size_t)h * (a.C + a.G * a.W) + slot] = (zz > 0.f) ? l2 * 0.69314718055994531f : -INFINITY;
        }
    }
    if (a.row_lse) {  // empty beacon slots have no row
        const int32_t* cnt = a.counts + (size_t)h * a.C;
        for (int c = tid; c < a.C; c += kThreads)
            if (cnt[c] <= 0) a.row_lse[(size_t)h * (a.C + a.G * a.W) + c] = -INFINITY;
    }
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) dev::st_flag(hc + kHcReady, 1);
}

// Count this S item's statistics in; true for the head's last S item, which
// then folds them.
__device__ __forceinline__ bool count_stats(const Args& a, int h, int* s_flag) {
    dev::wait_all_memory();  // statistics stored before the counter moves
    __syncthreads();
    int* hc = a.hctl + (size_t)h * kHcWords;
    if (threadIdx.x == 0) *s_flag = (dev::fetch_add_relaxed(hc + kHcP1Count, 1) == a.nch - 1);
    __syncthreads();
    return *s_flag != 0;
}

// Block until the head's lse is published (one thread waits, then all).
__device__ __forceinline__ bool await_lse(const Args& a, int h, int* s_flag) {
    if (threadIdx.x == 0) {
        *s_flag = dev::wait_flag(a.hctl + (size_t)h * kHcWords + kHcReady);
        if (!*s_flag) dev::raise_error(a.hdr, kErrScoreWait);
    }
    __syncthreads();
    return *s_flag != 0;
}

// ---- S(h, chunk): row statistics over one key chunk -------------------------
//
// Wave w takes keys [kw, kw + 64*KGN) in groups of 64 (four 16-key tiles).
// MFMA rows are keys and columns observation rows, so a lane owns one row
// (lane & 15 within the tile) and 16 keys of each group.  (key, row) pairs
// outside the mask (keys at or past N, the causal window) enter with the
// accumulator seeded at -inf, so they add exp2(-inf) = 0.
template <typename T, int D, int KGN>
__device__ void stats_item(const Args& a, int h, int chunk, Smem<T, D>& sm, int* s_flag) {
    constexpr int RG = Tr<T>::RG, LD = D + Tr<T>::PAD, RTM = RG / 16;
    constexpr int KC = kWaves * 64 * KGN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    active_slots(a, h, sm.act, &sm.nact);
    const int nact = sm.nact;
    const int R = nact + a.G * a.W;
    const int Rp = (R + 15) & ~15;
    const T* Kh = reinterpret_cast<const T*>(a.K) + (size_t)h * a.N_cap * D;
    const int kw = chunk * KC + wave * 64 * KGN;  // this wave's first key
    const int N = a.N;
    const float s2 = a.s2;
    const size_t pbase = ((size_t)h * a.nch + chunk) * a.R_pad_max;
    const KeyMask mk = key_mask(a, nact);

    for (int r0 = 0; r0 < Rp; r0 += RG) {
        const int nr = min(RG, Rp - r0), RT = nr / 16;
        __syncthreads();
        build_rows<T, D, LD>(a, h, r0, nr, sm.act, nact, sm.y);
        __syncthreads();
        float m[RTM], z[RTM];
#pragma unroll
        for (int i = 0; i < RTM; ++i) {
            m[i] = -INFINITY;
            z[i] = 0.f;
        }
        const int ngroups = max(0, min(KGN, (N - kw + 63) / 64));
#pragma unroll 1
        for (int kg = 0; kg < ngroups; ++kg) {
            const int kb = kw + kg * 64;
            Op<T, D> kop[4];
            load_group<T, D>(kop, Kh, kb, N, c16, g);
            const bool masked = kb + 64 > mk.all_see_below();  // some (key, row) pair is out
#pragma unroll
            for (int rt = 0; rt < RTM; ++rt) {
                if (rt < RT) {
                    Op<T, D> yop;
                    load_row_tile<T, D>(yop, sm.y + (rt * 16 + c16) * LD, g);
                    // 0, or -inf for keys this lane's row does not see
                    const int lim = masked ? mk.limit(r0 + rt * 16 + c16) : N;
                    f32x4 acc[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
#pragma unroll
                        for (int v = 0; v < 4; ++v) acc[t][v] = (kb + t * 16 + 4 * g + v <= lim) ? 0.f : -INFINITY;
                        mma(acc[t], kop[t], yop);  // rows = keys, columns = observation rows
                    }
                    float gm = fmaxf(fmaxf(acc[0][0], acc[0][1]), fmaxf(acc[0][2], acc[0][3]));
#pragma unroll
                    for (int t = 1; t < 4; ++t)
                        gm = fmaxf(gm, fmaxf(fmaxf(acc[t][0], acc[t][1]), fmaxf(acc[t][2], acc[t][3])));
                    const float mnew = fmaxf(m[rt], gm * s2);
                    // a lane may see no valid key yet: keep its sums at 0, not NaN
                    const float ms = (mnew == -INFINITY) ? 0.f : mnew;
                    float zz = z[rt] * fast_exp2(m[rt] - ms);
#pragma unroll
                    for (int t = 0; t < 4; ++t)
#pragma unroll
                        for (int v = 0; v < 4; ++v) zz += fast_exp2(__builtin_fmaf(acc[t][v], s2, -ms));
                    z[rt] = zz;
                    m[rt] = mnew;
                }
            }
        }
        // lanes sharing a row: g = 0..3 (lane bits 4, 5)
#pragma unroll
        for (int rt = 0; rt < RTM; ++rt) {
            if (rt < RT) {
                merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 16), dev::shfl_xor_f(z[rt], 16));
                merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 32), dev::shfl_xor_f(z[rt], 32));
                if (g == 0) {
                    sm.red_m[wave][rt * 16 + c16] = m[rt];
                    sm.red_z[wave][rt * 16 + c16] = z[rt];
                }
            }
        }
        __syncthreads();
        for (int r = tid; r < nr; r += kThreads) {
            float mm = sm.red_m[0][r], zz = sm.red_z[0][r];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) merge_mz(mm, zz, sm.red_m[w][r], sm.red_z[w][r]);
            dev::st_coherent(a.part_m + pbase + r0 + r, mm);
            dev::st_coherent(a.part_z + pbase + r0 + r, zz);
        }
    }
    if (count_stats(a, h, s_flag)) fold_and_publish(a, h, sm.act, nact, a.hctl + (size_t)h * kHcWords);
}

// ---- F(h, chunk): final scores over one key chunk ----------------------
//
// MFMA rows are observation rows and columns keys; the accumulator starts at
// -lse2_r / s2, so each output is (l_rj - lse_r) / (s2 ln 2) and a key's
// score is the max down its column (or, for the mean, the log of the mean
// of the weights exp2(s2 * output)).  Per-key maxima (sums) collect in LDS
// across row groups and are written out coalesced at the end.
template <typename T, int D, int KGN>
__device__ void final_item(const Args& a, int h, int chunk, Smem<T, D>& sm, int* s_flag) {
    constexpr int RG = Tr<T>::RG, LD = D + Tr<T>::PAD, RTM = RG / 16;
    constexpr int KC = kWaves * 64 * KGN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    if (!await_lse(a, h, s_flag)) return;
    active_slots(a, h, sm.act, &sm.nact);
    const int R = sm.nact + a.G * a.W;
    const int Rp = (R + 15) & ~15;
    const T* Kh = reinterpret_cast<const T*>(a.K) + (size_t)h * a.N_cap * D;
    const int k0 = chunk * KC;
    const int kw = k0 + wave * 64 * KGN;
    const int N = a.N;
    const float inv_s2 = 1.0f / a.s2, s2 = a.s2;
    const KeyMask mk = key_mask(a, sm.nact);
    const bool mean = a.mean != 0;
    for (int i = tid; i < KC; i += kThreads) {
        sm.best[i] = -INFINITY;
        sm.bests[i] = 0.f;
    }
    const int ngroups = max(0, min(KGN, (N - kw + 63) / 64));

    for (int r0 = 0; r0 < Rp; r0 += RG) {
        const int nr = min(RG, Rp - r0), RT = nr / 16;
        __syncthreads();
        build_rows<T, D, LD>(a, h, r0, nr, sm.act, sm.nact, sm.y);
        for (int r = tid; r < nr; r += kThreads)
            sm.nlse[r] = -dev::ld_coherent(a.lse2 + (size_t)h * a.R_pad_max + r0 + r) * inv_s2;
        __syncthreads();
#pragma unroll 1
        for (int kg = 0; kg < ngroups; ++kg) {
            const int kb = kw + kg * 64;
            Op<T, D> kop[4];
            load_group<T, D>(kop, Kh, kb, N, c16, g);
            const bool masked = kb + 64 > mk.all_see_below();
            // per key of this lane: the max over rows of acc * s2 (log2 of the
            // weight) and, for the mean, the sum of the weights relative to it
            float best[4], bsum[4];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                best[t] = -INFINITY;
                bsum[t] = 0.f;
            }
#pragma unroll
            for (int rt = 0; rt < RTM; ++rt) {
                if (rt < RT) {
                    Op<T, D> yop;
                    load_row_tile<T, D>(yop, sm.y + (rt * 16 + c16) * LD, g);
                    const f32x4 c0 = *reinterpret_cast<const f32x4*>(sm.nlse + rt * 16 + 4 * g);
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        f32x4 acc = c0;
                        if (masked) {  // (key, row) pairs outside the mask start at -inf
                            const int key = kb + t * 16 + c16;
#pragma unroll
                            for (int v = 0; v < 4; ++v)
                                if (key > mk.limit(r0 + rt * 16 + 4 * g + v)) acc[v] = -INFINITY;
                        }
                        mma(acc, yop, kop[t]);  // rows = observation rows, columns = keys
                        if (mean)
                            add_weights(best[t], bsum[t], acc * s2);
                        else
                            best[t] = fmaxf(best[t], fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
                    }
                }
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                float b = best[t];
                float* slot = sm.best + (kb - k0) + t * 16 + c16;  // this wave's own keys
                if (mean) {
                    float bs = bsum[t];
                    merge_mz(b, bs, dev::shfl_xor_f(b, 16), dev::shfl_xor_f(bs, 16));
                    merge_mz(b, bs, dev::shfl_xor_f(b, 32), dev::shfl_xor_f(bs, 32));
                    if (g == t) merge_mz(*slot, sm.bests[slot - sm.best], b, bs);
                } else {
                    b = fmaxf(b, dev::shfl_xor_f(b, 16));
                    b = fmaxf(b, dev::shfl_xor_f(b, 32));
                    if (g == t) *slot = fmaxf(*slot, b);
                }
            }
        }
    }
    __syncthreads();
    float* out = a.scores + (size_t)h * N;
    const float log2R = log2f((float)R);
    for (int i = tid; i < KC; i += kThreads)
        if (k0 + i < N)
            out[k0 + i] = mean ? (sm.best[i] + log2f(sm.bests[i]) - log2R) * 0.69314718055994531f
                               : sm.best[i] * a.s2ln2;
}

// Workgroup -> head.  The grid lists, for s = 0, 1, ..., nch workgroups of
// head s (if s < P) and then nch workgroups of head s - lag (if s >= lag),
// so each head's second half starts about `lag` heads after its first.
__device__ __forceinline__ int head_of_block(const Args& a, int b) {
    const int P = a.P, nch = a.nch, L = a.lag;
    if (b < L * nch) return b / nch;
    b -= L * nch;
    if (b < (P - L) * 2 * nch) {
        const int s = L + b / (2 * nch);
        return (b % (2 * nch) < nch) ? s : s - L;
    }
    b -= (P - L) * 2 * nch;
    return P - L + b / nch;
}

// ---- work-item protocol shared by both paths --------------------------------
// Take the next work ticket of head h (tickets below nch are S items, the
// rest F items); false if the workspace stamp or control line is bad.  The
// request is issued first and completed separately, so that loads issued in
// between (the fast path's rows) are in flight while the atomic returns; the
// ticket is taken before the stamp is known, which only matters when the
// item then does nothing and reports the bad stamp.
struct TicketReq {
    int t;
    dev::u32x4 hdr;  // magic, P, budget, error bits
};
__device__ __forceinline__ TicketReq request_ticket(const Args& a, int h) {
    TicketReq r{0, {0u, 0u, 0u, 0u}};
    if (threadIdx.x == 0) {
        r.t = dev::fetch_add_relaxed(a.hctl + (size_t)h * kHcWords + kHcScTicket, 1);
        r.hdr = *reinterpret_cast<const dev::u32x4*>(a.hdr);  // one load, checked on completion
    }
    return r;
}
__device__ __forceinline__ bool complete_ticket(const Args& a, const TicketReq& r, int* s_ticket, int* s_ok) {
    if (threadIdx.x == 0) {
        int ok = r.hdr[kHdrMagic] == kWsMagic && (int)r.hdr[kHdrP] == a.P && (int)r.hdr[kHdrBudget] == a.budget;
        *s_ticket = r.t;
        if (ok && r.t >= a.tickets) ok = 0;  // control line was not clear: do nothing
        if (!ok) dev::raise_error(a.hdr, kErrStamp);
        *s_ok = ok;
    }
    __syncthreads();
    return *s_ok != 0;
}

// Clear head h's score control words (thread 0).  Every score launch does
// this for all heads in a kernel of its own, before any work item takes a
// ticket, so work items never wait at the end to find the head's last one.
__device__ __forceinline__ void reset_head_control(const Args& a, int h) {
    int* hc = a.hctl + (size_t)h * kHcWords;
    if (threadIdx.x == 0) {
        dev::st_flag(hc + kHcScTicket, 0);
        dev::st_flag(hc + kHcP1Count, 0);
        dev::st_flag(hc + kHcReady, 0);
        if (a.fused) {
            dev::st_flag(hc + kHcFcDone, 0);
            dev::st_flag(hc + kHcFDone, 0);
            dev::st_flag(hc + kHcScReady, 0);
            dev::st_flag(hc + kHcKept, 0);
        }
    }
    if (a.fused)
        for (int i = threadIdx.x; i < a.nsegF; i += blockDim.x) dev::st_flag(a.cflags + (size_t)h * a.nseg_cap + i, 0);
}

__global__ void reset_control_kernel(Args a) {
    const int h = blockIdx.x * blockDim.x + threadIdx.x;
    if (h < a.P) {
        int* hc = a.hctl + (size_t)h * kHcWords;
        dev::st_flag(hc + kHcScTicket, 0);
        dev::st_flag(hc + kHcP1Count, 0);
        dev::st_flag(hc + kHcReady, 0);
    }
}

template <typename T, int D, int KGN>
__global__ __launch_bounds__(kThreads, 2) void score_kernel(Args a) {
    __shared__ Smem<T, D> sm;
    __shared__ int s_ticket, s_ok, s_flag;
    const int h = head_of_block(a, blockIdx.x);
    if (!complete_ticket(a, request_ticket(a, h), &s_ticket, &s_ok)) return;
    if (s_ticket < a.nch)
        stats_item<T, D, KGN>(a, h, s_ticket, sm, &s_flag);
    else
        final_item<T, D, KGN>(a, h, s_ticket - a.nch, sm, &s_flag);
}

// ---- fast path: bf16 cache, rows in groups of at most 144 ------------------
//
// A small kernel first writes each head's observation rows to the workspace
// in MFMA operand order, so that a work item loads them straight into
// registers with coalesced 16-byte loads.  When all rows fit in one group of
// at most 144 (9 tiles) they are loaded before the item's ticket returns and
// stay in registers for the whole item.  Wider heads (up to 8 groups) split
// the rows into equal groups: an item takes them one after the other,
// streaming its key chunk again for each (from L2 or the memory-side cache);
// S items store each group's row statistics, F items keep each key's max
// (or sum) over the groups so far in LDS and write it after the last.  Key tiles are staged through
// LDS with coalesced global_load_lds_dwordx4 (direct to LDS, no registers),
// double-buffered per wave so the next group of 32 keys is in flight while
// this one is computed; a 16-lane ds_read_b128 of a staged tile is
// conflict-free thanks to an XOR swizzle of the 16-byte chunks of each key
// row.
//
// The two stages are distinct __shared__ variables and the key loop is
// unrolled by two, so every LDS read names one stage; the compiler then
// waits only for the loads into that stage, not for the group in flight
// into the other one.
constexpr int kFRT = kFastTiles;  // at most this many 16-row tiles per row group
constexpr int kFKG = 32;  // keys per group: two 16-key tiles

template <int D>
struct KeyStage {
    static constexpr int CPR = D * 2 / 16;       // 16-byte chunks per key row
    static constexpr int RPI = 64 / CPR;         // key rows per load instruction
    static constexpr int NI = kFKG / RPI;        // load instructions per group
    static constexpr int ELEMS = kFKG * D;       // bf16 elements per group
    // chunk position of logical chunk c of row r is c ^ swz(r)
    __device__ static int swz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
};

template <int D>
struct alignas(16) StageBuf {
    uint16_t k[kWaves][KeyStage<D>::ELEMS];
};

constexpr int kMaxKeyChunk = 1024;  // keys per work item at most

struct alignas(16) FastSmem {
    union {
        struct {
            float m[kWaves][kFRT * 16];
            float z[kWaves][kFRT * 16];
        } red;  // S items: per-wave row statistics
        struct {
            float nlse[kFRT * 16];      // -lse of each row (raw-dot units)
            float kacc[kMaxKeyChunk];   // each key's result (with several row groups: so far)
            float kaccs[kMaxKeyChunk];  // mean form, several row groups: each key's weight sum so far
        } fin;  // F items
    } v;
    int lim[kFRT * 16];  // last key each row sees (KeyMask::limit)
};

// Each row's key limit into LDS (rows r0 .. r0 + 16 RT - 1), for the groups
// that mask (key, row) pairs.
template <int RT>
__device__ __forceinline__ void fill_limits(const KeyMask& mk, int r0, int* lim) {
    for (int r = threadIdx.x; r < RT * 16; r += kThreads) lim[r] = mk.limit(r0 + r);
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Rows of head h into the workspace: row tile rt, vector v, lane l holds the
// 16 bytes lane l presents to the MFMA, i.e. chunk 4 v + l / 16 of row
// 16 rt + l % 16; plus the head's occupied-slot list.
template <int D>
__global__ __launch_bounds__(kThreads) void rows_kernel(Args a) {
    constexpr int LD = D + 8, NV = Op<uint16_t, D>::NV;
    __shared__ uint16_t y[kFRT * 16 * LD];
    __shared__ int act[kMaxC];
    __shared__ int nact;
    const int h = blockIdx.x, tid = threadIdx.x;
    reset_head_control(a, h);
    active_slots(a, h, act, &nact);
    // up to 144 rows at a time through LDS
    for (int r0 = 0; r0 < a.R_pad_max; r0 += kFRT * 16) {
        const int nr = min(kFRT * 16, a.R_pad_max - r0);
        build_rows<uint16_t, D, LD>(a, h, r0, nr, act, nact, y);
        __syncthreads();
        dev::u32x4* out = reinterpret_cast<dev::u32x4*>(a.rows) + ((size_t)h * a.R_pad_max + r0) * D / 8;
        const int n = nr / 16 * NV * 64;
        for (int i = tid; i < n; i += kThreads) {
            const int lane = i & 63, v = (i >> 6) % NV, rt = (i >> 6) / NV;
            out[i] = *reinterpret_cast<const dev::u32x4*>(y + (rt * 16 + (lane & 15)) * LD + (4 * v + (lane >> 4)) * 8);
        }
        __syncthreads();
    }
    int* meta = a.rmeta + (size_t)h * kMetaWords;
    if (tid == 0) meta[0] = nact;
    for (int c = tid; c < nact; c += kThreads) meta[kMetaAct + c] = act[c];
}

// Row group rg (rows 16 RT rg .. 16 RT (rg + 1) - 1) of head h into registers.
template <int D, int RT>
__device__ __forceinline__ void load_rows(const Args& a, int h, int rg, Op<uint16_t, D>* yr, int lane) {
    constexpr int NV = Op<uint16_t, D>::NV;
    const dev::u32x4* src =
        reinterpret_cast<const dev::u32x4*>(a.rows) + ((size_t)h * a.R_pad_max + (size_t)rg * RT * 16) * D / 8 + lane;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int v = 0; v < NV; ++v) yr[rt].v[v] = src[(rt * NV + v) * 64];
}

// Byte offset, within a group, of what lane `lane` loads with instruction
// j: load instruction j writes 1 KB contiguous at stage + 1 KB * j, lane
// l's 16 bytes at offset 16 l, which is key row r = j*RPI + l / CPR at
// swizzled position l % CPR, holding logical chunk (l % CPR) ^ swz(r).
// Each group of CPR lanes reads one whole key row.
template <int D>
__device__ __forceinline__ int group_offset(int j, int lane) {
    using KS = KeyStage<D>;
    const int r = j * KS::RPI + lane / KS::CPR;
    return r * D * 2 + (((lane % KS::CPR) ^ KS::swz(r)) * 16);
}

// Start loading keys [kb, kb + 32) of the head into a wave's stage.  The
// buffer resource covers keys [kb, min(N, kb + 32)) only, so rows past N
// read as zero.  AUX is the load's cache policy: F items, the last readers
// of their keys, load them non-temporal (2), which measured about 2 %
// faster on the 32K layer than the default policy.
template <int D, int AUX = 0>
__device__ __forceinline__ void issue_group(const uint16_t* Kh, int kb, int N, uint16_t* stage, int lane) {
#if defined(__HIP_DEVICE_COMPILE__)  // buffer resources exist in device code only
    using KS = KeyStage<D>;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)(Kh + (size_t)kb * D), (short)0, min(N - kb, kFKG) * D * 2, 0x00020000);
    // the offsets are recomputed at every issue: hoisted out of the key
    // loop they would hold NI registers for the whole item
    int l = lane;
    asm volatile("" : "+v"(l));
#pragma unroll
    for (int j = 0; j < KS::NI; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)(stage + j * 512),
                                                 16, group_offset<D>(j, l), 0, 0, AUX);
#endif
}

// MFMA operand of staged key tile t for lane (c16, g): vector v holds
// logical chunk 4 v + g of key row 16 t + c16.
template <int D>
__device__ __forceinline__ void read_key_tile(Op<uint16_t, D>& op, const uint16_t* stage, int t, int c16, int g) {
    using KS = KeyStage<D>;
    const int r = t * 16 + c16;
    const uint16_t* row = stage + r * D;
#pragma unroll
    for (int v = 0; v < Op<uint16_t, D>::NV; ++v)
        op.v[v] = *reinterpret_cast<const dev::u32x4*>(row + ((4 * v + g) ^ KS::swz(r)) * 8);
}

// Running (max, sum) of one S item over one staged group of 32 keys.
// In groups holding keys some row may not see (TAIL: keys at or past N, or
// the causal window) those (key, row) pairs enter with the accumulator
// seeded at -inf, so they add exp2(-inf) = 0.
//
// Software-pipelined by one row tile: the MFMAs of tile rt + 1 are issued
// in the same scheduling region as the exp/max work on tile rt and
// interleaved with it (one MFMA, then four VALU instructions), so the
// matrix core is not left idle while the wave waits on its results.  Only
// two tiles of accumulators are live at a time; hoisting more would spill
// the registers that hold the rows.
template <int D, int RT, bool TAIL>
__device__ __forceinline__ void stats_group(const uint16_t* st, int kb, const int* lim, const Op<uint16_t, D>* yr,
                                            float s2, float* m, float* z, int c16, int g) {
    Op<uint16_t, D> kop[2];
    read_key_tile<D>(kop[0], st, 0, c16, g);
    read_key_tile<D>(kop[1], st, 1, c16, g);
    f32x4 acc[2][2];
    auto issue = [&](int rt, f32x4* a) {
        const int l = TAIL ? lim[rt * 16 + c16] : 0;  // this lane's row
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int v = 0; v < 4; ++v) a[t][v] = (!TAIL || kb + t * 16 + 4 * g + v <= l) ? 0.f : -INFINITY;
            mma(a[t], kop[t], yr[rt]);  // rows = keys, columns = observation rows
        }
    };
    issue(0, acc[0]);
    dev::static_for<RT>([&](auto rt) {
        if constexpr (rt + 1 < RT) issue(rt + 1, acc[(rt + 1) & 1]);
        f32x4* a = acc[rt & 1];
        const float gm = fmaxf(fmaxf(fmaxf(a[0][0], a[0][1]), fmaxf(a[0][2], a[0][3])),
                               fmaxf(fmaxf(a[1][0], a[1][1]), fmaxf(a[1][2], a[1][3])));
        const float mnew = fmaxf(m[rt], gm * s2);
        const float ms = (mnew == -INFINITY) ? 0.f : mnew;  // no valid key yet: sums stay 0
        float zz = z[rt] * fast_exp2(m[rt] - ms);
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) zz += fast_exp2(__builtin_fmaf(a[t][v], s2, -ms));
        z[rt] = zz;
        m[rt] = mnew;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // four VALU
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// The same statistics with each lane's offset fixed: after an item's first
// group every lane holds a finite offset per row tile (fix_offsets), and
// later groups only add exp2(y - offset).  A later key more than 127 (log2
// units) above the offset overflows the sum to +inf; the item then redoes
// its statistics with the running max.  Two VALU instructions and one exp2
// per (row, key) instead of about four and a bit.
// Offsets of the fixed-offset statistics, taken after an item's first
// group: per row, the largest logit (log2 units) any of the row's four lanes
// has seen in that group, plus a margin of 64, or 0 for a row that has seen
// no key; each lane's sum so far is rescaled to it.  The margin lets later
// keys lie up to 191 above the first group's maximum before a sum overflows
// (keys far above the first ones are common where queries revisit a few
// keys); it costs nothing in precision: the sums stay above 2^-64, and a term
// that flushes to zero lies more than 62 below the row's maximum.
constexpr float kOffsetMargin = 64.f;

// A lane's statistics before they are merged: the sum's binary exponent
// moves into the offset, so z lies in [0.5, 1) and m is within one of the
// lane's log2-sum.  A sum taken against a fixed offset can be as large as
// 2^127, and merges scale sums by exp2(m - M): without this, a chunk whose
// offset lies more than 126 below another chunk's would lose its sum to a
// factor that underflows, however large the sum.  A lane that saw no key
// (z = 0) gets m = -inf.
__device__ __forceinline__ void normalise_mz(float& m, float& z) {
    if (z == 0.f) {
        m = -INFINITY;
        return;
    }
    int e;
    z = frexpf(z, &e);
    m += (float)e;
}

template <int RT>
__device__ __forceinline__ void fix_offsets(float* m, float* z, float* nms) {
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        float mr = fmaxf(m[i], dev::shfl_xor_f(m[i], 16));
        mr = fmaxf(mr, dev::shfl_xor_f(mr, 32));
        const float off = (mr == -INFINITY) ? 0.f : mr + kOffsetMargin;
        z[i] *= fast_exp2(m[i] - off);  // m = -inf: the sum is 0 and stays 0
        m[i] = off;
        nms[i] = -off;
    }
}

template <int D, int RT, bool TAIL>
__device__ __forceinline__ void stats_group_fixed(const uint16_t* st, int kb, const int* lim,
                                                  const Op<uint16_t, D>* yr, float s2, const float* nms, float* z,
                                                  int c16, int g) {
    Op<uint16_t, D> kop[2];
    read_key_tile<D>(kop[0], st, 0, c16, g);
    read_key_tile<D>(kop[1], st, 1, c16, g);
    f32x4 acc[2][2];
    auto issue = [&](int rt, f32x4* a) {
        const int l = TAIL ? lim[rt * 16 + c16] : 0;  // this lane's row
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int v = 0; v < 4; ++v) a[t][v] = (!TAIL || kb + t * 16 + 4 * g + v <= l) ? 0.f : -INFINITY;
            mma(a[t], kop[t], yr[rt]);  // rows = keys, columns = observation rows
        }
    };
    issue(0, acc[0]);
    dev::static_for<RT>([&](auto rt) {
        if constexpr (rt + 1 < RT) issue(rt + 1, acc[(rt + 1) & 1]);
        f32x4* a = acc[rt & 1];
        const float nm = nms[rt];
        float e[8];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) e[4 * t + v] = fast_exp2(__builtin_fmaf(a[t][v], s2, nm));
        z[rt] += ((e[0] + e[1]) + (e[2] + e[3])) + ((e[4] + e[5]) + (e[6] + e[7]));
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);  // three VALU
        }
        __builtin_amdgcn_sched_barrier(0);
    });
}

// Scores of one F item's staged group of 32 keys: per key the maximum over
// rows (or the log of the mean weight), written straight out (64 contiguous
// bytes per 16-key tile).  TAIL groups mask (key, row) pairs as in S.
// Pipelined like stats_group; each tile's -lse seed is read from LDS two
// tiles ahead (re-read every group through an offset the compiler cannot
// hoist: kept for the whole item these would hold 4 * RT registers).
// Row-group phase of an F item: its only group, or the first, a middle or
// the last of several (then each key's result is combined in kacc).
enum RowPhase : int { kOnlyGroup = 0, kFirstGroup = 1, kMidGroup = 2, kLastGroup = 3 };

template <int D, int RT, bool MEAN, bool TAIL>
__device__ __forceinline__ void final_group(const uint16_t* st, int kb, int N, const int* lim, const Op<uint16_t, D>* yr,
                                            const float* nlse, float* out, float s2, float log2R, int c16, int g,
                                            int phase, float* kacc, float* kaccs, int k0) {
    Op<uint16_t, D> kop[2];
    read_key_tile<D>(kop[0], st, 0, c16, g);
    read_key_tile<D>(kop[1], st, 1, c16, g);
    // per key of this lane: max over rows of (l - lse) / s2; for the mean,
    // the max of the log2 weights s2 * acc and the weights' sum relative to it
    float best[2] = {-INFINITY, -INFINITY};
    float bsum[2] = {0.f, 0.f};
    f32x4 acc[2][2];
    f32x4 cn[2];
    auto load_c = [&](int rt) {
        int off = rt * 16 + 4 * g;
        asm volatile("" : "+v"(off));
        return *reinterpret_cast<const f32x4*>(nlse + off);
    };
    auto accumulate = [&](const f32x4* a) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            if constexpr (MEAN)
                add_weights(best[t], bsum[t], a[t] * s2);
            else
                best[t] = fmaxf(best[t], fmaxf(fmaxf(a[t][0], a[t][1]), fmaxf(a[t][2], a[t][3])));
        }
    };
    if constexpr (TAIL) {
        // a head's last groups only: one row tile at a time, (key, row)
        // pairs outside the mask seeded at -inf
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 c0 = load_c(rt);
            const int4 l4 = *reinterpret_cast<const int4*>(lim + rt * 16 + 4 * g);
            f32x4* a = acc[0];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int key = kb + t * 16 + c16;
                a[t][0] = key > l4.x ? -INFINITY : c0[0];
                a[t][1] = key > l4.y ? -INFINITY : c0[1];
                a[t][2] = key > l4.z ? -INFINITY : c0[2];
                a[t][3] = key > l4.w ? -INFINITY : c0[3];
                mma(a[t], yr[rt], kop[t]);  // rows = observation rows, columns = keys
            }
            accumulate(a);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
    auto issue = [&](int rt, f32x4* a, const f32x4& c0) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            a[t] = c0;
            mma(a[t], yr[rt], kop[t]);  // rows = observation rows, columns = keys
        }
    };
    cn[0] = load_c(0);
    if constexpr (RT > 1) cn[1] = load_c(1);
    issue(0, acc[0], cn[0]);
    dev::static_for<RT>([&](auto rt) {
        if constexpr (rt + 2 < RT) cn[rt & 1] = load_c(rt + 2);
        if constexpr (rt + 1 < RT) issue(rt + 1, acc[(rt + 1) & 1], cn[(rt + 1) & 1]);
        accumulate(acc[rt & 1]);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x002, MEAN ? 6 : 1, 0);  // VALU
        }
        __builtin_amdgcn_sched_barrier(0);
    });
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        float b = best[t], bs = bsum[t];
        if constexpr (MEAN) {
            merge_mz(b, bs, dev::shfl_xor_f(b, 16), dev::shfl_xor_f(bs, 16));
            merge_mz(b, bs, dev::shfl_xor_f(b, 32), dev::shfl_xor_f(bs, 32));
        } else {
            b = fmaxf(b, dev::shfl_xor_f(b, 16));
            b = fmaxf(b, dev::shfl_xor_f(b, 32));
        }
        const int key = kb + t * 16 + c16;
        if (g == t && key < N) {
            // several row groups: the key's (max, sum) or max so far, kept by this lane
            if (phase == kMidGroup || phase == kLastGroup) {
                if constexpr (MEAN)
                    merge_mz(b, bs, kacc[key - k0], kaccs[key - k0]);
                else
                    b = fmaxf(b, kacc[key - k0]);
            }
            if (phase == kOnlyGroup || phase == kLastGroup) {
                if constexpr (MEAN)
                    b = (b + log2f(bs) - log2R) * 0.69314718055994531f;  // ln of the mean weight
                else
                    b *= s2 * 0.69314718055994531f;
            } else if constexpr (MEAN) {
                kaccs[key - k0] = bs;
            }
            // the item's scores are stored after its key loop: a store here
            // would count in vmcnt, and the next group's wait would wait for it
            kacc[key - k0] = b;
        }
    }
}

// Row split (below): each wave holds one row group and takes every key of
// the item, so a key's maximum over the head's rows meets across the four
// waves; this body folds the wave's maximum into kmax[key - k0] (order
// keys, atomic max).  Max form only.
template <int D, int RT, bool TAIL>
__device__ __forceinline__ void final_group_split(const uint16_t* st, int kb, int N, const int* lim,
                                                  const Op<uint16_t, D>* yr, const float* nlse, int c16, int g,
                                                  unsigned* kmax, int k0) {
    Op<uint16_t, D> kop[2];
    read_key_tile<D>(kop[0], st, 0, c16, g);
    read_key_tile<D>(kop[1], st, 1, c16, g);
    float best[2] = {-INFINITY, -INFINITY};
    f32x4 acc[2][2];
    auto load_c = [&](int rt) {
        int off = rt * 16 + 4 * g;
        asm volatile("" : "+v"(off));
        return *reinterpret_cast<const f32x4*>(nlse + off);
    };
    auto accumulate = [&](const f32x4* a) {
#pragma unroll
        for (int t = 0; t < 2; ++t) best[t] = fmaxf(best[t], fmaxf(fmaxf(a[t][0], a[t][1]), fmaxf(a[t][2], a[t][3])));
    };
    if constexpr (TAIL) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            const f32x4 c0 = load_c(rt);
            const int4 l4 = *reinterpret_cast<const int4*>(lim + rt * 16 + 4 * g);
            f32x4* a = acc[0];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int key = kb + t * 16 + c16;
                a[t][0] = key > l4.x ? -INFINITY : c0[0];
                a[t][1] = key > l4.y ? -INFINITY : c0[1];
                a[t][2] = key > l4.z ? -INFINITY : c0[2];
                a[t][3] = key > l4.w ? -INFINITY : c0[3];
                mma(a[t], yr[rt], kop[t]);
            }
            accumulate(a);
            __builtin_amdgcn_sched_barrier(0);
        }
    } else {
        f32x4 cn[2];
        auto issue = [&](int rt, f32x4* a, const f32x4& c0) {
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                a[t] = c0;
                mma(a[t], yr[rt], kop[t]);
            }
        };
        cn[0] = load_c(0);
        if constexpr (RT > 1) cn[1] = load_c(1);
        issue(0, acc[0], cn[0]);
        dev::static_for<RT>([&](auto rt) {
            if constexpr (rt + 2 < RT) cn[rt & 1] = load_c(rt + 2);
            if constexpr (rt + 1 < RT) issue(rt + 1, acc[(rt + 1) & 1], cn[(rt + 1) & 1]);
            accumulate(acc[rt & 1]);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        });
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        float b = best[t];
        b = fmaxf(b, dev::shfl_xor_f(b, 16));
        b = fmaxf(b, dev::shfl_xor_f(b, 32));
        const int key = kb + t * 16 + c16;
        if (g == t && key < N) atomicMax(kmax + (key - k0), dev::ord_key(b));
    }
}

// Wait until the group read next has landed in this wave's stage; `more`
// says whether the following group is still in flight behind it.
template <int D>
__device__ __forceinline__ void wait_group(bool more) {
    if (more)
        wait_vmem<KeyStage<D>::NI>();
    else
        wait_vmem<0>();
}

// MULTI: the rows come in several row groups, each loaded here (else the
// item's only group was loaded with its ticket).
template <int D, int RT, bool MULTI>
__device__ __forceinline__ void fast_stats(const Args& a, int h, int chunk, FastSmem& sm, StageBuf<D>& sa, StageBuf<D>& sb,
                           Op<uint16_t, D>* yr, int* s_flag) {
    const int KC = a.key_chunk, KPW = KC / kWaves, GPW = KPW / kFKG;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const uint16_t* Kh = reinterpret_cast<const uint16_t*>(a.K) + (size_t)h * a.N_cap * D;
    const int N = a.N;
    const int kw = chunk * KC + wave * KPW;
    const int ngroups = max(0, min(GPW, (N - kw + kFKG - 1) / kFKG));
    uint16_t* stA = sa.k[wave];
    uint16_t* stB = sb.k[wave];
    if (!MULTI) {
        if (ngroups > 0) issue_group<D>(Kh, kw, N, stA, lane);
        if (ngroups > 1) issue_group<D>(Kh, kw + kFKG, N, stB, lane);
    }
    const float s2 = a.s2;
    const KeyMask mk = key_mask(a, a.rmeta[(size_t)h * kMetaWords]);
    const int clear_below = mk.all_see_below();
    const size_t pbase = ((size_t)h * a.nch + chunk) * a.R_pad_max;
    // Rows in groups of 16 RT; the chunk's keys are streamed again for every
    // further group.
    const int nrg = MULTI ? a.R_pad_max / (RT * 16) : 1;
    for (int rg = 0; rg < nrg; ++rg) {
        if (MULTI) {
            load_rows<D, RT>(a, h, rg, yr, lane);
            if (ngroups > 0) issue_group<D>(Kh, kw, N, stA, lane);
            if (ngroups > 1) issue_group<D>(Kh, kw + kFKG, N, stB, lane);
        }
        fill_limits<RT>(mk, rg * RT * 16, sm.lim);
        __syncthreads();
        float m[RT], z[RT], nms[RT];
#pragma unroll
        for (int i = 0; i < RT; ++i) {
            m[i] = -INFINITY;
            z[i] = 0.f;
        }
        // the first group keeps a running max and fixes each lane's offset;
        // the others add exp2(y - offset) only
        auto fixed_body = [&](const uint16_t* st, int kb) {
            if (kb + kFKG <= clear_below)
                stats_group_fixed<D, RT, false>(st, kb, sm.lim, yr, s2, nms, z, c16, g);
            else
                stats_group_fixed<D, RT, true>(st, kb, sm.lim, yr, s2, nms, z, c16, g);
        };
        auto running_body = [&](const uint16_t* st, int kb) {
            if (kb + kFKG <= clear_below)
                stats_group<D, RT, false>(st, kb, sm.lim, yr, s2, m, z, c16, g);
            else
                stats_group<D, RT, true>(st, kb, sm.lim, yr, s2, m, z, c16, g);
        };
#pragma unroll 1
        for (int kg = 0; kg < ngroups; kg += 2) {
            const int kb = kw + kg * kFKG;
            wait_group<D>(kg + 1 < ngroups);
            if (kg == 0) {
                running_body(stA, kb);
                fix_offsets<RT>(m, z, nms);
            } else {
                fixed_body(stA, kb);
            }
            if (kg + 2 < ngroups) issue_group<D>(Kh, kb + 2 * kFKG, N, stA, lane);
            if (kg + 1 < ngroups) {
                wait_group<D>(kg + 2 < ngroups);
                fixed_body(stB, kb + kFKG);
                if (kg + 3 < ngroups) issue_group<D>(Kh, kb + 3 * kFKG, N, stB, lane);
            }
        }
        // a key far above its lane's offset overflowed a sum: redo this
        // wave's statistics with the running max (not met on real data)
        bool over = false;
#pragma unroll
        for (int i = 0; i < RT; ++i) over |= (z[i] == INFINITY);
        if (__builtin_amdgcn_ballot_w64(over) != 0) {
#pragma unroll
            for (int i = 0; i < RT; ++i) {
                m[i] = -INFINITY;
                z[i] = 0.f;
            }
#pragma unroll 1
            for (int kg = 0; kg < ngroups; ++kg) {
                const int kb = kw + kg * kFKG;
                issue_group<D>(Kh, kb, N, stA, lane);
                wait_vmem<0>();
                running_body(stA, kb);
            }
        }
#pragma unroll
        for (int i = 0; i < RT; ++i) normalise_mz(m[i], z[i]);
        // lanes sharing a row: g = 0..3, then waves
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 16), dev::shfl_xor_f(z[rt], 16));
            merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 32), dev::shfl_xor_f(z[rt], 32));
            if (g == 0) {
                sm.v.red.m[wave][rt * 16 + c16] = m[rt];
                sm.v.red.z[wave][rt * 16 + c16] = z[rt];
            }
        }
        __syncthreads();
        for (int r = tid; r < RT * 16; r += kThreads) {
            float mm = sm.v.red.m[0][r], zz = sm.v.red.z[0][r];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) merge_mz(mm, zz, sm.v.red.m[w][r], sm.v.red.z[w][r]);
            dev::st_coherent(a.part_m + pbase + rg * RT * 16 + r, mm);
            dev::st_coherent(a.part_z + pbase + rg * RT * 16 + r, zz);
        }
        __syncthreads();  // the statistics and limits are rewritten by the next group
    }
    if (count_stats(a, h, s_flag)) {
        const int* meta = a.rmeta + (size_t)h * kMetaWords;
        fold_and_publish(a, h, meta + kMetaAct, meta[0], a.hctl + (size_t)h * kHcWords);
    }
}

// The F item's key loop (both stages already in flight).
template <int D, int RT, bool MEAN>
__device__ __forceinline__ void final_loop(const uint16_t* Kh, int kw, int ngroups, int N, int clear_below,
                                           const int* lim, uint16_t* stA, uint16_t* stB, const Op<uint16_t, D>* yr,
                                           const float* nlse, float* out, float s2, float log2R, int lane, int c16,
                                           int g, int phase, float* kacc, float* kaccs, int k0) {
    auto body = [&](const uint16_t* st, int kb) {
        if (kb + kFKG <= clear_below)
            final_group<D, RT, MEAN, false>(st, kb, N, lim, yr, nlse, out, s2, log2R, c16, g, phase, kacc, kaccs,
                                            k0);
        else
            final_group<D, RT, MEAN, true>(st, kb, N, lim, yr, nlse, out, s2, log2R, c16, g, phase, kacc, kaccs,
                                           k0);
    };
#pragma unroll 1
    for (int kg = 0; kg < ngroups; kg += 2) {
        const int kb = kw + kg * kFKG;
        wait_group<D>(kg + 1 < ngroups);
        body(stA, kb);
        if (kg + 2 < ngroups) issue_group<D, 2>(Kh, kb + 2 * kFKG, N, stA, lane);
        if (kg + 1 < ngroups) {
            wait_group<D>(kg + 2 < ngroups);
            body(stB, kb + kFKG);
            if (kg + 3 < ngroups) issue_group<D, 2>(Kh, kb + 3 * kFKG, N, stB, lane);
        }
    }
}

template <int D, int RT, bool MULTI>
__device__ __forceinline__ void fast_final(const Args& a, int h, int chunk, FastSmem& sm, StageBuf<D>& sa, StageBuf<D>& sb,
                           Op<uint16_t, D>* yr, int* s_flag) {
    const int KC = a.key_chunk, KPW = KC / kWaves, GPW = KPW / kFKG;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const uint16_t* Kh = reinterpret_cast<const uint16_t*>(a.K) + (size_t)h * a.N_cap * D;
    const int N = a.N;
    const int kw = chunk * KC + wave * KPW;
    const int ngroups = max(0, min(GPW, (N - kw + kFKG - 1) / kFKG));
    uint16_t* stA = sa.k[wave];
    uint16_t* stB = sb.k[wave];
    // both stages in flight while lse is awaited
    if (ngroups > 0) issue_group<D, 2>(Kh, kw, N, stA, lane);
    if (ngroups > 1) issue_group<D, 2>(Kh, kw + kFKG, N, stB, lane);
    if (!await_lse(a, h, s_flag)) {
        wait_vmem<0>();  // no load may land in LDS after this workgroup ends
        return;
    }
    const float inv_s2 = 1.0f / a.s2;
    const KeyMask mk = key_mask(a, a.rmeta[(size_t)h * kMetaWords]);
    float* out = a.scores + (size_t)h * N;
    const int clear_below = mk.all_see_below();
    const float log2R = log2f((float)mk.R);
    const int nrg = MULTI ? a.R_pad_max / (RT * 16) : 1;
    for (int rg = 0; rg < nrg; ++rg) {
        if (MULTI) {
            load_rows<D, RT>(a, h, rg, yr, lane);
            if (rg > 0 && ngroups > 0) issue_group<D, 2>(Kh, kw, N, stA, lane);
            if (rg > 0 && ngroups > 1) issue_group<D, 2>(Kh, kw + kFKG, N, stB, lane);
        }
        for (int r = tid; r < RT * 16; r += kThreads)
            sm.v.fin.nlse[r] = -dev::ld_coherent(a.lse2 + (size_t)h * a.R_pad_max + rg * RT * 16 + r) * inv_s2;
        fill_limits<RT>(mk, rg * RT * 16, sm.lim);
        __syncthreads();
        const int phase = nrg == 1 ? kOnlyGroup : rg == 0 ? kFirstGroup : rg == nrg - 1 ? kLastGroup : kMidGroup;
        if (a.mean)
            final_loop<D, RT, true>(Kh, kw, ngroups, N, clear_below, sm.lim, stA, stB, yr, sm.v.fin.nlse, out, a.s2,
                                    log2R, lane, c16, g, phase, sm.v.fin.kacc, sm.v.fin.kaccs, chunk * KC);
        else
            final_loop<D, RT, false>(Kh, kw, ngroups, N, clear_below, sm.lim, stA, stB, yr, sm.v.fin.nlse, out, a.s2,
                                     0.f, lane, c16, g, phase, sm.v.fin.kacc, sm.v.fin.kaccs, chunk * KC);
        __syncthreads();  // the normalisers and limits are rewritten by the next group
    }
    // the item's scores, kept in LDS by the key loop, go out coalesced
    const int k0 = chunk * KC, nk = min(KC, N - k0);
    if (!a.fused) {
        for (int i = tid; i < nk; i += kThreads) out[k0 + i] = sm.v.fin.kacc[i];
        return;
    }
    // fused launch: the head's selection item (maybe on another XCD) reads
    // them, so they are written through coherently and counted in; the last
    // item of the head marks its scores complete
    for (int i = tid; i < nk; i += kThreads) dev::st_coherent(out + k0 + i, sm.v.fin.kacc[i]);
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) {
        int* hc = a.hctl + (size_t)h * kHcWords;
        if (dev::fetch_add_relaxed(hc + kHcFDone, 1) == a.nch - 1) dev::st_flag(hc + kHcScReady, 1);
    }
}

// ---- row split: four row groups, one per wave, sharing the key stream ----
//
// Heads whose rows span four groups of at most kFRT tiles (R of about 450
// to 576) would stream each key chunk four times through one wave's
// registers.  Here wave w holds row group w and every wave computes every
// key of the item from one shared stream: super-stages of four 32-key
// groups (sa, then sb; group q of a super-stage is loaded by wave q), one
// barrier per super-stage, the next super-stage in flight while one is
// computed.  S items store each wave's own rows' statistics; F items (max
// form) meet each key's maximum across the waves with an LDS atomic max.
constexpr int kSplitGroups = 4;
constexpr int kSuper = kWaves * kFKG;  // keys per super-stage
static_assert(kSplitGroups == kWaves && kMaxKeyChunk % kSuper == 0, "one row group per wave");

struct SplitLds {  // overlays FastSmem::v (S items use lim only)
    int lim[kSplitGroups][kFRT * 16];
    float nlse[kSplitGroups][kFRT * 16];
    unsigned kmax[kMaxKeyChunk];
};

// Issue super-stage s of an item (keys k0 + s kSuper ...): wave w loads its group.
template <int D, int AUX>
__device__ __forceinline__ void issue_super(const uint16_t* Kh, int k0, int s, int N, StageBuf<D>& st, int wave,
                                            int lane) {
    const int kb = k0 + s * kSuper + wave * kFKG;
    if (kb < N) issue_group<D, AUX>(Kh, kb, N, st.k[wave], lane);
}

template <int D, int RT>
__device__ void split_stats(const Args& a, int h, int chunk, FastSmem& sm, StageBuf<D>& sa, StageBuf<D>& sb,
                            int* s_flag) {
    static_assert(sizeof(SplitLds) <= sizeof(FastSmem::v), "row-split LDS fits the overlay");
    SplitLds& sl = *reinterpret_cast<SplitLds*>(&sm.v);
    const int KC = a.key_chunk;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const uint16_t* Kh = reinterpret_cast<const uint16_t*>(a.K) + (size_t)h * a.N_cap * D;
    const int N = a.N, k0 = chunk * KC;
    const int nsup = (min(KC, N - k0) + kSuper - 1) / kSuper;
    Op<uint16_t, D> yr[RT];
    load_rows<D, RT>(a, h, wave, yr, lane);
    issue_super<D, 0>(Kh, k0, 0, N, sa, wave, lane);
    if (nsup > 1) issue_super<D, 0>(Kh, k0, 1, N, sb, wave, lane);
    const float s2 = a.s2;
    const KeyMask mk = key_mask(a, a.rmeta[(size_t)h * kMetaWords]);
    const int clear_below = mk.all_see_below();
    for (int r = tid; r < kSplitGroups * RT * 16; r += kThreads) sl.lim[r / (RT * 16)][r % (RT * 16)] = mk.limit(r);
    const int* lim = sl.lim[wave];
    float m[RT], z[RT], nms[RT];
#pragma unroll
    for (int i = 0; i < RT; ++i) {
        m[i] = -INFINITY;
        z[i] = 0.f;
    }
    auto running_body = [&](const uint16_t* st, int kb) {
        if (kb + kFKG <= clear_below)
            stats_group<D, RT, false>(st, kb, lim, yr, s2, m, z, c16, g);
        else
            stats_group<D, RT, true>(st, kb, lim, yr, s2, m, z, c16, g);
    };
    auto fixed_body = [&](const uint16_t* st, int kb) {
        if (kb + kFKG <= clear_below)
            stats_group_fixed<D, RT, false>(st, kb, lim, yr, s2, nms, z, c16, g);
        else
            stats_group_fixed<D, RT, true>(st, kb, lim, yr, s2, nms, z, c16, g);
    };
    auto super_body = [&](StageBuf<D>& st, int sidx) {
#pragma unroll 1
        for (int q = 0; q < kWaves; ++q) {
            const int kb = k0 + sidx * kSuper + q * kFKG;
            if (kb >= N) break;
            if (sidx == 0 && q == 0) {  // the first group fixes each lane's offset
                running_body(st.k[q], kb);
                fix_offsets<RT>(m, z, nms);
            } else {
                fixed_body(st.k[q], kb);
            }
        }
    };
#pragma unroll 1
    for (int sidx = 0; sidx < nsup; sidx += 2) {
        wait_vmem<0>();
        __syncthreads();  // every wave's group landed; the other stage is free
        if (sidx >= 2 && sidx + 1 < nsup) issue_super<D, 0>(Kh, k0, sidx + 1, N, sb, wave, lane);
        super_body(sa, sidx);
        if (sidx + 1 < nsup) {
            wait_vmem<0>();
            __syncthreads();
            if (sidx + 2 < nsup) issue_super<D, 0>(Kh, k0, sidx + 2, N, sa, wave, lane);
            super_body(sb, sidx + 1);
        }
    }
    // a key far above its lane's offset overflowed a sum: this wave redoes
    // its rows with the running max, streaming through its own group stage
    __syncthreads();  // the shared stages are free
    bool over = false;
#pragma unroll
    for (int i = 0; i < RT; ++i) over |= (z[i] == INFINITY);
    if (__builtin_amdgcn_ballot_w64(over) != 0) {
#pragma unroll
        for (int i = 0; i < RT; ++i) {
            m[i] = -INFINITY;
            z[i] = 0.f;
        }
#pragma unroll 1
        for (int kb = k0; kb < min(k0 + KC, N); kb += kFKG) {
            issue_group<D>(Kh, kb, N, sa.k[wave], lane);
            wait_vmem<0>();
            running_body(sa.k[wave], kb);
        }
    }
#pragma unroll
    for (int i = 0; i < RT; ++i) normalise_mz(m[i], z[i]);
    // this wave's rows: lanes sharing a row (g = 0..3) meet, then go out
    const size_t pbase = ((size_t)h * a.nch + chunk) * a.R_pad_max + (size_t)wave * RT * 16;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 16), dev::shfl_xor_f(z[rt], 16));
        merge_mz(m[rt], z[rt], dev::shfl_xor_f(m[rt], 32), dev::shfl_xor_f(z[rt], 32));
        if (g == 0) {
            dev::st_coherent(a.part_m + pbase + rt * 16 + c16, m[rt]);
            dev::st_coherent(a.part_z + pbase + rt * 16 + c16, z[rt]);
        }
    }
    if (count_stats(a, h, s_flag)) {
        const int* meta = a.rmeta + (size_t)h * kMetaWords;
        fold_and_publish(a, h, meta + kMetaAct, meta[0], a.hctl + (size_t)h * kHcWords);
    }
}

template <int D, int RT>
__device__ void split_final(const Args& a, int h, int chunk, FastSmem& sm, StageBuf<D>& sa, StageBuf<D>& sb,
                            int* s_flag) {
    SplitLds& sl = *reinterpret_cast<SplitLds*>(&sm.v);
    const int KC = a.key_chunk;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c16 = lane & 15;
    const uint16_t* Kh = reinterpret_cast<const uint16_t*>(a.K) + (size_t)h * a.N_cap * D;
    const int N = a.N, k0 = chunk * KC, nk = min(KC, N - k0);
    const int nsup = (nk + kSuper - 1) / kSuper;
    Op<uint16_t, D> yr[RT];
    load_rows<D, RT>(a, h, wave, yr, lane);
    issue_super<D, 2>(Kh, k0, 0, N, sa, wave, lane);
    if (nsup > 1) issue_super<D, 2>(Kh, k0, 1, N, sb, wave, lane);
    for (int i = tid; i < nk; i += kThreads) sl.kmax[i] = 0u;  // below every score's order key
    if (!await_lse(a, h, s_flag)) {
        wait_vmem<0>();
        return;
    }
    const float inv_s2 = 1.0f / a.s2;
    const KeyMask mk = key_mask(a, a.rmeta[(size_t)h * kMetaWords]);
    const int clear_below = mk.all_see_below();
    for (int r = tid; r < kSplitGroups * RT * 16; r += kThreads) {
        sl.nlse[r / (RT * 16)][r % (RT * 16)] = -dev::ld_coherent(a.lse2 + (size_t)h * a.R_pad_max + r) * inv_s2;
        sl.lim[r / (RT * 16)][r % (RT * 16)] = mk.limit(r);
    }
    const int* lim = sl.lim[wave];
    const float* nlse = sl.nlse[wave];
    auto super_body = [&](StageBuf<D>& st, int sidx) {
#pragma unroll 1
        for (int q = 0; q < kWaves; ++q) {
            const int kb = k0 + sidx * kSuper + q * kFKG;
            if (kb >= N) break;
            if (kb + kFKG <= clear_below)
                final_group_split<D, RT, false>(st.k[q], kb, N, lim, yr, nlse, c16, g, sl.kmax, k0);
            else
                final_group_split<D, RT, true>(st.k[q], kb, N, lim, yr, nlse, c16, g, sl.kmax, k0);
        }
    };
#pragma unroll 1
    for (int sidx = 0; sidx < nsup; sidx += 2) {
        wait_vmem<0>();
        __syncthreads();  // (the first also: the normalisers, limits and kmax are set)
        if (sidx >= 2 && sidx + 1 < nsup) issue_super<D, 2>(Kh, k0, sidx + 1, N, sb, wave, lane);
        super_body(sa, sidx);
        if (sidx + 1 < nsup) {
            wait_vmem<0>();
            __syncthreads();
            if (sidx + 2 < nsup) issue_super<D, 2>(Kh, k0, sidx + 2, N, sa, wave, lane);
            super_body(sb, sidx + 1);
        }
    }
    __syncthreads();
    float* out = a.scores + (size_t)h * N;
    const float sc = a.s2 * 0.69314718055994531f;
    auto score_of = [&](int i) {
        const unsigned u = sl.kmax[i];  // inverse of the order key
        return __uint_as_float((u & 0x80000000u) ? (u & 0x7fffffffu) : ~u) * sc;
    };
    if (!a.fused) {
        for (int i = tid; i < nk; i += kThreads) out[k0 + i] = score_of(i);
        return;
    }
    for (int i = tid; i < nk; i += kThreads) dev::st_coherent(out + k0 + i, score_of(i));
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) {
        int* hc = a.hctl + (size_t)h * kHcWords;
        if (dev::fetch_add_relaxed(hc + kHcFDone, 1) == a.nch - 1) dev::st_flag(hc + kHcScReady, 1);
    }
}

// S or F item of a row-split head (F items of the mean form take the
// row-group loop: their per-key (max, sum) pairs do not merge by atomics).
template <int D, int RT>
__device__ __forceinline__ void split_item(const Args& a, int h, int ticket, FastSmem& sm, StageBuf<D>& sa,
                                           StageBuf<D>& sb, int* s_flag) {
    if (ticket < a.nch) {
        split_stats<D, RT>(a, h, ticket, sm, sa, sb, s_flag);
    } else if (!a.mean) {
        split_final<D, RT>(a, h, ticket - a.nch, sm, sa, sb, s_flag);
    } else {
        Op<uint16_t, D> yr[RT];
        fast_final<D, RT, true>(a, h, ticket - a.nch, sm, sa, sb, yr, s_flag);
    }
}

// SPLIT: four row groups, one per wave (MULTI is then true as well).
template <int D, int RT, bool MULTI, bool SPLIT>
__global__ __launch_bounds__(kThreads, 2) void fast_score_kernel(Args a) {
    __shared__ FastSmem sm;
    __shared__ StageBuf<D> sa;
    __shared__ StageBuf<D> sb;
    __shared__ int s_ticket, s_ok, s_flag;
    const int h = head_of_block(a, blockIdx.x);
    const TicketReq req = request_ticket(a, h);
    if constexpr (SPLIT) {
        if (!complete_ticket(a, req, &s_ticket, &s_ok)) return;
        split_item<D, RT>(a, h, __builtin_amdgcn_readfirstlane(s_ticket), sm, sa, sb, &s_flag);
        return;
    } else {
    Op<uint16_t, D> yr[RT];
    if (!MULTI) load_rows<D, RT>(a, h, 0, yr, threadIdx.x & 63);  // in flight with the ticket
    if (!complete_ticket(a, req, &s_ticket, &s_ok)) {
        wait_vmem<0>();
        return;
    }
    const int ticket = __builtin_amdgcn_readfirstlane(s_ticket);
    if (ticket < a.nch)
        fast_stats<D, RT, MULTI>(a, h, ticket, sm, sa, sb, yr, &s_flag);
    else
        fast_final<D, RT, MULTI>(a, h, ticket - a.nch, sm, sa, sb, yr, &s_flag);
    }
}

// ---- the fused eviction: score, select and compact under one ticket ------
//
// Each head's work items, in ticket order: nch S items, nch F items, one
// selection item (once every F item of the head has stored its scores) and
// nsegF compaction items (once the head's kept indices are stored).  Every
// wait is on lower tickets of the same head, which have started and never
// wait on higher ones, so the launch cannot deadlock whatever the
// residency.  The grid lists a head's selection and compaction workgroups
// lag2 heads after its first, so that the HBM-bound compaction of earlier
// heads runs while later heads are being scored.

// Workgroup -> head in the fused grid: slot s holds the S workgroups of head
// s (s < P), the F workgroups of head s - lag (lag <= s < P + lag), the
// selection workgroup of head s - lag2 and the compaction workgroups of
// head s - lag3, in that order; the host lists the slot ranges of equal
// size.  Workgroups that start early only wait (holding their slot), so
// each kind comes a few machine-fulls after what it needs.
__device__ __forceinline__ int head_of_block_fused(const Args& a, int b) {
    int i = 0;
    while (i + 1 < a.nreg && b >= a.rb[i + 1]) ++i;
    const int per = a.rper[i];
    const int s = a.rs[i] + (b - a.rb[i]) / per;
    int r = (b - a.rb[i]) % per;
    if (s < a.P) {
        if (r < a.nch) return s;
        r -= a.nch;
    }
    if (s >= a.lag && s < a.P + a.lag) {
        if (r < a.nch) return s - a.lag;
        r -= a.nch;
    }
    if (s >= a.lag2 && s < a.P + a.lag2) {
        if (r < 1) return s - a.lag2;
    }
    return s - a.lag3;
}

template <int D, int RT, bool MULTI, bool SPLIT>
__global__ __launch_bounds__(kThreads, 2) void evict_kernel(Args a) {
    __shared__ FastSmem sm;
    __shared__ StageBuf<D> sa;
    __shared__ StageBuf<D> sb;
    __shared__ int s_ticket, s_ok, s_flag;
    const int h = head_of_block_fused(a, blockIdx.x);
    const TicketReq req = request_ticket(a, h);
    if (!complete_ticket(a, req, &s_ticket, &s_ok)) return;
    const int ticket = __builtin_amdgcn_readfirstlane(s_ticket);
    if (ticket < 2 * a.nch) {
        if constexpr (SPLIT) {
            split_item<D, RT>(a, h, ticket, sm, sa, sb, &s_flag);
            return;
        }
        Op<uint16_t, D> yr[RT];
        if (!MULTI) load_rows<D, RT>(a, h, 0, yr, threadIdx.x & 63);
        if (ticket < a.nch)
            fast_stats<D, RT, MULTI>(a, h, ticket, sm, sa, sb, yr, &s_flag);
        else
            fast_final<D, RT, MULTI>(a, h, ticket - a.nch, sm, sa, sb, yr, &s_flag);
        return;
    }
    const int tid = threadIdx.x;
    int* hc = a.hctl + (size_t)h * kHcWords;
    if (ticket == 2 * a.nch) {
        // selection: every F item of the head has stored its scores
        if (tid == 0) {
            s_flag = dev::wait_flag(hc + kHcScReady);
            if (!s_flag) dev::raise_error(a.hdr, kErrScoreWait);
        }
        __syncthreads();
        constexpr int BINS = sizeof(StageBuf<D>) >= sizeof(roles::SelLds<4096>) ? 4096 : 2048;
        static_assert(sizeof(roles::SelLds<BINS>) <= sizeof(StageBuf<D>), "selection LDS");
        if (s_flag)
            roles::select_item<BINS>(a.scores + (size_t)h * a.N, a.kept + (size_t)h * a.n_keep, a.N, a.budget, a.W,
                                     a.n_prefix, *reinterpret_cast<roles::SelLds<BINS>*>(&sa));
        dev::wait_all_memory();
        __syncthreads();
        if (tid == 0) dev::st_flag(hc + kHcKept, s_flag ? 1 : 2);  // 2: no valid kept set
        return;
    }
    // compaction segment: the head's kept indices are stored
    const int seg = ticket - 2 * a.nch - 1;
    if (tid == 0) {
        s_flag = dev::wait_flag(hc + kHcKept) && dev::ld_flag(hc + kHcKept) == 1;
        if (!s_flag) dev::raise_error(a.hdr, kErrCompactWait);
    }
    __syncthreads();
    int* lds = reinterpret_cast<int*>(&sa);
    int* flags = a.cflags + (size_t)h * a.nseg_cap;
    bool ok = true;
    if (s_flag) {
        const size_t hs = (size_t)a.N_cap * D * 2;
        ok = roles::compact_item<D * 2>(a.Kc + (size_t)h * hs, a.Vc + (size_t)h * hs, a.kept + (size_t)h * a.n_keep,
                                        flags, seg, a.n_keep, a.N, lds, lds + roles::kSegF, a.hdr);
    } else if (tid == 0) {
        dev::st_flag(flags + seg, 1);  // lower-ticket waits of later segments end
    }
    if (!ok && tid == 0) dev::raise_error(a.hdr, kErrBadIndex);
    // the head's last segment leaves its flags clear for later launches
    __syncthreads();
    if (tid == 0) s_ok = dev::fetch_add_relaxed(hc + kHcFcDone, 1) == a.nsegF - 1;
    __syncthreads();
    if (s_ok) {
        for (int i = tid; i < a.nsegF; i += kThreads) dev::st_flag(flags + i, 0);
        if (tid == 0) dev::st_flag(hc + kHcFcDone, 0);
    }
}

template <int D, int RT>
hipError_t launch_fast_rt(const Args& a, hipStream_t s) {
    hipLaunchKernelGGL((rows_kernel<D>), dim3(a.P), dim3(kThreads), 0, s, a);
    const bool multi = a.R_pad_max > RT * 16;
    // four row groups of 7 to 9 tiles (R of about 400 to 576): one per wave
    if constexpr (RT >= 7) {
        if (a.R_pad_max == kSplitGroups * RT * 16 && a.key_chunk == kMaxKeyChunk) {
            if (a.fused)
                hipLaunchKernelGGL((evict_kernel<D, RT, true, true>), dim3(a.total), dim3(kThreads), 0, s, a);
            else
                hipLaunchKernelGGL((fast_score_kernel<D, RT, true, true>), dim3(a.total), dim3(kThreads), 0, s, a);
            return hipGetLastError();
        }
    }
    if (a.fused) {
        if (multi)
            hipLaunchKernelGGL((evict_kernel<D, RT, true, false>), dim3(a.total), dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL((evict_kernel<D, RT, false, false>), dim3(a.total), dim3(kThreads), 0, s, a);
    } else if (multi) {
        hipLaunchKernelGGL((fast_score_kernel<D, RT, true, false>), dim3(a.total), dim3(kThreads), 0, s, a);
    } else {
        hipLaunchKernelGGL((fast_score_kernel<D, RT, false, false>), dim3(a.total), dim3(kThreads), 0, s, a);
    }
    return hipGetLastError();
}

template <int D>
hipError_t launch_fast(const Args& a, int rtg, hipStream_t s) {
    switch (rtg) {
        case 1: return launch_fast_rt<D, 1>(a, s);
        case 2: return launch_fast_rt<D, 2>(a, s);
        case 3: return launch_fast_rt<D, 3>(a, s);
        case 4: return launch_fast_rt<D, 4>(a, s);
        case 5: return launch_fast_rt<D, 5>(a, s);
        case 6: return launch_fast_rt<D, 6>(a, s);
        case 7: return launch_fast_rt<D, 7>(a, s);
        case 8: return launch_fast_rt<D, 8>(a, s);
        default: return launch_fast_rt<D, 9>(a, s);
    }
}

template <typename T, int D, int KGN>
hipError_t launch_t(const Args& a, hipStream_t s) {
    hipLaunchKernelGGL(reset_control_kernel, dim3((a.P + 255) / 256), dim3(256), 0, s, a);
    hipLaunchKernelGGL((score_kernel<T, D, KGN>), dim3(a.total), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

namespace {

// Grid of the fused launch: the slot ranges of equal composition (see
// head_of_block_fused).
void fused_regions(Args& a) {
    const int P = a.P;
    int bp[8] = {0, a.lag, a.lag2, a.lag3, P, P + a.lag, P + a.lag2, P + a.lag3};
    for (int i = 1; i < 8; ++i)  // sort the breakpoints
        for (int j = i; j > 0 && bp[j] < bp[j - 1]; --j) {
            const int t = bp[j];
            bp[j] = bp[j - 1];
            bp[j - 1] = t;
        }
    a.nreg = 0;
    int b = 0;
    for (int i = 0; i + 1 < 8; ++i) {
        const int x = bp[i], y = bp[i + 1];
        if (x >= y) continue;
        const int per = (x < P ? a.nch : 0) + (x >= a.lag && x < P + a.lag ? a.nch : 0) +
                        (x >= a.lag2 && x < P + a.lag2 ? 1 : 0) + (x >= a.lag3 && x < P + a.lag3 ? a.nsegF : 0);
        if (per == 0) continue;
        a.rs[a.nreg] = x;
        a.rb[a.nreg] = b;
        a.rper[a.nreg] = per;
        ++a.nreg;
        b += per * (y - x);
    }
    a.total = b;
}

hipError_t launch_score_impl(const bkv_dims& d, const WsLayout& L, int flags, const void* K, void* V,
                             const void* q_win, const float* beacons, const int32_t* counts, const float* rope_cos,
                             const float* rope_sin, float scale, float* scores, float* row_lse, int32_t* kept,
                             void* ws, hipStream_t s) {
    char* w = static_cast<char*>(ws);
    Args a;
    memset(&a, 0, sizeof a);
    a.K = K;
    a.qwin = q_win;
    a.beacons = beacons;
    a.counts = counts;
    a.rope_cos = rope_cos;
    a.rope_sin = rope_sin;
    a.scores = scores;
    a.row_lse = row_lse;
    a.hdr = reinterpret_cast<int*>(w);
    a.hctl = reinterpret_cast<int*>(w + L.hctl);
    a.part_m = reinterpret_cast<float*>(w + L.part_m);
    a.part_z = reinterpret_cast<float*>(w + L.part_z);
    a.lse2 = reinterpret_cast<float*>(w + L.lse2);
    a.B = d.B;
    a.Hq = d.Hq;
    a.Hkv = d.Hkv;
    a.G = d.Hq / d.Hkv;
    a.N = d.N;
    a.N_cap = d.N_cap;
    a.W = d.W;
    a.C = d.C;
    a.P = L.P;
    a.budget = d.budget;
    a.R_pad_max = L.R_pad_max;
    a.nch = L.nch;
    a.key_chunk = L.key_chunk;
    // Lag between a head's S and F items: about two machine-fulls of items
    // (two resident workgroups per CU).  The F items, whose key loads are
    // non-temporal, then find their head's normalisers ready more often
    // while the re-read still comes from the memory-side cache: on the 32K
    // layer lags of 14 to 24 heads scored about 4 % faster than 8 and 32.
    int dev_id = 0, cus = 256;
    if (hipGetDevice(&dev_id) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id) != hipSuccess)
        cus = 256;
    int lag = (4 * cus + 2 * L.nch - 1) / (2 * L.nch);
    a.lag = lag < 1 ? 1 : (lag > L.P ? L.P : lag);
    a.total = 2 * L.P * L.nch;
    a.tickets = 2 * L.nch;
    if (V) {  // the fused eviction (fast path only)
        a.fused = 1;
        a.Kc = static_cast<char*>(const_cast<void*>(K));
        a.Vc = static_cast<char*>(V);
        a.kept = kept;
        a.cflags = reinterpret_cast<int*>(w + L.cflags);
        a.n_prefix = d.n_prefix;
        a.n_keep = d.N < d.budget ? d.N : d.budget;
        a.nsegF = (a.n_keep + roles::kSegF - 1) / roles::kSegF;
        a.nseg_cap = L.nseg;
        a.tickets = 2 * L.nch + 1 + a.nsegF;
        // the selection about two machine-fulls of workgroups after the
        // head's F items, the compaction about four more after the selection
        const int step = (4 * cus + a.tickets - 1) / a.tickets;
        a.lag2 = a.lag + step > L.P ? L.P : a.lag + step;
        a.lag3 = a.lag2 + 2 * step > L.P ? L.P : a.lag2 + 2 * step;
        fused_regions(a);
    }
    const float sc = (scale == 0.0f) ? (float)(1.0 / sqrt((double)d.D)) : scale;
    a.s2 = sc * 1.4426950408889634f;
    a.s2ln2 = a.s2 * 0.69314718055994531f;
    a.mean = (flags & BKV_SCORE_MEAN) != 0;
    a.causal = (flags & BKV_SCORE_CAUSAL) != 0;
    const bool bf = d.dtype == BKV_BF16;
    if (L.rtg > 0) {  // bf16: each row group's rows fit in registers
        a.rows = reinterpret_cast<uint16_t*>(w + L.rows);
        a.rmeta = reinterpret_cast<int*>(w + L.rmeta);
        return d.D == 128 ? launch_fast<128>(a, L.rtg, s) : launch_fast<64>(a, L.rtg, s);
    }
    if (a.fused) return hipErrorNotSupported;  // the caller checks evict_fusable first
    const bool k4 = L.kgn == 4;  // 1024-key items (else 256)
    if (bf && d.D == 128) return k4 ? launch_t<uint16_t, 128, 4>(a, s) : launch_t<uint16_t, 128, 1>(a, s);
    if (bf) return k4 ? launch_t<uint16_t, 64, 4>(a, s) : launch_t<uint16_t, 64, 1>(a, s);
    if (d.D == 128) return k4 ? launch_t<float, 128, 4>(a, s) : launch_t<float, 128, 1>(a, s);
    return k4 ? launch_t<float, 64, 4>(a, s) : launch_t<float, 64, 1>(a, s);
}

}  // namespace

hipError_t launch_score(const bkv_dims& d, const WsLayout& L, int flags, const void* K, const void* q_win,
                        const float* beacons, const int32_t* counts, const float* rope_cos,
                        const float* rope_sin, float scale, float* scores, float* row_lse, void* ws,
                        hipStream_t s) {
    return launch_score_impl(d, L, flags, K, nullptr, q_win, beacons, counts, rope_cos, rope_sin, scale, scores,
                             row_lse, nullptr, ws, s);
}

// Shorter heads have few score items per head, so the selection and
// compaction items come at the end of the grid and run with little to
// overlap (the 4224-token steady state measured 217 us fused against 210
// chained); longer heads take the selection's streaming path; heads of
// several row groups leave the score items long and few (the R = 464 16K
// layer measured 293 us fused against 213 chained).
bool evict_fusable(const bkv_dims& d, const WsLayout& L) {
    return L.rtg > 0 && L.R_pad_max == L.rtg * 16 && L.nch >= 16 && d.N <= 32768;
}

hipError_t launch_evict_fused(const bkv_dims& d, const WsLayout& L, int flags, void* K, void* V, const void* q_win,
                              const float* beacons, const int32_t* counts, const float* rope_cos,
                              const float* rope_sin, float scale, float* scores, float* row_lse, int32_t* kept,
                              void* ws, hipStream_t s) {
    return launch_score_impl(d, L, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale, scores, row_lse,
                             kept, ws, s);
}

}  // namespace bkv
