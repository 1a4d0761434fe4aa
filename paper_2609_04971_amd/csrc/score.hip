// (a2)+(a3) Observation rows and key scores for gfx950.
//
// For every (batch, kv-head) the observation rows y_r are the occupied
// beacons rotated to the current step plus the recent queries of the GQA
// group (Section 4.3; Algorithm 2).  With l_rj = scale * <y_r, k_j>, the
// key score is  s_j = max_r (l_rj - lse_r),  lse_r = log sum_j exp(l_rj):
// softmax attention normalised over all N keys (Eq. 4), aggregated by max
// over every query and head of the group (Eq. 6, max form).
//
// One launch does it all with ticketed work items:
//   S(h, c)  row statistics (running max m, sum z) of l over key chunk c;
//            the last S item of a head folds them into lse_r;
//   F(h, c)  recompute l for chunk c and write s_j = max_r (l_rj - lse_r).
// F(h, .) is ticketed `lag` heads after S(h, .), so the second read of a
// head's keys follows the first closely (it tends to hit the MI355X's
// memory-side cache rather than HBM).  An F item waits only for the S items
// of its head, which hold lower tickets, have started, and never wait, so
// the schedule cannot deadlock whatever the residency.
//
// Every item builds its own observation rows in LDS from the read-only
// inputs (RoPE, then rounding to the cache dtype), so the only data passed
// between work items are the per-chunk statistics and lse, a few KB per
// head.  Those go through agent-scope atomic loads and stores, which are
// coherent across the MI355X's per-XCD L2 caches by themselves; a producer
// waits for its stores to complete (s_waitcnt) before the counter or flag
// that publishes them, so no L2 write-back or invalidation is needed.
//
// Logits come from v_mfma_f32_16x16x32_bf16 (fp32 accumulation of exact
// bf16 products; fp32 caches use v_mfma_f32_16x16x4_f32).  A lane holds a
// contiguous quarter of a row (D/4 elements) of each 16-row operand tile,
// so the key tile is read straight from HBM with 16-byte loads, no LDS
// staging; the observation rows sit in LDS.  Statistics are kept in log2
// units (v_exp_f32 computes 2^x): s2 = scale * log2(e).  In F items the
// accumulator starts at -lse2_r / s2, so the MFMA yields l_rj - lse_r (up
// to the factor s2) directly and the epilogue is one max per element.
#include <math.h>

#include "device_common.h"
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
    static constexpr int RG = 160;  // observation rows resident in LDS at a time
};
template <>
struct Tr<float> {
    static constexpr int ES = 4;
    static constexpr int PAD = 4;
    static constexpr int RG = 80;
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
    int* p1cnt;     // [P] S items finished per head
    int* ready;     // [P] lse of the head published
    float* part_m;  // [P][nch][R_pad_max] chunk row maxima (log2 units)
    float* part_z;  // [P][nch][R_pad_max] chunk row sums relative to part_m
    float* lse2;    // [P][R_pad_max] row log2-normalisers
    int B, Hq, Hkv, G, N, N_cap, W, C, P, budget;
    int R_pad_max, nch, lag, total;
    float s2;     // scale * log2(e)
    float s2ln2;  // s2 * ln(2): log2-units-of-raw-dot -> natural log
};

// Per-lane operand slice: D/4 contiguous elements = NV 16-byte vectors.
template <typename T, int D>
struct Op {
    static constexpr int SL = D / 4;
    static constexpr int NV = SL * Tr<T>::ES / 16;
    dev::u32x4 v[NV];
};

template <typename T, int D>
__device__ __forceinline__ void load_key_tile(Op<T, D>& op, const T* Khead, int key, int g) {
    const dev::u32x4* src = reinterpret_cast<const dev::u32x4*>(Khead + (size_t)key * D + g * Op<T, D>::SL);
#pragma unroll
    for (int v = 0; v < Op<T, D>::NV; ++v) op.v[v] = src[v];
}

template <typename T, int D>
__device__ __forceinline__ void load_row_tile(Op<T, D>& op, const T* lds_row) {
    const dev::u32x4* src = reinterpret_cast<const dev::u32x4*>(lds_row);
#pragma unroll
    for (int v = 0; v < Op<T, D>::NV; ++v) op.v[v] = src[v];
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

template <typename T, int D>
struct alignas(16) Smem {
    T y[Tr<T>::RG * (D + Tr<T>::PAD)];
    float red_m[kWaves][Tr<T>::RG];
    float red_z[kWaves][Tr<T>::RG];
    float nlse[Tr<T>::RG];
    int act[kMaxC];
    int nact;
};

// Occupied beacon slots of head h, ascending, into sm.act / sm.nact.
template <typename T, int D>
__device__ __forceinline__ void active_slots(const Args& a, int h, Smem<T, D>& sm) {
    if (threadIdx.x == 0) {
        const int32_t* cnt = a.counts + (size_t)h * a.C;  // not read when C == 0
        int n = 0;
        for (int c = 0; c < a.C; ++c)
            if (cnt[c] > 0) sm.act[n++] = c;
        sm.nact = n;
    }
    __syncthreads();
}

// Observation rows [r0, r0 + nr) of head h into LDS: rows below nact are
// the occupied beacons rotated to the step and rounded to the cache dtype,
// then the G*W recent queries (contiguous in q_win), then zero padding.
template <typename T, int D>
__device__ void build_rows(const Args& a, int h, int r0, int nr, Smem<T, D>& sm) {
    constexpr int LD = D + Tr<T>::PAD;
    constexpr int VPR = D * Tr<T>::ES / 16;
    const int tid = threadIdx.x;
    const int b = h / a.Hkv, kh = h % a.Hkv;
    const int nact = sm.nact, R = nact + a.G * a.W;
    // beacon rows in this group
    const int bl = max(0, min(nact, r0 + nr) - r0);
    for (int idx = tid; idx < bl * (D / 2); idx += kThreads) {
        const int r = idx / (D / 2), i = idx % (D / 2);
        const float* beta = a.beacons + ((size_t)h * a.C + sm.act[r0 + r]) * D;
        float2 p = make_float2(beta[i], beta[i + D / 2]);
        if (a.rope_cos) p = rope_pair(p.x, p.y, a.rope_cos[i], a.rope_sin[i]);
        sm.y[r * LD + i] = to_elem<T>(p.x);
        sm.y[r * LD + i + D / 2] = to_elem<T>(p.y);
    }
    // recent rows and padding, 16 bytes at a time
    const T* q = reinterpret_cast<const T*>(a.qwin) + ((size_t)b * a.Hq + (size_t)kh * a.G) * a.W * D;
    for (int i = tid; i < (nr - bl) * VPR; i += kThreads) {
        const int r = bl + i / VPR, v = i % VPR;
        const int gr = r0 + r;  // row index within the head
        dev::u32x4 val = {0u, 0u, 0u, 0u};
        if (gr < R) val = reinterpret_cast<const dev::u32x4*>(q + (size_t)(gr - nact) * D)[v];
        *reinterpret_cast<dev::u32x4*>(sm.y + r * LD + v * (16 / Tr<T>::ES)) = val;
    }
}

// ---- S(h, chunk): row statistics over one key chunk -------------------------
template <typename T, int D, int KGN>
__device__ void stats_item(const Args& a, int h, int chunk, Smem<T, D>& sm, int* s_flag) {
    constexpr int RG = Tr<T>::RG, LD = D + Tr<T>::PAD, RTM = RG / 16;
    constexpr int KC = kWaves * 64 * KGN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    active_slots<T, D>(a, h, sm);
    const int nact = sm.nact;
    const int R = nact + a.G * a.W;
    const int Rp = (R + 15) & ~15;
    const T* Kh = reinterpret_cast<const T*>(a.K) + (size_t)h * a.N_cap * D;
    const int kw = chunk * KC + wave * 64 * KGN;  // this wave's first key
    const int N = a.N;
    const float s2 = a.s2;
    const size_t pbase = ((size_t)h * a.nch + chunk) * a.R_pad_max;

    for (int r0 = 0; r0 < Rp; r0 += RG) {
        const int nr = min(RG, Rp - r0), RT = nr / 16;
        __syncthreads();
        build_rows<T, D>(a, h, r0, nr, sm);
        __syncthreads();
        float m[RTM], z[RTM];
#pragma unroll
        for (int i = 0; i < RTM; ++i) {
            m[i] = -INFINITY;
            z[i] = 0.f;
        }
#pragma unroll
        for (int kg = 0; kg < KGN; ++kg) {
            const int kb = kw + kg * 64;
            if (kb < N) {
                Op<T, D> kop[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) load_key_tile<T, D>(kop[t], Kh, min(kb + t * 16 + c16, N - 1), g);
#pragma unroll
                for (int rt = 0; rt < RTM; ++rt) {
                    if (rt < RT) {
                        Op<T, D> yop;
                        load_row_tile<T, D>(yop, sm.y + (rt * 16 + c16) * LD + g * Op<T, D>::SL);
                        f32x4 acc[4];
                        float gm = -INFINITY;
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
                            mma(acc[t], kop[t], yop);  // rows = keys, columns = observation rows
#pragma unroll
                            for (int v = 0; v < 4; ++v) {
                                const int key = kb + t * 16 + 4 * g + v;
                                float x = (key < N) ? acc[t][v] : -INFINITY;
                                acc[t][v] = x;
                                gm = fmaxf(gm, x);
                            }
                        }
                        const float mnew = fmaxf(m[rt], gm * s2);
                        if (mnew != -INFINITY) {
                            float zz = (m[rt] == -INFINITY) ? 0.f : z[rt] * fast_exp2(m[rt] - mnew);
#pragma unroll
                            for (int t = 0; t < 4; ++t)
#pragma unroll
                                for (int v = 0; v < 4; ++v) zz += fast_exp2(__builtin_fmaf(acc[t][v], s2, -mnew));
                            z[rt] = zz;
                            m[rt] = mnew;
                        }
                    }
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
    // publish: statistics stored before the counter moves
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) *s_flag = (dev::fetch_add_relaxed(a.p1cnt + h, 1) == a.nch - 1);
    __syncthreads();
    if (!*s_flag) return;
    // last chunk of the head: fold the chunk statistics into lse
    const size_t hb = (size_t)h * a.nch * a.R_pad_max;
    for (int r = tid; r < Rp; r += kThreads) {
        float mm = -INFINITY, zz = 0.f;
        if (r < R)
            for (int c = 0; c < a.nch; ++c) {
                const size_t i = hb + (size_t)c * a.R_pad_max + r;
                merge_mz(mm, zz, dev::ld_coherent(a.part_m + i), dev::ld_coherent(a.part_z + i));
            }
        const float l2 = (r < R) ? mm + log2f(zz) : INFINITY;  // padding rows never win
        dev::st_coherent(a.lse2 + (size_t)h * a.R_pad_max + r, l2);
        if (a.row_lse && r < R) {
            const int slot = (r < nact) ? sm.act[r] : a.C + (r - nact);
            a.row_lse[(size_t)h * (a.C + a.G * a.W) + slot] = l2 * 0.69314718055994531f;
        }
    }
    if (a.row_lse) {  // empty beacon slots have no row
        const int32_t* cnt = a.counts + (size_t)h * a.C;
        for (int c = tid; c < a.C; c += kThreads)
            if (cnt[c] <= 0) a.row_lse[(size_t)h * (a.C + a.G * a.W) + c] = -INFINITY;
    }
    dev::wait_all_memory();
    __syncthreads();
    if (tid == 0) dev::st_flag(a.ready + h, 1);
}

// ---- F(h, chunk): final max-aggregated scores over one key chunk ----------
template <typename T, int D, int KGN>
__device__ void final_item(const Args& a, int h, int chunk, Smem<T, D>& sm) {
    constexpr int RG = Tr<T>::RG, LD = D + Tr<T>::PAD, RTM = RG / 16;
    constexpr int KC = kWaves * 64 * KGN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    active_slots<T, D>(a, h, sm);
    const int R = sm.nact + a.G * a.W;
    const int Rp = (R + 15) & ~15;
    const T* Kh = reinterpret_cast<const T*>(a.K) + (size_t)h * a.N_cap * D;
    const int kw = chunk * KC + wave * 64 * KGN;
    const int N = a.N;
    const float inv_s2 = 1.0f / a.s2;

    float best[4 * KGN];
#pragma unroll
    for (int i = 0; i < 4 * KGN; ++i) best[i] = -INFINITY;

    for (int r0 = 0; r0 < Rp; r0 += RG) {
        const int nr = min(RG, Rp - r0), RT = nr / 16;
        __syncthreads();
        build_rows<T, D>(a, h, r0, nr, sm);
        for (int r = tid; r < nr; r += kThreads)
            sm.nlse[r] = -dev::ld_coherent(a.lse2 + (size_t)h * a.R_pad_max + r0 + r) * inv_s2;
        __syncthreads();
#pragma unroll
        for (int kg = 0; kg < KGN; ++kg) {
            const int kb = kw + kg * 64;
            if (kb < N) {
                Op<T, D> kop[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) load_key_tile<T, D>(kop[t], Kh, min(kb + t * 16 + c16, N - 1), g);
#pragma unroll
                for (int rt = 0; rt < RTM; ++rt) {
                    if (rt < RT) {
                        Op<T, D> yop;
                        load_row_tile<T, D>(yop, sm.y + (rt * 16 + c16) * LD + g * Op<T, D>::SL);
                        const f32x4 c0 = *reinterpret_cast<const f32x4*>(sm.nlse + rt * 16 + 4 * g);
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            f32x4 acc = c0;
                            mma(acc, yop, kop[t]);  // rows = observation rows, columns = keys
                            best[kg * 4 + t] =
                                fmaxf(best[kg * 4 + t], fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3])));
                        }
                    }
                }
            }
        }
    }
    float* out = a.scores + (size_t)h * N;
#pragma unroll
    for (int i = 0; i < 4 * KGN; ++i) {
        float b = best[i];
        b = fmaxf(b, dev::shfl_xor_f(b, 16));
        b = fmaxf(b, dev::shfl_xor_f(b, 32));
        const int key = kw + (i >> 2) * 64 + (i & 3) * 16 + c16;
        if (g == (i & 3) && key < N) out[key] = b * a.s2ln2;
    }
}

// Ticket -> work item.  kind 1 = S, 2 = F.  The S items of head h come
// `lag` heads before its F items.
__device__ __forceinline__ void decode(const Args& a, int t, int& kind, int& h, int& c) {
    const int P = a.P, nch = a.nch, L = a.lag;
    if (t < L * nch) {
        kind = 1;
        h = t / nch;
        c = t % nch;
        return;
    }
    t -= L * nch;
    if (t < (P - L) * 2 * nch) {
        const int s = L + t / (2 * nch), r = t % (2 * nch);
        if (r < nch) {
            kind = 1;
            h = s;
            c = r;
        } else {
            kind = 2;
            h = s - L;
            c = r - nch;
        }
        return;
    }
    t -= (P - L) * 2 * nch;
    kind = 2;
    h = P - L + t / nch;
    c = t % nch;
}

template <typename T, int D, int KGN>
__global__ __launch_bounds__(kThreads) void score_kernel(Args a) {
    __shared__ Smem<T, D> sm;
    __shared__ int s_ticket, s_ok, s_flag;
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_ok = dev::stamp_ok(a.hdr, a.P, a.budget);
        if (s_ok)
            s_ticket = dev::fetch_add_relaxed(a.hdr + kHdrScTicket, 1);
        else
            dev::raise_error(a.hdr, kErrStamp);
    }
    __syncthreads();
    if (!s_ok) return;
    if (s_ticket >= a.total) {  // control block was not clear: do nothing
        if (tid == 0) dev::raise_error(a.hdr, kErrStamp);
        return;
    }
    int kind, h, c;
    decode(a, s_ticket, kind, h, c);
    if (kind == 1) {
        stats_item<T, D, KGN>(a, h, c, sm, &s_flag);
    } else {
        if (tid == 0) {
            s_flag = dev::wait_flag(a.ready + h);
            if (!s_flag) dev::raise_error(a.hdr, kErrScoreWait);
        }
        __syncthreads();
        if (s_flag) final_item<T, D, KGN>(a, h, c, sm);
    }
    // The last item to finish clears the control block for the next launch.
    __syncthreads();
    if (tid == 0) s_flag = (dev::fetch_add_relaxed(a.hdr + kHdrScDone, 1) == a.total - 1);
    __syncthreads();
    if (s_flag) {
        for (int i = tid; i < a.P; i += kThreads) {
            dev::st_flag(a.p1cnt + i, 0);
            dev::st_flag(a.ready + i, 0);
        }
        if (tid == 0) {
            dev::st_flag(a.hdr + kHdrScTicket, 0);
            dev::st_flag(a.hdr + kHdrScDone, 0);
        }
    }
}

template <typename T, int D, int KGN>
hipError_t launch_t(const Args& a, hipStream_t s) {
    hipLaunchKernelGGL((score_kernel<T, D, KGN>), dim3(a.total), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const bkv_dims& d, const WsLayout& L, const void* K, const void* q_win,
                        const float* beacons, const int32_t* counts, const float* rope_cos,
                        const float* rope_sin, float scale, float* scores, float* row_lse, void* ws,
                        hipStream_t s) {
    char* w = static_cast<char*>(ws);
    Args a;
    a.K = K;
    a.qwin = q_win;
    a.beacons = beacons;
    a.counts = counts;
    a.rope_cos = rope_cos;
    a.rope_sin = rope_sin;
    a.scores = scores;
    a.row_lse = row_lse;
    a.hdr = reinterpret_cast<int*>(w);
    a.p1cnt = reinterpret_cast<int*>(w + L.p1cnt);
    a.ready = reinterpret_cast<int*>(w + L.ready);
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
    // Lag between a head's S and F items: about one machine-full of items.
    int dev_id = 0, cus = 256;
    if (hipGetDevice(&dev_id) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev_id) != hipSuccess)
        cus = 256;
    int lag = (2 * cus + 2 * L.nch - 1) / (2 * L.nch);
    a.lag = lag < 1 ? 1 : (lag > L.P ? L.P : lag);
    a.total = 2 * L.P * L.nch;
    const float sc = (scale == 0.0f) ? (float)(1.0 / sqrt((double)d.D)) : scale;
    a.s2 = sc * 1.4426950408889634f;
    a.s2ln2 = a.s2 * 0.69314718055994531f;
    const bool bf = d.dtype == BKV_BF16;
    if (bf && d.D == 128) return L.kgn == 4 ? launch_t<uint16_t, 128, 4>(a, s) : launch_t<uint16_t, 128, 1>(a, s);
    if (bf && d.D == 64) return L.kgn == 4 ? launch_t<uint16_t, 64, 4>(a, s) : launch_t<uint16_t, 64, 1>(a, s);
    if (d.D == 128) return L.kgn == 4 ? launch_t<float, 128, 4>(a, s) : launch_t<float, 128, 1>(a, s);
    return L.kgn == 4 ? launch_t<float, 64, 4>(a, s) : launch_t<float, 64, 1>(a, s);
}

}  // namespace bkv
