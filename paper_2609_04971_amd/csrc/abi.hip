// C ABI of the eviction-step library (declared in include/bkv.h): host-side
// validation, workspace layout, and the enqueue of each operation's kernels.
// Nothing here allocates device memory or synchronises, except
// bkv_device_status, which is documented to.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "bkv.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

constexpr int kMaxRows = 1024;  // observation rows per head (C + G*W)
constexpr int kMaxC = 64;
constexpr int kFpsMaxN = 32768;     // rows per FPS head
constexpr int kFpsMaxGather = 128;  // rows an FPS gather writes per head

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

__global__ void ws_init_kernel(int* ws, int nwords, int P, int budget) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < nwords; i += gridDim.x * blockDim.x) {
        int v = 0;
        if (i == kHdrMagic) v = (int)kWsMagic;
        if (i == kHdrP) v = P;
        if (i == kHdrBudget) v = budget;
        ws[i] = v;
    }
}

}  // namespace

WsLayout ws_layout(const bkv_dims& d) {
    WsLayout L;
    memset(&L, 0, sizeof L);
    const int P = d.B * d.Hkv;
    const int G = d.Hkv > 0 ? d.Hq / d.Hkv : 0;
    L.P = P;
    L.nseg = (d.budget + kSegRows - 1) / kSegRows;
    size_t off = kHdrWords * sizeof(int);
    L.hctl = off;
    off = align_up(off + sizeof(int) * (size_t)P * kHcWords);
    L.cflags = off;
    off = align_up(off + sizeof(int) * (size_t)P * L.nseg);
    if (d.N > d.budget && d.N > kTkMinN && P <= kTkMaxHeads) {  // heads may be split for selection
        L.tk_hist = off;
        off = align_up(off + sizeof(int) * (size_t)P * 4096);
        L.tk_head = off;
        off = align_up(off + sizeof(int) * (size_t)P * kTkHeadWords);
        L.tk_cand = off;
        off = align_up(off + sizeof(uint32_t) * 2 * (size_t)P * 512);
        L.tk_cnt = off;
        off = align_up(off + sizeof(int) * (size_t)P * kTkMaxSlices);
    }
    L.ctl_end = off;
    // data (depends on N, W, C as well)
    const int R = d.C + G * d.W;
    const int tiles = (R + 15) / 16;
    L.rtg = 0;
    L.R_pad_max = tiles * 16;
    if (d.dtype == BKV_BF16 && tiles <= kFastTiles * kFastRowGroups) {
        // fast path: rows in equal groups of at most kFastTiles tiles, padded
        // with rows that never win
        const int nrg = max(1, (tiles + kFastTiles - 1) / kFastTiles);
        L.rtg = max(1, (tiles + nrg - 1) / nrg);
        L.R_pad_max = nrg * L.rtg * 16;
    }
    // key chunk per score work item: 1024 keys once there are enough chunks
    // to fill the machine about twice (shorter items spend their time on the
    // ticket, the rows and the epilogue: at 4K tokens and 128 heads 1024-key
    // items score 30 % faster than 256-key ones), or when the rows span
    // several row groups (each group streams the chunk again); else 256
    const long long big = (long long)P * ((d.N + 1023) / 1024);
    L.kgn = (big >= 512 || tiles > kFastTiles) ? 4 : 1;
    L.key_chunk = 256 * L.kgn;
    L.nch = (d.N + L.key_chunk - 1) / L.key_chunk;
    L.part_m = off;
    off = align_up(off + sizeof(float) * (size_t)P * L.nch * L.R_pad_max);
    L.part_z = off;
    off = align_up(off + sizeof(float) * (size_t)P * L.nch * L.R_pad_max);
    L.lse2 = off;
    off = align_up(off + sizeof(float) * (size_t)P * L.R_pad_max);
    L.rows = off;
    off = align_up(off + sizeof(uint16_t) * (size_t)P * L.R_pad_max * d.D);
    L.rmeta = off;
    off = align_up(off + sizeof(int32_t) * (size_t)P * kMetaWords);
    L.score_end = off;
    L.scores = off;
    off = align_up(off + sizeof(float) * (size_t)P * d.N);
    L.kept = off;
    off = align_up(off + sizeof(int32_t) * (size_t)P * d.budget);
    L.evict_end = off;
    return L;
}

}  // namespace bkv

using namespace bkv;

namespace {

bkv_status map_hip(hipError_t e) { return e == hipSuccess ? BKV_OK : BKV_ERR_HIP; }

bool empty_batch(const bkv_dims* d) { return d->B == 0; }

}  // namespace

extern "C" {

bkv_status bkv_validate(const bkv_dims* d, int32_t op) {
    if (!d) return BKV_ERR_INVALID;
    if (op < BKV_OP_BEACON_UPDATE || op > BKV_OP_EVICT) return BKV_ERR_INVALID;
    if (d->dtype != BKV_F32 && d->dtype != BKV_BF16) return BKV_ERR_DTYPE;
    if (d->B < 0 || d->Hkv < 1 || d->Hq < 1 || d->Hq % d->Hkv != 0) return BKV_ERR_SHAPE;
    if (d->D != 64 && d->D != 128) return BKV_ERR_SHAPE;
    if (d->N_cap < 1 || d->N < 0 || d->N > d->N_cap) return BKV_ERR_SHAPE;
    if (d->W < 0 || d->C < 0 || d->C > kMaxC || d->n_prefix < 0) return BKV_ERR_SHAPE;
    if ((long long)d->W + d->n_prefix > d->budget || d->budget < 1) return BKV_ERR_SHAPE;
    const long long G = d->Hq / d->Hkv;
    // index arithmetic stays in 32 bits where the kernels use int
    if ((long long)d->B * d->Hkv * d->N_cap > 0x7fffffffLL || (long long)d->B * d->Hq * d->W > 0x7fffffffLL)
        return BKV_ERR_SHAPE;
    if (op == BKV_OP_SCORE || op == BKV_OP_EVICT) {
        const long long R = d->C + G * d->W;
        if (R < 1 || R > kMaxRows) return BKV_ERR_SHAPE;
    }
    if (op == BKV_OP_BEACON_UPDATE && d->C < 1) return BKV_ERR_SHAPE;
    return BKV_OK;
}

size_t bkv_workspace_bytes(const bkv_dims* d, int32_t op) {
    if (bkv_validate(d, op) != BKV_OK) return 0;
    const WsLayout L = ws_layout(*d);
    switch (op) {
        case BKV_OP_SCORE: return L.score_end;
        case BKV_OP_TOPK: return L.tk_hist ? L.ctl_end : 0;
        case BKV_OP_COMPACT: return L.ctl_end;
        case BKV_OP_EVICT: return L.evict_end;
        default: return 0;
    }
}

bkv_status bkv_workspace_init(const bkv_dims* d, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!d || !ws) return BKV_ERR_INVALID;
    bkv_status st = bkv_validate(d, BKV_OP_COMPACT);
    if (st != BKV_OK) return st;
    const WsLayout L = ws_layout(*d);
    if (ws_bytes < L.ctl_end) return BKV_ERR_WORKSPACE;
    const int nwords = (int)(L.ctl_end / sizeof(int));
    int blocks = (nwords + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(ws_init_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<int*>(ws), nwords, L.P,
                       d->budget);
    return map_hip(hipGetLastError());
}

bkv_status bkv_device_status(const void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!ws || ws_bytes < kHdrWords * sizeof(int)) return BKV_ERR_INVALID;
    if (hipStreamSynchronize(stream) != hipSuccess) return BKV_ERR_HIP;
    int hdr[4];
    if (hipMemcpy(hdr, ws, sizeof hdr, hipMemcpyDeviceToHost) != hipSuccess) return BKV_ERR_HIP;
    if ((uint32_t)hdr[kHdrMagic] != kWsMagic) return BKV_ERR_WORKSPACE;
    return hdr[kHdrErr] ? BKV_ERR_DEVICE : BKV_OK;
}

bkv_status bkv_beacon_update(const bkv_dims* d, const void* q_new, int32_t T, float* beacons, int32_t* counts,
                             int32_t* assign, hipStream_t stream) {
    bkv_status st = bkv_validate(d, BKV_OP_BEACON_UPDATE);
    if (st != BKV_OK) return st;
    if (T < 0) return BKV_ERR_SHAPE;
    if (empty_batch(d) || T == 0) return BKV_OK;
    if (!q_new || !beacons || !counts) return BKV_ERR_INVALID;
    if ((long long)d->B * d->Hq * T * d->D > 0x7fffffffLL) return BKV_ERR_SHAPE;
    return map_hip(launch_beacon_update(*d, q_new, T, beacons, counts, assign, stream));
}

static bkv_status check_score_args(const bkv_dims* d, const void* K, const void* q_win, const float* beacons,
                                   const int32_t* counts, const float* rope_cos, const float* rope_sin,
                                   float scale) {
    if (!K || ((!beacons || !counts) && d->C > 0) || (!q_win && d->W > 0)) return BKV_ERR_INVALID;
    if ((rope_cos == nullptr) != (rope_sin == nullptr)) return BKV_ERR_INVALID;
    if (!aligned16(K) || (q_win && !aligned16(q_win))) return BKV_ERR_INVALID;
    if (!(scale >= 0.0f) || isinf(scale)) return BKV_ERR_INVALID;
    return BKV_OK;
}

bkv_status bkv_score(const bkv_dims* d, const void* K, const void* q_win, const float* beacons,
                     const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                     float* scores, float* row_lse, void* ws, size_t ws_bytes, hipStream_t stream) {
    return bkv_score_ex(d, 0, K, q_win, beacons, counts, rope_cos, rope_sin, scale, scores, row_lse, ws, ws_bytes,
                        stream);
}

bkv_status bkv_score_ex(const bkv_dims* d, int32_t flags, const void* K, const void* q_win, const float* beacons,
                        const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                        float* scores, float* row_lse, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (flags & ~(BKV_SCORE_MEAN | BKV_SCORE_CAUSAL)) return BKV_ERR_INVALID;
    bkv_status st = bkv_validate(d, BKV_OP_SCORE);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    st = check_score_args(d, K, q_win, beacons, counts, rope_cos, rope_sin, scale);
    if (st != BKV_OK) return st;
    if (!scores) return BKV_ERR_INVALID;
    const WsLayout L = ws_layout(*d);
    if (!ws || ws_bytes < L.score_end || !aligned16(ws)) return BKV_ERR_WORKSPACE;
    return map_hip(launch_score(*d, L, flags, K, q_win, beacons, counts, rope_cos, rope_sin, scale, scores, row_lse, ws,
                                stream));
}

bkv_status bkv_topk(const bkv_dims* d, const float* scores, int32_t* kept, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
    bkv_status st = bkv_validate(d, BKV_OP_TOPK);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    if (!scores || !kept) return BKV_ERR_INVALID;
    const WsLayout L = ws_layout(*d);
    // the split selection needs the workspace's control block; without it
    // (or with a smaller buffer) every head takes one workgroup
    void* w = (ws && L.tk_hist && ws_bytes >= L.ctl_end) ? ws : nullptr;
    return map_hip(launch_topk(*d, L, scores, kept, w, stream));
}

bkv_status bkv_compact(const bkv_dims* d, void* K, void* V, const int32_t* kept, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
    bkv_status st = bkv_validate(d, BKV_OP_COMPACT);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    if (!K || !V || !kept) return BKV_ERR_INVALID;
    if (!aligned16(K) || !aligned16(V)) return BKV_ERR_INVALID;
    const WsLayout L = ws_layout(*d);
    if (!ws || ws_bytes < L.ctl_end || !aligned16(ws)) return BKV_ERR_WORKSPACE;
    return map_hip(launch_compact(*d, L, K, V, kept, ws, stream));
}

bkv_status bkv_compact_fill(const bkv_dims* d, void* K, void* V, const int32_t* kept, int32_t* src_of, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
    bkv_status st = bkv_validate(d, BKV_OP_COMPACT);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    if (!K || !V || !kept || !src_of) return BKV_ERR_INVALID;
    if (!aligned16(K) || !aligned16(V)) return BKV_ERR_INVALID;
    if ((d->N < d->budget ? d->N : d->budget) > kMaxFillKeep) return BKV_ERR_SHAPE;
    const WsLayout L = ws_layout(*d);
    if (!ws || ws_bytes < L.ctl_end || !aligned16(ws)) return BKV_ERR_WORKSPACE;
    return map_hip(launch_compact_fill(*d, K, V, kept, src_of, ws, stream));
}

bkv_status bkv_evict(const bkv_dims* d, void* K, void* V, const void* q_win, const float* beacons,
                     const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                     int32_t* kept, float* scores, float* row_lse, void* ws, size_t ws_bytes,
                     hipStream_t stream) {
    return bkv_evict_ex(d, 0, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale, kept, scores, row_lse, ws,
                        ws_bytes, stream);
}

bkv_status bkv_evict_ex(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win, const float* beacons,
                        const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                        int32_t* kept, float* scores, float* row_lse, void* ws, size_t ws_bytes,
                        hipStream_t stream) {
    bkv_status st = bkv::evict_check(d, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    const WsLayout L = ws_layout(*d);
    if (!ws || ws_bytes < L.evict_end || !aligned16(ws)) return BKV_ERR_WORKSPACE;
    return bkv::evict_enqueue(d, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale, kept, scores,
                              row_lse, ws, stream);
}

}  // extern "C"

namespace bkv {

bkv_status evict_check(const bkv_dims* d, int32_t flags, const void* K, const void* V, const void* q_win,
                       const float* beacons, const int32_t* counts, const float* rope_cos, const float* rope_sin,
                       float scale) {
    if (flags & ~(BKV_SCORE_MEAN | BKV_SCORE_CAUSAL)) return BKV_ERR_INVALID;
    bkv_status st = bkv_validate(d, BKV_OP_EVICT);
    if (st != BKV_OK) return st;
    if (empty_batch(d) || d->N == 0) return BKV_OK;
    st = check_score_args(d, K, q_win, beacons, counts, rope_cos, rope_sin, scale);
    if (st != BKV_OK) return st;
    if (!V || !aligned16(V)) return BKV_ERR_INVALID;
    return BKV_OK;
}

bkv_status evict_enqueue(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win, const float* beacons,
                         const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                         int32_t* kept, float* scores, float* row_lse, void* ws, hipStream_t stream) {
    const WsLayout L = ws_layout(*d);
    char* w = static_cast<char*>(ws);
    float* sc = scores ? scores : reinterpret_cast<float*>(w + L.scores);
    int32_t* kp = kept ? kept : reinterpret_cast<int32_t*>(w + L.kept);
    if (evict_fusable(*d, L))
        return map_hip(launch_evict_fused(*d, L, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale, sc,
                                          row_lse, kp, ws, stream));
    hipError_t e =
        launch_score(*d, L, flags, K, q_win, beacons, counts, rope_cos, rope_sin, scale, sc, row_lse, ws, stream);
    if (e != hipSuccess) return BKV_ERR_HIP;
    e = launch_topk(*d, L, sc, kp, ws, stream);
    if (e != hipSuccess) return BKV_ERR_HIP;
    return map_hip(launch_compact(*d, L, K, V, kp, ws, stream));
}

}  // namespace bkv

extern "C" {

static bkv_status check_fps_args(int32_t H, int32_t n, int32_t m, int32_t D, int32_t dtype, const void* q,
                                 int32_t q_rows) {
    if (dtype != BKV_F32 && dtype != BKV_BF16) return BKV_ERR_DTYPE;
    if (D != 64 && D != 128) return BKV_ERR_SHAPE;
    if (H < 0 || n < 0 || m < 0 || n > kFpsMaxN || q_rows < n) return BKV_ERR_SHAPE;
    if ((long long)H * q_rows > 0x7fffffffLL) return BKV_ERR_SHAPE;
    if (H > 0 && n > 0 && m > 0 && (!q || !aligned16(q))) return BKV_ERR_INVALID;
    return BKV_OK;
}

bkv_status bkv_fps(int32_t H, int32_t n, int32_t m, int32_t D, int32_t dtype, const void* q, int32_t q_rows,
                   int32_t* picks, hipStream_t stream) {
    bkv_status st = check_fps_args(H, n, m, D, dtype, q, q_rows);
    if (st != BKV_OK) return st;
    if (H == 0 || n == 0 || m == 0) return BKV_OK;
    if (!picks) return BKV_ERR_INVALID;
    const int k = m < n ? m : n;
    return map_hip(launch_fps(H, n, k, D, dtype, q, q_rows, picks, nullptr, dtype, 0, nullptr, stream));
}

bkv_status bkv_fps_gather(int32_t H, int32_t n, int32_t m, int32_t D, int32_t dtype, const void* src,
                          int32_t src_rows, void* dst, int32_t dst_dtype, int32_t dst_rows, int32_t* picks,
                          int32_t* counts, hipStream_t stream) {
    bkv_status st = check_fps_args(H, n, m, D, dtype, src, src_rows);
    if (st != BKV_OK) return st;
    if (dst_dtype != BKV_F32 && dst_dtype != dtype) return BKV_ERR_DTYPE;
    const int k = m < n ? m : n;
    if (k > kFpsMaxGather || dst_rows < k || (long long)H * dst_rows > 0x7fffffffLL) return BKV_ERR_SHAPE;
    if (H == 0 || n == 0 || m == 0) return BKV_OK;
    if (!dst || !aligned16(dst)) return BKV_ERR_INVALID;
    // dst is either src itself, with the same layout, or disjoint from it
    const size_t src_bytes = (size_t)H * src_rows * D * (dtype == BKV_BF16 ? 2 : 4);
    const size_t dst_bytes = (size_t)H * dst_rows * D * (dst_dtype == BKV_BF16 ? 2 : 4);
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
    const bool overlap = s0 < d0 + dst_bytes && d0 < s0 + src_bytes;
    if (overlap && !(s0 == d0 && dst_dtype == dtype && dst_rows == src_rows)) return BKV_ERR_INVALID;
    return map_hip(launch_fps(H, n, k, D, dtype, src, src_rows, picks, dst, dst_dtype, dst_rows, counts, stream));
}

const char* bkv_status_string(bkv_status s) {
    switch (s) {
        case BKV_OK: return "ok";
        case BKV_ERR_INVALID: return "invalid argument";
        case BKV_ERR_SHAPE: return "invalid or unsupported shape";
        case BKV_ERR_DTYPE: return "unsupported dtype";
        case BKV_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
        case BKV_ERR_HIP: return "HIP runtime error";
        case BKV_ERR_DEVICE: return "device-side check failed";
    }
    return "unknown status";
}

int32_t bkv_abi_version(void) { return 1; }

}  // extern "C"
