// Internal interface between the C ABI (abi.hip) and the kernel files.
// Not installed; the public contract is include/bkv.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "bkv.h"

namespace bkv {

// ---- workspace --------------------------------------------------------------
// Control block (zeroed by init except the stamp; the score words are also
// reset by every score launch before it starts, the compaction words are
// left zero by every compaction), then data.
// The control block's size and offsets depend only on P = B*Hkv and budget,
// so one initialised workspace stays valid while N, W or C change.
constexpr uint32_t kWsMagic = 0x424b5631u;  // "BKV1"

enum HdrWord : int {
    kHdrMagic = 0,
    kHdrP = 1,
    kHdrBudget = 2,
    kHdrErr = 3,     // sticky device error bits, cleared only by init
    kHdrWords = 64   // header is 256 bytes
};

// One 128-byte control line per (batch, kv-head), so that work items of
// different heads never contend for one address.
enum HeadWord : int {
    kHcScTicket = 0,  // score: work ticket within the head
    kHcP1Count = 2,   // score: statistics items of the head finished
    kHcReady = 3,     // score: the head's row normalisers are published
    kHcCpTicket = 4,  // compaction: work ticket within the head
    kHcCpDone = 5,    // compaction: segments of the head finished
    // the fused eviction launch (score, select and compaction work items of
    // every head under the score ticket)
    kHcFcDone = 6,    // fused: compaction segments of the head finished
    kHcFDone = 7,     // fused: final-score items of the head finished
    kHcScReady = 8,   // fused: the head's scores are all stored
    kHcKept = 9,      // fused: the head's kept indices are stored
    kHcWords = 32
};

enum DevErr : int { kErrScoreWait = 1, kErrCompactWait = 2, kErrStamp = 4, kErrBadIndex = 8 };

constexpr int kSegRows = 128;  // compaction rows per work item
constexpr int kMaxFillKeep = 65536;  // hole-filling compaction: kept rows per head at most (LDS bitmap)

// Per-head row metadata written before scoring: word 0 = number of occupied
// beacon slots, words kMetaAct.. = those slots, ascending.
constexpr int kMetaAct = 16;
constexpr int kMetaWords = 128;

struct WsLayout {
    // control block
    size_t hctl;    // per-head control lines (int32 [P][kHcWords])
    size_t cflags;  // compaction: per-segment read-done flags (int32 [P][nseg])
    // selection split over several workgroups per head (0: not laid out)
    size_t tk_hist;  // int32 [P][4096] bin counts, left zero after each selection
    size_t tk_head;  // int32 [P][kTkHeadWords]
    size_t tk_cand;  // uint32 [P][512][2] threshold-bin (order key, token)
    size_t tk_cnt;   // int32 [P][kTkMaxSlices] per-slice counts
    size_t ctl_end;
    // data
    size_t part_m, part_z;  // score: per-chunk row statistics (fp32 [P][nch][R_pad_max])
    size_t lse2;            // score: row log2-normalisers (fp32 [P][R_pad_max])
    size_t rows;            // score: observation rows in MFMA operand order (bf16 [P][R_pad_max][D])
    size_t rmeta;           // score: per-head occupied-slot list (int32 [P][kMetaWords])
    size_t score_end;
    size_t scores;          // evict: scores when the caller passes none [P][N]
    size_t kept;            // evict: kept indices when the caller passes none [P][budget]
    size_t evict_end;
    int P, nseg, R_pad_max, nch, kgn, key_chunk;
    int rtg;  // score fast path: row tiles (16 rows) per row group; 0 selects the generic path
};

// The score fast path (bf16) holds the rows of one row group in registers:
// at most kFastTiles tiles per group and kFastRowGroups groups.
constexpr int kFastTiles = 9;

// Split selection: words per head, slices per head at most, heads at most
// for which the regions are laid out, and the shortest head it takes.
constexpr int kTkHeadWords = 4;
constexpr int kTkMaxSlices = 64;
constexpr int kTkMaxHeads = 64;
constexpr int kTkMinN = 8192;
constexpr int kFastRowGroups = 8;

WsLayout ws_layout(const bkv_dims& d);

// ---- the whole eviction (bkv_evict_ex), split so that a caller can check the
// arguments before it enqueues anything of its own -----------------------------
bkv_status evict_check(const bkv_dims* d, int32_t flags, const void* K, const void* V, const void* q_win,
                       const float* beacons, const int32_t* counts, const float* rope_cos, const float* rope_sin,
                       float scale);
// Arguments already checked, N > 0 and B > 0, ws holds ws_layout(d).evict_end bytes.
bkv_status evict_enqueue(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win, const float* beacons,
                         const int32_t* counts, const float* rope_cos, const float* rope_sin, float scale,
                         int32_t* kept, float* scores, float* row_lse, void* ws, hipStream_t stream);

// ---- launches (enqueue only; arguments already validated) --------------------

hipError_t launch_beacon_update(const bkv_dims& d, const void* q_new, int T, float* beacons,
                                int32_t* counts, int32_t* assign, hipStream_t s);

hipError_t launch_score(const bkv_dims& d, const WsLayout& L, int flags, const void* K, const void* q_win,
                        const float* beacons, const int32_t* counts, const float* rope_cos,
                        const float* rope_sin, float scale, float* scores, float* row_lse,
                        void* ws, hipStream_t s);

// The whole eviction in one launch (score, select and compact work items
// under one per-head ticket); only where evict_fusable (the bf16 fast path,
// heads of 16K to 32K tokens, where it measured at least as fast as the
// chained launches).  kept and scores are required (the workspace's own may
// be passed).
bool evict_fusable(const bkv_dims& d, const WsLayout& L);
hipError_t launch_evict_fused(const bkv_dims& d, const WsLayout& L, int flags, void* K, void* V, const void* q_win,
                              const float* beacons, const int32_t* counts, const float* rope_cos,
                              const float* rope_sin, float scale, float* scores, float* row_lse, int32_t* kept,
                              void* ws, hipStream_t s);

// Selection; with a workspace holding the split-selection regions (ws
// non-null, L.tk_hist set) a layer of few heads is split over several
// workgroups per head.
hipError_t launch_topk(const bkv_dims& d, const WsLayout& L, const float* scores, int32_t* kept, void* ws,
                       hipStream_t s);
hipError_t launch_compact_fill(const bkv_dims& d, void* K, void* V, const int32_t* kept, int32_t* src_of, void* ws,
                               hipStream_t s);

hipError_t launch_compact(const bkv_dims& d, const WsLayout& L, void* K, void* V,
                          const int32_t* kept, void* ws, hipStream_t s);

// FPS over H heads of src [H][src_rows][D], k = min(m, n) picks per head;
// dst (optional) receives the picked rows, counts (optional) the occupancy.
hipError_t launch_fps(int H, int n, int kmax, int D, int dtype, const void* src, int src_rows, int32_t* picks,
                      void* dst, int dst_dtype, int dst_rows, int32_t* counts, hipStream_t s);

}  // namespace bkv
