/*
 * bkv.h -- C ABI of the BeaconKV eviction step on AMD Instinct MI355X (gfx950).
 *
 * Paper: "BeaconKV: Key-Value Cache Compression Guided by Beacon Queries for
 * Efficient Large Reasoning Model Inference" (arXiv 2609.04971).
 *
 * One KV-cache layer is evicted per call, every (batch, kv-head) pair
 * independently.  Notation: P = B*Hkv heads, G = Hq/Hkv query heads per
 * kv-head, and query head hq belongs to kv-head hq / G (contiguous GQA
 * grouping).  All layouts are dense row-major with the last dimension
 * contiguous:
 *
 *   K, V      [B, Hkv, N_cap, D]  cache (post-RoPE keys), dtype of the dims
 *   q_new     [B, Hq,  T,     D]  newest pre-RoPE queries, dtype of the dims
 *   q_win     [B, Hq,  W,     D]  recent queries, already rotated at their own
 *                                 positions, dtype of the dims; any order
 *   beacons   [B, Hkv, C,     D]  fp32 beacon vectors (pre-RoPE)
 *   counts    [B, Hkv, C]         int32 members per beacon; 0 = empty slot
 *   rope_cos, rope_sin [D/2]      fp32 rotation table for the current step
 *   scores    [B, Hkv, N]         fp32 log-domain key scores
 *   row_lse   [B, Hkv, C + G*W]   fp32 per-row log-normaliser, slot-indexed
 *   kept      [B, Hkv, min(budget, N)]  int32 kept token indices, ascending
 *
 * Conventions for every entry point:
 *   - Pointers to tensors are device pointers owned by the caller.  The
 *     library allocates nothing; scratch comes from the caller's workspace
 *     (bkv_evict_noalloc alone uses a fixed array of the library instead).
 *   - Work is enqueued on `stream` and is asynchronous; no call synchronises
 *     except bkv_device_status.
 *   - Arguments are validated on the host before anything is enqueued; on an
 *     error no work is enqueued and no buffer changes.  Launch failures map to
 *     BKV_ERR_HIP.
 *   - Inputs must be finite.  Non-finite values give an unspecified ranking,
 *     but never an out-of-bounds access and always an exact kept count.
 *   - Calls that share a workspace must be ordered on one stream.
 */
#ifndef BKV_H
#define BKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BKV_OK = 0,
    BKV_ERR_INVALID = 1,   /* NULL pointer or value out of range */
    BKV_ERR_SHAPE = 2,     /* inconsistent or unsupported dimensions */
    BKV_ERR_DTYPE = 3,     /* unsupported element type */
    BKV_ERR_WORKSPACE = 4, /* workspace missing, too small or not initialised */
    BKV_ERR_HIP = 5,       /* a HIP runtime call failed */
    BKV_ERR_DEVICE = 6     /* a device-side check tripped (see bkv_device_status) */
} bkv_status;

typedef enum { BKV_F32 = 0, BKV_BF16 = 1 } bkv_dtype;

typedef enum {
    BKV_OP_BEACON_UPDATE = 0,
    BKV_OP_SCORE = 1,
    BKV_OP_TOPK = 2,
    BKV_OP_COMPACT = 3,
    BKV_OP_EVICT = 4
} bkv_op;

typedef struct {
    int32_t B;        /* batch, >= 0 (0 makes every call a no-op) */
    int32_t Hq;       /* query heads, a positive multiple of Hkv */
    int32_t Hkv;      /* kv heads, >= 1 */
    int32_t D;        /* head dimension, 64 or 128 */
    int32_t N;        /* valid cached tokens per head, 0 <= N <= N_cap */
    int32_t N_cap;    /* allocated tokens per head: the head stride of K and V */
    int32_t W;        /* recent queries per query head, and recent tokens always kept */
    int32_t C;        /* beacon slots per kv-head, 0..64 */
    int32_t budget;   /* tokens kept per kv-head (B_KV^min), >= max(1, W + n_prefix) */
    int32_t n_prefix; /* leading tokens always kept, counted inside the budget */
    int32_t dtype;    /* bkv_dtype of K, V, q_new and q_win */
} bkv_dims;

/* Host-only check of `d` for operation `op` (a bkv_op).  Enqueues nothing.
 * Rules: Hkv >= 1, Hq % Hkv == 0, D in {64, 128}, 0 <= N <= N_cap,
 * N_cap >= 1, W >= 0, 0 <= C <= 64, n_prefix >= 0,
 * budget >= max(1, W + n_prefix), dtype in {BKV_F32, BKV_BF16};
 * scoring (SCORE, EVICT) also needs 1 <= C + G*W <= 1024; the beacon
 * update needs C >= 1. */
bkv_status bkv_validate(const bkv_dims* d, int32_t op);

/* Bytes of workspace `op` needs for `d` (0 when it needs none).  One
 * workspace sized for BKV_OP_EVICT serves every operation on those dims. */
size_t bkv_workspace_bytes(const bkv_dims* d, int32_t op);

/* Enqueue the initialisation of a workspace: clears its control block and
 * stamps it with (B*Hkv, budget).  Required once after allocation, again
 * whenever B*Hkv or budget change, and after a BKV_ERR_DEVICE.  Calls in
 * between need nothing: every score launch resets its own control words
 * before its work starts, and compaction leaves its words clear.  A kernel
 * that finds a workspace not stamped for its dims does no work and raises
 * BKV_ERR_DEVICE. */
bkv_status bkv_workspace_init(const bkv_dims* d, void* ws, size_t ws_bytes, hipStream_t stream);

/* Synchronise `stream`, then report the device-side error word of `ws`:
 * BKV_OK, or BKV_ERR_DEVICE if a bounded wait timed out or the workspace
 * stamp did not match (the affected outputs are then unspecified). */
bkv_status bkv_device_status(const void* ws, size_t ws_bytes, hipStream_t stream);

/* (a1) Beacon maintenance.  For each (b, kv-head), the T*G new pre-RoPE
 * queries of its query heads are taken in order t-major, then g ascending.
 * Each one fills the lowest empty slot if there is one (count 1); otherwise
 * it joins the slot of largest cosine similarity (ties -> lowest slot;
 * cosine 0 when a norm is 0), whose count grows by one and whose vector
 * moves to the running mean: beta += (x - beta) / count.  Beacons represent
 * clusters of pre-RoPE queries under cosine similarity (Section 3.2,
 * "Beacon queries"; Section 4.2; Appendix D.1, the nearest-representative
 * similarity of Algorithm 1).
 *   q_new   [B,Hq,T,D] read;  beacons, counts  read and written in place.
 *   assign  optional [B,Hkv,T*G] int32 output: the slot each query joined,
 *           in processing order; NULL to skip.
 *   T >= 0 (0 is a no-op).  Needs no workspace. */
bkv_status bkv_beacon_update(const bkv_dims* d, const void* q_new, int32_t T, float* beacons,
                             int32_t* counts, int32_t* assign, hipStream_t stream);

/* (a2)+(a3) Scores.  Per (b, kv-head) the observation rows are: every
 * occupied beacon slot c in ascending order, rotated to the current step
 * with rotate-half RoPE (pair (i, i+D/2) turned by rope_cos[i], rope_sin[i];
 * products rounded to fp32, then the sum, no fused multiply-add) and then
 * rounded to the cache dtype (bf16: nearest-even); then the G*W recent
 * queries as given (Section 4.3, "Query Construction and Alignment";
 * Algorithm 2, the union of beacon and recent queries).  Both tables NULL
 * means no rotation.  With l_rj = scale * <y_r, k_j> (fp32 accumulation;
 * scale 0 selects fp32(1/sqrt(D))), every row is normalised over all N keys
 * (Eq. 4) and the key score is the max over rows (Eq. 6, max form;
 * Section 4.3 "Importance Scoring via Max-Aggregation"):
 *   lse_r = log sum_j exp(l_rj),   scores[j] = max_r (l_rj - lse_r) <= 0,
 * so exp(scores[j]) is the largest attention weight key j receives.  With
 * no occupied slot and W == 0 every score is -inf.
 *   row_lse optional (NULL to skip): entry c for beacon slot c (-inf when
 *           empty), entry C + g*W + w for recent query w of head h*G+g.
 *   N == 0: nothing is written.  Workspace: bkv_workspace_bytes(d, SCORE). */
bkv_status bkv_score(const bkv_dims* d, const void* K, const void* q_win, const float* beacons,
                     const int32_t* counts, const float* rope_cos, const float* rope_sin,
                     float scale, float* scores, float* row_lse, void* ws, size_t ws_bytes,
                     hipStream_t stream);

/* Scoring options (bit flags) for bkv_score_ex and bkv_evict_ex.
 *   BKV_SCORE_MEAN    the mean form of Eq. (6) instead of the max: the
 *                     paper's Table 2 ablation.  scores[j] =
 *                     ln((1/R) sum_r exp(l_rj - lse_r)) <= 0, R the number
 *                     of rows (occupied beacon slots plus G*W).
 *   BKV_SCORE_CAUSAL  the W recent queries of each query head are taken
 *                     oldest first, the last one at the current step, and
 *                     recent query w sees only the keys j <= N - W + w: its
 *                     lse runs over those keys and its weight on later keys
 *                     is 0 (a causal attention row).  Beacon rows see every
 *                     key.  A row that sees no key has row_lse -inf and
 *                     weight 0; a key that no row sees scores -inf. */
#define BKV_SCORE_MEAN 1
#define BKV_SCORE_CAUSAL 2

/* bkv_score with options; flags 0 is bkv_score.  Unknown flag bits are
 * BKV_ERR_INVALID. */
bkv_status bkv_score_ex(const bkv_dims* d, int32_t flags, const void* K, const void* q_win,
                        const float* beacons, const int32_t* counts, const float* rope_cos,
                        const float* rope_sin, float scale, float* scores, float* row_lse, void* ws,
                        size_t ws_bytes, hipStream_t stream);

/* (a4) Selection.  If N <= budget, kept = 0..N-1.  Otherwise the first
 * n_prefix and the last W tokens are always kept and the remaining
 * budget - n_prefix - W places go to the other tokens of highest score,
 * ties to the lower index (-0 equals +0); kept is emitted in ascending
 * order (Section 2.2 TopK; Algorithm 2, the I_keep, k_sel, TopK and Sort
 * steps).  scores [B,Hkv,N] read; kept [B,Hkv,min(budget,N)] written.
 * ws is optional (NULL: one workgroup per head).  With a workspace of at
 * least bkv_workspace_bytes(d, BKV_OP_TOPK) bytes (0 when the dims never
 * split), initialised by bkv_workspace_init, a layer of few heads of more
 * than 8192 tokens splits each head over several workgroups (three kernel
 * launches); the result is the same. */
bkv_status bkv_topk(const bkv_dims* d, const float* scores, int32_t* kept, void* ws,
                    size_t ws_bytes, hipStream_t stream);

/* (a5) In-place, order-preserving compaction: for i < n = min(budget, N),
 * row i of K and of V becomes original row kept[i] (Section 2.2, Eq. 8;
 * Algorithm 2, Gather after Sort), bit for bit.  kept must be strictly
 * ascending within [0, N) per head (as bkv_topk emits); rows from n on are
 * left as they were.  Workspace: bkv_workspace_bytes(d, COMPACT). */
bkv_status bkv_compact(const bkv_dims* d, void* K, void* V, const int32_t* kept, void* ws,
                       size_t ws_bytes, hipStream_t stream);

/* Hole-filling compaction: another layout for the kept set of bkv_compact.
 * For n = min(budget, N): every kept row below n stays where it is, and the
 * m-th evicted position below n (ascending) receives the m-th kept row at
 * or above n (ascending), bit for bit, so rows [0, n) of K and V hold the
 * kept set, not in token order, and only the kept rows past n move.
 * Algorithm 2 sorts and gathers (bkv_compact, order preserved); with the
 * periodic eviction of Section 5.1 (B_max -> 7/8 B_max) this layout moves
 * at most 1/8 of the cache instead of every row after the first evicted
 * one.  The forcing rules of bkv_topk still hold across evictions: prefix
 * rows are always kept and so never move, and tokens appended after an
 * eviction stay at the end in order.  Scores do not depend on row order
 * (RoPE is in the cached keys); top-k ties then go to the lower cache row.
 *   kept    [B,Hkv,n] int32 read, strictly ascending within [0, N).
 *   src_of  [B,Hkv,n] int32 written: the old row now at each row j < n
 *           (j itself for rows that stayed).
 * n <= 65536, else BKV_ERR_SHAPE.  A head whose kept indices are not
 * ascending within [0, N) moves nothing (src_of = identity) and raises
 * BKV_ERR_DEVICE.  Workspace: bkv_workspace_bytes(d, COMPACT). */
bkv_status bkv_compact_fill(const bkv_dims* d, void* K, void* V, const int32_t* kept, int32_t* src_of,
                            void* ws, size_t ws_bytes, hipStream_t stream);

/* (a6) The whole eviction of one layer: bkv_score, bkv_topk, bkv_compact in
 * order on `stream`.  scores, row_lse and kept are optional outputs (NULL:
 * scores and kept live in the workspace).  Afterwards each head holds
 * min(budget, N) rows.  Workspace: bkv_workspace_bytes(d, EVICT). */
bkv_status bkv_evict(const bkv_dims* d, void* K, void* V, const void* q_win, const float* beacons,
                     const int32_t* counts, const float* rope_cos, const float* rope_sin,
                     float scale, int32_t* kept, float* scores, float* row_lse, void* ws,
                     size_t ws_bytes, hipStream_t stream);

/* ---- Continual FPS: the paper's own beacon selection ------------------------
 * Farthest point sampling under cosine similarity (Appendix D.1, Algorithm 1)
 * of H independent query sets ("heads"), each the first n rows of
 * q [H, q_rows, D] (pre-RoPE queries, dtype BKV_BF16 or BKV_F32, row stride D,
 * head stride q_rows*D elements, 16-byte aligned).  Per head, with cos = 0
 * whenever either norm is 0:
 *   avg_i = mean over all n rows j (j = i included) of cos(q_i, q_j);
 *   the first pick is argmin_i avg_i; S_j = cos(q_j, first pick);
 *   each further pick is r = argmin over unpicked j of S_j, after which
 *   S_j <- max(S_j, cos(q_j, q_r)) for the unpicked j;
 * every argmin takes the lowest index among equal values, and the picks are
 * emitted in selection order, k = min(m, n) of them (m >= n returns every
 * row).  Cosines are computed in fp32 (exact bf16 products, fp32 sums).
 * Limits: D in {64, 128}; 0 <= n <= q_rows; n <= 32768; H, m >= 0
 * (H, n or m of 0 enqueue nothing).  Needs no workspace. */

/* picks [H, min(m, n)] int32 written: the selected row indices of each head. */
bkv_status bkv_fps(int32_t H, int32_t n, int32_t m, int32_t D, int32_t dtype, const void* q,
                   int32_t q_rows, int32_t* picks, hipStream_t stream);

/* FPS followed by the gather of the selection, which is the fill-and-compress
 * step Q_obs <- FPS(Q_obs, B_Q^min) of Section 4.2 (Eq. fps_q) and also serves
 * the prefill initialisation and the post-eviction re-selection of
 * Algorithm 2: rows 0..k-1 of each head of dst [H, dst_rows, D] become the
 * picked rows of src in selection order, k = min(m, n), converted to
 * dst_dtype (BKV_F32 always; otherwise equal to dtype), bit for bit when
 * the type is unchanged; rows k..dst_rows-1 are left as they were.
 * dst may be src itself (then dst_dtype == dtype and dst_rows == src_rows:
 * every picked row is read before any is written); any other overlap is
 * BKV_ERR_INVALID.  picks [H, k] int32 is an optional output (NULL to skip).
 * counts, optional [H, dst_rows] int32, is set to 1 for rows < k and 0 for
 * the rest, so that for H = B*Hq and dst_rows = n_beacon, dst written as
 * fp32 is directly the beacons [B, Hkv, G*n_beacon, D] and counts argument
 * of bkv_score: the union of the query heads' beacon sets of each group
 * (Algorithm 2, the group-level beacon set).  Limits: those of bkv_fps,
 * plus k <= 128 and dst_rows >= k. */
bkv_status bkv_fps_gather(int32_t H, int32_t n, int32_t m, int32_t D, int32_t dtype, const void* src,
                          int32_t src_rows, void* dst, int32_t dst_dtype, int32_t dst_rows, int32_t* picks,
                          int32_t* counts, hipStream_t stream);

/* bkv_evict with scoring options (see bkv_score_ex); flags 0 is bkv_evict. */
bkv_status bkv_evict_ex(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win,
                        const float* beacons, const int32_t* counts, const float* rope_cos,
                        const float* rope_sin, float scale, int32_t* kept, float* scores, float* row_lse,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- An eviction that allocates nothing ---------------------------------------
 * For callers that cannot allocate device memory or pass a workspace: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  bkv_evict_ex's work (flags as there; scores, kept and row_lse
 * optional outputs as there) with its workspace in a fixed array of this
 * library, BKV_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU, held from the first
 * call on that GPU until the process ends.  The call allocates nothing: no
 * hipMalloc, hipFree or allocating library routine.  Every call on a GPU
 * reuses that GPU's array, so calls that overlap in time on one GPU race:
 * order them on one stream.  Each call first re-stamps and clears the
 * array's control block with a fill kernel (no memset), so no
 * initialisation call is needed and nothing carries over between calls.
 *   device_status  optional device int32 output: BKV_OK, or BKV_ERR_DEVICE
 *                  if a device-side check of this call tripped (the outputs
 *                  are then unspecified); NULL to skip.
 * Dims whose bkv_workspace_bytes(d, BKV_OP_EVICT) exceeds the array are
 * BKV_ERR_WORKSPACE (checked on the host, nothing enqueued).  The first
 * call on a GPU looks up the array's device address (hipGetSymbolAddress);
 * failure there is BKV_ERR_HIP. */
#define BKV_NOALLOC_SCRATCH_BYTES (32u << 20)
bkv_status bkv_evict_noalloc(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win,
                             const float* beacons, const int32_t* counts, const float* rope_cos,
                             const float* rope_sin, float scale, int32_t* kept, float* scores, float* row_lse,
                             int32_t* device_status, hipStream_t stream);

/* Static description of a status code. */
const char* bkv_status_string(bkv_status s);

/* ABI version of this header, 1. */
int32_t bkv_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BKV_H */
