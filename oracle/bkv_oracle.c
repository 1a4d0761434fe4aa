/*
 * CPU oracle for the BeaconKV eviction step -- TEST INFRASTRUCTURE ONLY.
 *
 * This file is the plain, slow, obviously-correct statement of what the GPU
 * library computes.  It exists so that tests, the smoke check and the
 * benchmark's CPU baseline can compare against it.  Product code never links,
 * loads or calls it, and it shares no source with the GPU path.
 *
 * Paper: "BeaconKV: Key-Value Cache Compression Guided by Beacon Queries for
 * Efficient Large Reasoning Model Inference" (arXiv 2609.04971).
 *
 * Everything is computed per (batch, kv-head) pair on the exact values of
 * the inputs (bf16 and fp32 widen exactly to double); arithmetic is double
 * precision unless a step is defined in fp32 below.  Build with
 * -ffp-contract=off: the RoPE step relies on separately rounded fp32
 * multiplies and adds.
 *
 * Pins (what checks this file against something other than itself) live in
 * tests/test_oracle_*.py: hand-worked examples, closed forms, library
 * special cases (scipy log_softmax, numpy mean), brute force and invariants.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_BF16 1

/* ---- element access --------------------------------------------------- */

/* bf16 is the upper half of an IEEE binary32, so widening is a shift. */
static float bf16_bits_to_float(uint16_t h) {
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Round a binary32 to the nearest bf16, ties to even (NaN stays NaN). */
static float round_to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) {
        u |= 0x00400000u; /* quiet NaN */
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    float r;
    memcpy(&r, &u, sizeof r);
    return r;
}

static double elem(const void* base, size_t i, int dtype) {
    if (dtype == ORC_BF16) return (double)bf16_bits_to_float(((const uint16_t*)base)[i]);
    return (double)((const float*)base)[i];
}

/* ---- (a1) beacon maintenance --------------------------------------------
 *
 * Beacons are representatives of clusters of pre-RoPE queries compared by
 * cosine similarity (Section 3.2 "Beacon queries"; the cosine geometry of
 * Section 4.2 and the nearest-representative similarity S_j of Appendix D.1,
 * Algorithm 1).  The online rule built here: every new query joins the beacon
 * it is most cosine-similar to and that beacon becomes the running mean of
 * its members (sequential k-means; a streaming form of the "K-Means
 * Centroids" selector the paper compares in Figure 7).  Empty slots are
 * seeded first, lowest slot first, so counts always sum to queries seen.
 *
 * One kv-head: q_block holds the G query heads of the group, [G][T][D];
 * queries are taken in order t-major, then g ascending, and each one sees
 * the beacons left by the previous one.  cos(x, b) = x.b / (|x||b|), and 0
 * when either norm is 0.  argmax ties go to the lowest slot.  A near tie
 * (best two cosines within 1e-6) is flagged in near_tie.
 * The mean is formed in double and stored back to fp32 after every query.
 * ------------------------------------------------------------------------ */
int orc_beacon_update(int dtype, int D, int C, int G, int T, const void* q_block,
                      float* beacons, int32_t* counts, int32_t* assign, int32_t* near_tie) {
    if (D <= 0 || C <= 0 || G <= 0 || T < 0) return -1;
    double* x = (double*)malloc(sizeof(double) * (size_t)D);
    if (!x) return -2;
    int q = 0;
    for (int t = 0; t < T; ++t) {
        for (int g = 0; g < G; ++g, ++q) {
            for (int d = 0; d < D; ++d) x[d] = elem(q_block, ((size_t)g * T + t) * D + d, dtype);
            int chosen = -1, tie = 0;
            for (int c = 0; c < C; ++c) {
                if (counts[c] == 0) { chosen = c; break; }
            }
            if (chosen >= 0) {
                for (int d = 0; d < D; ++d) beacons[(size_t)chosen * D + d] = (float)x[d];
                counts[chosen] = 1;
            } else {
                double xn = 0.0;
                for (int d = 0; d < D; ++d) xn += x[d] * x[d];
                xn = sqrt(xn);
                double best = -INFINITY, second = -INFINITY;
                for (int c = 0; c < C; ++c) {
                    const float* b = beacons + (size_t)c * D;
                    double dot = 0.0, bn = 0.0;
                    for (int d = 0; d < D; ++d) {
                        dot += x[d] * (double)b[d];
                        bn += (double)b[d] * (double)b[d];
                    }
                    bn = sqrt(bn);
                    double cs = (xn == 0.0 || bn == 0.0) ? 0.0 : dot / (xn * bn);
                    if (cs > best) {
                        second = best;
                        best = cs;
                        chosen = c;
                    } else if (cs > second) {
                        second = cs;
                    }
                }
                tie = (C > 1) && (best - second <= 1e-6);
                int32_t n = ++counts[chosen];
                float* b = beacons + (size_t)chosen * D;
                for (int d = 0; d < D; ++d) {
                    double bd = (double)b[d];
                    b[d] = (float)(bd + (x[d] - bd) / (double)n);
                }
            }
            if (assign) assign[q] = chosen;
            if (near_tie) near_tie[q] = tie;
        }
    }
    free(x);
    return 0;
}

/* ---- (a2) observation rows ------------------------------------------------
 *
 * Beacon queries are rotated to the current step t, recent queries keep their
 * own positions (Section 4.3 "Query Construction and Alignment"; Algorithm 2,
 * the construction of Q_obs).  Recent queries arrive already rotated.  RoPE is
 * the rotate-half form: pair (d, d + D/2) is turned by the angle whose
 * cosine and sine the caller tabulates for step t.
 *
 * Reading of the precision: each product is rounded to fp32, then the sum or
 * difference is rounded to fp32 (no fused multiply-add), and for bf16 caches
 * the row is then rounded to bf16 (nearest, ties to even).  A NULL table is
 * the identity.  Only occupied slots (count > 0) become rows, in slot order;
 * the G*W recent rows follow, g-major, w-minor.
 * ------------------------------------------------------------------------ */
void orc_rope_row(int D, const float* beta, const float* cos_t, const float* sin_t, int to_bf16,
                  float* out) {
    int h = D / 2;
    for (int d = 0; d < h; ++d) {
        float lo, hi;
        if (cos_t && sin_t) {
            float a = beta[d] * cos_t[d];
            float b = beta[d + h] * sin_t[d];
            float c = beta[d + h] * cos_t[d];
            float e = beta[d] * sin_t[d];
            lo = a - b;
            hi = c + e;
        } else {
            lo = beta[d];
            hi = beta[d + h];
        }
        out[d] = to_bf16 ? round_to_bf16(lo) : lo;
        out[d + h] = to_bf16 ? round_to_bf16(hi) : hi;
    }
}

/* Y is [(C + G*W)][D]; row_slot[r] names the slot a row came from: the
 * beacon index c, or C + g*W + w for a recent query.  Returns R. */
int orc_assemble_rows(int dtype, int D, int C, int G, int W, const float* beacons,
                      const int32_t* counts, const float* cos_t, const float* sin_t,
                      const void* qwin_block, double* Y, int32_t* row_slot) {
    float* tmp = (float*)malloc(sizeof(float) * (size_t)D);
    if (!tmp) return -2;
    int r = 0;
    for (int c = 0; c < C; ++c) {
        if (counts[c] <= 0) continue;
        orc_rope_row(D, beacons + (size_t)c * D, cos_t, sin_t, dtype == ORC_BF16, tmp);
        for (int d = 0; d < D; ++d) Y[(size_t)r * D + d] = (double)tmp[d];
        row_slot[r++] = c;
    }
    for (int g = 0; g < G; ++g) {
        for (int w = 0; w < W; ++w) {
            for (int d = 0; d < D; ++d)
                Y[(size_t)r * D + d] = elem(qwin_block, ((size_t)g * W + w) * D + d, dtype);
            row_slot[r++] = C + g * W + w;
        }
    }
    free(tmp);
    return r;
}

/* ---- (a3) scores -------------------------------------------------------------
 *
 * Attention weight of observation row r on cached key j (Eq. 4):
 *   w_rj = exp(l_rj) / sum_l exp(l_rl),   l_rj = scale * <y_r, k_j>,
 * normalised over all N cached keys.  The key score is the max of w_rj over
 * every observation row, i.e. over all queries and all heads of the GQA group
 * (Eq. 6, max form; Section 4.3 "Importance Scoring via Max-Aggregation";
 * Algorithm 2, the Score step).  It is kept in the log domain:
 *   lse_r = m_r + ln sum_j exp(l_rj - m_r),   m_r = max_j l_rj,
 *   s_j   = max_r (l_rj - lse_r),  so exp(s_j) = max_r w_rj.
 * With no rows at all every s_j is -inf.
 * ------------------------------------------------------------------------ */
/* Scoring variants (the next step after the max form).
 *
 * agg = 1 takes the other aggregation Eq. (6) defines, the mean over the
 * observation queries, s_j^mean = (1/R) sum_r w_rj (the paper ablates it
 * against the max in Table 2), kept in the log domain as
 *   s_j = ln((1/R) sum_r exp(l_rj - lse_r)).
 * With `limit` given, row r sees only the keys j <= limit[r] (a causal
 * restriction for recent queries): its lse runs over those keys alone and
 * its weight on every later key is 0.  A row that sees no key has
 * lse = -inf and weight 0 everywhere; R still counts it in the mean.  A key
 * no row sees scores -inf.  agg = 0, limit = NULL is orc_score.
 */
int orc_score_ex(int R, int N, int D, const double* Y, const void* Khead, int dtype, double scale, int agg,
                 const int32_t* limit, double* lse, double* s) {
    if (R == 0) {
        for (int j = 0; j < N; ++j) s[j] = -INFINITY;
        return 0;
    }
    double* logit = (double*)malloc(sizeof(double) * (size_t)R * (size_t)(N > 0 ? N : 1));
    double* krow = (double*)malloc(sizeof(double) * (size_t)D);
    if (!logit || !krow) {
        free(logit);
        free(krow);
        return -2;
    }
    for (int j = 0; j < N; ++j) {
        for (int d = 0; d < D; ++d) krow[d] = elem(Khead, (size_t)j * D + d, dtype);
        for (int r = 0; r < R; ++r) {
            double dot = 0.0;
            for (int d = 0; d < D; ++d) dot += Y[(size_t)r * D + d] * krow[d];
            logit[(size_t)r * N + j] = scale * dot;
        }
    }
    /* keys j < seen(r) are the ones row r sees */
#define ORC_SEEN(r) (limit ? (limit[r] + 1 < 0 ? 0 : (limit[r] + 1 < N ? limit[r] + 1 : N)) : N)
    for (int r = 0; r < R; ++r) {
        const double* l = logit + (size_t)r * N;
        const int n = ORC_SEEN(r);
        double m = -INFINITY;
        for (int j = 0; j < n; ++j)
            if (l[j] > m) m = l[j];
        double z = 0.0;
        for (int j = 0; j < n; ++j) z += exp(l[j] - m);
        lse[r] = (n > 0) ? m + log(z) : -INFINITY;
    }
    for (int j = 0; j < N; ++j) {
        double best = -INFINITY, sum = 0.0;
        for (int r = 0; r < R; ++r) {
            if (j >= ORC_SEEN(r)) continue;
            const double v = logit[(size_t)r * N + j] - lse[r];
            if (v > best) best = v;
            sum += exp(v);
        }
        s[j] = agg ? log(sum / (double)R) : best;
    }
#undef ORC_SEEN
    free(logit);
    free(krow);
    return 0;
}

int orc_score(int R, int N, int D, const double* Y, const void* Khead, int dtype, double scale,
              double* lse, double* s) {
    return orc_score_ex(R, N, D, Y, Khead, dtype, scale, 0, NULL, lse, s);
}

/* Score one kv-head from raw inputs: rows (a2) then (a3).  lse_slot is
 * indexed by slot (C beacon slots, then G*W recent rows); empty beacon
 * slots read -inf. */
/* causal = 1 limits recent query w of each query head (slot C + g*W + w,
 * the W recent queries taken oldest first, the newest at the current step
 * N - 1) to the keys up to its own position N - W + w; beacon rows see all
 * keys. */
int orc_score_head_ex(int dtype, int D, int N, int C, int G, int W, const void* Khead,
                      const void* qwin_block, const float* beacons, const int32_t* counts,
                      const float* cos_t, const float* sin_t, float scale, int agg, int causal,
                      double* lse_slot, double* s) {
    int Rmax = C + G * W;
    double* Y = (double*)malloc(sizeof(double) * (size_t)(Rmax > 0 ? Rmax : 1) * D);
    int32_t* slot = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Rmax > 0 ? Rmax : 1));
    int32_t* limit = (int32_t*)malloc(sizeof(int32_t) * (size_t)(Rmax > 0 ? Rmax : 1));
    double* lse = (double*)malloc(sizeof(double) * (size_t)(Rmax > 0 ? Rmax : 1));
    if (!Y || !slot || !limit || !lse) {
        free(Y);
        free(slot);
        free(limit);
        free(lse);
        return -2;
    }
    int R = orc_assemble_rows(dtype, D, C, G, W, beacons, counts, cos_t, sin_t, qwin_block, Y, slot);
    for (int r = 0; r < R; ++r) limit[r] = (slot[r] < C) ? N - 1 : N - W + (slot[r] - C) % W;
    double sc = (scale == 0.0f) ? (double)(float)(1.0 / sqrt((double)D)) : (double)scale;
    int rc = orc_score_ex(R, N, D, Y, Khead, dtype, sc, agg, causal ? limit : NULL, lse, s);
    for (int i = 0; i < Rmax; ++i) lse_slot[i] = -INFINITY;
    for (int r = 0; r < R; ++r) lse_slot[slot[r]] = lse[r];
    free(Y);
    free(slot);
    free(limit);
    free(lse);
    return rc;
}

int orc_score_head(int dtype, int D, int N, int C, int G, int W, const void* Khead,
                   const void* qwin_block, const float* beacons, const int32_t* counts,
                   const float* cos_t, const float* sin_t, float scale, double* lse_slot,
                   double* s) {
    return orc_score_head_ex(dtype, D, N, C, G, W, Khead, qwin_block, beacons, counts, cos_t, sin_t, scale, 0,
                             0, lse_slot, s);
}

/* ---- (a4) selection -------------------------------------------------------
 *
 * Forced keep = the first n_prefix tokens and the last W tokens; the rest of
 * the budget, k_sel = budget - |forced|, goes to the best-scoring other
 * tokens, and the result is sorted (Section 2.2 TopK; Algorithm 2, the
 * I_keep / k_sel / TopK / Sort steps).  "Best" is the order (score
 * descending, index ascending): ties go to the lower index.  If N <= budget
 * every token is kept.  Returns the number kept, min(budget, N).
 * ------------------------------------------------------------------------ */
typedef struct {
    double s;
    int32_t idx;
} orc_cand;

static int orc_cand_cmp(const void* pa, const void* pb) {
    const orc_cand* a = (const orc_cand*)pa;
    const orc_cand* b = (const orc_cand*)pb;
    if (a->s > b->s) return -1;
    if (a->s < b->s) return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

int orc_topk(int N, const double* s, int budget, int W, int n_prefix, int32_t* kept) {
    if (N <= budget) {
        for (int j = 0; j < N; ++j) kept[j] = j;
        return N;
    }
    unsigned char* keep = (unsigned char*)calloc((size_t)N, 1);
    orc_cand* cand = (orc_cand*)malloc(sizeof(orc_cand) * (size_t)N);
    if (!keep || !cand) {
        free(keep);
        free(cand);
        return -2;
    }
    int nforced = 0;
    for (int j = 0; j < N; ++j) {
        if (j < n_prefix || j >= N - W) {
            keep[j] = 1;
            ++nforced;
        }
    }
    int ncand = 0;
    for (int j = 0; j < N; ++j) {
        if (!keep[j]) {
            cand[ncand].s = s[j];
            cand[ncand].idx = j;
            ++ncand;
        }
    }
    qsort(cand, (size_t)ncand, sizeof(orc_cand), orc_cand_cmp);
    int ksel = budget - nforced;
    for (int i = 0; i < ksel && i < ncand; ++i) keep[cand[i].idx] = 1;
    int n = 0;
    for (int j = 0; j < N; ++j)
        if (keep[j]) kept[n++] = j;
    free(keep);
    free(cand);
    return n;
}

/* ---- (a5) compaction ---------------------------------------------------
 *
 * Gather along the sequence axis, K^ = K[:, I, :] and V^ = V[:, I, :]
 * (Section 2.2, Eq. 8; Algorithm 2, Gather after Sort).  Rows are copied
 * bit for bit from a snapshot of the original head, so the in-place result
 * equals the out-of-place gather.  Rows at n_keep and beyond are untouched.
 * ------------------------------------------------------------------------ */
int orc_compact(int esize, int D, int n_keep, const int32_t* kept, void* Khead, void* Vhead) {
    size_t row = (size_t)esize * (size_t)D;
    unsigned char* tk = (unsigned char*)malloc(row * (size_t)(n_keep > 0 ? n_keep : 1));
    unsigned char* tv = (unsigned char*)malloc(row * (size_t)(n_keep > 0 ? n_keep : 1));
    if (!tk || !tv) {
        free(tk);
        free(tv);
        return -2;
    }
    for (int i = 0; i < n_keep; ++i) {
        memcpy(tk + row * i, (unsigned char*)Khead + row * (size_t)kept[i], row);
        memcpy(tv + row * i, (unsigned char*)Vhead + row * (size_t)kept[i], row);
    }
    memcpy(Khead, tk, row * (size_t)n_keep);
    memcpy(Vhead, tv, row * (size_t)n_keep);
    free(tk);
    free(tv);
    return 0;
}

/* ---- hole-filling compaction: another layout for the same kept set -----
 *
 * Algorithm 2 sorts the kept indices and gathers, so the cache stays in
 * token order (orc_compact).  This variant leaves every kept row that lies
 * below n_keep where it is and moves only the kept rows at or above n_keep:
 * the m-th evicted position below n_keep (ascending) receives the m-th kept
 * row at or above n_keep (ascending).  Rows [0, n_keep) then hold the kept
 * set, not in token order; src_of[j] (j < n_keep) is the old position of
 * the row now at j.  kept must be strictly ascending within [0, N).
 * Returns the number of rows moved, or a negative error. */
int orc_compact_fill(int esize, int D, int N, int n_keep, const int32_t* kept, void* Khead, void* Vhead,
                     int32_t* src_of) {
    size_t row = (size_t)esize * (size_t)D;
    for (int i = 0; i < n_keep; ++i)
        if (kept[i] < 0 || kept[i] >= N || (i > 0 && kept[i] <= kept[i - 1])) return -1;
    unsigned char* in_place = (unsigned char*)calloc((size_t)(n_keep > 0 ? n_keep : 1), 1);
    if (!in_place) return -2;
    int c = 0;  /* kept rows already below n_keep: the first c entries of kept */
    while (c < n_keep && kept[c] < n_keep) in_place[kept[c++]] = 1;
    int m = 0;  /* holes filled so far */
    for (int p = 0; p < n_keep; ++p) {
        if (in_place[p]) {
            src_of[p] = p;
            continue;
        }
        const int src = kept[c + m++];
        memcpy((unsigned char*)Khead + row * (size_t)p, (unsigned char*)Khead + row * (size_t)src, row);
        memcpy((unsigned char*)Vhead + row * (size_t)p, (unsigned char*)Vhead + row * (size_t)src, row);
        src_of[p] = src;
    }
    free(in_place);
    return m;
}

/* ---- (a6) the whole eviction of one kv-head: (a2) -> (a3) -> (a4) -> (a5).
 * Returns the number of rows kept (or a negative error). */
int orc_evict_head_ex(int dtype, int D, int N, int C, int G, int W, int budget, int n_prefix,
                      void* Khead, void* Vhead, const void* qwin_block, const float* beacons,
                      const int32_t* counts, const float* cos_t, const float* sin_t, float scale, int agg,
                      int causal, double* lse_slot, double* s, int32_t* kept) {
    int rc = orc_score_head_ex(dtype, D, N, C, G, W, Khead, qwin_block, beacons, counts, cos_t,
                               sin_t, scale, agg, causal, lse_slot, s);
    if (rc) return rc;
    int n = orc_topk(N, s, budget, W, n_prefix, kept);
    if (n < 0) return n;
    rc = orc_compact(dtype == ORC_BF16 ? 2 : 4, D, n, kept, Khead, Vhead);
    return rc ? rc : n;
}

int orc_evict_head(int dtype, int D, int N, int C, int G, int W, int budget, int n_prefix,
                   void* Khead, void* Vhead, const void* qwin_block, const float* beacons,
                   const int32_t* counts, const float* cos_t, const float* sin_t, float scale,
                   double* lse_slot, double* s, int32_t* kept) {
    return orc_evict_head_ex(dtype, D, N, C, G, W, budget, n_prefix, Khead, Vhead, qwin_block, beacons, counts,
                             cos_t, sin_t, scale, 0, 0, lse_slot, s, kept);
}

/* ---- farthest point sampling over pre-RoPE queries ----------------------
 *
 * Appendix D.1 (Algorithm 1), the selection step of Continual FPS
 * (Section 4.2; Algorithm 2 calls it as FPS(Q, B_Q^min)).  From n queries
 * of dimension D pick min(m, n) of them, in selection order:
 *
 *   avg_i = (1/n) sum_j cos(q_i, q_j)     (j = i included)
 *   p     = argmin_i avg_i                (first pick)
 *   S_j   = cos(q_j, q_p)
 *   then repeatedly r = argmin over unpicked j of S_j, pick r, and
 *   S_j <- max(S_j, cos(q_j, q_r)) for the unpicked j.
 *
 * cos(x, y) = x.y / (|x| |y|), taken as 0 when either norm is 0.  Ties go
 * to the lowest index.  The cosines are computed here pairwise, straight
 * from the definition (O(n^2 D)).
 *
 * forced (optional): a selection to follow instead of the argmins, as long
 * as each forced pick is within tie_tol of that step's minimum (else the
 * function returns -(step + 1)); near_tie (optional) flags the steps whose
 * minimum is shared, within tie_tol, by another candidate.  This lets a
 * test check a selection made in another precision step by step.
 * Returns the number of picks.
 */
static double orc_cos(const void* q, int dtype, int D, int i, int j) {
    double dot = 0.0, ni = 0.0, nj = 0.0;
    for (int d = 0; d < D; ++d) {
        const double a = elem(q, (size_t)i * D + d, dtype), b = elem(q, (size_t)j * D + d, dtype);
        dot += a * b;
        ni += a * a;
        nj += b * b;
    }
    if (ni == 0.0 || nj == 0.0) return 0.0;
    return dot / (sqrt(ni) * sqrt(nj));
}

int orc_fps(int dtype, int D, int n, int m, const void* q, const int32_t* forced, double tie_tol,
            int32_t* out, int32_t* near_tie) {
    const int k_max = m < n ? m : n;
    if (k_max <= 0) return 0;
    double* val = (double*)malloc(sizeof(double) * (size_t)n);
    unsigned char* picked = (unsigned char*)calloc((size_t)n, 1);
    if (!val || !picked) {
        free(val);
        free(picked);
        return -1000000;
    }
    /* average cosine of each query against all of them */
    for (int i = 0; i < n; ++i) {
        double s = 0.0;
        for (int j = 0; j < n; ++j) s += orc_cos(q, dtype, D, i, j);
        val[i] = s / (double)n;
    }
    int rc = k_max;
    for (int k = 0; k < k_max; ++k) {
        /* the step's minimum over unpicked candidates (val = avg for the
           first pick, S afterwards), lowest index on ties */
        int best = -1;
        for (int j = 0; j < n; ++j)
            if (!picked[j] && (best < 0 || val[j] < val[best])) best = j;
        int tie = 0;
        for (int j = 0; j < n; ++j)
            if (!picked[j] && j != best && val[j] <= val[best] + tie_tol) tie = 1;
        int r = best;
        if (forced) {
            r = forced[k];
            if (r < 0 || r >= n || picked[r] || val[r] > val[best] + tie_tol) {
                rc = -(k + 1);
                break;
            }
        }
        out[k] = r;
        if (near_tie) near_tie[k] = tie;
        picked[r] = 1;
        /* nearest-picked similarity: S_j = cos(q_j, q_r) after the first
           pick, then the running maximum */
        for (int j = 0; j < n; ++j) {
            if (picked[j]) continue;
            const double c = orc_cos(q, dtype, D, j, r);
            val[j] = (k == 0) ? c : (c > val[j] ? c : val[j]);
        }
    }
    free(val);
    free(picked);
    return rc;
}
