/*
 * CPU oracle for the DualGCN aggregation path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, single-threaded C99 that states what the path computes, for the
 * parity tests, the smoke check and the CPU baseline of the benchmark.  It
 * shares no code, header or constant table with the GPU library and must never
 * be called by it.  Built with -O2 -ffp-contract=off, no fast-math.
 *
 * Contents
 *   philox4x64_10      counter-based generator of Salmon, Moraes, Dror & Shaw,
 *                      "Parallel random numbers: as easy as 1, 2, 3" (SC'11),
 *                      Philox-4x64 with 10 rounds, written from that paper.
 *   oracle_walk        one anonymous random walk (Sec. 3.2, "Theoretical
 *                      Foundation"): step to uniformly drawn neighbours and label
 *                      each visited node by the order of its first occurrence.
 *   oracle_density     S_v = sum over the k walks of v of the number of distinct
 *                      nodes, so the neighbour density of Sec. 3.2 is
 *                      N_v = sum_i i P_i = S_v / k (Theorem 1).
 *   oracle_spmm_rows   y_i = sum_p val_p x_{col_p} in float64 (the aggregation
 *                      SpMM of Sec. 1 / Sec. 2.1) with its magnitude bound
 *                      b_i = sum_p |val_p| |x_{col_p}|.
 *   oracle_xw_rows     t_i = x_i W in float64 (the update phase, Sec. 1) with
 *                      its magnitude bound |x_i| |W|.
 *
 * Random stream of a walk (the paper does not say how a neighbour is drawn):
 * walk w of node v takes, at step s (0-based), the 32-bit half r of 64-bit
 * word floor(s/2) mod 4 of the Philox block with counter (v, w, floor(s/8), 0)
 * and key (seed, 0) -- the low half for even s, the high half for odd s --;
 * the neighbour is entry floor(r * deg / 2^32) of the current row, i.e.
 * uniform over the row's entries as stored (self-loops and duplicates
 * included).  One block serves eight steps.  A row with no entries keeps the
 * walk in place.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

/* ---------------- Philox-4x64-10 (Salmon et al., SC'11) ---------------- */

/* Round multipliers and key increments of Philox-4x64 as published. */
#define PHILOX_M0 0xD2E7470EE14C6C93ULL
#define PHILOX_M1 0xCA5A826395121157ULL
#define PHILOX_W0 0x9E3779B97F4A7C15ULL /* golden ratio */
#define PHILOX_W1 0xBB67AE8584CAA73BULL /* sqrt(3) - 1 */

static void mul_hi_lo(uint64_t a, uint64_t b, uint64_t *hi, uint64_t *lo)
{
    /* schoolbook 64x64 -> 128 product on 32-bit halves */
    uint64_t a0 = a & 0xFFFFFFFFu, a1 = a >> 32;
    uint64_t b0 = b & 0xFFFFFFFFu, b1 = b >> 32;
    uint64_t p00 = a0 * b0, p01 = a0 * b1, p10 = a1 * b0, p11 = a1 * b1;
    uint64_t mid = (p00 >> 32) + (p01 & 0xFFFFFFFFu) + (p10 & 0xFFFFFFFFu);
    *lo = (p00 & 0xFFFFFFFFu) | (mid << 32);
    *hi = p11 + (p01 >> 32) + (p10 >> 32) + (mid >> 32);
}

void philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t hi0, lo0, hi1, lo1;
        mul_hi_lo(PHILOX_M0, x0, &hi0, &lo0);
        mul_hi_lo(PHILOX_M1, x2, &hi1, &lo1);
        uint64_t y0 = hi1 ^ x1 ^ k0;
        uint64_t y1 = lo1;
        uint64_t y2 = hi0 ^ x3 ^ k1;
        uint64_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* floor(r * m / 2^32): maps a uniform 32-bit word onto [0, m), m < 2^32. */
static uint64_t scale_half(uint32_t r, uint64_t m)
{
    return ((uint64_t)r * m) >> 32;
}

/* ---------------- anonymous random walks (Sec. 3.2) ---------------- */

/* labels are bytes, so a walk has at most 255 steps (256 labels) */
#define ORACLE_MAX_STEPS 255

/*
 * Walk `walk` from `start`, `steps` steps.  Returns the number of distinct
 * nodes visited (start included).  If `labels` is not NULL it receives the
 * anonymous walk: labels[s] = 1 + (index of the s-th visited node in the list
 * of distinct nodes in order of first visit), for s = 0..steps.
 */
uint32_t oracle_walk(const int32_t *rowptr, const int32_t *col, int32_t n,
                     int32_t start, uint32_t walk, uint64_t seed, uint32_t steps,
                     uint8_t *labels)
{
    (void)n;
    int32_t seen[ORACLE_MAX_STEPS + 1];
    uint32_t distinct = 0;
    if (steps > ORACLE_MAX_STEPS) return 0;
    int32_t cur = start;
    seen[distinct++] = cur;
    if (labels) labels[0] = 1;
    uint64_t key[2] = {seed, 0};
    uint64_t block[4] = {0, 0, 0, 0};
    for (uint32_t s = 0; s < steps; ++s) {
        if (s % 8 == 0) {
            uint64_t ctr[4] = {(uint64_t)(uint32_t)start, walk, s / 8, 0};
            philox4x64_10(ctr, key, block);
        }
        uint64_t word = block[(s / 2) % 4];
        uint32_t r = (s % 2 == 0) ? (uint32_t)(word & 0xFFFFFFFFu) : (uint32_t)(word >> 32);
        int64_t deg = (int64_t)rowptr[cur + 1] - rowptr[cur];
        int32_t next = cur;
        if (deg > 0)
            next = col[rowptr[cur] + (int64_t)scale_half(r, (uint64_t)deg)];
        uint32_t label = 0;
        for (uint32_t i = 0; i < distinct; ++i)
            if (seen[i] == next) { label = i + 1; break; }
        if (label == 0) {
            seen[distinct++] = next;
            label = distinct;
        }
        if (labels) labels[s + 1] = (uint8_t)label;
        cur = next;
    }
    return distinct;
}

/* S[i] = sum over walks w < k of the distinct-node count of walk w from nodes[i]. */
void oracle_density(const int32_t *rowptr, const int32_t *col, int32_t n,
                    uint64_t seed, uint32_t k, uint32_t steps,
                    const int32_t *nodes, int64_t count, uint32_t *S)
{
    for (int64_t i = 0; i < count; ++i) {
        uint32_t total = 0;
        for (uint32_t w = 0; w < k; ++w)
            total += oracle_walk(rowptr, col, n, nodes[i], w, seed, steps, NULL);
        S[i] = total;
    }
}

/* out[(v*k + w)*(steps+1) + s] = labels of walk w from node v, for every node. */
void oracle_patterns(const int32_t *rowptr, const int32_t *col, int32_t n,
                     uint64_t seed, uint32_t k, uint32_t steps, uint8_t *out)
{
    for (int32_t v = 0; v < n; ++v)
        for (uint32_t w = 0; w < k; ++w)
            oracle_walk(rowptr, col, n, v, w, seed, steps,
                        out + ((int64_t)v * k + w) * (steps + 1));
}

/* ---------------- aggregation SpMM (Sec. 1, Sec. 2.1) ---------------- */

/*
 * For each listed row r = rows[i]:
 *   Y[i*F + f] = sum_{p in row r} val[p] * X[col[p]*F + f]          (float64)
 *   B[i*F + f] = sum_{p in row r} |val[p]| * |X[col[p]*F + f]|      (float64)
 * B may be NULL.
 */
void oracle_spmm_rows(const int32_t *rowptr, const int32_t *col, const float *val,
                      const float *X, int32_t F, const int32_t *rows, int64_t count,
                      double *Y, double *B)
{
    for (int64_t i = 0; i < count; ++i) {
        int32_t r = rows[i];
        double *y = Y + i * (int64_t)F;
        double *b = B ? B + i * (int64_t)F : NULL;
        for (int32_t f = 0; f < F; ++f) {
            y[f] = 0.0;
            if (b) b[f] = 0.0;
        }
        for (int64_t p = rowptr[r]; p < rowptr[r + 1]; ++p) {
            double a = (double)val[p];
            const float *x = X + (int64_t)col[p] * F;
            for (int32_t f = 0; f < F; ++f) {
                y[f] += a * (double)x[f];
                if (b) b[f] += fabs(a) * fabs((double)x[f]);
            }
        }
    }
}

/* Same product with a float64 right operand (used to chain GCN layers). */
void oracle_spmm_rows_f64(const int32_t *rowptr, const int32_t *col, const float *val,
                          const double *X, int32_t F, const int32_t *rows, int64_t count,
                          const int64_t *slot, double *Y)
{
    /* slot[c] = row of X holding node c (X is compacted to the needed nodes) */
    for (int64_t i = 0; i < count; ++i) {
        int32_t r = rows[i];
        double *y = Y + i * (int64_t)F;
        for (int32_t f = 0; f < F; ++f) y[f] = 0.0;
        for (int64_t p = rowptr[r]; p < rowptr[r + 1]; ++p) {
            double a = (double)val[p];
            const double *x = X + slot[col[p]] * F;
            for (int32_t f = 0; f < F; ++f) y[f] += a * x[f];
        }
    }
}

/* ---------------- update phase X W (Sec. 1) ---------------- */

/*
 * For each listed row r = rows[i]:
 *   T[i*Fout + j]  = sum_c X[r*Fin + c] * W[c*Fout + j]        (float64)
 *   BT[i*Fout + j] = sum_c |X[r*Fin + c]| * |W[c*Fout + j]|    (may be NULL)
 */
void oracle_xw_rows(const float *X, const float *W, int32_t Fin, int32_t Fout,
                    const int32_t *rows, int64_t count, double *T, double *BT)
{
    for (int64_t i = 0; i < count; ++i) {
        const float *x = X + (int64_t)rows[i] * Fin;
        double *t = T + i * (int64_t)Fout;
        double *bt = BT ? BT + i * (int64_t)Fout : NULL;
        for (int32_t j = 0; j < Fout; ++j) {
            double s = 0.0, m = 0.0;
            for (int32_t c = 0; c < Fin; ++c) {
                double a = (double)x[c], w = (double)W[(int64_t)c * Fout + j];
                s += a * w;
                m += fabs(a) * fabs(w);
            }
            t[j] = s;
            if (bt) bt[j] = m;
        }
    }
}
