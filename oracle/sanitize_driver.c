/*
 * Runs every function of oracle.c on small graphs, edge cases included (an empty
 * row, a single node, repeated columns, a hub, the longest walks), for a build with
 * AddressSanitizer and UndefinedBehaviorSanitizer: any out-of-bounds access,
 * overflow or uninitialised shift aborts the run.  Test infrastructure only.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

uint32_t oracle_walk(const int32_t *rowptr, const int32_t *col, int32_t n, int32_t start,
                     uint32_t walk, uint64_t seed, uint32_t steps, uint8_t *labels);
void oracle_density(const int32_t *rowptr, const int32_t *col, int32_t n, uint64_t seed,
                    uint32_t k, uint32_t steps, const int32_t *nodes, int64_t count, uint32_t *S);
void oracle_patterns(const int32_t *rowptr, const int32_t *col, int32_t n, uint64_t seed,
                     uint32_t k, uint32_t steps, uint8_t *out);
void oracle_spmm_rows(const int32_t *rowptr, const int32_t *col, const float *val,
                      const float *X, int32_t F, const int32_t *rows, int64_t count,
                      double *Y, double *B);
void oracle_spmm_rows_f64(const int32_t *rowptr, const int32_t *col, const float *val,
                          const double *X, int32_t F, const int32_t *rows, int64_t count,
                          const int64_t *slot, double *Y);
void oracle_xw_rows(const float *X, const float *W, int32_t Fin, int32_t Fout,
                    const int32_t *rows, int64_t count, double *T, double *BT);

static int32_t *alloc_i32(size_t n) { return (int32_t *)malloc(sizeof(int32_t) * (n ? n : 1)); }

/* a hub (node 0 linked to all), a repeated column, an empty row, self-loops elsewhere */
static void build(int32_t n, int32_t **rowptr, int32_t **col, float **val, int64_t *nnz) {
    int64_t cap = 4 * (int64_t)n + 8, e = 0;
    *rowptr = alloc_i32((size_t)n + 1);
    *col = alloc_i32((size_t)cap);
    (*rowptr)[0] = 0;
    for (int32_t r = 0; r < n; ++r) {
        if (r == 0) {
            for (int32_t c = 0; c < n; ++c) (*col)[e++] = c;
        } else if (r == n - 1 && n > 2) {
            /* empty row */
        } else {
            (*col)[e++] = r;
            (*col)[e++] = 0;
            (*col)[e++] = 0;   /* repeated column */
        }
        (*rowptr)[r + 1] = (int32_t)e;
    }
    *nnz = e;
    *val = (float *)malloc(sizeof(float) * (size_t)(e ? e : 1));
    for (int64_t i = 0; i < e; ++i) (*val)[i] = (float)(i % 7) - 3.0f;
}

int main(void) {
    const int32_t sizes[] = {1, 2, 3, 17, 64};
    for (size_t si = 0; si < sizeof(sizes) / sizeof(sizes[0]); ++si) {
        const int32_t n = sizes[si];
        int32_t *rowptr, *col;
        float *val;
        int64_t nnz;
        build(n, &rowptr, &col, &val, &nnz);
        const uint32_t steps_list[] = {1, 4, 8, 9, 30, 255};
        for (size_t di = 0; di < sizeof(steps_list) / sizeof(steps_list[0]); ++di) {
            const uint32_t d = steps_list[di];
            uint8_t *labels = (uint8_t *)malloc(d + 1);
            for (int32_t v = 0; v < n; ++v) (void)oracle_walk(rowptr, col, n, v, 3, 11, d, labels);
            free(labels);
            const uint32_t k = 5;
            uint8_t *pat = (uint8_t *)malloc((size_t)n * k * (d + 1));
            oracle_patterns(rowptr, col, n, 7, k, d, pat);
            free(pat);
            int32_t *nodes = alloc_i32((size_t)n);
            uint32_t *S = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n);
            for (int32_t v = 0; v < n; ++v) nodes[v] = v;
            oracle_density(rowptr, col, n, 5, k, d, nodes, n, S);
            free(nodes);
            free(S);
        }
        const int32_t F = 3;
        float *X = (float *)malloc(sizeof(float) * (size_t)n * F);
        double *Xd = (double *)malloc(sizeof(double) * (size_t)n * F);
        for (int64_t i = 0; i < (int64_t)n * F; ++i) X[i] = Xd[i] = (float)(i % 5) - 2.0f;
        int32_t *rows = alloc_i32((size_t)n);
        int64_t *slot = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
        for (int32_t r = 0; r < n; ++r) rows[r] = slot[r] = r;
        double *Y = (double *)malloc(sizeof(double) * (size_t)n * F);
        double *B = (double *)malloc(sizeof(double) * (size_t)n * F);
        oracle_spmm_rows(rowptr, col, val, X, F, rows, n, Y, B);
        oracle_spmm_rows(rowptr, col, val, X, F, rows, n, Y, NULL);
        oracle_spmm_rows_f64(rowptr, col, val, Xd, F, rows, n, slot, Y);
        float W[3 * 2] = {1, 2, 3, 4, 5, 6};
        double *T = (double *)malloc(sizeof(double) * (size_t)n * 2);
        double *BT = (double *)malloc(sizeof(double) * (size_t)n * 2);
        oracle_xw_rows(X, W, F, 2, rows, n, T, BT);
        oracle_xw_rows(X, W, F, 2, rows, n, T, NULL);
        free(X); free(Xd); free(rows); free(slot); free(Y); free(B); free(T); free(BT);
        free(rowptr); free(col); free(val);
    }
    puts("oracle sanitizer run: ok");
    return 0;
}
