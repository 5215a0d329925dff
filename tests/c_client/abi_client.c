/* A plain C99 client of the library: compiled with the C compiler against include/dualgcn.h
 * and linked with libdualgcn.so, it checks that the header is valid C and that the entry
 * points resolve and answer argument errors without a device.  Exit status 0 = all checks
 * passed; otherwise the number of the first failed check. */
#include <stdio.h>
#include <string.h>

#include "dualgcn.h"

int main(void) {
    int32_t rowptr[3] = {0, 1, 2};
    int32_t col[2] = {0, 1};
    float val[2] = {1.0f, 1.0f};
    dualgcn_csr csr;
    dualgcn_plan *plan = (dualgcn_plan *)&csr;   /* must be reset to NULL on error */
    size_t bytes = 0;

    if (strcmp(dualgcn_status_str(DUALGCN_OK), "ok") != 0) return 1;
    if (dualgcn_status_str(12345) == NULL) return 2;
    if (dualgcn_partition(NULL, 0, 16, 5, NULL, NULL, &plan) != DUALGCN_ERR_INVALID_ARG) return 3;
    if (plan != NULL) return 4;
    csr.n = 2;
    csr.nnz = 2;
    csr.rowptr = rowptr;
    csr.col = col;
    csr.val = val;
    if (dualgcn_partition(&csr, 0, 0, 5, NULL, NULL, &plan) != DUALGCN_ERR_INVALID_ARG) return 5;
    if (dualgcn_spmm(NULL, NULL, NULL, 4, NULL) != DUALGCN_ERR_INVALID_ARG) return 6;
    if (dualgcn_spmm_update(NULL, NULL, NULL, NULL, NULL, 128, 64, DUALGCN_RELU, NULL) !=
        DUALGCN_ERR_INVALID_ARG)
        return 7;
    if (dualgcn_gcn_layer_workspace(NULL, 32, 32, &bytes) != DUALGCN_ERR_INVALID_ARG) return 8;
    dualgcn_plan_destroy(NULL);
    printf("c client: ok\n");
    return 0;
}
