// Values of other aggregation matrices on the same structure (DualGCN Sec. 2.1: the
// aggregation phase of a message-passing layer multiplies by a matrix derived from the
// adjacency; the GCN normalisation is one choice).  The SpMM kernels take any values, so
// switching aggregator means filling `val` again: GCN 1/sqrt(d_r d_c), mean 1/d_r, sum 1
// with 1 + eps on self-loop entries (the GIN form).  d is the row length of the matrix as
// given.  Values are computed in float64 and rounded once to float32.
#include "internal.h"

#include <algorithm>

namespace dgc {
namespace {

constexpr int kThreads = 256;

// Row of entry e: the last r with rowptr[r] <= e (rows may be empty).
__device__ __forceinline__ int32_t row_of(const int32_t *__restrict__ rowptr, int32_t n, int64_t e) {
    int32_t lo = 0, hi = n;           // answer in [lo, hi)
    while (hi - lo > 1) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (static_cast<int64_t>(rowptr[mid]) <= e) lo = mid;
        else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kThreads) void aggregator_kernel(const int32_t *__restrict__ rowptr,
                                                              const int32_t *__restrict__ col,
                                                              int32_t n, int64_t nnz, int kind,
                                                              double one_plus_eps,
                                                              float *__restrict__ val) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < nnz;
         e += stride) {
        const int32_t r = row_of(rowptr, n, e);
        const int32_t c = col[e];
        const double dr = static_cast<double>(rowptr[r + 1] - rowptr[r]);
        double v = 0.0;
        if (kind == DUALGCN_AGG_MEAN) {
            v = 1.0 / dr;
        } else if (kind == DUALGCN_AGG_SUM) {
            v = c == r ? one_plus_eps : 1.0;
        } else if (c >= 0 && c < n) {
            const double dc = static_cast<double>(rowptr[c + 1] - rowptr[c]);
            v = 1.0 / sqrt(dr * dc);
        }
        val[e] = static_cast<float>(v);
    }
}

}  // namespace

int launch_aggregator_values(const dualgcn_csr *csr, int kind, float eps, float *val,
                             hipStream_t s) {
    if (csr->nnz == 0) return DUALGCN_OK;
    const int64_t blocks = std::min<int64_t>((csr->nnz + kThreads - 1) / kThreads, 65536);
    hipLaunchKernelGGL(aggregator_kernel, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s,
                       csr->rowptr, csr->col, csr->n, csr->nnz, kind,
                       1.0 + static_cast<double>(eps), val);
    return hip_status(hipGetLastError());
}

}  // namespace dgc
