// Attainable memory bandwidth of the device, for reading the SpMM's rates against what the
// memory system delivers to a plain streaming kernel (next to the nominal HBM peak).
//
// copy: dst = src, 16-byte loads and non-temporal 16-byte stores, every byte read once and
//       written once;
// read: every 16-byte word of src read once and folded into one float per workgroup
//       (written to dst), so the loads cannot be removed.
// Grid-strided over the buffer with up to kMaxProbeGrid workgroups (many per CU, so that
// the next workgroups' loads are queued while the first ones finish).
#include "internal.h"

#include <algorithm>

namespace dgc {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

typedef float f32x4 __attribute__((ext_vector_type(4)));

// Each workgroup moves kUnroll consecutive 4 KiB pieces (256 lanes x 16 bytes) per
// iteration, then strides by the whole grid.
__global__ __launch_bounds__(kThreads) void copy_probe_kernel(const f32x4 *__restrict__ src,
                                                              f32x4 *__restrict__ dst, int64_t words) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads * kUnroll;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads * kUnroll + threadIdx.x; i < words;
         i += stride) {
        f32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (i + u * kThreads < words) v[u] = src[i + u * kThreads];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (i + u * kThreads < words) __builtin_nontemporal_store(v[u], dst + i + u * kThreads);
    }
}

__global__ __launch_bounds__(kThreads) void read_probe_kernel(const f32x4 *__restrict__ src,
                                                              float *__restrict__ out, int64_t words) {
    __shared__ float sh[kThreads];
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads * kUnroll;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads * kUnroll + threadIdx.x; i < words;
         i += stride) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (i + u * kThreads < words) acc += src[i + u * kThreads];
    }
    sh[threadIdx.x] = acc[0] + acc[1] + acc[2] + acc[3];
    __syncthreads();
    for (int m = kThreads / 2; m > 0; m >>= 1) {
        if (static_cast<int>(threadIdx.x) < m) sh[threadIdx.x] += sh[threadIdx.x + m];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[blockIdx.x] = sh[0];
}

}  // namespace

int probe_grid() { return kMaxProbeGrid; }

int launch_bandwidth_probe(int kind, const void *src, void *dst, size_t bytes, hipStream_t s) {
    const int64_t words = static_cast<int64_t>(bytes / 16);
    const int64_t per_block = static_cast<int64_t>(kThreads) * kUnroll;
    const unsigned grid = static_cast<unsigned>(std::max<int64_t>(
        1, std::min<int64_t>(probe_grid(), (words + per_block - 1) / per_block)));
    if (kind == DUALGCN_PROBE_COPY)
        hipLaunchKernelGGL(copy_probe_kernel, dim3(grid), dim3(kThreads), 0, s,
                           static_cast<const f32x4 *>(src), static_cast<f32x4 *>(dst), words);
    else
        hipLaunchKernelGGL(read_probe_kernel, dim3(grid), dim3(kThreads), 0, s,
                           static_cast<const f32x4 *>(src), static_cast<float *>(dst), words);
    return hip_status(hipGetLastError());
}

}  // namespace dgc
