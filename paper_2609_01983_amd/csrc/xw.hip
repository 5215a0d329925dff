// Update phase T = X W of a GCN layer on the gfx950 matrix cores (DualGCN Sec. 1:
// after aggregation a layer multiplies by a small dense weight matrix), followed
// by the aggregation Y = act(A T) of spmm.hip.
//
// X (n x F_in, float32) is rounded to bfloat16 (nearest-even) in registers, W is
// rounded once into a transposed bfloat16 copy, and v_mfma_f32_16x16x32_bf16
// accumulates in float32.  The product is memory-bound (it reads 4 F_in and
// writes 4 F_out bytes per row for 2 F_in F_out flops), so the kernel streams X
// once: every wavefront owns 16-row tiles, loads all of a tile's K fragments
// before its first MFMA, and reads W^T from LDS, where each workgroup stages it
// once for all the tiles it processes.
//
// MFMA 16x16x32 operand layout (64 lanes, l = lane):
//   A (16 x 32):  lane l supplies row l % 16, eight consecutive k of group l / 16
//   B (32 x 16):  lane l supplies column l % 16, the same eight k
//   D (16 x 16):  lane l holds rows 4 (l / 16) + j, j < 4, column l % 16
// Both operands use the same (lane group, element) -> k assignment, so the sum
// over k is correct for any such assignment.
#include "internal.h"

#include <algorithm>

namespace dgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerWave = 16;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kLdsElems = 32768;     // bf16 elements of W^T one workgroup stages (64 KiB)
constexpr int kPad = 8;              // bf16 padding per LDS row (spreads LDS banks)

// float32 -> bfloat16 bits, round to nearest even; NaNs stay NaN.
__device__ __forceinline__ unsigned short to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<unsigned short>((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<unsigned short>(u >> 16);
}

// Wt[j][c] = bf16(W[c][j]): the transposed weight matrix, row stride F_in.
__global__ __launch_bounds__(kThreads) void weight_bf16_kernel(const float *__restrict__ W,
                                                               int32_t F_in, int32_t F_out,
                                                               unsigned short *__restrict__ Wt) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= static_cast<int64_t>(F_in) * F_out) return;
    const int32_t j = static_cast<int32_t>(i / F_in), c = static_cast<int32_t>(i % F_in);
    Wt[i] = to_bf16(W[static_cast<int64_t>(c) * F_out + j]);
}

// T[:, c0 : c0 + 16 ntiles] = bf16(X) * Wt[c0 : ..]^T for every row tile; F_in % 32 == 0.
template <int NTMAX>
__global__ __launch_bounds__(kThreads) void xw_mfma_kernel(const float *__restrict__ X,
                                                           const unsigned short *__restrict__ Wt,
                                                           float *__restrict__ T, int32_t n,
                                                           int32_t F_in, int32_t F_out,
                                                           int32_t c0, int32_t ntiles) {
    extern __shared__ unsigned short w_lds[];   // [16 ntiles][F_in + kPad]
    const int ldw = F_in + kPad;
    const int ncols = 16 * ntiles;
    // stage W^T rows c0 .. c0 + ncols in LDS, 16 bytes per lane
    for (int idx = threadIdx.x; idx < ncols * (F_in / 8); idx += kThreads) {
        const int j = idx / (F_in / 8), c8 = idx % (F_in / 8);
        const uint4 v = *reinterpret_cast<const uint4 *>(Wt + static_cast<int64_t>(c0 + j) * F_in + c8 * 8);
        *reinterpret_cast<uint4 *>(w_lds + j * ldw + c8 * 8) = v;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lrow = lane & 15;          // A row / B column / D column inside the tile
    const int kgrp = lane >> 4;          // which 8-wide k group this lane supplies
    const int ksteps = F_in / 32;
    const int64_t tiles = (static_cast<int64_t>(n) + kRowsPerBlock - 1) / kRowsPerBlock;

    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t row0 = tile * kRowsPerBlock + wave * kRowsPerWave;
        const int64_t arow = row0 + lrow;
        const bool arow_ok = arow < n;
        f32x4 acc[NTMAX];
#pragma unroll
        for (int t = 0; t < NTMAX; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        const float *xr = X + arow * F_in + kgrp * 8;
        for (int ks = 0; ks < ksteps; ++ks) {
            float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
            if (arow_ok) {
                lo = *reinterpret_cast<const float4 *>(xr + ks * 32);
                hi = *reinterpret_cast<const float4 *>(xr + ks * 32 + 4);
            }
            u16x8 a16;
            a16[0] = to_bf16(lo.x); a16[1] = to_bf16(lo.y); a16[2] = to_bf16(lo.z); a16[3] = to_bf16(lo.w);
            a16[4] = to_bf16(hi.x); a16[5] = to_bf16(hi.y); a16[6] = to_bf16(hi.z); a16[7] = to_bf16(hi.w);
            const bf16x8 a = __builtin_bit_cast(bf16x8, a16);
#pragma unroll
            for (int t = 0; t < NTMAX; ++t) {
                if (t < ntiles) {
                    const u16x8 b16 = *reinterpret_cast<const u16x8 *>(
                        w_lds + (t * 16 + lrow) * ldw + ks * 32 + kgrp * 8);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        a, __builtin_bit_cast(bf16x8, b16), acc[t], 0, 0, 0);
                }
            }
        }
#pragma unroll
        for (int t = 0; t < NTMAX; ++t) {
            if (t < ntiles) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int64_t orow = row0 + kgrp * 4 + j;
                    if (orow < n) T[orow * F_out + c0 + t * 16 + lrow] = acc[t][j];
                }
            }
        }
    }
}

int num_cus() {
    static int cus = 0;
    if (cus == 0) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
    }
    return cus;
}

// Dynamic LDS above 64 KiB must be requested per kernel.
int allow_lds(const void *kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return DUALGCN_OK;
    return hip_status(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                          static_cast<int>(bytes)));
}

}  // namespace

size_t xw_workspace_bytes(int32_t n, int32_t F_in, int32_t F_out) {
    const size_t t_bytes = (static_cast<size_t>(n) * F_out * sizeof(float) + 255) / 256 * 256;
    return t_bytes + static_cast<size_t>(F_in) * F_out * sizeof(unsigned short);
}

int launch_gcn_layer(const Plan &p, const float *X, const float *W, float *Y, int32_t F_in,
                     int32_t F_out, bool relu, void *workspace, hipStream_t s) {
    const size_t t_bytes = (static_cast<size_t>(p.n) * F_out * sizeof(float) + 255) / 256 * 256;
    float *T = static_cast<float *>(workspace);
    unsigned short *Wt = reinterpret_cast<unsigned short *>(static_cast<char *>(workspace) + t_bytes);
    {
        const int64_t count = static_cast<int64_t>(F_in) * F_out;
        hipLaunchKernelGGL(weight_bf16_kernel, dim3(static_cast<unsigned>((count + kThreads - 1) / kThreads)),
                           dim3(kThreads), 0, s, W, F_in, F_out, Wt);
    }
    // column blocks whose W^T slice fits the LDS budget
    int cb = std::min<int>(F_out, (kLdsElems / F_in) / 16 * 16);
    if (cb < 16) return DUALGCN_ERR_UNSUPPORTED;
    const int64_t tiles = (static_cast<int64_t>(p.n) + kRowsPerBlock - 1) / kRowsPerBlock;
    for (int c0 = 0; c0 < F_out; c0 += cb) {
        const int width = std::min(cb, F_out - c0);
        const int ntiles = width / 16;
        const size_t lds = static_cast<size_t>(width) * (F_in + kPad) * sizeof(unsigned short);
        const int per_cu = lds <= 80 * 1024 ? 2 : 1;
        int st = DUALGCN_OK;
        if (ntiles <= 4) st = allow_lds(reinterpret_cast<const void *>(&xw_mfma_kernel<4>), lds);
        else if (ntiles <= 8) st = allow_lds(reinterpret_cast<const void *>(&xw_mfma_kernel<8>), lds);
        else st = allow_lds(reinterpret_cast<const void *>(&xw_mfma_kernel<16>), lds);
        if (st) return st;
        const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(tiles, static_cast<int64_t>(num_cus()) * per_cu));
        if (ntiles <= 4)
            hipLaunchKernelGGL((xw_mfma_kernel<4>), dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                               lds, s, X, Wt, T, p.n, F_in, F_out, c0, ntiles);
        else if (ntiles <= 8)
            hipLaunchKernelGGL((xw_mfma_kernel<8>), dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                               lds, s, X, Wt, T, p.n, F_in, F_out, c0, ntiles);
        else
            hipLaunchKernelGGL((xw_mfma_kernel<16>), dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                               lds, s, X, Wt, T, p.n, F_in, F_out, c0, ntiles);
        st = hip_status(hipGetLastError());
        if (st) return st;
    }
    return launch_spmm(p, T, Y, F_out, relu, s);
}

}  // namespace dgc
