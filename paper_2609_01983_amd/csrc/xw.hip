// Update phase T = X W of a GCN layer on the gfx950 matrix cores (DualGCN Sec. 1:
// after aggregation a layer multiplies by a small dense weight matrix), and the same
// kernel for the backward product dX = (G_T W^T) * [M > 0] of training, which reads W
// transposed and zeroes the outputs that the previous layer's ReLU did not pass.
//
// X (n x F_in, float32) is rounded to bfloat16 (nearest-even) in registers -- or is
// read as stored when it already holds bfloat16 (the output of a previous layer's
// aggregation written in bfloat16: the same values this rounding would give) --, W is
// rounded to bfloat16 while each workgroup stages its transpose in LDS, and
// v_mfma_f32_16x16x32_bf16 accumulates in float32.  The product is memory-bound
// (it reads 4 F_in and writes 4 F_out bytes per row for 2 F_in F_out flops, far
// below the ridge of the bf16 matrix cores), so the kernel is built to stream X:
// 512-thread workgroups (eight wavefronts share one staged W, so a CU holds 16
// wavefronts even when W^T takes 64 KiB of LDS), every wavefront owns 16-row
// tiles and requests the next 32-wide k-step of its tile while the MFMAs of the
// current one run, and the grid is persistent (one pass over the row tiles).
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

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kRowsPerWave = 16;
constexpr int kRowsPerBlock = kWaves * kRowsPerWave;
constexpr int kLdsElems = 32768;     // bf16 elements of W^T one workgroup stages (64 KiB)
constexpr int kPad = 8;              // bf16 padding per LDS row (spreads LDS banks)
constexpr int kMaxTiles = 16;        // 16-column output tiles per wavefront and launch

// The bfloat16 A fragment of a lane at k-step ks: eight consecutive k of row `arow`
// (zeros past the last row), from float32 X rounded here or from bfloat16 X as stored.
template <bool XBF>
struct XFrag {
    f32x4 lo, hi;      // float32 X
    uint4 raw;         // bfloat16 X

    __device__ __forceinline__ void load(const void *X, int64_t arow, bool ok, int ld, int kk) {
        if constexpr (XBF) {
            raw = make_uint4(0u, 0u, 0u, 0u);
            if (ok) raw = *reinterpret_cast<const uint4 *>(static_cast<const unsigned short *>(X) + arow * ld + kk);
        } else {
            lo = f32x4{0.f, 0.f, 0.f, 0.f};
            hi = lo;
            if (ok) {
                const float *xr = static_cast<const float *>(X) + arow * ld + kk;
                lo = *reinterpret_cast<const f32x4 *>(xr);
                hi = *reinterpret_cast<const f32x4 *>(xr + 4);
            }
        }
    }
    __device__ __forceinline__ bf16x8 bf16() const {
        if constexpr (XBF) {
            return __builtin_bit_cast(bf16x8, raw);
        } else {
            u16x8 a16;
            a16[0] = to_bf16(lo[0]); a16[1] = to_bf16(lo[1]);
            a16[2] = to_bf16(lo[2]); a16[3] = to_bf16(lo[3]);
            a16[4] = to_bf16(hi[0]); a16[5] = to_bf16(hi[1]);
            a16[6] = to_bf16(hi[2]); a16[7] = to_bf16(hi[3]);
            return __builtin_bit_cast(bf16x8, a16);
        }
    }
};

// Where the output keeps a product: no mask, or M > 0 for a float32 or bfloat16 M.
enum MaskKind { kNoMask = 0, kMaskF32 = 1, kMaskBF16 = 2 };

// Masked products leave the matrix cores through LDS: each wavefront stages its 16-row
// tile 64 columns at a time (rows padded to 68 words), and every lane then finishes 16
// consecutive outputs of one row -- the mask read and the output written with 16-byte
// accesses instead of one element per lane and instruction.
constexpr int kEpiCols = 64;
constexpr int kEpiLd = kEpiCols + 4;
constexpr int kEpiWaveWords = kRowsPerWave * kEpiLd;

size_t epilogue_lds_bytes(int mask) {
    return mask == kNoMask ? 0 : static_cast<size_t>(kWaves) * kEpiWaveWords * sizeof(float);
}

// Sixteen consecutive mask elements from `at` (16-byte aligned) as float32.
template <int MASK>
__device__ __forceinline__ void load_mask16(const void *M, int64_t at, float (&m)[16]) {
    if constexpr (MASK == kMaskF32) {
        const f32x4 *p = reinterpret_cast<const f32x4 *>(static_cast<const float *>(M) + at);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const f32x4 v = p[q];
            m[4 * q] = v[0];
            m[4 * q + 1] = v[1];
            m[4 * q + 2] = v[2];
            m[4 * q + 3] = v[3];
        }
    } else {
        const uint4 *p = reinterpret_cast<const uint4 *>(static_cast<const unsigned short *>(M) + at);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const uint4 v = p[q];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                m[8 * q + 2 * i] = __builtin_bit_cast(float, w[i] << 16);
                m[8 * q + 2 * i + 1] = __builtin_bit_cast(float, w[i] & 0xFFFF0000u);
            }
        }
    }
}

// Out[:, c0 : c0 + 16 ntiles] = bf16(A) bf16(B[:, c0 : ..]) for every row tile, where A is
// n x K (row-major) and B(k, j) = W[k sk + j sn] is K x N: (sk, sn) = (N, 1) multiplies by
// W, (1, K) by the transpose of a row-major N x K matrix W.  With a mask, outputs whose
// M element (n x N, row-major) is not positive are written as zeros.  K % 32 == 0.
template <int NTMAX, bool XBF, int MASK>
__global__ __launch_bounds__(kThreads) void xw_mfma_kernel(const void *__restrict__ X,
                                                           const float *__restrict__ W,
                                                           const void *__restrict__ M,
                                                           float *__restrict__ T, int32_t n,
                                                           int32_t K, int32_t N, int32_t sk,
                                                           int32_t sn, int32_t c0, int32_t ntiles) {
    extern __shared__ unsigned short w_lds[];   // [16 ntiles][K + kPad]: B^T in bf16
    const int ldw = K + kPad;
    const int ncols = 16 * ntiles;
    if (sn == 1) {          // consecutive threads read consecutive columns of W
        for (int idx = threadIdx.x; idx < K * ncols; idx += kThreads) {
            const int c = idx / ncols, j = idx % ncols;
            w_lds[j * ldw + c] = to_bf16(W[static_cast<int64_t>(c) * sk + c0 + j]);
        }
    } else {                // consecutive threads read consecutive k of W's rows
        for (int idx = threadIdx.x; idx < K * ncols; idx += kThreads) {
            const int j = idx / K, c = idx % K;
            w_lds[j * ldw + c] = to_bf16(W[static_cast<int64_t>(c0 + j) * sn + c]);
        }
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lrow = lane & 15;          // A row / B column / D column inside the tile
    const int kgrp = lane >> 4;          // which 8-wide k group this lane supplies
    const int ksteps = K / 32;
    const int64_t tiles = (static_cast<int64_t>(n) + kRowsPerBlock - 1) / kRowsPerBlock;

    for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        const int64_t row0 = tile * kRowsPerBlock + wave * kRowsPerWave;
        const int64_t arow = row0 + lrow;
        const bool arow_ok = arow < n;
        f32x4 acc[NTMAX];
#pragma unroll
        for (int t = 0; t < NTMAX; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        // k-step ks + 1 is requested while the MFMAs of k-step ks run
        XFrag<XBF> cur, nxt;
        cur.load(X, arow, arow_ok, K, kgrp * 8);
        for (int ks = 0; ks < ksteps; ++ks) {
            nxt.load(X, arow, arow_ok && ks + 1 < ksteps, K, (ks + 1) * 32 + kgrp * 8);
            const bf16x8 av = cur.bf16();
            const int kk = ks * 32 + kgrp * 8;
#pragma unroll
            for (int t = 0; t < NTMAX; ++t) {
                if (t < ntiles) {
                    const u16x8 b16 = *reinterpret_cast<const u16x8 *>(w_lds + (t * 16 + lrow) * ldw + kk);
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        av, __builtin_bit_cast(bf16x8, b16), acc[t], 0, 0, 0);
                }
            }
            cur = nxt;
        }
        if constexpr (MASK == kNoMask) {
#pragma unroll
            for (int t = 0; t < NTMAX; ++t) {
                if (t < ntiles) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int64_t orow = row0 + kgrp * 4 + j;
                        if (orow < n) T[orow * N + c0 + t * 16 + lrow] = acc[t][j];
                    }
                }
            }
        } else {
            float *epi = reinterpret_cast<float *>(w_lds + ncols * ldw) + wave * kEpiWaveWords;
            const int er = lane >> 2;                  // staged row this lane finishes
            const int ec = (lane & 3) * 16;            // its first column inside a pass
            const int64_t orow = row0 + er;
#pragma unroll
            for (int h = 0; h < (NTMAX + 3) / 4; ++h) {
                if (4 * h < ntiles) {                  // uniform over the workgroup
                    const int cl = h * kEpiCols + ec;  // column inside this launch's block
                    const bool ok = orow < n && cl < ncols;
                    const int64_t at = orow * N + c0 + cl;
                    float mk[16];
                    if (ok) load_mask16<MASK>(M, at, mk);
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int t = 4 * h + u;
                        if (t < NTMAX && t < ntiles) {
#pragma unroll
                            for (int j = 0; j < 4; ++j) epi[(kgrp * 4 + j) * kEpiLd + u * 16 + lrow] = acc[t][j];
                        }
                    }
                    __syncthreads();
                    if (ok) {
                        const f32x4 *src = reinterpret_cast<const f32x4 *>(epi + er * kEpiLd + ec);
                        f32x4 *dst = reinterpret_cast<f32x4 *>(T + at);
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            f32x4 v = src[q];
#pragma unroll
                            for (int i = 0; i < 4; ++i) v[i] = mk[4 * q + i] > 0.f ? v[i] : 0.f;
                            dst[q] = v;
                        }
                    }
                    __syncthreads();
                }
            }
        }
    }
}

// Dynamic LDS above 64 KiB must be requested per kernel.
int allow_lds(const void *kernel, size_t bytes) {
    if (bytes <= 64 * 1024) return DUALGCN_OK;
    return hip_status(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                          static_cast<int>(bytes)));
}

template <int NT, bool XBF, int MASK>
int launch_tiles(const void *X, const float *W, const void *M, float *T, int32_t n, int32_t K,
                 int32_t N, int32_t sk, int32_t sn, int c0, int ntiles, size_t lds, hipStream_t s) {
    lds += epilogue_lds_bytes(MASK);
    int st = allow_lds(reinterpret_cast<const void *>(&xw_mfma_kernel<NT, XBF, MASK>), lds);
    if (st) return st;
    // workgroups per CU allowed by the LDS of one CU (160 KiB) and by 2048 threads per CU
    const int per_cu = std::max<int>(1, std::min<int>(2048 / kThreads, static_cast<int>((160 * 1024) / lds)));
    const int64_t tiles = (static_cast<int64_t>(n) + kRowsPerBlock - 1) / kRowsPerBlock;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(tiles, static_cast<int64_t>(device_cus()) * per_cu));
    hipLaunchKernelGGL((xw_mfma_kernel<NT, XBF, MASK>), dim3(static_cast<unsigned>(grid)),
                       dim3(kThreads), lds, s, X, W, M, T, n, K, N, sk, sn, c0, ntiles);
    return hip_status(hipGetLastError());
}

template <bool XBF, int MASK>
int launch_nt(const void *X, const float *W, const void *M, float *T, int32_t n, int32_t K,
              int32_t N, int32_t sk, int32_t sn, int c0, int ntiles, size_t lds, hipStream_t s) {
    if (ntiles <= 4) return launch_tiles<4, XBF, MASK>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
    if (ntiles <= 8) return launch_tiles<8, XBF, MASK>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
    return launch_tiles<16, XBF, MASK>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
}

// Out (n x N) = A (n x K) B (K x N) with B(k, j) = W[k sk + j sn], in column blocks whose
// B^T slice fits the LDS budget.
int launch_mm(const void *X, bool in_bf16, const float *W, int32_t sk, int32_t sn,
              const void *M, int mask, float *T, int32_t n, int32_t K, int32_t N, hipStream_t s) {
    const int cb = std::min<int>(std::min<int>(N, 16 * kMaxTiles), (kLdsElems / K) / 16 * 16);
    if (cb < 16) return DUALGCN_ERR_UNSUPPORTED;
    for (int c0 = 0; c0 < N; c0 += cb) {
        const int width = std::min(cb, N - c0);
        const int ntiles = width / 16;
        const size_t lds = static_cast<size_t>(width) * (K + kPad) * sizeof(unsigned short);
        int st;
        if (in_bf16) {
            if (mask == kMaskF32) st = launch_nt<true, kMaskF32>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
            else if (mask == kMaskBF16) st = launch_nt<true, kMaskBF16>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
            else st = launch_nt<true, kNoMask>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
        } else {
            if (mask == kMaskF32) st = launch_nt<false, kMaskF32>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
            else if (mask == kMaskBF16) st = launch_nt<false, kMaskBF16>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
            else st = launch_nt<false, kNoMask>(X, W, M, T, n, K, N, sk, sn, c0, ntiles, lds, s);
        }
        if (st) return st;
    }
    return DUALGCN_OK;
}

}  // namespace

size_t xw_workspace_bytes(int32_t n, int32_t F_out) {
    return (static_cast<size_t>(n) * F_out * sizeof(float) + 255) / 256 * 256;
}

int launch_xw(const void *X, bool in_bf16, const float *W, float *T, int32_t n, int32_t F_in,
              int32_t F_out, hipStream_t s) {
    return launch_mm(X, in_bf16, W, F_out, 1, nullptr, kNoMask, T, n, F_in, F_out, s);
}

int launch_backward_data(const void *G, bool g_bf16, const float *W, const void *M, bool m_bf16,
                         float *dX, int32_t n, int32_t F_in, int32_t F_out, hipStream_t s) {
    const int mask = M == nullptr ? kNoMask : (m_bf16 ? kMaskBF16 : kMaskF32);
    return launch_mm(G, g_bf16, W, 1, F_out, M, mask, dX, n, F_out, F_in, s);
}

int launch_gcn_layer(const Plan &p, const void *X, bool in_bf16, const float *W, void *Y,
                     bool out_bf16, int32_t F_in, int32_t F_out, bool relu, void *workspace,
                     hipStream_t s) {
    float *T = static_cast<float *>(workspace);
    const int st = launch_xw(X, in_bf16, W, T, p.n, F_in, F_out, s);
    if (st) return st;
    return launch_spmm(p, T, Y, F_out, relu, out_bf16, s);
}

}  // namespace dgc
