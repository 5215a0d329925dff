// Training-side kernels of a GCN on gfx950 (DualGCN Sec. 1: the paper accelerates GCN
// training, whose backward pass repeats the aggregation on the gradients).
//
// For a layer H = act(A (X W)) and G = dL/dH the chain rule gives
//   G_P = G * act'(P),  G_T = A^T G_P (the aggregation SpMM on a plan of A^T, which for
//   the symmetric normalised adjacency is the forward plan),  dW = X^T G_T  and
//   dX = G_T W^T (masked by the previous layer's ReLU; the matrix-core kernel of the
//   update phase computes it).  This file holds the two remaining pieces:
//
// * the mean softmax cross-entropy over labeled rows and its gradient, one 16-lane
//   group per row, float32 arithmetic with the loss summed in float64 per workgroup
//   and then over workgroups in a fixed order;
// * the weight gradient dW = X^T G on the matrix cores.  The contraction runs over the
//   n rows, so every workgroup owns a fixed set of 64-row chunks, stages each chunk
//   transposed in LDS as bfloat16 (the same rounding as the update phase), multiplies
//   with v_mfma_f32_16x16x32_bf16 into float32 accumulators and writes one partial
//   dW; a second kernel sums the partials in workgroup order in float64 (so the result
//   does not depend on timing) and can apply the SGD step W -= lr dW.
#include "internal.h"

#include <algorithm>

namespace dgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// ------------------------------------------------------------------ softmax cross-entropy

constexpr int kGroup = 16;                       // lanes per row
constexpr int kRowsPerBlock = kThreads / kGroup;

__device__ __forceinline__ float group_max(float v) {
#pragma unroll
    for (int o = kGroup / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kGroup));
    return v;
}

__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
    for (int o = kGroup / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kGroup);
    return v;
}

__global__ __launch_bounds__(kThreads) void softmax_xent_kernel(
    const float *__restrict__ Y, const int32_t *__restrict__ labels, int32_t n, int32_t C,
    float scale, float *__restrict__ G, double *__restrict__ partial) {
    __shared__ double sh[kThreads];
    const int g = threadIdx.x / kGroup, l = threadIdx.x % kGroup;
    double acc = 0.0;
    for (int64_t row = static_cast<int64_t>(blockIdx.x) * kRowsPerBlock + g; row < n;
         row += static_cast<int64_t>(gridDim.x) * kRowsPerBlock) {
        const float *y = Y + row * C;
        float *gr = G + row * C;
        const int32_t lab = labels[row];
        const bool labeled = lab >= 0 && lab < C;
        float m = -INFINITY;
        for (int j = l; j < C; j += kGroup) m = fmaxf(m, y[j]);
        m = group_max(m);
        float s = 0.f;
        for (int j = l; j < C; j += kGroup) s += expf(y[j] - m);
        s = group_sum(s);
        const float inv = 1.f / s;
        for (int j = l; j < C; j += kGroup) {
            const float p = expf(y[j] - m) * inv;
            gr[j] = labeled ? scale * (p - (j == lab ? 1.f : 0.f)) : 0.f;
        }
        if (labeled && l == 0) acc += static_cast<double>(logf(s) + m - y[lab]);
    }
    const int t = threadIdx.x;
    sh[t] = acc;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) sh[t] += sh[t + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[blockIdx.x] = sh[0];
}

// loss[0] = scale * sum of the partials, in workgroup order.
__global__ void loss_total_kernel(double *__restrict__ loss, int32_t count, float scale) {
    double s = 0.0;
    for (int i = 0; i < count; ++i) s += loss[1 + i];
    loss[0] = static_cast<double>(scale) * s;
}

// ------------------------------------------------------------------ weight gradient

constexpr int kWgThreads = 512;
constexpr int kWgWaves = kWgThreads / 64;
constexpr int kChunk = 64;                       // rows per LDS stage (two k-steps of 32)
constexpr int kLdsPad = 8;                       // bf16 padding per transposed row
constexpr int kLdsRow = kChunk + kLdsPad;
constexpr int kMaxIB = 256;                      // dW rows (X columns) per pass
constexpr int kMaxJB = 128;                      // dW columns (G columns) per pass
constexpr int kMaxPartials = 512;                // workgroups, hence partial dW matrices

// Four consecutive elements of one row as float32, from float32 or bfloat16 storage.
template <bool BF>
__device__ __forceinline__ f32x4 load4(const void *base, int64_t at) {
    if constexpr (BF) {
        const uint2 r = *reinterpret_cast<const uint2 *>(static_cast<const unsigned short *>(base) + at);
        return f32x4{__builtin_bit_cast(float, r.x << 16), __builtin_bit_cast(float, r.x & 0xFFFF0000u),
                     __builtin_bit_cast(float, r.y << 16), __builtin_bit_cast(float, r.y & 0xFFFF0000u)};
    } else {
        return *reinterpret_cast<const f32x4 *>(static_cast<const float *>(base) + at);
    }
}

// One staged operand: `width` columns (starting at col0) of a 64-row chunk, held by each
// thread as up to ITEMS (row pair, column quad) items between the global load and the
// transposed LDS write t[col][row].
template <bool BF, int ITEMS>
struct Stage {
    f32x4 v[ITEMS][2];

    __device__ __forceinline__ void load(const void *src, int64_t ld, int64_t n, int64_t r0,
                                         int col0, int width) {
        const int quads = width / 4;
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            const int w = threadIdx.x + it * kWgThreads;
            const int rp = w / quads, cq = w % quads;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t r = r0 + 2 * rp + h;
                v[it][h] = f32x4{0.f, 0.f, 0.f, 0.f};
                if (rp < kChunk / 2 && r < n) v[it][h] = load4<BF>(src, r * ld + col0 + 4 * cq);
            }
        }
    }

    __device__ __forceinline__ void store(uint32_t *t, int width) const {
        const int quads = width / 4;
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            const int w = threadIdx.x + it * kWgThreads;
            const int rp = w / quads, cq = w % quads;
            if (rp < kChunk / 2) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t lo = to_bf16(v[it][0][c]), hi = to_bf16(v[it][1][c]);
                    t[((4 * cq + c) * kLdsRow + 2 * rp) / 2] = lo | (hi << 16);
                }
            }
        }
    }
};

// partial[blockIdx.x] (F_in x F_out, only the block [i0, i0 + IB) x [j0, j0 + JB)) =
// sum over this workgroup's chunks of bf16(X)^T bf16(G).  Tiles of 16 x 16 go to the
// wavefronts in row-major order, NT per wavefront.
template <int NT, bool XBF, bool GBF>
__global__ __launch_bounds__(kWgThreads) void wgrad_kernel(const void *__restrict__ X,
                                                           const void *__restrict__ G,
                                                           float *__restrict__ partial, int32_t n,
                                                           int32_t F_in, int32_t F_out, int32_t i0,
                                                           int32_t IB, int32_t j0, int32_t JB) {
    extern __shared__ uint32_t lds[];
    uint32_t *xt = lds;                                    // [IB][kLdsRow] bf16
    uint32_t *gt = lds + IB * kLdsRow / 2;                 // [JB][kLdsRow] bf16
    const unsigned short *xt16 = reinterpret_cast<const unsigned short *>(xt);
    const unsigned short *gt16 = reinterpret_cast<const unsigned short *>(gt);

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lrow = lane & 15, kgrp = lane >> 4;
    const int jt_count = JB / 16;
    const int tiles = (IB / 16) * jt_count;

    f32x4 acc[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};

    constexpr int kXItems = (kChunk / 2) * (kMaxIB / 4) / kWgThreads;   // 4
    constexpr int kGItems = (kChunk / 2) * (kMaxJB / 4) / kWgThreads;   // 2
    Stage<XBF, kXItems> xs;
    Stage<GBF, kGItems> gs;
    const int64_t chunks = (static_cast<int64_t>(n) + kChunk - 1) / kChunk;
    int64_t c = blockIdx.x;
    if (c < chunks) {
        xs.load(X, F_in, n, c * kChunk, i0, IB);
        gs.load(G, F_out, n, c * kChunk, j0, JB);
    }
    for (; c < chunks; c += gridDim.x) {
        __syncthreads();                     // the previous chunk's MFMAs are done with LDS
        xs.store(xt, IB);
        gs.store(gt, JB);
        __syncthreads();
        const int64_t next = c + gridDim.x;
        if (next < chunks) {                 // the next chunk is requested during the MFMAs
            xs.load(X, F_in, n, next * kChunk, i0, IB);
            gs.load(G, F_out, n, next * kChunk, j0, JB);
        }
#pragma unroll
        for (int ks = 0; ks < kChunk / 32; ++ks) {
            const int kk = ks * 32 + kgrp * 8;
#pragma unroll
            for (int u = 0; u < NT; ++u) {
                const int t = wave * NT + u;
                if (t < tiles) {
                    const int it = t / jt_count, jt = t % jt_count;
                    const u16x8 a = *reinterpret_cast<const u16x8 *>(xt16 + (it * 16 + lrow) * kLdsRow + kk);
                    const u16x8 b = *reinterpret_cast<const u16x8 *>(gt16 + (jt * 16 + lrow) * kLdsRow + kk);
                    acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), acc[u], 0, 0, 0);
                }
            }
        }
    }
    float *out = partial + static_cast<int64_t>(blockIdx.x) * F_in * F_out;
#pragma unroll
    for (int u = 0; u < NT; ++u) {
        const int t = wave * NT + u;
        if (t < tiles) {
            const int it = t / jt_count, jt = t % jt_count;
#pragma unroll
            for (int r = 0; r < 4; ++r)
                out[static_cast<int64_t>(i0 + it * 16 + kgrp * 4 + r) * F_out + j0 + jt * 16 + lrow] = acc[u][r];
        }
    }
}

// dW[e] = sum over workgroups b (in order) of partial[b][e]; with W, also W[e] -= lr dW[e].
__global__ __launch_bounds__(kThreads) void wgrad_reduce_kernel(const float *__restrict__ partial,
                                                                int32_t count, int64_t elems,
                                                                float *__restrict__ dW, float lr,
                                                                float *__restrict__ W) {
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; e < elems;
         e += static_cast<int64_t>(gridDim.x) * kThreads) {
        double s = 0.0;
        for (int b = 0; b < count; ++b) s += static_cast<double>(partial[b * elems + e]);
        const float d = static_cast<float>(s);
        dW[e] = d;
        if (W) W[e] -= lr * d;
    }
}

int wgrad_blocks(int32_t n) {
    const int64_t chunks = (static_cast<int64_t>(n) + kChunk - 1) / kChunk;
    return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(chunks, kMaxPartials)));
}

template <int NT, bool XBF, bool GBF>
int launch_wgrad_pass(const void *X, const void *G, float *partial, int blocks, int32_t n,
                      int32_t F_in, int32_t F_out, int i0, int IB, int j0, int JB, hipStream_t s) {
    const size_t lds = static_cast<size_t>(IB + JB) * kLdsRow * sizeof(unsigned short);
    hipLaunchKernelGGL((wgrad_kernel<NT, XBF, GBF>), dim3(blocks), dim3(kWgThreads), lds, s, X, G,
                       partial, n, F_in, F_out, i0, IB, j0, JB);
    return hip_status(hipGetLastError());
}

template <bool XBF, bool GBF>
int launch_wgrad_nt(const void *X, const void *G, float *partial, int blocks, int32_t n,
                    int32_t F_in, int32_t F_out, int i0, int IB, int j0, int JB, hipStream_t s) {
    const int per_wave = ((IB / 16) * (JB / 16) + kWgWaves - 1) / kWgWaves;
    if (per_wave <= 4) return launch_wgrad_pass<4, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
    if (per_wave <= 8) return launch_wgrad_pass<8, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
    return launch_wgrad_pass<16, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
}

}  // namespace

int launch_softmax_xent(const float *Y, const int32_t *labels, int32_t n, int32_t C, float scale,
                        float *G, double *loss, hipStream_t s) {
    const int64_t need = (static_cast<int64_t>(n) + kRowsPerBlock - 1) / kRowsPerBlock;
    const int blocks = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(need, kLossBlocks)));
    hipLaunchKernelGGL(softmax_xent_kernel, dim3(blocks), dim3(kThreads), 0, s, Y, labels, n, C,
                       scale, G, loss + 1);
    hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(1), 0, s, loss, blocks, scale);
    return hip_status(hipGetLastError());
}

size_t wgrad_workspace_bytes(int32_t n, int32_t F_in, int32_t F_out) {
    return static_cast<size_t>(wgrad_blocks(n)) * F_in * F_out * sizeof(float);
}

int launch_weight_grad(const void *X, bool x_bf16, const void *G, bool g_bf16, float *dW,
                       int32_t n, int32_t F_in, int32_t F_out, float lr, float *W, void *workspace,
                       hipStream_t s) {
    float *partial = static_cast<float *>(workspace);
    const int blocks = wgrad_blocks(n);
    const int JB = std::min<int>(F_out, kMaxJB);
    const int IB = std::min<int>(F_in, kMaxIB);
    for (int j0 = 0; j0 < F_out; j0 += JB) {
        for (int i0 = 0; i0 < F_in; i0 += IB) {
            const int ib = std::min(IB, F_in - i0), jb = std::min(JB, F_out - j0);
            int st;
            if (x_bf16) {
                st = g_bf16 ? launch_wgrad_nt<true, true>(X, G, partial, blocks, n, F_in, F_out, i0, ib, j0, jb, s)
                            : launch_wgrad_nt<true, false>(X, G, partial, blocks, n, F_in, F_out, i0, ib, j0, jb, s);
            } else {
                st = g_bf16 ? launch_wgrad_nt<false, true>(X, G, partial, blocks, n, F_in, F_out, i0, ib, j0, jb, s)
                            : launch_wgrad_nt<false, false>(X, G, partial, blocks, n, F_in, F_out, i0, ib, j0, jb, s);
            }
            if (st) return st;
        }
    }
    const int64_t elems = static_cast<int64_t>(F_in) * F_out;
    const int rblocks = static_cast<int>(std::min<int64_t>((elems + kThreads - 1) / kThreads, 4096));
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(rblocks), dim3(kThreads), 0, s, partial, blocks,
                       elems, dW, lr, W);
    return hip_status(hipGetLastError());
}

}  // namespace dgc
