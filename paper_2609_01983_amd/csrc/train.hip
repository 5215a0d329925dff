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
#include <type_traits>

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
        if (!labeled) {                     // zero gradient, whatever the logits: Y is not read
            for (int j = l; j < C; j += kGroup) gr[j] = 0.f;
            continue;
        }
        float m = -INFINITY;
        for (int j = l; j < C; j += kGroup) m = fmaxf(m, y[j]);
        m = group_max(m);
        float s = 0.f;
        for (int j = l; j < C; j += kGroup) s += expf(y[j] - m);
        s = group_sum(s);
        const float inv = 1.f / s;
        for (int j = l; j < C; j += kGroup) {
            const float p = expf(y[j] - m) * inv;
            gr[j] = scale * (p - (j == lab ? 1.f : 0.f));
        }
        if (l == 0) acc += static_cast<double>(logf(s) + m - y[lab]);
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

// The same for C % 4 == 0, C <= 64 QPL, 16-byte aligned rows: every lane keeps QPL float4 of
// each of RPG rows in registers (one read of Y on labeled rows, one write of G), and a group
// has the loads of all RPG rows in flight before it reduces any of them.
template <int QPL, int RPG>
__global__ __launch_bounds__(kThreads) void softmax_xent_vec_kernel(
    const float *__restrict__ Y, const int32_t *__restrict__ labels, int32_t n, int32_t C,
    float scale, float *__restrict__ G, double *__restrict__ partial) {
    __shared__ double sh[kThreads];
    const int g = threadIdx.x / kGroup, l = threadIdx.x % kGroup;
    const int quads = C / 4;
    constexpr int kRowsPerIter = kRowsPerBlock * RPG;
    double acc = 0.0;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * kRowsPerIter; base < n;
         base += static_cast<int64_t>(gridDim.x) * kRowsPerIter) {
        f32x4 v[RPG][QPL];
        int32_t lab[RPG];
#pragma unroll
        for (int r = 0; r < RPG; ++r) {
            const int64_t row = base + r * kRowsPerBlock + g;
            lab[r] = row < n ? labels[row] : -1;
        }
        // an unlabeled row's gradient is zero whatever its logits: Y is read on labeled rows only
#pragma unroll
        for (int r = 0; r < RPG; ++r) {
            const int64_t row = base + r * kRowsPerBlock + g;
            const bool want = lab[r] >= 0 && lab[r] < C;
#pragma unroll
            for (int q = 0; q < QPL; ++q) {
                const int j = l + q * kGroup;
                v[r][q] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
                if (want && j < quads) v[r][q] = *reinterpret_cast<const f32x4 *>(Y + row * C + 4 * j);
            }
        }
#pragma unroll
        for (int r = 0; r < RPG; ++r) {
            const int64_t row = base + r * kRowsPerBlock + g;
            float m = -INFINITY;
#pragma unroll
            for (int q = 0; q < QPL; ++q)
                m = fmaxf(m, fmaxf(fmaxf(v[r][q][0], v[r][q][1]), fmaxf(v[r][q][2], v[r][q][3])));
            m = group_max(m);
            float s = 0.f;
            float ylab = 0.f;
#pragma unroll
            for (int q = 0; q < QPL; ++q) {
                const int j = l + q * kGroup;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    if (4 * j + c == lab[r]) ylab = v[r][q][c];
                    const float e = j < quads ? expf(v[r][q][c] - m) : 0.f;
                    v[r][q][c] = e;
                    s += e;
                }
            }
            s = group_sum(s);
            ylab = group_sum(ylab);
            const bool labeled = lab[r] >= 0 && lab[r] < C;
            const float inv = 1.f / s;
            if (row < n) {
#pragma unroll
                for (int q = 0; q < QPL; ++q) {
                    const int j = l + q * kGroup;
                    if (j < quads) {
                        f32x4 o;
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            o[c] = labeled ? scale * (v[r][q][c] * inv - (4 * j + c == lab[r] ? 1.f : 0.f)) : 0.f;
                        __builtin_nontemporal_store(o, reinterpret_cast<f32x4 *>(G + row * C + 4 * j));
                    }
                }
                if (labeled && l == 0) acc += static_cast<double>(logf(s) + m - ylab);
            }
        }
    }
    const int t = threadIdx.x;
    sh[t] = acc;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) sh[t] += sh[t + h];
        __syncthreads();
    }
    if (t == 0) partial[blockIdx.x] = sh[0];
}

// loss[0] = scale * sum of the partials, by a fixed tree over workgroup order.
__global__ __launch_bounds__(kThreads) void loss_total_kernel(double *__restrict__ loss,
                                                              int32_t count, float scale) {
    __shared__ double sh[kThreads];
    const int t = threadIdx.x;
    double s = 0.0;
    for (int i = t; i < count; i += kThreads) s += loss[1 + i];
    sh[t] = s;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) sh[t] += sh[t + h];
        __syncthreads();
    }
    if (t == 0) loss[0] = static_cast<double>(scale) * sh[0];
}

// ------------------------------------------------------------------ weight gradient

constexpr int kWgThreads = 1024;
constexpr int kWgWaves = kWgThreads / 64;
constexpr int kChunk = 64;                       // rows per LDS stage (two k-steps of 32)
// A transposed LDS row holds the chunk's 64 rows of one column as bfloat16, padded to 68:
// consecutive lanes of a store then hit 64 different banks, and every 8-byte fragment
// read stays aligned.
constexpr int kLdsRow = 68;
constexpr int kLdsRow2 = kLdsRow / 2;            // the same row in 32-bit words
constexpr int kMaxIB = 256;                      // dW rows (X columns) per pass
constexpr int kMaxJB = 128;                      // dW columns (G columns) per pass
constexpr int kMaxPartials = 1024;               // workgroups, hence partial dW matrices

template <bool BF>
struct RawQuad {           // four consecutive elements of a row as stored
    using type = f32x4;
};
template <>
struct RawQuad<true> {
    using type = uint2;
};

// One staged operand: `width` columns (from col0, width % 32 == 0) of a 64-row chunk, held
// by each thread as up to ITEMS items of (row pair, column quad) between the global load
// and the transposed LDS store t[col][row].  Items come in blocks of 8 row pairs x 8
// quads, one block per wavefront instruction: each row's 8 quads are one contiguous
// 128-byte (float32) or 64-byte (bfloat16) segment of memory, and the 64 LDS words a
// store instruction writes fall in 64 different banks.
template <bool BF, int ITEMS>
struct Stage {
    typename RawQuad<BF>::type v[ITEMS][2];

    __device__ __forceinline__ static bool item(int it, int width, int &rp, int &cq) {
        const int w = static_cast<int>(threadIdx.x) + it * kWgThreads;
        const int blk = w >> 6, sub = w & 63;
        const int qb = blk >> 2;
        rp = 8 * (blk & 3) + (sub & 7);
        cq = 8 * qb + (sub >> 3);
        return qb < width / 32;
    }

    // Every lane issues every load, without branches: a row past the end reads row n - 1
    // (n >= 1) and an item outside `width` reads its row's first quad.  With no load under
    // a condition, the compiler counts the loads in flight exactly and waits only for the
    // chunk being stored while the next chunk's loads are still on their way.  store()
    // writes zeros for rows past the end.
    __device__ __forceinline__ void load(const void *src, int64_t ld, int64_t n, int64_t r0,
                                         int col0, int width) {
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            int rp, cq;
            const bool ok = item(it, width, rp, cq);
            const int64_t c = col0 + (ok ? 4 * cq : 0);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t r = r0 + 2 * rp + h;
                const int64_t at = (r < n ? r : n - 1) * ld + c;
                if constexpr (BF)
                    v[it][h] = *reinterpret_cast<const uint2 *>(static_cast<const unsigned short *>(src) + at);
                else
                    v[it][h] = *reinterpret_cast<const f32x4 *>(static_cast<const float *>(src) + at);
            }
        }
    }

    __device__ __forceinline__ static uint32_t bits(const typename RawQuad<BF>::type &q, int c) {
        if constexpr (BF) {
            const uint32_t word = c < 2 ? q.x : q.y;
            return (c & 1) ? word >> 16 : word & 0xFFFFu;
        } else {
            return to_bf16(q[c]);
        }
    }

    // The chunk of rows from r0 into t[col][row] (bfloat16 pairs), zeros past row n.
    __device__ __forceinline__ void store(uint32_t *t, int width, int64_t r0, int64_t n) const {
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            int rp, cq;
            if (item(it, width, rp, cq)) {
                const bool in0 = r0 + 2 * rp < n, in1 = r0 + 2 * rp + 1 < n;
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    t[(4 * cq + c) * kLdsRow2 + rp] = (in0 ? bits(v[it][0], c) : 0u) |
                                                      ((in1 ? bits(v[it][1], c) : 0u) << 16);
            }
        }
    }
};

// Eight consecutive k (rows of the chunk) of transposed row `row`, from two aligned 8-byte
// LDS reads.
__device__ __forceinline__ bf16x8 fragment(const uint32_t *t, int row, int kk) {
    const uint2 *q = reinterpret_cast<const uint2 *>(t + row * kLdsRow2 + kk / 2);
    const uint2 a = q[0], b = q[1];
    return __builtin_bit_cast(bf16x8, make_uint4(a.x, a.y, b.x, b.y));
}

// partial[blockIdx.x] (F_in x F_out, only the block [i0, i0 + IB) x [j0, j0 + JB)) =
// sum over this workgroup's chunks c = blockIdx.x, + gridDim.x, + 2 gridDim.x, ... of
// bf16(X)^T bf16(G), accumulated in that order (two k-steps of 32 rows per chunk).  Tiles
// of 16 x 16 go to the wavefronts in row-major order, NT per wavefront.  The loads of
// chunk c + gridDim.x are in flight while chunk c is stored to LDS and multiplied.
template <int NT, bool XBF, bool GBF>
__global__ __launch_bounds__(kWgThreads) void wgrad_kernel(const void *__restrict__ X,
                                                           const void *__restrict__ G,
                                                           float *__restrict__ partial, int32_t n,
                                                           int32_t F_in, int32_t F_out, int32_t i0,
                                                           int32_t IB, int32_t j0, int32_t JB) {
    extern __shared__ uint32_t lds[];
    uint32_t *xt = lds;                                    // [IB][kLdsRow] bf16
    uint32_t *gt = lds + IB * kLdsRow2;                    // [JB][kLdsRow] bf16

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int lrow = lane & 15, kgrp = lane >> 4;
    const int jt_count = JB / 16;
    const int tiles = (IB / 16) * jt_count;

    f32x4 acc[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u) acc[u] = f32x4{0.f, 0.f, 0.f, 0.f};

    constexpr int kXItems = (kChunk / 2) * (kMaxIB / 4) / kWgThreads;   // 2
    constexpr int kGItems = (kChunk / 2) * (kMaxJB / 4) / kWgThreads;   // 1
    Stage<XBF, kXItems> xs, xn;
    Stage<GBF, kGItems> gs, gn;
    const int64_t chunks = (static_cast<int64_t>(n) + kChunk - 1) / kChunk;
    int64_t c = blockIdx.x;                  // the launch has at most one workgroup per chunk
    xs.load(X, F_in, n, c * kChunk, i0, IB);
    gs.load(G, F_out, n, c * kChunk, j0, JB);
    for (; c < chunks; c += gridDim.x) {
        const int64_t next = c + gridDim.x;  // past the last chunk: rows n - 1, never stored
        xn.load(X, F_in, n, next * kChunk, i0, IB);
        gn.load(G, F_out, n, next * kChunk, j0, JB);
        __syncthreads();                     // the previous chunk's MFMAs are done with LDS
        xs.store(xt, IB, c * kChunk, n);
        gs.store(gt, JB, c * kChunk, n);
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kChunk / 32; ++ks) {
            const int kk = ks * 32 + kgrp * 8;
#pragma unroll
            for (int u = 0; u < NT; ++u) {
                const int t = wave * NT + u;
                if (t < tiles) {
                    const int it = t / jt_count, jt = t % jt_count;
                    acc[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        fragment(xt, it * 16 + lrow, kk), fragment(gt, jt * 16 + lrow, kk), acc[u], 0, 0, 0);
                }
            }
        }
        xs = xn;
        gs = gn;
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

// ------------------------------------------------ both operands bfloat16: transposing reads
//
// The same product (same chunks, k-steps and order of accumulation, hence the same bits)
// when X and G are both stored in bfloat16.  A chunk is copied to LDS row-major, 16 bytes
// per lane, and the matrix-core operands, which need eight consecutive rows of one column
// per lane, come from gfx950's transposing LDS read (ds_read_b64_tr_b16): within each group
// of 16 lanes, lane i receives element i % 4 of the 4-element pieces that lanes
// i / 4, 4 + i / 4, 8 + i / 4 and 12 + i / 4 point at.  So lane 4t + u of a group points at
// row t of its four, columns 4u .. 4u + 3 of the 16-column tile, and receives one column
// over four consecutive rows.
//
// 512 threads: eight wavefronts as 4 x 2 over the dW block, each with up to 4 x 4 tiles of
// 16 x 16 (tile rows wm, wm + 4, ..; tile columns wn, wn + 2, ..), so that a k-step reads
// 4 + 4 fragments per wavefront for 16 products (the row-per-wavefront split of
// wgrad_kernel reads 9 for 8).  LDS rows are kMaxIB (X) and kMaxJB (G) elements long; the
// 16-element blocks of row r are XOR-permuted by (r % 4) + 4 ((r / 8) % 2), which puts the
// 16 rows one transposing read touches on eight different 32-byte bank groups, two each.
constexpr int kTrThreads = 512;
constexpr int kTrTiles = 4;                       // tile rows and tile columns per wavefront
constexpr int kTrXItems = kChunk * kMaxIB / 8 / kTrThreads;   // 16-byte pieces per thread: 4
constexpr int kTrGItems = kChunk * kMaxJB / 8 / kTrThreads;   // 2
constexpr int kTrBufElems = kChunk * (kMaxIB + kMaxJB);       // one chunk of X and G in LDS

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int tr_swizzle(int r) {
    return (r & 3) | ((r >> 1) & 4);
}

// `width` columns (from col0) of a 64-row chunk of a bfloat16 matrix, 16 bytes per item.
// Loads are unconditional (rows past the end read row n - 1, items past the chunk read its
// first piece), so the compiler waits only for the chunk it stores; rows past the end are
// stored as zeros.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int ITEMS>
struct RowStage {
    u32x4 v[ITEMS];

    __device__ __forceinline__ void load(const unsigned short *src, int64_t ld, int64_t n,
                                         int64_t r0, int col0, int width) {
        const int per_row = width / 8, total = kChunk * per_row;
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            int p = static_cast<int>(threadIdx.x) + it * kTrThreads;
            p = p < total ? p : 0;
            const int64_t r = r0 + p / per_row;
            v[it] = *reinterpret_cast<const u32x4 *>(src + (r < n ? r : n - 1) * ld + col0 + (p % per_row) * 8);
        }
    }

    // t: [kChunk][pitch] bfloat16, blocks of 16 elements permuted per row
    __device__ __forceinline__ void store(unsigned short *t, int pitch, int64_t r0, int64_t n,
                                          int width) const {
        const int per_row = width / 8, total = kChunk * per_row;
#pragma unroll
        for (int it = 0; it < ITEMS; ++it) {
            const int p = static_cast<int>(threadIdx.x) + it * kTrThreads;
            if (p < total) {                                  // uniform over a wavefront
                const int row = p / per_row, c8 = p % per_row;
                const uint32_t keep = r0 + row < n ? ~0u : 0u;
                *reinterpret_cast<u32x4 *>(t + row * pitch + (((c8 >> 1) ^ tr_swizzle(row)) << 4) + (c8 & 1) * 8) =
                    v[it] & keep;
            }
        }
    }
};

// The 16 x 32 operand of tile columns [c0, c0 + 16) over rows [kb, kb + 32) of t: lane
// (16 g + s) gets column c0 + s at rows kb + 8 g .. kb + 8 g + 7.
__device__ __forceinline__ bf16x8 tr_fragment(const unsigned short *t, int pitch, int kb, int c0,
                                              int lane) {
    const int s = lane & 15, g = lane >> 4;
    const int r = kb + 8 * g + (s >> 2);
    const int col = (((c0 >> 4) ^ tr_swizzle(r)) << 4) + 4 * (s & 3);   // rows r and r + 4 share the permutation
    typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(t + r * pitch + col));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(t + (r + 4) * pitch + col));
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

__global__ __launch_bounds__(kTrThreads) void wgrad_tr_kernel(const unsigned short *__restrict__ X,
                                                              const unsigned short *__restrict__ G,
                                                              float *__restrict__ partial, int32_t n,
                                                              int32_t F_in, int32_t F_out, int32_t i0,
                                                              int32_t IB, int32_t j0, int32_t JB) {
    extern __shared__ uint4 lds4[];
    unsigned short *xt = reinterpret_cast<unsigned short *>(lds4);   // [kChunk][kMaxIB]
    unsigned short *gt = xt + kChunk * kMaxIB;                         // [kChunk][kMaxJB]

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int it_count = IB / 16, jt_count = JB / 16;

    f32x4 acc[kTrTiles][kTrTiles];
#pragma unroll
    for (int a = 0; a < kTrTiles; ++a)
#pragma unroll
        for (int b = 0; b < kTrTiles; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

    RowStage<kTrXItems> xs, xn;
    RowStage<kTrGItems> gs, gn;
    const int64_t chunks = (static_cast<int64_t>(n) + kChunk - 1) / kChunk;
    int64_t c = blockIdx.x;                  // the launch has at most one workgroup per chunk
    xs.load(X, F_in, n, c * kChunk, i0, IB);
    gs.load(G, F_out, n, c * kChunk, j0, JB);
    for (; c < chunks; c += gridDim.x) {
        const int64_t next = c + gridDim.x;  // past the last chunk: rows n - 1, never stored
        xn.load(X, F_in, n, next * kChunk, i0, IB);
        gn.load(G, F_out, n, next * kChunk, j0, JB);
        __syncthreads();                     // the previous chunk's products are done with LDS
        xs.store(xt, kMaxIB, c * kChunk, n, IB);
        gs.store(gt, kMaxJB, c * kChunk, n, JB);
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kChunk / 32; ++ks) {
            bf16x8 af[kTrTiles], bf[kTrTiles];
#pragma unroll
            for (int a = 0; a < kTrTiles; ++a)
                if (wm + 4 * a < it_count) af[a] = tr_fragment(xt, kMaxIB, ks * 32, (wm + 4 * a) * 16, lane);
#pragma unroll
            for (int b = 0; b < kTrTiles; ++b)
                if (wn + 2 * b < jt_count) bf[b] = tr_fragment(gt, kMaxJB, ks * 32, (wn + 2 * b) * 16, lane);
#pragma unroll
            for (int a = 0; a < kTrTiles; ++a)
#pragma unroll
                for (int b = 0; b < kTrTiles; ++b)
                    if (wm + 4 * a < it_count && wn + 2 * b < jt_count)
                        acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bf[b], acc[a][b], 0, 0, 0);
        }
        xs = xn;
        gs = gn;
    }
    float *out = partial + static_cast<int64_t>(blockIdx.x) * F_in * F_out;
    const int s = lane & 15, g = lane >> 4;
#pragma unroll
    for (int a = 0; a < kTrTiles; ++a)
#pragma unroll
        for (int b = 0; b < kTrTiles; ++b) {
            const int it = wm + 4 * a, jt = wn + 2 * b;
            if (it < it_count && jt < jt_count) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    out[static_cast<int64_t>(i0 + it * 16 + g * 4 + r) * F_out + j0 + jt * 16 + s] = acc[a][b][r];
            }
        }
}

// dW[e] = sum over workgroups b of partial[b][e] in float64: eight threads sum consecutive
// eighths of the partials in order, then the eight sums are added in order; with W, also
// W[e] -= lr dW[e].  A workgroup covers 32 consecutive elements.
constexpr int kReduceSegs = 8;
constexpr int kReduceElems = kThreads / kReduceSegs;
__global__ __launch_bounds__(kThreads) void wgrad_reduce_kernel(const float *__restrict__ partial,
                                                                int32_t count, int64_t elems,
                                                                float *__restrict__ dW, float lr,
                                                                float *__restrict__ W) {
    __shared__ double sh[kReduceSegs][kReduceElems];
    const int el = threadIdx.x % kReduceElems, seg = threadIdx.x / kReduceElems;
    const int per = (count + kReduceSegs - 1) / kReduceSegs;
    for (int64_t e0 = static_cast<int64_t>(blockIdx.x) * kReduceElems; e0 < elems;
         e0 += static_cast<int64_t>(gridDim.x) * kReduceElems) {
        const int64_t e = e0 + el;
        double s = 0.0;
        if (e < elems) {
            const int b1 = min(count, (seg + 1) * per);
            for (int b = seg * per; b < b1; ++b) s += static_cast<double>(partial[b * elems + e]);
        }
        sh[seg][el] = s;
        __syncthreads();
        if (seg == 0 && e < elems) {
            double t = 0.0;
#pragma unroll
            for (int k = 0; k < kReduceSegs; ++k) t += sh[k][el];
            const float d = static_cast<float>(t);
            dW[e] = d;
            if (W) W[e] -= lr * d;
        }
        __syncthreads();
    }
}

// Upper bound of the workgroups (partials) of one product over n rows.
int wgrad_max_blocks(int32_t n) {
    const int64_t chunks = (static_cast<int64_t>(n) + kChunk - 1) / kChunk;
    return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(chunks, kMaxPartials)));
}

size_t wgrad_lds_bytes(int IB, int JB) {
    return static_cast<size_t>(IB + JB) * kLdsRow * sizeof(unsigned short);
}
static_assert((kMaxIB + kMaxJB) * kLdsRow * sizeof(unsigned short) <= 64 * 1024 &&
                  kTrBufElems * sizeof(unsigned short) <= 64 * 1024,
              "weight-gradient LDS within the default dynamic limit");

// One pass over the rows for the dW block [i0, i0 + IB) x [j0, j0 + JB).
template <int NT, bool XBF, bool GBF>
int launch_wgrad_pass(const void *X, const void *G, float *partial, int blocks, int32_t n,
                      int32_t F_in, int32_t F_out, int i0, int IB, int j0, int JB, hipStream_t s) {
    hipLaunchKernelGGL((wgrad_kernel<NT, XBF, GBF>), dim3(blocks), dim3(kWgThreads),
                       wgrad_lds_bytes(IB, JB), s, X, G, partial, n, F_in, F_out, i0, IB, j0, JB);
    return hip_status(hipGetLastError());
}

template <bool XBF, bool GBF>
int launch_wgrad_nt(const void *X, const void *G, float *partial, int blocks, int32_t n,
                    int32_t F_in, int32_t F_out, int i0, int IB, int j0, int JB, hipStream_t s) {
    const int per_wave = ((IB / 16) * (JB / 16) + kWgWaves - 1) / kWgWaves;
    if (per_wave <= 2)
        return launch_wgrad_pass<2, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
    if (per_wave <= 4)
        return launch_wgrad_pass<4, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
    return launch_wgrad_pass<8, XBF, GBF>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
}

int launch_wgrad_any(bool x_bf16, bool g_bf16, const void *X, const void *G, float *partial,
                     int blocks, int32_t n, int32_t F_in, int32_t F_out, int i0, int IB, int j0,
                     int JB, hipStream_t s) {
    if (x_bf16 && g_bf16) {
        hipLaunchKernelGGL(wgrad_tr_kernel, dim3(blocks), dim3(kTrThreads),
                           kTrBufElems * sizeof(unsigned short), s, static_cast<const unsigned short *>(X),
                           static_cast<const unsigned short *>(G), partial, n, F_in, F_out, i0, IB, j0, JB);
        return hip_status(hipGetLastError());
    }
    if (x_bf16)
        return launch_wgrad_nt<true, false>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
    return g_bf16 ? launch_wgrad_nt<false, true>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s)
                  : launch_wgrad_nt<false, false>(X, G, partial, blocks, n, F_in, F_out, i0, IB, j0, JB, s);
}

}  // namespace

int launch_softmax_xent(const float *Y, const int32_t *labels, int32_t n, int32_t C, float scale,
                        float *G, double *loss, hipStream_t s) {
    const bool vec = C % 4 == 0 && C <= 4 * 4 * kGroup && reinterpret_cast<uintptr_t>(Y) % 16 == 0 &&
                     reinterpret_cast<uintptr_t>(G) % 16 == 0;
    const int rows_per_block = vec && C <= 4 * kGroup ? kRowsPerBlock * 4 : kRowsPerBlock;
    const int64_t need = (static_cast<int64_t>(n) + rows_per_block - 1) / rows_per_block;
    const int blocks = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(need, kLossBlocks)));
    if (vec && C <= 4 * kGroup)
        hipLaunchKernelGGL((softmax_xent_vec_kernel<1, 4>), dim3(blocks), dim3(kThreads), 0, s, Y,
                           labels, n, C, scale, G, loss + 1);
    else if (vec)
        hipLaunchKernelGGL((softmax_xent_vec_kernel<4, 1>), dim3(blocks), dim3(kThreads), 0, s, Y,
                           labels, n, C, scale, G, loss + 1);
    else
        hipLaunchKernelGGL(softmax_xent_kernel, dim3(blocks), dim3(kThreads), 0, s, Y, labels, n, C,
                           scale, G, loss + 1);
    hipLaunchKernelGGL(loss_total_kernel, dim3(1), dim3(kThreads), 0, s, loss, blocks, scale);
    return hip_status(hipGetLastError());
}

size_t wgrad_workspace_bytes(int32_t n, int32_t F_in, int32_t F_out) {
    return static_cast<size_t>(wgrad_max_blocks(n)) * F_in * F_out * sizeof(float);
}

// Workgroups (partial dW matrices) of one weight-gradient product on the current device:
// one per CU (each kernel's workgroup fills a CU's registers: 16 wavefronts of up to 128
// VGPRs, or 8 of up to 256), at most one per chunk and kMaxPartials.  The count depends
// only on the device and n, never on the operand types, so every kernel sums the same
// chunks into the same partials in the same order.
int wgrad_blocks(int32_t n) {
    return std::max(1, std::min(wgrad_max_blocks(n), device_cus()));
}

int launch_weight_grad(const void *X, bool x_bf16, const void *G, bool g_bf16, float *dW,
                       int32_t n, int32_t F_in, int32_t F_out, float lr, float *W, void *workspace,
                       hipStream_t s) {
    float *partial = static_cast<float *>(workspace);
    const int JB = std::min<int>(F_out, kMaxJB);
    const int IB = std::min<int>(F_in, kMaxIB);
    const int blocks = wgrad_blocks(n);
    for (int j0 = 0; j0 < F_out; j0 += JB) {
        for (int i0 = 0; i0 < F_in; i0 += IB) {
            const int ib = std::min(IB, F_in - i0), jb = std::min(JB, F_out - j0);
            const int st = launch_wgrad_any(x_bf16, g_bf16, X, G, partial, blocks, n, F_in, F_out,
                                            i0, ib, j0, jb, s);
            if (st) return st;
        }
    }
    const int64_t elems = static_cast<int64_t>(F_in) * F_out;
    const int rblocks = static_cast<int>(std::min<int64_t>((elems + kReduceElems - 1) / kReduceElems, 8192));
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3(rblocks), dim3(kThreads), 0, s, partial, blocks,
                       elems, dW, lr, W);
    return hip_status(hipGetLastError());
}

// ------------------------------------------------------------------ without allocation
//
// The partial dW matrices of launch_weight_grad in a static device array instead of a
// caller's workspace, for callers that cannot allocate.  Each device holds its own copy
// of the array (for the life of the process); host code must not pass the array's name to
// a kernel (in host code it is only a stand-in for the symbol), so its address on each
// device is looked up once, with that device current, and kept.  Every partial a product
// uses is written in full before it is read, so the array needs no clearing; two calls that
// overlap on one device share it and race.
namespace {

__device__ __align__(256) float scratch[DUALGCN_WGRAD_NOALLOC_BYTES / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device (looked up on first use there).
int scratch_address(void **out) {
    int dev = 0;
    int st = hip_status(hipGetDevice(&dev));
    if (st) return st;
    if (dev < 0 || dev >= kMaxDevices) return DUALGCN_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void *p = nullptr;
        if ((st = hip_status(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))))) return st;
        if (!p) return DUALGCN_ERR_HIP;
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return DUALGCN_OK;
}

}  // namespace

int wgrad_noalloc_bytes(bool x_bf16, bool g_bf16, int32_t n, int32_t F_in, int32_t F_out,
                        size_t *bytes) {
    *bytes = static_cast<size_t>(wgrad_blocks(n)) * F_in * F_out * sizeof(float);
    return DUALGCN_OK;
}

int launch_weight_grad_noalloc(const void *X, bool x_bf16, const void *G, bool g_bf16, float *dW,
                               int32_t n, int32_t F_in, int32_t F_out, float lr, float *W,
                               hipStream_t s) {
    size_t need = 0;
    int st = wgrad_noalloc_bytes(x_bf16, g_bf16, n, F_in, F_out, &need);
    if (st) return st;
    if (need > DUALGCN_WGRAD_NOALLOC_BYTES) return DUALGCN_ERR_UNSUPPORTED;
    void *partial = nullptr;
    if ((st = scratch_address(&partial))) return st;
    return launch_weight_grad(X, x_bf16, G, g_bf16, dW, n, F_in, F_out, lr, W, partial, s);
}

}  // namespace dgc

