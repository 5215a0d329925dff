// Dual-path aggregation SpMM Y = A X on gfx950 (DualGCN Sec. 3.3).
//
// One launch; every workgroup picks its path from its index (Eq. (1) was
// applied when the plan was built, so the paths are contiguous index ranges):
//
//   [0, n_parts)                    parts of dense rows longer than one chunk,
//                                   heaviest row first
//   [n_parts, n_parts + n_dense)    whole dense rows, heaviest first
//   [.., + sparse blocks)           sparse rows, several per workgroup
//
// Feature layout (both paths): a row of X is read by a lane group of LPR lanes,
// each lane holding VEC consecutive features (float4 loads when VEC = 4), so one
// neighbour costs one coalesced load of LPR*VEC*4 bytes per group.  The group
// loads LPR (column, value) pairs of its batch with one coalesced load and
// passes them lane to lane with shuffles; up to 8 neighbour rows are in flight
// per lane (the ILP of the paper's dense path, re-derived for 64-lane waves).
//
// Sparse path (paper: several rows per block, warp-feature association): one
// row per lane group, 64/LPR rows per wavefront; each row is written once.
//
// Dense path (paper: one row per block, 4-way ILP, shared-memory reduction):
// the workgroup's 256/LPR lane groups take the row's batches round robin and
// the group partials are summed in LDS in group order.  Rows longer than one
// chunk are split over several workgroups: each writes a float64 partial, and
// the last one to arrive (integer counter) sums the parts in part order, writes
// the row and clears the counter.  No floating-point atomics: Y is
// bit-reproducible.
//
// Summation: products and the sum of one batch (<= LPR <= 64 terms) are float32;
// batch sums, group sums and part sums are float64; the output is rounded once.
// The error of every element is then below ~(LPR + 2) * 2^-24 * sum |a||x|.
#include "internal.h"

namespace dgc {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int VEC>
__device__ __forceinline__ void load_row(const float *__restrict__ p, float (&x)[VEC]) {
    if constexpr (VEC == 4) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(p);
        x[0] = v[0];
        x[1] = v[1];
        x[2] = v[2];
        x[3] = v[3];
    } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) x[j] = p[j];
    }
}

template <int VEC>
__device__ __forceinline__ void store_row(float *__restrict__ p, const double (&s)[VEC], bool relu) {
    float o[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        o[j] = static_cast<float>(s[j]);
        if (relu) o[j] = o[j] > 0.f ? o[j] : 0.f;
    }
    if constexpr (VEC == 4) {
        const f32x4 v = {o[0], o[1], o[2], o[3]};
        __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
    } else {
#pragma unroll
        for (int j = 0; j < VEC; ++j) __builtin_nontemporal_store(o[j], p + j);
    }
}

// Accumulates entries [first, last) of one CSR row, in batches of LPR entries
// starting at `first` and then every `step` entries, into tot (float64).
template <int LPR, int VEC>
__device__ __forceinline__ void gather_rows(const int32_t *__restrict__ col,
                                            const float *__restrict__ val,
                                            const float *__restrict__ X, int64_t ldx, int f,
                                            bool fin, int li, int32_t first, int32_t last,
                                            int32_t step, double (&tot)[VEC]) {
    constexpr int U = LPR < 8 ? LPR : 8;
    for (int32_t base = first; base < last; base += step) {
        const int cnt = min(LPR, last - base);
        int32_t c = 0;
        float a = 0.f;
        if (li < cnt) {
            c = col[base + li];
            a = val[base + li];
        }
        float acc[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
        for (int t = 0; t < cnt; t += U) {
            float xs[U][VEC];
            float as[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int src = t + u;
                const int32_t cc = __shfl(c, src, LPR);
                as[u] = __shfl(a, src, LPR);
                if (src < cnt && fin) {
                    load_row<VEC>(X + static_cast<int64_t>(cc) * ldx + f, xs[u]);
                } else {
                    as[u] = 0.f;
#pragma unroll
                    for (int j = 0; j < VEC; ++j) xs[u][j] = 0.f;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int j = 0; j < VEC; ++j) acc[j] = fmaf(as[u], xs[u][j], acc[j]);
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) tot[j] += static_cast<double>(acc[j]);
    }
}

struct Args {
    const int32_t *perm;
    int32_t n, n_sparse;
    const SplitPart *parts;
    int32_t n_parts;
    int32_t n_dense_blocks;     // n_parts + (n - n_sparse)
    int32_t *counters;
    double *partials;
    const int32_t *rowptr;
    const int32_t *col;
    const float *val;
    const float *X;
    float *Y;
    int32_t F;                  // leading dimension of X and Y
    int32_t f0;                 // first feature of this slice
    int32_t relu;
};

template <int LPR, int VEC>
__global__ __launch_bounds__(kThreads) void spmm_dual_kernel(const Args a) {
    constexpr int G = kThreads / LPR;       // lane groups per workgroup
    constexpr int SW = LPR * VEC;           // features per slice
    __shared__ double red[G][SW];
    __shared__ int last_flag;

    const int b = static_cast<int>(blockIdx.x);
    const int li = static_cast<int>(threadIdx.x) % LPR;
    const int f = a.f0 + li * VEC;
    const bool fin = (VEC == 1) ? (f < a.F) : true;

    if (b >= a.n_dense_blocks) {
        // ---------------- sparse path: one row per lane group
        constexpr int GPW = 64 / LPR;
        const int lane = static_cast<int>(threadIdx.x) & 63;
        const int64_t gid = (static_cast<int64_t>(b - a.n_dense_blocks) * kWaves +
                             (threadIdx.x >> 6)) * GPW + lane / LPR;
        if (gid >= a.n_sparse) return;
        const int32_t r = a.perm[gid];
        double tot[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) tot[j] = 0.0;
        gather_rows<LPR, VEC>(a.col, a.val, a.X, a.F, f, fin, li, a.rowptr[r], a.rowptr[r + 1],
                              LPR, tot);
        if (fin) store_row<VEC>(a.Y + static_cast<int64_t>(r) * a.F + f, tot, a.relu);
        return;
    }

    // ---------------- dense path: one workgroup per row (or per part of a long row)
    int32_t r, p0, p1;
    int part = -1, nparts = 1, first = 0;
    if (b < a.n_parts) {
        const SplitPart sp = a.parts[a.n_parts - 1 - b];
        r = sp.row;
        part = sp.part;
        nparts = sp.nparts;
        first = sp.first;
        const int32_t row_end = a.rowptr[r + 1];
        p0 = a.rowptr[r] + part * kDenseChunk;
        p1 = min(p0 + kDenseChunk, row_end);
    } else {
        const int32_t i = a.n - 1 - (b - a.n_parts);
        r = a.perm[i];
        p0 = a.rowptr[r];
        p1 = a.rowptr[r + 1];
        if (p1 - p0 > kDenseChunk) return;   // this row is covered by its parts
    }
    const int g = static_cast<int>(threadIdx.x) / LPR;
    double tot[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) tot[j] = 0.0;
    gather_rows<LPR, VEC>(a.col, a.val, a.X, a.F, f, fin, li, p0 + g * LPR, p1, G * LPR, tot);
#pragma unroll
    for (int j = 0; j < VEC; ++j) red[g][li * VEC + j] = tot[j];
    __syncthreads();
    const int t = static_cast<int>(threadIdx.x);
    const int ft = a.f0 + t;
    if (part < 0) {
        if (t < SW && ft < a.F) {
            double s = 0.0;
#pragma unroll 4
            for (int q = 0; q < G; ++q) s += red[q][t];
            float o = static_cast<float>(s);
            if (a.relu) o = o > 0.f ? o : 0.f;
            __builtin_nontemporal_store(o, a.Y + static_cast<int64_t>(r) * a.F + ft);
        }
        return;
    }
    if (t < SW) {
        double s = 0.0;
#pragma unroll 4
        for (int q = 0; q < G; ++q) s += red[q][t];
        __hip_atomic_store(a.partials + static_cast<int64_t>(first + part) * kMaxSlice + t, s,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __threadfence();      // publish this part before counting it
    __syncthreads();
    if (t == 0) last_flag = atomicAdd(&a.counters[first], 1) == nparts - 1;
    __syncthreads();
    if (!last_flag) return;
    __threadfence();      // see every other part
    if (t < SW && ft < a.F) {
        double s = 0.0;
        for (int q = 0; q < nparts; ++q)
            s += __hip_atomic_load(a.partials + static_cast<int64_t>(first + q) * kMaxSlice + t,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        float o = static_cast<float>(s);
        if (a.relu) o = o > 0.f ? o : 0.f;
        __builtin_nontemporal_store(o, a.Y + static_cast<int64_t>(r) * a.F + ft);
    }
    if (t == 0) a.counters[first] = 0;   // ready for the next call on this plan
}

template <int LPR, int VEC>
int launch_slice(Args a, hipStream_t s) {
    constexpr int rows_per_block = kWaves * (64 / LPR);
    const int64_t sparse_blocks = (static_cast<int64_t>(a.n_sparse) + rows_per_block - 1) / rows_per_block;
    const int64_t blocks = static_cast<int64_t>(a.n_dense_blocks) + sparse_blocks;
    if (blocks == 0) return DUALGCN_OK;
    if (blocks > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    hipLaunchKernelGGL((spmm_dual_kernel<LPR, VEC>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kThreads), 0, s, a);
    return hip_status(hipGetLastError());
}

}  // namespace

int launch_spmm(const Plan &p, const float *X, float *Y, int32_t F, bool relu, hipStream_t s) {
    Args a{};
    a.perm = p.perm;
    a.n = p.n;
    a.n_sparse = p.n_sparse;
    a.parts = p.parts;
    a.n_parts = p.n_split_parts;
    a.n_dense_blocks = p.n_split_parts + (p.n - p.n_sparse);
    a.counters = p.counters;
    a.partials = p.partials;
    a.rowptr = p.rowptr;
    a.col = p.col;
    a.val = p.val;
    a.X = X;
    a.Y = Y;
    a.F = F;
    a.relu = relu ? 1 : 0;

    const bool aligned = (reinterpret_cast<uintptr_t>(X) % 16 == 0) &&
                         (reinterpret_cast<uintptr_t>(Y) % 16 == 0) && (F % 4 == 0);
    int st = DUALGCN_OK;
    if (aligned && (F == 4 || F == 8 || F == 16 || F == 32 || F == 64 || F == 128 || F == 256)) {
        a.f0 = 0;
        switch (F) {
            case 4: return launch_slice<1, 4>(a, s);
            case 8: return launch_slice<2, 4>(a, s);
            case 16: return launch_slice<4, 4>(a, s);
            case 32: return launch_slice<8, 4>(a, s);
            case 64: return launch_slice<16, 4>(a, s);
            case 128: return launch_slice<32, 4>(a, s);
            default: return launch_slice<64, 4>(a, s);
        }
    }
    if (aligned && F % 256 == 0) {
        for (int32_t f0 = 0; f0 < F && !st; f0 += 256) {
            a.f0 = f0;
            st = launch_slice<64, 4>(a, s);
        }
        return st;
    }
    for (int32_t f0 = 0; f0 < F && !st; f0 += 64) {
        a.f0 = f0;
        st = launch_slice<64, 1>(a, s);
    }
    return st;
}

}  // namespace dgc
