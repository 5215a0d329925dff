// Dual-path aggregation SpMM Y = A X on gfx950 (DualGCN Sec. 3.3), and the same
// aggregation fused with the next layer's update, T = bf16(act(A X)) W (further below).
//
// The kernels stream the plan's sorted copy of the matrix: row i of the copy is
// row order[i] of A, the sparse region is rows [0, n_sparse) and the dense region
// rows [n_sparse, n) (Eq. (1) was applied when the plan was built; inside a region
// rows go by row-length octave, then node id).  One launch
// covers both paths; every workgroup picks its path from its index:
//
//   parts      rows of the dense region longer than one chunk, split into parts
//              of the plan's dense chunk (512 to 4096 entries, by the matrix's size;
//              heaviest row first), one wavefront per part
//   long       the other dense rows of at least 2^kLongRowOctave entries (one to
//              three octaves fewer for groups narrower than 32 lanes), one
//              wavefront per row, heaviest first
//   medium     the remaining dense rows, one lane group per row, heaviest first
//   sparse     tasks of up to kTaskRows short consecutive rows, one lane group per
//              task (the paper's "several rows per block")
//
// Feature layout.  A lane group of LPR lanes covers SW = LPR * VEC consecutive
// features of a row: with VEC = 4 every lane makes one 16-byte load, so one
// neighbour costs one coalesced load of the whole row (512 bytes = four 128-byte
// lines at F = 128, 32 lanes).  Features beyond 256 are processed in windows of
// 256; a window may be cut into S slices, workgroup b working on slice b % S
// (used by the one-feature-per-lane path for arbitrary F).  Measured on c4/c5
// (F = 128): cutting rows into 128-byte slices so that each XCD reads only its
// own slice raises the L2 hit rate of a plain gather, but costs more in the SpMM
// than it saves (every slice re-reads the indices and repeats the shuffles), so
// rows are read whole.
//
// Gathers.  A group takes the entries of its row (or task) in rounds of kRound:
// each lane loads kRound / LPR (column, value) pairs with coalesced loads, the
// pairs are broadcast inside the group with shuffles, and all kRound neighbour
// slices are requested before the first product, so every group keeps kRound
// loads in flight (the ILP of the paper's dense path, Alg. 1, deepened).  On large
// operands the rows of cold columns (marked by the plan) are read non-temporally
// (the cache classes below).
//
// Dense path (paper: one row per block, 4-way ILP and a shared reduction): a long
// row gets a wavefront whose groups take rounds of the row in turn and are summed
// with a butterfly over the lanes; a dense row shorter than 2^kLongRowOctave
// entries gets one lane group, which fills its rounds better (measured: the SBM
// workload's dense rows of 100-250 entries run 9% faster than with a wavefront).
// A split row's parts each write a float64 partial, and a small second kernel
// sums them in part order and writes the row.  The kernel boundary makes the
// partials visible: a fence inside the SpMM would write back and invalidate the
// XCD's L2 once per part, which the gathers live on.  No floating-point atomics:
// Y is bit-reproducible.
//
// Sparse path (tasks): the group walks the task's entries as one stream, so even
// rows with one or two entries share a round of kRound gathers; a row is written
// as soon as its last entry has been added.
//
// Summation: products and the sum of one round (<= kRound terms) are float32,
// rounds are added in float64, and each output is rounded once to float32.  The
// error of every element is below ~(kRound + 2) * 2^-24 * sum |a||x|.
#include "internal.h"

#include <algorithm>

namespace dgc {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kRound = 16;            // entries a lane group gathers per round

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

template <int VEC>
__device__ __forceinline__ void load_x(const float *__restrict__ p, float (&x)[VEC]) {
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

// Stores the rounded sums of one lane's VEC features at element offset `at` of Y
// (float32, or bfloat16 rounded from the float32 value when BF).
template <int VEC, bool BF>
__device__ __forceinline__ void store_y(void *__restrict__ Y, int64_t at, const double (&s)[VEC],
                                        bool relu) {
    float o[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        o[j] = static_cast<float>(s[j]);
        if (relu) o[j] = o[j] > 0.f ? o[j] : 0.f;
    }
    if constexpr (BF) {
        unsigned short *p = static_cast<unsigned short *>(Y) + at;
        if constexpr (VEC == 4) {
            const uint2 v = make_uint2(static_cast<uint32_t>(to_bf16(o[0])) | (static_cast<uint32_t>(to_bf16(o[1])) << 16),
                                       static_cast<uint32_t>(to_bf16(o[2])) | (static_cast<uint32_t>(to_bf16(o[3])) << 16));
            __builtin_nontemporal_store(v.x, reinterpret_cast<uint32_t *>(p));
            __builtin_nontemporal_store(v.y, reinterpret_cast<uint32_t *>(p) + 1);
        } else {
#pragma unroll
            for (int j = 0; j < VEC; ++j) __builtin_nontemporal_store(to_bf16(o[j]), p + j);
        }
    } else {
        float *p = static_cast<float *>(Y) + at;
        if constexpr (VEC == 4) {
            const f32x4 v = {o[0], o[1], o[2], o[3]};
            __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
        } else {
#pragma unroll
            for (int j = 0; j < VEC; ++j) __builtin_nontemporal_store(o[j], p + j);
        }
    }
}

struct Args {
    const int32_t *pptr;        // sorted copy of the matrix
    const int32_t *pcol;
    const float *pval;
    const int32_t *perm;        // output row of each sorted row (the plan's order)
    const int32_t *tasks;
    const SplitPart *parts;
    double *partials;
    const float *X;
    void *Y;                    // float32, or bfloat16 when the kernel's BF is set (fused: H or null)
    uint32_t x_bytes;           // bytes of X that gathers may read (cache-class loads)
    int32_t n, n_sparse, n_tasks, n_parts, n_long;
    int32_t dense_chunk;        // entries per part of a split dense row (the plan's)
    int32_t ld;                 // leading dimension of X and Y (= F)
    int32_t f0;                 // first feature of this launch window
    int32_t fend;               // end of the valid features of the window
    int32_t S;                  // feature slices in the window
    int32_t nb_parts;           // logical workgroups of hub-row parts
    int32_t nb_long;            // logical workgroups of long dense rows (a wavefront each)
    int32_t nb_dense;           // nb_long + those of the other dense rows (a group each)
    int32_t relu;
};

// Where a finished row goes.  Rows are emitted by whole lane groups (every lane of
// the group calls row() with the same arguments except its features): `slot` numbers
// the row inside the wavefront's current block of work (group gw, row j of its task:
// gw * kTaskRows + j; a wavefront's long row: 0).
//
// StoreRows writes the row to Y at output row `out`.
template <int VEC, bool BF>
struct StoreRows {
    void *Y;
    int32_t ld;
    bool relu;
    __device__ __forceinline__ void row(int64_t out, int slot, const double (&tot)[VEC], int f,
                                        bool fin) const {
        (void)slot;
        if (fin) store_y<VEC, BF>(Y, out * ld + f, tot, relu);
    }
};

// StageRows keeps the row for the fused update instead: act(row) rounded to bfloat16
// in the wavefront's LDS tile (row `slot`, ld elements apart), its output row in
// outs[slot]; when H is set, the same bfloat16 row is also stored to H (row `out`,
// ldH elements apart), as the plain kernel stores a bfloat16 Y.  VEC = 4; the window
// starts at feature 0.
struct StageRows {
    unsigned short *h;
    int32_t *outs;
    int32_t ld;
    bool relu;
    bool lead;          // the group's first lane records the output row
    unsigned short *H;
    int32_t ldH;
    __device__ __forceinline__ void row(int64_t out, int slot, const double (&tot)[4], int f,
                                        bool fin) const {
        if (fin) {
            float o[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                o[j] = static_cast<float>(tot[j]);
                if (relu) o[j] = o[j] > 0.f ? o[j] : 0.f;
            }
            const uint2 pk =
                make_uint2(static_cast<uint32_t>(to_bf16(o[0])) | (static_cast<uint32_t>(to_bf16(o[1])) << 16),
                           static_cast<uint32_t>(to_bf16(o[2])) | (static_cast<uint32_t>(to_bf16(o[3])) << 16));
            *reinterpret_cast<uint2 *>(h + static_cast<int64_t>(slot) * ld + f) = pk;
            if (H) {
                uint32_t *g = reinterpret_cast<uint32_t *>(H + out * ldH + f);
                __builtin_nontemporal_store(pk.x, g);
                __builtin_nontemporal_store(pk.y, g + 1);
            }
        }
        if (lead) outs[slot] = static_cast<int32_t>(out);
    }
};

// Cache classes of the gathers (kernels instantiated with CP): a gathered row is read
// with the default policy when its column is among the hottest (rows the L2s keep), and
// non-temporal otherwise, so that rows read a few times per launch do not push the hot
// rows out of the L2.  The plan marks the other columns with bit 31 of the sorted copy's
// column (a column is below 2^31 - 1, so a marked one never reads as the invalid -1);
// every kernel masks it off, and it never changes which row is read.
constexpr int kCpolNt = 2;                    // the nt field of a gfx950 buffer load
constexpr uint32_t kRowMask = 0x7FFFFFFFu;

// Entries [e, min(e + kRound, e_end)) of the sorted copy, as seen by lane li of a
// group whose first lane is gbase: lane li loads entries e + li + k LPR; entry u is
// then held by lane u % LPR in register u / LPR.  An invalid entry holds column -1.
template <int LPR>
struct Round {
    static constexpr int EPL = (kRound + LPR - 1) / LPR;   // entries per lane
    int32_t c[EPL];
    float v[EPL];

    __device__ __forceinline__ void load(const Args &a, int32_t e, int32_t e_end, int li) {
#pragma unroll
        for (int k = 0; k < EPL; ++k) {
            const int slot = li + k * LPR;
            const int32_t idx = e + slot;
            const bool ok = slot < kRound && idx < e_end;
            c[k] = ok ? a.pcol[idx] : -1;
            v[k] = ok ? a.pval[idx] : 0.f;
        }
    }
};

template <int POLICY>
__device__ __forceinline__ void load_x_cp(__amdgpu_buffer_rsrc_t rx, uint32_t off, float (&x)[4]) {
    const f32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, POLICY);
    x[0] = v[0];
    x[1] = v[1];
    x[2] = v[2];
    x[3] = v[3];
}

// Requests the kRound neighbour slices of a round (invalid entries read nothing and
// get weight zero).
// The broadcasts read lane gbase + u % LPR with ds_bpermute: the group's base byte
// address is hidden from the optimiser, so that the constant u % LPR lanes go into the
// instruction's offset field instead of one precomputed address register per u
// (sixteen registers held through the whole kernel otherwise).
template <int LPR, int VEC, bool CP>
__device__ __forceinline__ void gather(const Args &a, const Round<LPR> &r, int gbase, int f,
                                       bool fin, float (&as)[kRound], float (&xs)[kRound][VEC]) {
    static_assert(!CP || VEC == 4, "cache classes need 16-byte loads");
    int base4 = gbase * 4;
    asm volatile("" : "+v"(base4));
#pragma unroll
    for (int u = 0; u < kRound; ++u) {
        const int src = base4 + (u % LPR) * 4;
        const int32_t cc = __builtin_amdgcn_ds_bpermute(src, r.c[u / LPR]);
        as[u] = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(r.v[u / LPR])));
        if constexpr (CP) {
            if (cc != -1 && fin) {
                // the host checked that n ld 4 bytes fit the 32-bit range of the buffer
                const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<float *>(a.X), 0, static_cast<int>(a.x_bytes), 0x00020000);
                const uint32_t row = static_cast<uint32_t>(cc) & kRowMask;
                const uint32_t off = (row * static_cast<uint32_t>(a.ld) + static_cast<uint32_t>(f)) * 4u;
                if (cc >= 0) load_x_cp<0>(rx, off, xs[u]);
                else load_x_cp<kCpolNt>(rx, off, xs[u]);      // a marked (cold) column
            } else {
                as[u] = 0.f;
#pragma unroll
                for (int j = 0; j < VEC; ++j) xs[u][j] = 0.f;
            }
        } else {
            if (cc != -1 && fin) {
                load_x<VEC>(a.X + static_cast<int64_t>(static_cast<uint32_t>(cc) & kRowMask) * a.ld + f, xs[u]);
            } else {
                as[u] = 0.f;
#pragma unroll
                for (int j = 0; j < VEC; ++j) xs[u][j] = 0.f;
            }
        }
    }
}

// Dense path: one wavefront accumulates entries [e0, e1) of one row; on return every
// lane holds the row's sums for its features (groups reduced by a butterfly).
template <int LPR, int VEC, bool CP>
__device__ __forceinline__ void dense_row(const Args &a, int32_t e0, int32_t e1, int li, int gw,
                                          int gbase, int f, bool fin, double (&tot)[VEC]) {
    constexpr int GPW = 64 / LPR;
#pragma unroll
    for (int j = 0; j < VEC; ++j) tot[j] = 0.0;
    for (int32_t e = e0 + gw * kRound; e < e1; e += GPW * kRound) {
        Round<LPR> r;
        r.load(a, e, e1, li);
        float as[kRound], xs[kRound][VEC];
        gather<LPR, VEC, CP>(a, r, gbase, f, fin, as, xs);
        float acc[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
#pragma unroll
        for (int u = 0; u < kRound; ++u)
#pragma unroll
            for (int j = 0; j < VEC; ++j) acc[j] = fmaf(as[u], xs[u][j], acc[j]);
#pragma unroll
        for (int j = 0; j < VEC; ++j) tot[j] += static_cast<double>(acc[j]);
    }
#pragma unroll
    for (int m = LPR; m < 64; m <<= 1)
#pragma unroll
        for (int j = 0; j < VEC; ++j) tot[j] += __shfl_xor(tot[j], m, 64);
}

// Selects register j / LPR of a per-lane array and reads it from lane j % LPR.
template <int LPR, int N>
__device__ __forceinline__ int32_t task_meta(const int32_t (&m)[N], int j, int gbase) {
    int32_t x = m[0];
#pragma unroll
    for (int k = 1; k < N; ++k)
        if (j / LPR == k) x = m[k];
    return __shfl(x, gbase + j % LPR, 64);
}

// The work of logical workgroup lb (feature slice `slice`) for wavefront `wave` of a
// workgroup of WAVES wavefronts; finished rows go to `emit`.
template <int LPR, int VEC, int WAVES, bool CP, class Emit>
__device__ __forceinline__ void spmm_block(const Args &a, int lb, int slice, int wave,
                                           const Emit &emit) {
    constexpr int GPW = 64 / LPR;                 // lane groups per wavefront
    constexpr int SW = LPR * VEC;                 // features per slice
    constexpr int RPL = (kTaskRows + LPR - 1) / LPR;

    const int lane = static_cast<int>(threadIdx.x) & 63;
    const int li = lane % LPR;
    const int gw = lane / LPR;
    const int gbase = lane - li;
    const int f = a.f0 + slice * SW + li * VEC;
    const bool fin = f < a.fend;

    if (lb >= a.nb_parts + a.nb_long && lb < a.nb_parts + a.nb_dense) {
        // ---------------- dense path, shorter rows: one lane group per row
        const int64_t gi = (static_cast<int64_t>(lb - a.nb_parts - a.nb_long) * WAVES + wave) * GPW + gw;
        const int64_t i = a.n - a.n_long - 1 - gi;
        if (i < a.n_sparse) return;           // the whole group leaves together
        const int32_t e0 = a.pptr[i], e1 = a.pptr[i + 1];
        double tot[VEC];
#pragma unroll
        for (int j = 0; j < VEC; ++j) tot[j] = 0.0;
        for (int32_t e = e0; e < e1; e += kRound) {
            Round<LPR> r;
            r.load(a, e, e1, li);
            float as[kRound], xs[kRound][VEC];
            gather<LPR, VEC, CP>(a, r, gbase, f, fin, as, xs);
            float acc[VEC];
#pragma unroll
            for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
#pragma unroll
            for (int u = 0; u < kRound; ++u)
#pragma unroll
                for (int j = 0; j < VEC; ++j) acc[j] = fmaf(as[u], xs[u][j], acc[j]);
#pragma unroll
            for (int j = 0; j < VEC; ++j) tot[j] += static_cast<double>(acc[j]);
        }
        emit.row(a.perm[i], gw * kTaskRows, tot, f, fin);
        return;
    }
    if (lb < a.nb_parts + a.nb_long) {
        // ---------------- dense path, long rows: one wavefront per row or per part of a split row
        const int w = lb * WAVES + wave;
        int32_t i, e0, e1;
        int part = -1, first = 0;
        if (lb < a.nb_parts) {
            if (w >= a.n_parts) return;
            const SplitPart sp = a.parts[a.n_parts - 1 - w];
            i = sp.row;
            part = sp.part;
            first = sp.first;
            e0 = a.pptr[i] + part * a.dense_chunk;
            e1 = min(e0 + a.dense_chunk, a.pptr[i + 1]);
        } else {
            i = a.n - 1 - (w - a.nb_parts * WAVES);
            if (i < a.n - a.n_long) return;
            e0 = a.pptr[i];
            e1 = a.pptr[i + 1];
            if (e1 - e0 > a.dense_chunk) return;   // covered by its parts
        }
        double tot[VEC];
        dense_row<LPR, VEC, CP>(a, e0, e1, li, gw, gbase, f, fin, tot);
        if (part < 0) {
            if (gw == 0) emit.row(a.perm[i], 0, tot, f, fin);
            return;
        }
        // a part of a split row: its float64 partial, summed by combine_kernel after this launch
        if (gw == 0 && fin) {
            double *pp = a.partials + static_cast<int64_t>(first + part) * kMaxSlice + (f - a.f0);
#pragma unroll
            for (int j = 0; j < VEC; ++j) pp[j] = tot[j];
        }
        return;
    }

    // ---------------- sparse path: one task (up to kTaskRows short rows) per lane group
    const int64_t t = (static_cast<int64_t>(lb - a.nb_parts - a.nb_dense) * WAVES + wave) * GPW + gw;
    if (t >= a.n_tasks) return;               // the whole group leaves together
    const int32_t r0 = a.tasks[t];
    const int m = a.tasks[t + 1] - r0;        // 1 .. kTaskRows rows
    int32_t rend[RPL], rout[RPL];             // row j: lane j % LPR, register j / LPR
#pragma unroll
    for (int k = 0; k < RPL; ++k) {
        const int j = li + k * LPR;
        rend[k] = j < m ? a.pptr[r0 + j + 1] : 0;
        rout[k] = j < m ? a.perm[r0 + j] : 0;
    }
    const int32_t e_begin = a.pptr[r0];
    const int32_t e_end = task_meta<LPR>(rend, m - 1, gbase);
    if (e_begin == e_end) {                   // a task of empty rows (a run of them is cut
        double z[VEC];                        // into tasks of at most kTaskRows)
#pragma unroll
        for (int j = 0; j < VEC; ++j) z[j] = 0.0;
        for (int j = 0; j < m; ++j) emit.row(task_meta<LPR>(rout, j, gbase), gw * kTaskRows + j, z, f, fin);
        return;
    }
    int cur = 0;                              // every row of a task with entries is non-empty
    int32_t cur_end = task_meta<LPR>(rend, 0, gbase);
    int32_t cur_out = task_meta<LPR>(rout, 0, gbase);
    double tot[VEC];
    float part[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
        tot[j] = 0.0;
        part[j] = 0.f;
    }
    for (int32_t e = e_begin; e < e_end; e += kRound) {
        Round<LPR> r;
        r.load(a, e, e_end, li);
        float as[kRound], xs[kRound][VEC];
        gather<LPR, VEC, CP>(a, r, gbase, f, fin, as, xs);
#pragma unroll
        for (int u = 0; u < kRound; ++u) {
#pragma unroll
            for (int j = 0; j < VEC; ++j) part[j] = fmaf(as[u], xs[u][j], part[j]);
            if (e + u + 1 == cur_end) {       // the current row ends with this entry
#pragma unroll
                for (int j = 0; j < VEC; ++j) {
                    tot[j] += static_cast<double>(part[j]);
                    part[j] = 0.f;
                }
                emit.row(cur_out, gw * kTaskRows + cur, tot, f, fin);
#pragma unroll
                for (int j = 0; j < VEC; ++j) tot[j] = 0.0;
                if (++cur < m) {
                    cur_end = task_meta<LPR>(rend, cur, gbase);
                    cur_out = task_meta<LPR>(rout, cur, gbase);
                }
            }
        }
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
            tot[j] += static_cast<double>(part[j]);
            part[j] = 0.f;
        }
    }
}

template <int LPR, int VEC, bool BF, bool CP>
__global__ __launch_bounds__(kThreads) void spmm_dual_kernel(const Args a) {
    const StoreRows<VEC, BF> emit{a.Y, a.ld, a.relu != 0};
    spmm_block<LPR, VEC, kWaves, CP>(a, static_cast<int>(blockIdx.x) / a.S,
                                 static_cast<int>(blockIdx.x) % a.S,
                                 static_cast<int>(threadIdx.x) >> 6, emit);
}

// The rows split into parts: row = the sum of its parts' float64 partials, in part order.
// One workgroup per part; only a row's first part does the work (a kernel boundary after
// the SpMM makes every partial visible, so no fence or counter is needed).
template <bool BF>
__global__ __launch_bounds__(kThreads) void combine_kernel(const Args a) {
    const SplitPart sp = a.parts[blockIdx.x];
    if (sp.part != 0) return;
    const int t = static_cast<int>(threadIdx.x);
    const int f = a.f0 + t;
    if (f >= a.fend) return;
    const double *pp = a.partials + static_cast<int64_t>(sp.first) * kMaxSlice + t;
    double s[1] = {0.0};
    for (int q = 0; q < sp.nparts; ++q) s[0] += pp[static_cast<int64_t>(q) * kMaxSlice];
    store_y<1, BF>(a.Y, static_cast<int64_t>(a.perm[sp.row]) * a.ld + f, s, a.relu);
}

// ---------------- the aggregation fused with the next layer's update
//
// T = bf16(act(A X)) bf16(W), float32 accumulation: the product of a GCN layer's
// aggregated output with the next layer's weights without storing the aggregated
// features.  The aggregation is the plain kernel's (same schedule, same sums); a
// finished row is rounded to bfloat16 into its wavefront's LDS tile (and, if asked,
// also stored to H as the plain kernel's bfloat16 output) instead of Y.
// Every workgroup stages W^T in bfloat16 once and then takes logical workgroups
// blockIdx.x, blockIdx.x + gridDim.x, ... of the plain kernel's schedule (heaviest
// first as before); after each one, the wavefront multiplies its tile by W^T on the
// matrix cores (v_mfma_f32_16x16x32_bf16, 16-row tiles, k in the update kernel's
// order) and writes the finished rows of T.  Rows go through the same bfloat16
// values and the same MFMA sequence as dualgcn_spmm_act with a bfloat16 output
// followed by dualgcn_update, so both routes give identical T.
//
// MFMA 16x16x32 operands (l = lane): A row l % 16 and B column l % 16, eight
// consecutive k of group l / 16; D rows 4 (l / 16) + j, j < 4, column l % 16.
//
// Occupancy.  A wavefront loads its A fragments of a 16-row tile into registers before
// the tile's products, so the tile's LDS rows are free while its results are staged:
// when a 16-row tile of bfloat16 rows is at least as large as the output staging
// (K >= 128), the staging lives in the tile.  At K = 128, N = 64 that takes a workgroup
// from 51 to 35 KiB of LDS, and the kernel is compiled for 4 wavefronts per SIMD
// (at most 128 registers), so four workgroups share a CU instead of three.
constexpr int kXwPad = 8;                     // bfloat16 padding per LDS row
constexpr int kXwBlocksPerGroup = 8;          // logical workgroups per launched workgroup
constexpr int kXwStageLd = 68;                // floats per staged output row (64 + padding)
constexpr int kXwStageWords = 16 * kXwStageLd; // a wavefront's output staging

template <int LPR>
struct XwTile {
    static constexpr int kSlots = (64 / LPR) * kTaskRows;   // rows a wavefront finishes per block
    static constexpr int kRows = kSlots < 16 ? 16 : kSlots; // rows of its LDS tile
};

// Does a 16-row tile of bfloat16 rows K + kXwPad apart hold a wavefront's output staging?
__host__ __device__ constexpr bool xw_stage_in_tile(int K) {
    return (K + kXwPad) * 2 >= kXwStageLd * 4;
}

size_t xw_lds_bytes(int lpr, int K, int N) {
    const int slots = (64 / lpr) * kTaskRows;
    const size_t rows = slots < 16 ? 16 : slots;
    const size_t ld = static_cast<size_t>(K) + kXwPad;
    return (static_cast<size_t>(N) + kWaves * rows) * ld * sizeof(unsigned short) +
           kWaves * rows * sizeof(int32_t) +
           (xw_stage_in_tile(K) ? 0 : static_cast<size_t>(kWaves) * kXwStageWords * sizeof(float));
}

template <int LPR, bool CP>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4)))
void spmm_xw_kernel(const Args a, const float *__restrict__ W,
                                                           float *__restrict__ T, int32_t K,
                                                           int32_t N, int32_t nblocks) {
    constexpr int ROWS = XwTile<LPR>::kRows;
    extern __shared__ unsigned short xw_lds[];
    const int ld = K + kXwPad;
    const int ntiles = N / 16;
    const int lane = static_cast<int>(threadIdx.x) & 63;
    const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
    unsigned short *wt = xw_lds;                                   // [N][ld]: W^T in bfloat16
    unsigned short *h = xw_lds + (N + wave * ROWS) * ld;           // this wavefront's rows
    int32_t *outs = reinterpret_cast<int32_t *>(xw_lds + (N + kWaves * ROWS) * ld) + wave * ROWS;
    const bool stage_in_tile = xw_stage_in_tile(K);
    float *stage_own = reinterpret_cast<float *>(reinterpret_cast<int32_t *>(xw_lds + (N + kWaves * ROWS) * ld) +
                                                 kWaves * ROWS) + wave * kXwStageWords;
    for (int idx = static_cast<int>(threadIdx.x); idx < K * N; idx += kThreads) {
        const int c = idx / N, j = idx % N;   // consecutive threads read consecutive columns
        wt[j * ld + c] = to_bf16(W[idx]);
    }
    if (lane < ROWS) outs[lane] = -1;
    __syncthreads();

    const StageRows emit{h, outs, ld, a.relu != 0, lane % LPR == 0, static_cast<unsigned short *>(a.Y), a.ld};
    constexpr int KF = LPR / 8;               // A fragments of a row: K <= 4 LPR, 32 k each
    for (int lb = static_cast<int>(blockIdx.x); lb < nblocks; lb += static_cast<int>(gridDim.x)) {
        spmm_block<LPR, 4, kWaves, CP>(a, lb, 0, wave, emit);
        __syncwarp();
        // the lane's MFMA coordinates, recomputed here (hidden from the optimiser) rather
        // than held in registers through the aggregation
        int ln = static_cast<int>(threadIdx.x) & 63;
        asm volatile("" : "+v"(ln));
        const int lrow = ln & 15, kgrp = ln >> 4;
        const int sr = ln >> 4, sc = (ln & 15) * 4;        // first staged row and the columns a lane stores
#pragma unroll
        for (int rt = 0; rt < ROWS / 16; ++rt) {
            if (__ballot(outs[rt * 16 + lrow] >= 0) == 0) continue;   // no row in this tile
            int32_t orow[4];                                          // rows sr + 4 q of the tile
#pragma unroll
            for (int q = 0; q < 4; ++q) orow[q] = outs[rt * 16 + sr + 4 * q];
            const unsigned short *hrow = h + (rt * 16 + lrow) * ld + kgrp * 8;
            u16x8 afrag[KF];
#pragma unroll
            for (int q = 0; q < KF; ++q)
                afrag[q] = q * 32 < K ? *reinterpret_cast<const u16x8 *>(hrow + q * 32) : u16x8{};
            __syncwarp();
            float *stage = stage_in_tile ? reinterpret_cast<float *>(h + rt * 16 * ld) : stage_own;
            // one 16-column tile of T at a time (the k order of each tile is the update's),
            // staged in LDS and stored 64 columns at a time: each store instruction writes
            // four whole 256-byte row pieces (16 lanes x 16 bytes each)
            for (int t = 0; t < ntiles; ++t) {
                const unsigned short *wrow = wt + (t * 16 + lrow) * ld + kgrp * 8;
                f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int q = 0; q < KF; ++q) {
                    if (q * 32 >= K) break;
                    const u16x8 b16 = *reinterpret_cast<const u16x8 *>(wrow + q * 32);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, afrag[q]),
                                                                  __builtin_bit_cast(bf16x8, b16), acc,
                                                                  0, 0, 0);
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) stage[(kgrp * 4 + j) * kXwStageLd + (t & 3) * 16 + lrow] = acc[j];
                if ((t & 3) == 3 || t == ntiles - 1) {
                    __syncwarp();
                    const int c0 = (t & ~3) * 16;                      // first column of this pass
                    if (c0 + sc < N) {
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            if (orow[q] >= 0) {
                                const f32x4 v = *reinterpret_cast<const f32x4 *>(stage + (sr + 4 * q) * kXwStageLd + sc);
                                __builtin_nontemporal_store(
                                    v, reinterpret_cast<f32x4 *>(T + static_cast<int64_t>(orow[q]) * N + c0 + sc));
                            }
                        }
                    }
                    __syncwarp();
                }
            }
        }
        __syncwarp();
        if (lane < ROWS) outs[lane] = -1;
        __syncwarp();
    }
}

// The split rows of the fused product: the row from its parts' partials (as in
// combine_kernel), rounded to bfloat16 as row 0 of a tile whose other rows are zero,
// then the same MFMA sequence on the first wavefront with W read from memory.
__global__ __launch_bounds__(kThreads) void combine_xw_kernel(const Args a, const float *__restrict__ W,
                                                              float *__restrict__ T, int32_t K,
                                                              int32_t N) {
    __shared__ unsigned short hrow[kMaxSlice];
    const SplitPart sp = a.parts[blockIdx.x];
    if (sp.part != 0) return;
    const int t = static_cast<int>(threadIdx.x);
    if (t < K) {
        const double *pp = a.partials + static_cast<int64_t>(sp.first) * kMaxSlice + t;
        double sum = 0.0;
        for (int q = 0; q < sp.nparts; ++q) sum += pp[static_cast<int64_t>(q) * kMaxSlice];
        float o = static_cast<float>(sum);
        if (a.relu) o = o > 0.f ? o : 0.f;
        hrow[t] = to_bf16(o);
        if (a.Y) static_cast<unsigned short *>(a.Y)[static_cast<int64_t>(a.perm[sp.row]) * K + t] = hrow[t];
    }
    __syncthreads();
    if (t >= 64) return;
    const int lrow = t & 15, kgrp = t >> 4;
    const int64_t out = static_cast<int64_t>(a.perm[sp.row]) * N;
    for (int u = 0; u < N / 16; ++u) {
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int kk = kgrp * 8; kk < K; kk += 32) {
            u16x8 a16, b16;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                a16[e] = lrow == 0 ? hrow[kk + e] : static_cast<unsigned short>(0);
                b16[e] = to_bf16(W[static_cast<int64_t>(kk + e) * N + u * 16 + lrow]);
            }
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a16),
                                                          __builtin_bit_cast(bf16x8, b16), acc, 0, 0, 0);
        }
        if (kgrp == 0) T[out + u * 16 + lrow] = acc[0];
    }
}

// Logical workgroups of the plain kernel's schedule (sets the nb_* fields).
template <int LPR>
int64_t schedule_blocks(Args &a) {
    constexpr int GPB = kThreads / LPR;       // sparse tasks per workgroup
    a.nb_parts = (a.n_parts + kWaves - 1) / kWaves;
    a.nb_long = (a.n_long + kWaves - 1) / kWaves;
    a.nb_dense = a.nb_long + (a.n - a.n_sparse - a.n_long + GPB - 1) / GPB;
    const int64_t nb_sparse = (static_cast<int64_t>(a.n_tasks) + GPB - 1) / GPB;
    return static_cast<int64_t>(a.nb_parts) + a.nb_dense + nb_sparse;
}

template <int LPR, bool CP>
int launch_xw_window(Args a, const float *W, float *T, int32_t K, int32_t N, hipStream_t s) {
    const int64_t blocks = schedule_blocks<LPR>(a);
    if (blocks > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    if (blocks > 0) {
        const size_t lds = xw_lds_bytes(LPR, K, N);
        const void *kern = reinterpret_cast<const void *>(&spmm_xw_kernel<LPR, CP>);
        if (lds > 64 * 1024) {
            const int st = hip_status(hipFuncSetAttribute(
                kern, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)));
            if (st) return st;
        }
        // about kXwBlocksPerGroup logical workgroups each, and at least as many workgroups
        // as fit at once (LDS of one CU: 160 KiB; 2048 threads).  Measured on c5 (F 128 -> 64):
        // one pass of resident workgroups over all blocks is 12% slower than this (its static
        // share of blocks finishes unevenly); blocks of ~4 or fewer pay the W staging again.
        const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(2048 / kThreads, (160 * 1024) / lds));
        const int64_t grid = std::min<int64_t>(
            blocks, std::max<int64_t>(per_cu * device_cus(), (blocks + kXwBlocksPerGroup - 1) / kXwBlocksPerGroup));
        hipLaunchKernelGGL((spmm_xw_kernel<LPR, CP>), dim3(static_cast<unsigned>(grid)), dim3(kThreads),
                           lds, s, a, W, T, K, N, static_cast<int32_t>(blocks));
    }
    if (a.n_parts > 0)
        hipLaunchKernelGGL(combine_xw_kernel, dim3(static_cast<unsigned>(a.n_parts)), dim3(kThreads),
                           0, s, a, W, T, K, N);
    return hip_status(hipGetLastError());
}

template <int LPR, int VEC, bool CP = false>
int launch_window(Args a, bool bf, hipStream_t s) {
    const int64_t blocks = schedule_blocks<LPR>(a) * a.S;
    if (blocks == 0) return DUALGCN_OK;
    if (blocks > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    if (bf)
        hipLaunchKernelGGL((spmm_dual_kernel<LPR, VEC, true, CP>), dim3(static_cast<unsigned>(blocks)),
                           dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL((spmm_dual_kernel<LPR, VEC, false, CP>), dim3(static_cast<unsigned>(blocks)),
                           dim3(kThreads), 0, s, a);
    if (a.n_parts > 0) {
        if (bf)
            hipLaunchKernelGGL((combine_kernel<true>), dim3(static_cast<unsigned>(a.n_parts)),
                               dim3(kThreads), 0, s, a);
        else
            hipLaunchKernelGGL((combine_kernel<false>), dim3(static_cast<unsigned>(a.n_parts)),
                               dim3(kThreads), 0, s, a);
    }
    return hip_status(hipGetLastError());
}

Args plan_args(const Plan &p, const float *X, void *Y, int32_t F, bool relu) {
    Args a{};
    a.pptr = p.pptr;
    a.pcol = p.pcol;
    a.pval = p.pval;
    a.perm = p.order;
    a.tasks = p.tasks;
    a.parts = p.parts;
    a.partials = p.partials;
    a.X = X;
    a.Y = Y;
    a.n = p.n;
    a.n_sparse = p.n_sparse;
    a.n_tasks = p.n_tasks;
    a.n_parts = p.n_split_parts;
    a.dense_chunk = p.dense_chunk;
    a.n_long = p.n_long[0];
    a.ld = F;
    a.relu = relu ? 1 : 0;
    return a;
}

// Lane-group width for a window of w features with four features per lane, and the
// class of the long-row bound that goes with it.
int window_lpr(int32_t w) {
    return w <= 4 ? 1 : w <= 8 ? 2 : w <= 16 ? 4 : w <= 32 ? 8 : w <= 64 ? 16 : w <= 128 ? 32 : 64;
}

int long_row_class(int lpr) {
    int cls = 0;
    for (int g = lpr; g < 32 && cls < kLongRowClasses - 1; g *= 2) ++cls;
    return cls;
}

// Cache classes of a launch's gathers (the plan marks every column outside the hottest
// kHotRows; classes apply from operands larger than the 256 MiB memory-side cache, below
// which non-temporal loads would only lose rows that cache holds).  Measured on R-MAT
// graphs with shuffled ids (c5: n = 2^22, 67M entries; c4: n = 2^21, 63M entries),
// F = 128: the layer-1 aggregation fused with the next update 4.27 -> 4.03 ms (c5) and
// 3.72 -> 3.45 ms (c4), the plain SpMM 4.46 -> 4.24 and 3.70 -> 3.47 ms; the L2 hit rate of
// the fused kernel rose from 22.5% to 26.8% and its fetched bytes fell from 28.6 to 27.0 GB.
// Hot sets of 16 MiB or less, or a third class loading warm rows with sc0, were slower.
//
// gather_classes sets the class fields of `a` for gathers of w features of rows ld apart
// and returns true when the launch should use them: the plan marked its cold columns, rows
// are read whole with 16-byte loads, the operand fits the 32-bit offsets of a buffer load,
// and it is larger than the memory-side cache.
bool gather_classes(const Plan &p, int32_t ld, int32_t w, bool vec, Args &a) {
    if (!vec || !p.cold_marked) return false;
    const uint64_t bytes = static_cast<uint64_t>(p.n) * static_cast<uint64_t>(ld) * sizeof(float);
    const uint64_t row_bytes = static_cast<uint64_t>(w) * sizeof(float);
    if (bytes > 0xFFFFFFFFull || static_cast<uint64_t>(p.n) * row_bytes <= kGatherClassMinBytes) return false;
    a.x_bytes = static_cast<uint32_t>(bytes);
    return true;
}

}  // namespace

size_t spmm_xw_lds_bytes(int32_t F_in, int32_t F_out) {
    return xw_lds_bytes(window_lpr(F_in), F_in, F_out);
}

// The fused junction pays where the aggregation is bound by the memory fabric: the
// operand is larger than the memory-side cache (then the n x F_in intermediate it never
// writes or reads back is traffic saved), and the kernel's LDS still lets at least
// kFusedMinGroups workgroups share a CU.  Measured (F_in -> F_out): R-MAT c4 (n = 2^21)
// 128 -> 64 fused 3.42 ms against 3.66 ms for the two calls, 64 -> 32 1.76 against 1.85;
// the SBM c3 (n = 2^18, 128 MiB operand) 0.76 against 0.62 and R-MAT c2 (n = 2^17) 0.33
// against 0.29; 256 -> 128, where one workgroup fills a CU's LDS, 16.0 against 7.85 ms (c4).
constexpr int kFusedMinGroups = 3;

bool fused_junction_pays(const Plan &p, int32_t F_in, int32_t F_out) {
    const size_t lds = xw_lds_bytes(window_lpr(F_in), F_in, F_out);
    const uint64_t groups = (160 * 1024) / lds;
    return static_cast<uint64_t>(p.n) * F_in * sizeof(float) > kGatherClassMinBytes && groups >= kFusedMinGroups;
}

namespace {

// Orders work on stream s after the plan's sorted copy (written on the partition's stream);
// once the copy has been seen complete, launches need no wait (and no barrier packet).
int after_plan(const Plan &p, hipStream_t s) {
    if (!p.ready || p.ready_seen.load(std::memory_order_acquire)) return DUALGCN_OK;
    const hipError_t q = hipEventQuery(p.ready);
    if (q == hipSuccess) {
        p.ready_seen.store(true, std::memory_order_release);
        release_pending(p);
        return DUALGCN_OK;
    }
    if (q != hipErrorNotReady) return hip_status(q);
    return hip_status(hipStreamWaitEvent(s, p.ready, 0));
}

}  // namespace

int launch_spmm_xw(const Plan &p, const float *X, const float *W, float *T, void *H,
                   int32_t F_in, int32_t F_out, bool relu, hipStream_t s) {
    if (const int st = after_plan(p, s)) return st;
    Args a = plan_args(p, X, H, F_in, relu);
    a.f0 = 0;
    a.fend = F_in;
    a.S = 1;
    const int lpr = window_lpr(F_in);
    a.n_long = p.n_long[long_row_class(lpr)];
    const bool cp = gather_classes(p, F_in, F_in, true, a);
    int st = DUALGCN_ERR_UNSUPPORTED;
    if (lpr == 8) st = cp ? launch_xw_window<8, true>(a, W, T, F_in, F_out, s)
                          : launch_xw_window<8, false>(a, W, T, F_in, F_out, s);
    else if (lpr == 16) st = cp ? launch_xw_window<16, true>(a, W, T, F_in, F_out, s)
                                : launch_xw_window<16, false>(a, W, T, F_in, F_out, s);
    else if (lpr == 32) st = cp ? launch_xw_window<32, true>(a, W, T, F_in, F_out, s)
                                : launch_xw_window<32, false>(a, W, T, F_in, F_out, s);
    else if (lpr == 64) st = cp ? launch_xw_window<64, true>(a, W, T, F_in, F_out, s)
                                : launch_xw_window<64, false>(a, W, T, F_in, F_out, s);
    if (st) return st;
    return note_use(p, s);
}

int launch_spmm(const Plan &p, const float *X, void *Y, int32_t F, bool relu, bool bf,
                hipStream_t s) {
    if (const int st = after_plan(p, s)) return st;
    Args a = plan_args(p, X, Y, F, relu);

    const bool vec = (reinterpret_cast<uintptr_t>(X) % 16 == 0) &&
                     (reinterpret_cast<uintptr_t>(Y) % (bf ? 8 : 16) == 0) && (F % 4 == 0);
    int st = DUALGCN_OK;
    for (int32_t f0 = 0; f0 < F && !st; f0 += kMaxSlice) {
        const int32_t w = F - f0 < kMaxSlice ? F - f0 : kMaxSlice;
        a.f0 = f0;
        a.fend = f0 + w;
        if (vec) {
            // whole rows: the smallest power-of-two lane group with 4 features per lane;
            // groups under 32 lanes hand rows from a lower length bound to wavefronts
            a.S = 1;
            a.n_long = p.n_long[long_row_class(window_lpr(w))];
            // cache classes for the widths whose rows fill whole 128-byte lines
            const bool cp = w > 16 && gather_classes(p, F, w, true, a);
            if (w <= 4) st = launch_window<1, 4>(a, bf, s);
            else if (w <= 8) st = launch_window<2, 4>(a, bf, s);
            else if (w <= 16) st = launch_window<4, 4>(a, bf, s);
            else if (w <= 32) st = cp ? launch_window<8, 4, true>(a, bf, s) : launch_window<8, 4>(a, bf, s);
            else if (w <= 64) st = cp ? launch_window<16, 4, true>(a, bf, s) : launch_window<16, 4>(a, bf, s);
            else if (w <= 128) st = cp ? launch_window<32, 4, true>(a, bf, s) : launch_window<32, 4>(a, bf, s);
            else st = cp ? launch_window<64, 4, true>(a, bf, s) : launch_window<64, 4>(a, bf, s);
        } else {
            // any other width or alignment: one feature per lane, 64-feature slices
            a.S = (w + 63) / 64;
            st = launch_window<64, 1>(a, bf, s);
        }
    }
    if (st) return st;
    return note_use(p, s);
}

}  // namespace dgc
