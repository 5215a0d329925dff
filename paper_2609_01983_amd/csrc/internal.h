// Internal declarations shared by the translation units of libdualgcn.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstddef>
#include <cstdint>
#include <mutex>
#include <utility>
#include <vector>

#include "dualgcn.h"

#include <rocprofiler-sdk-roctx/roctx.h>

namespace dgc {

// A named range for tracers (roctx; a call into the marker library and nothing more when
// no tool listens).  next() closes the current range and opens the following one.
class TraceRange {
   public:
    explicit TraceRange(const char *name) { roctxRangePush(name); }
    ~TraceRange() { roctxRangePop(); }
    TraceRange(const TraceRange &) = delete;
    TraceRange &operator=(const TraceRange &) = delete;
    void next(const char *name) {
        roctxRangePop();
        roctxRangePush(name);
    }
};

using u128 = unsigned __int128;

// Entries of one dense row handled by one wavefront (a plan's dense chunk); longer rows are
// split into parts of this many entries and combined in a fixed order.  A wavefront takes a
// part in C / 64 rounds of dependent loads (F = 128), while the whole matrix spread over the
// ~4096 wavefronts the chip holds needs about nnz / 2^18 rounds: the chunk is the largest
// power of two up to kMaxDenseChunk with C <= nnz / 2048, so that no part takes more than
// about twice the launch's rounds, and at least kMinDenseChunk (the long-row bound, below
// which a dense row is a lane group's).  Matrices of fewer than kSplitMinEntries entries keep
// the largest chunk: their launches last a few microseconds, less than splitting would add
// (the kernel that combines the parts).
constexpr int kMaxDenseChunk = 4096;
constexpr int kMinDenseChunk = 512;
constexpr int64_t kSplitMinEntries = int64_t{1} << 20;
inline int32_t dense_chunk_for(int64_t nnz) {
    int32_t c = kMaxDenseChunk;
    if (nnz < kSplitMinEntries) return c;
    while (c > kMinDenseChunk && static_cast<int64_t>(c) * 2048 > nnz) c >>= 1;
    return c;
}
// Widest feature window one SpMM launch covers; wider F is processed in windows.
constexpr int kMaxSlice = 256;
// Dense rows of at least 2^kLongRowOctave entries get a wavefront each; shorter dense
// rows get one lane group each.  Narrow features mean small lane groups (more of them per
// wavefront), so the SpMM lowers the bound by one octave per halving of the group below
// 32 lanes, down to 2^(kLongRowOctave - kLongRowClasses + 1) entries: a group then never
// walks more than 64 / (groups per wavefront) rounds of 16 entries alone.
constexpr int kLongRowOctave = 9;
constexpr int kLongRowClasses = 4;
// A sparse-region task is a run of at most kTaskRows consecutive rows of the sorted
// order whose first entries fall in one window of kTaskEntries entries.
constexpr int kTaskRows = 8;
constexpr int kTaskEntries = 32;

// Gather heat of a node: how often the SpMM reads its feature row, on a log scale with
// eight steps per octave (8 floor(log2 d) + the three bits below the leading one of d,
// 0 for d = 0).  d is the node's row length, which for the symmetric aggregation matrix
// is also the number of entries in its column, i.e. the number of times its row of X is
// gathered.  It only steers cache policies of the gathers, never a result.
constexpr int kHeatLevels = 256;
// Gathers use cache classes only on operands larger than the memory-side cache (256 MiB);
// a launch reads rows of at most kMaxSlice floats, so smaller plans mark no columns.
constexpr uint64_t kGatherClassMinBytes = 256ull << 20;
// Rows of X whose gathers keep the default cache policy: the hottest kHotRows columns
// (32 MiB of 128-float rows, the L2s' share of the hottest rows).
constexpr uint32_t kHotRows = 65536;
__host__ __device__ inline uint32_t heat_of(uint32_t d) {
    if (d == 0) return 0;
    const uint32_t o = 31u - static_cast<uint32_t>(__builtin_clz(d));
    const uint32_t frac = o >= 3 ? (d >> (o - 3)) & 7u : (d << (3 - o)) & 7u;
    return 8u * o + frac;
}

// One part of a split dense row: position of the row in the sorted order, part index,
// number of parts, index of the row's first part.
struct SplitPart {
    int32_t row;
    int32_t part;
    int32_t nparts;
    int32_t first;
};

struct Plan {
    int device = 0;
    void *mem = nullptr;               // one device block holding every array below
    size_t mem_bytes = 0;
    int32_t n = 0;
    int64_t nnz = 0;
    const int32_t *rowptr = nullptr;   // borrowed
    const int32_t *col = nullptr;      // borrowed
    const float *val = nullptr;        // borrowed

    uint32_t *S = nullptr;             // [n] density sums
    uint64_t *K = nullptr;             // [n] hybrid keys
    int32_t *perm = nullptr;           // [n] nodes sorted by (K, v)
    // [n] processing order: sparse rows then dense rows (the same split as perm),
    // each region by row-length octave, then node id
    int32_t *order = nullptr;

    // The matrix with its rows in processing order (row i of this copy is row order[i]):
    // the contiguous sparse and dense regions the SpMM kernels stream through.
    int32_t *pptr = nullptr;           // [n + 1]
    int32_t *pcol = nullptr;           // [nnz]
    float *pval = nullptr;             // [nnz]
    int32_t *tasks = nullptr;          // [n_tasks + 1] first sorted row of each sparse task
    bool cold_marked = false;          // bit 31 of pcol marks columns outside the hottest
                                       // kHotRows (plans on which gathers may use classes)

    int32_t n_sparse = 0;
    int32_t n_tasks = 0;
    int32_t n_long[kLongRowClasses] = {};   // dense rows of >= 2^(kLongRowOctave - c) entries
                                            // (the last ones of the order)
    int32_t dense_chunk = kMaxDenseChunk;   // entries per part of a split dense row
    int32_t n_split_rows = 0;
    int32_t n_split_parts = 0;
    SplitPart *parts = nullptr;        // [n_split_parts]
    double *partials = nullptr;        // [n_split_parts][kMaxSlice]
    int32_t *tile_row = nullptr;       // [nnz / 4096 + 2] rows of the sorted copy's tiles
    hipEvent_t ready = nullptr;        // recorded after the sorted copy was written
    mutable std::atomic<bool> ready_seen{false};   // `ready` was found complete
    // the last launch that used the plan on each stream (destroy waits for these)
    mutable std::mutex use_mu;
    mutable std::vector<std::pair<hipStream_t, hipEvent_t>> uses;
    // the build's scratch block while the sorted copy may still read it (plans that mark
    // cold columns): released once `ready` has been seen complete, or with the plan
    mutable void *pending = nullptr;
    mutable size_t pending_bytes = 0;

    uint64_t kstar = 0, kmax = 0;
    u128 s1 = 0, s2 = 0;
    dualgcn_thresholds th{};
    uint64_t seed = 0;
    uint32_t k = 0, d = 0;
    int32_t max_degree = 0;
};

// ---- status helpers (api.hip)
int hip_status(hipError_t e);          // records e; returns DUALGCN_OK or DUALGCN_ERR_HIP
int device_status();                   // DUALGCN_OK or DUALGCN_ERR_NO_DEVICE / _HIP
int alloc_bytes(void **p, size_t bytes);  // DUALGCN_OK or DUALGCN_ERR_OOM / _HIP
// A device block of at least `bytes` on the current device, possibly a cached one;
// *capacity receives its real size, to be passed back to release_block.
int alloc_block(void **p, size_t *capacity, size_t bytes);
// Returns a block to the cache (or to HIP); the device must no longer use it.
void release_block(void *p, size_t capacity);

// Compute units of the current device, queried once per device (256 if the query fails).
int device_cus();

// ---- anonymous walks (arw.hip)
// S[v] = sum over k walks of distinct-node counts; patterns (may be null) receives labels.
int launch_arw(const int32_t *rowptr, const int32_t *col, int32_t n, uint64_t seed, uint32_t k,
               uint32_t d, uint32_t *S, uint8_t *patterns, const int32_t *bad_flag,
               hipStream_t stream);
// The same sums from nodeinfo (every node's (first entry, degree), as validate_csr writes
// it), two walks per lane advanced in lockstep.  With succ (succ[e] = (first entry, degree)
// of the node in column e) each step reads one record instead of a node's bounds and then
// a column.  DUALGCN_ERR_UNSUPPORTED (nothing launched) when d > 32.
int launch_density(const int2 *nodeinfo, const int32_t *col, const int2 *succ, int32_t n,
                   uint64_t seed, uint32_t k, uint32_t d, uint32_t *S, const int32_t *bad_flag,
                   hipStream_t stream);

// ---- partition (partition.hip)
// Checks the CSR on the device: flags[0] |= 1 (row pointers) | 2 (columns); flags must
// start at zero.  nodeinfo (may be null, n entries) receives (rowptr[v], rowptr[v+1] -
// rowptr[v]); blockmax (may be null, kValidateBlocks entries) each workgroup's largest
// row length; heat_hist (may be null, kHeatLevels counters that start at zero) the number
// of nodes per heat_of(row length).  check_cols = false leaves the columns to a later pass
// over them (the partition's successor pass, which sets bit 2 the same way).
constexpr int kValidateBlocks = 2048;
int validate_csr(const dualgcn_csr *csr, int32_t *flags, int2 *nodeinfo, int32_t *blockmax,
                 uint32_t *heat_hist, hipStream_t stream, bool check_cols = true);
// S_host (host, n sums), when given, replaces the walks: the density sums of a saved plan.
int build_plan(const dualgcn_csr *csr, uint64_t seed, uint32_t k, uint32_t d,
               const dualgcn_thresholds &th, const uint32_t *S_host, hipStream_t stream,
               Plan **out);
// An order-free 64-bit checksum of a CSR structure (row pointers and columns); waits.
int structure_checksum(const int32_t *rowptr, const int32_t *col, int32_t n, int64_t nnz,
                       hipStream_t stream, uint64_t *out);
void free_plan(Plan *p);

// float32 -> bfloat16 bits, round to nearest even; NaNs stay NaN.
__device__ __forceinline__ unsigned short to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return static_cast<unsigned short>((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<unsigned short>(u >> 16);
}

// ---- SpMM (spmm.hip): Y = A X on one plan, optional ReLU on the result; with out_bf16
// Y holds the bfloat16 rounding (nearest-even) of the float32 results.
// Host waits that poll instead of blocking (partition.hip): for the work queued on a
// stream so far, or for an event.
int wait_stream(hipStream_t stream);
int wait_event(hipEvent_t event);
// Records that work using the plan was queued on `stream` (spmm.hip), and waits for every
// such use and for the plan's own build (partition.hip).
int note_use(const Plan &p, hipStream_t stream);
int wait_plan_idle(const Plan &p);
// Returns the plan's pending scratch block to the block cache; only once `ready` has completed.
void release_pending(const Plan &p);

int launch_spmm(const Plan &p, const float *X, void *Y, int32_t F, bool relu, bool out_bf16,
                hipStream_t stream);
// T = bf16(act(A X)) bf16(W) (float32 accumulation), act(A X) stored as bfloat16 to H
// only if H is not null: 32 <= F_in <= 256 and 32 <= F_out <= 256 multiples of 32,
// X and T 16-byte aligned, H 8-byte aligned.
int launch_spmm_xw(const Plan &p, const float *X, const float *W, float *T, void *H,
                   int32_t F_in, int32_t F_out, bool relu, hipStream_t stream);
// LDS bytes a workgroup of launch_spmm_xw takes (at most 160 KiB are supported).
size_t spmm_xw_lds_bytes(int32_t F_in, int32_t F_out);
// Is launch_spmm_xw faster than launch_spmm (bfloat16 output) followed by launch_xw on this
// plan and shape?  (A cost rule from measurements; both routes give the same bits.)
bool fused_junction_pays(const Plan &p, int32_t F_in, int32_t F_out);

// ---- update phase (xw.hip)
// Bytes of the float32 T = X W buffer a layer keeps in its workspace (256-byte multiple).
size_t xw_workspace_bytes(int32_t n, int32_t F_out);
// T = bf16(X) bf16(W) with float32 accumulation; X is float32, or bfloat16 if in_bf16.
int launch_xw(const void *X, bool in_bf16, const float *W, float *T, int32_t n, int32_t F_in,
              int32_t F_out, hipStream_t stream);
// Y = act(A (X W)): launch_xw into the workspace, then launch_spmm.
int launch_gcn_layer(const Plan &p, const void *X, bool in_bf16, const float *W, void *Y,
                     bool out_bf16, int32_t F_in, int32_t F_out, bool relu, void *workspace,
                     hipStream_t stream);

// dX = (bf16(G) bf16(W)^T) * [M > 0] (no mask when M is null); G is n x F_out (float32,
// or bfloat16 if g_bf16), W is F_in x F_out, M and dX are n x F_in.
int launch_backward_data(const void *G, bool g_bf16, const float *W, const void *M, bool m_bf16,
                         float *dX, int32_t n, int32_t F_in, int32_t F_out, hipStream_t stream);

// ---- aggregator values (aggregate.hip): val[e] for the structure of csr (no validation;
// out-of-range columns read nothing).
int launch_aggregator_values(const dualgcn_csr *csr, int kind, float eps, float *val,
                             hipStream_t stream);

// ---- training (train.hip)
// Workgroups of the loss kernel; loss[1 .. kLossBlocks] hold their partial sums.
constexpr int kLossBlocks = DUALGCN_LOSS_SLOTS - 1;
int launch_softmax_xent(const float *Y, const int32_t *labels, int32_t n, int32_t C, float scale,
                        float *G, double *loss, hipStream_t stream);
// Bytes of the partial dW matrices of launch_weight_grad.
size_t wgrad_workspace_bytes(int32_t n, int32_t F_in, int32_t F_out);
// dW = bf16(X)^T bf16(G), summed over rows in a fixed order; with W, W -= lr dW.
int launch_weight_grad(const void *X, bool x_bf16, const void *G, bool g_bf16, float *dW,
                       int32_t n, int32_t F_in, int32_t F_out, float lr, float *W, void *workspace,
                       hipStream_t stream);
// The same with the partials in the library's static device array (no workspace, no
// allocation): DUALGCN_ERR_UNSUPPORTED when they need more than its
// DUALGCN_WGRAD_NOALLOC_BYTES.  wgrad_noalloc_bytes gives what they need on the current
// device.
int wgrad_noalloc_bytes(bool x_bf16, bool g_bf16, int32_t n, int32_t F_in, int32_t F_out,
                        size_t *bytes);
int launch_weight_grad_noalloc(const void *X, bool x_bf16, const void *G, bool g_bf16, float *dW,
                               int32_t n, int32_t F_in, int32_t F_out, float lr, float *W,
                               hipStream_t stream);

// ---- attainable bandwidth (probe.hip): kind DUALGCN_PROBE_COPY or DUALGCN_PROBE_READ; the
// read probe writes one float per workgroup (probe_grid() <= kMaxProbeGrid) to dst.
constexpr int kMaxProbeGrid = 16384;
int probe_grid();
int launch_bandwidth_probe(int kind, const void *src, void *dst, size_t bytes, hipStream_t stream);

}  // namespace dgc
