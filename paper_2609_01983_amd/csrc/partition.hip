// Dual-metric partition on gfx950 (DualGCN Sec. 3.2 and Sec. 3.3 Eq. (1)).
//
// Pipeline (one stream, two host waits; three with an adaptive or balanced alpha):
//   validate        rowptr / col checks, the largest degree, node records -> flag
//   successors      (when walks outnumber entries twice) one record per entry:
//                   the first entry and degree of the node in that column
//   walks           S_v (arw.hip), or S from a saved plan
//   adaptive alpha  (optional; also the balanced one) moments of S and D -> extra host wait
//   keys            K_v = p S_v + (q - p) k D_v, D_v from the row pointers, and the
//                   exact 128-bit sums of K and K^2 per workgroup, then one
//                   workgroup folds them                              -> host wait 1
//   host            K* = least integer >= mu_K + beta sigma_K (exact integers)
//   radix sort      stable LSD sort of (K_v, v) on 8-bit digits      -> perm
//   split           n_sparse = lower_bound(sorted K, K*)
//   processing order  (region, row-length octave, node id): one stable radix pass
//                   over the node ids on a key of (region, octave) below 64
//   row pointers    of the rows in processing order, by a scan
//   schedule        sparse tasks (runs of at most kTaskRows short rows) and the
//                   parts of dense rows longer than one dense chunk
//   sorted copy     the rows of the matrix in processing order, so that both regions
//                   are contiguous streams (Sec. 3.2: the sorted nodes are cut into
//                   contiguous blocks); host wait 2 reads the schedule sizes while it
//                   runs, and the call returns with it queued (plan users wait for
//                   the plan's ready event)
//
// Everything is integer arithmetic, so the plan does not depend on launch order
// or reduction order: it is the unique sort of (K_v, v) cut at K*.
#include "internal.h"

#include <chrono>

#include <algorithm>
#include <cstring>
#include <thread>

namespace dgc {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;                    // items per thread in tiled kernels
constexpr int kTile = kThreads * kItems;      // 4096
constexpr int kRadixBits = 8;
constexpr int kRadix = 1 << kRadixBits;

// ------------------------------------------------------------------ validation

// Checks the row pointers and (with check_cols; otherwise the successor pass checks them)
// the columns, records the largest degree, writes every node's (first entry, degree)
// record for the walks (one 8-byte read per step) and counts the nodes per gather heat
// (per workgroup in LDS, then one atomic per non-empty value and workgroup).
__global__ __launch_bounds__(kThreads) void validate_kernel(const int32_t *__restrict__ rowptr,
                                                            const int32_t *__restrict__ col,
                                                            int32_t n, int64_t nnz,
                                                            int32_t *__restrict__ flag,
                                                            int2 *__restrict__ nodeinfo,
                                                            int32_t *__restrict__ blockmax,
                                                            uint32_t *__restrict__ heat_hist,
                                                            int32_t check_cols) {
    __shared__ int32_t sh_bad[kThreads / 64], sh_max[kThreads / 64];
    __shared__ uint32_t sh_hist[kHeatLevels];
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (heat_hist) {
        for (int h = static_cast<int>(threadIdx.x); h < kHeatLevels; h += kThreads) sh_hist[h] = 0;
        __syncthreads();
    }
    int32_t bad = 0, dmax = 0;
    for (int64_t i = t0; i < n; i += stride) {
        const int32_t a = rowptr[i], b = rowptr[i + 1];
        if (b < a) bad |= 1;
        dmax = max(dmax, b - a);
        if (nodeinfo) nodeinfo[i] = make_int2(a, b - a);
        if (heat_hist) atomicAdd(&sh_hist[heat_of(b > a ? static_cast<uint32_t>(b - a) : 0u)], 1u);
    }
    if (heat_hist) {
        __syncthreads();
        for (int h = static_cast<int>(threadIdx.x); h < kHeatLevels; h += kThreads)
            if (sh_hist[h]) atomicAdd(&heat_hist[h], sh_hist[h]);
    }
    if (t0 == 0) {
        if (rowptr[0] != 0) bad |= 1;
        if (static_cast<int64_t>(rowptr[n]) != nnz) bad |= 1;
    }
    // columns: scalar head up to a 16-byte boundary, 16-byte loads, scalar tail
    if (!check_cols) nnz = 0;
    const int64_t head = std::min<int64_t>(nnz, ((16 - (reinterpret_cast<uintptr_t>(col) & 15)) & 15) / 4);
    const int64_t body = (nnz - head) / 4;
    const int4 *__restrict__ c4 = reinterpret_cast<const int4 *>(col + head);
#pragma unroll 4
    for (int64_t q = t0; q < body; q += stride) {
        const int4 c = c4[q];
        if (c.x < 0 || c.x >= n || c.y < 0 || c.y >= n || c.z < 0 || c.z >= n || c.w < 0 || c.w >= n)
            bad |= 2;
    }
    if (t0 < head) {
        const int32_t c = col[t0];
        if (c < 0 || c >= n) bad |= 2;
    }
    for (int64_t p = head + 4 * body + t0; p < nnz; p += stride) {
        const int32_t c = col[p];
        if (c < 0 || c >= n) bad |= 2;
    }
    // one result per workgroup: the flag by an atomic only when something is wrong, the
    // largest degree into blockmax (folded later), so no address is contended
    for (int off = 32; off > 0; off >>= 1) {
        bad |= __shfl_xor(bad, off, 64);
        dmax = max(dmax, __shfl_xor(dmax, off, 64));
    }
    if ((threadIdx.x & 63) == 0) {
        sh_bad[threadIdx.x >> 6] = bad;
        sh_max[threadIdx.x >> 6] = dmax;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kThreads / 64; ++w) {
            bad |= sh_bad[w];
            dmax = max(dmax, sh_max[w]);
        }
        if (bad) atomicOr(flag, bad);
        if (blockmax) blockmax[blockIdx.x] = dmax;
    }
}

// Successor records of the walks: succ[e] = (first entry of c, degree of c) for
// c = col[e], the node record validate_kernel wrote.  With marked, also the column with
// bit 31 set when c is outside the hottest columns (heat below *hot_heat), in the
// matrix's entry order: the sorted copy then reads it in place of the column, and the
// mark costs it nothing.  This pass reads every column, so it also checks them (the
// validation then checks only the row pointers): a column out of range sets bit 2 of
// the flag (nothing walks or copies then) and gets a record without reading them.
__global__ __launch_bounds__(kThreads) void successor_kernel(const int2 *__restrict__ nodeinfo,
                                                             const int32_t *__restrict__ col,
                                                             int32_t n, int64_t nnz,
                                                             int2 *__restrict__ succ,
                                                             const uint32_t *__restrict__ hot_heat,
                                                             int32_t *__restrict__ marked,
                                                             int32_t *__restrict__ flag) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const uint32_t hot = marked ? *hot_heat : 0u;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < nnz;
         e += stride) {
        const int32_t c = col[e];
        const bool in = c >= 0 && c < n;
        if (!in) atomicOr(flag, 2);
        const int2 r = in ? nodeinfo[c] : make_int2(0, 0);
        if (succ) succ[e] = r;
        if (marked) {
            const bool cold = heat_of(static_cast<uint32_t>(r.y)) < hot;
            marked[e] = static_cast<int32_t>(static_cast<uint32_t>(c) | (cold ? 0x80000000u : 0u));
        }
    }
}

// *hot_heat = the smallest heat h whose nodes of heat >= h number at most hot_rows
// (kHeatLevels if even the hottest value has more); hist counts the nodes per heat value.
// One workgroup of kHeatLevels threads: a suffix sum in LDS, then the smallest qualifying
// value by an LDS minimum.
__global__ __launch_bounds__(kHeatLevels) void hot_heat_kernel(const uint32_t *__restrict__ hist,
                                                               uint32_t hot_rows,
                                                               uint32_t *__restrict__ hot_heat) {
    __shared__ uint64_t above[kHeatLevels];
    __shared__ uint32_t best;
    const int h = static_cast<int>(threadIdx.x);
    above[h] = hist[h];
    if (h == 0) best = kHeatLevels;
    __syncthreads();
    for (int d = 1; d < kHeatLevels; d <<= 1) {      // above[h] = sum of hist[h..]
        const uint64_t add = h + d < kHeatLevels ? above[h + d] : 0;
        __syncthreads();
        above[h] += add;
        __syncthreads();
    }
    if (above[h] <= hot_rows) atomicMin(&best, static_cast<uint32_t>(h));
    __syncthreads();
    if (h == 0) *hot_heat = best;
}

// ------------------------------------------------------------------ structure checksum

// splitmix64's output function (Steele, Lea & Flood, OOPSLA'14): a bijective mix of one
// 64-bit word.
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

constexpr int kSumBlocks = 1024;

// partial[b] = sum (mod 2^64) of mix64 over this workgroup's entries of rowptr (tagged by
// position) and col (tagged by position and a different constant): order-free, exact.
__global__ __launch_bounds__(kThreads) void checksum_kernel(const int32_t *__restrict__ rowptr,
                                                            const int32_t *__restrict__ col,
                                                            int32_t n, int64_t nnz,
                                                            uint64_t *__restrict__ partial) {
    __shared__ uint64_t sh[kThreads];
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    uint64_t acc = 0;
    for (int64_t i = t0; i <= n; i += stride)
        acc += mix64((static_cast<uint64_t>(i) << 32) ^ static_cast<uint32_t>(rowptr[i]));
    for (int64_t e = t0; e < nnz; e += stride)
        acc += mix64(((static_cast<uint64_t>(e) << 32) ^ static_cast<uint32_t>(col[e])) +
                     0x9E3779B97F4A7C15ull);
    const int t = threadIdx.x;
    sh[t] = acc;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) sh[t] += sh[t + h];
        __syncthreads();
    }
    if (t == 0) partial[blockIdx.x] = sh[0];
}

__global__ void checksum_fold_kernel(uint64_t *__restrict__ partial) {
    uint64_t s = 0;
    for (int i = 0; i < kSumBlocks; ++i) s += partial[i];
    partial[kSumBlocks] = s;
}

// ------------------------------------------------------------------ keys and moments

struct Moments {
    uint64_t s1_lo, s1_hi, s2_lo, s2_hi, kmax;
};

__host__ __device__ __forceinline__ u128 join(uint64_t lo, uint64_t hi) {
    return (static_cast<u128>(hi) << 64) | lo;
}

__global__ __launch_bounds__(kThreads) void keys_kernel(
    const int32_t *__restrict__ rowptr, const uint32_t *__restrict__ S, int32_t n, uint64_t p,
    uint64_t qmp_k, uint64_t *__restrict__ K, Moments *__restrict__ partial,
    const int32_t *__restrict__ bad_flag) {
    __shared__ u128 sh1[kThreads], sh2[kThreads];
    __shared__ uint64_t shm[kThreads];
    u128 s1 = 0, s2 = 0;
    uint64_t kmax = 0;
    if (*bad_flag == 0) {
        const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
        for (int64_t v = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; v < n;
             v += stride) {
            const uint64_t deg = static_cast<uint64_t>(rowptr[v + 1] - rowptr[v]);
            const uint64_t key = p * S[v] + qmp_k * deg;
            K[v] = key;
            s1 += key;
            s2 += static_cast<u128>(key) * key;
            kmax = key > kmax ? key : kmax;
        }
    }
    const int t = threadIdx.x;
    sh1[t] = s1;
    sh2[t] = s2;
    shm[t] = kmax;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) {
            sh1[t] += sh1[t + h];
            sh2[t] += sh2[t + h];
            shm[t] = shm[t] > shm[t + h] ? shm[t] : shm[t + h];
        }
        __syncthreads();
    }
    if (t == 0) {
        partial[blockIdx.x] = Moments{static_cast<uint64_t>(sh1[0]),
                                      static_cast<uint64_t>(sh1[0] >> 64),
                                      static_cast<uint64_t>(sh2[0]),
                                      static_cast<uint64_t>(sh2[0] >> 64), shm[0]};
    }
}

struct Summary {
    Moments m;
    int32_t flag;
    int32_t maxdeg;
};

__global__ __launch_bounds__(kThreads) void fold_kernel(const Moments *__restrict__ partial,
                                                        int32_t count,
                                                        const int32_t *__restrict__ flag,
                                                        const int32_t *__restrict__ blockmax,
                                                        Summary *__restrict__ out) {
    __shared__ u128 sh1[kThreads], sh2[kThreads];
    __shared__ uint64_t shm[kThreads];
    __shared__ int32_t shd[kThreads];
    const int t = threadIdx.x;
    u128 s1 = 0, s2 = 0;
    uint64_t kmax = 0;
    int32_t dmax = 0;
    for (int i = t; i < count; i += kThreads) {
        s1 += join(partial[i].s1_lo, partial[i].s1_hi);
        s2 += join(partial[i].s2_lo, partial[i].s2_hi);
        kmax = partial[i].kmax > kmax ? partial[i].kmax : kmax;
    }
    for (int i = t; i < kValidateBlocks; i += kThreads) dmax = max(dmax, blockmax[i]);
    sh1[t] = s1;
    sh2[t] = s2;
    shm[t] = kmax;
    shd[t] = dmax;
    __syncthreads();
    for (int h = kThreads / 2; h > 0; h >>= 1) {
        if (t < h) {
            sh1[t] += sh1[t + h];
            sh2[t] += sh2[t + h];
            shm[t] = shm[t] > shm[t + h] ? shm[t] : shm[t + h];
            shd[t] = max(shd[t], shd[t + h]);
        }
        __syncthreads();
    }
    if (t == 0) {
        out->m = Moments{static_cast<uint64_t>(sh1[0]), static_cast<uint64_t>(sh1[0] >> 64),
                         static_cast<uint64_t>(sh2[0]), static_cast<uint64_t>(sh2[0] >> 64),
                         shm[0]};
        out->flag = *flag;
        out->maxdeg = shd[0];
    }
}

// ------------------------------------------------------------------ block scan helpers

// Exclusive scan of one value per thread across a 256-thread workgroup.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t *total,
                                                         uint32_t *sh_waves) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t inc = x;
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(inc, off, 64);
        if (lane >= off) inc += y;
    }
    if (lane == 63) sh_waves[wave] = inc;
    __syncthreads();
    uint32_t wave_base = 0, sum = 0;
    for (int i = 0; i < kThreads / 64; ++i) {
        if (i < wave) wave_base += sh_waves[i];
        sum += sh_waves[i];
    }
    __syncthreads();
    *total = sum;
    return wave_base + inc - x;
}

// Tile sums of a u32 array (tiles of kTile elements).  Full tiles of a 16-byte aligned array
// are read with coalesced 16-byte loads (thread t takes quads t, t + kThreads, ...; the
// order of a sum of integers does not matter), others element by element.
__global__ __launch_bounds__(kThreads) void scan_reduce_kernel(const uint32_t *__restrict__ in,
                                                               int64_t count,
                                                               uint32_t *__restrict__ sums) {
    __shared__ uint32_t shw[kThreads / 64];
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kTile;
    uint32_t s = 0;
    if (base + kTile <= count && reinterpret_cast<uintptr_t>(in) % 16 == 0) {
        const uint4 *q = reinterpret_cast<const uint4 *>(in + base);
#pragma unroll
        for (int i = 0; i < kItems / 4; ++i) {
            const uint4 v = q[threadIdx.x + i * kThreads];
            s += v.x + v.y + v.z + v.w;
        }
    } else {
        for (int i = 0; i < kItems; ++i) {
            const int64_t idx = base + static_cast<int64_t>(i) * kThreads + threadIdx.x;
            if (idx < count) s += in[idx];
        }
    }
    uint32_t total;
    block_exclusive_scan(s, &total, shw);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Exclusive scan of the tile sums by one workgroup (in place); writes the grand total.
__global__ __launch_bounds__(kThreads) void scan_top_kernel(uint32_t *__restrict__ sums,
                                                            int32_t count,
                                                            uint32_t *__restrict__ grand) {
    __shared__ uint32_t shw[kThreads / 64];
    uint32_t carry = 0;
    for (int32_t base = 0; base < count; base += kThreads) {
        const int32_t i = base + threadIdx.x;
        const uint32_t x = i < count ? sums[i] : 0;
        uint32_t total;
        const uint32_t ex = block_exclusive_scan(x, &total, shw);
        if (i < count) sums[i] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0 && grand) *grand = carry;
}

// Exclusive scan inside each tile plus the tile's offset; out may alias in.  A full tile is
// taken as kTile / 4 quads in index order, quad c held by thread c % kThreads in round
// c / kThreads: round by round, a block scan of the quad sums gives each quad its offset,
// so loads and stores stay coalesced 16-byte accesses (arrays 16-byte aligned).  Other
// tiles go element by element, each thread scanning kItems consecutive elements.
__global__ __launch_bounds__(kThreads) void scan_apply_kernel(const uint32_t *in, int64_t count,
                                                              const uint32_t *__restrict__ sums,
                                                              uint32_t *out) {
    __shared__ uint32_t shw[kThreads / 64];
    const int64_t tile = static_cast<int64_t>(blockIdx.x) * kTile;
    if (tile + kTile <= count && (reinterpret_cast<uintptr_t>(in) | reinterpret_cast<uintptr_t>(out)) % 16 == 0) {
        const uint4 *q = reinterpret_cast<const uint4 *>(in + tile);
        uint4 v[kItems / 4];
#pragma unroll
        for (int i = 0; i < kItems / 4; ++i) v[i] = q[threadIdx.x + i * kThreads];
        uint32_t carry = sums[blockIdx.x];
#pragma unroll
        for (int i = 0; i < kItems / 4; ++i) {
            const uint32_t qs = v[i].x + v[i].y + v[i].z + v[i].w;
            uint32_t total;
            const uint32_t ex = carry + block_exclusive_scan(qs, &total, shw);
            carry += total;
            reinterpret_cast<uint4 *>(out + tile)[threadIdx.x + i * kThreads] =
                make_uint4(ex, ex + v[i].x, ex + v[i].x + v[i].y, ex + v[i].x + v[i].y + v[i].z);
        }
        return;
    }
    const int64_t base = tile + static_cast<int64_t>(threadIdx.x) * kItems;
    uint32_t v[kItems];
    uint32_t s = 0;
    for (int i = 0; i < kItems; ++i) {
        v[i] = base + i < count ? in[base + i] : 0;
        s += v[i];
    }
    uint32_t total;
    uint32_t run = block_exclusive_scan(s, &total, shw) + sums[blockIdx.x];
    for (int i = 0; i < kItems; ++i) {
        if (base + i < count) out[base + i] = run;
        run += v[i];
    }
}

// ------------------------------------------------------------------ radix sort of (K, v)

// Sort tiles hold kThreads * ITEMS keys: 16 per thread on large inputs, 4 below
// kSortSmallKeys keys, where 4096-key tiles would leave most CUs idle and make every
// wavefront walk 16 rounds in a row (c2, 2^17 keys: 32 workgroups).
constexpr int kSortItemsSmall = 4;
constexpr int64_t kSortSmallKeys = int64_t{1} << 20;

template <int ITEMS>
__global__ __launch_bounds__(kThreads) void radix_hist_kernel(const uint64_t *__restrict__ keys,
                                                              int32_t n, int shift,
                                                              uint32_t *__restrict__ hist,
                                                              int32_t nblocks) {
    __shared__ uint32_t h[kRadix];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kThreads * ITEMS;
    for (int i = 0; i < ITEMS; ++i) {
        const int64_t idx = base + static_cast<int64_t>(i) * kThreads + threadIdx.x;
        if (idx < n) atomicAdd(&h[(keys[idx] >> shift) & (kRadix - 1)], 1u);
    }
    __syncthreads();
    hist[static_cast<int64_t>(threadIdx.x) * nblocks + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one 8-bit digit.  Wave w owns items [base + 64 ITEMS w, base + 64 ITEMS
// (w+1)), taken in rounds of 64 consecutive items; lanes with equal digits find each other
// with eight ballots, so an item's rank is (earlier items of its digit in this wave) +
// (earlier lanes of its digit in this round).  Tile order = index order, hence stable.
template <int ITEMS>
__global__ __launch_bounds__(kThreads) void radix_scatter_kernel(
    const uint64_t *__restrict__ keys_in, const int32_t *__restrict__ vals_in, int32_t n,
    int shift, const uint32_t *__restrict__ offsets, int32_t nblocks,
    uint64_t *__restrict__ keys_out, int32_t *__restrict__ vals_out) {
    __shared__ uint32_t cnt[kThreads / 64][kRadix];
    __shared__ uint32_t goff[kRadix];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int w = 0; w < kThreads / 64; ++w) cnt[w][threadIdx.x] = 0;
    goff[threadIdx.x] = offsets[static_cast<int64_t>(threadIdx.x) * nblocks + blockIdx.x];
    __syncthreads();

    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kThreads * ITEMS +
                         static_cast<int64_t>(wave) * (ITEMS * 64);
    uint32_t rank[ITEMS];
    for (int j = 0; j < ITEMS; ++j) {
        const int64_t idx = base + static_cast<int64_t>(j) * 64 + lane;
        const bool valid = idx < n;
        const uint32_t dg = valid ? static_cast<uint32_t>((keys_in[idx] >> shift) & (kRadix - 1)) : 0;
        uint64_t m = __ballot(valid);
        for (int b = 0; b < kRadixBits; ++b) {
            const bool bit = (dg >> b) & 1u;
            const uint64_t bal = __ballot(valid && bit);
            m &= bit ? bal : ~bal;
        }
        const uint32_t below = static_cast<uint32_t>(__popcll(m & lt_mask));
        const uint32_t before = valid ? cnt[wave][dg] : 0;
        __builtin_amdgcn_wave_barrier();
        if (valid && below == 0) cnt[wave][dg] = before + static_cast<uint32_t>(__popcll(m));
        __builtin_amdgcn_wave_barrier();
        rank[j] = before + below;
    }
    __syncthreads();
    {   // exclusive prefix of the per-wave counts, digit by digit
        uint32_t run = 0;
        for (int w = 0; w < kThreads / 64; ++w) {
            const uint32_t c = cnt[w][threadIdx.x];
            cnt[w][threadIdx.x] = run;
            run += c;
        }
    }
    __syncthreads();
    for (int j = 0; j < ITEMS; ++j) {
        const int64_t idx = base + static_cast<int64_t>(j) * 64 + lane;
        if (idx < n) {
            const uint64_t key = keys_in[idx];
            const uint32_t dg = static_cast<uint32_t>((key >> shift) & (kRadix - 1));
            const uint32_t dest = goff[dg] + cnt[wave][dg] + rank[j];
            if (dest < static_cast<uint32_t>(n)) {   // always true for a consistent histogram
                keys_out[dest] = key;
                vals_out[dest] = vals_in ? vals_in[idx] : static_cast<int32_t>(idx);
            }
        }
    }
}

__global__ void iota_kernel(int32_t *__restrict__ out, int32_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) out[i] = static_cast<int32_t>(i);
}

// ------------------------------------------------------------------ split and schedule

struct SplitSummary {
    int32_t n_sparse;
    int32_t split_rows;
    uint32_t parts;
    uint32_t tasks;
    int32_t long_rows[kLongRowClasses];   // dense rows of >= 2^(kLongRowOctave - c) entries
};

// First index i of the sorted array a[0, n) with a[i] >= x (n if none), found by one
// wavefront: each round probes 64 evenly spaced positions strictly inside the candidate
// range [lo, hi] (a[i] < x below lo, a[i] >= x from hi on) and keeps the gap between the
// last probe below x and the first one at or above it, until at most 64 candidates are left.
__device__ int32_t wave_lower_bound(const uint64_t *__restrict__ a, int32_t n, uint64_t x) {
    const int lane = static_cast<int>(threadIdx.x) & 63;
    int32_t lo = 0, hi = n;
    while (hi - lo > 64) {
        const int64_t span = hi - lo;
        const int32_t p = lo + static_cast<int32_t>(span * (lane + 1) / 65);
        const uint64_t m = __ballot(a[p] >= x);
        if (m == 0) {
            lo = lo + static_cast<int32_t>(span * 64 / 65) + 1;
        } else {
            const int f = __ffsll(static_cast<unsigned long long>(m)) - 1;
            hi = lo + static_cast<int32_t>(span * (f + 1) / 65);
            if (f > 0) lo = lo + static_cast<int32_t>(span * f / 65) + 1;
        }
    }
    const int32_t p = lo + lane;
    const uint64_t m = __ballot(p >= hi || a[p] >= x);
    return m ? lo + __ffsll(static_cast<unsigned long long>(m)) - 1 : hi;
}

// n_sparse = first position whose key is >= K* (one wavefront; keys are sorted).
__global__ void lower_bound_kernel(const uint64_t *__restrict__ sorted, int32_t n, uint64_t kstar,
                                   int32_t force_sparse_count, SplitSummary *__restrict__ out) {
    const int32_t lo = wave_lower_bound(sorted, n, kstar);
    if (threadIdx.x != 0) return;
    out->n_sparse = force_sparse_count >= 0 ? force_sparse_count : lo;
    out->split_rows = 0;
    out->parts = 0;
    out->tasks = 0;
    for (int c = 0; c < kLongRowClasses; ++c) out->long_rows[c] = 0;
}

// long_rows[c] = rows of the dense region with at least 2^(kLongRowOctave - c) entries: the
// rows whose processing-order key is at least that class's, i.e. n minus the number of
// smaller keys, which the scanned histogram of the order pass holds (digit-major: entry
// d * nblocks is the count of keys below d).
__global__ void long_rows_kernel(const uint32_t *__restrict__ scanned_hist, int32_t nblocks,
                                 int32_t n, SplitSummary *__restrict__ out) {
    const int c = static_cast<int>(threadIdx.x);
    if (c >= kLongRowClasses) return;
    const uint32_t first_long = 32u + kLongRowOctave - c;
    out->long_rows[c] = n - static_cast<int32_t>(scanned_hist[static_cast<int64_t>(first_long) * nblocks]);
}

// Processing order of the SpMM (the row order of the sorted copy): region first (sparse
// rows, then dense rows, Eq. (1)), then the octave of the row length, then node id.  Rows
// that share an octave cost about the same (the balance the paper sorts for); keeping node
// ids in order inside an octave keeps whatever locality the numbering has (e.g. the
// contiguous communities of a block-structured graph).  forced = 0 / 1 puts every row in
// one region, -1 applies K >= K*.
__global__ __launch_bounds__(kThreads) void order_key_kernel(const uint64_t *__restrict__ K,
                                                             uint64_t kstar, int32_t forced,
                                                             const int32_t *__restrict__ rowptr,
                                                             int32_t n, uint64_t *__restrict__ key) {
    const int64_t v = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const uint32_t deg = static_cast<uint32_t>(rowptr[v + 1] - rowptr[v]);
    const uint64_t octave = deg ? 31u - static_cast<uint32_t>(__clz(deg)) : 0u;
    const uint64_t dense = forced >= 0 ? static_cast<uint64_t>(forced) : (K[v] >= kstar ? 1u : 0u);
    key[v] = dense * 32u + octave;
}

// pptr[i] = length of row order[i] for i < n and pptr[n] = 0; an exclusive scan then turns
// pptr into the row pointers of the sorted copy.
__global__ __launch_bounds__(kThreads) void sorted_degree_kernel(const int32_t *__restrict__ order,
                                                                 const int32_t *__restrict__ rowptr,
                                                                 int32_t n, uint32_t *__restrict__ pptr) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) {
        const int32_t r = order[i];
        pptr[i] = static_cast<uint32_t>(rowptr[r + 1] - rowptr[r]);
    } else if (i == n) {
        pptr[n] = 0;
    }
}

// Last row r in [lo, hi] with ptr[r] <= e (the row whose entries contain e when ptr
// holds row pointers and lo's range starts at or before e).
template <typename P>
__device__ __forceinline__ int32_t row_of(const P &ptr, int32_t lo, int32_t hi, int64_t e) {
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo + 1) / 2;
        if (static_cast<int64_t>(ptr[mid]) <= e) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

constexpr int kCopyTile = 4096;     // entries of the sorted copy one workgroup fills

// tile_row[t] = the sorted row that holds entry t kCopyTile (for every tile start below nnz):
// each non-empty row writes the tiles that start inside it.
__global__ __launch_bounds__(kThreads) void tile_row_kernel(const int32_t *__restrict__ pptr,
                                                            int32_t n, int32_t *__restrict__ tile_row) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t b = pptr[i], e = pptr[i + 1];
    for (int64_t t = (b + kCopyTile - 1) / kCopyTile; t * kCopyTile < e; ++t)
        tile_row[t] = static_cast<int32_t>(i);
}

// Fills entries [b kCopyTile, (b + 1) kCopyTile) of the sorted copy: entry e of sorted
// row i is entry e - pptr[i] of row order[i], i.e. entry e + delta[i] of the matrix with
// delta[i] = rowptr[order[i]] - pptr[i].  The tile's rows come from tile_row; each counts
// itself at the tile position where it starts (its first entry, or the tile's start), and
// an inclusive scan of those counts gives every entry the index of its row (rows of no
// entries start where the next row does and count before it).  Thread t then copies entries
// e0 + t + 256 k, so reads inside a row and all writes are coalesced.
__global__ __launch_bounds__(kThreads) void sorted_copy_kernel(
    const int32_t *__restrict__ order, const int32_t *__restrict__ rowptr,
    const int32_t *__restrict__ col, const float *__restrict__ val,
    const int32_t *__restrict__ pptr, const int32_t *__restrict__ tile_row, int32_t n,
    int64_t nnz, int32_t *__restrict__ pcol, float *__restrict__ pval) {
    constexpr int kPer = kCopyTile / kThreads;          // counters one thread scans
    __shared__ int32_t sh_delta[kCopyTile + 1];
    __shared__ __align__(16) uint32_t sh_cnt[kCopyTile];
    __shared__ uint32_t sh_waves[kThreads / 64];
    const int t = static_cast<int>(threadIdx.x);
    const int64_t e0 = static_cast<int64_t>(blockIdx.x) * kCopyTile;
    const int64_t e1 = e0 + kCopyTile < nnz ? e0 + kCopyTile : nnz;
    const int32_t r_lo = tile_row[blockIdx.x];
    const int32_t r_hi = e1 < nnz ? tile_row[blockIdx.x + 1] : n - 1;   // holds e1 or the end
    const int32_t rows = r_hi - r_lo + 1;
    if (rows <= kCopyTile + 1) {
        for (int k = t; k < kCopyTile; k += kThreads) sh_cnt[k] = 0;
        __syncthreads();
        for (int32_t k = t; k < rows; k += kThreads) {
            const int32_t b = pptr[r_lo + k];
            sh_delta[k] = rowptr[order[r_lo + k]] - b;
            const int64_t pos = b > e0 ? b - e0 : 0;
            if (pos < e1 - e0) atomicAdd(&sh_cnt[pos], 1u);
        }
        __syncthreads();
        uint32_t c[kPer];
        uint32_t sum = 0;
#pragma unroll
        for (int q = 0; q < kPer / 4; ++q) {
            const uint4 v = reinterpret_cast<const uint4 *>(sh_cnt + t * kPer)[q];
            c[4 * q] = v.x;
            c[4 * q + 1] = v.y;
            c[4 * q + 2] = v.z;
            c[4 * q + 3] = v.w;
        }
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            sum += c[q];
            c[q] = sum;
        }
        uint32_t total;
        const uint32_t base = block_exclusive_scan(sum, &total, sh_waves);
#pragma unroll
        for (int q = 0; q < kPer / 4; ++q)
            reinterpret_cast<uint4 *>(sh_cnt + t * kPer)[q] =
                make_uint4(base + c[4 * q], base + c[4 * q + 1], base + c[4 * q + 2], base + c[4 * q + 3]);
        __syncthreads();
        for (int64_t e = e0 + t; e < e1; e += kThreads) {
            const int64_t src = e + sh_delta[sh_cnt[e - e0] - 1];
            pcol[e] = col[src];
            pval[e] = val[src];
        }
    } else {
        // more rows than entries (empty rows): search the row pointers in memory
        for (int64_t e = e0 + t; e < e1; e += kThreads) {
            const int32_t r = row_of(pptr, r_lo, r_hi, e);
            const int64_t src = rowptr[order[r]] + (e - pptr[r]);
            pcol[e] = col[src];
            pval[e] = val[src];
        }
    }
}

constexpr int32_t kTaskProbe = 64;

// Does row i of the sorted order start a sparse-region task?  A task is a run of at most
// kTaskRows consecutive rows whose first entries lie in one window of kTaskEntries entries,
// or a run of at most kTaskRows consecutive empty rows: a run of empty rows (they share
// their first entry) is cut into tasks of kTaskRows from its first row, and the row after
// an empty row starts a task.
__device__ __forceinline__ bool starts_task(const int32_t *__restrict__ pptr, int32_t i) {
    const int32_t b = pptr[i];
    if (i == 0) return true;
    const bool empty = pptr[i + 1] == b;
    if (!empty && pptr[i - 1] == b) return true;      // the first row after empty rows
    // window start: empty rows count from the first row starting at b (the first of their
    // run: an earlier row ending at b is not empty, so it starts before b)
    const int32_t w0 = empty ? b : (b / kTaskEntries) * kTaskEntries;
    // first row whose first entry is >= w0: it lies within the last kTaskProbe rows unless
    // the window holds that many empty rows, so probe there before searching all of [0, i]
    int32_t lo = 0, hi = i;
    if (i >= kTaskProbe) {
        if (pptr[i - kTaskProbe] < w0) lo = i - kTaskProbe + 1;
        else hi = i - kTaskProbe;
    }
    while (lo < hi) {
        const int32_t mid = lo + (hi - lo) / 2;
        if (pptr[mid] < w0) lo = mid + 1;
        else hi = mid;
    }
    return (i - lo) % kTaskRows == 0;
}

// flags[i] = offsets[i] = 1 if row i starts a task (offsets is scanned afterwards).
__global__ __launch_bounds__(kThreads) void task_flag_kernel(const int32_t *__restrict__ pptr,
                                                             int32_t n,
                                                             const SplitSummary *__restrict__ sum,
                                                             uint32_t *__restrict__ flags,
                                                             uint32_t *__restrict__ offsets) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t f = (i < sum->n_sparse && starts_task(pptr, static_cast<int32_t>(i))) ? 1u : 0u;
    flags[i] = f;
    offsets[i] = f;
}

// tasks[offsets[i]] = i for every task start i; tasks[n_tasks] = n_sparse.
__global__ __launch_bounds__(kThreads) void task_fill_kernel(int32_t n,
                                                             const SplitSummary *__restrict__ sum,
                                                             const uint32_t *__restrict__ flags,
                                                             const uint32_t *__restrict__ offsets,
                                                             int32_t *__restrict__ tasks) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i == 0) tasks[sum->tasks] = sum->n_sparse;
    if (i < n && flags[i]) tasks[offsets[i]] = static_cast<int32_t>(i);
}

// Dense rows of the sorted order longer than one chunk: counts[i] = offsets[i] = number of
// parts (offsets is scanned afterwards).
__global__ __launch_bounds__(kThreads) void split_count_kernel(const int32_t *__restrict__ pptr,
                                                               int32_t n, int32_t chunk,
                                                               SplitSummary *__restrict__ sum,
                                                               uint32_t *__restrict__ counts,
                                                               uint32_t *__restrict__ offsets) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    uint32_t c = 0;
    if (i >= sum->n_sparse) {
        const int32_t deg = pptr[i + 1] - pptr[i];
        if (deg > chunk) {
            c = static_cast<uint32_t>((deg + chunk - 1) / chunk);
            atomicAdd(&sum->split_rows, 1);
        }
    }
    counts[i] = c;
    offsets[i] = c;        // scanned afterwards
}

__global__ __launch_bounds__(kThreads) void split_fill_kernel(const uint32_t *__restrict__ counts,
                                                              const uint32_t *__restrict__ offsets,
                                                              int32_t n,
                                                              SplitPart *__restrict__ parts,
                                                              uint32_t n_parts) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const uint32_t c = counts[i];
    if (c == 0) return;
    const uint32_t off = offsets[i];
    for (uint32_t j = 0; j < c && off + j < n_parts; ++j)
        parts[off + j] = SplitPart{static_cast<int32_t>(i), static_cast<int32_t>(j),
                                   static_cast<int32_t>(c), static_cast<int32_t>(off)};
}

// ------------------------------------------------------------------ host helpers

// Offsets of sub-arrays of one device block, each 256-byte aligned.
struct Layout {
    size_t bytes = 0;
    size_t take(size_t count_bytes) {
        const size_t o = bytes;
        bytes += (count_bytes + 255) / 256 * 256;
        return o;
    }
};

// A scratch block returned to the block cache once `stream` has finished with it.
struct ScratchBlock {
    void *p = nullptr;
    size_t bytes = 0;
    hipStream_t stream = nullptr;
    hipEvent_t done = nullptr;     // recorded after its last use, when that is known
    ~ScratchBlock() {
        if (p) {
            (void)(done ? wait_event(done) : wait_stream(stream));
            release_block(p, bytes);
        }
        if (done) (void)hipEventDestroy(done);
    }
};

}  // namespace

// Waits until an event has completed by polling it: a wait that blocks in the runtime
// resumes 50-150 us after the last kernel, which the partition's host waits would
// otherwise add to every build (the GPU idles meanwhile).  Polling stops after
// kPollLimit (the waits of a build take a few milliseconds at the sizes measured here);
// a longer wait blocks in the runtime instead of keeping a host core busy.
constexpr auto kPollLimit = std::chrono::milliseconds(20);
int wait_event(hipEvent_t e) {
    const auto t0 = std::chrono::steady_clock::now();
    for (;;) {
        const hipError_t q = hipEventQuery(e);
        if (q == hipSuccess) return DUALGCN_OK;
        if (q != hipErrorNotReady) return hip_status(q);
        if (std::chrono::steady_clock::now() - t0 > kPollLimit) return hip_status(hipEventSynchronize(e));
        std::this_thread::yield();
    }
}

int wait_stream(hipStream_t s) {
    hipEvent_t e = nullptr;
    int st = hip_status(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    if (st) return st;
    st = hip_status(hipEventRecord(e, s));
    if (!st) st = wait_event(e);
    (void)hipEventDestroy(e);
    return st;
}

namespace {

// A small pinned host buffer per host thread for the partition's read-backs: the copies
// into it are asynchronous, so the host waits only by polling (wait_stream, wait_event).
// It lives until the process ends (one buffer per thread that builds plans).
constexpr size_t kReadbackBytes = 256;
void *readback_buffer() {
    thread_local void *buf = nullptr;
    if (!buf && hipHostMalloc(&buf, kReadbackBytes, hipHostMallocPortable) != hipSuccess) buf = nullptr;
    return buf;
}

// Copies `bytes` of device memory to *dst through the pinned buffer and waits for them.
int read_back(void *dst, const void *src, size_t bytes, hipStream_t s) {
    void *pin = readback_buffer();
    if (!pin) return DUALGCN_ERR_OOM;
    int st = hip_status(hipMemcpyAsync(pin, src, bytes, hipMemcpyDeviceToHost, s));
    if (!st) st = wait_stream(s);
    if (!st) std::memcpy(dst, pin, bytes);
    return st;
}

// Exclusive scan of `count` u32 values in place; `sums` holds one word per tile.
// Writes the grand total to *grand (device) when grand is not null.
int exclusive_scan(uint32_t *data, int64_t count, uint32_t *sums, uint32_t *grand,
                   hipStream_t s) {
    const int64_t tiles = (count + kTile - 1) / kTile;
    if (tiles > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    if (tiles > 0) {
        hipLaunchKernelGGL(scan_reduce_kernel, dim3(static_cast<unsigned>(tiles)), dim3(kThreads),
                           0, s, data, count, sums);
    }
    hipLaunchKernelGGL(scan_top_kernel, dim3(1), dim3(kThreads), 0, s, sums,
                       static_cast<int32_t>(tiles), grand);
    if (tiles > 0) {
        hipLaunchKernelGGL(scan_apply_kernel, dim3(static_cast<unsigned>(tiles)), dim3(kThreads),
                           0, s, data, count, sums, data);
    }
    return hip_status(hipGetLastError());
}

int bit_length(uint64_t x) {
    int b = 0;
    while (x) {
        ++b;
        x >>= 1;
    }
    return b;
}

// Integer square root rounded up: least r with r*r >= x (digit-by-digit method).
u128 isqrt_ceil(u128 x) {
    u128 rem = x, root = 0, bit = static_cast<u128>(1) << 126;
    while (bit > rem) bit >>= 2;
    while (bit != 0) {
        if (rem >= root + bit) {
            rem -= root + bit;
            root = (root >> 1) + bit;
        } else {
            root >>= 1;
        }
        bit >>= 2;
    }
    return root * root == x ? root : root + 1;
}

bool mul_overflows(u128 a, u128 b, u128 *out) {
    if (a != 0 && b > (~static_cast<u128>(0)) / a) return true;
    *out = a * b;
    return false;
}

// K* = least integer K >= mu + (b/c) sigma over the n keys with sums s1, s2:
//   c (n K - s1) >= b sqrt(V),  V = n s2 - s1^2  (= n^2 sigma^2)
//   <=>  n K - s1 >= t := ceil(ceil(sqrt(b^2 V)) / c)  <=>  K >= ceil((s1 + t) / n).
int threshold_key(int32_t n, u128 s1, u128 s2, uint32_t b, uint32_t c, uint64_t *kstar) {
    u128 ns2, s1sq, bb, bbv;
    if (mul_overflows(static_cast<u128>(n), s2, &ns2)) return DUALGCN_ERR_UNSUPPORTED;
    if (mul_overflows(s1, s1, &s1sq)) return DUALGCN_ERR_UNSUPPORTED;
    if (ns2 < s1sq) return DUALGCN_ERR_HIP;  // impossible for exact sums
    const u128 V = ns2 - s1sq;
    bb = static_cast<u128>(b) * b;
    if (mul_overflows(bb, V, &bbv)) return DUALGCN_ERR_UNSUPPORTED;
    const u128 root = isqrt_ceil(bbv);
    const u128 t = (root + c - 1) / c;
    const u128 num = s1 + t;
    const u128 k = (num + static_cast<u128>(n) - 1) / static_cast<u128>(n);
    *kstar = k > static_cast<u128>(~0ull) ? ~0ull : static_cast<uint64_t>(k);
    return DUALGCN_OK;
}

// n^2 times the population variance of values with sums s1, s2: V = n s2 - s1^2.
int scaled_variance(int32_t n, u128 s1, u128 s2, u128 *V) {
    u128 ns2, s1sq;
    if (mul_overflows(static_cast<u128>(n), s2, &ns2)) return DUALGCN_ERR_UNSUPPORTED;
    if (mul_overflows(s1, s1, &s1sq)) return DUALGCN_ERR_UNSUPPORTED;
    if (ns2 < s1sq) return DUALGCN_ERR_HIP;  // impossible for exact sums
    *V = ns2 - s1sq;
    return DUALGCN_OK;
}

// Adaptive weight p/q = Var(N) / (Var(N) + Var(D)) rounded down (N = S / k), and
// q / 2 when neither metric varies: since Var(N) / Var(D) = V_S / (k^2 V_D),
// p = floor(q V_S / (V_S + k^2 V_D)).
int adaptive_weight(int32_t n, uint32_t k, uint32_t q, const Moments &ms, const Moments &md,
                    uint64_t *p) {
    u128 vs, vd, kvd, num;
    int st;
    if ((st = scaled_variance(n, join(ms.s1_lo, ms.s1_hi), join(ms.s2_lo, ms.s2_hi), &vs)))
        return st;
    if ((st = scaled_variance(n, join(md.s1_lo, md.s1_hi), join(md.s2_lo, md.s2_hi), &vd)))
        return st;
    if (mul_overflows(static_cast<u128>(k) * k, vd, &kvd)) return DUALGCN_ERR_UNSUPPORTED;
    const u128 den = vs + kvd;
    if (den < vs) return DUALGCN_ERR_UNSUPPORTED;
    if (den == 0) {
        *p = q / 2;
        return DUALGCN_OK;
    }
    if (mul_overflows(static_cast<u128>(q), vs, &num)) return DUALGCN_ERR_UNSUPPORTED;
    *p = static_cast<uint64_t>(num / den);
    return DUALGCN_OK;
}

// Balanced weight p/q: the largest multiple of 1/q with alpha sigma_N <= (1 - alpha) sigma_D
// (N = S / k), i.e. alpha = sigma_D / (sigma_N + sigma_D) rounded down, so that the two terms
// of H spread alike.  Squared and scaled by n^2 k^2 q^2:  p^2 V_S <= (q - p)^2 k^2 V_D, which
// is monotone in p (left side grows, right side shrinks): a binary search over [0, q].
// A metric that does not vary carries no information and gets no weight (p = 0 when S is
// constant, p = q when D is), and p = q / 2 when neither varies.
int balanced_weight(int32_t n, uint32_t k, uint32_t q, const Moments &ms, const Moments &md,
                    uint64_t *p) {
    u128 vs, vd, kvd;
    int st;
    if ((st = scaled_variance(n, join(ms.s1_lo, ms.s1_hi), join(ms.s2_lo, ms.s2_hi), &vs)))
        return st;
    if ((st = scaled_variance(n, join(md.s1_lo, md.s1_hi), join(md.s2_lo, md.s2_hi), &vd)))
        return st;
    if (vs == 0 || vd == 0) {
        *p = vs == 0 && vd == 0 ? q / 2 : (vs == 0 ? 0 : q);
        return DUALGCN_OK;
    }
    if (mul_overflows(static_cast<u128>(k) * k, vd, &kvd)) return DUALGCN_ERR_UNSUPPORTED;
    uint64_t lo = 0, hi = q;          // p = lo satisfies the inequality, p = q does not
    while (hi - lo > 1) {
        const uint64_t mid = lo + (hi - lo) / 2;
        u128 left, right;
        if (mul_overflows(static_cast<u128>(mid) * mid, vs, &left) ||
            mul_overflows(static_cast<u128>(q - mid) * (q - mid), kvd, &right))
            return DUALGCN_ERR_UNSUPPORTED;
        if (left <= right) lo = mid;
        else hi = mid;
    }
    *p = lo;
    return DUALGCN_OK;
}

// s2 = sum K^2 is accumulated modulo 2^128; it cannot have wrapped when
// kmax * s1 (an upper bound of it) fits.
bool square_sum_fits(const Moments &m) {
    u128 bound;
    return !mul_overflows(static_cast<u128>(m.kmax), join(m.s1_lo, m.s1_hi), &bound);
}

}  // namespace

int validate_csr(const dualgcn_csr *csr, int32_t *flags, int2 *nodeinfo, int32_t *blockmax,
                 uint32_t *heat_hist, hipStream_t s, bool check_cols) {
    hipLaunchKernelGGL(validate_kernel, dim3(kValidateBlocks), dim3(kThreads), 0, s, csr->rowptr,
                       csr->col, csr->n, csr->nnz, flags, nodeinfo, blockmax, heat_hist,
                       check_cols ? 1 : 0);
    return hip_status(hipGetLastError());
}

void free_plan(Plan *p) {
    if (!p) return;
    if (p->pending) release_block(p->pending, p->pending_bytes);
    release_block(p->mem, p->mem_bytes);
    if (p->ready) (void)hipEventDestroy(p->ready);
    for (auto &u : p->uses) (void)hipEventDestroy(u.second);
    delete p;
}

int note_use(const Plan &p, hipStream_t s) {
    std::lock_guard<std::mutex> lock(p.use_mu);
    for (auto &u : p.uses)
        if (u.first == s) return hip_status(hipEventRecord(u.second, s));
    hipEvent_t e = nullptr;
    int st = hip_status(hipEventCreateWithFlags(&e, hipEventDisableTiming));
    if (st) return st;
    if ((st = hip_status(hipEventRecord(e, s)))) {
        (void)hipEventDestroy(e);
        return st;
    }
    p.uses.emplace_back(s, e);
    return DUALGCN_OK;
}

void release_pending(const Plan &p) {
    std::lock_guard<std::mutex> lock(p.use_mu);
    if (!p.pending) return;
    release_block(p.pending, p.pending_bytes);
    p.pending = nullptr;
    p.pending_bytes = 0;
}

int wait_plan_idle(const Plan &p) {
    int st = p.ready ? wait_event(p.ready) : DUALGCN_OK;
    if (!st) release_pending(p);
    std::lock_guard<std::mutex> lock(p.use_mu);
    for (auto &u : p.uses)
        if (!st) st = wait_event(u.second);
    return st;
}

int structure_checksum(const int32_t *rowptr, const int32_t *col, int32_t n, int64_t nnz,
                       hipStream_t s, uint64_t *out) {
    void *buf = nullptr;
    int st = alloc_bytes(&buf, sizeof(uint64_t) * (kSumBlocks + 1));
    if (st) return st;
    uint64_t *partial = static_cast<uint64_t *>(buf);
    hipLaunchKernelGGL(checksum_kernel, dim3(kSumBlocks), dim3(kThreads), 0, s, rowptr, col, n, nnz,
                       partial);
    hipLaunchKernelGGL(checksum_fold_kernel, dim3(1), dim3(1), 0, s, partial);
    st = hip_status(hipGetLastError());
    if (!st) st = hip_status(hipMemcpyAsync(out, partial + kSumBlocks, sizeof(uint64_t),
                                            hipMemcpyDeviceToHost, s));
    if (!st) st = hip_status(hipStreamSynchronize(s));
    (void)hipFree(buf);
    return st;
}

int build_plan(const dualgcn_csr *csr, uint64_t seed, uint32_t k, uint32_t d,
               const dualgcn_thresholds &th, const uint32_t *S_host, hipStream_t s, Plan **out) {
    const int32_t n = csr->n;
    const int64_t nnz = csr->nnz;
    const size_t un = static_cast<size_t>(n), unnz = static_cast<size_t>(nnz);
    Plan *p = new (std::nothrow) Plan();
    if (!p) return DUALGCN_ERR_OOM;
    struct Guard {   // on an error return: wait for the queued work, then release
        Plan *p;
        hipStream_t s;
        ~Guard() {
            if (!p) return;
            (void)hipStreamSynchronize(s);
            free_plan(p);
        }
    } guard{p, s};
    int st;
    if ((st = hip_status(hipGetDevice(&p->device)))) return st;
    p->n = n;
    p->nnz = nnz;
    p->rowptr = csr->rowptr;
    p->col = csr->col;
    p->val = csr->val;
    p->th = th;
    p->seed = seed;
    p->k = k;
    p->d = d;

    // Every array of the plan lives in one device block, every scratch array of the
    // build in another: two allocations per plan.  Split parts are bounded by
    // sum over rows longer than C of ceil(deg / C) < 2 nnz / C + 1.
    p->dense_chunk = dense_chunk_for(nnz);
    const size_t max_parts = unnz / static_cast<size_t>(p->dense_chunk) * 2 + 1;
    // The lockstep walker reads successor records (8 bytes per entry, scratch) when the
    // walks take at least twice as many steps as the matrix has entries: building them
    // costs one random read per entry and saves one dependent random read per step.
    const bool use_succ = S_host == nullptr &&
                          static_cast<u128>(n) * k * d >= 2 * static_cast<u128>(unnz);
    // columns outside the hottest kHotRows are marked (bit 31 of the sorted copy's columns)
    // for the cache classes of the gathers, only when a launch on the plan can use them
    // (an operand of rows up to kMaxSlice floats larger than kGatherClassMinBytes): the
    // successor pass writes the marked columns and the sorted copy reads them
    const bool mark = nnz > 0 && static_cast<uint64_t>(n) * kMaxSlice * sizeof(float) > kGatherClassMinBytes;
    const int32_t nb_keys = static_cast<int32_t>(std::min<int64_t>((n + kThreads - 1) / kThreads, 1024));
    const int sort_items = n < kSortSmallKeys ? kSortItemsSmall : kItems;
    const int64_t sort_tile = static_cast<int64_t>(kThreads) * sort_items;
    const int32_t nblocks = static_cast<int32_t>((static_cast<int64_t>(n) + sort_tile - 1) / sort_tile);
    const int64_t scan_tiles = std::max((static_cast<int64_t>(kRadix) * nblocks + kTile - 1) / kTile,
                                        (static_cast<int64_t>(n) + 1 + kTile - 1) / kTile) + 1;
    Layout lp, ls;
    const size_t o_S = lp.take(sizeof(uint32_t) * un), o_K = lp.take(sizeof(uint64_t) * un),
                 o_perm = lp.take(sizeof(int32_t) * un), o_order = lp.take(sizeof(int32_t) * un),
                 o_pptr = lp.take(sizeof(int32_t) * (un + 1)),
                 o_pcol = lp.take(sizeof(int32_t) * unnz), o_pval = lp.take(sizeof(float) * unnz),
                 o_tasks = lp.take(sizeof(int32_t) * (un + 1)),
                 o_parts = lp.take(sizeof(SplitPart) * max_parts),
                 o_partials = lp.take(sizeof(double) * max_parts * kMaxSlice),
                 o_tiles = lp.take(sizeof(int32_t) * (unnz / kCopyTile + 2));
    // the validation flags and the heat histogram are cleared by one fill; the hot heat
    // value follows them
    constexpr size_t kFlagBytes = 2 * sizeof(int32_t), kHistBytes = sizeof(uint32_t) * kHeatLevels;
    const size_t o_flags = ls.take(kFlagBytes + kHistBytes + sizeof(uint32_t)), o_mom = ls.take(sizeof(Moments) * nb_keys),
                 o_sum = ls.take(2 * sizeof(Summary)), o_kb0 = ls.take(sizeof(uint64_t) * un),
                 o_kb1 = ls.take(sizeof(uint64_t) * un), o_vb0 = ls.take(sizeof(int32_t) * un),
                 o_scan = ls.take(sizeof(uint32_t) * static_cast<size_t>(scan_tiles)),
                 o_hist = ls.take(sizeof(uint32_t) * kRadix * static_cast<size_t>(nblocks)),
                 o_ssum = ls.take(sizeof(SplitSummary)), o_counts = ls.take(sizeof(uint32_t) * 2 * ((un + 3) / 4 * 4)),
                 o_info = ls.take(sizeof(int2) * un),
                 o_succ = ls.take(use_succ ? sizeof(int2) * unnz : 0),
                 o_marked = ls.take(mark ? sizeof(int32_t) * unnz : 0),
                 o_bmax = ls.take(sizeof(int32_t) * kValidateBlocks);
    if ((st = alloc_block(&p->mem, &p->mem_bytes, lp.bytes))) return st;
    ScratchBlock scratch;
    scratch.stream = s;
    if ((st = alloc_block(&scratch.p, &scratch.bytes, ls.bytes))) return st;
    char *pm = static_cast<char *>(p->mem);
    char *sm = static_cast<char *>(scratch.p);
    p->S = reinterpret_cast<uint32_t *>(pm + o_S);
    p->K = reinterpret_cast<uint64_t *>(pm + o_K);
    p->perm = reinterpret_cast<int32_t *>(pm + o_perm);
    p->order = reinterpret_cast<int32_t *>(pm + o_order);
    p->pptr = reinterpret_cast<int32_t *>(pm + o_pptr);
    p->pcol = reinterpret_cast<int32_t *>(pm + o_pcol);
    p->pval = reinterpret_cast<float *>(pm + o_pval);
    p->tasks = reinterpret_cast<int32_t *>(pm + o_tasks);
    p->parts = reinterpret_cast<SplitPart *>(pm + o_parts);
    p->partials = reinterpret_cast<double *>(pm + o_partials);
    p->tile_row = reinterpret_cast<int32_t *>(pm + o_tiles);
    p->cold_marked = mark;
    int32_t *marked = mark ? reinterpret_cast<int32_t *>(sm + o_marked) : nullptr;
    int32_t *bad = reinterpret_cast<int32_t *>(sm + o_flags);
    uint32_t *heat_hist = reinterpret_cast<uint32_t *>(sm + o_flags + kFlagBytes);
    uint32_t *hot_heat = heat_hist + kHeatLevels;
    Moments *moments = reinterpret_cast<Moments *>(sm + o_mom);
    Summary *summary = reinterpret_cast<Summary *>(sm + o_sum);
    uint64_t *kb0 = reinterpret_cast<uint64_t *>(sm + o_kb0);
    uint64_t *kb1 = reinterpret_cast<uint64_t *>(sm + o_kb1);
    int32_t *vb0 = reinterpret_cast<int32_t *>(sm + o_vb0);
    uint32_t *scan_sums = reinterpret_cast<uint32_t *>(sm + o_scan);
    uint32_t *hist = reinterpret_cast<uint32_t *>(sm + o_hist);
    // one pass of the radix sort: the digit histogram of `keys` at `shift`, or the scatter
    auto radix_hist = [&](const uint64_t *keys, int shift) {
        if (sort_items == kItems)
            hipLaunchKernelGGL(radix_hist_kernel<kItems>, dim3(nblocks), dim3(kThreads), 0, s, keys, n,
                               shift, hist, nblocks);
        else
            hipLaunchKernelGGL(radix_hist_kernel<kSortItemsSmall>, dim3(nblocks), dim3(kThreads), 0, s,
                               keys, n, shift, hist, nblocks);
    };
    auto radix_scatter = [&](const uint64_t *kin, const int32_t *vin, int shift, uint64_t *kout,
                             int32_t *vout) {
        if (sort_items == kItems)
            hipLaunchKernelGGL(radix_scatter_kernel<kItems>, dim3(nblocks), dim3(kThreads), 0, s, kin,
                               vin, n, shift, hist, nblocks, kout, vout);
        else
            hipLaunchKernelGGL(radix_scatter_kernel<kSortItemsSmall>, dim3(nblocks), dim3(kThreads), 0,
                               s, kin, vin, n, shift, hist, nblocks, kout, vout);
    };
    SplitSummary *dsum = reinterpret_cast<SplitSummary *>(sm + o_ssum);
    uint32_t *cnt = reinterpret_cast<uint32_t *>(sm + o_counts);
    uint32_t *off = cnt + (static_cast<int64_t>(n) + 3) / 4 * 4;    // 16-byte aligned
    int2 *nodeinfo = reinterpret_cast<int2 *>(sm + o_info);
    int32_t *blockmax = reinterpret_cast<int32_t *>(sm + o_bmax);

    TraceRange phase("partition: validate + walks");
    if ((st = hip_status(hipMemsetAsync(bad, 0, kFlagBytes + kHistBytes, s)))) return st;
    // the successor pass reads every column: where it runs, it checks them in place of the
    // validation (which then reads only the row pointers)
    const bool succ_pass = (use_succ || mark) && nnz > 0;
    if ((st = validate_csr(csr, bad, nodeinfo, blockmax, mark ? heat_hist : nullptr, s, !succ_pass)))
        return st;
    if (mark) hipLaunchKernelGGL(hot_heat_kernel, dim3(1), dim3(kHeatLevels), 0, s, heat_hist, kHotRows, hot_heat);
    int2 *succ = nullptr;
    if (succ_pass) {
        if (use_succ) succ = reinterpret_cast<int2 *>(sm + o_succ);
        const int64_t sblocks = std::min<int64_t>((nnz + kThreads - 1) / kThreads, 65536);
        hipLaunchKernelGGL(successor_kernel, dim3(static_cast<unsigned>(sblocks)), dim3(kThreads), 0,
                           s, nodeinfo, csr->col, n, nnz, succ, hot_heat, marked, bad);
    }
    if (S_host) {
        // the density sums of a saved plan of this matrix: no walks
        if ((st = hip_status(hipMemcpyAsync(p->S, S_host, sizeof(uint32_t) * un,
                                            hipMemcpyHostToDevice, s))))
            return st;
    } else {
        // walks: the lockstep walker where it applies, else one walk per lane
        st = launch_density(nodeinfo, csr->col, succ, n, seed, k, d, p->S, bad, s);
        if (st == DUALGCN_ERR_UNSUPPORTED)
            st = launch_arw(csr->rowptr, csr->col, n, seed, k, d, p->S, nullptr, bad, s);
        if (st) return st;
    }
    // adaptive or balanced alpha: moments of S and of D (two passes of the key kernel with
    // the weights (1, 0) and (0, 1)), one more host wait, the weight chosen on the host
    uint64_t pa = th.alpha_num;
    const uint64_t qa = th.alpha_den;
    if (th.alpha_num == DUALGCN_ALPHA_ADAPTIVE || th.alpha_num == DUALGCN_ALPHA_BALANCED) {
        const uint64_t weights[2][2] = {{1, 0}, {0, 1}};
        for (int m = 0; m < 2; ++m) {
            hipLaunchKernelGGL(keys_kernel, dim3(nb_keys), dim3(kThreads), 0, s, csr->rowptr, p->S,
                               n, weights[m][0], weights[m][1], p->K, moments, bad);
            hipLaunchKernelGGL(fold_kernel, dim3(1), dim3(kThreads), 0, s, moments, nb_keys, bad,
                               blockmax, summary + m);
        }
        if ((st = hip_status(hipGetLastError()))) return st;
        Summary two[2];
        static_assert(sizeof(two) <= kReadbackBytes, "read-back buffer");
        if ((st = read_back(two, summary, sizeof(two), s))) return st;    // adaptive alphas only
        if (two[0].flag) return DUALGCN_ERR_BAD_CSR;
        if (!square_sum_fits(two[0].m) || !square_sum_fits(two[1].m)) return DUALGCN_ERR_UNSUPPORTED;
        st = th.alpha_num == DUALGCN_ALPHA_ADAPTIVE
                 ? adaptive_weight(n, k, th.alpha_den, two[0].m, two[1].m, &pa)
                 : balanced_weight(n, k, th.alpha_den, two[0].m, two[1].m, &pa);
        if (st) return st;
        p->th.alpha_num = static_cast<uint32_t>(pa);
    }
    phase.next("partition: keys + threshold");
    // keys and moments
    hipLaunchKernelGGL(keys_kernel, dim3(nb_keys), dim3(kThreads), 0, s, csr->rowptr, p->S, n,
                       pa, (qa - pa) * k, p->K, moments, bad);
    hipLaunchKernelGGL(fold_kernel, dim3(1), dim3(kThreads), 0, s, moments, nb_keys, bad, blockmax,
                       summary);
    if ((st = hip_status(hipGetLastError()))) return st;
    Summary sum{};
    {
        // host wait 1 reads the sums; the work that needs no threshold is queued behind the
        // read-back so that it runs while the host wakes up: perm cleared (every entry is a
        // valid node id even before the sort writes it), and the histogram and scan of the
        // sort's first digit
        void *pin = readback_buffer();
        if (!pin) return DUALGCN_ERR_OOM;
        if ((st = hip_status(hipMemcpyAsync(pin, summary, sizeof(sum), hipMemcpyDeviceToHost, s))))
            return st;
        struct Event {
            hipEvent_t e = nullptr;
            ~Event() {
                if (e) (void)hipEventDestroy(e);
            }
        } sums_read;
        if ((st = hip_status(hipEventCreateWithFlags(&sums_read.e, hipEventDisableTiming)))) return st;
        if ((st = hip_status(hipEventRecord(sums_read.e, s)))) return st;
        if ((st = hip_status(hipMemsetAsync(p->perm, 0, sizeof(int32_t) * un, s)))) return st;
        radix_hist(p->K, 0);
        if ((st = hip_status(hipGetLastError()))) return st;
        if ((st = exclusive_scan(hist, static_cast<int64_t>(kRadix) * nblocks, scan_sums, nullptr, s)))
            return st;
        if ((st = wait_event(sums_read.e))) return st;
        std::memcpy(&sum, pin, sizeof(sum));
    }
    if (sum.flag) return DUALGCN_ERR_BAD_CSR;

    p->max_degree = sum.maxdeg;
    p->s1 = join(sum.m.s1_lo, sum.m.s1_hi);
    p->s2 = join(sum.m.s2_lo, sum.m.s2_hi);
    p->kmax = sum.m.kmax;
    if (!square_sum_fits(sum.m)) return DUALGCN_ERR_UNSUPPORTED;
    if ((st = threshold_key(n, p->s1, p->s2, th.beta_num, th.beta_den, &p->kstar))) return st;

    phase.next("partition: sort");
    // stable radix sort of (K, v) on the bits the keys use (the first digit's histogram and
    // scan are already queued)
    const int passes = (bit_length(p->kmax) + kRadixBits - 1) / kRadixBits;
    uint64_t *sorted = nullptr;
    if (passes == 0) {
        hipLaunchKernelGGL(iota_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, s,
                           p->perm, n);
        if ((st = hip_status(hipMemcpyAsync(kb0, p->K, sizeof(uint64_t) * un,
                                            hipMemcpyDeviceToDevice, s))))
            return st;
        sorted = kb0;
    } else {
        // ping-pong so that the last pass lands its values in p->perm
        int32_t *vbuf[2];
        uint64_t *kbuf[2] = {kb0, kb1};
        if (passes % 2 == 1) {
            vbuf[0] = p->perm;
            vbuf[1] = vb0;
        } else {
            vbuf[0] = vb0;
            vbuf[1] = p->perm;
        }
        const uint64_t *kin = p->K;
        const int32_t *vin = nullptr;   // identity on the first pass
        for (int pass = 0; pass < passes; ++pass) {
            const int shift = pass * kRadixBits;
            uint64_t *kout = kbuf[pass % 2];
            int32_t *vout = vbuf[pass % 2];
            if (pass > 0) {
                radix_hist(kin, shift);
                if ((st = hip_status(hipGetLastError()))) return st;
                if ((st = exclusive_scan(hist, static_cast<int64_t>(kRadix) * nblocks, scan_sums,
                                         nullptr, s)))
                    return st;
            }
            radix_scatter(kin, vin, shift, kout, vout);
            if ((st = hip_status(hipGetLastError()))) return st;
            kin = kout;
            vin = vout;
        }
        sorted = const_cast<uint64_t *>(kin);
    }

    // region split, the sorted copy of the matrix, sparse tasks and dense-row parts
    int32_t forced = -1;
    if (th.force_mode == DUALGCN_FORCE_SPARSE) forced = n;
    if (th.force_mode == DUALGCN_FORCE_DENSE) forced = 0;
    hipLaunchKernelGGL(lower_bound_kernel, dim3(1), dim3(64), 0, s, sorted, n, p->kstar, forced, dsum);
    const unsigned grid_n1 = static_cast<unsigned>((static_cast<int64_t>(n) + 1 + kThreads - 1) / kThreads);
    const unsigned grid_n = static_cast<unsigned>((static_cast<int64_t>(n) + kThreads - 1) / kThreads);
    // processing order: one stable 8-bit pass over the node ids (keys < 64); the buffer of
    // the sorted keys is free again once lower_bound has run (same stream)
    {
        const int32_t region = th.force_mode == DUALGCN_FORCE_SPARSE ? 0
                               : th.force_mode == DUALGCN_FORCE_DENSE ? 1 : -1;
        uint64_t *okey = sorted == kb0 ? kb1 : kb0;
        uint64_t *okey_out = sorted == kb0 ? kb0 : kb1;
        hipLaunchKernelGGL(order_key_kernel, dim3(grid_n), dim3(kThreads), 0, s, p->K, p->kstar,
                           region, csr->rowptr, n, okey);
        radix_hist(okey, 0);
        if ((st = exclusive_scan(hist, static_cast<int64_t>(kRadix) * nblocks, scan_sums, nullptr, s)))
            return st;
        radix_scatter(okey, nullptr, 0, okey_out, p->order);
        hipLaunchKernelGGL(long_rows_kernel, dim3(1), dim3(64), 0, s, hist, nblocks, n, dsum);
        if ((st = hip_status(hipGetLastError()))) return st;
    }
    uint32_t *pptr_u = reinterpret_cast<uint32_t *>(p->pptr);
    phase.next("partition: sorted copy + schedule");
    hipLaunchKernelGGL(sorted_degree_kernel, dim3(grid_n1), dim3(kThreads), 0, s, p->order, csr->rowptr,
                       n, pptr_u);
    if ((st = exclusive_scan(pptr_u, static_cast<int64_t>(n) + 1, scan_sums, nullptr, s))) return st;
    hipLaunchKernelGGL(task_flag_kernel, dim3(grid_n), dim3(kThreads), 0, s, p->pptr, n, dsum, cnt,
                       off);
    if ((st = exclusive_scan(off, n, scan_sums, &dsum->tasks, s))) return st;
    hipLaunchKernelGGL(task_fill_kernel, dim3(grid_n), dim3(kThreads), 0, s, n, dsum, cnt, off,
                       p->tasks);
    hipLaunchKernelGGL(split_count_kernel, dim3(grid_n), dim3(kThreads), 0, s, p->pptr, n,
                       p->dense_chunk, dsum, cnt, off);
    if ((st = exclusive_scan(off, n, scan_sums, &dsum->parts, s))) return st;
    hipLaunchKernelGGL(split_fill_kernel, dim3(grid_n), dim3(kThreads), 0, s, cnt, off, n, p->parts,
                       static_cast<uint32_t>(max_parts));
    if ((st = hip_status(hipGetLastError()))) return st;
    // the schedule sizes are read back while the sorted copy, the last kernel and the only
    // one after them, runs: it reads the plan and the caller's matrix, not the scratch block
    static_assert(sizeof(SplitSummary) <= kReadbackBytes, "read-back buffer");
    void *pin = readback_buffer();
    if (!pin) return DUALGCN_ERR_OOM;
    if ((st = hip_status(hipMemcpyAsync(pin, dsum, sizeof(SplitSummary), hipMemcpyDeviceToHost, s))))
        return st;
    {
        // host wait 2 reads the sizes at this point; the scratch block's last use is here
        // too, unless the sorted copy reads the marked columns from it: then the plan keeps
        // the block until its `ready` event (after the copy) is seen complete, so that the
        // host does not wait for the copy (an early return from here on synchronises the
        // stream before the plan and the block are released)
        hipEvent_t done = nullptr;
        if ((st = hip_status(hipEventCreateWithFlags(&done, hipEventDisableTiming)))) return st;
        if ((st = hip_status(hipEventRecord(done, s)))) {
            (void)hipEventDestroy(done);
            return st;
        }
        scratch.done = done;
        if (marked) {
            p->pending = scratch.p;
            p->pending_bytes = scratch.bytes;
            scratch.p = nullptr;
        }
    }
    if (nnz > 0) {
        const unsigned grid_e = static_cast<unsigned>((nnz + kCopyTile - 1) / kCopyTile);
        hipLaunchKernelGGL(tile_row_kernel, dim3(grid_n), dim3(kThreads), 0, s, p->pptr, n, p->tile_row);
        hipLaunchKernelGGL(sorted_copy_kernel, dim3(grid_e), dim3(kThreads), 0, s, p->order,
                           csr->rowptr, marked ? marked : csr->col, csr->val, p->pptr, p->tile_row,
                           n, nnz, p->pcol, p->pval);
        if ((st = hip_status(hipGetLastError()))) return st;
    }
    // every use of the plan's sorted copy waits for this event (its stream, or any other)
    if ((st = hip_status(hipEventCreateWithFlags(&p->ready, hipEventDisableTiming)))) return st;
    if ((st = hip_status(hipEventRecord(p->ready, s)))) return st;
    // host wait 2: the region and schedule sizes; the scratch block is released after it
    if ((st = wait_event(scratch.done))) return st;
    SplitSummary ss{};
    std::memcpy(&ss, pin, sizeof(ss));
    if (ss.parts > max_parts) return DUALGCN_ERR_HIP;    // impossible: bounded above
    p->n_sparse = ss.n_sparse;
    p->n_tasks = static_cast<int32_t>(ss.tasks);
    for (int c = 0; c < kLongRowClasses; ++c) p->n_long[c] = ss.long_rows[c];
    p->n_split_rows = ss.split_rows;
    p->n_split_parts = static_cast<int32_t>(ss.parts);
    guard.p = nullptr;
    *out = p;
    return DUALGCN_OK;
}

}  // namespace dgc
