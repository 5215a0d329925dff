// Anonymous random walks and neighbour-density sums on gfx950.
//
// DualGCN Sec. 3.2 ("Theoretical Foundation", Theorem 1, "Neighbor Density"):
// a walk repeatedly moves to a random neighbour and labels every visited node
// by the order of its first occurrence; the density of node v is the mean
// number of distinct nodes over its k walks, N_v = S_v / k.
//
// When only the sums are needed (the partition) and d <= 32, one lane runs two
// walks of a node in lockstep, so that both walks' reads are in flight together;
// the lanes of a node are adjacent and their counts are summed across lanes.  For
// the walk patterns, or longer walks, one lane runs one (node, walk) pair.  Counts
// that cannot be summed inside one wavefront are added with integer atomics
// (order-independent, hence exact).
//
// Random stream: step s of walk w from v uses the 32-bit half r (low for even s,
// high for odd s) of 64-bit word floor(s/2) mod 4 of the Philox-4x64-10 block
// (Salmon, Moraes, Dror & Shaw, SC'11) with counter (v, w, floor(s/8), 0) and key
// (seed, 0); one block serves eight steps.  The neighbour is entry
// floor(r * deg / 2^32) of the current row (uniform over stored entries); an
// empty row keeps the walk in place.  A walk of up to eight steps thus costs one
// Philox evaluation; what bounds the kernel is the chain of dependent random reads
// (row bounds, then a column entry) at every step.
#include "internal.h"

namespace dgc {
namespace {

// Philox-4x64 multipliers and Weyl key increments, as published.
constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;

struct Block4 {
    uint64_t w[4];
};

// The 32-bit half of the block spent on step s (s is a compile-time index after unrolling).
__device__ __forceinline__ uint32_t half_word(const Block4 &b, int s) {
    const uint64_t word = b.w[(s >> 1) & 3];
    return (s & 1) ? static_cast<uint32_t>(word >> 32) : static_cast<uint32_t>(word);
}

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                                uint64_t c3, uint64_t k0, uint64_t k1) {
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t lo0 = kPhiloxM0 * c0;
        const uint64_t hi0 = __umul64hi(kPhiloxM0, c0);
        const uint64_t lo1 = kPhiloxM1 * c2;
        const uint64_t hi1 = __umul64hi(kPhiloxM1, c2);
        const uint64_t n0 = hi1 ^ c1 ^ k0;
        const uint64_t n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += kPhiloxW0;
        k1 += kPhiloxW1;
    }
    return Block4{{c0, c1, c2, c3}};
}

// One walk of `d` steps (d <= MAXD).  Returns the number of distinct nodes.
// path[i] is the i-th visited node and lab[i] its label; a revisited node takes
// the label of any earlier position holding it.  With UNROLL the arrays are
// indexed only by compile-time positions and stay in registers.
template <int MAXD, bool UNROLL>
__device__ __forceinline__ uint32_t walk_one(const int32_t *__restrict__ rowptr,
                                             const int32_t *__restrict__ col, uint32_t v,
                                             uint32_t w, uint32_t d, uint64_t seed,
                                             uint8_t *__restrict__ pat) {
    int32_t path[MAXD + 1];
    uint8_t lab[MAXD + 1];
    path[0] = static_cast<int32_t>(v);
    lab[0] = 1;
    if (pat) pat[0] = 1;
    uint32_t distinct = 1;
    int32_t cur = static_cast<int32_t>(v);
    Block4 blk{};
    constexpr int kUnrollSteps = UNROLL ? MAXD : 1;
#pragma unroll kUnrollSteps
    for (int s = 0; s < MAXD; ++s) {
        if (static_cast<uint32_t>(s) >= d) break;
        if ((s & 7) == 0) blk = philox4x64_10(v, w, static_cast<uint64_t>(s >> 3), 0, seed, 0);
        const uint32_t r = half_word(blk, s);
        const int32_t b = rowptr[cur];
        const int32_t e = rowptr[cur + 1];
        int32_t nxt = cur;
        if (e > b) nxt = col[b + static_cast<int32_t>(__umulhi(r, static_cast<uint32_t>(e - b)))];
        uint8_t label = 0;
#pragma unroll kUnrollSteps
        for (int i = 0; i <= s; ++i)
            if (path[i] == nxt) label = lab[i];
        if (label == 0) label = static_cast<uint8_t>(++distinct);
        path[s + 1] = nxt;
        lab[s + 1] = label;
        if (pat) pat[s + 1] = label;
        cur = nxt;
    }
    return distinct;
}

// Walks w0 .. w0 + nw - 1 (nw <= WPL) of d steps (d <= MAXD) from node v advanced in
// lockstep, so that their memory reads are in flight together; u[j] receives the
// distinct-node count of walk w0 + j (0 for j >= nw).  Same stream and counts as walk_one (no pattern output).  A walk that
// steps onto a node whose only entry is a self-loop (or that has no entry) can never
// leave it nor meet a new node, so it stops reading memory there: its lane is masked
// off for the remaining steps, which saves L2 requests without changing any count.
template <int MAXD, int WPL>
__device__ __forceinline__ void walk_lockstep(const int2 *__restrict__ nodeinfo,
                                              const int32_t *__restrict__ col, uint32_t v,
                                              uint32_t w0, uint32_t nw, uint32_t d, uint64_t seed,
                                              uint32_t (&u)[WPL]) {
    int32_t path[WPL][MAXD + 1];
    int32_t cur[WPL];
    bool live[WPL];
    Block4 blk[WPL];
#pragma unroll
    for (int j = 0; j < WPL; ++j) {       // walks w0 + j for j < nw; the others count 0
        path[j][0] = static_cast<int32_t>(v);
        cur[j] = static_cast<int32_t>(v);
        live[j] = static_cast<uint32_t>(j) < nw;
        u[j] = live[j] ? 1 : 0;
    }
#pragma unroll MAXD
    for (int s = 0; s < MAXD; ++s) {
        if (static_cast<uint32_t>(s) >= d) break;
        int2 ni[WPL];             // (first entry, degree) of the current nodes
#pragma unroll
        for (int j = 0; j < WPL; ++j) {
            ni[j] = make_int2(0, 0);
            if (live[j]) {
                if ((s & 7) == 0) blk[j] = philox4x64_10(v, w0 + j, static_cast<uint64_t>(s >> 3), 0, seed, 0);
                ni[j] = nodeinfo[cur[j]];
            }
        }
        int32_t nxt[WPL];
#pragma unroll
        for (int j = 0; j < WPL; ++j) {
            nxt[j] = cur[j];
            if (live[j] && ni[j].y > 0) {
                const uint32_t r = half_word(blk[j], s);
                nxt[j] = col[ni[j].x + static_cast<int32_t>(__umulhi(r, static_cast<uint32_t>(ni[j].y)))];
            }
        }
#pragma unroll
        for (int j = 0; j < WPL; ++j) {
            if (live[j]) {
                bool seen = false;
#pragma unroll MAXD
                for (int i = 0; i <= s; ++i) seen |= path[j][i] == nxt[j];
                if (!seen) ++u[j];
                live[j] = !(ni[j].y <= 1 && nxt[j] == cur[j]);   // absorbed: stays put for good
            }
            path[j][s + 1] = nxt[j];
            cur[j] = nxt[j];
        }
    }
}

// The same lockstep walks over successor records: succ[e] = (first entry, degree) of
// the node in column e, so one 8-byte read per step yields the next node together with
// what the step after it needs -- one dependent random read per step instead of two.
// A node is identified by its first entry, which is unique among nodes with entries;
// a node without entries (it shares its first entry with the next node that has some)
// gets bit 31 set.  A walk meets at most one such node, as its last, since it never
// leaves it, so the keys tell apart every pair of nodes one walk can visit.
__device__ __forceinline__ int32_t node_key(int2 rec) {
    return rec.y > 0 ? rec.x : static_cast<int32_t>(static_cast<uint32_t>(rec.x) | 0x80000000u);
}

template <int MAXD, int WPL>
__device__ __forceinline__ void walk_lockstep_succ(const int2 *__restrict__ nodeinfo,
                                                   const int2 *__restrict__ succ, uint32_t v,
                                                   uint32_t w0, uint32_t nw, uint32_t d,
                                                   uint64_t seed, uint32_t (&u)[WPL]) {
    int32_t path[WPL][MAXD + 1];
    int2 cur[WPL];                // (first entry, degree) of the current node
    bool live[WPL];
    Block4 blk[WPL];
    const int2 start = nodeinfo[v];
#pragma unroll
    for (int j = 0; j < WPL; ++j) {
        path[j][0] = node_key(start);
        cur[j] = start;
        live[j] = static_cast<uint32_t>(j) < nw;
        u[j] = live[j] ? 1 : 0;
    }
#pragma unroll MAXD
    for (int s = 0; s < MAXD; ++s) {
        if (static_cast<uint32_t>(s) >= d) break;
        int2 nxt[WPL];
#pragma unroll
        for (int j = 0; j < WPL; ++j) {
            nxt[j] = cur[j];
            if (live[j] && cur[j].y > 0) {
                if ((s & 7) == 0) blk[j] = philox4x64_10(v, w0 + j, static_cast<uint64_t>(s >> 3), 0, seed, 0);
                const uint32_t r = half_word(blk[j], s);
                nxt[j] = succ[cur[j].x + static_cast<int32_t>(__umulhi(r, static_cast<uint32_t>(cur[j].y)))];
            }
        }
#pragma unroll
        for (int j = 0; j < WPL; ++j) {
            const int32_t key = node_key(nxt[j]);
            if (live[j]) {
                bool seen = false;
#pragma unroll MAXD
                for (int i = 0; i <= s; ++i) seen |= path[j][i] == key;
                if (!seen) ++u[j];
                live[j] = !(cur[j].y <= 1 && key == path[j][s]);   // absorbed: stays put for good
            }
            path[j][s + 1] = key;
            cur[j] = nxt[j];
        }
    }
}

// One lane per (node, walk); with `patterns` the labels are written out.
template <int MAXD, bool UNROLL>
__global__ __launch_bounds__(256) void arw_kernel(const int32_t *__restrict__ rowptr,
                                                  const int32_t *__restrict__ col, int32_t n,
                                                  uint64_t seed, uint32_t k, uint32_t d,
                                                  int k_log2, uint32_t *__restrict__ S,
                                                  uint8_t *__restrict__ patterns,
                                                  const int32_t *__restrict__ bad_flag) {
    if (*bad_flag) return;  // the CSR failed validation: touch nothing
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t total = static_cast<int64_t>(n) * k;
    const bool valid = gid < total;
    uint32_t v = 0, w = 0, u = 0;
    if (valid) {
        if (k_log2 >= 0) {
            v = static_cast<uint32_t>(gid >> k_log2);
            w = static_cast<uint32_t>(gid & ((1 << k_log2) - 1));
        } else {
            v = static_cast<uint32_t>(gid / k);
            w = static_cast<uint32_t>(gid - static_cast<int64_t>(v) * k);
        }
        uint8_t *pat = patterns ? patterns + gid * (d + 1) : nullptr;
        u = walk_one<MAXD, UNROLL>(rowptr, col, v, w, d, seed, pat);
    }
    if (k_log2 >= 0 && k_log2 <= 6) {
        // the k lanes of a node are adjacent and aligned inside the wavefront
        for (int off = 1; off < (1 << k_log2); off <<= 1) u += __shfl_xor(u, off, 64);
        if (valid && w == 0) S[v] = u;
    } else if (valid) {
        atomicAdd(&S[v], u);
    }
}

// Density sums only, two walks per lane: lane p of node v (L = ceil(k / 2) adjacent
// lanes per node) runs walks 2p and 2p + 1, or only 2p when that is the node's last
// walk.  When L is a power of two up to 64 the lanes of a node are aligned inside the
// wavefront: their counts are summed with shuffles and stored once.  Otherwise the
// counts are summed per node inside the wavefront (a segmented scan) and the node's
// last lane in the wavefront adds the sum to S[v], which starts at zero.
template <int MAXD>
__global__ __launch_bounds__(256) void arw_sum_kernel(const int2 *__restrict__ nodeinfo,
                                                      const int32_t *__restrict__ col,
                                                      const int2 *__restrict__ succ,
                                                      int32_t n, uint64_t seed, uint32_t k,
                                                      uint32_t d, uint32_t L, int L_log2,
                                                      uint32_t *__restrict__ S,
                                                      const int32_t *__restrict__ bad_flag) {
    if (*bad_flag) return;
    const int64_t gid = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const bool valid = gid < static_cast<int64_t>(n) * L;
    int64_t v64, p;
    if (L_log2 >= 0) {
        v64 = gid >> L_log2;
        p = gid & ((static_cast<int64_t>(1) << L_log2) - 1);
    } else {
        v64 = gid / L;
        p = gid - v64 * L;
    }
    const uint32_t v = static_cast<uint32_t>(v64);
    const uint32_t w0 = static_cast<uint32_t>(p) * 2;
    uint32_t u = 0;
    if (valid) {
        const uint32_t nw = k - w0 >= 2 ? 2 : 1;
        uint32_t uj[2];
        if (succ)
            walk_lockstep_succ<MAXD, 2>(nodeinfo, succ, v, w0, nw, d, seed, uj);
        else
            walk_lockstep<MAXD, 2>(nodeinfo, col, v, w0, nw, d, seed, uj);
        u = uj[0] + uj[1];
    }
    if (L_log2 >= 0 && L_log2 <= 6) {
        for (int off = 1; off < (1 << L_log2); off <<= 1) u += __shfl_xor(u, off, 64);
        if (valid && p == 0) S[v] = u;
        return;
    }
    const int lane = static_cast<int>(threadIdx.x) & 63;
    const int first = lane - static_cast<int>(p < lane ? p : lane);   // node's first lane here
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(u, off, 64);
        if (lane - off >= first) u += t;
    }
    if (valid && (p == static_cast<int64_t>(L) - 1 || lane == 63)) atomicAdd(&S[v], u);
}

}  // namespace

int launch_density(const int2 *nodeinfo, const int32_t *col, const int2 *succ, int32_t n,
                   uint64_t seed, uint32_t k, uint32_t d, uint32_t *S, const int32_t *bad_flag,
                   hipStream_t stream) {
    if (d > 32 || k < 1) return DUALGCN_ERR_UNSUPPORTED;
    const uint32_t L = k / 2 + (k & 1);                 // lanes per node, two walks each
    int L_log2 = -1;
    if ((L & (L - 1)) == 0) {
        L_log2 = 0;
        while ((1u << L_log2) < L) ++L_log2;
    }
    const int64_t blocks = (static_cast<int64_t>(n) * L + 255) / 256;
    if (blocks > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    if (L_log2 < 0 || L_log2 > 6) {                     // summed with atomics
        const int st = hip_status(hipMemsetAsync(S, 0, sizeof(uint32_t) * static_cast<size_t>(n), stream));
        if (st) return st;
    }
    const dim3 grid(static_cast<unsigned>(blocks)), block(256);
    if (d <= 8)
        hipLaunchKernelGGL((arw_sum_kernel<8>), grid, block, 0, stream, nodeinfo, col, succ, n, seed,
                           k, d, L, L_log2, S, bad_flag);
    else
        hipLaunchKernelGGL((arw_sum_kernel<32>), grid, block, 0, stream, nodeinfo, col, succ, n,
                           seed, k, d, L, L_log2, S, bad_flag);
    return hip_status(hipGetLastError());
}

int launch_arw(const int32_t *rowptr, const int32_t *col, int32_t n, uint64_t seed, uint32_t k,
               uint32_t d, uint32_t *S, uint8_t *patterns, const int32_t *bad_flag,
               hipStream_t stream) {
    int k_log2 = -1;
    if ((k & (k - 1)) == 0) {
        k_log2 = 0;
        while ((1u << k_log2) < k) ++k_log2;
    }
    const bool shuffle_sum = k_log2 >= 0 && k_log2 <= 6;
    if (!shuffle_sum) {
        int st = hip_status(hipMemsetAsync(S, 0, sizeof(uint32_t) * static_cast<size_t>(n), stream));
        if (st) return st;
    }
    const int64_t total = static_cast<int64_t>(n) * k;
    const int64_t blocks = (total + 255) / 256;
    if (blocks > 0x7FFFFFFF) return DUALGCN_ERR_UNSUPPORTED;
    const dim3 grid(static_cast<unsigned>(blocks)), block(256);
    if (d <= 8)
        hipLaunchKernelGGL((arw_kernel<8, true>), grid, block, 0, stream, rowptr, col, n, seed, k,
                           d, k_log2, S, patterns, bad_flag);
    else if (d <= 32)
        hipLaunchKernelGGL((arw_kernel<32, true>), grid, block, 0, stream, rowptr, col, n, seed,
                           k, d, k_log2, S, patterns, bad_flag);
    else
        hipLaunchKernelGGL((arw_kernel<255, false>), grid, block, 0, stream, rowptr, col, n,
                           seed, k, d, k_log2, S, patterns, bad_flag);
    return hip_status(hipGetLastError());
}

}  // namespace dgc
