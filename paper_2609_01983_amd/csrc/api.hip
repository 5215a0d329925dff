// C ABI of libdualgcn: argument checks, status codes and dispatch to the kernels.
// Every check that needs no device runs before the device is touched.
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <new>
#include <vector>

#include "internal.h"

namespace dgc {

namespace {
thread_local int g_last_hip_error = 0;
}

int hip_status(hipError_t e) {
    if (e == hipSuccess) return DUALGCN_OK;
    g_last_hip_error = static_cast<int>(e);
    if (e == hipErrorOutOfMemory) return DUALGCN_ERR_OOM;
    if (e == hipErrorNoDevice || e == hipErrorInvalidDevice) return DUALGCN_ERR_NO_DEVICE;
    return DUALGCN_ERR_HIP;
}

int device_status() {
    int count = 0;
    const hipError_t e = hipGetDeviceCount(&count);
    if (e != hipSuccess || count <= 0) {
        if (e != hipSuccess) g_last_hip_error = static_cast<int>(e);
        return DUALGCN_ERR_NO_DEVICE;
    }
    return DUALGCN_OK;
}

int device_cus() {
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cached[kMaxDevices];    // zero-initialised: not queried yet
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    const bool slot = dev >= 0 && dev < kMaxDevices;
    if (slot) {
        const int c = cached[dev].load(std::memory_order_relaxed);
        if (c > 0) return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    if (slot) cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

// Allocation-failure injection for tests: while DUALGCN_TEST_FAIL_ALLOC holds N > 0 (any
// text may follow the number), the N-th device allocation request counted from the
// moment the variable took its current text fails with DUALGCN_ERR_OOM (once) before HIP
// is called.
bool injected_failure() {
    static std::mutex mu;
    static std::string last;
    static long count = 0;
    const char *e = std::getenv("DUALGCN_TEST_FAIL_ALLOC");
    const std::string cur = e ? e : "";
    std::lock_guard<std::mutex> lock(mu);
    if (cur != last) {
        last = cur;
        count = 0;
    }
    const long target = cur.empty() ? 0 : std::atol(cur.c_str());
    return target > 0 && ++count == target;
}

int alloc_bytes(void **p, size_t bytes) {
    *p = nullptr;
    if (injected_failure()) return DUALGCN_ERR_OOM;
    const hipError_t e = hipMalloc(p, bytes ? bytes : 1);
    if (e != hipSuccess) {
        *p = nullptr;
        g_last_hip_error = static_cast<int>(e);
        return e == hipErrorOutOfMemory ? DUALGCN_ERR_OOM : DUALGCN_ERR_HIP;
    }
    return DUALGCN_OK;
}

// ---- cached device blocks
//
// A plan takes one large block and its build one scratch block.  Released blocks are
// kept (per device, at most kCachedBlocks) and handed out again to a request of at
// most their size and at least half of it, so that rebuilding a plan of the same
// matrix does not pay hipMalloc and hipFree of gigabytes every time.  The cache holds
// its blocks until the process ends; a failed hipMalloc first returns the device's
// cached blocks to HIP and tries again.
namespace {
struct CachedBlock {
    int device;
    size_t bytes;
    void *ptr;
};
std::mutex g_cache_mu;
std::vector<CachedBlock> g_cache;
constexpr size_t kCachedBlocks = 4;
}  // namespace

int alloc_block(void **p, size_t *capacity, size_t bytes) {
    *p = nullptr;
    *capacity = 0;
    if (injected_failure()) return DUALGCN_ERR_OOM;
    if (bytes == 0) bytes = 1;
    int dev = 0;
    int st = hip_status(hipGetDevice(&dev));
    if (st) return st;
    {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        size_t best = g_cache.size();
        for (size_t i = 0; i < g_cache.size(); ++i) {
            const CachedBlock &b = g_cache[i];
            if (b.device == dev && b.bytes >= bytes && b.bytes / 2 <= bytes &&
                (best == g_cache.size() || b.bytes < g_cache[best].bytes))
                best = i;
        }
        if (best < g_cache.size()) {
            *p = g_cache[best].ptr;
            *capacity = g_cache[best].bytes;
            g_cache.erase(g_cache.begin() + static_cast<std::ptrdiff_t>(best));
            return DUALGCN_OK;
        }
    }
    hipError_t e = hipMalloc(p, bytes);
    if (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        std::vector<void *> drop;
        {
            std::lock_guard<std::mutex> lock(g_cache_mu);
            for (size_t i = g_cache.size(); i-- > 0;) {
                if (g_cache[i].device == dev) {
                    drop.push_back(g_cache[i].ptr);
                    g_cache.erase(g_cache.begin() + static_cast<std::ptrdiff_t>(i));
                }
            }
        }
        for (void *q : drop) (void)hipFree(q);
        e = hipMalloc(p, bytes);
    }
    if (e != hipSuccess) {
        *p = nullptr;
        g_last_hip_error = static_cast<int>(e);
        return e == hipErrorOutOfMemory ? DUALGCN_ERR_OOM : DUALGCN_ERR_HIP;
    }
    *capacity = bytes;
    return DUALGCN_OK;
}

void release_block(void *p, size_t capacity) {
    if (!p) return;
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess) {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        if (g_cache.size() < kCachedBlocks) {
            g_cache.push_back(CachedBlock{dev, capacity, p});
            return;
        }
    }
    (void)hipFree(p);
}

}  // namespace dgc

using dgc::Plan;

namespace {

constexpr uint32_t kMaxRational = 1u << 16;
// Largest number of entries: 32-bit entry offsets keep some headroom for the
// kernels' round arithmetic.
constexpr int64_t kMaxNnz = (static_cast<int64_t>(1) << 31) - (1 << 16);

int check_csr(const dualgcn_csr *c) {
    if (!c || !c->rowptr) return DUALGCN_ERR_INVALID_ARG;
    if (c->n < 1) return DUALGCN_ERR_INVALID_ARG;
    if (c->nnz < 0) return DUALGCN_ERR_INVALID_ARG;
    if (c->nnz > kMaxNnz) return DUALGCN_ERR_UNSUPPORTED;
    if (c->nnz > 0 && (!c->col || !c->val)) return DUALGCN_ERR_INVALID_ARG;
    return DUALGCN_OK;
}

int check_walks(uint32_t k, uint32_t d) {
    if (k < 1 || d < 1) return DUALGCN_ERR_INVALID_ARG;
    if (d > 255) return DUALGCN_ERR_UNSUPPORTED;
    // S_v <= k (d + 1) is held in 32 bits
    if (static_cast<uint64_t>(k) * (static_cast<uint64_t>(d) + 1) >= (static_cast<uint64_t>(1) << 32))
        return DUALGCN_ERR_UNSUPPORTED;
    return DUALGCN_OK;
}

// q k max(d + 1, nnz) < 2^63 keeps every key K_v = p S_v + (q - p) k D_v in 63 bits.
bool keys_fit(uint32_t q, uint32_t k, uint32_t d, int64_t nnz) {
    const dgc::u128 m = static_cast<dgc::u128>(q) * k *
                        static_cast<dgc::u128>(nnz > static_cast<int64_t>(d) + 1 ? nnz : d + 1);
    return m < (static_cast<dgc::u128>(1) << 63);
}

// Thresholds of a partition: rationals below 2^16 with non-zero denominators, alpha <= 1
// (or an adaptive marker when `adaptive_ok`), a known force mode.
int check_thresholds(const dualgcn_thresholds &t, bool adaptive_ok) {
    if (t.alpha_den == 0 || t.beta_den == 0) return DUALGCN_ERR_INVALID_ARG;
    if (t.alpha_num > t.alpha_den &&
        !(adaptive_ok && (t.alpha_num == DUALGCN_ALPHA_ADAPTIVE || t.alpha_num == DUALGCN_ALPHA_BALANCED)))
        return DUALGCN_ERR_INVALID_ARG;
    if (t.alpha_den >= kMaxRational || t.beta_den >= kMaxRational || t.beta_num >= kMaxRational)
        return DUALGCN_ERR_INVALID_ARG;
    if (t.force_mode < DUALGCN_FORCE_AUTO || t.force_mode > DUALGCN_FORCE_DENSE)
        return DUALGCN_ERR_INVALID_ARG;
    return DUALGCN_OK;
}

int check_plan(const dualgcn_plan *plan) {
    return plan ? DUALGCN_OK : DUALGCN_ERR_INVALID_ARG;
}

const Plan *as_plan(const dualgcn_plan *p) { return reinterpret_cast<const Plan *>(p); }

// Do [a, a + abytes) and [b, b + bbytes) share a byte?
bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes) {
    const char *x = static_cast<const char *>(a);
    const char *y = static_cast<const char *>(b);
    return x < y + bbytes && y < x + abytes;
}

// Shapes of the update phase T = X W handled by the matrix-core kernel.
int check_update(const void *X, const float *W, const void *T, int32_t F_in, int32_t F_out) {
    if (!X || !W || !T || F_in < 1 || F_out < 1) return DUALGCN_ERR_INVALID_ARG;
    if (F_in % 32 || F_out % 32 || F_in > 1024 || F_out > 256) return DUALGCN_ERR_UNSUPPORTED;
    if (reinterpret_cast<uintptr_t>(X) % 16) return DUALGCN_ERR_INVALID_ARG;
    return DUALGCN_OK;
}

}  // namespace

extern "C" {

const char *dualgcn_status_str(int status) {
    switch (status) {
        case DUALGCN_OK: return "ok";
        case DUALGCN_ERR_INVALID_ARG: return "invalid argument";
        case DUALGCN_ERR_BAD_CSR: return "malformed CSR matrix";
        case DUALGCN_ERR_UNSUPPORTED: return "unsupported size or parameter";
        case DUALGCN_ERR_OOM: return "device out of memory";
        case DUALGCN_ERR_HIP: return "HIP runtime error";
        case DUALGCN_ERR_NO_DEVICE: return "no HIP device";
        default: return "unknown status";
    }
}

int dualgcn_last_hip_error(void) { return dgc::g_last_hip_error; }

int dualgcn_partition(const dualgcn_csr *csr, uint64_t seed, uint32_t walks_per_node,
                      uint32_t walk_len, const dualgcn_thresholds *th, void *stream,
                      dualgcn_plan **out) {
    dgc::TraceRange trace("dualgcn_partition");
    if (!out) return DUALGCN_ERR_INVALID_ARG;
    *out = nullptr;
    int st = check_csr(csr);
    if (st) return st;
    if ((st = check_walks(walks_per_node, walk_len))) return st;
    dualgcn_thresholds t{1, 2, 1, 2, DUALGCN_FORCE_AUTO};
    if (th) t = *th;
    if ((st = check_thresholds(t, true))) return st;
    if (!keys_fit(t.alpha_den, walks_per_node, walk_len, csr->nnz)) return DUALGCN_ERR_UNSUPPORTED;
    if ((st = dgc::device_status())) return st;
    Plan *p = nullptr;
    st = dgc::build_plan(csr, seed, walks_per_node, walk_len, t, nullptr,
                         static_cast<hipStream_t>(stream), &p);
    if (st) return st;
    *out = reinterpret_cast<dualgcn_plan *>(p);
    return DUALGCN_OK;
}

void dualgcn_plan_destroy(dualgcn_plan *plan) {
    if (!plan) return;
    Plan *p = reinterpret_cast<Plan *>(plan);
    // the plan's own build and every launch that used it; on a failed wait (a device
    // error), wait for the whole device before the memory can be handed out again
    if (dgc::wait_plan_idle(*p)) (void)hipDeviceSynchronize();
    dgc::free_plan(p);
}

int dualgcn_spmm(const dualgcn_plan *plan, const float *X, float *Y, int32_t F, void *stream) {
    return dualgcn_spmm_act(plan, X, Y, F, 0u, stream);
}

int dualgcn_spmm_act(const dualgcn_plan *plan, const float *X, void *Y, int32_t F,
                     uint32_t flags, void *stream) {
    dgc::TraceRange trace("dualgcn_spmm");
    int st = check_plan(plan);
    if (st) return st;
    if (!X || !Y || F < 1) return DUALGCN_ERR_INVALID_ARG;
    if (flags & ~(DUALGCN_RELU | DUALGCN_OUT_BF16)) return DUALGCN_ERR_INVALID_ARG;
    if (F >= (1 << 20)) return DUALGCN_ERR_UNSUPPORTED;
    const Plan *p = as_plan(plan);
    const bool bf = (flags & DUALGCN_OUT_BF16) != 0;
    const size_t elems = static_cast<size_t>(p->n) * F;
    if (overlaps(X, elems * sizeof(float), Y, elems * (bf ? 2 : 4))) return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_spmm(*p, X, Y, F, (flags & DUALGCN_RELU) != 0, bf,
                            static_cast<hipStream_t>(stream));
}

int dualgcn_spmm_update(const dualgcn_plan *plan, const float *X, const float *W, float *T,
                        void *H, int32_t F_in, int32_t F_out, uint32_t flags, void *stream) {
    dgc::TraceRange trace("dualgcn_spmm_update");
    int st = check_plan(plan);
    if (st) return st;
    if (!X || !W || !T || F_in < 1 || F_out < 1) return DUALGCN_ERR_INVALID_ARG;
    if (flags & ~DUALGCN_RELU) return DUALGCN_ERR_INVALID_ARG;
    if (F_in % 32 || F_out % 32 || F_in > 256 || F_out > 256 ||
        dgc::spmm_xw_lds_bytes(F_in, F_out) > 160 * 1024)
        return DUALGCN_ERR_UNSUPPORTED;
    if (reinterpret_cast<uintptr_t>(X) % 16 || reinterpret_cast<uintptr_t>(T) % 16)
        return DUALGCN_ERR_INVALID_ARG;
    const Plan *p = as_plan(plan);
    const size_t n = static_cast<size_t>(p->n);
    const size_t tbytes = n * F_out * sizeof(float);
    const size_t xbytes = n * F_in * sizeof(float), wbytes = static_cast<size_t>(F_in) * F_out * sizeof(float);
    if (overlaps(X, xbytes, T, tbytes) || overlaps(W, wbytes, T, tbytes))
        return DUALGCN_ERR_INVALID_ARG;
    if (H) {
        const size_t hbytes = n * F_in * sizeof(uint16_t);
        if (reinterpret_cast<uintptr_t>(H) % 8 || overlaps(H, hbytes, X, xbytes) ||
            overlaps(H, hbytes, W, wbytes) || overlaps(H, hbytes, T, tbytes))
            return DUALGCN_ERR_INVALID_ARG;
    }
    if ((st = dgc::device_status())) return st;
    const bool relu = (flags & DUALGCN_RELU) != 0;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    if (H && reinterpret_cast<uintptr_t>(H) % 16 == 0 && !dgc::fused_junction_pays(*p, F_in, F_out)) {
        // the two calls are faster here, and H holds their intermediate: the same bits
        if ((st = dgc::launch_spmm(*p, X, H, F_in, relu, true, s))) return st;
        return dgc::launch_xw(H, true, W, T, p->n, F_in, F_out, s);
    }
    return dgc::launch_spmm_xw(*p, X, W, T, H, F_in, F_out, relu, s);
}

int dualgcn_spmm_update_route(const dualgcn_plan *plan, int32_t F_in, int32_t F_out,
                              int32_t *fused) {
    int st = check_plan(plan);
    if (st) return st;
    if (!fused || F_in < 1 || F_out < 1) return DUALGCN_ERR_INVALID_ARG;
    if (F_in % 32 || F_out % 32 || F_in > 256 || F_out > 256 ||
        dgc::spmm_xw_lds_bytes(F_in, F_out) > 160 * 1024)
        return DUALGCN_ERR_UNSUPPORTED;
    *fused = dgc::fused_junction_pays(*as_plan(plan), F_in, F_out) ? 1 : 0;
    return DUALGCN_OK;
}

int dualgcn_update(const void *X, const float *W, float *T, int32_t n, int32_t F_in,
                   int32_t F_out, uint32_t flags, void *stream) {
    dgc::TraceRange trace("dualgcn_update");
    if (n < 1) return DUALGCN_ERR_INVALID_ARG;
    int st = check_update(X, W, T, F_in, F_out);
    if (st) return st;
    if (flags & ~DUALGCN_IN_BF16) return DUALGCN_ERR_INVALID_ARG;
    const bool bf = (flags & DUALGCN_IN_BF16) != 0;
    const size_t un = static_cast<size_t>(n);
    if (overlaps(X, un * F_in * (bf ? 2 : 4), T, un * F_out * sizeof(float)))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_xw(X, bf, W, T, n, F_in, F_out, static_cast<hipStream_t>(stream));
}

int dualgcn_gcn_layer_workspace(const dualgcn_plan *plan, int32_t F_in, int32_t F_out,
                                size_t *bytes) {
    int st = check_plan(plan);
    if (st) return st;
    if (!bytes || F_in < 1 || F_out < 1) return DUALGCN_ERR_INVALID_ARG;
    *bytes = dgc::xw_workspace_bytes(as_plan(plan)->n, F_out);
    return DUALGCN_OK;
}

int dualgcn_gcn_layer(const dualgcn_plan *plan, const void *X, const float *W, void *Y,
                      int32_t F_in, int32_t F_out, uint32_t flags, void *workspace,
                      size_t workspace_bytes, void *stream) {
    dgc::TraceRange trace("dualgcn_gcn_layer");
    int st = check_plan(plan);
    if (st) return st;
    if (!Y || !workspace) return DUALGCN_ERR_INVALID_ARG;
    if ((st = check_update(X, W, Y, F_in, F_out))) return st;
    if (flags & ~(DUALGCN_RELU | DUALGCN_IN_BF16 | DUALGCN_OUT_BF16)) return DUALGCN_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(workspace) % 256) return DUALGCN_ERR_INVALID_ARG;
    const Plan *p = as_plan(plan);
    const size_t ws = dgc::xw_workspace_bytes(p->n, F_out);
    if (workspace_bytes < ws) return DUALGCN_ERR_INVALID_ARG;
    const size_t n = static_cast<size_t>(p->n);
    const bool in_bf = (flags & DUALGCN_IN_BF16) != 0, out_bf = (flags & DUALGCN_OUT_BF16) != 0;
    if (overlaps(X, n * F_in * (in_bf ? 2 : 4), workspace, ws) ||
        overlaps(Y, n * F_out * (out_bf ? 2 : 4), workspace, ws))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_gcn_layer(*p, X, in_bf, W, Y, out_bf, F_in, F_out,
                                 (flags & DUALGCN_RELU) != 0, workspace,
                                 static_cast<hipStream_t>(stream));
}

int dualgcn_softmax_xent(const float *Y, const int32_t *labels, int32_t n, int32_t C,
                         float scale, float *G, double *loss, void *stream) {
    dgc::TraceRange trace("dualgcn_softmax_xent");
    if (!Y || !labels || !G || !loss || n < 1 || C < 1) return DUALGCN_ERR_INVALID_ARG;
    if (C >= (1 << 20)) return DUALGCN_ERR_UNSUPPORTED;
    const size_t elems = static_cast<size_t>(n) * C;
    const size_t lbytes = sizeof(double) * DUALGCN_LOSS_SLOTS;
    if (overlaps(Y, elems * sizeof(float), G, elems * sizeof(float)) ||
        overlaps(loss, lbytes, Y, elems * sizeof(float)) ||
        overlaps(loss, lbytes, G, elems * sizeof(float)) ||
        overlaps(loss, lbytes, labels, sizeof(int32_t) * n) ||
        overlaps(G, elems * sizeof(float), labels, sizeof(int32_t) * n))
        return DUALGCN_ERR_INVALID_ARG;
    int st = dgc::device_status();
    if (st) return st;
    return dgc::launch_softmax_xent(Y, labels, n, C, scale, G, loss, static_cast<hipStream_t>(stream));
}

int dualgcn_weight_grad_workspace(int32_t n, int32_t F_in, int32_t F_out, size_t *bytes) {
    if (!bytes || n < 1 || F_in < 1 || F_out < 1) return DUALGCN_ERR_INVALID_ARG;
    *bytes = dgc::wgrad_workspace_bytes(n, F_in, F_out);
    return DUALGCN_OK;
}

int dualgcn_weight_grad(const void *X, const void *G, float *dW, int32_t n, int32_t F_in,
                        int32_t F_out, uint32_t flags, float lr, float *W, void *workspace,
                        size_t workspace_bytes, void *stream) {
    dgc::TraceRange trace("dualgcn_weight_grad");
    if (!G || !dW || !workspace || n < 1) return DUALGCN_ERR_INVALID_ARG;
    int st = check_update(X, W ? W : dW, dW, F_in, F_out);
    if (st) return st;
    if (flags & ~(DUALGCN_IN_BF16 | DUALGCN_GRAD_BF16)) return DUALGCN_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(G) % 16 || reinterpret_cast<uintptr_t>(workspace) % 256)
        return DUALGCN_ERR_INVALID_ARG;
    const size_t ws = dgc::wgrad_workspace_bytes(n, F_in, F_out);
    if (workspace_bytes < ws) return DUALGCN_ERR_INVALID_ARG;
    const bool xbf = (flags & DUALGCN_IN_BF16) != 0, gbf = (flags & DUALGCN_GRAD_BF16) != 0;
    const size_t un = static_cast<size_t>(n);
    const size_t xb = un * F_in * (xbf ? 2 : 4), gb = un * F_out * (gbf ? 2 : 4);
    const size_t wb = static_cast<size_t>(F_in) * F_out * sizeof(float);
    if (overlaps(dW, wb, X, xb) || overlaps(dW, wb, G, gb) || overlaps(dW, wb, workspace, ws) ||
        overlaps(workspace, ws, X, xb) || overlaps(workspace, ws, G, gb))
        return DUALGCN_ERR_INVALID_ARG;
    if (W && (overlaps(W, wb, X, xb) || overlaps(W, wb, G, gb) || overlaps(W, wb, dW, wb) ||
              overlaps(W, wb, workspace, ws)))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_weight_grad(X, xbf, G, gbf, dW, n, F_in, F_out, lr, W, workspace,
                                   static_cast<hipStream_t>(stream));
}

int dualgcn_weight_grad_noalloc(const void *X, const void *G, float *dW, int32_t n, int32_t F_in,
                                int32_t F_out, uint32_t flags, float lr, float *W, void *stream) {
    dgc::TraceRange trace("dualgcn_weight_grad_noalloc");
    if (!G || !dW || n < 1) return DUALGCN_ERR_INVALID_ARG;
    int st = check_update(X, W ? W : dW, dW, F_in, F_out);
    if (st) return st;
    if (flags & ~(DUALGCN_IN_BF16 | DUALGCN_GRAD_BF16)) return DUALGCN_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(G) % 16) return DUALGCN_ERR_INVALID_ARG;
    const bool xbf = (flags & DUALGCN_IN_BF16) != 0, gbf = (flags & DUALGCN_GRAD_BF16) != 0;
    const size_t un = static_cast<size_t>(n);
    const size_t xb = un * F_in * (xbf ? 2 : 4), gb = un * F_out * (gbf ? 2 : 4);
    const size_t wb = static_cast<size_t>(F_in) * F_out * sizeof(float);
    if (overlaps(dW, wb, X, xb) || overlaps(dW, wb, G, gb)) return DUALGCN_ERR_INVALID_ARG;
    if (W && (overlaps(W, wb, X, xb) || overlaps(W, wb, G, gb) || overlaps(W, wb, dW, wb)))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_weight_grad_noalloc(X, xbf, G, gbf, dW, n, F_in, F_out, lr, W,
                                           static_cast<hipStream_t>(stream));
}

int dualgcn_backward_data(const void *G, const float *W, const void *M, float *dX, int32_t n,
                          int32_t F_in, int32_t F_out, uint32_t flags, void *stream) {
    dgc::TraceRange trace("dualgcn_backward_data");
    if (!G || n < 1) return DUALGCN_ERR_INVALID_ARG;
    int st = check_update(G, W, dX, F_in, F_out);
    if (st) return st;
    if (flags & ~(DUALGCN_IN_BF16 | DUALGCN_GRAD_BF16)) return DUALGCN_ERR_INVALID_ARG;
    const bool mbf = (flags & DUALGCN_IN_BF16) != 0, gbf = (flags & DUALGCN_GRAD_BF16) != 0;
    const size_t un = static_cast<size_t>(n);
    const size_t xb = un * F_in * sizeof(float);
    if (overlaps(dX, xb, G, un * F_out * (gbf ? 2 : 4))) return DUALGCN_ERR_INVALID_ARG;
    if (M && overlaps(dX, xb, M, un * F_in * (mbf ? 2 : 4))) return DUALGCN_ERR_INVALID_ARG;
    if (M && (reinterpret_cast<uintptr_t>(M) % 16 || reinterpret_cast<uintptr_t>(dX) % 16))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    return dgc::launch_backward_data(G, gbf, W, M, mbf, dX, n, F_in, F_out,
                                     static_cast<hipStream_t>(stream));
}

int dualgcn_plan_query(const dualgcn_plan *plan, dualgcn_plan_info *out) {
    int st = check_plan(plan);
    if (st) return st;
    if (!out) return DUALGCN_ERR_INVALID_ARG;
    const Plan *p = as_plan(plan);
    dualgcn_plan_info i{};
    i.n = p->n;
    i.nnz = p->nnz;
    i.n_sparse = p->n_sparse;
    i.n_dense = p->n - p->n_sparse;
    i.kstar = p->kstar;
    i.s1_hi = static_cast<uint64_t>(p->s1 >> 64);
    i.s1_lo = static_cast<uint64_t>(p->s1);
    i.s2_hi = static_cast<uint64_t>(p->s2 >> 64);
    i.s2_lo = static_cast<uint64_t>(p->s2);
    i.kmax = p->kmax;
    i.alpha_num = p->th.alpha_num;
    i.alpha_den = p->th.alpha_den;
    i.beta_num = p->th.beta_num;
    i.beta_den = p->th.beta_den;
    i.force_mode = p->th.force_mode;
    i.seed = p->seed;
    i.walks_per_node = p->k;
    i.walk_len = p->d;
    i.max_degree = p->max_degree;
    i.dense_chunk = p->dense_chunk;
    i.n_split_rows = p->n_split_rows;
    i.n_split_parts = p->n_split_parts;
    i.n_tasks = p->n_tasks;
    i.n_long_rows = p->n_long[0];
    i.cold_marked = p->cold_marked ? 1 : 0;
    *out = i;
    return DUALGCN_OK;
}

int dualgcn_plan_export(const dualgcn_plan *plan, int32_t *perm_h, uint32_t *S_h, uint64_t *K_h) {
    int st = check_plan(plan);
    if (st) return st;
    if ((st = dgc::device_status())) return st;
    const Plan *p = as_plan(plan);
    const size_t n = static_cast<size_t>(p->n);
    if ((st = dgc::hip_status(hipDeviceSynchronize()))) return st;
    if (perm_h && (st = dgc::hip_status(hipMemcpy(perm_h, p->perm, n * 4, hipMemcpyDeviceToHost))))
        return st;
    if (S_h && (st = dgc::hip_status(hipMemcpy(S_h, p->S, n * 4, hipMemcpyDeviceToHost)))) return st;
    if (K_h && (st = dgc::hip_status(hipMemcpy(K_h, p->K, n * 8, hipMemcpyDeviceToHost)))) return st;
    return DUALGCN_OK;
}

int dualgcn_arw_patterns(const dualgcn_csr *csr, uint64_t seed, uint32_t walks_per_node,
                         uint32_t walk_len, uint8_t *out, void *stream) {
    dgc::TraceRange trace("dualgcn_arw_patterns");
    int st = check_csr(csr);
    if (st) return st;
    if ((st = check_walks(walks_per_node, walk_len))) return st;
    if (!out) return DUALGCN_ERR_INVALID_ARG;
    const dgc::u128 total = static_cast<dgc::u128>(csr->n) * walks_per_node * (walk_len + 1);
    if (total >= (static_cast<dgc::u128>(1) << 40)) return DUALGCN_ERR_UNSUPPORTED;
    if ((st = dgc::device_status())) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *scratch = nullptr;   // [n] sums + 2 validation words
    if ((st = dgc::alloc_bytes(&scratch, sizeof(uint32_t) * (static_cast<size_t>(csr->n) + 2))))
        return st;
    uint32_t *S = static_cast<uint32_t *>(scratch);
    int32_t *flags = reinterpret_cast<int32_t *>(S + csr->n);
    st = dgc::hip_status(hipMemsetAsync(flags, 0, 2 * sizeof(int32_t), s));
    if (!st) st = dgc::validate_csr(csr, flags, nullptr, nullptr, nullptr, s);
    if (!st)
        st = dgc::launch_arw(csr->rowptr, csr->col, csr->n, seed, walks_per_node, walk_len, S, out,
                             flags, s);
    int32_t bad = 0;
    if (!st) st = dgc::hip_status(hipMemcpyAsync(&bad, flags, sizeof(bad), hipMemcpyDeviceToHost, s));
    if (!st) st = dgc::hip_status(hipStreamSynchronize(s));
    (void)hipFree(scratch);
    if (!st && bad) st = DUALGCN_ERR_BAD_CSR;
    return st;
}

// Saved plans: this header, then the n density sums S (uint32).
struct PlanFileHeader {
    char magic[8];
    uint32_t version;
    uint32_t header_bytes;
    int32_t n;
    int32_t reserved;
    int64_t nnz;
    uint64_t seed;
    uint32_t k, d;
    dualgcn_thresholds th;
    int32_t reserved2;
    uint64_t checksum;
};
constexpr char kPlanMagic[8] = {'D', 'G', 'C', 'N', 'P', 'L', 'A', 'N'};
constexpr uint32_t kPlanVersion = 1;

int dualgcn_plan_save(const dualgcn_plan *plan, void *buf, size_t *bytes) {
    dgc::TraceRange trace("dualgcn_plan_save");
    int st = check_plan(plan);
    if (st) return st;
    if (!bytes) return DUALGCN_ERR_INVALID_ARG;
    const Plan *p = as_plan(plan);
    const size_t need = sizeof(PlanFileHeader) + sizeof(uint32_t) * static_cast<size_t>(p->n);
    if (!buf) {
        *bytes = need;
        return DUALGCN_OK;
    }
    if (*bytes < need) {
        *bytes = need;
        return DUALGCN_ERR_INVALID_ARG;
    }
    PlanFileHeader h{};
    std::memcpy(h.magic, kPlanMagic, sizeof(h.magic));
    h.version = kPlanVersion;
    h.header_bytes = sizeof(PlanFileHeader);
    h.n = p->n;
    h.nnz = p->nnz;
    h.seed = p->seed;
    h.k = p->k;
    h.d = p->d;
    h.th = p->th;               // with an adaptive alpha: the weight it chose
    if ((st = dgc::structure_checksum(p->rowptr, p->col, p->n, p->nnz, nullptr, &h.checksum)))
        return st;
    std::memcpy(buf, &h, sizeof(h));
    if ((st = dgc::hip_status(hipMemcpy(static_cast<char *>(buf) + sizeof(h), p->S,
                                        sizeof(uint32_t) * static_cast<size_t>(p->n),
                                        hipMemcpyDeviceToHost))))
        return st;
    *bytes = need;
    return DUALGCN_OK;
}

int dualgcn_plan_load(const dualgcn_csr *csr, const void *buf, size_t bytes, void *stream,
                      dualgcn_plan **out) {
    dgc::TraceRange trace("dualgcn_plan_load");
    if (!out) return DUALGCN_ERR_INVALID_ARG;
    *out = nullptr;
    int st = check_csr(csr);
    if (st) return st;
    if (!buf || bytes < sizeof(PlanFileHeader)) return DUALGCN_ERR_INVALID_ARG;
    PlanFileHeader h;
    std::memcpy(&h, buf, sizeof(h));
    if (std::memcmp(h.magic, kPlanMagic, sizeof(h.magic)) || h.version != kPlanVersion ||
        h.header_bytes != sizeof(PlanFileHeader))
        return DUALGCN_ERR_INVALID_ARG;
    if (h.n != csr->n || h.nnz != csr->nnz ||
        bytes != sizeof(PlanFileHeader) + sizeof(uint32_t) * static_cast<size_t>(h.n))
        return DUALGCN_ERR_INVALID_ARG;
    const dualgcn_thresholds &t = h.th;
    if ((st = check_walks(h.k, h.d))) return st;
    if ((st = check_thresholds(t, false))) return st;     // a saved plan holds a resolved alpha
    if (!keys_fit(t.alpha_den, h.k, h.d, csr->nnz)) return DUALGCN_ERR_UNSUPPORTED;
    if ((st = dgc::device_status())) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint64_t sum = 0;
    if ((st = dgc::structure_checksum(csr->rowptr, csr->col, csr->n, csr->nnz, s, &sum))) return st;
    if (sum != h.checksum) return DUALGCN_ERR_INVALID_ARG;
    const uint32_t *S = reinterpret_cast<const uint32_t *>(static_cast<const char *>(buf) + sizeof(h));
    Plan *p = nullptr;
    if ((st = dgc::build_plan(csr, h.seed, h.k, h.d, t, S, s, &p))) return st;
    *out = reinterpret_cast<dualgcn_plan *>(p);
    return DUALGCN_OK;
}

int dualgcn_aggregator_values(const dualgcn_csr *csr, int32_t kind, float eps, float *val,
                              void *stream) {
    dgc::TraceRange trace("dualgcn_aggregator_values");
    int st = check_csr(csr);
    if (st) return st;
    if (!val || kind < DUALGCN_AGG_GCN || kind > DUALGCN_AGG_SUM) return DUALGCN_ERR_INVALID_ARG;
    if (overlaps(val, sizeof(float) * static_cast<size_t>(csr->nnz), csr->rowptr,
                 sizeof(int32_t) * (static_cast<size_t>(csr->n) + 1)) ||
        (csr->nnz > 0 && overlaps(val, sizeof(float) * static_cast<size_t>(csr->nnz), csr->col,
                                  sizeof(int32_t) * static_cast<size_t>(csr->nnz))))
        return DUALGCN_ERR_INVALID_ARG;
    if ((st = dgc::device_status())) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *scratch = nullptr;   // 2 validation words
    if ((st = dgc::alloc_bytes(&scratch, 2 * sizeof(int32_t)))) return st;
    int32_t *flags = static_cast<int32_t *>(scratch);
    st = dgc::hip_status(hipMemsetAsync(flags, 0, 2 * sizeof(int32_t), s));
    if (!st) st = dgc::validate_csr(csr, flags, nullptr, nullptr, nullptr, s);
    if (!st) st = dgc::launch_aggregator_values(csr, kind, eps, val, s);
    int32_t bad = 0;
    if (!st) st = dgc::hip_status(hipMemcpyAsync(&bad, flags, sizeof(bad), hipMemcpyDeviceToHost, s));
    if (!st) st = dgc::hip_status(hipStreamSynchronize(s));
    (void)hipFree(scratch);
    if (!st && bad) st = DUALGCN_ERR_BAD_CSR;
    return st;
}

}  // extern "C"

int dualgcn_bandwidth_probe(int32_t kind, const void *src, void *dst, size_t bytes, void *stream) {
    dgc::TraceRange trace("dualgcn_bandwidth_probe");
    if (!src || !dst || bytes == 0 || bytes % 16 || reinterpret_cast<uintptr_t>(src) % 16 ||
        reinterpret_cast<uintptr_t>(dst) % 16)
        return DUALGCN_ERR_INVALID_ARG;
    if (kind != DUALGCN_PROBE_COPY && kind != DUALGCN_PROBE_READ) return DUALGCN_ERR_INVALID_ARG;
    if (kind == DUALGCN_PROBE_COPY && overlaps(src, bytes, dst, bytes)) return DUALGCN_ERR_INVALID_ARG;
    const int st = dgc::device_status();
    if (st) return st;
    return dgc::launch_bandwidth_probe(kind, src, dst, bytes, static_cast<hipStream_t>(stream));
}

int32_t dualgcn_bandwidth_probe_out_floats(void) { return dgc::kMaxProbeGrid; }
