// Parameter update of the training step: SGD whose step is scaled down when
// the L2 norm over all gradients of the step exceeds a threshold.
//
// JANUS inserts the update into the generated graph after the operations of
// automatic differentiation (Section 3.1).  The paper names no optimizer; the
// rule used is plain SGD, p <- p - lr s g, with the clipping coefficient
// s = min(1, max_norm / (norm + 1e-6)), s = 1 when clipping is off.  Model
// state changes all-or-nothing (Section 4.2.3): a non-finite norm leaves
// every parameter as it was.
//
// Three launches, each bound by HBM traffic:
//   sgd_sumsq_kernel   block b of kSgdBlocks sums g^2 (in float64) over its
//                      range of the concatenation of the tensors;
//   sgd_scale_kernel   one block adds the block sums in block order and forms
//                      the norm, lr s and the skip flag;
//   sgd_update_kernel  p <- p - (lr s) g over the same ranges.
// Every sum runs in a fixed order, so the norm does not depend on timing.
#include <algorithm>
#include <cmath>
#include <mutex>

#include "device.hpp"
#include "runtime.hpp"

namespace janus {
namespace {

constexpr int kSgdThreads = 256;
constexpr int kSgdBlocks = 1024;
constexpr int kSgdTable = 64;   // tensors per launch

// Up to kSgdTable tensors of one launch, passed by value.
struct SgdTable {
    int n;
    int64_t off[kSgdTable + 1];   // element offsets of the tensors in their concatenation
    const float* g[kSgdTable];
    void* p[kSgdTable];
};

struct SgdCtrl {
    float ls;        // lr * s (0 when skipped)
    int skip;        // 1: the norm is not finite, nothing changes
    int pad[62];
};

// [lo, hi) of the concatenation for block b of nb
__device__ __forceinline__ void block_range(int64_t total, int b, int nb, int64_t& lo, int64_t& hi) {
    const int64_t base = total / nb, rem = total % nb;
    lo = int64_t(b) * base + (b < rem ? b : rem);
    hi = lo + base + (b < rem ? 1 : 0);
}

// fixed-order sum of one double per thread of the block; thread 0 gets it
__device__ __forceinline__ double block_sum(double v, double* red) {
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    double s = 0.0;
    if (threadIdx.x == 0)
        for (int w = 0; w < kSgdThreads / 64; ++w) s += red[w];
    return s;
}

__global__ __launch_bounds__(kSgdThreads) void sgd_sumsq_kernel(SgdTable t, double* partial) {
    __shared__ double red[kSgdThreads / 64];
    const int tid = threadIdx.x;
    int64_t lo, hi;
    block_range(t.off[t.n], blockIdx.x, gridDim.x, lo, hi);
    double acc = 0.0;
    for (int i = 0; i < t.n; ++i) {
        const int64_t s0 = lo > t.off[i] ? lo : t.off[i];
        const int64_t s1 = hi < t.off[i + 1] ? hi : t.off[i + 1];
        if (s0 >= s1) continue;
        const float* g = t.g[i] + (s0 - t.off[i]);
        const int64_t len = s1 - s0;
        // elements before the first 16-byte boundary, then float4s, then the rest
        int64_t head = int64_t((16u - (reinterpret_cast<uintptr_t>(g) & 15u)) & 15u) / 4;
        if (head > len) head = len;
        if (tid < head) {
            const double v = g[tid];
            acc += v * v;
        }
        const int64_t n4 = (len - head) / 4;
        const float4* g4 = reinterpret_cast<const float4*>(g + head);
#pragma unroll 4
        for (int64_t k = tid; k < n4; k += kSgdThreads) {
            const float4 v = g4[k];
            acc += double(v.x) * v.x + double(v.y) * v.y + double(v.z) * v.z + double(v.w) * v.w;
        }
        const int64_t r0 = head + 4 * n4;
        if (r0 + tid < len) {
            const double v = g[r0 + tid];
            acc += v * v;
        }
    }
    const double s = block_sum(acc, red);
    if (tid == 0) partial[blockIdx.x] = s;
}

__global__ __launch_bounds__(kSgdThreads) void sgd_scale_kernel(const double* partial, int n, float lr,
                                                                float max_norm, const uint32_t* hold, SgdCtrl* ctrl,
                                                                float* stats) {
    __shared__ double red[kSgdThreads / 64];
    double acc = 0.0;
    for (int k = threadIdx.x; k < n; k += kSgdThreads) acc += partial[k];
    const double total = block_sum(acc, red);
    if (threadIdx.x == 0) {
        const double norm = sqrt(total);
        const bool finite = isfinite(norm);
        // a held update (the step that produced the gradients failed) writes
        // nothing, as for a non-finite norm
        const bool held = hold != nullptr && *hold != 0u;
        double s = 1.0;
        if (!finite || held) s = 0.0;
        else if (max_norm > 0.f && isfinite(max_norm)) s = fmin(1.0, double(max_norm) / (norm + 1e-6));
        ctrl->ls = float(double(lr) * s);
        ctrl->skip = (finite && !held) ? 0 : 1;
        if (stats) {
            stats[0] = float(norm);
            stats[1] = float(s);
        }
    }
}

template <typename T>
__global__ __launch_bounds__(kSgdThreads) void sgd_update_kernel(SgdTable t, const SgdCtrl* ctrl) {
    if (ctrl->skip) return;
    const float ls = ctrl->ls;
    const int tid = threadIdx.x;
    int64_t lo, hi;
    block_range(t.off[t.n], blockIdx.x, gridDim.x, lo, hi);
    for (int i = 0; i < t.n; ++i) {
        const int64_t s0 = lo > t.off[i] ? lo : t.off[i];
        const int64_t s1 = hi < t.off[i + 1] ? hi : t.off[i + 1];
        if (s0 >= s1) continue;
        const float* g = t.g[i] + (s0 - t.off[i]);
        T* p = static_cast<T*>(t.p[i]) + (s0 - t.off[i]);
        const int64_t len = s1 - s0;
        int64_t head = int64_t((16u - (reinterpret_cast<uintptr_t>(g) & 15u)) & 15u) / 4;
        if (head > len) head = len;
        // vector body only when the parameters line up with the gradients
        const bool vec = (reinterpret_cast<uintptr_t>(p + head) % (4 * sizeof(T))) == 0;
        const int64_t n4 = vec ? (len - head) / 4 : 0;
        if (!vec) head = 0;
        if (tid < head) p[tid] = from_f<T>(to_f<T>(p[tid]) - ls * g[tid]);
        const float4* g4 = reinterpret_cast<const float4*>(g + head);
#pragma unroll 4
        for (int64_t k = tid; k < n4; k += kSgdThreads) {
            const float4 v = g4[k];
            T* q = p + head + 4 * k;
            if constexpr (sizeof(T) == 4) {
                float4 w = *reinterpret_cast<const float4*>(q);
                w.x -= ls * v.x;
                w.y -= ls * v.y;
                w.z -= ls * v.z;
                w.w -= ls * v.w;
                *reinterpret_cast<float4*>(q) = w;
            } else {
                const uint2 w = *reinterpret_cast<const uint2*>(q);
                const float a = bf2f(bf16_t(w.x & 0xffffu)) - ls * v.x, b = bf2f(bf16_t(w.x >> 16)) - ls * v.y;
                const float c = bf2f(bf16_t(w.y & 0xffffu)) - ls * v.z, d = bf2f(bf16_t(w.y >> 16)) - ls * v.w;
                *reinterpret_cast<uint2*>(q) = make_uint2(uint32_t(f2bf(a)) | (uint32_t(f2bf(b)) << 16),
                                                          uint32_t(f2bf(c)) | (uint32_t(f2bf(d)) << 16));
            }
        }
        for (int64_t k = head + 4 * n4 + tid; k < len; k += kSgdThreads) p[k] = from_f<T>(to_f<T>(p[k]) - ls * g[k]);
    }
}

constexpr int sgd_chunks(int n) { return (n + kSgdTable - 1) / kSgdTable; }

constexpr size_t sgd_ws_bytes(int n) {
    return ((size_t(sgd_chunks(n)) * kSgdBlocks * sizeof(double) + 255) / 256) * 256 + 256;
}

// The allocation-free update keeps its block sums and control word in this
// file-scope array (one copy per device, alive until the process ends)
// instead of a caller workspace: room for kNoAllocMaxTensors tensors.  Every
// call writes all of it that it reads (each block its sum, the scale kernel
// the control word), so nothing is cleared between calls.
constexpr int kNoAllocMaxTensors = JANUS_SGD_NOALLOC_MAX_TENSORS;
constexpr size_t kNoAllocScratchBytes = sgd_ws_bytes(kNoAllocMaxTensors);
static_assert(kNoAllocScratchBytes <= 64 * 1024, "a modest fixed array");
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, looked up once per
// device (hipGetSymbolAddress with that device current) and kept.  The
// array's name in host code is only a stand-in for the symbol; kernels and
// copies get this address.
janus_status scratch_address(void** out) {
    int dev = 0;
    JANUS_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return JANUS_ERR_UNSUPPORTED;
    static std::mutex m;
    static void* addr[kMaxDevices] = {};
    std::lock_guard<std::mutex> lock(m);
    if (!addr[dev]) {
        void* p = nullptr;
        JANUS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return JANUS_ERR_DEVICE;
        addr[dev] = p;
    }
    *out = addr[dev];
    return JANUS_OK;
}

SgdTable sgd_table(int c, int n, void* const* params, const float* const* grads, const int64_t* sizes) {
    SgdTable t{};
    const int i0 = c * kSgdTable, i1 = std::min(n, i0 + kSgdTable);
    t.n = i1 - i0;
    t.off[0] = 0;
    for (int i = i0; i < i1; ++i) {
        t.g[i - i0] = grads[i];
        t.p[i - i0] = params[i];
        t.off[i - i0 + 1] = t.off[i - i0] + sizes[i];
    }
    return t;
}

}  // namespace
}  // namespace janus

using namespace janus;

extern "C" size_t janus_sgd_workspace_bytes(const janus_sgd_desc* d) {
    if (!d || d->n < 1) return 0;
    return sgd_ws_bytes(d->n);
}

namespace janus {
namespace {

janus_status sgd_check(const janus_sgd_desc* d, void* const* params, const float* const* grads, const int64_t* sizes) {
    if (!d || d->n < 1 || !params || !grads || !sizes) return JANUS_ERR_INVALID_ARG;
    if (!dtype_ok(d->dtype)) return JANUS_ERR_UNSUPPORTED;
    if (!std::isfinite(d->lr) || std::isnan(d->max_norm)) return JANUS_ERR_INVALID_ARG;
    for (int i = 0; i < d->n; ++i) {
        if (sizes[i] < 0) return JANUS_ERR_INVALID_ARG;
        if (sizes[i] > 0 && (!params[i] || !grads[i])) return JANUS_ERR_INVALID_ARG;
        if (reinterpret_cast<uintptr_t>(grads[i]) % 4 != 0 ||
            reinterpret_cast<uintptr_t>(params[i]) % dtype_size(d->dtype) != 0)
            return JANUS_ERR_INVALID_ARG;
    }
    return JANUS_OK;
}

// The three launches of the update on `ws` (sgd_ws_bytes(d->n) bytes, block
// sums then the control word in its last 256 bytes).  `traced`: record the
// launches for janus_trace_end (which creates events, so the
// allocation-free entry point passes false).
janus_status sgd_run(const janus_sgd_desc* d, void* const* params, const float* const* grads, const int64_t* sizes,
                     float* stats, const uint32_t* hold, void* ws, hipStream_t st, bool traced) {
    const int nc = sgd_chunks(d->n);
    double* partial = static_cast<double*>(ws);
    SgdCtrl* ctrl = reinterpret_cast<SgdCtrl*>(static_cast<char*>(ws) + sgd_ws_bytes(d->n) - 256);
    const char* no_label = nullptr;
    for (int c = 0; c < nc; ++c) {
        const SgdTable t = sgd_table(c, d->n, params, grads, sizes);
        TraceScope trace(traced ? "sgd_sumsq" : no_label, 2.0 * double(t.off[t.n]), 4.0 * double(t.off[t.n]), st);
        hipLaunchKernelGGL(sgd_sumsq_kernel, dim3(kSgdBlocks), dim3(kSgdThreads), 0, st, t,
                           partial + int64_t(c) * kSgdBlocks);
        JANUS_LAUNCH_CHECK();
    }
    {
        TraceScope trace(traced ? "sgd_scale" : no_label, 0.0, 8.0 * nc * kSgdBlocks, st);
        hipLaunchKernelGGL(sgd_scale_kernel, dim3(1), dim3(kSgdThreads), 0, st, partial, nc * kSgdBlocks, d->lr,
                           d->max_norm, hold, ctrl, stats);
        JANUS_LAUNCH_CHECK();
    }
    const size_t es = dtype_size(d->dtype);
    for (int c = 0; c < nc; ++c) {
        const SgdTable t = sgd_table(c, d->n, params, grads, sizes);
        TraceScope trace(traced ? "sgd_update" : no_label, 2.0 * double(t.off[t.n]),
                         (4.0 + 2.0 * es) * double(t.off[t.n]), st);
        if (d->dtype == JANUS_BF16)
            hipLaunchKernelGGL(sgd_update_kernel<bf16_t>, dim3(kSgdBlocks), dim3(kSgdThreads), 0, st, t, ctrl);
        else
            hipLaunchKernelGGL(sgd_update_kernel<float>, dim3(kSgdBlocks), dim3(kSgdThreads), 0, st, t, ctrl);
        JANUS_LAUNCH_CHECK();
    }
    return JANUS_OK;
}

}  // namespace
}  // namespace janus

extern "C" janus_status janus_sgd_clip_update(const janus_sgd_desc* d, void* const* params, const float* const* grads,
                                              const int64_t* sizes, float* stats, const uint32_t* hold, void* ws,
                                              size_t ws_bytes, void* stream) {
    janus_status e = sgd_check(d, params, grads, sizes);
    if (e != JANUS_OK) return e;
    if (!ws || ws_bytes < sgd_ws_bytes(d->n) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    return sgd_run(d, params, grads, sizes, stats, hold, ws, static_cast<hipStream_t>(stream), true);
}

extern "C" janus_status janus_sgd_clip_update_noalloc(const janus_sgd_desc* d, void* const* params,
                                                      const float* const* grads, const int64_t* sizes, float* stats,
                                                      const uint32_t* hold, void* stream) {
    janus_status e = sgd_check(d, params, grads, sizes);
    if (e != JANUS_OK) return e;
    if (d->n > kNoAllocMaxTensors) return JANUS_ERR_WORKSPACE;
    void* ws = nullptr;
    if ((e = scratch_address(&ws)) != JANUS_OK) return e;
    return sgd_run(d, params, grads, sizes, stats, hold, ws, static_cast<hipStream_t>(stream), false);
}
