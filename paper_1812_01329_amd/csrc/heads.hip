// Embedding lookup and its gradient, softmax cross-entropy, the projection +
// mean-squared-error head, and scalar losses: the inputs and the
// ``compute_loss(outputs)`` of the training programs (Figure 1).
//
// Reductions are deterministic: every sum is taken in a fixed order (wave
// shuffles in a fixed butterfly, then a fixed sequence of partials), so two
// runs on the same inputs give identical bits.
#include <algorithm>
#include <mutex>
#include <cstdlib>
#include <vector>

#include "device.hpp"
#include "ops.hpp"

namespace janus {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// block-wide sum (blockDim.x a multiple of 64, at most 1024); result in all threads
__device__ float block_sum(float v, float* red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float s = 0.f;
    for (int i = 0; i < nw; ++i) s += red[i];
    return s;
}
__device__ float block_max(float v, float* red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    v = wave_max(v);
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float m = red[0];
    for (int i = 1; i < nw; ++i) m = fmaxf(m, red[i]);
    return m;
}

// --------------------------------------------------------------- embedding
template <typename T, bool VEC>
__global__ void embed_fwd_kernel(const T* E, const int32_t* ids, int V, int H, T* out) {
    const int r = blockIdx.x;
    // ids were range-checked on the host; the clamp only keeps a mismatched
    // device copy from reading outside the table
    const int64_t id = min(max(ids[r], 0), V - 1);
    const T* src = E + id * H;
    T* dst = out + int64_t(r) * H;
    if (VEC) {
        constexpr int V = 16 / sizeof(T);
        for (int j = threadIdx.x; j < H / V; j += blockDim.x)
            reinterpret_cast<uint4*>(dst)[j] = reinterpret_cast<const uint4*>(src)[j];
    } else {
        for (int j = threadIdx.x; j < H; j += blockDim.x) dst[j] = src[j];
    }
}

// dE[id] = sum of dx over the rows of one group of equal ids, in ascending
// row order.  seg = [order (rows) | off (nseg + 1) | sid (nseg)]: group g
// covers order[off[g] .. off[g + 1]) and has id sid[g].  One workgroup per
// group, threads over the columns; the rows of a frequent id are loaded eight
// at a time and added in order, so the loads overlap and the sum is fixed.
template <typename T>
__global__ void embed_bwd_seg_kernel(const T* dx, const int32_t* seg, int rows, int nseg, int H, float* dE) {
    const int g = blockIdx.x;
    const int32_t* order = seg;
    const int32_t* off = seg + rows;
    const int32_t* sid = off + nseg + 1;
    const int k0 = off[g], k1 = off[g + 1];
    const int64_t id = sid[g];
    for (int j = threadIdx.x; j < H; j += blockDim.x) {
        float s = 0.f;
        int k = k0;
        for (; k + 8 <= k1; k += 8) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = to_f(dx[int64_t(order[k + e]) * H + j]);
#pragma unroll
            for (int e = 0; e < 8; ++e) s += v[e];
        }
        for (; k < k1; ++k) s += to_f(dx[int64_t(order[k]) * H + j]);
        dE[id * H + j] = s;
    }
}

// --------------------------------------------------------------- softmax xent
// per row: loss_r = logsumexp(z) - z[target]; dz = (softmax(z) - onehot) / rows
constexpr int kXentLdsMax = 12288;   // vocabulary whose row a block keeps in LDS (48 KB)

template <typename T>
__global__ __launch_bounds__(256) void xent_row_kernel(const float* logits, int64_t ld, const int32_t* tgt, int V,
                                                       int rows, T* dz, int64_t ldz, float* loss_rows) {
    // With dynamic LDS for the row (V floats), the row is read from memory
    // once: the first pass keeps it, the second replaces it by exp(z - max),
    // the third writes dz from it.  Every thread touches only its own
    // entries (v = tid mod 256), so the passes need no barrier between them
    // beyond the reductions.  Without LDS (a row past 48 KB) each pass reads
    // the row again.  Both give the same values.
    extern __shared__ float zs[];
    const bool keep = (V <= kXentLdsMax);
    __shared__ float red[16];
    const int r = blockIdx.x;
    const float* z = logits + int64_t(r) * ld;
    float m = -INFINITY;
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        const float x = z[v];
        if (keep) zs[v] = x;
        m = fmaxf(m, x);
    }
    m = block_max(m, red);
    float s = 0.f;
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        const float e = __expf((keep ? zs[v] : z[v]) - m);
        if (keep) zs[v] = e;
        s += e;
    }
    s = block_sum(s, red);
    const float lse = m + __logf(s);
    const int t = min(max(tgt[r], 0), V - 1);
    const float inv = 1.f / float(rows);
    for (int v = threadIdx.x; v < V; v += blockDim.x) {
        const float p = (keep ? zs[v] : __expf(z[v] - m)) / s;
        dz[int64_t(r) * ldz + v] = from_f<T>((p - (v == t ? 1.f : 0.f)) * inv);
    }
    if (threadIdx.x == 0) loss_rows[r] = lse - z[t];
}

// loss = scale * sum of n partials, in index order by one block
__global__ __launch_bounds__(1024) void finish_sum_kernel(const float* part, int64_t n, float scale, float* loss) {
    __shared__ float red[16];
    float s = 0.f;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) s += part[i];
    s = block_sum(s, red);
    if (threadIdx.x == 0) *loss = s * scale;
}

// --------------------------------------------------------------- MSE head
// yp = h W^T + b for a tile, then d = yp - target; writes dY = 2 d / count
// (dtype) and one partial sum of d^2 per workgroup.
template <typename T, class Cfg, bool AL>
__global__ __launch_bounds__(Cfg::NT) void mse_gemm_kernel(int M, int N, int K, const T* h, const T* W, const T* b,
                                                           const T* tgt, T* dY, float scale, float* part) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ float red[16];
    T* sA = reinterpret_cast<T*>(smem_raw);
    T* sB = sA + Cfg::BM * Cfg::LD;
    const int tid = threadIdx.x;
    const int n0 = blockIdx.x * Cfg::BN, m0 = blockIdx.y * Cfg::BM;
    LoaderK<T, Cfg::BM, Cfg::BK, Cfg::NT, AL> la;
    LoaderK<T, Cfg::BN, Cfg::BK, Cfg::NT, AL> lb;
    la.init(h + int64_t(m0) * K, K, 0, RowsContig{M - m0}, tid);
    lb.init(W + int64_t(n0) * K, K, 0, RowsContig{N - n0}, tid);
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop<Cfg>(acc, la, lb, K, sA, sB, tid);
    const int lane = tid & 63, wave = tid >> 6;
    float sq = 0.f;
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
        const int col = n0 + Cfg::wave_col0(wave) + j * 32 + acc_col(lane);
        if (col >= N) continue;
        const float bv = to_f(b[col]);
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane);
                if (row >= M) continue;
                const int64_t o = int64_t(row) * N + col;
                const float d = acc[i][j][v] + bv - to_f(tgt[o]);
                sq += d * d;
                dY[o] = from_f<T>(scale * d);
            }
    }
    sq = block_sum(sq, red);
    if (tid == 0) part[blockIdx.y * gridDim.x + blockIdx.x] = sq;
}

// --------------------------------------------------------------- scalar losses
// One workgroup: 16-byte loads, eight in flight per thread (the loop is
// unrolled), four running sums per thread added in a fixed order, then the
// fixed-order workgroup sum.  The result does not depend on timing.
__global__ __launch_bounds__(1024) void loss_reduce_kernel(int kind, const float* h, int64_t n, float* loss) {
    __shared__ float red[16];
    const bool vec = (reinterpret_cast<uintptr_t>(h) & 15u) == 0;
    const int64_t n4 = vec ? n / 4 : 0;
    const float4* h4 = reinterpret_cast<const float4*>(h);
    float s0 = 0.f, s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll 8
    for (int64_t i = threadIdx.x; i < n4; i += 1024) {
        const float4 v = h4[i];
        if (kind == 0) {
            s0 += v.x * v.x;
            s1 += v.y * v.y;
            s2 += v.z * v.z;
            s3 += v.w * v.w;
        } else {
            s0 += v.x;
            s1 += v.y;
            s2 += v.z;
            s3 += v.w;
        }
    }
    for (int64_t i = 4 * n4 + threadIdx.x; i < n; i += 1024) s0 += kind == 0 ? h[i] * h[i] : h[i];
    float s = (s0 + s1) + (s2 + s3);
    s = block_sum(s, red);
    if (threadIdx.x == 0) *loss = kind == 0 ? s : s / float(n);
}

__global__ void loss_grad_kernel(int kind, const float* h, int64_t n, float* dh) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) dh[i] = kind == 0 ? 2.f * h[i] : 1.f / float(n);
}

using HeadBF16 = TileCfg<bf16_t, 128, 128, 32, 2, 2>;
using HeadF32 = TileCfg<float, 64, 64, 32, 2, 2>;

struct XentWs {
    int32_t* seg = nullptr;      // EMBED_BWD: the rows grouped by id
    float* logits = nullptr;
    void* dz = nullptr;
    float* loss_rows = nullptr;
    float* part = nullptr;
    void* gs = nullptr;          // contraction scratch
    size_t gs_bytes = 0;
    int64_t ldv = 0;
};

// scratch bound of the head's contractions: logits = h Wout^T, dh = dz Wout,
// dWout = dz^T h (run one after another, so one buffer serves all)
size_t head_gemm_scratch(janus_dtype dt, int rows, int H, int V) {
    if (dt != JANUS_BF16) return 0;
    GemmDesc g;
    g.dtype = dt;
    g.M = rows; g.N = V; g.K = H;
    size_t m = gemm_scratch_bound(g);
    g.N = H; g.K = V; g.b_t = true;
    m = std::max(m, gemm_scratch_bound(g));
    g.M = V; g.N = H; g.K = rows; g.a_t = true;
    return std::max(m, gemm_scratch_bound(g));
}

size_t carve_xent(const janus_xent_desc& d, janus_xent_op op, void* base, XentWs& w) {
    Carver c(base);
    if (op == JANUS_XENT_FWD_BWD) {
        w.ldv = round_up(d.V, 8);
        w.logits = c.take<float>(int64_t(d.rows) * w.ldv);
        w.dz = c.take<char>(int64_t(d.rows) * w.ldv * dtype_size(d.dtype));
        w.loss_rows = c.take<float>(d.rows);
        w.part = c.take<float>(colsum_partial_floats(d.V));
        w.gs_bytes = head_gemm_scratch(d.dtype, d.rows, d.H, d.V);
        w.gs = c.take<char>(int64_t(w.gs_bytes));
    }
    if (op == JANUS_EMBED_BWD) w.seg = c.take<int32_t>(int64_t(embed_seg_ints(d.rows)));
    return c.off + 256;
}

struct MseWs {
    void* dY = nullptr;
    float* part = nullptr;
    float* cpart = nullptr;
    void* gs = nullptr;          // contraction scratch
    size_t gs_bytes = 0;
    int nparts = 0;
};

template <class Cfg>
int mse_parts(const janus_mse_desc& d) {
    return ((d.P + Cfg::BN - 1) / Cfg::BN) * ((d.rows + Cfg::BM - 1) / Cfg::BM);
}

size_t carve_mse(const janus_mse_desc& d, void* base, MseWs& w) {
    Carver c(base);
    w.dY = c.take<char>(int64_t(d.rows) * d.P * dtype_size(d.dtype));
    w.nparts = d.dtype == JANUS_BF16 ? mse_parts<HeadBF16>(d) : mse_parts<HeadF32>(d);
    w.part = c.take<float>(d.dtype == JANUS_BF16 ? std::max<size_t>(size_t(w.nparts), gemm_mse_partials(d.rows, d.P))
                                                 : size_t(w.nparts));
    w.cpart = c.take<float>(colsum_partial_floats(d.P));
    w.gs_bytes = head_gemm_scratch(d.dtype, d.rows, d.H, d.P);
    w.gs = c.take<char>(int64_t(w.gs_bytes));
    return c.off + 256;
}

template <typename T, class Cfg>
janus_status mse_impl(const janus_mse_desc& d, const void* h, const void* W, const void* b, const void* tgt,
                      void* dh, float* dW, float* db, float* loss, const MseWs& w, hipStream_t st) {
    const float count = float(int64_t(d.rows) * d.P);
    dim3 grid((d.P + Cfg::BN - 1) / Cfg::BN, (d.rows + Cfg::BM - 1) / Cfg::BM);
    // large bf16 shapes: the fast contraction with the loss in its epilogue,
    // which also forms db
    const bool fused = d.dtype == JANUS_BF16 && gemm_mse_fast(d.rows, d.P, d.H, h, W) &&
                       reinterpret_cast<uintptr_t>(tgt) % 16 == 0 && reinterpret_cast<uintptr_t>(b) % 16 == 0;
    if (fused) {
        janus_status e = gemm_mse(d.rows, d.P, d.H, h, W, b, tgt, w.dY, 2.f / count, w.part, db, st);
        if (e != JANUS_OK) return e;
        const int64_t nparts = int64_t((d.rows + 255) / 256) * ((d.P + 255) / 256);
        TraceScope trace("finish_sum", 0.0, 4.0 * nparts, st);
        hipLaunchKernelGGL(finish_sum_kernel, dim3(1), dim3(1024), 0, st, w.part, nparts, 1.f / count, loss);
        JANUS_LAUNCH_CHECK();
    } else {
        {
            TraceScope trace("mse_gemm", 2.0 * d.rows * double(d.P) * d.H,
                             double(sizeof(T)) * (double(d.rows) * d.H + double(d.P) * d.H + 2.0 * d.rows * double(d.P)),
                             st);
            const bool al = (int64_t(d.H) * int64_t(sizeof(T))) % 16 == 0 &&
                            reinterpret_cast<uintptr_t>(h) % 16 == 0 && reinterpret_cast<uintptr_t>(W) % 16 == 0;
            if (al)
                hipLaunchKernelGGL((mse_gemm_kernel<T, Cfg, true>), grid, dim3(Cfg::NT), Cfg::SMEM_BYTES, st, d.rows,
                                   d.P, d.H, static_cast<const T*>(h), static_cast<const T*>(W),
                                   static_cast<const T*>(b), static_cast<const T*>(tgt), static_cast<T*>(w.dY),
                                   2.f / count, w.part);
            else
                hipLaunchKernelGGL((mse_gemm_kernel<T, Cfg, false>), grid, dim3(Cfg::NT), Cfg::SMEM_BYTES, st, d.rows,
                                   d.P, d.H, static_cast<const T*>(h), static_cast<const T*>(W),
                                   static_cast<const T*>(b), static_cast<const T*>(tgt), static_cast<T*>(w.dY),
                                   2.f / count, w.part);
            JANUS_LAUNCH_CHECK();
        }
        TraceScope trace("finish_sum", 0.0, 4.0 * w.nparts, st);
        hipLaunchKernelGGL(finish_sum_kernel, dim3(1), dim3(1024), 0, st, w.part, int64_t(w.nparts), 1.f / count,
                           loss);
        JANUS_LAUNCH_CHECK();
    }
    // dh = dY W
    GemmDesc g;
    g.dtype = d.dtype;
    g.M = d.rows;
    g.N = d.H;
    g.K = d.P;
    g.A = w.dY;
    g.lda = d.P;
    g.b_t = true;
    g.B = W;
    g.ldb = d.H;
    g.C = dh;
    g.ldc = d.H;
    g.c_f32 = false;
    g.scratch = w.gs;
    g.scratch_bytes = w.gs_bytes;
    janus_status e = gemm(g, st);
    if (e != JANUS_OK) return e;
    // dW = dY^T h
    GemmDesc q;
    q.dtype = d.dtype;
    q.M = d.P;
    q.N = d.H;
    q.K = d.rows;
    q.a_t = true;
    q.A = w.dY;
    q.lda = d.P;
    q.b_t = true;
    q.B = h;
    q.ldb = d.H;
    q.C = dW;
    q.ldc = d.H;
    q.c_f32 = true;
    q.scratch = w.gs;
    q.scratch_bytes = w.gs_bytes;
    e = gemm(q, st);
    if (e != JANUS_OK) return e;
    if (fused) return JANUS_OK;
    return colsum(d.dtype, w.dY, d.rows, d.P, d.P, db, w.cpart, st);
}

template <typename T>
janus_status xent_impl(const janus_xent_desc& d, const int32_t* ids_dev, const void* Wout, const void* bout,
                       const void* h, void* dh, float* dWout, float* dbout, float* loss, const XentWs& w,
                       hipStream_t st) {
    GemmDesc g;
    g.dtype = d.dtype;
    g.M = d.rows;
    g.N = d.V;
    g.K = d.H;
    g.A = h;
    g.lda = d.H;
    g.B = Wout;
    g.ldb = d.H;
    g.C = w.logits;
    g.ldc = w.ldv;
    g.c_f32 = true;
    g.bias = bout;
    g.scratch = w.gs;
    g.scratch_bytes = w.gs_bytes;
    janus_status e = gemm(g, st);
    if (e != JANUS_OK) return e;
    {
        TraceScope trace_row("xent_row", 0.0, double(d.rows) * d.V * (4.0 + sizeof(T)), st);
        const size_t zsm = d.V <= kXentLdsMax ? sizeof(float) * size_t(d.V) : 0;
        hipLaunchKernelGGL(xent_row_kernel<T>, dim3(d.rows), dim3(256), zsm, st, w.logits, w.ldv, ids_dev, d.V, d.rows,
                           static_cast<T*>(w.dz), w.ldv, w.loss_rows);
        JANUS_LAUNCH_CHECK();
    }
    {
        TraceScope trace_fin("finish_sum", 0.0, 4.0 * d.rows, st);
        hipLaunchKernelGGL(finish_sum_kernel, dim3(1), dim3(1024), 0, st, w.loss_rows, int64_t(d.rows),
                           1.f / float(d.rows), loss);
        JANUS_LAUNCH_CHECK();
    }
    // dh = dz Wout
    GemmDesc q;
    q.dtype = d.dtype;
    q.M = d.rows;
    q.N = d.H;
    q.K = d.V;
    q.A = w.dz;
    q.lda = w.ldv;
    q.b_t = true;
    q.B = Wout;
    q.ldb = d.H;
    q.C = dh;
    q.ldc = d.H;
    q.c_f32 = false;
    q.scratch = w.gs;
    q.scratch_bytes = w.gs_bytes;
    e = gemm(q, st);
    if (e != JANUS_OK) return e;
    // dWout = dz^T h
    GemmDesc r;
    r.dtype = d.dtype;
    r.M = d.V;
    r.N = d.H;
    r.K = d.rows;
    r.a_t = true;
    r.A = w.dz;
    r.lda = w.ldv;
    r.b_t = true;
    r.B = h;
    r.ldb = d.H;
    r.C = dWout;
    r.ldc = d.H;
    r.c_f32 = true;
    r.scratch = w.gs;
    r.scratch_bytes = w.gs_bytes;
    e = gemm(r, st);
    if (e != JANUS_OK) return e;
    return colsum(d.dtype, w.dz, d.rows, d.V, w.ldv, dbout, w.part, st);
}

}  // namespace

size_t embed_seg_ints(int rows) { return rows > 0 ? size_t(3) * rows + 1 : 1; }

int embed_segments(const int32_t* ids_host, int rows, int V, std::vector<int32_t>& seg) {
    // stable counting sort by id: count, exclusive scan, place rows in
    // ascending order within each id
    std::vector<int32_t> count(size_t(V) + 1, 0);
    for (int r = 0; r < rows; ++r) ++count[size_t(ids_host[r]) + 1];
    int nseg = 0;
    for (int v = 0; v < V; ++v) {
        nseg += count[size_t(v) + 1] != 0;
        count[size_t(v) + 1] += count[size_t(v)];
    }
    seg.assign(size_t(rows) + 2 * size_t(nseg) + 1, 0);
    int32_t* order = seg.data();
    int32_t* off = order + rows;
    int32_t* sid = off + nseg + 1;
    std::vector<int32_t> next(count.begin(), count.end() - 1);
    for (int r = 0; r < rows; ++r) order[next[size_t(ids_host[r])]++] = r;
    int g = 0;
    for (int v = 0; v < V; ++v)
        if (count[size_t(v) + 1] != count[size_t(v)]) {
            off[g] = count[size_t(v)];
            sid[g] = v;
            ++g;
        }
    off[nseg] = rows;
    return nseg;
}

janus_status embed_backward(janus_dtype dt, const void* dx, const int32_t* ids_host, int rows, int H, float* dE, int V,
                            int32_t* seg_dev, hipStream_t st) {
    janus_status e = zero_fill(dE, size_t(V) * H * sizeof(float), st);
    if (e != JANUS_OK) return e;
    if (rows <= 0) return JANUS_OK;
    std::vector<int32_t> seg;
    const int nseg = embed_segments(ids_host, rows, V, seg);
    if ((e = upload(seg_dev, seg.data(), seg.size() * sizeof(int32_t), st)) != JANUS_OK) return e;
    TraceScope trace("embed_bwd", 0.0, double(rows) * H * dtype_size(dt) + double(nseg) * H * 4.0, st);
    if (dt == JANUS_BF16)
        hipLaunchKernelGGL(embed_bwd_seg_kernel<bf16_t>, dim3(unsigned(nseg)), dim3(256), 0, st,
                           static_cast<const bf16_t*>(dx), seg_dev, rows, nseg, H, dE);
    else
        hipLaunchKernelGGL(embed_bwd_seg_kernel<float>, dim3(unsigned(nseg)), dim3(256), 0, st,
                           static_cast<const float*>(dx), seg_dev, rows, nseg, H, dE);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

// ------------------------------------------------------- small softmax head
// The whole softmax cross-entropy head of a small problem (a few hundred
// rows, at most 64 classes, e.g. the 5-class sentiment head at the tree
// roots) in one workgroup: h and Wout in LDS, the logits, per-row
// log-sum-exp, loss, dz = (softmax - onehot) / rows, dh = dz Wout,
// dWout = dz^T h and dbout = column sums of dz, each summed in a fixed
// order.  One launch instead of three contractions, two reductions and
// the column sums.
constexpr int kXentSmallV = 64;
constexpr size_t kXentSmallLds = 64 * 1024;

size_t xent_small_lds(const janus_xent_desc& d) {
    return sizeof(float) * (size_t(d.rows) * d.H + size_t(d.V) * d.H + size_t(d.rows) * d.V + size_t(d.rows));
}
bool xent_small_fits(const janus_xent_desc& d) {
    const char* e = getenv("JANUS_XENT_SMALL");
    if (e && e[0] == '0') return false;
    return d.V <= kXentSmallV && xent_small_lds(d) <= kXentSmallLds;
}

template <typename T>
__global__ __launch_bounds__(256) void xent_small_kernel(const T* h, const T* W, const T* b, const int32_t* tgt,
                                                         int rows, int V, int H, T* dh, float* dW, float* db,
                                                         float* loss) {
    extern __shared__ float xs[];
    float* hs = xs;                    // [rows][H]
    float* wsm = hs + rows * H;        // [V][H]
    float* zs = wsm + V * H;           // [rows][V]: logits, then dz
    float* ls = zs + rows * V;         // [rows] loss of each row
    const int tid = threadIdx.x;
    // h and W into LDS, NB elements in flight per thread: the raw values are
    // loaded first and converted only after the last load of the batch is
    // issued, so a batch costs one memory round trip, not one per element
    auto stage = [&](float* dst, const T* src, int n) {
        constexpr int NB = 32;
        for (int base = tid; base < n; base += 256 * NB) {
            T v[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const int idx = base + i * 256;
                v[i] = idx < n ? src[idx] : T(0);
            }
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const int idx = base + i * 256;
                if (idx < n) dst[idx] = to_f(v[i]);
            }
        }
    };
    stage(hs, h, rows * H);
    stage(wsm, W, V * H);
    __syncthreads();
    for (int i = tid; i < rows * V; i += blockDim.x) {
        const int r = i / V, v = i - r * V;
        float s = to_f(b[v]);
        for (int k = 0; k < H; ++k) s += hs[r * H + k] * wsm[v * H + k];
        zs[i] = s;
    }
    __syncthreads();
    const float inv = 1.f / float(rows);
    for (int r = tid; r < rows; r += blockDim.x) {
        float* z = zs + r * V;
        float m = -INFINITY;
        for (int v = 0; v < V; ++v) m = fmaxf(m, z[v]);
        float se = 0.f;
        for (int v = 0; v < V; ++v) se += __expf(z[v] - m);
        const int t = min(max(tgt[r], 0), V - 1);
        ls[r] = m + __logf(se) - z[t];
        const float rs = 1.f / se;
        for (int v = 0; v < V; ++v) z[v] = (__expf(z[v] - m) * rs - (v == t ? 1.f : 0.f)) * inv;
    }
    __syncthreads();
    if (tid == 0) {
        float s = 0.f;
        for (int r = 0; r < rows; ++r) s += ls[r];
        *loss = s * inv;
    }
    for (int i = tid; i < rows * H; i += blockDim.x) {
        const int r = i / H, k = i - r * H;
        float s = 0.f;
        for (int v = 0; v < V; ++v) s += zs[r * V + v] * wsm[v * H + k];
        dh[i] = from_f<T>(s);
    }
    for (int i = tid; i < V * H; i += blockDim.x) {
        const int v = i / H, k = i - v * H;
        float s = 0.f;
        for (int r = 0; r < rows; ++r) s += zs[r * V + v] * hs[r * H + k];
        dW[i] = s;
    }
    for (int v = tid; v < V; v += blockDim.x) {
        float s = 0.f;
        for (int r = 0; r < rows; ++r) s += zs[r * V + v];
        db[v] = s;
    }
}

template <typename T>
janus_status xent_small(const janus_xent_desc& d, const int32_t* ids_dev, const void* Wout, const void* bout,
                        const void* h, void* dh, float* dWout, float* dbout, float* loss, hipStream_t st) {
    static std::mutex m;
    static size_t attr = 0;
    const size_t smem = xent_small_lds(d);
    {
        std::lock_guard<std::mutex> lock(m);
        if (smem > attr) {
            JANUS_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(xent_small_kernel<T>),
                                          hipFuncAttributeMaxDynamicSharedMemorySize, int(smem)));
            attr = smem;
        }
    }
    TraceScope trace("xent_small", 2.0 * 3.0 * d.rows * double(d.V) * d.H,
                     double(dtype_size(d.dtype)) * (2.0 * d.rows * d.H + double(d.V) * d.H), st);
    hipLaunchKernelGGL(xent_small_kernel<T>, dim3(1), dim3(256), smem, st, static_cast<const T*>(h),
                       static_cast<const T*>(Wout), static_cast<const T*>(bout), ids_dev, d.rows, d.V, d.H,
                       static_cast<T*>(dh), dWout, dbout, loss);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

}  // namespace janus

using namespace janus;

extern "C" size_t janus_xent_workspace_bytes(const janus_xent_desc* d, janus_xent_op op) {
    if (!d || d->V <= 0 || d->H <= 0 || d->rows <= 0) return 0;
    XentWs w;
    return carve_xent(*d, op, nullptr, w);
}

extern "C" janus_status janus_embed_softmax_xent(const janus_xent_desc* d, janus_xent_op op, const int32_t* ids_host,
                                                 const int32_t* ids_dev, const void* table, const void* bias,
                                                 const void* in, void* out, float* dtable, float* dbias, float* loss,
                                                 void* ws, size_t ws_bytes, void* stream) {
    if (!d || d->V <= 0 || d->H <= 0 || d->rows <= 0 || !ids_host || !ids_dev) return JANUS_ERR_INVALID_ARG;
    if (!dtype_ok(d->dtype)) return JANUS_ERR_UNSUPPORTED;
    if (op != JANUS_EMBED_FWD && op != JANUS_XENT_FWD_BWD && op != JANUS_EMBED_BWD) return JANUS_ERR_INVALID_ARG;
    if (op == JANUS_EMBED_FWD && (!table || !out)) return JANUS_ERR_INVALID_ARG;
    if (op == JANUS_XENT_FWD_BWD && (!table || !bias || !in || !out || !dtable || !dbias || !loss))
        return JANUS_ERR_INVALID_ARG;
    if (op == JANUS_EMBED_BWD && (!in || !dtable)) return JANUS_ERR_INVALID_ARG;
    for (int32_t r = 0; r < d->rows; ++r)
        if (ids_host[r] < 0 || ids_host[r] >= d->V) return JANUS_ERR_TOKEN;
    XentWs w;
    const size_t need = carve_xent(*d, op, nullptr, w);
    if (op != JANUS_EMBED_FWD) {
        if (!ws || ws_bytes < need || reinterpret_cast<uintptr_t>(ws) % 256 != 0) return JANUS_ERR_WORKSPACE;
        carve_xent(*d, op, ws, w);
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    const size_t es = dtype_size(d->dtype);
    if (op == JANUS_EMBED_FWD) {
        TraceScope trace("embed_fwd", 0.0, 2.0 * d->rows * double(d->H) * es, st);
        const bool vec = (int64_t(d->H) * int64_t(es)) % 16 == 0 && reinterpret_cast<uintptr_t>(table) % 16 == 0 &&
                         reinterpret_cast<uintptr_t>(out) % 16 == 0;
        if (d->dtype == JANUS_BF16) {
            if (vec)
                hipLaunchKernelGGL((embed_fwd_kernel<bf16_t, true>), dim3(d->rows), dim3(128), 0, st,
                                   static_cast<const bf16_t*>(table), ids_dev, d->V, d->H, static_cast<bf16_t*>(out));
            else
                hipLaunchKernelGGL((embed_fwd_kernel<bf16_t, false>), dim3(d->rows), dim3(128), 0, st,
                                   static_cast<const bf16_t*>(table), ids_dev, d->V, d->H, static_cast<bf16_t*>(out));
        } else {
            if (vec)
                hipLaunchKernelGGL((embed_fwd_kernel<float, true>), dim3(d->rows), dim3(128), 0, st,
                                   static_cast<const float*>(table), ids_dev, d->V, d->H, static_cast<float*>(out));
            else
                hipLaunchKernelGGL((embed_fwd_kernel<float, false>), dim3(d->rows), dim3(128), 0, st,
                                   static_cast<const float*>(table), ids_dev, d->V, d->H, static_cast<float*>(out));
        }
        JANUS_LAUNCH_CHECK();
        return JANUS_OK;
    }
    if (op == JANUS_EMBED_BWD) return embed_backward(d->dtype, in, ids_host, d->rows, d->H, dtable, d->V, w.seg, st);
    if (xent_small_fits(*d)) {
        if (d->dtype == JANUS_BF16)
            return xent_small<bf16_t>(*d, ids_dev, table, bias, in, out, dtable, dbias, loss, st);
        return xent_small<float>(*d, ids_dev, table, bias, in, out, dtable, dbias, loss, st);
    }
    if (d->dtype == JANUS_BF16)
        return xent_impl<bf16_t>(*d, ids_dev, table, bias, in, out, dtable, dbias, loss, w, st);
    return xent_impl<float>(*d, ids_dev, table, bias, in, out, dtable, dbias, loss, w, st);
}

extern "C" size_t janus_mse_workspace_bytes(const janus_mse_desc* d) {
    if (!d || d->rows <= 0 || d->H <= 0 || d->P <= 0 || !dtype_ok(d->dtype)) return 0;
    MseWs w;
    return carve_mse(*d, nullptr, w);
}

extern "C" janus_status janus_linear_mse(const janus_mse_desc* d, const void* h, const void* W, const void* b,
                                         const void* target, void* dh, float* dW, float* db, float* loss, void* ws,
                                         size_t ws_bytes, void* stream) {
    if (!d || d->rows <= 0 || d->H <= 0 || d->P <= 0) return JANUS_ERR_INVALID_ARG;
    if (!dtype_ok(d->dtype)) return JANUS_ERR_UNSUPPORTED;
    if (!h || !W || !b || !target || !dh || !dW || !db || !loss) return JANUS_ERR_INVALID_ARG;
    MseWs w;
    if (!ws || ws_bytes < carve_mse(*d, nullptr, w) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    carve_mse(*d, ws, w);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (d->dtype == JANUS_BF16) return mse_impl<bf16_t, HeadBF16>(*d, h, W, b, target, dh, dW, db, loss, w, st);
    return mse_impl<float, HeadF32>(*d, h, W, b, target, dh, dW, db, loss, w, st);
}

extern "C" janus_status janus_loss_reduce(janus_loss_kind kind, const float* h, int64_t n, float* loss, float* dh,
                                          void* stream) {
    if (!h || !loss || n <= 0) return JANUS_ERR_INVALID_ARG;
    if (kind != JANUS_LOSS_SUMSQ && kind != JANUS_LOSS_MEAN) return JANUS_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    TraceScope trace("loss_reduce", 0.0, 4.0 * n * (dh ? 2.0 : 1.0), st);
    hipLaunchKernelGGL(loss_reduce_kernel, dim3(1), dim3(1024), 0, st, int(kind), h, n, loss);
    JANUS_LAUNCH_CHECK();
    if (dh) {
        hipLaunchKernelGGL(loss_grad_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, int(kind), h, n, dh);
        JANUS_LAUNCH_CHECK();
    }
    return JANUS_OK;
}
