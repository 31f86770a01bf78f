// General MFMA contraction with optional row gathers and scatters, plus the
// small reductions used around it.  Every dense contraction of the training
// step that has no fused epilogue goes through here: the hoisted input
// projection of all time steps, the weight gradients (one contraction over
// all packed time steps), input gradients, and the head contractions.
#include "device.hpp"
#include "ops.hpp"

namespace janus {

namespace {

// Epilogue: C = alpha * acc + bias, optional row scatter.  Specialised on the
// output type and the scatter so that every accumulator index is a
// compile-time constant (the 256-register accumulator stays in registers).
template <typename T, class Cfg, typename OutT, bool SCATTER>
__device__ __forceinline__ void store_tile_impl(const GemmDesc& g, f32x16_t (&acc)[Cfg::FM][Cfg::FN], int m0, int n0,
                                                int tid) {
    const int lane = tid & 63, wave = tid >> 6;
    const T* bias = static_cast<const T*>(g.bias);
    OutT* C = static_cast<OutT*>(g.C);
    float bv[Cfg::FN];
    int col[Cfg::FN];
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
        col[j] = n0 + Cfg::wave_col0(wave) + j * 32 + acc_col(lane);
        bv[j] = (bias && col[j] < g.N) ? to_f(bias[col[j]]) : 0.f;
    }
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int row = m0 + Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane);
            const bool rok = row < g.M;
            const int64_t crow = SCATTER ? (rok ? int64_t(g.c_idx[row]) : 0) : int64_t(row);
#pragma unroll
            for (int j = 0; j < Cfg::FN; ++j) {
                if (rok && col[j] < g.N) {
                    const float val = g.alpha * acc[i][j][v] + bv[j];
                    C[crow * g.ldc + col[j]] = from_f<OutT>(val);
                }
            }
        }
    }
}

template <typename T, class Cfg>
__device__ __forceinline__ void store_tile(const GemmDesc& g, f32x16_t (&acc)[Cfg::FM][Cfg::FN], int m0, int n0,
                                           int tid) {
    if (g.c_f32) {
        if (g.c_idx) store_tile_impl<T, Cfg, float, true>(g, acc, m0, n0, tid);
        else store_tile_impl<T, Cfg, float, false>(g, acc, m0, n0, tid);
    } else {
        if (g.c_idx) store_tile_impl<T, Cfg, T, true>(g, acc, m0, n0, tid);
        else store_tile_impl<T, Cfg, T, false>(g, acc, m0, n0, tid);
    }
}

template <typename T, class Cfg, bool AT, bool BT, bool AL>
__global__ __launch_bounds__(Cfg::NT) void gemm_kernel(GemmDesc g) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    T* sA = reinterpret_cast<T*>(smem_raw);
    T* sB = sA + Cfg::BM * Cfg::LD;
    const int tid = threadIdx.x;
    const int n0 = blockIdx.x * Cfg::BN;
    const int m0 = blockIdx.y * Cfg::BM;
    const T* A = static_cast<const T*>(g.A);
    const T* B = static_cast<const T*>(g.B);

    using LA = typename std::conditional<AT, LoaderT<T, Cfg::BM, Cfg::BK, Cfg::NT, AL>,
                                         LoaderK<T, Cfg::BM, Cfg::BK, Cfg::NT, AL>>::type;
    using LB = typename std::conditional<BT, LoaderT<T, Cfg::BN, Cfg::BK, Cfg::NT, AL>,
                                         LoaderK<T, Cfg::BN, Cfg::BK, Cfg::NT, AL>>::type;
    LA la;
    LB lb;
    if constexpr (AT) {
        la.init(A, g.lda, g.a_idx, m0, g.M);
    } else {
        if (g.a_idx) la.init(A, g.lda, 0, RowsIndexed{g.a_idx + m0, g.M - m0}, tid);
        else la.init(A + int64_t(m0) * g.lda, g.lda, 0, RowsContig{g.M - m0}, tid);
    }
    if constexpr (BT) {
        lb.init(B, g.ldb, g.b_idx, n0, g.N);
    } else {
        if (g.b_idx) lb.init(B, g.ldb, 0, RowsIndexed{g.b_idx + n0, g.N - n0}, tid);
        else lb.init(B + int64_t(n0) * g.ldb, g.ldb, 0, RowsContig{g.N - n0}, tid);
    }
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop<Cfg>(acc, la, lb, g.K, sA, sB, tid);

    store_tile<T, Cfg>(g, acc, m0, n0, tid);
}

// Large bf16 contractions: 256 x 256 tiles, four waves of 128 x 128, two LDS
// stages.  Tiles are numbered so that each XCD (blocks are dealt to the 8
// XCDs round robin) works on a contiguous range, grouped 8 M-tiles at a time
// so that neighbouring workgroups share B tiles in that XCD's L2.
template <class Cfg, bool AT, bool BT, bool AL>
__global__ __launch_bounds__(Cfg::NT) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gemm_big_kernel(GemmDesc g, int mtiles, int ntiles) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);
    const int tid = threadIdx.x;
    const int ntot = mtiles * ntiles;
    int t = blockIdx.x;
    if (ntot % 8 == 0) t = (t % 8) * (ntot / 8) + t / 8;
    constexpr int GM = 8;
    const int in_group = GM * ntiles;
    const int first_m = (t / in_group) * GM;
    const int gsz = min(mtiles - first_m, GM);
    const int tm = first_m + (t % in_group) % gsz;
    const int tn = (t % in_group) / gsz;
    const int m0 = tm * Cfg::BM, n0 = tn * Cfg::BN;
    const bf16_t* A = static_cast<const bf16_t*>(g.A);
    const bf16_t* B = static_cast<const bf16_t*>(g.B);
    using LA = typename std::conditional<AT, LoaderT<bf16_t, Cfg::BM, Cfg::BK, Cfg::NT, AL, true>,
                                         LoaderK<bf16_t, Cfg::BM, Cfg::BK, Cfg::NT, AL, true>>::type;
    using LB = typename std::conditional<BT, LoaderT<bf16_t, Cfg::BN, Cfg::BK, Cfg::NT, AL, true>,
                                         LoaderK<bf16_t, Cfg::BN, Cfg::BK, Cfg::NT, AL, true>>::type;
    LA la;
    LB lb;
    if constexpr (AT) {
        la.init(A, g.lda, g.a_idx, m0, g.M);
    } else {
        if (g.a_idx) la.init(A, g.lda, 0, RowsIndexed{g.a_idx + m0, g.M - m0}, tid);
        else la.init(A + int64_t(m0) * g.lda, g.lda, 0, RowsContig{g.M - m0}, tid);
    }
    if constexpr (BT) {
        lb.init(B, g.ldb, g.b_idx, n0, g.N);
    } else {
        if (g.b_idx) lb.init(B, g.ldb, 0, RowsIndexed{g.b_idx + n0, g.N - n0}, tid);
        else lb.init(B + int64_t(n0) * g.ldb, g.ldb, 0, RowsContig{g.N - n0}, tid);
    }
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop_swz<Cfg>(acc, la, lb, g.K, smem, tid);
    store_tile<bf16_t, Cfg>(g, acc, m0, n0, tid);
}

const char* gemm_label(bool at, bool bt, bool bf16) {
    if (!at && !bt) return bf16 ? "gemm_nt_bf16" : "gemm_nt_f32";
    if (!at && bt) return bf16 ? "gemm_nn_bf16" : "gemm_nn_f32";
    return bf16 ? "gemm_tn_bf16" : "gemm_tn_f32";
}

template <typename T, class Cfg, bool AT, bool BT, bool AL>
janus_status launch(const GemmDesc& g, hipStream_t s) {
    dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM);
    const double es = sizeof(T);
    TraceScope trace(gemm_label(AT, BT, sizeof(T) == 2), 2.0 * g.M * g.N * double(g.K),
                     (double(g.M) * g.K + double(g.N) * g.K) * es + double(g.M) * g.N * (g.c_f32 ? 4.0 : es), s);
    hipLaunchKernelGGL((gemm_kernel<T, Cfg, AT, BT, AL>), grid, dim3(Cfg::NT), Cfg::SMEM_BYTES, s, g);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

template <class Cfg, bool AT, bool BT, bool AL>
janus_status launch_big(const GemmDesc& g, hipStream_t s) {
    constexpr int smem = 2 * (Cfg::BM + Cfg::BN) * Cfg::BK * int(sizeof(bf16_t));
    static bool attr = false;
    if (!attr) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_big_kernel<Cfg, AT, BT, AL>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, smem) != hipSuccess)
            return JANUS_ERR_DEVICE;
        attr = true;
    }
    const int mt = (g.M + Cfg::BM - 1) / Cfg::BM, nt = (g.N + Cfg::BN - 1) / Cfg::BN;
    TraceScope trace(gemm_label(AT, BT, true), 2.0 * g.M * g.N * double(g.K),
                     (double(g.M) * g.K + double(g.N) * g.K) * 2.0 + double(g.M) * g.N * (g.c_f32 ? 4.0 : 2.0), s);
    hipLaunchKernelGGL((gemm_big_kernel<Cfg, AT, BT, AL>), dim3(mt * nt), dim3(Cfg::NT), smem, s, g, mt, nt);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

template <class Cfg>
janus_status dispatch_big(const GemmDesc& g, bool aligned, hipStream_t s) {
    if (!g.a_t && !g.b_t) return aligned ? launch_big<Cfg, false, false, true>(g, s) : launch_big<Cfg, false, false, false>(g, s);
    if (!g.a_t && g.b_t) return aligned ? launch_big<Cfg, false, true, true>(g, s) : launch_big<Cfg, false, true, false>(g, s);
    if (g.a_t && g.b_t) return aligned ? launch_big<Cfg, true, true, true>(g, s) : launch_big<Cfg, true, true, false>(g, s);
    return JANUS_ERR_UNSUPPORTED;
}

template <typename T, class Cfg>
janus_status dispatch(const GemmDesc& g, bool aligned, hipStream_t s) {
    if (!g.a_t && !g.b_t) return aligned ? launch<T, Cfg, false, false, true>(g, s) : launch<T, Cfg, false, false, false>(g, s);
    if (!g.a_t && g.b_t) return aligned ? launch<T, Cfg, false, true, true>(g, s) : launch<T, Cfg, false, true, false>(g, s);
    if (g.a_t && g.b_t) return aligned ? launch<T, Cfg, true, true, true>(g, s) : launch<T, Cfg, true, true, false>(g, s);
    return JANUS_ERR_UNSUPPORTED;
}

bool aligned16(const void* p, int64_t ld, size_t es) {
    return (reinterpret_cast<uintptr_t>(p) % 16 == 0) && ((ld * int64_t(es)) % 16 == 0);
}

// ---------------------------------------------------------------- colsum
constexpr int kColTile = 256;
constexpr int kRowChunks = 64;

template <typename T>
__global__ __launch_bounds__(kColTile) void colsum_partial_kernel(const T* in, int64_t R, int C, int64_t ld,
                                                                  float* partial) {
    const int c = blockIdx.x * kColTile + threadIdx.x;
    const int chunk = blockIdx.y;
    const int64_t per = (R + kRowChunks - 1) / kRowChunks;
    const int64_t r0 = chunk * per, r1 = r0 + per < R ? r0 + per : R;
    if (c >= C) return;
    float s = 0.f;
    for (int64_t r = r0; r < r1; ++r) s += to_f(in[r * ld + c]);
    partial[int64_t(chunk) * C + c] = s;
}

__global__ __launch_bounds__(kColTile) void colsum_final_kernel(const float* partial, int C, float* out,
                                                                const int32_t* out_idx) {
    const int c = blockIdx.x * kColTile + threadIdx.x;
    if (c >= C) return;
    float s = 0.f;
    for (int k = 0; k < kRowChunks; ++k) s += partial[int64_t(k) * C + c];
    out[out_idx ? out_idx[c] : c] = s;
}

__global__ void zero_kernel(unsigned char* p, size_t head, uint4* mid, size_t n16, unsigned char* tail, size_t ntail) {
    size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (; i < n16; i += stride) mid[i] = make_uint4(0, 0, 0, 0);
    if (blockIdx.x == 0 && threadIdx.x < head) p[threadIdx.x] = 0;
    if (blockIdx.x == 0 && threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

}  // namespace

// bf16: 128x128 tiles, 4 waves of 64x64; fp32: 64x64 tiles, 4 waves of 32x32
using CfgBF16 = TileCfg<bf16_t, 128, 128, 32, 2, 2>;
using CfgF32 = TileCfg<float, 64, 64, 32, 2, 2>;
using CfgBig = TileCfg<bf16_t, 256, 256, 64, 2, 2>;

janus_status gemm(const GemmDesc& g, hipStream_t stream) {
    if (g.M <= 0 || g.N <= 0) return JANUS_OK;
    const size_t es = dtype_size(g.dtype);
    const bool aligned = aligned16(g.A, g.lda, es) && aligned16(g.B, g.ldb, es);
    if (g.K <= 0) {
        // empty contraction: C = bias (or 0); handled by the kernel with K = 0
    }
    if (g.dtype == JANUS_BF16) {
        if (g.M >= 256 && g.N >= 256) return dispatch_big<CfgBig>(g, aligned, stream);
        return dispatch<bf16_t, CfgBF16>(g, aligned, stream);
    }
    if (g.dtype == JANUS_F32) return dispatch<float, CfgF32>(g, aligned, stream);
    return JANUS_ERR_UNSUPPORTED;
}

size_t colsum_partial_floats(int C) { return size_t(kRowChunks) * size_t(C); }

janus_status colsum(janus_dtype dt, const void* in, int64_t R, int C, int64_t ld, float* out, float* partial,
                    hipStream_t stream, const int32_t* out_idx) {
    if (C <= 0) return JANUS_OK;
    dim3 g1((C + kColTile - 1) / kColTile, kRowChunks);
    TraceScope trace("colsum", 0.0, double(R) * C * double(dtype_size(dt)) + 4.0 * C, stream);
    if (dt == JANUS_BF16)
        hipLaunchKernelGGL(colsum_partial_kernel<bf16_t>, g1, dim3(kColTile), 0, stream,
                           static_cast<const bf16_t*>(in), R, C, ld, partial);
    else
        hipLaunchKernelGGL(colsum_partial_kernel<float>, g1, dim3(kColTile), 0, stream,
                           static_cast<const float*>(in), R, C, ld, partial);
    JANUS_LAUNCH_CHECK();
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + kColTile - 1) / kColTile), dim3(kColTile), 0, stream,
                       partial, C, out, out_idx);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

janus_status zero_fill(void* p, size_t bytes, hipStream_t stream) {
    if (bytes == 0) return JANUS_OK;
    unsigned char* b = static_cast<unsigned char*>(p);
    size_t head = (16 - reinterpret_cast<uintptr_t>(b) % 16) % 16;
    if (head > bytes) head = bytes;
    const size_t n16 = (bytes - head) / 16;
    const size_t nt = bytes - head - n16 * 16;
    unsigned blocks = unsigned(n16 / 256 + 1 < 4096 ? n16 / 256 + 1 : 4096);
    TraceScope trace("zero_fill", 0.0, double(bytes), stream);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, stream, b, head,
                       reinterpret_cast<uint4*>(b + head), n16, b + head + n16 * 16, nt);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

}  // namespace janus
