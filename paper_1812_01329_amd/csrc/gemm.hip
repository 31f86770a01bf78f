// General MFMA contraction with optional row gathers and scatters, plus the
// small reductions used around it.  Every dense contraction of the training
// step that has no fused epilogue goes through here: the hoisted input
// projection of all time steps, the weight gradients (one contraction over
// all packed time steps), input gradients, and the head contractions.
#include "device.hpp"
#include "ops.hpp"

namespace janus {

namespace {

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

    using LA = typename std::conditional<AT, LoaderR<T, Cfg::BM, Cfg::BK, Cfg::NT, AL>,
                                         LoaderK<T, Cfg::BM, Cfg::BK, Cfg::NT, AL>>::type;
    using LB = typename std::conditional<BT, LoaderR<T, Cfg::BN, Cfg::BK, Cfg::NT, AL>,
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

    const int lane = tid & 63, wave = tid >> 6;
    const T* bias = static_cast<const T*>(g.bias);
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
        const int col = n0 + Cfg::wave_col0(wave) + j * 32 + acc_col(lane);
        if (col >= g.N) continue;
        const float bv = bias ? to_f(bias[col]) : 0.f;
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane);
                if (row >= g.M) continue;
                const int64_t crow = g.c_idx ? int64_t(g.c_idx[row]) : int64_t(row);
                const float val = g.alpha * acc[i][j][v] + bv;
                if (g.c_f32) static_cast<float*>(g.C)[crow * g.ldc + col] = val;
                else static_cast<T*>(g.C)[crow * g.ldc + col] = from_f<T>(val);
            }
        }
    }
}

template <typename T, class Cfg, bool AT, bool BT, bool AL>
janus_status launch(const GemmDesc& g, hipStream_t s) {
    dim3 grid((g.N + Cfg::BN - 1) / Cfg::BN, (g.M + Cfg::BM - 1) / Cfg::BM);
    hipLaunchKernelGGL((gemm_kernel<T, Cfg, AT, BT, AL>), grid, dim3(Cfg::NT), Cfg::SMEM_BYTES, s, g);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
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

__global__ __launch_bounds__(kColTile) void colsum_final_kernel(const float* partial, int C, float* out) {
    const int c = blockIdx.x * kColTile + threadIdx.x;
    if (c >= C) return;
    float s = 0.f;
    for (int k = 0; k < kRowChunks; ++k) s += partial[int64_t(k) * C + c];
    out[c] = s;
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

janus_status gemm(const GemmDesc& g, hipStream_t stream) {
    if (g.M <= 0 || g.N <= 0) return JANUS_OK;
    const size_t es = dtype_size(g.dtype);
    const bool aligned = aligned16(g.A, g.lda, es) && aligned16(g.B, g.ldb, es);
    if (g.K <= 0) {
        // empty contraction: C = bias (or 0); handled by the kernel with K = 0
    }
    if (g.dtype == JANUS_BF16) return dispatch<bf16_t, CfgBF16>(g, aligned, stream);
    if (g.dtype == JANUS_F32) return dispatch<float, CfgF32>(g, aligned, stream);
    return JANUS_ERR_UNSUPPORTED;
}

size_t colsum_partial_floats(int C) { return size_t(kRowChunks) * size_t(C); }

janus_status colsum(janus_dtype dt, const void* in, int64_t R, int C, int64_t ld, float* out, float* partial,
                    hipStream_t stream) {
    if (C <= 0) return JANUS_OK;
    dim3 g1((C + kColTile - 1) / kColTile, kRowChunks);
    if (dt == JANUS_BF16)
        hipLaunchKernelGGL(colsum_partial_kernel<bf16_t>, g1, dim3(kColTile), 0, stream,
                           static_cast<const bf16_t*>(in), R, C, ld, partial);
    else
        hipLaunchKernelGGL(colsum_partial_kernel<float>, g1, dim3(kColTile), 0, stream,
                           static_cast<const float*>(in), R, C, ld, partial);
    JANUS_LAUNCH_CHECK();
    hipLaunchKernelGGL(colsum_final_kernel, dim3((C + kColTile - 1) / kColTile), dim3(kColTile), 0, stream,
                       partial, C, out);
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
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, stream, b, head,
                       reinterpret_cast<uint4*>(b + head), n16, b + head + n16 * 16, nt);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

}  // namespace janus
