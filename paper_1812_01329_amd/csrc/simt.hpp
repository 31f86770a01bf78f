// Small float32 contractions for the tree steps (SIMT, K split over waves)
// and a float32 transpose, shared by the TreeLSTM, TreeRNN and Child-Sum
// TreeLSTM.
#pragma once

#include "device.hpp"
#include "runtime.hpp"

namespace janus {
namespace {

// The contractions of the tree step are small: per level a few to a few
// hundred rows against a 750 x 300 weight, and the weight gradients with
// K = a few hundred nodes.  Tiles that walk K serially leave most of the GPU
// idle and wait on one load round trip after another.  Instead each block
// computes 8 rows x 64 columns of C = a . B with K split over its 8 waves:
//   a(m, k) = A[arow(m) * lda + k]  (arow(m) = a_idx[m] or m), or with AT
//             A[k * lda + m];
//   B row k = B + brow(k) * ldb      (brow(k) = b_idx[k] or k), N contiguous.
// The block's slab of a (8 rows, K in chunks of 1024) is staged in LDS and
// read as broadcasts; each lane owns one column and streams its B entries
// from the L2 (every row block reads the same B), 16 loads in flight.  The
// waves' partial sums are added through LDS in wave order.  Epilogues: rows
// of C (+ bias); the backward's [dh_L; dh_R], whose two halves go to the
// rows of the two children; or (TreeRNN forward) h = tanh(. + bias), saved
// in C and sent to the parent's [h_L; h_R] row or to h_root.  With
// kSimtTanhGrad the a slab is da = a (1 - s^2) for a second operand s of
// a's layout (TreeRNN backward: dh and h), and column block 0 also stores da.
constexpr int kSimtRows = 8, kSimtCols = 64, kSimtWaves = 8, kSimtKc = 1024;
enum SimtEpi { kSimtStore = 0, kSimtChildren = 1, kSimtTanhSend = 2 };
enum SimtAMode { kSimtPlain = 0, kSimtTanhGrad = 1 };

// operands of the TreeRNN epilogue and a-transform
struct SimtExtra {
    float* HLR = nullptr;        // kSimtTanhSend: [h_L; h_R] rows of internal nodes
    float* root = nullptr;       //                h_root
    int M0 = 0;                  //                first internal position
    const float* S = nullptr;    // kSimtTanhGrad: h, same layout as a
    float* D = nullptr;          //                da out, same layout as a
};

template <bool AT, int EPI, int AMODE = kSimtPlain>
__global__ __launch_bounds__(64 * kSimtWaves) void simt_gemm_kernel(int M, int N, int K, const float* A, int64_t lda,
                                                                    const int32_t* a_idx, const float* B, int64_t ldb,
                                                                    const int32_t* b_idx, const float* bias, float* C,
                                                                    int64_t ldc, const int32_t* lchild,
                                                                    const int32_t* rchild, int H, SimtExtra x) {
    __shared__ __align__(16) float sA[kSimtKc][kSimtRows];
    __shared__ float red[kSimtWaves][kSimtRows][kSimtCols];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = blockIdx.x * kSimtCols + lane;
    const int m0 = blockIdx.y * kSimtRows;
    float acc[kSimtRows];
#pragma unroll
    for (int r = 0; r < kSimtRows; ++r) acc[r] = 0.f;
    for (int k0 = 0; k0 < K; k0 += kSimtKc) {
        const int kc = min(kSimtKc, K - k0);
        __syncthreads();
        for (int i = tid; i < kSimtKc * kSimtRows; i += 64 * kSimtWaves) {
            // AT: consecutive threads read consecutive m of one k; otherwise
            // consecutive k of one row
            const int r = AT ? i % kSimtRows : i / kSimtKc, kk = AT ? i / kSimtRows : i % kSimtKc;
            const int m = m0 + r;
            float v = 0.f;
            if (m < M && kk < kc) {
                if constexpr (AMODE == kSimtTanhGrad) {
                    const int64_t o = int64_t(m) * lda + k0 + kk;
                    const float h = x.S[o];
                    v = A[o] * (1.f - h * h);
                    if (blockIdx.x == 0) x.D[o] = v;
                } else if (AT) {
                    v = A[int64_t(k0 + kk) * lda + m];
                } else {
                    v = A[(a_idx ? int64_t(a_idx[m]) : int64_t(m)) * lda + k0 + kk];
                }
            }
            sA[kk][r] = v;
        }
        __syncthreads();
        const int kb = wave * kc / kSimtWaves, ke = (wave + 1) * kc / kSimtWaves;
        if (n < N) {
#pragma unroll 16
            for (int kk = kb; kk < ke; ++kk) {
                const int k = k0 + kk;
                const float bv = B[(b_idx ? int64_t(b_idx[k]) : int64_t(k)) * ldb + n];
                const float4 a0 = *reinterpret_cast<const float4*>(&sA[kk][0]);
                const float4 a1 = *reinterpret_cast<const float4*>(&sA[kk][4]);
                acc[0] += a0.x * bv; acc[1] += a0.y * bv; acc[2] += a0.z * bv; acc[3] += a0.w * bv;
                acc[4] += a1.x * bv; acc[5] += a1.y * bv; acc[6] += a1.z * bv; acc[7] += a1.w * bv;
            }
        }
    }
#pragma unroll
    for (int r = 0; r < kSimtRows; ++r) red[wave][r][lane] = acc[r];
    __syncthreads();
    // thread (row r = wave, column lane) adds the waves' parts in order
    const int r = wave, m = m0 + r;
    if (m >= M || n >= N) return;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kSimtWaves; ++w) sum += red[w][r][lane];
    if constexpr (EPI == kSimtTanhSend) {
        // lchild / rchild carry the parent slot and the tree index of each row
        const float h = tanhf_(sum + bias[n]);
        C[int64_t(m) * ldc + n] = h;
        const int par = lchild[m];
        if (par >= 0) x.HLR[int64_t((par >> 1) - x.M0) * 2 * N + (par & 1) * N + n] = h;
        else x.root[int64_t(rchild[m]) * N + n] = h;
    } else if constexpr (EPI == kSimtChildren) {
        if (n < H) C[int64_t(lchild[m]) * H + n] = sum;
        else C[int64_t(rchild[m]) * H + n - H] = sum;
    } else {
        C[int64_t(m) * ldc + n] = sum + (bias ? bias[n] : 0.f);
    }
}

template <bool AT, int EPI, int AMODE = kSimtPlain>
janus_status simt_gemm(const char* label, int M, int N, int K, const float* A, int64_t lda, const int32_t* a_idx,
                       const float* B, int64_t ldb, const int32_t* b_idx, const float* bias, float* C, int64_t ldc,
                       hipStream_t st, const int32_t* lchild = nullptr, const int32_t* rchild = nullptr, int H = 0,
                       SimtExtra x = SimtExtra()) {
    if (M <= 0 || N <= 0) return JANUS_OK;
    dim3 grid(unsigned((N + kSimtCols - 1) / kSimtCols), unsigned((M + kSimtRows - 1) / kSimtRows));
    TraceScope trace(label, 2.0 * M * N * double(K), 4.0 * (double(M) * K + double(K) * N + double(M) * N), st);
    hipLaunchKernelGGL((simt_gemm_kernel<AT, EPI, AMODE>), grid, dim3(64 * kSimtWaves), 0, st, M, N, K, A, lda, a_idx,
                       B, ldb, b_idx, bias, C, ldc, lchild, rchild, H, x);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

// out[c * R + r] = in[r * C + c], float32
__global__ void transpose_f32_kernel(const float* in, int R, int C, float* out) {
    __shared__ float t[32][33];
    const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
    for (int i = threadIdx.y; i < 32; i += 8) {
        const int r = r0 + i, c = c0 + threadIdx.x;
        if (r < R && c < C) t[i][threadIdx.x] = in[int64_t(r) * C + c];
    }
    __syncthreads();
    for (int i = threadIdx.y; i < 32; i += 8) {
        const int c = c0 + i, r = r0 + threadIdx.x;
        if (r < R && c < C) out[int64_t(c) * R + r] = t[threadIdx.x][i];
    }
}

janus_status transpose_f32(const float* in, int R, int C, float* out, hipStream_t st) {
    TraceScope trace("transpose_f32", 0.0, 8.0 * R * double(C), st);
    hipLaunchKernelGGL(transpose_f32_kernel, dim3(unsigned((C + 31) / 32), unsigned((R + 31) / 32)), dim3(32, 8), 0, st,
                       in, R, C, out);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

}  // namespace
}  // namespace janus
