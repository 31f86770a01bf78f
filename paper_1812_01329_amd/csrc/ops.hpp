// Internal launchers shared between the library's translation units.
#pragma once

#include <vector>

#include "runtime.hpp"

namespace janus {

// C[M, N] = alpha * sum_k A(m, k) B(n, k) + bias[n]
//  A(m, k) = A[a_row(m) * lda + k]        (a_t = false; a_idx maps m, or NULL)
//          = A[a_row(k) * lda + m]        (a_t = true;  a_idx maps k, or NULL)
//  B(n, k) = B[b_row(n) * ldb + k]        (b_t = false; b_idx maps n, or NULL)
//          = B[b_row(k) * ldb + n]        (b_t = true;  b_idx maps k, or NULL)
//  C row m is written at C[c_row(m) * ldc + n] (c_idx maps m, or NULL), in
//  float32 when c_f32, else in the operand dtype.  bias (dtype) may be NULL.
// Supported layouts: (a_t, b_t) = (0, 0), (0, 1), (1, 1).
struct GemmDesc {
    janus_dtype dtype = JANUS_BF16;
    int M = 0, N = 0, K = 0;
    bool a_t = false;
    const void* A = nullptr;
    int64_t lda = 0;
    const int32_t* a_idx = nullptr;
    bool b_t = false;
    const void* B = nullptr;
    int64_t ldb = 0;
    const int32_t* b_idx = nullptr;
    void* C = nullptr;
    int64_t ldc = 0;
    const int32_t* c_idx = nullptr;
    bool c_f32 = true;
    const void* bias = nullptr;
    float alpha = 1.0f;
    // rows of A / B behind a_idx / b_idx (bounds the gathered offsets; 0 =
    // unknown, which keeps a gathered operand off the fast path)
    int64_t a_src_rows = 0, b_src_rows = 0;
    // (a_t / b_t false only) rows of A / B hold zeros from K up to the next
    // multiple of 8, so they may be read in whole 16-byte chunks
    bool a_zero_pad = false, b_zero_pad = false;
    // device scratch for transposed operand copies and split-K partials,
    // gemm_scratch_bytes(g) bytes; with less, a slower path that needs none
    // is taken
    void* scratch = nullptr;
    size_t scratch_bytes = 0;
};

janus_status gemm(const GemmDesc& g, hipStream_t stream);
size_t gemm_scratch_bytes(const GemmDesc& g);
// scratch enough for the contraction with any K up to g.K, any operand
// alignment and any gathered-row count (for sizing workspaces in advance)
size_t gemm_scratch_bound(const GemmDesc& g);

// Projection + MSE in one pass (bf16, K-contiguous h [M, K] and W [N, K]):
// d = h W^T + bias - tgt, dY = scale d (bf16, [M, N]), part[0, mt * nt) =
// per-workgroup sums of d^2 (mt, nt = tiles of 256 rows / columns), db[N] =
// column sums of dY (float32, fixed order).  part needs gemm_mse_partials
// floats.  gemm_mse_fast tells whether the shape and operands qualify.
bool gemm_mse_fast(int M, int N, int K, const void* h, const void* W);
size_t gemm_mse_partials(int M, int N);
janus_status gemm_mse(int M, int N, int K, const void* h, const void* W, const void* bias, const void* tgt, void* dY,
                      float scale, float* part, float* db, hipStream_t stream);

// out[c * ld_out + r] = in[row(r) * ld_in + c] (bf16), row(r) = idx[r] or r,
// for r < R, c < C; columns [R, R_pad) of each output row are zero.  C,
// ld_in, ld_out, R_pad must be multiples of 8 and pointers 16-byte aligned.
janus_status transpose_bf16(const void* in, int64_t ld_in, const int32_t* idx, int64_t R, int C, void* out,
                            int64_t ld_out, int64_t R_pad, hipStream_t stream);

// out[c] = sum over rows r < R of in[r * ld + c] (float32 result), for
// c < C; deterministic two-pass reduction using `partial` scratch of
// colsum_partial_floats(C) floats.
size_t colsum_partial_floats(int C);
janus_status colsum(janus_dtype dt, const void* in, int64_t R, int C, int64_t ld, float* out,
                    float* partial, hipStream_t stream, const int32_t* out_idx = nullptr);

// clear `bytes` bytes of device memory (a kernel, so it may be captured)
janus_status zero_fill(void* p, size_t bytes, hipStream_t stream);

// dE [V, H] float32 = 0, then dE[ids[r]] = sum of dx[r] over the rows with
// that id, in ascending r (deterministic, no atomics).  The rows are grouped
// by id on the host (a stable counting sort of ids_host, already range
// checked) and the groups go to the device in `seg_dev`, a region of
// embed_seg_ints(rows) int32 of device memory the caller provides (a
// workspace piece); one workgroup then sums each group.
size_t embed_seg_ints(int rows);
// The host part: rows grouped by id into seg = order[rows], off[nseg + 1],
// sid[nseg] (ids ascending, rows ascending within an id); returns nseg.
int embed_segments(const int32_t* ids_host, int rows, int V, std::vector<int32_t>& seg);
janus_status embed_backward(janus_dtype dt, const void* dx, const int32_t* ids_host, int rows, int H, float* dE, int V,
                            int32_t* seg_dev, hipStream_t stream);

}  // namespace janus
