// Device-side building blocks: bf16 conversion, activations, MFMA
// fragments, global->LDS tile loaders and the MFMA main loop shared by all
// contraction kernels.
//
// Matrix-core mapping (gfx950, wave64):
//   bf16: v_mfma_f32_32x32x16_bf16, one instruction per 16-deep k-step;
//   fp32: v_mfma_f32_32x32x2_f32, eight instructions per 16-deep k-step.
// In both cases lane l of a wave supplies row (l % 32) of the 32x16 operand
// slab and the eight consecutive k values 8 * (l / 32) + [0, 8): A and B use
// the same k assignment, so the contraction is exact whichever physical k
// the hardware pairs.  Accumulator element v of lane l is output row
// 8 * (v / 4) + 4 * (l / 32) + (v % 4), column l % 32.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace janus {

typedef uint16_t bf16_t;   // raw bf16 bit pattern in memory

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// float -> bf16, round to nearest even (NaN kept quiet)
__device__ __forceinline__ bf16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return bf16_t((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return bf16_t(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// logistic sigmoid and tanh from the exponential (accurate to a few ulp of
// float32, far inside the tolerances the path is checked to)
// The reciprocals use the hardware approximation (v_rcp_f32, about 1 ulp)
// rather than an IEEE-rounded division, which costs ten instructions.
__device__ __forceinline__ float sigmoidf_(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }
__device__ __forceinline__ float tanhf_(float x) {
    // tanh(x) = 1 - 2 / (exp(2x) + 1), saturating cleanly for large |x|
    float e = __expf(2.0f * x);
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(e + 1.0f);
}

// ------------------------------------------------------------------ MFMA
template <typename T> struct Frag;
template <> struct Frag<bf16_t> {
    uint4 v;   // 8 bf16
    __device__ __forceinline__ void load(const bf16_t* p) { v = *reinterpret_cast<const uint4*>(p); }
};
template <> struct Frag<float> {
    float4 v0, v1;   // 8 floats
    __device__ __forceinline__ void load(const float* p) {
        v0 = *reinterpret_cast<const float4*>(p);
        v1 = *reinterpret_cast<const float4*>(p + 4);
    }
};

__device__ __forceinline__ void mfma(f32x16_t& acc, const Frag<bf16_t>& a, const Frag<bf16_t>& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                  __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}
__device__ __forceinline__ void mfma(f32x16_t& acc, const Frag<float>& a, const Frag<float>& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v0.x, b.v0.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v0.y, b.v0.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v0.z, b.v0.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v0.w, b.v0.w, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v1.x, b.v1.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v1.y, b.v1.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v1.z, b.v1.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.v1.w, b.v1.w, acc, 0, 0, 0);
}

// accumulator element v of this lane -> row / column inside the 32x32 tile
__device__ __forceinline__ int acc_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }
__device__ __forceinline__ int acc_col(int lane) { return lane & 31; }

// ------------------------------------------------------------- row maps
// A row map turns a tile-relative row into a global row index, or -1 when
// the row is outside the operand.
struct RowsContig {          // rows [0, n) of a dense matrix
    int n;
    __device__ __forceinline__ int64_t operator()(int r) const { return r < n ? int64_t(r) : -1; }
};
struct RowsIndexed {         // rows idx[0 .. n) of a matrix
    const int32_t* idx;
    int n;
    __device__ __forceinline__ int64_t operator()(int r) const { return r < n ? int64_t(idx[r]) : -1; }
};
struct RowsGateMajor {       // rows g * H + u0 + j of a [4H or 5H, K] gate-major matrix
    int H, u0, U;            // tile column n -> gate n / U, unit u0 + n % U
    int gates;
    __device__ __forceinline__ int64_t operator()(int n) const {
        int g = n / U, j = n - g * U;
        return (g < gates && u0 + j < H) ? int64_t(g) * H + u0 + j : -1;
    }
};

// ---------------------------------------------------------- tile loaders
// Swizzled (unpadded) LDS tile: rows of BK elements split into CPR 16-byte
// chunks; chunk q of row r lives at chunk q ^ ((r ^ (r >> 3)) & (CPR - 1)).
// K-contiguous stores (8 lanes per row), transposed block stores (lanes 8
// rows apart) and MFMA fragment reads (32 consecutive rows) then all spread
// over distinct banks.
template <typename T, int BK>
struct Swz {
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int CPR = BK / VEC;
    static_assert((CPR & (CPR - 1)) == 0, "chunks per row must be a power of two");
    __device__ static __forceinline__ int sw(int row) { return (row ^ (row >> 3)) & (CPR - 1); }
    __device__ static __forceinline__ int off(int row, int chunk) { return row * BK + ((chunk ^ sw(row)) * VEC); }
};

// Shared-memory tiles are stored [rows][BK + PAD] with k contiguous so that
// every MFMA fragment is one 16- or 32-byte LDS read.
template <typename T> struct Lds { static constexpr int PAD = 16 / sizeof(T); };

// Operand whose k index is contiguous in memory: elem(r, k) = p[row(r) * ld + k].
template <typename T, int ROWS, int BK, int NT, bool AL, bool SWZ = false>
struct LoaderK {
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int CPR = BK / VEC;
    static constexpr int CH = ROWS * CPR;
    static constexpr int PER = (CH + NT - 1) / NT;
    static constexpr int LD = BK + Lds<T>::PAD;
    const T* rowp[PER];
    uint4 r[PER];

    template <class RowMap>
    __device__ __forceinline__ void init(const T* base, int64_t ld, int r0, const RowMap& rows, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            int c = tid + i * NT;
            int rr = c / CPR;
            int64_t g = (CH % NT == 0 || c < CH) ? rows(r0 + rr) : -1;
            rowp[i] = g >= 0 ? base + g * ld + (c % CPR) * VEC : nullptr;
        }
    }
    __device__ __forceinline__ void load(int k0, int K, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            int c = tid + i * NT;
            int kk = k0 + (c % CPR) * VEC;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (rowp[i]) {
                const T* p = rowp[i] + k0;
                if (AL && kk + VEC <= K) {
                    v = *reinterpret_cast<const uint4*>(p);
                } else {
                    T tmp[VEC];
#pragma unroll
                    for (int j = 0; j < VEC; ++j) tmp[j] = (kk + j < K) ? p[j] : T(0);
                    __builtin_memcpy(&v, tmp, 16);
                }
            }
            r[i] = v;
        }
    }
    __device__ __forceinline__ void store(T* s, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            int c = tid + i * NT;
            if (CH % NT == 0 || c < CH) {
                const int o = SWZ ? Swz<T, BK>::off(c / CPR, c % CPR) : (c / CPR) * LD + (c % CPR) * VEC;
                *reinterpret_cast<uint4*>(s + o) = r[i];
            }
        }
    }
};

// Transposed operand read in square VEC x VEC blocks: each task loads VEC
// consecutive k rows of VEC contiguous elements (16 bytes each) and writes
// VEC rows of VEC consecutive k values (16 bytes each) into the k-contiguous
// tile, transposing in registers.  elem(r, k) = p[krow(k) * ld + r0 + r].
template <typename T, int ROWS, int BK, int NT, bool AL, bool SWZ = false>
struct LoaderT {
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr int RCH = ROWS / VEC;
    static constexpr int KCH = BK / VEC;
    static constexpr int TASKS = RCH * KCH;
    static constexpr int PER = (TASKS + NT - 1) / NT;
    static constexpr int LD = BK + Lds<T>::PAD;
    static_assert(ROWS % VEC == 0 && BK % VEC == 0, "tile must be a multiple of the vector width");
    const T* base;
    int64_t ld;
    const int32_t* kidx;
    int rbase, nrows;
    uint4 r[PER][VEC];

    __device__ __forceinline__ void init(const T* b, int64_t l, const int32_t* ki, int r0, int n) {
        base = b; ld = l; kidx = ki; rbase = r0; nrows = n;
    }
    __device__ __forceinline__ void load(int k0, int K, int tid) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int c = tid + i * NT;
            const int rc = (c % RCH) * VEC;
            const int kb = (c / RCH) * VEC;
            const int gr = rbase + rc;
            const bool task = (TASKS % NT == 0 || c < TASKS);
#pragma unroll
            for (int j = 0; j < VEC; ++j) {
                uint4 v = make_uint4(0, 0, 0, 0);
                const int k = k0 + kb + j;
                if (task && k < K && gr < nrows) {
                    const int64_t krow = kidx ? int64_t(kidx[k]) : int64_t(k);
                    const T* p = base + krow * ld + gr;
                    if (AL && gr + VEC <= nrows) {
                        v = *reinterpret_cast<const uint4*>(p);
                    } else {
                        T tmp[VEC];
#pragma unroll
                        for (int e = 0; e < VEC; ++e) tmp[e] = (gr + e < nrows) ? p[e] : T(0);
                        __builtin_memcpy(&v, tmp, 16);
                    }
                }
                r[i][j] = v;
            }
        }
    }
    __device__ __forceinline__ void store(T* s, int tid) const {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int c = tid + i * NT;
            if (!(TASKS % NT == 0 || c < TASKS)) continue;
            const int rc = (c % RCH) * VEC;
            const int kb = (c / RCH) * VEC;
            const uint32_t* w[VEC];
#pragma unroll
            for (int j = 0; j < VEC; ++j) w[j] = reinterpret_cast<const uint32_t*>(&r[i][j]);
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                uint4 o;
                uint32_t* od = reinterpret_cast<uint32_t*>(&o);
                if constexpr (sizeof(T) == 2) {
                    const int sh = 16 * (e & 1);
#pragma unroll
                    for (int d = 0; d < 4; ++d)
                        od[d] = ((w[2 * d][e >> 1] >> sh) & 0xffffu) | (((w[2 * d + 1][e >> 1] >> sh) & 0xffffu) << 16);
                } else {
#pragma unroll
                    for (int d = 0; d < 4; ++d) od[d] = w[d][e];
                }
                const int so = SWZ ? Swz<T, BK>::off(rc + e, kb / VEC) : (rc + e) * LD + kb;
                *reinterpret_cast<uint4*>(s + so) = o;
            }
        }
    }
};

// ------------------------------------------------------------ main loop
// C_tile[BM x BN] = sum_k A(m, k) B(n, k) for one workgroup tile, WGM x WGN
// waves, each owning a (BM / WGM) x (BN / WGN) block of 32x32 MFMA tiles.
template <typename T, int BM_, int BN_, int BK_, int WGM_, int WGN_>
struct TileCfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WGM = WGM_, WGN = WGN_;
    static constexpr int NT = WGM * WGN * 64;
    static constexpr int WTM = BM / WGM, WTN = BN / WGN;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int LD = BK + Lds<T>::PAD;
    static constexpr int SMEM_BYTES = (BM + BN) * LD * int(sizeof(T));
    static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be a multiple of 32");
    static_assert(BK % 16 == 0, "BK must be a multiple of 16");
    __device__ static __forceinline__ int wave_row0(int wave) { return (wave / WGN) * WTM; }
    __device__ static __forceinline__ int wave_col0(int wave) { return (wave % WGN) * WTN; }
};

template <class Cfg, typename T, class LA, class LB>
__device__ __forceinline__ void mma_mainloop(f32x16_t (&acc)[Cfg::FM][Cfg::FN], LA& la, LB& lb,
                                             int K, T* sA, T* sB, int tid) {
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    if (K <= 0) return;
    const int row_in = lane & 31, kq = (lane >> 5) * 8;
    const T* pa = sA + (Cfg::wave_row0(wave) + row_in) * Cfg::LD + kq;
    const T* pb = sB + (Cfg::wave_col0(wave) + row_in) * Cfg::LD + kq;
    la.load(0, K, tid);
    lb.load(0, K, tid);
    for (int k0 = 0; k0 < K; k0 += Cfg::BK) {
        __syncthreads();
        la.store(sA, tid);
        lb.store(sB, tid);
        __syncthreads();
        if (k0 + Cfg::BK < K) {
            la.load(k0 + Cfg::BK, K, tid);
            lb.load(k0 + Cfg::BK, K, tid);
        }
#pragma unroll
        for (int ks = 0; ks < Cfg::BK / 16; ++ks) {
            Frag<T> fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i) fa[i].load(pa + i * 32 * Cfg::LD + ks * 16);
#pragma unroll
            for (int j = 0; j < Cfg::FN; ++j) fb[j].load(pb + j * 32 * Cfg::LD + ks * 16);
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
                for (int j = 0; j < Cfg::FN; ++j) mfma(acc[i][j], fa[i], fb[j]);
        }
    }
}

// Double-buffered variant: two LDS stages, one barrier per k tile.  The
// next tile's global loads are in flight while the current tile is
// multiplied; `smem` holds 2 * (BM + BN) * LD elements.
template <class Cfg, typename T, class LA, class LB>
__device__ __forceinline__ void mma_mainloop_db(f32x16_t (&acc)[Cfg::FM][Cfg::FN], LA& la, LB& lb, int K, T* smem,
                                                int tid) {
    constexpr int STAGE = (Cfg::BM + Cfg::BN) * Cfg::LD;
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    if (K <= 0) return;
    const int row_in = lane & 31, kq = (lane >> 5) * 8;
    const int a_off = (Cfg::wave_row0(wave) + row_in) * Cfg::LD + kq;
    const int b_off = Cfg::BM * Cfg::LD + (Cfg::wave_col0(wave) + row_in) * Cfg::LD + kq;
    la.load(0, K, tid);
    lb.load(0, K, tid);
    la.store(smem, tid);
    lb.store(smem + Cfg::BM * Cfg::LD, tid);
    __syncthreads();
    const int nk = (K + Cfg::BK - 1) / Cfg::BK;
    for (int it = 0; it < nk; ++it) {
        T* cur = smem + (it & 1) * STAGE;
        T* nxt = smem + ((it + 1) & 1) * STAGE;
        const bool more = it + 1 < nk;
        if (more) {
            la.load((it + 1) * Cfg::BK, K, tid);
            lb.load((it + 1) * Cfg::BK, K, tid);
        }
#pragma unroll
        for (int ks = 0; ks < Cfg::BK / 16; ++ks) {
            Frag<T> fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i) fa[i].load(cur + a_off + i * 32 * Cfg::LD + ks * 16);
#pragma unroll
            for (int j = 0; j < Cfg::FN; ++j) fb[j].load(cur + b_off + j * 32 * Cfg::LD + ks * 16);
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
                for (int j = 0; j < Cfg::FN; ++j) mfma(acc[i][j], fa[i], fb[j]);
        }
        if (more) {
            la.store(nxt, tid);
            lb.store(nxt + Cfg::BM * Cfg::LD, tid);
        }
        __syncthreads();
    }
}

// Double-buffered main loop over swizzled, unpadded LDS tiles (bf16).
// `smem` holds 2 * (BM + BN) * BK elements.
template <class Cfg, class LA, class LB>
__device__ __forceinline__ void mma_mainloop_swz(f32x16_t (&acc)[Cfg::FM][Cfg::FN], LA& la, LB& lb, int K,
                                                 bf16_t* smem, int tid) {
    using S = Swz<bf16_t, Cfg::BK>;
    constexpr int STAGE = (Cfg::BM + Cfg::BN) * Cfg::BK;
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
    if (K <= 0) return;
    int arow[Cfg::FM], asw[Cfg::FM], brow[Cfg::FN], bsw[Cfg::FN];
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i) {
        const int r = Cfg::wave_row0(wave) + i * 32 + (lane & 31);
        arow[i] = r * Cfg::BK;
        asw[i] = S::sw(r);
    }
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
        const int r = Cfg::wave_col0(wave) + j * 32 + (lane & 31);
        brow[j] = Cfg::BM * Cfg::BK + r * Cfg::BK;
        bsw[j] = S::sw(r);
    }
    const int kh = lane >> 5;
    la.load(0, K, tid);
    lb.load(0, K, tid);
    la.store(smem, tid);
    lb.store(smem + Cfg::BM * Cfg::BK, tid);
    __syncthreads();
    const int nk = (K + Cfg::BK - 1) / Cfg::BK;
    for (int it = 0; it < nk; ++it) {
        bf16_t* cur = smem + (it & 1) * STAGE;
        bf16_t* nxt = smem + ((it + 1) & 1) * STAGE;
        const bool more = it + 1 < nk;
        if (more) {
            la.load((it + 1) * Cfg::BK, K, tid);
            lb.load((it + 1) * Cfg::BK, K, tid);
        }
#pragma unroll
        for (int ks = 0; ks < Cfg::BK / 16; ++ks) {
            const int q = 2 * ks + kh;
            Frag<bf16_t> fa[Cfg::FM], fb[Cfg::FN];
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i) fa[i].load(cur + arow[i] + ((q ^ asw[i]) << 3));
#pragma unroll
            for (int j = 0; j < Cfg::FN; ++j) fb[j].load(cur + brow[j] + ((q ^ bsw[j]) << 3));
#pragma unroll
            for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
                for (int j = 0; j < Cfg::FN; ++j) mfma(acc[i][j], fa[i], fb[j]);
        }
        if (more) {
            la.store(nxt, tid);
            lb.store(nxt + Cfg::BM * Cfg::BK, tid);
        }
        __syncthreads();
    }
}

}  // namespace janus
