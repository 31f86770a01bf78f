// General MFMA contraction with optional row gathers and scatters, plus the
// small reductions used around it.  Every dense contraction of the training
// step that has no fused epilogue goes through here: the hoisted input
// projection of all time steps, the weight gradients (one contraction over
// all packed time steps), input gradients, and the head contractions.
#include <algorithm>
#include <cstdlib>

#include "device.hpp"
#include "ops.hpp"

namespace janus {

namespace {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

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

// ------------------------------------------------------------ fast NT path
// C[M, N] = A[M, K] . B[N, K]^T for bf16 operands whose K runs contiguously
// (rows of A and B), the one layout every large contraction of the step is
// brought into.  256 x 256 x 64 tiles, 8 waves in a 2 x 4 grid (128 x 64
// each), two LDS stages filled by buffer loads that write LDS directly (no
// register staging), 16-byte chunks XOR-swizzled by row so that the MFMA
// fragment reads are conflict-free.  Rows past M / N and k past K read as
// zero through the buffer range check, so ragged shapes need no separate
// path.  Optional K split: each split writes float32 partials that a second
// kernel sums in split order (deterministic).
struct NtCfg {
    static constexpr int BM = 256, BN = 256, BK = 64, NT = 512;
    static constexpr int WGM = 2, WGN = 4, WTM = BM / WGM, WTN = BN / WGN;
    static constexpr int FM = WTM / 32, FN = WTN / 32;
    static constexpr int CPR = BK / 8;                        // 16-byte chunks per tile row
    static constexpr int RPI = 64 / CPR;                      // tile rows per wave-wide load
    static constexpr int LOADS = BM / RPI / (NT / 64 / 2);    // loads per wave per stage
    static constexpr int STAGE = (BM + BN) * BK;              // bf16 elements per stage
    __device__ static __forceinline__ int wave_row0(int wave) { return (wave / WGN) * WTM; }
    __device__ static __forceinline__ int wave_col0(int wave) { return (wave % WGN) * WTN; }
};
static_assert(NtCfg::LOADS == 8, "load schedule assumes 8 loads per wave per stage");

struct NtArgs {
    const bf16_t* A;
    const bf16_t* B;
    int64_t lda, ldb;
    const int32_t* a_idx;       // gathered rows (whole-matrix buffer base), or NULL
    const int32_t* b_idx;
    int M, N, K;
    int mt, nt, splits, ktiles_per_split;
    float* partial;             // [splits, M, N] when splits > 1
    // MSE epilogue: d = C + bias - tgt; dY = scale d (bf16); per workgroup
    // sum of d^2 into part_sq[block] and column sums of dY into
    // part_col[m-tile * N + col]
    const bf16_t* tgt;
    bf16_t* dY;
    float scale;
    float* part_sq;
    float* part_col;
    // plain store epilogue in 16-byte row pieces through LDS (N and ldc
    // multiples of 8, C and the bias 16-byte aligned)
    int vec_store;
    // persistent launch: the number of tiles; the grid (a multiple of 8)
    // walks them
    int ntiles;
};

enum NtEpilogue { kEpiStore = 0, kEpiPartial = 1, kEpiMse = 2 };

// Element v (0..15) of a 32 x 32 block held as four 16x16x32 MFMA products:
// sub-block v / 4 = (a, b) covers rows 16 a + [0, 16), columns 16 b + [0, 16),
// and its element v % 4 of lane l sits at row 4 (l / 16) + v % 4, column l % 16.
__device__ __forceinline__ int nt_row(int v, int lane) { return 16 * (v >> 3) + 4 * (lane >> 4) + (v & 3); }
__device__ __forceinline__ int nt_col(int v, int lane) { return 16 * ((v >> 2) & 1) + (lane & 15); }

constexpr uint32_t kNtOutOfRange = 0x80000000u;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// PERSIST (plain store epilogue through LDS only): a grid of one workgroup
// per CU walks the tiles, and each workgroup issues the first K block of its
// next tile before the epilogue of the current one, so the load latency of a
// tile's start hides behind the previous tile's stores.
template <typename OutT, bool SCATTER, int EPI, bool PERSIST = false>
__global__ __launch_bounds__(NtCfg::NT) __attribute__((amdgpu_waves_per_eu(2, 2)))
void gemm_nt_fast_kernel(NtArgs p, GemmDesc g) {
    static_assert(!PERSIST || EPI == kEpiStore, "persistent tiles: plain store epilogue only");
    using C_ = NtCfg;
    // The two stages are separate LDS objects and the main loop is unrolled
    // by two, so every fragment read names the stage it reads: the compiler
    // can then tell them apart from the direct-to-LDS loads filling the other
    // stage and does not wait for those loads before reading.
    __shared__ __align__(16) bf16_t stage0[C_::STAGE];
    __shared__ __align__(16) bf16_t stage1[C_::STAGE];
    // wave index made visibly uniform, so that everything derived from it
    // (operand choice, buffer descriptor, LDS destinations) stays scalar
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // block -> (split, tile): consecutive blocks go to the 8 XCDs in turn, so
    // renumber to give each XCD a contiguous range, then walk the tiles in
    // groups of 4 M-tiles so neighbours share B tiles in that XCD's L2.  A
    // persistent workgroup w (on XCD w mod 8) takes blocks w / 8 + i G / 8 of
    // its XCD's range (grid G), in the same order.
    const int ntot = PERSIST ? p.ntiles : int(gridDim.x);
    const int per_xcd = ntot / 8, xstep = int(gridDim.x) / 8;
    int vb;
    if constexpr (PERSIST) {
        vb = int(blockIdx.x / 8);   // index within the XCD's range
    } else {
        vb = blockIdx.x;
        if (ntot % 8 == 0) vb = (vb % 8) * (ntot / 8) + vb / 8;
    }
    const int tiles = p.mt * p.nt;
    constexpr int GM = 4;
    const int in_group = GM * p.nt;
    int split = 0, m0 = 0, n0 = 0, kt0 = 0, nk = 0;
    auto map_tile = [&](int b, int& sp, int& tm0, int& tn0, int& tk0, int& tnk) {
        sp = b / tiles;
        const int t = b % tiles;
        const int first_m = (t / in_group) * GM;
        const int gsz = min(p.mt - first_m, GM);
        tm0 = (first_m + (t % in_group) % gsz) * C_::BM;
        tn0 = ((t % in_group) / gsz) * C_::BN;
        tk0 = sp * p.ktiles_per_split;
        tnk = max(0, min(p.ktiles_per_split, (p.K + C_::BK - 1) / C_::BK - tk0));
    };
    auto block_of = [&](int i) { return PERSIST ? int(blockIdx.x % 8) * per_xcd + i : i; };
    map_tile(block_of(vb), split, m0, n0, kt0, nk);

    // this lane's loads: waves 0-3 fill the A tile, 4-7 the B tile; load j
    // of wave w covers tile rows 64 (w % 4) + 8 j + lane / 8, physical chunk
    // lane % 8, holding logical chunk (lane % 8) ^ (row % 8)
    const bool isA = wave < 4;
    const int lw = wave & 3;
    const int rows = isA ? p.M : p.N;
    const int64_t ld = isA ? p.lda : p.ldb;
    const int32_t* idx = isA ? p.a_idx : p.b_idx;
    const bf16_t* src = isA ? p.A : p.B;
    const int kchunk = ((lane & 7) ^ (lane >> 3)) * 8;
    uint32_t rowoff[C_::LOADS];
    __amdgpu_buffer_rsrc_t rs;
    auto setup_loads = [&](int tm0, int tn0) {
        const int row0 = isA ? tm0 : tn0;
#pragma unroll
        for (int j = 0; j < C_::LOADS; ++j) {
            const int r = lw * 64 + j * 8 + (lane >> 3);
            const int gr = row0 + r;
            const int64_t src_row = idx ? int64_t(idx[min(gr, rows - 1)]) : int64_t(r);
            rowoff[j] = gr < rows ? uint32_t(src_row * ld * 2) : kNtOutOfRange;
        }
        const bf16_t* base = idx ? src : src + int64_t(row0) * ld;
        rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(base), (short)0, 0x7fffffff, 0x00020000);
    };
    setup_loads(m0, n0);
    const int lds_op = (isA ? 0 : C_::BM * C_::BK) + lw * 64 * C_::BK;

    // Offsets with bit 31 set are out of range (the descriptor covers 2^31 - 1
    // bytes and every in-range offset is below 2^31), so masking is an OR.
    auto issue = [&](int kt, bf16_t* stage) {
        const int k = kt * C_::BK + kchunk;
        const uint32_t kbad = k < p.K ? 0u : kNtOutOfRange;
        bf16_t* dst = stage + lds_op;
#pragma unroll
        for (int j = 0; j < C_::LOADS; ++j) {
            const uint32_t off = (rowoff[j] + uint32_t(k) * 2u) | kbad;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t)(dst + j * 8 * C_::BK), 16, off, 0, 0, 0);
        }
    };

    const int wr0 = C_::wave_row0(wave), wc0 = C_::wave_col0(wave);
    // A wave's 128 x 64 block is 8 x 4 products of 16 x 16 (16x16x32 MFMA:
    // the same operand bytes per flop as 32x32x16, measured 5-7 % faster on
    // the step's shapes).  acc[i][j][s] holds sub-block (s / 2, s % 2) of the
    // 32 x 32 block (i, j); element v of a 32 x 32 block is acc[i][j][v / 4][v % 4],
    // at row nt_row(v, lane), column nt_col(v, lane).
    f32x4_t acc[C_::FM][C_::FN][4];
    // fragment rows; the row swizzle is row % 8 = lane % 8 for every fragment
    const int sw = lane & 7, kq = lane >> 4;
    int arow[2 * C_::FM], brow[2 * C_::FN];
#pragma unroll
    for (int i = 0; i < 2 * C_::FM; ++i) arow[i] = (wr0 + i * 16 + (lane & 15)) * C_::BK;
#pragma unroll
    for (int j = 0; j < 2 * C_::FN; ++j) brow[j] = C_::BM * C_::BK + (wc0 + j * 16 + (lane & 15)) * C_::BK;

    auto compute = [&](const bf16_t* cur) {
#pragma unroll
        for (int ks = 0; ks < C_::BK / 32; ++ks) {
            const int q = 4 * ks + kq;
            // the B fragments, then the A fragments in two halves (fewer live
            // registers: the persistent variant holds the next tile's loads too)
            uint4 fb[2 * C_::FN];
#pragma unroll
            for (int j = 0; j < 2 * C_::FN; ++j) fb[j] = *reinterpret_cast<const uint4*>(cur + brow[j] + ((q ^ sw) << 3));
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint4 fa[C_::FM];
#pragma unroll
                for (int i = 0; i < C_::FM; ++i)
                    fa[i] = *reinterpret_cast<const uint4*>(cur + arow[h * C_::FM + i] + ((q ^ sw) << 3));
#pragma unroll
                for (int i = 0; i < C_::FM; ++i)
#pragma unroll
                    for (int j = 0; j < 2 * C_::FN; ++j) {
                        const int ii = h * C_::FM + i;
                        f32x4_t& a = acc[ii / 2][j / 2][2 * (ii % 2) + j % 2];
                        a = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, fa[i]),
                                                                    __builtin_bit_cast(bf16x8_t, fb[j]), a, 0, 0, 0);
                    }
            }
        }
    };

    // Each half: wait until this wave's loads of the current stage have
    // landed and its reads of the other stage have returned, barrier (so the
    // same holds for every wave), refill the other stage, compute on the
    // current one.  The scheduling barriers keep the compiler from moving
    // LDS reads across the barrier or sinking the refill below the compute
    // (which would leave nothing to overlap); a plain __syncthreads would
    // instead wait for the refill too.
    auto sync = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
    };
    if (nk > 0) issue(kt0, stage0);
    while (true) {
#pragma unroll
    for (int i = 0; i < C_::FM; ++i)
#pragma unroll
        for (int j = 0; j < C_::FN; ++j)
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) acc[i][j][s4] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    int it = 0;
    for (; it + 1 < nk; it += 2) {
        sync();
        issue(kt0 + it + 1, stage1);
        __builtin_amdgcn_sched_barrier(0);
        compute(stage0);
        sync();
        if (it + 2 < nk) issue(kt0 + it + 2, stage0);
        __builtin_amdgcn_sched_barrier(0);
        compute(stage1);
    }
    if (it < nk) {
        sync();
        compute(stage0);
    }
    // persistent: the next tile's first K block goes to stage 0 before this
    // tile's epilogue (which then stages through stage 1 only)
    bool more = false;
    int nsplit = 0, nm0 = 0, nn0 = 0, nkt0 = 0, nnk = 0;
    if constexpr (PERSIST) {
        vb += xstep;
        more = vb < per_xcd;
        sync();   // every wave is done reading both stages
        if (more) {
            map_tile(block_of(vb), nsplit, nm0, nn0, nkt0, nnk);
            setup_loads(nm0, nn0);
            if (nnk > 0) issue(nkt0, stage0);
        }
    }
    if constexpr (EPI == kEpiMse) {
        // Stage each wave's accumulators through LDS (the stages are free now)
        // so that the target is read and dY written in 16-byte row pieces:
        // two halves of 64 rows x 64 columns (float32, 16 KB per wave), 8-column
        // chunks XOR-swizzled by row.  Lane l then takes chunk l % 8 of rows
        // l / 8 + 8 q.  Requires N % 8 == 0 (checked by the caller).
        const bf16_t* bias = static_cast<const bf16_t*>(g.bias);
        __syncthreads();
        float* tile = reinterpret_cast<float*>(wave < 4 ? stage0 : stage1) + (wave & 3) * 4096;
        const int c8 = lane & 7, rq = lane >> 3;
        const int ccol = n0 + wc0 + c8 * 8;   // first global column of this lane's chunk
        const bool cok = ccol < p.N;
        float bv[8];
        {
            uint4 braw = make_uint4(0, 0, 0, 0);
            if (bias && cok) braw = *reinterpret_cast<const uint4*>(bias + ccol);
            const uint32_t bw[4] = {braw.x, braw.y, braw.z, braw.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bv[2 * e] = bf2f(bf16_t(bw[e] & 0xffffu));
                bv[2 * e + 1] = bf2f(bf16_t(bw[e] >> 16));
            }
        }
        float sq = 0.f;
        float cs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int ii = 0; ii < 2; ++ii)
#pragma unroll
                for (int j = 0; j < C_::FN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int r = ii * 32 + nt_row(v, lane), c = j * 32 + nt_col(v, lane);
                        tile[r * 64 + (c ^ ((r & 7) << 3))] = acc[2 * half + ii][j][v >> 2][v & 3];
                    }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int r = rq + 8 * q;
                const int row = m0 + wr0 + half * 64 + r;
                const float4 v0 = *reinterpret_cast<const float4*>(tile + r * 64 + ((c8 ^ (r & 7)) << 3));
                const float4 v1 = *reinterpret_cast<const float4*>(tile + r * 64 + ((c8 ^ (r & 7)) << 3) + 4);
                if (row < p.M && cok) {
                    const int64_t o = int64_t(row) * p.N + ccol;
                    const uint4 tr = *reinterpret_cast<const uint4*>(p.tgt + o);
                    const uint32_t tw[4] = {tr.x, tr.y, tr.z, tr.w};
                    const float val[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
                    uint32_t ow[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float d0 = val[2 * e] + bv[2 * e] - bf2f(bf16_t(tw[e] & 0xffffu));
                        const float d1 = val[2 * e + 1] + bv[2 * e + 1] - bf2f(bf16_t(tw[e] >> 16));
                        sq += d0 * d0 + d1 * d1;
                        const float y0 = p.scale * d0, y1 = p.scale * d1;
                        cs[2 * e] += y0;
                        cs[2 * e + 1] += y1;
                        ow[e] = uint32_t(f2bf(y0)) | (uint32_t(f2bf(y1)) << 16);
                    }
                    *reinterpret_cast<uint4*>(p.dY + o) = make_uint4(ow[0], ow[1], ow[2], ow[3]);
                }
            }
        }
        // column sums: lanes with the same chunk (l % 8) in order of xor steps,
        // then the two wave rows meet in LDS, in a fixed order
#pragma unroll
        for (int e = 0; e < 8; ++e)
#pragma unroll
            for (int m = 8; m < 64; m <<= 1) cs[e] += __shfl_xor(cs[e], m);
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) sq += __shfl_xor(sq, m);
        __syncthreads();
        float* red = reinterpret_cast<float*>(stage0);   // [WGM][BN] column sums, then [8] squares
        if (lane < 8) {
#pragma unroll
            for (int e = 0; e < 8; ++e) red[(wave / C_::WGN) * C_::BN + wc0 + lane * 8 + e] = cs[e];
        }
        if (lane == 0) red[C_::WGM * C_::BN + wave] = sq;
        __syncthreads();
        if (tid < C_::BN && n0 + tid < p.N) {
            float c = 0.f;
#pragma unroll
            for (int r = 0; r < C_::WGM; ++r) c += red[r * C_::BN + tid];
            p.part_col[int64_t(m0 / C_::BM) * p.N + n0 + tid] = c;
        }
        if (tid == 0) {
            float q = 0.f;
            for (int w = 0; w < C_::NT / 64; ++w) q += red[C_::WGM * C_::BN + w];
            p.part_sq[blockIdx.x] = q;
        }
    } else if constexpr (EPI == kEpiPartial) {
        float* P = p.partial + int64_t(split) * p.M * p.N;
#pragma unroll
        for (int j = 0; j < C_::FN; ++j)
#pragma unroll
            for (int i = 0; i < C_::FM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = m0 + wr0 + i * 32 + nt_row(v, lane), col = n0 + wc0 + j * 32 + nt_col(v, lane);
                    if (row < p.M && col < p.N) P[int64_t(row) * p.N + col] = acc[i][j][v >> 2][v & 3];
                }
    } else {
        if (p.vec_store) {
            // Stage each wave's accumulators through LDS as in the MSE epilogue
            // (passes of 64 rows x 64 columns, 8-column chunks swizzled by
            // row); lane l then writes columns 8 (l % 8) .. + 7 of rows
            // l / 8 + 8 q: 16 bytes (bf16) or 32 bytes (float32) per store.
            // Persistent: stage 0 is filling with the next tile, so every wave
            // stages 32 rows at a time in its 8 KB of stage 1.
            constexpr int RP = PERSIST ? 32 : 64;   // rows per pass
            const bf16_t* bias = static_cast<const bf16_t*>(g.bias);
            OutT* C = static_cast<OutT*>(g.C);
            if constexpr (!PERSIST) __syncthreads();
            float* tile = PERSIST ? reinterpret_cast<float*>(stage1) + wave * 2048
                                  : reinterpret_cast<float*>(wave < 4 ? stage0 : stage1) + (wave & 3) * 4096;
            const int c8 = lane & 7, rq = lane >> 3;
            const int ccol = n0 + wc0 + c8 * 8;
            const bool cok = ccol < p.N;
            float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            if (bias && cok) {
                const uint4 braw = *reinterpret_cast<const uint4*>(bias + ccol);
                const uint32_t bw[4] = {braw.x, braw.y, braw.z, braw.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    bv[2 * e] = bf2f(bf16_t(bw[e] & 0xffffu));
                    bv[2 * e + 1] = bf2f(bf16_t(bw[e] >> 16));
                }
            }
#pragma unroll
            for (int pass = 0; pass < C_::WTM / RP; ++pass) {
#pragma unroll
                for (int ii = 0; ii < RP / 32; ++ii)
#pragma unroll
                    for (int j = 0; j < C_::FN; ++j)
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int r = ii * 32 + nt_row(v, lane), c = j * 32 + nt_col(v, lane);
                            tile[r * 64 + (c ^ ((r & 7) << 3))] = acc[pass * (RP / 32) + ii][j][v >> 2][v & 3];
                        }
#pragma unroll
                for (int q = 0; q < RP / 8; ++q) {
                    const int r = rq + 8 * q;
                    const int row = m0 + wr0 + pass * RP + r;
                    const float4 v0 = *reinterpret_cast<const float4*>(tile + r * 64 + ((c8 ^ (r & 7)) << 3));
                    const float4 v1 = *reinterpret_cast<const float4*>(tile + r * 64 + ((c8 ^ (r & 7)) << 3) + 4);
                    if (row < p.M && cok) {
                        const int64_t crow = SCATTER ? int64_t(g.c_idx[row]) : int64_t(row);
                        const float val[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
                        float o[8];
#pragma unroll
                        for (int e = 0; e < 8; ++e) o[e] = g.alpha * val[e] + bv[e];
                        OutT* dst = C + crow * g.ldc + ccol;
                        if constexpr (sizeof(OutT) == 2) {
                            uint32_t w[4];
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                w[e] = uint32_t(f2bf(o[2 * e])) | (uint32_t(f2bf(o[2 * e + 1])) << 16);
                            *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
                        } else {
                            *reinterpret_cast<float4*>(dst) = make_float4(o[0], o[1], o[2], o[3]);
                            *reinterpret_cast<float4*>(dst + 4) = make_float4(o[4], o[5], o[6], o[7]);
                        }
                    }
                }
            }
        } else {
            // C = alpha acc + bias element by element (any N, ldc, alignment)
            const bf16_t* bias = static_cast<const bf16_t*>(g.bias);
            OutT* C = static_cast<OutT*>(g.C);
            // a lane's columns: 16 b + l % 16 of each 32-column block j
            float bv[C_::FN][2];
#pragma unroll
            for (int j = 0; j < C_::FN; ++j)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int col = n0 + wc0 + j * 32 + 16 * b + (lane & 15);
                    bv[j][b] = (bias && col < p.N) ? bf2f(bias[col]) : 0.f;
                }
#pragma unroll
            for (int i = 0; i < C_::FM; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = m0 + wr0 + i * 32 + nt_row(v, lane);
                    if (row >= p.M) continue;
                    const int64_t crow = SCATTER ? int64_t(g.c_idx[row]) : int64_t(row);
#pragma unroll
                    for (int j = 0; j < C_::FN; ++j) {
                        const int col = n0 + wc0 + j * 32 + nt_col(v, lane);
                        if (col < p.N)
                            C[crow * g.ldc + col] = from_f<OutT>(g.alpha * acc[i][j][v >> 2][v & 3] + bv[j][(v >> 2) & 1]);
                    }
                }
        }
    }
    if (!more) break;
    split = nsplit;
    m0 = nm0;
    n0 = nn0;
    kt0 = nkt0;
    nk = nnk;
    }
}

// C = alpha * (sum over splits of the partials, in split order) + bias
template <typename OutT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* partial, int splits, int M, int N,
                                                            GemmDesc g) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i >= int64_t(M) * N) return;
    const int row = int(i / N), col = int(i % N);
    float s = 0.f;
    for (int k = 0; k < splits; ++k) s += partial[int64_t(k) * M * N + i];
    const float bv = g.bias ? to_f(static_cast<const bf16_t*>(g.bias)[col]) : 0.f;
    const int64_t crow = g.c_idx ? int64_t(g.c_idx[row]) : int64_t(row);
    static_cast<OutT*>(g.C)[crow * g.ldc + col] = from_f<OutT>(g.alpha * s + bv);
}

// out[c * ld_out + r] = in[row(r) * ld_in + c] for r < R, c < C (row(r) =
// idx[r] or r), bf16; columns r in [R, R_pad) of out are written as zero.
// Each thread moves one 8 x 8 block: eight 16-byte row loads, a transpose of
// 16-bit lanes in registers (byte permutes), eight 16-byte stores.  A wave
// covers 64 rows x 64 columns; lanes 8q..8q+7 read one 128-byte row piece
// and write one 128-byte output row piece.  Needs C, ld_in, ld_out, R_pad
// multiples of 8 and 16-byte aligned pointers.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const bf16_t* in, int64_t ld_in, const int32_t* idx,
                                                             int64_t R, int C, bf16_t* out, int64_t ld_out,
                                                             int64_t R_pad) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t r0 = int64_t(blockIdx.x) * 64 + (lane >> 3) * 8;
    const int c0 = (blockIdx.y * 4 + wave) * 64 + (lane & 7) * 8;
    if (c0 >= C || r0 >= R_pad) return;
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const int64_t r = r0 + j;
        v[j] = make_uint4(0, 0, 0, 0);
        if (r < R) v[j] = *reinterpret_cast<const uint4*>(in + (idx ? int64_t(idx[r]) : r) * ld_in + c0);
    }
    // w[e] dword q = (row 2q, column e) | (row 2q + 1, column e) << 16
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        uint32_t d[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint4& lo = v[2 * q];
            const uint4& hi = v[2 * q + 1];
            const uint32_t a = (e >> 1) == 0 ? lo.x : (e >> 1) == 1 ? lo.y : (e >> 1) == 2 ? lo.z : lo.w;
            const uint32_t b = (e >> 1) == 0 ? hi.x : (e >> 1) == 1 ? hi.y : (e >> 1) == 2 ? hi.z : hi.w;
            d[q] = __builtin_amdgcn_perm(b, a, (e & 1) ? 0x07060302u : 0x05040100u);
        }
        *reinterpret_cast<uint4*>(out + int64_t(c0 + e) * ld_out + r0) = make_uint4(d[0], d[1], d[2], d[3]);
    }
}

// The same as transpose_bf16_kernel for any alignment and C: a 64 x 64 tile
// through LDS, one element per access.
__global__ __launch_bounds__(256) void transpose_any_kernel(const bf16_t* in, int64_t ld_in, const int32_t* idx,
                                                            int64_t R, int C, bf16_t* out, int64_t ld_out,
                                                            int64_t R_pad) {
    __shared__ bf16_t tile[64][65];
    const int64_t r0 = int64_t(blockIdx.x) * 64;
    const int c0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int rr = ty; rr < 64; rr += 4) {
        const int64_t r = r0 + rr;
        const int c = c0 + tx;
        bf16_t v = 0;
        if (r < R && c < C) v = in[(idx ? int64_t(idx[r]) : r) * ld_in + c];
        tile[rr][tx] = v;
    }
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        const int c = c0 + cc;
        const int64_t r = r0 + tx;
        if (c < C && r < R_pad) out[int64_t(c) * ld_out + r] = tile[tx][cc];
    }
}

// out[r * ld_out + k] = in[row(r) * ld_in + k] for k < K, 0 for K <= k < K_pad
__global__ __launch_bounds__(256) void copy_rows_kernel(const bf16_t* in, int64_t ld_in, const int32_t* idx,
                                                        int64_t R, int K, bf16_t* out, int64_t ld_out, int K_pad) {
    const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (i >= R * K_pad) return;
    const int64_t r = i / K_pad;
    const int k = int(i % K_pad);
    out[r * ld_out + k] = k < K ? in[(idx ? int64_t(idx[r]) : r) * ld_in + k] : bf16_t(0);
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

namespace {

// How a contraction runs on the fast NT path, and the scratch it needs.
// How an operand reaches the kernel: read in place, or first written to
// scratch as a K-contiguous copy (transposed when stored K-major, padded with
// zeros to a 16-byte multiple of K when its rows cannot be read in 16-byte
// chunks).
enum OperandMode { kInPlace = 0, kCopyRows = 1, kCopyTransposed = 2 };

struct NtPlan {
    bool fast = false;
    int64_t ldt = 0;                 // leading dimension of copies (K rounded to 64)
    int amode = kInPlace, bmode = kInPlace;
    int splits = 1, ktiles_per_split = 0;
    size_t a_off = 0, b_off = 0, p_off = 0, bytes = 0;
};

bool rows16(const void* p, int64_t ld) { return reinterpret_cast<uintptr_t>(p) % 16 == 0 && ld % 8 == 0; }

NtPlan plan_nt(const GemmDesc& g) {
    NtPlan p;
    if (g.dtype != JANUS_BF16 || g.M < 128 || g.N < 128 || g.K < 64) return p;
    constexpr int64_t kMaxOff = int64_t(1) << 31;
    // an operand read in place: 16-byte chunks along K (K a multiple of 8, or
    // rows zero-padded past K), byte offsets in 31 bits
    auto in_place_ok = [&](const void* ptr, int64_t ld, const int32_t* idx, int64_t src_rows, bool zero_pad) {
        if (!rows16(ptr, ld) || (g.K % 8 != 0 && !zero_pad)) return false;
        if (idx) return src_rows > 0 && src_rows * ld * 2 < kMaxOff;
        return int64_t(NtCfg::BM) * ld * 2 < kMaxOff;
    };
    p.amode = g.a_t ? kCopyTransposed
                    : in_place_ok(g.A, g.lda, g.a_idx, g.a_src_rows, g.a_zero_pad) ? kInPlace : kCopyRows;
    p.bmode = g.b_t ? kCopyTransposed
                    : in_place_ok(g.B, g.ldb, g.b_idx, g.b_src_rows, g.b_zero_pad) ? kInPlace : kCopyRows;
    p.ldt = round_up(int64_t(g.K), 64);
    if (int64_t(NtCfg::BM) * p.ldt * 2 >= kMaxOff) return p;
    const int tiles = ((g.M + NtCfg::BM - 1) / NtCfg::BM) * ((g.N + NtCfg::BN - 1) / NtCfg::BN);
    const int ktiles = (g.K + NtCfg::BK - 1) / NtCfg::BK;
    int splits = 1;
    if (tiles < 160 && ktiles >= 32) splits = std::max(1, std::min({8, 256 / tiles, ktiles / 16}));
    p.ktiles_per_split = (ktiles + splits - 1) / splits;
    p.splits = (ktiles + p.ktiles_per_split - 1) / p.ktiles_per_split;
    size_t off = 0;
    auto take = [&](size_t bytes) { const size_t o = off; off += (bytes + 255) / 256 * 256; return o; };
    if (p.amode != kInPlace) p.a_off = take(size_t(g.M) * p.ldt * 2);
    if (p.bmode != kInPlace) p.b_off = take(size_t(g.N) * p.ldt * 2);
    if (p.splits > 1) p.p_off = take(size_t(p.splits) * g.M * g.N * 4);
    p.bytes = off;
    p.fast = true;
    return p;
}

const char* nt_label(bool f32out, bool scatter, bool partial) {
    if (partial) return "gemm_nt_splitk";
    if (f32out) return scatter ? "gemm_nt_f32out_scatter" : "gemm_nt_f32out";
    return scatter ? "gemm_nt_bf16out_scatter" : "gemm_nt_bf16out";
}

// JANUS_GEMM_PERSIST=1 switches the persistent tile loop on
bool getenv_on(const char* name) {
    const char* e = getenv(name);
    return e && e[0] == '1';
}

// compute units of the current device (0 if the query fails)
int device_cus() {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
        (void)hipGetLastError();
        return 0;
    }
    return v;
}

template <typename OutT, bool SCATTER, int EPI>
janus_status launch_nt(const NtArgs& args, const GemmDesc& g, hipStream_t s) {
    auto kern = &gemm_nt_fast_kernel<OutT, SCATTER, EPI>;
    NtArgs a = args;
    a.vec_store = (EPI == kEpiStore && g.N % 8 == 0 && g.ldc % 8 == 0 && reinterpret_cast<uintptr_t>(g.C) % 16 == 0 &&
                   (!g.bias || reinterpret_cast<uintptr_t>(g.bias) % 16 == 0))
                      ? 1
                      : 0;
    const int ntot = a.mt * a.nt * a.splits;
    // persistent tiles where every workgroup gets two or more: one per CU
    // (a multiple of 8, so each XCD holds the same number).  Off unless asked
    // for: with the 16x16x32 products that variant spills registers around
    // its tile loop and runs slower than one workgroup per tile.
    int grid = 0;
    if constexpr (EPI == kEpiStore) {
        const int cus = device_cus() / 8 * 8;
        if (a.vec_store && cus >= 8 && ntot % 8 == 0 && ntot >= 2 * cus && getenv_on("JANUS_GEMM_PERSIST")) grid = cus;
    }
    const double out_bytes = EPI == kEpiPartial ? 4.0 * a.splits : EPI == kEpiMse ? 4.0 : (sizeof(OutT) == 4 ? 4.0 : 2.0);
    TraceScope trace(EPI == kEpiMse ? "gemm_nt_mse" : nt_label(sizeof(OutT) == 4, SCATTER, EPI == kEpiPartial),
                     2.0 * g.M * g.N * double(g.K),
                     (double(g.M) * g.K + double(g.N) * g.K) * 2.0 + double(g.M) * g.N * out_bytes, s);
    bool launched = false;
    if constexpr (EPI == kEpiStore) {
        if (grid > 0) {
            a.ntiles = ntot;
            hipLaunchKernelGGL((gemm_nt_fast_kernel<OutT, SCATTER, EPI, true>), dim3(unsigned(grid)),
                               dim3(NtCfg::NT), 0, s, a, g);
            launched = true;
        }
    }
    if (!launched) hipLaunchKernelGGL(kern, dim3(unsigned(ntot)), dim3(NtCfg::NT), 0, s, a, g);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

janus_status transpose_launch(const bf16_t* in, int64_t ld_in, const int32_t* idx, int64_t R, int C, bf16_t* out,
                              int64_t ld_out, int64_t R_pad, hipStream_t s) {
    if (R_pad <= 0 || C <= 0) return JANUS_OK;
    TraceScope trace("transpose_bf16", 0.0, 2.0 * (double(R) * C + double(R_pad) * C), s);
    if (rows16(in, ld_in) && rows16(out, ld_out) && C % 8 == 0 && R_pad % 8 == 0) {
        dim3 grid(unsigned((R_pad + 63) / 64), unsigned((C + 255) / 256));
        hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, s, in, ld_in, idx, R, C, out, ld_out, R_pad);
    } else {
        dim3 grid(unsigned((R_pad + 63) / 64), unsigned((C + 63) / 64));
        hipLaunchKernelGGL(transpose_any_kernel, grid, dim3(256), 0, s, in, ld_in, idx, R, C, out, ld_out, R_pad);
    }
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

janus_status copy_rows_launch(const bf16_t* in, int64_t ld_in, const int32_t* idx, int64_t R, int K, bf16_t* out,
                              int64_t ld_out, int K_pad, hipStream_t s) {
    const int64_t n = R * K_pad;
    if (n <= 0) return JANUS_OK;
    TraceScope trace("copy_rows_bf16", 0.0, 2.0 * (double(R) * K + double(n)), s);
    hipLaunchKernelGGL(copy_rows_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s, in, ld_in, idx, R, K, out,
                       ld_out, K_pad);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

janus_status gemm_fast(const GemmDesc& g, const NtPlan& p, hipStream_t s) {
    char* scratch = static_cast<char*>(g.scratch);
    NtArgs a{};
    a.M = g.M;
    a.N = g.N;
    a.K = g.K;
    janus_status e;
    // each operand as the kernel reads it: rows of K contiguous elements
    auto prepare = [&](int mode, const void* src, int64_t ld, const int32_t* idx, int rows, size_t off,
                       const bf16_t*& op, int64_t& op_ld, const int32_t*& op_idx) -> janus_status {
        if (mode == kInPlace) {
            op = static_cast<const bf16_t*>(src);
            op_ld = ld;
            op_idx = idx;
            return JANUS_OK;
        }
        bf16_t* t = reinterpret_cast<bf16_t*>(scratch + off);
        op = t;
        op_ld = p.ldt;
        op_idx = nullptr;
        if (mode == kCopyTransposed)   // element (row, k) at src[idx(k) * ld + row]
            return transpose_launch(static_cast<const bf16_t*>(src), ld, idx, g.K, rows, t, p.ldt, p.ldt, s);
        return copy_rows_launch(static_cast<const bf16_t*>(src), ld, idx, rows, g.K, t, p.ldt, int(p.ldt), s);
    };
    if ((e = prepare(p.amode, g.A, g.lda, g.a_idx, g.M, p.a_off, a.A, a.lda, a.a_idx)) != JANUS_OK) return e;
    if ((e = prepare(p.bmode, g.B, g.ldb, g.b_idx, g.N, p.b_off, a.B, a.ldb, a.b_idx)) != JANUS_OK) return e;
    a.mt = (g.M + NtCfg::BM - 1) / NtCfg::BM;
    a.nt = (g.N + NtCfg::BN - 1) / NtCfg::BN;
    a.splits = p.splits;
    a.ktiles_per_split = p.ktiles_per_split;
    if (p.splits > 1) {
        a.partial = reinterpret_cast<float*>(scratch + p.p_off);
        if ((e = launch_nt<float, false, kEpiPartial>(a, g, s)) != JANUS_OK) return e;
        const int64_t n = int64_t(g.M) * g.N;
        TraceScope trace("splitk_reduce", 0.0, 4.0 * n * p.splits + n * (g.c_f32 ? 4.0 : 2.0), s);
        if (g.c_f32)
            hipLaunchKernelGGL(splitk_reduce_kernel<float>, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s,
                               a.partial, p.splits, g.M, g.N, g);
        else
            hipLaunchKernelGGL(splitk_reduce_kernel<bf16_t>, dim3(unsigned((n + 255) / 256)), dim3(256), 0, s,
                               a.partial, p.splits, g.M, g.N, g);
        JANUS_LAUNCH_CHECK();
        return JANUS_OK;
    }
    if (g.c_f32) return g.c_idx ? launch_nt<float, true, kEpiStore>(a, g, s) : launch_nt<float, false, kEpiStore>(a, g, s);
    return g.c_idx ? launch_nt<bf16_t, true, kEpiStore>(a, g, s) : launch_nt<bf16_t, false, kEpiStore>(a, g, s);
}

}  // namespace

// out[c] = sum over k < n of part[k * C + c], in order k = 0, 1, ...
__global__ __launch_bounds__(256) void colpart_reduce_kernel(const float* part, int n, int C, float* out) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= C) return;
    float s = 0.f;
    for (int k = 0; k < n; ++k) s += part[int64_t(k) * C + c];
    out[c] = s;
}

size_t gemm_mse_partials(int M, int N) {
    const size_t mt = (M + NtCfg::BM - 1) / NtCfg::BM, nt = (N + NtCfg::BN - 1) / NtCfg::BN;
    return mt * nt + mt * size_t(N);
}

bool gemm_mse_fast(int M, int N, int K, const void* h, const void* W) {
    GemmDesc g;
    g.dtype = JANUS_BF16;
    g.M = M;
    g.N = N;
    g.K = K;
    g.A = h;
    g.lda = K;
    g.B = W;
    g.ldb = K;
    const NtPlan p = plan_nt(g);
    // the epilogue reads the target and writes dY in 16-byte row pieces
    return p.fast && p.bytes == 0 && p.splits == 1 && N % 8 == 0;
}

janus_status gemm_mse(int M, int N, int K, const void* h, const void* W, const void* bias, const void* tgt, void* dY,
                      float scale, float* part, float* db, hipStream_t s) {
    if (!gemm_mse_fast(M, N, K, h, W)) return JANUS_ERR_UNSUPPORTED;
    GemmDesc g;
    g.dtype = JANUS_BF16;
    g.M = M;
    g.N = N;
    g.K = K;
    g.A = h;
    g.lda = K;
    g.B = W;
    g.ldb = K;
    g.bias = bias;
    NtArgs a{};
    a.A = static_cast<const bf16_t*>(h);
    a.B = static_cast<const bf16_t*>(W);
    a.lda = K;
    a.ldb = K;
    a.M = M;
    a.N = N;
    a.K = K;
    a.mt = (M + NtCfg::BM - 1) / NtCfg::BM;
    a.nt = (N + NtCfg::BN - 1) / NtCfg::BN;
    a.splits = 1;
    a.ktiles_per_split = (K + NtCfg::BK - 1) / NtCfg::BK;
    a.tgt = static_cast<const bf16_t*>(tgt);
    a.dY = static_cast<bf16_t*>(dY);
    a.scale = scale;
    a.part_sq = part;
    a.part_col = part + size_t(a.mt) * a.nt;
    janus_status e = launch_nt<float, false, kEpiMse>(a, g, s);
    if (e != JANUS_OK) return e;
    TraceScope trace("colpart_reduce", 0.0, 4.0 * double(a.mt) * N + 4.0 * N, s);
    hipLaunchKernelGGL(colpart_reduce_kernel, dim3(unsigned((N + 255) / 256)), dim3(256), 0, s, a.part_col, a.mt, N,
                       db);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

size_t gemm_scratch_bytes(const GemmDesc& g) {
    const NtPlan p = plan_nt(g);
    return p.fast ? p.bytes : 0;
}

size_t gemm_scratch_bound(const GemmDesc& g) {
    GemmDesc q = g;
    q.A = q.B = nullptr;            // 16-byte aligned stand-ins (unaligned caller tensors may need more;
                                    // gemm() then takes the slower path that needs none)
    q.a_src_rows = q.a_idx ? int64_t(1) : 0;
    q.b_src_rows = q.b_idx ? int64_t(1) : 0;
    const NtPlan p = plan_nt(q);
    if (!p.fast) return 0;
    const int tiles = ((g.M + NtCfg::BM - 1) / NtCfg::BM) * ((g.N + NtCfg::BN - 1) / NtCfg::BN);
    size_t b = 0;
    if (p.amode != kInPlace) b += (size_t(g.M) * p.ldt * 2 + 255) / 256 * 256;
    if (p.bmode != kInPlace) b += (size_t(g.N) * p.ldt * 2 + 255) / 256 * 256;
    if (tiles < 160) b += (size_t(8) * g.M * g.N * 4 + 255) / 256 * 256;
    return b;
}

janus_status gemm(const GemmDesc& g, hipStream_t stream) {
    if (g.M <= 0 || g.N <= 0) return JANUS_OK;
    const size_t es = dtype_size(g.dtype);
    const bool aligned = aligned16(g.A, g.lda, es) && aligned16(g.B, g.ldb, es);
    if (g.dtype == JANUS_BF16) {
        const NtPlan p = plan_nt(g);
        if (p.fast && (p.bytes == 0 || (g.scratch && g.scratch_bytes >= p.bytes))) return gemm_fast(g, p, stream);
        return dispatch<bf16_t, CfgBF16>(g, aligned, stream);
    }
    if (g.dtype == JANUS_F32) return dispatch<float, CfgF32>(g, aligned, stream);
    return JANUS_ERR_UNSUPPORTED;
}

janus_status transpose_bf16(const void* in, int64_t ld_in, const int32_t* idx, int64_t R, int C, void* out,
                            int64_t ld_out, int64_t R_pad, hipStream_t stream) {
    if (!rows16(in, ld_in) || !rows16(out, ld_out) || C % 8 != 0 || R_pad % 8 != 0 || R_pad < R)
        return JANUS_ERR_UNSUPPORTED;
    return transpose_launch(static_cast<const bf16_t*>(in), ld_in, idx, R, C, static_cast<bf16_t*>(out), ld_out,
                            R_pad, stream);
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
