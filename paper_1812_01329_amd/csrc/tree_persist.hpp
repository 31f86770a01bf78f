// Persistent level programs of the binary TreeLSTM: the whole forward pass
// of a tree batch in one launch, and the whole backward pass (levels, weight
// gradients, input gradients and the embedding gradient) in another.
//
// The recursion over a tree (Section 4.2.1: recursive calls become graph
// invocations; Section 6.1: the TreeNN models) visits a node after both of
// its subtrees.  Nodes of equal height are independent, so a level is one
// batched step over all trees of the batch (the parallel execution of
// independent nodes, "+PARL" in Section 6.3.1).  Here the levels run inside
// one kernel, separated by a device-wide barrier, instead of one or two
// launches per level: the per-level cost drops from launch and drain to one
// barrier, and each workgroup's weight slice stays in LDS for all levels.
//
// Node rows are level-ordered positions p (a level is a contiguous range,
// leaves first, M0 of them).  Gate blocks are (i, f_L, f_R, o, u); the gate
// q of unit j sits at column q * H + j of G and dA.
//
// Forward.  The 5H gate columns are split in groups of 6 units (30 of the
// 32 columns of an MFMA tile); workgroup w keeps the W and U columns of
// group w mod G in LDS and takes the 32-node row tiles r = w / G, r + R, ...
// of every level.  A tile's operand rows (the leaves' embedding rows, the
// internal nodes' [h_L; h_R]) are staged in LDS, contracted with fp32 MFMA
// (K split over the four waves, partial tiles summed in LDS), and the cell
// update runs in the same workgroup: c goes to its row, h to the parent's
// [h_L; h_R] row (or to h_root), the gates to G for the backward.
//
// Backward, levels from the top down.  Workgroup w keeps the 32 columns
// w mod NC of U (the columns of [dh_L; dh_R]) in LDS and takes row tiles of
// each internal level; per tile it recomputes the cell backward of its rows
// for all units, in chunks of 32 units, into LDS, and contracts the chunk
// with its U columns: [dh_L; dh_R] = dA U, sent to the two children (each
// node has one parent, so the rows are plain stores).  The workgroup of
// column tile c also stores dA and the children's dc of the unit chunks
// c, c + NC, ... (spread so no column tile carries all the stores).  Level
// 0 (the leaves) only stores dA.  After a barrier the workgroups share the contractions over
// nodes: dU = dA_int^T [h_L; h_R], dW = dA_leaf^T x_leaf, db = column sums
// of dA, dx_leaf = dA_leaf W; after another the embedding gradient, row by
// row of the table (the leaves grouped by word on the host; rows no leaf
// uses are zero), so each row is written once.
//
// Memory between workgroups follows the rule of the persistent recurrence
// kernels: a value another workgroup reads in the same launch is stored
// write-through and read only after a barrier that follows the store, at an
// address no workgroup read earlier in the launch.  Rows that cross
// workgroups are padded to whole 128-byte lines, so a line never mixes a row
// that is already read with one that is not yet written.
#pragma once

#include "tree_common.hpp"

namespace janus {
namespace tpersist {

// ---------------------------------------------------------------- forward
struct FwdArgs {
    int E, H, N, M0, nlev, ngroups;
    const int32_t* loff;       // [nlev + 1] level offsets
    const int32_t* lword;      // [N] word of a leaf
    const int32_t* lchild;     // [N] position of the left child, -1 for leaves
    const int32_t* rchild;
    const int32_t* parent;     // [N] 2 * parent position + side, -1 for roots
    const int32_t* rootk;      // [N] tree index of a root, -1 otherwise
    const float* emb;          // [V x E]
    const float* W;            // [5H x E]
    const float* U;            // [5H x 2H]
    const float* b;            // [5H]
    float* G;                  // [N x ldg] gates after activation
    int64_t ldg;
    float* C;                  // [N x ldc]
    int64_t ldc;
    float* HLR;                // [(N - M0) x ldl]: row p - M0 holds [h_L ; h_R] of node p
    int64_t ldl;
    float* h_root;             // [trees x H]
    TreeSync* sync;
};

__host__ __device__ inline int fwd_lds_floats(int E, int H) {
    const int sE = pad16(E) + 4, sU = pad16(2 * H) + 4, sA = (sE > sU ? sE : sU);
    return 32 * (sE + sU + sA) + kWaves * 32 * kRed + 64;   // + the row offsets of a tile (int64)
}

// Stage a [32 x K] weight slice (row c = tile column c: gate c / 6 of unit
// 6 g + c % 6) into LDS rows of pitch ld, zero past K and for absent units.
__device__ __forceinline__ void stage_fwd_slice(float* dst, int ld, const float* src, int K, int KP, int H, int g) {
    auto row_of = [&](int c) -> int64_t {
        const int q = c / kUG, j = kUG * g + c % kUG;
        return (q < 5 && j < H) ? int64_t(q) * H + j : -1;
    };
    if (K % 4 == 0) {
        const int KP4 = KP / 4;
        stage4<8>(32 * KP4,
                  [&](int idx) {
                      const int c = idx / KP4, k = 4 * (idx - c * KP4);
                      const int64_t r = row_of(c);
                      return (r >= 0 && k < K) ? ld4(src + r * K + k) : make_float4(0.f, 0.f, 0.f, 0.f);
                  },
                  [&](int idx, float4 v) {
                      const int c = idx / KP4, k = 4 * (idx - c * KP4);
                      *reinterpret_cast<float4*>(dst + c * ld + k) = v;
                  });
    } else {
        stage<16>(32 * KP,
                  [&](int idx) {
                      const int c = idx / KP, k = idx - c * KP;
                      const int64_t r = row_of(c);
                      return (r >= 0 && k < K) ? src[r * K + k] : 0.f;
                  },
                  [&](int idx, float v) {
                      const int c = idx / KP, k = idx - c * KP;
                      dst[c * ld + k] = v;
                  });
    }
}

__global__ __launch_bounds__(kThreads) void treelstm_fwd_persistent(FwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int E = a.E, H = a.H;
    const int KE = pad16(E), KU = pad16(2 * H), KA = KE > KU ? KE : KU;
    const int sE = KE + 4, sU = KU + 4, sA = KA + 4;
    float* Wl = sm;                 // [32 tile columns][sE]
    float* Ul = Wl + 32 * sE;       // [32][sU]
    float* At = Ul + 32 * sU;       // [32 node rows][sA]
    float* red = At + 32 * sA;      // [waves][32][kRed]
    int64_t* rowsrc = reinterpret_cast<int64_t*>(red + kWaves * 32 * kRed);   // [32] source row offset, -1 = none
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int g = int(blockIdx.x) % a.ngroups, r0 = int(blockIdx.x) / a.ngroups;
    const int R = int(gridDim.x) / a.ngroups;

    stage_fwd_slice(Wl, sE, a.W, E, KE, H, g);
    stage_fwd_slice(Ul, sU, a.U, 2 * H, KU, H, g);
    tree_census_wait(bar);
    // threads below 32 * 6 update one cell each: row cm of the tile, unit cj
    const int cm = tid / kUG, cu = tid % kUG, cj = kUG * g + cu;
    const bool cell_thread = tid < 32 * kUG && cj < H;
    float bias[5];
#pragma unroll
    for (int q = 0; q < 5; ++q) bias[q] = cell_thread ? a.b[q * H + cj] : 0.f;

    // the cell's links (children, parent, root slot) of row cm of tile t at
    // level L; those of a workgroup's first tile of a level are loaded
    // before the barrier that precedes the level
    int lc = -1, rc = -1, par = -1, rk = -1;
    auto links = [&](int L, int t) {
        const int pt = a.loff[L] + 32 * t, p = pt + cm;
        const bool cell = cell_thread && p < a.loff[L + 1];
        lc = cell ? a.lchild[p] : -1;
        rc = cell ? a.rchild[p] : -1;
        par = cell ? a.parent[p] : -1;
        rk = cell ? a.rootk[p] : -1;
    };
    auto level_tiles = [&](int L) { return (a.loff[L + 1] - a.loff[L] + 31) / 32; };
    if (r0 < level_tiles(0)) links(0, r0);
    for (int L = 0; L < a.nlev; ++L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        const int ntile = level_tiles(L);
        const bool leaf = L == 0;
        const int K = leaf ? E : 2 * H, KP = leaf ? KE : KU, sW = leaf ? sE : sU;
        const float* Wsrc = leaf ? Wl : Ul;
        const float* src = leaf ? a.emb : a.HLR;
        for (int t = r0; t < ntile; t += R) {
            const int pt = p0 + 32 * t, rows = min(32, p1 - pt);
            const int p = pt + cm;
            const bool cell = cell_thread && cm < rows;
            if (t != r0) links(L, t);
            __syncthreads();   // the previous tile's reads of At, red and rowsrc are done
            if (tid < 32) {
                const int q = pt + tid;
                rowsrc[tid] = tid < rows ? (leaf ? int64_t(a.lword[q]) * E : int64_t(q - a.M0) * a.ldl) : -1;
            }
            __syncthreads();
            // the children's c, in flight with the tile's rows
            const float cl = a.C[int64_t(lc >= 0 ? lc : 0) * a.ldc + (cell ? cj : 0)];
            const float cr = a.C[int64_t(rc >= 0 ? rc : 0) * a.ldc + (cell ? cj : 0)];
            if (!leaf || aligned16(a.emb)) {
                // every row in one round trip (16-byte pieces where K % 4 == 0)
                stage_tile_rows(At, sA, src, rowsrc, K);
            } else {
                stage<16>(32 * KP,
                          [&](int idx) {
                              const int m = idx / KP, k = idx - m * KP;
                              const int64_t r = rowsrc[m];
                              return (r >= 0 && k < K) ? src[r + k] : 0.f;
                          },
                          [&](int idx, float v) {
                              const int m = idx / KP, k = idx - m * KP;
                              At[m * sA + k] = v;
                          });
            }
            __syncthreads();
            // D[node m][tile column c] = sum_k rows[m][k] * Wslice[c][k], the
            // k-steps of 16 dealt to the waves in turn
            f32x16_t acc;
            zero_acc(acc);
            for (int ks = wave; ks < KP / 16; ks += kWaves) {
                Frag<float> fa, fb;
                fa.load(At + (lane & 31) * sA + ks * 16 + 8 * (lane >> 5));
                fb.load(Wsrc + (lane & 31) * sW + ks * 16 + 8 * (lane >> 5));
                mfma(acc, fa, fb);
            }
            spill_acc(acc, red, wave, lane);
            __syncthreads();
            if (cell) {
                float z[5];
#pragma unroll
                for (int q = 0; q < 5; ++q) z[q] = bias[q] + red_sum(red, cm, q * kUG + cu);
                const float gi = sigmoidf_(z[0]), gl = sigmoidf_(z[1]), gr = sigmoidf_(z[2]), go = sigmoidf_(z[3]);
                const float gu = tanhf_(z[4]);
                const float c = gi * gu + gl * (lc >= 0 ? cl : 0.f) + gr * (rc >= 0 ? cr : 0.f);
                const float h = go * tanhf_(c);
                store_through(a.C, int64_t(p) * a.ldc + cj, c);
                float* gp = a.G + int64_t(p) * a.ldg + cj;
                gp[0] = gi;
                gp[H] = gl;
                gp[2 * H] = gr;
                gp[3 * H] = go;
                gp[4 * H] = gu;
                if (par >= 0) store_through(a.HLR, int64_t((par >> 1) - a.M0) * a.ldl + (par & 1) * H + cj, h);
                else a.h_root[int64_t(rk) * H + cj] = h;
            }
        }
        if (L + 1 < a.nlev) {
            if (r0 < level_tiles(L + 1)) links(L + 1, r0);
            persist::barrier_arrive(bar);
            persist::barrier_wait(bar);
        }
    }
}

// --------------------------------------------------------------- backward
struct BwdArgs {
    int E, H, N, M0, nlev, ncol, nseg, V;
    const int32_t* loff;
    const int32_t* lword;
    const int32_t* lchild;
    const int32_t* rchild;
    const int32_t* rootk;
    const int32_t* seg;        // order[M0], off[nseg + 1], sid[nseg], first[grid]: the leaves grouped by word
                               // (ids ascending), and each workgroup's first group of the embedding rows
    const float* emb;          // [V x E]
    const float* W;            // [5H x E]
    const float* U;            // [5H x 2H]
    const float* G;            // the forward's gates, cells and [h_L ; h_R] rows
    int64_t ldg;
    const float* C;
    int64_t ldc;
    const float* HLR;
    int64_t ldl;
    const float* dh_root;      // [trees x H]
    float* dh;                 // [N x ldc] gradient of h from the parent's level
    float* dc;                 // [N x ldc]
    float* dA;                 // [N x lda] gradient of the gate pre-activations
    int64_t lda;
    float* dxl;                // [M0 x ldx] gradient of the leaves' inputs
    int64_t ldx;
    float* demb;               // [V x E], every row written
    float* dW;                 // [5H x E]
    float* dU;                 // [5H x 2H]
    float* db;                 // [5H]
    TreeSync* sync;
};

__host__ __device__ inline int bwd_hp(int H) { return padto(H, kUC); }
// chunk depth of the backward's 16-byte contractions over nodes
constexpr int kKCB = kKC;
__host__ __device__ inline int bwd_lds_floats(int H) {
    const int sUs = 5 * bwd_hp(H) + 4, sC = 5 * kUC + 4;
    const int level = 32 * sUs + 32 * sC;
    const int tail = 2 * 64 * (kKCB + 4);   // the contractions over nodes (64 x 64 tiles) reuse the front
    return (level > tail ? level : tail) + kWaves * 32 * kRed;
}

// The internal levels run in 16-row tiles: thread rows tid / 32 + 8 i
// (i < 2), unit lane tid % 32 of each 32-unit chunk.  A thread holds the
// inputs of all its cells at once (H at most 32 kMaxCh), so a tile costs
// one memory round trip for its inputs.
constexpr int kLR = 16;
constexpr int kLRows = kLR * kUC / kThreads;   // 2
constexpr int kMaxCh = 6;
struct LevLinks {
    int p[kLRows], lc[kLRows], rc[kLRows], rk[kLRows];
};
struct LevIn {
    float g[kLRows][kMaxCh][5], c[kLRows][kMaxCh], cl[kLRows][kMaxCh], cr[kLRows][kMaxCh];
    float dh[kLRows][kMaxCh], dc[kLRows][kMaxCh];
};
__device__ __forceinline__ LevLinks lev_links(const BwdArgs& a, int pt, int rows) {
    LevLinks r;
#pragma unroll
    for (int i = 0; i < kLRows; ++i) {
        const int m = int(threadIdx.x) / 32 + 8 * i;
        r.p[i] = m < rows ? pt + m : -1;
        const int q = m < rows ? pt + m : pt;
        r.lc[i] = a.lchild[q];
        r.rc[i] = a.rchild[q];
        r.rk[i] = a.rootk[q];
    }
    return r;
}
// Every load is issued before any value is used (indices clamped to valid
// rows and units, absent cells masked afterwards by the caller).
__device__ __forceinline__ void lev_inputs(const BwdArgs& a, const LevLinks& r, int nch, LevIn& x) {
    const int H = a.H, u = int(threadIdx.x) % 32;
#pragma unroll
    for (int ch = 0; ch < kMaxCh; ++ch) {
        if (ch >= nch) break;
        const int j = min(32 * ch + u, H - 1);
#pragma unroll
        for (int i = 0; i < kLRows; ++i) {
            const int64_t p = r.p[i] >= 0 ? r.p[i] : 0;
            const int64_t pl = r.lc[i] >= 0 ? r.lc[i] : p, pr = r.rc[i] >= 0 ? r.rc[i] : p;
            const float* gp = a.G + p * a.ldg + j;
#pragma unroll
            for (int q = 0; q < 5; ++q) x.g[i][ch][q] = gp[q * H];
            x.c[i][ch] = a.C[p * a.ldc + j];
            x.cl[i][ch] = a.C[pl * a.ldc + j];
            x.cr[i][ch] = a.C[pr * a.ldc + j];
            x.dh[i][ch] = r.rk[i] >= 0 ? a.dh_root[int64_t(r.rk[i]) * H + j] : a.dh[p * a.ldc + j];
            x.dc[i][ch] = a.dc[p * a.ldc + j];
        }
    }
}

__global__ __launch_bounds__(kThreads) void treelstm_bwd_persistent(BwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int E = a.E, H = a.H, H2 = 2 * a.H, G5 = 5 * a.H;
    const int Hp = bwd_hp(H);
    const int sUs = 5 * Hp + 4, sC = 5 * kUC + 4;
    float* Us = sm;                         // [32 columns of [dh_L; dh_R]][5 Hp]: U[q H + j][col] at q Hp + j
    float* dAc = Us + 32 * sUs;             // [32 node rows][5 kUC]: gate q of chunk unit u at q kUC + u
    const int front = bwd_lds_floats(H) - kWaves * 32 * kRed;
    float* red = sm + front;                // [waves][32][kRed]
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int col = int(blockIdx.x) % a.ncol, r0 = int(blockIdx.x) / a.ncol;
    const int R = int(gridDim.x) / a.ncol;
    // U[q H + j][32 col + c] -> Us[c][q Hp + j]: 32 consecutive columns of a
    // row of U are one 128-byte piece
    if (H2 % 4 == 0) {
        stage4<16>(8 * 5 * Hp,
                  [&](int idx) {
                      const int row = idx / 8, c4 = 4 * (idx % 8), q = row / Hp, j = row - q * Hp, n = 32 * col + c4;
                      return (j < H && n < H2) ? ld4(a.U + (int64_t(q) * H + j) * H2 + n) : make_float4(0.f, 0.f, 0.f, 0.f);
                  },
                  [&](int idx, float4 v) {
                      const int row = idx / 8, c4 = 4 * (idx % 8);
                      Us[(c4 + 0) * sUs + row] = v.x;
                      Us[(c4 + 1) * sUs + row] = v.y;
                      Us[(c4 + 2) * sUs + row] = v.z;
                      Us[(c4 + 3) * sUs + row] = v.w;
                  });
    } else {
        stage<16>(32 * 5 * Hp,
                  [&](int idx) {
                      const int row = idx / 32, c = idx % 32, q = row / Hp, j = row - q * Hp, n = 32 * col + c;
                      return (j < H && n < H2) ? a.U[(int64_t(q) * H + j) * H2 + n] : 0.f;
                  },
                  [&](int idx, float v) { Us[(idx % 32) * sUs + idx / 32] = v; });
    }
    tree_census_wait(bar);
    const int u = tid % 32;   // this thread's unit lane within a chunk

    const int nch = (H + kUC - 1) / kUC;
    auto level_tiles = [&](int L) { return (a.loff[L + 1] - a.loff[L] + kLR - 1) / kLR; };
    // the links of this workgroup's first tile of a level are loaded before
    // the barrier that precedes the level
    LevLinks lk{};
    if (a.nlev > 1 && r0 < level_tiles(a.nlev - 1)) {
        const int pt = a.loff[a.nlev - 1] + kLR * r0;
        lk = lev_links(a, pt, min(kLR, a.loff[a.nlev] - pt));
    }
    for (int L = a.nlev - 1; L >= 1; --L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        const int ntile = level_tiles(L);
        for (int t = r0; t < ntile; t += R) {
            const int pt = p0 + kLR * t, rows = min(kLR, p1 - pt);
            if (t != r0) lk = lev_links(a, pt, rows);
            LevIn x;
            lev_inputs(a, lk, nch, x);
            // D[node m][column 16 b + c] over the gate columns as 16x16x4
            // products: k step jj of lane l takes gate column 8 (l / 16) + jj
            // of a 32-column group in both operands, so eight steps cover the
            // group once
            f32x4_t acc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
            // the cells of chunk ch into dA buffer ch % 2 (zero past H and
            // for absent rows); the chunk's column tile also stores dA and
            // the children's dc
            auto cells = [&](int ch) {
                const int j = ch * kUC + u;
                float* dAb = dAc + (ch & 1) * kLR * sC;
#pragma unroll
                for (int i = 0; i < kLRows; ++i) {
                    const int m = tid / 32 + 8 * i;
                    const float gi = x.g[i][ch][0], gl = x.g[i][ch][1], gr = x.g[i][ch][2], go = x.g[i][ch][3];
                    const float gu = x.g[i][ch][4];
                    const float tau = tanhf_(x.c[i][ch]);
                    const float dh = x.dh[i][ch], dc = lk.rk[i] >= 0 ? 0.f : x.dc[i][ch];
                    const float d_o = dh * tau;
                    const float dct = dc + dh * go * (1.f - tau * tau);
                    float da[5];
                    da[0] = dct * gu * gi * (1.f - gi);
                    da[1] = dct * x.cl[i][ch] * gl * (1.f - gl);
                    da[2] = dct * x.cr[i][ch] * gr * (1.f - gr);
                    da[3] = d_o * go * (1.f - go);
                    da[4] = dct * gi * (1.f - gu * gu);
                    if (lk.p[i] < 0 || j >= H) {
#pragma unroll
                        for (int q = 0; q < 5; ++q) da[q] = 0.f;
                    } else if (ch % a.ncol == col) {
#pragma unroll
                        for (int q = 0; q < 5; ++q) store_through(a.dA, int64_t(lk.p[i]) * a.lda + q * H + j, da[q]);
                        store_through(a.dc, int64_t(lk.lc[i]) * a.ldc + j, dct * gl);
                        store_through(a.dc, int64_t(lk.rc[i]) * a.ldc + j, dct * gr);
                    }
#pragma unroll
                    for (int q = 0; q < 5; ++q) dAb[m * sC + q * kUC + u] = da[q];
                }
            };
            // the chunk's gates dealt to the waves in turn; per gate both
            // 16-column blocks, two independent accumulator chains
            auto contract = [&](int ch) {
                const int j0 = ch * kUC;
                const float* dAb = dAc + (ch & 1) * kLR * sC;
#pragma unroll
                for (int q = 0; q < 5; ++q) {
                    if ((ch * 5 + q) % kWaves != wave) continue;
                    const float* ap = dAb + (lane & 15) * sC + q * kUC + 8 * (lane >> 4);
                    const float* bp = Us + (lane & 15) * sUs + q * Hp + j0 + 8 * (lane >> 4);
                    const float4 a0 = *reinterpret_cast<const float4*>(ap), a1 = *reinterpret_cast<const float4*>(ap + 4);
                    const float4 b0 = *reinterpret_cast<const float4*>(bp), b1 = *reinterpret_cast<const float4*>(bp + 4);
                    const float4 c0 = *reinterpret_cast<const float4*>(bp + 16 * sUs);
                    const float4 c1 = *reinterpret_cast<const float4*>(bp + 16 * sUs + 4);
                    const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
                    const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
                    const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
                    for (int jj = 0; jj < 8; ++jj) {
                        acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[jj], bv[jj], acc[0], 0, 0, 0);
                        acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[jj], cv[jj], acc[1], 0, 0, 0);
                    }
                }
            };
            // software pipeline over the chunks: the cells of chunk ch + 1 go
            // to the other buffer while chunk ch is contracted; one barrier
            // per chunk orders both buffers
            cells(0);
            __syncthreads();
#pragma unroll
            for (int ch = 0; ch < kMaxCh; ++ch) {
                if (ch >= nch) break;
                contract(ch);
                if (ch + 1 < kMaxCh && ch + 1 < nch) cells(ch + 1);
                __syncthreads();
            }
            // element v of acc[b] of lane l: row 4 (l / 16) + v, column 16 b + l % 16
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    red[(wave * 32 + 4 * (lane >> 4) + v) * kRed + 16 * b + (lane & 15)] = acc[b][v];
            __syncthreads();
            // [dh_L; dh_R] of the tile's rows to the two children
            for (int idx = tid; idx < kLR * 32; idx += kThreads) {
                const int m = idx / 32, c = idx % 32, n = 32 * col + c;
                if (m < rows && n < H2) {
                    const int p = pt + m;
                    const float v = red_sum(red, m, c);
                    if (n < H) store_through(a.dh, int64_t(a.lchild[p]) * a.ldc + n, v);
                    else store_through(a.dh, int64_t(a.rchild[p]) * a.ldc + (n - H), v);
                }
            }
            __syncthreads();   // red and the dA buffers are read before the next tile overwrites them
        }
        if (L > 1 && r0 < level_tiles(L - 1)) {
            const int pt = a.loff[L - 1] + kLR * r0;
            lk = lev_links(a, pt, min(kLR, a.loff[L] - pt));
        }
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
    }
    // the leaves: dA only (no children, so the forget gates' entries are
    // 0); 16-row tiles dealt to all workgroups, each tile's inputs in one
    // round trip after its links
    {
        const int ntile = (a.M0 + kLR - 1) / kLR;
        for (int t = int(blockIdx.x); t < ntile; t += int(gridDim.x)) {
            const LevLinks ll = lev_links(a, kLR * t, min(kLR, a.M0 - kLR * t));
            LevIn x;
            lev_inputs(a, ll, nch, x);
#pragma unroll
            for (int ch = 0; ch < kMaxCh; ++ch) {
                if (ch >= nch) break;
                const int j = ch * kUC + u;
#pragma unroll
                for (int i = 0; i < kLRows; ++i) {
                    if (ll.p[i] < 0 || j >= H) continue;
                    const float gi = x.g[i][ch][0], go = x.g[i][ch][3], gu = x.g[i][ch][4];
                    const float tau = tanhf_(x.c[i][ch]);
                    const float dh = x.dh[i][ch], dc = ll.rk[i] >= 0 ? 0.f : x.dc[i][ch];
                    const float d_o = dh * tau;
                    const float dct = dc + dh * go * (1.f - tau * tau);
                    float* row = a.dA + int64_t(ll.p[i]) * a.lda + j;
                    store_through(row, 0, dct * gu * gi * (1.f - gi));
                    store_through(row, H, 0.f);
                    store_through(row, 2 * H, 0.f);
                    store_through(row, 3 * H, d_o * go * (1.f - go));
                    store_through(row, 4 * H, dct * gi * (1.f - gu * gu));
                }
            }
        }
    }
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    // contractions over nodes, dealt to the workgroups in turn: 64 x 64
    // tiles where every operand can be read in 16-byte pieces (always for dU,
    // whose rows are padded to 32 floats), else 32 x 32
    {
        const bool vec = E % 4 == 0 && aligned16(a.emb) && aligned16(a.W);
        const int T = vec ? 64 : 32;      // tile edge of the dW and dx items
        float* Ac = sm;
        float* Bc = sm + 64 * (kKCB + 4);   // the scalar contraction's pitch kKC + 4 fits below
        const int ne = (E + T - 1) / T, nl = (a.M0 + T - 1) / T;
        const int n_dU = ((G5 + 63) / 64) * ((H2 + 63) / 64), n_dW = ((G5 + T - 1) / T) * ne, n_dx = nl * ne;
        const int n_db = (G5 + 31) / 32, nh2 = (H2 + 63) / 64;
        const int total = n_dU + n_dW + n_dx + n_db;
        const int Nint = a.N - a.M0;
        for (int it = int(blockIdx.x); it < total; it += int(gridDim.x)) {
            if (it >= n_dU + n_dW + n_dx) {
                // db over all nodes for 32 columns: 32 row groups of 16-byte
                // pieces (8 per row), 16 loads in flight per thread, then the
                // groups in order
                const int i = it - (n_dU + n_dW + n_dx);
                const int c4 = 4 * (tid % 8), rg = tid / 8, n = 32 * i + c4;
                constexpr int RG = kThreads / 8;
                float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f);
                const bool vecb = a.lda % 4 == 0;
                for (int p0 = rg; p0 < a.N; p0 += RG * 16) {
                    float4 v[16];
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const int p = p0 + q * RG;
                        v[q] = make_float4(0.f, 0.f, 0.f, 0.f);
                        if (p < a.N) {
                            const float* row = a.dA + int64_t(p) * a.lda + n;
                            if (vecb && n + 3 < G5) v[q] = ld4(row);
                            else {
                                v[q].x = n < G5 ? row[0] : 0.f;
                                v[q].y = n + 1 < G5 ? row[1] : 0.f;
                                v[q].z = n + 2 < G5 ? row[2] : 0.f;
                                v[q].w = n + 3 < G5 ? row[3] : 0.f;
                            }
                        }
                    }
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        s4.x += v[q].x; s4.y += v[q].y; s4.z += v[q].z; s4.w += v[q].w;
                    }
                }
                __syncthreads();
                red[rg * 32 + c4 + 0] = s4.x;
                red[rg * 32 + c4 + 1] = s4.y;
                red[rg * 32 + c4 + 2] = s4.z;
                red[rg * 32 + c4 + 3] = s4.w;
                __syncthreads();
                if (tid < 32 && 32 * i + tid < G5) {
                    float t2 = 0.f;
                    for (int q = 0; q < RG; ++q) t2 += red[q * 32 + tid];
                    a.db[32 * i + tid] = t2;
                }
                continue;
            }
            f32x16_t acc;
            zero_acc(acc);
            int kind, ti, tj;
            if (it < n_dU) { kind = 0; ti = it / nh2; tj = it % nh2; }
            else if (it < n_dU + n_dW) { kind = 1; ti = (it - n_dU) / ne; tj = (it - n_dU) % ne; }
            else { kind = 2; ti = (it - n_dU - n_dW) / ne; tj = (it - n_dU - n_dW) % ne; }
            if (vec || kind == 0) {
                // rows of dA and [h_L; h_R] are padded to 32 floats, and rows of
                // emb and W are 16-byte aligned where vec holds: 16-byte pieces
                const int m0 = 64 * ti, n0 = 64 * tj;
                if (kind == 0) {
                    // dU[m][n] = sum over internal nodes of dA[p][m] [h_L; h_R][p][n]
                    node_contraction64<false, kKCB>(acc, Ac, Bc, Nint, min(64, G5 - m0), min(64, H2 - n0),
                        [&](int r4, int k) { return ld4(a.dA + int64_t(a.M0 + k) * a.lda + m0 + r4); },
                        [&](int c4, int k) { return ld4(a.HLR + int64_t(k) * a.ldl + n0 + c4); });
                } else if (kind == 1) {
                    // dW = sum over leaves of dA[p][.] x_p[.]
                    node_contraction64<false, kKCB>(acc, Ac, Bc, a.M0, min(64, G5 - m0), min(64, E - n0),
                        [&](int r4, int k) { return ld4(a.dA + int64_t(k) * a.lda + m0 + r4); },
                        [&](int c4, int k) { return ld4(a.emb + int64_t(a.lword[k]) * E + n0 + c4); });
                } else {
                    // dx_leaf[p][.] = sum over gate columns of dA[p][k] W[k][.]
                    node_contraction64<true, kKCB>(acc, Ac, Bc, G5, min(64, a.M0 - m0), min(64, E - n0),
                        [&](int r, int k4) { return ld4(a.dA + int64_t(m0 + r) * a.lda + k4); },
                        [&](int c4, int k) { return ld4(a.W + int64_t(k) * E + n0 + c4); });
                }
                // each wave holds the quadrant at rows 32 (wave / 2), columns 32 (wave % 2)
                const int qm = m0 + 32 * (wave >> 1), qn = n0 + 32 * (wave & 1) + acc_col(lane);
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = qm + acc_row(v, lane);
                    if (kind == 0) {
                        if (m < G5 && qn < H2) a.dU[int64_t(m) * H2 + qn] = acc[v];
                    } else if (kind == 1) {
                        if (m < G5 && qn < E) a.dW[int64_t(m) * E + qn] = acc[v];
                    } else {
                        if (m < a.M0 && qn < E) store_through(a.dxl, int64_t(m) * a.ldx + qn, acc[v]);
                    }
                }
                continue;
            }
            if (kind == 1) {
                // dW = sum over leaves of dA[p][.] x_p[.]
                node_contraction<false>(acc, Ac, Bc, a.M0,
                    [&](int r, int k) {
                        const int n = 32 * ti + r;
                        return n < G5 ? a.dA[int64_t(k) * a.lda + n] : 0.f;
                    },
                    [&](int c, int k) {
                        const int n = 32 * tj + c;
                        return n < E ? a.emb[int64_t(a.lword[k]) * E + n] : 0.f;
                    });
            } else {
                // dx_leaf[p][.] = sum over gate columns of dA[p][k] W[k][.]
                node_contraction<true>(acc, Ac, Bc, G5,
                    [&](int r, int k) {
                        const int p = 32 * ti + r;
                        return p < a.M0 ? a.dA[int64_t(p) * a.lda + k] : 0.f;
                    },
                    [&](int c, int k) {
                        const int n = 32 * tj + c;
                        return n < E ? a.W[int64_t(k) * E + n] : 0.f;
                    });
            }
            spill_acc(acc, red, wave, lane);
            __syncthreads();
            for (int idx = tid; idx < 32 * 32; idx += kThreads) {
                const int r = idx / 32, c = idx % 32;
                const float v = red_sum(red, r, c);
                if (kind == 1) {
                    const int m = 32 * ti + r, n = 32 * tj + c;
                    if (m < G5 && n < E) a.dW[int64_t(m) * E + n] = v;
                } else {
                    const int p = 32 * ti + r, n = 32 * tj + c;
                    if (p < a.M0 && n < E) store_through(a.dxl, int64_t(p) * a.ldx + n, v);
                }
            }
            __syncthreads();   // red is read before the next item overwrites it
        }
    }
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    // the embedding gradient.  Rows without leaves are zero: each workgroup
    // zeroes those of an equal share of the table (first[w] is the first group
    // whose id is at least its first row).  Rows with leaves are the sum of
    // their dx rows in ascending leaf order, one group per workgroup in turn,
    // so a frequent word's many leaves do not all fall to one workgroup.
    {
        const int32_t* order = a.seg;
        const int32_t* off = order + a.M0;
        const int32_t* sid = off + a.nseg + 1;
        const int32_t* first = sid + a.nseg;
        const int64_t v0 = int64_t(a.V) * blockIdx.x / gridDim.x, v1 = int64_t(a.V) * (blockIdx.x + 1) / gridDim.x;
        int gi = first[blockIdx.x];
        int64_t next_id = gi < a.nseg ? sid[gi] : a.V;
        for (int64_t v = v0; v < v1; ++v) {
            if (v == next_id) {
                ++gi;
                next_id = gi < a.nseg ? sid[gi] : a.V;
                continue;
            }
            for (int e = tid; e < E; e += kThreads) a.demb[v * E + e] = 0.f;
        }
        int* lorder = reinterpret_cast<int*>(sm);   // the leaves of the current row, kThreads at a time
        for (int g = int(blockIdx.x); g < a.nseg; g += int(gridDim.x)) {
            const int64_t v = sid[g];
            const int k0 = off[g], k1 = off[g + 1];
            float s[2] = {0.f, 0.f};   // columns tid and tid + kThreads (E <= kMaxE)
            for (int kb = k0; kb < k1; kb += kThreads) {
                const int nk = min(kThreads, k1 - kb);
                __syncthreads();   // the previous batch of leaves is read
                if (tid < nk) lorder[tid] = order[kb + tid];
                __syncthreads();
                constexpr int LB = 32;   // leaves per round trip
                for (int k = 0; k < nk; k += LB) {
                    float x0[LB], x1[LB];
#pragma unroll
                    for (int q = 0; q < LB; ++q) {
                        const int64_t r = k + q < nk ? int64_t(lorder[k + q]) * a.ldx : -1;
                        x0[q] = (r >= 0 && tid < E) ? a.dxl[r + tid] : 0.f;
                        x1[q] = (r >= 0 && tid + kThreads < E) ? a.dxl[r + tid + kThreads] : 0.f;
                    }
#pragma unroll
                    for (int q = 0; q < LB; ++q) {
                        s[0] += x0[q];
                        s[1] += x1[q];
                    }
                }
            }
            if (tid < E) a.demb[v * E + tid] = s[0];
            if (tid + kThreads < E) a.demb[v * E + tid + kThreads] = s[1];
        }
    }
}

}  // namespace tpersist
}  // namespace janus
