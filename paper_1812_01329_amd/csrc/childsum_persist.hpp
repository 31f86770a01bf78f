// Persistent level programs of the Child-Sum TreeLSTM: the forward pass of a
// batch of trees of any arity in one launch, and the backward pass (levels,
// weight gradients, input gradients and the embedding gradient) in another.
//
// Every node reads its word vector x; h~ is the sum of its children's h, and
// child k has its own forget gate:
//     i, o, u = s, s, tanh (W_iou x + U_iou h~ + b_iou)
//     f_k = s(W_f x + U_f h_k + b_f),  c = i u + sum_k f_k c_k,  h = o tanh(c).
// Levels group nodes by height, the frontiers of the recursion (Section
// 4.2.1; the independent nodes of a level run together, "+PARL" in Section
// 6.3.1), with a device-wide barrier where a level needs another's results.
//
// Forward.  XW = X W^T + b of every node comes first (32 x 32 tiles, fp32
// MFMA; workgroup w keeps the 32 rows w mod NC of W and of U in LDS).  Then,
// per level: the cells, one (node, unit) pair per thread over the whole
// grid, each gathering its children's G rows and c (by linearity U_iou h~ is
// the sum of the children's G_iou rows, and child k's forget gate reads
// G_f of row k); a barrier; G = h U^T of the level's rows as tiles, for
// their parents; a barrier.
//
// Backward, levels from the top down.  The roots' dG and dc rows are zeroed
// first.  Per level, one barrier: dh = dG U of the level's rows as 16-node
// tiles (workgroup w keeps the 32 columns w mod NC of U, K = 4H, in LDS; a
// row's dG is complete once all its parents' levels are done, and a root's
// is zero), and in the same workgroup the cell backward of the tile's
// (node, unit) pairs, dh taken from LDS, which writes into the row of each
// child k dG(k) = [da_iou; da_f(k)] and its dc, and into its own row
// dXW = [da_iou; sum_k da_f].  Then dW = dXW^T X,
// dU = dG^T H, db (column sums of dXW) and dX = dXW W shared by the
// workgroups; a barrier; the embedding gradient, word by word.
//
// Memory between workgroups follows the rule of the other persistent
// kernels (write-through stores, read after a barrier, fresh addresses,
// rows padded to whole 128-byte lines).  Every row that crosses workgroups
// is written once and read only after that.
#pragma once

#include "tree_common.hpp"

namespace janus {
namespace tpersist {

// ---------------------------------------------------------------- forward
struct CsFwdArgs {
    int E, H, N, nlev, ncol;   // ncol: 32-column tiles of the 4H gate columns
    const int32_t* loff;       // [nlev + 1] level offsets
    const int32_t* pword;      // [N] word of the node at each position
    const int32_t* pcoff;      // [N + 1] children of p: pkids[pcoff[p] .. pcoff[p + 1])
    const int32_t* pkids;      // child positions
    const int32_t* rootk;      // [N] tree index of a root, -1 otherwise
    const float* emb;          // [V x E]
    const float* W;            // [4H x E] blocks (i, o, u, f)
    const float* U;            // [4H x H]
    const float* b;            // [4H]
    float* XW;                 // [N x ld4] X W^T + b
    float* G;                  // [N x ld4] h U^T
    int64_t ld4;
    float* Gt;                 // [N x ld3] gates i, o, u
    int64_t ld3;
    float* F;                  // [N x ldh] forget gate of a node towards its parent
    float* C;                  // [N x ldh]
    float* Hn;                 // [N x ldh]
    int64_t ldh;
    float* h_root;             // [trees x H]
    TreeSync* sync;
};

__host__ __device__ inline int cs_fwd_lds_floats(int E, int H) {
    const int sE = pad16(E) + 4, sH = pad16(H) + 4, sA = sE > sH ? sE : sH;
    const int slab = 32 * sA, red = kWaves * 32 * kRed;   // the partial tiles reuse the operand slab
    return 32 * sE + 32 * sH + (slab > red ? slab : red) + 64;   // + the tile's source row offsets (int64)
}

__global__ __launch_bounds__(kThreads) void childsum_fwd_persistent(CsFwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int E = a.E, H = a.H, G4 = 4 * a.H;
    const int KE = pad16(E), KH = pad16(H), sE = KE + 4, sH = KH + 4, sA = sE > sH ? sE : sH;
    float* Wl = sm;                  // [32][sE]: W row 32 col + c
    float* Ul = Wl + 32 * sE;        // [32][sH]: U row 32 col + c
    float* At = Ul + 32 * sH;        // [32 node rows][sA], then the partial tiles
    float* red = At;
    int64_t* rowsrc = reinterpret_cast<int64_t*>(sm + cs_fwd_lds_floats(E, H) - 64);
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int col = int(blockIdx.x) % a.ncol, r0 = int(blockIdx.x) / a.ncol;
    const int R = int(gridDim.x) / a.ncol;
    stage_weight_rows(Wl, sE, a.W, G4, E, col);
    stage_weight_rows(Ul, sH, a.U, G4, H, col);

    // a tile of 32 rows against this workgroup's 32 weight rows; the result
    // goes to dst[row p][32 col + c] (+ bias), written through
    auto tile = [&](int pt, int rows, const float* src, int K, const float* Wsl, int sW, const float* bias,
                    float* dst) {
        __syncthreads();   // the previous tile's reads of At (the partial tiles) and rowsrc are done
        if (tid < 32) {
            int64_t r = -1;
            if (tid < rows) r = src == a.emb ? int64_t(a.pword[pt + tid]) * E : int64_t(pt + tid) * a.ldh;
            rowsrc[tid] = r;
        }
        __syncthreads();
        stage_tile_rows(At, sA, src, rowsrc, K);
        __syncthreads();
        f32x16_t acc;
        tile_mfma(acc, At, sA, Wsl, sW, pad16(K), wave, lane);
        __syncthreads();   // every wave is done reading At before the partial tiles overwrite it
        spill_acc(acc, red, wave, lane);
        __syncthreads();
        for (int idx = tid; idx < 32 * 32; idx += kThreads) {
            const int m = idx / 32, c = idx % 32, n = 32 * col + c;
            if (m < rows && n < G4)
                store_through(dst, int64_t(pt + m) * a.ld4 + n, red_sum(red, m, c) + (bias ? bias[n] : 0.f));
        }
    };

    // XW = X W^T + b for every node
    {
        const int ntile = (a.N + 31) / 32;
        for (int t = r0; t < ntile; t += R) tile(32 * t, min(32, a.N - 32 * t), a.emb, E, Wl, sE, a.b, a.XW);
    }
    tree_census_wait(bar);
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    const int64_t stride = int64_t(gridDim.x) * kThreads;
    for (int L = 0; L < a.nlev; ++L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        // the cells of the level: (node, unit) pairs over the whole grid
        const int64_t total = int64_t(p1 - p0) * H;
        for (int64_t g = int64_t(blockIdx.x) * kThreads + tid; g < total; g += stride) {
            const int m = int(g / H), j = int(g - int64_t(m) * H), p = p0 + m;
            const float* xw = a.XW + int64_t(p) * a.ld4 + j;
            float ai = xw[0], ao = xw[H], au = xw[2 * H];
            const float af = xw[3 * H];
            const int c0 = a.pcoff[p], c1 = a.pcoff[p + 1], rk = a.rootk[p];
            float csum = 0.f;
            for (int e0 = c0; e0 < c1; e0 += 4) {
                int kid[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) kid[i] = e0 + i < c1 ? a.pkids[e0 + i] : -1;
                float gv[4][4], ck[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    gv[i][0] = gv[i][1] = gv[i][2] = gv[i][3] = ck[i] = 0.f;
                    if (kid[i] >= 0) {
                        const float* g4 = a.G + int64_t(kid[i]) * a.ld4 + j;
                        gv[i][0] = g4[0];
                        gv[i][1] = g4[H];
                        gv[i][2] = g4[2 * H];
                        gv[i][3] = g4[3 * H];
                        ck[i] = a.C[int64_t(kid[i]) * a.ldh + j];
                    }
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    if (kid[i] < 0) continue;
                    ai += gv[i][0];
                    ao += gv[i][1];
                    au += gv[i][2];
                    const float f = sigmoidf_(af + gv[i][3]);
                    a.F[int64_t(kid[i]) * a.ldh + j] = f;
                    csum += f * ck[i];
                }
            }
            const float gi = sigmoidf_(ai), go = sigmoidf_(ao), gu = tanhf_(au);
            const float c = gi * gu + csum;
            const float h = go * tanhf_(c);
            store_through(a.C, int64_t(p) * a.ldh + j, c);
            store_through(a.Hn, int64_t(p) * a.ldh + j, h);
            float* gt = a.Gt + int64_t(p) * a.ld3 + j;
            gt[0] = gi;
            gt[H] = go;
            gt[2 * H] = gu;
            if (rk >= 0) a.h_root[int64_t(rk) * H + j] = h;
        }
        if (L + 1 == a.nlev) break;   // the top level has no parents
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
        // G = h U^T of the level's rows, for their parents
        const int ntile = (p1 - p0 + 31) / 32;
        for (int t = r0; t < ntile; t += R) tile(p0 + 32 * t, min(32, p1 - p0 - 32 * t), a.Hn, H, Ul, sH, nullptr, a.G);
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
    }
}

// --------------------------------------------------------------- backward
struct CsBwdArgs {
    int E, H, N, nlev, ncol, nseg, V;   // ncol: 32-column tiles of H (dh)
    const int32_t* loff;
    const int32_t* pword;
    const int32_t* pcoff;
    const int32_t* pkids;
    const int32_t* rootk;
    const int32_t* seg;        // order[N], off[nseg + 1], sid[nseg], first[grid]: the nodes grouped by word
    const float* emb;          // [V x E]
    const float* W;            // [4H x E]
    const float* U;            // [4H x H]
    const float* Gt;           // the forward's gates, forget gates, cells and h
    int64_t ld3;
    const float* F;
    const float* C;
    const float* Hn;
    int64_t ldh;
    const float* dh_root;      // [trees x H]
    float* dG;                 // [N x ld4] gradient of the row's G (from its parent's cell)
    float* dXW;                // [N x ld4]
    int64_t ld4;
    float* dc;                 // [N x ldh]
    float* dx;                 // [N x ldx] gradient of the nodes' inputs
    int64_t ldx;
    float* demb;               // [V x E], every row written
    float* dW;                 // [4H x E]
    float* dU;                 // [4H x H]
    float* db;                 // [4H]
    TreeSync* sync;
};

// the backward's level tiles: 16 node rows, contracted as 16x16x4 products
constexpr int kCsRT = 16;
__host__ __device__ inline int cs_bwd_pitch(int H) { return pad16(4 * H) + 4; }
__host__ __device__ inline int cs_bwd_front(int H) {
    const int slab = 32 * cs_bwd_pitch(H), red = kWaves * 32 * kRed;
    const int level = slab + (slab > red ? slab : red);   // U columns, then the dG tile (and the partial tiles)
    const int tail = 2 * 32 * (kKC + 4) + red;            // the contractions over nodes and their partial tiles
    return level > tail ? level : tail;
}
__host__ __device__ inline int cs_bwd_lds_floats(int H) { return cs_bwd_front(H) + 64; }

__global__ __launch_bounds__(kThreads) void childsum_bwd_persistent(CsBwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int E = a.E, H = a.H, G4 = 4 * a.H;
    const int K4 = pad16(G4), sK = cs_bwd_pitch(H);
    float* Us = sm;                  // [32 columns of H][sK]: Us[c][k] = U[k][32 col + c]
    float* At = Us + 32 * sK;        // [32 node rows][sK] dG tile (16 used), then the partial tiles
    int64_t* rowsrc = reinterpret_cast<int64_t*>(sm + cs_bwd_front(H));
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int col = int(blockIdx.x) % a.ncol, r0 = int(blockIdx.x) / a.ncol;
    const int R = int(gridDim.x) / a.ncol;
    const int64_t stride = int64_t(gridDim.x) * kThreads;

    // U[k][32 col + c] -> Us[c][k]
    if (H % 4 == 0) {
        stage4_2d<10>(K4, 8,
                      [&](int k, int q) {
                          const int n = 32 * col + 4 * q;
                          return (k < G4 && n < H) ? ld4(a.U + int64_t(k) * H + n) : make_float4(0.f, 0.f, 0.f, 0.f);
                      },
                      [&](int k, int q, float4 v) {
                          Us[(4 * q + 0) * sK + k] = v.x;
                          Us[(4 * q + 1) * sK + k] = v.y;
                          Us[(4 * q + 2) * sK + k] = v.z;
                          Us[(4 * q + 3) * sK + k] = v.w;
                      });
    } else {
        stage<16>(32 * K4,
                  [&](int idx) {
                      const int k = idx / 32, c = idx % 32, n = 32 * col + c;
                      return (k < G4 && n < H) ? a.U[int64_t(k) * H + n] : 0.f;
                  },
                  [&](int idx, float v) { Us[(idx % 32) * sK + idx / 32] = v; });
    }
    // the roots have no parent: their dG and dc rows are zero
    for (int64_t g = int64_t(blockIdx.x) * kThreads + tid; g < int64_t(a.N) * H; g += stride) {
        const int p = int(g / H), j = int(g - int64_t(p) * H);
        if (a.rootk[p] < 0) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q) store_through(a.dG, int64_t(p) * a.ld4 + q * H + j, 0.f);
        store_through(a.dc, int64_t(p) * a.ldh + j, 0.f);
    }
    tree_census_wait(bar);
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    for (int L = a.nlev - 1; L >= 0; --L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        // Per 16-node tile: dh = dG U for the workgroup's 32 units, then the
        // cell backward of those (node, unit) pairs in the same workgroup
        // (dh stays in LDS): thread rows tid / 32 + 8 i, unit 32 col + tid % 32.
        const int ntile = (p1 - p0 + kCsRT - 1) / kCsRT;
        for (int t = r0; t < ntile; t += R) {
            const int pt = p0 + kCsRT * t, rows = min(kCsRT, p1 - pt);
            const int c = tid % 32, j = 32 * col + c;
            // the cells' own inputs, in flight while the tile is staged and
            // contracted (indices clamped to a valid node and unit)
            int rk[2], c0[2], c1[2];
            float gi[2], go[2], gu[2], cp[2], dcp[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int m = tid / 32 + 8 * i;
                const int p = pt + min(m, rows - 1), jj = min(j, H - 1);
                rk[i] = a.rootk[p];
                c0[i] = a.pcoff[p];
                c1[i] = a.pcoff[p + 1];
                const float* gt = a.Gt + int64_t(p) * a.ld3 + jj;
                gi[i] = gt[0];
                go[i] = gt[H];
                gu[i] = gt[2 * H];
                cp[i] = a.C[int64_t(p) * a.ldh + jj];
                dcp[i] = a.dc[int64_t(p) * a.ldh + jj];
            }
            __syncthreads();   // the previous tile's reads of At (the partial tiles) and rowsrc are done
            if (tid < 32) rowsrc[tid] = tid < rows ? int64_t(pt + tid) * a.ld4 : -1;
            __syncthreads();
            stage_tile_rows(At, sK, a.dG, rowsrc, G4);
            __syncthreads();
            f32x4_t acc[2];
            tile_mfma16(acc, At, sK, Us, sK, K4, wave, lane);
            __syncthreads();   // every wave is done reading At before the partial tiles overwrite it
            spill_acc16(acc, At, wave, lane);
            __syncthreads();
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int m = tid / 32 + 8 * i, p = pt + m;
                if (m >= rows || j >= H) continue;
                const float dhp = red_sum(At, m, c);
                const float dhr = rk[i] >= 0 ? a.dh_root[int64_t(rk[i]) * H + j] : 0.f;
                const float dhv = dhp + dhr;
                const float tau = tanhf_(cp[i]);
                const float dct = dcp[i] + dhv * go[i] * (1.f - tau * tau);
                const float dai = dct * gu[i] * gi[i] * (1.f - gi[i]);
                const float dao = dhv * tau * go[i] * (1.f - go[i]);
                const float dau = dct * gi[i] * (1.f - gu[i] * gu[i]);
                float dafs = 0.f;
                for (int e0 = c0[i]; e0 < c1[i]; e0 += 4) {
                    int kid[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) kid[q] = e0 + q < c1[i] ? a.pkids[e0 + q] : -1;
                    float fk[4], ck[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int64_t o = int64_t(kid[q] >= 0 ? kid[q] : p) * a.ldh + j;
                        fk[q] = a.F[o];
                        ck[q] = a.C[o];
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        if (kid[q] < 0) continue;
                        const float daf = dct * ck[q] * fk[q] * (1.f - fk[q]);
                        dafs += daf;
                        const int64_t o = int64_t(kid[q]) * a.ld4 + j;
                        store_through(a.dG, o, dai);
                        store_through(a.dG, o + H, dao);
                        store_through(a.dG, o + 2 * H, dau);
                        store_through(a.dG, o + 3 * H, daf);
                        store_through(a.dc, int64_t(kid[q]) * a.ldh + j, dct * fk[q]);
                    }
                }
                const int64_t o = int64_t(p) * a.ld4 + j;
                store_through(a.dXW, o, dai);
                store_through(a.dXW, o + H, dao);
                store_through(a.dXW, o + 2 * H, dau);
                store_through(a.dXW, o + 3 * H, dafs);
            }
        }
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
    }

    // contractions over nodes, dealt to the workgroups in turn
    {
        float* Ac = sm;
        float* Bc = sm + 32 * (kKC + 4);
        float* red = sm + 2 * 32 * (kKC + 4);
        const int n4 = (G4 + 31) / 32, ne = (E + 31) / 32, nh = (H + 31) / 32, nn = (a.N + 31) / 32;
        const int n_dW = n4 * ne, n_dU = n4 * nh, n_dx = nn * ne, n_db = n4;
        const int total = n_dW + n_dU + n_dx + n_db;
        for (int it = int(blockIdx.x); it < total; it += int(gridDim.x)) {
            if (it >= n_dW + n_dU + n_dx) {
                // db for 32 gate columns over all nodes: 16-byte pieces (rows
                // padded to 32 floats), 32 row groups, 16 rows in flight per
                // thread, then the groups in order
                const int i = it - (n_dW + n_dU + n_dx), c4 = 4 * (tid % 8), rg = tid / 8, n = 32 * i + c4;
                constexpr int RG = kThreads / 8;
                float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int q0 = rg; q0 < a.N; q0 += RG * 16) {
                    float4 v[16];
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const int k = q0 + q * RG;
                        v[q] = (k < a.N && n < G4) ? ld4(a.dXW + int64_t(k) * a.ld4 + n) : make_float4(0.f, 0.f, 0.f, 0.f);
                    }
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        s4.x += v[q].x; s4.y += v[q].y; s4.z += v[q].z; s4.w += v[q].w;
                    }
                }
                __syncthreads();   // the previous item's reads of red are done
                red[rg * 32 + c4 + 0] = s4.x;
                red[rg * 32 + c4 + 1] = s4.y;
                red[rg * 32 + c4 + 2] = s4.z;
                red[rg * 32 + c4 + 3] = s4.w;
                __syncthreads();
                if (tid < 32 && 32 * i + tid < G4) {
                    float t2 = 0.f;
                    for (int q = 0; q < RG; ++q) t2 += red[q * 32 + tid];
                    a.db[32 * i + tid] = t2;
                }
                __syncthreads();
                continue;
            }
            f32x16_t acc;
            zero_acc(acc);
            int kind, ti, tj;
            if (it < n_dW) { kind = 0; ti = it / ne; tj = it % ne; }
            else if (it < n_dW + n_dU) { kind = 1; ti = (it - n_dW) / nh; tj = (it - n_dW) % nh; }
            else { kind = 2; ti = (it - n_dW - n_dU) / ne; tj = (it - n_dW - n_dU) % ne; }
            // rows of dXW, dG and h are padded to 32 floats: 16-byte pieces
            // always; rows of emb and W when E % 4 == 0 and both are 16-byte aligned
            const bool vec = E % 4 == 0 && aligned16(a.emb) && aligned16(a.W);
            if (kind == 0 && vec) {
                node_contraction4<false>(acc, Ac, Bc, a.N, min(32, G4 - 32 * ti), min(32, E - 32 * tj),
                    [&](int r4, int k) { return ld4(a.dXW + int64_t(k) * a.ld4 + 32 * ti + r4); },
                    [&](int c4, int k) { return ld4(a.emb + int64_t(a.pword[k]) * E + 32 * tj + c4); });
            } else if (kind == 1) {
                // dU = sum over nodes of dG[p][.] h_p[.]
                node_contraction4<false>(acc, Ac, Bc, a.N, min(32, G4 - 32 * ti), min(32, H - 32 * tj),
                    [&](int r4, int k) { return ld4(a.dG + int64_t(k) * a.ld4 + 32 * ti + r4); },
                    [&](int c4, int k) { return ld4(a.Hn + int64_t(k) * a.ldh + 32 * tj + c4); });
            } else if (kind == 2 && vec) {
                node_contraction4<true>(acc, Ac, Bc, G4, min(32, a.N - 32 * ti), min(32, E - 32 * tj),
                    [&](int r, int k4) { return ld4(a.dXW + int64_t(32 * ti + r) * a.ld4 + k4); },
                    [&](int c4, int k) { return ld4(a.W + int64_t(k) * E + 32 * tj + c4); });
            } else if (kind == 0) {
                // dW[32 ti + r][32 tj + c] = sum over nodes of dXW[p][.] x_p[.]
                node_contraction<false>(acc, Ac, Bc, a.N,
                    [&](int r, int k) {
                        const int n = 32 * ti + r;
                        return n < G4 ? a.dXW[int64_t(k) * a.ld4 + n] : 0.f;
                    },
                    [&](int c, int k) {
                        const int n = 32 * tj + c;
                        return n < E ? a.emb[int64_t(a.pword[k]) * E + n] : 0.f;
                    });
            } else {
                // dx[p][.] = sum over gate columns of dXW[p][k] W[k][.]
                node_contraction<true>(acc, Ac, Bc, G4,
                    [&](int r, int k) {
                        const int p = 32 * ti + r;
                        return p < a.N ? a.dXW[int64_t(p) * a.ld4 + k] : 0.f;
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
                if (kind == 0) {
                    const int m = 32 * ti + r, n = 32 * tj + c;
                    if (m < G4 && n < E) a.dW[int64_t(m) * E + n] = v;
                } else if (kind == 1) {
                    const int m = 32 * ti + r, n = 32 * tj + c;
                    if (m < G4 && n < H) a.dU[int64_t(m) * H + n] = v;
                } else {
                    const int p = 32 * ti + r, n = 32 * tj + c;
                    if (p < a.N && n < E) store_through(a.dx, int64_t(p) * a.ldx + n, v);
                }
            }
            __syncthreads();   // red is read before the next item overwrites it
        }
    }
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    // the embedding gradient: rows of words no node uses are zero (each
    // workgroup zeroes those of an equal share of the table); a used row is
    // the sum of its nodes' dx rows in ascending position order, one word per
    // workgroup in turn
    {
        const int32_t* order = a.seg;
        const int32_t* off = order + a.N;
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
        int* lorder = reinterpret_cast<int*>(sm);   // the nodes of the current row, kThreads at a time
        for (int g = int(blockIdx.x); g < a.nseg; g += int(gridDim.x)) {
            const int64_t v = sid[g];
            const int k0 = off[g], k1 = off[g + 1];
            float s[2] = {0.f, 0.f};   // columns tid and tid + kThreads (E <= kMaxE)
            for (int kb = k0; kb < k1; kb += kThreads) {
                const int nk = min(kThreads, k1 - kb);
                __syncthreads();   // the previous batch of nodes is read
                if (tid < nk) lorder[tid] = order[kb + tid];
                __syncthreads();
                constexpr int LB = 32;   // nodes per round trip
                for (int k = 0; k < nk; k += LB) {
                    float x0[LB], x1[LB];
#pragma unroll
                    for (int q = 0; q < LB; ++q) {
                        const int64_t r = k + q < nk ? int64_t(lorder[k + q]) * a.ldx : -1;
                        x0[q] = (r >= 0 && tid < E) ? a.dx[r + tid] : 0.f;
                        x1[q] = (r >= 0 && tid + kThreads < E) ? a.dx[r + tid + kThreads] : 0.f;
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
