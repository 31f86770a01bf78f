// Persistent level programs of the binary TreeRNN: the whole forward pass of
// a tree batch in one launch, and the whole backward pass (levels, weight
// gradients and the embedding gradient) in another.
//
// The model composes a node from its two subtrees, h = tanh(W [h_L; h_R] + b),
// and a leaf's h is its word vector (Section 6.1 trains it on the TreeNN
// workload next to the TreeLSTM).  The frontier schedule is the TreeLSTM's:
// level-ordered node positions, leaves first (M0 of them), one device-wide
// barrier between levels instead of one launch per level (Section 4.2.1
// recursion as graph invocations; independent nodes of a level run together,
// "+PARL" in Section 6.3.1).
//
// Forward.  Workgroup w keeps the 32 rows w mod NC of W (32 output units,
// all 2H inputs) in LDS and takes the 16-node row tiles r = w / NC, r + R, ...
// of each internal level: it stages the tile's [h_L; h_R] rows, contracts
// them as fp32 16x16x4 products (K split over the four waves, partial tiles
// summed in LDS), and applies bias and tanh; h goes to its row (for the backward) and
// to the parent's [h_L; h_R] row or to h_root.  The leaves only copy their
// word vectors to their parents' rows; those rows are dealt to all
// workgroups before the first barrier.
//
// Backward, levels from the top down.  Workgroup w keeps the 32 columns
// w mod NC2 of W (of [dh_L; dh_R]) in LDS.  Per row tile it forms
// da = dh (1 - h^2) for all units in LDS (the workgroup of column tile c
// also stores the units of chunks c, c + NC2, ... to dA), contracts it with
// its W columns and sends [dh_L; dh_R] to the two children.  After the last
// level the workgroups share dW = dA_int^T [h_L; h_R] and db (column sums
// of dA over internal nodes), then the embedding gradient: the sum of the
// leaves' dh per word, in ascending leaf order, and zero rows for words no
// leaf uses.
//
// Memory between workgroups follows the rule of the other persistent
// kernels: what another workgroup reads in the same launch is stored
// write-through and read only after a barrier that follows the store, at an
// address nobody read earlier in the launch; rows that cross workgroups are
// padded to whole 128-byte lines.
#pragma once

#include "tree_common.hpp"

namespace janus {
namespace tpersist {

// ---------------------------------------------------------------- forward
struct RnnFwdArgs {
    int H, N, M0, nlev, ncol;
    const int32_t* loff;       // [nlev + 1] level offsets
    const int32_t* lword;      // [N] word of a leaf
    const int32_t* parent;     // [N] 2 * parent position + side, -1 for roots
    const int32_t* rootk;      // [N] tree index of a root, -1 otherwise
    const float* emb;          // [V x H]
    const float* W;            // [H x 2H]
    const float* b;            // [H]
    float* Hn;                 // [N x ldh] h of the internal nodes
    int64_t ldh;
    float* HLR;                // [(N - M0) x ldl]: row p - M0 holds [h_L ; h_R] of node p
    int64_t ldl;
    float* h_root;             // [trees x H]
    TreeSync* sync;
};

// Node rows per level tile: 16, contracted as 16x16x4 products.
constexpr int kRT = 16;

// Row pitch of the staged operands (K = 2H, padded to the MFMA k-step).
__host__ __device__ inline int rnn_fwd_pitch(int H) { return pad16(2 * H) + 4; }
__host__ __device__ inline int rnn_fwd_lds_floats(int H) {
    const int slab = 32 * rnn_fwd_pitch(H);
    const int red = kWaves * 32 * kRed;   // the partial tiles reuse the operand slab
    return slab + (slab > red ? slab : red) + 128;   // + the tile's source and destination row offsets (int64)
}

__global__ __launch_bounds__(kThreads) void treernn_fwd_persistent(RnnFwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int H = a.H, K = 2 * a.H, KP = pad16(K), sK = rnn_fwd_pitch(H);
    float* Wl = sm;                       // [32 units][sK]: row c = W row 32 col + c
    float* At = Wl + 32 * sK;             // [32 node rows][sK] (16 used), then the partial tiles
    float* red = At;
    // [32] source row offset of each tile row (-1: none), and where its h
    // goes: >= 0 an offset into HLR, else -1 - (offset into h_root)
    int64_t* rowsrc = reinterpret_cast<int64_t*>(sm + rnn_fwd_lds_floats(H) - 128);
    int64_t* rowdst = rowsrc + 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int col = int(blockIdx.x) % a.ncol, r0 = int(blockIdx.x) / a.ncol;
    const int R = int(gridDim.x) / a.ncol;

    // the leaves: word vectors to the parents' rows (or to h_root), spread
    // over every thread of the grid, NB pieces in flight per thread
    {
        constexpr int NB = 4;
        const int V4 = H % 4 == 0 ? 4 : 1, HV = H / V4;
        const int64_t total = int64_t(a.M0) * HV, stride = int64_t(gridDim.x) * kThreads;
        for (int64_t base = int64_t(blockIdx.x) * kThreads + tid; base < total; base += stride * NB) {
            int p[NB], par[NB], rk[NB];
            float4 v[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const int64_t q = base + i * stride;
                p[i] = q < total ? int(q / HV) : -1;
                par[i] = p[i] >= 0 ? a.parent[p[i]] : -1;
                rk[i] = p[i] >= 0 ? a.rootk[p[i]] : -1;
                v[i] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (p[i] >= 0) {
                    const int j = V4 * int(q - int64_t(p[i]) * HV);
                    const float* src = a.emb + int64_t(a.lword[p[i]]) * H + j;
                    if (V4 == 4) v[i] = ld4(src);
                    else v[i].x = src[0];
                }
            }
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                if (p[i] < 0) continue;
                const int j = V4 * int(base + i * stride - int64_t(p[i]) * HV);
                const float e[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
                for (int c = 0; c < V4; ++c) {
                    if (par[i] >= 0)
                        store_through(a.HLR, int64_t((par[i] >> 1) - a.M0) * a.ldl + (par[i] & 1) * H + j + c, e[c]);
                    else
                        a.h_root[int64_t(rk[i]) * H + j + c] = e[c];
                }
            }
        }
    }
    // W rows of this column tile, zero past K and past H
    if (K % 4 == 0) {
        stage4_2d<10>(32, KP / 4,
                      [&](int c, int q) {
                          const int n = 32 * col + c, k = 4 * q;
                          return (n < H && k < K) ? ld4(a.W + int64_t(n) * K + k) : make_float4(0.f, 0.f, 0.f, 0.f);
                      },
                      [&](int c, int q, float4 v) { *reinterpret_cast<float4*>(Wl + c * sK + 4 * q) = v; });
    } else {
        stage<16>(32 * KP,
                  [&](int idx) {
                      const int c = idx / KP, k = idx - c * KP, n = 32 * col + c;
                      return (n < H && k < K) ? a.W[int64_t(n) * K + k] : 0.f;
                  },
                  [&](int idx, float v) { Wl[(idx / KP) * sK + idx % KP] = v; });
    }
    tree_census_wait(bar);
    if (a.nlev > 1) {
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
    }

    for (int L = 1; L < a.nlev; ++L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        const int ntile = (p1 - p0 + kRT - 1) / kRT;
        for (int t = r0; t < ntile; t += R) {
            const int pt = p0 + kRT * t, rows = min(kRT, p1 - pt);
            __syncthreads();   // the previous tile's reads of At (the partial tiles), rowsrc and rowdst are done
            // the destinations of the tile's h, loaded while the rows are staged
            int par = -1, rk = -1;
            if (tid < rows) {
                par = a.parent[pt + tid];
                rk = a.rootk[pt + tid];
            }
            if (tid < 32) rowsrc[tid] = tid < rows ? int64_t(pt + tid - a.M0) * a.ldl : -1;
            __syncthreads();
            stage_tile_rows(At, sK, a.HLR, rowsrc, K);
            if (tid < rows)
                rowdst[tid] = par >= 0 ? int64_t((par >> 1) - a.M0) * a.ldl + (par & 1) * H : -1 - int64_t(rk) * H;
            __syncthreads();
            // D[node m][unit c] = sum_k rows[m][k] W[32 col + c][k]
            f32x4_t acc[2];
            tile_mfma16(acc, At, sK, Wl, sK, KP, wave, lane);
            __syncthreads();   // every wave is done reading At before the partial tiles overwrite it
            spill_acc16(acc, red, wave, lane);
            __syncthreads();
            for (int idx = tid; idx < kRT * 32; idx += kThreads) {
                const int m = idx / 32, c = idx % 32, n = 32 * col + c;
                if (m >= rows || n >= H) continue;
                const int p = pt + m;
                const float h = tanhf_(red_sum(red, m, c) + a.b[n]);
                a.Hn[int64_t(p) * a.ldh + n] = h;
                const int64_t dst = rowdst[m];
                if (dst >= 0) store_through(a.HLR, dst + n, h);
                else a.h_root[-1 - dst + n] = h;
            }
        }
        if (L + 1 < a.nlev) {
            persist::barrier_arrive(bar);
            persist::barrier_wait(bar);
        }
    }
}

// --------------------------------------------------------------- backward
struct RnnBwdArgs {
    int H, N, M0, nlev, ncol, nseg, V, ntrees;
    const int32_t* loff;
    const int32_t* lword;
    const int32_t* lchild;
    const int32_t* rchild;
    const int32_t* rootk;
    const int32_t* rootpos;    // [ntrees] position of root k
    const int32_t* seg;        // order[M0], off[nseg + 1], sid[nseg], first[grid]: the leaves grouped by word
    const float* W;            // [H x 2H]
    const float* Hn;           // the forward's h of internal nodes and [h_L ; h_R] rows
    int64_t ldh;
    const float* HLR;
    int64_t ldl;
    const float* dh_root;      // [trees x H]
    float* dh;                 // [N x ldh] gradient of h from the parent's level
    float* dA;                 // [N x lda] da of internal nodes
    int64_t lda;
    float* demb;               // [V x H], every row written
    float* dW;                 // [H x 2H]
    float* db;                 // [H]
    TreeSync* sync;
};

__host__ __device__ inline int rnn_bwd_pitch(int H) { return pad16(H) + 4; }
__host__ __device__ inline int rnn_bwd_front(int H) {
    const int level = 2 * 32 * rnn_bwd_pitch(H);
    const int tail = 2 * 32 * (kKC + 4);   // the contractions over nodes reuse the front
    return level > tail ? level : tail;
}
__host__ __device__ inline int rnn_bwd_lds_floats(int H) {
    return rnn_bwd_front(H) + kWaves * 32 * kRed + 64;   // + the tile's child links
}

__global__ __launch_bounds__(kThreads) void treernn_bwd_persistent(RnnBwdArgs a) {
    extern __shared__ __align__(16) float sm[];
    const int H = a.H, H2 = 2 * a.H, KP = pad16(a.H), sH = rnn_bwd_pitch(a.H);
    float* Ws = sm;                  // [32 columns of [dh_L; dh_R]][sH]: Ws[c][k] = W[k][32 col + c]
    float* dAt = Ws + 32 * sH;       // [32 node rows][sH] (16 used): da of the tile
    float* red = sm + rnn_bwd_front(H);
    int* links = reinterpret_cast<int*>(red + kWaves * 32 * kRed);   // [32] left, [32] right child of the tile rows
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    TreeBarrier bar;
    tree_census_arrive(bar, a.sync);
    const int col = int(blockIdx.x) % a.ncol, r0 = int(blockIdx.x) / a.ncol;
    const int R = int(gridDim.x) / a.ncol;
    // W[k][32 col + c] -> Ws[c][k]: 32 consecutive columns of a row of W are
    // one 128-byte piece
    if (H2 % 4 == 0) {
        stage4<8>(8 * KP,
                  [&](int idx) {
                      const int k = idx / 8, c4 = 4 * (idx % 8), n = 32 * col + c4;
                      return (k < H && n < H2) ? ld4(a.W + int64_t(k) * H2 + n) : make_float4(0.f, 0.f, 0.f, 0.f);
                  },
                  [&](int idx, float4 v) {
                      const int k = idx / 8, c4 = 4 * (idx % 8);
                      Ws[(c4 + 0) * sH + k] = v.x;
                      Ws[(c4 + 1) * sH + k] = v.y;
                      Ws[(c4 + 2) * sH + k] = v.z;
                      Ws[(c4 + 3) * sH + k] = v.w;
                  });
    } else {
        stage<16>(32 * KP,
                  [&](int idx) {
                      const int k = idx / 32, c = idx % 32, n = 32 * col + c;
                      return (k < H && n < H2) ? a.W[int64_t(k) * H2 + n] : 0.f;
                  },
                  [&](int idx, float v) { Ws[(idx % 32) * sH + idx / 32] = v; });
    }
    // the roots' dh into their dh rows (a root has no parent to send it), so
    // every level reads dh from one place; spread over the grid
    {
        const int K = a.ntrees;
        const int64_t total = int64_t(K) * H, stride = int64_t(gridDim.x) * kThreads;
        for (int64_t q = int64_t(blockIdx.x) * kThreads + tid; q < total; q += stride) {
            const int k = int(q / H), j = int(q - int64_t(k) * H);
            store_through(a.dh, int64_t(a.rootpos[k]) * a.ldh + j, a.dh_root[q]);
        }
    }
    tree_census_wait(bar);
    persist::barrier_arrive(bar);
    persist::barrier_wait(bar);

    // dA is stored in 16-byte write-through pieces (its rows are padded to 32
    // floats, so a piece past H stays inside the row); the first piece of
    // each thread, stepped without a division as in stage4_2d
    const auto rsA = persist::make_rsrc(a.dA, uint32_t(a.N) * uint32_t(a.lda) * 4u);
    const int KP4 = KP / 4, dm = kThreads / KP4, dq = kThreads - dm * KP4;
    const int m_first = tid / KP4, q_first = tid - m_first * KP4;

    for (int L = a.nlev - 1; L >= 1; --L) {
        const int p0 = a.loff[L], p1 = a.loff[L + 1];
        const int ntile = (p1 - p0 + kRT - 1) / kRT;
        for (int t = r0; t < ntile; t += R) {
            const int pt = p0 + kRT * t, rows = min(kRT, p1 - pt);
            __syncthreads();   // the previous tile's reads of dAt and red are done
            // da = dh (1 - h^2) of the tile's rows in 16-byte pieces (rows are
            // padded to 32 floats, so a piece never crosses a row), NB pieces
            // of dh and of h in flight per thread: one round trip for the tile
            // at H <= 320.  Units of chunk j are also stored by column tile
            // j mod NC2.
            // the children of the tile's rows, loaded with the tile
            int lc = -1, rc = -1;
            if (tid < rows) {
                lc = a.lchild[pt + tid];
                rc = a.rchild[pt + tid];
            }
            {
                constexpr int NB = 10;
                int m = m_first, q = q_first;
                while (m < kRT) {
                    float4 dv[NB], hv[NB];
                    int mm[NB], qq[NB];
#pragma unroll
                    for (int i = 0; i < NB; ++i) {
                        mm[i] = m;
                        qq[i] = q;
                        dv[i] = hv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
                        if (m < rows && 4 * q < H) {
                            const int64_t o = int64_t(pt + m) * a.ldh + 4 * q;
                            dv[i] = ld4(a.dh + o);
                            hv[i] = ld4(a.Hn + o);
                        }
                        q += dq;
                        m += dm;
                        if (q >= KP4) {
                            q -= KP4;
                            ++m;
                        }
                    }
                    // (no use of a loaded value above: every load of the batch
                    // is in flight before the first wait)
#pragma unroll
                    for (int i = 0; i < NB; ++i) {
                        if (mm[i] >= kRT) continue;
                        const int k = 4 * qq[i];
                        // columns past H (the row's padding, never written) count as 0
                        if (k + 1 >= H) dv[i].y = hv[i].y = 0.f;
                        if (k + 2 >= H) dv[i].z = hv[i].z = 0.f;
                        if (k + 3 >= H) dv[i].w = hv[i].w = 0.f;
                        float4 da;
                        da.x = dv[i].x * (1.f - hv[i].x * hv[i].x);
                        da.y = dv[i].y * (1.f - hv[i].y * hv[i].y);
                        da.z = dv[i].z * (1.f - hv[i].z * hv[i].z);
                        da.w = dv[i].w * (1.f - hv[i].w * hv[i].w);
                        *reinterpret_cast<float4*>(dAt + mm[i] * sH + k) = da;
                        // unit chunk k / 32 (below NC2, since 2H >= H) is stored by column tile k / 32
                        if (mm[i] < rows && k < H && (k >> 5) == col)
                            persist::store16<persist::kStoreThrough>(
                                rsA, uint32_t((int64_t(pt + mm[i]) * a.lda + k) * 4),
                                make_uint4(__float_as_uint(da.x), __float_as_uint(da.y), __float_as_uint(da.z),
                                           __float_as_uint(da.w)));
                    }
                }
            }
            if (tid < rows) {
                links[tid] = lc;
                links[32 + tid] = rc;
            }
            __syncthreads();
            // D[node m][column c] = sum_k da[m][k] W[k][32 col + c]
            f32x4_t acc[2];
            tile_mfma16(acc, dAt, sH, Ws, sH, KP, wave, lane);
            spill_acc16(acc, red, wave, lane);
            __syncthreads();
            // [dh_L; dh_R] of the tile's rows to the two children
            for (int idx = tid; idx < kRT * 32; idx += kThreads) {
                const int m = idx / 32, c = idx % 32, n = 32 * col + c;
                if (m < rows && n < H2) {
                    const float v = red_sum(red, m, c);
                    if (n < H) store_through(a.dh, int64_t(links[m]) * a.ldh + n, v);
                    else store_through(a.dh, int64_t(links[32 + m]) * a.ldh + (n - H), v);
                }
            }
        }
        persist::barrier_arrive(bar);
        persist::barrier_wait(bar);
    }

    // dW and db over the internal nodes, dealt to the workgroups in turn
    {
        float* Ac = sm;
        float* Bc = sm + 32 * (kKC + 4);
        const int nh = (H + 31) / 32, nh2 = (H2 + 31) / 32;
        const int n_dW = nh * nh2, total = n_dW + nh;
        const int Nint = a.N - a.M0;
        for (int it = int(blockIdx.x); it < total; it += int(gridDim.x)) {
            if (it >= n_dW) {
                // db for 32 units: 16-byte pieces (8 per row, the row padded to
                // 32 floats), 32 row groups, 16 rows in flight per thread, then
                // the groups in order
                const int i = it - n_dW, c4 = 4 * (tid % 8), rg = tid / 8, n = 32 * i + c4;
                constexpr int RG = kThreads / 8;
                float4 s4 = make_float4(0.f, 0.f, 0.f, 0.f);
                for (int q0 = rg; q0 < Nint; q0 += RG * 16) {
                    float4 v[16];
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const int k = q0 + q * RG;
                        v[q] = (k < Nint && n < H) ? ld4(a.dA + int64_t(a.M0 + k) * a.lda + n)
                                                   : make_float4(0.f, 0.f, 0.f, 0.f);
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
                if (tid < 32 && 32 * i + tid < H) {
                    float t2 = 0.f;
                    for (int q = 0; q < RG; ++q) t2 += red[q * 32 + tid];
                    a.db[32 * i + tid] = t2;
                }
                __syncthreads();
                continue;
            }
            const int ti = it / nh2, tj = it % nh2;
            f32x16_t acc;
            zero_acc(acc);
            // dW[32 ti + r][32 tj + c] = sum over internal nodes of da[p][.] [h_L; h_R][p][.]
            node_contraction4<false>(acc, Ac, Bc, Nint, min(32, H - 32 * ti), min(32, H2 - 32 * tj),
                [&](int r4, int k) { return ld4(a.dA + int64_t(a.M0 + k) * a.lda + 32 * ti + r4); },
                [&](int c4, int k) { return ld4(a.HLR + int64_t(k) * a.ldl + 32 * tj + c4); });
            spill_acc(acc, red, wave, lane);
            __syncthreads();
            for (int idx = tid; idx < 32 * 32; idx += kThreads) {
                const int r = idx / 32, c = idx % 32, m = 32 * ti + r, n = 32 * tj + c;
                if (m < H && n < H2) a.dW[int64_t(m) * H2 + n] = red_sum(red, r, c);
            }
            __syncthreads();   // red is read before the next item overwrites it
        }
    }

    // the embedding gradient (reads only the leaves' dh, complete after the
    // last barrier: the roots' copy, or the last level).  Rows without leaves
    // are zero: each workgroup zeroes those of an equal share of the table.
    // Rows with leaves are the sum of their dh rows in ascending leaf order,
    // one group per workgroup in turn.
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
            for (int e = tid; e < H; e += kThreads) a.demb[v * H + e] = 0.f;
        }
        // the leaves of the current row, kThreads at a time: each leaf's dh row
        const float** lsrc = reinterpret_cast<const float**>(sm);
        for (int g = int(blockIdx.x); g < a.nseg; g += int(gridDim.x)) {
            const int64_t v = sid[g];
            const int k0 = off[g], k1 = off[g + 1];
            float s[2] = {0.f, 0.f};   // columns tid and tid + kThreads (H <= kMaxE)
            for (int kb = k0; kb < k1; kb += kThreads) {
                const int nk = min(kThreads, k1 - kb);
                __syncthreads();   // the previous batch of leaves is read
                if (tid < nk) lsrc[tid] = a.dh + int64_t(order[kb + tid]) * a.ldh;
                __syncthreads();
                constexpr int LB = 32;   // leaves per round trip
                for (int k = 0; k < nk; k += LB) {
                    float x0[LB], x1[LB];
#pragma unroll
                    for (int q = 0; q < LB; ++q) {
                        const float* r = k + q < nk ? lsrc[k + q] : nullptr;
                        x0[q] = (r && tid < H) ? r[tid] : 0.f;
                        x1[q] = (r && tid + kThreads < H) ? r[tid + kThreads] : 0.f;
                    }
#pragma unroll
                    for (int q = 0; q < LB; ++q) {
                        s[0] += x0[q];
                        s[1] += x1[q];
                    }
                }
            }
            if (tid < H) a.demb[v * H + tid] = s[0];
            if (tid + kThreads < H) a.demb[v * H + tid + kThreads] = s[1];
        }
    }
}

}  // namespace tpersist
}  // namespace janus
