// Binary TreeLSTM over a batch of trees, evaluated as level-wise frontiers.
//
// The recursive TreeNN program (Section 6.1, footnote 6; recursion turned
// into graph invocations, Section 4.2.1) visits a node after both of its
// subtrees.  Grouping nodes by height gives frontiers of independent cell
// applications: every node of level k depends only on levels < k, so a
// level is one batched contraction plus one pointwise kernel, across all
// trees of the batch at once (the paper's largest gain on TreeNNs comes from
// running independent nodes together, Section 6.3.1 "+PARL").
//
// Node state is stored by level-ordered position p (nodes of a level are
// contiguous), so each level's contraction reads a dense block of rows:
//   level 0 (all leaves):  A_0 = emb[word] W^T + b   (row gather of emb)
//   level k >= 1:          A_k = HLR_k U^T + b       (HLR row = [h_L; h_R])
// The pointwise kernel of a level writes each node's h straight into its
// parent's HLR row (left or right half) or into h_root, so the next level's
// operand is ready without a gather.
//
// Backward, levels from the top down: the pointwise backward of a level
// writes its da rows and its children's dc; the contraction da U sends
// [dh_L; dh_R] to the two children (each node has one parent, so these are
// plain stores).  After the loop: dU = da_int^T HLR, dW = da_leaf^T X_leaf,
// db = column sums of da, dx_leaf = da_leaf W, then the embedding gradient.
#include <vector>

#include "device.hpp"
#include "ops.hpp"

namespace janus {

namespace {

struct TreeWs {
    // level-ordered device schedule
    int32_t* lword = nullptr;    // [N] word of a leaf, -1 otherwise
    int32_t* lchild = nullptr;   // [N] position of left child, -1 for leaves
    int32_t* rchild = nullptr;   // [N]
    int32_t* parent = nullptr;   // [N] 2 * position of parent + side, -1 for roots
    int32_t* rootk = nullptr;    // [N] tree index of a root, -1 otherwise
    int32_t* rootpos = nullptr;  // [K] position of root k
    float* A = nullptr;          // [N x ld5] pre-activations (forward), da (backward)
    float* G = nullptr;          // [N x ld5] gates (i, f_L, f_R, o, u) after activation
    float* C = nullptr;          // [N x H]   cell memory
    float* HLR = nullptr;        // [N x 2H]  children's h of internal nodes (row p - M0)
    float* dh = nullptr;         // [N x H]
    float* dc = nullptr;         // [N x H]
    float* dxl = nullptr;        // [N x E]   gradient of leaf inputs
    float* part = nullptr;
    int64_t ld5 = 0;
};

size_t carve(const janus_treelstm_desc& d, int32_t N, int32_t K, void* base, TreeWs& w) {
    Carver c(base);
    const int H = d.H;
    w.ld5 = round_up(int64_t(5) * H, 4);
    w.lword = c.take<int32_t>(N);
    w.lchild = c.take<int32_t>(N);
    w.rchild = c.take<int32_t>(N);
    w.parent = c.take<int32_t>(N);
    w.rootk = c.take<int32_t>(N);
    w.rootpos = c.take<int32_t>(K);
    w.A = c.take<float>(int64_t(N) * w.ld5);
    w.G = c.take<float>(int64_t(N) * w.ld5);
    w.C = c.take<float>(int64_t(N) * H);
    w.HLR = c.take<float>(int64_t(N) * 2 * H);
    w.dh = c.take<float>(int64_t(N) * H);
    w.dc = c.take<float>(int64_t(N) * H);
    w.dxl = c.take<float>(int64_t(N) * d.E);
    w.part = c.take<float>(colsum_partial_floats(5 * H));
    return c.off + 256;
}

// one schedule array set per call, in level order
struct TreeHost {
    std::vector<int32_t> lword, lchild, rchild, parent, rootk, rootpos;
};

void build_host(const janus_tree_batch* t, const TreeSchedule& s, TreeHost& h) {
    const int32_t N = s.N;
    h.lword.assign(N, -1);
    h.lchild.assign(N, -1);
    h.rchild.assign(N, -1);
    h.parent.assign(N, -1);
    h.rootk.assign(N, -1);
    h.rootpos.assign(t->num_trees, 0);
    for (int32_t p = 0; p < N; ++p) {
        const int32_t n = s.level_nodes[p];
        if (t->left[n] < 0) {
            h.lword[p] = t->word[n];
        } else {
            const int32_t pl = s.pos[t->left[n]], pr = s.pos[t->right[n]];
            h.lchild[p] = pl;
            h.rchild[p] = pr;
            h.parent[pl] = 2 * p;
            h.parent[pr] = 2 * p + 1;
        }
    }
    for (int32_t k = 0; k < t->num_trees; ++k) {
        const int32_t p = s.pos[t->root[k]];
        h.rootk[p] = k;
        h.rootpos[k] = p;
    }
}

__device__ __forceinline__ float sig(float x) { return sigmoidf_(x); }

__global__ void tree_fwd_point_kernel(int p0, int rows, int H, int M0, int64_t ld5, const float* A, float* G,
                                      float* C, const int32_t* lchild, const int32_t* rchild, const int32_t* parent,
                                      const int32_t* rootk, float* HLR, float* h_root) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(rows) * H) return;
    const int p = p0 + int(i / H), j = int(i % H);
    const float* a = A + int64_t(p) * ld5 + j;
    const float gi = sig(a[0]), gl = sig(a[H]), gr = sig(a[2 * H]), go = sig(a[3 * H]), gu = tanhf_(a[4 * H]);
    const int lc = lchild[p], rc = rchild[p];
    const float cl = lc >= 0 ? C[int64_t(lc) * H + j] : 0.f;
    const float cr = rc >= 0 ? C[int64_t(rc) * H + j] : 0.f;
    const float c = gi * gu + gl * cl + gr * cr;
    const float h = go * tanhf_(c);
    C[int64_t(p) * H + j] = c;
    float* g = G + int64_t(p) * ld5 + j;
    g[0] = gi;
    g[H] = gl;
    g[2 * H] = gr;
    g[3 * H] = go;
    g[4 * H] = gu;
    const int par = parent[p];
    if (par >= 0) HLR[int64_t((par >> 1) - M0) * 2 * H + (par & 1) * H + j] = h;
    else h_root[int64_t(rootk[p]) * H + j] = h;
}

__global__ void tree_bwd_init_kernel(int K, int H, const int32_t* rootpos, const float* dh_root, float* dh, float* dc) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(K) * H) return;
    const int k = int(i / H), j = int(i % H);
    const int p = rootpos[k];
    dh[int64_t(p) * H + j] = dh_root[i];
    dc[int64_t(p) * H + j] = 0.f;
}

__global__ void tree_bwd_point_kernel(int p0, int rows, int H, int64_t ld5, const float* G, const float* C,
                                      const float* dh, float* dc, const int32_t* lchild, const int32_t* rchild,
                                      float* dA) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(rows) * H) return;
    const int p = p0 + int(i / H), j = int(i % H);
    const float* g = G + int64_t(p) * ld5 + j;
    const float gi = g[0], gl = g[H], gr = g[2 * H], go = g[3 * H], gu = g[4 * H];
    const int lc = lchild[p], rc = rchild[p];
    const float cl = lc >= 0 ? C[int64_t(lc) * H + j] : 0.f;
    const float cr = rc >= 0 ? C[int64_t(rc) * H + j] : 0.f;
    const float c = C[int64_t(p) * H + j];
    const float dhv = dh[int64_t(p) * H + j];
    const float tau = tanhf_(c);
    const float d_o = dhv * tau;
    const float dct = dc[int64_t(p) * H + j] + dhv * go * (1.f - tau * tau);
    float* da = dA + int64_t(p) * ld5 + j;
    da[0] = dct * gu * gi * (1.f - gi);
    da[H] = dct * cl * gl * (1.f - gl);
    da[2 * H] = dct * cr * gr * (1.f - gr);
    da[3 * H] = d_o * go * (1.f - go);
    da[4 * H] = dct * gi * (1.f - gu * gu);
    if (lc >= 0) {
        dc[int64_t(lc) * H + j] = dct * gl;
        dc[int64_t(rc) * H + j] = dct * gr;
    }
}

// [dh_L; dh_R] = da U for the nodes of one level, scattered to the children
template <class Cfg, bool AL>
__global__ __launch_bounds__(Cfg::NT) void tree_dh_kernel(int p0, int rows, int H, int64_t ld5, const float* dA,
                                                          const float* U, const int32_t* lchild,
                                                          const int32_t* rchild, float* dh) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    float* sA = reinterpret_cast<float*>(smem_raw);
    float* sB = sA + Cfg::BM * Cfg::LD;
    const int tid = threadIdx.x;
    const int n0 = blockIdx.x * Cfg::BN, m0 = blockIdx.y * Cfg::BM;
    const int N = 2 * H;
    LoaderK<float, Cfg::BM, Cfg::BK, Cfg::NT, AL> la;
    LoaderT<float, Cfg::BN, Cfg::BK, Cfg::NT, AL> lb;
    la.init(dA + int64_t(p0 + m0) * ld5, ld5, 0, RowsContig{rows - m0}, tid);
    lb.init(U, N, nullptr, n0, N);
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop<Cfg>(acc, la, lb, 5 * H, sA, sB, tid);
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int j = 0; j < Cfg::FN; ++j) {
        const int col = n0 + Cfg::wave_col0(wave) + j * 32 + acc_col(lane);
        if (col >= N) continue;
#pragma unroll
        for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = m0 + Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane);
                if (row >= rows) continue;
                const int p = p0 + row;
                if (col < H) dh[int64_t(lchild[p]) * H + col] = acc[i][j][v];
                else dh[int64_t(rchild[p]) * H + col - H] = acc[i][j][v];
            }
    }
}

using TreeCfg = TileCfg<float, 64, 64, 32, 2, 2>;

janus_status check(const janus_treelstm_desc* d) {
    if (!d || d->E <= 0 || d->H <= 0 || d->V <= 0) return JANUS_ERR_INVALID_ARG;
    if (d->dtype != JANUS_F32) return JANUS_ERR_UNSUPPORTED;
    return JANUS_OK;
}

janus_status upload_tree(const janus_tree_batch* t, const TreeSchedule& s, const TreeWs& w, hipStream_t st) {
    TreeHost h;
    build_host(t, s, h);
    const size_t nb = sizeof(int32_t) * s.N;
    janus_status e;
    if ((e = upload(w.lword, h.lword.data(), nb, st)) != JANUS_OK) return e;
    if ((e = upload(w.lchild, h.lchild.data(), nb, st)) != JANUS_OK) return e;
    if ((e = upload(w.rchild, h.rchild.data(), nb, st)) != JANUS_OK) return e;
    if ((e = upload(w.parent, h.parent.data(), nb, st)) != JANUS_OK) return e;
    if ((e = upload(w.rootk, h.rootk.data(), nb, st)) != JANUS_OK) return e;
    return upload(w.rootpos, h.rootpos.data(), sizeof(int32_t) * t->num_trees, st);
}

janus_status prepare(const janus_treelstm_desc* d, const janus_tree_batch* t, void* ws, size_t ws_bytes,
                     TreeSchedule& s, TreeWs& w) {
    janus_status e = check(d);
    if (e != JANUS_OK) return e;
    if ((e = build_tree_schedule(t, d->V, s)) != JANUS_OK) return e;
    if (!ws || ws_bytes < carve(*d, s.N, t->num_trees, nullptr, w) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    carve(*d, s.N, t->num_trees, ws, w);
    return JANUS_OK;
}

}  // namespace

}  // namespace janus

using namespace janus;

extern "C" size_t janus_treelstm_workspace_bytes(const janus_treelstm_desc* d, int32_t max_nodes,
                                                 int32_t max_trees) {
    if (check(d) != JANUS_OK || max_nodes <= 0 || max_trees <= 0) return 0;
    TreeWs w;
    return carve(*d, max_nodes, max_trees, nullptr, w);
}

extern "C" janus_status janus_treelstm_fwd(const janus_treelstm_desc* d, const janus_tree_batch* t, const void* emb,
                                           const void* W, const void* U, const void* b, void* h_root, void* ws,
                                           size_t ws_bytes, void* stream) {
    if (!emb || !W || !U || !b || !h_root) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeWs w;
    janus_status e = prepare(d, t, ws, ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if ((e = upload_tree(t, s, w, st)) != JANUS_OK) return e;
    const int H = d->H, E = d->E;
    const int M0 = s.level_offsets[1];
    for (int k = 0; k < s.num_levels; ++k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        GemmDesc g;
        g.dtype = JANUS_F32;
        g.M = rows;
        g.N = 5 * H;
        if (k == 0) {
            g.K = E;
            g.A = emb;
            g.lda = E;
            g.a_idx = w.lword;
            g.B = W;
            g.ldb = E;
        } else {
            g.K = 2 * H;
            g.A = w.HLR + int64_t(p0 - M0) * 2 * H;
            g.lda = 2 * H;
            g.B = U;
            g.ldb = 2 * H;
        }
        g.C = w.A + int64_t(p0) * w.ld5;
        g.ldc = w.ld5;
        g.c_f32 = true;
        g.bias = b;
        if ((e = gemm(g, st)) != JANUS_OK) return e;
        const int64_t n = int64_t(rows) * H;
        TraceScope trace("tree_fwd_point", 0.0, 4.0 * n * 14.0, st);
        hipLaunchKernelGGL(tree_fwd_point_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows, H, M0,
                           w.ld5, w.A, w.G, w.C, w.lchild, w.rchild, w.parent, w.rootk, w.HLR,
                           static_cast<float*>(h_root));
        JANUS_LAUNCH_CHECK();
    }
    return JANUS_OK;
}

extern "C" janus_status janus_treelstm_bwd(const janus_treelstm_desc* d, const janus_tree_batch* t, const void* emb,
                                           const void* W, const void* U, void* ws, size_t ws_bytes,
                                           const void* dh_root, float* demb, float* dW, float* dU, float* db,
                                           void* stream) {
    if (!emb || !W || !U || !dh_root || !demb || !dW || !dU || !db) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeWs w;
    janus_status e = prepare(d, t, ws, ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    const int M0 = s.level_offsets[1];
    if (M0 > kMaxEmbedBwdRows) return JANUS_ERR_UNSUPPORTED;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if ((e = upload_tree(t, s, w, st)) != JANUS_OK) return e;
    const int H = d->H, E = d->E, N = s.N;
    const int64_t kh = int64_t(t->num_trees) * H;
    {
    TraceScope trace("tree_bwd_init", 0.0, 12.0 * kh, st);
    hipLaunchKernelGGL(tree_bwd_init_kernel, dim3(unsigned((kh + 255) / 256)), dim3(256), 0, st, t->num_trees, H,
                       w.rootpos, static_cast<const float*>(dh_root), w.dh, w.dc);
    JANUS_LAUNCH_CHECK();
    }
    const bool al = (int64_t(2) * H * 4) % 16 == 0 && reinterpret_cast<uintptr_t>(U) % 16 == 0;
    for (int k = s.num_levels - 1; k >= 0; --k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        const int64_t n = int64_t(rows) * H;
        {
        TraceScope trace("tree_bwd_point", 0.0, 4.0 * n * 17.0, st);
        hipLaunchKernelGGL(tree_bwd_point_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows, H,
                           w.ld5, w.G, w.C, w.dh, w.dc, w.lchild, w.rchild, w.A);
        JANUS_LAUNCH_CHECK();
        }
        if (k == 0) break;
        dim3 grid((2 * H + TreeCfg::BN - 1) / TreeCfg::BN, (rows + TreeCfg::BM - 1) / TreeCfg::BM);
        TraceScope trace("tree_dh_gemm", 2.0 * rows * 2.0 * H * 5.0 * H,
                         4.0 * (double(rows) * 5 * H + 10.0 * H * H + 2.0 * rows * H), st);
        if (al)
            hipLaunchKernelGGL((tree_dh_kernel<TreeCfg, true>), grid, dim3(TreeCfg::NT), TreeCfg::SMEM_BYTES, st, p0,
                               rows, H, w.ld5, w.A, static_cast<const float*>(U), w.lchild, w.rchild, w.dh);
        else
            hipLaunchKernelGGL((tree_dh_kernel<TreeCfg, false>), grid, dim3(TreeCfg::NT), TreeCfg::SMEM_BYTES, st, p0,
                               rows, H, w.ld5, w.A, static_cast<const float*>(U), w.lchild, w.rchild, w.dh);
        JANUS_LAUNCH_CHECK();
    }
    // dU = da_int^T HLR  (K = internal nodes)
    GemmDesc g;
    g.dtype = JANUS_F32;
    g.M = 5 * H;
    g.N = 2 * H;
    g.K = N - M0;
    g.a_t = true;
    g.A = w.A + int64_t(M0) * w.ld5;
    g.lda = w.ld5;
    g.b_t = true;
    g.B = w.HLR;
    g.ldb = 2 * H;
    g.C = dU;
    g.ldc = 2 * H;
    g.c_f32 = true;
    if ((e = gemm(g, st)) != JANUS_OK) return e;
    // dW = da_leaf^T emb[word]  (K = leaves, gathered rows of emb)
    g.N = E;
    g.K = M0;
    g.A = w.A;
    g.B = emb;
    g.ldb = E;
    g.b_idx = w.lword;
    g.C = dW;
    g.ldc = E;
    if ((e = gemm(g, st)) != JANUS_OK) return e;
    if ((e = colsum(JANUS_F32, w.A, N, 5 * H, w.ld5, db, w.part, st)) != JANUS_OK) return e;
    // dx_leaf = da_leaf W, then the embedding gradient
    GemmDesc q;
    q.dtype = JANUS_F32;
    q.M = M0;
    q.N = E;
    q.K = 5 * H;
    q.A = w.A;
    q.lda = w.ld5;
    q.b_t = true;
    q.B = W;
    q.ldb = E;
    q.C = w.dxl;
    q.ldc = E;
    q.c_f32 = true;
    if ((e = gemm(q, st)) != JANUS_OK) return e;
    return embed_backward(JANUS_F32, w.dxl, w.lword, M0, E, demb, d->V, st);
}
