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
#include <algorithm>
#include <cstdlib>
#include <mutex>
#include <vector>

#include "device.hpp"
#include "ops.hpp"
#include "simt.hpp"
#include "tree_persist.hpp"
#include "treernn_persist.hpp"

namespace janus {

namespace {

using tpersist::kMaxTreeGrid;
using tpersist::TreeDev;
using tpersist::tree_dev;
using tpersist::tree_persistent_launch;

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
    float* Wt = nullptr;         // [E x 5H]  W transposed (forward)
    float* Ut = nullptr;         // [2H x 5H] U transposed (forward)
    float* part = nullptr;
    int32_t* seg = nullptr;      // the leaves grouped by word, for the embedding gradient
    int64_t ld5 = 0;
    // persistent path: level offsets and the barrier's counters (carved right
    // after the schedule arrays and before `seg`, so that each direction's
    // upload is one copy), and node rows padded to whole 128-byte lines
    int32_t* loff = nullptr;     // [N + 1]
    tpersist::TreeSync* tsync = nullptr;
    float* Gp = nullptr;         // [N x ldg] gates
    float* Cp = nullptr;         // [N x ldc]
    float* HLRp = nullptr;       // [N x ldl]
    float* dhp = nullptr;        // [N x ldc]
    float* dcp = nullptr;        // [N x ldc]
    float* dAp = nullptr;        // [N x lda]
    float* dxp = nullptr;        // [N x ldx]
    int64_t ldg = 0, ldc = 0, ldl = 0, lda = 0, ldx = 0;
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
    w.loff = c.take<int32_t>(int64_t(N) + 1);
    w.tsync = c.take<tpersist::TreeSync>(1);
    // the leaves grouped by word, and (persistent backward) each workgroup's
    // first group of the embedding rows: one entry per workgroup, at most one
    // per CU of the devices the library plans for
    w.seg = c.take<int32_t>(int64_t(embed_seg_ints(N)) + kMaxTreeGrid);
    w.A = c.take<float>(int64_t(N) * w.ld5);
    w.G = c.take<float>(int64_t(N) * w.ld5);
    w.C = c.take<float>(int64_t(N) * H);
    w.HLR = c.take<float>(int64_t(N) * 2 * H);
    w.dh = c.take<float>(int64_t(N) * H);
    w.dc = c.take<float>(int64_t(N) * H);
    w.dxl = c.take<float>(int64_t(N) * d.E);
    w.Wt = c.take<float>(int64_t(d.E) * 5 * H);
    w.Ut = c.take<float>(int64_t(2) * H * 5 * H);
    w.part = c.take<float>(colsum_partial_floats(5 * H));
    w.ldg = w.lda = round_up(int64_t(5) * H, 32);
    w.ldc = round_up(H, 32);
    w.ldl = round_up(int64_t(2) * H, 32);
    w.ldx = round_up(d.E, 32);
    w.Gp = c.take<float>(int64_t(N) * w.ldg);
    w.Cp = c.take<float>(int64_t(N) * w.ldc);
    w.HLRp = c.take<float>(int64_t(N) * w.ldl);
    w.dhp = c.take<float>(int64_t(N) * w.ldc);
    w.dcp = c.take<float>(int64_t(N) * w.ldc);
    w.dAp = c.take<float>(int64_t(N) * w.lda);
    w.dxp = c.take<float>(int64_t(N) * w.ldx);
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

// One backward level k >= 1 in one launch: block (x, y) first applies the
// cell backward to the 8 rows y*8.. of the level (all 5H gate columns; every
// column block does this, block x = 0 also writes da and the children's dc
// to memory), straight into the LDS slab, then computes columns x*64.. of
// [dh_L; dh_R] = da U with K = 5H split over its waves, as simt_gemm_kernel.
__global__ __launch_bounds__(64 * kSimtWaves) void tree_bwd_level_kernel(int p0, int rows, int H, int64_t ld5,
                                                                         const float* G, const float* C,
                                                                         const float* dh_in, float* dc,
                                                                         const int32_t* lchild, const int32_t* rchild,
                                                                         float* dA, const float* U, float* dh) {
    __shared__ __align__(16) float sA[kSimtKc][kSimtRows];
    __shared__ float red[kSimtWaves][kSimtRows][kSimtCols];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int N = 2 * H, K = 5 * H;
    const int n = blockIdx.x * kSimtCols + lane;
    const int m0 = blockIdx.y * kSimtRows;
    const bool writer = blockIdx.x == 0;
    for (int i = tid; i < kSimtRows * H; i += 64 * kSimtWaves) {
        const int r = i / H, j = i - r * H, m = m0 + r;
        float da[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
        if (m < rows) {
            const int p = p0 + m;
            const float* g = G + int64_t(p) * ld5 + j;
            const float gi = g[0], gl = g[H], gr = g[2 * H], go = g[3 * H], gu = g[4 * H];
            const int lc = lchild[p], rc = rchild[p];
            const float cl = C[int64_t(lc) * H + j], cr = C[int64_t(rc) * H + j];
            const float c = C[int64_t(p) * H + j];
            const float dhv = dh_in[int64_t(p) * H + j];
            const float tau = tanhf_(c);
            const float d_o = dhv * tau;
            const float dct = dc[int64_t(p) * H + j] + dhv * go * (1.f - tau * tau);
            da[0] = dct * gu * gi * (1.f - gi);
            da[1] = dct * cl * gl * (1.f - gl);
            da[2] = dct * cr * gr * (1.f - gr);
            da[3] = d_o * go * (1.f - go);
            da[4] = dct * gi * (1.f - gu * gu);
            if (writer) {
                float* dst = dA + int64_t(p) * ld5 + j;
#pragma unroll
                for (int q = 0; q < 5; ++q) dst[q * H] = da[q];
                dc[int64_t(lc) * H + j] = dct * gl;
                dc[int64_t(rc) * H + j] = dct * gr;
            }
        }
#pragma unroll
        for (int q = 0; q < 5; ++q) sA[q * H + j][r] = da[q];
    }
    __syncthreads();
    float acc[kSimtRows];
#pragma unroll
    for (int r = 0; r < kSimtRows; ++r) acc[r] = 0.f;
    const int kb = wave * K / kSimtWaves, ke = (wave + 1) * K / kSimtWaves;
    if (n < N) {
#pragma unroll 16
        for (int k = kb; k < ke; ++k) {
            const float bv = U[int64_t(k) * N + n];
            const float4 a0 = *reinterpret_cast<const float4*>(&sA[k][0]);
            const float4 a1 = *reinterpret_cast<const float4*>(&sA[k][4]);
            acc[0] += a0.x * bv; acc[1] += a0.y * bv; acc[2] += a0.z * bv; acc[3] += a0.w * bv;
            acc[4] += a1.x * bv; acc[5] += a1.y * bv; acc[6] += a1.z * bv; acc[7] += a1.w * bv;
        }
    }
#pragma unroll
    for (int r = 0; r < kSimtRows; ++r) red[wave][r][lane] = acc[r];
    __syncthreads();
    const int r = wave, m = m0 + r;
    if (m >= rows || n >= N) return;
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < kSimtWaves; ++w) sum += red[w][r][lane];
    const int p = p0 + m;
    if (n < H) dh[int64_t(lchild[p]) * H + n] = sum;
    else dh[int64_t(rchild[p]) * H + n - H] = sum;
}

janus_status check(const janus_treelstm_desc* d) {
    if (!d || d->E <= 0 || d->H <= 0 || d->V <= 0) return JANUS_ERR_INVALID_ARG;
    if (d->dtype != JANUS_F32) return JANUS_ERR_UNSUPPORTED;
    return JANUS_OK;
}

// `keep`: receives the host arrays (the backward groups the leaves by word
// from them)
janus_status upload_tree(const janus_tree_batch* t, const TreeSchedule& s, const TreeWs& w, hipStream_t st,
                         TreeHost* keep = nullptr) {
    TreeHost local;
    TreeHost& h = keep ? *keep : local;
    build_host(t, s, h);
    const size_t nb = sizeof(int32_t) * s.N;
    // carved one after another (only the level offsets between them): one
    // copy.  The barrier block is zeroed too, so the device report of a call
    // on this path reads no stale flag.
    const std::vector<char> zero_sync(sizeof(tpersist::TreeSync), 0);
    const UploadPiece pieces[] = {{w.lword, h.lword.data(), nb},   {w.lchild, h.lchild.data(), nb},
                                  {w.rchild, h.rchild.data(), nb}, {w.parent, h.parent.data(), nb},
                                  {w.rootk, h.rootk.data(), nb},
                                  {w.rootpos, h.rootpos.data(), sizeof(int32_t) * t->num_trees},
                                  {w.tsync, zero_sync.data(), zero_sync.size()}};
    return upload_pieces(pieces, 7, st);
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


// ------------------------------------------------------- persistent path

// Grid and LDS of the persistent TreeLSTM kernels: one workgroup per CU at
// most, the grid a multiple of the unit groups (forward) and of the column
// tiles (backward) so every workgroup holds one weight slice.  Off with
// JANUS_TREE_PERSIST=0, where a slice does not fit the LDS (about H > 170
// for the backward's U columns) or for inputs wider than 512; the
// level-by-level kernels run then.
struct TreePlan {
    bool on = false;
    int ngroups = 0, fwd_grid = 0, ncol = 0, bwd_grid = 0;
    size_t fwd_lds = 0, bwd_lds = 0;
};
TreePlan tree_plan(const janus_treelstm_desc& d) {
    TreePlan p;
    const char* e = getenv("JANUS_TREE_PERSIST");
    if (e && e[0] == '0') return p;
    const TreeDev dev = tree_dev();
    if (dev.cus <= 0 || dev.lds == 0) return p;
    if (d.E > tpersist::kMaxE || d.H > tpersist::kUC * tpersist::kMaxCh) return p;
    p.ngroups = (d.H + tpersist::kUG - 1) / tpersist::kUG;
    p.ncol = (2 * d.H + 31) / 32;
    if (p.ngroups > dev.cus || p.ncol > dev.cus) return p;
    const int cus = dev.cus < kMaxTreeGrid ? dev.cus : kMaxTreeGrid;
    p.fwd_grid = p.ngroups * (cus / p.ngroups);
    p.bwd_grid = p.ncol * (cus / p.ncol);
    p.fwd_lds = size_t(tpersist::fwd_lds_floats(d.E, d.H)) * sizeof(float);
    p.bwd_lds = size_t(tpersist::bwd_lds_floats(d.H)) * sizeof(float);
    p.on = p.fwd_lds <= dev.lds && p.bwd_lds <= dev.lds;
    return p;
}


// Forward on the persistent path: the schedule, the level offsets and the
// barrier's counters (with its error flag) go over in one copy, then one
// launch runs every level.
janus_status treelstm_fwd_persistent_call(const janus_treelstm_desc& d, const janus_tree_batch* t,
                                          const TreeSchedule& s, const TreeWs& w, const TreePlan& plan,
                                          const void* emb, const void* W, const void* U, const void* b, void* h_root,
                                          hipStream_t st) {
    TreeHost h;
    build_host(t, s, h);
    const size_t nb = sizeof(int32_t) * s.N;
    const std::vector<char> zero_sync(sizeof(tpersist::TreeSync), 0);
    const UploadPiece pieces[] = {{w.lword, h.lword.data(), nb},
                                  {w.lchild, h.lchild.data(), nb},
                                  {w.rchild, h.rchild.data(), nb},
                                  {w.parent, h.parent.data(), nb},
                                  {w.rootk, h.rootk.data(), nb},
                                  {w.rootpos, h.rootpos.data(), sizeof(int32_t) * t->num_trees},
                                  {w.loff, s.level_offsets.data(), sizeof(int32_t) * s.level_offsets.size()},
                                  {w.tsync, zero_sync.data(), zero_sync.size()}};
    janus_status e = upload_pieces(pieces, 8, st);
    if (e != JANUS_OK) return e;
    tpersist::FwdArgs a;
    a.E = d.E;
    a.H = d.H;
    a.N = s.N;
    a.M0 = s.level_offsets[1];
    a.nlev = s.num_levels;
    a.ngroups = plan.ngroups;
    a.loff = w.loff;
    a.lword = w.lword;
    a.lchild = w.lchild;
    a.rchild = w.rchild;
    a.parent = w.parent;
    a.rootk = w.rootk;
    a.emb = static_cast<const float*>(emb);
    a.W = static_cast<const float*>(W);
    a.U = static_cast<const float*>(U);
    a.b = static_cast<const float*>(b);
    a.G = w.Gp;
    a.ldg = w.ldg;
    a.C = w.Cp;
    a.ldc = w.ldc;
    a.HLR = w.HLRp;
    a.ldl = w.ldl;
    a.h_root = static_cast<float*>(h_root);
    a.sync = w.tsync;
    static size_t attr = 0;
    const double flops = 2.0 * 5.0 * d.H * (double(a.M0) * d.E + double(s.N - a.M0) * 2.0 * d.H);
    TraceScope trace("treelstm_fwd_persistent", flops, 0.0, st);
    return tree_persistent_launch(tpersist::treelstm_fwd_persistent, plan.fwd_grid, plan.fwd_lds, a, st, attr);
}

// Backward on the persistent path: the schedule is the forward's (the
// workspace is unchanged between the two calls); the leaves grouped by word
// and the barrier's counters (not its error flag) go over in one copy, then
// one launch runs the levels, the weight and input gradients and the
// embedding gradient.
janus_status treelstm_bwd_persistent_call(const janus_treelstm_desc& d, const janus_tree_batch* t,
                                          const TreeSchedule& s, const TreeWs& w, const TreePlan& plan,
                                          const void* emb, const void* W, const void* U, const void* dh_root,
                                          float* demb, float* dW, float* dU, float* db, hipStream_t st) {
    TreeHost h;
    build_host(t, s, h);
    const int M0 = s.level_offsets[1];
    std::vector<int32_t> seg;
    const int nseg = embed_segments(h.lword.data(), M0, d.V, seg);
    // first group of each workgroup's rows [V w / grid, V (w + 1) / grid)
    const int32_t* sid = seg.data() + M0 + nseg + 1;
    for (int g = 0; g < plan.bwd_grid; ++g) {
        const int64_t v0 = int64_t(d.V) * g / plan.bwd_grid;
        seg.push_back(int32_t(std::lower_bound(sid, sid + nseg, v0) - sid));
        sid = seg.data() + M0 + nseg + 1;   // push_back may move the array
    }
    const size_t counters = sizeof(tpersist::TreeSync) - tpersist::kTreeSyncCounters;
    const std::vector<char> zero_counters(counters, 0);
    const UploadPiece pieces[] = {
        {reinterpret_cast<char*>(w.tsync) + tpersist::kTreeSyncCounters, zero_counters.data(), counters},
        {w.seg, seg.data(), seg.size() * sizeof(int32_t)}};
    janus_status e = upload_pieces(pieces, 2, st);
    if (e != JANUS_OK) return e;
    tpersist::BwdArgs a;
    a.E = d.E;
    a.H = d.H;
    a.N = s.N;
    a.M0 = M0;
    a.nlev = s.num_levels;
    a.ncol = plan.ncol;
    a.nseg = nseg;
    a.V = d.V;
    a.loff = w.loff;
    a.lword = w.lword;
    a.lchild = w.lchild;
    a.rchild = w.rchild;
    a.rootk = w.rootk;
    a.seg = w.seg;
    a.emb = static_cast<const float*>(emb);
    a.W = static_cast<const float*>(W);
    a.U = static_cast<const float*>(U);
    a.G = w.Gp;
    a.ldg = w.ldg;
    a.C = w.Cp;
    a.ldc = w.ldc;
    a.HLR = w.HLRp;
    a.ldl = w.ldl;
    a.dh_root = static_cast<const float*>(dh_root);
    a.dh = w.dhp;
    a.dc = w.dcp;
    a.dA = w.dAp;
    a.lda = w.lda;
    a.dxl = w.dxp;
    a.ldx = w.ldx;
    a.demb = demb;
    a.dW = dW;
    a.dU = dU;
    a.db = db;
    a.sync = w.tsync;
    static size_t attr = 0;
    // [dh_L; dh_R] = dA U on internal nodes, dU, dW and dx_leaf
    const double Nint = double(s.N - M0);
    const double flops = 2.0 * 5.0 * d.H * (Nint * 2.0 * d.H * 2.0 + double(M0) * d.E * 2.0);
    TraceScope trace("treelstm_bwd_persistent", flops, 0.0, st);
    return tree_persistent_launch(tpersist::treelstm_bwd_persistent, plan.bwd_grid, plan.bwd_lds, a, st, attr);
}

// ------------------------------------------------------------------ TreeRNN
// Binary TreeRNN on the same frontier schedule: a leaf's h is its word
// vector (embedding width = H), an internal node h = tanh(W [h_L; h_R] + b).
// Forward: the leaves copy their embedding rows into their parents' [h_L;
// h_R] rows; each internal level is one contraction with W^T whose epilogue
// adds the bias, applies tanh, saves h and sends it to the parent.
// Backward, levels from the top down, one contraction per level: its a slab
// is da = dh (1 - h^2) (column block 0 also stores da) and its epilogue sends
// [dh_L; dh_R] = da W to the two children; after the loop dW = da^T HLR and
// db = column sums of da over the internal nodes, and the leaves' dh is the
// gradient of their word vectors.
struct TreeRnnWs {
    TreeWs s;                    // schedule arrays (lword .. rootpos, loff, tsync, seg) only
    float* A = nullptr;          // [N x H] pre-activations (forward), da (backward)
    float* Hn = nullptr;         // [N x H] h of every node
    float* HLR = nullptr;        // [N - M0 x 2H] children's h of internal nodes
    float* dh = nullptr;         // [N x H]
    float* Wt = nullptr;         // [2H x H] W transposed
    float* part = nullptr;
    // persistent path: node rows padded to whole 128-byte lines
    float* Hnp = nullptr;        // [N x ldh]
    float* HLRp = nullptr;       // [N x ldl]
    float* dhp = nullptr;        // [N x ldh]
    float* dAp = nullptr;        // [N x ldh]
    int64_t ldh = 0, ldl = 0;
};

size_t carve_rnn(const janus_treelstm_desc& d, int32_t N, int32_t K, void* base, TreeRnnWs& w) {
    Carver c(base);
    const int H = d.H;
    w.s.lword = c.take<int32_t>(N);
    w.s.lchild = c.take<int32_t>(N);
    w.s.rchild = c.take<int32_t>(N);
    w.s.parent = c.take<int32_t>(N);
    w.s.rootk = c.take<int32_t>(N);
    w.s.rootpos = c.take<int32_t>(K);
    // the persistent path's level offsets, barrier counters and leaf groups
    // follow the schedule arrays, so each direction's upload is one copy
    w.s.loff = c.take<int32_t>(int64_t(N) + 1);
    w.s.tsync = c.take<tpersist::TreeSync>(1);
    w.s.seg = c.take<int32_t>(int64_t(embed_seg_ints(N)) + kMaxTreeGrid);
    w.A = c.take<float>(int64_t(N) * H);
    w.Hn = c.take<float>(int64_t(N) * H);
    w.HLR = c.take<float>(int64_t(N) * 2 * H);
    w.dh = c.take<float>(int64_t(N) * H);
    w.Wt = c.take<float>(int64_t(2) * H * H);
    w.part = c.take<float>(colsum_partial_floats(H));
    w.ldh = round_up(H, 32);
    w.ldl = round_up(int64_t(2) * H, 32);
    w.Hnp = c.take<float>(int64_t(N) * w.ldh);
    w.HLRp = c.take<float>(int64_t(N) * w.ldl);
    w.dhp = c.take<float>(int64_t(N) * w.ldh);
    w.dAp = c.take<float>(int64_t(N) * w.ldh);
    return c.off + 256;
}

// h of node p (level-ordered) to its parent's [h_L; h_R] row or to h_root
__device__ __forceinline__ void rnn_send(int p, int j, int H, int M0, float h, const int32_t* parent,
                                         const int32_t* rootk, float* HLR, float* h_root) {
    const int par = parent[p];
    if (par >= 0) HLR[int64_t((par >> 1) - M0) * 2 * H + (par & 1) * H + j] = h;
    else h_root[int64_t(rootk[p]) * H + j] = h;
}

__global__ void treernn_leaf_kernel(int rows, int H, int M0, const int32_t* lword, const float* emb,
                                    const int32_t* parent, const int32_t* rootk, float* Hn, float* HLR,
                                    float* h_root) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(rows) * H) return;
    const int p = int(i / H), j = int(i % H);
    const float h = emb[int64_t(lword[p]) * H + j];
    Hn[i] = h;
    rnn_send(p, j, H, M0, h, parent, rootk, HLR, h_root);
}

janus_status check_rnn(const janus_treelstm_desc* d) {
    janus_status e = check(d);
    if (e != JANUS_OK) return e;
    return d->E == d->H ? JANUS_OK : JANUS_ERR_INVALID_ARG;
}

janus_status prepare_rnn(const janus_treelstm_desc* d, const janus_tree_batch* t, void* ws, size_t ws_bytes,
                         TreeSchedule& s, TreeRnnWs& w) {
    janus_status e = check_rnn(d);
    if (e != JANUS_OK) return e;
    if ((e = build_tree_schedule(t, d->V, s)) != JANUS_OK) return e;
    if (!ws || ws_bytes < carve_rnn(*d, s.N, t->num_trees, nullptr, w) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    carve_rnn(*d, s.N, t->num_trees, ws, w);
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
    const TreePlan plan = tree_plan(*d);
    if (plan.on) return treelstm_fwd_persistent_call(*d, t, s, w, plan, emb, W, U, b, h_root, st);
    if ((e = upload_tree(t, s, w, st)) != JANUS_OK) return e;
    const int H = d->H, E = d->E;
    const int M0 = s.level_offsets[1];
    // the level contractions read W and U transposed (N = 5H contiguous)
    if ((e = transpose_f32(static_cast<const float*>(W), 5 * H, E, w.Wt, st)) != JANUS_OK) return e;
    if ((e = transpose_f32(static_cast<const float*>(U), 5 * H, 2 * H, w.Ut, st)) != JANUS_OK) return e;
    const float* bias = static_cast<const float*>(b);
    for (int k = 0; k < s.num_levels; ++k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        // A_k = a . W^T + b over the rows of level k: leaves gather their
        // embedding rows, internal nodes read [h_L; h_R]
        if (k == 0)
            e = simt_gemm<false, kSimtStore>("tree_level_gemm", rows, 5 * H, E, static_cast<const float*>(emb), E,
                                             w.lword, w.Wt, 5 * H, nullptr, bias, w.A, w.ld5, st);
        else
            e = simt_gemm<false, kSimtStore>("tree_level_gemm", rows, 5 * H, 2 * H,
                                             w.HLR + int64_t(p0 - M0) * 2 * H, 2 * H, nullptr, w.Ut, 5 * H, nullptr,
                                             bias, w.A + int64_t(p0) * w.ld5, w.ld5, st);
        if (e != JANUS_OK) return e;
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
    hipStream_t st = static_cast<hipStream_t>(stream);
    const TreePlan plan = tree_plan(*d);
    if (plan.on)
        return treelstm_bwd_persistent_call(*d, t, s, w, plan, emb, W, U, dh_root, demb, dW, dU, db, st);
    TreeHost host;
    if ((e = upload_tree(t, s, w, st, &host)) != JANUS_OK) return e;
    const int H = d->H, E = d->E, N = s.N;
    const int64_t kh = int64_t(t->num_trees) * H;
    {
    TraceScope trace("tree_bwd_init", 0.0, 12.0 * kh, st);
    hipLaunchKernelGGL(tree_bwd_init_kernel, dim3(unsigned((kh + 255) / 256)), dim3(256), 0, st, t->num_trees, H,
                       w.rootpos, static_cast<const float*>(dh_root), w.dh, w.dc);
    JANUS_LAUNCH_CHECK();
    }
    for (int k = s.num_levels - 1; k >= 0; --k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        const int64_t n = int64_t(rows) * H;
        if (k == 0) {
            TraceScope trace("tree_bwd_point", 0.0, 4.0 * n * 17.0, st);
            hipLaunchKernelGGL(tree_bwd_point_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows, H,
                               w.ld5, w.G, w.C, w.dh, w.dc, w.lchild, w.rchild, w.A);
            JANUS_LAUNCH_CHECK();
            break;
        }
        if (5 * H > kSimtKc) {
            // gate columns do not fit one LDS slab: pointwise, then the contraction
            {
                TraceScope trace("tree_bwd_point", 0.0, 4.0 * n * 17.0, st);
                hipLaunchKernelGGL(tree_bwd_point_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows,
                                   H, w.ld5, w.G, w.C, w.dh, w.dc, w.lchild, w.rchild, w.A);
                JANUS_LAUNCH_CHECK();
            }
            e = simt_gemm<false, kSimtChildren>("tree_dh_gemm", rows, 2 * H, 5 * H, w.A + int64_t(p0) * w.ld5, w.ld5,
                                                nullptr, static_cast<const float*>(U), 2 * H, nullptr, nullptr, w.dh,
                                                0, st, w.lchild + p0, w.rchild + p0, H);
            if (e != JANUS_OK) return e;
            continue;
        }
        // cell backward of the level and [dh_L; dh_R] = da U to the children
        dim3 grid(unsigned((2 * H + kSimtCols - 1) / kSimtCols), unsigned((rows + kSimtRows - 1) / kSimtRows));
        TraceScope trace("tree_bwd_level", 2.0 * rows * 2.0 * H * 5.0 * H,
                         4.0 * (double(rows) * 17.0 * H + 10.0 * H * H + 2.0 * rows * H), st);
        hipLaunchKernelGGL(tree_bwd_level_kernel, grid, dim3(64 * kSimtWaves), 0, st, p0, rows, H, w.ld5, w.G, w.C,
                           w.dh, w.dc, w.lchild, w.rchild, w.A, static_cast<const float*>(U), w.dh);
        JANUS_LAUNCH_CHECK();
    }
    // dU = da_int^T HLR  (K = internal nodes)
    e = simt_gemm<true, kSimtStore>("tree_dU_gemm", 5 * H, 2 * H, N - M0, w.A + int64_t(M0) * w.ld5, w.ld5, nullptr,
                                    w.HLR, 2 * H, nullptr, nullptr, dU, 2 * H, st);
    if (e != JANUS_OK) return e;
    // dW = da_leaf^T emb[word]  (K = leaves, gathered rows of emb)
    e = simt_gemm<true, kSimtStore>("tree_dW_gemm", 5 * H, E, M0, w.A, w.ld5, nullptr, static_cast<const float*>(emb),
                                    E, w.lword, nullptr, dW, E, st);
    if (e != JANUS_OK) return e;
    if ((e = colsum(JANUS_F32, w.A, N, 5 * H, w.ld5, db, w.part, st)) != JANUS_OK) return e;
    // dx_leaf = da_leaf W, then the embedding gradient
    e = simt_gemm<false, kSimtStore>("tree_dx_gemm", M0, E, 5 * H, w.A, w.ld5, nullptr, static_cast<const float*>(W), E,
                                     nullptr, nullptr, w.dxl, E, st);
    if (e != JANUS_OK) return e;
    return embed_backward(JANUS_F32, w.dxl, host.lword.data(), M0, E, demb, d->V, w.seg, st);
}

extern "C" janus_status janus_treelstm_device_report(const janus_treelstm_desc* d, const janus_tree_batch* t,
                                                     const void* ws, size_t ws_bytes, int32_t* timed_out,
                                                     void* stream) {
    if (!timed_out) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeWs w;
    janus_status e = prepare(d, t, const_cast<void*>(ws), ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    unsigned flag = 0;
    JANUS_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    JANUS_HIP(hipMemcpy(&flag, &w.tsync->error, sizeof(flag), hipMemcpyDeviceToHost));
    *timed_out = flag != 0u ? 1 : 0;
    return flag != 0u ? JANUS_ERR_DEVICE : JANUS_OK;
}

namespace janus {
namespace {

// Grid and LDS of the persistent TreeRNN kernels: one workgroup per CU at
// most, the grid a multiple of the column tiles of W (forward: H / 32 output
// units; backward: 2H / 32 columns of [dh_L; dh_R]).  Off with
// JANUS_TREE_PERSIST=0, for H above 512 (the embedding gradient's two
// columns per thread), or where the forward's operand slabs do not fit the
// LDS (about H > 312); the level-by-level kernels run then.
struct RnnPlan {
    bool on = false;
    int ncol = 0, fwd_grid = 0, ncol2 = 0, bwd_grid = 0;
    size_t fwd_lds = 0, bwd_lds = 0;
};
RnnPlan rnn_plan(const janus_treelstm_desc& d) {
    RnnPlan p;
    const char* e = getenv("JANUS_TREE_PERSIST");
    if (e && e[0] == '0') return p;
    const TreeDev dev = tree_dev();
    if (dev.cus <= 0 || dev.lds == 0 || d.H > tpersist::kMaxE) return p;
    p.ncol = (d.H + 31) / 32;
    p.ncol2 = (2 * d.H + 31) / 32;
    if (p.ncol2 > dev.cus) return p;
    const int cus = dev.cus < kMaxTreeGrid ? dev.cus : kMaxTreeGrid;
    p.fwd_grid = p.ncol * (cus / p.ncol);
    p.bwd_grid = p.ncol2 * (cus / p.ncol2);
    p.fwd_lds = size_t(tpersist::rnn_fwd_lds_floats(d.H)) * sizeof(float);
    p.bwd_lds = size_t(tpersist::rnn_bwd_lds_floats(d.H)) * sizeof(float);
    p.on = p.fwd_lds <= dev.lds && p.bwd_lds <= dev.lds;
    return p;
}
// The backward addresses dA through one buffer descriptor (byte offsets
// below 2^31); larger batches run the level-by-level kernels.
bool rnn_persist_fits(const RnnPlan& p, const janus_treelstm_desc& d, int32_t N) {
    return p.on && int64_t(N) * round_up(d.H, 32) * 4 < (int64_t(1) << 31);
}

// Forward: schedule, level offsets and the zeroed barrier block (error flag
// included) in one copy, then one launch for every level.
janus_status treernn_fwd_persistent_call(const janus_treelstm_desc& d, const janus_tree_batch* t,
                                         const TreeSchedule& s, const TreeRnnWs& w, const RnnPlan& plan,
                                         const void* emb, const void* W, const void* b, void* h_root,
                                         hipStream_t st) {
    TreeHost h;
    build_host(t, s, h);
    const size_t nb = sizeof(int32_t) * s.N;
    const std::vector<char> zero_sync(sizeof(tpersist::TreeSync), 0);
    const UploadPiece pieces[] = {{w.s.lword, h.lword.data(), nb},
                                  {w.s.lchild, h.lchild.data(), nb},
                                  {w.s.rchild, h.rchild.data(), nb},
                                  {w.s.parent, h.parent.data(), nb},
                                  {w.s.rootk, h.rootk.data(), nb},
                                  {w.s.rootpos, h.rootpos.data(), sizeof(int32_t) * t->num_trees},
                                  {w.s.loff, s.level_offsets.data(), sizeof(int32_t) * s.level_offsets.size()},
                                  {w.s.tsync, zero_sync.data(), zero_sync.size()}};
    janus_status e = upload_pieces(pieces, 8, st);
    if (e != JANUS_OK) return e;
    tpersist::RnnFwdArgs a;
    a.H = d.H;
    a.N = s.N;
    a.M0 = s.level_offsets[1];
    a.nlev = s.num_levels;
    a.ncol = plan.ncol;
    a.loff = w.s.loff;
    a.lword = w.s.lword;
    a.parent = w.s.parent;
    a.rootk = w.s.rootk;
    a.emb = static_cast<const float*>(emb);
    a.W = static_cast<const float*>(W);
    a.b = static_cast<const float*>(b);
    a.Hn = w.Hnp;
    a.ldh = w.ldh;
    a.HLR = w.HLRp;
    a.ldl = w.ldl;
    a.h_root = static_cast<float*>(h_root);
    a.sync = w.s.tsync;
    static size_t attr = 0;
    const double flops = 2.0 * d.H * 2.0 * d.H * double(s.N - a.M0);
    TraceScope trace("treernn_fwd_persistent", flops, 0.0, st);
    return tree_persistent_launch(tpersist::treernn_fwd_persistent, plan.fwd_grid, plan.fwd_lds, a, st, attr);
}

// Backward: the forward's schedule (the workspace is unchanged between the
// calls); the leaves grouped by word and the barrier's counters (not its
// error flag) in one copy, then one launch for the levels, dW, db and the
// embedding gradient.
janus_status treernn_bwd_persistent_call(const janus_treelstm_desc& d, const janus_tree_batch* t,
                                         const TreeSchedule& s, const TreeRnnWs& w, const RnnPlan& plan,
                                         const void* W, const void* dh_root, float* demb, float* dW, float* db,
                                         hipStream_t st) {
    TreeHost h;
    build_host(t, s, h);
    const int M0 = s.level_offsets[1];
    std::vector<int32_t> seg;
    const int nseg = embed_segments(h.lword.data(), M0, d.V, seg);
    // first group of each workgroup's rows [V w / grid, V (w + 1) / grid)
    for (int g = 0; g < plan.bwd_grid; ++g) {
        const int32_t* sid = seg.data() + M0 + nseg + 1;
        const int64_t v0 = int64_t(d.V) * g / plan.bwd_grid;
        const int32_t first = int32_t(std::lower_bound(sid, sid + nseg, v0) - sid);
        seg.push_back(first);
    }
    const size_t counters = sizeof(tpersist::TreeSync) - tpersist::kTreeSyncCounters;
    const std::vector<char> zero_counters(counters, 0);
    const UploadPiece pieces[] = {
        {reinterpret_cast<char*>(w.s.tsync) + tpersist::kTreeSyncCounters, zero_counters.data(), counters},
        {w.s.seg, seg.data(), seg.size() * sizeof(int32_t)}};
    janus_status e = upload_pieces(pieces, 2, st);
    if (e != JANUS_OK) return e;
    tpersist::RnnBwdArgs a;
    a.H = d.H;
    a.N = s.N;
    a.M0 = M0;
    a.nlev = s.num_levels;
    a.ncol = plan.ncol2;
    a.nseg = nseg;
    a.V = d.V;
    a.ntrees = t->num_trees;
    a.loff = w.s.loff;
    a.lword = w.s.lword;
    a.lchild = w.s.lchild;
    a.rchild = w.s.rchild;
    a.rootk = w.s.rootk;
    a.rootpos = w.s.rootpos;
    a.seg = w.s.seg;
    a.W = static_cast<const float*>(W);
    a.Hn = w.Hnp;
    a.ldh = w.ldh;
    a.HLR = w.HLRp;
    a.ldl = w.ldl;
    a.dh_root = static_cast<const float*>(dh_root);
    a.dh = w.dhp;
    a.dA = w.dAp;
    a.lda = w.ldh;
    a.demb = demb;
    a.dW = dW;
    a.db = db;
    a.sync = w.s.tsync;
    static size_t attr = 0;
    // [dh_L; dh_R] = da W and dW, both 2 H 2H per internal node
    const double flops = 2.0 * 2.0 * d.H * 2.0 * d.H * double(s.N - M0);
    TraceScope trace("treernn_bwd_persistent", flops, 0.0, st);
    return tree_persistent_launch(tpersist::treernn_bwd_persistent, plan.bwd_grid, plan.bwd_lds, a, st, attr);
}

}  // namespace
}  // namespace janus

extern "C" size_t janus_treernn_workspace_bytes(const janus_treernn_desc* d, int32_t max_nodes, int32_t max_trees) {
    if (check_rnn(d) != JANUS_OK || max_nodes <= 0 || max_trees <= 0) return 0;
    TreeRnnWs w;
    return carve_rnn(*d, max_nodes, max_trees, nullptr, w);
}

extern "C" janus_status janus_treernn_fwd(const janus_treernn_desc* d, const janus_tree_batch* t, const void* emb,
                                          const void* W, const void* b, void* h_root, void* ws, size_t ws_bytes,
                                          void* stream) {
    if (!emb || !W || !b || !h_root) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeRnnWs w;
    janus_status e = prepare_rnn(d, t, ws, ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const RnnPlan plan = rnn_plan(*d);
    if (rnn_persist_fits(plan, *d, s.N)) return treernn_fwd_persistent_call(*d, t, s, w, plan, emb, W, b, h_root, st);
    if ((e = upload_tree(t, s, w.s, st)) != JANUS_OK) return e;
    const int H = d->H;
    const int M0 = s.level_offsets[1];
    float* hr = static_cast<float*>(h_root);
    // the level contractions read W transposed (N = H contiguous)
    if ((e = transpose_f32(static_cast<const float*>(W), H, 2 * H, w.Wt, st)) != JANUS_OK) return e;
    {
        const int64_t n = int64_t(M0) * H;
        TraceScope trace("treernn_leaf", 0.0, 12.0 * n, st);
        hipLaunchKernelGGL(treernn_leaf_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, M0, H, M0,
                           w.s.lword, static_cast<const float*>(emb), w.s.parent, w.s.rootk, w.Hn, w.HLR, hr);
        JANUS_LAUNCH_CHECK();
    }
    SimtExtra send;
    send.HLR = w.HLR;
    send.root = hr;
    send.M0 = M0;
    for (int k = 1; k < s.num_levels; ++k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        // h = tanh([h_L; h_R] W^T + b), saved and sent on (parent slot and tree
        // index of each row through the epilogue's index arguments)
        e = simt_gemm<false, kSimtTanhSend>("treernn_level", rows, H, 2 * H, w.HLR + int64_t(p0 - M0) * 2 * H, 2 * H,
                                            nullptr, w.Wt, H, nullptr, static_cast<const float*>(b),
                                            w.Hn + int64_t(p0) * H, H, st, w.s.parent + p0, w.s.rootk + p0, H, send);
        if (e != JANUS_OK) return e;
    }
    return JANUS_OK;
}

extern "C" janus_status janus_treernn_bwd(const janus_treernn_desc* d, const janus_tree_batch* t, const void* W,
                                          void* ws, size_t ws_bytes, const void* dh_root, float* demb, float* dW,
                                          float* db, void* stream) {
    if (!W || !dh_root || !demb || !dW || !db) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeRnnWs w;
    janus_status e = prepare_rnn(d, t, ws, ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    const int M0 = s.level_offsets[1];
    hipStream_t st = static_cast<hipStream_t>(stream);
    const RnnPlan plan = rnn_plan(*d);
    if (rnn_persist_fits(plan, *d, s.N))
        return treernn_bwd_persistent_call(*d, t, s, w, plan, W, dh_root, demb, dW, db, st);
    TreeHost host;
    if ((e = upload_tree(t, s, w.s, st, &host)) != JANUS_OK) return e;
    const int H = d->H, N = s.N;
    const int64_t kh = int64_t(t->num_trees) * H;
    {
        // dh of the roots (the dc half of this kernel's output is unused here)
        TraceScope trace("tree_bwd_init", 0.0, 12.0 * kh, st);
        hipLaunchKernelGGL(tree_bwd_init_kernel, dim3(unsigned((kh + 255) / 256)), dim3(256), 0, st, t->num_trees, H,
                           w.s.rootpos, static_cast<const float*>(dh_root), w.dh, w.A);
        JANUS_LAUNCH_CHECK();
    }
    for (int k = s.num_levels - 1; k >= 1; --k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        // da = dh (1 - h^2) as the a slab (stored by column block 0), and
        // [dh_L; dh_R] = da W to the children (W rows are N = 2H contiguous)
        SimtExtra tg;
        tg.S = w.Hn + int64_t(p0) * H;
        tg.D = w.A + int64_t(p0) * H;
        e = simt_gemm<false, kSimtChildren, kSimtTanhGrad>("treernn_level_bwd", rows, 2 * H, H, w.dh + int64_t(p0) * H,
                                                           H, nullptr, static_cast<const float*>(W), 2 * H, nullptr,
                                                           nullptr, w.dh, 0, st, w.s.lchild + p0, w.s.rchild + p0, H,
                                                           tg);
        if (e != JANUS_OK) return e;
    }
    // dW = da_int^T HLR  (K = internal nodes), db = column sums of da_int
    e = simt_gemm<true, kSimtStore>("treernn_dW_gemm", H, 2 * H, N - M0, w.A + int64_t(M0) * H, H, nullptr, w.HLR,
                                    2 * H, nullptr, nullptr, dW, 2 * H, st);
    if (e != JANUS_OK) return e;
    if (N > M0) {
        if ((e = colsum(JANUS_F32, w.A + int64_t(M0) * H, N - M0, H, H, db, w.part, st)) != JANUS_OK) return e;
    } else if ((e = zero_fill(db, sizeof(float) * H, st)) != JANUS_OK) {
        return e;
    }
    // the leaves' dh is the gradient of their word vectors
    return embed_backward(JANUS_F32, w.dh, host.lword.data(), M0, H, demb, d->V, w.s.seg, st);
}

extern "C" janus_status janus_treernn_device_report(const janus_treernn_desc* d, const janus_tree_batch* t,
                                                    const void* ws, size_t ws_bytes, int32_t* timed_out,
                                                    void* stream) {
    if (!timed_out) return JANUS_ERR_INVALID_ARG;
    TreeSchedule s;
    TreeRnnWs w;
    janus_status e = prepare_rnn(d, t, const_cast<void*>(ws), ws_bytes, s, w);
    if (e != JANUS_OK) return e;
    unsigned flag = 0;
    JANUS_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    JANUS_HIP(hipMemcpy(&flag, &w.s.tsync->error, sizeof(flag), hipMemcpyDeviceToHost));
    *timed_out = flag != 0u ? 1 : 0;
    return flag != 0u ? JANUS_ERR_DEVICE : JANUS_OK;
}
