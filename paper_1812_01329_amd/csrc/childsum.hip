// Child-Sum TreeLSTM over a batch of trees of any arity, evaluated as
// level-wise frontiers.
//
// The cited TreeLSTM paper defines this variant next to the binary one: every
// node reads its word vector x, h~ is the sum of its children's h, and each
// child k has its own forget gate,
//     i, o = s(W x + U h~ + b),  u = tanh(W x + U h~ + b)   (blocks i, o, u)
//     f_k  = s(W_f x + U_f h_k + b_f)
//     c = i u + sum_k f_k c_k,   h = o tanh(c).
// Levels group nodes by height (a node after all of its children), the same
// frontiers as the binary TreeNNs (Section 6.3.1, "+PARL").
//
// Forward.  x does not depend on the recursion, so XW = X W^T + b is one
// contraction over all nodes first.  After a level is computed, one
// contraction G = h U^T (all four blocks) serves its parents: by linearity
// U_iou h~ of a parent is the sum of its children's G_iou rows, and child k's
// forget gate reads G_f of row k.  A level is thus one cell kernel (which
// gathers its children's G and c) and one contraction.
//
// Backward, levels from the top down.  A node's cell backward writes, into
// the row of each child k, dG(k) = [da_iou(parent); da_f(parent, k)] and the
// child's dc; into its own row dXW = [da_iou; sum_k da_f].  When a level is
// reached all its rows of dG are complete, so its dh = dG U is one
// contraction over the level's contiguous rows (roots have dG = 0 and add
// the head's gradient).  Then dW = dXW^T X, dU = dG^T H, db = sum of dXW,
// and dX = dXW W for the embedding gradient.
#include <algorithm>
#include <vector>

#include "childsum_persist.hpp"
#include "device.hpp"
#include "ops.hpp"
#include "simt.hpp"

namespace janus {

namespace {

struct CsWs {
    int32_t* pword = nullptr;    // [N] word of the node at each position
    int32_t* pcoff = nullptr;    // [N + 1] children of position p: pkids[pcoff[p] .. pcoff[p + 1])
    int32_t* pkids = nullptr;    // [N] child positions
    int32_t* rootk = nullptr;    // [N] tree index of a root, -1 otherwise
    float* XW = nullptr;         // [N x 4H] X W^T + b
    float* G = nullptr;          // [N x 4H] h U^T (forward), dG (backward)
    float* Gt = nullptr;         // [N x 3H] gates i, o, u
    float* F = nullptr;          // [N x H]  forget gate of each node towards its parent
    float* C = nullptr;          // [N x H]
    float* Hn = nullptr;         // [N x H]
    float* dXW = nullptr;        // [N x 4H]
    float* dh = nullptr;         // [N x H]
    float* dc = nullptr;         // [N x H]
    float* dx = nullptr;         // [N x E]
    float* Wt = nullptr;         // [E x 4H]
    float* Ut = nullptr;         // [H x 4H]
    float* part = nullptr;
    int32_t* seg = nullptr;      // the nodes grouped by word, for the embedding gradient
    // persistent path: level offsets and the barrier's counters (carved right
    // after the schedule arrays and before `seg`, so that each direction's
    // upload is one copy), and node rows padded to whole 128-byte lines
    int32_t* loff = nullptr;     // [N + 1]
    tpersist::TreeSync* tsync = nullptr;
    float* XWp = nullptr;        // [N x ld4]
    float* Gp = nullptr;         // [N x ld4] h U^T (forward)
    float* dGp = nullptr;        // [N x ld4]
    float* dXWp = nullptr;       // [N x ld4]
    float* Gtp = nullptr;        // [N x ld3]
    float* Fp = nullptr;         // [N x ldh]
    float* Cp = nullptr;         // [N x ldh]
    float* Hnp = nullptr;        // [N x ldh]
    float* dcp = nullptr;        // [N x ldh]
    float* dhp = nullptr;        // [N x ldh]
    float* dxp = nullptr;        // [N x ldx]
    int64_t ld4 = 0, ld3 = 0, ldh = 0, ldx = 0;
};

size_t carve_cs(const janus_treelstm_desc& d, int32_t N, void* base, CsWs& w) {
    Carver c(base);
    const int H = d.H, E = d.E;
    w.pword = c.take<int32_t>(N);
    w.pcoff = c.take<int32_t>(int64_t(N) + 1);
    w.pkids = c.take<int32_t>(N);
    w.rootk = c.take<int32_t>(N);
    w.loff = c.take<int32_t>(int64_t(N) + 1);
    w.tsync = c.take<tpersist::TreeSync>(1);
    // the nodes grouped by word, and (persistent backward) each workgroup's
    // first group of the embedding rows
    w.seg = c.take<int32_t>(int64_t(embed_seg_ints(N)) + tpersist::kMaxTreeGrid);
    w.XW = c.take<float>(int64_t(N) * 4 * H);
    w.G = c.take<float>(int64_t(N) * 4 * H);
    w.Gt = c.take<float>(int64_t(N) * 3 * H);
    w.F = c.take<float>(int64_t(N) * H);
    w.C = c.take<float>(int64_t(N) * H);
    w.Hn = c.take<float>(int64_t(N) * H);
    w.dXW = c.take<float>(int64_t(N) * 4 * H);
    w.dh = c.take<float>(int64_t(N) * H);
    w.dc = c.take<float>(int64_t(N) * H);
    w.dx = c.take<float>(int64_t(N) * E);
    w.Wt = c.take<float>(int64_t(E) * 4 * H);
    w.Ut = c.take<float>(int64_t(H) * 4 * H);
    w.part = c.take<float>(colsum_partial_floats(4 * H));
    w.ld4 = round_up(int64_t(4) * H, 32);
    w.ld3 = round_up(int64_t(3) * H, 32);
    w.ldh = round_up(H, 32);
    w.ldx = round_up(E, 32);
    w.XWp = c.take<float>(int64_t(N) * w.ld4);
    w.Gp = c.take<float>(int64_t(N) * w.ld4);
    w.dGp = c.take<float>(int64_t(N) * w.ld4);
    w.dXWp = c.take<float>(int64_t(N) * w.ld4);
    w.Gtp = c.take<float>(int64_t(N) * w.ld3);
    w.Fp = c.take<float>(int64_t(N) * w.ldh);
    w.Cp = c.take<float>(int64_t(N) * w.ldh);
    w.Hnp = c.take<float>(int64_t(N) * w.ldh);
    w.dcp = c.take<float>(int64_t(N) * w.ldh);
    w.dhp = c.take<float>(int64_t(N) * w.ldh);
    w.dxp = c.take<float>(int64_t(N) * w.ldx);
    return c.off + 256;
}

__global__ void cs_fwd_cell_kernel(int p0, int rows, int H, const float* XW, const float* G, const int32_t* pcoff,
                                   const int32_t* pkids, const int32_t* rootk, float* Gt, float* F, float* C,
                                   float* Hn, float* h_root) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(rows) * H) return;
    const int p = p0 + int(i / H), j = int(i % H);
    const float* xw = XW + int64_t(p) * 4 * H;
    float ai = xw[j], ao = xw[H + j], au = xw[2 * H + j];
    const float af = xw[3 * H + j];
    float csum = 0.f;
    for (int e = pcoff[p]; e < pcoff[p + 1]; ++e) {
        const int k = pkids[e];
        const float* g = G + int64_t(k) * 4 * H;
        ai += g[j];
        ao += g[H + j];
        au += g[2 * H + j];
        const float f = sigmoidf_(af + g[3 * H + j]);
        F[int64_t(k) * H + j] = f;
        csum += f * C[int64_t(k) * H + j];
    }
    const float gi = sigmoidf_(ai), go = sigmoidf_(ao), gu = tanhf_(au);
    const float c = gi * gu + csum;
    const float h = go * tanhf_(c);
    C[int64_t(p) * H + j] = c;
    Hn[int64_t(p) * H + j] = h;
    float* gt = Gt + int64_t(p) * 3 * H;
    gt[j] = gi;
    gt[H + j] = go;
    gt[2 * H + j] = gu;
    if (rootk[p] >= 0) h_root[int64_t(rootk[p]) * H + j] = h;
}

__global__ void cs_bwd_cell_kernel(int p0, int rows, int H, const float* dh, const float* dh_root,
                                   const int32_t* rootk, const float* Gt, const float* F, const float* C,
                                   const int32_t* pcoff, const int32_t* pkids, float* dc, float* dG, float* dXW) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(rows) * H) return;
    const int p = p0 + int(i / H), j = int(i % H);
    const int rk = rootk[p];
    const float dhv = dh[int64_t(p) * H + j] + (rk >= 0 ? dh_root[int64_t(rk) * H + j] : 0.f);
    const float* gt = Gt + int64_t(p) * 3 * H;
    const float gi = gt[j], go = gt[H + j], gu = gt[2 * H + j];
    const float tau = tanhf_(C[int64_t(p) * H + j]);
    const float dct = dc[int64_t(p) * H + j] + dhv * go * (1.f - tau * tau);
    const float dai = dct * gu * gi * (1.f - gi);
    const float dao = dhv * tau * go * (1.f - go);
    const float dau = dct * gi * (1.f - gu * gu);
    float dafs = 0.f;
    for (int e = pcoff[p]; e < pcoff[p + 1]; ++e) {
        const int k = pkids[e];
        const float f = F[int64_t(k) * H + j];
        const float daf = dct * C[int64_t(k) * H + j] * f * (1.f - f);
        dafs += daf;
        float* g = dG + int64_t(k) * 4 * H;
        g[j] = dai;
        g[H + j] = dao;
        g[2 * H + j] = dau;
        g[3 * H + j] = daf;
        dc[int64_t(k) * H + j] = dct * f;
    }
    float* x = dXW + int64_t(p) * 4 * H;
    x[j] = dai;
    x[H + j] = dao;
    x[2 * H + j] = dau;
    x[3 * H + j] = dafs;
}

janus_status check_cs(const janus_treelstm_desc* d) {
    if (!d || d->E <= 0 || d->H <= 0 || d->V <= 0) return JANUS_ERR_INVALID_ARG;
    if (d->dtype != JANUS_F32) return JANUS_ERR_UNSUPPORTED;
    return JANUS_OK;
}

// Validates the call and carves the workspace; `upload` also copies the
// schedule arrays (carved one after another: one copy) for the level-by-level
// kernels.
janus_status prepare_cs(const janus_treelstm_desc* d, const janus_nary_tree_batch* t, void* ws, size_t ws_bytes,
                        NarySchedule& s, CsWs& w, hipStream_t st, bool upload = true) {
    janus_status e = check_cs(d);
    if (e != JANUS_OK) return e;
    if ((e = build_nary_schedule(t, d->V, s)) != JANUS_OK) return e;
    if (!ws || ws_bytes < carve_cs(*d, s.N, nullptr, w) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    carve_cs(*d, s.N, ws, w);
    if (!upload) return JANUS_OK;
    const size_t nb = sizeof(int32_t) * s.N;
    // the barrier block is zeroed too, so the device report of a call on
    // this path reads no stale flag
    const std::vector<char> zero_sync(sizeof(tpersist::TreeSync), 0);
    const UploadPiece pieces[] = {{w.pword, s.pword.data(), nb},
                                  {w.pcoff, s.pcoff.data(), nb + sizeof(int32_t)},
                                  {w.pkids, s.pkids.data(), sizeof(int32_t) * s.pkids.size()},
                                  {w.rootk, s.rootk.data(), nb},
                                  {w.tsync, zero_sync.data(), zero_sync.size()}};
    return upload_pieces(pieces, 5, st);
}

// ------------------------------------------------------- persistent path
// Grid and LDS of the persistent Child-Sum kernels: one workgroup per CU at
// most, the grid a multiple of the column tiles (forward: 4H / 32 gate
// columns; backward: H / 32 columns of dh).  Off with JANUS_TREE_PERSIST=0,
// for inputs wider than 512 (the embedding gradient's two columns per
// thread), or where the backward's U columns and dG tile (two 32 x 4H slabs)
// do not fit the LDS (about H > 156); the level-by-level kernels run then.
struct CsPlan {
    bool on = false;
    int ncolf = 0, fwd_grid = 0, ncolb = 0, bwd_grid = 0;
    size_t fwd_lds = 0, bwd_lds = 0;
};
CsPlan cs_plan(const janus_treelstm_desc& d) {
    CsPlan p;
    const char* e = getenv("JANUS_TREE_PERSIST");
    if (e && e[0] == '0') return p;
    const tpersist::TreeDev dev = tpersist::tree_dev();
    if (dev.cus <= 0 || dev.lds == 0 || d.E > tpersist::kMaxE) return p;
    p.ncolf = (4 * d.H + 31) / 32;
    p.ncolb = (d.H + 31) / 32;
    if (p.ncolf > dev.cus) return p;
    const int cus = dev.cus < tpersist::kMaxTreeGrid ? dev.cus : tpersist::kMaxTreeGrid;
    p.fwd_grid = p.ncolf * (cus / p.ncolf);
    p.bwd_grid = p.ncolb * (cus / p.ncolb);
    p.fwd_lds = size_t(tpersist::cs_fwd_lds_floats(d.E, d.H)) * sizeof(float);
    p.bwd_lds = size_t(tpersist::cs_bwd_lds_floats(d.H)) * sizeof(float);
    p.on = p.fwd_lds <= dev.lds && p.bwd_lds <= dev.lds;
    return p;
}

// Forward: schedule, level offsets and the zeroed barrier block (error flag
// included) in one copy, then one launch for every level.
janus_status cs_fwd_persistent_call(const janus_treelstm_desc& d, const NarySchedule& s, const CsWs& w,
                                    const CsPlan& plan, const void* emb, const void* W, const void* U, const void* b,
                                    void* h_root, hipStream_t st) {
    const size_t nb = sizeof(int32_t) * s.N;
    const std::vector<char> zero_sync(sizeof(tpersist::TreeSync), 0);
    const UploadPiece pieces[] = {{w.pword, s.pword.data(), nb},
                                  {w.pcoff, s.pcoff.data(), nb + sizeof(int32_t)},
                                  {w.pkids, s.pkids.data(), sizeof(int32_t) * s.pkids.size()},
                                  {w.rootk, s.rootk.data(), nb},
                                  {w.loff, s.level_offsets.data(), sizeof(int32_t) * s.level_offsets.size()},
                                  {w.tsync, zero_sync.data(), zero_sync.size()}};
    janus_status e = upload_pieces(pieces, 6, st);
    if (e != JANUS_OK) return e;
    tpersist::CsFwdArgs a;
    a.E = d.E;
    a.H = d.H;
    a.N = s.N;
    a.nlev = int(s.level_offsets.size()) - 1;
    a.ncol = plan.ncolf;
    a.loff = w.loff;
    a.pword = w.pword;
    a.pcoff = w.pcoff;
    a.pkids = w.pkids;
    a.rootk = w.rootk;
    a.emb = static_cast<const float*>(emb);
    a.W = static_cast<const float*>(W);
    a.U = static_cast<const float*>(U);
    a.b = static_cast<const float*>(b);
    a.XW = w.XWp;
    a.G = w.Gp;
    a.ld4 = w.ld4;
    a.Gt = w.Gtp;
    a.ld3 = w.ld3;
    a.F = w.Fp;
    a.C = w.Cp;
    a.Hn = w.Hnp;
    a.ldh = w.ldh;
    a.h_root = static_cast<float*>(h_root);
    a.sync = w.tsync;
    static size_t attr = 0;
    const double flops = 2.0 * s.N * 4.0 * d.H * (double(d.E) + double(d.H));
    TraceScope trace("childsum_fwd_persistent", flops, 0.0, st);
    return tpersist::tree_persistent_launch(tpersist::childsum_fwd_persistent, plan.fwd_grid, plan.fwd_lds, a, st,
                                            attr);
}

// Backward: the forward's schedule (the workspace is unchanged between the
// calls); the nodes grouped by word and the barrier's counters (not its
// error flag) in one copy, then one launch.
janus_status cs_bwd_persistent_call(const janus_treelstm_desc& d, const NarySchedule& s, const CsWs& w,
                                    const CsPlan& plan, const void* emb, const void* W, const void* U,
                                    const void* dh_root, float* demb, float* dW, float* dU, float* db,
                                    hipStream_t st) {
    std::vector<int32_t> seg;
    const int nseg = embed_segments(s.pword.data(), s.N, d.V, seg);
    // first group of each workgroup's rows [V w / grid, V (w + 1) / grid)
    for (int g = 0; g < plan.bwd_grid; ++g) {
        const int32_t* sid = seg.data() + s.N + nseg + 1;
        const int64_t v0 = int64_t(d.V) * g / plan.bwd_grid;
        const int32_t first = int32_t(std::lower_bound(sid, sid + nseg, v0) - sid);
        seg.push_back(first);
    }
    const size_t counters = sizeof(tpersist::TreeSync) - tpersist::kTreeSyncCounters;
    const std::vector<char> zero_counters(counters, 0);
    const UploadPiece pieces[] = {
        {reinterpret_cast<char*>(w.tsync) + tpersist::kTreeSyncCounters, zero_counters.data(), counters},
        {w.seg, seg.data(), seg.size() * sizeof(int32_t)}};
    janus_status e = upload_pieces(pieces, 2, st);
    if (e != JANUS_OK) return e;
    tpersist::CsBwdArgs a;
    a.E = d.E;
    a.H = d.H;
    a.N = s.N;
    a.nlev = int(s.level_offsets.size()) - 1;
    a.ncol = plan.ncolb;
    a.nseg = nseg;
    a.V = d.V;
    a.loff = w.loff;
    a.pword = w.pword;
    a.pcoff = w.pcoff;
    a.pkids = w.pkids;
    a.rootk = w.rootk;
    a.seg = w.seg;
    a.emb = static_cast<const float*>(emb);
    a.W = static_cast<const float*>(W);
    a.U = static_cast<const float*>(U);
    a.Gt = w.Gtp;
    a.ld3 = w.ld3;
    a.F = w.Fp;
    a.C = w.Cp;
    a.Hn = w.Hnp;
    a.ldh = w.ldh;
    a.dh_root = static_cast<const float*>(dh_root);
    a.dG = w.dGp;
    a.dXW = w.dXWp;
    a.ld4 = w.ld4;
    a.dc = w.dcp;
    a.dx = w.dxp;
    a.ldx = w.ldx;
    a.demb = demb;
    a.dW = dW;
    a.dU = dU;
    a.db = db;
    a.sync = w.tsync;
    static size_t attr = 0;
    // dh = dG U, dW, dU and dx over every node
    const double flops = 2.0 * s.N * 4.0 * d.H * (2.0 * d.H + 2.0 * d.E);
    TraceScope trace("childsum_bwd_persistent", flops, 0.0, st);
    return tpersist::tree_persistent_launch(tpersist::childsum_bwd_persistent, plan.bwd_grid, plan.bwd_lds, a, st,
                                            attr);
}

}  // namespace

}  // namespace janus

using namespace janus;

extern "C" size_t janus_childsum_workspace_bytes(const janus_childsum_desc* d, int32_t max_nodes) {
    if (check_cs(d) != JANUS_OK || max_nodes <= 0) return 0;
    CsWs w;
    return carve_cs(*d, max_nodes, nullptr, w);
}

extern "C" janus_status janus_childsum_fwd(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                           const void* emb, const void* W, const void* U, const void* b, void* h_root,
                                           void* ws, size_t ws_bytes, void* stream) {
    if (!emb || !W || !U || !b || !h_root) return JANUS_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    NarySchedule s;
    CsWs w;
    const CsPlan plan = cs_plan(*d);
    janus_status e = prepare_cs(d, t, ws, ws_bytes, s, w, st, !plan.on);
    if (e != JANUS_OK) return e;
    if (plan.on) return cs_fwd_persistent_call(*d, s, w, plan, emb, W, U, b, h_root, st);
    const int H = d->H, E = d->E, N = s.N;
    const int L = int(s.level_offsets.size()) - 1;
    if ((e = transpose_f32(static_cast<const float*>(W), 4 * H, E, w.Wt, st)) != JANUS_OK) return e;
    if ((e = transpose_f32(static_cast<const float*>(U), 4 * H, H, w.Ut, st)) != JANUS_OK) return e;
    // the input part of every node's gates at once
    e = simt_gemm<false, kSimtStore>("childsum_x_gemm", N, 4 * H, E, static_cast<const float*>(emb), E, w.pword, w.Wt,
                                     4 * H, nullptr, static_cast<const float*>(b), w.XW, 4 * H, st);
    if (e != JANUS_OK) return e;
    for (int k = 0; k < L; ++k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        const int64_t n = int64_t(rows) * H;
        {
            TraceScope trace("childsum_fwd_cell", 0.0, 4.0 * n * 16.0, st);
            hipLaunchKernelGGL(cs_fwd_cell_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows, H,
                               w.XW, w.G, w.pcoff, w.pkids, w.rootk, w.Gt, w.F, w.C, w.Hn,
                               static_cast<float*>(h_root));
            JANUS_LAUNCH_CHECK();
        }
        if (k + 1 < L) {   // the top level has no parents
            e = simt_gemm<false, kSimtStore>("childsum_level_gemm", rows, 4 * H, H, w.Hn + int64_t(p0) * H, H, nullptr,
                                             w.Ut, 4 * H, nullptr, nullptr, w.G + int64_t(p0) * 4 * H, 4 * H, st);
            if (e != JANUS_OK) return e;
        }
    }
    return JANUS_OK;
}

extern "C" janus_status janus_childsum_bwd(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                           const void* emb, const void* W, const void* U, void* ws, size_t ws_bytes,
                                           const void* dh_root, float* demb, float* dW, float* dU, float* db,
                                           void* stream) {
    if (!emb || !W || !U || !dh_root || !demb || !dW || !dU || !db) return JANUS_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    NarySchedule s;
    CsWs w;
    const CsPlan plan = cs_plan(*d);
    janus_status e = prepare_cs(d, t, ws, ws_bytes, s, w, st, !plan.on);
    if (e != JANUS_OK) return e;
    if (plan.on) return cs_bwd_persistent_call(*d, s, w, plan, emb, W, U, dh_root, demb, dW, dU, db, st);
    const int H = d->H, E = d->E, N = s.N;
    const int L = int(s.level_offsets.size()) - 1;
    // roots have no parent: their dG rows and dc stay 0
    if ((e = zero_fill(w.G, sizeof(float) * size_t(N) * 4 * H, st)) != JANUS_OK) return e;
    if ((e = zero_fill(w.dc, sizeof(float) * size_t(N) * H, st)) != JANUS_OK) return e;
    for (int k = L - 1; k >= 0; --k) {
        const int p0 = s.level_offsets[k], rows = s.level_offsets[k + 1] - p0;
        // dh of the level from the dG rows its parents wrote
        e = simt_gemm<false, kSimtStore>("childsum_dh_gemm", rows, H, 4 * H, w.G + int64_t(p0) * 4 * H, 4 * H, nullptr,
                                         static_cast<const float*>(U), H, nullptr, nullptr, w.dh + int64_t(p0) * H, H,
                                         st);
        if (e != JANUS_OK) return e;
        const int64_t n = int64_t(rows) * H;
        TraceScope trace("childsum_bwd_cell", 0.0, 4.0 * n * 20.0, st);
        hipLaunchKernelGGL(cs_bwd_cell_kernel, dim3(unsigned((n + 255) / 256)), dim3(256), 0, st, p0, rows, H, w.dh,
                           static_cast<const float*>(dh_root), w.rootk, w.Gt, w.F, w.C, w.pcoff, w.pkids, w.dc, w.G,
                           w.dXW);
        JANUS_LAUNCH_CHECK();
    }
    // dW = dXW^T X (rows of emb gathered by word), dU = dG^T H, db = sum dXW
    e = simt_gemm<true, kSimtStore>("childsum_dW_gemm", 4 * H, E, N, w.dXW, 4 * H, nullptr,
                                    static_cast<const float*>(emb), E, w.pword, nullptr, dW, E, st);
    if (e != JANUS_OK) return e;
    e = simt_gemm<true, kSimtStore>("childsum_dU_gemm", 4 * H, H, N, w.G, 4 * H, nullptr, w.Hn, H, nullptr, nullptr,
                                    dU, H, st);
    if (e != JANUS_OK) return e;
    if ((e = colsum(JANUS_F32, w.dXW, N, 4 * H, 4 * H, db, w.part, st)) != JANUS_OK) return e;
    // dX = dXW W, then the embedding gradient
    e = simt_gemm<false, kSimtStore>("childsum_dx_gemm", N, E, 4 * H, w.dXW, 4 * H, nullptr,
                                     static_cast<const float*>(W), E, nullptr, nullptr, w.dx, E, st);
    if (e != JANUS_OK) return e;
    return embed_backward(JANUS_F32, w.dx, s.pword.data(), N, E, demb, d->V, w.seg, st);
}

extern "C" janus_status janus_childsum_device_report(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                                     const void* ws, size_t ws_bytes, int32_t* timed_out,
                                                     void* stream) {
    if (!timed_out) return JANUS_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    NarySchedule s;
    CsWs w;
    janus_status e = prepare_cs(d, t, const_cast<void*>(ws), ws_bytes, s, w, st, false);
    if (e != JANUS_OK) return e;
    unsigned flag = 0;
    JANUS_HIP(hipStreamSynchronize(st));
    JANUS_HIP(hipMemcpy(&flag, &w.tsync->error, sizeof(flag), hipMemcpyDeviceToHost));
    *timed_out = flag != 0u ? 1 : 0;
    return flag != 0u ? JANUS_ERR_DEVICE : JANUS_OK;
}
