// LSTM over variable-length sequences: forward and backward through time.
//
// The loop of Figure 1 (``state = rnn_cell(state, item)``) with one trip
// count per sequence (Section 4.2.1).  The batch is sorted longest first, so
// the sequences still running at step t are the first active[t] sorted rows
// and their activations are stored "packed": packed row off[t] + r holds
// sorted row r at step t.  Work per step is then a dense block of active[t]
// rows; finished rows cost nothing.
//
// Per layer, forward:
//   1. hoisted input projection for every packed row:  XG = X Wx^T + b
//      (one contraction over all time steps; no dependence on h)
//   2. for t < t_eff, one fused step kernel: the recurrent contraction
//      h_{t-1} Wh^T for a tile of rows x (4 gates of U hidden units), then the
//      cell pointwise on the same tile (gates, c_t, h_t, outputs).
// Per layer, backward (reverse t):
//   one fused step kernel per t: dh_rec = dG_{t+1} Wh for a tile of rows x
//   hidden units, then the cell backward pointwise for step t on the same
//   tile, writing dG_t and the carried dc.  After the loop, the weight
//   gradients are single contractions over all packed rows:
//   dWx = dG^T X, dWh = dG^T H_prev, db = column sums of dG, dX = dG Wx.
//
// Workspace layout (identical for forward and backward; see carve()):
//   perm [B], xrow [T*B], prevrow [T*B]        int32 (variable lengths only)
//   per layer: Hs [(B + T*B) x ldh] dtype      rows [0, B): h0 (sorted rows),
//                                               row B + p: h at packed row p
//              Cs [(B + T*B) x ldh] float32     same for c
//              Gs [T*B x ldg] dtype             post-activation gates i, f, g, o
//   XG [T*B x ldg] dtype                        XG in forward, dG in backward
//   dY [T*B x ldh] dtype                        gradient of a lower layer's output
//   dh, dc [B x H] float32                      carried gradients (sorted rows)
//   colsum scratch
#include <algorithm>
#include <mutex>
#include <vector>

#include "device.hpp"
#include "lstm_persist.hpp"
#include "ops.hpp"

namespace janus {

namespace {

struct LstmWs {
    int32_t* perm = nullptr;
    int32_t* xrow = nullptr;
    int32_t* prevrow = nullptr;
    std::vector<void*> Hs;
    std::vector<float*> Cs;
    std::vector<void*> Gs;
    void* XG = nullptr;
    void* dY = nullptr;
    float* dh = nullptr;
    float* dc = nullptr;
    float* part = nullptr;
    // persistent path
    std::vector<void*> Wxi;             // per layer: Wx with gate-interleaved rows
    std::vector<void*> bi;              // per layer: b, gate-interleaved
    int32_t* perm4 = nullptr;           // [4H] interleaved row -> gate-major row
    int32_t* act_dev = nullptr;         // [T + 1]
    int32_t* off_dev = nullptr;         // [T + 2]
    float* dpart = nullptr;             // [T + 1] slots of partial recurrent gradients, NS x B x (H rounded to 8 NS)
    bf16_t* Gf = nullptr;               // [T] slots of dG in fragment layout (persistent backward)
    int64_t gf_slot = 0;                // elements per slot
    persist::Sync* sync = nullptr;
    void* GT = nullptr;                 // dG^T [4H x ldk] (bf16), K-contiguous operand of the weight gradients
    std::vector<bf16_t*> HT;            // per layer: h transposed [H x ldht], columns [0, B) = h0 (persistent forward)
    int64_t ldht = 0;
    bf16_t* Hf = nullptr;               // [T + 1] slots of h in fragment layout (persistent forward)
    int64_t hf_slot = 0;                // elements per slot
    void* gs = nullptr;                 // contraction scratch (transposed operands, split-K partials)
    size_t gs_bytes = 0;
    int64_t ldh = 0, ldg = 0, ldk = 0;
};

// ------------------------------------------------------- persistent path
struct DeviceInfo {
    int cus = 0;
    size_t lds = 0;
    int xccs = 0;
};

// Properties of the current device, queried once per device (under a lock,
// so concurrent first calls from several host threads do not race).
DeviceInfo device_info() {
    static std::mutex m;
    static DeviceInfo cache[64];
    static bool have[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DeviceInfo{};
    std::lock_guard<std::mutex> lock(m);
    if (!have[dev]) {
        DeviceInfo d;
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess) d.cus = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess) d.lds = size_t(v);
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeNumberOfXccs, dev) == hipSuccess) d.xccs = v;
        // a failed query must not surface as the error of a later launch check
        (void)hipGetLastError();
        cache[dev] = d;
        have[dev] = true;
    }
    return cache[dev];
}

// Forward K split (persistent path): the k-groups of 16 columns of h (Kp / 16)
// are split in `ns` slices and the units in groups of 8 ns; one workgroup per
// (slice, group) holds the rows of the group's units for its slice.
int persist_fwd_nkg(const janus_lstm_desc& d) { return int(round_up(d.H, 64) / 16); }
int persist_fwd_ksp(const janus_lstm_desc& d, int ns) { return 16 * ((persist_fwd_nkg(d) + ns - 1) / ns); }
int persist_fwd_groups(const janus_lstm_desc& d, int ns) { return (d.H + 8 * ns - 1) / (8 * ns); }
int persist_fwd_blocks(const janus_lstm_desc& d, int ns) { return ns * persist_fwd_groups(d, ns); }

// Groups whose members may straddle an XCD boundary: at most one fewer than
// the XCDs (all the census can tell apart when the count is unknown).
int persist_straddle_slots() {
    const int x = device_info().xccs;
    return (x > 0 && x <= persist::kMaxXcds ? x : persist::kMaxXcds) - 1;
}

// Floats of the forward's partial sums at `ns` slices: one slot reused by
// groups on one XCD, then per step and straddling group a slot of its own.
int64_t persist_fwd_part_local(const janus_lstm_desc& d, int ns) {
    return int64_t(ns) * persist_fwd_groups(d, ns) * ns * ((d.B + 31) / 32) * 1024;
}
int64_t persist_fwd_part_floats(const janus_lstm_desc& d, int ns) {
    if (ns <= 1) return 0;
    return persist_fwd_part_local(d, ns) +
           int64_t(d.T) * persist_straddle_slots() * ns * ns * ((d.B + 31) / 32) * 1024;
}

// Contraction scratch for every contraction of the forward and backward
// passes (they run one after another on one stream, so one buffer serves all).
size_t lstm_gemm_scratch(const janus_lstm_desc& d) {
    const int64_t TB = int64_t(d.T) * d.B;
    if (d.dtype != JANUS_BF16 || TB > INT32_MAX) return 0;
    size_t m = 0;
    for (int l = 0; l < d.L; ++l) {
        const int Il = l == 0 ? d.I : d.H;
        GemmDesc g;
        g.dtype = d.dtype;
        g.M = int(TB); g.N = 4 * d.H; g.K = Il;            // input projection
        g.a_idx = reinterpret_cast<const int32_t*>(16);
        m = std::max(m, gemm_scratch_bound(g));
        g = GemmDesc();
        g.dtype = d.dtype;
        g.M = 4 * d.H; g.N = Il; g.K = int(TB);             // dWx, dWh (dG^T in place, rows transposed)
        g.a_zero_pad = true;
        g.b_t = true;
        m = std::max(m, gemm_scratch_bound(g));
        g.N = d.H;
        m = std::max(m, gemm_scratch_bound(g));
        g = GemmDesc();
        g.dtype = d.dtype;
        g.M = int(TB); g.N = Il; g.K = 4 * d.H;             // dX = dG Wx
        g.b_t = true;
        m = std::max(m, gemm_scratch_bound(g));
    }
    return m;
}

size_t carve(const janus_lstm_desc& d, void* base, LstmWs& w) {
    Carver c(base);
    const size_t es = dtype_size(d.dtype);
    const int64_t TB = int64_t(d.T) * d.B;
    // rows padded to whole 128-byte lines (see the persistent kernels' barrier)
    w.ldh = round_up(d.H, 64);
    w.ldg = round_up(int64_t(4) * d.H, 64);
    w.perm = c.take<int32_t>(d.B);
    w.xrow = c.take<int32_t>(TB);
    w.prevrow = c.take<int32_t>(TB);
    w.Hs.assign(d.L, nullptr);
    w.Cs.assign(d.L, nullptr);
    w.Gs.assign(d.L, nullptr);
    for (int l = 0; l < d.L; ++l) {
        w.Hs[l] = c.take<char>((d.B + TB) * w.ldh * es);
        w.Cs[l] = c.take<float>((d.B + TB) * w.ldh);
        w.Gs[l] = c.take<char>(TB * w.ldg * es);
    }
    w.XG = c.take<char>(TB * w.ldg * es);
    w.dY = c.take<char>(TB * w.ldh * es);
    w.dh = c.take<float>(int64_t(d.B) * d.H);
    w.dc = c.take<float>(int64_t(d.B) * d.H);
    w.part = c.take<float>(colsum_partial_floats(4 * d.H));
    w.Wxi.assign(d.L, nullptr);
    w.bi.assign(d.L, nullptr);
    for (int l = 0; l < d.L; ++l) {
        const int64_t Il = l == 0 ? d.I : d.H;
        w.Wxi[l] = c.take<char>(int64_t(4) * d.H * Il * es);
        w.bi[l] = c.take<char>(int64_t(4) * d.H * es);
    }
    w.perm4 = c.take<int32_t>(int64_t(4) * d.H);
    w.act_dev = c.take<int32_t>(int64_t(d.T) + 1);
    w.off_dev = c.take<int32_t>(int64_t(d.T) + 2);
    w.sync = c.take<persist::Sync>(1);
    if (d.dtype == JANUS_BF16) {
        // partial sums of the persistent backward, and of the forward (the two
        // never run at the same time)
        const int64_t bwd_part = (int64_t(d.T) + 1) * persist::kMaxSlices * d.B * round_up(d.H, 8 * persist::kMaxSlices);
        w.dpart = c.take<float>(std::max({bwd_part, persist_fwd_part_floats(d, 2), persist_fwd_part_floats(d, 4)}));
        w.gf_slot = round_up(d.B, 32) * int64_t(4) * d.H;
        w.Gf = c.take<bf16_t>(int64_t(d.T) * w.gf_slot);
        w.ldht = round_up(int64_t(d.B) + TB, 64);
        w.HT.assign(d.L, nullptr);
        for (int l = 0; l < d.L; ++l) w.HT[l] = c.take<bf16_t>(int64_t(d.H) * w.ldht);
        w.hf_slot = round_up(d.B, 32) * round_up(d.H, 64);
        w.Hf = c.take<bf16_t>((int64_t(d.T) + 1) * w.hf_slot);
        w.ldk = round_up(TB, 64);
        w.GT = c.take<char>(int64_t(4) * d.H * w.ldk * es);
        w.gs_bytes = lstm_gemm_scratch(d);
        w.gs = c.take<char>(int64_t(w.gs_bytes));
    }
    return c.off + 256;
}

int persist_kw(int B) { return B <= 32 ? 8 : B <= 64 ? 4 : B <= 128 ? 2 : 1; }

size_t persist_red_bytes(int kw) { return size_t(kw - 1) * (persist::kWaves / kw) * 4096; }

size_t persist_fwd_lds(const janus_lstm_desc& d, int ns) {
    return size_t(32 * ns) * (persist_fwd_ksp(d, ns) + 8) * 2 + persist_red_bytes(persist_kw(d.B));
}
// Backward: the k-groups of 16 interleaved gate columns (4H / 16) are split
// in `ns` slices and the units in groups of 8 ns; one workgroup per (slice,
// group) holds that part of Wh^T in LDS.
int persist_bwd_nkg(const janus_lstm_desc& d) { return d.H / 4; }
int persist_bwd_ksp(const janus_lstm_desc& d, int ns) { return 16 * ((persist_bwd_nkg(d) + ns - 1) / ns); }
size_t persist_bwd_lds(const janus_lstm_desc& d, int ns) {
    return size_t(8 * ns) * (persist_bwd_ksp(d, ns) + 8) * 2 + persist_red_bytes(persist_kw(d.B));
}
int persist_bwd_groups(const janus_lstm_desc& d, int ns) { return (d.H + 8 * ns - 1) / (8 * ns); }
int persist_bwd_blocks(const janus_lstm_desc& d, int ns) { return ns * persist_bwd_groups(d, ns); }

size_t device_lds(const DeviceInfo& info) { return info.lds > 0 ? info.lds : 65536; }

bool persist_bwd_fits(const janus_lstm_desc& d, int ns, const DeviceInfo& info) {
    return persist_bwd_blocks(d, ns) <= info.cus && persist_bwd_groups(d, ns) <= persist::kMaxGroups &&
           persist_bwd_lds(d, ns) <= device_lds(info);
}

bool persist_fwd_fits(const janus_lstm_desc& d, int ns, const DeviceInfo& info) {
    return persist_fwd_blocks(d, ns) <= info.cus && (ns == 1 || persist_fwd_groups(d, ns) <= persist::kMaxGroups) &&
           persist_fwd_lds(d, ns) <= device_lds(info);
}

// Slices of the persistent forward.  Two slices halve each workgroup's
// share of the h stream but add the exchange of partial pre-activations
// (about 2.5 us per step); they pay where the h slot (B x H bf16) is 1 MB
// and up: at H = 2048, B = 256 the two forward layers of a training step
// take 8.0 against 8.3 ms.  Below, the stream is short and one slice is
// faster (B 128, H 1024: 1.26 against 1.48 ms; PTB, B 20: 0.40 against
// 0.56 ms).  Four slices lose everywhere: at H = 2048 their partial sums
// (3 MB per XCD) no longer stay in the L2.  One slice is taken when two do
// not fit; JANUS_FWD_SLICES=1, 2 or 4 asks for a count.
int persist_fwd_slices(const janus_lstm_desc& d) {
    const DeviceInfo info = device_info();
    const char* e = getenv("JANUS_FWD_SLICES");
    if (e && (e[0] == '1' || e[0] == '2' || e[0] == '4')) {
        const int forced = e[0] - '0';
        return persist_fwd_fits(d, forced, info) ? forced : 0;
    }
    const bool big = int64_t(d.B) * d.H * 2 >= (int64_t(1) << 20);
    if (big && persist_fwd_fits(d, 2, info)) return 2;
    return persist_fwd_fits(d, 1, info) ? 1 : 0;
}

// Slices of the persistent backward.  8 slices halve each workgroup's
// share of the dG stream but double the partial sums it exchanges; they pay
// where the per-step dG slot (B x 4H bf16) is large, 2 MB and up (0.5 ms of
// a 35 ms step at H = 2048, B = 256), and 4 slices are faster below (PTB,
// B 20: 0.55 against 0.66 ms of backward per step; B 128, H 1024: 1.48
// against 1.55 ms).  The other count is taken when the preferred one does
// not fit; 0 when neither does.  JANUS_BWD_SLICES=4 or 8 asks for one of
// them only.
int persist_bwd_slices(const janus_lstm_desc& d) {
    const DeviceInfo info = device_info();
    const char* e = getenv("JANUS_BWD_SLICES");
    const int forced = (e && e[0] == '4') ? 4 : (e && e[0] == '8') ? 8 : 0;
    const bool big = int64_t(d.B) * 4 * d.H * 2 >= (int64_t(2) << 20);
    for (int ns : {big ? 8 : 4, big ? 4 : 8}) {
        if (forced && ns != forced) continue;
        if (persist_bwd_fits(d, ns, info)) return ns;
    }
    return 0;
}

// The persistent path needs bf16, H a multiple of 8, one co-resident
// workgroup per slice and the weight slice in LDS; a batch of more than 256
// rows runs in parts of 256 sorted rows, one launch each.  It can be
// switched off with JANUS_PERSIST=0 (the per-step kernels then run).
bool use_persistent(const janus_lstm_desc& d) {
    const char* e = getenv("JANUS_PERSIST");
    const bool env = !(e && e[0] == '0');
    if (!env || d.dtype != JANUS_BF16 || d.H % 8 != 0) return false;
    const DeviceInfo info = device_info();
    if (info.cus <= 0) return false;
    return persist_fwd_slices(d) > 0 && persist_bwd_slices(d) > 0;
}

__global__ void perm4_kernel(int H, int32_t* perm4) {
    const int n = blockIdx.x * blockDim.x + threadIdx.x;
    if (n < 4 * H) perm4[n] = (n & 3) * H + (n >> 2);
}

// dst row n (interleaved) = src row (n % 4) * H + n / 4, rows of `cols` elements
template <typename T>
__global__ void interleave_rows_kernel(const T* src, T* dst, int H, int cols) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(4) * H * cols) return;
    const int n = int(i / cols), k = int(i % cols);
    dst[i] = src[(int64_t(n & 3) * H + (n >> 2)) * cols + k];
}

// ------------------------------------------------------------ init kernels
// initial state of the sorted rows into Hs / Cs rows [0, B) (and, for the
// persistent forward, into slot 0 of the fragment-layout copy Hf)
template <typename T>
__global__ void fwd_init_kernel(int B, int H, int64_t ldh, const int32_t* perm, const float* h0, const float* c0,
                                T* Hs, float* Cs, int active0, float* hT, float* cT, T* Hf, int Kp, T* HT,
                                int64_t ldht) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(B) * H) return;
    const int r = int(i / H), u = int(i % H);
    const int b = perm ? perm[r] : r;
    const float hv = h0 ? h0[int64_t(b) * H + u] : 0.f;
    const float cv = c0 ? c0[int64_t(b) * H + u] : 0.f;
    Hs[int64_t(r) * ldh + u] = from_f<T>(hv);
    Cs[int64_t(r) * ldh + u] = cv;
    if (Hf) Hf[persist::frag_index(r, u, Kp)] = from_f<T>(hv);
    if (HT) HT[int64_t(u) * ldht + r] = from_f<T>(hv);
    if (r >= active0) {   // a length-0 sequence ends in its initial state
        if (hT) hT[int64_t(b) * H + u] = hv;
        if (cT) cT[int64_t(b) * H + u] = cv;
    }
}

__global__ void bwd_init_kernel(int B, int H, const int32_t* perm, const float* dhT, const float* dcT, float* dh,
                                float* dc) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= int64_t(B) * H) return;
    const int r = int(i / H), u = int(i % H);
    const int b = perm ? perm[r] : r;
    dh[i] = dhT ? dhT[int64_t(b) * H + u] : 0.f;
    dc[i] = dcT ? dcT[int64_t(b) * H + u] : 0.f;
}

// ------------------------------------------------------------ forward step
template <typename T>
struct FwdStep {
    int H, B, t, active, active_next, U;
    int64_t off_t, prev_base, ldh, ldg;
    T* Hs;
    float* Cs;
    const T* Wh;
    const T* XG;
    T* Gs;
    T* y;
    const int32_t* perm;
    float* hT;
    float* cT;
};

template <typename T, class Cfg, bool AL>
__global__ __launch_bounds__(Cfg::NT) void fwd_step_kernel(FwdStep<T> a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    T* sA = reinterpret_cast<T*>(smem_raw);
    T* sB = sA + Cfg::BM * Cfg::LD;
    const int tid = threadIdx.x;
    const int U = a.U;
    const int u0 = blockIdx.x * U;
    const int m0 = blockIdx.y * Cfg::BM;

    LoaderK<T, Cfg::BM, Cfg::BK, Cfg::NT, AL> la;
    LoaderK<T, Cfg::BN, Cfg::BK, Cfg::NT, AL> lb;
    la.init(a.Hs + (a.prev_base + m0) * a.ldh, a.ldh, 0, RowsContig{a.active - m0}, tid);
    lb.init(a.Wh, a.H, 0, RowsGateMajor{a.H, u0, U, 4}, tid);
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop<Cfg>(acc, la, lb, a.H, sA, sB, tid);

    // stage the tile so that the four gates of a unit meet in one thread
    __syncthreads();
    constexpr int SLD = Cfg::BN + 1;
    float* sT = reinterpret_cast<float*>(smem_raw);
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sT[(Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane)) * SLD + Cfg::wave_col0(wave) + j * 32 +
                   acc_col(lane)] = acc[i][j][v];
    __syncthreads();

    const int H = a.H;
    for (int idx = tid; idx < Cfg::BM * U; idx += Cfg::NT) {
        const int r = idx / U, j = idx - (idx / U) * U;
        const int row = m0 + r, u = u0 + j;
        if (row >= a.active || u >= H) continue;
        const int64_t p = a.off_t + row;
        const T* xg = a.XG + p * a.ldg + u;
        const float ai = sT[r * SLD + 0 * U + j] + to_f(xg[0]);
        const float af = sT[r * SLD + 1 * U + j] + to_f(xg[H]);
        const float ag = sT[r * SLD + 2 * U + j] + to_f(xg[2 * H]);
        const float ao = sT[r * SLD + 3 * U + j] + to_f(xg[3 * H]);
        const float gi = sigmoidf_(ai), gf = sigmoidf_(af), gg = tanhf_(ag), go = sigmoidf_(ao);
        const float cp = a.Cs[(a.prev_base + row) * a.ldh + u];
        const float c = gf * cp + gi * gg;
        const float h = go * tanhf_(c);
        a.Cs[(a.B + p) * a.ldh + u] = c;
        a.Hs[(a.B + p) * a.ldh + u] = from_f<T>(h);
        T* gs = a.Gs + p * a.ldg + u;
        gs[0] = from_f<T>(gi);
        gs[H] = from_f<T>(gf);
        gs[2 * H] = from_f<T>(gg);
        gs[3 * H] = from_f<T>(go);
        const int b = a.perm ? a.perm[row] : row;
        if (a.y) a.y[(int64_t(a.t) * a.B + b) * H + u] = from_f<T>(h);
        if (row >= a.active_next) {   // last step of this sequence
            if (a.hT) a.hT[int64_t(b) * H + u] = h;
            if (a.cT) a.cT[int64_t(b) * H + u] = c;
        }
    }
}

// ----------------------------------------------------------- backward step
template <typename T>
struct BwdStep {
    int H, B, active, active_next;      // rows of step t; rows with a recurrent product
    int final_step;                     // 1: write dh0 / dc0 instead of a cell backward
    int64_t off_t, off_next, prev_base, ldh, ldg;
    const T* Wh;
    T* G;                               // dG store: read rows off_next + r, write rows off_t + r
    const T* Gs;                        // saved gates
    const float* Cs;
    const T* dy;                        // gradient of this layer's output, or NULL
    int64_t dy_ld;
    const int32_t* dy_rows;             // packed row -> dy row, NULL = identity
    float* dh;
    float* dc;
    const int32_t* perm;
    float* dh0;
    float* dc0;
};

template <typename T, class Cfg, bool AL>
__global__ __launch_bounds__(Cfg::NT) void bwd_step_kernel(BwdStep<T> a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    T* sA = reinterpret_cast<T*>(smem_raw);
    T* sB = sA + Cfg::BM * Cfg::LD;
    const int tid = threadIdx.x;
    const int u0 = blockIdx.x * Cfg::BN;
    const int m0 = blockIdx.y * Cfg::BM;
    const int H = a.H;

    // dh_rec[r, u] = sum_k dG_{t+1}[r, k] Wh[k, u]   (k over the 4H gate rows)
    LoaderK<T, Cfg::BM, Cfg::BK, Cfg::NT, AL> la;
    LoaderT<T, Cfg::BN, Cfg::BK, Cfg::NT, AL> lb;
    la.init(a.G + (a.off_next + m0) * a.ldg, a.ldg, 0, RowsContig{a.active_next - m0}, tid);
    lb.init(a.Wh, H, nullptr, u0, H);
    f32x16_t acc[Cfg::FM][Cfg::FN];
    mma_mainloop<Cfg>(acc, la, lb, a.active_next > m0 ? 4 * H : 0, sA, sB, tid);

    __syncthreads();
    constexpr int SLD = Cfg::BN + 1;
    float* sT = reinterpret_cast<float*>(smem_raw);
    const int lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < Cfg::FM; ++i)
#pragma unroll
        for (int j = 0; j < Cfg::FN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sT[(Cfg::wave_row0(wave) + i * 32 + acc_row(v, lane)) * SLD + Cfg::wave_col0(wave) + j * 32 +
                   acc_col(lane)] = acc[i][j][v];
    __syncthreads();

    for (int idx = tid; idx < Cfg::BM * Cfg::BN; idx += Cfg::NT) {
        const int r = idx / Cfg::BN, j = idx % Cfg::BN;
        const int row = m0 + r, u = u0 + j;
        if (row >= a.active || u >= H) continue;
        const int64_t hu = int64_t(row) * H + u;
        float dhv = row < a.active_next ? sT[r * SLD + j] : a.dh[hu];
        if (a.final_step) {
            const int b = a.perm ? a.perm[row] : row;
            if (a.dh0) a.dh0[int64_t(b) * H + u] = dhv;
            if (a.dc0) a.dc0[int64_t(b) * H + u] = a.dc[hu];
            continue;
        }
        const int64_t p = a.off_t + row;
        if (a.dy) {
            const int64_t yr = a.dy_rows ? int64_t(a.dy_rows[p]) : p;
            dhv += to_f(a.dy[yr * a.dy_ld + u]);
        }
        const T* gs = a.Gs + p * a.ldg + u;
        const float gi = to_f(gs[0]), gf = to_f(gs[H]), gg = to_f(gs[2 * H]), go = to_f(gs[3 * H]);
        const float c = a.Cs[(a.B + p) * a.ldh + u];
        const float cp = a.Cs[(a.prev_base + row) * a.ldh + u];
        const float tau = tanhf_(c);
        const float d_o = dhv * tau;
        const float dct = a.dc[hu] + dhv * go * (1.f - tau * tau);
        const float d_i = dct * gg, d_g = dct * gi, d_f = dct * cp;
        a.dc[hu] = dct * gf;
        T* dg = a.G + p * a.ldg + u;
        dg[0] = from_f<T>(d_i * gi * (1.f - gi));
        dg[H] = from_f<T>(d_f * gf * (1.f - gf));
        dg[2 * H] = from_f<T>(d_g * (1.f - gg * gg));
        dg[3 * H] = from_f<T>(d_o * go * (1.f - go));
    }
}

// ------------------------------------------------- one-workgroup recurrence
// A problem whose recurrent weights fit one CU's LDS (as float32) runs the
// whole time loop of a layer in one workgroup: Wh, h and c (forward) or
// dG_{t+1}, dh and dc (backward) stay in LDS, and steps are separated by
// workgroup barriers instead of kernel launches.  The state of step t and
// t + 1 sits in two LDS buffers used in turn, so a step needs one barrier
// and no cell holds its result in registers across it.  Work item j of a
// step takes cell (row, unit) j / S and the terms k = j % S (mod S) of its
// contraction; the S adjacent lanes of a cell add their parts with shuffles
// in a fixed order, so a cell's four gates meet in one lane and the cell
// update needs no exchange.  Weight rows are S floats longer than their
// length, which puts the S parts of the 64 / S cells of a wave in distinct
// LDS banks.  The operands of a step that do not depend on the recurrence
// (the input projection; the saved gates, cell states and dy) are loaded
// one step ahead, across the barrier.  The values the step kernels pass
// between steps through memory in T (h, dG) are rounded to T here too, and
// every buffer the step kernels write is written.
constexpr int kSmallThreads = 1024;
constexpr int kSmallCells = 8;   // cells per thread at most: B H <= 8192

template <int S>
__device__ __forceinline__ float small_group_sum(float v) {
#pragma unroll
    for (int m = 1; m < S; m <<= 1) v += __shfl_xor(v, m);
    return v;
}

template <typename T>
struct FwdSmall {
    int H, B, t_eff, fixed;
    const int32_t* active;
    const int32_t* offsets;
    int64_t ldh, ldg;
    const T* Wh;
    const T* XG;
    T* Hs;
    float* Cs;
    T* Gs;
    T* y;
    const int32_t* perm;
    float* hT;
    float* cT;
};

template <typename T, int S>
__global__ __launch_bounds__(kSmallThreads) void fwd_small_kernel(FwdSmall<T> a) {
    extern __shared__ float smem_f[];
    const int H = a.H, B = a.B, ldw = H + S, BH = B * H;
    float* Wl = smem_f;              // [4H][H + S]: row k = gate-major row k of Wh
    float* hl = Wl + 4 * H * ldw;    // [2][B][H]: h of steps t - 1 and t, in turn
    float* cl = hl + 2 * BH;         // [2][B][H]
    const int tid = threadIdx.x, part = tid % S;
    for (int i = tid; i < 4 * H * H; i += kSmallThreads) Wl[(i / H) * ldw + i % H] = to_f(a.Wh[i]);
    for (int i = tid; i < BH; i += kSmallThreads) {
        const int r = i / H, u = i % H;
        hl[i] = to_f(a.Hs[int64_t(r) * a.ldh + u]);
        cl[i] = a.Cs[int64_t(r) * a.ldh + u];
    }
    // input projection of cell i of step t (lane part 0 only)
    auto load_x = [&](int64_t off, int i, float* x) {
        const T* xg = a.XG + (off + i / H) * a.ldg + i % H;
#pragma unroll
        for (int g = 0; g < 4; ++g) x[g] = to_f(xg[g * H]);
    };
    float xpre[4] = {0.f, 0.f, 0.f, 0.f};   // of the first cell of this thread, one step ahead
    if (part == 0 && tid / S < persist::act_at(a.active, a.fixed, B, 0, a.t_eff) * H)
        load_x(persist::off_at(a.offsets, a.fixed, B, 0), tid / S, xpre);
    __syncthreads();
    for (int t = 0; t < a.t_eff; ++t) {
        const int act = persist::act_at(a.active, a.fixed, B, t, a.t_eff);
        const int act_next = persist::act_at(a.active, a.fixed, B, t + 1, a.t_eff);
        const int64_t off = persist::off_at(a.offsets, a.fixed, B, t);
        const float* hp = hl + (t & 1) * BH;
        const float* cp = cl + (t & 1) * BH;
        float* hn = hl + ((t + 1) & 1) * BH;
        float* cn = cl + ((t + 1) & 1) * BH;
        // rows past act stop here for good, so their slots are never read again
        for (int j = tid; j / S < act * H; j += kSmallThreads) {   // uniform over a cell's S lanes
            const int i = j / S, r = i / H, u = i % H;
            const int64_t p = off + r;
            float x[4] = {xpre[0], xpre[1], xpre[2], xpre[3]};
            if (part == 0 && j != tid) load_x(off, i, x);
            const float* hr = hp + r * H;
            const float *wi = Wl + u * ldw, *wf = Wl + (H + u) * ldw;
            const float *wg = Wl + (2 * H + u) * ldw, *wo = Wl + (3 * H + u) * ldw;
            float ai = 0.f, af = 0.f, ag = 0.f, ao = 0.f;
#pragma unroll 4
            for (int k = part; k < H; k += S) {
                const float hk = hr[k];
                ai += hk * wi[k];
                af += hk * wf[k];
                ag += hk * wg[k];
                ao += hk * wo[k];
            }
            ai = small_group_sum<S>(ai);
            af = small_group_sum<S>(af);
            ag = small_group_sum<S>(ag);
            ao = small_group_sum<S>(ao);
            if (part == 0) {
                const float gi = sigmoidf_(ai + x[0]), gf = sigmoidf_(af + x[1]);
                const float gg = tanhf_(ag + x[2]), go = sigmoidf_(ao + x[3]);
                const float c = gf * cp[i] + gi * gg;
                const float h = go * tanhf_(c);
                const T hq = from_f<T>(h);
                hn[i] = to_f(hq);
                cn[i] = c;
                a.Cs[(a.B + p) * a.ldh + u] = c;
                a.Hs[(a.B + p) * a.ldh + u] = hq;
                T* gs = a.Gs + p * a.ldg + u;
                gs[0] = from_f<T>(gi);
                gs[H] = from_f<T>(gf);
                gs[2 * H] = from_f<T>(gg);
                gs[3 * H] = from_f<T>(go);
                const int b = a.perm ? a.perm[r] : r;
                if (a.y) a.y[(int64_t(t) * B + b) * H + u] = hq;
                if (r >= act_next) {   // last step of this sequence
                    if (a.hT) a.hT[int64_t(b) * H + u] = h;
                    if (a.cT) a.cT[int64_t(b) * H + u] = c;
                }
            }
        }
        if (part == 0 && tid / S < act_next * H) load_x(persist::off_at(a.offsets, a.fixed, B, t + 1), tid / S, xpre);
        __syncthreads();   // step t + 1 reads what step t wrote
    }
}

template <typename T>
struct BwdSmall {
    int H, B, t_eff, fixed;
    const int32_t* active;
    const int32_t* offsets;
    int64_t ldh, ldg;
    const T* Wh;
    T* G;                     // dG rows of every step (for the contractions after the loop)
    const T* Gs;
    const float* Cs;
    const T* dy;
    int64_t dy_ld;
    const int32_t* dy_rows;
    const float* dh;          // initial dh, dc of the sorted rows (from dhT, dcT)
    const float* dc;
    const int32_t* perm;
    float* dh0;
    float* dc0;
};

template <typename T, int S>
__global__ __launch_bounds__(kSmallThreads) void bwd_small_kernel(BwdSmall<T> a) {
    extern __shared__ float smem_f[];
    const int H = a.H, B = a.B, G4 = 4 * H, ldk = G4 + S, BH = B * H;
    float* Wt = smem_f;              // [H][4H + S]: Wt[u][k] = Wh[k][u]
    float* gl = Wt + H * ldk;        // [2][B][4H]: dG of steps t + 1 and t, in turn
    float* dcl = gl + 2 * B * G4;    // [2][B][H]
    float* dhl = dcl + 2 * BH;       // [B][H]: dh of rows not yet started
    const int tid = threadIdx.x, part = tid % S;
    for (int i = tid; i < G4 * H; i += kSmallThreads) Wt[(i % H) * ldk + i / H] = to_f(a.Wh[i]);
    // a row's dc enters from either buffer at the step its sequence ends
    for (int i = tid; i < BH; i += kSmallThreads) {
        dhl[i] = a.dh[i];
        dcl[i] = dcl[BH + i] = a.dc[i];
    }
    // saved gates, c_t, c_{t-1} and dy of cell i of step t (lane part 0 only)
    auto load_ops = [&](int t, int i, float* v) {
        const int r = i / H, u = i % H;
        const int64_t p = persist::off_at(a.offsets, a.fixed, B, t) + r;
        const int64_t prev_base = t == 0 ? 0 : int64_t(B) + persist::off_at(a.offsets, a.fixed, B, t - 1);
        const T* gs = a.Gs + p * a.ldg + u;
#pragma unroll
        for (int g = 0; g < 4; ++g) v[g] = to_f(gs[g * H]);
        v[4] = a.Cs[(a.B + p) * a.ldh + u];
        v[5] = a.Cs[(prev_base + r) * a.ldh + u];
        v[6] = a.dy ? to_f(a.dy[(a.dy_rows ? int64_t(a.dy_rows[p]) : p) * a.dy_ld + u]) : 0.f;
    };
    float pre[7] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};   // of the first cell of this thread, one step ahead
    if (part == 0 && a.t_eff > 0 && tid / S < persist::act_at(a.active, a.fixed, B, a.t_eff - 1, a.t_eff) * H)
        load_ops(a.t_eff - 1, tid / S, pre);
    __syncthreads();
    // dh of cell i = (r, u): sum_k dG_{t+1}[r, k] Wh[k, u] over the S parts
    // for a row that ran at t + 1, else the carried dh (all lanes of a cell
    // take the same branch)
    auto dh_of = [&](const float* gnext, int i, int act_next) -> float {
        const int r = i / H, u = i % H;
        if (r >= act_next) return dhl[i];
        const float* gr = gnext + r * G4;
        const float* wr = Wt + u * ldk;
        float s0 = 0.f, s1 = 0.f;
        int k = part;
#pragma unroll 2
        for (; k + S < G4; k += 2 * S) {
            s0 += gr[k] * wr[k];
            s1 += gr[k + S] * wr[k + S];
        }
        if (k < G4) s0 += gr[k] * wr[k];
        return small_group_sum<S>(s0 + s1);
    };
    int cur = 0;   // buffer that holds dG_{t+1} and dc_{t+1}
    for (int t = a.t_eff - 1; t >= 0; --t, cur ^= 1) {
        const int act = persist::act_at(a.active, a.fixed, B, t, a.t_eff);
        const int act_next = persist::act_at(a.active, a.fixed, B, t + 1, a.t_eff);
        const int64_t off = persist::off_at(a.offsets, a.fixed, B, t);
        const float* gc = gl + cur * B * G4;
        const float* dcc = dcl + cur * BH;
        float* gn = gl + (cur ^ 1) * B * G4;
        float* dcn = dcl + (cur ^ 1) * BH;
        for (int j = tid; j / S < act * H; j += kSmallThreads) {
            const int i = j / S, r = i / H, u = i % H;
            const int64_t p = off + r;
            float v[7];
#pragma unroll
            for (int e = 0; e < 7; ++e) v[e] = pre[e];
            if (part == 0 && j != tid) load_ops(t, i, v);
            const float dhv = dh_of(gc, i, act_next) + v[6];
            if (part == 0) {
                const float gi = v[0], gf = v[1], gg = v[2], go = v[3], c = v[4], cprev = v[5];
                const float tau = tanhf_(c);
                const float d_o = dhv * tau;
                const float dct = dcc[i] + dhv * go * (1.f - tau * tau);
                dcn[i] = dct * gf;
                const float dg[4] = {dct * gg * gi * (1.f - gi), dct * cprev * gf * (1.f - gf),
                                     dct * gi * (1.f - gg * gg), d_o * go * (1.f - go)};
                T* gp = a.G + p * a.ldg + u;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const T q = from_f<T>(dg[g]);
                    gp[g * H] = q;
                    gn[r * G4 + g * H + u] = to_f(q);
                }
            }
        }
        if (part == 0 && t > 0 && tid / S < persist::act_at(a.active, a.fixed, B, t - 1, a.t_eff) * H)
            load_ops(t - 1, tid / S, pre);
        __syncthreads();   // step t - 1 reads what step t wrote
    }
    // gradient of the initial state
    const int act0 = persist::act_at(a.active, a.fixed, B, 0, a.t_eff);
    const float* gc = gl + cur * B * G4;
    const float* dcc = dcl + cur * BH;
    for (int j = tid; j / S < BH; j += kSmallThreads) {
        const int i = j / S, r = i / H, u = i % H;
        const float dhv = dh_of(gc, i, act0);
        if (part == 0) {
            const int b = a.perm ? a.perm[r] : r;
            if (a.dh0) a.dh0[int64_t(b) * H + u] = dhv;
            if (a.dc0) a.dc0[int64_t(b) * H + u] = dcc[i];
        }
    }
}

// bf16: 128 rows x 32 columns per tile, 4 waves of 32x32
using StepBF16 = TileCfg<bf16_t, 128, 32, 32, 4, 1>;
// fp32: 64 rows x 32 columns per tile, 2 waves of 32x32
using StepF32 = TileCfg<float, 64, 32, 32, 2, 1>;

template <class Cfg>
constexpr int step_smem() {
    return Cfg::SMEM_BYTES > Cfg::BM * (Cfg::BN + 1) * 4 ? Cfg::SMEM_BYTES : Cfg::BM * (Cfg::BN + 1) * 4;
}

template <typename T, class Cfg>
janus_status launch_fwd_step(const FwdStep<T>& a, bool al, hipStream_t s) {
    dim3 grid((a.H + a.U - 1) / a.U, (a.active + Cfg::BM - 1) / Cfg::BM);
    TraceScope trace(sizeof(T) == 2 ? "lstm_fwd_step_bf16" : "lstm_fwd_step_f32",
                     2.0 * a.active * 4.0 * a.H * a.H,
                     double(sizeof(T)) * (double(a.active) * a.H + 4.0 * a.H * a.H), s);
    if (al)
        hipLaunchKernelGGL((fwd_step_kernel<T, Cfg, true>), grid, dim3(Cfg::NT), step_smem<Cfg>(), s, a);
    else
        hipLaunchKernelGGL((fwd_step_kernel<T, Cfg, false>), grid, dim3(Cfg::NT), step_smem<Cfg>(), s, a);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

template <typename T, class Cfg>
janus_status launch_bwd_step(const BwdStep<T>& a, bool al, hipStream_t s) {
    dim3 grid((a.H + Cfg::BN - 1) / Cfg::BN, (a.active + Cfg::BM - 1) / Cfg::BM);
    if (grid.y == 0) return JANUS_OK;
    TraceScope trace(sizeof(T) == 2 ? "lstm_bwd_step_bf16" : "lstm_bwd_step_f32",
                     2.0 * a.active_next * 4.0 * a.H * a.H,
                     double(sizeof(T)) * (4.0 * a.active_next * a.H + 4.0 * a.H * a.H), s);
    if (al)
        hipLaunchKernelGGL((bwd_step_kernel<T, Cfg, true>), grid, dim3(Cfg::NT), step_smem<Cfg>(), s, a);
    else
        hipLaunchKernelGGL((bwd_step_kernel<T, Cfg, false>), grid, dim3(Cfg::NT), step_smem<Cfg>(), s, a);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

// lanes per cell of a one-workgroup kernel whose contraction has K terms:
// a power of two, as many as the threads allow while each lane keeps at
// least 32 terms (fewer leave the lanes waiting on LDS latency more than
// the split saves), at most 8
int small_split(const janus_lstm_desc& d, int K) {
    int S = 1;
    while (S < 8 && int64_t(d.B) * d.H * (2 * S) <= kSmallThreads && K >= 64 * S) S *= 2;
    return S;
}
int small_fwd_split(const janus_lstm_desc& d) { return small_split(d, d.H); }
int small_bwd_split(const janus_lstm_desc& d) { return small_split(d, 4 * d.H); }

size_t small_fwd_lds(const janus_lstm_desc& d) {
    return sizeof(float) * (size_t(4) * d.H * (d.H + small_fwd_split(d)) + size_t(4) * d.B * d.H);
}
size_t small_bwd_lds(const janus_lstm_desc& d) {
    return sizeof(float) * (size_t(d.H) * (4 * d.H + small_bwd_split(d)) + size_t(11) * d.B * d.H);
}

// The one-workgroup recurrence replaces the per-step kernels (it is never
// taken where the persistent path applies) when every cell has a thread
// slot and Wh (float32), the state and dG fit one workgroup's LDS.
// JANUS_SMALL=0 switches it off.
bool use_small(const janus_lstm_desc& d) {
    const char* e = getenv("JANUS_SMALL");
    if (e && e[0] == '0') return false;
    if (int64_t(d.B) * d.H > int64_t(kSmallThreads) * kSmallCells) return false;
    const size_t cap = device_lds(device_info());
    return small_fwd_lds(d) <= cap && small_bwd_lds(d) <= cap;
}

// Raise a kernel's dynamic LDS limit when a launch needs more than the
// largest size set so far (cached per kernel in `attr_smem`).  The cache and
// the attribute change together under one lock, so calls from several host
// threads neither race on the cache nor lower the limit under each other.
template <class K>
janus_status raise_lds_limit(K kernel, size_t smem, size_t& attr_smem) {
    static std::mutex m;
    std::lock_guard<std::mutex> lock(m);
    if (smem > attr_smem) {
        JANUS_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                      int(smem)));
        attr_smem = smem;
    }
    return JANUS_OK;
}

template <class K, class A>
janus_status small_launch(K kernel, size_t smem, const A& args, hipStream_t st, size_t& attr_smem) {
    if (janus_status e = raise_lds_limit(kernel, smem, attr_smem); e != JANUS_OK) return e;
    hipLaunchKernelGGL(kernel, dim3(1), dim3(kSmallThreads), smem, st, args);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

template <typename T>
janus_status launch_fwd_small(const janus_lstm_desc& d, const FwdSmall<T>& a, hipStream_t st) {
    static size_t attr[4] = {};
    const size_t smem = small_fwd_lds(d);
    switch (small_fwd_split(d)) {
        case 1: return small_launch(fwd_small_kernel<T, 1>, smem, a, st, attr[0]);
        case 2: return small_launch(fwd_small_kernel<T, 2>, smem, a, st, attr[1]);
        case 4: return small_launch(fwd_small_kernel<T, 4>, smem, a, st, attr[2]);
        default: return small_launch(fwd_small_kernel<T, 8>, smem, a, st, attr[3]);
    }
}

template <typename T>
janus_status launch_bwd_small(const janus_lstm_desc& d, const BwdSmall<T>& a, hipStream_t st) {
    static size_t attr[4] = {};
    const size_t smem = small_bwd_lds(d);
    switch (small_bwd_split(d)) {
        case 1: return small_launch(bwd_small_kernel<T, 1>, smem, a, st, attr[0]);
        case 2: return small_launch(bwd_small_kernel<T, 2>, smem, a, st, attr[1]);
        case 4: return small_launch(bwd_small_kernel<T, 4>, smem, a, st, attr[2]);
        default: return small_launch(bwd_small_kernel<T, 8>, smem, a, st, attr[3]);
    }
}

janus_status check_desc(const janus_lstm_desc* d) {
    if (!d) return JANUS_ERR_INVALID_ARG;
    if (d->L <= 0 || d->I <= 0 || d->H <= 0 || d->B <= 0 || d->T < 0) return JANUS_ERR_INVALID_ARG;
    if (!dtype_ok(d->dtype)) return JANUS_ERR_UNSUPPORTED;
    return JANUS_OK;
}

bool all_nonnull(const void* const* p, int n) {
    if (!p) return false;
    for (int i = 0; i < n; ++i)
        if (!p[i]) return false;
    return true;
}

bool weight_aligned(const janus_lstm_desc& d) {
    // vector loads of Wh rows need 16-byte aligned rows
    return (int64_t(d.H) * int64_t(dtype_size(d.dtype))) % 16 == 0;
}

// Launch of a persistent kernel: an ordinary dispatch on the caller's stream.
// The grid barrier needs every workgroup resident at once.  The fit checks
// allow at most one workgroup per CU and no more workgroups than CUs, and the
// occupancy query below confirms that the registers and LDS of one workgroup
// fit a CU, so on a device that runs nothing else every workgroup is placed
// at launch.  Should some not be (another process holding CUs), the waits are
// bounded: they set the error flag, the grid drains, and the device report
// returns JANUS_ERR_DEVICE.
//
// A cooperative launch would make the runtime check residency itself, but it
// dispatches through a second hardware queue, ordered against the caller's
// stream with extra barrier packets around every launch; under a profiler
// that queue's teardown ended the process with a segmentation fault at exit.
template <class K, class A>
janus_status persistent_launch(K kernel, int blocks, size_t smem, const A& args, hipStream_t st, size_t& attr_smem) {
    if (janus_status e = raise_lds_limit(kernel, smem, attr_smem); e != JANUS_OK) return e;
    const DeviceInfo info = device_info();
    int per_cu = 0;
    JANUS_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel),
                                                           persist::kThreads, smem));
    if (per_cu < 1 || int64_t(per_cu) * info.cus < blocks) return JANUS_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(kernel, dim3(blocks), dim3(persist::kThreads), smem, st, args);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

janus_status launch_fwd_persistent(const janus_lstm_desc& d, int ns, persist::FwdArgs& a, double flops,
                                   double bytes, hipStream_t st) {
    static size_t attr[3][4] = {};
    const int kw = persist_kw(d.B);
    const size_t smem = persist_fwd_lds(d, ns);
    const int blocks = persist_fwd_blocks(d, ns);
    TraceScope trace("lstm_fwd_persistent", flops, bytes, st);
#define JANUS_FWD_CASES(NS, I)                                                                               \
    switch (kw) {                                                                                            \
        case 1: return persistent_launch(persist::lstm_fwd_persistent<1, NS>, blocks, smem, a, st, attr[I][0]); \
        case 2: return persistent_launch(persist::lstm_fwd_persistent<2, NS>, blocks, smem, a, st, attr[I][1]); \
        case 4: return persistent_launch(persist::lstm_fwd_persistent<4, NS>, blocks, smem, a, st, attr[I][2]); \
        default: return persistent_launch(persist::lstm_fwd_persistent<8, NS>, blocks, smem, a, st, attr[I][3]); \
    }
    if (ns == 4) JANUS_FWD_CASES(4, 2)
    if (ns == 2) JANUS_FWD_CASES(2, 1)
    JANUS_FWD_CASES(1, 0)
#undef JANUS_FWD_CASES
}

janus_status launch_bwd_persistent(const janus_lstm_desc& d, int ns, persist::BwdArgs& a, double flops,
                                   double bytes, hipStream_t st) {
    static size_t attr[8] = {};
    const int kw = persist_kw(d.B);
    const size_t smem = persist_bwd_lds(d, ns);
    const int blocks = persist_bwd_blocks(d, ns);
    TraceScope trace("lstm_bwd_persistent", flops, bytes, st);
    if (ns == 8) {
        switch (kw) {
            case 1: return persistent_launch(persist::lstm_bwd_persistent<1, 8>, blocks, smem, a, st, attr[4]);
            case 2: return persistent_launch(persist::lstm_bwd_persistent<2, 8>, blocks, smem, a, st, attr[5]);
            case 4: return persistent_launch(persist::lstm_bwd_persistent<4, 8>, blocks, smem, a, st, attr[6]);
            default: return persistent_launch(persist::lstm_bwd_persistent<8, 8>, blocks, smem, a, st, attr[7]);
        }
    }
    switch (kw) {
        case 1: return persistent_launch(persist::lstm_bwd_persistent<1, 4>, blocks, smem, a, st, attr[0]);
        case 2: return persistent_launch(persist::lstm_bwd_persistent<2, 4>, blocks, smem, a, st, attr[1]);
        case 4: return persistent_launch(persist::lstm_bwd_persistent<4, 4>, blocks, smem, a, st, attr[2]);
        default: return persistent_launch(persist::lstm_bwd_persistent<8, 4>, blocks, smem, a, st, attr[3]);
    }
}

// sum over steps of rows with a recurrent product: forward rows t < t_eff,
// backward rows of the contractions from dG_{t+1}
double recurrent_rows(const SeqSchedule& s) {
    double r = 0;
    for (int t = 0; t < s.t_eff; ++t) r += s.active[t];
    return r;
}

// Recurrent rows of the batch part starting at sorted row rb (at most kMaxB rows).
double part_rows(const SeqSchedule& s, int rb) {
    double rows = 0;
    for (int t = 0; t < s.t_eff; ++t) rows += std::min(std::max(s.active[t] - rb, 0), persist::kMaxB);
    return rows;
}

// Algorithmic bytes of one persistent launch over `rows` active rows: every
// value the recurrence must read or write, counted once, plus the recurrent
// weight (4H x H bf16) read once.
//   forward, per row:  XG (4H bf16), h_{t-1} (H bf16), c_t (H fp32), the
//                      gates (4H bf16), h_t for the next step (H bf16), and
//                      the optional copies (h row-major, h transposed, y)
//   backward, per row: the saved gates (4H bf16), c_{t-1} (H fp32), dy
//                      (H bf16), dG_{t+1} (4H bf16), dG_t for the next step
//                      (4H bf16), and the optional dG copies (transposed,
//                      row-major)
double fwd_persistent_bytes(const persist::FwdArgs& a, double rows) {
    const double H = a.H;
    const double per_row = (8.0 + 2.0 + 4.0 + 8.0 + 2.0) * H + (a.Hs ? 2.0 * H : 0.0) + (a.HT ? 2.0 * H : 0.0) +
                           (a.y ? 2.0 * H : 0.0);
    return rows * per_row + 8.0 * H * H;
}
double bwd_persistent_bytes(const persist::BwdArgs& a, double rows) {
    const double H = a.H;
    const double per_row = (8.0 + 4.0 + 8.0 + 8.0) * H + (a.dy ? 2.0 * H : 0.0) + (a.GT ? 8.0 * H : 0.0) +
                           (a.G ? 8.0 * H : 0.0);
    return rows * per_row + 8.0 * H * H;
}

// With equal lengths the persistent forward also writes h transposed (HT,
// h0 in the first B columns): HT is then h_{t-1} transposed for every
// packed row (the dWh operand) and HT + B is the layer output transposed
// (the next layer's dWx operand), both read in place (K = T B a multiple of 8).
bool use_ht(const janus_lstm_desc& d, const SeqSchedule& s, bool persistent) {
    return persistent && s.fixed && (int64_t(d.T) * d.B) % 8 == 0;
}

// The persistent backward writes dG transposed itself when the padded tail of
// each row (past the packed count, to a multiple of 8) needs no zeros.
bool gt_by_kernel(const SeqSchedule& s, bool persistent) { return persistent && s.packed % 8 == 0; }

// One layer of the forward pass on the persistent path (bf16 only).
janus_status fwd_layer_persistent(const janus_lstm_desc& d, const SeqSchedule& s, const LstmWs& w, int l,
                                  const void* x, const int32_t* xrow, const void* Wx, const void* Wh, const void* b,
                                  const int32_t* perm, void* y, float* hT, float* cT, hipStream_t st) {
    const int H = d.H, B = d.B;
    const int Il = l == 0 ? d.I : H;
    const int64_t rows4 = int64_t(4) * H * Il;
    {
        TraceScope trace("interleave_weights", 0.0, 4.0 * double(rows4 + 4 * H), st);
        hipLaunchKernelGGL(interleave_rows_kernel<bf16_t>, dim3(unsigned((rows4 + 255) / 256)), dim3(256), 0, st,
                           static_cast<const bf16_t*>(Wx), static_cast<bf16_t*>(w.Wxi[l]), H, Il);
        JANUS_LAUNCH_CHECK();
        hipLaunchKernelGGL(interleave_rows_kernel<bf16_t>, dim3(unsigned((4 * H + 255) / 256)), dim3(256), 0, st,
                           static_cast<const bf16_t*>(b), static_cast<bf16_t*>(w.bi[l]), H, 1);
        JANUS_LAUNCH_CHECK();
    }
    GemmDesc g;
    g.dtype = JANUS_BF16;
    g.M = int(s.packed);
    g.N = 4 * H;
    g.K = Il;
    if (l == 0) {
        g.A = x;
        g.lda = d.I;
        g.a_idx = xrow;
    } else {
        g.A = static_cast<const bf16_t*>(w.Hs[l - 1]) + int64_t(B) * w.ldh;
        g.lda = w.ldh;
    }
    g.a_src_rows = int64_t(d.T) * B;
    g.B = w.Wxi[l];
    g.ldb = Il;
    g.C = w.XG;
    g.ldc = w.ldg;
    g.c_f32 = false;
    g.bias = w.bi[l];
    g.scratch = w.gs;
    g.scratch_bytes = w.gs_bytes;
    janus_status e = gemm(g, st);
    if (e != JANUS_OK) return e;
    if ((e = zero_fill(w.sync, persist::kSyncCounterBytes, st)) != JANUS_OK) return e;
    persist::FwdArgs a = {};
    a.H = H;
    a.B = B;
    a.t_eff = s.t_eff;
    a.fixed = s.fixed ? 1 : 0;
    a.Kp = int(round_up(H, 64));
    const int ns = persist_fwd_slices(d);
    a.nkg = persist_fwd_nkg(d);
    a.ksp = persist_fwd_ksp(d, ns);
    a.part = w.dpart;
    a.part_local = persist_fwd_part_local(d, ns);
    a.nstraddle = persist_straddle_slots();
    a.active = w.act_dev;
    a.offsets = w.off_dev;
    a.perm = perm;
    a.Wh = static_cast<const bf16_t*>(Wh);
    a.Hs = static_cast<bf16_t*>(w.Hs[l]);
    a.Cs = w.Cs[l];
    a.XG = static_cast<const bf16_t*>(w.XG);
    a.Gs = static_cast<bf16_t*>(w.Gs[l]);
    a.y = static_cast<bf16_t*>(y);
    a.hT = hT;
    a.cT = cT;
    a.ldh = w.ldh;
    a.ldg = w.ldg;
    a.Hf = w.Hf;
    a.hf_slot = w.hf_slot;
    a.HT = use_ht(d, s, true) ? w.HT[l] : nullptr;
    // the top layer's row-major h is read only by its weight gradients, and
    // only when they cannot take the transposed copy
    if (l == d.L - 1 && a.HT) a.Hs = nullptr;
    a.ldht = w.ldht;
    a.sync = w.sync;
    // batches past kMaxB rows run in parts of kMaxB sorted rows, one launch
    // each (rows are independent sequences; the counters restart per launch)
    for (int rb = 0; rb < B; rb += persist::kMaxB) {
        if (rb > 0 && (e = zero_fill(w.sync, persist::kSyncCounterBytes, st)) != JANUS_OK) return e;
        a.rbase = rb;
        const double rows = part_rows(s, rb);
        e = launch_fwd_persistent(d, ns, a, 2.0 * 4.0 * H * double(H) * rows, fwd_persistent_bytes(a, rows), st);
        if (e != JANUS_OK) return e;
    }
    return JANUS_OK;
}

template <typename T, class Cfg>
janus_status lstm_fwd_impl(const janus_lstm_desc& d, const SeqSchedule& s, const LstmWs& w, const void* x,
                           const void* const* Wx, const void* const* Wh, const void* const* b, const float* h0,
                           const float* c0, void* y, float* hT, float* cT, hipStream_t st) {
    const int B = d.B, H = d.H;
    const int64_t TB = int64_t(d.T) * B;
    const int32_t* perm = s.fixed ? nullptr : w.perm;
    const int32_t* xrow = s.fixed ? nullptr : w.xrow;
    if (!s.fixed) {
        janus_status e = zero_fill(y, size_t(TB) * H * sizeof(T), st);
        if (e != JANUS_OK) return e;
    }
    const bool al = weight_aligned(d);
    const bool persistent = use_persistent(d);
    if (persistent && H % 64 != 0) {
        // columns [H, Kp) of the fragment-layout copy are never written and
        // take part in the contraction against zero weights: make them 0
        janus_status e = zero_fill(w.Hf, size_t(d.T + 1) * size_t(w.hf_slot) * 2, st);
        if (e != JANUS_OK) return e;
    }
    for (int l = 0; l < d.L; ++l) {
        const int64_t bh = int64_t(B) * H;
        {
            TraceScope trace("lstm_fwd_init", 0.0, double(bh) * (8.0 + 4.0 + sizeof(T)), st);
            hipLaunchKernelGGL(fwd_init_kernel<T>, dim3(unsigned((bh + 255) / 256)), dim3(256), 0, st, B, H, w.ldh,
                               perm, h0 ? h0 + l * bh : nullptr, c0 ? c0 + l * bh : nullptr,
                               static_cast<T*>(w.Hs[l]), w.Cs[l], s.active[0], hT ? hT + l * bh : nullptr,
                               cT ? cT + l * bh : nullptr, persistent ? reinterpret_cast<T*>(w.Hf) : nullptr,
                               int(round_up(H, 64)), use_ht(d, s, persistent) ? reinterpret_cast<T*>(w.HT[l]) : nullptr,
                               w.ldht);
            JANUS_LAUNCH_CHECK();
        }
        if (s.packed == 0) continue;
        if (persistent) {
            janus_status e = fwd_layer_persistent(d, s, w, l, x, xrow, Wx[l], Wh[l], b[l], perm,
                                                  l == d.L - 1 ? y : nullptr, hT ? hT + l * bh : nullptr,
                                                  cT ? cT + l * bh : nullptr, st);
            if (e != JANUS_OK) return e;
            continue;
        }
        // hoisted input projection of every running (t, b)
        GemmDesc g;
        g.dtype = d.dtype;
        g.M = int(s.packed);
        g.N = 4 * H;
        g.K = l == 0 ? d.I : H;
        if (l == 0) {
            g.A = x;
            g.lda = d.I;
            g.a_idx = xrow;
        } else {
            g.A = static_cast<const T*>(w.Hs[l - 1]) + int64_t(B) * w.ldh;
            g.lda = w.ldh;
        }
        g.a_src_rows = TB;
        g.B = Wx[l];
        g.ldb = g.K;
        g.C = w.XG;
        g.ldc = w.ldg;
        g.c_f32 = false;
        g.bias = b[l];
        g.scratch = w.gs;
        g.scratch_bytes = w.gs_bytes;
        janus_status e = gemm(g, st);
        if (e != JANUS_OK) return e;
        if (use_small(d)) {
            FwdSmall<T> a = {};
            a.H = H;
            a.B = B;
            a.t_eff = s.t_eff;
            a.fixed = s.fixed ? 1 : 0;
            a.active = w.act_dev;
            a.offsets = w.off_dev;
            a.ldh = w.ldh;
            a.ldg = w.ldg;
            a.Wh = static_cast<const T*>(Wh[l]);
            a.XG = static_cast<const T*>(w.XG);
            a.Hs = static_cast<T*>(w.Hs[l]);
            a.Cs = w.Cs[l];
            a.Gs = static_cast<T*>(w.Gs[l]);
            a.y = l == d.L - 1 ? static_cast<T*>(y) : nullptr;
            a.perm = perm;
            a.hT = hT ? hT + l * bh : nullptr;
            a.cT = cT ? cT + l * bh : nullptr;
            TraceScope trace("lstm_fwd_small", 2.0 * 4.0 * H * double(H) * double(s.packed), 0.0, st);
            if ((e = launch_fwd_small(d, a, st)) != JANUS_OK) return e;
            continue;
        }
        for (int t = 0; t < s.t_eff; ++t) {
            FwdStep<T> a;
            a.H = H;
            a.B = B;
            a.t = t;
            a.active = s.active[t];
            a.active_next = s.active[t + 1];
            a.U = Cfg::BN / 4;
            a.off_t = s.offsets[t];
            a.prev_base = t == 0 ? 0 : int64_t(B) + s.offsets[t - 1];
            a.ldh = w.ldh;
            a.ldg = w.ldg;
            a.Hs = static_cast<T*>(w.Hs[l]);
            a.Cs = w.Cs[l];
            a.Wh = static_cast<const T*>(Wh[l]);
            a.XG = static_cast<const T*>(w.XG);
            a.Gs = static_cast<T*>(w.Gs[l]);
            a.y = l == d.L - 1 ? static_cast<T*>(y) : nullptr;
            a.perm = perm;
            a.hT = hT ? hT + l * bh : nullptr;
            a.cT = cT ? cT + l * bh : nullptr;
            e = launch_fwd_step<T, Cfg>(a, al, st);
            if (e != JANUS_OK) return e;
        }
    }
    return JANUS_OK;
}

template <typename T, class Cfg>
janus_status lstm_bwd_impl(const janus_lstm_desc& d, const SeqSchedule& s, const LstmWs& w, const void* x,
                           const void* const* Wx, const void* const* Wh, const void* dy, const float* dhT,
                           const float* dcT, void* dx, float* dh0, float* dc0, float* const* dWx,
                           float* const* dWh, float* const* db, hipStream_t st) {
    const int B = d.B, H = d.H;
    const int64_t TB = int64_t(d.T) * B;
    const int32_t* perm = s.fixed ? nullptr : w.perm;
    const int32_t* xrow = s.fixed ? nullptr : w.xrow;
    const int32_t* prevrow = s.fixed ? nullptr : w.prevrow;
    const bool al = weight_aligned(d);
    if (dx && !s.fixed) {
        janus_status e = zero_fill(dx, size_t(TB) * d.I * sizeof(T), st);
        if (e != JANUS_OK) return e;
    }
    const int64_t bh = int64_t(B) * H;
    const bool persistent = use_persistent(d);
    if (persistent) {
        TraceScope trace("perm4", 0.0, 16.0 * H, st);
        hipLaunchKernelGGL(perm4_kernel, dim3(unsigned((4 * H + 255) / 256)), dim3(256), 0, st, H, w.perm4);
        JANUS_LAUNCH_CHECK();
    }
    for (int l = d.L - 1; l >= 0; --l) {
        const bool top = l == d.L - 1;
        if (persistent) {
            janus_status e = zero_fill(w.sync, persist::kSyncCounterBytes, st);
            if (e != JANUS_OK) return e;
            persist::BwdArgs a = {};
            a.H = H;
            a.B = B;
            a.t_eff = s.t_eff;
            a.fixed = s.fixed ? 1 : 0;
            const int ns = persist_bwd_slices(d);
            a.nkg = persist_bwd_nkg(d);
            a.ksp = persist_bwd_ksp(d, ns);
            a.Gf = w.Gf;
            a.gf_slot = w.gf_slot;
            a.active = w.act_dev;
            a.offsets = w.off_dev;
            a.perm = perm;
            a.Wh = static_cast<const bf16_t*>(Wh[l]);
            a.G = static_cast<bf16_t*>(w.XG);
            a.Gs = static_cast<const bf16_t*>(w.Gs[l]);
            a.Cs = w.Cs[l];
            if (top) {
                a.dy = static_cast<const bf16_t*>(dy);
                a.dy_ld = H;
                a.dy_rows = xrow;
            } else {
                a.dy = static_cast<const bf16_t*>(w.dY);
                a.dy_ld = w.ldh;
                a.dy_rows = nullptr;
            }
            a.dhT = dhT ? dhT + l * bh : nullptr;
            a.dcT = dcT ? dcT + l * bh : nullptr;
            a.dh0 = dh0 ? dh0 + l * bh : nullptr;
            a.dc0 = dc0 ? dc0 + l * bh : nullptr;
            a.part = w.dpart;
            a.db = db[l];
            a.GT = gt_by_kernel(s, persistent) ? static_cast<bf16_t*>(w.GT) : nullptr;
            // row-major dG only where something reads it: dX (the layer below,
            // or dx asked for), or the weight gradients when dG^T is not here
            if (l == 0 && !dx && a.GT) a.G = nullptr;
            a.ldk = w.ldk;
            a.gt_pairs = (s.fixed && B % 2 == 0) ? 1 : 0;   // packed offsets t B all even
            a.ldh = w.ldh;
            a.ldg = w.ldg;
            a.sync = w.sync;
            // parts of kMaxB sorted rows, as in the forward; the bias
            // gradient of a later part is added to the earlier parts' sum
            for (int rb = 0; rb < B; rb += persist::kMaxB) {
                if (rb > 0 && (e = zero_fill(w.sync, persist::kSyncCounterBytes, st)) != JANUS_OK) return e;
                a.rbase = rb;
                a.db_add = rb > 0 ? 1 : 0;
                const double rows = part_rows(s, rb);
                e = launch_bwd_persistent(d, ns, a, 2.0 * 4.0 * H * double(H) * rows, bwd_persistent_bytes(a, rows), st);
                if (e != JANUS_OK) return e;
            }
        } else {
        {
        TraceScope trace("lstm_bwd_init", 0.0, double(bh) * 16.0, st);
        hipLaunchKernelGGL(bwd_init_kernel, dim3(unsigned((bh + 255) / 256)), dim3(256), 0, st, B, H, perm,
                           dhT ? dhT + l * bh : nullptr, dcT ? dcT + l * bh : nullptr, w.dh, w.dc);
        JANUS_LAUNCH_CHECK();
        }
        BwdStep<T> a;
        a.H = H;
        a.B = B;
        a.ldh = w.ldh;
        a.ldg = w.ldg;
        a.Wh = static_cast<const T*>(Wh[l]);
        a.G = static_cast<T*>(w.XG);
        a.Gs = static_cast<const T*>(w.Gs[l]);
        a.Cs = w.Cs[l];
        if (top) {
            a.dy = static_cast<const T*>(dy);
            a.dy_ld = H;
            a.dy_rows = xrow;
        } else {
            a.dy = static_cast<const T*>(w.dY);
            a.dy_ld = w.ldh;
            a.dy_rows = nullptr;
        }
        a.dh = w.dh;
        a.dc = w.dc;
        a.perm = perm;
        a.dh0 = dh0 ? dh0 + l * bh : nullptr;
        a.dc0 = dc0 ? dc0 + l * bh : nullptr;
        if (use_small(d)) {
            if (s.t_eff > 0 || a.dh0 || a.dc0) {
                BwdSmall<T> q = {};
                q.H = H;
                q.B = B;
                q.t_eff = s.t_eff;
                q.fixed = s.fixed ? 1 : 0;
                q.active = w.act_dev;
                q.offsets = w.off_dev;
                q.ldh = w.ldh;
                q.ldg = w.ldg;
                q.Wh = a.Wh;
                q.G = a.G;
                q.Gs = a.Gs;
                q.Cs = a.Cs;
                q.dy = a.dy;
                q.dy_ld = a.dy_ld;
                q.dy_rows = a.dy_rows;
                q.dh = w.dh;
                q.dc = w.dc;
                q.perm = perm;
                q.dh0 = a.dh0;
                q.dc0 = a.dc0;
                TraceScope trace("lstm_bwd_small", 2.0 * 4.0 * H * double(H) * double(recurrent_rows(s)), 0.0, st);
                janus_status e = launch_bwd_small(d, q, st);
                if (e != JANUS_OK) return e;
            }
        } else {
        for (int t = s.t_eff - 1; t >= 0; --t) {
            a.final_step = 0;
            a.active = s.active[t];
            a.active_next = s.active[t + 1];
            a.off_t = s.offsets[t];
            a.off_next = s.offsets[t + 1];
            a.prev_base = t == 0 ? 0 : int64_t(B) + s.offsets[t - 1];
            janus_status e = launch_bwd_step<T, Cfg>(a, al, st);
            if (e != JANUS_OK) return e;
        }
        if (a.dh0 || a.dc0) {
            a.final_step = 1;
            a.active = B;
            a.active_next = s.active[0];
            a.off_t = 0;
            a.off_next = 0;
            a.prev_base = 0;
            janus_status e = launch_bwd_step<T, Cfg>(a, al, st);
            if (e != JANUS_OK) return e;
        }
        }
        }
        const int32_t* rowmap = persistent ? w.perm4 : nullptr;   // interleaved gate rows -> torch rows
        const int Il = l == 0 ? d.I : H;
        // dG^T once for both weight gradients, so that they read it in place
        // (written by the persistent backward itself when it can)
        const bool gt = w.GT && (4 * H) % 8 == 0;
        if (gt && !gt_by_kernel(s, persistent)) {
            janus_status e = transpose_bf16(w.XG, w.ldg, nullptr, s.packed, 4 * H, w.GT, w.ldk,
                                            round_up(s.packed, 64), st);
            if (e != JANUS_OK) return e;
        }
        // dWx = dG^T X
        GemmDesc g;
        g.dtype = d.dtype;
        g.M = 4 * H;
        g.N = Il;
        g.K = int(s.packed);
        if (gt) {
            g.A = w.GT;
            g.lda = w.ldk;
            g.a_zero_pad = true;
        } else {
            g.a_t = true;
            g.A = w.XG;
            g.lda = w.ldg;
        }
        g.scratch = w.gs;
        g.scratch_bytes = w.gs_bytes;
        const bool ht = use_ht(d, s, persistent);
        g.b_t = true;
        if (l == 0) {
            g.B = x;
            g.ldb = d.I;
            g.b_idx = xrow;
        } else if (ht) {
            g.b_t = false;   // the layer below's output, transposed, in place
            g.B = w.HT[l - 1] + B;
            g.ldb = w.ldht;
        } else {
            g.B = static_cast<const T*>(w.Hs[l - 1]) + int64_t(B) * w.ldh;
            g.ldb = w.ldh;
        }
        g.C = dWx[l];
        g.ldc = Il;
        g.c_idx = rowmap;
        g.c_f32 = true;
        janus_status e = gemm(g, st);
        if (e != JANUS_OK) return e;
        // dWh = dG^T H_prev
        g.N = H;
        if (ht) {
            g.b_t = false;   // h_{t-1} transposed, in place
            g.B = w.HT[l];
            g.ldb = w.ldht;
            g.b_idx = nullptr;
        } else {
            g.b_t = true;
            g.B = w.Hs[l];
            g.ldb = w.ldh;
            g.b_idx = prevrow;
        }
        g.C = dWh[l];
        g.ldc = H;
        e = gemm(g, st);
        if (e != JANUS_OK) return e;
        if (!persistent) {   // the persistent backward forms db itself
            e = colsum(d.dtype, w.XG, s.packed, 4 * H, w.ldg, db[l], w.part, st, rowmap);
            if (e != JANUS_OK) return e;
        }
        // gradient of this layer's input: dG Wx
        if (l > 0 || dx) {
            GemmDesc q;
            q.dtype = d.dtype;
            q.M = int(s.packed);
            q.N = Il;
            q.K = 4 * H;
            q.A = w.XG;
            q.lda = w.ldg;
            q.b_t = true;
            q.B = persistent ? w.Wxi[l] : Wx[l];
            q.ldb = Il;
            q.c_f32 = false;
            q.scratch = w.gs;
            q.scratch_bytes = w.gs_bytes;
            if (l > 0) {
                q.C = w.dY;
                q.ldc = w.ldh;
            } else {
                q.C = dx;
                q.ldc = d.I;
                q.c_idx = xrow;
            }
            e = gemm(q, st);
            if (e != JANUS_OK) return e;
        }
    }
    return JANUS_OK;
}

janus_status upload_schedule(const SeqSchedule& s, const LstmWs& w, hipStream_t st) {
    if (s.fixed) return JANUS_OK;
    janus_status e = upload(w.perm, s.perm.data(), sizeof(int32_t) * s.B, st);
    if (e != JANUS_OK) return e;
    if (s.packed > 0) {
        e = upload(w.xrow, s.xrow.data(), sizeof(int32_t) * s.packed, st);
        if (e != JANUS_OK) return e;
        e = upload(w.prevrow, s.prevrow.data(), sizeof(int32_t) * s.packed, st);
        if (e != JANUS_OK) return e;
    }
    e = upload(w.act_dev, s.active.data(), sizeof(int32_t) * (s.T + 1), st);
    if (e != JANUS_OK) return e;
    return upload(w.off_dev, s.offsets.data(), sizeof(int32_t) * (s.T + 2), st);
}

// ------------------------------------------------------- padded problems
// A bf16 problem whose hidden size is not a multiple of 16 or whose input
// size is not a multiple of 8 runs as the same problem with those sizes
// rounded up (zero weights, inputs and initial state in the added units and
// input features), so that every row is a whole number of 16-byte chunks and
// the fast paths apply.  An added unit then stays exactly 0 (its gates are
// i = f = o = 1/2, g = 0, so c and h stay 0), feeds nothing (its weight
// columns are 0) and receives zero gradients, so the results on the real
// units are those of the unpadded problem.  Parameters and inputs are copied
// in (padded) and results copied out on every call.
bool needs_padding(const janus_lstm_desc& d) { return d.dtype == JANUS_BF16 && (d.H % 16 != 0 || d.I % 8 != 0); }

janus_lstm_desc padded_desc(const janus_lstm_desc& d) {
    janus_lstm_desc p = d;
    p.H = int(round_up(d.H, 16));
    p.I = int(round_up(d.I, 8));
    return p;
}

struct PadWs {
    std::vector<void*> Wx, Wh, b;      // padded parameters (bf16, gate-major rows of Hp units)
    std::vector<float*> dWx, dWh, db;  // padded gradients (float32)
    void* x = nullptr;                 // [T*B x Ip]
    void* y = nullptr;                 // [T*B x Hp], and dy in the backward
    void* dx = nullptr;                // [T*B x Ip]
    float* s0 = nullptr;               // four [L*B x Hp] float32 state buffers
    float* s1 = nullptr;
    float* s2 = nullptr;
    float* s3 = nullptr;
};

// the padded problem's own workspace comes first, then the copies
size_t carve_pad(const janus_lstm_desc& d, void* base, PadWs& w) {
    const janus_lstm_desc p = padded_desc(d);
    LstmWs inner;
    Carver c(base);
    c.take<char>(carve(p, nullptr, inner));
    const int64_t TB = int64_t(d.T) * d.B, LB = int64_t(d.L) * d.B;
    w.Wx.assign(d.L, nullptr);
    w.Wh.assign(d.L, nullptr);
    w.b.assign(d.L, nullptr);
    w.dWx.assign(d.L, nullptr);
    w.dWh.assign(d.L, nullptr);
    w.db.assign(d.L, nullptr);
    for (int l = 0; l < d.L; ++l) {
        const int64_t Il = l == 0 ? p.I : p.H;
        w.Wx[l] = c.take<bf16_t>(int64_t(4) * p.H * Il);
        w.Wh[l] = c.take<bf16_t>(int64_t(4) * p.H * p.H);
        w.b[l] = c.take<bf16_t>(int64_t(4) * p.H);
        w.dWx[l] = c.take<float>(int64_t(4) * p.H * Il);
        w.dWh[l] = c.take<float>(int64_t(4) * p.H * p.H);
        w.db[l] = c.take<float>(int64_t(4) * p.H);
    }
    w.x = c.take<bf16_t>(TB * p.I);
    w.y = c.take<bf16_t>(TB * p.H);
    w.dx = c.take<bf16_t>(TB * p.I);
    w.s0 = c.take<float>(LB * p.H);
    w.s1 = c.take<float>(LB * p.H);
    w.s2 = c.take<float>(LB * p.H);
    w.s3 = c.take<float>(LB * p.H);
    return c.off + 256;
}

// A batch of padding copies in one launch.  Copy o:
//   dst[r, c] (r < rows, c < cols) = src[sr, c] for c < scols, else 0,
// where the source row sr is r (gate_dH == 0) or, for gate-major parameter
// rows, gate g = r / gate_dH, unit u = r % gate_dH, sr = g * gate_sH + u (no
// source row, i.e. 0, when u >= gate_sH).  Elements are es = 2 or 4 bytes.
// blockIdx.y selects the copy; blocks stride over its elements.
constexpr int kMaxRemaps = 16;
struct RemapOp {
    const void* src;
    void* dst;
    int64_t sld, dld, rows;
    int scols, cols, gate_sH, gate_dH, es;
};
struct RemapBatch {
    RemapOp op[kMaxRemaps];
};

template <typename T>
__device__ __forceinline__ void remap_one(const RemapOp& o, int64_t i) {
    const int64_t r = i / o.cols;
    const int c = int(i % o.cols);
    int64_t sr = r;
    bool ok = c < o.scols;
    if (o.gate_dH > 0) {
        const int64_t g = r / o.gate_dH, u = r % o.gate_dH;
        ok = ok && u < o.gate_sH;
        sr = g * o.gate_sH + u;
    }
    static_cast<T*>(o.dst)[r * o.dld + c] = ok ? static_cast<const T*>(o.src)[sr * o.sld + c] : T(0);
}

__global__ __launch_bounds__(256) void remap_batch_kernel(RemapBatch b) {
    const RemapOp& o = b.op[blockIdx.y];
    const int64_t n = o.rows * o.cols;
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
        if (o.es == 2) remap_one<uint16_t>(o, i);
        else remap_one<uint32_t>(o, i);
    }
}

// Collects copies and launches them together (in groups of kMaxRemaps).
struct RemapList {
    RemapBatch b{};
    int n = 0;
    int64_t most = 0;
    template <typename T>
    janus_status add(const void* src, int64_t sld, int scols, void* dst, int64_t dld, int64_t rows, int cols,
                     int gate_sH, int gate_dH, hipStream_t st) {
        if (rows * cols <= 0) return JANUS_OK;
        if (n == kMaxRemaps) {
            janus_status e = launch(st);
            if (e != JANUS_OK) return e;
        }
        b.op[n++] = RemapOp{src, dst, sld, dld, rows, scols, cols, gate_sH, gate_dH, int(sizeof(T))};
        most = std::max(most, rows * cols);
        return JANUS_OK;
    }
    janus_status launch(hipStream_t st) {
        if (n == 0) return JANUS_OK;
        double bytes = 0;
        for (int i = 0; i < n; ++i) bytes += 2.0 * double(b.op[i].rows) * b.op[i].cols * b.op[i].es;
        TraceScope trace("pad_copy", 0.0, bytes, st);
        const unsigned gx = unsigned(std::min<int64_t>((most + 255) / 256, 1024));
        hipLaunchKernelGGL(remap_batch_kernel, dim3(gx, unsigned(n)), dim3(256), 0, st, b);
        JANUS_LAUNCH_CHECK();
        n = 0;
        most = 0;
        return JANUS_OK;
    }
};

// padded copies of the parameters and x, made by the forward call and kept in
// the workspace for its backward
janus_status pad_params(const janus_lstm_desc& d, const janus_lstm_desc& p, const PadWs& w, const void* x,
                        const void* const* Wx, const void* const* Wh, const void* const* b, RemapList& q,
                        hipStream_t st) {
    janus_status e;
    for (int l = 0; l < d.L; ++l) {
        const int Il = l == 0 ? d.I : d.H, Ilp = l == 0 ? p.I : p.H;
        if ((e = q.add<bf16_t>(Wx[l], Il, Il, w.Wx[l], Ilp, int64_t(4) * p.H, Ilp, d.H, p.H, st)) != JANUS_OK) return e;
        if ((e = q.add<bf16_t>(Wh[l], d.H, d.H, w.Wh[l], p.H, int64_t(4) * p.H, p.H, d.H, p.H, st)) != JANUS_OK)
            return e;
        if ((e = q.add<bf16_t>(b[l], 1, 1, w.b[l], 1, int64_t(4) * p.H, 1, d.H, p.H, st)) != JANUS_OK) return e;
    }
    if (x && d.T > 0) return q.add<bf16_t>(x, d.I, d.I, w.x, p.I, int64_t(d.T) * d.B, p.I, 0, 0, st);
    return JANUS_OK;
}

// [L*B x H] float32 state in / out of the padded layout
janus_status pad_state(const janus_lstm_desc& d, const janus_lstm_desc& p, const float* src, float* dst,
                       RemapList& q, hipStream_t st) {
    return q.add<float>(src, d.H, d.H, dst, p.H, int64_t(d.L) * d.B, p.H, 0, 0, st);
}
janus_status unpad_state(const janus_lstm_desc& d, const janus_lstm_desc& p, const float* src, float* dst,
                         RemapList& q, hipStream_t st) {
    return q.add<float>(src, p.H, p.H, dst, d.H, int64_t(d.L) * d.B, d.H, 0, 0, st);
}

janus_status lstm_fwd_padded(const janus_lstm_desc& d, const SeqSchedule& s, void* ws, const void* x,
                             const void* const* Wx, const void* const* Wh, const void* const* b, const float* h0,
                             const float* c0, void* y, float* hT, float* cT, hipStream_t st) {
    const janus_lstm_desc p = padded_desc(d);
    PadWs w;
    carve_pad(d, ws, w);
    LstmWs inner;
    carve(p, ws, inner);
    RemapList q;
    janus_status e = pad_params(d, p, w, x, Wx, Wh, b, q, st);
    if (e != JANUS_OK) return e;
    if (h0 && (e = pad_state(d, p, h0, w.s0, q, st)) != JANUS_OK) return e;
    if (c0 && (e = pad_state(d, p, c0, w.s1, q, st)) != JANUS_OK) return e;
    if ((e = q.launch(st)) != JANUS_OK) return e;
    std::vector<const void*> Wxp(w.Wx.begin(), w.Wx.end()), Whp(w.Wh.begin(), w.Wh.end()), bp(w.b.begin(), w.b.end());
    e = lstm_fwd_impl<bf16_t, StepBF16>(p, s, inner, w.x, Wxp.data(), Whp.data(), bp.data(), h0 ? w.s0 : nullptr,
                                        c0 ? w.s1 : nullptr, w.y, w.s2, w.s3, st);
    if (e != JANUS_OK) return e;
    if (d.T > 0 && (e = q.add<bf16_t>(w.y, p.H, p.H, y, d.H, int64_t(d.T) * d.B, d.H, 0, 0, st)) != JANUS_OK)
        return e;
    if (hT && (e = unpad_state(d, p, w.s2, hT, q, st)) != JANUS_OK) return e;
    if (cT && (e = unpad_state(d, p, w.s3, cT, q, st)) != JANUS_OK) return e;
    return q.launch(st);
}

janus_status lstm_bwd_padded(const janus_lstm_desc& d, const SeqSchedule& s, void* ws, const void* x,
                             const void* const* Wx, const void* const* Wh, const void* dy, const float* dhT,
                             const float* dcT, void* dx, float* dh0, float* dc0, float* const* dWx, float* const* dWh,
                             float* const* db, hipStream_t st) {
    const janus_lstm_desc p = padded_desc(d);
    PadWs w;
    carve_pad(d, ws, w);
    LstmWs inner;
    carve(p, ws, inner);
    // the padded Wx, Wh and x are still in the workspace from the forward call
    (void)x;
    (void)Wx;
    (void)Wh;
    RemapList q;
    janus_status e;
    const int64_t TB = int64_t(d.T) * d.B;
    if (dy && TB > 0 && (e = q.add<bf16_t>(dy, d.H, d.H, w.y, p.H, TB, p.H, 0, 0, st)) != JANUS_OK) return e;
    if (dhT && (e = pad_state(d, p, dhT, w.s0, q, st)) != JANUS_OK) return e;
    if (dcT && (e = pad_state(d, p, dcT, w.s1, q, st)) != JANUS_OK) return e;
    if ((e = q.launch(st)) != JANUS_OK) return e;
    std::vector<const void*> Wxp(w.Wx.begin(), w.Wx.end()), Whp(w.Wh.begin(), w.Wh.end());
    e = lstm_bwd_impl<bf16_t, StepBF16>(p, s, inner, w.x, Wxp.data(), Whp.data(), dy ? w.y : nullptr,
                                        dhT ? w.s0 : nullptr, dcT ? w.s1 : nullptr, dx ? w.dx : nullptr, w.s2, w.s3,
                                        w.dWx.data(), w.dWh.data(), w.db.data(), st);
    if (e != JANUS_OK) return e;
    if (dx && TB > 0 && (e = q.add<bf16_t>(w.dx, p.I, p.I, dx, d.I, TB, d.I, 0, 0, st)) != JANUS_OK) return e;
    if (dh0 && (e = unpad_state(d, p, w.s2, dh0, q, st)) != JANUS_OK) return e;
    if (dc0 && (e = unpad_state(d, p, w.s3, dc0, q, st)) != JANUS_OK) return e;
    for (int l = 0; l < d.L; ++l) {
        const int Il = l == 0 ? d.I : d.H, Ilp = l == 0 ? p.I : p.H;
        if ((e = q.add<float>(w.dWx[l], Ilp, Ilp, dWx[l], Il, int64_t(4) * d.H, Il, p.H, d.H, st)) != JANUS_OK)
            return e;
        if ((e = q.add<float>(w.dWh[l], p.H, p.H, dWh[l], d.H, int64_t(4) * d.H, d.H, p.H, d.H, st)) != JANUS_OK)
            return e;
        if ((e = q.add<float>(w.db[l], 1, 1, db[l], 1, int64_t(4) * d.H, 1, p.H, d.H, st)) != JANUS_OK) return e;
    }
    return q.launch(st);
}

}  // namespace

}  // namespace janus

using namespace janus;

extern "C" size_t janus_lstm_workspace_bytes(const janus_lstm_desc* d) {
    if (check_desc(d) != JANUS_OK) return 0;
    if (needs_padding(*d)) {
        PadWs w;
        return carve_pad(*d, nullptr, w);
    }
    LstmWs w;
    return carve(*d, nullptr, w);
}

extern "C" janus_status janus_lstm_seq_fwd(const janus_lstm_desc* d, const void* x, const int32_t* lengths,
                                           const void* const* Wx, const void* const* Wh, const void* const* b,
                                           const float* h0, const float* c0, void* y, float* hT, float* cT,
                                           void* ws, size_t ws_bytes, void* stream) {
    janus_status e = check_desc(d);
    if (e != JANUS_OK) return e;
    if ((!x && d->T > 0) || (!y && d->T > 0) || !all_nonnull(Wx, d->L) || !all_nonnull(Wh, d->L) ||
        !all_nonnull(b, d->L))
        return JANUS_ERR_INVALID_ARG;
    if (!ws) return JANUS_ERR_WORKSPACE;
    SeqSchedule s;
    e = build_seq_schedule(d->B, d->T, lengths, s);
    if (e != JANUS_OK) return e;
    if (ws_bytes < janus_lstm_workspace_bytes(d) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    const bool pad = needs_padding(*d);
    LstmWs w;
    carve(pad ? padded_desc(*d) : *d, ws, w);
    hipStream_t st = static_cast<hipStream_t>(stream);
    e = upload_schedule(s, w, st);
    if (e != JANUS_OK) return e;
    // a step starts: the report, timeout flag included, covers this call and
    // the backward calls after it
    if ((e = zero_fill(w.sync, sizeof(persist::Sync), st)) != JANUS_OK) return e;
    if (pad) return lstm_fwd_padded(*d, s, ws, x, Wx, Wh, b, h0, c0, y, hT, cT, st);
    if (d->dtype == JANUS_BF16)
        return lstm_fwd_impl<bf16_t, StepBF16>(*d, s, w, x, Wx, Wh, b, h0, c0, y, hT, cT, st);
    return lstm_fwd_impl<float, StepF32>(*d, s, w, x, Wx, Wh, b, h0, c0, y, hT, cT, st);
}

extern "C" janus_status janus_lstm_seq_bwd(const janus_lstm_desc* d, const void* x, const int32_t* lengths,
                                           const void* const* Wx, const void* const* Wh, void* ws, size_t ws_bytes,
                                           const void* dy, const float* dhT, const float* dcT, void* dx, float* dh0,
                                           float* dc0, float* const* dWx, float* const* dWh, float* const* db,
                                           void* stream) {
    janus_status e = check_desc(d);
    if (e != JANUS_OK) return e;
    if ((!x && d->T > 0) || !all_nonnull(Wx, d->L) || !all_nonnull(Wh, d->L) ||
        !all_nonnull(reinterpret_cast<const void* const*>(dWx), d->L) ||
        !all_nonnull(reinterpret_cast<const void* const*>(dWh), d->L) ||
        !all_nonnull(reinterpret_cast<const void* const*>(db), d->L))
        return JANUS_ERR_INVALID_ARG;
    if (!ws) return JANUS_ERR_WORKSPACE;
    SeqSchedule s;
    e = build_seq_schedule(d->B, d->T, lengths, s);
    if (e != JANUS_OK) return e;
    if (ws_bytes < janus_lstm_workspace_bytes(d) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    const bool pad = needs_padding(*d);
    LstmWs w;
    carve(pad ? padded_desc(*d) : *d, ws, w);
    hipStream_t st = static_cast<hipStream_t>(stream);
    e = upload_schedule(s, w, st);
    if (e != JANUS_OK) return e;
    // The backward's own report fields start at zero; the timeout flag and
    // the forward's fields stay as the forward left them, so a wait that ran
    // out in the forward is still reported after the backward (and the
    // backward's kernels drain at once instead of computing on its garbage).
    if ((e = zero_fill(w.sync, persist::kSyncCounterBytes, st)) != JANUS_OK) return e;
    if ((e = zero_fill(&w.sync->groups, 2 * sizeof(unsigned), st)) != JANUS_OK) return e;
    if (pad) return lstm_bwd_padded(*d, s, ws, x, Wx, Wh, dy, dhT, dcT, dx, dh0, dc0, dWx, dWh, db, st);
    if (d->dtype == JANUS_BF16)
        return lstm_bwd_impl<bf16_t, StepBF16>(*d, s, w, x, Wx, Wh, dy, dhT, dcT, dx, dh0, dc0, dWx, dWh, db, st);
    return lstm_bwd_impl<float, StepF32>(*d, s, w, x, Wx, Wh, dy, dhT, dcT, dx, dh0, dc0, dWx, dWh, db, st);
}

namespace janus {
namespace {
// h0[l, r, :] = hT[l, r, :] for r < Bp, else 0 (the same for c); i runs over
// the h half, then the c half
__global__ void state_carry_kernel(int L, int Bp, int Bn, int H, const float* hT, const float* cT, float* h0,
                                   float* c0) {
    const int64_t n = int64_t(L) * Bn * H;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < 2 * n; i += int64_t(gridDim.x) * blockDim.x) {
        const bool cpart = i >= n;
        const int64_t j = cpart ? i - n : i;
        const int64_t u = j % H, r = (j / H) % Bn, l = j / (int64_t(H) * Bn);
        const float* src = cpart ? cT : hT;
        float* dst = cpart ? c0 : h0;
        dst[j] = r < Bp ? src[(l * Bp + r) * H + u] : 0.f;
    }
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return na > 0 && nb > 0 && x < y + nb && y < x + na;
}
}  // namespace
}  // namespace janus

extern "C" janus_status janus_lstm_state_carry(const janus_lstm_desc* d, int32_t B_prev, const float* hT,
                                               const float* cT, float* h0, float* c0, void* stream) {
    janus_status e = check_desc(d);
    if (e != JANUS_OK) return e;
    if (B_prev < 0 || !h0 || !c0 || (B_prev > 0 && (!hT || !cT))) return JANUS_ERR_INVALID_ARG;
    const size_t nn = size_t(d->L) * d->B * d->H * sizeof(float), np = size_t(d->L) * B_prev * d->H * sizeof(float);
    if (overlaps(h0, nn, c0, nn) || overlaps(h0, nn, hT, np) || overlaps(h0, nn, cT, np) || overlaps(c0, nn, hT, np) ||
        overlaps(c0, nn, cT, np))
        return JANUS_ERR_INVALID_ARG;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int64_t n = 2 * int64_t(d->L) * d->B * d->H;
    TraceScope trace("state_carry", 0.0, 4.0 * double(n) * 2.0, st);
    const unsigned blocks = unsigned(std::min<int64_t>((n + 255) / 256, 4096));
    hipLaunchKernelGGL(state_carry_kernel, dim3(blocks), dim3(256), 0, st, d->L, int(B_prev), d->B, d->H, hT, cT, h0,
                       c0);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

extern "C" janus_status janus_lstm_device_report(const janus_lstm_desc* d, const void* ws, size_t ws_bytes,
                                                 janus_lstm_report* out, void* stream) {
    janus_status e = check_desc(d);
    if (e != JANUS_OK) return e;
    if (!out) return JANUS_ERR_INVALID_ARG;
    if (!ws) return JANUS_ERR_WORKSPACE;
    if (ws_bytes < janus_lstm_workspace_bytes(d) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    LstmWs w;
    carve(needs_padding(*d) ? padded_desc(*d) : *d, const_cast<void*>(ws), w);
    unsigned rep[5] = {0u, 0u, 0u, 0u, 0u};
    JANUS_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
    JANUS_HIP(hipMemcpy(rep, &w.sync->error, sizeof(rep), hipMemcpyDeviceToHost));
    out->timed_out = rep[0] != 0u ? 1 : 0;
    out->bwd_groups = int32_t(rep[1]);
    out->bwd_local_groups = int32_t(rep[2]);
    out->fwd_groups = int32_t(rep[3]);
    out->fwd_local_groups = int32_t(rep[4]);
    return out->timed_out ? JANUS_ERR_DEVICE : JANUS_OK;
}

extern "C" janus_status janus_lstm_fault_flag(const janus_lstm_desc* d, const void* ws, size_t ws_bytes,
                                              const uint32_t** out) {
    janus_status e = check_desc(d);
    if (e != JANUS_OK) return e;
    if (!out) return JANUS_ERR_INVALID_ARG;
    if (!ws) return JANUS_ERR_WORKSPACE;
    if (ws_bytes < janus_lstm_workspace_bytes(d) || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return JANUS_ERR_WORKSPACE;
    LstmWs w;
    carve(needs_padding(*d) ? padded_desc(*d) : *d, const_cast<void*>(ws), w);
    static_assert(sizeof(w.sync->error) == sizeof(uint32_t), "one 32-bit word");
    *out = reinterpret_cast<const uint32_t*>(&w.sync->error);
    return JANUS_OK;
}
