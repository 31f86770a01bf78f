// Persistent recurrence kernels: the whole time loop of one layer in one
// cooperative launch, with each workgroup's slice of the recurrent weight
// resident in LDS for all steps and steps separated by a device-wide barrier.
//
// Gate-interleaved layout: activations are stored with column 4u + g for
// hidden unit u and gate g (i, f, g, o), so the four gates of a cell are one
// 8-byte access.  The recurrent weight is read in that order from the
// caller's gate-major Wh ([4H, H], row g*H + u) while it is staged into LDS.
//
// Forward (one barrier per step).  Workgroup j owns units [8j, 8j + 8): the
// 32 interleaved rows of Wh for them stay in LDS.  Per step it computes
//     D[32 gate rows x batch] = Wslice [32 x H] . h_{t-1}^T [H x batch]
// with Wslice as the MFMA A operand (from LDS) and rows of h_{t-1} as the B
// operand (straight from global memory).  In the 32x32 accumulator layout a
// lane then holds all four gates of four units for one batch row, so the
// cell update runs in registers.
//
// Backward (two barriers per step).  dh_{t-1} = dG_t Wh contracts over 4H.
// Workgroup (s, v) holds Wh^T for 32 units v and the quarter s of the 4H
// interleaved gate columns, and writes a partial dh for those units; after a
// barrier, workgroup q sums the four partials (in order s = 0..3) for units
// [8q, 8q + 8), applies the cell backward for step t-1 and writes dG_{t-1};
// after a second barrier the next contraction may read it.  The carried dc
// (and dh of rows whose sequence has not started in reverse) stay in
// registers of the owning thread for the whole launch.
#pragma once

#include "device.hpp"

namespace janus {
namespace persist {

constexpr int kThreads = 512;          // 8 waves
constexpr int kWaves = kThreads / 64;
constexpr int kUnitsFwd = 8;           // hidden units per forward workgroup (32 gate rows)
constexpr int kUnitsBwd = 32;          // hidden units per backward workgroup
constexpr int kSlices = 4;             // K-split of the backward contraction
constexpr int kMaxB = 256;             // batch rows handled by one pass of 8 waves
constexpr int kCellsPerThread = 4;     // (kMaxB * 8 units) / kThreads
constexpr int kSpinLimit = 1 << 22;    // bounded wait at each barrier (~0.1 s)

// Device-wide barrier state (zeroed before every launch).  Counters sit in
// separate 256-byte lines.
struct Sync {
    unsigned count;                    // global arrivals (census first, then one per XCD per barrier)
    unsigned error;                    // set when a wait exceeds its spin limit
    unsigned pad0[62];
    unsigned xcd[16][64];              // per-XCD arrivals
    unsigned census[16][64];           // workgroups resident on each XCD
};

__device__ __forceinline__ unsigned xcc_id() {
    // hardware register XCC_ID (20), bits [3:0]: the XCD this wave runs on
    return __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11)) & 0xfu;
}

// Per-workgroup barrier bookkeeping, meaningful in thread 0 only.
struct Barrier {
    Sync* s;
    unsigned x, xsize, nx, nb, phase;
};

__device__ __forceinline__ bool spin_until(Sync* s, const unsigned* p, unsigned target) {
    int spins = 0;
    while (__hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (__hip_atomic_load(&s->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) return false;
        if (++spins > kSpinLimit) {
            __hip_atomic_store(&s->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
    }
    return true;
}

// Census of the workgroups on every XCD (their L2 is shared), once per launch.
__device__ __forceinline__ void barrier_init(Barrier& b, Sync* s) {
    b.s = s;
    b.nb = gridDim.x;
    b.phase = 0;
    b.x = 0;
    b.xsize = 1;
    b.nx = 1;
    if (threadIdx.x == 0) {
        b.x = xcc_id();
        __hip_atomic_fetch_add(&s->census[b.x][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&s->count, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        spin_until(s, &s->count, b.nb);
        b.xsize = __hip_atomic_load(&s->census[b.x][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        b.nx = 0;
        for (int q = 0; q < 16; ++q)
            b.nx += __hip_atomic_load(&s->census[q][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u;
    }
    __syncthreads();
}

// Device-wide barrier.  Workgroups on one XCD share its L2, so only the last
// of them to arrive releases (one L2 write-back per XCD) and signals the
// global count; every workgroup waits until all XCDs have signalled.
//
// There is no per-workgroup acquire (an acquire would invalidate the XCD's
// shared L2 once per workgroup and throw away the lines the other 31
// workgroups are reading).  This is safe because of how the kernels address
// memory within one launch: every location one workgroup reads after a
// barrier that another workgroup wrote before it is either (a) a row written
// during this launch for the first time and never read before the barrier
// (h and dG rows of a step; rows are padded to whole 128-byte lines so that
// no line is shared between steps), so no cache can hold an old copy, or
// (b) read with the cache-bypassing policy (the reused partial-sum buffer).
// Caches are invalidated by the dispatch at kernel start.
//
// After a timeout every later wait returns at once, so all waves still
// reach the end of the kernel (results are then garbage and `error` is set).
__device__ __forceinline__ void grid_barrier(Barrier& b) {
    ++b.phase;
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_s_waitcnt(0);   // this workgroup's stores have reached the L2
        const unsigned old =
            __hip_atomic_fetch_add(&b.s->xcd[b.x][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == b.phase * b.xsize - 1u)
            __hip_atomic_fetch_add(&b.s->count, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        spin_until(b.s, &b.s->count, b.nb + b.phase * b.nx);
    }
    __syncthreads();
}

// ---------------------------------------------------------------- forward
struct FwdArgs {
    int H, B, t_eff, fixed;
    int Kp;                            // H rounded up to 64
    const int32_t* active;             // [T + 1] (ignored when fixed)
    const int32_t* offsets;            // [T + 2] (ignored when fixed)
    const int32_t* perm;               // [B] or NULL
    const bf16_t* Wh;                  // [4H, H] gate-major
    bf16_t* Hs;                        // [(B + T*B) x ldh]
    float* Cs;                         // [(B + T*B) x ldh]
    const bf16_t* XG;                  // [T*B x ldg] interleaved, bias included
    bf16_t* Gs;                        // [T*B x ldg] interleaved gates
    bf16_t* y;                         // [T, B, H] or NULL
    float* hT;
    float* cT;
    int64_t ldh, ldg;
    bf16_t* Hf;                        // [T + 1] slots of h in fragment layout (slot t = h_{t-1}; slot 0 = h0)
    int64_t hf_slot;                   // elements per slot: round_up(B, 32) * Kp
    Sync* sync;
};

// Fragment layout of a [rows x Kp] bf16 operand (Kp a multiple of 16):
// element (r, k) sits at
//   ((r / 32) * (Kp / 16) + k / 16) * 512 + (((k % 16) / 8) * 32 + r % 32) * 8 + k % 8,
// so the 16 bytes lane l supplies to a 32x32x16 MFMA as the B operand (row
// l % 32, k = 16 j + 8 (l / 32) + [0, 8)) are contiguous and one wave-wide
// load reads 1 KB in one piece, instead of 16 bytes from each of 32 rows.
__host__ __device__ __forceinline__ int64_t frag_index(int64_t r, int k, int Kp) {
    return ((r >> 5) * (Kp >> 4) + (k >> 4)) * 512 + ((((k & 15) >> 3) << 5) + (r & 31)) * 8 + (k & 7);
}

// Schedule values are the same for every lane; readfirstlane keeps them in
// scalar registers so that buffer descriptors built from them stay uniform.
__device__ __forceinline__ int act_at(const int32_t* active, int fixed, int B, int t, int t_eff) {
    if (t >= t_eff || t < 0) return 0;
    return fixed ? B : __builtin_amdgcn_readfirstlane(active[t]);
}
__device__ __forceinline__ int64_t off_at(const int32_t* offsets, int fixed, int B, int t) {
    return fixed ? int64_t(t) * B : int64_t(__builtin_amdgcn_readfirstlane(offsets[t]));
}

// LDS row i = 8a + 4h + b of the forward weight slice holds gate b of unit
// 4h + a: in the 32x32 accumulator layout lane l then holds all four gates
// of the four consecutive units 4 (l / 32) + [0, 4) of its batch row, so the
// cell update reads and writes 16- and 32-byte pieces.
__device__ __forceinline__ int fwd_row_unit(int i) { return 4 * ((i >> 2) & 1) + (i >> 3); }

// Load the 32 rows of the forward weight slice into LDS (k contiguous,
// padded pitch `wld`, zeros past H).
__device__ __forceinline__ void stage_fwd_weights(const FwdArgs& a, bf16_t* Ws, int wld, int u0) {
    const int chunks = a.Kp / 8;
    for (int idx = threadIdx.x; idx < 32 * chunks; idx += kThreads) {
        const int i = idx / chunks, kc = (idx - i * chunks) * 8;
        const int u = u0 + fwd_row_unit(i), g = i & 3;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (u < a.H && kc < a.H) {
            const bf16_t* src = a.Wh + (int64_t(g) * a.H + u) * a.H + kc;
            if (kc + 8 <= a.H && (a.H % 8) == 0) {
                v = *reinterpret_cast<const uint4*>(src);
            } else {
                bf16_t tmp[8];
                for (int e = 0; e < 8; ++e) tmp[e] = (kc + e < a.H) ? src[e] : bf16_t(0);
                __builtin_memcpy(&v, tmp, 16);
            }
        }
        *reinterpret_cast<uint4*>(Ws + i * wld + kc) = v;
    }
}

// acc += Wslice . rows^T over k-blocks [kb0, kb1) of 64.
//
// The operand rows are read with buffer loads through a descriptor that
// covers exactly the rows of this step, so a row past the end reads zeros
// without a branch; a chunk at or past `kmax` (the valid k, a multiple of 8)
// is sent out of range the same way.  `roff` is the byte offset of element
// (row, 32 * (lane / 32)) of this lane's row inside the descriptor.  Rows
// stream through a ring of DEPTH k-blocks kept in flight, so the memory
// latency is paid once per step and each MFMA waits only for its own block.
constexpr int kDepthFwd = 8;
constexpr int kDepthBwd = 4;
constexpr uint32_t kOutOfRange = 0x80000000u;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, int(bytes), 0x00020000);
}

// Stores of per-step results that no other workgroup reads in this launch
// use the sc0|sc1 cache policy (written through), so that the release at the
// next barrier has little dirty data left to write back.
constexpr int kStoreThrough = 1 | 16;
constexpr int kLoadBypass = 1 | 16;    // sc0 | sc1: read from the coherence point, not the caches

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float load4_bypass(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, int(off), 0, kLoadBypass));
}
template <int POLICY>
__device__ __forceinline__ void store4(__amdgpu_buffer_rsrc_t rs, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), rs, int(off), 0, POLICY);
}
template <int POLICY>
__device__ __forceinline__ void store16(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint4 v) {
    const u32x4_t w = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(w, rs, int(off), 0, POLICY);
}
template <int POLICY>
__device__ __forceinline__ void store8(__amdgpu_buffer_rsrc_t rs, uint32_t off, uint2 v) {
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    const u32x2_t w = {v.x, v.y};
    __builtin_amdgcn_raw_buffer_store_b64(w, rs, int(off), 0, POLICY);
}

__device__ __forceinline__ void load_block(uint4 (&hv)[4], __amdgpu_buffer_rsrc_t rs, uint32_t roff, int kb, int kb1,
                                           int kmax, int kofs) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const bool ok = kb < kb1 && kb * 64 + kofs + 8 * s < kmax;
        const uint32_t off = ok ? roff + uint32_t(kb * 64 + 8 * s) * 2u : kOutOfRange;
        const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, 0);
        hv[s] = make_uint4(v.x, v.y, v.z, v.w);
    }
}

__device__ __forceinline__ void mfma_block(f32x16_t& acc, const bf16_t* wrow, const uint4 (&hv)[4], int kb,
                                           int kofs) {
    Frag<bf16_t> fw[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) fw[s].v = *reinterpret_cast<const uint4*>(wrow + kb * 64 + kofs + 8 * s);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        Frag<bf16_t> fh;
        fh.v = hv[s];
        mfma(acc, fw[s], fh);
    }
}

template <int DEPTH>
__device__ __forceinline__ void contract_rows(f32x16_t& acc, const bf16_t* wrow, __amdgpu_buffer_rsrc_t rs,
                                              uint32_t roff, int kb0, int kb1, int kmax, int kofs) {
    uint4 ring[DEPTH][4];
#pragma unroll
    for (int i = 0; i < DEPTH; ++i) load_block(ring[i], rs, roff, kb0 + i, kb1, kmax, kofs);
    int kb = kb0;
    for (; kb + DEPTH <= kb1; kb += DEPTH) {
#pragma unroll
        for (int i = 0; i < DEPTH; ++i) {
            mfma_block(acc, wrow, ring[i], kb + i, kofs);
            load_block(ring[i], rs, roff, kb + i + DEPTH, kb1, kmax, kofs);
        }
    }
    // remaining blocks (fewer than DEPTH) are already in the ring
#pragma unroll
    for (int i = 0; i < DEPTH; ++i)
        if (kb + i < kb1) mfma_block(acc, wrow, ring[i], kb + i, kofs);
}

// Sum the K parts of the waves that share a batch tile (KW > 1) through
// LDS, in a fixed order; afterwards waves with kw == 0 hold the totals.
template <int KW>
__device__ __forceinline__ void reduce_kparts(f32x16_t& acc, float* red, int wave, int lane) {
    if constexpr (KW > 1) {
        constexpr int NB = kWaves / KW;
        const int kw = wave / NB, bt = wave % NB;
        if (kw > 0) {
            float* dst = red + ((kw - 1) * NB + bt) * 1024 + lane * 16;
#pragma unroll
            for (int v = 0; v < 16; ++v) dst[v] = acc[v];
        }
        __syncthreads();
        if (kw == 0) {
            for (int q = 1; q < KW; ++q) {
                const float* src = red + ((q - 1) * NB + bt) * 1024 + lane * 16;
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[v] += src[v];
            }
        }
    }
}

// acc += Wslice . R^T for one 32-row group R of an operand in fragment
// layout, over n k-groups of 16.  `off` is the byte offset of this lane's
// 16 bytes of the first k-group (k-groups are 1 KB apart); `wrow` is this
// lane's LDS weight row at the first k-group (16 elements per k-group).
// Loads stream through a ring of DEPTH k-groups in flight; two accumulators
// alternate so consecutive MFMAs do not wait on each other.
template <int DEPTH>
__device__ __forceinline__ void contract_frag(f32x16_t& acc, const bf16_t* wrow, __amdgpu_buffer_rsrc_t rs,
                                              uint32_t off, int n) {
    uint4 ring[DEPTH];
    f32x16_t acc1;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc1[v] = 0.f;
#pragma unroll
    for (int i = 0; i < DEPTH; ++i) ring[i] = load16(rs, i < n ? off + uint32_t(i) * 1024u : kOutOfRange);
    int kg = 0;
    for (; kg + DEPTH <= n; kg += DEPTH) {
#pragma unroll
        for (int i = 0; i < DEPTH; ++i) {
            Frag<bf16_t> fw, fh;
            fw.v = *reinterpret_cast<const uint4*>(wrow + (kg + i) * 16);
            fh.v = ring[i];
            if (i & 1) mfma(acc1, fw, fh);
            else mfma(acc, fw, fh);
            const int nx = kg + i + DEPTH;
            ring[i] = load16(rs, nx < n ? off + uint32_t(nx) * 1024u : kOutOfRange);
        }
    }
#pragma unroll
    for (int i = 0; i < DEPTH; ++i) {
        if (kg + i < n) {
            Frag<bf16_t> fw, fh;
            fw.v = *reinterpret_cast<const uint4*>(wrow + (kg + i) * 16);
            fh.v = ring[i];
            if (i & 1) mfma(acc1, fw, fh);
            else mfma(acc, fw, fh);
        }
    }
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] += acc1[v];
}

constexpr int kDepthFrag = 16;

template <int KW>
__global__ __launch_bounds__(kThreads) void lstm_fwd_persistent(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wld = a.Kp + 8;
    bf16_t* Ws = reinterpret_cast<bf16_t*>(smem_raw);
    float* red = reinterpret_cast<float*>(smem_raw + size_t(32) * wld * sizeof(bf16_t));
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int u0 = blockIdx.x * kUnitsFwd;
    constexpr int NB = kWaves / KW;
    const int bt = wave % NB, kw = wave / NB;
    const int nkg = a.Kp / 16;
    const int kg0 = kw * nkg / KW, kg1 = (kw + 1) * nkg / KW;
    const bf16_t* wrow = Ws + (lane & 31) * wld + 8 * (lane >> 5) + kg0 * 16;
    const uint32_t hoff = (uint32_t(bt * nkg + kg0) * 512u + uint32_t(lane) * 8u) * 2u;
    const int H = a.H;
    const int row = bt * 32 + (lane & 31);   // this lane's batch row (sorted order)
    const int ub = u0 + 4 * (lane >> 5);      // its four consecutive units
    const bool owner = kw == 0;               // lanes of these waves own cells
    Barrier bar;
    barrier_init(bar, a.sync);

    stage_fwd_weights(a, Ws, wld, u0);
    // the cell state of the owned cells stays in registers for the launch
    float creg[4] = {0.f, 0.f, 0.f, 0.f};
    if (owner && row < a.B) {
        const float4 c0 = *reinterpret_cast<const float4*>(a.Cs + int64_t(row) * a.ldh + ub);
        creg[0] = c0.x; creg[1] = c0.y; creg[2] = c0.z; creg[3] = c0.w;
    }
    __syncthreads();

    for (int t = 0; t < a.t_eff; ++t) {
        const int act = act_at(a.active, a.fixed, a.B, t, a.t_eff);
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        const int64_t off_t = off_at(a.offsets, a.fixed, a.B, t);
        // operand of the cell update that does not depend on h_{t-1}: load it
        // first (branch-free; lanes without a cell read out of range, i.e. 0)
        const bool cell = owner && row < act;
        const auto rxg = make_rsrc(a.XG + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
        const uint32_t oxg = cell ? (uint32_t(row) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u : kOutOfRange;
        const uint4 xg0 = load16(rxg, oxg), xg1 = load16(rxg, oxg + 16u);
        f32x16_t acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.f;
        if (bt * 32 < act) {
            // h_{t-1} is slot t of the fragment-layout copy
            const auto rs = make_rsrc(a.Hf + int64_t(t) * a.hf_slot, uint32_t(a.hf_slot) * 2u);
            contract_frag<kDepthFrag>(acc, wrow, rs, hoff, kg1 - kg0);
        }
        reduce_kparts<KW>(acc, red, wave, lane);
        if (cell) {
            const uint32_t xw[8] = {xg0.x, xg0.y, xg0.z, xg0.w, xg1.x, xg1.y, xg1.z, xg1.w};
            float hn[4];
            uint32_t gw[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t w0 = xw[2 * q], w1 = xw[2 * q + 1];
                const float ai = acc[4 * q + 0] + bf2f(bf16_t(w0 & 0xffffu));
                const float af = acc[4 * q + 1] + bf2f(bf16_t(w0 >> 16));
                const float ag = acc[4 * q + 2] + bf2f(bf16_t(w1 & 0xffffu));
                const float ao = acc[4 * q + 3] + bf2f(bf16_t(w1 >> 16));
                const float gi = sigmoidf_(ai), gf = sigmoidf_(af), gg = tanhf_(ag), go = sigmoidf_(ao);
                creg[q] = gf * creg[q] + gi * gg;
                hn[q] = go * tanhf_(creg[q]);
                gw[2 * q] = uint32_t(f2bf(gi)) | (uint32_t(f2bf(gf)) << 16);
                gw[2 * q + 1] = uint32_t(f2bf(gg)) | (uint32_t(f2bf(go)) << 16);
            }
            const uint2 hb = make_uint2(uint32_t(f2bf(hn[0])) | (uint32_t(f2bf(hn[1])) << 16),
                                        uint32_t(f2bf(hn[2])) | (uint32_t(f2bf(hn[3])) << 16));
            // h_t for the next step (fragment layout, slot t + 1)
            if (t + 1 < a.t_eff && row < act_next) {
                const auto rhf = make_rsrc(a.Hf + int64_t(t + 1) * a.hf_slot, uint32_t(a.hf_slot) * 2u);
                store8<kStoreThrough>(rhf, uint32_t(frag_index(row, ub, a.Kp)) * 2u, hb);
            }
            const int64_t nrow = int64_t(a.B) + off_t;   // first row of step t in Hs / Cs
            const auto rcs = make_rsrc(a.Cs + nrow * a.ldh, uint32_t(act) * uint32_t(a.ldh) * 4u);
            const auto rhs = make_rsrc(a.Hs + nrow * a.ldh, uint32_t(act) * uint32_t(a.ldh) * 2u);
            const auto rgs = make_rsrc(a.Gs + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
            store16<kStoreThrough>(rcs, (uint32_t(row) * uint32_t(a.ldh) + uint32_t(ub)) * 4u,
                    make_uint4(__float_as_uint(creg[0]), __float_as_uint(creg[1]), __float_as_uint(creg[2]),
                               __float_as_uint(creg[3])));
            store8<kStoreThrough>(rhs, (uint32_t(row) * uint32_t(a.ldh) + uint32_t(ub)) * 2u, hb);
            const uint32_t og = (uint32_t(row) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u;
            store16<kStoreThrough>(rgs, og, make_uint4(gw[0], gw[1], gw[2], gw[3]));
            store16<kStoreThrough>(rgs, og + 16u, make_uint4(gw[4], gw[5], gw[6], gw[7]));
            const int b = a.perm ? a.perm[row] : row;
            if (a.y) {
                const auto ry = make_rsrc(a.y + int64_t(t) * a.B * H, uint32_t(a.B) * uint32_t(H) * 2u);
                store8<kStoreThrough>(ry, (uint32_t(b) * uint32_t(H) + uint32_t(ub)) * 2u, hb);
            }
            if (row >= act_next) {   // last step of this sequence
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (a.hT) a.hT[int64_t(b) * H + ub + q] = hn[q];
                    if (a.cT) a.cT[int64_t(b) * H + ub + q] = creg[q];
                }
            }
        }
        if (t + 1 < a.t_eff) grid_barrier(bar);
    }
}

// ---------------------------------------------------------------- backward
struct BwdArgs {
    int H, B, t_eff, fixed;
    int Ks;                            // interleaved gate columns per K slice (= H)
    int Ksp;                           // Ks rounded up to 64
    const int32_t* active;
    const int32_t* offsets;
    const int32_t* perm;
    const bf16_t* Wh;                  // [4H, H] gate-major
    bf16_t* G;                         // dG store [T*B x ldg] interleaved
    const bf16_t* Gs;                  // saved gates, interleaved
    const float* Cs;
    const bf16_t* dy;                  // gradient of this layer's output or NULL
    int64_t dy_ld;
    const int32_t* dy_rows;            // packed row -> dy row, NULL = identity
    const float* dhT;
    const float* dcT;
    float* dh0;
    float* dc0;
    float* part;                       // [kSlices x B x H]
    int64_t ldh, ldg;
    Sync* sync;
};

// WT[uu][kk] = (Wh interleaved)[s * Ks + kk][v0 + uu] = Wh[(c % 4) * H + c / 4][v0 + uu], c = s * Ks + kk
__device__ __forceinline__ void stage_bwd_weights(const BwdArgs& a, bf16_t* Ws, int wld, int s, int v0) {
    const int H = a.H;
#pragma unroll 8
    for (int idx = threadIdx.x; idx < kUnitsBwd * a.Ksp; idx += kThreads) {
        const int kk = idx / kUnitsBwd, uu = idx - kk * kUnitsBwd;
        const int c = s * a.Ks + kk;
        const int u = v0 + uu;
        bf16_t v = 0;
        if (kk < a.Ks && c < 4 * H && u < H) v = a.Wh[(int64_t(c & 3) * H + (c >> 2)) * H + u];
        Ws[uu * wld + kk] = v;
    }
}

// partial dh for units [v0, v0 + 32) from slice s of dG rows [off, off + rows)
template <int KW>
__device__ __forceinline__ void bwd_contract(const BwdArgs& a, const bf16_t* Ws, int wld, float* red, int s, int v0,
                                             int64_t off, int rows) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int NB = kWaves / KW;
    const int bt = wave % NB, kw = wave / NB;
    const int nkb = a.Ksp / 64;
    const int kb0 = kw * nkb / KW, kb1 = (kw + 1) * nkb / KW;
    const int kofs = (lane >> 5) * 32;
    const int row = bt * 32 + (lane & 31);
    f32x16_t acc;
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
    if (bt * 32 < rows) {
        const auto rs = make_rsrc(a.G + off * a.ldg, uint32_t(rows) * uint32_t(a.ldg) * 2u);
        const uint32_t roff = (uint32_t(row) * uint32_t(a.ldg) + uint32_t(s) * uint32_t(a.Ks) + uint32_t(kofs)) * 2u;
        contract_rows<kDepthBwd>(acc, Ws + (lane & 31) * wld, rs, roff, kb0, kb1, a.Ks, kofs);
    }
    reduce_kparts<KW>(acc, red, wave, lane);
    if (kw == 0 && row < rows) {
        // the partial-sum buffer is rewritten every step: write through
        const auto rp = make_rsrc(a.part + int64_t(s) * a.B * a.H, uint32_t(a.B) * uint32_t(a.H) * 4u);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int u = v0 + acc_row(v, lane);
            const uint32_t o = u < a.H ? (uint32_t(row) * uint32_t(a.H) + uint32_t(u)) * 4u : kOutOfRange;
            store4<kStoreThrough>(rp, o, acc[v]);
        }
    }
}

template <int KW>
__global__ __launch_bounds__(kThreads) void lstm_bwd_persistent(BwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wld = a.Ksp + 8;
    bf16_t* Ws = reinterpret_cast<bf16_t*>(smem_raw);
    float* red = reinterpret_cast<float*>(smem_raw + size_t(kUnitsBwd) * wld * sizeof(bf16_t));
    const int tid = threadIdx.x;
    const int q = blockIdx.x;
    const int s = q % kSlices, v0 = (q / kSlices) * kUnitsBwd;
    const int H = a.H;
    Barrier bar;
    barrier_init(bar, a.sync);

    stage_bwd_weights(a, Ws, wld, s, v0);

    // cells owned for the pointwise part: units [8q, 8q + 8) x rows
    float dhp[kCellsPerThread], dcr[kCellsPerThread];
#pragma unroll
    for (int k = 0; k < kCellsPerThread; ++k) {
        const int idx = tid + k * kThreads;
        const int r = idx >> 3, u = q * 8 + (idx & 7);
        dhp[k] = 0.f;
        dcr[k] = 0.f;
        if (r < a.B && u < H) {
            const int b = a.perm ? a.perm[r] : r;
            if (a.dhT) dhp[k] = a.dhT[int64_t(b) * H + u];
            if (a.dcT) dcr[k] = a.dcT[int64_t(b) * H + u];
        }
    }
    __syncthreads();

    for (int t = a.t_eff - 1; t >= -1; --t) {
        const int act = t >= 0 ? act_at(a.active, a.fixed, a.B, t, a.t_eff) : a.B;
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        // partial sums of dh_t from dG_{t+1}
        if (act_next > 0) {
            bwd_contract<KW>(a, Ws, wld, red, s, v0, off_at(a.offsets, a.fixed, a.B, t + 1), act_next);
            grid_barrier(bar);
        }
        const int64_t off_t = t >= 0 ? off_at(a.offsets, a.fixed, a.B, t) : 0;
        const int64_t prev_base = t <= 0 ? 0 : int64_t(a.B) + off_at(a.offsets, a.fixed, a.B, t - 1);
#pragma unroll
        for (int k = 0; k < kCellsPerThread; ++k) {
            const int idx = tid + k * kThreads;
            const int r = idx >> 3, u = q * 8 + (idx & 7);
            if (r >= act || u >= H) continue;
            float dhv = dhp[k];
            if (r < act_next) {
                // reused every step: read past the caches, sum in slice order
                const auto rp = make_rsrc(a.part, uint32_t(kSlices) * uint32_t(a.B) * uint32_t(H) * 4u);
                dhv = 0.f;
#pragma unroll
                for (int j = 0; j < kSlices; ++j)
                    dhv += load4_bypass(rp, ((uint32_t(j) * uint32_t(a.B) + uint32_t(r)) * uint32_t(H) + uint32_t(u)) * 4u);
            }
            if (t < 0) {
                const int b = a.perm ? a.perm[r] : r;
                if (a.dh0) a.dh0[int64_t(b) * H + u] = dhv;
                if (a.dc0) a.dc0[int64_t(b) * H + u] = dcr[k];
                continue;
            }
            const int64_t p = off_t + r;
            if (a.dy) {
                const int64_t yr = a.dy_rows ? int64_t(a.dy_rows[p]) : p;
                dhv += bf2f(a.dy[yr * a.dy_ld + u]);
            }
            const uint2 gv = *reinterpret_cast<const uint2*>(a.Gs + p * a.ldg + 4 * u);
            const float gi = bf2f(bf16_t(gv.x & 0xffffu)), gf = bf2f(bf16_t(gv.x >> 16));
            const float gg = bf2f(bf16_t(gv.y & 0xffffu)), go = bf2f(bf16_t(gv.y >> 16));
            const float c = a.Cs[(a.B + p) * a.ldh + u];
            const float cp = a.Cs[(prev_base + r) * a.ldh + u];
            const float tau = tanhf_(c);
            const float d_o = dhv * tau;
            const float dct = dcr[k] + dhv * go * (1.f - tau * tau);
            dcr[k] = dct * gf;
            uint2 dg;
            dg.x = uint32_t(f2bf(dct * gg * gi * (1.f - gi))) | (uint32_t(f2bf(dct * cp * gf * (1.f - gf))) << 16);
            dg.y = uint32_t(f2bf(dct * gi * (1.f - gg * gg))) | (uint32_t(f2bf(d_o * go * (1.f - go))) << 16);
            const auto rg = make_rsrc(a.G + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
            store8<kStoreThrough>(rg, (uint32_t(r) * uint32_t(a.ldg) + 4u * uint32_t(u)) * 2u, dg);
        }
        if (t >= 0 && act > 0) grid_barrier(bar);
    }
}

}  // namespace persist
}  // namespace janus
