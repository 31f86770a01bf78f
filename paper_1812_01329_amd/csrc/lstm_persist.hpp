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

struct Sync {
    unsigned count;                    // arrivals, monotonically increasing within a launch
    unsigned error;                    // set when a wait exceeds its spin limit
};

// Device-wide barrier for a cooperative launch of `nblocks` workgroups.
// `phase` counts barriers passed so far; after a timeout every later wait
// returns at once so that all waves still reach the end of the kernel.
__device__ __forceinline__ void grid_barrier(Sync* s, unsigned nblocks, unsigned& phase) {
    ++phase;
    __syncthreads();
    if (threadIdx.x == 0) {
        __threadfence();
        __hip_atomic_fetch_add(&s->count, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        const unsigned target = phase * nblocks;
        int spins = 0;
        while (__hip_atomic_load(&s->count, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
            if (__hip_atomic_load(&s->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) break;
            __builtin_amdgcn_s_sleep(1);
            if (++spins > kSpinLimit) {
                __hip_atomic_store(&s->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
        __threadfence();
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
    Sync* sync;
};

// Schedule values are the same for every lane; readfirstlane keeps them in
// scalar registers so that buffer descriptors built from them stay uniform.
__device__ __forceinline__ int act_at(const int32_t* active, int fixed, int B, int t, int t_eff) {
    if (t >= t_eff || t < 0) return 0;
    return fixed ? B : __builtin_amdgcn_readfirstlane(active[t]);
}
__device__ __forceinline__ int64_t off_at(const int32_t* offsets, int fixed, int B, int t) {
    return fixed ? int64_t(t) * B : int64_t(__builtin_amdgcn_readfirstlane(offsets[t]));
}

// Load rows of a gate-interleaved slice of W into LDS: LDS row i (0..31)
// holds W row `row_of(i)` (or zeros), k contiguous, padded pitch `wld`.
__device__ __forceinline__ void stage_fwd_weights(const FwdArgs& a, bf16_t* Ws, int wld, int u0) {
    const int chunks = a.Kp / 8;
    for (int idx = threadIdx.x; idx < 32 * chunks; idx += kThreads) {
        const int i = idx / chunks, kc = (idx - i * chunks) * 8;
        const int u = u0 + (i >> 2), g = i & 3;
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
// stream through a ring of kDepth k-blocks kept in flight, so the memory
// latency is paid once per step and each MFMA waits only for its own block.
constexpr int kDepth = 8;
constexpr uint32_t kOutOfRange = 0x80000000u;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, int(bytes), 0x00020000);
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

__device__ __forceinline__ void contract_rows(f32x16_t& acc, const bf16_t* wrow, __amdgpu_buffer_rsrc_t rs,
                                              uint32_t roff, int kb0, int kb1, int kmax, int kofs) {
    uint4 ring[kDepth][4];
#pragma unroll
    for (int i = 0; i < kDepth; ++i) load_block(ring[i], rs, roff, kb0 + i, kb1, kmax, kofs);
    int kb = kb0;
    for (; kb + kDepth <= kb1; kb += kDepth) {
#pragma unroll
        for (int i = 0; i < kDepth; ++i) {
            mfma_block(acc, wrow, ring[i], kb + i, kofs);
            load_block(ring[i], rs, roff, kb + i + kDepth, kb1, kmax, kofs);
        }
    }
    // remaining blocks (fewer than kDepth) are already in the ring
#pragma unroll
    for (int i = 0; i < kDepth; ++i)
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

template <int KW>
__global__ __launch_bounds__(kThreads) void lstm_fwd_persistent(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wld = a.Kp + 8;
    bf16_t* Ws = reinterpret_cast<bf16_t*>(smem_raw);
    float* red = reinterpret_cast<float*>(smem_raw + size_t(32) * wld * sizeof(bf16_t));
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int u0 = blockIdx.x * kUnitsFwd;
    constexpr int NB = kWaves / KW;
    const int bt = wave % NB, kw = wave / NB;
    const int nkb = a.Kp / 64;
    const int kb0 = kw * nkb / KW, kb1 = (kw + 1) * nkb / KW;
    const int kofs = (lane >> 5) * 32;
    const bf16_t* wrow = Ws + (lane & 31) * wld;
    const int H = a.H;
    unsigned phase = 0;

    stage_fwd_weights(a, Ws, wld, u0);
    __syncthreads();

    for (int t = 0; t < a.t_eff; ++t) {
        const int act = act_at(a.active, a.fixed, a.B, t, a.t_eff);
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        const int64_t off_t = off_at(a.offsets, a.fixed, a.B, t);
        const int64_t prev_base = t == 0 ? 0 : int64_t(a.B) + off_at(a.offsets, a.fixed, a.B, t - 1);
        const int row = bt * 32 + (lane & 31);
        // operands of the cell update do not depend on h_{t-1}: load them first
        const bool cell = kw == 0 && row < act;
        const int64_t p = off_t + row;
        uint2 xg[4];
        float cprev[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int u = u0 + 2 * q + (lane >> 5);
            xg[q] = make_uint2(0, 0);
            cprev[q] = 0.f;
            if (cell && u < H) {
                xg[q] = *reinterpret_cast<const uint2*>(a.XG + p * a.ldg + 4 * u);
                cprev[q] = a.Cs[(prev_base + row) * a.ldh + u];
            }
        }
        f32x16_t acc;
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[v] = 0.f;
        if (bt * 32 < act) {
            // rows [0, act) of h_{t-1} start at Hs row prev_base
            const auto rs = make_rsrc(a.Hs + prev_base * a.ldh, uint32_t(act) * uint32_t(a.ldh) * 2u);
            contract_rows(acc, wrow, rs, (uint32_t(row) * uint32_t(a.ldh) + uint32_t(kofs)) * 2u, kb0, kb1, H, kofs);
        }
        reduce_kparts<KW>(acc, red, wave, lane);
        if (cell) {
            const int b = a.perm ? a.perm[row] : row;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int u = u0 + 2 * q + (lane >> 5);
                if (u >= H) continue;
                const float ai = acc[4 * q + 0] + bf2f(bf16_t(xg[q].x & 0xffffu));
                const float af = acc[4 * q + 1] + bf2f(bf16_t(xg[q].x >> 16));
                const float ag = acc[4 * q + 2] + bf2f(bf16_t(xg[q].y & 0xffffu));
                const float ao = acc[4 * q + 3] + bf2f(bf16_t(xg[q].y >> 16));
                const float gi = sigmoidf_(ai), gf = sigmoidf_(af), gg = tanhf_(ag), go = sigmoidf_(ao);
                const float cp = cprev[q];
                const float c = gf * cp + gi * gg;
                const float h = go * tanhf_(c);
                a.Cs[(a.B + p) * a.ldh + u] = c;
                const bf16_t hb = f2bf(h);
                a.Hs[(a.B + p) * a.ldh + u] = hb;
                uint2 gs;
                gs.x = uint32_t(f2bf(gi)) | (uint32_t(f2bf(gf)) << 16);
                gs.y = uint32_t(f2bf(gg)) | (uint32_t(f2bf(go)) << 16);
                *reinterpret_cast<uint2*>(a.Gs + p * a.ldg + 4 * u) = gs;
                if (a.y) a.y[(int64_t(t) * a.B + b) * H + u] = hb;
                if (row >= act_next) {
                    if (a.hT) a.hT[int64_t(b) * H + u] = h;
                    if (a.cT) a.cT[int64_t(b) * H + u] = c;
                }
            }
        }
        if (t + 1 < a.t_eff) grid_barrier(a.sync, gridDim.x, phase);
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
        contract_rows(acc, Ws + (lane & 31) * wld, rs, roff, kb0, kb1, a.Ks, kofs);
    }
    reduce_kparts<KW>(acc, red, wave, lane);
    if (kw == 0 && row < rows) {
        float* dst = a.part + (int64_t(s) * a.B + row) * a.H;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int u = v0 + acc_row(v, lane);
            if (u < a.H) dst[u] = acc[v];
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
    unsigned phase = 0;

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
            grid_barrier(a.sync, gridDim.x, phase);
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
                dhv = 0.f;
#pragma unroll
                for (int j = 0; j < kSlices; ++j) dhv += a.part[(int64_t(j) * a.B + r) * H + u];
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
            *reinterpret_cast<uint2*>(a.G + p * a.ldg + 4 * u) = dg;
        }
        if (t >= 0 && act > 0) grid_barrier(a.sync, gridDim.x, phase);
    }
}

}  // namespace persist
}  // namespace janus
