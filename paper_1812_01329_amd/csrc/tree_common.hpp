// Shared pieces of the persistent tree level programs (binary TreeLSTM,
// TreeRNN, Child-Sum TreeLSTM): the workgroup shape, the counter block of the
// device-wide barrier, staging helpers that keep many loads in flight, the
// 32 x 32 fp32 MFMA contraction over nodes, and the host-side launch of a
// grid whose workgroups must all be resident.
#pragma once

#include <mutex>

#include "device.hpp"
#include "lstm_persist.hpp"
#include "runtime.hpp"

namespace janus {
namespace tpersist {

constexpr int kThreads = 256;          // 4 waves
constexpr int kWaves = kThreads / 64;
constexpr int kUG = 6;                 // units per forward group: 5 x 6 = 30 of 32 tile columns
constexpr int kUC = 32;                // units per chunk of the backward's cell recompute
constexpr int kKC = 128;               // k per staged chunk of the contractions over nodes
constexpr int kRed = 33;               // row pitch of the per-wave partial tiles
constexpr int kMaxE = 2 * kThreads;    // input width the embedding-gradient phase handles

__host__ __device__ constexpr int pad16(int x) { return (x + 15) & ~15; }
__host__ __device__ constexpr int padto(int x, int m) { return (x + m - 1) / m * m; }

// Counter block of the grid barrier.  `error` comes first: the backward's
// upload zeroes the counters that follow it and leaves a flag the forward
// set.
struct TreeSync {
    unsigned error;
    unsigned pad_e[63];
    unsigned count;
    unsigned pad0[63];
    unsigned xcd[16][64];
    unsigned census[16][64];
};
constexpr size_t kTreeSyncCounters = offsetof(TreeSync, count);   // byte offset of the counters

using TreeBarrier = persist::BarrierT<TreeSync>;

// The census of the workgroups on each XCD (which the grid barrier's waits
// need), in two halves so that a kernel stages its weight slices while the
// other workgroups arrive: tree_census_arrive counts this workgroup on its
// XCD and in the total (thread 0, without waiting for the replies);
// tree_census_wait waits until every workgroup has counted itself, then
// lane q < 16 of wave 0 reads XCD q's count, all in one round trip.  The
// fields the level barrier uses (x in thread 0, xcount in lanes 0-15) are
// then set as the one-call census sets them.
__device__ __forceinline__ void tree_census_arrive(TreeBarrier& b, TreeSync* s) {
    b.s = s;
    b.nb = gridDim.x;
    b.phase = 0;
    b.x = 0;
    b.xsize = 1;
    b.nx = 1;
    b.xidx = 0;
    b.xfirst = 0;
    b.xcount = 0;
    if (threadIdx.x == 0) {
        b.x = persist::xcc_id();
        __hip_atomic_fetch_add(&s->census[b.x][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&s->count, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
}
__device__ __forceinline__ void tree_census_wait(TreeBarrier& b) {
    if (threadIdx.x < 64) {
        if (threadIdx.x == 0) persist::spin_until(b.s, &b.s->count, b.nb);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        if (threadIdx.x < 16)
            b.xcount = __hip_atomic_load(&b.s->census[threadIdx.x][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
}

// A store other workgroups read later in the launch: device-scope, so it is
// written through the L2 of this XCD to memory (the L2s of the XCDs are not
// coherent with each other), and counted like any store by the wait at the
// barrier's arrival.
__device__ __forceinline__ void store_through(float* base, int64_t idx, float v) {
    __hip_atomic_store(base + idx, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void zero_acc(f32x16_t& acc) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[v] = 0.f;
}

// Sum the four waves' 32 x 32 tiles: every wave writes its accumulator to
// red[wave][row][col]; after the barrier red holds the parts, summed by the
// reader in wave order.
__device__ __forceinline__ void spill_acc(const f32x16_t& acc, float* red, int wave, int lane) {
#pragma unroll
    for (int v = 0; v < 16; ++v) red[(wave * 32 + acc_row(v, lane)) * kRed + acc_col(lane)] = acc[v];
}
__device__ __forceinline__ float red_sum(const float* red, int m, int c) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += red[(w * 32 + m) * kRed + c];
    return s;
}

// Copy n elements into LDS: element i is ld(i) (which returns 0 outside its
// operand) and goes where st(i, v) puts it.  Each thread issues NB loads
// before it writes any, so it pays one memory round trip per NB elements
// rather than one per element.
template <int NB, class Ld, class St>
__device__ __forceinline__ void stage(int n, Ld ld, St st) {
    for (int base = int(threadIdx.x); base < n; base += kThreads * NB) {
        float v[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int idx = base + i * kThreads;
            v[i] = idx < n ? ld(idx) : 0.f;
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int idx = base + i * kThreads;
            if (idx < n) st(idx, v[i]);
        }
    }
}
// The same with 16-byte pieces (ld4 returns a float4).
template <int NB, class Ld, class St>
__device__ __forceinline__ void stage4(int n, Ld ld, St st) {
    for (int base = int(threadIdx.x); base < n; base += kThreads * NB) {
        float4 v[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int idx = base + i * kThreads;
            v[i] = idx < n ? ld(idx) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int idx = base + i * kThreads;
            if (idx < n) st(idx, v[i]);
        }
    }
}
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Copy an nrow x KQ grid of 16-byte pieces into LDS: piece (m, q) is
// ld(m, q) (0 outside its operand) and goes where st(m, q, v) puts it.
// Thread t takes pieces t, t + kThreads, ... in row-major order, stepping
// (m, q) without a division, and issues NB loads before it writes any.
template <int NB, class Ld, class St>
__device__ __forceinline__ void stage4_2d(int nrow, int KQ, Ld ld, St st) {
    const int dm = kThreads / KQ, dq = kThreads - dm * KQ;
    int m = int(threadIdx.x) / KQ, q = int(threadIdx.x) - m * KQ;
    while (m < nrow) {
        float4 v[NB];
        int mm[NB], qq[NB];
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            mm[i] = m;
            qq[i] = q;
            v[i] = m < nrow ? ld(m, q) : make_float4(0.f, 0.f, 0.f, 0.f);
            q += dq;
            m += dm;
            if (q >= KQ) {
                q -= KQ;
                ++m;
            }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i)
            if (mm[i] < nrow) st(mm[i], qq[i], v[i]);
    }
}


// acc += sum over k in [0, K) of Aop(row, k) Bop(col, k) for a 32 x 32 tile,
// staged kKC k at a time through LDS (A and B chunks [32][kKC + 4]); the
// waves take its k-steps of 16 in turn, and the next chunk is loaded into
// registers while the current one is contracted.  fa(r, k) / fb(c, k)
// return the operand value (0 outside).  AK: A is contiguous in k in memory
// (consecutive threads then take consecutive k), else in r (consecutive
// threads take consecutive rows of one k); B is always contiguous in c.
template <bool AK, class FA, class FB>
__device__ __forceinline__ void node_contraction(f32x16_t& acc, float* Ac, float* Bc, int K, FA fa, FB fb) {
    constexpr int sK = kKC + 4, PER = 32 * kKC / kThreads;   // 8 elements of each operand per thread
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float va[PER], vb[PER];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx / 32, r = idx % 32;
            vb[i] = k0 + kk < K ? fb(r, k0 + kk) : 0.f;
            if constexpr (AK) {
                const int ra = idx / kKC, ka = idx % kKC;
                va[i] = k0 + ka < K ? fa(ra, k0 + ka) : 0.f;
            } else {
                va[i] = k0 + kk < K ? fa(r, k0 + kk) : 0.f;
            }
        }
    };
    if (K > 0) fetch(0);
    for (int k0 = 0; k0 < K; k0 += kKC) {
        __syncthreads();   // the previous chunk's reads are done
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx / 32, r = idx % 32;
            Bc[r * sK + kk] = vb[i];
            if constexpr (AK) Ac[(idx / kKC) * sK + idx % kKC] = va[i];
            else Ac[r * sK + kk] = va[i];
        }
        if (k0 + kKC < K) fetch(k0 + kKC);
        __syncthreads();
        for (int ks = wave; ks < kKC / 16; ks += kWaves) {
            Frag<float> xa, xb;
            xa.load(Ac + (lane & 31) * sK + ks * 16 + 8 * (lane >> 5));
            xb.load(Bc + (lane & 31) * sK + ks * 16 + 8 * (lane >> 5));
            mfma(acc, xa, xb);
        }
    }
}

// The same with 16-byte pieces, for operands whose rows are 16-byte aligned
// and padded so that four elements read from a valid start never leave the
// row: fa4(i, k) returns A[i][k .. k + 3] (AK) or A[i .. i + 3][k], and
// fb4(j, k) returns B[j .. j + 3][k], as loaded.  nA and nB count the valid
// rows of A and columns of B in this tile; the elements past them (and past
// K) are zeroed when the chunk is written to LDS, after the chunk's loads
// are all issued.  A thread then issues 8 loads per chunk instead of 32.
// KC is the chunk depth (Ac and Bc hold 32 rows of pitch KC + 4).
template <bool AK, int KC = kKC, class FA, class FB>
__device__ __forceinline__ void node_contraction4(f32x16_t& acc, float* Ac, float* Bc, int K, int nA, int nB,
                                                  FA fa4, FB fb4) {
    constexpr int sK = KC + 4, PER = 32 * KC / 4 / kThreads;   // pieces of each operand per thread
    constexpr int CQ = KC / 4;                                  // 16-byte pieces per row of a chunk
    static_assert(PER * kThreads * 4 == 32 * KC, "a chunk is whole passes of the workgroup");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float4 va[PER], vb[PER];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx >> 3, c4 = 4 * (idx & 7);
            vb[i] = (k0 + kk < K && c4 < nB) ? fb4(c4, k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
            if constexpr (AK) {
                const int r = idx / CQ, k4 = 4 * (idx % CQ);
                va[i] = (k0 + k4 < K && r < nA) ? fa4(r, k0 + k4) : make_float4(0.f, 0.f, 0.f, 0.f);
            } else {
                va[i] = (k0 + kk < K && c4 < nA) ? fa4(c4, k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    };
    // keep the first n elements of a piece
    auto keep = [](float4 v, int n) {
        if (n < 4) v.w = 0.f;
        if (n < 3) v.z = 0.f;
        if (n < 2) v.y = 0.f;
        return v;
    };
    if (K > 0) fetch(0);
    for (int k0 = 0; k0 < K; k0 += KC) {
        __syncthreads();   // the previous chunk's reads are done
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx >> 3, c4 = 4 * (idx & 7);
            const float4 b = keep(vb[i], nB - c4);
            Bc[(c4 + 0) * sK + kk] = b.x;
            Bc[(c4 + 1) * sK + kk] = b.y;
            Bc[(c4 + 2) * sK + kk] = b.z;
            Bc[(c4 + 3) * sK + kk] = b.w;
            if constexpr (AK) {
                const int r = idx / CQ, k4 = 4 * (idx % CQ);
                *reinterpret_cast<float4*>(Ac + r * sK + k4) = keep(va[i], K - (k0 + k4));
            } else {
                const float4 v = keep(va[i], nA - c4);
                Ac[(c4 + 0) * sK + kk] = v.x;
                Ac[(c4 + 1) * sK + kk] = v.y;
                Ac[(c4 + 2) * sK + kk] = v.z;
                Ac[(c4 + 3) * sK + kk] = v.w;
            }
        }
        if (k0 + KC < K) fetch(k0 + KC);
        __syncthreads();
        for (int ks = wave; ks < KC / 16; ks += kWaves) {
            Frag<float> xa, xb;
            xa.load(Ac + (lane & 31) * sK + ks * 16 + 8 * (lane >> 5));
            xb.load(Bc + (lane & 31) * sK + ks * 16 + 8 * (lane >> 5));
            mfma(acc, xa, xb);
        }
    }
}


// A 64 x 64 tile of the same sum, for operands in 16-byte pieces (the
// conventions of node_contraction4; nA and nB count the valid rows of A and
// columns of B, up to 64).  Chunks of KC k pass through LDS (A and B chunks
// [64][KC + 4]) with the next chunk loaded into registers meanwhile.  Wave w
// contracts the whole chunk for the 32 x 32 quadrant at rows 32 (w / 2) and
// columns 32 (w % 2) of the tile, so acc needs no sum over the waves, and a
// chunk's MFMA work (about as long as a load round trip) hides the next
// chunk's loads.  Against four 32 x 32 tiles, the operands are read from
// memory half as often.
template <bool AK, int KC, class FA, class FB>
__device__ __forceinline__ void node_contraction64(f32x16_t& acc, float* Ac, float* Bc, int K, int nA, int nB,
                                                   FA fa4, FB fb4) {
    constexpr int sK = KC + 4, PER = 64 * KC / 4 / kThreads;   // pieces of each operand per thread and chunk
    constexpr int CQ = KC / 4;                                  // 16-byte pieces per row of a chunk
    static_assert(PER * kThreads * 4 == 64 * KC, "a chunk is whole passes of the workgroup");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float4 va[PER], vb[PER];
    auto fetch = [&](int k0) {
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx >> 4, c4 = 4 * (idx & 15);
            vb[i] = (k0 + kk < K && c4 < nB) ? fb4(c4, k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
            if constexpr (AK) {
                const int r = idx / CQ, k4 = 4 * (idx % CQ);
                va[i] = (k0 + k4 < K && r < nA) ? fa4(r, k0 + k4) : make_float4(0.f, 0.f, 0.f, 0.f);
            } else {
                va[i] = (k0 + kk < K && c4 < nA) ? fa4(c4, k0 + kk) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    };
    auto keep = [](float4 v, int n) {
        if (n < 4) v.w = 0.f;
        if (n < 3) v.z = 0.f;
        if (n < 2) v.y = 0.f;
        return v;
    };
    const float* ar = Ac + (32 * (wave >> 1) + (lane & 31)) * sK + 8 * (lane >> 5);
    const float* br = Bc + (32 * (wave & 1) + (lane & 31)) * sK + 8 * (lane >> 5);
    if (K > 0) fetch(0);
    for (int k0 = 0; k0 < K; k0 += KC) {
        __syncthreads();   // the previous chunk's reads are done
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            const int idx = tid + i * kThreads;
            const int kk = idx >> 4, c4 = 4 * (idx & 15);
            const float4 b = keep(vb[i], nB - c4);
            Bc[(c4 + 0) * sK + kk] = b.x;
            Bc[(c4 + 1) * sK + kk] = b.y;
            Bc[(c4 + 2) * sK + kk] = b.z;
            Bc[(c4 + 3) * sK + kk] = b.w;
            if constexpr (AK) {
                const int r = idx / CQ, k4 = 4 * (idx % CQ);
                *reinterpret_cast<float4*>(Ac + r * sK + k4) = keep(va[i], K - (k0 + k4));
            } else {
                const float4 v = keep(va[i], nA - c4);
                Ac[(c4 + 0) * sK + kk] = v.x;
                Ac[(c4 + 1) * sK + kk] = v.y;
                Ac[(c4 + 2) * sK + kk] = v.z;
                Ac[(c4 + 3) * sK + kk] = v.w;
            }
        }
        if (k0 + KC < K) fetch(k0 + KC);
        __syncthreads();
        const int nks = (K - k0 < KC ? K - k0 + 15 : KC) / 16;   // k-steps of 16 holding data
        for (int ks = 0; ks < nks; ++ks) {
            Frag<float> xa, xb;
            xa.load(ar + ks * 16);
            xb.load(br + ks * 16);
            mfma(acc, xa, xb);
        }
    }
}

// Stage 32 weight rows 32 col + c (c < 32) of a [rows x K] matrix into LDS
// rows of pitch ld, zero past K and past the last row.
__device__ __forceinline__ void stage_weight_rows(float* dst, int ld, const float* src, int nrows, int K, int col) {
    const int KP = pad16(K);
    if (K % 4 == 0) {
        stage4_2d<10>(32, KP / 4,
                      [&](int c, int q) {
                          const int n = 32 * col + c, k = 4 * q;
                          return (n < nrows && k < K) ? ld4(src + int64_t(n) * K + k) : make_float4(0.f, 0.f, 0.f, 0.f);
                      },
                      [&](int c, int q, float4 v) { *reinterpret_cast<float4*>(dst + c * ld + 4 * q) = v; });
    } else {
        stage<16>(32 * KP,
                  [&](int idx) {
                      const int c = idx / KP, k = idx - c * KP, n = 32 * col + c;
                      return (n < nrows && k < K) ? src[int64_t(n) * K + k] : 0.f;
                  },
                  [&](int idx, float v) { dst[(idx / KP) * ld + idx % KP] = v; });
    }
}

// Stage the rows rowsrc[m] (element offsets into src, -1 = zero row) of K
// columns into At (pitch ld), zero up to pad16(K).  K % 4 == 0 (16-byte
// aligned rows): thread t owns the 16-byte column q = t mod KQ of the rows
// t / KQ, t / KQ + RP, ... (RP = kThreads / KQ rows per pass), reads those
// rows' offsets, then issues all its loads before it writes any.
__device__ __forceinline__ void stage_tile_rows(float* At, int ld, const float* src, const int64_t* rowsrc, int K) {
    const int KP = pad16(K);
    if (K % 4 == 0 && KP / 4 <= kThreads) {
        constexpr int NB = 16;
        const int KQ = KP / 4, RP = kThreads / KQ;
        const int q = int(threadIdx.x) % KQ, m0 = int(threadIdx.x) / KQ;
        if (m0 >= RP) return;
        const bool colok = 4 * q < K;
        for (int mb = m0; mb < 32; mb += RP * NB) {
            int64_t r[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const int m = mb + i * RP;
                r[i] = (m < 32 && colok) ? rowsrc[m] : -1;
            }
            float4 v[NB];
#pragma unroll
            for (int i = 0; i < NB; ++i) v[i] = r[i] >= 0 ? ld4(src + r[i] + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int i = 0; i < NB; ++i) {
                const int m = mb + i * RP;
                if (m < 32) *reinterpret_cast<float4*>(At + m * ld + 4 * q) = v[i];
            }
        }
    } else {
        stage<16>(32 * KP,
                  [&](int idx) {
                      const int m = idx / KP, k = idx - m * KP;
                      const int64_t r = rowsrc[m];
                      return (r >= 0 && k < K) ? src[r + k] : 0.f;
                  },
                  [&](int idx, float v) { At[(idx / KP) * ld + idx % KP] = v; });
    }
}

// acc = the tile's rows At [32 x KP] times the weight slice Wl [32 x KP]
// (transposed), k-steps of 16 dealt to the waves in turn.
__device__ __forceinline__ void tile_mfma(f32x16_t& acc, const float* At, int lda, const float* Wl, int ldw, int KP,
                                          int wave, int lane) {
    zero_acc(acc);
    for (int ks = wave; ks < KP / 16; ks += kWaves) {
        Frag<float> fa, fb;
        fa.load(At + (lane & 31) * lda + ks * 16 + 8 * (lane >> 5));
        fb.load(Wl + (lane & 31) * ldw + ks * 16 + 8 * (lane >> 5));
        mfma(acc, fa, fb);
    }
}

// The same for a 16-row tile, as 16x16x4 products: D[16 x 32] (two 16 x 16
// blocks, columns 16 b + .) = A[16 x KP] B[32 x KP]^T, KP a multiple of 16.
// The 32-column k groups are dealt to the waves in turn; step jj of lane l
// takes column 32 g + 8 (l / 16) + jj of both operands, so eight steps cover
// the group once and each lane reads 8 consecutive floats per operand.  When
// KP is 16 past a multiple of 32, the last group's upper two lane quarters
// take zeros (their columns lie past the rows' end).
__device__ __forceinline__ void tile_mfma16(f32x4_t (&acc)[2], const float* A, int lda, const float* B, int ldb,
                                            int KP, int wave, int lane) {
    acc[0] = acc[1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    auto group = [&](int g, bool tail) {
        const int k = 32 * g + 8 * (lane >> 4);
        const bool ok = !tail || k < KP;
        const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
        const float* ap = A + (lane & 15) * lda + k;
        const float* bp = B + (lane & 15) * ldb + k;
        const float4 a0 = ok ? *reinterpret_cast<const float4*>(ap) : z;
        const float4 a1 = ok ? *reinterpret_cast<const float4*>(ap + 4) : z;
        const float4 b0 = ok ? *reinterpret_cast<const float4*>(bp) : z;
        const float4 b1 = ok ? *reinterpret_cast<const float4*>(bp + 4) : z;
        const float4 c0 = ok ? *reinterpret_cast<const float4*>(bp + 16 * ldb) : z;
        const float4 c1 = ok ? *reinterpret_cast<const float4*>(bp + 16 * ldb + 4) : z;
        const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
        const float bv[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
        const float cv[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) {
            acc[0] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[jj], bv[jj], acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[jj], cv[jj], acc[1], 0, 0, 0);
        }
    };
    const int nfull = KP / 32;
    for (int g = wave; g < nfull; g += kWaves) group(g, false);
    if (KP % 32 != 0 && nfull % kWaves == wave) group(nfull, true);
}
// element v of acc[b] of lane l sits at row 4 (l / 16) + v, column 16 b + l % 16
__device__ __forceinline__ void spill_acc16(const f32x4_t (&acc)[2], float* red, int wave, int lane) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int v = 0; v < 4; ++v) red[(wave * 32 + 4 * (lane >> 4) + v) * kRed + 16 * b + (lane & 15)] = acc[b][v];
}

// ------------------------------------------------------------ host side
constexpr int kMaxTreeGrid = 4096;   // workgroups of a persistent tree launch (the leaf groups' tail is sized for it)

struct TreeDev {
    int cus = 0;
    size_t lds = 0;
};
// Properties of the current device, queried once per device under a lock.
inline TreeDev tree_dev() {
    static std::mutex m;
    static TreeDev cache[64];
    static bool have[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return TreeDev{};
    std::lock_guard<std::mutex> lock(m);
    if (!have[dev]) {
        TreeDev t;
        int v = 0;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess) t.cus = v;
        if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) == hipSuccess) t.lds = size_t(v);
        (void)hipGetLastError();
        cache[dev] = t;
        have[dev] = true;
    }
    return cache[dev];
}

// An ordinary launch of a grid whose workgroups must all be resident (the
// plan allows one per CU and no more than the CUs; the occupancy query
// confirms one fits a CU).  The barrier's waits are bounded.
template <class K, class A>
inline janus_status tree_persistent_launch(K kernel, int blocks, size_t smem, const A& args, hipStream_t st,
                                    size_t& attr_smem) {
    static std::mutex m;
    {
        std::lock_guard<std::mutex> lock(m);
        if (smem > attr_smem) {
            JANUS_HIP(hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                          hipFuncAttributeMaxDynamicSharedMemorySize, int(smem)));
            attr_smem = smem;
        }
    }
    int per_cu = 0;
    JANUS_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel),
                                                           kThreads, smem));
    if (per_cu < 1 || int64_t(per_cu) * tree_dev().cus < blocks) return JANUS_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kThreads), smem, st, args);
    JANUS_LAUNCH_CHECK();
    return JANUS_OK;
}

}  // namespace tpersist
}  // namespace janus
