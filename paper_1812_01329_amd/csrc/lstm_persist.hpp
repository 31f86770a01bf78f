// Persistent recurrence kernels: the whole time loop of one layer in one
// launch of co-resident workgroups, with each workgroup's slice of the recurrent weight
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
// The 4H interleaved gate columns are split in NS slices (4 or 8) and the
// units in groups of 8 NS.  Workgroup (s, v) holds Wh^T for the units of
// group v and the columns of slice s, and writes a partial dh for those
// units; after a barrier among the NS workgroups of the group, member s sums
// the NS partials (in order) for its 8 units [8 NS v + 8 s, + 8), applies
// the cell backward and writes dG; after a grid barrier the next
// contraction may read it.  Each workgroup streams 1/NS of dG per step, so
// more slices mean less operand traffic per CU and more partial sums.  The carried dc
// (and dh of rows whose sequence has not started in reverse) stay in
// registers of the owning thread for the whole launch.
#pragma once

#include <cstddef>

#include "device.hpp"

namespace janus {
namespace persist {

constexpr int kThreads = 512;          // 8 waves
constexpr int kWaves = kThreads / 64;
constexpr int kMaxSlices = 8;          // largest K-split of the backward contraction
constexpr int kMaxB = 256;             // batch rows handled by one pass of 8 waves
constexpr int kSpinLimit = 1 << 22;    // bounded wait at each barrier (~0.1 s)
constexpr int kMaxGroups = 128;        // unit groups (H / (8 NS)) a launch may have
constexpr int kMaxXcds = 16;           // XCDs the census can tell apart (XCC_ID is 4 bits)

// Device-wide barrier state.  The counters (up to `error`) are zeroed before
// every launch; the report that follows them is zeroed once per library call
// and accumulates over its launches.  Counters sit in separate 256-byte lines.
struct Sync {
    unsigned count;                    // global arrivals (census first, then one per XCD per barrier)
    unsigned pad0[63];
    unsigned xcd[16][64];              // per-XCD arrivals
    unsigned census[16][64];           // workgroups resident on each XCD
    unsigned group[kMaxGroups][64];    // arrivals of each unit group
    unsigned ready[kMaxGroups][64];    // backward: members of each unit group whose dG_t is stored
    unsigned error;                    // set when a wait exceeds its spin limit
    unsigned groups;                   // backward unit groups launched
    unsigned local_groups;             // of which kept their partial sums in one XCD's L2
    unsigned fwd_groups;               // the same for the forward
    unsigned fwd_local_groups;
    unsigned pad1[59];
};
constexpr size_t kSyncCounterBytes = offsetof(Sync, error);

__device__ __forceinline__ unsigned xcc_id() {
    // hardware register XCC_ID (20), bits [3:0]: the XCD this wave runs on
    return __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11)) & 0xfu;
}

// Per-workgroup barrier bookkeeping, meaningful in thread 0 only (xcount:
// in the first 16 lanes of wave 0).  S is the counter block: Sync here, or
// any struct with the same count / xcd / census / error members.
template <class S>
struct BarrierT {
    S* s;
    unsigned x, xsize, nx, nb, phase;
    unsigned xidx;                     // arrival order of this workgroup among those on its XCD
    unsigned xfirst;                   // workgroups on the XCDs numbered below this one
    unsigned xcount;                   // lane q < 16 of wave 0: workgroups on XCD q
};

using Barrier = BarrierT<Sync>;

template <class S>
__device__ __forceinline__ bool spin_until(S* s, const unsigned* p, unsigned target) {
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
// Ordering the workgroups by (XCD, arrival order on it) gives each a rank
// xfirst + xidx in [0, gridDim.x) under which consecutive ranks share an XCD
// wherever possible, whatever order the hardware placed them in.
template <class S>
__device__ __forceinline__ void barrier_init(BarrierT<S>& b, S* s) {
    b.s = s;
    b.nb = gridDim.x;
    b.phase = 0;
    b.x = 0;
    b.xsize = 1;
    b.nx = 1;
    b.xidx = 0;
    b.xfirst = 0;
    if (threadIdx.x == 0) {
        b.x = xcc_id();
        b.xidx = __hip_atomic_fetch_add(&s->census[b.x][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(&s->count, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
        spin_until(s, &s->count, b.nb);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        b.xsize = __hip_atomic_load(&s->census[b.x][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        b.nx = 0;
        for (unsigned q = 0; q < 16; ++q) {
            const unsigned c = __hip_atomic_load(&s->census[q][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            b.nx += c != 0u;
            if (q < b.x) b.xfirst += c;
        }
    }
    __syncthreads();
    b.xcount = 0;
    if (threadIdx.x < 16)
        b.xcount = __hip_atomic_load(&s->census[threadIdx.x][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Device-wide barrier, in two halves so that work no other workgroup waits
// for can run while it completes:
//   barrier_arrive: every wave waits for its own memory operations, then the
//     workgroup arrives on its XCD's counter;
//   barrier_wait:   lane q of wave 0 polls XCD q's counter until all of that
//     XCD's workgroups have arrived, all XCDs at once (one round trip per
//     poll, and no second hop through a global count).
// Between the two a workgroup may issue stores that nobody reads in this
// launch and loads of data it owns.  The halves use the raw s_barrier (no
// fence), so memory operations issued between them stay in flight across the
// wait.
//
// Arrivals are relaxed, with no L2 write-back and no invalidate.  That is
// safe because of how the kernels address memory within one launch.  Every
// value one workgroup reads after a barrier that another workgroup wrote
// before it is:
//   * stored with the write-through policy and acknowledged before the
//     writer arrives, so it is in memory by then; and
//   * at an address written for the first time in this launch and never read
//     before that barrier (a fresh slot per step; slots and rows are whole
//     128-byte lines), so no cache on the reading side holds a copy.
// Results that only later kernels read are stored write-back; the end of the
// kernel writes them back.  Caches are invalidated by the dispatch at kernel
// start.
//
// After a timeout every later wait returns at once, so all waves still reach
// the end of the kernel (results are then garbage and `error` is set).
template <class S>
__device__ __forceinline__ void barrier_arrive(BarrierT<S>& b) {
    ++b.phase;
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (threadIdx.x == 0) __hip_atomic_fetch_add(&b.s->xcd[b.x][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <class S>
__device__ __forceinline__ void barrier_wait(BarrierT<S>& b) {
    if (threadIdx.x < 64) {
        const unsigned q = threadIdx.x & 15u;
        const unsigned target = b.phase * b.xcount;   // 0 past lane 15 and for empty XCDs
        bool done = threadIdx.x >= 16 || b.xcount == 0u;
        int spins = 0;
        while (true) {
            if (!done) done = __hip_atomic_load(&b.s->xcd[q][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target;
            if (__all(done)) break;
            if (__hip_atomic_load(&b.s->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) break;
            if (++spins > kSpinLimit) {
                if (threadIdx.x == 0) __hip_atomic_store(&b.s->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
    }
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Barrier among the `members` workgroups of one unit group (they exchange
// partial sums only among themselves).  When all members run on one XCD they
// share its L2: the sums are stored write-back (the L2 acknowledges them
// before the arrival) and read with device-scope loads, which miss in the L1
// and return the L2's copy, so one slot serves every step in the forward (a
// step's sums are read before the grid barrier after which the next step
// overwrites them) and two slots, used in turn, in the backward (which has
// no grid barrier).
// Otherwise they are written through to memory into a slot fresh for each
// step, as for the grid barrier.
//
// Every wave waits for its own stores before the workgroup barrier: the
// workgroup-scope fence of __syncthreads does not wait for global stores
// (the waves share the CU's L1), so without it the arrival could overtake
// another wave's partial sums.
__device__ __forceinline__ void group_barrier(Sync* s, unsigned* cnt, unsigned& phase, unsigned members) {
    ++phase;
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_s_waitcnt(0);
        __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        spin_until(s, cnt, phase * members);
    }
    __syncthreads();
}

// The same barrier for a group whose members all run on one XCD, whose
// partial sums therefore go through that XCD's L2: each member publishes the
// phase it reached in a flag word of its own (word 8 m + 4 of the group's
// 64-word line, member m) with an ordinary store once its partial sums are
// acknowledged, and lane q < members of wave 0 polls member q's flag with
// loads that skip the L1, as the partial sums are read.  A barrier is then an
// L2 round trip, not an atomic performed in memory and polls of it.  The
// flags start at zero with the counters of every launch.
__device__ __forceinline__ void group_barrier_l2(Sync* s, unsigned* line, unsigned& phase, unsigned members,
                                                 int me) {
    ++phase;
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x < 64) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(line, (short)0, int(64 * sizeof(unsigned)),
                                                                            0x00020000);
        const unsigned q = threadIdx.x;
        if (q == 0) {
            __builtin_amdgcn_s_waitcnt(0);
            __builtin_amdgcn_raw_buffer_store_b32(phase, rs, int(4 * (8 * me + 4)), 0, 0);   // written back
        }
        bool done = q >= members;
        int spins = 0;
        while (true) {
            if (!done) done = __builtin_amdgcn_raw_buffer_load_b32(rs, int(4 * (8 * q + 4)), 0, 16) >= phase;
            if (__all(done)) break;
            if ((++spins & 63) == 0 &&
                __hip_atomic_load(&s->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u)
                break;
            if (spins > kSpinLimit) {
                if (q == 0) __hip_atomic_store(&s->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
        }
    }
    __syncthreads();
}

// Place of a workgroup in the unit groups of NS members, from its census
// rank p = xfirst + xidx: member s = p mod NS of group v = p / NS.  The
// members hold consecutive ranks, so they run on one XCD (`local`) unless
// the group contains an XCD boundary (a rank at which the next nonempty
// XCD's workgroups begin).  Such a group is numbered by the boundaries at or
// before its first rank (`straddle`, below the number of XCDs minus one),
// which indexes the slots it needs per step.  All members compute the same
// values from the census, which is complete after barrier_init.
struct GroupPlace {
    int s, v, local, straddle;
};
template <int NS>
__device__ __forceinline__ GroupPlace group_place(const Barrier& bar, Sync* sync) {
    __shared__ int place[4];
    if (threadIdx.x == 0) {
        const unsigned p = bar.xfirst + bar.xidx;
        const unsigned g0 = p - p % NS;
        unsigned end = 0, before = 0;
        bool cross = false;
        for (unsigned q = 0; q < unsigned(kMaxXcds); ++q) {
            const unsigned c = __hip_atomic_load(&sync->census[q][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (c == 0u) continue;
            end += c;
            if (end >= bar.nb) break;   // the end of the last XCD is no boundary
            if (end <= g0) ++before;
            else if (end < g0 + NS) cross = true;
        }
        place[0] = int(p % NS);
        place[1] = int(p / NS);
        place[2] = cross ? 0 : 1;
        place[3] = int(before);
    }
    __syncthreads();
    return GroupPlace{place[0], place[1], place[2], place[3]};
}

// ---------------------------------------------------------------- forward
struct FwdArgs {
    int H, B, t_eff, fixed;
    int rbase;                         // first (sorted) batch row of this launch: rows rbase + [0, kMaxB)
    int Kp;                            // H rounded up to 64
    int nkg;                           // k-groups of 16 columns of h (Kp / 16)
    int ksp;                           // columns of the widest K slice (multiple of 16)
    const int32_t* active;             // [T + 1] (ignored when fixed)
    const int32_t* offsets;            // [T + 2] (ignored when fixed)
    const int32_t* perm;               // [B] or NULL
    const bf16_t* Wh;                  // [4H, H] gate-major
    bf16_t* Hs;                        // [(B + T*B) x ldh], or NULL (not stored)
    float* Cs;                         // [(B + T*B) x ldh]
    const bf16_t* XG;                  // [T*B x ldg] interleaved, bias included
    bf16_t* Gs;                        // [T*B x ldg] interleaved gates
    bf16_t* y;                         // [T, B, H] or NULL
    float* hT;
    float* cT;
    int64_t ldh, ldg;
    bf16_t* Hf;                        // [T + 1] slots of h in fragment layout (slot t = h_{t-1}; slot 0 = h0)
    int64_t hf_slot;                   // elements per slot: round_up(B, 32) * Kp
    bf16_t* HT;                        // [H x ldht] h transposed, column B + p = h at packed row p, or NULL
    int64_t ldht;
    // K-split (NS > 1): partial gate pre-activations exchanged in each unit
    // group.  `part` holds one slot [writer][group][reader][batch tile][1024]
    // reused every step by groups on one XCD (part_local floats), then, per
    // step and straddling group, [t][straddle][writer][reader][batch tile][1024].
    float* part;
    int64_t part_local;
    int nstraddle;                     // straddling groups the slots are sized for
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

// Load the forward weights of a workgroup into LDS: for each member m of its
// unit group (units v0 + 8 m + [0, 8)), 32 rows in the order above, columns
// [c0, c1) of Wh (its K slice) at LDS columns [0, c1 - c0); k contiguous,
// pitch `wld`, zeros past H.  Tile m starts at row 32 m.
template <int NS>
__device__ __forceinline__ void stage_fwd_weights(const FwdArgs& a, bf16_t* Ws, int wld, int v0, int c0, int c1) {
    const int chunks = a.ksp / 8;
    for (int idx = threadIdx.x; idx < 32 * NS * chunks; idx += kThreads) {
        const int i = idx / chunks, kl = (idx - i * chunks) * 8, kc = c0 + kl;
        const int m = i >> 5, ii = i & 31;
        const int u = v0 + 8 * m + fwd_row_unit(ii), g = ii & 3;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (u < a.H && kc < a.H && kc < c1) {
            const bf16_t* src = a.Wh + (int64_t(g) * a.H + u) * a.H + kc;
            if (kc + 8 <= a.H && (a.H % 8) == 0) {
                v = *reinterpret_cast<const uint4*>(src);
            } else {
                bf16_t tmp[8];
                for (int e = 0; e < 8; ++e) tmp[e] = (kc + e < a.H) ? src[e] : bf16_t(0);
                __builtin_memcpy(&v, tmp, 16);
            }
        }
        *reinterpret_cast<uint4*>(Ws + i * wld + kl) = v;
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
constexpr uint32_t kOutOfRange = 0x80000000u;

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, int(bytes), 0x00020000);
}

// Store policies: values other workgroups read later in the same launch are
// written through (sc0 | sc1) to memory; values only later kernels read are
// written back through the L2 as usual.
constexpr int kStoreThrough = 1 | 16;
constexpr int kStoreBack = 0;

__device__ __forceinline__ uint4 load16(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}
// device-scope load (sc1): misses in the L1, so it returns what the L2 holds
__device__ __forceinline__ uint4 load16_l2(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, int(off), 0, 16);
    return make_uint4(v.x, v.y, v.z, v.w);
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

// The same for MT weight tiles of 32 rows (`wtile` elements apart in LDS)
// that share each operand fragment: one load feeds MT MFMAs, whose
// accumulators are independent.  The weight fragments of the next k-group
// are read from LDS while the MFMAs of this one run, and a scheduling
// barrier after each refill keeps the compiler from sinking the refills to
// the end of the unrolled block (which empties the ring).
template <int DEPTH, int MT>
__device__ __forceinline__ void contract_frag_mt(f32x16_t (&acc)[MT], const bf16_t* wrow, int wtile,
                                                 __amdgpu_buffer_rsrc_t rs, uint32_t off, int n) {
    if constexpr (MT == 1) {
        contract_frag<DEPTH>(acc[0], wrow, rs, off, n);
    } else {
        static_assert(DEPTH % 2 == 0, "even ring depth");
        const int last = n > 0 ? n - 1 : 0;
        uint4 w[2][MT];
        auto wload = [&](uint4 (&dst)[MT], int kg) {
            const int k = kg < last ? kg : last;
#pragma unroll
            for (int m = 0; m < MT; ++m) dst[m] = *reinterpret_cast<const uint4*>(wrow + m * wtile + k * 16);
        };
        auto step = [&](const uint4 (&wf)[MT], uint4 h) {
            Frag<bf16_t> fh;
            fh.v = h;
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                Frag<bf16_t> fw;
                fw.v = wf[m];
                mfma(acc[m], fw, fh);
            }
        };
        uint4 ring[DEPTH];
#pragma unroll
        for (int i = 0; i < DEPTH; ++i) ring[i] = load16(rs, i < n ? off + uint32_t(i) * 1024u : kOutOfRange);
        wload(w[0], 0);
        int kg = 0;
        for (; kg + DEPTH <= n; kg += DEPTH) {
#pragma unroll
            for (int i = 0; i < DEPTH; ++i) {
                wload(w[(i + 1) & 1], kg + i + 1);
                step(w[i & 1], ring[i]);
                const int nx = kg + i + DEPTH;
                ring[i] = load16(rs, nx < n ? off + uint32_t(nx) * 1024u : kOutOfRange);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
#pragma unroll
        for (int i = 0; i < DEPTH; ++i) {
            if (kg + i < n) {
                wload(w[(i + 1) & 1], kg + i + 1);
                step(w[i & 1], ring[i]);
            }
        }
    }
}

// ring depth with two weight tiles (each fragment feeds two MFMAs)
constexpr int kDepthFrag2 = 8;
constexpr int kDepthFrag = 12;

// One layer's forward recurrence.  NS == 1: workgroup q owns units
// [8 q, 8 q + 8) and contracts all of h_{t-1} against their 32 rows of Wh.
// NS > 1 (K split): the units are split in groups of 8 NS and the columns of
// Wh in NS slices; member s of group v holds the rows of all 8 NS units for
// slice s, contracts slice s of h_{t-1} (1 / NS of the stream) into partial
// pre-activations of the whole group, and owns the cells of units
// v0 + 8 s + [0, 8).  The members exchange partial sums as the backward does.
template <int KW, int NS>
__global__ __launch_bounds__(kThreads) void lstm_fwd_persistent(FwdArgs a) {
    static_assert(NS == 1 || NS == 2 || NS == 4, "slices of the forward contraction");
    constexpr int MT = NS;            // 32-row weight tiles per wave: one per member of the group
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wld = a.ksp + 8;
    bf16_t* Ws = reinterpret_cast<bf16_t*>(smem_raw);
    float* red = reinterpret_cast<float*>(smem_raw + size_t(32 * NS) * wld * sizeof(bf16_t));
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    Barrier bar;
    barrier_init(bar, a.sync);
    int s = 0, v = int(blockIdx.x), straddle = 0;
    bool plocal = true;
    if constexpr (NS > 1) {
        const GroupPlace gp = group_place<NS>(bar, a.sync);
        s = gp.s;
        v = gp.v;
        plocal = gp.local != 0;
        straddle = gp.straddle;
        if (threadIdx.x == 0 && s == 0) {
            __hip_atomic_fetch_add(&a.sync->fwd_groups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (plocal)
                __hip_atomic_fetch_add(&a.sync->fwd_local_groups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            // slots were sized for fewer straddling groups than the census found:
            // report it, and the partial sums below go nowhere
            if (!plocal && straddle >= a.nstraddle)
                __hip_atomic_store(&a.sync->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    const int ngroups = int(gridDim.x) / NS;
    const int v0 = v * 8 * NS;                // first unit of the group
    const int u0 = v0 + 8 * s;                // first unit whose cells this workgroup owns
    constexpr int NB = kWaves / KW;
    const int bt = wave % NB, kw = wave / NB;
    const int sg0 = s * a.nkg / NS, sgn = (s + 1) * a.nkg / NS - sg0;   // k-groups of slice s
    const int kg0 = kw * sgn / KW, kg1 = (kw + 1) * sgn / KW;
    const bf16_t* wrow = Ws + (lane & 31) * wld + 8 * (lane >> 5) + kg0 * 16;
    const int tb = a.rbase / 32 + bt;        // this wave's batch tile of the whole batch
    const uint32_t hoff = (uint32_t(tb * a.nkg + sg0 + kg0) * 512u + uint32_t(lane) * 8u) * 2u;
    const int H = a.H;
    const int row = tb * 32 + (lane & 31);   // this lane's batch row (sorted order)
    const int ub = u0 + 4 * (lane >> 5);      // its four consecutive units
    // lanes of the kw == 0 waves own cells; with NS > 1 the last group may
    // extend past H, and its units there have none
    const bool owner = kw == 0 && ub < H;
    const int b = (owner && row < a.B && a.perm) ? a.perm[row] : row;   // caller's batch index
    unsigned* gcnt = NS > 1 ? &a.sync->group[v][0] : nullptr;
    unsigned gphase = 0;
    const int nbt = (a.B + 31) / 32;          // batch tiles of 32 rows
    const uint32_t tile_bytes = uint32_t(nbt) * 4096u;
    // tile (writer j, reader m) of this group's partial sums at step t
    auto part_tile = [&](int j, int m, int t) -> __amdgpu_buffer_rsrc_t {
        if (plocal)
            return make_rsrc(a.part + ((int64_t(j) * ngroups + v) * NS + m) * nbt * 1024, tile_bytes);
        const bool room = straddle < a.nstraddle;
        return make_rsrc(a.part + a.part_local +
                             ((((int64_t(t) * a.nstraddle + (room ? straddle : 0)) * NS + j) * NS + m) * nbt) * 1024,
                         room ? tile_bytes : 0u);
    };

    stage_fwd_weights<NS>(a, Ws, wld, v0, 16 * sg0, 16 * (sg0 + sgn));
    // the cell state of the owned cells stays in registers for the launch
    float creg[4] = {0.f, 0.f, 0.f, 0.f};
    if (owner && row < a.B) {
        const float4 c0 = *reinterpret_cast<const float4*>(a.Cs + int64_t(row) * a.ldh + ub);
        creg[0] = c0.x; creg[1] = c0.y; creg[2] = c0.z; creg[3] = c0.w;
    }
    __syncthreads();

    // operand of the cell update that does not depend on h_{t-1}, loaded one
    // step ahead (branch-free; lanes without a cell read out of range, i.e. 0)
    uint4 xg0, xg1;
    auto prefetch_xg = [&](int t) {
        const int act = act_at(a.active, a.fixed, a.B, t, a.t_eff);
        const int64_t off = off_at(a.offsets, a.fixed, a.B, t);
        const auto rxg = make_rsrc(a.XG + off * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
        const uint32_t o = (owner && row < act) ? (uint32_t(row) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u
                                                : kOutOfRange;
        xg0 = load16(rxg, o);
        xg1 = load16(rxg, o + 16u);
    };
    prefetch_xg(0);

    for (int t = 0; t < a.t_eff; ++t) {
        const int act = act_at(a.active, a.fixed, a.B, t, a.t_eff);
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        const int64_t off_t = off_at(a.offsets, a.fixed, a.B, t);
        const bool cell = owner && row < act;
        const bool more = t + 1 < a.t_eff;
        f32x16_t accs[MT];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int e = 0; e < 16; ++e) accs[m][e] = 0.f;
        if (tb * 32 < act) {
            // h_{t-1} is slot t of the fragment-layout copy
            const auto rs = make_rsrc(a.Hf + int64_t(t) * a.hf_slot, uint32_t(a.hf_slot) * 2u);
            contract_frag_mt<MT == 1 ? kDepthFrag : kDepthFrag2, MT>(accs, wrow, 32 * wld, rs, hoff, kg1 - kg0);
        }
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (KW > 1 && m > 0) __syncthreads();   // the previous tile's K parts have been read
            reduce_kparts<KW>(accs[m], red, wave, lane);
        }
        f32x16_t acc = accs[0];
        if constexpr (NS > 1) {
            // tile m of a wave holds the pre-activations of member m's units for
            // its 32 batch rows; lane l's 16 values are stored as four 16-byte
            // pieces q, so each store of a wave is 1 KB in one piece
            const uint32_t po = uint32_t((tb * 4) * 64 + lane) * 16u;
            if (kw == 0 && tb * 32 < act) {
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    if (m == s) continue;
                    const auto rp = part_tile(s, m, t);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const uint4 pv = make_uint4(__float_as_uint(accs[m][4 * q]), __float_as_uint(accs[m][4 * q + 1]),
                                                    __float_as_uint(accs[m][4 * q + 2]),
                                                    __float_as_uint(accs[m][4 * q + 3]));
                        if (plocal) store16<kStoreBack>(rp, po + uint32_t(q) * 1024u, pv);
                        else store16<kStoreThrough>(rp, po + uint32_t(q) * 1024u, pv);
                    }
                }
            }
            if (plocal) group_barrier_l2(a.sync, gcnt, gphase, unsigned(NS), s);
            else group_barrier(a.sync, gcnt, gphase, unsigned(NS));
            // this workgroup's own tile, then the members' sums in member order
            f32x16_t own = accs[0];
#pragma unroll
            for (int m = 1; m < MT; ++m)
                if (m == s) own = accs[m];
            uint4 pin[NS][4];
#pragma unroll
            for (int j = 0; j < NS; ++j) {
                const auto rp = part_tile(j, s, t);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t o = (owner && row < act && j != s) ? po + uint32_t(q) * 1024u : kOutOfRange;
                    pin[j][q] = plocal ? load16_l2(rp, o) : load16(rp, o);
                }
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
            for (int j = 0; j < NS; ++j) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float pj[4] = {__uint_as_float(pin[j][q].x), __uint_as_float(pin[j][q].y),
                                         __uint_as_float(pin[j][q].z), __uint_as_float(pin[j][q].w)};
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[4 * q + e] += j == s ? own[4 * q + e] : pj[e];
                }
            }
        }
        float hn[4] = {0.f, 0.f, 0.f, 0.f};
        uint32_t gw[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
        uint2 hb = make_uint2(0u, 0u);
        if (cell) {
            const uint32_t xw[8] = {xg0.x, xg0.y, xg0.z, xg0.w, xg1.x, xg1.y, xg1.z, xg1.w};
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
            hb = make_uint2(uint32_t(f2bf(hn[0])) | (uint32_t(f2bf(hn[1])) << 16),
                            uint32_t(f2bf(hn[2])) | (uint32_t(f2bf(hn[3])) << 16));
            // h_t for the next step (fragment layout, slot t + 1): the only
            // value other workgroups read in this launch
            if (more && row < act_next) {
                const auto rhf = make_rsrc(a.Hf + int64_t(t + 1) * a.hf_slot, uint32_t(a.hf_slot) * 2u);
                store8<kStoreThrough>(rhf, uint32_t(frag_index(row, ub, a.Kp)) * 2u, hb);
            }
        }
        if (more) barrier_arrive(bar);
        // results for later kernels and the next step's operand, while the
        // barrier completes
        if (cell) {
            const int64_t nrow = int64_t(a.B) + off_t;   // first row of step t in Hs / Cs
            const auto rcs = make_rsrc(a.Cs + nrow * a.ldh, uint32_t(act) * uint32_t(a.ldh) * 4u);
            const auto rgs = make_rsrc(a.Gs + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
            store16<kStoreBack>(rcs, (uint32_t(row) * uint32_t(a.ldh) + uint32_t(ub)) * 4u,
                    make_uint4(__float_as_uint(creg[0]), __float_as_uint(creg[1]), __float_as_uint(creg[2]),
                               __float_as_uint(creg[3])));
            if (a.Hs) {
                const auto rhs = make_rsrc(a.Hs + nrow * a.ldh, uint32_t(act) * uint32_t(a.ldh) * 2u);
                store8<kStoreBack>(rhs, (uint32_t(row) * uint32_t(a.ldh) + uint32_t(ub)) * 2u, hb);
            }
            if (a.HT) {
                // transposed copy, the K-contiguous operand of the weight gradients
                bf16_t* ht = a.HT + int64_t(ub) * a.ldht + a.B + off_t + row;
#pragma unroll
                for (int q = 0; q < 4; ++q) ht[q * a.ldht] = f2bf(hn[q]);
            }
            const uint32_t og = (uint32_t(row) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u;
            store16<kStoreBack>(rgs, og, make_uint4(gw[0], gw[1], gw[2], gw[3]));
            store16<kStoreBack>(rgs, og + 16u, make_uint4(gw[4], gw[5], gw[6], gw[7]));
            if (a.y) {
                const auto ry = make_rsrc(a.y + int64_t(t) * a.B * H, uint32_t(a.B) * uint32_t(H) * 2u);
                store8<kStoreBack>(ry, (uint32_t(b) * uint32_t(H) + uint32_t(ub)) * 2u, hb);
            }
            if (row >= act_next) {   // last step of this sequence
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (a.hT) a.hT[int64_t(b) * H + ub + q] = hn[q];
                    if (a.cT) a.cT[int64_t(b) * H + ub + q] = creg[q];
                }
            }
        }
        if (more) {
            prefetch_xg(t + 1);
            barrier_wait(bar);
        }
    }
}

// ---------------------------------------------------------------- backward
struct BwdArgs {
    int H, B, t_eff, fixed;
    int rbase;                         // first (sorted) batch row of this launch: rows rbase + [0, kMaxB)
    int db_add;                        // 1: add this launch's bias gradient to db (a later batch part)
    int nkg;                           // k-groups of 16 interleaved gate columns (4H / 16)
    int ksp;                           // columns of the widest K slice (multiple of 16)
    const int32_t* active;
    const int32_t* offsets;
    const int32_t* perm;
    const bf16_t* Wh;                  // [4H, H] gate-major
    bf16_t* G;                         // dG store [T*B x ldg] interleaved (for dX after the loop), or NULL
    bf16_t* Gf;                        // [T] slots of dG in fragment layout (slot t = dG_t), K = 4H
    int64_t gf_slot;                   // elements per slot: round_up(B, 32) * 4H
    const bf16_t* Gs;                  // saved gates, interleaved
    const float* Cs;
    const bf16_t* dy;                  // gradient of this layer's output or NULL
    int64_t dy_ld;
    const int32_t* dy_rows;            // packed row -> dy row, NULL = identity
    const float* dhT;
    const float* dcT;
    float* dh0;
    float* dc0;
    float* part;                       // [t_eff + 1] slots of NS x B x (8 NS groups) partial sums of dh
    float* db;                         // [4H] gate-major bias gradient (overwritten), or NULL
    bf16_t* GT;                        // [4H x ldk] dG transposed (interleaved rows), or NULL
    int64_t ldk;
    int gt_pairs;                      // 1: every step's packed offset is even (row pairs as 4-byte stores)
    int64_t ldh, ldg;
    Sync* sync;
};

// Slice s of the K = 4H interleaved gate columns: k-groups [s nkg / NS, (s + 1) nkg / NS).
template <int NS>
__device__ __forceinline__ int slice_kg0(int nkg, int s) { return s * nkg / NS; }

// WT[uu][kk] = (Wh interleaved)[c][v0 + uu] = Wh[(c % 4) * H + c / 4][v0 + uu],  c = 16 kg0 + kk
template <int NS>
__device__ __forceinline__ void stage_bwd_weights(const BwdArgs& a, bf16_t* Ws, int wld, int s, int v0) {
    constexpr int UNITS = 8 * NS;
    const int H = a.H;
    const int c0 = 16 * slice_kg0<NS>(a.nkg, s), c1 = 16 * slice_kg0<NS>(a.nkg, s + 1);
#pragma unroll 8
    for (int idx = threadIdx.x; idx < UNITS * a.ksp; idx += kThreads) {
        const int kk = idx / UNITS, uu = idx - kk * UNITS;
        const int c = c0 + kk;
        const int u = v0 + uu;
        bf16_t v = 0;
        if (c < c1 && c < 4 * H && u < H) v = a.Wh[(int64_t(c & 3) * H + (c >> 2)) * H + u];
        Ws[uu * wld + kk] = v;
    }
}

template <int KW, int NS>
__global__ __launch_bounds__(kThreads) void lstm_bwd_persistent(BwdArgs a) {
    static_assert(NS == 4 || NS == 8, "slices of the backward contraction");
    constexpr int UNITS = 8 * NS;     // units of a group
    constexpr int MT = UNITS / 32;    // 32-row weight tiles per wave
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wld = a.ksp + 8;
    bf16_t* Ws = reinterpret_cast<bf16_t*>(smem_raw);
    float* red = reinterpret_cast<float*>(smem_raw + size_t(UNITS) * wld * sizeof(bf16_t));
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    Barrier bar;
    barrier_init(bar, a.sync);
    // Unit group v and K slice s of this workgroup from its census rank p:
    // the members of a group hold consecutive ranks, so they run on one XCD
    // unless the group straddles the end of an XCD's workgroups.  The
    // partial sums of such a local group stay in the L2 its members share.
    __shared__ int assign[3];
    if (threadIdx.x == 0) {
        const unsigned p = bar.xfirst + bar.xidx;
        const unsigned g0 = p - p % NS;   // rank of the group's first member
        assign[0] = int(p % NS);
        assign[1] = int(p / NS);
        assign[2] = (g0 >= bar.xfirst && g0 + NS <= bar.xfirst + bar.xsize) ? 1 : 0;
    }
    __syncthreads();
    const int s = assign[0], v = assign[1];
    const bool plocal = assign[2] != 0;
    if (threadIdx.x == 0 && s == 0) {
        __hip_atomic_fetch_add(&a.sync->groups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (plocal) __hip_atomic_fetch_add(&a.sync->local_groups, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int v0 = v * UNITS;
    const int ngroups = int(gridDim.x) / NS;
    const int H = a.H;
    unsigned* gcnt = &a.sync->group[v][0];
    unsigned gphase = 0;

    stage_bwd_weights<NS>(a, Ws, wld, s, v0);

    // contraction geometry: wave (bt, kw) takes batch rows [32 bt, 32 bt + 32)
    // and part kw of this slice's k-groups
    constexpr int NB = kWaves / KW;
    const int bt = wave % NB, kw = wave / NB;
    const int sg0 = slice_kg0<NS>(a.nkg, s), sgn = slice_kg0<NS>(a.nkg, s + 1) - sg0;
    const int kg0 = kw * sgn / KW, kg1 = (kw + 1) * sgn / KW;

    // Step-to-step dependency.  The contraction of step t reads slice s of
    // dG_{t+1}: k-groups [sg0, sg0 + sgn), i.e. units [4 sg0, 4 (sg0 + sgn)),
    // whose cells belong to unit groups [vr0, vr1].  Instead of a grid
    // barrier, each workgroup counts itself into its group's `ready` once its
    // dG_t is stored (written through and acknowledged, as for the grid
    // barrier), and waits only for the groups its slice reads: NS arrivals
    // per step each.
    const int vr0 = (4 * sg0) / UNITS;
    const int vr1 = min(ngroups - 1, (4 * (sg0 + sgn) - 1) / UNITS);
    unsigned rphase = 0;
    auto ready_arrive = [&]() {
        ++rphase;
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (threadIdx.x == 0)
            __hip_atomic_fetch_add(&a.sync->ready[v][0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    // lane q of wave 0 polls group vr0 + q, so the counters are read in
    // parallel (one round trip per poll, not one per group).  A slice spans
    // at most ngroups / NS + 1 groups, within one wave for NS >= 4.
    static_assert(kMaxGroups / 4 + 1 <= 64, "the groups of a slice fit one wave");
    auto ready_wait = [&]() {
        if (wave == 0) {
            const int q = vr0 + lane;
            const unsigned target = rphase * unsigned(NS);
            bool done = q > vr1;
            int spins = 0;
            while (true) {
                if (!done) done = __hip_atomic_load(&a.sync->ready[q][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= target;
                if (__all(done)) break;
                if (__hip_atomic_load(&a.sync->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) break;
                if (++spins > kSpinLimit) {
                    if (lane == 0) __hip_atomic_store(&a.sync->error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
            }
        }
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
    };
    const bf16_t* wrow = Ws + (lane & 31) * wld + 8 * (lane >> 5) + kg0 * 16;
    const int tb = a.rbase / 32 + bt;        // this wave's batch tile of the whole batch
    const uint32_t goff = (uint32_t(tb * a.nkg + sg0 + kg0) * 512u + uint32_t(lane) * 8u) * 2u;
    const int crow = tb * 32 + (lane & 31);   // batch row of this lane's accumulator column

    // pointwise ownership: row r, units [ub, ub + 4) (member s of the group
    // takes units [v0 + 8 s, v0 + 8 s + 8))
    const int r = a.rbase + (tid >> 1);
    const int ub = v0 + 8 * s + 4 * (tid & 1);
    const bool mine = r < a.B && ub < H;
    const int b = mine ? (a.perm ? a.perm[r] : r) : 0;
    float dhp[4] = {0.f, 0.f, 0.f, 0.f}, dcr[4] = {0.f, 0.f, 0.f, 0.f}, cnx[4] = {0.f, 0.f, 0.f, 0.f};
    float dbs[16];   // running sum over steps of this thread's dG (unit k, gate g at 4 k + g)
#pragma unroll
    for (int e = 0; e < 16; ++e) dbs[e] = 0.f;
    if (mine) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (a.dhT) dhp[k] = a.dhT[int64_t(b) * H + ub + k];
            if (a.dcT) dcr[k] = a.dcT[int64_t(b) * H + ub + k];
        }
    }
    __syncthreads();

    // operands of the cell backward that do not depend on dh, loaded one step
    // ahead (lanes without a cell read out of range, i.e. 0)
    uint4 g0, g1, cpv, cnv;
    uint2 dyv;
    auto prefetch = [&](int t) {
        const int act = t >= 0 ? act_at(a.active, a.fixed, a.B, t, a.t_eff) : a.B;
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        const int64_t off_t = t >= 0 ? off_at(a.offsets, a.fixed, a.B, t) : 0;
        const int64_t prev_base = t <= 0 ? 0 : int64_t(a.B) + off_at(a.offsets, a.fixed, a.B, t - 1);
        const bool cell = mine && r < act && t >= 0;
        const auto rgs = make_rsrc(a.Gs + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
        const uint32_t ogs = cell ? (uint32_t(r) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u : kOutOfRange;
        g0 = load16(rgs, ogs);
        g1 = load16(rgs, ogs + 16u);
        const auto rcp = make_rsrc(a.Cs + prev_base * a.ldh, uint32_t(a.B) * uint32_t(a.ldh) * 4u);
        cpv = load16(rcp, cell ? (uint32_t(r) * uint32_t(a.ldh) + uint32_t(ub)) * 4u : kOutOfRange);
        // c_t is carried from the later step when the row was active there
        const bool fresh = cell && r >= act_next;
        const auto rcn = make_rsrc(a.Cs + (int64_t(a.B) + off_t) * a.ldh, uint32_t(a.B) * uint32_t(a.ldh) * 4u);
        cnv = load16(rcn, fresh ? (uint32_t(r) * uint32_t(a.ldh) + uint32_t(ub)) * 4u : kOutOfRange);
        dyv = make_uint2(0, 0);
        if (cell && a.dy) {
            const int64_t p = off_t + r;
            const int64_t yr = a.dy_rows ? int64_t(a.dy_rows[p]) : p;
            dyv = *reinterpret_cast<const uint2*>(a.dy + yr * a.dy_ld + ub);
        }
    };
    prefetch(a.t_eff - 1);

    for (int t = a.t_eff - 1; t >= -1; --t) {
        const int act = t >= 0 ? act_at(a.active, a.fixed, a.B, t, a.t_eff) : a.B;
        const int act_next = act_at(a.active, a.fixed, a.B, t + 1, a.t_eff);
        const int64_t off_t = t >= 0 ? off_at(a.offsets, a.fixed, a.B, t) : 0;
        const bool cell = mine && r < act && t >= 0;
        const bool fresh = cell && r >= act_next;
        const bool sync_after = t >= 0 && act > 0;

        // partial sums of dh_t from dG_{t+1} (slot t + 1 of the fragment copy).
        // Slot layout [writer slice][group][reader member][row][8 units]: what
        // one wave stores, and what one wave of a reader loads, is 1 KB in one
        // piece (32 rows x 32 bytes).
        // A local group alternates between slots 0 and 1: without a grid
        // barrier a member may store step t's sums while another still reads
        // those of step t + 1, but not those of step t + 2 (its sums of step
        // t + 1 entered the group barrier first).
        const int64_t pslot = int64_t(NS) * ngroups * NS * a.B * 8;
        float* part = plocal ? a.part + int64_t((t + 1) & 1) * pslot : a.part + int64_t(t + 1) * pslot;
        if (act_next > 0) {
            f32x16_t acc[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[m][e] = 0.f;
            if (tb * 32 < act_next) {
                const auto rs = make_rsrc(a.Gf + int64_t(t + 1) * a.gf_slot, uint32_t(a.gf_slot) * 2u);
                contract_frag_mt<MT == 1 ? kDepthFrag : kDepthFrag2, MT>(acc, wrow, 32 * wld, rs, goff, kg1 - kg0);
            }
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if (KW > 1 && m > 0) __syncthreads();   // the previous tile's K parts have been read
                reduce_kparts<KW>(acc[m], red, wave, lane);
            }
            if (kw == 0 && crow < act_next) {
                // tile m of a lane holds units v0 + 32 m + 8 j + 4 (lane / 32) + [0, 4) of row crow:
                // reader member 4 m + j, unit offset 4 (lane / 32) in its octet
                const auto rp = make_rsrc(part + (int64_t(s) * ngroups + v) * NS * a.B * 8,
                                          uint32_t(NS) * uint32_t(a.B) * 32u);
#pragma unroll
                for (int m = 0; m < MT; ++m)
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int u = v0 + 32 * m + 8 * j + 4 * (lane >> 5);
                        const uint32_t o =
                            u < H ? ((uint32_t(4 * m + j) * uint32_t(a.B) + uint32_t(crow)) * 8u + 4u * uint32_t(lane >> 5)) * 4u
                                  : kOutOfRange;
                        const uint4 pv = make_uint4(__float_as_uint(acc[m][4 * j]), __float_as_uint(acc[m][4 * j + 1]),
                                                    __float_as_uint(acc[m][4 * j + 2]),
                                                    __float_as_uint(acc[m][4 * j + 3]));
                        if (plocal) store16<kStoreBack>(rp, o, pv);
                        else store16<kStoreThrough>(rp, o, pv);
                    }
            }
            if (plocal) group_barrier_l2(a.sync, gcnt, gphase, unsigned(NS), s);
            else group_barrier(a.sync, gcnt, gphase, unsigned(NS));
        }

        uint32_t dgl[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};   // this step's dG, zero without a cell
        float dh[4] = {dhp[0], dhp[1], dhp[2], dhp[3]};
        if (mine && r < act) {
            if (r < act_next) {
                // sum the slices in order
                dh[0] = dh[1] = dh[2] = dh[3] = 0.f;
#pragma unroll
                for (int j = 0; j < NS; ++j) {
                    const auto rp = make_rsrc(part + ((int64_t(j) * ngroups + v) * NS + s) * a.B * 8,
                                              uint32_t(a.B) * 32u);
                    const uint32_t o = (uint32_t(r) * 8u + 4u * uint32_t(tid & 1)) * 4u;
                    const uint4 pv = plocal ? load16_l2(rp, o) : load16(rp, o);
                    dh[0] += __uint_as_float(pv.x); dh[1] += __uint_as_float(pv.y);
                    dh[2] += __uint_as_float(pv.z); dh[3] += __uint_as_float(pv.w);
                }
            }
        }
        if (cell) {
            const uint32_t gw[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
            const float cpr[4] = {__uint_as_float(cpv.x), __uint_as_float(cpv.y), __uint_as_float(cpv.z),
                                  __uint_as_float(cpv.w)};
            if (fresh) {
                cnx[0] = __uint_as_float(cnv.x); cnx[1] = __uint_as_float(cnv.y);
                cnx[2] = __uint_as_float(cnv.z); cnx[3] = __uint_as_float(cnv.w);
            }
            const float dyf[4] = {bf2f(bf16_t(dyv.x & 0xffffu)), bf2f(bf16_t(dyv.x >> 16)),
                                  bf2f(bf16_t(dyv.y & 0xffffu)), bf2f(bf16_t(dyv.y >> 16))};
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float dhv = dh[k] + dyf[k];
                const uint32_t w0 = gw[2 * k], w1 = gw[2 * k + 1];
                const float gi = bf2f(bf16_t(w0 & 0xffffu)), gf = bf2f(bf16_t(w0 >> 16));
                const float gg = bf2f(bf16_t(w1 & 0xffffu)), go = bf2f(bf16_t(w1 >> 16));
                const float tau = tanhf_(cnx[k]);
                const float d_o = dhv * tau;
                const float dct = dcr[k] + dhv * go * (1.f - tau * tau);
                dcr[k] = dct * gf;
                const float dai = dct * gg * gi * (1.f - gi), daf = dct * cpr[k] * gf * (1.f - gf);
                const float dag = dct * gi * (1.f - gg * gg), dao = d_o * go * (1.f - go);
                dbs[4 * k] += dai;
                dbs[4 * k + 1] += daf;
                dbs[4 * k + 2] += dag;
                dbs[4 * k + 3] += dao;
                dgl[2 * k] = uint32_t(f2bf(dai)) | (uint32_t(f2bf(daf)) << 16);
                dgl[2 * k + 1] = uint32_t(f2bf(dag)) | (uint32_t(f2bf(dao)) << 16);
                cnx[k] = cpr[k];   // c_{t-1} is the next (earlier) step's c_t
            }
            // dG_t in fragment layout (columns 4 ub .. 4 ub + 15: one k-group):
            // the only value other workgroups read in this launch
            const auto rf = make_rsrc(a.Gf + int64_t(t) * a.gf_slot, uint32_t(a.gf_slot) * 2u);
            const uint32_t of = uint32_t(frag_index(r, 4 * ub, 4 * H)) * 2u;
            store16<kStoreThrough>(rf, of, make_uint4(dgl[0], dgl[1], dgl[2], dgl[3]));
            store16<kStoreThrough>(rf, of + 512u, make_uint4(dgl[4], dgl[5], dgl[6], dgl[7]));
        }
        if (sync_after) ready_arrive();

        // results for later kernels and the next (earlier) step's operands,
        // while the producers of this slice finish the step
        if (t < 0 && mine) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if (a.dh0) a.dh0[int64_t(b) * H + ub + k] = dh[k];
                if (a.dc0) a.dc0[int64_t(b) * H + ub + k] = dcr[k];
            }
        }
        if (cell) {
            if (a.G) {
                // dG_t row-major (for the contractions after the loop)
                const auto rg = make_rsrc(a.G + off_t * a.ldg, uint32_t(act) * uint32_t(a.ldg) * 2u);
                const uint32_t og = (uint32_t(r) * uint32_t(a.ldg) + 4u * uint32_t(ub)) * 2u;
                store16<kStoreBack>(rg, og, make_uint4(dgl[0], dgl[1], dgl[2], dgl[3]));
                store16<kStoreBack>(rg, og + 16u, make_uint4(dgl[4], dgl[5], dgl[6], dgl[7]));
            }
            if (a.GT && !a.gt_pairs) {
                // transposed copy: the K-contiguous operand of the weight gradients
                bf16_t* gt = a.GT + int64_t(4) * ub * a.ldk + off_t + r;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    gt[(2 * e) * a.ldk] = bf16_t(dgl[e] & 0xffffu);
                    gt[(2 * e + 1) * a.ldk] = bf16_t(dgl[e] >> 16);
                }
            }
        }
        if (a.GT && a.gt_pairs && t >= 0) {
            // transposed copy with row pairs: lanes l and l ^ 2 hold rows r and
            // r ^ 1 of the same units; the even row writes columns 4 ub + [0, 8)
            // and the odd row columns 4 ub + [8, 16), 4 bytes (two rows) each.
            const bool odd = r & 1;
            uint32_t own[4], other[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                own[i] = odd ? dgl[4 + i] : dgl[i];
                other[i] = __shfl_xor(odd ? dgl[i] : dgl[4 + i], 2);
            }
            if (cell) {
                const int64_t p0 = off_t + (r & ~1);
                bf16_t* gt = a.GT + (int64_t(4) * ub + (odd ? 8 : 0)) * a.ldk + p0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t lo = odd ? other[i] : own[i];    // even row's dword
                    const uint32_t hi = odd ? own[i] : other[i];    // odd row's dword
                    *reinterpret_cast<uint32_t*>(gt + (2 * i) * a.ldk) = (lo & 0xffffu) | (hi << 16);
                    *reinterpret_cast<uint32_t*>(gt + (2 * i + 1) * a.ldk) = (lo >> 16) | (hi & 0xffff0000u);
                }
            }
        }
        if (t >= 0) prefetch(t - 1);
        if (sync_after) ready_wait();
    }

    // bias gradient: sum dbs over the rows of this workgroup's units, in a
    // fixed order (lanes of a wave by xor steps, then waves in order); the
    // weight slice in LDS is no longer needed and holds the wave totals
    if (a.db) {
        // lanes 2 r' + half of a wave hold rows r' of one half: reduce over r'
#pragma unroll
        for (int e = 0; e < 16; ++e) {
#pragma unroll
            for (int m = 2; m < 64; m <<= 1) dbs[e] += __shfl_xor(dbs[e], m);
        }
        __syncthreads();
        float* wsum = reinterpret_cast<float*>(smem_raw);   // [8 waves][2 halves][16]
        if (lane < 2) {
#pragma unroll
            for (int e = 0; e < 16; ++e) wsum[(wave * 2 + lane) * 16 + e] = dbs[e];
        }
        __syncthreads();
        if (tid < 32) {
            const int half = tid >> 4, e = tid & 15;
            float sum = 0.f;
            for (int w = 0; w < kWaves; ++w) sum += wsum[(w * 2 + half) * 16 + e];
            const int u = v0 + 8 * s + 4 * half + (e >> 2), g = e & 3;
            if (u < H) a.db[int64_t(g) * H + u] = a.db_add ? a.db[int64_t(g) * H + u] + sum : sum;
        }
    }
}

}  // namespace persist
}  // namespace janus
