// Internal host-side declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime_api.h>

#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/janus.h"

namespace janus {

// ---------------------------------------------------------------- schedules
struct SeqSchedule {
    int32_t B = 0, T = 0, t_eff = 0;
    int64_t packed = 0;              // sum of lengths = rows of all running steps
    bool fixed = true;               // every length equals T (identity maps)
    std::vector<int32_t> perm;       // [B]
    std::vector<int32_t> active;     // [T + 1], active[t] = 0 for t >= t_eff
    std::vector<int32_t> offsets;    // [T + 2]
    std::vector<int32_t> xrow;       // [packed] row of x for each packed row (varlen only)
    std::vector<int32_t> prevrow;    // [packed] row of h_{t-1} in the h store (varlen only)
};

struct TreeSchedule {
    int32_t N = 0, num_trees = 0, num_levels = 0, max_level_size = 0;
    std::vector<int32_t> level;          // [N]
    std::vector<int32_t> level_offsets;  // [L + 1]
    std::vector<int32_t> level_nodes;    // [N] node at each level-ordered position
    std::vector<int32_t> pos;            // [N] level-ordered position of each node
};

// Trees of any arity (child lists): nodes ordered by (level, id), a node's
// level one more than its highest child's; children lists by position.
struct NarySchedule {
    int32_t N = 0;
    std::vector<int32_t> level_offsets;   // [num_levels + 1]
    std::vector<int32_t> pword;           // [N] word of the node at each position
    std::vector<int32_t> pcoff;           // [N + 1] children of position p: pkids[pcoff[p] .. pcoff[p + 1])
    std::vector<int32_t> pkids;           // [max(E, 1)] child positions
    std::vector<int32_t> rootk;           // [N] tree index of a root position, -1 otherwise
    std::vector<int32_t> rootpos;         // [K] position of root k
};

janus_status build_seq_schedule(int32_t B, int32_t T, const int32_t* lengths, SeqSchedule& s);
janus_status validate_tree_batch(const janus_tree_batch* t, int32_t V);
janus_status build_tree_schedule(const janus_tree_batch* t, int32_t V, TreeSchedule& s);
janus_status build_nary_schedule(const janus_nary_tree_batch* t, int32_t V, NarySchedule& s);

// ---------------------------------------------------------------- workspace
// Bump allocator used both to size a workspace (base == nullptr) and to
// carve it; identical call sequences give identical layouts.
struct Carver {
    char* base;
    size_t off = 0;
    explicit Carver(void* b) : base(static_cast<char*>(b)) {}
    template <typename T>
    T* take(size_t count) {
        off = (off + 255) & ~size_t(255);
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }
inline size_t dtype_size(janus_dtype d) { return d == JANUS_BF16 ? 2 : 4; }
inline bool dtype_ok(janus_dtype d) { return d == JANUS_F32 || d == JANUS_BF16; }

// Copies small host arrays (schedules, index maps) into device memory
// through a pinned staging ring, so that the source may be a temporary and
// the copy stays asynchronous on the caller's stream.
janus_status upload(void* dst_dev, const void* src_host, size_t bytes, hipStream_t stream);

// Several host arrays for device buffers that lie one after another in one
// region (carved in order, with padding between them): one copy of a host
// image of the whole span instead of one copy per array; the padding is
// written with zeros.  Pieces out of order, further apart than
// kUploadMaxGap bytes, or spanning more than the staging capacity are
// copied one by one.
constexpr size_t kUploadMaxGap = size_t(64) << 10;
struct UploadPiece {
    void* dst;
    const void* src;
    size_t bytes;
};
janus_status upload_pieces(const UploadPiece* pieces, int n, hipStream_t stream);

// Brackets one kernel launch with trace events while tracing is on (see
// janus_trace_begin); a no-op otherwise, and for a NULL label (a launch that
// must not create events).  flops / bytes: algorithmic work.
class TraceScope {
  public:
    TraceScope(const char* label, double flops, double bytes, hipStream_t stream);
    ~TraceScope();
    TraceScope(const TraceScope&) = delete;
    TraceScope& operator=(const TraceScope&) = delete;

  private:
    int slot_ = -1;
    hipStream_t stream_ = nullptr;
};

// Records which HIP call failed, with its error, for janus_last_error on
// this thread, and returns JANUS_ERR_DEVICE.
janus_status device_error(hipError_t e, const char* what, const char* file, int line);

#define JANUS_HIP(call)                                                                 \
    do {                                                                                \
        const hipError_t janus_e_ = (call);                                             \
        if (janus_e_ != hipSuccess) return ::janus::device_error(janus_e_, #call, __FILE__, __LINE__); \
    } while (0)

#define JANUS_LAUNCH_CHECK() JANUS_HIP(hipGetLastError())

}  // namespace janus
