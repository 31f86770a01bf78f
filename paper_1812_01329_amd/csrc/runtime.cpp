// Host runtime: pinned staging ring for schedule uploads, status strings.
#include "runtime.hpp"

#include <cstdio>
#include <cstring>
#include <deque>
#include <vector>
#include <mutex>

namespace janus {

namespace {
thread_local char g_last_error[512] = "";
}

janus_status device_error(hipError_t e, const char* what, const char* file, int line) {
    const char* base = std::strrchr(file, '/');
    std::snprintf(g_last_error, sizeof(g_last_error), "%s (%d) from %s at %s:%d", hipGetErrorName(e), int(e), what,
                  base ? base + 1 : file, line);
    return JANUS_ERR_DEVICE;
}

namespace {

// A ring of pinned host memory.  Each upload copies its bytes into the next
// free region, enqueues an asynchronous host-to-device copy on the caller's
// stream and records an event; a region is reused only after its event has
// completed.  The ring is allocated once per process.
class PinnedRing {
  public:
    static constexpr size_t kCapacity = size_t(64) << 20;

    janus_status put(void* dst, const void* src, size_t bytes, hipStream_t stream) {
        std::lock_guard<std::mutex> lock(mu_);
        if (!base_) {
            const hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&base_), kCapacity, hipHostMallocDefault);
            if (e != hipSuccess) {
                base_ = nullptr;
                return device_error(e, "hipHostMalloc", __FILE__, __LINE__);
            }
        }
        const size_t need = (bytes + 255) & ~size_t(255);
        if (need > kCapacity) return JANUS_ERR_UNSUPPORTED;
        if (head_ + need > kCapacity) head_ = 0;
        // wait for every in-flight copy that still reads the target region
        for (auto it = inflight_.begin(); it != inflight_.end();) {
            const bool overlap = it->off < head_ + need && head_ < it->off + it->len;
            if (overlap) {
                JANUS_HIP(hipEventSynchronize(it->ev));
                free_events_.push_back(it->ev);
                it = inflight_.erase(it);
            } else {
                ++it;
            }
        }
        std::memcpy(base_ + head_, src, bytes);
        JANUS_HIP(hipMemcpyAsync(dst, base_ + head_, bytes, hipMemcpyHostToDevice, stream));
        hipEvent_t ev;
        if (!free_events_.empty()) {
            ev = free_events_.back();
            free_events_.pop_back();
        } else {
            JANUS_HIP(hipEventCreateWithFlags(&ev, hipEventDisableTiming));
        }
        JANUS_HIP(hipEventRecord(ev, stream));
        inflight_.push_back({head_, need, ev});
        // retire completed copies so the list stays short
        while (!inflight_.empty() && hipEventQuery(inflight_.front().ev) == hipSuccess) {
            free_events_.push_back(inflight_.front().ev);
            inflight_.pop_front();
        }
        head_ += need;
        return JANUS_OK;
    }

  private:
    struct Use {
        size_t off, len;
        hipEvent_t ev;
    };
    std::mutex mu_;
    char* base_ = nullptr;
    size_t head_ = 0;
    std::deque<Use> inflight_;
    std::vector<hipEvent_t> free_events_;
};

PinnedRing& ring() {
    static PinnedRing r;
    return r;
}

}  // namespace

janus_status upload(void* dst_dev, const void* src_host, size_t bytes, hipStream_t stream) {
    if (bytes == 0) return JANUS_OK;
    return ring().put(dst_dev, src_host, bytes, stream);
}

janus_status upload_pieces(const UploadPiece* pieces, int n, hipStream_t stream) {
    if (n <= 0) return JANUS_OK;
    char* const base = static_cast<char*>(pieces[0].dst);
    size_t span = 0;
    bool ordered = true;
    for (int i = 0; i < n; ++i) {
        char* d = static_cast<char*>(pieces[i].dst);
        // overlaps or precedes the previous piece, or leaves more than
        // alignment padding between them (the image writes the gaps, with
        // zeros, so they must hold nothing)
        if (d < base + span || size_t(d - (base + span)) > kUploadMaxGap) ordered = false;
        if (ordered) span = size_t(d - base) + pieces[i].bytes;
    }
    if (!ordered || span > (size_t(16) << 20)) {
        for (int i = 0; i < n; ++i) {
            const janus_status e = upload(pieces[i].dst, pieces[i].src, pieces[i].bytes, stream);
            if (e != JANUS_OK) return e;
        }
        return JANUS_OK;
    }
    std::vector<char> image(span, 0);
    for (int i = 0; i < n; ++i)
        if (pieces[i].bytes) std::memcpy(image.data() + (static_cast<char*>(pieces[i].dst) - base), pieces[i].src,
                                         pieces[i].bytes);
    return upload(base, image.data(), span, stream);
}

// ------------------------------------------------------------------ tracing
namespace {

struct TraceRec {
    const char* label;
    double flops, bytes;
    hipEvent_t start, stop;
};

struct TraceState {
    std::mutex mu;
    bool on = false;
    bool failed = false;
    std::vector<TraceRec> recs;
    std::vector<hipEvent_t> pool;

    hipEvent_t get() {
        if (!pool.empty()) {
            hipEvent_t e = pool.back();
            pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) {
            failed = true;
            return nullptr;
        }
        return e;
    }
};

TraceState& trace() {
    static TraceState t;
    return t;
}

}  // namespace

TraceScope::TraceScope(const char* label, double flops, double bytes, hipStream_t stream) {
    if (!label) return;   // an untraced launch
    TraceState& t = trace();
    if (!t.on) return;
    std::lock_guard<std::mutex> lock(t.mu);
    hipEvent_t a = t.get(), b = t.get();
    if (!a || !b) return;
    if (hipEventRecord(a, stream) != hipSuccess) {
        t.failed = true;
        return;
    }
    t.recs.push_back({label, flops, bytes, a, b});
    slot_ = int(t.recs.size()) - 1;
    stream_ = stream;
}

TraceScope::~TraceScope() {
    if (slot_ < 0) return;
    TraceState& t = trace();
    std::lock_guard<std::mutex> lock(t.mu);
    if (hipEventRecord(t.recs[slot_].stop, stream_) != hipSuccess) t.failed = true;
}

}  // namespace janus

extern "C" janus_status janus_trace_begin(void) {
    janus::TraceState& t = janus::trace();
    std::lock_guard<std::mutex> lock(t.mu);
    for (auto& r : t.recs) {
        t.pool.push_back(r.start);
        t.pool.push_back(r.stop);
    }
    t.recs.clear();
    t.failed = false;
    t.on = true;
    return JANUS_OK;
}

extern "C" janus_status janus_trace_end(janus_trace_stat* out, int32_t max_out, int32_t* n_out) {
    if (!n_out) return JANUS_ERR_INVALID_ARG;
    janus::TraceState& t = janus::trace();
    std::lock_guard<std::mutex> lock(t.mu);
    t.on = false;
    std::vector<janus_trace_stat> agg;
    janus_status st = t.failed ? JANUS_ERR_DEVICE : JANUS_OK;
    for (auto& r : t.recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
            st = JANUS_ERR_DEVICE;
            continue;
        }
        janus_trace_stat* s = nullptr;
        for (auto& a : agg)
            if (std::strncmp(a.label, r.label, sizeof(a.label)) == 0) s = &a;
        if (!s) {
            agg.push_back(janus_trace_stat{});
            s = &agg.back();
            std::strncpy(s->label, r.label, sizeof(s->label) - 1);
        }
        s->launches += 1;
        s->total_ms += ms;
        s->flops += r.flops;
        s->bytes += r.bytes;
    }
    for (auto& r : t.recs) {
        t.pool.push_back(r.start);
        t.pool.push_back(r.stop);
    }
    t.recs.clear();
    *n_out = int32_t(agg.size());
    for (int32_t i = 0; i < int32_t(agg.size()) && i < max_out && out; ++i) out[i] = agg[i];
    return st;
}

extern "C" const char* janus_status_string(janus_status s) {
    switch (s) {
        case JANUS_OK: return "ok";
        case JANUS_ERR_INVALID_ARG: return "invalid argument";
        case JANUS_ERR_LENGTH: return "sequence length outside [0, T]";
        case JANUS_ERR_TREE: return "malformed tree batch";
        case JANUS_ERR_TOKEN: return "id outside [0, V)";
        case JANUS_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
        case JANUS_ERR_UNSUPPORTED: return "unsupported dtype or shape";
        case JANUS_ERR_DEVICE: return "HIP call failed";
    }
    return "unknown status";
}

extern "C" const char* janus_last_error(void) { return janus::g_last_error; }

extern "C" const char* janus_version(void) { return "janus-mi355x 0.1.0 (gfx950)"; }
