// Kernel-level tracing: when enabled, every kernel the library launches is
// bracketed by two HIP events recorded on its launch stream (or only the
// launches a name filter lists), so a caller can read the device duration of
// each launch.  Events are created once by
// cogdl_trace_enable; the launch path only records them (nothing allocates).
// The tracer is process-wide and not thread-safe.
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"
#include "internal.hpp"

namespace cogdl {
namespace {

struct Tracer {
    bool on = false;
    int32_t cap = 0;
    int32_t n = 0;
    std::vector<hipEvent_t> start, stop;
    std::vector<const char *> names;
    std::vector<std::string> only;   // empty: record every launch
};

Tracer g_trace;

bool traced(const char *name)
{
    if (g_trace.only.empty()) return true;
    for (const std::string &o : g_trace.only)
        if (o == name) return true;
    return false;
}

void trace_free()
{
    for (auto e : g_trace.start) (void)hipEventDestroy(e);
    for (auto e : g_trace.stop) (void)hipEventDestroy(e);
    g_trace.start.clear();
    g_trace.stop.clear();
    g_trace.names.clear();
    g_trace.cap = g_trace.n = 0;
    g_trace.on = false;
}

}  // namespace

int trace_begin(const char *name, hipStream_t s)
{
    if (!g_trace.on || g_trace.n >= g_trace.cap || !traced(name)) return -1;
    const int i = g_trace.n++;
    g_trace.names[i] = name;
    (void)hipEventRecord(g_trace.start[i], s);
    return i;
}

void trace_end(int slot, hipStream_t s)
{
    if (slot >= 0) (void)hipEventRecord(g_trace.stop[slot], s);
}

int resident_blocks(const void *kernel, int block)
{
    struct Entry { const void *kernel; int device, block, blocks; };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) { (void)hipGetLastError(); return 2048; }
    std::lock_guard<std::mutex> lock(mu);
    for (const Entry &e : cache)
        if (e.kernel == kernel && e.device == dev && e.block == block) return e.blocks;
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, block, 0) != hipSuccess ||
        cus < 1 || per_cu < 1) {
        (void)hipGetLastError();
        return 2048;
    }
    cache.push_back(Entry{kernel, dev, block, cus * per_cu});
    return cus * per_cu;
}

}  // namespace cogdl

extern "C" {

cogdl_status cogdl_trace_enable(int32_t capacity)
{
    using cogdl::g_trace;
    if (capacity < 0) return COGDL_ERR_INVALID;
    cogdl::trace_free();
    if (capacity == 0) return COGDL_OK;
    g_trace.start.resize(capacity);
    g_trace.stop.resize(capacity);
    g_trace.names.assign(capacity, nullptr);
    for (int32_t i = 0; i < capacity; ++i) {
        if (hipEventCreate(&g_trace.start[i]) != hipSuccess ||
            hipEventCreate(&g_trace.stop[i]) != hipSuccess) {
            g_trace.start.resize(i);
            g_trace.stop.resize(i);
            cogdl::trace_free();
            return COGDL_ERR_NOMEM;
        }
    }
    g_trace.cap = capacity;
    g_trace.n = 0;
    g_trace.on = true;
    return COGDL_OK;
}

cogdl_status cogdl_trace_filter(const char *names)
{
    std::vector<std::string> only;
    if (names) {
        if (strlen(names) > 1023) return COGDL_ERR_INVALID;
        const char *p = names;
        while (*p) {
            const char *q = strchr(p, ',');
            const size_t len = q ? (size_t)(q - p) : strlen(p);
            if (len > 63) return COGDL_ERR_INVALID;
            if (len > 0) only.emplace_back(p, len);
            p += len;
            if (*p == ',') ++p;
        }
    }
    cogdl::g_trace.only.swap(only);
    return COGDL_OK;
}

cogdl_status cogdl_trace_reset(void)
{
    cogdl::g_trace.n = 0;
    return COGDL_OK;
}

int32_t cogdl_trace_count(void) { return cogdl::g_trace.n; }

cogdl_status cogdl_trace_get(int32_t i, const char **name, float *ms)
{
    using cogdl::g_trace;
    if (i < 0 || i >= g_trace.n || !name || !ms) return COGDL_ERR_INVALID;
    *name = g_trace.names[i];
    if (hipEventSynchronize(g_trace.stop[i]) != hipSuccess) return COGDL_ERR_LAUNCH;
    if (hipEventElapsedTime(ms, g_trace.start[i], g_trace.stop[i]) != hipSuccess)
        return COGDL_ERR_LAUNCH;
    return COGDL_OK;
}

}  // extern "C"
