// Optional per-kernel timing with HIP events recorded on the launch stream.
#include <mutex>
#include <vector>

#include "moe_internal.h"

namespace moe {
namespace {

struct Record {
    int kind;
    hipEvent_t start, stop;
};

constexpr size_t kMaxRecords = 1 << 16;

std::mutex g_mu;
uint32_t g_mask = 0;  // bit k set: kernels of kind k are timed
std::vector<Record> g_pool;  // events are created once and reused
size_t g_used = 0;

}  // namespace

KernelTimer::KernelTimer(int kind, hipStream_t stream) : slot(-1), s(stream)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!((g_mask >> kind) & 1u) || g_used >= kMaxRecords) return;
    if (g_used == g_pool.size()) {
        Record r{kind, nullptr, nullptr};
        if (hipEventCreate(&r.start) != hipSuccess) return;
        if (hipEventCreate(&r.stop) != hipSuccess) {
            (void)hipEventDestroy(r.start);
            return;
        }
        g_pool.push_back(r);
    }
    // not under stream capture: a captured record would only order the graph,
    // it would not time anything
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;
    Record &r = g_pool[g_used];
    r.kind = kind;
    if (hipEventRecord(r.start, s) != hipSuccess) return;
    slot = (int)g_used++;
}

KernelTimer::~KernelTimer()
{
    if (slot < 0) return;
    std::lock_guard<std::mutex> lk(g_mu);
    (void)hipEventRecord(g_pool[slot].stop, s);
}

}  // namespace moe

using namespace moe;

extern "C" moe_status moe_timing_enable(int enable)
{
    std::lock_guard<std::mutex> lk(g_mu);
    g_mask = enable ? (1u << MOE_K_COUNT) - 1u : 0u;
    return MOE_OK;
}

extern "C" moe_status moe_timing_enable_mask(uint32_t kinds)
{
    if (kinds >> MOE_K_COUNT) return set_error(MOE_ERR_INVALID_ARG, "moe_timing_enable_mask: 0x%x", kinds);
    std::lock_guard<std::mutex> lk(g_mu);
    g_mask = kinds;
    return MOE_OK;
}

extern "C" moe_status moe_timing_reset(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    for (size_t i = 0; i < g_used; ++i) {
        const hipError_t err = hipEventSynchronize(g_pool[i].stop);
        if (err != hipSuccess) return set_error(MOE_ERR_HIP, "moe_timing_reset: %s", hipGetErrorString(err));
    }
    g_used = 0;
    return MOE_OK;
}

extern "C" moe_status moe_timing_read(int kind, double *total_ms, int64_t *launches)
{
    if (total_ms == nullptr || launches == nullptr || kind < 0 || kind >= MOE_K_COUNT)
        return set_error(MOE_ERR_INVALID_ARG, "moe_timing_read: bad kind %d or null output", kind);
    std::lock_guard<std::mutex> lk(g_mu);
    double sum = 0.0;
    int64_t n = 0;
    for (size_t i = 0; i < g_used; ++i) {
        if (g_pool[i].kind != kind) continue;
        hipError_t err = hipEventSynchronize(g_pool[i].stop);
        float ms = 0.f;
        if (err == hipSuccess) err = hipEventElapsedTime(&ms, g_pool[i].start, g_pool[i].stop);
        if (err != hipSuccess) return set_error(MOE_ERR_HIP, "moe_timing_read: %s", hipGetErrorString(err));
        sum += ms;
        ++n;
    }
    *total_ms = sum;
    *launches = n;
    return MOE_OK;
}
