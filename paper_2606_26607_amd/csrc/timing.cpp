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
bool g_enabled = false;
std::vector<Record> g_pool;  // events are created once and reused
size_t g_used = 0;

}  // namespace

KernelTimer::KernelTimer(int kind, hipStream_t stream) : slot(-1), s(stream)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_enabled || g_used >= kMaxRecords) return;
    if (g_used == g_pool.size()) {
        Record r{kind, nullptr, nullptr};
        if (hipEventCreate(&r.start) != hipSuccess) return;
        if (hipEventCreate(&r.stop) != hipSuccess) {
            (void)hipEventDestroy(r.start);
            return;
        }
        g_pool.push_back(r);
    }
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
    g_enabled = enable != 0;
    return MOE_OK;
}

extern "C" moe_status moe_timing_reset(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    for (size_t i = 0; i < g_used; ++i)
        if (hipEventSynchronize(g_pool[i].stop) != hipSuccess) return MOE_ERR_HIP;
    g_used = 0;
    return MOE_OK;
}

extern "C" moe_status moe_timing_read(int kind, double *total_ms, int64_t *launches)
{
    if (total_ms == nullptr || launches == nullptr || kind < 0 || kind >= MOE_K_COUNT)
        return MOE_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(g_mu);
    double sum = 0.0;
    int64_t n = 0;
    for (size_t i = 0; i < g_used; ++i) {
        if (g_pool[i].kind != kind) continue;
        if (hipEventSynchronize(g_pool[i].stop) != hipSuccess) return MOE_ERR_HIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, g_pool[i].start, g_pool[i].stop) != hipSuccess) return MOE_ERR_HIP;
        sum += ms;
        ++n;
    }
    *total_ms = sum;
    *launches = n;
    return MOE_OK;
}
