// api.hip -- host-only entry points of libams: status text, build info and
// per-kernel event timing.
#include <string.h>

#include <mutex>
#include <vector>

#include "ams_device.h"

extern "C" const char *ams_status_str(ams_status s)
{
    switch (s) {
    case AMS_OK: return "ok";
    case AMS_ERR_NULL: return "a required pointer is NULL";
    case AMS_ERR_SIZE: return "a size is negative, too large, or inconsistent";
    case AMS_ERR_DTYPE: return "unknown storage dtype";
    case AMS_ERR_DIMS: return "unsupported layer widths";
    case AMS_ERR_WORKSPACE: return "workspace too small";
    case AMS_ERR_HIP: return "HIP launch or runtime error";
    case AMS_ERR_ID_RANGE: return "image ID out of range";
    case AMS_ERR_MODE: return "unknown pooling mode";
    case AMS_ERR_CAPACITY: return "size beyond the fixed scratch of the no-allocation call";
    }
    return "unknown status";
}

extern "C" const char *ams_build_info(void)
{
    return "libams 0.1.0 gfx950 wave64";
}

// ------------------------------------------------------------- timing ----

int ams_timing_flag = 0;

namespace {

struct TimedLaunch {
    const char *name;                 // static string at the launch site
    hipEvent_t start, stop;
};

std::mutex g_timing_mu;
std::vector<TimedLaunch> g_launches;  // recorded since the last read
std::vector<hipEvent_t> g_free;       // events kept for reuse
bool g_timing_failed = false;

hipEvent_t take_event()
{
    if (!g_free.empty()) {
        hipEvent_t e = g_free.back();
        g_free.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

void ams_timing_begin(const char *name, hipStream_t st)
{
    std::lock_guard<std::mutex> lk(g_timing_mu);
    TimedLaunch t{name, take_event(), nullptr};
    if (!t.start || hipEventRecord(t.start, st) != hipSuccess) g_timing_failed = true;
    g_launches.push_back(t);
}

void ams_timing_end(hipStream_t st)
{
    std::lock_guard<std::mutex> lk(g_timing_mu);
    if (g_launches.empty() || g_launches.back().stop) {
        g_timing_failed = true;
        return;
    }
    TimedLaunch &t = g_launches.back();
    t.stop = take_event();
    if (!t.stop || hipEventRecord(t.stop, st) != hipSuccess) g_timing_failed = true;
}

extern "C" ams_status ams_timing_enable(int on)
{
    __atomic_store_n(&ams_timing_flag, on ? 1 : 0, __ATOMIC_RELAXED);
    return AMS_OK;
}

extern "C" ams_status ams_timing_read(ams_kernel_time *out, int cap, int *n_out)
{
    if (cap < 0 || (cap > 0 && !out) || !n_out) return AMS_ERR_NULL;
    std::lock_guard<std::mutex> lk(g_timing_mu);
    bool failed = g_timing_failed;
    std::vector<ams_kernel_time> acc;
    for (const TimedLaunch &t : g_launches) {
        float ms = 0.f;
        const bool ok = t.start && t.stop && hipEventSynchronize(t.stop) == hipSuccess &&
                        hipEventElapsedTime(&ms, t.start, t.stop) == hipSuccess;
        if (!ok) failed = true;
        size_t k = 0;
        while (k < acc.size() && strncmp(acc[k].name, t.name, sizeof(acc[k].name)) != 0) ++k;
        if (k == acc.size()) {
            ams_kernel_time z{};
            strncpy(z.name, t.name, sizeof(z.name) - 1);
            acc.push_back(z);
        }
        if (ok) {
            acc[k].launches += 1;
            acc[k].total_ms += ms;
        }
        if (t.start) g_free.push_back(t.start);
        if (t.stop) g_free.push_back(t.stop);
    }
    g_launches.clear();
    g_timing_failed = false;
    for (int k = 0; k < cap && k < (int)acc.size(); ++k) out[k] = acc[k];
    *n_out = (int)acc.size();
    return failed ? AMS_ERR_HIP : AMS_OK;
}
