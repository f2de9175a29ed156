// dd_prof.hip -- the dd_prof_* timing ABI: HIP event pairs around launches.
#include "dd_prof.hpp"
#include "dd_attn.h"

#include <mutex>
#include <vector>

namespace dd {
namespace {

struct Record {
    hipEvent_t start, stop;
    int kernel;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Record> g_recs;  // records [0, g_used) are live; the rest are reusable
size_t g_used = 0;

const char *const kNames[K_COUNT] = {"forward", "backward_short", "backward_dkdv", "backward_dq",
                                     "rope"};

}  // namespace

ProfScope::ProfScope(KernelId id, hipStream_t stream) : slot_(-1), stream_(stream)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_on)
        return;
    if (g_used == g_recs.size()) {
        Record r{nullptr, nullptr, 0};
        if (hipEventCreate(&r.start) != hipSuccess || hipEventCreate(&r.stop) != hipSuccess)
            return;
        g_recs.push_back(r);
    }
    Record &r = g_recs[g_used];
    r.kernel = id;
    if (hipEventRecord(r.start, stream_) != hipSuccess)
        return;
    slot_ = static_cast<int>(g_used++);
}

ProfScope::~ProfScope()
{
    if (slot_ < 0)
        return;
    std::lock_guard<std::mutex> lk(g_mu);
    (void)hipEventRecord(g_recs[slot_].stop, stream_);
}

}  // namespace dd

extern "C" {

int dd_prof_enable(int on)
{
    std::lock_guard<std::mutex> lk(dd::g_mu);
    if (on)
        dd::g_used = 0;
    dd::g_on = on != 0;
    return DD_OK;
}

int dd_prof_read(int kernel, double *total_ms, long long *launches)
{
    if (!total_ms || !launches)
        return DD_ERR_NULL;
    if (kernel < 0 || kernel >= dd::K_COUNT)
        return DD_ERR_SHAPE;
    std::lock_guard<std::mutex> lk(dd::g_mu);
    double sum = 0.0;
    long long n = 0;
    for (size_t i = 0; i < dd::g_used; ++i) {
        const dd::Record &r = dd::g_recs[i];
        if (r.kernel != kernel)
            continue;
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
            return DD_ERR_HIP;
        sum += ms;
        ++n;
    }
    *total_ms = sum;
    *launches = n;
    return DD_OK;
}

int dd_prof_launches(int *kernels, double *ms, long long capacity, long long *count)
{
    if (!count || (capacity > 0 && (!kernels || !ms)))
        return DD_ERR_NULL;
    std::lock_guard<std::mutex> lk(dd::g_mu);
    const long long n = static_cast<long long>(dd::g_used);
    for (long long i = 0; i < n && i < capacity; ++i) {
        const dd::Record &r = dd::g_recs[static_cast<size_t>(i)];
        float t = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess)
            return DD_ERR_HIP;
        kernels[i] = r.kernel;
        ms[i] = t;
    }
    *count = n;
    return DD_OK;
}

const char *dd_prof_kernel_name(int kernel)
{
    return (kernel >= 0 && kernel < dd::K_COUNT) ? dd::kNames[kernel] : nullptr;
}

}  // extern "C"
