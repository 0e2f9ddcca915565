// Status strings, device-error bookkeeping and host-side helpers.
#include <atomic>
#include <cstring>
#include <map>
#include <string>

#include "common.h"

namespace tgm {

namespace {
struct ProfRec {
    const char *name;
    hipEvent_t a, b;
};
struct Profiler {
    bool on = false;
    std::vector<hipEvent_t> free_events;
    std::vector<ProfRec> pending;
    std::map<std::string, std::pair<int64_t, double>> totals;
    std::vector<std::string> names;   // stable order for tgm_profile_get
} g_prof;

hipEvent_t take_event()
{
    if (g_prof.free_events.empty()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess)
            return nullptr;
        return e;
    }
    hipEvent_t e = g_prof.free_events.back();
    g_prof.free_events.pop_back();
    return e;
}

void fold_pending()
{
    for (auto &r : g_prof.pending) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
            auto &t = g_prof.totals[r.name];
            t.first += 1;
            t.second += ms;
        }
        g_prof.free_events.push_back(r.a);
        g_prof.free_events.push_back(r.b);
    }
    g_prof.pending.clear();
    g_prof.names.clear();
    for (auto &kv : g_prof.totals)
        g_prof.names.push_back(kv.first);
}
}  // namespace

int prof_begin(const char *kernel, hipStream_t s)
{
    if (!g_prof.on)
        return -1;
    ProfRec r{kernel, take_event(), take_event()};
    if (!r.a || !r.b || hipEventRecord(r.a, s) != hipSuccess)
        return -1;
    g_prof.pending.push_back(r);
    return (int)g_prof.pending.size() - 1;
}

void prof_end(int id, hipStream_t s)
{
    if (id < 0)
        return;
    hipEventRecord(g_prof.pending[id].b, s);
}

static std::atomic<int> g_device_error{hipSuccess};
static std::atomic<int64_t> g_allocs{0};

void count_alloc() { g_allocs.fetch_add(1, std::memory_order_relaxed); }

void record_error(hipError_t e)
{
    int expected = hipSuccess;
    g_device_error.compare_exchange_strong(expected, (int)e);
}

std::vector<float> pack_b(const float *W, int n_out, int ldw, int c0, int K, int KC, int NB)
{
    std::vector<float> out((size_t)KC * NB * kWave * 4, 0.f);
    for (int kc = 0; kc < KC; ++kc)
        for (int nb = 0; nb < NB; ++nb)
            for (int lane = 0; lane < kWave; ++lane)
                for (int j = 0; j < 4; ++j) {
                    const int k = 16 * kc + 4 * (lane >> 4) + j;
                    const int n = 16 * nb + (lane & 15);
                    if (k < K && n < n_out)
                        out[(((size_t)kc * NB + nb) * kWave + lane) * 4 + j] =
                            W[(size_t)n * ldw + c0 + k];
                }
    return out;
}

tgm_status_t upload(void *dst, const void *src, size_t bytes)
{
    if (bytes == 0)
        return TGM_OK;
    hipError_t e = hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        record_error(e);
        return TGM_EDEVICE;
    }
    return TGM_OK;
}

}  // namespace tgm

extern "C" const char *tgm_status_str(tgm_status_t s)
{
    switch (s) {
    case TGM_OK: return "ok";
    case TGM_EINVAL: return "invalid argument";
    case TGM_ERANGE: return "input content out of range";
    case TGM_EORDER: return "iteration protocol violated";
    case TGM_ESIZE: return "capacity exceeded";
    case TGM_EDEVICE: return "HIP runtime error";
    case TGM_ENOMEM: return "device allocation failed";
    default: return "unknown status";
    }
}

extern "C" tgm_status_t tgm_last_device_error(void)
{
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        tgm::record_error(e);
    const int prev = tgm::g_device_error.exchange(hipSuccess);
    return prev == hipSuccess ? TGM_OK : TGM_EDEVICE;
}

extern "C" int32_t tgm_version(void) { return 100; }

extern "C" tgm_status_t tgm_alloc_count(int64_t *count)
{
    if (!count)
        return TGM_EINVAL;
    *count = tgm::g_allocs.load(std::memory_order_relaxed);
    return TGM_OK;
}

extern "C" tgm_status_t tgm_profile_enable(int32_t on)
{
    tgm::g_prof.on = on != 0;
    return TGM_OK;
}

extern "C" tgm_status_t tgm_profile_reset(void)
{
    tgm::fold_pending();
    tgm::g_prof.totals.clear();
    tgm::g_prof.names.clear();
    return TGM_OK;
}

extern "C" int32_t tgm_profile_count(void)
{
    tgm::fold_pending();
    return (int32_t)tgm::g_prof.names.size();
}

extern "C" tgm_status_t tgm_profile_get(int32_t k, const char **name, int64_t *launches,
                                        double *total_ms)
{
    if (k < 0 || k >= (int32_t)tgm::g_prof.names.size())
        return TGM_EINVAL;
    const std::string &n = tgm::g_prof.names[k];
    const auto &t = tgm::g_prof.totals[n];
    if (name) {
        static std::map<std::string, std::string> keep;
        *name = keep.emplace(n, n).first->second.c_str();
    }
    if (launches) *launches = t.first;
    if (total_ms) *total_ms = t.second;
    return TGM_OK;
}
