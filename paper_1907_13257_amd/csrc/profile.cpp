// profile.cpp -- optional per-kernel timing: when enabled, each launch of the
// library is bracketed by two HIP events on the stream it runs on, tagged with
// its kernel class and algorithmic FLOPs / bytes.  Durations are resolved when
// the caller reads the statistics.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <vector>

#include "../../include/lstm355.h"
#include "kernels.hpp"

namespace lstm355 {

namespace {

struct Rec {
    int k;
    hipEvent_t a, b;
    double flops, bytes;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;   // recycled events

// Timing-only events: no system-scope fence (cache write-back) when they
// complete, so recording them barely perturbs the kernels they bracket.
hipEvent_t take_event()
{
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

const char *const kNames[K_NCLASS] = {"gemm_input_proj", "recurrent_fwd", "recurrent_bwd", "gemm_dx",
                                       "gemm_dw",         "gemm_dr",       "gemm_dp",       "small",
                                       "gemm_dw_dr"};

}  // namespace

const char *kclass_name(int k) { return (k >= 0 && k < K_NCLASS) ? kNames[k] : "?"; }

ProfScope::ProfScope(int kclass, hipStream_t st, double fl, double by) : k(kclass), s(st), flops(fl), bytes(by), ev0(nullptr)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_on) return;
    hipEvent_t e = take_event();
    if (!e) return;
    if (hipEventRecord(e, s) != hipSuccess) {
        g_pool.push_back(e);
        return;
    }
    ev0 = e;
}

ProfScope::~ProfScope()
{
    if (!ev0) return;
    std::lock_guard<std::mutex> lk(g_mu);
    hipEvent_t e1 = take_event();
    if (!e1 || hipEventRecord(e1, s) != hipSuccess) {
        if (e1) g_pool.push_back(e1);
        (void)hipEventSynchronize(static_cast<hipEvent_t>(ev0));
        g_pool.push_back(static_cast<hipEvent_t>(ev0));
        return;
    }
    g_recs.push_back(Rec{k, static_cast<hipEvent_t>(ev0), e1, flops, bytes});
}

}  // namespace lstm355

using namespace lstm355;

extern "C" lstm_status_t lstm_profile_enable(int on)
{
    std::lock_guard<std::mutex> lk(g_mu);
    g_on = on != 0;
    return LSTM_OK;
}

extern "C" lstm_status_t lstm_profile_reset(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto &r : g_recs) {
        (void)hipEventSynchronize(r.b);
        g_pool.push_back(r.a);
        g_pool.push_back(r.b);
    }
    g_recs.clear();
    return LSTM_OK;
}

extern "C" lstm_status_t lstm_profile_read(lstm_kernel_stat_t *out, int cap, int *n)
{
    if (!n || (cap > 0 && !out)) return LSTM_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(g_mu);
    lstm_kernel_stat_t acc[K_NCLASS];
    std::memset(acc, 0, sizeof(acc));
    for (int k = 0; k < K_NCLASS; ++k) std::strncpy(acc[k].name, kNames[k], sizeof(acc[k].name) - 1);
    for (auto &r : g_recs) {
        float ms = 0.0f;
        if (hipEventSynchronize(r.b) != hipSuccess) return LSTM_ERR_HIP;
        if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return LSTM_ERR_HIP;
        acc[r.k].launches += 1;
        acc[r.k].total_ms += ms;
        acc[r.k].flops += r.flops;
        acc[r.k].bytes += r.bytes;
    }
    int m = 0;
    for (int k = 0; k < K_NCLASS && m < cap; ++k)
        if (acc[k].launches) out[m++] = acc[k];
    *n = m;
    return LSTM_OK;
}
