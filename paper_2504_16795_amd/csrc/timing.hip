// Optional per-kernel timing: while enabled, every kernel launch of the library (or only
// those of one selected kernel) is bracketed by a pair of HIP events recorded on the launch
// stream.  Collecting waits for the recorded
// events and accumulates, per kernel name, the launch count and the total milliseconds.
// Disabled (the default), a launch costs one relaxed atomic load.
#include <atomic>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "hsa.h"

namespace hsa {
namespace {

struct Rec {
    const char* name;
    hipEvent_t a, b;
};

std::atomic<bool> g_on{false};
std::atomic<bool> g_filtered{false};
std::mutex g_mu;
std::string g_only;                                       // timed kernel when filtered
std::vector<Rec> g_pending;
std::vector<hipEvent_t> g_free;
std::map<std::string, std::pair<long, double>> g_acc;   // name -> (launches, total ms)

hipEvent_t take_event() {
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

KernelTimer::KernelTimer(const char* name, hipStream_t st) : name_(name), st_(st) {
    if (!g_on.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_filtered.load(std::memory_order_relaxed) && g_only != name) return;
    a_ = take_event();
    b_ = take_event();
    if (a_ && b_) (void)hipEventRecord(a_, st_);
}

KernelTimer::~KernelTimer() {
    if (!a_ || !b_) return;
    (void)hipEventRecord(b_, st_);
    std::lock_guard<std::mutex> lk(g_mu);
    g_pending.push_back(Rec{name_, a_, b_});
}

}  // namespace hsa

extern "C" {

hsa_attn_status_t hsa_attn_timing_enable(int on) {
    hsa::g_on.store(on != 0);
    return HSA_ATTN_OK;
}

hsa_attn_status_t hsa_attn_timing_select(const char* name) {
    std::lock_guard<std::mutex> lk(hsa::g_mu);
    hsa::g_only = name ? name : "";
    hsa::g_filtered.store(!hsa::g_only.empty());
    return HSA_ATTN_OK;
}

int hsa_attn_timing_collect(char* buf, size_t len) {
    std::lock_guard<std::mutex> lk(hsa::g_mu);
    for (auto& r : hsa::g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(r.b) == hipSuccess &&
            hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
            auto& e = hsa::g_acc[r.name];
            e.first += 1;
            e.second += ms;
        }
        hsa::g_free.push_back(r.a);
        hsa::g_free.push_back(r.b);
    }
    hsa::g_pending.clear();
    std::string out;
    char line[256];
    for (auto& kv : hsa::g_acc) {
        snprintf(line, sizeof(line), "%s %ld %.6f\n", kv.first.c_str(), kv.second.first,
                 kv.second.second);
        out += line;
    }
    const size_t need = out.size() + 1;
    if (buf && len >= need) {        // delivered: start a new accumulation
        std::memcpy(buf, out.c_str(), need);
        hsa::g_acc.clear();
    } else if (buf && len) {
        buf[0] = '\0';
    }
    return (int)need;
}

}  // extern "C"
