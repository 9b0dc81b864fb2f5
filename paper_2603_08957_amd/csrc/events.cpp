// A pool of timing events per device.  Phase timing records a handful of
// events per call; creating and destroying them each time cost tens of
// microseconds of host time per call on small inputs, so released events
// go back to a free list of the device they were created on and are reused.
#include <mutex>
#include <unordered_map>
#include <vector>

#include "tre_internal.h"

namespace tre {

namespace {

constexpr size_t kPoolMax = 256;  // free events kept per device

std::mutex g_mu;
std::unordered_map<int, std::vector<hipEvent_t>> g_free;  // device -> free events
std::unordered_map<hipEvent_t, int> g_owner;              // event -> its device

}  // namespace

thread_local KernelEvents* t_kernel_events = nullptr;

hipEvent_t event_acquire() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto& f = g_free[dev];
        if (!f.empty()) {
            hipEvent_t e = f.back();
            f.pop_back();
            return e;
        }
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    g_owner[e] = dev;
    return e;
}

void event_release(hipEvent_t e) {
    if (!e) return;
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_owner.find(e);
    if (it == g_owner.end()) {
        (void)hipEventDestroy(e);
        return;
    }
    auto& f = g_free[it->second];
    if (f.size() < kPoolMax) {
        f.push_back(e);
        return;
    }
    g_owner.erase(it);
    (void)hipEventDestroy(e);
}

KernelEvents::~KernelEvents() {
    if (keep) return;
    event_release(start);
    event_release(stop);
}

}  // namespace tre
