// Per-device helper streams of libpgf (see pgf_stream.h).  They live until
// the process ends.
#include "pgf_stream.h"

namespace pgf {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
Helper *g_helpers[kMaxDevices] = {};
bool g_failed[kMaxDevices] = {};
}  // namespace

Helper *helper() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_helpers[dev] || g_failed[dev]) return g_helpers[dev];
    Helper *h = new Helper;
    if (hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&h->fork, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&h->join, hipEventDisableTiming) != hipSuccess) {
        // Leave no half-made helper behind; clear the error for the caller.
        if (h->fork) (void)hipEventDestroy(h->fork);
        if (h->side) (void)hipStreamDestroy(h->side);
        delete h;
        (void)hipGetLastError();
        g_failed[dev] = true;
        return nullptr;
    }
    g_helpers[dev] = h;
    return h;
}

}  // namespace pgf
