// Helper stream of libpgf: per device one extra stream (default priority,
// non-blocking) and two events, with which a call runs the projection of
// its next host block while the scans of the current one run on the
// caller's stream.  Host code only.
#pragma once

#include <hip/hip_runtime.h>

#include <mutex>

namespace pgf {

struct Helper {
    hipStream_t side = nullptr;
    hipEvent_t fork = nullptr;   // recorded on the caller's stream, waited for on side
    hipEvent_t join = nullptr;   // recorded on side, waited for on the caller's stream
    std::mutex mu;               // held by one call while it enqueues work on side
};

// The current device's helper, created on first use; nullptr if HIP cannot
// create it (the caller then runs everything on its own stream).
Helper *helper();

}  // namespace pgf
