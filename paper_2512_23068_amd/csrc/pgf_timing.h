// Launch timing of libpgf (a measurement aid behind pgf_timing_enable):
// while timing is on, a Timed object brackets one kernel launch with HIP
// events on the launch's stream; pgf_timing_read sums the elapsed times per
// kind (the PGF_TIMING_KINDS slots of include/pgf.h).
#pragma once

#include <hip/hip_runtime.h>

namespace pgf {

class Timed {
public:
    // on = false: records nothing whatever pgf_timing_enable says (calls
    // that may not create events).
    Timed(int kind, hipStream_t st, bool on = true);
    ~Timed();
    Timed(const Timed &) = delete;
    Timed &operator=(const Timed &) = delete;

private:
    int kind_;
    hipStream_t st_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

}  // namespace pgf
