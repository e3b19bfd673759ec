// Launch-timing registry of libpgf (see pgf_timing.h and pgf_timing_* in
// include/pgf.h).  Host code only.
#include "pgf_timing.h"

#include <mutex>
#include <vector>

#include "../../include/pgf.h"

namespace pgf {
namespace {

struct Registry {
    std::mutex mu;
    bool on = false;
    struct Rec {
        int kind;
        hipEvent_t a, b;
    };
    std::vector<Rec> recs;
    std::vector<hipEvent_t> pool;
};

Registry &registry() {
    static Registry r;
    return r;
}

// Caller holds the registry lock.
hipEvent_t take_event(Registry &r) {
    if (!r.pool.empty()) {
        hipEvent_t e = r.pool.back();
        r.pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

Timed::Timed(int kind, hipStream_t st, bool on) : kind_(kind), st_(st) {
    if (!on) return;
    Registry &r = registry();
    std::lock_guard<std::mutex> lk(r.mu);
    if (!r.on) return;
    a_ = take_event(r);
    b_ = take_event(r);
    if (a_) (void)hipEventRecord(a_, st_);
}

Timed::~Timed() {
    if (!a_ || !b_) return;
    (void)hipEventRecord(b_, st_);
    Registry &r = registry();
    std::lock_guard<std::mutex> lk(r.mu);
    r.recs.push_back({kind_, a_, b_});
}

}  // namespace pgf

extern "C" int pgf_timing_enable(int on) {
    pgf::Registry &r = pgf::registry();
    std::lock_guard<std::mutex> lk(r.mu);
    r.on = on != 0;
    return PGF_OK;
}

extern "C" int pgf_timing_read(double *ms, int64_t *launches) {
    pgf::Registry &r = pgf::registry();
    std::lock_guard<std::mutex> lk(r.mu);
    for (int i = 0; i < PGF_TIMING_KINDS; ++i) {
        if (ms) ms[i] = 0.0;
        if (launches) launches[i] = 0;
    }
    int rc = PGF_OK;
    for (auto &rec : r.recs) {
        float t = 0.0f;
        if (hipEventSynchronize(rec.b) != hipSuccess || hipEventElapsedTime(&t, rec.a, rec.b) != hipSuccess)
            rc = PGF_ERR_HIP;
        if (rec.kind >= 0 && rec.kind < PGF_TIMING_KINDS) {
            if (ms) ms[rec.kind] += t;
            if (launches) launches[rec.kind] += 1;
        }
        r.pool.push_back(rec.a);
        r.pool.push_back(rec.b);
    }
    r.recs.clear();
    return rc;
}
