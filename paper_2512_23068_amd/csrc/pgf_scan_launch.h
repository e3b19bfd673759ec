// Launch sequence of one planned libpgf call (the kernels are in
// pgf_scan_kernels.h, instantiated once per input type in pgf_scan_f32.hip
// and pgf_scan_bf16.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pgf_plan.h"

namespace pgf {

// Enqueues every kernel of the call planned in q on stream st.  x, dx are
// f32 (InT = float) or bf16 bit patterns (InT = uint16_t); d2y is the
// second-order output, gy and gA, gB, gC the parameter flows' adjoint input
// and gradient outputs (NULL where the order does not use them).  The
// arguments have passed the entry points' checks.  Returns PGF_OK,
// PGF_ERR_UNSUPPORTED (no kernel for the planned tiling) or PGF_ERR_HIP.
template <typename InT>
int launch(const Plan &q, const pgf_params &p, const InT *x, const InT *dx, float *y, float *dy, float *d2y,
           hipStream_t st, const float *gy, float *gA, float *gB, float *gC);

// Whether launch() has a kernel for every step of the plan (no device
// work; the planner and the kernel tables must agree, and pgf_plan checks).
template <typename InT>
bool launch_supported(const Plan &q, const pgf_params &p);

extern template bool launch_supported<float>(const Plan &, const pgf_params &);
extern template bool launch_supported<uint16_t>(const Plan &, const pgf_params &);
extern template int launch<float>(const Plan &, const pgf_params &, const float *, const float *, float *, float *,
                                  float *, hipStream_t, const float *, float *, float *, float *);
extern template int launch<uint16_t>(const Plan &, const pgf_params &, const uint16_t *, const uint16_t *, float *,
                                     float *, float *, hipStream_t, const float *, float *, float *, float *);

}  // namespace pgf
