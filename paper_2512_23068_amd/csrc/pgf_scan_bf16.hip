// The scan kernels and their launch sequence for bf16 (uint16_t bit patterns) inputs.
#include "pgf_scan_kernels.h"

namespace pgf {

template int launch<uint16_t>(const Plan &, const pgf_params &, const uint16_t *, const uint16_t *, float *, float *, float *,
                        hipStream_t, const float *, float *, float *, float *);

template bool launch_supported<uint16_t>(const Plan &, const pgf_params &);

}  // namespace pgf
