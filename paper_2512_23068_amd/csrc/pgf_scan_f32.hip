// The scan kernels and their launch sequence for f32 inputs.
#include "pgf_scan_kernels.h"

namespace pgf {

template int launch<float>(const Plan &, const pgf_params &, const float *, const float *, float *, float *, float *,
                        hipStream_t, const float *, float *, float *, float *);

template bool launch_supported<float>(const Plan &, const pgf_params &);

}  // namespace pgf
