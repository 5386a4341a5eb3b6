// launch_f32_hi.hip -- kernels and launch sequence for float inputs with
// F = 9..16 harmonics per axis (one translation unit per range so that
// the instantiations compile in parallel).
#include "launch.hpp"

namespace cpe {
CPE_LAUNCH_RANGE(launch_f32_hi, float, 9)
}  // namespace cpe
