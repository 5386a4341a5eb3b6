// launch_f16_hi.hip -- kernels and launch sequence for _Float16 inputs with
// F = 9..16 harmonics per axis (one translation unit per range so that
// the instantiations compile in parallel).
#include "launch.hpp"

namespace cpe {
CPE_LAUNCH_RANGE(launch_f16_hi, _Float16, 9)
}  // namespace cpe
