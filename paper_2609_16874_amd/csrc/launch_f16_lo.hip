// launch_f16_lo.hip -- kernels and launch sequence for _Float16 inputs with
// F = 1..8 harmonics per axis (one translation unit per range so that
// the instantiations compile in parallel).
#include "launch.hpp"

namespace cpe {
CPE_LAUNCH_RANGE(launch_f16_lo, _Float16, 1)
}  // namespace cpe
