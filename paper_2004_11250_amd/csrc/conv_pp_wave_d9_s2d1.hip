// Pruned 3x3 conv, wave-pipeline kernel, all-ones (dense 3x3) library, stride 2, dilation 1.
#include "conv_pp_wave_inst.hpp"

namespace pp {
PP_WAVE_INSTANTIATE(kLibDense9, 2, 1)
}  // namespace pp
