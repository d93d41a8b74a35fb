// Pruned 3x3 conv, wave-pipeline kernel, canonical library, stride 2, dilation 2.
#include "conv_pp_wave_inst.hpp"

namespace pp {
PP_WAVE_INSTANTIATE(kLibCanon8, 2, 2)
}  // namespace pp
