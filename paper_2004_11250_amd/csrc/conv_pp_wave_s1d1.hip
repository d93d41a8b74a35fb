// Pruned 3x3 conv, wave-pipeline kernel, canonical library, stride 1, dilation 1.
#include "conv_pp_wave_inst.hpp"

namespace pp {
PP_WAVE_INSTANTIATE(kLibCanon8, 1, 1)
}  // namespace pp
