// Pruned 3x3 conv, canonical 8-pattern library, stride 2, dilation 2.
#include "conv_pp_inst.hpp"

namespace pp {
PP_INSTANTIATE(kLibCanon8, 2, 2)
}  // namespace pp
