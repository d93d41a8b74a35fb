// Pruned 3x3 conv for the dense library {0x1FF} and for any other pattern
// library (taps tested at run time), all strides and dilations.
#include "conv_pp_inst.hpp"

namespace pp {
PP_INSTANTIATE(kLibDense9, 1, 1)
PP_INSTANTIATE(kLibDense9, 2, 1)
PP_INSTANTIATE(kLibDense9, 1, 2)
PP_INSTANTIATE(kLibDense9, 2, 2)
PP_INSTANTIATE(kLibGeneric, 1, 1)
PP_INSTANTIATE(kLibGeneric, 2, 1)
PP_INSTANTIATE(kLibGeneric, 1, 2)
PP_INSTANTIATE(kLibGeneric, 2, 2)
}  // namespace pp
