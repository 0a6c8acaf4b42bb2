// Instantiations: float32 operands, head width 128 (built without VGPR-form accumulators,
// which the compiler cannot build for this unit).
#include "bla_forward_inst.h"
BLA_INSTANTIATE(float, 128, 16, 32)
BLA_INSTANTIATE(float, 128, 32, 32)
BLA_INSTANTIATE(float, 128, 32, 64)
BLA_INSTANTIATE(float, 128, 64, 32)
BLA_INSTANTIATE(float, 128, 64, 64)
BLA_INSTANTIATE(float, 128, 64, 128)
BLA_INSTANTIATE(float, 128, 128, 32)
BLA_INSTANTIATE(float, 128, 128, 64)
BLA_INSTANTIATE(float, 128, 128, 128)
BLA_INSTANTIATE(float, 128, 128, 256)
