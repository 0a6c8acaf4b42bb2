// Instantiations: float operands, head width 64.
#include "bla_forward_inst.h"
BLA_INSTANTIATE(float, 64, 16, 32)
BLA_INSTANTIATE(float, 64, 32, 32)
BLA_INSTANTIATE(float, 64, 32, 64)
BLA_INSTANTIATE(float, 64, 64, 32)
BLA_INSTANTIATE(float, 64, 64, 64)
BLA_INSTANTIATE(float, 64, 64, 128)
BLA_INSTANTIATE(float, 64, 128, 32)
BLA_INSTANTIATE(float, 64, 128, 64)
BLA_INSTANTIATE(float, 64, 128, 128)
BLA_INSTANTIATE(float, 64, 128, 256)
