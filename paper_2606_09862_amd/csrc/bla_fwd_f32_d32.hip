// Instantiations: float operands, head width 32.
#include "bla_forward_inst.h"
BLA_INSTANTIATE(float, 32, 16, 32)
BLA_INSTANTIATE(float, 32, 32, 32)
BLA_INSTANTIATE(float, 32, 32, 64)
BLA_INSTANTIATE(float, 32, 64, 32)
BLA_INSTANTIATE(float, 32, 64, 64)
BLA_INSTANTIATE(float, 32, 64, 128)
BLA_INSTANTIATE(float, 32, 128, 32)
BLA_INSTANTIATE(float, 32, 128, 64)
BLA_INSTANTIATE(float, 32, 128, 128)
BLA_INSTANTIATE(float, 32, 128, 256)
