// Instantiations: bf16 operands, head width 128.
#include "bla_forward_inst.h"
BLA_INSTANTIATE(bf16, 128, 16, 32)
BLA_INSTANTIATE(bf16, 128, 32, 32)
BLA_INSTANTIATE(bf16, 128, 32, 64)
BLA_INSTANTIATE(bf16, 128, 64, 32)
BLA_INSTANTIATE(bf16, 128, 64, 64)
BLA_INSTANTIATE(bf16, 128, 64, 128)
