// Instantiations: bf16 operands, head width 128, M padded to 128 (every slot padding).
// Built without VGPR-form accumulators (the compiler cannot build these with them).
#include "bla_forward_inst.h"
BLA_INSTANTIATE(bf16, 128, 128, 32)
BLA_INSTANTIATE(bf16, 128, 128, 64)
BLA_INSTANTIATE(bf16, 128, 128, 128)
BLA_INSTANTIATE(bf16, 128, 128, 256)
