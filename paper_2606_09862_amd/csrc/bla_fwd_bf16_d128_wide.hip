// Instantiations: bf16 operands, head width 128, M padded to 128 with S padded to 32, 64
// or 256.  Built without VGPR-form accumulators (the compiler cannot build these three).
#include "bla_forward_inst.h"
BLA_INSTANTIATE(bf16, 128, 128, 32)
BLA_INSTANTIATE(bf16, 128, 128, 64)
BLA_INSTANTIATE(bf16, 128, 128, 256)
