// Backward instantiations, bf16 operands (head widths 32 and 64): the kernels of
// bla_backward_bf16.h, with every table of the chunk loop in LDS.
#include "bla_backward_bf16.h"

namespace bla {

hipError_t launch_backward_bf16(int D, int MP, int SP, const BwdArgs& a, hipStream_t s, void* const* ev)
{
#define BLA_BWD(DD, MM, SS) \
    if (D == DD && MP == MM && SP == SS) return launch_backward16_shape<DD, MM, SS>(a, s, ev);
    BLA_BWD(32, 16, 32)
    BLA_BWD(32, 32, 32)
    BLA_BWD(32, 32, 64)
    BLA_BWD(32, 64, 32)
    BLA_BWD(32, 64, 64)
    BLA_BWD(32, 64, 128)
    BLA_BWD(64, 16, 32)
    BLA_BWD(64, 32, 32)
    BLA_BWD(64, 32, 64)
    BLA_BWD(64, 64, 32)
    BLA_BWD(64, 64, 64)
    BLA_BWD(64, 64, 128)
#undef BLA_BWD
    return hipErrorInvalidValue;
}

}  // namespace bla
