// Backward instantiations, float32 operands (head width 32), and the dispatch by dtype.
#include "bla_backward.h"

namespace bla {

hipError_t launch_backward_bf16(int D, int MP, int SP, const BwdArgs& a, hipStream_t s, void* const* ev);

hipError_t launch_backward(int is_bf16, int D, int MP, int SP, const BwdArgs& a, hipStream_t s, void* const* ev)
{
    if (is_bf16) return launch_backward_bf16(D, MP, SP, a, s, ev);
#define BLA_BWD(DD, MM, SS) \
    if (D == DD && MP == MM && SP == SS) return launch_backward_shape<float, DD, MM, SS>(a, s, ev);
    BLA_BWD(32, 16, 32)
    BLA_BWD(32, 32, 32)
    BLA_BWD(32, 32, 64)
#undef BLA_BWD
    return hipErrorInvalidValue;
}

}  // namespace bla
