// Run-time selection of the forward / summary kernel instantiation for a plan.
#include "bla_forward_inst.h"

namespace bla {

#define BLA_FWD_CASE(TT, DD, MMP, SSP) \
    if (p.D == DD && p.MP == MMP && p.SP == SSP) return Launch<TT, DD, MMP, SSP>::forward(p, a, s);
#define BLA_SUM_CASE(TT, DD, MMP, SSP) \
    if (p.D == DD && p.MP == MMP && p.SP == SSP) return Launch<TT, DD, MMP, SSP>::summary(p, a, s);
#define BLA_SUP_CASE(TT, DD, MMP, SSP)                                                             \
    if (D == DD && MP == MMP && SP == SSP)                                                          \
        return one_unit_fits<TT, DD, MMP, SSP>(C) || (C == kChunk && pair_units<TT, DD, MMP, SSP>() > 0);

hipError_t launch_forward(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    if (p.bf16) {
        BLA_FOR_EACH_SHAPE(BLA_FWD_CASE, bf16)
    } else {
        BLA_FOR_EACH_SHAPE(BLA_FWD_CASE, float)
    }
    return hipErrorInvalidValue;
}

hipError_t launch_summary(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    if (p.bf16) {
        BLA_FOR_EACH_SHAPE(BLA_SUM_CASE, bf16)
    } else {
        BLA_FOR_EACH_SHAPE(BLA_SUM_CASE, float)
    }
    return hipErrorInvalidValue;
}

#define BLA_UNITS_CASE(TT, DD, MMP, SSP) \
    if (D == DD && MP == MMP && SP == SSP) return pair_units<TT, DD, MMP, SSP>();

int forward_units_per_wg(int is_bf16, int D, int MP, int SP)
{
    if (is_bf16) {
        BLA_FOR_EACH_SHAPE(BLA_UNITS_CASE, bf16)
    }
    return 0;
}

bool forward_supported(int is_bf16, int D, int MP, int SP, int C)
{
    if (is_bf16) {
        BLA_FOR_EACH_SHAPE(BLA_SUP_CASE, bf16)
    } else {
        BLA_FOR_EACH_SHAPE(BLA_SUP_CASE, float)
    }
    return false;
}

}  // namespace bla
