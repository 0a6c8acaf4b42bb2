// Dispatch over the instantiated forward shapes for one operand type.
//
// Shapes: head width D in {32, 64, 128}; padded modes MP in {16, 32, 64, 128};
// padded slots SP in {32, 64, 128, 256} with SP <= max(32, 2 MP).  A shape whose
// LDS tiles exceed the 160 KB of a gfx950 workgroup is reported unsupported.
#pragma once

#include "bla_forward.h"

#define BLA_FOR_EACH_MS(X, T, D) \
    X(T, D, 16, 32)              \
    X(T, D, 32, 32)              \
    X(T, D, 32, 64)              \
    X(T, D, 64, 32)              \
    X(T, D, 64, 64)              \
    X(T, D, 64, 128)             \
    X(T, D, 128, 32)             \
    X(T, D, 128, 64)             \
    X(T, D, 128, 128)            \
    X(T, D, 128, 256)

#define BLA_FOR_EACH_SHAPE(X, T) \
    BLA_FOR_EACH_MS(X, T, 32)    \
    BLA_FOR_EACH_MS(X, T, 64)    \
    BLA_FOR_EACH_MS(X, T, 128)

namespace bla {

template <typename T, int D, int MP, int SP> constexpr bool fits()
{
    return Fwd<T, D, MP, SP>::LDS_BYTES <= kMaxLds;
}

template <typename T, int D, int MP, int SP>
hipError_t launch_forward_t(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    if constexpr (fits<T, D, MP, SP>()) {
        hipLaunchKernelGGL((forward_kernel<T, D, MP, SP>), dim3((unsigned)(p.B * p.H * p.nseg)),
                           dim3(kThreads), 0, s, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <typename T, int D, int MP>
hipError_t launch_summary_t(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    hipLaunchKernelGGL((summary_kernel<T, D, MP>), dim3((unsigned)(p.B * p.H * p.nbs)), dim3(kThreads),
                       0, s, a);
    return hipGetLastError();
}

}  // namespace bla

// Defines launch_forward_<NAME>, launch_summary_<NAME>, forward_supported_<NAME>.
#define BLA_DEFINE_DISPATCH(T, NAME)                                                         \
    namespace bla {                                                                          \
    hipError_t launch_forward_##NAME(const Plan& p, const FwdArgs& a, hipStream_t s)         \
    {                                                                                        \
        BLA_FOR_EACH_SHAPE(BLA_FWD_CASE, T)                                                  \
        return hipErrorInvalidValue;                                                         \
    }                                                                                        \
    hipError_t launch_summary_##NAME(const Plan& p, const FwdArgs& a, hipStream_t s)         \
    {                                                                                        \
        BLA_FOR_EACH_SHAPE(BLA_SUM_CASE, T)                                                  \
        return hipErrorInvalidValue;                                                         \
    }                                                                                        \
    bool forward_supported_##NAME(int D, int MP, int SP)                                     \
    {                                                                                        \
        BLA_FOR_EACH_SHAPE(BLA_SUP_CASE, T)                                                  \
        return false;                                                                        \
    }                                                                                        \
    }

#define BLA_FWD_CASE(TT, DD, MMP, SSP) \
    if (p.D == DD && p.MP == MMP && p.SP == SSP) return launch_forward_t<TT, DD, MMP, SSP>(p, a, s);
#define BLA_SUM_CASE(TT, DD, MMP, SSP) \
    if (p.D == DD && p.MP == MMP && p.SP == SSP) return launch_summary_t<TT, DD, MMP>(p, a, s);
#define BLA_SUP_CASE(TT, DD, MMP, SSP) \
    if (D == DD && MP == MMP && SP == SSP) return fits<TT, DD, MMP, SSP>();
