// Launch wrappers of the forward kernels and the list of instantiated shapes.
//
// Shapes: head width D in {32, 64, 128}; padded modes MP in {16, 32, 64, 128};
// padded slots SP in {32, 64, 128, 256} with SP <= max(32, 2 MP).  A shape whose
// LDS tiles exceed the 160 KB of a gfx950 workgroup is reported unsupported.
// Each group of shapes is instantiated in its own translation unit (bla_fwd_*.hip)
// so that the units compile in parallel and can take their own compiler options;
// bla_forward_dispatch.hip selects the instantiation at run time.
#pragma once

#include "bla_forward.h"
#include "bla_forward_pair.h"

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

template <typename T, int D, int MP, int SP, int CC = kChunk> constexpr bool fits()
{
    return Fwd<T, D, MP, SP, CC>::LDS_BYTES <= kMaxLds;
}

// Chunk lengths other than the default 64 run on the one-unit kernels and are built for
// M <= 64 (padded modes up to 64), where their tiles and registers fit.
template <int MP, int CC> constexpr bool chunk_built() { return CC == kChunk || MP <= 64; }

template <typename T, int D, int MP, int SP, int CC>
hipError_t launch_one_unit(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    if constexpr (chunk_built<MP, CC>() && fits<T, D, MP, SP, CC>()) {
        const dim3 grid((unsigned)(p.B * p.H * p.nseg));
        if (a.anchor)
            hipLaunchKernelGGL((forward_kernel<T, D, MP, SP, true, CC>), grid, dim3(Geo<T, D, MP, CC>::NTHR), 0, s, a);
        else
            hipLaunchKernelGGL((forward_kernel<T, D, MP, SP, false, CC>), grid, dim3(Geo<T, D, MP, CC>::NTHR), 0, s, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

template <typename T, int D, int MP, int CC>
hipError_t launch_one_summary(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    if constexpr (chunk_built<MP, CC>()) {
        hipLaunchKernelGGL((summary_kernel<T, D, MP, CC>), dim3((unsigned)(p.B * p.H * p.nbs)),
                           dim3(Geo<T, D, MP, CC>::NTHR), 0, s, a);
        return hipGetLastError();
    } else {
        return hipErrorInvalidValue;
    }
}

// Whether the one-unit forward kernel exists for a shape and chunk length.
template <typename T, int D, int MP, int SP> bool one_unit_fits(int C)
{
    switch (C) {
    case 16: return chunk_built<MP, 16>() && fits<T, D, MP, SP, 16>();
    case 32: return chunk_built<MP, 32>() && fits<T, D, MP, SP, 32>();
    case 64: return fits<T, D, MP, SP, 64>();
    case 128: return chunk_built<MP, 128>() && fits<T, D, MP, SP, 128>();
    }
    return false;
}

template <typename T, int D, int MP, int SP> struct Launch {
    static hipError_t forward(const Plan& p, const FwdArgs& a, hipStream_t s);
    static hipError_t summary(const Plan& p, const FwdArgs& a, hipStream_t s);
};

// Units per workgroup of the bf16 pair kernel for a shape (0: the shape uses forward_kernel).
template <typename T, int D, int MP, int SP> constexpr int pair_units()
{
    if constexpr (sizeof(T) == 2) {
        return Pair<D, MP, SP>::FITS ? Pair<D, MP, SP>::U : 0;
    } else {
        return 0;
    }
}

}  // namespace bla

// Defines the launchers of one shape (used by the bla_fwd_*.hip units).
#define BLA_INSTANTIATE(T, D, MP, SP)                                                                   \
    namespace bla {                                                                                     \
    template <> hipError_t Launch<T, D, MP, SP>::forward(const Plan& p, const FwdArgs& a, hipStream_t s) \
    {                                                                                                   \
        if constexpr (pair_units<T, D, MP, SP>() > 0) {                                                 \
            if (p.pair) {                                                                               \
                constexpr int UU = pair_units<T, D, MP, SP>();                                          \
                dim3 grid((unsigned)((p.B * p.nseg + UU - 1) / UU), (unsigned)p.H);                     \
                if (a.anchor)                                                                           \
                    hipLaunchKernelGGL((forward_pair_kernel<D, MP, SP, true>), grid, dim3(256 * UU), 0, s, a); \
                else                                                                                    \
                    hipLaunchKernelGGL((forward_pair_kernel<D, MP, SP, false>), grid, dim3(256 * UU), 0, s, a); \
                return hipGetLastError();                                                               \
            }                                                                                           \
        }                                                                                               \
        switch (p.C) {                                                                                  \
        case 16: return launch_one_unit<T, D, MP, SP, 16>(p, a, s);                                     \
        case 32: return launch_one_unit<T, D, MP, SP, 32>(p, a, s);                                     \
        case 64: return launch_one_unit<T, D, MP, SP, 64>(p, a, s);                                     \
        case 128: return launch_one_unit<T, D, MP, SP, 128>(p, a, s);                                   \
        }                                                                                               \
        return hipErrorInvalidValue;                                                                    \
    }                                                                                                   \
    template <> hipError_t Launch<T, D, MP, SP>::summary(const Plan& p, const FwdArgs& a, hipStream_t s) \
    {                                                                                                   \
        if constexpr (pair_units<T, D, MP, SP>() > 0) {                                                 \
            if (p.pair) {                                                                               \
                hipLaunchKernelGGL((summary_pair_kernel<D, MP>),                                        \
                                   dim3((unsigned)summary_grid_x<D, MP>((long long)p.B * p.nbs), (unsigned)p.H),  \
                                   dim3(summary_threads<D, MP>()), 0, s, a);                            \
                return hipGetLastError();                                                               \
            }                                                                                           \
        }                                                                                               \
        if constexpr (sizeof(T) == 2) {                                                                 \
            if (p.C == kChunk) { /* bf16, 64-token chunks: the sliced summary kernel */                 \
                hipLaunchKernelGGL((summary_pair_kernel<D, MP, true>),                                  \
                                   dim3((unsigned)summary_grid_x<D, MP>((long long)p.B * p.nbs), (unsigned)p.H),  \
                                   dim3(summary_threads<D, MP>()), 0, s, a);                            \
                return hipGetLastError();                                                               \
            }                                                                                           \
        }                                                                                               \
        switch (p.C) {                                                                                  \
        case 16: return launch_one_summary<T, D, MP, 16>(p, a, s);                                      \
        case 32: return launch_one_summary<T, D, MP, 32>(p, a, s);                                      \
        case 64: return launch_one_summary<T, D, MP, 64>(p, a, s);                                      \
        case 128: return launch_one_summary<T, D, MP, 128>(p, a, s);                                    \
        }                                                                                               \
        return hipErrorInvalidValue;                                                                    \
    }                                                                                                   \
    }
