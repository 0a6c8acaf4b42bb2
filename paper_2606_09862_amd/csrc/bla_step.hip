// Single-token recurrent decode (one iteration of Alg. 2's loop) for gfx950.
//
// One 256-thread workgroup per (b, h).  The step is bound by HBM: it streams the
// float32 states in and out once (4 M d floats each way) and does ~1 flop per
// byte.  Threads own (mode, 4-wide d slice) pieces of the states, so every state
// access is a coalesced 16-byte load/store and every state element is read and
// written exactly once:
//   Z[m] <- rho_m Z[m] + x                       (Sec. 3.1 Eq. recurrence)
//   u[m] = <q, Z_k[m]>                           (reduced over d across lanes)
//   z_s = scale sum_m A[s,m] Re u[m] + B[s,m] Im u[m], masked (Eq. compressed/output)
//   p = softmax(z);  a = A^T p, b = B^T p;  o = sum_m a_m Vcos[m] + b_m Vsin[m]
#include <math.h>
#include <stdint.h>

#include "bla_device.h"
#include "bla_plan.h"

namespace bla {

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void step_kernel(StepArgs a, int MP, int SP)
{
    constexpr int NQ = D / 4;             // 4-wide slices per row
    constexpr int RPP = kThreads / NQ;    // rows (modes) per pass
    constexpr int MAXPASS = 128 / RPP;    // enough passes for MP <= 128
    __shared__ float su[2 * 128];
    __shared__ float sz[256];
    __shared__ float sab[2 * 128];
    __shared__ __attribute__((aligned(16))) float sred[RPP * D];

    const int bh = blockIdx.x, b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x, rg = tid / NQ, qd = tid % NQ;
    const int M = a.M;
    const long long pos = a.pos ? (long long)a.pos[b] : a.t0;
    const floatx4 q4 = to_f4(ld4<T>((const T*)a.q + (size_t)bh * D + 4 * qd));
    const floatx4 k4 = to_f4(ld4<T>((const T*)a.k + (size_t)bh * D + 4 * qd));
    const floatx4 v4 = to_f4(ld4<T>((const T*)a.v + (size_t)bh * D + 4 * qd));
    const float* E1 = a.E32 + ((size_t)h * (kChunk + 1) + 1) * 2 * MP;
    float* skb = a.sk + (size_t)bh * 2 * M * D;
    float* svb = a.sv + (size_t)bh * 2 * M * D;

    floatx4 vc[MAXPASS], vs[MAXPASS];
#pragma unroll
    for (int ps = 0; ps < MAXPASS; ++ps) {
        vc[ps] = vs[ps] = zero4();
        const int m = ps * RPP + rg;
        if (m < MP) {
            float uc = 0.f, us = 0.f;
            if (m < M) {
                const float rc = E1[m], rs = E1[MP + m];
                const floatx4 c = ld4f(skb + (size_t)m * D + 4 * qd);
                const floatx4 s = ld4f(skb + (size_t)(M + m) * D + 4 * qd);
                const floatx4 nc = rc * c - rs * s + k4;
                const floatx4 ns = rs * c + rc * s;
                st4f(skb + (size_t)m * D + 4 * qd, nc);
                st4f(skb + (size_t)(M + m) * D + 4 * qd, ns);
                uc = q4[0] * nc[0] + q4[1] * nc[1] + q4[2] * nc[2] + q4[3] * nc[3];
                us = q4[0] * ns[0] + q4[1] * ns[1] + q4[2] * ns[2] + q4[3] * ns[3];
                const floatx4 c2 = ld4f(svb + (size_t)m * D + 4 * qd);
                const floatx4 s2 = ld4f(svb + (size_t)(M + m) * D + 4 * qd);
                vc[ps] = rc * c2 - rs * s2 + v4;
                vs[ps] = rs * c2 + rc * s2;
                st4f(svb + (size_t)m * D + 4 * qd, vc[ps]);
                st4f(svb + (size_t)(M + m) * D + 4 * qd, vs[ps]);
            }
#pragma unroll
            for (int off = NQ / 2; off > 0; off >>= 1) {
                uc += __shfl_xor(uc, off);
                us += __shfl_xor(us, off);
            }
            if (qd == 0) {
                su[m] = uc;
                su[MP + m] = us;
            }
        }
    }
    __syncthreads();

    for (int s = tid; s < SP; s += kThreads) {
        const float* row = a.AB32 + (size_t)s * 2 * MP;
        float z = 0.f;
        for (int m = 0; m < MP; ++m) z += row[m] * su[m] + row[MP + m] * su[MP + m];
        z *= a.scale;
        if (pos < (long long)a.theta[(size_t)h * SP + s]) z = -INFINITY;
        sz[s] = z;
    }
    __syncthreads();
    if (tid < 64) {
        float mx = -INFINITY;
        for (int s = tid; s < SP; s += 64) mx = fmaxf(mx, sz[s]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float sum = 0.f;
        for (int s = tid; s < SP; s += 64) {
            const float e = __expf(sz[s] - mx);
            sz[s] = e;
            sum += e;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
        const float inv = 1.f / sum;
        for (int s = tid; s < SP; s += 64) sz[s] *= inv;
    }
    __syncthreads();
    for (int m = tid; m < MP; m += kThreads) {
        float am = 0.f, bm = 0.f;
        for (int s = 0; s < SP; ++s) {
            am += sz[s] * a.AB32[(size_t)s * 2 * MP + m];
            bm += sz[s] * a.AB32[(size_t)s * 2 * MP + MP + m];
        }
        sab[m] = am;
        sab[MP + m] = bm;
    }
    __syncthreads();
    floatx4 o4 = zero4();
#pragma unroll
    for (int ps = 0; ps < MAXPASS; ++ps) {
        const int m = ps * RPP + rg;
        if (m < M) o4 += sab[m] * vc[ps] + sab[MP + m] * vs[ps];
    }
    st4f(sred + (size_t)rg * D + 4 * qd, o4);
    __syncthreads();
    for (int d = tid; d < D; d += kThreads) {
        float acc = 0.f;
        for (int g = 0; g < RPP; ++g) acc += sred[(size_t)g * D + d];
        ((T*)a.o)[(size_t)bh * D + d] = (T)acc;
    }
}

hipError_t launch_step(const Plan& p, const StepArgs& a, hipStream_t s)
{
    dim3 grid((unsigned)(p.B * p.H));
    const int MP = p.MP, SP = p.SP;
#define BLA_STEP_CASE(TT, DD)                                                              \
    hipLaunchKernelGGL((step_kernel<TT, DD>), grid, dim3(kThreads), 0, s, a, MP, SP);      \
    return hipGetLastError();
    if (p.bf16) {
        if (p.D == 32) { BLA_STEP_CASE(bf16, 32) }
        if (p.D == 64) { BLA_STEP_CASE(bf16, 64) }
        if (p.D == 128) { BLA_STEP_CASE(bf16, 128) }
    } else {
        if (p.D == 32) { BLA_STEP_CASE(float, 32) }
        if (p.D == 64) { BLA_STEP_CASE(float, 64) }
        if (p.D == 128) { BLA_STEP_CASE(float, 128) }
    }
#undef BLA_STEP_CASE
    return hipErrorInvalidValue;
}

}  // namespace bla
