// Single-token recurrent decode (one iteration of Alg. 2's loop) for gfx950.
//
// One workgroup per (b, h).  The step streams the float32 states in and out once
// (4 M d floats each way) and is bound by HBM; everything else is kept off the
// memory path:
//   Z[m] <- rho_m Z[m] + x                          (Sec. 3.1, the mode recurrence)
//   u[m] = <q, Z_k[m]>                              (reduced over d across lanes)
//   z_s = scale sum_m c_m (cos_k Re u[m] + sin_k Im u[m]),  k = m s mod S, masked
//   p = softmax(z);  a_m = c_m sum_s p_s cos_k,  b_m = c_m sum_s p_s sin_k
//   o = sum_m a_m Re Z_v[m] + b_m Im Z_v[m]
// The slot matrices A[s,m] = c_m cos(2 pi m s / S), B[s,m] = c_m sin(2 pi m s / S)
// (Eq. for the interpolation at tau_s = s T / S) are generated from one table of
// cos | sin(2 pi k / S), k < S, held in LDS; the slot and mode sums are split over
// all waves of the workgroup.
//
// Anchored slots (Sec. 3.3, Alg. 1) read the same mode state at the absolute phase of the
// token: with rho^p = exp(i m w p), the anchored mode state is rho^p conj(Z), so
//   u <- rho^p conj(u)                         before the scores, and
//   (a_m, b_m) <- (a c + b s, a s - b c)        (c + i s = rho^p) before the output sum.
#include <math.h>
#include <stdint.h>

#include "bla_device.h"
#include "bla_plan.h"

namespace bla {

template <int D, int MP> struct StepGeo {
    static constexpr int NT = MP * D <= 4096 ? 256 : 512;
    static constexpr int NQ = D / 4;                        // threads per state row (4 floats each)
    static constexpr int RPP = NT / NQ;                     // state rows (modes) per pass
    static constexpr int PASSES = (MP + RPP - 1) / RPP;     // passes over the modes
};

template <int D, int MP> constexpr int step_threads() { return StepGeo<D, MP>::NT; }

template <typename T, int D, int MP>
__global__ __launch_bounds__((StepGeo<D, MP>::NT)) void step_kernel(StepArgs a)
{
    using G = StepGeo<D, MP>;
    constexpr int NT = G::NT, NQ = G::NQ, RPP = G::RPP, PASSES = G::PASSES;
    __shared__ float strig[2 * 256];       // cos | sin of 2 pi k / S
    __shared__ float su[2 * MP];           // Re u | Im u
    __shared__ float spart[2 * NT];        // partial sums (scores, then readout coefficients)
    __shared__ float sp[256];              // slot probabilities
    __shared__ float sab[2 * MP];          // a | b
    __shared__ __attribute__((aligned(16))) float sred[RPP * D];

    const int bh = blockIdx.x, b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x, rg = tid / NQ, qd = tid % NQ;
    const int M = a.M, S = a.S, SP = a.SP;
    const long long pos = a.pos ? (long long)a.pos[b] : a.t0;
    const float* E1 = a.E32 + ((size_t)h * (kChunk + 1) + 1) * 2 * MP;
    float* skb = a.sk + (size_t)bh * 2 * M * D;
    float* svb = a.sv + (size_t)bh * 2 * M * D;

    // every state load of the workgroup up front (16-byte, coalesced along d); the loads
    // are unconditional (rows past M re-read row M - 1 and are ignored), so none of them
    // waits for another.  Offsets within one (b, h) state are 32-bit on a uniform base.
    floatx4 kc[PASSES], ks[PASSES], vc[PASSES], vs[PASSES];
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int mc = min(ps * RPP + rg, M - 1);
        kc[ps] = ld4f(skb + (unsigned)(mc * D + 4 * qd));
        ks[ps] = ld4f(skb + (unsigned)((M + mc) * D + 4 * qd));
        vc[ps] = ld4f(svb + (unsigned)(mc * D + 4 * qd));
        vs[ps] = ld4f(svb + (unsigned)((M + mc) * D + 4 * qd));
    }
    const floatx4 q4 = to_f4(ld4<T>((const T*)a.q + (size_t)bh * D + 4 * qd));
    const floatx4 k4 = to_f4(ld4<T>((const T*)a.k + (size_t)bh * D + 4 * qd));
    const floatx4 v4 = to_f4(ld4<T>((const T*)a.v + (size_t)bh * D + 4 * qd));
    for (int i = tid; i < 2 * SP; i += NT) strig[i] = a.trig[i];

    // state update, written back, and the per-mode query products
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int m = ps * RPP + rg;
        const bool valid = m < M;
        const int mc = min(m, M - 1);
        const float rc = E1[mc], rs = E1[MP + mc];
        const floatx4 nc = rc * kc[ps] - rs * ks[ps] + k4;
        const floatx4 ns = rs * kc[ps] + rc * ks[ps];
        const floatx4 wc = rc * vc[ps] - rs * vs[ps] + v4;
        const floatx4 ws = rs * vc[ps] + rc * vs[ps];
        float uc = q4[0] * nc[0] + q4[1] * nc[1] + q4[2] * nc[2] + q4[3] * nc[3];
        float us = q4[0] * ns[0] + q4[1] * ns[1] + q4[2] * ns[2] + q4[3] * ns[3];
        vc[ps] = wc;
        vs[ps] = ws;
        if (valid) {
            st4f(skb + (unsigned)(m * D + 4 * qd), nc);
            st4f(skb + (unsigned)((M + m) * D + 4 * qd), ns);
            st4f(svb + (unsigned)(m * D + 4 * qd), wc);
            st4f(svb + (unsigned)((M + m) * D + 4 * qd), ws);
        } else {
            uc = us = 0.f;
        }
        // the NQ threads of a row are consecutive lanes of one wave
#pragma unroll
        for (int off = NQ / 2; off > 0; off >>= 1) {
            uc += __shfl_xor(uc, off);
            us += __shfl_xor(us, off);
        }
        if (qd == 0 && m < MP) {
            if (a.anchor) {
                float c = 0.f, s = 0.f;
                if (m < M) anchor_phase(m, pos, a.rperiod[h], c, s);
                const float rc_ = c * uc + s * us, rs_ = s * uc - c * us;
                uc = rc_;
                us = rs_;
            }
            su[m] = uc;
            su[MP + m] = us;
        }
    }
    __syncthreads();

    // scores: thread (p, s) sums modes [p * mlen, (p + 1) * mlen) of slot s
    const float cnorm = 1.f / (2.f * M - 1.f);
    {
        const int parts = NT / SP, s = tid % SP, p = tid / SP;
        const int mlen = (M + parts - 1) / parts, m0 = p * mlen, m1 = min(M, m0 + mlen);
        float z = 0.f;
        if (s < S && m0 < m1) {
            int k = (int)(((long long)m0 * s) % S);
#pragma unroll 4
            for (int m = m0; m < m1; ++m) {
                const float c = m == 0 ? cnorm : 2.f * cnorm;
                z += c * (strig[k] * su[m] + strig[SP + k] * su[MP + m]);
                k += s;
                if (k >= S) k -= S;
            }
        }
        spart[p * SP + s] = z;
    }
    __syncthreads();
    if (tid < SP) {
        float z = 0.f;
        for (int p = 0; p < NT / SP; ++p) z += spart[p * SP + tid];
        z *= a.scale;
        if (tid >= S || pos < (long long)a.theta[(size_t)h * SP + tid]) z = -INFINITY;
        sp[tid] = z;
    }
    __syncthreads();
    if (tid < 64) {
        float mx = -INFINITY;
        for (int s = tid; s < SP; s += 64) mx = fmaxf(mx, sp[s]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float sum = 0.f;
        for (int s = tid; s < SP; s += 64) {
            const float e = __expf(sp[s] - mx);
            sp[s] = e;
            sum += e;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off);
        const float inv = 1.f / sum;
        for (int s = tid; s < SP; s += 64) sp[s] *= inv;
    }
    __syncthreads();

    // readout coefficients: thread (p, m) sums slots [p * slen, (p + 1) * slen) of mode m
    {
        const int parts = NT / MP, m = tid % MP, p = tid / MP;
        const int slen = (S + parts - 1) / parts, s0 = p * slen, s1 = min(S, s0 + slen);
        float ca = 0.f, cb = 0.f;
        if (m < M && s0 < s1) {
            int k = (int)(((long long)m * s0) % S);
#pragma unroll 4
            for (int s = s0; s < s1; ++s) {
                ca += sp[s] * strig[k];
                cb += sp[s] * strig[SP + k];
                k += m;
                if (k >= S) k -= S;
            }
        }
        spart[p * MP + m] = ca;
        spart[NT + p * MP + m] = cb;
    }
    __syncthreads();
    if (tid < MP) {
        float ca = 0.f, cb = 0.f;
        for (int p = 0; p < NT / MP; ++p) {
            ca += spart[p * MP + tid];
            cb += spart[NT + p * MP + tid];
        }
        const float c = tid == 0 ? cnorm : 2.f * cnorm;
        if (a.anchor) {
            float pc = 0.f, ps = 0.f;
            if (tid < M) anchor_phase(tid, pos, a.rperiod[h], pc, ps);
            const float na = pc * ca + ps * cb, nb = ps * ca - pc * cb;
            ca = na;
            cb = nb;
        }
        sab[tid] = c * ca;
        sab[MP + tid] = c * cb;
    }
    __syncthreads();

    floatx4 o4 = zero4();
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int m = ps * RPP + rg;
        if (m < M) o4 += sab[m] * vc[ps] + sab[MP + m] * vs[ps];
    }
    st4f(sred + (size_t)rg * D + 4 * qd, o4);
    __syncthreads();
    for (int d = tid; d < D; d += NT) {
        float acc = 0.f;
        for (int g = 0; g < RPP; ++g) acc += sred[(size_t)g * D + d];
        ((T*)a.o)[(size_t)bh * D + d] = (T)acc;
    }
}

template <typename T, int D>
hipError_t launch_step_d(const Plan& p, const StepArgs& a, hipStream_t s)
{
    dim3 grid((unsigned)(p.B * p.H));
#define BLA_STEP_MP(MMP)                                                                                 \
    if (p.MP == MMP) {                                                                                   \
        hipLaunchKernelGGL((step_kernel<T, D, MMP>), grid, dim3(step_threads<D, MMP>()), 0, s, a);       \
        return hipGetLastError();                                                                        \
    }
    BLA_STEP_MP(16)
    BLA_STEP_MP(32)
    BLA_STEP_MP(64)
    BLA_STEP_MP(128)
#undef BLA_STEP_MP
    return hipErrorInvalidValue;
}

hipError_t launch_step(const Plan& p, const StepArgs& a, hipStream_t s)
{
    if (p.bf16) {
        if (p.D == 32) return launch_step_d<bf16, 32>(p, a, s);
        if (p.D == 64) return launch_step_d<bf16, 64>(p, a, s);
        if (p.D == 128) return launch_step_d<bf16, 128>(p, a, s);
    } else {
        if (p.D == 32) return launch_step_d<float, 32>(p, a, s);
        if (p.D == 64) return launch_step_d<float, 64>(p, a, s);
        if (p.D == 128) return launch_step_d<float, 128>(p, a, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace bla
