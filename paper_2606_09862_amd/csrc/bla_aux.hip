// Table construction, the scan over block summaries, and state copies.
//
// Tables are built on the device in double precision (library sincos) from the
// exact integer phase m*j mod T, then rounded once to float32 / the operand type.
#include <math.h>
#include <stdint.h>

#include "bla_device.h"
#include "bla_plan.h"

namespace bla {

// 2 pi (m j mod T) / T, exact up to the final rounding of the division.
__device__ __forceinline__ double mode_phase(long long mj, double T)
{
    return 2.0 * M_PI * fmod((double)mj, T) / T;
}

// One thread per angle: a (head, j, m) phase with j = 0..C for the per-head tables,
// an (s, m) phase for the slot matrices, plus the per-head mask thresholds and
// block rotations.  Each sincos result is written to every table that uses it.
template <typename T>
__global__ __launch_bounds__(kThreads) void tables_kernel(TableArgs a)
{
    const int MP = a.MP, MP2 = 2 * MP, C = a.C;
    const int J = a.jrows;                                      // rows j = 0..J-1 (stride C + 1)
    const long long n_head = (long long)a.nh * J * MP;          // (h, j, m)
    const long long n_misc = (long long)a.nh * (a.SP + MP);     // theta, rotblk
    const long long n_ab = a.with_shared ? (long long)a.SP * MP : 0;
    const long long n_trig = a.with_shared ? (long long)a.SP : 0;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < n_head) {
        const int hl = (int)(gid / (J * MP));
        const int rem = (int)(gid % (J * MP));
        const int j = rem / MP, m = rem % MP, h = a.h0 + hl;
        double sn = 0.0, cs = 0.0;
        if (m < a.M) sincos(mode_phase((long long)m * j, a.T[hl]), &sn, &cs);
        float* E32 = a.E32 + (size_t)h * (C + 1) * MP2;
        E32[(size_t)j * MP2 + m] = (float)cs;
        E32[(size_t)j * MP2 + MP + m] = (float)sn;
        T* Etab = (T*)a.Etab + (size_t)h * C * MP2;
        if (j < C) {
            Etab[(size_t)j * MP2 + m] = (T)(float)cs;
            Etab[(size_t)j * MP2 + MP + m] = (T)(float)(a.conj_tab ? -sn : sn);
        }
        if (!a.conj_tab) {
            // the transposed tables of the one-unit kernels (the pair kernels read Etab transposed)
            T* EbarT = (T*)a.EbarT + (size_t)h * MP2 * C;
            T* ErevT = (T*)a.ErevT + (size_t)h * MP2 * C;
            if (j < C) {
                EbarT[(size_t)m * C + j] = (T)(float)cs;           // conj(rho^j)
                EbarT[(size_t)(MP + m) * C + j] = (T)(float)(-sn);
            }
            if (j >= 1) {                                          // rho^{C-i} at i = C - j
                ErevT[(size_t)m * C + (C - j)] = (T)(float)cs;
                ErevT[(size_t)(MP + m) * C + (C - j)] = (T)(float)sn;
            }
        }
        return;
    }
    if (gid < n_head + n_misc) {
        const long long e = gid - n_head;
        const int hl = (int)(e / (a.SP + MP)), k = (int)(e % (a.SP + MP)), h = a.h0 + hl;
        const double Tp = a.T[hl];
        if (k < a.SP) {
            a.theta[(size_t)h * a.SP + k] = k < a.S ? (int)rint((double)k * Tp / (double)a.S) : INT32_MAX;
            if (k == 0) {
                a.rperiod[h] = 1.0 / Tp;
                a.period[h] = Tp;
            }
        } else {
            const int m = k - a.SP;
            double sn = 0.0, cs = 0.0;
            if (m < a.M) sincos(mode_phase((long long)m * a.Lblk, Tp), &sn, &cs);
            a.rotblk[(size_t)h * MP2 + m] = (float)cs;
            a.rotblk[(size_t)h * MP2 + MP + m] = (float)sn;
        }
        return;
    }
    if (gid < n_head + n_misc + n_ab) {
        // Interpolation matrices (Eq. translated at tau_s = s T / S): the phase
        // m w tau_s = 2 pi m s / S does not depend on the head's period.
        const long long e = gid - n_head - n_misc;
        const int s = (int)(e / MP), m = (int)(e % MP);
        float ca = 0.f, sa = 0.f;
        if (s < a.S && m < a.M) {
            const double cm = (m == 0 ? 1.0 : 2.0) / (2.0 * a.M - 1.0);
            const double ph = 2.0 * M_PI * (double)(((long long)m * s) % a.S) / (double)a.S;
            double sn, cs;
            sincos(ph, &sn, &cs);
            ca = (float)(cm * cs);
            sa = (float)(a.negB ? -cm * sn : cm * sn);
        }
        ((T*)a.ABs)[(size_t)s * MP2 + m] = (T)(ca * a.scale);
        ((T*)a.ABs)[(size_t)s * MP2 + MP + m] = (T)(sa * a.scale);
        if (!a.conj_tab) {
            ((T*)a.ABm)[(size_t)m * a.SP + s] = (T)ca;
            ((T*)a.ABm)[(size_t)(MP + m) * a.SP + s] = (T)sa;
        }
        return;
    }
    if (gid < n_head + n_misc + n_ab + n_trig) {
        // cos | sin of 2 pi k / S: the slot matrices are c_m times these at k = m s mod S
        const int k = (int)(gid - n_head - n_misc - n_ab);
        double sn = 0.0, cs = 0.0;
        if (k < a.S) sincos(2.0 * M_PI * (double)k / (double)a.S, &sn, &cs);
        a.trig[k] = (float)cs;
        a.trig[a.SP + k] = (float)sn;
    }
}

// One thread per 16-byte piece of a fragment-ordered table (see FragTabArgs): the shared slot
// matrices, each head's Etab, EbarT and ErevT, then the heads' twiddle tables.
__global__ __launch_bounds__(kThreads) void fragtab_kernel(FragTabArgs a)
{
    const long long MP2 = 2 * a.MP;
    const long long nab = (long long)a.SP * MP2 / 8, nh = (long long)a.C * MP2 / 8;
    long long u = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const bf16* src;
    bf16* dst;
    int K;  // columns of the source table
    if (u < nab) {
        src = (const bf16*)a.ABs, dst = (bf16*)a.fABs, K = (int)MP2;
    } else if ((u -= nab) < nab) {
        src = (const bf16*)a.ABm, dst = (bf16*)a.fABm, K = a.SP;
    } else if ((u -= nab) >= 3 * nh * a.H) {
        // twiddle pieces: (h, mt, ct, lane) -> cos | sin of the lane's token and four modes
        u -= 3 * nh * a.H;
        const int NMT = a.MP / 16, NT = a.C / 16;
        const long long h = u / (nh);
        if (h >= a.H) return;
        const int l = (int)(u % 64), ct = (int)((u / 64) % NT), mt = (int)((u / (64 * NT)) % NMT);
        const bf16* row = (const bf16*)a.Etab + (size_t)h * nh * 8 + (size_t)(16 * ct + (l & 15)) * MP2;
        const int m = 16 * mt + 4 * (l >> 4);
        bf16x8 x;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            x[e] = row[m + e];
            x[4 + e] = row[a.MP + m + e];
        }
        *reinterpret_cast<bf16x8*>((bf16*)a.fTw + (size_t)u * 8) = x;
        return;
    } else {
        const long long h = u / (3 * nh);
        if (h >= a.H) return;
        const int which = (int)((u % (3 * nh)) / nh);
        u %= nh;
        const size_t off = (size_t)h * nh * 8;
        K = which == 0 ? (int)MP2 : a.C;
        src = (const bf16*)(which == 0 ? a.Etab : which == 1 ? a.EbarT : a.ErevT) + off;
        dst = (bf16*)(which == 0 ? a.fEtab : which == 1 ? a.fEbar : a.fErev) + off;
    }
    const int l = (int)(u % 64), f = (int)(u / 64), kb = f % (K / 32), i = f / (K / 32);
    const bf16x8 x = *reinterpret_cast<const bf16x8*>(src + (size_t)(16 * i + (l & 15)) * K + 32 * kb + 8 * (l >> 4));
    *reinterpret_cast<bf16x8*>(dst + (size_t)u * 8) = x;
}

hipError_t launch_fragtab(const FragTabArgs& a, hipStream_t s)
{
    const long long n = 2ll * a.SP * 2 * a.MP / 8 + (long long)a.H * 4 * a.C * 2 * a.MP / 8;
    hipLaunchKernelGGL(fragtab_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_tables(const TableArgs& a, int is_bf16, hipStream_t s)
{
    const long long n = (long long)a.nh * a.jrows * a.MP + (long long)a.nh * (a.SP + a.MP) +
                        (a.with_shared ? (long long)a.SP * a.MP + a.SP : 0);
    dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
    if (is_bf16)
        hipLaunchKernelGGL(tables_kernel<bf16>, grid, dim3(kThreads), 0, s, a);
    else
        hipLaunchKernelGGL(tables_kernel<float>, grid, dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

// Scan over per-block summaries: carry'_g is the pre-rotated state at the start of
// segment g (g >= 1).  Z' <- rho^Lblk o Z' + S'_j block after block, starting from
// rho o state_in (or zero).  One thread per complex state element.
__global__ __launch_bounds__(kThreads) void scan_kernel(FwdArgs a, int MP, int D, int bps)
{
    const int per = 2 * MP * D;  // complex elements per (b,h): keys then values
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long long)a.B * a.H * per) return;
    const int bh = (int)(gid / per);
    const int e = (int)(gid % per);
    const int h = bh % a.H;
    const size_t U = (size_t)4 * MP * D;
    int m, d;
    size_t re, im;  // offsets inside one unit
    const float* sin_ = nullptr;
    if (e < MP * D) {
        m = e / D;
        d = e % D;
        re = (size_t)m * D + d;
        im = (size_t)MP * D + re;
        sin_ = a.sk_in;
    } else {
        int e2 = e - MP * D;
        d = e2 / MP;
        m = e2 % MP;
        re = (size_t)2 * MP * D + (size_t)d * MP + m;
        im = re + (size_t)MP * D;
        sin_ = a.sv_in;
    }
    const float* E1 = a.E32 + ((size_t)h * (a.C + 1) + 1) * 2 * MP;
    float zr = 0.f, zi = 0.f;
    if (sin_ && m < a.M) {
        float xr = sin_[(((size_t)bh * 2 + 0) * a.M + m) * D + d];
        float xi = sin_[(((size_t)bh * 2 + 1) * a.M + m) * D + d];
        float c1 = E1[m], s1 = E1[MP + m];
        zr = c1 * xr - s1 * xi;
        zi = s1 * xr + c1 * xi;
    }
    const float cb = a.rotblk[(size_t)h * 2 * MP + m];
    const float sb = a.rotblk[(size_t)h * 2 * MP + MP + m];
    const float* __restrict__ S = a.summ + (size_t)bh * a.nbs * U;
    float* __restrict__ Cy = a.carry + (size_t)bh * (a.nseg - 1) * U;
    // blocks in groups of 4 so that their loads are in flight together
    for (int j0 = 0; j0 < a.nbs; j0 += 4) {
        float sr[4], si[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int j = j0 + u;
            sr[u] = j < a.nbs ? S[(size_t)j * U + re] : 0.f;
            si[u] = j < a.nbs ? S[(size_t)j * U + im] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int j = j0 + u;
            if (j < a.nbs) {
                const float nr = cb * zr - sb * zi + sr[u];
                const float ni = sb * zr + cb * zi + si[u];
                zr = nr;
                zi = ni;
                if ((j + 1) % bps == 0) {
                    const int g = (j + 1) / bps;  // segment that starts after this block
                    Cy[(size_t)(g - 1) * U + re] = zr;
                    Cy[(size_t)(g - 1) * U + im] = zi;
                }
            }
        }
    }
}

hipError_t launch_scan(const Plan& p, const FwdArgs& a, hipStream_t s)
{
    long long n = (long long)p.B * p.H * 2 * p.MP * p.D;
    dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(scan_kernel, grid, dim3(kThreads), 0, s, a, p.MP, p.D, p.cps / p.cpb);
    return hipGetLastError();
}

__global__ __launch_bounds__(kThreads) void state_copy_kernel(const float* src, float* dst, size_t n)
{
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) dst[i] = src ? src[i] : 0.f;
}

hipError_t launch_state_copy(const float* src, float* dst, size_t n, hipStream_t s)
{
    if (n == 0 || dst == nullptr) return hipSuccess;
    dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(state_copy_kernel, grid, dim3(kThreads), 0, s, src, dst, n);
    return hipGetLastError();
}

}  // namespace bla
