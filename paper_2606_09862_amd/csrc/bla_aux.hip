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

template <typename T>
__global__ __launch_bounds__(kThreads) void tables_kernel(TableArgs a)
{
    const int MP2 = 2 * a.MP;
    const int C = a.C;
    if ((int)blockIdx.x < a.nh) {
        const int h = a.h0 + blockIdx.x;
        const double Tp = a.T[blockIdx.x];
        // E32: (C+1) x 2MP
        float* E32 = a.E32 + (size_t)h * (C + 1) * MP2;
        for (int idx = threadIdx.x; idx < (C + 1) * MP2; idx += blockDim.x) {
            int j = idx / MP2, col = idx % MP2, m = col % a.MP;
            float val = 0.f;
            if (m < a.M) {
                double sn, cs;
                sincos(mode_phase((long long)m * j, Tp), &sn, &cs);
                val = (float)(col < a.MP ? cs : sn);
            }
            E32[idx] = val;
        }
        T* EbarT = (T*)a.EbarT + (size_t)h * MP2 * C;
        T* ErevT = (T*)a.ErevT + (size_t)h * MP2 * C;
        for (int idx = threadIdx.x; idx < MP2 * C; idx += blockDim.x) {
            int row = idx / C, i = idx % C, m = row % a.MP;
            float eb = 0.f, er = 0.f;
            if (m < a.M) {
                double sn, cs, sr, cr;
                sincos(mode_phase((long long)m * i, Tp), &sn, &cs);
                sincos(mode_phase((long long)m * (C - i), Tp), &sr, &cr);
                eb = (float)(row < a.MP ? cs : -sn);
                er = (float)(row < a.MP ? cr : sr);
            }
            EbarT[idx] = (T)eb;
            ErevT[idx] = (T)er;
        }
        T* Etab = (T*)a.Etab + (size_t)h * C * MP2;
        for (int idx = threadIdx.x; idx < C * MP2; idx += blockDim.x) {
            int i = idx / MP2, col = idx % MP2, m = col % a.MP;
            float val = 0.f;
            if (m < a.M) {
                double sn, cs;
                sincos(mode_phase((long long)m * i, Tp), &sn, &cs);
                val = (float)(col < a.MP ? cs : sn);
            }
            Etab[idx] = (T)val;
        }
        for (int s = threadIdx.x; s < a.SP; s += blockDim.x)
            a.theta[(size_t)h * a.SP + s] =
                s < a.S ? (int)rint((double)s * Tp / (double)a.S) : INT32_MAX;
        for (int col = threadIdx.x; col < MP2; col += blockDim.x) {
            int m = col % a.MP;
            float val = 0.f;
            if (m < a.M) {
                double sn, cs;
                sincos(mode_phase((long long)m * a.Lblk, Tp), &sn, &cs);
                val = (float)(col < a.MP ? cs : sn);
            }
            a.rotblk[(size_t)h * MP2 + col] = val;
        }
    } else if (a.with_shared) {
        // Interpolation matrices (Eq. translated at tau_s = s T / S): the phase
        // m w tau_s = 2 pi m s / S does not depend on the head's period.
        const double inv = 1.0 / (2.0 * a.M - 1.0);
        for (int idx = threadIdx.x; idx < a.SP * MP2; idx += blockDim.x) {
            int s = idx / MP2, col = idx % MP2, m = col % a.MP;
            float val = 0.f;
            if (s < a.S && m < a.M) {
                double cm = (m == 0 ? 1.0 : 2.0) * inv;
                double ph = 2.0 * M_PI * (double)(((long long)m * s) % a.S) / (double)a.S;
                double sn, cs;
                sincos(ph, &sn, &cs);
                val = (float)(cm * (col < a.MP ? cs : sn));
            }
            a.AB32[idx] = val;
            ((T*)a.ABs)[idx] = (T)(val * a.scale);
            ((T*)a.ABm)[(size_t)col * a.SP + s] = (T)val;
        }
    }
}

hipError_t launch_tables(const TableArgs& a, int is_bf16, hipStream_t s)
{
    dim3 grid(a.nh + (a.with_shared ? 1 : 0));
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
    const float* E1 = a.E32 + ((size_t)h * (kChunk + 1) + 1) * 2 * MP;
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
    const float* S = a.summ + (size_t)bh * a.nbs * U;
    float* Cy = a.carry + (size_t)bh * (a.nseg - 1) * U;
    for (int j = 0; j < a.nbs; ++j) {
        float sr = S[(size_t)j * U + re], si = S[(size_t)j * U + im];
        float nr = cb * zr - sb * zi + sr;
        float ni = sb * zr + cb * zi + si;
        zr = nr;
        zi = ni;
        if ((j + 1) % bps == 0) {
            int g = (j + 1) / bps;  // segment that starts after this block
            Cy[(size_t)(g - 1) * U + re] = zr;
            Cy[(size_t)(g - 1) * U + im] = zi;
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
