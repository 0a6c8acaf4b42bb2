// State-decay form of BLA (Sec. 3.4) for gfx950: anchored slots (Sec. 3.3) whose previous
// state is multiplied by 1 - D before each write, the GSA-style gated recurrence
//     K~_t[s] = (1 - g_t[s]) K~_{t-1}[s] + g_t[s] k_t,   V~ likewise,
// with g_t[s] = D_M(p - tau_s) the slot's interpolation weight at the token's absolute
// position p (Eq. compressed_simplified).  The state is the slot state itself (the decay is
// diagonal in slots, not in modes): float32 [B, H, S, d].
//
// Sub-block form (every term a matrix-core contraction).  For a sub-block of c <= 16 tokens
// with gates a_j[s] = max(1 - g_j[s], eps), E_i[s] = prod_{l <= i} a_l[s] and
// Bq[j][s] = g_j[s] / E_j[s]:
//     K~_i = E_i o (K~_b + sum_{j <= i} Bq[j] k_j)
//     z^T  = scale E^T o (K~_b Q^T + Bq^T G^T),        G = tril(Q K^T)
//     O^T  = V~_b^T (P o E)^T + V^T tril(Bq (P o E)^T)
//     K~  <- E_{c-1} o (K~_b + Bq^T K),  V~ likewise.
// A gate is clamped at eps = 2^-40 where the decay flushes a slot (a = 0); the flushed
// state then survives with weight eps instead of 0.  Sub-blocks never cross a 16-token
// window of the sequence, and one ends before any slot's gate product drops below 2^-100,
// so E and 1/E stay inside the float32 (and bf16) range; the lengths depend on positions
// only (a whole window unless many small gates follow each other, as when M is small
// against T).  The gates, the sub-block lengths, E and Bq are the same for every batch row
// and every head of one period: decay_sched_kernel computes them once per call.
//
// Sequences are split into segments run by separate workgroups.  The recurrence is linear
// with data-independent gates, so a segment maps its entering state X to A_g o X + S_g:
// decay_forward_kernel<SUM = true> computes S_g (from a zero state) and A_g (the product
// of the segment's gates) for every segment but the last, decay_scan_kernel turns them in
// place into the entering states, and decay_forward_kernel<SUM = false> runs every segment
// from its entering state.
//
// Tiles are (slot x token) so that the softmax over the slots of a token is a reduction
// over the rows of the wave's tiles.  A workgroup of NWU waves runs one (b, h) sequence;
// wave w owns NSTW slot tiles and their fp32 state in registers (K~ as d x slot tiles, V~
// as slot x d tiles, the layouts the matrix cores read them in); with NWU > 1 the softmax
// and the output are reduced across the waves through LDS.
#include <math.h>
#include <stdint.h>

#include "bla_device.h"
#include "bla_forward_pair.h"
#include "bla_plan.h"

namespace bla {

constexpr float kDecayEps = 9.094947017729282e-13f;  // 2^-40

template <int D, int SP> struct DecayGeo {
    static constexpr int NDT = D / 16, KBD = D / 32, NST = SP / 16;
    // slot tiles per wave: the wave's fp32 state is 2 * NSTW * NDT tiles (at most 64 VGPRs,
    // so that two waves fit on a SIMD)
    static constexpr int NSTW = decay_slot_tiles_per_wave(D, SP);
    static constexpr int NWU = NST / NSTW;  // waves per workgroup
    static constexpr int NTH = 64 * NWU;
    static constexpr int LK = D + 12;       // K, V rows [16][LK] (bf16), conflict-free transposed reads
    static constexpr int LKF = D + 4;       // K rows [16][LKF] (float32)
    static constexpr int LKT = 16 + 4;      // K^T, V^T [D][LKT] (float32)
    static constexpr int LG = SP + 4;       // gate tables [16][LG] (float32)
    static_assert(NST % NSTW == 0, "slot tiles split evenly over the waves");
};

// sin(pi x) for |x| <= 1/2: the odd Taylor series of sin(pi x) through x^11, evaluated in
// float32 (relative error below 2e-7 on the whole range, so the Dirichlet ratio stays
// accurate near x = 0).
__device__ __forceinline__ float sinpi_half(float x)
{
    const float x2 = x * x;
    float p = -0.0073704309457143504f;           // -pi^11 / 11!
    p = p * x2 + 0.082145886611128228f;          //  pi^9 / 9!
    p = p * x2 - 0.59926452932079209f;           // -pi^7 / 7!
    p = p * x2 + 2.5501640398773455f;            //  pi^5 / 5!
    p = p * x2 - 5.1677127800499703f;            // -pi^3 / 3!
    p = p * x2 + 3.1415926535897932f;            //  pi
    return x * p;
}

// sin(pi a) for a in (-1, 1] from the half-range series (sin(pi a) = sin(pi (1 - a)), odd).
__device__ __forceinline__ float sinpi_one(float a)
{
    const float b = a > 0.5f ? 1.f - a : (a < -0.5f ? -1.f - a : a);
    return sinpi_half(b);
}

// Dirichlet kernel D_M at x = p - tau_s for the slot grid tau_s = s T / S, from the
// fractional revolutions fx = frac(p / T) (double): the closed form
// sin(N pi f) / (N sin(pi f)) with N = 2M - 1 and f = x / T reduced to (-1/2, 1/2].
__device__ __forceinline__ float dirichlet_at(double fx, int s, double rS, int N)
{
    double f = fx - (double)s * rS;
    f -= rint(f);
    if (f == 0.0) return 1.f;
    double a = (double)N * f;
    a -= 2.0 * rint(0.5 * a);
    return sinpif((float)a) / ((float)N * sinpif((float)f));
}

// Floats of one segment summary: K~ [SP][D], V~ [SP][D], gate product [SP].
template <int D, int SP> constexpr size_t decay_summary_floats() { return (size_t)2 * SP * D + SP; }

// Gate of slot s (s < S) at absolute position P: the interpolation weight D_M(P - tau_s) of
// Eq. compressed_simplified, with the phase f = (P - tau_s) / T reduced to (-1/2, 1/2] in
// double (P / T first, so that a position far past the period keeps a small one's accuracy)
// and the ratio sin(N pi f) / (N sin(pi f)) evaluated in float32 (D_M(0) = 1).
__device__ __forceinline__ float decay_gate(long long P, int s, double rT, double rS, int N)
{
    const double x = (double)P * rT;
    double fd = (x - floor(x)) - (double)s * rS;
    fd -= rint(fd);
    double ad = (double)N * fd;
    ad -= 2.0 * rint(0.5 * ad);
    const float den = sinpi_half((float)fd);
    return den == 0.f ? 1.f : sinpi_one((float)ad) * (1.f / (float)N) * __builtin_amdgcn_rcpf(den);
}

// The sub-block schedule of one forward call for period u and one 16-token window of the
// sequence (tokens w0 .. w0 + 15): the gates g_t[s] of Eq. compressed_simplified, the
// sub-blocks (greedy from the window start: each ends before any slot's product of
// a = max(1 - g, eps) falls below 2^-100, and takes at least one token), and per token the
// product E of a over its sub-block so far and Bq = g / E.  One workgroup of 256 threads per
// (window, period): all threads evaluate the window's gates into LDS, then wave 0 walks the
// sub-blocks with lane l holding slots l, l + 64, ...  Block (0, 0) also writes the head map.
template <int SPL>  // slots per lane: max(1, SP / 64)
__global__ __launch_bounds__(256) void decay_sched_kernel(GateArgs a)
{
    constexpr int MAXSPL = SPL;
    __shared__ float sg[16 * 64 * SPL];
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x < (unsigned)a.nh)
        a.gmap[a.h0 + threadIdx.x] = a.map[threadIdx.x];
    const int u = blockIdx.y, w0 = 16 * blockIdx.x, tid = threadIdx.x;
    const int nt = min(16, a.L - w0);
    const int N = 2 * a.M - 1;
    const double rT = a.rT[u];
    for (int x = tid; x < 16 * a.SP; x += 256) {
        const int i = x / a.SP, s = x % a.SP;
        sg[x] = (i < nt && s < a.S) ? decay_gate(a.t0 + w0 + i, s, rT, a.rS, N) : 0.f;
    }
    __syncthreads();
    if (tid >= 64) return;
    const int lane = tid;
    const size_t row0 = (size_t)(a.ubase + u) * a.L + w0;  // table row of the window's first token
    float gv[16][MAXSPL];
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
        for (int k = 0; k < MAXSPL; ++k) {
            const int s = lane + 64 * k;
            gv[i][k] = s < a.SP ? sg[i * a.SP + s] : 0.f;
        }
    for (int i0 = 0; i0 < nt;) {
        // first token of [i0, nt) whose prefix (from i0) of log2 a drops below -100
        int cut = nt;
#pragma unroll
        for (int k = 0; k < MAXSPL; ++k) {
            float lg = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                if (i >= i0 && i < nt) {
                    lg += __log2f(fmaxf(1.f - gv[i][k], kDecayEps));
                    if (lg < -100.f) cut = min(cut, i);
                }
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) cut = min(cut, __shfl_xor(cut, off));
        const int cs = max(1, cut - i0);
#pragma unroll
        for (int k = 0; k < MAXSPL; ++k) {
            const int s = lane + 64 * k;
            float run = 1.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                if (i >= i0 && i < i0 + cs && s < a.SP) {
                    run *= fmaxf(1.f - gv[i][k], kDecayEps);
                    const size_t idx = (row0 + i) * a.SP + s;
                    a.gE[idx] = run;
                    a.gB[idx] = gv[i][k] * __builtin_amdgcn_rcpf(run);  // run >= 2^-100: a normal float
                }
            }
        }
        if (lane == 0) a.glen[row0 + i0] = cs;
        i0 += cs;
    }
}

template <typename T, int D, int SP, bool SUM>
__global__ __launch_bounds__((DecayGeo<D, SP>::NTH)) void decay_forward_kernel(DecayArgs a)
{
    using G = DecayGeo<D, SP>;
    using F = typename Frag<T>::type;
    constexpr int NDT = G::NDT, KBD = G::KBD, NSTW = G::NSTW, NWU = G::NWU, NTH = G::NTH;
    constexpr int LG = G::LG;
    constexpr bool BF = sizeof(T) == 2;
    // LDS: K and V of the sub-block (bf16: row-major, read transposed with ds_read_tr;
    // float32: K row-major plus K^T, V^T), gate tables, thresholds, cross-wave buffers
    constexpr int KV_ELEMS = BF ? 2 * 16 * G::LK : 16 * G::LKF + 2 * D * G::LKT;
    __shared__ __attribute__((aligned(16))) T sKV[KV_ELEMS];
    // E and Bq rows of the sub-block for the outputs (the summary pass reads E from the schedule)
    __shared__ __attribute__((aligned(16))) float sE[SUM ? 4 : 16 * LG];
    __shared__ __attribute__((aligned(16))) float sB[SUM ? 4 : 16 * LG];
    __shared__ __attribute__((aligned(16))) int sTheta[SP];
    __shared__ float sRed[2][NWU][16];
    constexpr int LO = D + 4;  // sO row stride (floats)
    __shared__ __attribute__((aligned(16))) float sO[NWU > 1 ? NWU * 16 * LO : 4];

    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63, g = lane >> 4, r = lane & 15;
    const int nsu = SUM ? a.nseg - 1 : a.nseg;  // segments per sequence in this launch
    const int bh = blockIdx.x / nsu, seg = blockIdx.x % nsu, h = bh % a.H;
    constexpr size_t SF = decay_summary_floats<D, SP>();
    const int s0w = 16 * NSTW * wv;  // first slot of the wave
    const int S = a.S, L = a.L;
    const int tbeg = seg * a.seg_len, tend = min(L, tbeg + a.seg_len);
    const size_t grow = (size_t)a.gmap[h] * L;  // the head's schedule: rows grow + t of [L][SP]
    const T* qb = (const T*)a.q + (size_t)bh * L * D;
    const T* kb_ = (const T*)a.k + (size_t)bh * L * D;
    const T* vb = (const T*)a.v + (size_t)bh * L * D;
    T* ob = (T*)a.o + (size_t)bh * L * D;

    T* Ks = sKV;                                       // bf16: [16][LK]; float32: [16][LKF]
    T* Vs = BF ? sKV + 16 * G::LK : nullptr;           // bf16: [16][LK]
    T* KT = BF ? nullptr : sKV + 16 * G::LKF;          // float32: [D][LKT]
    T* VT = BF ? nullptr : KT + D * G::LKT;            // float32: [D][LKT]

    for (int i = tid; i < SP; i += NTH) sTheta[i] = a.theta[(size_t)h * SP + i];

    // ---- state: Kt[t][dt] = K~^T tile (d rows 16dt.., slot columns), Vt[t][dt] = V~ tile
    // (slot rows, d columns 16dt..) of the wave's slot tile t
    floatx4 Kst[NSTW][NDT], Vst[NSTW][NDT];
#pragma unroll
    for (int t = 0; t < NSTW; ++t) {
        const int sc = s0w + 16 * t + r;             // K~^T column slot
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            Kst[t][dt] = zero4();
            Vst[t][dt] = zero4();
            if (SUM) continue;
            if (seg > 0) {
                // entering state of the segment from the scanned summaries
                const float* cy = a.summ + ((size_t)bh * (a.nseg - 1) + (seg - 1)) * SF;
                Kst[t][dt] = ld4f(cy + (size_t)sc * D + 16 * dt + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    Vst[t][dt][e] = cy[(size_t)SP * D + (size_t)(s0w + 16 * t + 4 * g + e) * D + 16 * dt + r];
                continue;
            }
            if (a.sk_in && sc < S) Kst[t][dt] = ld4f(a.sk_in + ((size_t)bh * S + sc) * D + 16 * dt + 4 * g);
            if (a.sv_in) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int sr = s0w + 16 * t + 4 * g + e;
                    if (sr < S) Vst[t][dt][e] = a.sv_in[((size_t)bh * S + sr) * D + 16 * dt + r];
                }
            }
        }
    }

    // ---- staging of one sub-block's K and V (rows past c are zero)
    constexpr int PR = D * (int)sizeof(T) / 16;  // 16-byte pieces per row
    constexpr int EPP = 16 / (int)sizeof(T);     // elements per piece
    constexpr int PIECES = 2 * 16 * PR;
    constexpr int PPT = (PIECES + NTH - 1) / NTH;
    typedef typename Frag<T>::half Half;         // 4 elements (8 bytes bf16, 16 bytes float32)
    Half stg[PPT][BF ? 2 : 1];
    auto stage_load = [&](int t0s, int c) {
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int u = tid + NTH * i;
            const int which = u / (16 * PR), rem = u % (16 * PR);
            const int row = min(rem / PR, max(c - 1, 0)), pc = rem % PR;
            const T* src = (which == 0 ? kb_ : vb) + (size_t)(t0s + row) * D + EPP * pc;
            if (u < PIECES) {
                if constexpr (BF) {
                    stg[i][0] = ld4<T>(src);
                    stg[i][1] = ld4<T>(src + 4);
                } else {
                    stg[i][0] = ld4<T>(src);
                }
            }
        }
    };
    auto stage_store = [&](int c) {
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int u = tid + NTH * i;
            const int which = u / (16 * PR), rem = u % (16 * PR);
            const int row = rem / PR, pc = rem % PR;
            if (u < PIECES) {
                const bool live = row < c;
                if constexpr (BF) {
                    Half x0 = stg[i][0], x1 = stg[i][1];
                    if (!live) x0 = x1 = zero_half<T>();
                    T* dst = (which == 0 ? Ks : Vs) + row * G::LK + EPP * pc;
                    *reinterpret_cast<Half*>(dst) = x0;
                    *reinterpret_cast<Half*>(dst + 4) = x1;
                } else {
                    Half x0 = stg[i][0];
                    if (!live) x0 = zero_half<T>();
                    if (which == 0) *reinterpret_cast<Half*>(Ks + row * G::LKF + EPP * pc) = x0;
                    T* tr = which == 0 ? KT : VT;
#pragma unroll
                    for (int e = 0; e < 4; ++e) tr[(EPP * pc + e) * G::LKT + row] = x0[e];
                }
            }
        }
    };

    // schedule of the next sub-block (length, E and Bq of its first 16 tokens in the G
    // layout), loaded a sub-block ahead
    int lpf = 1;
    float Epf[NSTW][4], Bpf[NSTW][4];
    auto sched_load = [&](int t0s) {
        lpf = a.glen[grow + t0s];
#pragma unroll
        for (int t = 0; t < NSTW; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const size_t idx = (grow + min(t0s + 4 * g + e, L - 1)) * SP + s0w + 16 * t + r;
                if constexpr (!SUM) Epf[t][e] = a.gE[idx];
                Bpf[t][e] = a.gB[idx];
            }
    };
    // query rows of the next sub-block (columns: tokens), loaded a sub-block ahead; rows past
    // the sub-block's cut are other tokens of the sequence, whose columns are never stored
    F qpf[SUM ? 1 : KBD];
    auto q_load = [&](int t0s) {
        if constexpr (!SUM) {
            const int qrow = min(t0s + r, L - 1);
#pragma unroll
            for (int kb = 0; kb < KBD; ++kb) qpf[kb] = ld_frag<T>(qb + (size_t)qrow * D, 32 * kb, g);
        }
    };
    if (tbeg < tend) {
        stage_load(tbeg, min(16, tend - tbeg));
        sched_load(tbeg);
        q_load(tbeg);
    }
    float aprod[NSTW];  // product of the segment's gates for the K~^T column slot (summaries)
#pragma unroll
    for (int t = 0; t < NSTW; ++t) aprod[t] = 1.f;
    const float k2 = a.scale * 1.44269504088896341f;

    // Sub-blocks as scheduled (at most 16 tokens, never across a 16-token window); segment
    // starts are window starts.
    for (int tb = tbeg; tb < tend;) {
        const long long P = a.t0 + tb;  // absolute position of the sub-block's first token
        const int cmax = min(16, tend - tb);
        const int cs = max(1, min(lpf, cmax));
        F qf[SUM ? 1 : KBD];
#pragma unroll
        for (int kb = 0; kb < (SUM ? 0 : KBD); ++kb) qf[kb] = qpf[kb];
        // E and Bq of the sub-block's tokens in the G layout (lane (g, r): slot s0w + 16 t + r,
        // tokens 4g..4g+3); tokens past cs: factor 1, Bq 0
        float Ecur[NSTW][4], bq[NSTW][4];
#pragma unroll
        for (int t = 0; t < NSTW; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool live = 4 * g + e < cs;
                if constexpr (!SUM) Ecur[t][e] = live ? Epf[t][e] : 1.f;
                bq[t][e] = live ? Bpf[t][e] : 0.f;
            }
        // the summary pass: E of the sub-block's last token straight from the schedule
        float ecs[NSTW];
        floatx4 ers[NSTW];
        if constexpr (SUM) {
            const size_t last = (grow + tb + cs - 1) * SP + s0w;
#pragma unroll
            for (int t = 0; t < NSTW; ++t) {
                ecs[t] = a.gE[last + 16 * t + r];
                ers[t] = ld4f(a.gE + last + 16 * t + 4 * g);
            }
        }
        __syncthreads();  // previous sub-block done with the LDS tiles
        stage_store(cs);
        __syncthreads();  // K, V visible
        if (tb + cs < tend) {
            stage_load(tb + cs, min(16, tend - tb - cs));
            sched_load(tb + cs);
            q_load(tb + cs);
        }
        // the sub-block's E and Bq rows in LDS, each wave on its own slots (read below only by
        // the wave that wrote them)
        if constexpr (!SUM) {
#pragma unroll
            for (int t = 0; t < NSTW; ++t) {
                const int s = s0w + 16 * t + r;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sE[(4 * g + e) * LG + s] = Ecur[t][e];
                    sB[(4 * g + e) * LG + s] = bq[t][e];
                }
            }
        }

        // K^T and V^T fragments (rows: d, reduction: the sub-block's tokens)
        F vtf[NDT], ktf[NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            if constexpr (BF) {
                vtf[dt] = join(ld_tr(Vs + (4 * g + (r >> 2)) * G::LK + 16 * dt + 4 * (r & 3)), zero_half<T>());
                ktf[dt] = join(ld_tr(Ks + (4 * g + (r >> 2)) * G::LK + 16 * dt + 4 * (r & 3)), zero_half<T>());
            } else {
                vtf[dt] = ld_frag_lo<T>(VT + (16 * dt + r) * G::LKT, 0, g);
                ktf[dt] = ld_frag_lo<T>(KT + (16 * dt + r) * G::LKT, 0, g);
            }
        }

        if constexpr (!SUM) {
        // G^T = K Q^T (keys j rows, queries i columns), causal
        floatx4 gT = zero4();
        {
            const T* krow = BF ? Ks + r * G::LK : Ks + r * G::LKF;
#pragma unroll
            for (int kb = 0; kb < KBD; ++kb) gT = mma(ld_frag<T>(krow, 32 * kb, g), qf[kb], gT);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * g + e > r) gT[e] = 0.f;
        }
        const F gTf = join(cvt4(gT, T()), zero_half<T>());

        // ---- scores z^T (slots x tokens) = scale E^T o (K~ Q^T + Bq^T G^T), masked
        floatx4 z[NSTW];
        const long long pos_ll = P + r;
        const int pos = pos_ll < (1ll << 30) ? (int)pos_ll : (1 << 30);
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < NSTW; ++t) {
            floatx4 acc = zero4();
#pragma unroll
            for (int kb = 0; kb < KBD; ++kb)
                acc = mma(frag_from_acc<T>(Kst[t][2 * kb], Kst[t][2 * kb + 1]), qf[kb], acc);
            const F bqa = join(cvt4(floatx4{bq[t][0], bq[t][1], bq[t][2], bq[t][3]}, T()), zero_half<T>());
            acc = mma(bqa, gTf, acc);
            const floatx4 Ei = ld4f(sE + r * LG + s0w + 16 * t + 4 * g);
            const intx4 th = *reinterpret_cast<const intx4*>(sTheta + s0w + 16 * t + 4 * g);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float zz = pos < th[e] ? -INFINITY : acc[e] * Ei[e] * k2;
                z[t][e] = zz;
                mx = fmaxf(mx, zz);
            }
        }
        mx = rows_max(mx);
        if constexpr (NWU > 1) {
            if (g == 0) sRed[0][wv][r] = mx;
            __syncthreads();
#pragma unroll
            for (int w = 0; w < NWU; ++w) mx = fmaxf(mx, sRed[0][w][r]);
        }
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < NSTW; ++t)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float ex = __builtin_amdgcn_exp2f(z[t][e] - mx);
                z[t][e] = ex;
                sum += ex;
            }
        sum = rows_sum(sum);
        if constexpr (NWU > 1) {
            if (g == 0) sRed[1][wv][r] = sum;
            __syncthreads();
            sum = 0.f;
#pragma unroll
            for (int w = 0; w < NWU; ++w) sum += sRed[1][w][r];
        }
        const float inv = __builtin_amdgcn_rcpf(sum);  // sum >= 1 (the maximum contributes exp2(0))
        // (P o E)^T as B fragments over the wave's slots
#pragma unroll
        for (int t = 0; t < NSTW; ++t) {
            const floatx4 Ei = ld4f(sE + r * LG + s0w + 16 * t + 4 * g);
            z[t] = z[t] * inv * Ei;
        }
        constexpr int NPF = (NSTW + 1) / 2;
        F pf[NPF];
#pragma unroll
        for (int kp = 0; kp < NPF; ++kp)
            pf[kp] = 2 * kp + 1 < NSTW ? frag_from_acc<T>(z[2 * kp], z[2 * kp + 1])
                                       : join(cvt4(z[2 * kp], T()), zero_half<T>());

        // ---- H^T = tril(Bq (P o E)^T) (keys j rows, queries i columns), partial over the wave's slots
        floatx4 hT = zero4();
#pragma unroll
        for (int kp = 0; kp < NPF; ++kp) {
            const float* brow = sB + r * LG + s0w + 32 * kp;
            F ba;
            if (2 * kp + 1 < NSTW)
                ba = join(cvt4(ld4f(brow + 4 * g), T()), cvt4(ld4f(brow + 16 + 4 * g), T()));
            else
                ba = join(cvt4(ld4f(brow + 4 * g), T()), zero_half<T>());
            hT = mma(ba, pf[kp], hT);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (4 * g + e > r) hT[e] = 0.f;
        const F hTf = join(cvt4(hT, T()), zero_half<T>());

        // ---- O^T (d rows, tokens columns) = V~^T (P o E)^T + V^T H^T
        floatx4 oT[NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            floatx4 acc = zero4();
#pragma unroll
            for (int kp = 0; kp < NPF; ++kp) {
                const F va = 2 * kp + 1 < NSTW ? frag_from_acc<T>(Vst[2 * kp][dt], Vst[2 * kp + 1][dt])
                                               : join(cvt4(Vst[2 * kp][dt], T()), zero_half<T>());
                acc = mma(va, pf[kp], acc);
            }
            oT[dt] = mma(vtf[dt], hTf, acc);
        }
        if constexpr (NWU == 1) {
            if (r < cs) {
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) st4<T>(ob + (size_t)(tb + r) * D + 16 * dt + 4 * g, oT[dt]);
            }
        } else {
            // partial outputs of every wave through LDS: sO[w][token][d]; then each thread
            // sums eight consecutive d of one token over the waves and stores them at once
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) st4f(sO + ((size_t)wv * 16 + r) * LO + 16 * dt + 4 * g, oT[dt]);
            __syncthreads();
            constexpr int P8 = 16 * D / 8;  // 8-element pieces of the sub-block's output
            for (int u = tid; u < P8; u += NTH) {
                const int tok = u / (D / 8), d0 = 8 * (u % (D / 8));
                floatx4 lo = zero4(), hi = zero4();
#pragma unroll
                for (int w = 0; w < NWU; ++w) {
                    lo += ld4f(sO + ((size_t)w * 16 + tok) * LO + d0);
                    hi += ld4f(sO + ((size_t)w * 16 + tok) * LO + d0 + 4);
                }
                if (tok < cs) {
                    T* dst = ob + (size_t)(tb + tok) * D + d0;
                    st4<T>(dst, lo);
                    st4<T>(dst + 4, hi);
                }
            }
        }
        }  // !SUM

        // ---- state update: K~^T += K^T Bq, V~ += Bq^T V, then the decay E_{c-1} of the sub-block
#pragma unroll
        for (int t = 0; t < NSTW; ++t) {
            const F bqa = join(cvt4(floatx4{bq[t][0], bq[t][1], bq[t][2], bq[t][3]}, T()), zero_half<T>());
            const float ecol = SUM ? ecs[t] : sE[(cs - 1) * LG + s0w + 16 * t + r];
            const floatx4 erow = SUM ? ers[t] : ld4f(sE + (cs - 1) * LG + s0w + 16 * t + 4 * g);
            aprod[t] *= ecol;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                Kst[t][dt] = mma(ktf[dt], bqa, Kst[t][dt]) * ecol;
                Vst[t][dt] = mma(bqa, vtf[dt], Vst[t][dt]) * erow;
            }
        }
        tb += cs;
    }

    if constexpr (SUM) {
        // ---- segment summary: K~ rows, V~ rows, gate product
        float* sm = a.summ + ((size_t)bh * (a.nseg - 1) + seg) * SF;
#pragma unroll
        for (int t = 0; t < NSTW; ++t) {
            const int sc = s0w + 16 * t + r;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                st4f(sm + (size_t)sc * D + 16 * dt + 4 * g, Kst[t][dt]);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    sm[(size_t)SP * D + (size_t)(s0w + 16 * t + 4 * g + e) * D + 16 * dt + r] = Vst[t][dt][e];
            }
            if (g == 0) sm[(size_t)2 * SP * D + sc] = aprod[t];
        }
        return;
    }
    if (seg != a.nseg - 1) return;
    // ---- final slot states
#pragma unroll
    for (int t = 0; t < NSTW; ++t) {
        const int sc = s0w + 16 * t + r;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            if (a.sk_out && sc < S) st4f(a.sk_out + ((size_t)bh * S + sc) * D + 16 * dt + 4 * g, Kst[t][dt]);
            if (a.sv_out) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int sr = s0w + 16 * t + 4 * g + e;
                    if (sr < S) a.sv_out[((size_t)bh * S + sr) * D + 16 * dt + r] = Vst[t][dt][e];
                }
            }
        }
    }
}

// Entering states of the segments, in place over the summaries: thread (b,h, element)
// walks the segments, carry_{g+1} = A_g o carry_g + S_g from carry_0 = the input state,
// and stores carry_{g+1} where S_g was.
template <int D, int SP>
__global__ __launch_bounds__(256) void decay_scan_kernel(DecayArgs a)
{
    constexpr size_t PER = (size_t)2 * SP * D, SF = decay_summary_floats<D, SP>();
    const size_t gid = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (gid >= (size_t)a.B * a.H * PER) return;
    const size_t bh = gid / PER, e = gid % PER;
    const int half = (int)(e / ((size_t)SP * D));
    const int rem = (int)(e % ((size_t)SP * D)), s = rem / D, d = rem % D;
    float x = 0.f;
    const float* in = half ? a.sv_in : a.sk_in;
    if (in && s < a.S) x = in[(bh * a.S + s) * D + d];
    float* base = a.summ + bh * (size_t)(a.nseg - 1) * SF;
    for (int g = 0; g < a.nseg - 1; ++g) {
        float* sg = base + (size_t)g * SF;
        x = sg[PER + s] * x + sg[e];
        sg[e] = x;
    }
}

// ---------------------------------------------------------------------------------------
// One decode step of the decay form for every (b, h): one workgroup per (b, h); thread
// (slot row, d-quad) updates 4 state columns of a slot row in each of its passes.  Every
// state load is issued up front (at most 8 passes: the workgroup grows with S d).
template <int D, int SP> constexpr int decay_step_threads()
{
    return SP * D / 32 < 256 ? 256 : (SP * D / 32 > 1024 ? 1024 : SP * D / 32);
}

template <typename T, int D, int SP>
__global__ __launch_bounds__((decay_step_threads<D, SP>())) void decay_step_kernel(DecayStepArgs a)
{
    constexpr int NT = decay_step_threads<D, SP>();
    constexpr int NQ = D / 4, RPP = NT / NQ, PASSES = (SP + RPP - 1) / RPP;
    __shared__ float sg[SP];
    __shared__ float sz[SP];
    __shared__ __attribute__((aligned(16))) float sred[RPP * D];
    const int bh = blockIdx.x, b = bh / a.H, h = bh % a.H;
    const int tid = threadIdx.x, rg = tid / NQ, qd = tid % NQ;
    const int S = a.S, N = 2 * a.M - 1;
    const long long pos = a.pos ? (long long)a.pos[b] : a.t0;
    const double rT = a.rperiod[h], rS = 1.0 / (double)S;
    float* skb = a.sk + (size_t)bh * S * D;
    float* svb = a.sv + (size_t)bh * S * D;

    floatx4 kc[PASSES], vc[PASSES];
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int sc = min(ps * RPP + rg, S - 1);
        kc[ps] = ld4f(skb + (unsigned)(sc * D + 4 * qd));
        vc[ps] = ld4f(svb + (unsigned)(sc * D + 4 * qd));
    }
    const floatx4 q4 = to_f4(ld4<T>((const T*)a.q + (size_t)bh * D + 4 * qd));
    const floatx4 k4 = to_f4(ld4<T>((const T*)a.k + (size_t)bh * D + 4 * qd));
    const floatx4 v4 = to_f4(ld4<T>((const T*)a.v + (size_t)bh * D + 4 * qd));
    {
        const double x = (double)pos * rT;
        const double fx = x - floor(x);
        for (int s = tid; s < SP; s += NT) sg[s] = s < S ? dirichlet_at(fx, s, rS, N) : 0.f;
    }
    __syncthreads();

#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int s = ps * RPP + rg;
        const bool valid = s < S;
        const float gt = valid ? sg[s] : 0.f;
        const float keep = 1.f - gt;
        const floatx4 nk = keep * kc[ps] + gt * k4;
        const floatx4 nv = keep * vc[ps] + gt * v4;
        vc[ps] = nv;
        float zz = q4[0] * nk[0] + q4[1] * nk[1] + q4[2] * nk[2] + q4[3] * nk[3];
        if (valid) {
            st4f(skb + (unsigned)(s * D + 4 * qd), nk);
            st4f(svb + (unsigned)(s * D + 4 * qd), nv);
        }
#pragma unroll
        for (int off = NQ / 2; off > 0; off >>= 1) zz += __shfl_xor(zz, off);
        if (qd == 0 && s < SP) sz[s] = zz;
    }
    __syncthreads();
    if (tid < 64) {
        float mx = -INFINITY;
        for (int s = tid; s < SP; s += 64) {
            const float z = (s < S && pos >= (long long)a.theta[(size_t)h * SP + s]) ? sz[s] * a.scale : -INFINITY;
            sz[s] = z;
            mx = fmaxf(mx, z);
        }
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
    floatx4 o4 = zero4();
#pragma unroll
    for (int ps = 0; ps < PASSES; ++ps) {
        const int s = ps * RPP + rg;
        if (s < S) o4 += sz[s] * vc[ps];
    }
    st4f(sred + (size_t)rg * D + 4 * qd, o4);
    __syncthreads();
    for (int d = tid; d < D; d += NT) {
        float acc = 0.f;
        for (int gq = 0; gq < RPP; ++gq) acc += sred[(size_t)gq * D + d];
        ((T*)a.o)[(size_t)bh * D + d] = (T)acc;
    }
}

// ev (nullable, entries nullable): hipEvent_t recorded after the summary pass, after the scan
// and after the forward pass.
template <typename T, int D, int SP>
static hipError_t launch_decay_sp(const DecayArgs& a, hipStream_t s, void* const* ev)
{
    auto mark = [&](int i) -> hipError_t {
        return (ev && ev[i]) ? hipEventRecord((hipEvent_t)ev[i], s) : hipSuccess;
    };
    const unsigned units = (unsigned)(a.B * a.H);
    if (a.nseg > 1)
        hipLaunchKernelGGL((decay_forward_kernel<T, D, SP, true>), dim3(units * (a.nseg - 1)),
                           dim3(DecayGeo<D, SP>::NTH), 0, s, a);
    hipError_t e = mark(0);
    if (e != hipSuccess) return e;
    if (a.nseg > 1) {
        const size_t n = (size_t)units * 2 * SP * D;
        hipLaunchKernelGGL((decay_scan_kernel<D, SP>), dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
    }
    if ((e = mark(1)) != hipSuccess) return e;
    hipLaunchKernelGGL((decay_forward_kernel<T, D, SP, false>), dim3(units * a.nseg), dim3(DecayGeo<D, SP>::NTH),
                       0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return mark(2);
}

template <typename T, int D>
static hipError_t launch_decay_d(const DecayArgs& a, int SP, hipStream_t s, void* const* ev)
{
#define BLA_DECAY_SP(SSP) \
    if (SP == SSP) return launch_decay_sp<T, D, SSP>(a, s, ev);
    BLA_DECAY_SP(32)
    BLA_DECAY_SP(64)
    BLA_DECAY_SP(128)
    BLA_DECAY_SP(256)
#undef BLA_DECAY_SP
    return hipErrorInvalidValue;
}

hipError_t launch_decay_gates(const GateArgs& g, hipStream_t s)
{
    if (g.L <= 0 || g.nu == 0) return hipSuccess;
    if (g.SP > 256 || g.nh > kMaxHeadsPerTableLaunch || g.nu > g.nh) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((g.L + 15) / 16), (unsigned)g.nu);
    if (g.SP <= 64)
        hipLaunchKernelGGL(decay_sched_kernel<1>, grid, dim3(256), 0, s, g);
    else if (g.SP == 128)
        hipLaunchKernelGGL(decay_sched_kernel<2>, grid, dim3(256), 0, s, g);
    else
        hipLaunchKernelGGL(decay_sched_kernel<4>, grid, dim3(256), 0, s, g);
    return hipGetLastError();
}

hipError_t launch_decay_forward(int bf16_io, int D, int SP, const DecayArgs& a, hipStream_t s, void* const* ev)
{
    if (bf16_io) {
        if (D == 32) return launch_decay_d<bf16, 32>(a, SP, s, ev);
        if (D == 64) return launch_decay_d<bf16, 64>(a, SP, s, ev);
        if (D == 128) return launch_decay_d<bf16, 128>(a, SP, s, ev);
    } else {
        if (D == 32) return launch_decay_d<float, 32>(a, SP, s, ev);
        if (D == 64) return launch_decay_d<float, 64>(a, SP, s, ev);
        if (D == 128) return launch_decay_d<float, 128>(a, SP, s, ev);
    }
    return hipErrorInvalidValue;
}

template <typename T, int D>
static hipError_t launch_decay_step_d(const DecayStepArgs& a, int SP, hipStream_t s)
{
    const dim3 grid((unsigned)(a.B * a.H));
#define BLA_DSTEP_SP(SSP)                                                                \
    if (SP == SSP) {                                                                     \
        hipLaunchKernelGGL((decay_step_kernel<T, D, SSP>), grid, dim3(decay_step_threads<D, SSP>()), 0, s, a); \
        return hipGetLastError();                                                        \
    }
    BLA_DSTEP_SP(32)
    BLA_DSTEP_SP(64)
    BLA_DSTEP_SP(128)
    BLA_DSTEP_SP(256)
#undef BLA_DSTEP_SP
    return hipErrorInvalidValue;
}

hipError_t launch_decay_step(int bf16_io, int D, int SP, const DecayStepArgs& a, hipStream_t s)
{
    if (bf16_io) {
        if (D == 32) return launch_decay_step_d<bf16, 32>(a, SP, s);
        if (D == 64) return launch_decay_step_d<bf16, 64>(a, SP, s);
        if (D == 128) return launch_decay_step_d<bf16, 128>(a, SP, s);
    } else {
        if (D == 32) return launch_decay_step_d<float, 32>(a, SP, s);
        if (D == 64) return launch_decay_step_d<float, 64>(a, SP, s);
        if (D == 128) return launch_decay_step_d<float, 128>(a, SP, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace bla
