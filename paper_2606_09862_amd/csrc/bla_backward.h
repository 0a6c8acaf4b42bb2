// Backward pass of the chunked BLA operator for gfx950: the gradients of Alg. 2 (the
// rotating mode state of Sec. 3.1 Eq. recurrence read out through the blurry slots of
// Eq. compressed with the masked slot softmax of Eq. output) with respect to q, k, v and the
// input states, given dLoss/dO and dLoss/d(final states).
//
// Per chunk of c tokens (local index i), with rho_m = exp(i m w), E[i,m] = rho_m^i, the
// pre-rotated forward state Z' = rho Z entering the chunk, the pre-rotated adjoint
// Gam' = rho dLoss/dZ of the state after the chunk's last token, G = tril(Q K^T) and
// Gd = tril(dO V^T):
//
//   U   = E o (Q Z'_k^T + G conj(E)),   z = scale (Re U A^T + Im U B^T) masked, P = softmax
//   Y   = E o (dO Z'_v^T + Gd conj(E))          (y_i[m] = <dO_i, Z_v after token i>)
//   dP  = Re Y A^T + Im Y B^T,   dz = P o (dP - rowsum(P o dP))
//   W'' = (P A - i P B) o E,      Wq'' = scale (dz A - i dz B) o E       (Wq'' = conj(du) o E)
//   dq  = Re(Wq'' Z'_k) + tril(Re(Wq'' conj(E)^T)) K
//   dk  = tril(Re(Wq'' conj(E)^T))^T Q + Re(conj(Erev) Gam'_k),   Erev[j] = rho^{c-j}
//   dv  = tril(Re(W'' conj(E)^T))^T dO + Re(conj(Erev) Gam'_v)
//   Gam' <- conj(rho^c) o Gam' + [conj(Wq'')^T Q | conj(W'')^T dO]
//
// The walk goes over the chunks in reverse.  The forward state entering a chunk is rebuilt
// from the state after it, Z'_in = conj(rho^c) o (Z'_out - sum_i rho^{c-i} [k_i | v_i]): the
// rotation is unitary, so undoing it loses nothing, and the subtraction repeats the forward
// sum's own terms.  Sequences are cut into segments run by separate workgroups:
// bwd_fsum_kernel writes the forward summary of every segment (its pre-rotated state from
// zero), bwd_kernel<SUM = true> the adjoint summary of every segment but the first (the
// adjoint at its start from a zero adjoint at its end), and bwd_kernel<SUM = false> forms a
// segment's end state and end adjoint from them (Horner sums, the recurrences are linear)
// and walks the segment writing dq, dk, dv.
//
// Work split inside a 256-thread workgroup (4 waves): the state and adjoint tiles are
// split by mode tiles (both states held as [d rows][m columns] accumulator tiles, the
// adjoints as [m][d]); the per-token chain (scores, softmax, its gradient, dq) by query
// tiles; dk and dv by key tiles.  Everything a wave needs from another wave goes through
// LDS between barriers.
#pragma once

#include <math.h>

#include "bla_device.h"
#include "bla_forward.h"
#include "bla_plan.h"

namespace bla {

template <typename T, int D, int MP, int SP> struct Bwd : Geo<T, D, MP> {
    using G = Geo<T, D, MP>;
    static constexpr int NST = SP / 16;
    static constexpr int KBS = SP / 32;
    static constexpr int LDQ = D + G::PAD;          // row-major token tiles [C][LDQ]
    static constexpr int LDK = G::C + G::PAD;       // [D][LDK] transposed tiles, [C][LDK] G / H, [2MP][LDK] W
    static constexpr int LDU = 2 * MP + G::PAD;     // [C][LDU] U, Y; [D][LDU] state operands
    static constexpr size_t A_ELEMS = (size_t)4 * G::C * LDQ;
    static constexpr size_t T_ELEMS = (size_t)4 * D * LDK;
    static constexpr size_t G_ELEMS = (size_t)2 * G::C * LDK;
    static constexpr size_t B_ELEMS = (size_t)4 * MP * LDK > (size_t)2 * G::C * LDU
                                          ? (size_t)4 * MP * LDK : (size_t)2 * G::C * LDU;
    static_assert((size_t)2 * G::C * LDK <= A_ELEMS, "H tiles fit in the row-major token region");
    static constexpr size_t Z_ELEMS = (size_t)2 * D * LDU;
    static constexpr size_t LDS_BYTES = (A_ELEMS + T_ELEMS + G_ELEMS + B_ELEMS + Z_ELEMS) * sizeof(T) + (size_t)SP * 4;
    static_assert(LDS_BYTES == bwd_lds_bytes((int)sizeof(T), D, MP, SP), "host and device LDS layouts agree");
    static_assert(LDS_BYTES <= kBwdMaxLds, "backward tiles fit in LDS");
    static_assert(SP % 32 == 0, "slot padding");
};

// ---------------------------------------------------------------------------------
// Staging of NTEN token tensors of one chunk (tensor 0 = K, 1 = V, 2 = Q, 3 = dO) in units
// of 4 tokens x 8 elements: registers first (issued a chunk ahead), then LDS, transposed
// ([D][LDK], tokens contiguous) and, with ROW, row-major ([C][LDQ]).  Rows past c are zero.
// Consecutive threads take consecutive 8-element pieces of the same four rows, so the global
// reads are coalesced.
template <typename T, int D, int NTEN> struct BStage {
    static constexpr int UPT = (kChunk / 4) * (D / 8);   // units per tensor
    static constexpr int PT = (NTEN * UPT + kThreads - 1) / kThreads;
    typename Frag<T>::half x[PT][4][2];
};

template <typename T, int D, int NTEN>
__device__ __forceinline__ void bstage_load(BStage<T, D, NTEN>& st, const T* const* src, int c, int tid)
{
    using S = BStage<T, D, NTEN>;
#pragma unroll
    for (int i = 0; i < S::PT; ++i) {
        const int u = tid + i * kThreads;
        if ((NTEN * S::UPT) % kThreads == 0 || u < NTEN * S::UPT) {
            const int ten = u / S::UPT, uu = u % S::UPT, dq = uu % (D / 8), tq = uu / (D / 8);
            const T* base = src[ten] + 8 * dq;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int row = min(4 * tq + t, c - 1);
                st.x[i][t][0] = ld_global<typename Frag<T>::half>(base + (size_t)row * D);
                st.x[i][t][1] = ld_global<typename Frag<T>::half>(base + (size_t)row * D + 4);
            }
        }
    }
}

template <typename T, int D, int NTEN, bool ROW>
__device__ __forceinline__ void bstage_store(const BStage<T, D, NTEN>& st, T* const* rowdst, T* const* trdst,
                                             int ldq, int ldk, int c, int tid)
{
    using S = BStage<T, D, NTEN>;
    using H = typename Frag<T>::half;
    const H z = zero_half<T>();
#pragma unroll
    for (int i = 0; i < S::PT; ++i) {
        const int u = tid + i * kThreads;
        if ((NTEN * S::UPT) % kThreads == 0 || u < NTEN * S::UPT) {
            const int ten = u / S::UPT, uu = u % S::UPT, dq = uu % (D / 8), tq = uu / (D / 8);
            H x[4][2];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const bool ok = 4 * tq + t < c;
                x[t][0] = ok ? st.x[i][t][0] : z;
                x[t][1] = ok ? st.x[i][t][1] : z;
            }
            if constexpr (ROW) {
                T* rd = rowdst[ten] + 8 * dq;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    st_lds<H>(rd + (size_t)(4 * tq + t) * ldq, x[t][0]);
                    st_lds<H>(rd + (size_t)(4 * tq + t) * ldq + 4, x[t][1]);
                }
            }
            T* td = trdst[ten] + (size_t)(8 * dq) * ldk + 4 * tq;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                H lo{x[0][0][e], x[1][0][e], x[2][0][e], x[3][0][e]};
                H hi{x[0][1][e], x[1][1][e], x[2][1][e], x[3][1][e]};
                st_lds<H>(td + (size_t)e * ldk, lo);
                st_lds<H>(td + (size_t)(e + 4) * ldk, hi);
            }
        }
    }
}

// Z' (+ or -)= sum_i rho^{c-i} [k_i | v_i] on the wave's mode tiles; both states are held as
// [d rows][m columns] tiles.  Kt, Vt: [D][ldk] transposed chunk tiles; Erev: [2MP][C] table
// of rho^{C-i} (full chunks); E32: float32 phase table for a ragged c.
template <typename T, int D, int MP>
__device__ __forceinline__ void bwd_accumulate(StateTiles<T, D, MP>& Zk, StateTiles<T, D, MP>& Zv, const T* Kt,
                                               const T* Vt, int ldk, const T* Erev, const float* E32, int c, int w,
                                               int g, int r)
{
    using GG = Geo<T, D, MP>;
    using F = typename Frag<T>::type;
#pragma unroll
    for (int kb = 0; kb < GG::KBC; ++kb) {
        F kf[GG::NDT], vf[GG::NDT];
#pragma unroll
        for (int dt = 0; dt < GG::NDT; ++dt) {
            kf[dt] = ld_frag<T>(Kt + (size_t)(16 * dt + r) * ldk, 32 * kb, g);
            vf[dt] = ld_frag<T>(Vt + (size_t)(16 * dt + r) * ldk, 32 * kb, g);
        }
#pragma unroll
        for (int o = 0; o < GG::OWN; ++o) {
            const int mt = w + GG::NW * o;
            if (mt < GG::NMT) {
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const F ef = (c == GG::C) ? ld_frag<T>(Erev + (size_t)(16 * (p * GG::NMT + mt) + r) * GG::C, 32 * kb, g)
                                              : erev_frag<T, MP>(E32, 2 * MP, c, p, mt, kb, g, r);
#pragma unroll
                    for (int dt = 0; dt < GG::NDT; ++dt) {
                        Zk[o][p][dt] = mma(kf[dt], ef, Zk[o][p][dt]);
                        Zv[o][p][dt] = mma(vf[dt], ef, Zv[o][p][dt]);
                    }
                }
            }
        }
    }
}

// Multiply [d][m] state tiles by rot[m] = (cos, sin) (conjugated with CONJ).
template <typename T, int D, int MP, bool CONJ>
__device__ __forceinline__ void rotate_dm(StateTiles<T, D, MP>& Z, const float* rot, int w, int r)
{
    using GG = Geo<T, D, MP>;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o) {
        const int mt = w + GG::NW * o;
        if (mt < GG::NMT) {
            const float cc = rot[16 * mt + r], ss = CONJ ? -rot[MP + 16 * mt + r] : rot[MP + 16 * mt + r];
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) {
                const floatx4 re = Z[o][0][dt], im = Z[o][1][dt];
                Z[o][0][dt] = cc * re - ss * im;
                Z[o][1][dt] = ss * re + cc * im;
            }
        }
    }
}

// Pre-rotated phase (cos, sin) of m w n for one mode, n an exact token count.
__device__ __forceinline__ void bwd_phase(int m, long long n, double rT, float& c, float& s)
{
    anchor_phase(m, n, rT, c, s);
}

// ---------------------------------------------------------------------------------
// Forward summaries: per (b, h, segment) the pre-rotated state after the segment's tokens,
// from a zero state, stored as [k|v][re|im][MP][D].
template <typename T, int D, int MP>
__global__ __launch_bounds__(kThreads) void bwd_fsum_kernel(BwdArgs a)
{
    using GG = Geo<T, D, MP>;
    constexpr int C = GG::C, LDK = C + GG::PAD;
    __shared__ __attribute__((aligned(16))) T lds[2 * D * LDK];
    T* Kt = lds;
    T* Vt = lds + D * LDK;
    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int seg = blockIdx.x % a.nseg, bh = blockIdx.x / a.nseg, h = bh % a.H;
    const int ch0 = seg * a.cps, nch = min(a.cps, a.nch - ch0);
    const T* kb_ = (const T*)a.k + (size_t)bh * a.L * D;
    const T* vb = (const T*)a.v + (size_t)bh * a.L * D;
    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    const T* Erev = (const T*)a.ErevT + (size_t)h * 2 * MP * C;

    StateTiles<T, D, MP> Zk, Zv;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) Zk[o][p][dt] = Zv[o][p][dt] = zero4();

    BStage<T, D, 2> st;
    {
        const int tok0 = ch0 * C;
        const T* src[2] = {kb_ + (size_t)tok0 * D, vb + (size_t)tok0 * D};
        if (nch > 0) bstage_load<T, D, 2>(st, src, min(C, a.L - tok0), tid);
    }
    for (int n = 0; n < nch; ++n) {
        const int tok0 = (ch0 + n) * C, c = min(C, a.L - tok0);
        __syncthreads();
        T* tr[2] = {Kt, Vt};
        bstage_store<T, D, 2, false>(st, nullptr, tr, 0, LDK, c, tid);
        if (n + 1 < nch) {
            const int tn = tok0 + C;
            const T* src[2] = {kb_ + (size_t)tn * D, vb + (size_t)tn * D};
            bstage_load<T, D, 2>(st, src, min(C, a.L - tn), tid);
        }
        __syncthreads();
        rotate_dm<T, D, MP, false>(Zk, E32h + (size_t)c * 2 * MP, w, r);
        rotate_dm<T, D, MP, false>(Zv, E32h + (size_t)c * 2 * MP, w, r);
        bwd_accumulate<T, D, MP>(Zk, Zv, Kt, Vt, LDK, Erev, E32h, c, w, g, r);
    }
    float* S = a.fsum + ((size_t)bh * a.nseg + seg) * 4 * MP * D;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o) {
        const int mt = w + GG::NW * o;
        if (mt < GG::NMT) {
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < GG::NDT; ++dt) {
                    st4f(S + ((size_t)p * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zk[o][p][dt]);
                    st4f(S + ((size_t)(2 + p) * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zv[o][p][dt]);
                }
        }
    }
}

// ---------------------------------------------------------------------------------
// The reverse walk over one (b, h, segment).  SUM: adjoint summary only (segments 1..nseg-1,
// from a zero adjoint at the segment end; no dq / dk / dv).
template <typename T, int D, int MP, int SP, bool SUM>
__global__ __launch_bounds__(kThreads) void bwd_kernel(BwdArgs a)
{
    using GG = Geo<T, D, MP>;
    using P = Bwd<T, D, MP, SP>;
    using F = typename Frag<T>::type;
    constexpr int C = GG::C, NT = GG::NT, NW = GG::NW, NMT = GG::NMT, NDT = GG::NDT, OWN = GG::OWN;
    constexpr int KBD = GG::KBD, KBM = GG::KBM, KBC = GG::KBC, NST = P::NST, KBS = P::KBS;
    constexpr int LDQ = P::LDQ, LDK = P::LDK, LDU = P::LDU;
    __shared__ __attribute__((aligned(16))) char lds_raw[P::LDS_BYTES];
    // region A: row-major token tiles, then the H tiles [key][query]
    T* Qs = reinterpret_cast<T*>(lds_raw);
    T* Ks = Qs + (size_t)C * LDQ;
    T* Vs = Ks + (size_t)C * LDQ;
    T* dOs = Vs + (size_t)C * LDQ;
    T* HqT = Qs;
    T* HvT = HqT + (size_t)C * LDK;
    // region T: transposed token tiles
    T* Kt = Qs + P::A_ELEMS;
    T* Vt = Kt + (size_t)D * LDK;
    T* Qt = Vt + (size_t)D * LDK;
    T* dOt = Qt + (size_t)D * LDK;
    // region G: Gram tiles [query][key]
    T* GT = Kt + P::T_ELEMS;
    T* GdT = GT + (size_t)C * LDK;
    // region B: U and Y [token][Re m | Im m], then conj(Wq'')^T and conj(W'')^T [Re m | Im m][token]
    T* UT = GT + P::G_ELEMS;
    T* YT = UT + (size_t)C * LDU;
    T* WqT = UT;
    T* WvT = WqT + (size_t)2 * MP * LDK;
    // region Z: [d][Re m | -Im m] of Z'_k for dq, then [d][Re m | Im m] of the adjoints
    T* ZkT = WqT + P::B_ELEMS;
    T* GkT = ZkT;
    T* GvT = ZkT + (size_t)D * LDU;
    int* sTheta = reinterpret_cast<int*>(ZkT + P::Z_ELEMS);

    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nsu = SUM ? a.nseg - 1 : a.nseg;
    const int seg = blockIdx.x % nsu + (SUM ? 1 : 0), bh = blockIdx.x / nsu, h = bh % a.H;
    const int ch0 = seg * a.cps, nch = min(a.cps, a.nch - ch0);
    const T* qb = (const T*)a.q + (size_t)bh * a.L * D;
    const T* kb_ = (const T*)a.k + (size_t)bh * a.L * D;
    const T* vb = (const T*)a.v + (size_t)bh * a.L * D;
    const T* gb = (const T*)a.dO + (size_t)bh * a.L * D;
    const float* E32h0 = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    const T* Etab0 = (const T*)a.Etab + (size_t)h * C * 2 * MP;
    const T* Ebar0 = (const T*)a.EbarT + (size_t)h * 2 * MP * C;
    const T* Erev0 = (const T*)a.ErevT + (size_t)h * 2 * MP * C;
    const T* ABs0 = (const T*)a.ABs;
    const T* ABm0 = (const T*)a.ABm;
    const double rT = a.rperiod[h];
    const float* rho1 = E32h0 + 2 * MP;
    const float iscale = 1.f / a.scale;

    for (int i = tid; i < SP; i += kThreads) sTheta[i] = a.theta[(size_t)h * SP + i];

    // first (last in time) chunk's staging loads go out before the set-up
    BStage<T, D, 4> st;
    if (nch > 0) {
        const int tok0 = (ch0 + nch - 1) * C;
        const T* src[4] = {kb_ + (size_t)tok0 * D, vb + (size_t)tok0 * D, qb + (size_t)tok0 * D,
                           gb + (size_t)tok0 * D};
        bstage_load<T, D, 4>(st, src, min(C, a.L - tok0), tid);
    }

    // ---- forward state after the segment (pre-rotated, [d][m] tiles): Horner over the
    // forward summaries of segments 0..seg from the input state
    StateTiles<T, D, MP> Zk, Zv, Gk, Gv;
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = w + NW * o;
        const int m = 16 * mt + r;
        const bool live = mt < NMT;
        const float c1 = live ? rho1[m] : 0.f, s1 = live ? rho1[MP + m] : 0.f;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            floatx4 kr = zero4(), ki = zero4(), vr = zero4(), vi = zero4();
            if (live && m < a.M) {
                if (a.sk_in) {
                    kr = ld4f(a.sk_in + (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + 4 * g);
                    ki = ld4f(a.sk_in + (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + 4 * g);
                }
                if (a.sv_in) {
                    vr = ld4f(a.sv_in + (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + 4 * g);
                    vi = ld4f(a.sv_in + (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + 4 * g);
                }
            }
            Zk[o][0][dt] = c1 * kr - s1 * ki;
            Zk[o][1][dt] = s1 * kr + c1 * ki;
            Zv[o][0][dt] = c1 * vr - s1 * vi;
            Zv[o][1][dt] = s1 * vr + c1 * vi;
        }
    }
    for (int sg = 0; sg <= seg; ++sg) {
        const long long len = (long long)min(a.cps * C, a.L - sg * a.cps * C);
        const float* S = a.fsum + ((size_t)bh * a.nseg + sg) * 4 * MP * D;
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
            if (mt < NMT) {
                const int m = 16 * mt + r;
                float cc, ss;
                bwd_phase(m, len, rT, cc, ss);
#pragma unroll
                for (int p2 = 0; p2 < 2; ++p2) {
                    StateTiles<T, D, MP>& Z = p2 ? Zv : Zk;
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const floatx4 re = Z[o][0][dt], im = Z[o][1][dt];
                        const floatx4 sr = ld4f(S + ((size_t)(2 * p2 + 0) * MP + m) * D + 16 * dt + 4 * g);
                        const floatx4 si = ld4f(S + ((size_t)(2 * p2 + 1) * MP + m) * D + 16 * dt + 4 * g);
                        Z[o][0][dt] = cc * re - ss * im + sr;
                        Z[o][1][dt] = ss * re + cc * im + si;
                    }
                }
            }
        }
    }

    // ---- adjoint after the segment (pre-rotated, [m][d] tiles): Horner over the adjoint
    // summaries of the later segments from rho dLoss/d(final states)
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = w + NW * o;
        const bool live = mt < NMT;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            floatx4 kr = zero4(), ki = zero4(), vr = zero4(), vi = zero4();
            if (!SUM && live) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = 16 * mt + 4 * g + e;
                    if (m < a.M) {
                        float c1 = rho1[m], s1 = rho1[MP + m];
                        float xr = 0.f, xi = 0.f, yr = 0.f, yi = 0.f;
                        if (a.gk_out) {
                            xr = a.gk_out[(((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + r];
                            xi = a.gk_out[(((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + r];
                        }
                        if (a.gv_out) {
                            yr = a.gv_out[(((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + r];
                            yi = a.gv_out[(((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + r];
                        }
                        kr[e] = c1 * xr - s1 * xi;
                        ki[e] = s1 * xr + c1 * xi;
                        vr[e] = c1 * yr - s1 * yi;
                        vi[e] = s1 * yr + c1 * yi;
                    }
                }
            }
            Gk[o][0][dt] = kr;
            Gk[o][1][dt] = ki;
            Gv[o][0][dt] = vr;
            Gv[o][1][dt] = vi;
        }
    }
    if constexpr (!SUM) {
        for (int sg = a.nseg - 1; sg > seg; --sg) {
            const long long len = (long long)min(a.cps * C, a.L - sg * a.cps * C);
            const float* S = a.asum + ((size_t)bh * a.nseg + sg) * 4 * MP * D;
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt < NMT) {
                    floatx4 cc, ss;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float ce, se;
                        bwd_phase(16 * mt + 4 * g + e, len, rT, ce, se);
                        cc[e] = ce;
                        ss[e] = se;
                    }
#pragma unroll
                    for (int p2 = 0; p2 < 2; ++p2) {
                        StateTiles<T, D, MP>& Gm = p2 ? Gv : Gk;
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) {
                            floatx4 sr, si;
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                const int m = 16 * mt + 4 * g + e;
                                sr[e] = S[((size_t)(2 * p2 + 0) * MP + m) * D + 16 * dt + r];
                                si[e] = S[((size_t)(2 * p2 + 1) * MP + m) * D + 16 * dt + r];
                            }
                            const floatx4 re = Gm[o][0][dt], im = Gm[o][1][dt];
                            Gm[o][0][dt] = cc * re + ss * im + sr;
                            Gm[o][1][dt] = cc * im - ss * re + si;
                        }
                    }
                }
            }
        }
    }

    for (int n = nch - 1; n >= 0; --n) {
        const int tok0 = (ch0 + n) * C;
        const int c = min(C, a.L - tok0);
        // Table pointers made opaque to the optimiser once per chunk: the table fragments are
        // then re-read from the cache where they are used instead of being hoisted out of the
        // loop into registers (which would spill).
        const T* Etab = opaque(Etab0);
        const T* Ebar = opaque(Ebar0);
        const T* Erev = opaque(Erev0);
        const T* ABs = opaque(ABs0);
        const T* ABm = opaque(ABm0);
        const float* E32h = opaque(E32h0);
        const float* rhoc = E32h + (size_t)c * 2 * MP;
        __syncthreads();  // previous chunk done with every LDS region
        {
            T* rows[4] = {Ks, Vs, Qs, dOs};
            T* trs[4] = {Kt, Vt, Qt, dOt};
            bstage_store<T, D, 4, true>(st, rows, trs, LDQ, LDK, c, tid);
        }
        __syncthreads();  // staged tiles visible

        // ---- phase 1 (mode tiles): rebuild the entering state; publish Z'_k for dq; the
        // Gram tiles of key tile w
#pragma unroll
        for (int o = 0; o < OWN; ++o)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    Zk[o][p][dt] = -Zk[o][p][dt];
                    Zv[o][p][dt] = -Zv[o][p][dt];
                }
        bwd_accumulate<T, D, MP>(Zk, Zv, Kt, Vt, LDK, Erev, E32h, c, w, g, r);
#pragma unroll
        for (int o = 0; o < OWN; ++o)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    Zk[o][p][dt] = -Zk[o][p][dt];
                    Zv[o][p][dt] = -Zv[o][p][dt];
                }
        rotate_dm<T, D, MP, true>(Zk, rhoc, w, r);
        rotate_dm<T, D, MP, true>(Zv, rhoc, w, r);
        if constexpr (!SUM) {
            // [d][Re m | -Im m] of Z'_k (the A operand of Re(Wq'' Z'_k))
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt < NMT) {
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const size_t row = (size_t)(16 * dt + 4 * g + e) * LDU;
                            ZkT[row + 16 * mt + r] = (T)Zk[o][0][dt][e];
                            ZkT[row + MP + 16 * mt + r] = (T)(-Zk[o][1][dt][e]);
                        }
                }
            }
        }
        {
            F kf[KBD], vf[KBD];
#pragma unroll
            for (int kb = 0; kb < KBD; ++kb) {
                kf[kb] = ld_frag<T>(Ks + (size_t)(16 * w + r) * LDQ, 32 * kb, g);
                vf[kb] = ld_frag<T>(Vs + (size_t)(16 * w + r) * LDQ, 32 * kb, g);
            }
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) {
                if (ct < w) continue;
                const int j = 16 * ct + r;
                floatx4 ga = zero4(), gd = zero4();
#pragma unroll
                for (int kb = 0; kb < KBD; ++kb) {
                    ga = mma(kf[kb], ld_frag<T>(Qs + (size_t)j * LDQ, 32 * kb, g), ga);
                    gd = mma(vf[kb], ld_frag<T>(dOs + (size_t)j * LDQ, 32 * kb, g), gd);
                }
                if (ct == w) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (4 * g + e > r) ga[e] = gd[e] = 0.f;
                }
                st4<T>(GT + (size_t)j * LDK + 16 * w + 4 * g, ga);
                st4<T>(GdT + (size_t)j * LDK + 16 * w + 4 * g, gd);
            }
        }
        __syncthreads();  // Gram tiles visible

        // ---- phase 2 (mode tiles): U = E o (Q Z'_k^T + G conj(E)) and Y = E o (dO Z'_v^T +
        // Gd conj(E)), one query tile at a time, published as [token][Re m | Im m]
        {
            F zkf[OWN][2][KBD], zvf[OWN][2][KBD];
#pragma unroll
            for (int o = 0; o < OWN; ++o)
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int kb = 0; kb < KBD; ++kb) {
                        zkf[o][p][kb] = frag_from_acc<T>(Zk[o][p][2 * kb], Zk[o][p][2 * kb + 1]);
                        zvf[o][p][kb] = frag_from_acc<T>(Zv[o][p][2 * kb], Zv[o][p][2 * kb + 1]);
                    }
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) {
                const int j = 16 * ct + r;
                F qf[KBD], of[KBD];
#pragma unroll
                for (int kb = 0; kb < KBD; ++kb) {
                    qf[kb] = ld_frag<T>(Qs + (size_t)j * LDQ, 32 * kb, g);
                    of[kb] = ld_frag<T>(dOs + (size_t)j * LDQ, 32 * kb, g);
                }
#pragma unroll
                for (int o = 0; o < OWN; ++o) {
                    const int mt = w + NW * o;
                    if (mt >= NMT) continue;
                    floatx4 u[2], y[2];
#pragma unroll
                    for (int p = 0; p < 2; ++p) {
                        u[p] = y[p] = zero4();
#pragma unroll
                        for (int kb = 0; kb < KBD; ++kb) {
                            u[p] = mma(zkf[o][p][kb], qf[kb], u[p]);
                            y[p] = mma(zvf[o][p][kb], of[kb], y[p]);
                        }
                    }
#pragma unroll
                    for (int kb = 0; kb < KBC; ++kb) {
                        if (2 * kb <= ct) {
                            const T* grow = GT + (size_t)j * LDK;
                            const T* drow = GdT + (size_t)j * LDK;
                            const bool full = 2 * kb + 1 <= ct;
                            const F gf = full ? ld_frag<T>(grow, 32 * kb, g) : ld_frag_lo<T>(grow, 32 * kb, g);
                            const F df = full ? ld_frag<T>(drow, 32 * kb, g) : ld_frag_lo<T>(drow, 32 * kb, g);
#pragma unroll
                            for (int p = 0; p < 2; ++p) {
                                const F ef = ld_frag<T>(Ebar + (size_t)(16 * (p * NMT + mt) + r) * C, 32 * kb, g);
                                u[p] = mma(ef, gf, u[p]);
                                y[p] = mma(ef, df, y[p]);
                            }
                        }
                    }
                    const floatx4 cs = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + 16 * mt + 4 * g));
                    const floatx4 sn = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + MP + 16 * mt + 4 * g));
                    st4<T>(UT + (size_t)j * LDU + 16 * mt + 4 * g, cs * u[0] - sn * u[1]);
                    st4<T>(UT + (size_t)j * LDU + MP + 16 * mt + 4 * g, sn * u[0] + cs * u[1]);
                    st4<T>(YT + (size_t)j * LDU + 16 * mt + 4 * g, cs * y[0] - sn * y[1]);
                    st4<T>(YT + (size_t)j * LDU + MP + 16 * mt + 4 * g, sn * y[0] + cs * y[1]);
                }
            }
        }
        __syncthreads();  // U and Y visible; the row-major token tiles are no longer read

        // ---- phase 3 (query tile w): scores, softmax and its gradient, the readout weights
        // W'' and Wq'' (published conjugated and transposed), the H tiles, dq
        {
            const int j = 16 * w + r;
            const long long pos = a.t0 + tok0 + j;
            F uf[KBM], yf[KBM];
#pragma unroll
            for (int kb = 0; kb < KBM; ++kb) {
                uf[kb] = ld_frag<T>(UT + (size_t)j * LDU, 32 * kb, g);
                yf[kb] = ld_frag<T>(YT + (size_t)j * LDU, 32 * kb, g);
            }
            floatx4 sc[NST], dp[NST];
#pragma unroll
            for (int s4 = 0; s4 < NST; ++s4) {
                sc[s4] = dp[s4] = zero4();
#pragma unroll
                for (int kb = 0; kb < KBM; ++kb) {
                    const F af = ld_frag<T>(ABs + (size_t)(16 * s4 + r) * 2 * MP, 32 * kb, g);
                    sc[s4] = mma(af, uf[kb], sc[s4]);
                    dp[s4] = mma(af, yf[kb], dp[s4]);
                }
            }
            __syncthreads();  // every wave holds its U, Y rows: their buffer takes the weights
            float mx = -INFINITY;
#pragma unroll
            for (int s4 = 0; s4 < NST; ++s4) {
                const intx4 th = *reinterpret_cast<const intx4*>(sTheta + 16 * s4 + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (pos < (long long)th[e]) sc[s4][e] = -INFINITY;
                    mx = fmaxf(mx, sc[s4][e]);
                }
            }
            mx = rows_max(mx);
            float sum = 0.f;
#pragma unroll
            for (int s4 = 0; s4 < NST; ++s4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float ex = __expf(sc[s4][e] - mx);
                    sc[s4][e] = ex;
                    sum += ex;
                }
            sum = rows_sum(sum);
            const float inv = __builtin_amdgcn_rcpf(sum);  // sum >= 1: the maximum slot contributes exp(0)
            float pd = 0.f;
#pragma unroll
            for (int s4 = 0; s4 < NST; ++s4) {
                sc[s4] = sc[s4] * inv;
                dp[s4] = dp[s4] * iscale;
#pragma unroll
                for (int e = 0; e < 4; ++e) pd += sc[s4][e] * dp[s4][e];
            }
            pd = rows_sum(pd);
            F pf[KBS], zf[KBS];
#pragma unroll
            for (int kb = 0; kb < KBS; ++kb) {
                pf[kb] = frag_from_acc<T>(sc[2 * kb], sc[2 * kb + 1]);
                zf[kb] = frag_from_acc<T>(sc[2 * kb] * (dp[2 * kb] - pd), sc[2 * kb + 1] * (dp[2 * kb + 1] - pd));
            }
            // readout weights of the values, W'' = (P A - i P B) o E (E = rho^j), and H_v
            {
                floatx4 wa[2 * NMT];
#pragma unroll
                for (int t = 0; t < 2 * NMT; ++t) {
                    wa[t] = zero4();
#pragma unroll
                    for (int kb = 0; kb < KBS; ++kb)
                        wa[t] = mma(ld_frag<T>(ABm + (size_t)(16 * t + r) * SP, 32 * kb, g), pf[kb], wa[t]);
                }
#pragma unroll
                for (int mt = 0; mt < NMT; ++mt) {
                    const floatx4 cs = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + 16 * mt + 4 * g));
                    const floatx4 sn = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + MP + 16 * mt + 4 * g));
                    const floatx4 am = wa[mt], bm = wa[NMT + mt];
                    wa[mt] = am * cs + bm * sn;
                    wa[NMT + mt] = am * sn - bm * cs;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const size_t re = (size_t)(16 * mt + 4 * g + e) * LDK + j;
                        WvT[re] = (T)wa[mt][e];
                        WvT[re + (size_t)MP * LDK] = (T)(-wa[NMT + mt][e]);
                    }
                }
                if constexpr (!SUM) {
                    F wf[KBM];
#pragma unroll
                    for (int kb = 0; kb < KBM; ++kb) wf[kb] = frag_from_acc<T>(wa[2 * kb], wa[2 * kb + 1]);
#pragma unroll
                    for (int kt = 0; kt < NT; ++kt) {
                        floatx4 hv = zero4();
                        if (kt <= w) {
#pragma unroll
                            for (int kb = 0; kb < KBM; ++kb)
                                hv = mma(ld_frag<T>(Etab + (size_t)(16 * kt + r) * 2 * MP, 32 * kb, g), wf[kb], hv);
                            if (kt == w) {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (4 * g + e > r) hv[e] = 0.f;
                            }
                        }
#pragma unroll
                        for (int e = 0; e < 4; ++e) HvT[(size_t)(16 * kt + 4 * g + e) * LDK + j] = (T)hv[e];
                    }
                }
            }
            // score-gradient weights Wq'' = scale (dz A - i dz B) o E, H_q and dq
            {
                floatx4 wq[2 * NMT];
#pragma unroll
                for (int t = 0; t < 2 * NMT; ++t) {
                    wq[t] = zero4();
#pragma unroll
                    for (int kb = 0; kb < KBS; ++kb)
                        wq[t] = mma(ld_frag<T>(ABm + (size_t)(16 * t + r) * SP, 32 * kb, g), zf[kb], wq[t]);
                }
#pragma unroll
                for (int mt = 0; mt < NMT; ++mt) {
                    const floatx4 cs = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + 16 * mt + 4 * g));
                    const floatx4 sn = to_f4(ld4<T>(Etab + (size_t)j * 2 * MP + MP + 16 * mt + 4 * g));
                    const floatx4 am = wq[mt] * a.scale, bm = wq[NMT + mt] * a.scale;
                    wq[mt] = am * cs + bm * sn;
                    wq[NMT + mt] = am * sn - bm * cs;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const size_t re = (size_t)(16 * mt + 4 * g + e) * LDK + j;
                        WqT[re] = (T)wq[mt][e];
                        WqT[re + (size_t)MP * LDK] = (T)(-wq[NMT + mt][e]);
                    }
                }
                if constexpr (!SUM) {
                    F qf2[KBM];
#pragma unroll
                    for (int kb = 0; kb < KBM; ++kb) qf2[kb] = frag_from_acc<T>(wq[2 * kb], wq[2 * kb + 1]);
                    floatx4 oa[NDT];
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        oa[dt] = zero4();
#pragma unroll
                        for (int kb = 0; kb < KBM; ++kb)
                            oa[dt] = mma(ld_frag<T>(ZkT + (size_t)(16 * dt + r) * LDU, 32 * kb, g), qf2[kb], oa[dt]);
                    }
                    floatx4 hq[NT];
#pragma unroll
                    for (int kt = 0; kt < NT; ++kt) {
                        hq[kt] = zero4();
                        if (kt <= w) {
#pragma unroll
                            for (int kb = 0; kb < KBM; ++kb)
                                hq[kt] = mma(ld_frag<T>(Etab + (size_t)(16 * kt + r) * 2 * MP, 32 * kb, g), qf2[kb], hq[kt]);
                            if (kt == w) {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (4 * g + e > r) hq[kt][e] = 0.f;
                            }
                        }
#pragma unroll
                        for (int e = 0; e < 4; ++e) HqT[(size_t)(16 * kt + 4 * g + e) * LDK + j] = (T)hq[kt][e];
                    }
#pragma unroll
                    for (int kb = 0; kb < KBC; ++kb) {
                        if (2 * kb <= w) {
                            const F hf = frag_from_acc<T>(hq[2 * kb], hq[2 * kb + 1]);
#pragma unroll
                            for (int dt = 0; dt < NDT; ++dt)
                                oa[dt] = mma(ld_frag<T>(Kt + (size_t)(16 * dt + r) * LDK, 32 * kb, g), hf, oa[dt]);
                        }
                    }
                    if (j < c) {
                        T* dqb = (T*)a.dq + ((size_t)bh * a.L + tok0 + j) * D;
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) st4<T>(dqb + 16 * dt + 4 * g, oa[dt]);
                    }
                }
            }
        }
        __syncthreads();  // Z'_k no longer read; H tiles and weights visible

        // ---- phase 3b: publish the adjoints (after the chunk) as [d][Re m | Im m]; the next
        // chunk's loads go out
        if constexpr (!SUM) {
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt < NMT) {
#pragma unroll
                    for (int p = 0; p < 2; ++p)
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) {
                            st4<T>(GkT + (size_t)(16 * dt + r) * LDU + p * MP + 16 * mt + 4 * g, Gk[o][p][dt]);
                            st4<T>(GvT + (size_t)(16 * dt + r) * LDU + p * MP + 16 * mt + 4 * g, Gv[o][p][dt]);
                        }
                }
            }
        }
        if (n > 0) {
            const int tp = tok0 - C;
            const T* src[4] = {kb_ + (size_t)tp * D, vb + (size_t)tp * D, qb + (size_t)tp * D, gb + (size_t)tp * D};
            bstage_load<T, D, 4>(st, src, C, tid);
        }
        if constexpr (!SUM) __syncthreads();  // adjoint operands visible

        // ---- phase 4: dk, dv of key tile w; the adjoint advances to the chunk's start
        if constexpr (!SUM) {
            const int j = 16 * w + r;
            floatx4 ka[NDT], va[NDT];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) ka[dt] = va[dt] = zero4();
#pragma unroll
            for (int kb = 0; kb < KBC; ++kb) {
                const F hf = ld_frag<T>(HqT + (size_t)j * LDK, 32 * kb, g);
                const F vf2 = ld_frag<T>(HvT + (size_t)j * LDK, 32 * kb, g);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    ka[dt] = mma(ld_frag<T>(Qt + (size_t)(16 * dt + r) * LDK, 32 * kb, g), hf, ka[dt]);
                    va[dt] = mma(ld_frag<T>(dOt + (size_t)(16 * dt + r) * LDK, 32 * kb, g), vf2, va[dt]);
                }
            }
            // Re(conj(rho^{c-j}) Gam'): the B operand is row c - j of the float32 phase table
#pragma unroll
            for (int kb = 0; kb < KBM; ++kb) {
                F ef;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int col = 32 * kb + 16 * (e / 4) + 4 * g + (e % 4);
                    ef[e] = (T)(j < c ? E32h[(size_t)(c - j) * 2 * MP + col] : 0.f);
                }
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    ka[dt] = mma(ld_frag<T>(GkT + (size_t)(16 * dt + r) * LDU, 32 * kb, g), ef, ka[dt]);
                    va[dt] = mma(ld_frag<T>(GvT + (size_t)(16 * dt + r) * LDU, 32 * kb, g), ef, va[dt]);
                }
            }
            if (j < c) {
                T* dkb = (T*)a.dk + ((size_t)bh * a.L + tok0 + j) * D;
                T* dvb = (T*)a.dv + ((size_t)bh * a.L + tok0 + j) * D;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    st4<T>(dkb + 16 * dt + 4 * g, ka[dt]);
                    st4<T>(dvb + 16 * dt + 4 * g, va[dt]);
                }
            }
        }
        // Gam' <- conj(rho^c) o Gam' + [conj(Wq'')^T Q | conj(W'')^T dO]  ([m][d] tiles)
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
            if (mt < NMT) {
                const floatx4 cc = ld4f(rhoc + 16 * mt + 4 * g), ss = ld4f(rhoc + MP + 16 * mt + 4 * g);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    floatx4 re = Gk[o][0][dt], im = Gk[o][1][dt];
                    Gk[o][0][dt] = cc * re + ss * im;
                    Gk[o][1][dt] = cc * im - ss * re;
                    re = Gv[o][0][dt];
                    im = Gv[o][1][dt];
                    Gv[o][0][dt] = cc * re + ss * im;
                    Gv[o][1][dt] = cc * im - ss * re;
                }
#pragma unroll
                for (int kb = 0; kb < KBC; ++kb) {
                    F qt[NDT], ot[NDT];
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        qt[dt] = ld_frag<T>(Qt + (size_t)(16 * dt + r) * LDK, 32 * kb, g);
                        ot[dt] = ld_frag<T>(dOt + (size_t)(16 * dt + r) * LDK, 32 * kb, g);
                    }
#pragma unroll
                    for (int p = 0; p < 2; ++p) {
                        const F wkf = ld_frag<T>(WqT + (size_t)(p * MP + 16 * mt + r) * LDK, 32 * kb, g);
                        const F wvf = ld_frag<T>(WvT + (size_t)(p * MP + 16 * mt + r) * LDK, 32 * kb, g);
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) {
                            Gk[o][p][dt] = mma(wkf, qt[dt], Gk[o][p][dt]);
                            Gv[o][p][dt] = mma(wvf, ot[dt], Gv[o][p][dt]);
                        }
                    }
                }
            }
        }
    }

    // ---- the adjoint at the segment's start
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = w + NW * o;
        if (mt >= NMT) continue;
        if constexpr (SUM) {
            float* S = a.asum + ((size_t)bh * a.nseg + seg) * 4 * MP * D;
#pragma unroll
            for (int p2 = 0; p2 < 2; ++p2) {
                StateTiles<T, D, MP>& Gm = p2 ? Gv : Gk;
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            S[((size_t)(2 * p2 + p) * MP + 16 * mt + 4 * g + e) * D + 16 * dt + r] = Gm[o][p][dt][e];
            }
        } else {
            if (seg != 0) continue;
            // dLoss/d(input states) = conj(rho) Gam'
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int m = 16 * mt + 4 * g + e;
                if (m >= a.M) continue;
                const float c1 = rho1[m], s1 = rho1[MP + m];
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    const size_t o0 = (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + r;
                    const size_t o1 = (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + r;
                    if (a.gk_in) {
                        const float re = Gk[o][0][dt][e], im = Gk[o][1][dt][e];
                        a.gk_in[o0] = c1 * re + s1 * im;
                        a.gk_in[o1] = c1 * im - s1 * re;
                    }
                    if (a.gv_in) {
                        const float re = Gv[o][0][dt][e], im = Gv[o][1][dt][e];
                        a.gv_in[o0] = c1 * re + s1 * im;
                        a.gv_in[o1] = c1 * im - s1 * re;
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------
template <typename T, int D, int MP, int SP>
hipError_t launch_backward_shape(const BwdArgs& a, hipStream_t s, void* const* ev)
{
    if (a.nbk != a.nseg || a.cpb != a.cps) return hipErrorInvalidValue;  // one summary block per segment
    auto mark = [&](int i) -> hipError_t {
        return (ev && ev[i]) ? hipEventRecord((hipEvent_t)ev[i], s) : hipSuccess;
    };
    const unsigned units = (unsigned)(a.B * a.H);
    hipLaunchKernelGGL((bwd_fsum_kernel<T, D, MP>), dim3(units * a.nseg), dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || (e = mark(0)) != hipSuccess) return e;
    if (a.nseg > 1) {
        hipLaunchKernelGGL((bwd_kernel<T, D, MP, SP, true>), dim3(units * (a.nseg - 1)), dim3(kThreads), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = mark(1)) != hipSuccess) return e;
    hipLaunchKernelGGL((bwd_kernel<T, D, MP, SP, false>), dim3(units * a.nseg), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return mark(2);
}

}  // namespace bla
