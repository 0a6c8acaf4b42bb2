// Backward pass of the chunked BLA operator, bf16 operands: the same gradients and the same
// reverse walk as bla_backward.h (whose header states the per-chunk algebra), reorganised so
// that every table read inside the chunk loop comes from LDS.
//
//  * Token tiles (K, V, Q, dO) are staged once, row-major; the orientation with the reduction
//    over tokens is read with the transposing LDS load (ld_frag_tr).
//  * The head's phase table is held in LDS as conj(rho^i) = [cos | -sin] (row i).  It serves the
//    twiddles, the transposed operands of G conj(E), the state rebuilt by subtraction,
//        Z'_in = conj(rho^c) o Z'_out - sum_i conj(rho^i) [k_i | v_i],
//    the H tiles and the adjoint terms of dk and dv without a sign change, when the readout
//    weights are kept as [Re W'' | -Im W''] (which is also conj(W'') as the adjoint update uses
//    it).  The slot matrix scale (A | B) is held once; its transpose (the reduction over slots)
//    is read with ld_frag_tr.
//  * The adjoint is split by head-dim tiles (wave w owns d-tile w, for all modes), so the
//    adjoint terms of dk and dv, Re(rho^j o conj(rho^c) Gam'), are contractions of the wave's
//    own registers against the phase table: no adjoint is published through LDS.
//  * The forward summaries use Z' <- rho^c o (Z' + sum_i conj(rho^i) [k_i | v_i]).
#pragma once

#include "bla_backward.h"
#include "bla_forward_pair.h"

namespace bla {

template <int D, int MP, int SP> struct Bwd16 {
    static constexpr int C = kChunk, NT = C / 16, NW = kThreads / 64;
    static constexpr int NMT = MP / 16, NDT = D / 16, NST = SP / 16;
    static constexpr int KBD = D / 32, KBM = 2 * MP / 32, KBC = C / 32, KBS = SP / 32;
    static constexpr int OWN = (NMT + NW - 1) / NW;   // mode tiles of the forward state per wave
    static constexpr int ODT = (NDT + NW - 1) / NW;   // head-dim tiles of the adjoint per wave
    static constexpr int LDQ = D + 12;                // token tiles [C][LDQ] (read both ways)
    static constexpr int LDK = C + 4;                 // Gram tiles [C][LDK]
    static constexpr int LDU = 2 * MP + 4;            // U, Y [C][LDU]
    static constexpr int LE = 2 * MP + 12;            // phase table [C][LE]; slot matrix [SP][LE]
    // Tiles written row-major by the wave that produces them (8-byte stores) and read
    // transposed (ds_read_b64_tr_b16).  Where the LDS allows it without costing a workgroup
    // per compute unit (PS), they are piece-swizzled (pswz_col) at row strides of 8 x odd
    // (mod 64) dwords, so that neither the stores nor the transposed reads meet bank conflicts;
    // otherwise a stride of 2 (mod 32) dwords keeps the stores conflict-free.
    static constexpr size_t lds_bytes(int tp)
    {
        const int ldh = C + tp, ldw = 2 * MP + tp, ldz = D + tp;
        return ((size_t)4 * C * LDQ + (size_t)2 * C * (ldh > LDK ? ldh : LDK) +
                (size_t)2 * C * (ldw > LDU ? ldw : LDU) + (size_t)2 * MP * ldz + (size_t)C * LE + (size_t)SP * LE) * 2 +
               (size_t)SP * 4 + (size_t)2 * 2 * MP * 4;
    }
    static constexpr bool PS =
        lds_bytes(16) <= kBwdMaxLds && (2 * lds_bytes(16) <= kBwdMaxLds || 2 * lds_bytes(4) > kBwdMaxLds);
    static constexpr int TP = PS ? 16 : 4;
    static constexpr int LDH = C + TP;                // H tiles [query][key]
    static constexpr int LDW = 2 * MP + TP;           // readout weights [token][Re m | Im m]
    static constexpr int LDZ = D + TP;                // Z'_k [Re m | Im m][d]
    __device__ static int tcol(int row, int col) { return PS ? pswz_col(row, col) : col; }
    __device__ static bf16x8 ld_t(const bf16* M, int ld, int x0, int kb, int g, int r)
    {
        return PS ? ld_frag_tr_ps(M, ld, x0, kb, g, r) : ld_frag_tr(M, ld, x0, kb, g, r);
    }
    static constexpr size_t A_ELEMS = (size_t)4 * C * LDQ;
    static constexpr size_t G_ELEMS = (size_t)2 * C * (LDH > LDK ? LDH : LDK);
    static constexpr size_t B_ELEMS = (size_t)2 * C * (LDW > LDU ? LDW : LDU);
    static constexpr size_t Z_ELEMS = (size_t)2 * MP * LDZ;
    static constexpr size_t E_ELEMS = (size_t)C * LE;
    static constexpr size_t S_ELEMS = (size_t)SP * LE;
    static constexpr size_t LDS_BYTES =
        (A_ELEMS + G_ELEMS + B_ELEMS + Z_ELEMS + E_ELEMS + S_ELEMS) * 2 + (size_t)SP * 4 + (size_t)2 * 2 * MP * 4;
    static_assert(LDS_BYTES <= kBwdMaxLds, "backward tiles fit in LDS");
    static_assert((size_t)2 * C * LDH <= G_ELEMS, "H tiles fit in the Gram region");
};

__device__ __forceinline__ bf16x8 neg_frag(bf16x8 f)
{
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    u32x4 u = __builtin_bit_cast(u32x4, f);
    u ^= 0x80008000u;
    return __builtin_bit_cast(bf16x8, u);
}

// Row-major staging of NTEN tensors into [C][ld] tiles (rows past c are zero).
template <int D, int NTEN>
__device__ __forceinline__ void bstage_store_rows(const BStage<bf16, D, NTEN>& st, bf16* const* dst, int ld, int c,
                                                  int tid)
{
    using S = BStage<bf16, D, NTEN>;
    using H = bf16x4;
    const H z = zero_half<bf16>();
#pragma unroll
    for (int i = 0; i < S::PT; ++i) {
        const int u = tid + i * kThreads;
        if ((NTEN * S::UPT) % kThreads == 0 || u < NTEN * S::UPT) {
            const int ten = u / S::UPT, uu = u % S::UPT, dq = uu % (D / 8), tq = uu / (D / 8);
            bf16* rd = dst[ten] + 8 * dq;
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const bool ok = 4 * tq + t < c;
                st_lds<H>(rd + (size_t)(4 * tq + t) * ld, ok ? st.x[i][t][0] : z);
                st_lds<H>(rd + (size_t)(4 * tq + t) * ld + 4, ok ? st.x[i][t][1] : z);
            }
        }
    }
}

// The head's phase table as conj(rho^i) = [cos | -sin] rows into LDS ([C][ld]), from the
// workspace table [C][2MP] of rho^i.
template <int MP>
__device__ __forceinline__ void copy_conj_phase(bf16* dst, int ld, const bf16* src, int tid)
{
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    constexpr int PIECES = kChunk * 2 * MP / 4;
    for (int u = tid; u < PIECES; u += kThreads) {
        const int row = u / (2 * MP / 4), col = (u % (2 * MP / 4)) * 4;
        u32x2 x = *reinterpret_cast<const u32x2*>(src + (size_t)row * 2 * MP + col);
        if (col >= MP) x ^= 0x80008000u;
        *reinterpret_cast<u32x2*>(dst + (size_t)row * ld + col) = x;
    }
}

// cos | sin of m w c (float32, 2MP) for the chunk's length: the LDS row of rho^C, or the
// workspace's phase table for a ragged chunk.
__device__ __forceinline__ const float* rho_row(const float* sRho, int c, int MP)
{
    return c == kChunk ? sRho : sRho + 2 * MP;
}

// sRho[0 .. 2MP): rho^C; sRho[2MP .. 4MP): rho^c of the sequence's last chunk (c = L - (nch-1) C,
// the only chunk that can be shorter).  Both rows live in LDS, so the selected row is read
// with LDS loads (a row chosen between LDS and global memory would be read with flat loads,
// which hold every LDS wait until they return).
__device__ __forceinline__ void load_rho_rows(float* sRho, const float* E32h, const BwdArgs& a, int MP, int tid)
{
    const int c_last = a.L - (a.nch - 1) * kChunk;
    for (int i = tid; i < 2 * MP; i += kThreads) {
        sRho[i] = E32h[(size_t)kChunk * 2 * MP + i];
        sRho[2 * MP + i] = E32h[(size_t)c_last * 2 * MP + i];
    }
}

// ---------------------------------------------------------------------------------
// Forward summaries (bf16): per (b, h, summary block) the pre-rotated state after the block's
// tokens from zero, stored as [k|v][re|im][MP][D] (as bwd_fsum_kernel).
template <int D, int MP>
__global__ __launch_bounds__(kThreads) void bwd16_fsum_kernel(BwdArgs a)
{
    using G = Bwd16<D, MP, 32>;
    constexpr int C = kChunk, NMT = G::NMT, NDT = G::NDT, OWN = G::OWN, NW = G::NW;
    // K, V and the phase table are read only transposed here: row strides of 8 x odd (mod 64)
    // dwords keep those reads free of bank conflicts
    constexpr int LDQ = D + 16, LE = 2 * MP + 16;
    __shared__ __attribute__((aligned(16))) bf16 lds[2 * C * LDQ + C * LE];
    __shared__ __attribute__((aligned(16))) float sRhoC[2 * 2 * MP];
    bf16* Ks = lds;
    bf16* Vs = Ks + C * LDQ;
    bf16* sE = Vs + C * LDQ;
    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int blk = blockIdx.x % a.nbk, bh = blockIdx.x / a.nbk, h = bh % a.H;
    const int ch0 = blk * a.cpb, nch = min(a.cpb, a.nch - ch0);
    const bf16* kb_ = (const bf16*)a.k + (size_t)bh * a.L * D;
    const bf16* vb = (const bf16*)a.v + (size_t)bh * a.L * D;
    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    copy_conj_phase<MP>(sE, LE, (const bf16*)a.Etab + (size_t)h * C * 2 * MP, tid);
    load_rho_rows(sRhoC, E32h, a, MP, tid);

    StateTiles<bf16, D, MP> Zk, Zv;
#pragma unroll
    for (int o = 0; o < OWN; ++o)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) Zk[o][p][dt] = Zv[o][p][dt] = zero4();

    BStage<bf16, D, 2> st;
    if (nch > 0) {
        const int tok0 = ch0 * C;
        const bf16* src[2] = {kb_ + (size_t)tok0 * D, vb + (size_t)tok0 * D};
        bstage_load<bf16, D, 2>(st, src, min(C, a.L - tok0), tid);
    }
    for (int n = 0; n < nch; ++n) {
        const int tok0 = (ch0 + n) * C, c = min(C, a.L - tok0);
        __syncthreads();
        bf16* rows[2] = {Ks, Vs};
        bstage_store_rows<D, 2>(st, rows, LDQ, c, tid);
        if (n + 1 < nch) {
            const int tn = tok0 + C;
            const bf16* src[2] = {kb_ + (size_t)tn * D, vb + (size_t)tn * D};
            bstage_load<bf16, D, 2>(st, src, min(C, a.L - tn), tid);
        }
        __syncthreads();
        // Z' <- rho^c o (Z' + sum_i conj(rho^i) x_i)
#pragma unroll
        for (int kb = 0; kb < G::KBC; ++kb) {
            bf16x8 kf[NDT], vf[NDT];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                kf[dt] = ld_frag_tr(Ks, LDQ, 16 * dt, kb, g, r);
                vf[dt] = ld_frag_tr(Vs, LDQ, 16 * dt, kb, g, r);
            }
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt >= NMT) continue;
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const bf16x8 ef = ld_frag_tr(sE, LE, p * MP + 16 * mt, kb, g, r);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        Zk[o][p][dt] = mma(kf[dt], ef, Zk[o][p][dt]);
                        Zv[o][p][dt] = mma(vf[dt], ef, Zv[o][p][dt]);
                    }
                }
            }
        }
        const float* rc = rho_row(sRhoC, c, MP);
        rotate_dm<bf16, D, MP, false>(Zk, rc, w, r);
        rotate_dm<bf16, D, MP, false>(Zv, rc, w, r);
    }
    float* S = a.fsum + ((size_t)bh * a.nbk + blk) * 4 * MP * D;
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = w + NW * o;
        if (mt < NMT) {
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    st4f(S + ((size_t)p * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zk[o][p][dt]);
                    st4f(S + ((size_t)(2 + p) * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zv[o][p][dt]);
                }
        }
    }
}

// ---------------------------------------------------------------------------------
// The reverse walk over one (b, h, segment), bf16.  SUM: adjoint summary only.
template <int D, int MP, int SP, bool SUM>
__global__ __launch_bounds__(kThreads) void bwd16_kernel(BwdArgs a)
{
    using P = Bwd16<D, MP, SP>;
    using F = bf16x8;
    constexpr int C = P::C, NT = P::NT, NW = P::NW, NMT = P::NMT, NDT = P::NDT, OWN = P::OWN, ODT = P::ODT;
    constexpr int KBD = P::KBD, KBM = P::KBM, KBC = P::KBC, NST = P::NST, KBS = P::KBS;
    constexpr int LDQ = P::LDQ, LDK = P::LDK, LDU = P::LDU, LE = P::LE;
    __shared__ __attribute__((aligned(16))) char lds_raw[P::LDS_BYTES];
    bf16* Ks = reinterpret_cast<bf16*>(lds_raw);            // region A: token tiles, row-major
    bf16* Vs = Ks + (size_t)C * LDQ;
    bf16* Qs = Vs + (size_t)C * LDQ;
    bf16* dOs = Qs + (size_t)C * LDQ;
    bf16* GT = Ks + P::A_ELEMS;                              // region G: Gram tiles, then H tiles
    bf16* GdT = GT + (size_t)C * LDK;
    bf16* HqT = GT;                                          // [query][key], LDH
    bf16* HvT = GT + (size_t)C * P::LDH;
    bf16* UT = GT + P::G_ELEMS;                              // region B: U, Y, then the weights
    bf16* YT = UT + (size_t)C * LDU;
    bf16* WqT = UT;                                          // [token][Re m | Im m], LDW
    bf16* WvT = WqT + (size_t)C * P::LDW;
    bf16* ZkT = UT + P::B_ELEMS;                             // [Re m | Im m][d] of Z'_k, LDZ
    bf16* sE = ZkT + P::Z_ELEMS;                             // conj(rho^i) rows
    bf16* sAB = sE + P::E_ELEMS;                             // scale (A | B) rows
    int* sTheta = reinterpret_cast<int*>(sAB + P::S_ELEMS);
    float* sRhoC = reinterpret_cast<float*>(sTheta + SP);

    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int tid_ = tid, g_ = g, r_ = r;  // the chunk loop re-derives its own copies
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    // SUM: one summary block of a segment but the first; otherwise one segment.  last_blk:
    // the last summary block the walk covers.
    const int bps = a.nbk / a.nseg;
    const int nsu = SUM ? a.nbk - bps : a.nseg;
    const int seg = blockIdx.x % nsu + (SUM ? bps : 0), bh = blockIdx.x / nsu, h = bh % a.H;
    const int cpu = SUM ? a.cpb : a.cps;  // chunks per walked unit (block or segment)
    const int ch0 = seg * cpu, nch = min(cpu, a.nch - ch0);
    const int last_blk = SUM ? seg : (seg + 1) * bps - 1;
    const bf16* qb = (const bf16*)a.q + (size_t)bh * a.L * D;
    const bf16* kb_ = (const bf16*)a.k + (size_t)bh * a.L * D;
    const bf16* vb = (const bf16*)a.v + (size_t)bh * a.L * D;
    const bf16* gb = (const bf16*)a.dO + (size_t)bh * a.L * D;
    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    const double rT = a.rperiod[h];
    const float* rho1 = E32h + 2 * MP;
    const float iscale = 1.f / a.scale;

    // first (last in time) chunk's loads go out before the tables are copied
    BStage<bf16, D, 4> st;
    if (nch > 0) {
        const int tok0 = (ch0 + nch - 1) * C;
        const bf16* src[4] = {kb_ + (size_t)tok0 * D, vb + (size_t)tok0 * D, qb + (size_t)tok0 * D,
                              gb + (size_t)tok0 * D};
        bstage_load<bf16, D, 4>(st, src, min(C, a.L - tok0), tid);
    }
    copy_conj_phase<MP>(sE, LE, (const bf16*)a.Etab + (size_t)h * C * 2 * MP, tid);
    copy_table<bf16, SP, 2 * MP, LE>(sAB, (const bf16*)a.ABs, tid);
    for (int i = tid; i < SP; i += kThreads) sTheta[i] = a.theta[(size_t)h * SP + i];
    load_rho_rows(sRhoC, E32h, a, MP, tid);

    // ---- forward state after the segment (pre-rotated, [d][m] tiles, mode tiles split)
    StateTiles<bf16, D, MP> Zk, Zv;
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
    for (int sg = 0; sg <= last_blk; ++sg) {
        const long long len = (long long)min(a.cpb * C, a.L - sg * a.cpb * C);
        const float* S = a.fsum + ((size_t)bh * a.nbk + sg) * 4 * MP * D;
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
            if (mt < NMT) {
                const int m = 16 * mt + r;
                float cc, ss;
                bwd_phase(m, len, rT, cc, ss);
#pragma unroll
                for (int p2 = 0; p2 < 2; ++p2) {
                    StateTiles<bf16, D, MP>& Z = p2 ? Zv : Zk;
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

    // ---- adjoint after the segment (pre-rotated, [m][d] tiles; wave w owns d-tile w + NW od for
    // every mode tile): Horner over the adjoint summaries of the later segments from
    // rho dLoss/d(final states)
    floatx4 Gk[ODT][2][NMT], Gv[ODT][2][NMT];
#pragma unroll
    for (int od = 0; od < ODT; ++od) {
        const int dt = w + NW * od;
        const bool live = dt < NDT;
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) {
            floatx4 kr = zero4(), ki = zero4(), vr = zero4(), vi = zero4();
            if (!SUM && live) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = 16 * mt + 4 * g + e;
                    if (m < a.M) {
                        const float c1 = rho1[m], s1 = rho1[MP + m];
                        float xr = 0.f, xi = 0.f, yr = 0.f, yi = 0.f;
                        const size_t o0 = (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + r;
                        const size_t o1 = (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + r;
                        if (a.gk_out) {
                            xr = a.gk_out[o0];
                            xi = a.gk_out[o1];
                        }
                        if (a.gv_out) {
                            yr = a.gv_out[o0];
                            yi = a.gv_out[o1];
                        }
                        kr[e] = c1 * xr - s1 * xi;
                        ki[e] = s1 * xr + c1 * xi;
                        vr[e] = c1 * yr - s1 * yi;
                        vi[e] = s1 * yr + c1 * yi;
                    }
                }
            }
            Gk[od][0][mt] = kr;
            Gk[od][1][mt] = ki;
            Gv[od][0][mt] = vr;
            Gv[od][1][mt] = vi;
        }
    }
    if constexpr (!SUM) {
        for (int sg = a.nbk - 1; sg > last_blk; --sg) {
            const long long len = (long long)min(a.cpb * C, a.L - sg * a.cpb * C);
            const float* S = a.asum + ((size_t)bh * a.nbk + sg) * 4 * MP * D;
#pragma unroll
            for (int od = 0; od < ODT; ++od) {
                const int dt = w + NW * od;
                if (dt >= NDT) continue;
#pragma unroll
                for (int mt = 0; mt < NMT; ++mt) {
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
                        floatx4(&Gm)[2][NMT] = p2 ? Gv[od] : Gk[od];
                        floatx4 sr, si;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int m = 16 * mt + 4 * g + e;
                            sr[e] = S[((size_t)(2 * p2 + 0) * MP + m) * D + 16 * dt + r];
                            si[e] = S[((size_t)(2 * p2 + 1) * MP + m) * D + 16 * dt + r];
                        }
                        const floatx4 re = Gm[0][mt], im = Gm[1][mt];
                        Gm[0][mt] = cc * re + ss * im + sr;
                        Gm[1][mt] = cc * im - ss * re + si;
                    }
                }
            }
        }
    }
    __syncthreads();  // tables in LDS

    for (int n = nch - 1; n >= 0; --n) {
        // lane indices re-derived per chunk (opaque_lane): addresses stay inside the loop
        const int r = opaque_lane(r_), g = opaque_lane(g_), tid = opaque_lane(tid_);
        const int tok0 = (ch0 + n) * C;
        const int c = min(C, a.L - tok0);
        const float* rc = rho_row(sRhoC, c, MP);  // rho^c
        __syncthreads();  // previous chunk done with the token tiles and the weights
        {
            bf16* rows[4] = {Ks, Vs, Qs, dOs};
            bstage_store_rows<D, 4>(st, rows, LDQ, c, tid);
        }
        if (n > 0) {
            const int tp = tok0 - C;
            const bf16* src[4] = {kb_ + (size_t)tp * D, vb + (size_t)tp * D, qb + (size_t)tp * D, gb + (size_t)tp * D};
            bstage_load<bf16, D, 4>(st, src, C, tid);
        }
        __syncthreads();  // token tiles visible

        // ---- phase 1 (mode tiles): Z'_in = conj(rho^c) o Z'_out - sum_i conj(rho^i) x_i; publish
        // Z'_k for dq; Gram tiles of key tile w
        rotate_dm<bf16, D, MP, true>(Zk, rc, w, r);
        rotate_dm<bf16, D, MP, true>(Zv, rc, w, r);
#pragma unroll
        for (int kb = 0; kb < KBC; ++kb) {
            F kf[NDT], vf[NDT];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                kf[dt] = neg_frag(ld_frag_tr(Ks, LDQ, 16 * dt, kb, g, r));
                vf[dt] = neg_frag(ld_frag_tr(Vs, LDQ, 16 * dt, kb, g, r));
            }
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt >= NMT) continue;
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    const F ef = ld_frag_tr(sE, LE, p * MP + 16 * mt, kb, g, r);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        Zk[o][p][dt] = mma(kf[dt], ef, Zk[o][p][dt]);
                        Zv[o][p][dt] = mma(vf[dt], ef, Zv[o][p][dt]);
                    }
                }
            }
        }
        if constexpr (!SUM) {
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = w + NW * o;
                if (mt < NMT) {
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                        for (int p = 0; p < 2; ++p)
                            st_lds<bf16x4>(ZkT + (size_t)(p * MP + 16 * mt + r) * P::LDZ + P::tcol(p * MP + 16 * mt + r, 16 * dt + 4 * g),
                                           cvt4(Zk[o][p][dt], bf16()));
                }
            }
        }
        {
            F kf[KBD], vf[KBD];
#pragma unroll
            for (int kb = 0; kb < KBD; ++kb) {
                kf[kb] = ld_frag<bf16>(Ks + (size_t)(16 * w + r) * LDQ, 32 * kb, g);
                vf[kb] = ld_frag<bf16>(Vs + (size_t)(16 * w + r) * LDQ, 32 * kb, g);
            }
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) {
                if (ct < w) continue;
                const int j = 16 * ct + r;
                floatx4 ga = zero4(), gd = zero4();
#pragma unroll
                for (int kb = 0; kb < KBD; ++kb) {
                    ga = mma(kf[kb], ld_frag<bf16>(Qs + (size_t)j * LDQ, 32 * kb, g), ga);
                    gd = mma(vf[kb], ld_frag<bf16>(dOs + (size_t)j * LDQ, 32 * kb, g), gd);
                }
                if (ct == w) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (4 * g + e > r) ga[e] = gd[e] = 0.f;
                }
                st4<bf16>(GT + (size_t)j * LDK + 16 * w + 4 * g, ga);
                st4<bf16>(GdT + (size_t)j * LDK + 16 * w + 4 * g, gd);
            }
        }
        __syncthreads();  // Gram tiles visible

        // ---- phase 2 (mode tiles): U = E o (Q Z'_k^T + G conj(E)), Y = E o (dO Z'_v^T + Gd conj(E))
        {
            F zkf[OWN][2][KBD], zvf[OWN][2][KBD];
#pragma unroll
            for (int o = 0; o < OWN; ++o)
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int kb = 0; kb < KBD; ++kb) {
                        zkf[o][p][kb] = frag_from_acc<bf16>(Zk[o][p][2 * kb], Zk[o][p][2 * kb + 1]);
                        zvf[o][p][kb] = frag_from_acc<bf16>(Zv[o][p][2 * kb], Zv[o][p][2 * kb + 1]);
                    }
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) {
                const int j = 16 * ct + r;
                F qf[KBD], of[KBD];
#pragma unroll
                for (int kb = 0; kb < KBD; ++kb) {
                    qf[kb] = ld_frag<bf16>(Qs + (size_t)j * LDQ, 32 * kb, g);
                    of[kb] = ld_frag<bf16>(dOs + (size_t)j * LDQ, 32 * kb, g);
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
                            const bf16* grow = GT + (size_t)j * LDK;
                            const bf16* drow = GdT + (size_t)j * LDK;
                            const bool full = 2 * kb + 1 <= ct;
                            const F gf = full ? ld_frag<bf16>(grow, 32 * kb, g) : ld_frag_lo<bf16>(grow, 32 * kb, g);
                            const F df = full ? ld_frag<bf16>(drow, 32 * kb, g) : ld_frag_lo<bf16>(drow, 32 * kb, g);
#pragma unroll
                            for (int p = 0; p < 2; ++p) {
                                const F ef = ld_frag_tr(sE, LE, p * MP + 16 * mt, kb, g, r);
                                u[p] = mma(ef, gf, u[p]);
                                y[p] = mma(ef, df, y[p]);
                            }
                        }
                    }
                    // E o X with the stored row [c | -s] of token j
                    const floatx4 cs = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + 16 * mt + 4 * g));
                    const floatx4 ns = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + MP + 16 * mt + 4 * g));
                    st4<bf16>(UT + (size_t)j * LDU + 16 * mt + 4 * g, cs * u[0] + ns * u[1]);
                    st4<bf16>(UT + (size_t)j * LDU + MP + 16 * mt + 4 * g, cs * u[1] - ns * u[0]);
                    st4<bf16>(YT + (size_t)j * LDU + 16 * mt + 4 * g, cs * y[0] + ns * y[1]);
                    st4<bf16>(YT + (size_t)j * LDU + MP + 16 * mt + 4 * g, cs * y[1] - ns * y[0]);
                }
            }
        }
        __syncthreads();  // U and Y visible

        // ---- phase 3 (query tile w): scores, softmax and its gradient, the weights, H tiles, dq
        {
            const int j = 16 * w + r;
            const long long pos = a.t0 + tok0 + j;
            F uf[KBM], yf[KBM];
#pragma unroll
            for (int kb = 0; kb < KBM; ++kb) {
                uf[kb] = ld_frag<bf16>(UT + (size_t)j * LDU, 32 * kb, g);
                yf[kb] = ld_frag<bf16>(YT + (size_t)j * LDU, 32 * kb, g);
            }
            floatx4 sc[NST], dp[NST];
#pragma unroll
            for (int s4 = 0; s4 < NST; ++s4) {
                sc[s4] = dp[s4] = zero4();
#pragma unroll
                for (int kb = 0; kb < KBM; ++kb) {
                    const F af = ld_frag<bf16>(sAB + (size_t)(16 * s4 + r) * LE, 32 * kb, g);
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
                pf[kb] = frag_from_acc<bf16>(sc[2 * kb] * iscale, sc[2 * kb + 1] * iscale);
                zf[kb] = frag_from_acc<bf16>(sc[2 * kb] * (dp[2 * kb] - pd), sc[2 * kb + 1] * (dp[2 * kb + 1] - pd));
            }
            // [Re W'' | -Im W''] with W'' = (P A - i P B) o rho^j (the slot matrix holds scale (A | B):
            // pf carries 1 / scale), and H_v
            {
                floatx4 wa[2 * NMT];
#pragma unroll
                for (int t = 0; t < 2 * NMT; ++t) {
                    wa[t] = zero4();
#pragma unroll
                    for (int kb = 0; kb < KBS; ++kb) wa[t] = mma(ld_frag_tr(sAB, LE, 16 * t, kb, g, r), pf[kb], wa[t]);
                }
#pragma unroll
                for (int mt = 0; mt < NMT; ++mt) {
                    const floatx4 cs = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + 16 * mt + 4 * g));
                    const floatx4 ns = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + MP + 16 * mt + 4 * g));
                    const floatx4 am = wa[mt], bm = wa[NMT + mt];
                    wa[mt] = am * cs - bm * ns;
                    wa[NMT + mt] = am * ns + bm * cs;
                    st_lds<bf16x4>(WvT + (size_t)j * P::LDW + P::tcol(j, 16 * mt + 4 * g), cvt4(wa[mt], bf16()));
                    st_lds<bf16x4>(WvT + (size_t)j * P::LDW + P::tcol(j, MP + 16 * mt + 4 * g), cvt4(wa[NMT + mt], bf16()));
                }
                if constexpr (!SUM) {
                    F wf[KBM];
#pragma unroll
                    for (int kb = 0; kb < KBM; ++kb) wf[kb] = frag_from_acc<bf16>(wa[2 * kb], wa[2 * kb + 1]);
#pragma unroll
                    for (int kt = 0; kt < NT; ++kt) {
                        floatx4 hv = zero4();
                        if (kt <= w) {
#pragma unroll
                            for (int kb = 0; kb < KBM; ++kb)
                                hv = mma(ld_frag<bf16>(sE + (size_t)(16 * kt + r) * LE, 32 * kb, g), wf[kb], hv);
                            if (kt == w) {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (4 * g + e > r) hv[e] = 0.f;
                            }
                        }
                        st_lds<bf16x4>(HvT + (size_t)j * P::LDH + P::tcol(j, 16 * kt + 4 * g), cvt4(hv, bf16()));
                    }
                }
            }
            // [Re Wq'' | -Im Wq''] with Wq'' = scale (dz A - i dz B) o rho^j, H_q and dq
            {
                floatx4 wq[2 * NMT];
#pragma unroll
                for (int t = 0; t < 2 * NMT; ++t) {
                    wq[t] = zero4();
#pragma unroll
                    for (int kb = 0; kb < KBS; ++kb) wq[t] = mma(ld_frag_tr(sAB, LE, 16 * t, kb, g, r), zf[kb], wq[t]);
                }
#pragma unroll
                for (int mt = 0; mt < NMT; ++mt) {
                    const floatx4 cs = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + 16 * mt + 4 * g));
                    const floatx4 ns = to_f4(ld4_lds<bf16>(sE + (size_t)j * LE + MP + 16 * mt + 4 * g));
                    const floatx4 am = wq[mt], bm = wq[NMT + mt];
                    wq[mt] = am * cs - bm * ns;
                    wq[NMT + mt] = am * ns + bm * cs;
                    st_lds<bf16x4>(WqT + (size_t)j * P::LDW + P::tcol(j, 16 * mt + 4 * g), cvt4(wq[mt], bf16()));
                    st_lds<bf16x4>(WqT + (size_t)j * P::LDW + P::tcol(j, MP + 16 * mt + 4 * g), cvt4(wq[NMT + mt], bf16()));
                }
                if constexpr (!SUM) {
                    F qf2[KBM];
#pragma unroll
                    for (int kb = 0; kb < KBM; ++kb) qf2[kb] = frag_from_acc<bf16>(wq[2 * kb], wq[2 * kb + 1]);
                    floatx4 oa[NDT];
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        oa[dt] = zero4();
#pragma unroll
                        for (int kb = 0; kb < KBM; ++kb)
                            oa[dt] = mma(P::ld_t(ZkT, P::LDZ, 16 * dt, kb, g, r), qf2[kb], oa[dt]);
                    }
                    floatx4 hq[NT];
#pragma unroll
                    for (int kt = 0; kt < NT; ++kt) {
                        hq[kt] = zero4();
                        if (kt <= w) {
#pragma unroll
                            for (int kb = 0; kb < KBM; ++kb)
                                hq[kt] = mma(ld_frag<bf16>(sE + (size_t)(16 * kt + r) * LE, 32 * kb, g), qf2[kb], hq[kt]);
                            if (kt == w) {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (4 * g + e > r) hq[kt][e] = 0.f;
                            }
                        }
                        st_lds<bf16x4>(HqT + (size_t)j * P::LDH + P::tcol(j, 16 * kt + 4 * g), cvt4(hq[kt], bf16()));
                    }
#pragma unroll
                    for (int kb = 0; kb < KBC; ++kb) {
                        if (2 * kb <= w) {
                            const F hf = frag_from_acc<bf16>(hq[2 * kb], hq[2 * kb + 1]);
#pragma unroll
                            for (int dt = 0; dt < NDT; ++dt)
                                oa[dt] = mma(ld_frag_tr(Ks, LDQ, 16 * dt, kb, g, r), hf, oa[dt]);
                        }
                    }
                    if (j < c) {
                        bf16* dqb = (bf16*)a.dq + ((size_t)bh * a.L + tok0 + j) * D;
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) st4<bf16>(dqb + 16 * dt + 4 * g, oa[dt]);
                    }
                }
            }
        }
        __syncthreads();  // H tiles and weights visible

        // ---- phase 4 (head-dim tiles): Gam'' = conj(rho^c) o Gam'; dk, dv of the wave's d-tile for
        // every key; Gam' <- Gam'' + [conj(Wq'')^T Q | conj(W'')^T dO]
#pragma unroll
        for (int od = 0; od < ODT; ++od) {
            const int dt = w + NW * od;
            if (dt >= NDT) continue;
#pragma unroll
            for (int mt = 0; mt < NMT; ++mt) {
                const floatx4 cc = ld4f(rc + 16 * mt + 4 * g), ss = ld4f(rc + MP + 16 * mt + 4 * g);
                floatx4 re = Gk[od][0][mt], im = Gk[od][1][mt];
                Gk[od][0][mt] = cc * re + ss * im;
                Gk[od][1][mt] = cc * im - ss * re;
                re = Gv[od][0][mt];
                im = Gv[od][1][mt];
                Gv[od][0][mt] = cc * re + ss * im;
                Gv[od][1][mt] = cc * im - ss * re;
            }
            if constexpr (!SUM) {
                // A operands [Re Gam'' | Im Gam''] (rows d, reduction over the 2MP rows)
                F gkf[KBM], gvf[KBM];
#pragma unroll
                for (int kb = 0; kb < KBM; ++kb) {
                    // the block's two 16-row tiles in the order [Re tiles | Im tiles]
                    const int t0 = 2 * kb, t1 = 2 * kb + 1;
                    gkf[kb] = frag_from_acc<bf16>(Gk[od][t0 / NMT][t0 % NMT], Gk[od][t1 / NMT][t1 % NMT]);
                    gvf[kb] = frag_from_acc<bf16>(Gv[od][t0 / NMT][t0 % NMT], Gv[od][t1 / NMT][t1 % NMT]);
                }
                F qtf[KBC], otf[KBC];
#pragma unroll
                for (int kb = 0; kb < KBC; ++kb) {
                    qtf[kb] = ld_frag_tr(Qs, LDQ, 16 * dt, kb, g, r);
                    otf[kb] = ld_frag_tr(dOs, LDQ, 16 * dt, kb, g, r);
                }
#pragma unroll
                for (int kt = 0; kt < NT; ++kt) {
                    const int j = 16 * kt + r;
                    floatx4 ka = zero4(), va = zero4();
#pragma unroll
                    for (int kb = 0; kb < KBC; ++kb) {
                        ka = mma(qtf[kb], P::ld_t(HqT, P::LDH, 16 * kt, kb, g, r), ka);
                        va = mma(otf[kb], P::ld_t(HvT, P::LDH, 16 * kt, kb, g, r), va);
                    }
#pragma unroll
                    for (int kb = 0; kb < KBM; ++kb) {
                        const F ef = ld_frag<bf16>(sE + (size_t)j * LE, 32 * kb, g);
                        ka = mma(gkf[kb], ef, ka);
                        va = mma(gvf[kb], ef, va);
                    }
                    if (j < c) {
                        bf16* dkb = (bf16*)a.dk + ((size_t)bh * a.L + tok0 + j) * D;
                        bf16* dvb = (bf16*)a.dv + ((size_t)bh * a.L + tok0 + j) * D;
                        st4<bf16>(dkb + 16 * dt + 4 * g, ka);
                        st4<bf16>(dvb + 16 * dt + 4 * g, va);
                    }
                }
            }
#pragma unroll
            for (int kb = 0; kb < KBC; ++kb) {
                const F qtf = ld_frag_tr(Qs, LDQ, 16 * dt, kb, g, r);
                const F otf = ld_frag_tr(dOs, LDQ, 16 * dt, kb, g, r);
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int mt = 0; mt < NMT; ++mt) {
                        Gk[od][p][mt] = mma(P::ld_t(WqT, P::LDW, p * MP + 16 * mt, kb, g, r), qtf, Gk[od][p][mt]);
                        Gv[od][p][mt] = mma(P::ld_t(WvT, P::LDW, p * MP + 16 * mt, kb, g, r), otf, Gv[od][p][mt]);
                    }
            }
        }
    }

    // ---- the adjoint at the segment's start
#pragma unroll
    for (int od = 0; od < ODT; ++od) {
        const int dt = w + NW * od;
        if (dt >= NDT) continue;
        if constexpr (SUM) {
            float* S = a.asum + ((size_t)bh * a.nbk + seg) * 4 * MP * D;
#pragma unroll
            for (int p2 = 0; p2 < 2; ++p2)
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int mt = 0; mt < NMT; ++mt) {
                        const floatx4 x = p2 ? Gv[od][p][mt] : Gk[od][p][mt];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            S[((size_t)(2 * p2 + p) * MP + 16 * mt + 4 * g + e) * D + 16 * dt + r] = x[e];
                    }
        } else {
            if (seg != 0) continue;
#pragma unroll
            for (int mt = 0; mt < NMT; ++mt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = 16 * mt + 4 * g + e;
                    if (m >= a.M) continue;
                    const float c1 = rho1[m], s1 = rho1[MP + m];
                    const size_t o0 = (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + r;
                    const size_t o1 = (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + r;
                    if (a.gk_in) {
                        const float re = Gk[od][0][mt][e], im = Gk[od][1][mt][e];
                        a.gk_in[o0] = c1 * re + s1 * im;
                        a.gk_in[o1] = c1 * im - s1 * re;
                    }
                    if (a.gv_in) {
                        const float re = Gv[od][0][mt][e], im = Gv[od][1][mt][e];
                        a.gv_in[o0] = c1 * re + s1 * im;
                        a.gv_in[o1] = c1 * im - s1 * re;
                    }
                }
        }
    }
}

template <int D, int MP, int SP>
hipError_t launch_backward16_shape(const BwdArgs& a, hipStream_t s, void* const* ev)
{
    auto mark = [&](int i) -> hipError_t {
        return (ev && ev[i]) ? hipEventRecord((hipEvent_t)ev[i], s) : hipSuccess;
    };
    const unsigned units = (unsigned)(a.B * a.H);
    hipLaunchKernelGGL((bwd16_fsum_kernel<D, MP>), dim3(units * a.nbk), dim3(kThreads), 0, s, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || (e = mark(0)) != hipSuccess) return e;
    if (a.nseg > 1) {
        const unsigned sum_blocks = (unsigned)(a.nbk - a.nbk / a.nseg);  // blocks of segments 1..nseg-1
        hipLaunchKernelGGL((bwd16_kernel<D, MP, SP, true>), dim3(units * sum_blocks), dim3(kThreads), 0, s, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if ((e = mark(1)) != hipSuccess) return e;
    hipLaunchKernelGGL((bwd16_kernel<D, MP, SP, false>), dim3(units * a.nseg), dim3(kThreads), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return mark(2);
}

}  // namespace bla
