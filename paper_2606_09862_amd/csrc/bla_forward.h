// Chunked-parallel BLA forward kernels for gfx950 (templated; instantiated in
// bla_forward_bf16.hip and bla_forward_f32.hip).
//
// The operator is the mode-state recurrence (Sec. 3.1 Eq. recurrence) read out
// through blurry slots (Eq. compressed) with a masked slot softmax (Eq. output),
// i.e. Alg. 2.  The kernels compute it in chunks of C = 64 tokens with the state
// carried in registers.  Per chunk (local token j, key i, mode m), with
// rho_m = exp(i m w), E[j,m] = rho_m^j, G = tril(Q K^T) and the pre-rotated state
// Z' = rho Z (so every phase is a local power rho^j, j <= C):
//
//   (1+3)  U   = E o (Q Z'_k^T + G conj(E))            query-mode projection
//   (4)    z   = scale (Re U A^T + Im U B^T)            slot scores
//   (5)    P   = softmax(z masked where pos < theta)    start mask (Alg. 2)
//   (6)    W'' = (P A - i P B) o E                      readout weights per mode
//   (7-9)  O   = Re(W'' Z'_v) + tril(Re(W'' conj(E)^T)) V
//   (10)   Z' <- rho^c o Z' + sum_i rho^{c-i} [k_i | v_i]
//
// Work split inside a 256-thread workgroup (4 waves; 8 for d = M = 128, see Geo): contractions that produce
// per-mode rows (1+3, 10) are split by mode tiles, the Gram tile (2) by key
// tiles, and the per-token chain (4-9) by token tiles, so that the chain passes
// its intermediates in registers (see bla_device.h).  The fp32 state of the
// wave's own mode tiles lives in registers for the whole segment; its bf16 copy
// of Z'_v goes through LDS for (7).  The bf16 d = M = 128 shape with 64 or 128 slots
// splits (4)-(9) by output columns instead (Fwd::SPLIT: slot, mode and head-dim tiles
// per wave, the intermediates through LDS) and reads its tables as fragment-ordered
// copies in global memory (FragTabArgs).
//
// Data movement: the next chunk's Q, K, V are loaded into registers while the
// current chunk computes, and written to LDS (Q row-major, K and V transposed)
// at the top of the next iteration.  The head's tables (slot matrices, phase
// tables) are copied into LDS once per workgroup when they fit next to the
// per-chunk tiles; the wave's own rows of conj(E) and rho^{C-i} stay in
// registers for the whole segment.
//
// Anchored slots (Sec. 3.3, Alg. 1/3) share the mode state and steps (1), (2), (8)-(10);
// with P the chunk's absolute start and X = Q Z'_k^T + G conj(E), they read out
// U = rho^P o conj(X) and W'' = (P A + i P B) o conj(rho^P).  With -B in both slot
// matrices these are the twiddles of (3) and (6) applied with the single row
// conj(rho^P) = [cos | -sin](m w P) for every token of the chunk.
//
// A sequence is split into nseg segments processed by separate workgroups.  The
// state entering segment g >= 1 comes from a scan over per-block summaries
// (summary_kernel: step 10 alone, from a zero state) -- the recurrence is
// linear, so carry_g = sum of block summaries rotated to the segment start.
#pragma once

#include <math.h>

#include "bla_device.h"
#include "bla_plan.h"

namespace bla {

constexpr size_t kMaxLds = 160 * 1024;

// CC: tokens per chunk (16, 32, 64 or 128; Alg. 3 takes the chunk length as an input).
template <typename T, int D, int MP, int CC = kChunk> struct Geo {
    static constexpr int C = CC;
    static constexpr int NT = C / 16;           // token tiles per chunk
    // Threads per workgroup: 4 waves, or 8 for d = M = 128, where four waves would each hold
    // two mode tiles of both states (256 registers) and spill, and for 128-token chunks (one
    // token tile per wave); the token chain runs on waves 0..NT-1 and the other waves take
    // part in the mode-tile phases only, except in the split chain (Fwd::SPLIT), where every
    // wave takes a share of steps (4)-(9).
    static constexpr int NTHR = ((D == 128 && MP == 128) || NT > 4) ? 2 * kThreads : kThreads;
    static constexpr int NW = NTHR / 64;        // waves
    static constexpr int NMT = MP / 16;         // mode tiles
    static constexpr int NDT = D / 16;          // head-dim tiles
    static constexpr int KBD = D / 32;          // reduction blocks over d
    static constexpr int KBM = 2 * MP / 32;     // reduction blocks over [Re | Im] modes
    static constexpr int KBC = (C + 31) / 32;   // reduction blocks over chunk tokens
    // A 16-token chunk fills only the lower half of its one token-reduction block: every
    // fragment over chunk tokens then carries zeros in reduction indices 16..31.
    static constexpr bool HALF = C % 32 != 0;
    static constexpr int OWN = (NMT + NW - 1) / NW;  // mode tiles owned per wave
    // Row padding in LDS: rows of a fragment read (16 lanes, one row each, 8 bytes per
    // lane for bf16) land on distinct banks when the row stride is 8 bytes past a
    // multiple of 128 (4 elements); for float32 rows the same 4 elements keep the
    // 16-byte alignment of their 16-byte reads.
    static constexpr int PAD = 4;
    static constexpr int LDK = C + PAD;         // Kt, Vt: [D][LDK]
    static constexpr int LDQ = D + PAD;         // Qs: [C][LDQ]
    static constexpr int LDZ = 2 * MP + PAD;    // ZvT: [D][LDZ]
    static constexpr size_t KT_ELEMS = (size_t)D * LDK;
    static constexpr size_t Q_ELEMS = (size_t)C * LDQ;
    // staging units: Q rows in pieces of 8 elements, K/V in 4-token x 8-element blocks (consecutive
    // threads take consecutive 8-element pieces of the same four rows: coalesced global reads)
    static constexpr int QU = C * D / 8;
    static constexpr int KVU = 2 * (C / 4) * (D / 8);
    static constexpr int QPT = (QU + NTHR - 1) / NTHR;
    static constexpr int KVPT = (KVU + NTHR - 1) / NTHR;
    static_assert(NT <= NW, "one token tile per wave, for the first NT waves");
    static_assert(D % 32 == 0 && MP % 16 == 0, "tile shapes");
    static_assert(C == 16 || C == 32 || C == 64 || C == 128, "chunk length");
};

// Fragment over chunk tokens (reduction block kb) of a row-major tile whose rows hold the
// chunk's C tokens: for a 16-token chunk only the lower half exists.
template <typename T, int CC>
__device__ __forceinline__ typename Frag<T>::type ld_frag_c(const T* row, int kb, int g)
{
    if constexpr (CC % 32 != 0)
        return ld_frag_lo<T>(row, 32 * kb, g);
    else
        return ld_frag<T>(row, 32 * kb, g);
}

template <typename T, int D, int MP, int SP, int CC = kChunk> struct Fwd : Geo<T, D, MP, CC> {
    using G = Geo<T, D, MP, CC>;
    static constexpr int NST = SP / 16;
    static constexpr int KBS = SP / 32;
    static constexpr int LDG = G::C + G::PAD;    // GT:   [C tokens][LDG]
    static constexpr int LDU = 2 * MP + G::PAD;  // UT:   [C tokens][LDU]
    static constexpr int LDAS = 2 * MP + G::PAD; // ABs:  [SP][LDAS]
    static constexpr int LDAM = SP + G::PAD;     // ABm:  [2MP][LDAM]
    static constexpr int LDE = 2 * MP + G::PAD;  // Etab: [C][LDE]  (also the phase twiddles)
    static constexpr int LDR = G::C + G::PAD;    // EbarT, ErevT: [2MP][LDR]
    // Qs (read in phase A) and UT (written after the next barrier) share one buffer.
    static constexpr int LDQU = LDU > G::LDQ ? LDU : G::LDQ;
    // ... + the anchored twiddle row [2MP] of the chunk
    static constexpr size_t BASE_ELEMS = 2 * G::KT_ELEMS + (size_t)G::C * LDQU + (size_t)G::C * LDG +
                                         (size_t)D * G::LDZ + (size_t)2 * MP;
    static constexpr size_t TAB_ELEMS = (size_t)SP * LDAS + (size_t)2 * MP * LDAM + (size_t)G::C * LDE +
                                        (size_t)2 * 2 * MP * LDR;
    // float32 rows rho and rho^C, then the int32 mask thresholds
    static constexpr size_t SMALL_BYTES = (size_t)3 * 2 * MP * 4 + (size_t)SP * 4;
    static constexpr size_t BASE_BYTES = BASE_ELEMS * sizeof(T);
    static constexpr size_t FULL_BYTES = BASE_BYTES + TAB_ELEMS * sizeof(T) + SMALL_BYTES;
    static constexpr bool TL = FULL_BYTES <= kMaxLds;  // tables live in LDS
    // Split chain (bf16, eight waves, four token tiles, tables outside LDS): steps (4)-(9) are
    // split by output columns -- each wave forms one slot tile of the scores, one mode tile of
    // the readout weights and one head-dim tile of the output, for every token of the chunk,
    // so that each table fragment it loads serves all four token tiles.  The unnormalised slot
    // weights P~ ([C][LDP]) pass through LDS after the per-chunk buffers (later the H tiles);
    // the per-token (max, sum) of each slot tile use the Gram buffer, free by then.
    static constexpr int LDP = SP + G::PAD;
    static constexpr size_t SPLIT_BYTES = (size_t)G::C * LDP * sizeof(T);
    static constexpr bool SPLIT = sizeof(T) == 2 && G::NW == 2 * G::NT && SP % 64 == 0 && !TL &&
                                  BASE_BYTES + SPLIT_BYTES <= kMaxLds;
    static constexpr size_t LDS_BYTES = TL ? FULL_BYTES : BASE_BYTES + (SPLIT ? SPLIT_BYTES : 0);
    static_assert(SP % 32 == 0, "slot padding");
};

// The wave's fp32 state tiles: [owned mode tile][Re, Im][head-dim tile].
template <typename T, int D, int MP, int CC = kChunk> using StateTiles = floatx4[Geo<T, D, MP, CC>::OWN][2][D / 16];
// ---------------------------------------------------------------------------------
// Chunk staging: global -> registers (issued a chunk ahead) -> LDS.
template <typename T, int D, int MP, int CC = kChunk> struct Stage {
    using GG = Geo<T, D, MP, CC>;
    using H = typename Frag<T>::half;
    H q[GG::QPT][2];
    H kv[GG::KVPT][4][2];
};

// WQ: also stage the query rows.  c: valid tokens of the chunk.  The loads never
// depend on c (rows past c re-read row c-1, which exists); the zero fill past c is
// applied when the registers are written to LDS, so no wait on the loads is forced
// while they are in flight.
template <typename T, int D, int MP, bool WQ, int CC = kChunk>
__device__ __forceinline__ void stage_load(Stage<T, D, MP, CC>& st, const T* qc, const T* kc, const T* vc,
                                           int ts, int c, int tid)
{
    using GG = Geo<T, D, MP, CC>;
    constexpr int DO = D / 8;
#pragma unroll
    for (int i = 0; i < (WQ ? GG::QPT : 0); ++i) {
        const int u = tid + i * GG::NTHR;
        const int t = min(u / DO, c - 1), dq = u % DO;
        if (GG::QU % GG::NTHR == 0 || u < GG::QU) {
            st.q[i][0] = ld4<T>(qc + (size_t)t * ts + 8 * dq);
            st.q[i][1] = ld4<T>(qc + (size_t)t * ts + 8 * dq + 4);
        }
    }
    constexpr int UNITS = GG::KVU / 2;
#pragma unroll
    for (int i = 0; i < GG::KVPT; ++i) {
        const int u = tid + i * GG::NTHR;
        const int which = u / UNITS, uu = u % UNITS, dq = uu % (D / 8), tq = uu / (D / 8);
        const T* src = (which ? vc : kc) + 8 * dq;
        if (GG::KVU % GG::NTHR == 0 || u < GG::KVU) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int row = min(4 * tq + t, c - 1);
                st.kv[i][t][0] = ld4<T>(src + (size_t)row * ts);
                st.kv[i][t][1] = ld4<T>(src + (size_t)row * ts + 4);
            }
        }
    }
}

template <typename T, int D, int MP, bool WQ, int CC = kChunk>
__device__ __forceinline__ void stage_store(const Stage<T, D, MP, CC>& st, T* Qs, T* Kt, T* Vt, int c, int tid)
{
    using GG = Geo<T, D, MP, CC>;
    using H = typename Frag<T>::half;
    constexpr int DO = D / 8;
    const H z = zero_half<T>();
#pragma unroll
    for (int i = 0; i < (WQ ? GG::QPT : 0); ++i) {
        const int u = tid + i * GG::NTHR;
        if (GG::QU % GG::NTHR == 0 || u < GG::QU) {
            const int t = u / DO, dq = u % DO;
            const bool ok = t < c;
            *reinterpret_cast<H*>(Qs + (size_t)t * GG::LDQ + 8 * dq) = ok ? st.q[i][0] : z;
            *reinterpret_cast<H*>(Qs + (size_t)t * GG::LDQ + 8 * dq + 4) = ok ? st.q[i][1] : z;
        }
    }
    constexpr int UNITS = GG::KVU / 2;
#pragma unroll
    for (int i = 0; i < GG::KVPT; ++i) {
        const int u = tid + i * GG::NTHR;
        if (GG::KVU % GG::NTHR == 0 || u < GG::KVU) {
            const int which = u / UNITS, uu = u % UNITS, dq = uu % (D / 8), tq = uu / (D / 8);
            T* dst = (which ? Vt : Kt) + (8 * dq) * GG::LDK + 4 * tq;
            H x[4][2];
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const bool ok = 4 * tq + t < c;
                x[t][0] = ok ? st.kv[i][t][0] : z;
                x[t][1] = ok ? st.kv[i][t][1] : z;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                H lo{x[0][0][e], x[1][0][e], x[2][0][e], x[3][0][e]};
                H hi{x[0][1][e], x[1][1][e], x[2][1][e], x[3][1][e]};
                *reinterpret_cast<H*>(dst + e * GG::LDK) = lo;
                *reinterpret_cast<H*>(dst + (e + 4) * GG::LDK) = hi;
            }
        }
    }
}

// A table copied from the workspace into LDS: ROWS x COLS elements of E, source
// rows contiguous, destination row stride DSTRIDE (COLS * sizeof(E) a multiple of 8).
template <typename E, int ROWS, int COLS, int DSTRIDE, int NTHR = kThreads> struct TabCopy {
    static constexpr int PER = 8 / (int)sizeof(E);        // elements per 8-byte piece
    static constexpr int PIECES = ROWS * COLS / PER;
    static constexpr int ITER = (PIECES + NTHR - 1) / NTHR;
};

// Copy up to two tables with every load of the thread in flight before the first
// store (the copies run once per workgroup, so their latency is paid only once).
template <typename E, int ROWS, int COLS, int DSTRIDE, int NTHR = kThreads>
__device__ __forceinline__ void copy_table(E* dst, const E* src, int tid)
{
    typedef int intx2 __attribute__((ext_vector_type(2)));
    using TC = TabCopy<E, ROWS, COLS, DSTRIDE, NTHR>;
    intx2 buf[TC::ITER];
#pragma unroll
    for (int i = 0; i < TC::ITER; ++i) {
        const int u = tid + i * NTHR;
        if (TC::PIECES % NTHR == 0 || u < TC::PIECES)
            buf[i] = reinterpret_cast<const intx2*>(src)[u];
    }
#pragma unroll
    for (int i = 0; i < TC::ITER; ++i) {
        const int u = tid + i * NTHR;
        if (TC::PIECES % NTHR == 0 || u < TC::PIECES) {
            const int rr = u / (COLS / TC::PER), cc = (u % (COLS / TC::PER)) * TC::PER;
            *reinterpret_cast<intx2*>(dst + (size_t)rr * DSTRIDE + cc) = buf[i];
        }
    }
}

// Fragment of rho^{c-i} (i < c, zero past c) for a ragged last chunk, built from E32.
template <typename T, int MP>
__device__ __forceinline__ typename Frag<T>::type erev_frag(const float* E32, int ldE, int c, int p,
                                                            int mt, int kb, int g, int r)
{
    typename Frag<T>::type f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int i = 32 * kb + 16 * (e / 4) + 4 * g + (e % 4);
        float val = 0.f;
        if (i < c) val = E32[(size_t)(c - i) * ldE + p * MP + 16 * mt + r];
        f[e] = (T)val;
    }
    return f;
}

// Write the bf16/fp32 copy of Z'_v as ZvT[d][Re m | Im m] with the Im part negated
// (the A operand of O += Re(W'' Z'_v)).
template <typename T, int D, int MP, int CC = kChunk>
__device__ __forceinline__ void write_zvt(T* ZvT, const StateTiles<T, D, MP, CC>& Zv, int w, int g, int r)
{
    using GG = Geo<T, D, MP, CC>;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o) {
        const int mt = w + GG::NW * o;
        if (mt < GG::NMT) {
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) {
                st4<T>(ZvT + (size_t)(16 * dt + r) * GG::LDZ + 16 * mt + 4 * g, Zv[o][0][dt]);
                st4<T>(ZvT + (size_t)(16 * dt + r) * GG::LDZ + MP + 16 * mt + 4 * g, -Zv[o][1][dt]);
            }
        }
    }
}

// erev_frag in the reduction order 32kb + 8g + e (bf16).
template <int MP>
__device__ __forceinline__ bf16x8 erev_frag_nat(const float* E32, int ldE, int c, int p, int mt, int kb, int g, int r)
{
    bf16x8 f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int i = 32 * kb + 8 * g + e;
        float val = 0.f;
        if (i < c) val = E32[(size_t)(c - i) * ldE + p * MP + 16 * mt + r];
        f[e] = (bf16)val;
    }
    return f;
}

// Step 10 for a wave that owns one mode tile, with the rho^{c-i} fragments ef[kb][Re, Im]
// given in the reduction order 32kb + 8g + e (bf16), the rotation (cc, ss) of the lane's mode
// row (Z'_k) and (cv, sv) of its four mode columns (Z'_v).
template <typename T, int D, int MP, int CC = kChunk>
__device__ __forceinline__ void advance_owned(StateTiles<T, D, MP, CC>& Zk, StateTiles<T, D, MP, CC>& Zv,
                                              const T* Kt, const T* Vt, const bf16x8 (&ef)[Geo<T, D, MP, CC>::KBC][2],
                                              float cc, float ss, floatx4 cv, floatx4 sv, int g, int r)
{
    using GG = Geo<T, D, MP, CC>;
    static_assert(GG::OWN == 1 && sizeof(T) == 2 && !GG::HALF, "one owned mode tile, bf16, 32-token blocks");
#pragma unroll
    for (int dt = 0; dt < GG::NDT; ++dt) {
        const floatx4 kr = Zk[0][0][dt], ki = Zk[0][1][dt];
        Zk[0][0][dt] = cc * kr - ss * ki;
        Zk[0][1][dt] = ss * kr + cc * ki;
        const floatx4 vr = Zv[0][0][dt], vi = Zv[0][1][dt];
        Zv[0][0][dt] = cv * vr - sv * vi;
        Zv[0][1][dt] = sv * vr + cv * vi;
    }
#pragma unroll
    for (int kb = 0; kb < GG::KBC; ++kb)
#pragma unroll
        for (int dt = 0; dt < GG::NDT; ++dt) {
            const bf16x8 kf = ld_frag16_2x8((const bf16*)Kt + (size_t)(16 * dt + r) * GG::LDK, kb, g);
            const bf16x8 vf = ld_frag16_2x8((const bf16*)Vt + (size_t)(16 * dt + r) * GG::LDK, kb, g);
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                Zk[0][p][dt] = mma(kf, ef[kb][p], Zk[0][p][dt]);
                Zv[0][p][dt] = mma(ef[kb][p], vf, Zv[0][p][dt]);
            }
        }
}

// Step 10: Z' <- rho^c o Z' + sum_i rho^{c-i} [k_i | v_i] on the wave's own mode tiles.
// rhoC: the row rho^C (full chunks); rhoL: the row rho^c of the sequence's last chunk;
// E32 (row stride 2MP): phase table for the ragged chunk's rho^{c-i} fragments;
// Erev / ldR: the [2MP][C] table of rho^{C-i} (full chunks).
template <typename T, int D, int MP, int CC = kChunk>
__device__ __forceinline__ void advance_state(StateTiles<T, D, MP, CC>& Zk, StateTiles<T, D, MP, CC>& Zv,
                                              const T* Kt, const T* Vt, const float* rhoC,
                                              const float* rhoL, const float* E32, const T* Erev, int ldR,
                                              int c, int w, int g, int r)
{
    using GG = Geo<T, D, MP, CC>;
    using F = typename Frag<T>::type;
    // rho^c: a chunk shorter than C is the sequence's last one, whose row is rhoL (held where
    // rhoC is, so that the selected row is read with loads of one address space)
    const float* Ec = (c == GG::C) ? rhoC : rhoL;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o) {
        const int mt = w + GG::NW * o;
        if (mt < GG::NMT) {
            const float cc = Ec[16 * mt + r], ss = Ec[MP + 16 * mt + r];
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) {
                const floatx4 re = Zk[o][0][dt], im = Zk[o][1][dt];
                Zk[o][0][dt] = cc * re - ss * im;
                Zk[o][1][dt] = ss * re + cc * im;
            }
            const floatx4 cv = ld4f(Ec + 16 * mt + 4 * g), sv = ld4f(Ec + MP + 16 * mt + 4 * g);
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) {
                const floatx4 re = Zv[o][0][dt], im = Zv[o][1][dt];
                Zv[o][0][dt] = cv * re - sv * im;
                Zv[o][1][dt] = sv * re + cv * im;
            }
        }
    }
    // per reduction block: the phase fragments of the owned mode tiles first, then one
    // head-dim tile of K and V at a time (few fragments live next to the state)
#pragma unroll
    for (int kb = 0; kb < GG::KBC; ++kb) {
        F ef[GG::OWN][2];
#pragma unroll
        for (int o = 0; o < GG::OWN; ++o) {
            const int mt = min(w + GG::NW * o, GG::NMT - 1);
#pragma unroll
            for (int p = 0; p < 2; ++p)
                ef[o][p] = (c == GG::C) ? ld_frag_c<T, CC>(Erev + (size_t)(16 * (p * GG::NMT + mt) + r) * ldR, kb, g)
                                        : erev_frag<T, MP>(E32, 2 * MP, c, p, mt, kb, g, r);
        }
#pragma unroll
        for (int dt = 0; dt < GG::NDT; ++dt) {
            const F kf = ld_frag_c<T, CC>(Kt + (size_t)(16 * dt + r) * GG::LDK, kb, g);
            const F vf = ld_frag_c<T, CC>(Vt + (size_t)(16 * dt + r) * GG::LDK, kb, g);
#pragma unroll
            for (int o = 0; o < GG::OWN; ++o) {
                if (w + GG::NW * o < GG::NMT) {
#pragma unroll
                    for (int p = 0; p < 2; ++p) {
                        Zk[o][p][dt] = mma(kf, ef[o][p], Zk[o][p][dt]);
                        Zv[o][p][dt] = mma(ef[o][p], vf, Zv[o][p][dt]);
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------------
// Block summaries: the pre-rotated state after cpb full chunks, from zero.
template <typename T, int D, int MP, int CC = kChunk>
__global__ __launch_bounds__((Geo<T, D, MP, CC>::NTHR)) void summary_kernel(FwdArgs a)
{
    using GG = Geo<T, D, MP, CC>;
    __shared__ __attribute__((aligned(16))) T lds[2 * GG::KT_ELEMS];
    T* Kt = lds;
    T* Vt = lds + GG::KT_ELEMS;
    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, held in a scalar register
    const int blk = blockIdx.x % a.nbs, bh = blockIdx.x / a.nbs, h = bh % a.H;
    const T* kbase = (const T*)a.k + fwd_in_base(a, bh);
    const T* vbase = (const T*)a.v + fwd_in_base(a, bh);
    const int ts = a.in_t;
    const float* E32h = a.E32 + (size_t)h * (GG::C + 1) * 2 * MP;

    const T* ErevTh = (const T*)a.ErevT + (size_t)h * 2 * MP * GG::C;
    const float* rhoC = E32h + (size_t)GG::C * 2 * MP;
    StateTiles<T, D, MP, CC> Zk, Zv;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int dt = 0; dt < GG::NDT; ++dt) Zk[o][p][dt] = Zv[o][p][dt] = zero4();

    // Two chunks of K/V in flight ahead of the one being reduced: this kernel does
    // little arithmetic per byte, so it is bound by how much load latency it hides.
    Stage<T, D, MP, CC> st0, st1;
    const size_t first = (size_t)blk * a.cpb * GG::C;
    stage_load<T, D, MP, false, CC>(st0, nullptr, kbase + first * ts, vbase + first * ts, ts, GG::C, tid);
    if (a.cpb > 1)
        stage_load<T, D, MP, false, CC>(st1, nullptr, kbase + (first + GG::C) * ts, vbase + (first + GG::C) * ts, ts,
                                        GG::C, tid);
    const int tid_ = tid, g_ = g, r_ = r;
    for (int n = 0; n < a.cpb; ++n) {
        // lane indices re-derived per chunk (opaque_lane): addresses stay inside the loop
        const int r = opaque_lane(r_), g = opaque_lane(g_), tid = opaque_lane(tid_);
        __syncthreads();
        stage_store<T, D, MP, false, CC>(st0, nullptr, Kt, Vt, GG::C, tid);
        st0 = st1;
        if (n + 2 < a.cpb) {
            const size_t tok = first + (size_t)(n + 2) * GG::C;
            stage_load<T, D, MP, false, CC>(st1, nullptr, kbase + tok * ts, vbase + tok * ts, ts, GG::C, tid);
        }
        __syncthreads();
        advance_state<T, D, MP, CC>(Zk, Zv, Kt, Vt, rhoC, rhoC, E32h, ErevTh, GG::C, GG::C, w, g, r);
    }
    float* S = a.summ + ((size_t)bh * a.nbs + blk) * 4 * MP * D;
#pragma unroll
    for (int o = 0; o < GG::OWN; ++o) {
        const int mt = w + GG::NW * o;
        if (mt < GG::NMT) {
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < GG::NDT; ++dt) {
                    st4f(S + ((size_t)p * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zk[o][p][dt]);
                    st4f(S + (size_t)2 * MP * D + ((size_t)p * D + 16 * dt + r) * MP + 16 * mt + 4 * g,
                         Zv[o][p][dt]);
                }
        }
    }
}

// ---------------------------------------------------------------------------------
// One workgroup per (b, h, segment): the chunk loop over the segment.  AN: anchored slots
// (a separate instantiation, so that the rotating form keeps its own register allocation).
template <typename T, int D, int MP, int SP, bool AN, int CC = kChunk>
__global__ __launch_bounds__((Geo<T, D, MP, CC>::NTHR)) void forward_kernel(FwdArgs a)
{
    using P = Fwd<T, D, MP, SP, CC>;
    using GG = Geo<T, D, MP, CC>;
    using F = typename Frag<T>::type;
    constexpr int C = GG::C, NT = GG::NT, NW = GG::NW, NMT = GG::NMT, NDT = GG::NDT, OWN = GG::OWN;
    __shared__ __attribute__((aligned(16))) char lds_raw[P::LDS_BYTES];
    T* Kt = reinterpret_cast<T*>(lds_raw);
    T* Vt = Kt + GG::KT_ELEMS;
    T* Qs = Vt + GG::KT_ELEMS;  // query rows of the chunk (phase A) ...
    T* UT = Qs;                 // ... then U (phase B onwards)
    T* GT = Qs + (size_t)C * P::LDQU;
    T* ZvT = GT + (size_t)C * P::LDG;
    T* lPh = ZvT + (size_t)D * GG::LDZ;  // anchored twiddle row conj(rho^P) of the chunk
    // split chain: P~ rows (then the H tiles) and the per-token (max, sum) of every slot tile
    T* Pw = reinterpret_cast<T*>(lds_raw + P::BASE_BYTES);
    float* sStat = reinterpret_cast<float*>(GT);
    static_assert(!P::SPLIT || (size_t)C * P::NST * 2 * 4 <= (size_t)C * P::LDG * sizeof(T), "statistics fit");

    const int tid = threadIdx.x, g = (tid & 63) >> 4, r = tid & 15;
    const int tid_ = tid, g_ = g, r_ = r;  // the chunk loop re-derives its own copies
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, held in a scalar register
    const int seg = blockIdx.x % a.nseg, bh = blockIdx.x / a.nseg, h = bh % a.H;
    const int ch0 = seg * a.cps;
    const int nch = min(a.cps, a.nch - ch0);
    const T* qb = (const T*)a.q + fwd_in_base(a, bh);
    const T* kb_ = (const T*)a.k + fwd_in_base(a, bh);
    const T* vb = (const T*)a.v + fwd_in_base(a, bh);
    T* ob = (T*)a.o + fwd_out_base(a, bh);
    const int ts = a.in_t, tso = a.out_t;
    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    const int* thh = a.theta + (size_t)h * SP;

    // ---- tables: LDS copies when they fit, else straight from the workspace
    const T* tABs;
    const T* tABm;
    const T* tEtab;      // cos | sin of m w j, j < C: step 8 operand and the phase twiddles
    const T* tEbar;      // [2MP][C] conj(rho^i) rows
    const T* tErev;      // [2MP][C] rho^{C-i} rows
    const float* rho1;   // rho   (float32, 2MP)
    const float* rhoC;   // rho^C (float32, 2MP)
    const float* rhoL;   // rho^c of the sequence's last chunk (float32, 2MP)
    const int c_last = a.L - (a.nch - 1) * C;  // length of the last chunk (the only short one)
    const int* tTheta;   // start-mask thresholds [SP]
    constexpr int sABs = P::TL ? P::LDAS : 2 * MP;
    constexpr int sABm = P::TL ? P::LDAM : SP;
    constexpr int sEtab = P::TL ? P::LDE : 2 * MP;
    constexpr int sR = P::TL ? P::LDR : C;
    const T* gEbar = (const T*)a.EbarT + (size_t)h * 2 * MP * C;
    const T* gErev = (const T*)a.ErevT + (size_t)h * 2 * MP * C;
    const T* gEtab = (const T*)a.Etab + (size_t)h * C * 2 * MP;
    // fragment-ordered tables of the split chain (one contiguous 1 KB block per fragment)
    const T* fABs = (const T*)a.fABs;
    const T* fABm = (const T*)a.fABm;
    const T* fEtab = (const T*)a.fEtab + (size_t)h * C * 2 * MP;
    const T* fEbar = (const T*)a.fEbar + (size_t)h * C * 2 * MP;
    const T* fErev = (const T*)a.fErev + (size_t)h * C * 2 * MP;
    const T* fTw = (const T*)a.fTw + (size_t)h * C * 2 * MP;
    if constexpr (P::TL) {
        T* lABs = lPh + (size_t)2 * MP;
        T* lABm = lABs + (size_t)SP * P::LDAS;
        T* lEtab = lABm + (size_t)2 * MP * P::LDAM;
        T* lEbar = lEtab + (size_t)C * P::LDE;
        T* lErev = lEbar + (size_t)2 * MP * P::LDR;
        float* lRho = reinterpret_cast<float*>(lErev + (size_t)2 * MP * P::LDR);
        int* lTheta = reinterpret_cast<int*>(lRho + 6 * MP);
        copy_table<T, SP, 2 * MP, P::LDAS, GG::NTHR>(lABs, (const T*)a.ABs, tid);
        copy_table<T, 2 * MP, SP, P::LDAM, GG::NTHR>(lABm, (const T*)a.ABm, tid);
        copy_table<T, C, 2 * MP, P::LDE, GG::NTHR>(lEtab, gEtab, tid);
        copy_table<T, 2 * MP, C, P::LDR, GG::NTHR>(lEbar, gEbar, tid);
        copy_table<T, 2 * MP, C, P::LDR, GG::NTHR>(lErev, gErev, tid);
        copy_table<float, 1, 2 * MP, 2 * MP, GG::NTHR>(lRho, E32h + 2 * MP, tid);                    // rho
        copy_table<float, 1, 2 * MP, 2 * MP, GG::NTHR>(lRho + 2 * MP, E32h + (size_t)C * 2 * MP, tid);  // rho^C
        copy_table<float, 1, 2 * MP, 2 * MP, GG::NTHR>(lRho + 4 * MP, E32h + (size_t)c_last * 2 * MP, tid);  // rho^c_last
        copy_table<int, 1, SP, SP, GG::NTHR>(lTheta, thh, tid);
        tABs = lABs;
        tABm = lABm;
        tEtab = lEtab;
        tEbar = lEbar;
        tErev = lErev;
        rho1 = lRho;
        rhoC = lRho + 2 * MP;
        rhoL = lRho + 4 * MP;
        tTheta = lTheta;
    } else {
        tABs = (const T*)a.ABs;
        tABm = (const T*)a.ABm;
        tEtab = gEtab;
        tEbar = gEbar;
        tErev = gErev;
        rho1 = E32h + 2 * MP;
        rhoC = E32h + (size_t)C * 2 * MP;
        rhoL = E32h + (size_t)c_last * 2 * MP;
        tTheta = thh;
    }

    // Eight-wave geometry (bf16): the Gram tile's key rows are read transposed from the staged
    // K^T tile instead of being held in registers a chunk ahead.
    constexpr bool KROWS = GG::NTHR > kThreads && sizeof(T) == 2;
    // first chunk's staging loads go out before the state set-up
    Stage<T, D, MP, CC> st;
    F kpf[KROWS ? 1 : GG::KBD];  // key rows 16w..16w+15 of the next chunk (Gram tile A operand), unmasked
    {
        const int tok0 = ch0 * C, c0 = min(C, a.L - tok0), i = min(16 * w + r, c0 - 1);
        stage_load<T, D, MP, true, CC>(st, qb + (size_t)tok0 * ts, kb_ + (size_t)tok0 * ts, vb + (size_t)tok0 * ts,
                                       ts, c0, tid);
        if constexpr (!KROWS) {
#pragma unroll
            for (int kb = 0; kb < GG::KBD; ++kb) kpf[kb] = ld_frag<T>(kb_ + (size_t)(tok0 + i) * ts, 32 * kb, g);
        }
    }
    if constexpr (P::TL) __syncthreads();  // LDS tables visible

    // ---- state entering the segment (pre-rotated: Z' = rho Z)
    StateTiles<T, D, MP, CC> Zk, Zv;
    if (seg == 0) {
        const float* E1 = rho1;
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                floatx4 kr = zero4(), ki = zero4(), vr = zero4(), vi = zero4();
                if (mt < NMT) {
                    const int m = 16 * mt + r;
                    if (a.sk_in && m < a.M) {
                        kr = ld4f(a.sk_in + (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + 4 * g);
                        ki = ld4f(a.sk_in + (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + 4 * g);
                    }
                    if (a.sv_in) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int mv = 16 * mt + 4 * g + e;
                            if (mv < a.M) {
                                vr[e] = a.sv_in[(((size_t)bh * 2 + 0) * a.M + mv) * D + 16 * dt + r];
                                vi[e] = a.sv_in[(((size_t)bh * 2 + 1) * a.M + mv) * D + 16 * dt + r];
                            }
                        }
                    }
                    const float c1 = E1[m], s1 = E1[MP + m];
                    Zk[o][0][dt] = c1 * kr - s1 * ki;
                    Zk[o][1][dt] = s1 * kr + c1 * ki;
                    const floatx4 cv = ld4f(E1 + 16 * mt + 4 * g), sv = ld4f(E1 + MP + 16 * mt + 4 * g);
                    Zv[o][0][dt] = cv * vr - sv * vi;
                    Zv[o][1][dt] = sv * vr + cv * vi;
                } else {
                    Zk[o][0][dt] = Zk[o][1][dt] = Zv[o][0][dt] = Zv[o][1][dt] = zero4();
                }
            }
        }
    } else {
        const float* cy = a.carry + ((size_t)bh * (a.nseg - 1) + (seg - 1)) * 4 * MP * D;
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    if (mt < NMT) {
                        Zk[o][p][dt] = ld4f(cy + ((size_t)p * MP + 16 * mt + r) * D + 16 * dt + 4 * g);
                        Zv[o][p][dt] = ld4f(cy + (size_t)2 * MP * D +
                                            ((size_t)p * D + 16 * dt + r) * MP + 16 * mt + 4 * g);
                    } else {
                        Zk[o][p][dt] = Zv[o][p][dt] = zero4();
                    }
                }
        }
    }
    write_zvt<T, D, MP, CC>(ZvT, Zv, w, g, r);
    const double rT = AN ? a.rperiod[h] : 0.0;

    for (int n = 0; n < nch; ++n) {
        // lane indices re-derived per chunk (opaque_lane): addresses stay inside the loop
        const int r = opaque_lane(r_), g = opaque_lane(g_), tid = opaque_lane(tid_);
        const int tok0 = (ch0 + n) * C;
        const int c = min(C, a.L - tok0);
        if constexpr (!P::TL) {
            // tables in global memory: re-read per chunk rather than held in registers
            tABs = opaque(tABs);
            tABm = opaque(tABm);
            tEtab = opaque(tEtab);
            tEbar = opaque(tEbar);
            tErev = opaque(tErev);
            if constexpr (P::SPLIT) {
                fABs = opaque(fABs);
                fABm = opaque(fABm);
                fEtab = opaque(fEtab);
                fEbar = opaque(fEbar);
                fErev = opaque(fErev);
                fTw = opaque(fTw);
            }
        }
        __syncthreads();  // previous chunk done with Qs / Kt / Vt and the twiddle row
        stage_store<T, D, MP, true, CC>(st, Qs, Kt, Vt, c, tid);
        if constexpr (AN) {
            for (int m = tid; m < MP; m += GG::NTHR) {
                float cs = 0.f, sn = 0.f;
                if (m < a.M) anchor_phase(m, a.t0 + tok0, rT, cs, sn);
                lPh[m] = (T)cs;
                lPh[MP + m] = (T)(-sn);
            }
        }
        F kcur[KROWS ? 1 : GG::KBD];
        if constexpr (!KROWS) {
#pragma unroll
            for (int kb = 0; kb < GG::KBD; ++kb) kcur[kb] = (16 * w + r < c) ? kpf[kb] : zero_frag<T>();
        }
        if (n + 1 < nch) {
            const int tn = tok0 + C, cn = min(C, a.L - tn), i = min(16 * w + r, cn - 1);
            stage_load<T, D, MP, true, CC>(st, qb + (size_t)tn * ts, kb_ + (size_t)tn * ts, vb + (size_t)tn * ts, ts,
                                           cn, tid);
            if constexpr (!KROWS) {
#pragma unroll
                for (int kb = 0; kb < GG::KBD; ++kb) kpf[kb] = ld_frag<T>(kb_ + (size_t)(tn + i) * ts, 32 * kb, g);
            }
        }
        __syncthreads();  // staging and ZvT visible

        // ---- phase A: Gram tile (key tile w) and Q Z'_k^T on owned mode tiles
        floatx4 U[OWN][2][NT];
#pragma unroll
        for (int o = 0; o < OWN; ++o)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int ct = 0; ct < NT; ++ct) U[o][p][ct] = zero4();
        F zkf[OWN][2][GG::KBD];  // Z'_k^T tiles as A fragments (rows m, reduction over d)
#pragma unroll
        for (int o = 0; o < OWN; ++o)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int kb = 0; kb < GG::KBD; ++kb)
                    zkf[o][p][kb] = frag_from_acc<T>(Zk[o][p][2 * kb], Zk[o][p][2 * kb + 1]);
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
            const int j = 16 * ct + r;
            F qf[GG::KBD];
#pragma unroll
            for (int kb = 0; kb < GG::KBD; ++kb) qf[kb] = ld_frag<T>(Qs + (size_t)j * GG::LDQ, 32 * kb, g);
            if (ct >= w) {
                floatx4 acc = zero4();
#pragma unroll
                for (int kb = 0; kb < GG::KBD; ++kb) {
                    if constexpr (KROWS)
                        acc = mma(ld_frag_tr(Kt, GG::LDK, 16 * w, kb, g, r), qf[kb], acc);  // rows past c are 0
                    else
                        acc = mma(kcur[kb], qf[kb], acc);
                }
                if (ct == w) {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (4 * g + e > r) acc[e] = 0.f;
                }
                st4<T>(GT + (size_t)j * P::LDG + 16 * w + 4 * g, acc);
            }
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                if (w + NW * o < NMT) {
#pragma unroll
                    for (int p = 0; p < 2; ++p)
#pragma unroll
                        for (int kb = 0; kb < GG::KBD; ++kb)
                            U[o][p][ct] = mma(zkf[o][p][kb], qf[kb], U[o][p][ct]);
                }
            }
        }
        // Split chain (one owned mode tile): the conj(E) fragments and phase twiddles of phase
        // B are the same for every token tile; they are requested here, before the barrier, so
        // that their latency overlaps it (fragment-ordered table, reduction order 32kb + 8g + e,
        // matched by the Gram-tile reads below).
        F ebh[P::SPLIT ? 2 : 1][P::SPLIT ? GG::KBC : 1];
        F twh[P::SPLIT && !AN ? NT : 1];  // cos e = 0..3 | sin e = 0..3 of the lane's token, modes 16w + 4g + e
        if constexpr (P::SPLIT) {
            static_assert(OWN == 1 && !GG::HALF, "one owned mode tile, 32-token reduction blocks");
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int kb = 0; kb < GG::KBC; ++kb)
                    ebh[p][kb] = ld_global<F>(fEbar + ((size_t)((p * NMT + w) * GG::KBC + kb) * 64 + (tid & 63)) * 8);
            if constexpr (!AN) {
#pragma unroll
                for (int ct = 0; ct < NT; ++ct) twh[ct] = ld_global<F>(fTw + ((size_t)(w * NT + ct) * 64 + (tid & 63)) * 8);
            }
        }
        __syncthreads();

        // ---- phase B: + G conj(E), twiddle by E, publish U to LDS
        if constexpr (P::SPLIT) {
            const int mt = w;
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) {
#pragma unroll
                for (int kb = 0; kb < GG::KBC; ++kb) {
                    if (2 * kb <= ct) {
                        // keys 32kb + 8g + e; the half past the diagonal tile (g >= 2 when
                        // 2kb + 1 > ct) is not written this chunk: zero
                        F gf = ld_frag16_2x8(GT + (size_t)(16 * ct + r) * P::LDG, kb, g);
                        if (2 * kb + 1 > ct && g >= 2) gf = zero_frag<T>();
#pragma unroll
                        for (int p = 0; p < 2; ++p) U[0][p][ct] = mma(ebh[p][kb], gf, U[0][p][ct]);
                    }
                }
                const int j = 16 * ct + r;
                floatx4 cs, sn;
                if constexpr (AN) {
                    cs = to_f4(ld4_lds<T>(lPh + 16 * mt + 4 * g));
                    sn = to_f4(ld4_lds<T>(lPh + MP + 16 * mt + 4 * g));
                } else {
                    cs = to_f4(__builtin_shufflevector(twh[ct], twh[ct], 0, 1, 2, 3));
                    sn = to_f4(__builtin_shufflevector(twh[ct], twh[ct], 4, 5, 6, 7));
                }
                const floatx4 re = U[0][0][ct], im = U[0][1][ct];
                st4<T>(UT + (size_t)j * P::LDQU + 16 * mt + 4 * g, cs * re - sn * im);
                st4<T>(UT + (size_t)j * P::LDQU + MP + 16 * mt + 4 * g, sn * re + cs * im);
            }
        } else
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
            if (mt < NMT) {
#pragma unroll
                for (int ct = 0; ct < NT; ++ct) {
#pragma unroll
                    for (int kb = 0; kb < GG::KBC; ++kb) {
                        if (2 * kb <= ct) {
                            const T* grow = GT + (size_t)(16 * ct + r) * P::LDG;
                            const F gf = (2 * kb + 1 <= ct) ? ld_frag<T>(grow, 32 * kb, g)
                                                            : ld_frag_lo<T>(grow, 32 * kb, g);
#pragma unroll
                            for (int p = 0; p < 2; ++p)
                                U[o][p][ct] = mma(ld_frag_c<T, CC>(tEbar + (size_t)(16 * (p * NMT + mt) + r) * sR, kb, g),
                                                  gf, U[o][p][ct]);
                        }
                    }
                    const int j = 16 * ct + r;
                    floatx4 cs, sn;
                    if constexpr (AN) {
                        cs = to_f4(ld4_lds<T>(lPh + 16 * mt + 4 * g));
                        sn = to_f4(ld4_lds<T>(lPh + MP + 16 * mt + 4 * g));
                    } else {
                        cs = to_f4(ld4<T>(tEtab + (size_t)j * sEtab + 16 * mt + 4 * g));
                        sn = to_f4(ld4<T>(tEtab + (size_t)j * sEtab + MP + 16 * mt + 4 * g));
                    }
                    const floatx4 re = U[o][0][ct], im = U[o][1][ct];
                    st4<T>(UT + (size_t)j * P::LDQU + 16 * mt + 4 * g, cs * re - sn * im);
                    st4<T>(UT + (size_t)j * P::LDQU + MP + 16 * mt + 4 * g, sn * re + cs * im);
                }
            }
        }
        __syncthreads();

        // ---- per-token chain, split by output columns over the eight waves
        if constexpr (P::SPLIT) {
            static_assert(NT == 4 && NW == 8 && NMT == NW && NDT == NW, "eight waves, four token tiles");
            constexpr int NST = P::NST, NTT = NT * NST / NW;  // slot tiles; token tiles per wave
            const int lane = tid & 63;
            {
                // (4)-(5) scores of slot tile st for token tiles tt0 .. tt0 + NTT - 1, masked and
                // exponentiated against the tile's own maximum.  The slot-matrix fragment of
                // reduction block kb (fragment-ordered: one coalesced 1 KB load) is requested two
                // blocks ahead and serves every token tile of the wave.
                const int st = w % NST, tt0 = (w / NST) * NTT;
                F ab[2];
                auto ld_ab = [&](F& t, int kb) {
                    t = ld_global<F>(fABs + ((size_t)(st * GG::KBM + kb) * 64 + lane) * 8);
                };
                floatx4 sc[NTT];
#pragma unroll
                for (int i = 0; i < NTT; ++i) sc[i] = zero4();
                ld_ab(ab[0], 0);
                ld_ab(ab[1], 1);
#pragma unroll
                for (int kb = 0; kb < GG::KBM; ++kb) {
                    F uf[NTT];
#pragma unroll
                    for (int i = 0; i < NTT; ++i)
                        uf[i] = ld_frag16_2x8(UT + (size_t)(16 * (tt0 + i) + r) * P::LDQU, kb, g);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int i = 0; i < NTT; ++i) sc[i] = mma(ab[kb & 1], uf[i], sc[i]);
                    __builtin_amdgcn_sched_barrier(0);
                    if (kb + 2 < GG::KBM) ld_ab(ab[kb & 1], kb + 2);
                }
                __builtin_amdgcn_sched_barrier(0);
                const intx4 th = *reinterpret_cast<const intx4*>(tTheta + 16 * st + 4 * g);
#pragma unroll
                for (int i = 0; i < NTT; ++i) {
                    const int j = 16 * (tt0 + i) + r;
                    const long long pos = a.t0 + tok0 + j;
                    float mx = -INFINITY;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if (pos < (long long)th[e]) sc[i][e] = -INFINITY;
                        mx = fmaxf(mx, sc[i][e]);
                    }
                    mx = rows_max(mx);
                    // a slot tile can be fully masked (its weights are then zero); tile 0 holds
                    // slot 0, whose threshold is 0
                    const float mref = mx == -INFINITY ? 0.f : mx;
                    float sum = 0.f;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float ex = __expf(sc[i][e] - mref);
                        sc[i][e] = ex;
                        sum += ex;
                    }
                    sum = rows_sum(sum);
                    st4<T>(Pw + (size_t)j * P::LDP + 16 * st + 4 * g, sc[i]);
                    if (g == 0) {
                        sStat[(j * NST + st) * 2 + 0] = mx;
                        sStat[(j * NST + st) * 2 + 1] = sum;
                    }
                }
            }
            __syncthreads();  // P~ and the statistics visible; U no longer read
            {
                // (5) normalisation in place: wave w rescales the P~ rows of tokens 8w .. 8w + 7,
                // eight lanes per token, each lane SP/8 consecutive slots (within one slot tile):
                // P = P~ exp(m_tile - M) / sum_tiles exp(m_tile - M) s_tile, M the token's maximum
                constexpr int SPL = SP / 8;  // slots per lane
                static_assert(SPL == 8 || SPL == 16, "a lane's slots lie in one slot tile");
                const int jn = 8 * w + (lane >> 3), s0 = SPL * (lane & 7);
                float M = -INFINITY, mine = 0.f, tot = 0.f;
#pragma unroll
                for (int q = 0; q < NST; ++q) M = fmaxf(M, sStat[(jn * NST + q) * 2]);
#pragma unroll
                for (int q = 0; q < NST; ++q) {
                    const float e = __expf(sStat[(jn * NST + q) * 2] - M);  // 0 for a fully masked tile
                    tot += e * sStat[(jn * NST + q) * 2 + 1];
                    if (q == s0 / 16) mine = e;
                }
                const float f = mine * __builtin_amdgcn_rcpf(tot);
                T* prow = Pw + (size_t)jn * P::LDP + s0;
#pragma unroll
                for (int i = 0; i < SPL; i += 4) {
                    const typename Frag<T>::half x = ld4_lds<T>(prow + i);
                    st4<T>(prow + i, to_f4(x) * f);
                }
            }
            __syncthreads();  // P normalised

            {
                // (6)-(7) readout weights of mode tile w ([Re | Im] column tiles w, NMT + w) for
                // every token tile; the transposed slot-matrix fragments (fragment-ordered) are
                // loaded once and serve all four token tiles
                F am[2][P::KBS];
#pragma unroll
                for (int pp = 0; pp < 2; ++pp)
#pragma unroll
                    for (int ks = 0; ks < P::KBS; ++ks)
                        am[pp][ks] = ld_global<F>(fABm + ((size_t)((pp * NMT + w) * P::KBS + ks) * 64 + lane) * 8);
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    const int j = 16 * tt + r;
                    F pf[P::KBS];
#pragma unroll
                    for (int ks = 0; ks < P::KBS; ++ks) pf[ks] = ld_frag16_2x8(Pw + (size_t)j * P::LDP, ks, g);
                    floatx4 wa[2];
#pragma unroll
                    for (int pp = 0; pp < 2; ++pp) {
                        wa[pp] = zero4();
#pragma unroll
                        for (int ks = 0; ks < P::KBS; ++ks) wa[pp] = mma(am[pp][ks], pf[ks], wa[pp]);
                    }
                    floatx4 cs, sn;
                    if constexpr (AN) {
                        cs = to_f4(ld4_lds<T>(lPh + 16 * w + 4 * g));
                        sn = to_f4(ld4_lds<T>(lPh + MP + 16 * w + 4 * g));
                    } else {
                        const F tw = ld_global<F>(fTw + ((size_t)(w * NT + tt) * 64 + lane) * 8);
                        cs = to_f4(__builtin_shufflevector(tw, tw, 0, 1, 2, 3));
                        sn = to_f4(__builtin_shufflevector(tw, tw, 4, 5, 6, 7));
                    }
                    const floatx4 a0 = wa[0], b0 = wa[1];
                    st4<T>(UT + (size_t)j * P::LDQU + 16 * w + 4 * g, a0 * cs + b0 * sn);
                    st4<T>(UT + (size_t)j * P::LDQU + MP + 16 * w + 4 * g, a0 * sn - b0 * cs);
                }
            }
            __syncthreads();  // W'' rows visible; P~ no longer read

            {
                // (8)-(9) output head-dim tile w of every token tile.  The causal H tiles
                // (key tile kt <= token tile tt, ten of them) are shared out over the waves and
                // published to LDS over P~ as [token][key] rows (the tiles just past the
                // diagonal, which the 32-key blocks of the H V products also read, as zeros).
                T* Hs = Pw;
                auto h_tile = [&](int q, int& tt, int& kt) {
                    // q = 0..9 over (tt, kt), kt <= tt, in the order (0,0) (1,0) (1,1) (2,0) ...
                    tt = q < 1 ? 0 : q < 3 ? 1 : q < 6 ? 2 : 3;
                    kt = q - tt * (tt + 1) / 2;
                };
#pragma unroll
                for (int u2 = 0; u2 < 2; ++u2) {
                    const int q = w + NW * u2;
                    if (q < 12) {
                        int tt, kt;
                        floatx4 hh = zero4();
                        if (q < 10) {
                            h_tile(q, tt, kt);
                            const T* fe = fEtab + ((size_t)kt * GG::KBM * 64 + lane) * 8;
                            F ef[GG::KBM];
#pragma unroll
                            for (int kb = 0; kb < GG::KBM; ++kb) ef[kb] = ld_global<F>(fe + (size_t)kb * 64 * 8);
#pragma unroll
                            for (int kb = 0; kb < GG::KBM; ++kb)
                                hh = mma(ef[kb], ld_frag16_2x8(UT + (size_t)(16 * tt + r) * P::LDQU, kb, g), hh);
                            if (kt == tt) {
#pragma unroll
                                for (int e = 0; e < 4; ++e)
                                    if (4 * g + e > r) hh[e] = 0.f;
                            }
                        } else {
                            tt = 2 * (q - 10);  // the zero tiles (0, 1) and (2, 3)
                            kt = tt + 1;
                        }
                        st4<T>(Hs + (size_t)(16 * tt + r) * P::LDP + 16 * kt + 4 * g, hh);
                    }
                }
                // O^T tile (head dims 16w .., tokens of tile tt) = Re(W'' Z'_v) over the modes
                F zf[GG::KBM];
#pragma unroll
                for (int kb = 0; kb < GG::KBM; ++kb) zf[kb] = ld_frag16_2x8(ZvT + (size_t)(16 * w + r) * GG::LDZ, kb, g);
                floatx4 oa[NT];
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
                    oa[tt] = zero4();
#pragma unroll
                    for (int kb = 0; kb < GG::KBM; ++kb)
                        oa[tt] = mma(zf[kb], ld_frag16_2x8(UT + (size_t)(16 * tt + r) * P::LDQU, kb, g), oa[tt]);
                }
                __syncthreads();  // H tiles visible
#pragma unroll
                for (int tt = 0; tt < NT; ++tt) {
#pragma unroll
                    for (int kb = 0; kb < GG::KBC; ++kb) {
                        if (2 * kb <= tt)
                            oa[tt] = mma(ld_frag16_2x8(Vt + (size_t)(16 * w + r) * GG::LDK, kb, g),
                                         ld_frag16_2x8(Hs + (size_t)(16 * tt + r) * P::LDP, kb, g), oa[tt]);
                    }
                    const int j = 16 * tt + r;
                    if (j < c) st4<T>(ob + (size_t)(tok0 + j) * tso + 16 * w + 4 * g, oa[tt]);
                }
            }
        } else if (w < NT) {
        // ---- per-token chain on token tile w: scores, softmax, readout, output
            const int j = 16 * w + r;
            const long long pos = a.t0 + tok0 + j;
            F uf[GG::KBM];
#pragma unroll
            for (int kb = 0; kb < GG::KBM; ++kb) uf[kb] = ld_frag<T>(UT + (size_t)j * P::LDQU, 32 * kb, g);
            floatx4 sc[P::NST];
#pragma unroll
            for (int s4 = 0; s4 < P::NST; ++s4) {
                sc[s4] = zero4();
#pragma unroll
                for (int kb = 0; kb < GG::KBM; ++kb)
                    sc[s4] = mma(ld_frag<T>(tABs + (size_t)(16 * s4 + r) * sABs, 32 * kb, g), uf[kb], sc[s4]);
            }
            float mx = -INFINITY;
#pragma unroll
            for (int s4 = 0; s4 < P::NST; ++s4) {
                const intx4 th = *reinterpret_cast<const intx4*>(tTheta + 16 * s4 + 4 * g);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (pos < (long long)th[e]) sc[s4][e] = -INFINITY;
                    mx = fmaxf(mx, sc[s4][e]);
                }
            }
            mx = rows_max(mx);
            float sum = 0.f;
#pragma unroll
            for (int s4 = 0; s4 < P::NST; ++s4)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float ex = __expf(sc[s4][e] - mx);
                    sc[s4][e] = ex;
                    sum += ex;
                }
            sum = rows_sum(sum);
            const float inv = __builtin_amdgcn_rcpf(sum);  // sum >= 1: the maximum slot contributes exp(0)
            F pf[P::KBS];
#pragma unroll
            for (int kb = 0; kb < P::KBS; ++kb) pf[kb] = frag_from_acc<T>(sc[2 * kb] * inv, sc[2 * kb + 1] * inv);

            // W'' by groups of MG mode tiles: the Re and Im tiles of a group are produced,
            // twiddled and packed into their fragments together, so that only 2 MG accumulator
            // tiles are live at a time.  Fragment kb holds combined tiles 2kb, 2kb + 1 of
            // [Re tiles | Im tiles]: for MG = 2 those are Re (wf[kb']) and Im (wf[NMT/2 + kb'])
            // of the group's two mode tiles; for a single mode tile (NMT = 1) wf[0] = [Re | Im].
            constexpr int MG = (NMT % 2 == 0) ? 2 : 1;
            static_assert(MG == 2 || NMT == 1, "mode-tile grouping");
            F wf[GG::KBM];
#pragma unroll
            for (int kb = 0; kb < NMT / MG; ++kb) {
                floatx4 wa[2][MG];  // [Re, Im][mode tile MG kb + u]
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int u = 0; u < MG; ++u) {
                        const int t = p * NMT + MG * kb + u;
                        wa[p][u] = zero4();
#pragma unroll
                        for (int ks = 0; ks < P::KBS; ++ks)
                            wa[p][u] = mma(ld_frag<T>(tABm + (size_t)(16 * t + r) * sABm, 32 * ks, g), pf[ks], wa[p][u]);
                    }
#pragma unroll
                for (int u = 0; u < MG; ++u) {
                    const int mt = MG * kb + u;
                    floatx4 cs, sn;
                    if constexpr (AN) {
                        cs = to_f4(ld4_lds<T>(lPh + 16 * mt + 4 * g));
                        sn = to_f4(ld4_lds<T>(lPh + MP + 16 * mt + 4 * g));
                    } else {
                        cs = to_f4(ld4<T>(tEtab + (size_t)j * sEtab + 16 * mt + 4 * g));
                        sn = to_f4(ld4<T>(tEtab + (size_t)j * sEtab + MP + 16 * mt + 4 * g));
                    }
                    const floatx4 am = wa[0][u], bm = wa[1][u];
                    wa[0][u] = am * cs + bm * sn;
                    wa[1][u] = am * sn - bm * cs;
                }
                if constexpr (MG == 2) {
                    wf[kb] = frag_from_acc<T>(wa[0][0], wa[0][1]);
                    wf[NMT / 2 + kb] = frag_from_acc<T>(wa[1][0], wa[1][1]);
                } else {
                    wf[0] = frag_from_acc<T>(wa[0][0], wa[1][0]);
                }
            }

            floatx4 oa[NDT];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                oa[dt] = zero4();
#pragma unroll
                for (int kb = 0; kb < GG::KBM; ++kb)
                    oa[dt] = mma(ld_frag<T>(ZvT + (size_t)(16 * dt + r) * GG::LDZ, 32 * kb, g), wf[kb], oa[dt]);
            }
            floatx4 hh[NT < 2 ? 2 : NT];  // a 16-token chunk pairs its one tile with a zero tile
            hh[NT < 2 ? 1 : 0] = zero4();
#pragma unroll
            for (int kt = 0; kt < NT; ++kt) {
                hh[kt] = zero4();
                if (kt <= w) {
#pragma unroll
                    for (int kb = 0; kb < GG::KBM; ++kb)
                        hh[kt] = mma(ld_frag<T>(tEtab + (size_t)(16 * kt + r) * sEtab, 32 * kb, g), wf[kb], hh[kt]);
                    if (kt == w) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (4 * g + e > r) hh[kt][e] = 0.f;
                    }
                }
            }
#pragma unroll
            for (int kb = 0; kb < GG::KBC; ++kb) {
                if (2 * kb <= w) {
                    const F hf = frag_from_acc<T>(hh[2 * kb], hh[2 * kb + 1]);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt)
                        oa[dt] = mma(ld_frag_c<T, CC>(Vt + (size_t)(16 * dt + r) * GG::LDK, kb, g), hf, oa[dt]);
                }
            }
            if (j < c) {
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) st4<T>(ob + (size_t)(tok0 + j) * tso + 16 * dt + 4 * g, oa[dt]);
            }
        }
        __syncthreads();  // everyone done reading ZvT

        if constexpr (P::SPLIT) {
            // step (10) with rho^{c-i} from the fragment-ordered table (reduction order 32kb +
            // 8g + e, matched by the K and V reads); a ragged last chunk builds it from E32
            F ef[GG::KBC][2];
#pragma unroll
            for (int kb = 0; kb < GG::KBC; ++kb)
#pragma unroll
                for (int p = 0; p < 2; ++p)
                    ef[kb][p] = (c == C) ? ld_global<F>(fErev + ((size_t)((p * NMT + w) * GG::KBC + kb) * 64 + (tid & 63)) * 8)
                                         : erev_frag_nat<MP>(E32h, 2 * MP, c, p, w, kb, g, r);
            const float* Ec = (c == C) ? rhoC : rhoL;
            advance_owned<T, D, MP, CC>(Zk, Zv, Kt, Vt, ef, Ec[16 * w + r], Ec[MP + 16 * w + r], ld4f(Ec + 16 * w + 4 * g),
                                        ld4f(Ec + MP + 16 * w + 4 * g), g, r);
        } else {
            advance_state<T, D, MP, CC>(Zk, Zv, Kt, Vt, rhoC, rhoL, E32h, tErev, sR, c, w, g, r);
        }
        write_zvt<T, D, MP, CC>(ZvT, Zv, w, g, r);
    }

    // ---- final state (last segment): Z = conj(rho) Z'
    if (seg == a.nseg - 1) {
        const float* E1 = rho1;
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = w + NW * o;
            if (mt < NMT) {
                const int m = 16 * mt + r;
                const float c1 = E1[m], s1 = E1[MP + m];
                const floatx4 cv = ld4f(E1 + 16 * mt + 4 * g), sv = ld4f(E1 + MP + 16 * mt + 4 * g);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    if (a.sk_out && m < a.M) {
                        const floatx4 re = Zk[o][0][dt], im = Zk[o][1][dt];
                        st4f(a.sk_out + (((size_t)bh * 2 + 0) * a.M + m) * D + 16 * dt + 4 * g, c1 * re + s1 * im);
                        st4f(a.sk_out + (((size_t)bh * 2 + 1) * a.M + m) * D + 16 * dt + 4 * g, c1 * im - s1 * re);
                    }
                    if (a.sv_out) {
                        const floatx4 re = Zv[o][0][dt], im = Zv[o][1][dt];
                        const floatx4 nr = cv * re + sv * im, ni = cv * im - sv * re;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int mv = 16 * mt + 4 * g + e;
                            if (mv < a.M) {
                                a.sv_out[(((size_t)bh * 2 + 0) * a.M + mv) * D + 16 * dt + r] = nr[e];
                                a.sv_out[(((size_t)bh * 2 + 1) * a.M + mv) * D + 16 * dt + r] = ni[e];
                            }
                        }
                    }
                }
            }
        }
    }
}

}  // namespace bla
