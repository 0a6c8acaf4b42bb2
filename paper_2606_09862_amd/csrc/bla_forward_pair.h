// Chunked BLA forward for bf16 operands, two sequence units per workgroup.
//
// Same algebra as bla_forward.h (chunks of C = 64 tokens, pre-rotated state
// Z' = rho Z, steps (1)-(10) of that file), reorganised for latency hiding on
// gfx950:
//
//  * A workgroup of 8 waves runs U = 2 independent units (b, h, segment) of the
//    same head, 4 waves each, so every SIMD holds two waves whose dependency
//    chains interleave.  The head's tables are shared in LDS.
//  * Each table is stored once.  The second layout a contraction needs (slot
//    matrix [A|B] with the reduction over slots; the phase table with the
//    reduction over tokens; K and V with the reduction over tokens) is read with
//    the transposing LDS load ds_read_b64_tr_b16.
//  * The phase table holds conj(rho^i) = [cos | -sin] (row i, modes along the row).
//    It serves the twiddles, the transposed operands of steps (3) and (10) and the
//    rows of step (8) without sign changes: the readout weights are kept as
//    [Re W'' | -Im W''] and Z'_v is published as [Re | Im].
//  * The state update uses rho^{c-i} = rho^c conj(rho^i):
//        Z' <- rho^c o (Z' + sum_i conj(rho^i) [k_i | v_i]),
//    so one phase table serves steps (3), (8), (10) and the twiddles, and a
//    ragged last chunk needs no table of its own (rows past c are zero).
//  * Anchored slots (Sec. 3.3, Alg. 1/3) keep the same mode state and differ only in
//    the readout: with u = Q Z'_k^T + G conj(E) as above and P the chunk's absolute
//    start, the anchored query-mode products are rho^P o conj(u) instead of E o u, and
//    the readout weights (a + i b) o conj(rho^P) instead of (a - i b) o E.  With -B in
//    the slot matrix both are the rotating twiddles of steps (3) and (7) applied with
//    the one row [cos | sin](m w P) for every token of the chunk.
//  * Sequences are split into segments.  summary_pair_kernel reduces every segment
//    but the last to its summary (step (10) alone from a zero state); a unit then
//    starts from the preceding summaries combined in its prologue,
//        Z'_g = rho^{L_s} o (... (rho^{L_s} o (rho Z_in) + S_0) ...) + S_{g-1},
//    which is the state recurrence taken a whole segment (L_s tokens) at a time.
#pragma once

#include <math.h>

#include "bla_forward.h"

namespace bla {

// Lane-ordered segment summaries of the pair path: part p (Re Z_k, Im Z_k, Re Z_v, Im Z_v) of
// mode tile mt and head-dim tile dt is one accumulator tile, stored as 64 consecutive 16-byte
// pieces (lane l's four floats at 4 l), so that the summary kernel writes and the forward
// prologue reads it as one contiguous 1 KB block.  Lane (g, r) holds Z_k[16mt + r][16dt + 4g
// .. + 3] and Z_v[16dt + r][16mt + 4g .. + 3] (the two kernels' tile layouts).  The one-unit
// plans keep the row-major [4][..] layout that their scan reads.
template <int D, int MP>
__host__ __device__ constexpr size_t sum_tile(int p, int mt, int dt)
{
    return (((size_t)p * (MP / 16) + mt) * (D / 16) + dt) * 256;
}

template <int D, int MP, int SP> struct Pair {
    static constexpr int C = kChunk, NT = C / 16, WPU = 4;
    static constexpr int NMT = MP / 16, NDT = D / 16, NST = SP / 16;
    static constexpr int KBD = D / 32, KBM = 2 * MP / 32, KBC = C / 32, KBS = SP / 32;
    static constexpr int OWN = (NMT + WPU - 1) / WPU;
    // Row strides (elements): every row is 16 elements longer than its data, i.e. the stride
    // is 8 (mod 32) dwords.  With that stride a 16-lane group's 16-byte row-fragment reads
    // (16 rows, same columns) and its transposed reads (4 rows x 32 bytes) both run at the
    // full LDS rate on gfx950 (about 230 and 180 B/clk per compute unit, against about 120 at
    // strides of 2, 4 or 6 (mod 32) dwords).  K and V, whose row fragments pair with the
    // query rows, keep the natural order and use the reduction order 32kb + 8g + e (16-byte
    // reads as well).  The slot matrix and the phase table are read transposed more often
    // than row-wise, so they keep the natural order, whose transposed reads are conflict-free
    // at this stride, and their row fragments are two separate 8-byte reads.  The published
    // state is row-swizzled as well: every wave writes its owned tiles there once per chunk
    // as 8-byte pieces (16 rows x 4 consecutive pieces per instruction), which at these
    // strides put 4 rows on the same banks; swz4_col leaves 2.  Z'_k is read as 16-byte
    // fragments; Z'_v, read against accumulator-derived fragments, is stored fragment-ordered
    // (frag_col) under the same swizzle, so its fragments are 16-byte reads as well
    // (ld_frag16_sw4 for both, without conflicts).
    static constexpr int LAB = 2 * MP + 16;  // [A|B]:     [SP][LAB]
    static constexpr int LE = 2 * MP + 16;   // phase tab: [C][LE]
    static constexpr int LK = D + 16;        // K, V:      [C][LK]
    static constexpr int LZK = D + 16;       // Z'_k:      [2MP][LZK]  (Re rows, then Im rows)
    static constexpr int LZ = 2 * MP + 16;   // Z'_v:      [D][LZ]     (Re | Im along the row, fragment-ordered)
    // per unit, after Z'_v: the anchored twiddle row [cos | sin](m w P) of the chunk, [2MP]
    // (the queries do not pass through LDS: each lane loads its own token's fragments)
    static constexpr size_t AB_ELEMS = (size_t)SP * LAB;
    static constexpr size_t E_ELEMS = (size_t)C * LE;
    static constexpr size_t SHARED_BYTES = 2 * (AB_ELEMS + E_ELEMS) + 3 * 2 * MP * 4 + SP * 4;
    static constexpr size_t UNIT_ELEMS =
        2 * (size_t)C * LK + (size_t)2 * MP * LZK + (size_t)D * LZ + (size_t)2 * MP;
    static constexpr size_t UNIT_BYTES = 2 * UNIT_ELEMS;
    // two units per workgroup (two waves per SIMD) when their tiles fit in LDS and their
    // registers in half of the file (at most four owned state tiles per wave)
    static constexpr int U = (SHARED_BYTES + 2 * UNIT_BYTES <= kMaxLds && D <= 64 && MP <= 64) ? 2 : 1;
    static constexpr bool FITS = SHARED_BYTES + U * UNIT_BYTES <= kMaxLds;
    static constexpr size_t LDS_BYTES = SHARED_BYTES + U * UNIT_BYTES;
    // staging: K and V of one chunk in 16-byte pieces, spread over the unit's 256 threads
    static constexpr int PIECES = 2 * C * D / 8;
    static constexpr int PPT = (PIECES + 255) / 256;
    static_assert(NT == WPU, "one token tile per wave of a unit");
};

template <int D, int MP> using PStateDM = floatx4[(MP / 16 + 3) / 4][2][D / 16];
template <int D, int MP, int SP> using PState = PStateDM<D, MP>;
template <int D, int MP, int SP> using PStage = bf16x8[Pair<D, MP, SP>::PPT];

// ut: thread index within the unit (0..255); k, v: the chunk's first rows.
// ts: token stride of k, v (elements).
template <int D, int MP, int SP>
__device__ __forceinline__ void pair_stage_load(PStage<D, MP, SP>& st, const bf16* k, const bf16* v, int ts,
                                                int c, int ut)
{
    using P = Pair<D, MP, SP>;
    constexpr int PR = D / 8;  // pieces per row
#pragma unroll
    for (int i = 0; i < P::PPT; ++i) {
        const int u = ut + 256 * i;
        if (P::PIECES % 256 == 0 || u < P::PIECES) {
            const int which = u / (P::C * PR), rem = u % (P::C * PR);
            const int row = min(rem / PR, c - 1), pc = rem % PR;
            const unsigned off = (unsigned)(row * ts + 8 * pc);  // within one chunk
            const bf16* src = (which == 0 ? k : v) + off;
            st[i] = *reinterpret_cast<const bf16x8*>(src);
        }
    }
}

// FULL: the chunk has all C rows (no zero fill past c).  Rows are 16-byte aligned (LK is a
// multiple of 8 elements), so each piece is one 16-byte store.
template <int D, int MP, int SP, bool FULL>
__device__ __forceinline__ void pair_stage_store(const PStage<D, MP, SP>& st, bf16* Ks, bf16* Vs, int c, int ut)
{
    using P = Pair<D, MP, SP>;
    constexpr int PR = D / 8;
    static_assert(P::LK % 8 == 0, "16-byte rows");
#pragma unroll
    for (int i = 0; i < P::PPT; ++i) {
        const int u = ut + 256 * i;
        if (P::PIECES % 256 == 0 || u < P::PIECES) {
            const int which = u / (P::C * PR), rem = u % (P::C * PR);
            const int row = rem / PR, pc = rem % PR;
            bf16* dst = (which == 0 ? Ks : Vs) + (size_t)row * P::LK;
            const bf16x8 x = (FULL || row < c) ? st[i] : bf16x8{};
            *reinterpret_cast<bf16x8*>(dst + 8 * pc) = x;
        }
    }
}

// Copy a table of ROWS x COLS bf16 (source rows contiguous) into LDS rows of stride DST,
// all loads of a thread in flight before its stores.  FO: store the rows fragment-ordered
// (frag_col); SW: store them row-swizzled (swz_col); NEG_HI: negate the upper half of every
// row (columns COLS/2 ..), e.g. [cos | sin] -> [cos | -sin].
template <int ROWS, int COLS, int DST, int NTHR, bool FO = false, bool SW = false, bool NEG_HI = false>
__device__ __forceinline__ void pair_copy(bf16* dst, const bf16* src, int tid)
{
    typedef int intx2 __attribute__((ext_vector_type(2)));
    constexpr int PIECES = ROWS * COLS / 4, ITER = (PIECES + NTHR - 1) / NTHR;
    intx2 buf[ITER];
#pragma unroll
    for (int i = 0; i < ITER; ++i) {
        const int u = tid + i * NTHR;
        if (PIECES % NTHR == 0 || u < PIECES) buf[i] = reinterpret_cast<const intx2*>(src)[u];
    }
#pragma unroll
    for (int i = 0; i < ITER; ++i) {
        const int u = tid + i * NTHR;
        if (PIECES % NTHR == 0 || u < PIECES) {
            const int row = u / (COLS / 4), col = 4 * (u % (COLS / 4));
            intx2 x = buf[i];
            if (NEG_HI && col >= COLS / 2) x ^= (int)0x80008000;  // the sign bits of four bf16
            *reinterpret_cast<intx2*>(dst + (size_t)row * DST + (FO ? frag_col(col) : SW ? swz_col(row, col) : col)) = x;
        }
    }
}

// Publish the owned mode tiles of the state as bf16 operands: Z'_k as [2MP][LZK] rows
// (mode m, head-dim along the row, swz4_col) and Z'_v as [D][LZ] rows (head-dim d, modes along
// the row, fragment-ordered and swz4_col).
template <int D, int MP, int SP>
__device__ __forceinline__ void pair_write_zk(bf16* ZkT, const PState<D, MP, SP>& Zk, int wl, int g, int r)
{
    using P = Pair<D, MP, SP>;
#pragma unroll
    for (int o = 0; o < P::OWN; ++o) {
        const int mt = wl + P::WPU * o;
        if (mt < P::NMT) {
#pragma unroll
            for (int dt = 0; dt < P::NDT; ++dt) {
                st4<bf16>(ZkT + (size_t)(16 * mt + r) * P::LZK + swz4_col(r, 16 * dt + 4 * g), Zk[o][0][dt]);
                st4<bf16>(ZkT + (size_t)(MP + 16 * mt + r) * P::LZK + swz4_col(r, 16 * dt + 4 * g), Zk[o][1][dt]);
            }
        }
    }
}

template <int D, int MP, int SP>
__device__ __forceinline__ void pair_write_zv(bf16* ZvT, const PState<D, MP, SP>& Zv, int wl, int g, int r)
{
    using P = Pair<D, MP, SP>;
#pragma unroll
    for (int o = 0; o < P::OWN; ++o) {
        const int mt = wl + P::WPU * o;
        if (mt < P::NMT) {
#pragma unroll
            for (int dt = 0; dt < P::NDT; ++dt) {
                st4<bf16>(ZvT + (size_t)(16 * dt + r) * P::LZ + swz4_col(r, frag_col(16 * mt + 4 * g)), Zv[o][0][dt]);
                st4<bf16>(ZvT + (size_t)(16 * dt + r) * P::LZ + swz4_col(r, frag_col(MP + 16 * mt + 4 * g)), Zv[o][1][dt]);
            }
        }
    }
}

// Step (10) on the wave's owned mode tiles: Z' <- rho^c o (Z' + sum_i conj(rho^i) [k_i | v_i])
// with K, V ([C][LK], rows past c zero) and the phase table ([C][LE], row-swizzled) read
// transposed from LDS, and rho^c (cos | sin, float32) from Ec.
template <int D, int MP, int LK, int LE>
__device__ __forceinline__ void pair_advance(PStateDM<D, MP>& Zk, PStateDM<D, MP>& Zv, const bf16* Ks,
                                             const bf16* Vs, const bf16* sE, const float* Ec, int wl,
                                             int g, int r)
{
    using F = bf16x8;
    constexpr int NMT = MP / 16, NDT = D / 16, OWN = (NMT + 3) / 4, KBC = kChunk / 32;
#pragma unroll
    for (int kb = 0; kb < KBC; ++kb) {
        F ktf[NDT], vtf[NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            ktf[dt] = ld_frag_tr(Ks, LK, 16 * dt, kb, g, r);
            vtf[dt] = ld_frag_tr(Vs, LK, 16 * dt, kb, g, r);
        }
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = wl + 4 * o;
            if (mt < NMT) {
                const F ecf = ld_frag_tr_sw(sE, LE, 16 * mt, kb, g, r);
                const F esf = ld_frag_tr_sw(sE, LE, MP + 16 * mt, kb, g, r);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) {
                    Zk[o][0][dt] = mma(ktf[dt], ecf, Zk[o][0][dt]);
                    Zk[o][1][dt] = mma(ktf[dt], esf, Zk[o][1][dt]);
                    Zv[o][0][dt] = mma(ecf, vtf[dt], Zv[o][0][dt]);
                    Zv[o][1][dt] = mma(esf, vtf[dt], Zv[o][1][dt]);
                }
            }
        }
    }
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = wl + 4 * o;
        if (mt < NMT) {
            const float cc = Ec[16 * mt + r], ss = Ec[MP + 16 * mt + r];
            const floatx4 cv = ld4f(Ec + 16 * mt + 4 * g), sv = ld4f(Ec + MP + 16 * mt + 4 * g);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                const floatx4 kr = Zk[o][0][dt], ki = Zk[o][1][dt];
                Zk[o][0][dt] = cc * kr - ss * ki;
                Zk[o][1][dt] = ss * kr + cc * ki;
                const floatx4 vr = Zv[o][0][dt], vi = Zv[o][1][dt];
                Zv[o][0][dt] = cv * vr - sv * vi;
                Zv[o][1][dt] = sv * vr + cv * vi;
            }
        }
    }
}

// ---------------------------------------------------------------------------------
// Segment summaries: DS = D/32 workgroups per (b, h, summarised block), each reducing 32
// columns of K and V.  Every summarised chunk is full (only the last chunk of a sequence can
// be shorter, and the last segment is never summarised).
//
// K and V are streamed once.  Narrow column slices make many small workgroups (four waves
// and about 44 KB of LDS at MP = 64, three per compute unit), each staging NPF = 4 chunks
// ahead in registers plus one in LDS, so that many loads are in flight per compute unit.
// The DS slices of a block run on one XCD (see the index mapping in the kernel), so each
// 128-byte line of K and V is fetched from HBM once.
//
// Wave w owns column tile wd = w % 2 of its slice and mode tiles wm + WM*j (wm = w / 2).
// K and V are double-buffered in LDS (one barrier per chunk).
template <int D, int MP> struct SumPair {
    static constexpr int C = kChunk, KBC = C / 32;
    static constexpr int DW = 32, DS = D / DW;
    static constexpr int NDT = DW / 16, NMT = MP / 16;
    static constexpr int WD = NDT, WM = NMT < 2 ? NMT : 2, NW = WD * WM;
    static constexpr int NTHR = 64 * NW;
    static constexpr int ODT = 1, OMT = NMT / WM;
    static constexpr int MINB = MP <= 64 ? 3 : 2;  // workgroups per compute unit (launch bound)
    // row strides: the four rows of a transposed read's 16-lane group, and the two groups
    // of one LDS cycle, fall on distinct banks
    static constexpr int LK = DW + 16;
    static constexpr int LE = 2 * MP + 16;
    static constexpr size_t E_ELEMS = (size_t)C * LE, KV_ELEMS = (size_t)C * LK;
    static constexpr size_t LDS_BYTES = 2 * (E_ELEMS + 4 * KV_ELEMS) + 2 * MP * 4;
    static constexpr int PR = DW / 8;                 // 16-byte pieces per row of a tile
    static constexpr int PIECES = 2 * C * PR;         // pieces of K and V per chunk
    static constexpr int PPT = (PIECES + NTHR - 1) / NTHR;
    static constexpr int NPF = 4;  // chunks in flight in registers (plus one in LDS)
    static_assert(D % DW == 0 && NMT % WM == 0, "column and mode tiles split evenly over the waves");
    static_assert(NPF % 2 == 0, "the LDS buffer parity follows the unrolled stage index");
};
template <int D, int MP> using SStage = bf16x8[SumPair<D, MP>::PPT];
template <int D, int MP> using SState = floatx4[SumPair<D, MP>::OMT][SumPair<D, MP>::ODT][2];

// k, v: first row of the chunk, column offset of the workgroup's slice applied; ts: token
// stride; w: the wave (uniform).  A wave's 64 pieces come from one of K and V, so the base
// pointer of each load is uniform and the per-lane part a 32-bit offset.
template <int D, int MP>
__device__ __forceinline__ void sum_stage_load(SStage<D, MP>& st, const bf16* k, const bf16* v, int ts, int w,
                                               int lane)
{
    using P = SumPair<D, MP>;
    static_assert((P::C * P::PR) % 64 == 0, "a wave's pieces lie in one of K and V");
#pragma unroll
    for (int i = 0; i < P::PPT; ++i) {
        const int u0 = 64 * w + P::NTHR * i;  // the wave's first piece (uniform)
        if (P::PIECES % P::NTHR == 0 || u0 < P::PIECES) {
            const int which = u0 / (P::C * P::PR), rem = u0 % (P::C * P::PR) + lane;
            const unsigned off = (unsigned)((rem / P::PR) * ts + 8 * (rem % P::PR));
            st[i] = *reinterpret_cast<const bf16x8*>((which == 0 ? k : v) + off);
        }
    }
}

template <int D, int MP>
__device__ __forceinline__ void sum_stage_store(const SStage<D, MP>& st, bf16* Ks, bf16* Vs, int tid)
{
    using P = SumPair<D, MP>;
    static_assert(P::LK % 8 == 0, "16-byte rows");
#pragma unroll
    for (int i = 0; i < P::PPT; ++i) {
        const int u = tid + P::NTHR * i;
        if (P::PIECES % P::NTHR == 0 || u < P::PIECES) {
            const int which = u / (P::C * P::PR), rem = u % (P::C * P::PR);
            bf16* dst = (which == 0 ? Ks : Vs) + (size_t)(rem / P::PR) * P::LK + 8 * (rem % P::PR);
            *reinterpret_cast<bf16x8*>(dst) = st[i];
        }
    }
}

// Z <- rot o Z for the owned mode tiles; rot = (cos | sin) of the rotation, float32 in LDS.
// KMAJOR: the tiles hold (d rows, m columns) (Z_k); otherwise (m rows, d columns) (Z_v).
template <int D, int MP, bool KMAJOR>
__device__ __forceinline__ void sum_rotate(SState<D, MP>& Z, const float* rot, int wm, int g, int r)
{
    using P = SumPair<D, MP>;
#pragma unroll
    for (int j = 0; j < P::OMT; ++j) {
        const int mt = wm + P::WM * j;
        if constexpr (KMAJOR) {
            const float cc = rot[16 * mt + r], ss = rot[MP + 16 * mt + r];
#pragma unroll
            for (int i = 0; i < P::ODT; ++i) {
                const floatx4 kr = Z[j][i][0], ki = Z[j][i][1];
                Z[j][i][0] = cc * kr - ss * ki;
                Z[j][i][1] = ss * kr + cc * ki;
            }
        } else {
            const floatx4 cv = ld4f(rot + 16 * mt + 4 * g), sv = ld4f(rot + MP + 16 * mt + 4 * g);
#pragma unroll
            for (int i = 0; i < P::ODT; ++i) {
                const floatx4 vr = Z[j][i][0], vi = Z[j][i][1];
                Z[j][i][0] = cv * vr - sv * vi;
                Z[j][i][1] = sv * vr + cv * vi;
            }
        }
    }
}

template <int D, int MP> constexpr int summary_threads() { return SumPair<D, MP>::NTHR; }
// x extent of the summary grid for `jobs` (b, block) pairs: padded to a multiple of 8, times DS
template <int D, int MP> constexpr long long summary_grid_x(long long jobs)
{
    return (jobs + 7) / 8 * 8 * SumPair<D, MP>::DS;
}

// grid: summary_grid_x(B * nbs) x H workgroups of NTHR threads; every (b, summarised block)
// pair has DS workgroups, one per 32-column slice of K and V; the block covers chunks
// [blk * cpb, (blk + 1) * cpb).  PLAIN_E: the phase table holds [cos | sin] (the one-unit
// kernels' tables) instead of conj(rho^i) = [cos | -sin]; its sine half is negated on the
// copy into LDS.  The summaries are the same either way.
template <int D, int MP, bool PLAIN_E = false>
__global__ __launch_bounds__((SumPair<D, MP>::NTHR))
__attribute__((amdgpu_waves_per_eu(SumPair<D, MP>::MINB * SumPair<D, MP>::NW / 4))) void summary_pair_kernel(FwdArgs a)
{
    using P = SumPair<D, MP>;
    using F = bf16x8;
    constexpr int C = P::C, NMT = P::NMT, ODT = P::ODT, OMT = P::OMT, WD = P::WD, WM = P::WM, DS = P::DS;
    __shared__ __attribute__((aligned(16))) char lds_raw[P::LDS_BYTES];
    bf16* sE = reinterpret_cast<bf16*>(lds_raw);  // [C][LE]: conj(rho^i) = [cos | -sin]
    bf16* KV = sE + P::E_ELEMS;                   // [buffer][K | V][C][LK]
    float* sRhoC = reinterpret_cast<float*>(KV + 4 * P::KV_ELEMS);

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(w >= 0 && w < P::NW);
    const int wd = w % WD, wm = w / WD;
    const int g = (tid & 63) >> 4, r = tid & 15;
    // Workgroups are dealt to the eight XCDs by linear index (x mod 8 with a row length that
    // is a multiple of 8); the DS slices of a block take indices 8 apart, so they share an
    // XCD and its L2 and each 128-byte line of K and V is fetched from HBM once.
    const int xq = blockIdx.x / 8, ds = xq % DS, job = (xq / DS) * 8 + blockIdx.x % 8;
    if (job >= a.B * a.nbs) return;  // grid padding (whole workgroup, before any barrier)
    const int h = blockIdx.y, blk = job % a.nbs, b = job / a.nbs;
    const int bh = b * a.H + h;
    const size_t first = (size_t)blk * a.cpb * C;
    const int ts = a.in_t;
    const bf16* kb_ = (const bf16*)a.k + fwd_in_base(a, bh) + first * ts + ds * P::DW;
    const bf16* vb = (const bf16*)a.v + fwd_in_base(a, bh) + first * ts + ds * P::DW;

    // tables first: their loads are then the oldest in flight when they are stored
    pair_copy<C, 2 * MP, P::LE, P::NTHR, false, false, PLAIN_E>(sE, (const bf16*)a.Etab + (size_t)h * C * 2 * MP, tid);
    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    for (int i = tid; i < 2 * MP; i += P::NTHR) sRhoC[i] = E32h[(size_t)C * 2 * MP + i];

    // NPF chunks of K/V in flight ahead of the one being reduced.  The loop is unrolled
    // NPF times so that the staging registers keep fixed roles, and every load is
    // unconditional (chunk indices past the block re-read its last chunk), so the wait
    // before each store covers exactly the loads of that stage.
    constexpr int NPF = P::NPF;
    const int last = a.cpb - 1;
    SStage<D, MP> st[NPF];
#pragma unroll
    for (int i = 0; i < NPF; ++i) {
        const size_t off = (size_t)min(i, last) * C * ts;
        sum_stage_load<D, MP>(st[i], kb_ + off, vb + off, ts, w, tid & 63);
    }
    sum_stage_store<D, MP>(st[0], KV, KV + P::KV_ELEMS, tid);
    {
        const size_t off = (size_t)min(NPF, last) * C * ts;
        sum_stage_load<D, MP>(st[0], kb_ + off, vb + off, ts, w, tid & 63);
    }
    __syncthreads();  // tables and chunk 0 visible

    // conj(rho^i) fragments of the owned mode tiles ([cos | -sin], the reduction over i),
    // the same for every chunk: held in registers for the whole block
    F ef[OMT][P::KBC][2];
#pragma unroll
    for (int j = 0; j < OMT; ++j)
#pragma unroll
        for (int kb = 0; kb < P::KBC; ++kb) {
            ef[j][kb][0] = ld_frag_tr(sE, P::LE, 16 * (wm + WM * j), kb, g, r);
            ef[j][kb][1] = ld_frag_tr(sE, P::LE, MP + 16 * (wm + WM * j), kb, g, r);
        }

    SState<D, MP> Zk, Zv;  // [mode tile][column tile][Re, Im]
#pragma unroll
    for (int j = 0; j < OMT; ++j)
#pragma unroll
        for (int i = 0; i < ODT; ++i) Zk[j][i][0] = Zk[j][i][1] = Zv[j][i][0] = Zv[j][i][1] = zero4();

    // Per chunk: Zk <- rho^C o (Zk + Yk) and Zv <- rho^C o (Zv + Yv).  The rotation of Zv
    // is deferred to the start of the next chunk, so that each half below pairs the
    // matrix-core products of one state with the vector rotation of the other:
    //   1: Zk += Yk  with  Zv <- rho^C o Zv (the previous chunk's rotation; Zv = 0 at n = 0)
    //   2: Zv += Yv  with  Zk <- rho^C o Zk
    for (int n0 = 0; n0 < a.cpb; n0 += NPF) {
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            const int n = n0 + s;
            const bf16* Ks = KV + (size_t)(s & 1) * 2 * P::KV_ELEMS;  // chunk n (n and s share parity)
            const bf16* Vs = Ks + P::KV_ELEMS;
            // chunk n + 1 into the other buffer (last read by chunk n - 1, before the
            // previous barrier), then chunk n + 1 + NPF into the freed registers
            {
                const int s1 = (s + 1) % NPF;  // a constant once the loop is unrolled
                bf16* Kn = KV + (size_t)(s1 & 1) * 2 * P::KV_ELEMS;
                sum_stage_store<D, MP>(st[s1], Kn, Kn + P::KV_ELEMS, tid);
                const size_t off = (size_t)min(n + 1 + NPF, last) * C * ts;
                sum_stage_load<D, MP>(st[s1], kb_ + off, vb + off, ts, w, tid & 63);
            }
            if (n < a.cpb) {
                F ktf[P::KBC][ODT], vtf[P::KBC][ODT];
#pragma unroll
                for (int kb = 0; kb < P::KBC; ++kb)
#pragma unroll
                    for (int i = 0; i < ODT; ++i) {
                        ktf[kb][i] = ld_frag_tr(Ks, P::LK, 16 * (wd + WD * i), kb, g, r);
                        vtf[kb][i] = ld_frag_tr(Vs, P::LK, 16 * (wd + WD * i), kb, g, r);
                    }
                // 1
#pragma unroll
                for (int kb = 0; kb < P::KBC; ++kb)
#pragma unroll
                    for (int j = 0; j < OMT; ++j)
#pragma unroll
                        for (int i = 0; i < ODT; ++i) {
                            Zk[j][i][0] = mma(ktf[kb][i], ef[j][kb][0], Zk[j][i][0]);
                            Zk[j][i][1] = mma(ktf[kb][i], ef[j][kb][1], Zk[j][i][1]);
                        }
                sum_rotate<D, MP, false>(Zv, sRhoC, wm, g, r);
#pragma unroll
                for (int q = 0; q < 2 * P::KBC * ODT * OMT; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);  // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x2, 2, 0);  // two VALU
                }
                // 2
#pragma unroll
                for (int kb = 0; kb < P::KBC; ++kb)
#pragma unroll
                    for (int j = 0; j < OMT; ++j)
#pragma unroll
                        for (int i = 0; i < ODT; ++i) {
                            Zv[j][i][0] = mma(ef[j][kb][0], vtf[kb][i], Zv[j][i][0]);
                            Zv[j][i][1] = mma(ef[j][kb][1], vtf[kb][i], Zv[j][i][1]);
                        }
                sum_rotate<D, MP, true>(Zk, sRhoC, wm, g, r);
#pragma unroll
                for (int q = 0; q < 2 * P::KBC * ODT * OMT; ++q) {
                    __builtin_amdgcn_sched_group_barrier(0x8, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x2, 2, 0);
                }
            }
            __syncthreads();  // chunk n + 1 visible; chunk n's buffer free
        }
    }
    // the deferred rotation of the last chunk
    sum_rotate<D, MP, false>(Zv, sRhoC, wm, g, r);

    // Zk tiles hold (d rows, m columns), Zv tiles (m rows, d columns)
    float* S = a.summ + ((size_t)bh * a.nbs + blk) * 4 * MP * D;
#pragma unroll
    for (int j = 0; j < OMT; ++j) {
        const int mt = wm + WM * j;
#pragma unroll
        for (int i = 0; i < ODT; ++i) {
            const int dt = ds * P::NDT + wd + WD * i;
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                if constexpr (PLAIN_E) {  // one-unit plans: the scan's row-major layout
                    st4f(S + ((size_t)q * MP + 16 * mt + r) * D + 16 * dt + 4 * g, Zk[j][i][q]);
                    st4f(S + (size_t)2 * MP * D + ((size_t)q * D + 16 * dt + r) * MP + 16 * mt + 4 * g,
                         Zv[j][i][q]);
                } else {  // pair plans: lane order (sum_tile)
                    st4f(S + sum_tile<D, MP>(q, mt, dt) + 4 * (tid & 63), Zk[j][i][q]);
                    st4f(S + sum_tile<D, MP>(2 + q, mt, dt) + 4 * (tid & 63), Zv[j][i][q]);
                }
            }
        }
    }
}

// grid: ceil(B*nseg/U) x H workgroups of 256*U threads; workgroup (x, h) runs the
// units 2x and 2x+1 (U = 2) of head h.  Units are numbered over (b, i) with
// i = 0, 1, 2, 3, ... taking segments 0, nseg-1, 1, nseg-2, ..., so that the two units
// of a workgroup combine about nseg-1 segment summaries between them.
//
// Per chunk, two phases separated by barriers:
//   1. each wave runs the whole per-token chain of one token tile in registers (steps
//      (1)-(9), reading the published state of the chunk start), and independently
//      advances its owned mode tiles of the float32 state (step (10));
//   2. each wave publishes its state tiles for the next chunk and stages the next chunk.
// The second unit takes the token tiles in reverse order, so that every SIMD runs one
// short and one long causal tile.
template <int D, int MP, int SP, bool ANCHOR>
__global__ __launch_bounds__((256 * Pair<D, MP, SP>::U)) void forward_pair_kernel(FwdArgs a)
{
    using P = Pair<D, MP, SP>;
    using F = bf16x8;
    constexpr int C = P::C, NT = P::NT, NMT = P::NMT, NDT = P::NDT, OWN = P::OWN;
    __shared__ __attribute__((aligned(16))) char lds_raw[P::LDS_BYTES];
    bf16* sAB = reinterpret_cast<bf16*>(lds_raw);
    bf16* sE = sAB + P::AB_ELEMS;
    // rho, rho^C and rho^c_last (c_last: length of the last chunk, the same for every
    // unit of the workgroup)
    float* sRho = reinterpret_cast<float*>(sE + P::E_ELEMS);
    int* sTheta = reinterpret_cast<int*>(sRho + 6 * MP);

    const int tid = threadIdx.x;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int u = wv / P::WPU, wl = wv % P::WPU;  // unit and wave within the unit
    const int ut = tid & 255;                      // thread index within the unit
    const int g = (tid & 63) >> 4, r = tid & 15;
    const int tt = u == 0 ? wl : NT - 1 - wl;      // token tile of this wave's chain
    const int h = blockIdx.y;
    const int per_head = a.B * a.nseg;
    const int v_unit = blockIdx.x * P::U + u;
    const bool active = v_unit < per_head;
    const int b = active ? v_unit / a.nseg : 0, si = active ? v_unit % a.nseg : 0;
    const int seg = (si & 1) ? a.nseg - 1 - (si >> 1) : (si >> 1);
    const int bh = b * a.H + h;

    bf16* base = reinterpret_cast<bf16*>(lds_raw + P::SHARED_BYTES + (size_t)u * P::UNIT_BYTES);
    bf16* Ks = base;
    bf16* Vs = Ks + (size_t)C * P::LK;
    bf16* ZkT = Vs + (size_t)C * P::LK;
    bf16* ZvT = ZkT + (size_t)2 * MP * P::LZK;
    _Float16* sPh = reinterpret_cast<_Float16*>(ZvT + (size_t)D * P::LZ);  // anchored twiddle row

    const float* E32h = a.E32 + (size_t)h * (C + 1) * 2 * MP;
    // ---- shared tables
    pair_copy<SP, 2 * MP, P::LAB, 256 * P::U, false, true>(sAB, (const bf16*)a.ABs, tid);
    pair_copy<C, 2 * MP, P::LE, 256 * P::U, false, true>(sE, (const bf16*)a.Etab + (size_t)h * C * 2 * MP, tid);
    const int c_last = a.L - (a.nch - 1) * C;
    for (int i = tid; i < 2 * MP; i += 256 * P::U) {
        sRho[i] = E32h[2 * MP + i];
        sRho[2 * MP + i] = E32h[(size_t)C * 2 * MP + i];
        sRho[4 * MP + i] = E32h[(size_t)c_last * 2 * MP + i];
    }
    for (int i = tid; i < SP; i += 256 * P::U) sTheta[i] = a.theta[(size_t)h * SP + i];

    const int ch0 = seg * a.cps;
    const int nch = active ? min(a.cps, a.nch - ch0) : 0;
    const bf16* qb = (const bf16*)a.q + fwd_in_base(a, bh);
    const bf16* kb_ = (const bf16*)a.k + fwd_in_base(a, bh);
    const bf16* vb = (const bf16*)a.v + fwd_in_base(a, bh);
    bf16* ob = (bf16*)a.o + fwd_out_base(a, bh);
    const int ts = a.in_t, tso = a.out_t;
    // Chunk n + 1 is loaded into registers during chunk n; every load is unconditional
    // (an exhausted or idle unit re-reads a chunk that exists), so the wait before each
    // store to LDS covers only that stage's loads.
    const int last = max(nch - 1, 0);
    auto stage_chunk = [&](PStage<D, MP, SP>& st, int n) {
        const int tn = (ch0 + min(n, last)) * C, cn = min(C, a.L - tn);
        pair_stage_load<D, MP, SP>(st, kb_ + (size_t)tn * ts, vb + (size_t)tn * ts, ts, cn, ut);
    };
    // The query fragments of the wave's own token row j = 16 tt + r of chunk n (clamped to the
    // chunk's last token; rows past it are computed and never stored), elements 32kb + 8g ..
    // + 7: the reduction order of steps (1)-(2), whose other operands (Z'_k and K rows) are
    // stored in the natural order.  Loaded straight from memory one chunk ahead.
    auto load_q = [&](bf16x8 (&qd)[P::KBD], int n) {
        const int tn = (ch0 + min(n, last)) * C, cn = min(C, a.L - tn);
        const bf16* src = qb + (size_t)(tn + min(16 * tt + r, cn - 1)) * ts + 8 * g;
#pragma unroll
        for (int kb = 0; kb < P::KBD; ++kb) qd[kb] = *reinterpret_cast<const bf16x8*>(src + 32 * kb);
    };

    // anchored slots: the twiddle row of chunk n at its absolute start t0 + (ch0 + n) C
    const double rT = ANCHOR ? a.rperiod[h] : 0.0;
    auto phase_row = [&](int n) {
        if constexpr (ANCHOR) {
            for (int m = ut; m < MP; m += 256) {
                float cs = 0.f, sn = 0.f;
                if (m < a.M) anchor_phase(m, a.t0 + (long long)(ch0 + n) * C, rT, cs, sn);
                sPh[m] = (_Float16)cs;
                sPh[MP + m] = (_Float16)sn;
            }
        }
    };
    halfx4 twc[NMT], tws[NMT];
    auto twiddle_row = [&](int mt, halfx4& c, halfx4& n) {
        if constexpr (ANCHOR) {
            c = *reinterpret_cast<const halfx4*>(sPh + 16 * mt + 4 * g);
            n = *reinterpret_cast<const halfx4*>(sPh + MP + 16 * mt + 4 * g);
        } else {
            c = twc[mt];
            n = tws[mt];
        }
    };

    __syncthreads();  // tables visible

    // ---- state entering the unit's segment (pre-rotated: Z' = rho Z)
    PState<D, MP, SP> Zk, Zv;
    const float* E1 = sRho;
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
        const int mt = wl + P::WPU * o;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
            Zk[o][0][dt] = Zk[o][1][dt] = Zv[o][0][dt] = Zv[o][1][dt] = zero4();
            if (mt < NMT && active) {
                const int m = 16 * mt + r;
                floatx4 kr = zero4(), ki = zero4(), vr = zero4(), vi = zero4();
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
            }
        }
    }
    // combine the summaries of the blocks before this segment (Horner, block by block);
    // the next block's summary is loaded while the current one is combined (every load
    // unconditional, indices clamped, so each wait covers exactly one block's loads)
    if (active && seg > 0) {
        const int nblk = seg * (a.cps / a.cpb);
        const float* rb = a.rotblk + (size_t)h * 2 * MP;
        const float* Sb = a.summ + (size_t)bh * a.nbs * 4 * MP * D;
        floatx4 sj[2][OWN][NDT][4];  // [buffer][owned tile][head-dim tile][Re k, Im k, Re v, Im v]
        auto load_block = [&](floatx4 (&dst)[OWN][NDT][4], int j) {
            const float* Sj = Sb + (size_t)min(j, nblk - 1) * 4 * MP * D;
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = min(wl + P::WPU * o, NMT - 1);
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                    for (int pp = 0; pp < 4; ++pp) dst[o][dt][pp] = ld4f(Sj + sum_tile<D, MP>(pp, mt, dt) + 4 * (tid & 63));
            }
        };
        auto combine = [&](const floatx4 (&src)[OWN][NDT][4]) {
#pragma unroll
            for (int o = 0; o < OWN; ++o) {
                const int mt = wl + P::WPU * o;
                if (mt < NMT) {
                    const float cc = rb[16 * mt + r], ss = rb[MP + 16 * mt + r];
                    const floatx4 cv = ld4f(rb + 16 * mt + 4 * g), sv = ld4f(rb + MP + 16 * mt + 4 * g);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const floatx4 kr = Zk[o][0][dt], ki = Zk[o][1][dt];
                        Zk[o][0][dt] = cc * kr - ss * ki + src[o][dt][0];
                        Zk[o][1][dt] = ss * kr + cc * ki + src[o][dt][1];
                        const floatx4 vr = Zv[o][0][dt], vi = Zv[o][1][dt];
                        Zv[o][0][dt] = cv * vr - sv * vi + src[o][dt][2];
                        Zv[o][1][dt] = sv * vr + cv * vi + src[o][dt][3];
                    }
                }
            }
        };
        load_block(sj[0], 0);
        for (int j = 0; j < nblk; j += 2) {
            load_block(sj[1], j + 1);
            combine(sj[0]);
            if (j + 1 < nblk) {
                load_block(sj[0], j + 2);
                combine(sj[1]);
            }
        }
    }
    // Rotating slots: the twiddle row of steps (3) and (7) is the lane's own phase row
    // conj(rho^j) = [cos | -sin](m w j) of its token j = 16 tt + r, the same in every chunk,
    // so it is held in registers as half precision for the whole segment (modes 16 mt + 4 g
    // .. + 3 of each mode tile mt).  Loaded after the summary combination, whose buffers
    // need the registers.
    if constexpr (!ANCHOR) {
        const float* Ej = E32h + (size_t)(16 * tt + r) * 2 * MP;
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) {
            const floatx4 cv = ld4f(Ej + 16 * mt + 4 * g), sv = ld4f(Ej + MP + 16 * mt + 4 * g);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                twc[mt][e] = (_Float16)cv[e];
                tws[mt][e] = (_Float16)(-sv[e]);
            }
        }
    }
    PStage<D, MP, SP> st;
    F qf[P::KBD];
    load_q(qf, 0);
    stage_chunk(st, 0);
    pair_write_zk<D, MP, SP>(ZkT, Zk, wl, g, r);
    pair_write_zv<D, MP, SP>(ZvT, Zv, wl, g, r);
    {
        const int c0 = nch > 0 ? min(C, a.L - ch0 * C) : 0;
        if (c0 == C)
            pair_stage_store<D, MP, SP, true>(st, Ks, Vs, c0, ut);
        else
            pair_stage_store<D, MP, SP, false>(st, Ks, Vs, c0, ut);
    }
    phase_row(0);
    stage_chunk(st, 1);
    __syncthreads();  // chunk 0 and the initial state visible

    // both units run the same number of iterations (the barriers are workgroup-wide);
    // an exhausted or idle unit computes on zero-filled tiles and stores nothing
    const int nmax = a.cps;
    for (int n = 0; n < nmax; ++n) {
        const bool live = n < nch;
        const int tok0 = (ch0 + n) * C;
        const int c = live ? min(C, a.L - tok0) : 0;

        // ================= phase 1: the token chain of tile tt (steps 1-9)
        {
            const int j = 16 * tt + r;
            // (1)-(2) X = Q Z'_k^T + G conj(E): tiles over [Re | Im] modes (rows) x tokens (columns)
            floatx4 ua[2 * NMT];
#pragma unroll
            for (int t = 0; t < 2 * NMT; ++t) {
                ua[t] = zero4();
#pragma unroll
                for (int kb = 0; kb < P::KBD; ++kb)
                    ua[t] = mma(ld_frag16_sw4(ZkT + (size_t)(16 * t + r) * P::LZK, kb, g, r), qf[kb], ua[t]);
            }
            floatx4 ga[NT];  // Gram tiles: keys (rows) x this tile's queries (columns), keys <= query
#pragma unroll
            for (int kt = 0; kt < NT; ++kt) {
                ga[kt] = zero4();
                if (kt <= tt) {
#pragma unroll
                    for (int kb = 0; kb < P::KBD; ++kb)
                        ga[kt] = mma(ld_frag16(Ks + (size_t)(16 * kt + r) * P::LK, kb, g), qf[kb], ga[kt]);
                    if (kt == tt) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (4 * g + e > r) ga[kt][e] = 0.f;
                    }
                }
            }
            load_q(qf, n + 1);  // the queries of this chunk are no longer needed
#pragma unroll
            for (int kb = 0; kb < P::KBC; ++kb) {
                if (2 * kb <= tt) {
                    const F gf = frag_from_acc<bf16>(ga[2 * kb], ga[2 * kb + 1]);
#pragma unroll
                    for (int mt = 0; mt < NMT; ++mt) {
                        ua[mt] = mma(ld_frag_tr_sw(sE, P::LE, 16 * mt, kb, g, r), gf, ua[mt]);
                        ua[NMT + mt] = mma(ld_frag_tr_sw(sE, P::LE, MP + 16 * mt, kb, g, r), gf, ua[NMT + mt]);
                    }
                }
            }
            // (3) U = E o X  (anchored: [Re | -Im] of rho^P o conj(X))
#pragma unroll
            for (int mt = 0; mt < NMT; ++mt) {
                halfx4 cs, ns;
                twiddle_row(mt, cs, ns);
                twiddle_h<false>(cs, ns, ua[mt], ua[NMT + mt]);
            }
            F uf[P::KBM];
#pragma unroll
            for (int kb = 0; kb < P::KBM; ++kb) uf[kb] = frag_from_acc<bf16>(ua[2 * kb], ua[2 * kb + 1]);

            // (4) scores against the slot matrix (unscaled in LDS)
            const long long pos_ll = a.t0 + tok0 + j;
            const int pos = pos_ll < (1ll << 30) ? (int)pos_ll : (1 << 30);  // every threshold is below 2^30
            floatx4 sc[P::NST];
#pragma unroll
            for (int s4 = 0; s4 < P::NST; ++s4) {
                sc[s4] = zero4();
#pragma unroll
                for (int kb = 0; kb < P::KBM; ++kb)
                    sc[s4] = mma(ld_frag_2x8_sw(sAB + (size_t)(16 * s4 + r) * P::LAB, kb, g, r), uf[kb], sc[s4]);
            }
            // (5) masked softmax in base-2 units (z * scale * log2 e).  Thresholds grow with
            // the slot and padded slots carry INT32_MAX, so a chunk whose first position
            // reaches the last threshold needs no mask.
            const float k2 = a.scale * 1.44269504088896341f;
            float sum = 0.f;
            if (k2 > 0.f && a.t0 + tok0 >= (long long)sTheta[SP - 1]) {
                // no slot masked and a positive scale: the maximum of the raw scores, and the
                // scale folded into the exponent's argument, exp2(k2 z - k2 max z)
                float mx = -INFINITY;
#pragma unroll
                for (int s4 = 0; s4 < P::NST; ++s4)
#pragma unroll
                    for (int e = 0; e < 4; ++e) mx = fmaxf(mx, sc[s4][e]);
                const float nm = -k2 * rows_max(mx);
#pragma unroll
                for (int s4 = 0; s4 < P::NST; ++s4)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float ex = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[s4][e], k2, nm));
                        sc[s4][e] = ex;
                        sum += ex;
                    }
            } else {
                float mx = -INFINITY;
#pragma unroll
                for (int s4 = 0; s4 < P::NST; ++s4) {
                    const intx4 th = *reinterpret_cast<const intx4*>(sTheta + 16 * s4 + 4 * g);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        sc[s4][e] = pos < th[e] ? -INFINITY : sc[s4][e] * k2;
                        mx = fmaxf(mx, sc[s4][e]);
                    }
                }
                mx = rows_max(mx);
#pragma unroll
                for (int s4 = 0; s4 < P::NST; ++s4)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float ex = __builtin_amdgcn_exp2f(sc[s4][e] - mx);
                        sc[s4][e] = ex;
                        sum += ex;
                    }
            }
            sum = rows_sum(sum);
            const float inv = __builtin_amdgcn_rcpf(sum);  // sum >= 1: the maximum slot contributes exp(0)
            F pf[P::KBS];
#pragma unroll
            for (int kb = 0; kb < P::KBS; ++kb) pf[kb] = frag_from_acc<bf16>(sc[2 * kb] * inv, sc[2 * kb + 1] * inv);

            // (6) [a | b] = P [A | B], the slot matrix read transposed
            floatx4 wa[2 * NMT];
#pragma unroll
            for (int t = 0; t < 2 * NMT; ++t) {
                wa[t] = zero4();
#pragma unroll
                for (int kb = 0; kb < P::KBS; ++kb) wa[t] = mma(ld_frag_tr_sw(sAB, P::LAB, 16 * t, kb, g, r), pf[kb], wa[t]);
            }
            // (7) [Re W'' | -Im W''] with W'' = (a - i b) o E  (anchored: (a + i b) o conj(rho^P)):
            //     (a, b) <- (a c - b n, b c + a n)
#pragma unroll
            for (int mt = 0; mt < NMT; ++mt) {
                halfx4 cs, ns;
                twiddle_row(mt, cs, ns);
                twiddle_h<true>(cs, ns, wa[mt], wa[NMT + mt]);
            }
            F wf[P::KBM];
#pragma unroll
            for (int kb = 0; kb < P::KBM; ++kb) wf[kb] = frag_from_acc<bf16>(wa[2 * kb], wa[2 * kb + 1]);

            // (8) O = Re(W'' Z'_v) + V^T H^T with H = tril(Re(W'' conj(E)^T))
            floatx4 oa[NDT];
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                oa[dt] = zero4();
#pragma unroll
                for (int kb = 0; kb < P::KBM; ++kb)
                    oa[dt] = mma(ld_frag16_sw4(ZvT + (size_t)(16 * dt + r) * P::LZ, kb, g, r), wf[kb], oa[dt]);
            }
            floatx4 hh[NT];
#pragma unroll
            for (int kt = 0; kt < NT; ++kt) {
                hh[kt] = zero4();
                if (kt <= tt) {
#pragma unroll
                    for (int kb = 0; kb < P::KBM; ++kb)
                        hh[kt] = mma(ld_frag_2x8_sw(sE + (size_t)(16 * kt + r) * P::LE, kb, g, r), wf[kb], hh[kt]);
                    if (kt == tt) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (4 * g + e > r) hh[kt][e] = 0.f;
                    }
                }
            }
            // (9) O += V^T H^T, V read transposed
#pragma unroll
            for (int kb = 0; kb < P::KBC; ++kb) {
                if (2 * kb <= tt) {
                    const F hf = frag_from_acc<bf16>(hh[2 * kb], hh[2 * kb + 1]);
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) oa[dt] = mma(ld_frag_tr(Vs, P::LK, 16 * dt, kb, g, r), hf, oa[dt]);
                }
            }
            if (j < c) {
                bf16* oc = ob + (size_t)tok0 * tso;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt) st4<bf16>(oc + (unsigned)(j * tso + 16 * dt + 4 * g), oa[dt]);
            }
        }
        // ================= phase 1 (independent of the chain): step (10) on the owned mode tiles
        if (live) {
            const float* Ec = sRho + (c == C ? 2 * MP : 4 * MP);  // a chunk shorter than C is the last one
            pair_advance<D, MP, P::LK, P::LE>(Zk, Zv, Ks, Vs, sE, Ec, wl, g, r);
        }
        __syncthreads();  // chunk n and its published state no longer read

        // ================= phase 2: publish the state of chunk n + 1, stage chunk n + 1
        if (live) {
            pair_write_zk<D, MP, SP>(ZkT, Zk, wl, g, r);
            pair_write_zv<D, MP, SP>(ZvT, Zv, wl, g, r);
        }
        const int cn = n + 1 < nch ? min(C, a.L - (tok0 + C)) : 0;
        if (cn == C)
            pair_stage_store<D, MP, SP, true>(st, Ks, Vs, cn, ut);
        else
            pair_stage_store<D, MP, SP, false>(st, Ks, Vs, cn, ut);
        phase_row(n + 1);
        stage_chunk(st, n + 2);
        __syncthreads();  // chunk n + 1 and its state visible
    }

    // ---- final state (last segment): Z = conj(rho) Z'
    if (active && seg == a.nseg - 1) {
#pragma unroll
        for (int o = 0; o < OWN; ++o) {
            const int mt = wl + P::WPU * o;
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
