// Launch plan and kernel argument blocks shared by the host API and the kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "bla.h"

namespace bla {

constexpr int kChunk = 64;      // default tokens per chunk of the parallel form (the pair kernels' only one)
constexpr int kThreads = 256;   // 4 waves of 64 lanes per workgroup
constexpr int kMaxHeadsPerTableLaunch = 64;

// Sizes and workspace layout of one forward / step call.
struct Plan {
    int B, H, L, D, M, S;
    int MP, SP;          // M padded to 16/32/64/128, S padded to 32/64/128/256
    int C;               // chunk length
    int bf16;            // 1 if q,k,v,o are bfloat16
    int64_t t0;
    float scale;
    int nch;             // chunks per sequence
    int nseg, cps;       // segments per sequence, chunks per segment
    int upw;             // sequence units per forward workgroup (1, or 2 for the pair kernel)
    int pair;            // 1 if the bf16 pair kernel runs the forward pass
    int anchor;          // 1: slots anchored at absolute phase 0 (Sec. 3.3), 0: at the current token
    int cpb, nbs;        // chunks per summarised block, summarised blocks per sequence
    size_t unit_floats;  // floats of one full (k and v) pre-rotated state: 4*MP*D
    // 1: the tables read from global memory by the d = M = 128 forward kernel also exist in
    // operand-fragment order (see FragTabArgs)
    int fragtab;
    // workspace byte offsets
    size_t off_E32, off_EbarT, off_ErevT, off_Etab, off_ABs, off_ABm, off_theta,
        off_rotblk, off_trig, off_rperiod, off_period, off_summ, off_carry,
        off_fABs, off_fABm, off_fEtab, off_fEbar, off_fErev, off_fTw, total;
};

// Fragment-ordered copies of row-major bf16 tables M[R][K]: operand fragment (i, kb) of rows
// 16i..16i+15 and reduction block kb (columns 32kb + 8g + e for lane 16g + r) is stored as
// 64 consecutive 16-byte pieces, piece l = 16g + r holding M[16i + r][32kb + 8g .. + 7].  A
// wave then loads a fragment as one contiguous 1 KB block (coalesced), where the row-major
// table costs a separate 16-byte access per lane.
struct FragTabArgs {
    const void* ABs;   // [SP][2MP]
    const void* ABm;   // [2MP][SP]
    const void* Etab;  // [H][C][2MP]
    const void* EbarT; // [H][2MP][C]
    const void* ErevT; // [H][2MP][C]
    void* fABs;
    void* fABm;
    void* fEtab;
    void* fEbar;
    void* fErev;
    // phase twiddles in lane order: [H][MP/16 mode tiles][C/16 token tiles][64 lanes][8], lane
    // 16g + r holding cos | sin of m w j for j = 16 ct + r, m = 16 mt + 4g .. + 3
    void* fTw;
    int H, C, MP, SP;
};

struct TableArgs {
    float* E32;     // [H][C+1][2MP]  cos | sin of m w j, j = 0..C
    void* EbarT;    // [H][2MP][C]    cos(m w i) | -sin(m w i)       (operand type)
    void* ErevT;    // [H][2MP][C]    cos(m w (C-i)) | sin(m w (C-i)) (operand type)
    void* Etab;     // [H][C][2MP]    cos(m w i) | sin(m w i), or | -sin(m w i) if conj_tab (operand type)
    void* ABs;      // [SP][2MP]      scale * (A | B)                (operand type)
    void* ABm;      // [2MP][SP]      (A | B) transposed             (operand type)
    int* theta;     // [H][SP]        start-mask thresholds (INT32_MAX for padded slots)
    float* rotblk;  // [H][2MP]       cos | sin of m w Lblk
    float* trig;    // [2][SP]        cos | sin of 2 pi k / S, k < S (zero past S)
    double* rperiod; // [H]           1 / T of each head (clamped period)
    double* period;  // [H]           the clamped period T of each head
    int M, S, MP, SP, C, Lblk, h0, nh, with_shared;
    int conj_tab;   // Etab holds conj(rho^i) (the bf16 pair kernels' convention)
    int jrows;      // phase rows j = 0..jrows-1 computed (C + 1; 2 for a decode step)
    float scale;    // factor folded into ABs (1 when the kernel applies the score scale itself)
    int negB;       // store -B in ABs / ABm (the slot matrix of the anchored readout)
    double T[kMaxHeadsPerTableLaunch];  // clamped periods of heads h0..h0+nh-1
};

struct FwdArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    const float* sk_in;
    const float* sv_in;
    float* sk_out;
    float* sv_out;
    const float* E32;
    const void* EbarT;
    const void* ErevT;
    const void* Etab;
    const void* ABs;
    const void* ABm;
    // fragment-ordered copies (FragTabArgs), when the plan has them
    const void* fABs;
    const void* fABm;
    const void* fEtab;
    const void* fEbar;
    const void* fErev;
    const void* fTw;
    const int* theta;
    float* summ;
    float* carry;
    const float* rotblk;
    const double* rperiod;  // [H] 1 / T (anchored readout only)
    int B, H, L, M;
    int C;        // tokens per chunk (the per-head phase table E32 has C + 1 rows)
    int nch, nseg, cps, cpb, nbs;
    long long t0;
    float scale;  // score scale (applied by the pair kernel; folded into ABs otherwise)
    int anchor;   // 1: slots anchored at absolute phase 0 (Sec. 3.3)
    // Element strides of q, k, v (in_*) and o (out_*): row (b, h) starts at b * x_b + h * x_h,
    // token t of it at + t * x_t, and its d elements are contiguous.  [B, H, L, d] is
    // (H L d, L d, d); a fused projection output [B, L, 3, H, d] is (3 L H d, d, 3 H d).
    long long in_b, in_h, out_b, out_h;
    int in_t, out_t;
};

// Where row (b, h) = bh of q, k, v (in) or o (out) starts, in elements.
__host__ __device__ inline size_t fwd_in_base(const FwdArgs& a, int bh)
{
    return (size_t)(bh / a.H) * (size_t)a.in_b + (size_t)(bh % a.H) * (size_t)a.in_h;
}
__host__ __device__ inline size_t fwd_out_base(const FwdArgs& a, int bh)
{
    return (size_t)(bh / a.H) * (size_t)a.out_b + (size_t)(bh % a.H) * (size_t)a.out_h;
}

struct StepArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    const int64_t* pos;
    float* sk;
    float* sv;
    const float* E32;
    const float* trig;
    const int* theta;
    const double* rperiod;  // [H] 1 / T (anchored readout only)
    int B, H, M, S, SP;
    long long t0;
    float scale;
    int anchor;   // 1: slots anchored at absolute phase 0 (Sec. 3.3)
};

// State-decay form (Sec. 3.4): slot states [B][H][S][d] float32.
struct DecayArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    const float* sk_in;
    const float* sv_in;
    float* sk_out;
    float* sv_out;
    const int* theta;       // [H][SP] start-mask thresholds (INT32_MAX for padded slots)
    const double* period;   // [H] clamped period T
    const double* rperiod;  // [H] 1 / T
    float* summ;            // [B*H][nseg-1] segment summaries, scanned in place into entering states
    // Sub-block schedule of the call, per distinct period u (heads map to it through gmap):
    // sub-blocks never cross a 16-token window of the sequence; glen[u][t] is the length of
    // the sub-block that starts at token t, gE[u][t][s] the gate product E of token t within
    // its sub-block and gB[u][t][s] = g_t[s] / E (0 for padded slots).
    const float* gE;
    const float* gB;
    const int* glen;
    const int* gmap;        // [H] head -> its schedule (heads with one period share one)
    int B, H, L, M, S;
    int nseg, seg_len;      // segments per sequence and their length (a multiple of 16 tokens)
    long long t0;
    float scale;
};

// Slot tiles per wave of the decay forward kernel for (d, padded S): 8 / (d / 16) tiles (the
// wave's K~ and V~ state then takes 64 VGPRs), at least 1, at most all of them, and at
// least 1/8 of them (so a workgroup has at most 8 waves).
constexpr int decay_slot_tiles_per_wave(int D, int SP)
{
    const int nst = SP / 16, want = 8 / (D / 16) > 0 ? 8 / (D / 16) : 1;
    const int lo = (nst + 7) / 8;
    return want < lo ? lo : (want > nst ? nst : want);
}
// Waves per workgroup of the decay forward kernel.
inline int decay_waves(int D, int SP) { return (SP / 16) / decay_slot_tiles_per_wave(D, SP); }

struct DecayStepArgs {
    const void* q;
    const void* k;
    const void* v;
    void* o;
    const int64_t* pos;
    float* sk;
    float* sv;
    const int* theta;
    const double* rperiod;
    int B, H, M, S;
    long long t0;
    float scale;
};

// Backward of the chunked operator (gradients of Alg. 2).  Every [B,H,L,d] tensor in the
// io dtype; states and state gradients float32 [B,H,2,M,d].
struct BwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const void* dO;
    const float* sk_in;    // forward's input states (nullable: zero)
    const float* sv_in;
    const float* gk_out;   // dLoss / d(final states) (nullable: zero)
    const float* gv_out;
    void* dq;
    void* dk;
    void* dv;
    float* gk_in;          // dLoss / d(input states) (nullable: not wanted)
    float* gv_in;
    const float* E32;      // [H][C+1][2MP]
    const void* EbarT;     // [H][2MP][C]  conj(rho^i)
    const void* ErevT;     // [H][2MP][C]  rho^{C-i}
    const void* Etab;      // [H][C][2MP]  rho^i
    const void* ABs;       // [SP][2MP]    scale * (A | B)
    const void* ABm;       // [2MP][SP]    (A | B) transposed
    const int* theta;      // [H][SP]
    const double* rperiod; // [H] 1 / T
    float* fsum;           // [B*H][nbk][2][2][MP][D] forward summaries of the blocks
    float* asum;           // [B*H][nbk][2][2][MP][D] adjoint summaries (blocks of segment 0 unused)
    int B, H, L, M;
    int nch, nseg, cps;    // chunks per sequence, segments, chunks per segment
    int nbk, cpb;          // summary blocks per sequence (nseg times a power of two), chunks per block
    long long t0;
    float scale;
};

// LDS bytes of the backward kernel for an element size (2: bf16, 4: float32): token tiles
// row-major and transposed, Gram / H tiles, readout weights, state operands, thresholds.
constexpr size_t bwd_lds_bytes(int esz, int D, int MP, int SP)
{
    const size_t C = kChunk, PAD = 4, LDQ = D + PAD, LDK = C + PAD, LDU = 2 * (size_t)MP + PAD;
    const size_t A = 4 * C * LDQ, Tt = 4 * (size_t)D * LDK, G = 2 * C * LDK;
    const size_t Bw = 4 * (size_t)MP * LDK > 2 * C * LDU ? 4 * (size_t)MP * LDK : 2 * C * LDU;
    const size_t Z = 2 * (size_t)D * LDU;
    return (A + Tt + G + Bw + Z) * (size_t)esz + (size_t)SP * 4;
}
constexpr size_t kBwdMaxLds = 160 * 1024;

// Whether a backward kernel exists for (bf16, D, MP, SP): bf16 with D in {32, 64},
// float32 with D = 32; MP <= 64, SP <= max(32, 2 MP) <= 128, within the LDS of a workgroup.
inline bool backward_supported(int bf16, int D, int MP, int SP)
{
    if (bf16 ? (D != 32 && D != 64) : D != 32) return false;
    if (MP != 16 && MP != 32 && MP != 64) return false;
    if (SP != 32 && SP != 64 && SP != 128) return false;
    if (SP > (2 * MP > 32 ? 2 * MP : 32)) return false;
    return bwd_lds_bytes(bf16 ? 2 : 4, D, MP, SP) <= kBwdMaxLds;
}

// Launchers (defined in the .hip translation units).  They return a HIP error.
hipError_t launch_tables(const TableArgs& a, int bf16, hipStream_t s);
hipError_t launch_fragtab(const FragTabArgs& a, hipStream_t s);
hipError_t launch_summary(const Plan& p, const FwdArgs& a, hipStream_t s);
hipError_t launch_scan(const Plan& p, const FwdArgs& a, hipStream_t s);
hipError_t launch_forward(const Plan& p, const FwdArgs& a, hipStream_t s);
hipError_t launch_state_copy(const float* src, float* dst, size_t n, hipStream_t s);
hipError_t launch_step(const Plan& p, const StepArgs& a, hipStream_t s);
hipError_t launch_decay_forward(int bf16_io, int D, int SP, const DecayArgs& a, hipStream_t s,
                                void* const* events);
hipError_t launch_decay_step(int bf16_io, int D, int SP, const DecayStepArgs& a, hipStream_t s);
// The sub-block schedules of a decay forward call: one per distinct period, shared by every
// batch row and every head of that period, and the head map.
struct GateArgs {
    float* gE;    // schedules ubase .. ubase + nu - 1: [L][SP] each
    float* gB;    // [L][SP] each
    int* glen;    // [L] each
    int* gmap;    // [H]; entries h0 .. h0 + nh - 1 written from map
    int L, SP, S, M, h0, nh, ubase, nu;
    long long t0;
    double rS;                                 // 1 / S
    double rT[kMaxHeadsPerTableLaunch];        // 1 / T of table ubase + u
    int map[kMaxHeadsPerTableLaunch];          // table of head h0 + i
};
hipError_t launch_decay_gates(const GateArgs& g, hipStream_t s);

// Backward passes: forward summaries of every segment, adjoint summaries (segments 1..),
// and the reverse walk.  events[0..2] (nullable) are recorded after each pass.
hipError_t launch_backward(int bf16, int D, int MP, int SP, const BwdArgs& a, hipStream_t s,
                           void* const* events);

// Whether a forward kernel exists for (bf16, D, MP, SP) and chunk length C.
bool forward_supported(int bf16, int D, int MP, int SP, int C);

// bla_forward on q, k, v and o with the element strides of FwdArgs: in_strides and
// out_strides are {batch, head, token} (nullable: contiguous [B, H, L, d]).  Each stride
// must be a multiple of 8 elements.  Used by the layer to read the projection output and
// write the head-merged output in place.
bla_status forward_strided(const bla_params* p, const double* T, const void* q, const void* k, const void* v,
                           const long long* in_strides, const float* state_k_in, const float* state_v_in, void* o,
                           const long long* out_strides, float* state_k_out, float* state_v_out, void* workspace,
                           size_t workspace_bytes, void* stream, void* const* events);
// Sequence units per workgroup of the bf16 pair kernel (0: the one-unit forward kernel runs).
int forward_units_per_wg(int bf16, int D, int MP, int SP);

}  // namespace bla
