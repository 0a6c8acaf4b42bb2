/*
 * bla.h -- C ABI of the MI355X (gfx950) library for the forward operator of
 * Blurry Window Attention (BLA).
 *
 * The operator (Sec. 3.1; Appendix C, Alg. 2).  Per batch row b and head h the
 * layer keeps complex mode states Z_k[m] = Kcos[m] + i Ksin[m] (d_k wide) and
 * Z_v[m] = Vcos[m] + i Vsin[m] (d_v wide) for m = 0..M-1.  With the period
 * T_h clamped to at least 2M-1 and w = 2 pi / T_h, each token at absolute
 * position p does, in order:
 *   1. rotate and add (Eq. recurrence):  Z[m] <- exp(i m w) Z[m] + x_t   (x = k or v)
 *   2. rebuild S blurry slots (Eq. compressed, coefficients of Eq. translated at
 *      the slot lags tau_s = s T_h / S):
 *        K~[s] = sum_m c_m (cos(m w tau_s) Kcos[m] + sin(m w tau_s) Ksin[m]),
 *        c_0 = 1/(2M-1), c_m = 2/(2M-1);  V~ likewise
 *   3. attend over the slots (Eq. output) with the start-of-sequence mask:
 *        z_s = scale <q_t, K~[s]> if p >= rint(tau_s) else -inf,
 *        o_t = sum_s softmax(z)_s V~[s].
 * The paper's own slot count is S = 2M-1; any S >= 1 is accepted and places the
 * slots on the grid tau_s = s T / S (at S = 2M-1 this is the paper's dilated grid).
 *
 * Anchored slots (phase_anchor = 1; Sec. 3.3, Eqs. permuted and compressed_simplified,
 * Alg. 1 and Alg. 3).  The paper's "efficient" form places the slots at fixed phases
 * instead of at lags behind the current token: slot s holds
 *        K~[s] = sum_{t' <= t} D_M(p' - tau_s) k_t'     (p' the absolute position of t')
 * with D_M the Dirichlet kernel of step 2's coefficients, and step 3 is unchanged.  The
 * state buffers hold the SAME mode state Z in both forms (the anchored slots are read
 * from it at the token's absolute phase, K~[s] = sum_m c_m Re(exp(-i m w (p - tau_s)) Z[m])),
 * so state_k / state_v mean the same thing and may be handed between the two forms.  The
 * two forms give the same outputs exactly when S = T_h is an integer (the paper's case
 * T = S = 2M-1), where the anchored slots are a permutation of the rotating ones.
 *
 * Conventions shared by every entry point:
 *   - All tensors are row-major and contiguous, in device memory, 16-byte aligned:
 *       q, k: [B, H, L, d_k]   v, o: [B, H, L, d_v]   (bla_step: L is absent)
 *       states: float32 [B, H, 2, M, d] -- plane 0 = cos accumulator, plane 1 = sin.
 *   - io_dtype selects float32 or bfloat16 for q, k, v, o; states are float32.
 *   - T is a HOST array of H periods (double).  Each is clamped to >= 2M-1, as the
 *     paper's algorithms do; NaN, infinite, non-positive or > 1e9 is an error.
 *   - Every device buffer is owned by the caller.  The operator's calls allocate no
 *     device memory: scratch space (tables, per-block partial states) lives in the
 *     caller's workspace, sized by bla_workspace_size / bla_step_workspace_size.  Two
 *     exceptions, both outside the operator's own kernels: the first bla_layer_forward
 *     on a device creates a hipBLASLt handle (hipBLASLt allocates its own memory), and
 *     bla_forward_noalloc's workspace is a fixed device array of the library's code
 *     object (allocated with the module, once per device).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = default stream).
 *     Argument errors are reported synchronously before anything is launched;
 *     launch failures are reported as BLA_ERR_HIP.  Buffers must stay valid until
 *     the stream has executed the call.  Calls that share a workspace race unless
 *     they are ordered on one stream.
 *   - Supported shapes: d_k == d_v in {32, 64, 128}; 1 <= M <= 128; 1 <= S <= 256
 *     and S <= max(32, 2 P(M)) where P(M) is M rounded up to 16, 32, 64 or 128 (so
 *     the paper's S = 2M-1 is always accepted); chunk in {0 (= 64), 16, 32, 64, 128}
 *     (Alg. 3's chunk length: the result is the same up to rounding, only the work
 *     split changes); chunks other than 64 need P(M) <= 64 and run on the one-unit
 *     kernels (128-token chunks with register spills: 64 is the fast default);
 *     float32 I/O also needs the kernel's LDS tiles to fit (d = 128 with M > 64 does
 *     not, nor float32 128-token chunks at d = 64).  Anything else returns
 *     BLA_ERR_UNSUPPORTED; bla_supported() answers without launching.
 */
#ifndef BLA_H
#define BLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BLA_OK = 0,
    BLA_ERR_INVALID_ARG = 1, /* a null/misaligned pointer, a negative size, a bad period */
    BLA_ERR_UNSUPPORTED = 2, /* a valid shape the library has no kernel for           */
    BLA_ERR_WORKSPACE = 3,   /* workspace pointer null or smaller than required       */
    BLA_ERR_HIP = 4          /* the HIP runtime reported an error while launching     */
} bla_status;

typedef enum { BLA_F32 = 0, BLA_BF16 = 1 } bla_dtype;

typedef struct {
    int32_t B, H, L;     /* batch rows, heads, tokens in this call (L >= 0)              */
    int32_t d_k, d_v;    /* head widths of keys/queries and of values                    */
    int32_t M;           /* Fourier modes (Sec. 3.1), >= 1                               */
    int32_t S;           /* blurry slots, >= 1 (the paper's value is 2M-1)               */
    int32_t chunk;       /* tokens per chunk of the parallel form (16, 32, 64, 128);
                            0 = default (64)                                             */
    int64_t t0;          /* absolute position of token 0 (start mask only), >= 0         */
    float scale;         /* softmax scale; 0 selects 1/sqrt(d_k) (Eq. output)            */
    int32_t io_dtype;    /* bla_dtype of q, k, v, o                                      */
    int32_t phase_anchor; /* 0: slots at lags behind the current token (the operator above,
                            Sec. 3.1, Alg. 2); 1: slots anchored at absolute phase 0 (Sec. 3.3,
                            Alg. 1 / Alg. 3); any other value is BLA_ERR_INVALID_ARG        */
    int32_t reuse_tables; /* 0: build the phase and slot tables in the workspace (every call).
                            1: reuse them if this workspace already holds them.  Alg. 1 and
                            Alg. 3 take the interpolation matrices A, B as precomputed inputs;
                            with this flag the tables of an earlier call are kept.  The library
                            records, per device and workspace address, the key of the tables it
                            last built there (entry point, every field of *p that the tables
                            depend on, and the periods T); a call with reuse_tables = 1 skips
                            the table kernel only when that record matches, and builds the
                            tables otherwise.  The caller guarantees that nothing else has
                            written the workspace since that call (a workspace freed and
                            allocated again at the same address holds stale bytes: pass 0
                            then).  Any value other than 0 or 1 is BLA_ERR_INVALID_ARG.     */
} bla_params;

/* Human-readable name of a status code (static string, never NULL). */
const char* bla_status_string(bla_status s);

/* BLA_OK if the shape in *p has a kernel in the library, else the error it would get. */
bla_status bla_supported(const bla_params* p);

/*
 * Host-side float64 slot tables of one head (Sec. 3.1: the interpolation coefficients of
 * Eq. translated evaluated at the slot lags tau_s = s T / S, Alg. 2's dilated time grid):
 *   A[s*M + m] = c_m cos(2 pi m s / S),  B[s*M + m] = c_m sin(2 pi m s / S),
 *   c_0 = 1/(2M-1), c_m = 2/(2M-1) for m >= 1,
 *   theta[s] = rint(s T / S)  (round half to even), the first position at which slot s
 *   is visible (the start mask of Eq. output),
 * with T clamped to at least 2M-1 as the kernels do.  A and B are [S][M] row-major,
 * caller-owned host arrays; theta has S entries.  BLA_ERR_INVALID_ARG for M < 1, S < 1,
 * a null pointer, or T not finite and positive.  The device tables of bla_forward and
 * bla_step follow the same formulas (rounded to float32 / the operand type).
 */
bla_status bla_interp_tables(int32_t M, int32_t S, double T, double* A, double* B, int32_t* theta);

/*
 * Bytes of device workspace bla_forward needs for *p on the current device
 * (0 if *p is invalid or unsupported).  The value depends on B, H, L, d, M, S
 * and the device's compute-unit count, not on the data.
 */
size_t bla_workspace_size(const bla_params* p);

/*
 * Chunked-parallel forward over L tokens (Sec. 3.2's chunk mode; the operator is
 * Alg. 2's recurrence).  Writes o [B,H,L,d_v].  state_k_in / state_v_in
 * [B,H,2,M,d] give the states before token 0 (NULL = zero, a fresh sequence);
 * state_k_out / state_v_out receive the states after token L-1 (NULL = not
 * wanted).  The outputs must not alias the inputs.  L = 0 copies the input
 * states (or zeros) to the outputs.
 */
bla_status bla_forward(const bla_params* p, const double* T, const void* q, const void* k,
                       const void* v, const float* state_k_in, const float* state_v_in, void* o,
                       float* state_k_out, float* state_v_out, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * bla_forward with phase timing, for measurement tools: events[0..4] are
 * hipEvent_t handles created by the caller (any entry may be NULL; the array may
 * be NULL) and are recorded on `stream` before the table kernel, after it, after
 * the block-summary kernel, after the summary scan, and after the chunked forward
 * kernel (a phase that does not run for this shape still gets its event).  The
 * computation and every other convention are exactly those of bla_forward;
 * BLA_ERR_HIP is also returned if an event cannot be recorded.
 */
bla_status bla_forward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                             const void* v, const float* state_k_in, const float* state_v_in, void* o,
                             float* state_k_out, float* state_v_out, void* workspace,
                             size_t workspace_bytes, void* stream, void* const* events);

/*
 * bla_forward for callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops and harnesses that forbid hipMalloc).  The workspace is a fixed array inside
 * the library, BLA_NOALLOC_SCRATCH_BYTES bytes per device (each device the library runs on
 * holds its own copy until the process ends; its address is taken once per device, on the
 * first call there).  The call allocates nothing: no hipMalloc, hipFree or allocating library
 * routine.  Arguments and results are exactly those of bla_forward without the workspace
 * arguments; a shape whose bla_workspace_size exceeds BLA_NOALLOC_SCRATCH_BYTES returns
 * BLA_ERR_WORKSPACE before anything is launched.  Every call on a device shares that
 * device's array, which keeps the last call's contents (the forward writes every byte it
 * reads, so nothing needs clearing): calls that overlap in time on one device race, so
 * order them on one stream.  reuse_tables = 1 keeps the tables of the previous call
 * through this entry point, under the same rules as for a caller's workspace.
 */
#define BLA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
bla_status bla_forward_noalloc(const bla_params* p, const double* T, const void* q, const void* k,
                               const void* v, const float* state_k_in, const float* state_v_in, void* o,
                               float* state_k_out, float* state_v_out, void* stream);

/* Bytes of device workspace bla_step needs for *p (L is ignored). */
size_t bla_step_workspace_size(const bla_params* p);

/*
 * One recurrent decode step (one iteration of Alg. 2's loop) for every (b,h):
 * q, k [B,H,d_k], v, o [B,H,d_v].  The token of row b sits at absolute position
 * pos[b] (device int64 [B]; NULL = p->t0 for every row); the start mask uses it.
 * state_k / state_v [B,H,2,M,d] hold the states before the token and are updated
 * in place.  p->L is ignored.
 */
bla_status bla_step(const bla_params* p, const double* T, const void* q, const void* k,
                    const void* v, const int64_t* pos, float* state_k, float* state_v, void* o,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * State-decay form (Sec. 3.4).  Anchored slots (Sec. 3.3) whose previous state is
 * multiplied by 1 - D before each write, the gated recurrence the paper relates to GSA:
 *        K~[s] <- (1 - g[s]) K~[s] + g[s] k_t,   V~[s] likewise,
 *        g[s] = D_M(p - tau_s) = sum_m c_m cos(m w (p - tau_s))
 * at the token's absolute position p, followed by step 3 of the operator (masked slot
 * softmax and readout) on the decayed slots.  At T = S = 2M-1 a write replaces exactly the
 * slot of the current residue class, so the form is sliding-window attention with window
 * 2M-1.  The decay is diagonal in slots, so the state is the slot state itself:
 *        slot_k, slot_v: float32 [B, H, S, d] (row s of head (b,h) is slot s).
 * p->phase_anchor is ignored (the form is anchored by definition).  Shapes, dtypes, T,
 * alignment, ownership, streams and errors follow the conventions above (p->chunk is
 * accepted as for bla_forward; the kernels work in sub-blocks of at most 16 tokens that never
 * cross a 16-token window of the sequence and end early where a slot's product of decay
 * factors would fall below 2^-100).
 */

/* Bytes of device workspace bla_decay_forward and bla_decay_step need for *p.  For a forward
 * call it grows with L: the segment summaries plus a sub-block schedule of about
 * 8 * P(S) + 4 bytes per token and head (P(S): S padded as for bla_forward). */
size_t bla_decay_workspace_size(const bla_params* p);

/*
 * Decay-form forward over L tokens: o [B,H,L,d_v]; slot_k_in / slot_v_in [B,H,S,d] are the
 * slot states before token 0 (NULL = zero), slot_k_out / slot_v_out receive the states after
 * token L-1 (NULL = not wanted; they must not alias the inputs).  L = 0 copies the input
 * states (or zeros) to the outputs.
 */
bla_status bla_decay_forward(const bla_params* p, const double* T, const void* q, const void* k,
                             const void* v, const float* slot_k_in, const float* slot_v_in, void* o,
                             float* slot_k_out, float* slot_v_out, void* workspace,
                             size_t workspace_bytes, void* stream);

/*
 * bla_decay_forward with phase timing, for measurement tools: events[0..4] are hipEvent_t
 * handles created by the caller (any entry, or the array, may be NULL), recorded on
 * `stream` before the table kernel, after it, after the segment-summary pass, after the
 * scan of the summaries, and after the forward pass (a pass that does not run for this
 * shape still gets its event).  Everything else is exactly bla_decay_forward;
 * BLA_ERR_HIP is also returned if an event cannot be recorded.
 */
bla_status bla_decay_forward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                                   const void* v, const float* slot_k_in, const float* slot_v_in, void* o,
                                   float* slot_k_out, float* slot_v_out, void* workspace,
                                   size_t workspace_bytes, void* stream, void* const* events);

/*
 * One decay-form decode step for every (b,h): q, k [B,H,d_k], v, o [B,H,d_v], the token of
 * row b at absolute position pos[b] (device int64 [B]; NULL = p->t0); slot_k / slot_v
 * [B,H,S,d] are updated in place.
 */
bla_status bla_decay_step(const bla_params* p, const double* T, const void* q, const void* k,
                          const void* v, const int64_t* pos, float* slot_k, float* slot_v, void* o,
                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * Backward pass (gradients of the operator above, Alg. 2 with phase_anchor = 0).  The paper
 * trains every model through this operator (Sec. 4); the gradients are those of the loss
 * whose partial derivatives are dO = dLoss/dO [B,H,L,d_v] and dstate_k_out / dstate_v_out =
 * dLoss/d(final states) [B,H,2,M,d] (NULL = zero).  q, k, v, state_k_in, state_v_in are the
 * forward call's inputs (states NULL = zero); the forward outputs are not needed (the
 * states are rebuilt chunk by chunk).  Writes dq, dk [B,H,L,d_k] and dv [B,H,L,d_v] in the
 * io dtype, and dLoss/d(input states) into dstate_k_in / dstate_v_in [B,H,2,M,d] float32
 * (NULL = not wanted; they must not alias the other state arguments).  L = 0 copies the
 * final-state gradients (or zeros) to them.
 * Supported: phase_anchor = 0; chunk 0 or 64; bfloat16 with d in {32, 64} or float32 with d = 32;
 * M <= 64 (float32: M <= 32) and S <= max(32, 2 P(M)) <= 128; anything else BLA_ERR_UNSUPPORTED.
 * Every other convention (alignment, T, ownership, streams, errors) as for bla_forward.
 */
size_t bla_backward_workspace_size(const bla_params* p);
bla_status bla_backward(const bla_params* p, const double* T, const void* q, const void* k, const void* v,
                        const void* dO, const float* state_k_in, const float* state_v_in,
                        const float* dstate_k_out, const float* dstate_v_out, void* dq, void* dk, void* dv,
                        float* dstate_k_in, float* dstate_v_in, void* workspace, size_t workspace_bytes,
                        void* stream);

/*
 * bla_backward with phase timing, for measurement tools: events[0..4] (hipEvent_t, created by
 * the caller; any entry or the array may be NULL) are recorded before the table kernel, after
 * it, after the forward-summary pass, after the adjoint-summary pass and after the reverse walk.
 */
bla_status bla_backward_timed(const bla_params* p, const double* T, const void* q, const void* k,
                              const void* v, const void* dO, const float* state_k_in, const float* state_v_in,
                              const float* dstate_k_out, const float* dstate_v_out, void* dq, void* dk,
                              void* dv, float* dstate_k_in, float* dstate_v_in, void* workspace,
                              size_t workspace_bytes, void* stream, void* const* events);

/*
 * A whole BLA layer on hidden states (bfloat16 only).  The queries, keys and values are
 * linear projections of the hidden states (the attention layer of Sec. 2.1 whose softmax BLA
 * replaces), the H heads run the operator (bla_forward, either form by p->phase_anchor), and
 * an output projection mixes the heads back into the model width D = H * d_k:
 *     [q | k | v] = x W_qkv,   o = BLA(q, k, v),   y = o W_o
 * with x, y [B, L, D] row-major, W_qkv [D, 3D] (columns h d_k .. h d_k + d_k - 1 of block 0,
 * 1, 2 are head h's query, key and value projections), W_o [D, D] (row h d_k + e takes element
 * e of head h's output), all bf16; the products accumulate in float32 (hipBLASLt) and q, k, v
 * and o are rounded to bf16 between the steps.  p describes the operator (p->d_k = p->d_v is
 * the head width, p->L the tokens); states as for bla_forward.  The operator reads q, k, v in
 * place from the projection output [B, L, 3, H, d_k] and writes o in place as [B, L, H, d_k],
 * the output projection's input.  The workspace holds those two tensors, the operator's
 * workspace and 32 MB of GEMM scratch.  The first call on
 * a device creates a hipBLASLt handle that lives until the process ends.  Errors as for
 * bla_forward; a failing GEMM is BLA_ERR_HIP.
 */
size_t bla_layer_workspace_size(const bla_params* p);
bla_status bla_layer_forward(const bla_params* p, const double* T, const void* x, const void* w_qkv,
                             const void* w_o, const float* state_k_in, const float* state_v_in, void* y,
                             float* state_k_out, float* state_v_out, void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * bla_layer_forward with phase timing: events[0..3] (hipEvent_t or NULL) are recorded before
 * the QKV projection, after it, after the operator and after the output projection.
 */
bla_status bla_layer_forward_timed(const bla_params* p, const double* T, const void* x, const void* w_qkv,
                                   const void* w_o, const float* state_k_in, const float* state_v_in, void* y,
                                   float* state_k_out, float* state_v_out, void* workspace,
                                   size_t workspace_bytes, void* stream, void* const* events);

#ifdef __cplusplus
}
#endif

#endif /* BLA_H */
