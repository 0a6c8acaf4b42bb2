/*
 * Float64 CPU oracle for the forward operator of Blurry Window Attention (BLA).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or calls
 * this file: only the tests, the smoke check and the benchmark's CPU baseline
 * do.  It shares no code, header, table or constant with the HIP library.
 *
 * What it computes (per batch row b and head h, all in double precision):
 *
 *   period     T  <- max(T_h, 2M-1)                   (Alg. 1 / Alg. 3, "clamp period")
 *   frequency  w  = 2*pi / T                          (Sec. 3.1, text after Eq. compressed)
 *   Dirichlet coefficients c_0 = 1/(2M-1), c_m = 2/(2M-1) for 1 <= m < M
 *                                                     (Sec. 3.1 Eq. dirichlet)
 *   slot lags  tau_s = s*T/S for s in [0,S)  -- the dilated time grid of Alg. 1/2
 *              with 2M-1 replaced by the slot count S (S = 2M-1 is the paper's case)
 *   interpolation matrices (Sec. 3.1 Eq. translated, evaluated at Delta t = tau_s):
 *              A[s][m] = c_m cos(m w tau_s),   B[s][m] = c_m sin(m w tau_s)
 *   start-mask thresholds theta_s = rint(tau_s)       (Alg. 2 "dilated time grid")
 *
 *   for every token t (absolute position p = t0 + t), Alg. 2 loop body:
 *     state update (Sec. 3.1 Eq. recurrence):
 *        Kcos[m] <- cos(m w) Kcos[m] - sin(m w) Ksin[m] + k_t
 *        Ksin[m] <- sin(m w) Kcos[m] + cos(m w) Ksin[m]          (same for V)
 *     blurry slots (Sec. 3.1 Eq. compressed):  Kt[s] = sum_m A[s][m] Kcos[m] + B[s][m] Ksin[m]
 *     output (Sec. 3.1 Eq. output):
 *        z_s = scale * <q_t, Kt[s]>  if p >= theta_s else -inf
 *        o_t = sum_s softmax(z)_s Vt[s]
 *
 * The "factored" readout computes the same o_t with the sums over modes and
 * slots regrouped (z_s = scale * sum_m A[s][m] <q,Kcos[m]> + B[s][m] <q,Ksin[m]>,
 * o = sum_m (sum_s p_s A[s][m]) Vcos[m] + (sum_s p_s B[s][m]) Vsin[m]); it only
 * changes the rounding order and exists so that the long workloads finish in
 * seconds.  The "literal" readout materialises the slots exactly as written.
 *
 * Layouts: q,k [Bn][H][L][dk], v,o [Bn][H][L][dv]; states [Bn][H][2][M][d] with
 * plane 0 = cos accumulator and plane 1 = sin accumulator.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_PI 3.14159265358979323846264338327950288

static double clamp_period(double T, int M)
{
    double tmin = 2.0 * M - 1.0;
    return T < tmin ? tmin : T;
}

/* Interpolation matrices and mask thresholds for one head (Sec. 3.1 Eq. translated). */
void bla_oracle_interp(int M, int S, double T_in, double* A, double* Bm, int64_t* theta)
{
    double T = clamp_period(T_in, M);
    double w = 2.0 * ORACLE_PI / T;
    for (int s = 0; s < S; ++s) {
        double tau = (double)s * T / (double)S;
        for (int m = 0; m < M; ++m) {
            double c = (m == 0 ? 1.0 : 2.0) / (2.0 * M - 1.0);
            A[(size_t)s * M + m] = c * cos(m * w * tau);
            Bm[(size_t)s * M + m] = c * sin(m * w * tau);
        }
        if (theta) theta[s] = (int64_t)rint(tau);
    }
}

/* One (b,h) sequence, Alg. 2 token loop.  Work buffers are caller-provided. */
static void run_sequence(int L, int dk, int dv, int M, int S, double T_in, int64_t t0,
                         double scale, const double* q, const double* k, const double* v,
                         double* Kc, double* Ks, double* Vc, double* Vs, double* o,
                         int literal, double* work)
{
    double T = clamp_period(T_in, M);
    double w = 2.0 * ORACLE_PI / T;
    double* A = work;                       /* S*M */
    double* Bm = A + (size_t)S * M;         /* S*M */
    int64_t* theta = (int64_t*)(Bm + (size_t)S * M); /* S */
    double* rc = (double*)(theta + S);      /* M */
    double* rs = rc + M;                    /* M */
    double* z = rs + M;                     /* S */
    double* Kt = z + S;                     /* S*dk (literal) */
    double* Vt = Kt + (size_t)S * dk;       /* S*dv (literal) */
    double* uc = Vt + (size_t)S * dv;       /* M */
    double* us = uc + M;                    /* M */
    double* am = us + M;                    /* M */
    double* bm = am + M;                    /* M */

    bla_oracle_interp(M, S, T, A, Bm, theta);
    for (int m = 0; m < M; ++m) {
        rc[m] = cos(m * w);
        rs[m] = sin(m * w);
    }

    for (int t = 0; t < L; ++t) {
        const double* qt = q + (size_t)t * dk;
        const double* kt = k + (size_t)t * dk;
        const double* vt = v + (size_t)t * dv;
        double* ot = o + (size_t)t * dv;
        int64_t pos = t0 + t;

        /* Eq. recurrence for keys and values. */
        for (int m = 0; m < M; ++m) {
            for (int d = 0; d < dk; ++d) {
                double c = Kc[(size_t)m * dk + d], s = Ks[(size_t)m * dk + d];
                Kc[(size_t)m * dk + d] = rc[m] * c - rs[m] * s + kt[d];
                Ks[(size_t)m * dk + d] = rs[m] * c + rc[m] * s;
            }
            for (int d = 0; d < dv; ++d) {
                double c = Vc[(size_t)m * dv + d], s = Vs[(size_t)m * dv + d];
                Vc[(size_t)m * dv + d] = rc[m] * c - rs[m] * s + vt[d];
                Vs[(size_t)m * dv + d] = rs[m] * c + rc[m] * s;
            }
        }

        /* Scores with the start-of-sequence mask. */
        if (literal) {
            for (int s = 0; s < S; ++s) {
                for (int d = 0; d < dk; ++d) {
                    double acc = 0.0;
                    for (int m = 0; m < M; ++m)
                        acc += A[(size_t)s * M + m] * Kc[(size_t)m * dk + d] +
                               Bm[(size_t)s * M + m] * Ks[(size_t)m * dk + d];
                    Kt[(size_t)s * dk + d] = acc;
                }
                for (int d = 0; d < dv; ++d) {
                    double acc = 0.0;
                    for (int m = 0; m < M; ++m)
                        acc += A[(size_t)s * M + m] * Vc[(size_t)m * dv + d] +
                               Bm[(size_t)s * M + m] * Vs[(size_t)m * dv + d];
                    Vt[(size_t)s * dv + d] = acc;
                }
                double dot = 0.0;
                for (int d = 0; d < dk; ++d) dot += qt[d] * Kt[(size_t)s * dk + d];
                z[s] = scale * dot;
            }
        } else {
            for (int m = 0; m < M; ++m) {
                double a = 0.0, b = 0.0;
                for (int d = 0; d < dk; ++d) {
                    a += qt[d] * Kc[(size_t)m * dk + d];
                    b += qt[d] * Ks[(size_t)m * dk + d];
                }
                uc[m] = a;
                us[m] = b;
            }
            for (int s = 0; s < S; ++s) {
                double acc = 0.0;
                for (int m = 0; m < M; ++m)
                    acc += A[(size_t)s * M + m] * uc[m] + Bm[(size_t)s * M + m] * us[m];
                z[s] = scale * acc;
            }
        }

        /* Softmax over the slots; masked slots get probability zero. */
        double zmax = -INFINITY;
        for (int s = 0; s < S; ++s) {
            if (pos < theta[s]) z[s] = -INFINITY;
            if (z[s] > zmax) zmax = z[s];
        }
        double den = 0.0;
        for (int s = 0; s < S; ++s) {
            z[s] = (z[s] == -INFINITY) ? 0.0 : exp(z[s] - zmax);
            den += z[s];
        }
        for (int s = 0; s < S; ++s) z[s] /= den;

        /* Readout. */
        if (literal) {
            for (int d = 0; d < dv; ++d) {
                double acc = 0.0;
                for (int s = 0; s < S; ++s) acc += z[s] * Vt[(size_t)s * dv + d];
                ot[d] = acc;
            }
        } else {
            for (int m = 0; m < M; ++m) {
                double a = 0.0, b = 0.0;
                for (int s = 0; s < S; ++s) {
                    a += z[s] * A[(size_t)s * M + m];
                    b += z[s] * Bm[(size_t)s * M + m];
                }
                am[m] = a;
                bm[m] = b;
            }
            for (int d = 0; d < dv; ++d) {
                double acc = 0.0;
                for (int m = 0; m < M; ++m)
                    acc += am[m] * Vc[(size_t)m * dv + d] + bm[m] * Vs[(size_t)m * dv + d];
                ot[d] = acc;
            }
        }
    }
}

/*
 * Forward over Bn*H independent sequences.  state inputs may be NULL (zeros);
 * state outputs may be NULL.  Returns 0 on success, -1 on bad arguments or
 * allocation failure.  nthreads <= 0 means "OpenMP default".
 */
int bla_oracle_forward(int Bn, int H, int L, int dk, int dv, int M, int S, const double* T,
                       int64_t t0, double scale, const double* q, const double* k,
                       const double* v, const double* sk_in, const double* sv_in, double* o,
                       double* sk_out, double* sv_out, int literal, int nthreads)
{
    if (Bn < 0 || H < 0 || L < 0 || dk <= 0 || dv <= 0 || M <= 0 || S <= 0 || t0 < 0) return -1;
    size_t nseq = (size_t)Bn * H;
    size_t wlen = 2 * (size_t)S * M + (size_t)S + 2 * (size_t)M + (size_t)S +
                  (size_t)S * (dk + dv) + 4 * (size_t)M;
    size_t skl = 2 * (size_t)M * dk, svl = 2 * (size_t)M * dv;
    int err = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel
    {
        double* work = (double*)malloc(wlen * sizeof(double));
        double* st = (double*)malloc((skl + svl) * sizeof(double));
        if (!work || !st) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (long long i = 0; i < (long long)nseq; ++i) {
            if (!work || !st) continue;
            int h = (int)(i % H);
            double* Kc = st;
            double* Ks = st + (size_t)M * dk;
            double* Vc = st + skl;
            double* Vs = st + skl + (size_t)M * dv;
            if (sk_in) memcpy(st, sk_in + i * skl, skl * sizeof(double));
            else memset(st, 0, skl * sizeof(double));
            if (sv_in) memcpy(st + skl, sv_in + i * svl, svl * sizeof(double));
            else memset(st + skl, 0, svl * sizeof(double));
            run_sequence(L, dk, dv, M, S, T[h], t0, scale, q + i * (size_t)L * dk,
                         k + i * (size_t)L * dk, v + i * (size_t)L * dv, Kc, Ks, Vc, Vs,
                         o + i * (size_t)L * dv, literal, work);
            if (sk_out) memcpy(sk_out + i * skl, st, skl * sizeof(double));
            if (sv_out) memcpy(sv_out + i * svl, st + skl, svl * sizeof(double));
        }
        free(work);
        free(st);
    }
    return err ? -1 : 0;
}

/*
 * Single-token recurrent decode: one iteration of the Alg. 2 loop for every
 * (b,h), at absolute position pos[b], updating the states in place.
 */
int bla_oracle_step(int Bn, int H, int dk, int dv, int M, int S, const double* T,
                    const int64_t* pos, double scale, const double* q, const double* k,
                    const double* v, double* sk, double* sv, double* o, int nthreads)
{
    if (Bn < 0 || H < 0) return -1;
    for (int b = 0; b < Bn; ++b) {
        size_t off = (size_t)b * H;
        int rc = bla_oracle_forward(1, H, 1, dk, dv, M, S, T, pos[b], scale, q + off * dk,
                                    k + off * dk, v + off * dv, sk + off * 2 * M * dk,
                                    sv + off * 2 * M * dv, o + off * dv, sk + off * 2 * M * dk,
                                    sv + off * 2 * M * dv, 0, nthreads);
        if (rc) return rc;
    }
    return 0;
}

/*
 * Absolute-phase ("efficient") form of Sec. 3.3 (Eqs. permuted and
 * compressed_simplified; Alg. 1 recurrent, Alg. 3 chunked).  The slots are anchored
 * at phase 0 instead of at the current token, so the state is a plain cumulative sum
 * over slot vectors and needs no rotation.  Per token at absolute position p:
 *
 *   interpolation weights (Eq. compressed_simplified, the translated Dirichlet kernel
 *   evaluated at p):   g[s] = sum_m cos(m w p) A[s][m] + sin(m w p) B[s][m]
 *   slot states (Eq. permuted, accumulated):   Kt[s] += g[s] k_t,  Vt[s] += g[s] v_t
 *   output:   z_s = scale <q_t, Kt[s]> if p >= theta_s else -inf,
 *             o_t = sum_s softmax(z)_s Vt[s]
 *
 * With decay (Sec. 3.4, the GSA-style gated update with gate 1 - D): the previous
 * slot state is multiplied by (1 - g[s]) before the write,
 *             Kt[s] = (1 - g[s]) Kt[s] + g[s] k_t,  Vt[s] likewise,
 * which at T = S = 2M-1 replaces exactly the slot of the current residue class
 * (a ring buffer of the last 2M-1 tokens: sliding-window attention).
 *
 * m w p is reduced as w * fmod(m p, T): m p is an exact integer in double and fmod is
 * exact, so long positions lose no phase accuracy.  States are the slot states
 * [Bn][H][S][d] of Alg. 1 (K_prev, V_prev), not mode states.  Same argument rules
 * and return codes as bla_oracle_forward.
 */
static void run_sequence_anchored(int L, int dk, int dv, int M, int S, double T_in,
                                  int64_t t0, double scale, const double* q, const double* k,
                                  const double* v, double* Kt, double* Vt, double* o,
                                  int decay, double* work)
{
    double T = clamp_period(T_in, M);
    double w = 2.0 * ORACLE_PI / T;
    double* A = work;                              /* S*M */
    double* Bm = A + (size_t)S * M;                /* S*M */
    int64_t* theta = (int64_t*)(Bm + (size_t)S * M); /* S */
    double* cm = (double*)(theta + S);             /* M */
    double* sm = cm + M;                           /* M */
    double* g = sm + M;                            /* S */
    double* z = g + S;                             /* S */

    bla_oracle_interp(M, S, T, A, Bm, theta);
    for (int t = 0; t < L; ++t) {
        const double* qt = q + (size_t)t * dk;
        const double* kt = k + (size_t)t * dk;
        const double* vt = v + (size_t)t * dv;
        double* ot = o + (size_t)t * dv;
        int64_t pos = t0 + t;

        for (int m = 0; m < M; ++m) {
            double ph = w * fmod((double)m * (double)pos, T);
            cm[m] = cos(ph);
            sm[m] = sin(ph);
        }
        for (int s = 0; s < S; ++s) {
            double acc = 0.0;
            for (int m = 0; m < M; ++m)
                acc += cm[m] * A[(size_t)s * M + m] + sm[m] * Bm[(size_t)s * M + m];
            g[s] = acc;
        }
        for (int s = 0; s < S; ++s) {
            double keep = decay ? 1.0 - g[s] : 1.0;
            for (int d = 0; d < dk; ++d)
                Kt[(size_t)s * dk + d] = keep * Kt[(size_t)s * dk + d] + g[s] * kt[d];
            for (int d = 0; d < dv; ++d)
                Vt[(size_t)s * dv + d] = keep * Vt[(size_t)s * dv + d] + g[s] * vt[d];
        }

        double zmax = -INFINITY;
        for (int s = 0; s < S; ++s) {
            double dot = 0.0;
            for (int d = 0; d < dk; ++d) dot += qt[d] * Kt[(size_t)s * dk + d];
            z[s] = pos < theta[s] ? -INFINITY : scale * dot;
            if (z[s] > zmax) zmax = z[s];
        }
        double den = 0.0;
        for (int s = 0; s < S; ++s) {
            z[s] = (z[s] == -INFINITY) ? 0.0 : exp(z[s] - zmax);
            den += z[s];
        }
        for (int d = 0; d < dv; ++d) {
            double acc = 0.0;
            for (int s = 0; s < S; ++s) acc += z[s] * Vt[(size_t)s * dv + d];
            ot[d] = acc / den;
        }
    }
}

/* decay = 0: Alg. 1 (Sec. 3.3); decay = 1: with the state decay of Sec. 3.4. */
int bla_oracle_forward_anchored(int Bn, int H, int L, int dk, int dv, int M, int S,
                                const double* T, int64_t t0, double scale, const double* q,
                                const double* k, const double* v, const double* kt_in,
                                const double* vt_in, double* o, double* kt_out,
                                double* vt_out, int decay, int nthreads)
{
    if (Bn < 0 || H < 0 || L < 0 || dk <= 0 || dv <= 0 || M <= 0 || S <= 0 || t0 < 0) return -1;
    size_t nseq = (size_t)Bn * H;
    size_t wlen = 2 * (size_t)S * M + (size_t)S + 2 * (size_t)M + 2 * (size_t)S;
    size_t skl = (size_t)S * dk, svl = (size_t)S * dv;
    int err = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel
    {
        double* work = (double*)malloc(wlen * sizeof(double));
        double* st = (double*)malloc((skl + svl) * sizeof(double));
        if (!work || !st) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (long long i = 0; i < (long long)nseq; ++i) {
            if (!work || !st) continue;
            int h = (int)(i % H);
            if (kt_in) memcpy(st, kt_in + i * skl, skl * sizeof(double));
            else memset(st, 0, skl * sizeof(double));
            if (vt_in) memcpy(st + skl, vt_in + i * svl, svl * sizeof(double));
            else memset(st + skl, 0, svl * sizeof(double));
            run_sequence_anchored(L, dk, dv, M, S, T[h], t0, scale, q + i * (size_t)L * dk,
                                  k + i * (size_t)L * dk, v + i * (size_t)L * dv, st, st + skl,
                                  o + i * (size_t)L * dv, decay, work);
            if (kt_out) memcpy(kt_out + i * skl, st, skl * sizeof(double));
            if (vt_out) memcpy(vt_out + i * svl, st + skl, svl * sizeof(double));
        }
        free(work);
        free(st);
    }
    return err ? -1 : 0;
}

/*
 * Gradients of Alg. 2 (reverse-mode differentiation of the token loop; the paper trains
 * every model of Sec. 4 through this operator but states no backward pass, so this is the
 * chain rule applied to the forward definition above, step by step in reverse).
 *
 * Given dO = dLoss/dO and dZk_out, dZv_out = dLoss/d(final states) (zero if absent), for
 * t = L-1 down to 0, with the states after token t's update (stored by a forward pass) and
 * the adjoint gK, gV = dLoss/d(state after token t):
 *   slots:        Kt[s] = sum_m A[s][m] Kcos[m] + B[s][m] Ksin[m],  Vt likewise
 *   softmax:      p = softmax(z) with z_s = scale <q_t, Kt[s]> (masked slots: p_s = 0)
 *   readout:      dp_s = <dO_t, Vt[s]>,   dVt[s] = p_s dO_t
 *   softmax grad: dz_s = p_s (dp_s - sum_s' p_s' dp_s')
 *   scores:       dq_t = scale sum_s dz_s Kt[s],   dKt[s] = scale dz_s q_t
 *   slot grads into the adjoint:  gKcos[m] += sum_s A[s][m] dKt[s],  gKsin[m] += sum_s B[s][m] dKt[s]
 *                                 (gV from dVt likewise)
 *   recurrence:   k_t was added to every cos row, so dk_t = sum_m gKcos[m] (dv_t likewise);
 *                 the rotation (c, s) = (cos m w, sin m w) is orthogonal, so the adjoint of the
 *                 state before the token is  gcos' = c gcos + s gsin,  gsin' = -s gcos + c gsin.
 * After t = 0 the adjoint is dLoss/d(state_in).
 */
static void run_sequence_backward(int L, int dk, int dv, int M, int S, double T_in, int64_t t0,
                                  double scale, const double* q, const double* k, const double* v,
                                  const double* dO, const double* sk_in, const double* sv_in,
                                  double* gK, double* gV, double* dq, double* dkk, double* dvv,
                                  double* hist, double* work)
{
    double T = clamp_period(T_in, M);
    double w = 2.0 * ORACLE_PI / T;
    size_t skl = 2 * (size_t)M * dk, svl = 2 * (size_t)M * dv;
    double* A = work;                        /* S*M */
    double* Bm = A + (size_t)S * M;          /* S*M */
    int64_t* theta = (int64_t*)(Bm + (size_t)S * M); /* S */
    double* rc = (double*)(theta + S);       /* M */
    double* rs = rc + M;                     /* M */
    double* p = rs + M;                      /* S */
    double* dz = p + S;                      /* S */
    double* Kt = dz + S;                     /* S*dk */
    double* Vt = Kt + (size_t)S * dk;        /* S*dv */

    bla_oracle_interp(M, S, T, A, Bm, theta);
    for (int m = 0; m < M; ++m) {
        rc[m] = cos(m * w);
        rs[m] = sin(m * w);
    }

    /* forward pass: hist[t] = (Kcos, Ksin, Vcos, Vsin) after token t's update */
    for (int t = 0; t < L; ++t) {
        const double* prev = t ? hist + (size_t)(t - 1) * (skl + svl) : NULL;
        double* cur = hist + (size_t)t * (skl + svl);
        for (int m = 0; m < M; ++m) {
            for (int d = 0; d < dk; ++d) {
                double c = prev ? prev[(size_t)m * dk + d] : (sk_in ? sk_in[(size_t)m * dk + d] : 0.0);
                double s = prev ? prev[(size_t)(M + m) * dk + d]
                                : (sk_in ? sk_in[(size_t)(M + m) * dk + d] : 0.0);
                cur[(size_t)m * dk + d] = rc[m] * c - rs[m] * s + k[(size_t)t * dk + d];
                cur[(size_t)(M + m) * dk + d] = rs[m] * c + rc[m] * s;
            }
            for (int d = 0; d < dv; ++d) {
                double c = prev ? prev[skl + (size_t)m * dv + d] : (sv_in ? sv_in[(size_t)m * dv + d] : 0.0);
                double s = prev ? prev[skl + (size_t)(M + m) * dv + d]
                                : (sv_in ? sv_in[(size_t)(M + m) * dv + d] : 0.0);
                cur[skl + (size_t)m * dv + d] = rc[m] * c - rs[m] * s + v[(size_t)t * dv + d];
                cur[skl + (size_t)(M + m) * dv + d] = rs[m] * c + rc[m] * s;
            }
        }
    }

    /* reverse pass */
    for (int t = L - 1; t >= 0; --t) {
        const double* st = hist + (size_t)t * (skl + svl);
        const double* Kc = st;
        const double* Ks = st + (size_t)M * dk;
        const double* Vc = st + skl;
        const double* Vs = st + skl + (size_t)M * dv;
        const double* qt = q + (size_t)t * dk;
        const double* gt = dO + (size_t)t * dv;
        int64_t pos = t0 + t;

        /* slots, scores and softmax, as in the forward */
        for (int s = 0; s < S; ++s) {
            for (int d = 0; d < dk; ++d) {
                double acc = 0.0;
                for (int m = 0; m < M; ++m)
                    acc += A[(size_t)s * M + m] * Kc[(size_t)m * dk + d] + Bm[(size_t)s * M + m] * Ks[(size_t)m * dk + d];
                Kt[(size_t)s * dk + d] = acc;
            }
            for (int d = 0; d < dv; ++d) {
                double acc = 0.0;
                for (int m = 0; m < M; ++m)
                    acc += A[(size_t)s * M + m] * Vc[(size_t)m * dv + d] + Bm[(size_t)s * M + m] * Vs[(size_t)m * dv + d];
                Vt[(size_t)s * dv + d] = acc;
            }
            double dot = 0.0;
            for (int d = 0; d < dk; ++d) dot += qt[d] * Kt[(size_t)s * dk + d];
            p[s] = pos < theta[s] ? -INFINITY : scale * dot;
        }
        double zmax = -INFINITY;
        for (int s = 0; s < S; ++s)
            if (p[s] > zmax) zmax = p[s];
        double den = 0.0;
        for (int s = 0; s < S; ++s) {
            p[s] = (p[s] == -INFINITY) ? 0.0 : exp(p[s] - zmax);
            den += p[s];
        }
        for (int s = 0; s < S; ++s) p[s] /= den;

        /* readout and softmax gradients */
        double pdp = 0.0;
        for (int s = 0; s < S; ++s) {
            double dot = 0.0;
            for (int d = 0; d < dv; ++d) dot += gt[d] * Vt[(size_t)s * dv + d];
            dz[s] = dot;
            pdp += p[s] * dot;
        }
        for (int s = 0; s < S; ++s) dz[s] = p[s] * (dz[s] - pdp);

        /* query gradient */
        for (int d = 0; d < dk; ++d) {
            double acc = 0.0;
            for (int s = 0; s < S; ++s) acc += dz[s] * Kt[(size_t)s * dk + d];
            dq[(size_t)t * dk + d] = scale * acc;
        }

        /* slot gradients into the adjoint of the state after token t */
        for (int m = 0; m < M; ++m) {
            for (int d = 0; d < dk; ++d) {
                double ac = 0.0, as = 0.0;
                for (int s = 0; s < S; ++s) {
                    double g = scale * dz[s] * qt[d];
                    ac += A[(size_t)s * M + m] * g;
                    as += Bm[(size_t)s * M + m] * g;
                }
                gK[(size_t)m * dk + d] += ac;
                gK[(size_t)(M + m) * dk + d] += as;
            }
            for (int d = 0; d < dv; ++d) {
                double ac = 0.0, as = 0.0;
                for (int s = 0; s < S; ++s) {
                    double g = p[s] * gt[d];
                    ac += A[(size_t)s * M + m] * g;
                    as += Bm[(size_t)s * M + m] * g;
                }
                gV[(size_t)m * dv + d] += ac;
                gV[(size_t)(M + m) * dv + d] += as;
            }
        }

        /* the token entered every cos row */
        for (int d = 0; d < dk; ++d) {
            double acc = 0.0;
            for (int m = 0; m < M; ++m) acc += gK[(size_t)m * dk + d];
            dkk[(size_t)t * dk + d] = acc;
        }
        for (int d = 0; d < dv; ++d) {
            double acc = 0.0;
            for (int m = 0; m < M; ++m) acc += gV[(size_t)m * dv + d];
            dvv[(size_t)t * dv + d] = acc;
        }

        /* through the rotation to the state before the token */
        for (int m = 0; m < M; ++m) {
            for (int d = 0; d < dk; ++d) {
                double c = gK[(size_t)m * dk + d], s = gK[(size_t)(M + m) * dk + d];
                gK[(size_t)m * dk + d] = rc[m] * c + rs[m] * s;
                gK[(size_t)(M + m) * dk + d] = -rs[m] * c + rc[m] * s;
            }
            for (int d = 0; d < dv; ++d) {
                double c = gV[(size_t)m * dv + d], s = gV[(size_t)(M + m) * dv + d];
                gV[(size_t)m * dv + d] = rc[m] * c + rs[m] * s;
                gV[(size_t)(M + m) * dv + d] = -rs[m] * c + rc[m] * s;
            }
        }
    }
}

/*
 * Backward over Bn*H sequences: dq, dk [Bn][H][L][dk], dv [Bn][H][L][dv]; dsk_out, dsv_out
 * (nullable) receive dLoss/d(state_in).  sk_in, sv_in (nullable: zero) are the forward's
 * input states; dsk_in, dsv_in (nullable: zero) are dLoss/d(final states).  Same argument
 * rules and return codes as bla_oracle_forward.
 */
int bla_oracle_backward(int Bn, int H, int L, int dk, int dv, int M, int S, const double* T,
                        int64_t t0, double scale, const double* q, const double* k,
                        const double* v, const double* dO, const double* sk_in,
                        const double* sv_in, const double* dsk_in, const double* dsv_in,
                        double* dq, double* dkk, double* dvv, double* dsk_out, double* dsv_out,
                        int nthreads)
{
    if (Bn < 0 || H < 0 || L < 0 || dk <= 0 || dv <= 0 || M <= 0 || S <= 0 || t0 < 0) return -1;
    size_t nseq = (size_t)Bn * H;
    size_t wlen = 2 * (size_t)S * M + (size_t)S + 2 * (size_t)M + 2 * (size_t)S +
                  (size_t)S * (dk + dv);
    size_t skl = 2 * (size_t)M * dk, svl = 2 * (size_t)M * dv;
    int err = 0;
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel
    {
        double* work = (double*)malloc(wlen * sizeof(double));
        double* adj = (double*)malloc((skl + svl) * sizeof(double));
        double* hist = (double*)malloc(((size_t)(L > 0 ? L : 1)) * (skl + svl) * sizeof(double));
        if (!work || !adj || !hist) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(dynamic, 1)
        for (long long i = 0; i < (long long)nseq; ++i) {
            if (!work || !adj || !hist) continue;
            int h = (int)(i % H);
            if (dsk_in) memcpy(adj, dsk_in + i * skl, skl * sizeof(double));
            else memset(adj, 0, skl * sizeof(double));
            if (dsv_in) memcpy(adj + skl, dsv_in + i * svl, svl * sizeof(double));
            else memset(adj + skl, 0, svl * sizeof(double));
            run_sequence_backward(L, dk, dv, M, S, T[h], t0, scale, q + i * (size_t)L * dk,
                                  k + i * (size_t)L * dk, v + i * (size_t)L * dv,
                                  dO + i * (size_t)L * dv, sk_in ? sk_in + i * skl : NULL,
                                  sv_in ? sv_in + i * svl : NULL, adj, adj + skl,
                                  dq + i * (size_t)L * dk, dkk + i * (size_t)L * dk,
                                  dvv + i * (size_t)L * dv, hist, work);
            if (dsk_out) memcpy(dsk_out + i * skl, adj, skl * sizeof(double));
            if (dsv_out) memcpy(dsv_out + i * svl, adj + skl, svl * sizeof(double));
        }
        free(work);
        free(adj);
        free(hist);
    }
    return err ? -1 : 0;
}
