/*
 * oracle_attn.c -- plain fp64 CPU oracle for scaled dot-product attention.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no code, header, helper or
 * constant with the GPU library; the two meet only through the seeded inputs.
 *
 * What it computes (per batch b and head h independently, as the paper's
 * remark on higher-rank tensors partitions the problem, Sec. "MoA DNF
 * Derivation of Attention"):
 *
 *   Attention(Q, K, V) = softmax(scale * Q K^T) V          (eq. attention)
 *
 * with the numerically stable softmax of eq. stable_softmax.  For each query
 * row i the steps are taken in the paper's order (Steps I-IV and eq.
 * output_dnf; the per-row arrays s, e, w of Algorithm 1 are kept explicitly,
 * every intermediate is materialised, nothing is fused or reordered):
 *
 *   s[k] = scale * sum_{j=0}^{dk-1} Q[i][j] * K[k][j]     (eq. mm_psi: K read by
 *                                                            row, no K^T)
 *          or -inf when key k is masked
 *   m    = max_k s[k]                                      (Step I, eq. z_psi)
 *   e[k] = exp(s[k] - m)          (0 for masked keys)      (Step II, eq. num_psi)
 *   Z    = sum_k e[k]                                      (Step III, eq. den_psi)
 *   w[k] = e[k] / Z                                        (Step IV)
 *   O[i][c] = sum_k w[k] * V[k][c]                         (eq. output_dnf)
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *  - The paper divides by sqrt(dk); this oracle multiplies by a caller-given
 *    fp32 `scale` (1/sqrt(dk) by default in the callers), widened exactly.
 *  - Causal masking is not in the paper.  Key k is visible to query i iff
 *    k <= i + (Nk - Nq) (bottom-right aligned; equal to k <= i when Nq == Nk).
 *  - Masked logits are -inf, their e and w are exactly 0, and the max runs
 *    over visible keys only.
 *  - Sums run in increasing index order in IEEE fp64 with no contraction
 *    (built with -ffp-contract=off, no fast-math).
 *  - Inputs are fp32 or bf16 bit patterns; both widen exactly to fp64.
 *
 * Also returned on request: LSE[i] = m + ln(Z), the log of the softmax
 * denominator in natural-log units, and the full S and P matrices for tiny
 * shapes; the backward pass (dQ, dK, dV for a given dO, see oracle_attn_bwd
 * below); and the input projections that produce Q, K and V from the
 * sequence X (oracle_proj and oracle_bf16_round below).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_F32 = 0, ORACLE_BF16 = 1 };

typedef struct {
    const void* q;
    const void* k;
    const void* v;
    int dtype;
    int64_t B, H, Nq, Nk, dk, dv;
    double scale;
    int causal;
} problem_t;

/* Exact widening of one stored element to fp64. */
static double elem(const void* base, int dtype, int64_t idx) {
    if (dtype == ORACLE_F32) return (double)((const float*)base)[idx];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

static int visible(const problem_t* p, int64_t i, int64_t k) {
    return !p->causal || k <= i + (p->Nk - p->Nq);
}

/*
 * One query row: flat row index r = (b*H + h)*Nq + i.
 * s, e, w are caller-provided scratch of length Nk (Algorithm 1's vectors).
 * Writes O row (dv values), and optionally LSE, S row and P row.
 */
static void attend_row(const problem_t* p, int64_t r, double* s, double* e, double* w,
                       double* o_row, double* lse, double* s_row, double* p_row) {
    const int64_t bh = r / p->Nq;
    const int64_t i = r % p->Nq;
    const int64_t q_base = (bh * p->Nq + i) * p->dk;
    const int64_t k_base = bh * p->Nk * p->dk;
    const int64_t v_base = bh * p->Nk * p->dv;

    /* scores: inner product of Q row i with K row k (eq. mm_psi), then scaled */
    for (int64_t k = 0; k < p->Nk; ++k) {
        if (!visible(p, i, k)) {
            s[k] = -INFINITY;
            continue;
        }
        double acc = 0.0;
        for (int64_t j = 0; j < p->dk; ++j)
            acc += elem(p->q, p->dtype, q_base + j) * elem(p->k, p->dtype, k_base + k * p->dk + j);
        s[k] = p->scale * acc;
    }
    /* Step I: row maximum over visible keys */
    double m = -INFINITY;
    for (int64_t k = 0; k < p->Nk; ++k)
        if (s[k] > m) m = s[k];
    /* Step II: numerator */
    for (int64_t k = 0; k < p->Nk; ++k)
        e[k] = (s[k] == -INFINITY) ? 0.0 : exp(s[k] - m);
    /* Step III: denominator */
    double Z = 0.0;
    for (int64_t k = 0; k < p->Nk; ++k) Z += e[k];
    /* Step IV: attention weights */
    for (int64_t k = 0; k < p->Nk; ++k) w[k] = e[k] / Z;
    /* output row: weighted sum of V rows, each O[i][c] summed in increasing k */
    for (int64_t c = 0; c < p->dv; ++c) o_row[c] = 0.0;
    for (int64_t k = 0; k < p->Nk; ++k) {
        if (s[k] == -INFINITY) continue;   /* masked key: its weight is exactly 0 */
        for (int64_t c = 0; c < p->dv; ++c)
            o_row[c] += w[k] * elem(p->v, p->dtype, v_base + k * p->dv + c);
    }
    if (lse) *lse = m + log(Z);
    if (s_row) memcpy(s_row, s, (size_t)p->Nk * sizeof(double));
    if (p_row) memcpy(p_row, w, (size_t)p->Nk * sizeof(double));
}

static int check(const problem_t* p) {
    if (!p->q || !p->k || !p->v) return 1;
    if (p->dtype != ORACLE_F32 && p->dtype != ORACLE_BF16) return 1;
    if (p->B < 0 || p->H < 0 || p->Nq < 0 || p->Nk <= 0 || p->dk <= 0 || p->dv <= 0) return 1;
    if (p->causal && p->Nq > p->Nk) return 1;
    return 0;
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* Runs rows[0..n_rows) (flat row indices) or, if rows == NULL, all B*H*Nq rows. */
static int run_rows(const problem_t* p, const int64_t* rows, int64_t n_rows, double* O, double* LSE,
                    double* S, double* P, int nthreads) {
    if (check(p)) return 1;
    const int64_t total = p->B * p->H * p->Nq;
    if (rows)
        for (int64_t t = 0; t < n_rows; ++t)
            if (rows[t] < 0 || rows[t] >= total) return 1;
    set_threads(nthreads);
    int nt = 1;
#ifdef _OPENMP
    nt = omp_get_max_threads();
#endif
    /* per-thread copies of Algorithm 1's row vectors s, e, w */
    double* scratch = (double*)malloc((size_t)nt * 3 * (size_t)p->Nk * sizeof(double));
    if (!scratch) return 2;
#pragma omp parallel num_threads(nt)
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double* s = scratch + (size_t)tid * 3 * (size_t)p->Nk;
        double* e = s + p->Nk;
        double* w = e + p->Nk;
#pragma omp for schedule(dynamic, 4)
        for (int64_t t = 0; t < n_rows; ++t) {
            int64_t r = rows ? rows[t] : t;
            attend_row(p, r, s, e, w, O + t * p->dv, LSE ? LSE + t : NULL,
                       S ? S + t * p->Nk : NULL, P ? P + t * p->Nk : NULL);
        }
    }
    free(scratch);
    return 0;
}

/*
 * Full problem.  Q [B][H][Nq][dk], K [B][H][Nk][dk], V [B][H][Nk][dv] (row-major,
 * fp32 or bf16 bits per `dtype`).  O [B][H][Nq][dv] fp64; LSE [B][H][Nq] fp64 or NULL.
 * Returns 0 on success, 1 on bad arguments, 2 on host allocation failure.
 */
int oracle_attn_fwd(const void* Q, const void* K, const void* V, int dtype, int64_t B, int64_t H,
                    int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, float scale, int causal,
                    double* O, double* LSE, int nthreads) {
    problem_t p = {Q, K, V, dtype, B, H, Nq, Nk, dk, dv, (double)scale, causal};
    if (!O) return 1;
    return run_rows(&p, NULL, B * H * Nq, O, LSE, NULL, NULL, nthreads);
}

/*
 * Selected rows only: rows[t] is the flat row (b*H + h)*Nq + i.  O_rows is
 * [n_rows][dv], LSE_rows [n_rows] or NULL.  Used to check sampled outputs of
 * the large workloads.
 */
int oracle_attn_rows(const void* Q, const void* K, const void* V, int dtype, int64_t B, int64_t H,
                     int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, float scale, int causal,
                     const int64_t* rows, int64_t n_rows, double* O_rows, double* LSE_rows,
                     int nthreads) {
    problem_t p = {Q, K, V, dtype, B, H, Nq, Nk, dk, dv, (double)scale, causal};
    if (!O_rows || !rows || n_rows < 0) return 1;
    return run_rows(&p, rows, n_rows, O_rows, LSE_rows, NULL, NULL, nthreads);
}

/*
 * Full problem with the score matrix S (scaled, -inf where masked) and the
 * attention weights P, both [B][H][Nq][Nk] fp64, for tiny shapes.
 */
int oracle_attn_weights(const void* Q, const void* K, const void* V, int dtype, int64_t B,
                        int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv, float scale,
                        int causal, double* S, double* P, double* O, double* LSE) {
    problem_t p = {Q, K, V, dtype, B, H, Nq, Nk, dk, dv, (double)scale, causal};
    if (!S || !P || !O) return 1;
    return run_rows(&p, NULL, B * H * Nq, O, LSE, S, P, 1);
}

/*
 * Backward pass: the gradients of a scalar loss through O, given its
 * gradient dO = dL/dO, by the chain rule through the softmax Jacobian (the
 * derivative the paper's Stage 5 sets out to take).  Per (b, h) slice, with
 * w the attention weights of query row i (attend_row's Step IV output):
 *
 *   dV[k][c] = sum_i w_i[k] * dO[i][c]
 *   dP[k]    = sum_c dO[i][c] * V[k][c]                  (per row i)
 *   D        = sum_k w_i[k] * dP[k]
 *   dS[k]    = w_i[k] * (dP[k] - D)        (softmax Jacobian: dw/ds = diag(w) - w w^T)
 *   dQ[i][j] = scale * sum_k dS[k] * K[k][j]
 *   dK[k][j] = scale * sum_i dS_i[k] * Q[i][j]
 *
 * Masked keys have weight 0 and contribute nothing.  One (b, h) slice per
 * thread, so the sums over i of dK and dV run in increasing i within one
 * thread.  dO has the storage type of Q, K, V; dQ, dK, dV are fp64 in the
 * layouts of Q, K, V.
 */
int oracle_attn_bwd(const void* Q, const void* K, const void* V, const void* dO, int dtype,
                    int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                    float scale, int causal, double* dQ, double* dK, double* dV, int nthreads) {
    problem_t p = {Q, K, V, dtype, B, H, Nq, Nk, dk, dv, (double)scale, causal};
    if (check(&p) || !dO || !dQ || !dK || !dV) return 1;
    set_threads(nthreads);
    int nt = 1;
#ifdef _OPENMP
    nt = omp_get_max_threads();
#endif
    const size_t per = 4 * (size_t)Nk + (size_t)dv;
    double* scratch = (double*)malloc((size_t)nt * per * sizeof(double));
    if (!scratch) return 2;
    for (int64_t x = 0; x < B * H * Nk * dk; ++x) dK[x] = 0.0;
    for (int64_t x = 0; x < B * H * Nk * dv; ++x) dV[x] = 0.0;
#pragma omp parallel num_threads(nt)
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double* s = scratch + (size_t)tid * per;
        double* e = s + Nk;
        double* w = e + Nk;
        double* dp = w + Nk;
        double* o_row = dp + Nk;
#pragma omp for schedule(dynamic, 1)
        for (int64_t bh = 0; bh < B * H; ++bh) {
            const int64_t k_base = bh * Nk * dk, v_base = bh * Nk * dv;
            for (int64_t i = 0; i < Nq; ++i) {
                const int64_t r = bh * Nq + i;
                attend_row(&p, r, s, e, w, o_row, NULL, NULL, NULL);
                const int64_t q_row = r * dk, o_off = r * dv;
                double D = 0.0;
                for (int64_t k = 0; k < Nk; ++k) {
                    dp[k] = 0.0;
                    if (s[k] == -INFINITY) continue;
                    for (int64_t c = 0; c < dv; ++c)
                        dp[k] += elem(dO, dtype, o_off + c) * elem(V, dtype, v_base + k * dv + c);
                    D += w[k] * dp[k];
                }
                for (int64_t j = 0; j < dk; ++j) dQ[q_row + j] = 0.0;
                for (int64_t k = 0; k < Nk; ++k) {
                    if (s[k] == -INFINITY) continue;
                    const double ds = w[k] * (dp[k] - D);
                    for (int64_t j = 0; j < dk; ++j) {
                        dQ[q_row + j] += (double)scale * ds * elem(K, dtype, k_base + k * dk + j);
                        dK[k_base + k * dk + j] += (double)scale * ds * elem(Q, dtype, q_row + j);
                    }
                    for (int64_t c = 0; c < dv; ++c)
                        dV[v_base + k * dv + c] += w[k] * elem(dO, dtype, o_off + c);
                }
            }
        }
    }
    free(scratch);
    return 0;
}

/*
 * The same gradients at sampled outputs of one head slice bh (0 <= bh < B*H):
 * dQ at the query rows qrows[0..nq) and dK, dV at the key rows krows[0..nk)
 * of that slice (row indices within the slice).  Long sequences need this:
 * the full pass above costs O(Nq * Nk * d) per head with no shortcut.
 *
 * Every query row i of the slice first goes through attend_row (Steps I-IV,
 * its weights w[k] and output row O_i).  With dP_ik = <dO_i, V_k>:
 *   D_i  = sum_c dO_i[c] * O_i[c]      (= sum_k w_ik dP_ik, by the definition
 *                                        of O_i; taken in this form here so
 *                                        that a row needs dP only at the
 *                                        sampled keys)
 *   dS_ik = w_ik * (dP_ik - D_i)
 *   dQ_i  = scale * sum_k dS_ik K_k      (sampled i, all k, increasing k)
 *   dK_k  = scale * sum_i dS_ik Q_i      (sampled k, all i, increasing i)
 *   dV_k  =         sum_i w_ik dO_i      (sampled k, all i, increasing i)
 * Returns 0, 1 on invalid arguments, 2 when scratch memory is short.
 */
int oracle_attn_bwd_rows(const void* Q, const void* K, const void* V, const void* dO, int dtype,
                         int64_t B, int64_t H, int64_t Nq, int64_t Nk, int64_t dk, int64_t dv,
                         float scale, int causal, int64_t bh, const int64_t* qrows, int64_t nq,
                         const int64_t* krows, int64_t nk, double* dQ, double* dK, double* dV,
                         int nthreads) {
    problem_t p = {Q, K, V, dtype, B, H, Nq, Nk, dk, dv, (double)scale, causal};
    if (check(&p) || !dO || bh < 0 || bh >= B * H || nq < 0 || nk < 0) return 1;
    if ((nq && (!qrows || !dQ)) || (nk && (!krows || !dK || !dV))) return 1;
    for (int64_t x = 0; x < nq; ++x)
        if (qrows[x] < 0 || qrows[x] >= Nq) return 1;
    for (int64_t x = 0; x < nk; ++x)
        if (krows[x] < 0 || krows[x] >= Nk) return 1;
    set_threads(nthreads);
    int nt = 1;
#ifdef _OPENMP
    nt = omp_get_max_threads();
#endif
    const size_t per = 3 * (size_t)Nk + (size_t)dv;
    double* scratch = (double*)malloc((size_t)nt * per * sizeof(double));
    /* per query row and sampled key: the weight w_ik and dS_ik */
    double* wk = (double*)malloc(((size_t)Nq * (size_t)(nk ? nk : 1)) * sizeof(double));
    double* sk = (double*)malloc(((size_t)Nq * (size_t)(nk ? nk : 1)) * sizeof(double));
    if (!scratch || !wk || !sk) {
        free(scratch); free(wk); free(sk);
        return 2;
    }
    const int64_t k_base = bh * Nk * dk, v_base = bh * Nk * dv;
#pragma omp parallel num_threads(nt)
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double* s = scratch + (size_t)tid * per;
        double* e = s + Nk;
        double* w = e + Nk;
        double* o_row = w + Nk;
#pragma omp for schedule(dynamic, 16)
        for (int64_t i = 0; i < Nq; ++i) {
            const int64_t r = bh * Nq + i;
            attend_row(&p, r, s, e, w, o_row, NULL, NULL, NULL);
            const int64_t q_row = r * dk, o_off = r * dv;
            double D = 0.0;
            for (int64_t c = 0; c < dv; ++c) D += elem(dO, dtype, o_off + c) * o_row[c];
            for (int64_t x = 0; x < nk; ++x) {
                const int64_t k = krows[x];
                double ds = 0.0;
                if (s[k] != -INFINITY) {
                    double dp = 0.0;
                    for (int64_t c = 0; c < dv; ++c)
                        dp += elem(dO, dtype, o_off + c) * elem(V, dtype, v_base + k * dv + c);
                    ds = w[k] * (dp - D);
                }
                wk[(size_t)i * nk + x] = w[k];
                sk[(size_t)i * nk + x] = ds;
            }
            for (int64_t y = 0; y < nq; ++y) {
                if (qrows[y] != i) continue;
                double* dq_row = dQ + y * dk;
                for (int64_t j = 0; j < dk; ++j) dq_row[j] = 0.0;
                for (int64_t k = 0; k < Nk; ++k) {
                    if (s[k] == -INFINITY) continue;
                    double dp = 0.0;
                    for (int64_t c = 0; c < dv; ++c)
                        dp += elem(dO, dtype, o_off + c) * elem(V, dtype, v_base + k * dv + c);
                    const double ds = w[k] * (dp - D);
                    for (int64_t j = 0; j < dk; ++j)
                        dq_row[j] += (double)scale * ds * elem(K, dtype, k_base + k * dk + j);
                }
            }
            (void)q_row;
        }
#pragma omp for schedule(static)
        for (int64_t x = 0; x < nk; ++x) {
            double* dk_row = dK + x * dk;
            double* dv_row = dV + x * dv;
            for (int64_t j = 0; j < dk; ++j) dk_row[j] = 0.0;
            for (int64_t c = 0; c < dv; ++c) dv_row[c] = 0.0;
            for (int64_t i = 0; i < Nq; ++i) {
                const double wi = wk[(size_t)i * nk + x], ds = sk[(size_t)i * nk + x];
                if (wi == 0.0 && ds == 0.0) continue;
                const int64_t q_row = (bh * Nq + i) * dk, o_off = (bh * Nq + i) * dv;
                for (int64_t j = 0; j < dk; ++j) dk_row[j] += (double)scale * ds * elem(Q, dtype, q_row + j);
                for (int64_t c = 0; c < dv; ++c) dv_row[c] += wi * elem(dO, dtype, o_off + c);
            }
        }
    }
    free(scratch);
    free(wk);
    free(sk);
    return 0;
}

/* Threads OpenMP would use for a call with nthreads <= 0. */
int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * Input projections (the paper's problem statement: Q = X W_Q, K = X W_K,
 * V = X W_V).  X is [B][N][Dm] and each weight is given transposed, as
 * Wt[f][k] = W[k][f] with f over the H*d projected features (the layout of a
 * dense layer's weight); X and Wt are fp32 or bf16 bit patterns (same type).
 * Writes the exact projection, in fp64, in head-split form:
 *
 *   P[b][h][n][e] = sum_{k=0}^{Dm-1} X[b][n][k] * Wt[h*d + e][k]
 *
 * summed in increasing k, with no reordering.  Returns 0, or -1 on invalid
 * sizes.
 */
int oracle_proj(const void* X, const void* Wt, int dtype, int64_t B, int64_t N, int64_t Dm,
                int64_t H, int64_t d, double* P, int nthreads) {
    if (B < 0 || N < 0 || Dm < 1 || H < 0 || d < 1) return -1;
    set_threads(nthreads);
    const int64_t F = H * d;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < B * N; ++r) {
        const int64_t b = r / N, n = r % N;
        for (int64_t f = 0; f < F; ++f) {
            double acc = 0.0;
            for (int64_t k = 0; k < Dm; ++k)
                acc += elem(X, dtype, r * Dm + k) * elem(Wt, dtype, f * Dm + k);
            const int64_t h = f / d, e = f % d;
            P[((b * H + h) * N + n) * d + e] = acc;
        }
    }
    return 0;
}

/*
 * Round fp64 values to bf16, nearest with ties to even, directly from the fp64
 * value (no intermediate fp32, so no double rounding): the significand is
 * scaled to 8 bits and rounded by the FPU's default round-to-nearest-even.
 * Normal range only (|v| in [2^-126, 2^128)) and zero; that covers every value
 * the tests produce.  Writes bf16 bit patterns.
 */
void oracle_bf16_round(const double* v, int64_t n, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) {
        const double x = v[i];
        double y = 0.0;
        if (x != 0.0) {
            int e;
            const double m = frexp(fabs(x), &e);           /* |x| = m * 2^e, m in [0.5, 1) */
            y = ldexp(nearbyint(ldexp(m, 8)), e - 8);      /* 8 significant bits */
            if (x < 0) y = -y;
        } else if (signbit(x)) {
            y = -0.0;
        }
        const float f = (float)y;                          /* exact: 8 significant bits */
        uint32_t bits;
        memcpy(&bits, &f, sizeof bits);
        out[i] = (uint16_t)(bits >> 16);
    }
}
