/*
 * Parity oracle for the gated delta-rule recurrence -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  The product path (the HIP library) never calls it, shares
 * no source with it, and must fail loudly rather than fall back to it.
 *
 * What it computes (paper, section 2.2 "The model" and section 3.2 "A chunked
 * delta-rule scan for the recurrent layers"): every recurrent layer carries,
 * per head, a state matrix updated token by token.  With the state stored as
 * S in R^{dv x dk} (the transpose of the paper's H_k x H_v orientation), a scalar
 * log-decay g_t per (token, head) with alpha_t = exp(g_t), and a write strength
 * beta_t, the recurrence is
 *
 *     S_t = alpha_t * S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t (scale * q_t)                       (read after the update)
 *
 * This file writes that definition out literally, one state row at a time:
 * row j of S_t is  alpha_t * (s_j - beta_t (s_j . k_t) k_t) + beta_t v_t[j] k_t,
 * which is the j-th row of the matrix expression above (rows of S never mix).
 * Everything is fp64.  Inputs are the exact values the GPU receives, upcast.
 *
 * Layouts (row-major, contiguous, fp64):
 *   q, k      [Ttot, H, dk]     packed token axis (dense [B,T,H,d] == Ttot = B*T)
 *   v, o      [Ttot, H, dv]
 *   g, beta   [Ttot, H]
 *   S0, ST    [n_seq, H, dv, dk]  (S0 may be NULL: zero initial state;
 *                                  ST may be NULL: final state not stored)
 *   seq_start, seq_len [n_seq]   sequence s covers token rows
 *                                 [seq_start[s], seq_start[s] + seq_len[s]).
 *
 * Returns 0 on success, nonzero on an invalid argument.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_version(void) { return 1; }

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int oracle_gdn_recurrence(const double* q, const double* k, const double* v,
                          const double* g, const double* beta, const double* S0,
                          double* o, double* ST,
                          const int64_t* seq_start, const int64_t* seq_len, int n_seq,
                          int H, int dk, int dv, double scale, int n_threads)
{
    if (!q || !k || !v || !g || !beta || !o || !seq_start || !seq_len) return 1;
    if (n_seq < 0 || H < 1 || dk < 1 || dv < 1 || dk > 4096) return 2;
    const int64_t n_rows = (int64_t)n_seq * H * dv;   /* independent state rows */
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif

#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t task = 0; task < n_rows; ++task) {
        const int     j = (int)(task % dv);
        const int     h = (int)((task / dv) % H);
        const int64_t s = task / ((int64_t)dv * H);
        double row[4096];                                 /* s_j, one row of S */
        const int64_t srow = ((s * H + h) * (int64_t)dv + j) * dk;
        for (int c = 0; c < dk; ++c) row[c] = S0 ? S0[srow + c] : 0.0;

        for (int64_t t = seq_start[s]; t < seq_start[s] + seq_len[s]; ++t) {
            const double* kt = k + (t * H + h) * (int64_t)dk;
            const double* qt = q + (t * H + h) * (int64_t)dk;
            const double  vt = v[(t * H + h) * (int64_t)dv + j];
            const double  a  = exp(g[t * H + h]);
            const double  b  = beta[t * H + h];
            /* s_j (I - b k k^T) = s_j - b (s_j . k) k */
            double sk = 0.0;
            for (int c = 0; c < dk; ++c) sk += row[c] * kt[c];
            /* s_j <- a (s_j - b (s_j.k) k) + b v_j k */
            for (int c = 0; c < dk; ++c)
                row[c] = a * (row[c] - b * sk * kt[c]) + b * vt * kt[c];
            /* o_t[j] = s_j . (scale q_t) */
            double oj = 0.0;
            for (int c = 0; c < dk; ++c) oj += row[c] * (scale * qt[c]);
            o[(t * H + h) * (int64_t)dv + j] = oj;
        }
        if (ST)
            for (int c = 0; c < dk; ++c) ST[srow + c] = row[c];
    }
    return 0;
}
