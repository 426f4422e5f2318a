/*
 * CPU oracle for the SSD layer forward.  TEST INFRASTRUCTURE ONLY: the tests,
 * the smoke check and the benchmark's CPU baseline call it; the HIP library
 * never does, and the two share no code.
 *
 * It is the plain sequential recurrence, in float64, one token at a time:
 *
 *   selective SSM recurrence (Section 2, eq. s6):  h_t = A_t h_{t-1} + B_t x_t,
 *                                                  y_t = C_t^T h_t,
 *   with the scalar-times-identity transition of the SSD layer (Section 5,
 *   A_t = a_t I), broadcast over the head dimension P (Section 2, sequence
 *   transformations: P independent copies of the map).
 *
 * Discretisation (the paper defers it to prior work, Section 2, remark on
 * discretisation): per head A = -exp(A_log); transition exp(dt_t * A); input
 * dt_t * x_t.  So, per head h with state S (P x N):
 *
 *   S <- exp(dt_t A_h) S + (dt_t x_t) B_t^T        (outer product, P x N)
 *   y_t = S C_t + D_h x_t                          (contract over N)
 *
 * Head patterns (Section 7, multi-input / grouped-input SSM): B and C carry
 * G groups; head h reads group h / (H / G) (contiguous blocks of heads).
 *
 * Variable length (Section 8.3): with seq_idx, the single packed row holds
 * several sequences; the state entering the first token of every sequence is
 * replaced by that sequence's initial state (zero when none is given), so no
 * information crosses a boundary.  The initial state precedes the first token
 * and is decayed by it, as the state passed into the first chunk is in the
 * block decomposition (Section 6).  The final state of a sequence is the state
 * after its last token.
 *
 * Layouts (row-major): x,y (b,T,H,P); dt (b,T,H); A_log,D (H); B,C (b,T,G,N);
 * initial/final states (b,H,P,N), or (nseq,H,P,N) with seq_idx; seq_idx (1,T).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

int ssd_oracle_forward(int64_t batch, int64_t seqlen, int64_t nheads, int64_t headdim,
                       int64_t dstate, int64_t ngroups, const double* x, const double* dt,
                       const double* A_log, const double* B, const double* C,
                       const double* D, const double* initial_states,
                       const int32_t* seq_idx, int64_t nseq, double* y,
                       double* final_states, int nthreads)
{
    const int64_t T = seqlen, H = nheads, P = headdim, N = dstate, G = ngroups;
    if (batch <= 0 || T <= 0 || H <= 0 || P <= 0 || N <= 0 || G <= 0 || H % G)
        return -1;
    if (seq_idx && batch != 1)
        return -2;
    const int64_t heads_per_group = H / G;
    const int64_t units = batch * H;
    int bad = 0;

#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t u = 0; u < units; ++u) {
        const int64_t b = u / H, h = u % H, g = h / heads_per_group;
        const double A = -exp(A_log[h]);
        const double Dh = D ? D[h] : 0.0;
        double* S = (double*)malloc(sizeof(double) * P * N);
        if (!S) { bad = 1; continue; }
        for (int64_t t = 0; t < T; ++t) {
            /* state entering a unit: the row's (or the sequence's) initial state */
            int first = (t == 0) || (seq_idx && seq_idx[t] != seq_idx[t - 1]);
            if (first) {
                int64_t s = seq_idx ? seq_idx[t] : b;
                if (seq_idx && (s < 0 || s >= nseq)) { bad = 1; break; }
                if (initial_states)
                    memcpy(S, initial_states + (s * H + h) * P * N, sizeof(double) * P * N);
                else
                    memset(S, 0, sizeof(double) * P * N);
            }
            const double dtt = dt[(b * T + t) * H + h];
            const double decay = exp(dtt * A);
            const double* xt = x + ((b * T + t) * H + h) * P;
            const double* Bt = B + ((b * T + t) * G + g) * N;
            const double* Ct = C + ((b * T + t) * G + g) * N;
            double* yt = y + ((b * T + t) * H + h) * P;
            for (int64_t p = 0; p < P; ++p) {
                const double xin = dtt * xt[p];
                double* Sp = S + p * N;
                double acc = 0.0;
                for (int64_t n = 0; n < N; ++n) {
                    Sp[n] = decay * Sp[n] + xin * Bt[n];
                    acc += Sp[n] * Ct[n];
                }
                yt[p] = acc + Dh * xt[p];
            }
            int last = (t == T - 1) || (seq_idx && seq_idx[t + 1] != seq_idx[t]);
            if (last && final_states) {
                int64_t s = seq_idx ? seq_idx[t] : b;
                memcpy(final_states + (s * H + h) * P * N, S, sizeof(double) * P * N);
            }
        }
        free(S);
    }
    return bad ? -3 : 0;
}

/* Number of OpenMP threads the runtime would use by default (0 without OpenMP). */
int ssd_oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 0;
#endif
}
