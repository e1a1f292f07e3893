/*
 * Gated delta-rule oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, single-threaded CPU reference for the chunked gated
 * delta-rule prefill.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load it; it shares nothing with the HIP
 * path.
 *
 * The paper's hybrid model keeps a Gated DeltaNet state in its linear
 * layers (§2 "hybrid recurrent state", §7 model description) but never
 * writes the recurrence; the reading taken is the standard gated delta rule
 * of the Gated DeltaNet work the paper builds on, with S of shape dk x dv and
 * row vectors q_t, k_t (dk) and v_t (dv):
 *
 *   S_t = exp(g_t) (I - beta_t k_t^T k_t) S_{t-1} + beta_t k_t^T v_t
 *   o_t = scale * q_t S_t                         (state AFTER token t)
 *
 * with one log-gate g_t <= 0 and one write strength beta_t in [0, 1] per
 * (token, head).
 *
 * Two independent implementations:
 *   orc_gdn_sequential -- the recurrence token by token (the definition),
 *   orc_gdn_chunked    -- the chunked form, derived from unrolling the
 *     recurrence inside one chunk of C tokens with entering state S and
 *     inclusive in-chunk log-decay sums G_t (gamma_t = exp(G_t)).  Writing
 *     the update as S_t = exp(g_t) S_{t-1} + k_t^T u_t with the pseudo-value
 *     u_t = beta_t (v_t - exp(g_t) k_t S_{t-1}) and unrolling gives
 *       u_t = beta_t v_t - beta_t gamma_t k_t S
 *             - sum_{j<t} beta_t (gamma_t / gamma_j) (k_t . k_j) u_j,
 *     i.e. (I + A) U = diag(beta) V - diag(beta gamma) K S with A strictly
 *     lower triangular, A_tj = beta_t (gamma_t / gamma_j)(k_t . k_j).  With
 *     W = (I + A)^-1 diag(beta gamma) K and U' = (I + A)^-1 diag(beta) V
 *     (both independent of S):
 *       U     = U' - W S
 *       o_t   = scale (gamma_t q_t S + sum_{j<=t} (gamma_t / gamma_j)(q_t . k_j) u_j)
 *       S_new = gamma_last S + sum_j (gamma_last / gamma_j) k_j^T u_j
 *     (I + A) is solved by forward substitution, row by row.
 *
 * Precision: inputs are the exact fp32 values the device sees; every
 * accumulation is fp64; outputs fp64.
 *
 * Parity status: pinned (chunked against sequential; beta = 0 reduces to a
 * pure decay; with orthonormal keys and beta = 1 the state stores each value
 * exactly under its key; linearity in (v, S0); causality).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define AT3(p, t, h, d, H, D) ((p)[((int64_t)(t) * (H) + (h)) * (D) + (d)])
#define AT2(p, t, h, H) ((p)[(int64_t)(t) * (H) + (h)])

/*
 * The recurrence, token by token.  Returns 0, or -1 on a bad argument.
 *   q, k : [T, H, dk] fp32   v : [T, H, dv] fp32   g, beta : [T, H] fp32
 *   S0   : [H, dk, dv] fp64 or NULL   o : [T, H, dv] fp64   S_final : [H, dk, dv] or NULL
 */
int orc_gdn_sequential(int64_t T, int64_t H, int64_t dk, int64_t dv,
                       const float* q, const float* k, const float* v, const float* g,
                       const float* beta, double scale, const double* S0,
                       double* o, double* S_final)
{
    if (T < 0 || H <= 0 || dk <= 0 || dv <= 0) return -1;
    double* S = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    double* kS = (double*)malloc(sizeof(double) * (size_t)dv);
    if (!S || !kS) { free(S); free(kS); return -1; }
    for (int64_t h = 0; h < H; ++h) {
        for (int64_t i = 0; i < dk * dv; ++i)
            S[i] = S0 ? S0[h * dk * dv + i] : 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double a = exp((double)AT2(g, t, h, H));
            const double b = (double)AT2(beta, t, h, H);
            /* kS = k_t S_{t-1} (1 x dv) */
            for (int64_t j = 0; j < dv; ++j) {
                double acc = 0.0;
                for (int64_t i = 0; i < dk; ++i) acc += (double)AT3(k, t, h, i, H, dk) * S[i * dv + j];
                kS[j] = acc;
            }
            /* S_t = a (S - b k^T (k S)) + b k^T v */
            for (int64_t i = 0; i < dk; ++i) {
                const double ki = (double)AT3(k, t, h, i, H, dk);
                for (int64_t j = 0; j < dv; ++j)
                    S[i * dv + j] = a * (S[i * dv + j] - b * ki * kS[j]) + b * ki * (double)AT3(v, t, h, j, H, dv);
            }
            for (int64_t j = 0; j < dv; ++j) {
                double acc = 0.0;
                for (int64_t i = 0; i < dk; ++i) acc += (double)AT3(q, t, h, i, H, dk) * S[i * dv + j];
                AT3(o, t, h, j, H, dv) = scale * acc;
            }
        }
        if (S_final) memcpy(S_final + h * dk * dv, S, sizeof(double) * (size_t)(dk * dv));
    }
    free(S);
    free(kS);
    return 0;
}

/*
 * The chunked form (see the header comment).  chunk_states, when not NULL,
 * receives the state ENTERING each chunk ([ceil(T/C), H, dk, dv]).
 */
int orc_gdn_chunked(int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C,
                    const float* q, const float* k, const float* v, const float* g,
                    const float* beta, double scale, const double* S0,
                    double* o, double* chunk_states, double* S_final)
{
    if (T < 0 || H <= 0 || dk <= 0 || dv <= 0 || C <= 0) return -1;
    const int64_t n_chunks = (T + C - 1) / C;
    double* S = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    double* G = (double*)malloc(sizeof(double) * (size_t)C);
    double* A = (double*)malloc(sizeof(double) * (size_t)(C * C));
    double* W = (double*)malloc(sizeof(double) * (size_t)(C * dk));
    double* U = (double*)malloc(sizeof(double) * (size_t)(C * dv));
    double* Snew = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    if (!S || !G || !A || !W || !U || !Snew) {
        free(S); free(G); free(A); free(W); free(U); free(Snew);
        return -1;
    }
    for (int64_t h = 0; h < H; ++h) {
        for (int64_t i = 0; i < dk * dv; ++i)
            S[i] = S0 ? S0[h * dk * dv + i] : 0.0;
        for (int64_t c = 0; c < n_chunks; ++c) {
            const int64_t t0 = c * C;
            const int64_t L = (T - t0 < C) ? (T - t0) : C;
            if (chunk_states)
                memcpy(chunk_states + (c * H + h) * dk * dv, S, sizeof(double) * (size_t)(dk * dv));
            double run = 0.0;
            for (int64_t i = 0; i < L; ++i) {
                run += (double)AT2(g, t0 + i, h, H);
                G[i] = run;
            }
            /* A_tj = beta_t exp(G_t - G_j) (k_t . k_j), j < t */
            for (int64_t t = 0; t < L; ++t)
                for (int64_t j = 0; j < L; ++j) {
                    double kk = 0.0;
                    if (j < t)
                        for (int64_t d = 0; d < dk; ++d)
                            kk += (double)AT3(k, t0 + t, h, d, H, dk) * (double)AT3(k, t0 + j, h, d, H, dk);
                    A[t * C + j] = j < t ? (double)AT2(beta, t0 + t, h, H) * exp(G[t] - G[j]) * kk : 0.0;
                }
            /* forward substitution: (I + A) W = diag(beta gamma) K and
               (I + A) U' = diag(beta) V, row by row */
            for (int64_t t = 0; t < L; ++t) {
                const double bt = (double)AT2(beta, t0 + t, h, H);
                const double gt = exp(G[t]);
                for (int64_t d = 0; d < dk; ++d) {
                    double acc = bt * gt * (double)AT3(k, t0 + t, h, d, H, dk);
                    for (int64_t j = 0; j < t; ++j) acc -= A[t * C + j] * W[j * dk + d];
                    W[t * dk + d] = acc;
                }
                for (int64_t e = 0; e < dv; ++e) {
                    double acc = bt * (double)AT3(v, t0 + t, h, e, H, dv);
                    for (int64_t j = 0; j < t; ++j) acc -= A[t * C + j] * U[j * dv + e];
                    U[t * dv + e] = acc;
                }
            }
            /* U = U' - W S */
            for (int64_t t = 0; t < L; ++t)
                for (int64_t e = 0; e < dv; ++e) {
                    double acc = 0.0;
                    for (int64_t d = 0; d < dk; ++d) acc += W[t * dk + d] * S[d * dv + e];
                    U[t * dv + e] -= acc;
                }
            /* outputs */
            for (int64_t t = 0; t < L; ++t) {
                const double gt = exp(G[t]);
                for (int64_t e = 0; e < dv; ++e) {
                    double inter = 0.0;
                    for (int64_t d = 0; d < dk; ++d) inter += (double)AT3(q, t0 + t, h, d, H, dk) * S[d * dv + e];
                    double intra = 0.0;
                    for (int64_t j = 0; j <= t; ++j) {
                        double qk = 0.0;
                        for (int64_t d = 0; d < dk; ++d)
                            qk += (double)AT3(q, t0 + t, h, d, H, dk) * (double)AT3(k, t0 + j, h, d, H, dk);
                        intra += exp(G[t] - G[j]) * qk * U[j * dv + e];
                    }
                    AT3(o, t0 + t, h, e, H, dv) = scale * (gt * inter + intra);
                }
            }
            /* state at the chunk end */
            const double glast = exp(G[L - 1]);
            for (int64_t d = 0; d < dk; ++d)
                for (int64_t e = 0; e < dv; ++e) {
                    double acc = glast * S[d * dv + e];
                    for (int64_t j = 0; j < L; ++j)
                        acc += exp(G[L - 1] - G[j]) * (double)AT3(k, t0 + j, h, d, H, dk) * U[j * dv + e];
                    Snew[d * dv + e] = acc;
                }
            memcpy(S, Snew, sizeof(double) * (size_t)(dk * dv));
        }
        if (S_final) memcpy(S_final + h * dk * dv, S, sizeof(double) * (size_t)(dk * dv));
    }
    free(S); free(G); free(A); free(W); free(U); free(Snew);
    return 0;
}
