/*
 * Gated linear-attention oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, single-threaded CPU reference for what the chunked
 * linear-attention prefill computes.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it; the product library never
 * links, includes or calls anything in this directory, and this file shares
 * no code, header, table or helper with the HIP path.
 *
 * What is computed (paper: "Execution-State Capsules", §2 "hybrid recurrent
 * state is not prefix-addressable" -- the linear-attention state at position N
 * is a fold over all N tokens; §5 "chunk-alignment condition" -- the long
 * prefill folds that state once per chunk of C tokens, chunk boundaries at
 * multiples of C counted from the start of the prefill):
 *
 *   per head, with S_{-1} = S0 (dk x dv, zero when not given) and scale s
 *     S_t = exp(g_t) * S_{t-1} + k_t^T v_t          (outer product, dk x dv)
 *     o_t = s * q_t S_t                              (state AFTER token t)
 *
 * Two independent implementations of the same quantity live here:
 *   orc_linattn_sequential -- the recurrence itself, token by token (the
 *                             definition; pinned by closed forms),
 *   orc_linattn_chunked    -- the chunked form, written from the algebra of
 *                             one chunk (intra-chunk causal term plus the
 *                             decayed inter-chunk state term, then the state
 *                             fold at the chunk end); pinned by brute force
 *                             against the sequential form.
 *
 * Precision: inputs are the exact fp32 values the device sees (bf16 inputs are
 * widened exactly); every accumulation is fp64; outputs are fp64.
 *
 * Parity status: pinned (closed forms, brute force, composition, linearity,
 * head permutation, causality).  The paper prints no worked numeric example of
 * the scan, so absolute values are pinned by those invariants only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* [T, H, D] token-major layout, the same one the device path consumes. */
#define AT3(p, t, h, d, H, D) ((p)[((int64_t)(t) * (H) + (h)) * (D) + (d)])

/*
 * The recurrence, token by token.  Returns 0, or -1 on a bad argument.
 *   q, k : [T, H, dk] fp32      v : [T, H, dv] fp32      g : [T, H] fp32
 *   S0   : [H, dk, dv] fp64 or NULL (zeros)
 *   o    : [T, H, dv] fp64 out  S_final : [H, dk, dv] fp64 out (may be NULL)
 */
int orc_linattn_sequential(int64_t T, int64_t H, int64_t dk, int64_t dv,
                           const float* q, const float* k, const float* v,
                           const float* g, double scale, const double* S0,
                           double* o, double* S_final)
{
    if (T < 0 || H <= 0 || dk <= 0 || dv <= 0) return -1;
    double* S = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    if (!S) return -1;
    for (int64_t h = 0; h < H; ++h) {
        for (int64_t i = 0; i < dk * dv; ++i)
            S[i] = S0 ? S0[h * dk * dv + i] : 0.0;
        for (int64_t t = 0; t < T; ++t) {
            const double decay = exp((double)g[t * H + h]);
            /* state update: decay the whole state, then add the outer product */
            for (int64_t i = 0; i < dk; ++i) {
                const double ki = (double)AT3(k, t, h, i, H, dk);
                for (int64_t j = 0; j < dv; ++j)
                    S[i * dv + j] = decay * S[i * dv + j] + ki * (double)AT3(v, t, h, j, H, dv);
            }
            /* readout with the updated state */
            for (int64_t j = 0; j < dv; ++j) {
                double acc = 0.0;
                for (int64_t i = 0; i < dk; ++i)
                    acc += (double)AT3(q, t, h, i, H, dk) * S[i * dv + j];
                AT3(o, t, h, j, H, dv) = scale * acc;
            }
        }
        if (S_final)
            memcpy(S_final + h * dk * dv, S, sizeof(double) * (size_t)(dk * dv));
    }
    free(S);
    return 0;
}

/*
 * The chunked form.  Chunk j covers tokens [jC, min((j+1)C, T)) of this call,
 * length L; G_i is the inclusive prefix sum of the log-gates inside the chunk.
 *   o_i     = s * ( exp(G_i) q_i S_j  +  sum_{m<=i} exp(G_i - G_m) (q_i . k_m) v_m )
 *   S_{j+1} = exp(G_{L-1}) S_j  +  sum_{m<L} exp(G_{L-1} - G_m) k_m^T v_m
 * chunk_states (optional, [ceil(T/C), H, dk, dv]) receives S_j, the state
 * ENTERING chunk j, so chunk_states[0] is S0.  Returns 0 or -1.
 */
int orc_linattn_chunked(int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t C,
                        const float* q, const float* k, const float* v,
                        const float* g, double scale, const double* S0,
                        double* o, double* chunk_states, double* S_final)
{
    if (T < 0 || H <= 0 || dk <= 0 || dv <= 0 || C <= 0) return -1;
    const int64_t n_chunks = (T + C - 1) / C;
    double* S = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    double* Snew = (double*)malloc(sizeof(double) * (size_t)(dk * dv));
    double* G = (double*)malloc(sizeof(double) * (size_t)C);
    double* inter = (double*)malloc(sizeof(double) * (size_t)dv);
    if (!S || !Snew || !G || !inter) {
        free(S); free(Snew); free(G); free(inter);
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
            /* inclusive cumulative log-decay inside the chunk */
            double run = 0.0;
            for (int64_t i = 0; i < L; ++i) {
                run += (double)g[(t0 + i) * H + h];
                G[i] = run;
            }
            /* outputs: inter-chunk term through the entering state, plus the
               causal intra-chunk term (the diagonal m == i included) */
            for (int64_t i = 0; i < L; ++i) {
                const int64_t ti = t0 + i;
                for (int64_t j = 0; j < dv; ++j) {
                    double acc = 0.0;
                    for (int64_t d = 0; d < dk; ++d)
                        acc += (double)AT3(q, ti, h, d, H, dk) * S[d * dv + j];
                    inter[j] = exp(G[i]) * acc;
                }
                for (int64_t j = 0; j < dv; ++j) AT3(o, ti, h, j, H, dv) = inter[j];
                for (int64_t m = 0; m <= i; ++m) {
                    const int64_t tm = t0 + m;
                    double qk = 0.0;
                    for (int64_t d = 0; d < dk; ++d)
                        qk += (double)AT3(q, ti, h, d, H, dk) * (double)AT3(k, tm, h, d, H, dk);
                    const double w = exp(G[i] - G[m]) * qk;
                    for (int64_t j = 0; j < dv; ++j)
                        AT3(o, ti, h, j, H, dv) += w * (double)AT3(v, tm, h, j, H, dv);
                }
                for (int64_t j = 0; j < dv; ++j) AT3(o, ti, h, j, H, dv) *= scale;
            }
            /* state fold at the end of the chunk */
            const double chunk_decay = exp(G[L - 1]);
            for (int64_t i = 0; i < dk * dv; ++i) Snew[i] = chunk_decay * S[i];
            for (int64_t m = 0; m < L; ++m) {
                const int64_t tm = t0 + m;
                const double w = exp(G[L - 1] - G[m]);
                for (int64_t d = 0; d < dk; ++d) {
                    const double kd = w * (double)AT3(k, tm, h, d, H, dk);
                    for (int64_t j = 0; j < dv; ++j)
                        Snew[d * dv + j] += kd * (double)AT3(v, tm, h, j, H, dv);
                }
            }
            memcpy(S, Snew, sizeof(double) * (size_t)(dk * dv));
        }
        if (S_final)
            memcpy(S_final + h * dk * dv, S, sizeof(double) * (size_t)(dk * dv));
    }
    free(S); free(Snew); free(G); free(inter);
    return 0;
}
