// Chunked gated delta-rule (Gated DeltaNet) prefill on gfx950.
//
// The paper's hybrid model keeps a Gated DeltaNet state in its linear layers
// (§2 "hybrid recurrent state", §7 model description) without writing the
// recurrence; the standard gated delta rule is taken, per head, with S of
// shape dk x dv and row vectors q_t, k_t (dk) and v_t (dv):
//   S_t = exp(g_t) (I - beta_t k_t^T k_t) S_{t-1} + beta_t k_t^T v_t
//   o_t = scale * q_t S_t
// Chunked form: for a chunk with entering state S, inclusive in-chunk
// log-decay sums G_t and gamma_t = exp(G_t), the pseudo-values U solve
//   (I + A) U = diag(beta) (V - diag(gamma) K S),
//   A_tm = beta_t exp(G_t - G_m) (k_t . k_m) for m < t (strictly lower),
// and then
//   o_t   = scale (gamma_t q_t S + sum_{m<=t} exp(G_t - G_m)(q_t . k_m) u_m)
//   S_new = gamma_last S + sum_m exp(G_last - G_m) k_m^T u_m.
//
// Two launches.
//  1. gdn_prepare, one wave per (chunk, head), all chunks in parallel: A from
//     K K^T on MFMA and T = (I + A)^-1 blockwise in fp32 (the four 16 x 16
//     diagonal blocks by forward substitution, the blocks below them as
//     fp32 MFMA products), written to the workspace as ready MFMA operands.  T
//     depends on the chunk's inputs only -- not on S -- and is the same for
//     every value slice of the head, so it is computed once, off the
//     sequential path.
//  2. gdn_scan, one workgroup of eight waves per (head, 16-column slice of
//     the values), walks the chunks in order.  Column slices are
//     independent: U[:, J], o[:, J] and S[:, J] need only S[:, J] and
//     v[:, J].  Only K S -> R -> U -> S is a true recurrence; it runs on
//     four "chain" waves (row block r of the chunk, rows of S), with three
//     LDS barriers per chunk:
//       phase 1  R_r = beta (V_r - gamma K_r S) -> LDS
//       phase 2  U_r = sum_m T[r rows][m] R_m -> LDS, with w_m U_m
//       phase 3  S <- gamma_last S + K^T (w U) on the wave's rows of S,
//                published for the next chunk.
//     Four "output" waves do the rest beside it: the HBM loads of K, Q and
//     the gate tables (three chunks ahead) and the cooperative L2 prefetch,
//     then gamma Q_r S (from the published S) and the decayed scores
//     P = exp(G_i - G_m)(q_i . k_m), m <= i, of their rows (phase 1),
//     staging the next chunk's K and gate tables (phase 2), and
//     o_r = scale (gamma Q_r S + P U) (phase 3).  The scores are recomputed
//     by every value slice of a head rather than read from the workspace:
//     the slices already hold the chunk's Q and K, and the scan is bound by
//     the lines each workgroup asks L2 for, not by its arithmetic.  The
//     arithmetic applied to a chunk depends only on (S, that chunk's
//     inputs), so a call started at an aligned position from a restored
//     state reproduces one longer call bit for bit.
//
// Every product runs on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
// K and Q are exact bf16 operands; fp32 operands (S, R, U, w U, T, P) are
// split hi + lo in bf16 (three products, or two against an exact operand),
// ~2^-17 relative error per product.  All decays are exp2 of differences of
// G log2(e) with the later token first, so they lie in (0, 1] and nothing
// is divided by a decay.
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "internal.h"

namespace cap {
namespace {

using namespace dev;

constexpr int CH = 64;       // chunk length
constexpr int DVS = 16;      // value columns per scan workgroup
constexpr int NW = 4;        // waves per role of the scan workgroup
constexpr int ATP = CH + 4;  // pitch (floats) of the A^T rows in the prepare kernel

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ inline float f32_of(uint32_t u) { return __builtin_bit_cast(float, u); }

// ------------------------------------------------------------------ prepare
// One wave per (chunk c, head h): T = (I + A)^-1 and the gate tables into
// the workspace record of (c, h).  Rows past the last token have k = 0,
// beta = 0 and g = 0, so their rows and columns of A vanish and T is the
// identity there.  T does not depend on the state and is the same for every
// value slice of the head.
//
// Record layout (the scan's chain wave for row block r reads block (r, i)
// for i <= r / 2): block (r, i) = index r for r < 2, else 2 r - 2 + i;
// 2 KiB each, the bf16 hi plane then the lo plane, lane l = 16 grp + li at
// byte 16 l of its plane holding T[16 r + li][32 i + 8 grp + e], e = 0..7.
// Six blocks, then G log2(e) (64 fp32) and beta (64 fp32).
template <int DK>
__global__ __launch_bounds__(64) void gdn_prepare_kernel(const GdnParams p) {
    constexpr int NKK = DK / 32;
    __shared__ alignas(16) float at[CH * ATP];  // A^T [m][t]
    __shared__ alignas(16) float tg[CH];        // G_t log2(e)
    __shared__ alignas(16) float tb[CH];        // beta_t
    const int lane = threadIdx.x, li = lane & 15, grp = lane >> 4;
    const int H = p.H;
    const int64_t c = blockIdx.x / H;
    const int h = (int)(blockIdx.x - c * H);
    const int64_t t0 = c * CH, rows = p.T - t0;
    const int64_t krow = (int64_t)H * DK * 2;

    // key operands: kr[r][kk] holds k[16 r + li][32 kk + 8 grp .. +7], which is
    // both the A operand of row block r and the B operand of K_r^T
    const rsrc_t rk = make_rsrc(static_cast<const char*>(p.k) + t0 * krow, rows * krow);
    u32x4 kr[4][NKK];
    #pragma unroll
    for (int r = 0; r < 4; ++r)
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
            kr[r][kk] = __builtin_amdgcn_raw_buffer_load_b128(
                rk, (uint32_t)((16 * r + li) * krow + ((int64_t)h * DK + 32 * kk + 8 * grp) * 2), 0, 0);
    const rsrc_t rg = make_rsrc(p.g + t0 * H, rows * H * 4);
    const rsrc_t rb = make_rsrc(p.beta + t0 * H, rows * H * 4);
    const float gl = f32_of(__builtin_amdgcn_raw_buffer_load_b32(rg, (uint32_t)((lane * H + h) * 4), 0, 0));
    const float bl = f32_of(__builtin_amdgcn_raw_buffer_load_b32(rb, (uint32_t)((lane * H + h) * 4), 0, 0));
    tg[lane] = wave_inclusive_sum(gl) * LOG2E;
    tb[lane] = bl;
    __syncthreads();

    // A = diag(beta) (K K^T o exp(G_t - G_m)), strictly lower, stored as A^T
    #pragma unroll
    for (int r = 0; r < 4; ++r) {
        const f32x4 gt = *reinterpret_cast<const f32x4*>(&tg[16 * r + 4 * grp]);
        const f32x4 bt = *reinterpret_cast<const f32x4*>(&tb[16 * r + 4 * grp]);
        #pragma unroll
        for (int s = 0; s <= r; ++s) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk)
                acc = mma(__builtin_bit_cast(bf16x8, kr[r][kk]), __builtin_bit_cast(bf16x8, kr[s][kk]), acc);
            const int m = 16 * s + li;  // acc[q] = k_t . k_m, t = 16 r + 4 grp + q
            const float gm = tg[m];
            f32x4 a;
            #pragma unroll
            for (int q = 0; q < 4; ++q)
                a[q] = (16 * r + 4 * grp + q > m) ? bt[q] * __builtin_amdgcn_exp2f(gt[q] - gm) * acc[q] : 0.0f;
            *reinterpret_cast<f32x4*>(&at[m * ATP + 16 * r + 4 * grp]) = a;
        }
    }

    uint8_t* rec = p.ws + (c * H + h) * kGdnWsRecord;
    __syncthreads();

    // T = (I + A)^-1 by 16-row blocks.  `at` holds A^T above its diagonal
    // (at[m][t] = A[t][m], t > m); T is stored row-major on and below the
    // diagonal (at[t][m] = T[t][m], t >= m), so both live in one buffer.  T
    // is lower triangular: its entries above the diagonal are never stored
    // and every read of T masks them to zero.
    //  1. T_ii = (I + A_ii)^-1 for the four diagonal blocks by forward
    //     substitution in fp32, lane 16 i + j holding column j of block i;
    //  2. T_ij = -T_ii (sum_{k=j}^{i-1} A_ik T_kj) for i > j, one block
    //     diagonal d = i - j after the other, on v_mfma_f32_16x16x4_f32 (lane
    //     l feeds A[l % 16][l / 16] and B[l / 16][l % 16] and receives
    //     D[4 (l / 16) + r][l % 16]; fp32 products and sums).
    auto tval = [&](int row, int col) -> float { return col <= row ? at[row * ATP + col] : 0.0f; };
    {
        const int bi = grp, j = li;
        float x[16];
        #pragma unroll
        for (int t = 0; t < 16; ++t) x[t] = (t == j) ? 1.0f : 0.0f;
        #pragma unroll
        for (int m = 0; m < 15; ++m) {
            const float xm = x[m];
            #pragma unroll
            for (int t4 = (m + 1) / 4; t4 < 4; ++t4) {
                const f32x4 a = *reinterpret_cast<const f32x4*>(&at[(16 * bi + m) * ATP + 16 * bi + 4 * t4]);
                #pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * t4 + e > m) x[4 * t4 + e] = fmaf(-a[e], xm, x[4 * t4 + e]);
            }
        }
        #pragma unroll
        for (int t = 0; t < 16; ++t)
            if (t >= j) at[(16 * bi + t) * ATP + 16 * bi + j] = x[t];
    }
    __syncthreads();
    #pragma unroll
    for (int d = 1; d < 4; ++d) {
        // M_ij = sum_k A_ik T_kj, parked in T_ij's own place
        #pragma unroll
        for (int bj = 0; bj + d < 4; ++bj) {
            const int bi = bj + d;
            f32x4 m4 = {0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int k = bj; k < bi; ++k)
                #pragma unroll
                for (int s4 = 0; s4 < 4; ++s4) {
                    const int sx = 16 * k + 4 * s4 + grp;
                    m4 = __builtin_amdgcn_mfma_f32_16x16x4f32(at[sx * ATP + 16 * bi + li], tval(sx, 16 * bj + li), m4, 0,
                                                             0, 0);
                }
            #pragma unroll
            for (int r = 0; r < 4; ++r) at[(16 * bi + 4 * grp + r) * ATP + 16 * bj + li] = m4[r];
        }
        __syncthreads();
        // T_ij = -T_ii M_ij over M_ij (each lane's stores follow its reads)
        #pragma unroll
        for (int bj = 0; bj + d < 4; ++bj) {
            const int bi = bj + d;
            f32x4 t4 = {0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int sx = 4 * s4 + grp;
                t4 = __builtin_amdgcn_mfma_f32_16x16x4f32(tval(16 * bi + li, 16 * bi + sx),
                                                         at[(16 * bi + sx) * ATP + 16 * bj + li], t4, 0, 0, 0);
            }
            #pragma unroll
            for (int r = 0; r < 4; ++r) at[(16 * bi + 4 * grp + r) * ATP + 16 * bj + li] = -t4[r];
        }
        __syncthreads();
    }
    // the causal blocks of T in operand order, split hi/lo
    #pragma unroll
    for (int r = 0; r < 4; ++r)
        #pragma unroll
        for (int i = 0; i <= r / 2; ++i) {
            const int blk = r < 2 ? r : 2 * r - 2 + i;
            const int row = 16 * r + li, col = 32 * i + 8 * grp;
            float f[8];
            #pragma unroll
            for (int e = 0; e < 8; ++e) f[e] = tval(row, col + e);
            bf16x8 hi, lo;
            split_n<8>(f, hi, lo);
            *reinterpret_cast<bf16x8*>(rec + blk * 2048 + 16 * lane) = hi;
            *reinterpret_cast<bf16x8*>(rec + blk * 2048 + 1024 + 16 * lane) = lo;
        }
    float* tab = reinterpret_cast<float*>(rec + kGdnWsTabOff);
    tab[lane] = tg[lane];
    tab[CH + lane] = tb[lane];
}

// --------------------------------------------------------------------- scan
constexpr int NT = 2 * 64 * NW;  // threads per scan workgroup: output waves 0-3, chain waves 4-7
constexpr int NO_T = 64 * NW;    // threads of the output role

template <int DK>
struct alignas(16) GdnSmem {
    // K rows are read 16 rows x 16 B at a time and, transposed, 4 rows x
    // 32 B at a time: a pitch of 16 B times an odd number whose 4-row windows
    // do not overlap keeps both conflict-free.
    static constexpr int KP = DK == 128 ? 152 : 104;
    static constexpr int JP = DVS + 8;    // row pitch (elements) of the [*][j] tiles
    alignas(16) __bf16 k[2][CH * KP];     // K [m][d] by chunk parity
    alignas(16) __bf16 s[2][DK * JP];     // S [d][j]: hi, lo
    alignas(16) __bf16 r[2][CH * JP];     // R [m][j]: hi, lo
    alignas(16) __bf16 u[2][CH * JP];     // U [m][j]: hi, lo
    alignas(16) __bf16 wu[2][CH * JP];    // w U [m][j], w_m = exp(G_last - G_m): hi, lo
    alignas(16) float tab[2][2 * CH];     // by chunk parity: G_m log2(e) (0..63), beta_m (64..127)
    // decay factors of the scores below the diagonal blocks, by chunk
    // parity: exp(G_e - G_m) with e the last token of m's 16-token block,
    // and exp(G_i - G_e(M)) for the blocks M before i's (0 elsewhere)
    alignas(16) float bm[2][CH];
    alignas(16) float ai[2][CH][4];
};

struct GdnCtx {
    int h, j0, H, dv, lane, li, grp;
    int nfull, tail;               // full chunks, rows of the partial last one
    int64_t T, n;                  // tokens, chunks
    int64_t qk_row, v_row, o_row;  // bytes per token of q / k, v, o
};

// Valid rows of chunk c: CH up to the last full chunk, then the tail, then 0
// (chunks past the end), in 32-bit arithmetic (the host bounds the chunk
// count below 2^31 and a chunk's bytes of any tensor below 2^31).
__device__ inline uint32_t chunk_rows(const GdnCtx& x, int64_t c) {
    const int ci = (int)c;
    return ci < x.nfull ? (uint32_t)CH : (ci == x.nfull ? (uint32_t)x.tail : 0u);
}

// Every product is computed transposed, with the value column j as the row
// index of the accumulator: lane (grp, li) then holds four consecutive
// columns j = 4 grp .. 4 grp + 3 of one token or one row of S, so v is read,
// and o and the states are written, with one 8- or 16-byte access per lane
// instead of one per element (the memory pipeline, not the arithmetic, is
// what the scan waits on).  Tiles indexed [*][j] sit in LDS row-major and
// are read as operands with the transposing LDS load.
//
// The output role walks the chunks four steps per loop iteration, so its
// register stages (loads three chunks ahead) rotate without copies; the
// chain role loads one chunk ahead, by which time the output role's L2
// prefetch has the lines in L2.  Every global access of a step is issued
// unconditionally -- chunks past the end get empty buffer ranges: loads read
// zeros, stores are dropped -- so the in-order memory counters stay exact.
// A step past the end changes no state, writes only LDS buffers no live
// step reads, and skips its barriers.  A call of at most one chunk (ONE)
// runs the step once, without prefetch.

// ------------------------------------------------------------ output role
// Wave R owns rows i = 16 R..16 R + 15 of the chunk: in phase 1 it forms
// (gamma X)^T = (gamma Q_R S)^T from the published S and the decayed scores
// of its rows, P^T = (K Q_R^T) o exp(G_i - G_m) (m <= i), whose accumulators
// serve as they are as the B operand of U^T P^T; in phase 3,
// o^T = scale ((gamma X)^T + U^T P^T).  The role also loads K (all rows) and
// stages it in LDS, wave 0 stages the gate tables and waves 1 and 2 run the
// cooperative L2 prefetch.
template <int DK, int R>
struct OutStage {
    static constexpr int PK = CH * DK / 8 / NO_T;  // 16-byte K pieces per thread
    u32x4 kp[PK];       // K pieces, coalesced (consecutive threads: consecutive bytes of a row)
    u32x4 q[DK / 32];   // q[16 R + li][32 kk + 8 grp .. +7]
    float tab[2];       // wave 0: entries 2 lane, 2 lane + 1 of the gate tables
};

template <int DK, bool ONE, int R>
__device__ __forceinline__ void out_role(const GdnParams& p, GdnSmem<DK>& sm, const GdnCtx& x) {
    using Sm = GdnSmem<DK>;
    using St = OutStage<DK, R>;
    constexpr int KP = Sm::KP, JP = Sm::JP, PK = St::PK;
    constexpr int NKK = DK / 32, NT2 = R / 2 + 1;
    const int lane = x.lane, li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;
    const int ot = 64 * R + lane;

    auto load = [&](St& S_, int64_t c) {
        const int64_t t0 = c * CH;
        const uint32_t rows = chunk_rows(x, c);
        const rsrc_t rk = make_rsrc_u32(static_cast<const char*>(p.k) + t0 * x.qk_row, rows * (uint32_t)x.qk_row);
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = ot + NO_T * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            S_.kp[u] = __builtin_amdgcn_raw_buffer_load_b128(rk, (uint32_t)(m * x.qk_row + ((int64_t)h * DK + d0) * 2), 0, 0);
        }
        const rsrc_t rq = make_rsrc_u32(static_cast<const char*>(p.q) + t0 * x.qk_row, rows * (uint32_t)x.qk_row);
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
            S_.q[kk] = __builtin_amdgcn_raw_buffer_load_b128(
                rq, (uint32_t)((16 * R + li) * x.qk_row + ((int64_t)h * DK + 32 * kk + 8 * grp) * 2), 0, 0);
        const bool live = c < x.n;
        const uint8_t* rec = p.ws + (live ? (c * H + h) * kGdnWsRecord : 0);
        if constexpr (R == 0) {
            const rsrc_t rt = make_rsrc_u32(rec + kGdnWsTabOff, live ? 2u * CH * 4 : 0u);
            const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rt, (uint32_t)(8 * lane), 0, 0);
            const uint32_t v0 = v[0], v1 = v[1];
            S_.tab[0] = f32_of(v0);
            S_.tab[1] = f32_of(v1);
        }
    };

    // K rows into LDS buffer bk; wave 0 also the gate tables
    auto stage = [&](const St& S_, int bk) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = ot + NO_T * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            *reinterpret_cast<u32x4*>(&sm.k[bk][m * KP + d0]) = S_.kp[u];
        }
        if constexpr (R == 0) {
            sm.tab[bk][2 * lane] = S_.tab[0];
            sm.tab[bk][2 * lane + 1] = S_.tab[1];
            // the factored decay (lane t: token t); both factors in (0, 1]
            const float g = sm.tab[bk][lane];
            const int blk = lane >> 4;
            float ge[4];
            #pragma unroll
            for (int M = 0; M < 4; ++M) ge[M] = sm.tab[bk][16 * M + 15];
            sm.bm[bk][lane] = __builtin_amdgcn_exp2f(ge[blk] - g);
            f32x4 a;
            #pragma unroll
            for (int M = 0; M < 4; ++M) a[M] = (M < blk) ? __builtin_amdgcn_exp2f(g - ge[M]) : 0.0f;
            *reinterpret_cast<f32x4*>(&sm.ai[bk][lane][0]) = a;
        }
    };

    // Cooperative L2 prefetch.  The 16-column slices of a head all read the
    // head's K, Q and workspace lines and share the lines of V; requested by
    // every slice at the same moment, each miss costs every workgroup a full
    // HBM latency.  So waves 1 and 2 of each slice touch the slice's share of
    // the head's lines of chunk c + PREFETCH (the workspace record, then K,
    // Q and V rows; line L goes to slice L % NS), two chunks ahead of the
    // output role's loads, and the sibling slices' loads then hit in L2.  The
    // fetched word is consumed only as an asm operand four steps later,
    // which forces nothing but the load's completion.
    constexpr int PREFETCH = 5;
    uint32_t pf[4] = {0u, 0u, 0u, 0u};
    // The lane's line, fixed for the call: kind 0 the workspace record,
    // 1 K, 2 Q, 3 V, 4 none; its row in the chunk and byte offset in the row
    // (or in the record).
    int pkind = 4, prow = 0;
    int64_t poff = 0;
    if constexpr (R == 1 || R == 2) {
        const int ns = dv / DVS;
        const int L = j0 / DVS + ns * (64 * (R - 1) + lane);
        constexpr int LK = DK * 2 / 128;            // 128-byte lines per row of K or Q
        const int LV = (dv * 2 + 127) / 128;        // lines per row of the head's V
        constexpr int nR = (int)((kGdnWsRecord + 127) / 128);
        const int nK = CH * LK, nV = CH * LV;
        if (L < nR) {
            pkind = 0;
            poff = (int64_t)L * 128;
        } else if (L < nR + 2 * nK) {
            const int l = L - nR;
            const int lq = l < nK ? l : l - nK;
            pkind = l < nK ? 1 : 2;
            prow = lq / LK;
            poff = (int64_t)h * DK * 2 + (lq % LK) * 128;
        } else if (L < nR + 2 * nK + nV) {
            const int l = L - nR - 2 * nK;
            pkind = 3;
            prow = l / LV;
            poff = (int64_t)h * dv * 2 + (l % LV) * 128;
        }
    }
    const char* const pbase = pkind == 1 ? static_cast<const char*>(p.k)
                            : pkind == 2 ? static_cast<const char*>(p.q)
                                         : static_cast<const char*>(p.v);
    const int64_t prow_bytes = pkind == 3 ? x.v_row : x.qk_row;
    auto prefetch = [&](int slot, int64_t c) {
        __asm__ volatile("" : : "v"(pf[slot]));
        const char* a = static_cast<const char*>(p.k);  // in bounds whenever the loop runs
        if (pkind == 0) {
            if (c < x.n) a = reinterpret_cast<const char*>(p.ws) + (c * H + h) * kGdnWsRecord + poff;
        } else if (pkind < 4) {
            if (prow < (int)chunk_rows(x, c)) a = pbase + (c * CH + prow) * prow_bytes + poff;
        }
        pf[slot] = *reinterpret_cast<const uint32_t*>(a);
    };

    auto step = [&](int64_t c, const St& cur, const St& nxt, St& ld, int slot) {
        const bool live = c < x.n;
        const int b = (int)(c & 1);
        const __bf16* kb = sm.k[b];
        const int64_t t0 = c * CH;
        if constexpr (!ONE) load(ld, c + 3);
        if constexpr (!ONE && (R == 1 || R == 2)) prefetch(slot, c + PREFETCH);

        // ---- phase 1: (gamma X)^T = (gamma Q_R S)^T from the published S
        // (element e of the S^T operand of step kk is d = 32 kk + 8 grp + e),
        // and the scores K Q_R^T: accumulator mb holds (k_m . q_i) for
        // m = 16 mb + 4 grp + r, i = 16 R + li
        bf16x8 qo[NKK];
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) qo[kk] = __builtin_bit_cast(bf16x8, cur.q[kk]);
        f32x4 xh = {0.f, 0.f, 0.f, 0.f}, xl = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const int d0 = 32 * kk + 8 * grp;
            const bf16x8 sh = cat(tr4(sm.s[0], JP, d0, 0, li), tr4(sm.s[0], JP, d0 + 4, 0, li));
            const bf16x8 sl = cat(tr4(sm.s[1], JP, d0, 0, li), tr4(sm.s[1], JP, d0 + 4, 0, li));
            xh = mma(sh, qo[kk], xh);
            xl = mma(sl, qo[kk], xl);
        }
        f32x4 sc[R + 1];
        #pragma unroll
        for (int mb = 0; mb <= R; ++mb) {
            sc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk)
                sc[mb] = mma(*reinterpret_cast<const bf16x8*>(&kb[(16 * mb + li) * KP + 32 * kk + 8 * grp]), qo[kk],
                             sc[mb]);
        }
        // P^T = scores o exp(G_i - G_m) for m <= i, as the B operand of
        // U^T P^T: element e of step i2 is m = 32 i2 + 16 (e / 4) + 4 grp + e % 4
        // below the diagonal block exp(G_i - G_m) = exp(G_i - G_e) exp(G_e - G_m)
        // from the tables; on it exp2 of the difference, masked to m <= i
        const float g2i = sm.tab[b][16 * R + li];
        const f32x4 aiv = *reinterpret_cast<const f32x4*>(&sm.ai[b][16 * R + li][0]);
        bf16x8 ph[NT2], pl[NT2];
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            float f[8];
            #pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int mb = 2 * i2 + half;
                if (mb > R) {
                    #pragma unroll
                    for (int q = 0; q < 4; ++q) f[4 * half + q] = 0.0f;
                    continue;
                }
                if (mb < R) {
                    const f32x4 bmv = *reinterpret_cast<const f32x4*>(&sm.bm[b][16 * mb + 4 * grp]);
                    #pragma unroll
                    for (int q = 0; q < 4; ++q) f[4 * half + q] = (sc[mb][q] * aiv[mb]) * bmv[q];
                } else {
                    const f32x4 gm = *reinterpret_cast<const f32x4*>(&sm.tab[b][16 * mb + 4 * grp]);
                    #pragma unroll
                    for (int q = 0; q < 4; ++q)
                        f[4 * half + q] = (4 * grp + q <= li) ? sc[mb][q] * __builtin_amdgcn_exp2f(g2i - gm[q]) : 0.0f;
                }
            }
            split_n<8>(f, ph[i2], pl[i2]);
        }
        f32x4 oa;
        {
            const float gam = __builtin_amdgcn_exp2f(g2i);
            #pragma unroll
            for (int q = 0; q < 4; ++q) oa[q] = gam * (xh[q] + xl[q]);
        }
        if (live) lds_barrier();

        // ---- phase 2: stage chunk c+1
        if constexpr (!ONE) stage(nxt, b ^ 1);
        if (live) lds_barrier();

        // ---- phase 3: o^T = scale ((gamma X)^T + U^T P^T); element e of the
        // U^T operand of step i2 is m = 32 i2 + 16 (e / 4) + 4 grp + e % 4, the
        // order of the P^T operand
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            const int m0 = 32 * i2 + 4 * grp;
            const bf16x8 uh = cat(tr4(sm.u[0], JP, m0, 0, li), tr4(sm.u[0], JP, m0 + 16, 0, li));
            const bf16x8 ul = cat(tr4(sm.u[1], JP, m0, 0, li), tr4(sm.u[1], JP, m0 + 16, 0, li));
            oa = mma(uh, ph[i2], oa);
            oa = mma(ul, ph[i2], oa);
            oa = mma(uh, pl[i2], oa);
        }
        const rsrc_t ro = make_rsrc_u32(static_cast<char*>(static_cast<void*>(p.o)) + t0 * x.o_row,
                                        chunk_rows(x, c) * (uint32_t)x.o_row);
        f32x4 os;
        #pragma unroll
        for (int q = 0; q < 4; ++q) os[q] = oa[q] * p.scale;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, os), ro,
                                               (uint32_t)((16 * R + li) * x.o_row + ((int64_t)h * dv + j0 + 4 * grp) * 4), 0, 0);
        if (live) lds_barrier();
    };

    if constexpr (ONE) {
        St s0;
        load(s0, 0);
        stage(s0, 0);
        lds_barrier();
        if (x.n == 1) step(0, s0, s0, s0, 0);
    } else {
        St s0, s1, s2, s3;
        load(s0, 0);
        load(s1, 1);
        load(s2, 2);
        stage(s0, 0);
        lds_barrier();
        for (int64_t c = 0; c < x.n; c += 4) {
            step(c, s0, s1, s3, 0);
            step(c + 1, s1, s2, s0, 1);
            step(c + 2, s2, s3, s1, 2);
            step(c + 3, s3, s0, s2, 3);
        }
    }
}

// ------------------------------------------------------------- chain role
// Wave R owns rows 16 R..16 R + 15 of the chunk and rows
// 16 R NDW..16 (R + 1) NDW - 1 of S (fp32, in registers): (K_R S)^T -> R
// (phase 1), U_R^T = R^T T[R rows]^T (phase 2), S^T <- gamma_last S^T +
// (w U)^T K on its rows of S, published for the next chunk (phase 3).  Only
// this role's work is on the state's sequential path.
template <int DK, int R>
struct ChainStage {
    static constexpr int NT2 = R / 2 + 1;
    u32x4 t[NT2][2];    // T[16 R + li][32 i + 8 grp .. +7]: bf16 hi, lo
    u32x2 v;            // bf16 v[16 R + li][j0 + 4 grp .. +3]
};

template <int DK, bool ONE, int R>
__device__ __forceinline__ void chain_role(const GdnParams& p, GdnSmem<DK>& sm, const GdnCtx& x) {
    using Sm = GdnSmem<DK>;
    using St = ChainStage<DK, R>;
    constexpr int KP = Sm::KP, JP = Sm::JP;
    constexpr int NKK = DK / 32, NDW = DK / 64, NT2 = St::NT2;
    const int li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;

    // state tiles in transposed accumulator layout: S[u][q] = S[d][j0 + 4 grp
    // + q] with d = 16 (R NDW + u) + li -- 16 contiguous bytes of a state row
    f32x4 S[NDW];
    auto srow = [&](int u) -> int64_t {  // element offset of S[d][j0 + 4 grp] in a [H][dk][dv] state
        return ((int64_t)h * DK + 16 * (R * NDW + u) + li) * dv + j0 + 4 * grp;
    };
    #pragma unroll
    for (int u = 0; u < NDW; ++u)
        S[u] = p.state_in ? *reinterpret_cast<const f32x4*>(p.state_in + srow(u)) : f32x4{0.f, 0.f, 0.f, 0.f};

    auto load = [&](St& S_, int64_t c) {
        const int64_t t0 = c * CH;
        const rsrc_t rv = make_rsrc_u32(static_cast<const char*>(p.v) + t0 * x.v_row,
                                        chunk_rows(x, c) * (uint32_t)x.v_row);
        S_.v = __builtin_amdgcn_raw_buffer_load_b64(
            rv, (uint32_t)((16 * R + li) * x.v_row + ((int64_t)h * dv + j0 + 4 * grp) * 2), 0, 0);
        const bool live = c < x.n;
        const rsrc_t rt = make_rsrc_u32(p.ws + (live ? (c * H + h) * kGdnWsRecord : 0),
                                        live ? (uint32_t)kGdnWsTBytes : 0u);
        #pragma unroll
        for (int i = 0; i < NT2; ++i) {
            const int blk = R < 2 ? R : 2 * R - 2 + i;
            #pragma unroll
            for (int pl = 0; pl < 2; ++pl)
                S_.t[i][pl] = __builtin_amdgcn_raw_buffer_load_b128(rt, (uint32_t)(blk * 2048 + pl * 1024 + 16 * x.lane), 0, 0);
        }
    };

    // this wave's rows of S as bf16 hi/lo planes of S [d][j]
    auto publish_s = [&]() {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = 16 * (R * NDW + u) + li;
            const float f[4] = {S[u][0], S[u][1], S[u][2], S[u][3]};
            bf16x4 hi, lo;
            split_n<4>(f, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.s[0][d * JP + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.s[1][d * JP + 4 * grp]) = lo;
        }
    };

    // the chain waves carry the sequential path: issue their instructions
    // first when they compete with the output wave on the same SIMD
    __builtin_amdgcn_s_setprio(2);
    const int64_t state_elems = (int64_t)H * DK * dv;
    auto step = [&](int64_t c, const St& cur, St& ld) {
        const bool live = c < x.n;
        const int b = (int)(c & 1);
        const __bf16* kb = sm.k[b];

        // operands and decays that do not depend on S (token m = 16 R + li)
        bf16x8 th[NT2], tl[NT2];
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            th[i2] = __builtin_bit_cast(bf16x8, cur.t[i2][0]);
            tl[i2] = __builtin_bit_cast(bf16x8, cur.t[i2][1]);
        }
        const float g2 = sm.tab[b][16 * R + li], bt = sm.tab[b][CH + 16 * R + li];
        const float g2l = sm.tab[b][CH - 1];
        const float gam = __builtin_amdgcn_exp2f(g2), wm = __builtin_amdgcn_exp2f(g2l - g2), gl = __builtin_amdgcn_exp2f(g2l);
        const uint32_t v0 = cur.v[0], v1 = cur.v[1];
        const float vv[4] = {f32_of(v0 << 16), f32_of(v0 & 0xFFFF0000u), f32_of(v1 << 16), f32_of(v1 & 0xFFFF0000u)};

        // ---- phase 1: R^T = beta (V - gamma K_R S_c)^T (element e of the S^T
        // operand of step kk is d = 32 kk + 8 grp + e)
        f32x4 kh = {0.f, 0.f, 0.f, 0.f}, kl = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const int d0 = 32 * kk + 8 * grp;
            const bf16x8 sh = cat(tr4(sm.s[0], JP, d0, 0, li), tr4(sm.s[0], JP, d0 + 4, 0, li));
            const bf16x8 sl = cat(tr4(sm.s[1], JP, d0, 0, li), tr4(sm.s[1], JP, d0 + 4, 0, li));
            const bf16x8 ko = *reinterpret_cast<const bf16x8*>(&kb[(16 * R + li) * KP + d0]);
            kh = mma(sh, ko, kh);
            kl = mma(sl, ko, kl);
        }
        // the next chunk's loads go after this phase's LDS reads, so a full
        // memory pipeline cannot hold those reads back
        if constexpr (!ONE) load(ld, c + 1);
        {
            float rr[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) rr[q] = bt * (vv[q] - gam * (kh[q] + kl[q]));
            bf16x4 hi, lo;
            split_n<4>(rr, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.r[0][(16 * R + li) * JP + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.r[1][(16 * R + li) * JP + 4 * grp]) = lo;
        }
        if (live) lds_barrier();

        // ---- phase 2: U_R^T = R^T T[R rows]^T, and (w U_R)^T
        bf16x8 kt[NDW][2];  // K operands of the update (element e: m = 32 mm + 8 grp + e)
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            #pragma unroll
            for (int mm = 0; mm < 2; ++mm) {
                const int m0 = 32 * mm + 8 * grp, d0 = 16 * (R * NDW + u);
                kt[u][mm] = cat(tr4(kb, KP, m0, d0, li), tr4(kb, KP, m0 + 4, d0, li));
            }
        f32x4 ua = {0.f, 0.f, 0.f, 0.f}, ub = {0.f, 0.f, 0.f, 0.f}, uc = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            const int m0 = 32 * i2 + 8 * grp;
            const bf16x8 rh = cat(tr4(sm.r[0], JP, m0, 0, li), tr4(sm.r[0], JP, m0 + 4, 0, li));
            const bf16x8 rl = cat(tr4(sm.r[1], JP, m0, 0, li), tr4(sm.r[1], JP, m0 + 4, 0, li));
            ua = mma(rh, th[i2], ua);
            ub = mma(rl, th[i2], ub);
            uc = mma(rh, tl[i2], uc);
        }
        {
            float uf[4], wf[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) {
                uf[q] = ua[q] + (ub[q] + uc[q]);
                wf[q] = uf[q] * wm;
            }
            bf16x4 hi, lo;
            split_n<4>(uf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.u[0][(16 * R + li) * JP + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.u[1][(16 * R + li) * JP + 4 * grp]) = lo;
            split_n<4>(wf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.wu[0][(16 * R + li) * JP + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.wu[1][(16 * R + li) * JP + 4 * grp]) = lo;
        }
        if (live) lds_barrier();

        // ---- phase 3: S_c to chunk_states[c]; S^T <- gamma_last S^T + (w U)^T K
        const rsrc_t rc = make_rsrc_u32(p.chunk_states + (live ? c : 0) * state_elems,
                                        live && p.chunk_states ? (uint32_t)(state_elems * 4) : 0u);
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, S[u]), rc, (uint32_t)(srow(u) * 4), 0, 0);
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            f32x4 ah, al = {0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int q = 0; q < 4; ++q) ah[q] = gl * S[u][q];
            #pragma unroll
            for (int mm = 0; mm < 2; ++mm) {
                const int m0 = 32 * mm + 8 * grp;
                const bf16x8 wh = cat(tr4(sm.wu[0], JP, m0, 0, li), tr4(sm.wu[0], JP, m0 + 4, 0, li));
                const bf16x8 wl = cat(tr4(sm.wu[1], JP, m0, 0, li), tr4(sm.wu[1], JP, m0 + 4, 0, li));
                ah = mma(wh, kt[u][mm], ah);
                al = mma(wl, kt[u][mm], al);
            }
            if (live) S[u] = ah + al;
        }
        publish_s();
        if (live) lds_barrier();
    };

    if constexpr (ONE) {
        St s0;
        load(s0, 0);
        publish_s();
        lds_barrier();
        if (x.n == 1) step(0, s0, s0);
    } else {
        // one chunk ahead is enough here: the output role's prefetch has the
        // lines in L2 by then
        St s0, s1;
        load(s0, 0);
        publish_s();
        lds_barrier();
        for (int64_t c = 0; c < x.n; c += 2) {
            step(c, s0, s1);
            step(c + 1, s1, s0);
        }
    }
    if (p.final_state) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) *reinterpret_cast<f32x4*>(p.final_state + srow(u)) = S[u];
    }
}

template <int DK, bool ONE>
__global__ __launch_bounds__(NT) void gdn_scan_kernel(const GdnParams p) {
    __shared__ GdnSmem<DK> sm;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // workgroup -> (head, slice); slices of one head share an XCD (and its
    // L2) when the grid allows it (workgroups go round-robin over 8 XCDs)
    GdnCtx x;
    x.H = p.H;
    x.dv = p.dv;
    const int NS = x.dv / DVS;
    const int N = x.H * NS;
    int logical = blockIdx.x;
    if ((N % 8) == 0 && ((N / 8) % NS) == 0) logical = (blockIdx.x % 8) * (N / 8) + blockIdx.x / 8;
    x.h = logical / NS;
    x.j0 = (logical % NS) * DVS;
    x.lane = tid & 63;
    x.li = x.lane & 15;
    x.grp = x.lane >> 4;
    x.T = p.T;
    x.n = (p.T + CH - 1) / CH;
    x.nfull = (int)(p.T / CH);
    x.tail = (int)(p.T % CH);
    x.qk_row = (int64_t)x.H * DK * 2;
    x.v_row = (int64_t)x.H * x.dv * 2;
    x.o_row = (int64_t)x.H * x.dv * 4;

    // waves w and w + 4 share a SIMD: the chain wave with the most causal
    // rows (block 3) pairs with the output wave with the fewest (block 0)
    switch (wave) {
        case 0: out_role<DK, ONE, 0>(p, sm, x); break;
        case 1: out_role<DK, ONE, 1>(p, sm, x); break;
        case 2: out_role<DK, ONE, 2>(p, sm, x); break;
        case 3: out_role<DK, ONE, 3>(p, sm, x); break;
        case 4: chain_role<DK, ONE, 3>(p, sm, x); break;
        case 5: chain_role<DK, ONE, 2>(p, sm, x); break;
        case 6: chain_role<DK, ONE, 1>(p, sm, x); break;
        default: chain_role<DK, ONE, 0>(p, sm, x); break;
    }
}

template <int DK>
hipError_t launch_t(const GdnParams& p, hipStream_t stream) {
    const int64_t n = (p.T + CH - 1) / CH;
    if (n > 0) {
        const hipError_t e = launch_kernel(reinterpret_cast<const void*>(&gdn_prepare_kernel<DK>),
                                           dim3((unsigned)(n * p.H)), dim3(64), p, stream);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)(p.H * (p.dv / DVS)));
    const void* fn = p.T <= CH ? reinterpret_cast<const void*>(&gdn_scan_kernel<DK, true>)
                               : reinterpret_cast<const void*>(&gdn_scan_kernel<DK, false>);
    return launch_kernel(fn, grid, dim3(NT), p, stream);
}

}  // namespace

hipError_t launch_gdn(const GdnParams& p, hipStream_t stream) {
    if (p.dk == 128) return launch_t<128>(p, stream);
    if (p.dk == 64) return launch_t<64>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
