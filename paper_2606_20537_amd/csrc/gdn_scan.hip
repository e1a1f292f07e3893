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
//     K K^T on MFMA, then T = (I + A)^-1 by forward substitution in fp32
//     (lane j owns column j), written to the workspace.  T depends on the
//     chunk's keys, gates and write strengths only -- not on S -- and is the
//     same for every value slice of the head, so it is computed once, off
//     the sequential path.
//  2. gdn_scan, one workgroup of eight waves per (head, 16-column slice of
//     the values), walks the chunks in order.  Column slices are
//     independent: U[:, J], o[:, J] and S[:, J] need only S[:, J] and
//     v[:, J].  Only K S -> R -> U -> S is a true recurrence; it runs on
//     four "chain" waves (row block r of the chunk, rows of S), with three
//     LDS barriers per chunk:
//       phase 1  R_r = beta (V_r - gamma K_r S) -> LDS
//       phase 2  U_r = sum_m T[r rows][m] R_m -> LDS, with w_m U_m
//       phase 3  S <- gamma_last S + K^T (w U) on the wave's rows of S,
//                published as S^T for the next chunk.
//     Four "output" waves do everything else beside it: X = Q_r S
//     (phase 1), the decayed scores of their rows and the staging of the
//     next chunk's K and gate tables (phase 2), o_r = scale (gamma X + P U)
//     (phase 3), and the HBM loads three chunks ahead.  The arithmetic
//     applied to a chunk depends only on (S, that chunk's inputs), so a
//     call started at an aligned position from a restored state reproduces
//     one longer call bit for bit.
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
// identity there.
//
// Record layout (the scan's chain wave r reads block (r, i) for i <= r / 2):
// block (r, i) = index r for r < 2, else 2 r - 2 + i; 2 KiB each, the bf16
// hi plane then the lo plane, lane l = 16 grp + li holding
// T[16 r + li][32 i + 8 grp .. +7] at byte 16 l of its plane.  After the six
// blocks: G log2(e) (64 fp32) and beta (64 fp32).
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
                a[q] = (16 * r + 4 * grp + q > m) ? bt[q] * exp2f(gt[q] - gm) * acc[q] : 0.0f;
            *reinterpret_cast<f32x4*>(&at[m * ATP + 16 * r + 4 * grp]) = a;
        }
    }
    __syncthreads();

    // column `lane` of T: x_t = [t == lane] - sum_{m<t} A_tm x_m, applied
    // column by column of A (x_m is final once every earlier column is in)
    float xv[CH];
    #pragma unroll
    for (int t = 0; t < CH; ++t) xv[t] = (t == lane) ? 1.0f : 0.0f;
    #pragma unroll
    for (int m = 0; m < CH - 1; ++m) {
        const float xm = xv[m];
        #pragma unroll
        for (int t4 = (m + 1) / 4; t4 < CH / 4; ++t4) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(&at[m * ATP + 4 * t4]);
            #pragma unroll
            for (int e = 0; e < 4; ++e)
                if (4 * t4 + e > m) xv[4 * t4 + e] = fmaf(-a[e], xm, xv[4 * t4 + e]);
        }
    }
    // T row-major through LDS (the A^T rows are no longer needed), then the
    // causal blocks in operand order, split hi/lo
    __syncthreads();
    #pragma unroll
    for (int t = 0; t < CH; ++t) at[t * ATP + lane] = xv[t];
    __syncthreads();
    uint8_t* rec = p.ws + (c * H + h) * kGdnWsRecord;
    #pragma unroll
    for (int r = 0; r < 4; ++r)
        #pragma unroll
        for (int i = 0; i <= r / 2; ++i) {
            const int blk = r < 2 ? r : 2 * r - 2 + i;
            const float* src = &at[(16 * r + li) * ATP + 32 * i + 8 * grp];
            const f32x4 a0 = *reinterpret_cast<const f32x4*>(src);
            const f32x4 a1 = *reinterpret_cast<const f32x4*>(src + 4);
            const float f[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
            bf16x8 hi, lo;
            split_n<8>(f, hi, lo);
            *reinterpret_cast<bf16x8*>(rec + blk * 2048 + 16 * lane) = hi;
            *reinterpret_cast<bf16x8*>(rec + blk * 2048 + 1024 + 16 * lane) = lo;
        }
    float* tab = reinterpret_cast<float*>(rec + kGdnWsTBytes);
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
    static constexpr int SP = DK + 8;     // S^T row pitch (elements)
    static constexpr int RP = CH + 8;     // R^T / U^T row pitch (elements)
    alignas(16) __bf16 k[2][CH * KP];     // K [m][d] by chunk parity
    alignas(16) __bf16 q[2][CH * KP];     // Q [i][d] by chunk parity
    alignas(16) __bf16 s[2][DVS * SP];    // S^T [j][d]: hi, lo
    alignas(16) __bf16 r[2][DVS * RP];    // R^T [j][m]: hi, lo
    alignas(16) __bf16 u[2][DVS * RP];    // U^T [j][m]: hi, lo
    alignas(16) __bf16 wu[2][DVS * RP];   // (w U)^T [j][m], w_m = exp(G_last - G_m): hi, lo
    alignas(16) float tab[2][2 * CH];     // by chunk parity: G_m log2(e) (0..63), beta_m (64..127)
};

struct GdnCtx {
    int h, j0, H, dv, lane, li, grp;
    int64_t T, n;                  // tokens, chunks
    int64_t qk_row, v_row, o_row;  // bytes per token of q / k, v, o
};

// Both roles walk the chunks four steps per loop iteration, so the register
// stages (loads three chunks ahead) rotate without copies.  Every global
// access of a step is issued unconditionally -- chunks past the end get
// empty buffer ranges: loads read zeros, stores are dropped -- so the
// in-order memory counters stay exact and loads issued after a step's stores
// are waited for only three steps later.  A step past the end changes no
// state, writes only LDS buffers no live step reads, and skips its barriers.
// A call of at most one chunk (ONE) runs the step once, without prefetch.

// ------------------------------------------------------------ output role
// Wave R owns rows 16 R..16 R + 15 of the chunk: X = Q_R S (phase 1), the
// decayed scores of its rows (phase 2), o = scale (gamma X + P U) (phase 3).
// The role also loads K (all rows) and stages it in LDS, and wave 0 scans
// the log-gates into the decay tables.
template <int DK>
struct OutStage {
    static constexpr int PK = CH * DK / 8 / NO_T;  // 16-byte pieces of K and of Q per thread
    u32x4 kp[PK];     // K pieces, coalesced (consecutive threads: consecutive bytes of a row)
    u32x4 qp[PK];     // Q pieces, same order
    float tab[2];     // wave 0: entries 2 lane, 2 lane + 1 of the gate tables
};

template <int DK, bool ONE, int R>
__device__ __forceinline__ void out_role(const GdnParams& p, GdnSmem<DK>& sm, const GdnCtx& x) {
    using Sm = GdnSmem<DK>;
    using St = OutStage<DK>;
    constexpr int KP = Sm::KP, SP = Sm::SP, RP = Sm::RP, NKK = DK / 32, PK = St::PK;
    constexpr int NT2 = R / 2 + 1;  // 32-token steps of the causal rows of block R
    const int lane = x.lane, li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;
    const int ot = 64 * R + lane;

    auto load = [&](St& S_, int64_t c) {
        const int64_t t0 = c * CH, rows = x.T - t0;
        const rsrc_t rk = make_rsrc(static_cast<const char*>(p.k) + t0 * x.qk_row, rows * x.qk_row);
        const rsrc_t rq = make_rsrc(static_cast<const char*>(p.q) + t0 * x.qk_row, rows * x.qk_row);
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = ot + NO_T * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            const uint32_t off = (uint32_t)(m * x.qk_row + ((int64_t)h * DK + d0) * 2);
            S_.kp[u] = __builtin_amdgcn_raw_buffer_load_b128(rk, off, 0, 0);
            S_.qp[u] = __builtin_amdgcn_raw_buffer_load_b128(rq, off, 0, 0);
        }
        if constexpr (R == 0) {
            const bool live = c < x.n;
            const rsrc_t rt = make_rsrc(p.ws + (live ? (c * H + h) * kGdnWsRecord + kGdnWsTBytes : 0),
                                        live ? 2 * CH * 4 : 0);
            const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(rt, (uint32_t)(8 * lane), 0, 0);
            const uint32_t v0 = v[0], v1 = v[1];
            S_.tab[0] = f32_of(v0);
            S_.tab[1] = f32_of(v1);
        }
    };

    // K and Q rows into LDS buffer bk; wave 0 also the gate tables
    auto stage = [&](const St& S_, int bk) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = ot + NO_T * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            *reinterpret_cast<u32x4*>(&sm.k[bk][m * KP + d0]) = S_.kp[u];
            *reinterpret_cast<u32x4*>(&sm.q[bk][m * KP + d0]) = S_.qp[u];
        }
        if constexpr (R == 0) {
            sm.tab[bk][2 * lane] = S_.tab[0];
            sm.tab[bk][2 * lane + 1] = S_.tab[1];
        }
    };

    auto step = [&](int64_t c, const St& nxt, St& ld) {
        const bool live = c < x.n;
        const int b = (int)(c & 1);
        const int64_t t0 = c * CH, rows = x.T - t0;
        if constexpr (!ONE) load(ld, c + 3);

        // ---- phase 1: X = Q_R S_c (S^T published by the chain role)
        f32x4 xh = {0.f, 0.f, 0.f, 0.f}, xl = {0.f, 0.f, 0.f, 0.f};
        bf16x8 qo[NKK];  // q[16 R + li][32 kk + 8 grp .. +7]
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            qo[kk] = *reinterpret_cast<const bf16x8*>(&sm.q[b][(16 * R + li) * KP + 32 * kk + 8 * grp]);
            const bf16x8 sh = *reinterpret_cast<const bf16x8*>(&sm.s[0][li * SP + 32 * kk + 8 * grp]);
            const bf16x8 sl = *reinterpret_cast<const bf16x8*>(&sm.s[1][li * SP + 32 * kk + 8 * grp]);
            xh = mma(qo[kk], sh, xh);
            xl = mma(qo[kk], sl, xl);
        }
        if (live) lds_barrier();

        // ---- phase 2: stage chunk c+1; P[i][m] = exp(G_i - G_m) (q_i . k_m),
        // m <= i, i = 16 R + li, as the A operand of P U: element e of step i2
        // is m = 32 i2 + 16 (e / 4) + 4 grp + e % 4 -- the accumulator layout
        // of K_s Q_R^T, used as is
        if constexpr (!ONE) stage(nxt, b ^ 1);
        const __bf16* kb = sm.k[b];
        bf16x8 ph[NT2], pl[NT2];
        const float g2i = sm.tab[b][16 * R + li];
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            float pf[8];
            #pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int s = 2 * i2 + half;
                if (s > R) {
                    #pragma unroll
                    for (int q = 0; q < 4; ++q) pf[4 * half + q] = 0.0f;
                    continue;
                }
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                #pragma unroll
                for (int kk = 0; kk < NKK; ++kk) {
                    const bf16x8 ko = *reinterpret_cast<const bf16x8*>(&kb[(16 * s + li) * KP + 32 * kk + 8 * grp]);
                    acc = mma(ko, qo[kk], acc);
                }
                const f32x4 g2s = *reinterpret_cast<const f32x4*>(&sm.tab[b][16 * s + 4 * grp]);
                #pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bool keep = s < R || 4 * grp + q <= li;
                    pf[4 * half + q] = keep ? acc[q] * exp2f(g2i - g2s[q]) : 0.0f;
                }
            }
            split_n<8>(pf, ph[i2], pl[i2]);
        }
        const f32x4 g2m = *reinterpret_cast<const f32x4*>(&sm.tab[b][16 * R + 4 * grp]);
        f32x4 oa;
        #pragma unroll
        for (int q = 0; q < 4; ++q) oa[q] = exp2f(g2m[q]) * (xh[q] + xl[q]);
        if (live) lds_barrier();

        // ---- phase 3: o_R = scale (gamma X + P U)
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            const int m0 = li * RP + 32 * i2 + 4 * grp;
            const bf16x8 uh = cat(*reinterpret_cast<const bf16x4*>(&sm.u[0][m0]),
                                  *reinterpret_cast<const bf16x4*>(&sm.u[0][m0 + 16]));
            const bf16x8 ul = cat(*reinterpret_cast<const bf16x4*>(&sm.u[1][m0]),
                                  *reinterpret_cast<const bf16x4*>(&sm.u[1][m0 + 16]));
            oa = mma(ph[i2], uh, oa);
            oa = mma(ph[i2], ul, oa);
            oa = mma(pl[i2], uh, oa);
        }
        const rsrc_t ro = make_rsrc(static_cast<char*>(static_cast<void*>(p.o)) + t0 * x.o_row, rows * x.o_row);
        #pragma unroll
        for (int q = 0; q < 4; ++q)
            __builtin_amdgcn_raw_buffer_store_b32(
                __builtin_bit_cast(uint32_t, oa[q] * p.scale), ro,
                (uint32_t)((16 * R + 4 * grp + q) * x.o_row + ((int64_t)h * dv + j0 + li) * 4), 0, 0);
        if (live) lds_barrier();
    };

    if constexpr (ONE) {
        St s0;
        load(s0, 0);
        stage(s0, 0);
        lds_barrier();
        if (x.n == 1) step(0, s0, s0);
    } else {
        St s0, s1, s2, s3;
        load(s0, 0);
        load(s1, 1);
        load(s2, 2);
        stage(s0, 0);
        lds_barrier();
        for (int64_t c = 0; c < x.n; c += 4) {
            step(c, s1, s3);
            step(c + 1, s2, s0);
            step(c + 2, s3, s1);
            step(c + 3, s0, s2);
        }
    }
}

// ------------------------------------------------------------- chain role
// Wave R owns rows 16 R..16 R + 15 of the chunk and rows
// 16 R NDW..16 (R + 1) NDW - 1 of S (fp32, in registers): K_R S -> R
// (phase 1), U_R = T[R rows] R (phase 2), S <- gamma_last S + K^T (w U) on
// its rows of S and S^T published (phase 3).  Only this role's work is on
// the state's sequential path.
template <int R>
struct ChainStage {
    static constexpr int NT2 = R / 2 + 1;
    u32x4 t[NT2][2];    // T[16 R + li][32 i + 8 grp .. +7]: bf16 hi, lo
    uint32_t v[4];      // bf16 bits of v[16 R + 4 grp + q][j0 + li]
};

template <int DK, bool ONE, int R>
__device__ __forceinline__ void chain_role(const GdnParams& p, GdnSmem<DK>& sm, const GdnCtx& x) {
    using Sm = GdnSmem<DK>;
    using St = ChainStage<R>;
    constexpr int KP = Sm::KP, SP = Sm::SP, RP = Sm::RP;
    constexpr int NKK = DK / 32, NDW = DK / 64, NT2 = St::NT2;
    const int li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;

    // state tiles in accumulator layout: S[u][q] = S[d][j0 + li] with
    // d = 16 (R NDW + u) + 4 grp + q; for each q the 16 lanes of a group hold
    // 64 contiguous bytes of a state row
    f32x4 S[NDW];
    auto srow = [&](int u, int q) -> int64_t {
        return ((int64_t)h * DK + 16 * (R * NDW + u) + 4 * grp + q) * dv + j0 + li;
    };
    #pragma unroll
    for (int u = 0; u < NDW; ++u) {
        S[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (p.state_in) {
            #pragma unroll
            for (int q = 0; q < 4; ++q) S[u][q] = p.state_in[srow(u, q)];
        }
    }

    auto load = [&](St& S_, int64_t c) {
        const int64_t t0 = c * CH, rows = x.T - t0;
        const rsrc_t rv = make_rsrc(static_cast<const char*>(p.v) + t0 * x.v_row, rows * x.v_row);
        #pragma unroll
        for (int q = 0; q < 4; ++q)
            S_.v[q] = __builtin_amdgcn_raw_buffer_load_b16(
                rv, (uint32_t)((16 * R + 4 * grp + q) * x.v_row + ((int64_t)h * dv + j0 + li) * 2), 0, 0);
        const bool live = c < x.n;
        const rsrc_t rt = make_rsrc(p.ws + (live ? (c * H + h) * kGdnWsRecord : 0), live ? kGdnWsTBytes : 0);
        #pragma unroll
        for (int i = 0; i < NT2; ++i) {
            const int blk = R < 2 ? R : 2 * R - 2 + i;
            #pragma unroll
            for (int pl = 0; pl < 2; ++pl)
                S_.t[i][pl] = __builtin_amdgcn_raw_buffer_load_b128(rt, (uint32_t)(blk * 2048 + pl * 1024 + 16 * x.lane), 0, 0);
        }
    };

    // this wave's rows of S as bf16 hi/lo planes of S^T [j][d]
    auto publish_s = [&]() {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d0 = 16 * (R * NDW + u) + 4 * grp;
            const float f[4] = {S[u][0], S[u][1], S[u][2], S[u][3]};
            bf16x4 hi, lo;
            split_n<4>(f, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.s[0][li * SP + d0]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.s[1][li * SP + d0]) = lo;
        }
    };

    const uint64_t state_bytes = (uint64_t)H * DK * dv * 4;
    // the chain waves carry the sequential path: issue their instructions
    // first when they compete with the output wave on the same SIMD
    __builtin_amdgcn_s_setprio(2);
    auto step = [&](int64_t c, const St& cur, St& ld) {
        const bool live = c < x.n;
        const int b = (int)(c & 1);
        const __bf16* kb = sm.k[b];
        if constexpr (!ONE) load(ld, c + 3);

        // operands and decays that do not depend on S
        bf16x8 th[NT2], tl[NT2];
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            th[i2] = __builtin_bit_cast(bf16x8, cur.t[i2][0]);
            tl[i2] = __builtin_bit_cast(bf16x8, cur.t[i2][1]);
        }
        const f32x4 g2m = *reinterpret_cast<const f32x4*>(&sm.tab[b][16 * R + 4 * grp]);
        const f32x4 bm = *reinterpret_cast<const f32x4*>(&sm.tab[b][CH + 16 * R + 4 * grp]);
        const float g2l = sm.tab[b][CH - 1];
        float gam[4], wm[4], vv[4];
        #pragma unroll
        for (int q = 0; q < 4; ++q) {
            gam[q] = exp2f(g2m[q]);
            wm[q] = exp2f(g2l - g2m[q]);
            vv[q] = f32_of(cur.v[q] << 16);
        }
        const float gl = exp2f(g2l);

        // ---- phase 1: R_R = beta (V_R - gamma K_R S_c)
        f32x4 kh = {0.f, 0.f, 0.f, 0.f}, kl = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const bf16x8 ko = *reinterpret_cast<const bf16x8*>(&kb[(16 * R + li) * KP + 32 * kk + 8 * grp]);
            const bf16x8 sh = *reinterpret_cast<const bf16x8*>(&sm.s[0][li * SP + 32 * kk + 8 * grp]);
            const bf16x8 sl = *reinterpret_cast<const bf16x8*>(&sm.s[1][li * SP + 32 * kk + 8 * grp]);
            kh = mma(ko, sh, kh);
            kl = mma(ko, sl, kl);
        }
        {
            float rr[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) rr[q] = bm[q] * (vv[q] - gam[q] * (kh[q] + kl[q]));
            bf16x4 hi, lo;
            split_n<4>(rr, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.r[0][li * RP + 16 * R + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.r[1][li * RP + 16 * R + 4 * grp]) = lo;
        }
        if (live) lds_barrier();

        // ---- phase 2: U_R = T[R rows] R, and w U
        bf16x8 kt[NDW][2];  // K^T operands of the update (element e: m = 32 mm + 8 grp + e)
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
            const bf16x8 rh = *reinterpret_cast<const bf16x8*>(&sm.r[0][li * RP + 32 * i2 + 8 * grp]);
            const bf16x8 rl = *reinterpret_cast<const bf16x8*>(&sm.r[1][li * RP + 32 * i2 + 8 * grp]);
            ua = mma(th[i2], rh, ua);
            ub = mma(th[i2], rl, ub);
            uc = mma(tl[i2], rh, uc);
        }
        {
            float uf[4], wf[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) {
                uf[q] = ua[q] + (ub[q] + uc[q]);
                wf[q] = uf[q] * wm[q];
            }
            bf16x4 hi, lo;
            split_n<4>(uf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.u[0][li * RP + 16 * R + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.u[1][li * RP + 16 * R + 4 * grp]) = lo;
            split_n<4>(wf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.wu[0][li * RP + 16 * R + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.wu[1][li * RP + 16 * R + 4 * grp]) = lo;
        }
        if (live) lds_barrier();

        // ---- phase 3: S_c to chunk_states[c]; S <- gamma_last S + K^T (w U)
        const rsrc_t rc = make_rsrc(p.chunk_states + (live ? c : 0) * (int64_t)H * DK * dv,
                                    live && p.chunk_states ? (int64_t)state_bytes : 0);
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            #pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float sv = S[u][q];  // a bit_cast of a vector element reads element 0
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, sv), rc,
                                                      (uint32_t)(srow(u, q) * 4), 0, 0);
            }
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            f32x4 ah, al = {0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int q = 0; q < 4; ++q) ah[q] = gl * S[u][q];
            #pragma unroll
            for (int mm = 0; mm < 2; ++mm) {
                const int m0 = li * RP + 32 * mm + 8 * grp;
                const bf16x8 wh = *reinterpret_cast<const bf16x8*>(&sm.wu[0][m0]);
                const bf16x8 wl = *reinterpret_cast<const bf16x8*>(&sm.wu[1][m0]);
                ah = mma(kt[u][mm], wh, ah);
                al = mma(kt[u][mm], wl, al);
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
        St s0, s1, s2, s3;
        load(s0, 0);
        load(s1, 1);
        load(s2, 2);
        publish_s();
        lds_barrier();
        for (int64_t c = 0; c < x.n; c += 4) {
            step(c, s0, s3);
            step(c + 1, s1, s0);
            step(c + 2, s2, s1);
            step(c + 3, s3, s2);
        }
    }
    if (p.final_state) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            #pragma unroll
            for (int q = 0; q < 4; ++q) p.final_state[srow(u, q)] = S[u][q];
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
        hipLaunchKernelGGL((gdn_prepare_kernel<DK>), dim3((unsigned)(n * p.H)), dim3(64), 0, stream, p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)(p.H * (p.dv / DVS)));
    if (p.T <= CH) hipLaunchKernelGGL((gdn_scan_kernel<DK, true>), grid, dim3(NT), 0, stream, p);
    else hipLaunchKernelGGL((gdn_scan_kernel<DK, false>), grid, dim3(NT), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gdn(const GdnParams& p, hipStream_t stream) {
    if (p.dk == 128) return launch_t<128>(p, stream);
    if (p.dk == 64) return launch_t<64>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
