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
//  2. gdn_scan, one workgroup of four waves per (head, 16-column slice of
//     the values), walks the chunks in order.  Column slices are
//     independent: U[:, J], o[:, J] and S[:, J] need only S[:, J] and
//     v[:, J].  Wave w owns rows 16w..16w+15 of the chunk and rows
//     DK/4 w .. DK/4 (w+1) - 1 of S.  Per chunk, three LDS barriers:
//       phase 1  K_w S and Q_w S on MFMA (S from the published S^T planes),
//                R_w = beta (V_w - gamma K_w S) -> LDS; the decayed scores
//                of row block w, P = exp(G_i - G_m) (q_i . k_m), m <= i;
//       phase 2  U_w = sum_m T[w rows][m] R_m -> LDS, with w_m U_m;
//       phase 3  o_w = scale (gamma Q_w S + P U); S <- gamma_last S +
//                K^T (w U) on this wave's rows of d; publish S^T; stage the
//                next chunk's K and gate tables.
//     The next chunk's loads are issued at the start of phase 1.  The
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
constexpr int NW = 4;        // waves per scan workgroup
constexpr int ATP = CH + 4;  // pitch (floats) of the A^T rows in the prepare kernel

__device__ inline float f32_of(uint32_t u) { return __builtin_bit_cast(float, u); }

// ------------------------------------------------------------------ prepare
// One wave per (chunk c, head h): T = (I + A)^-1 into ws[c][h] (row-major,
// zeros above the diagonal).  Rows past the last token have k = 0, beta = 0
// and g = 0, so their rows and columns of A vanish and T is the identity
// there.
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
    float* tp = p.ws + ((c * H + h) * CH) * CH;
    #pragma unroll
    for (int t = 0; t < CH; ++t) tp[t * CH + lane] = xv[t];
}

// --------------------------------------------------------------------- scan
template <int DK>
struct alignas(16) GdnSmem {
    // K rows are read 16 rows x 16 B at a time and, transposed, 4 rows x
    // 32 B at a time: a pitch of 16 B times an odd number whose 4-row windows
    // do not overlap keeps both conflict-free.
    static constexpr int KP = DK == 128 ? 152 : 104;
    static constexpr int SP = DK + 8;     // S^T row pitch (elements)
    static constexpr int RP = CH + 8;     // R^T / U^T row pitch (elements)
    alignas(16) __bf16 k[2][CH * KP];     // K [m][d] by chunk parity
    alignas(16) __bf16 s[2][DVS * SP];    // S^T [j][d]: hi, lo
    alignas(16) __bf16 r[2][DVS * RP];    // R^T [j][m]: hi, lo
    alignas(16) __bf16 u[2][DVS * RP];    // U^T [j][m]: hi, lo
    alignas(16) __bf16 wu[2][DVS * RP];   // (w U)^T [j][m], w_m = exp(G_last - G_m): hi, lo
    alignas(16) float G2[2][CH];          // G_m log2(e) by chunk parity
    alignas(16) float B[2][CH];           // beta_m by chunk parity
};

// Register staging of one chunk for wave W.
template <int DK, int W>
struct GdnStage {
    static constexpr int PK = CH * DK / 8 / (64 * NW);  // 16-byte K pieces per thread
    static constexpr int NKK = DK / 32;
    static constexpr int NT2 = W / 2 + 1;                // 32-column steps of T's row block W
    u32x4 kp[PK];       // K pieces, coalesced (consecutive threads: consecutive bytes of a row)
    u32x4 q[NKK];       // q[16 W + li][32 kk + 8 grp .. +7]
    u32x4 t[NT2][2];    // T[16 W + li][32 i + 8 grp .. +7] (fp32)
    uint32_t v[4];      // bf16 bits of v[16 W + 4 grp + q][j0 + li]
    float g, b;         // wave 0: log-gate and beta of token `lane`
};

struct GdnCtx {
    int h, j0, H, dv, tid, lane, li, grp;
    int64_t T, n;                  // tokens, chunks
    int64_t qk_row, v_row, o_row;  // bytes per token of q / k, v, o
};

template <int DK, int W>
__device__ __forceinline__ void gdn_wave(const GdnParams& p, GdnSmem<DK>& sm, const GdnCtx& x) {
    using Sm = GdnSmem<DK>;
    using St = GdnStage<DK, W>;
    constexpr int KP = Sm::KP, SP = Sm::SP, RP = Sm::RP;
    constexpr int NKK = DK / 32, NDW = DK / 64, PK = St::PK, NT2 = St::NT2;
    const int lane = x.lane, li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;

    // state tiles in accumulator layout: S[u][q] = S[d][j0 + li] with
    // d = 16 (W NDW + u) + 4 grp + q; for each q the 16 lanes of a group hold
    // 64 contiguous bytes of a state row
    f32x4 S[NDW];
    auto srow = [&](int u, int q) -> int64_t {
        return ((int64_t)h * DK + 16 * (W * NDW + u) + 4 * grp + q) * dv + j0 + li;
    };
    #pragma unroll
    for (int u = 0; u < NDW; ++u) {
        S[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (p.state_in) {
            #pragma unroll
            for (int q = 0; q < 4; ++q) S[u][q] = p.state_in[srow(u, q)];
        }
    }

    // HBM loads of chunk c (chunks past the end get empty ranges: zeros)
    auto load_chunk = [&](St& R, int64_t c) {
        const int64_t t0 = c * CH, rows = x.T - t0;
        const rsrc_t rk = make_rsrc(static_cast<const char*>(p.k) + t0 * x.qk_row, rows * x.qk_row);
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = x.tid + 64 * NW * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            R.kp[u] = __builtin_amdgcn_raw_buffer_load_b128(rk, (uint32_t)(m * x.qk_row + ((int64_t)h * DK + d0) * 2), 0, 0);
        }
        const rsrc_t rq = make_rsrc(static_cast<const char*>(p.q) + t0 * x.qk_row, rows * x.qk_row);
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
            R.q[kk] = __builtin_amdgcn_raw_buffer_load_b128(
                rq, (uint32_t)((16 * W + li) * x.qk_row + ((int64_t)h * DK + 32 * kk + 8 * grp) * 2), 0, 0);
        const rsrc_t rv = make_rsrc(static_cast<const char*>(p.v) + t0 * x.v_row, rows * x.v_row);
        #pragma unroll
        for (int q = 0; q < 4; ++q)
            R.v[q] = __builtin_amdgcn_raw_buffer_load_b16(
                rv, (uint32_t)((16 * W + 4 * grp + q) * x.v_row + ((int64_t)h * dv + j0 + li) * 2), 0, 0);
        const bool live = c < x.n;
        const float* tb = p.ws + (live ? (c * H + h) * CH * CH : 0);
        const rsrc_t rt = make_rsrc(tb, live ? CH * CH * 4 : 0);
        #pragma unroll
        for (int i = 0; i < NT2; ++i)
            #pragma unroll
            for (int half = 0; half < 2; ++half)
                R.t[i][half] = __builtin_amdgcn_raw_buffer_load_b128(
                    rt, (uint32_t)(((16 * W + li) * CH + 32 * i + 8 * grp + 4 * half) * 4), 0, 0);
        if constexpr (W == 0) {
            const rsrc_t rg = make_rsrc(p.g + t0 * H, rows * H * 4);
            const rsrc_t rb = make_rsrc(p.beta + t0 * H, rows * H * 4);
            R.g = f32_of(__builtin_amdgcn_raw_buffer_load_b32(rg, (uint32_t)((lane * H + h) * 4), 0, 0));
            R.b = f32_of(__builtin_amdgcn_raw_buffer_load_b32(rb, (uint32_t)((lane * H + h) * 4), 0, 0));
        }
    };

    // K rows into LDS buffer bk; wave 0 also the gate tables
    auto stage = [&](const St& R, int bk) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = x.tid + 64 * NW * u;
            const int m = pc / (DK / 8), d0 = (pc % (DK / 8)) * 8;
            *reinterpret_cast<u32x4*>(&sm.k[bk][m * KP + d0]) = R.kp[u];
        }
        if constexpr (W == 0) {
            sm.G2[bk][lane] = wave_inclusive_sum(R.g) * LOG2E;
            sm.B[bk][lane] = R.b;
        }
    };

    // this wave's rows of S as bf16 hi/lo planes of S^T [j][d]
    auto publish_s = [&]() {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d0 = 16 * (W * NDW + u) + 4 * grp;
            const float f[4] = {S[u][0], S[u][1], S[u][2], S[u][3]};
            bf16x4 hi, lo;
            split_n<4>(f, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.s[0][li * SP + d0]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.s[1][li * SP + d0]) = lo;
        }
    };

    auto step = [&](int64_t c, const St& C, St& N) {
        const int b = (int)(c & 1);
        const int64_t t0 = c * CH, rows = x.T - t0;
        const __bf16* kb = sm.k[b];
        load_chunk(N, c + 1);
        if (p.chunk_states) {
            float* cs = p.chunk_states + c * (int64_t)H * DK * dv;
            #pragma unroll
            for (int u = 0; u < NDW; ++u)
                #pragma unroll
                for (int q = 0; q < 4; ++q) cs[srow(u, q)] = S[u][q];
        }

        // ---- phase 1: K_W S, Q_W S, R_W, decayed scores of row block W
        f32x4 ks = {0.f, 0.f, 0.f, 0.f}, qs = {0.f, 0.f, 0.f, 0.f};
        bf16x8 kw[NKK];
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            kw[kk] = *reinterpret_cast<const bf16x8*>(&kb[(16 * W + li) * KP + 32 * kk + 8 * grp]);
            const bf16x8 sh = *reinterpret_cast<const bf16x8*>(&sm.s[0][li * SP + 32 * kk + 8 * grp]);
            const bf16x8 sl = *reinterpret_cast<const bf16x8*>(&sm.s[1][li * SP + 32 * kk + 8 * grp]);
            ks = mma(kw[kk], sh, ks);
            ks = mma(kw[kk], sl, ks);
            const bf16x8 qo = __builtin_bit_cast(bf16x8, C.q[kk]);
            qs = mma(qo, sh, qs);
            qs = mma(qo, sl, qs);
        }
        const f32x4 g2m = *reinterpret_cast<const f32x4*>(&sm.G2[b][16 * W + 4 * grp]);
        const f32x4 bm = *reinterpret_cast<const f32x4*>(&sm.B[b][16 * W + 4 * grp]);
        {
            float rr[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) rr[q] = bm[q] * (f32_of(C.v[q] << 16) - exp2f(g2m[q]) * ks[q]);
            bf16x4 hi, lo;
            split_n<4>(rr, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.r[0][li * RP + 16 * W + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.r[1][li * RP + 16 * W + 4 * grp]) = lo;
        }
        // P[i][m] = exp(G_i - G_m) (q_i . k_m), m <= i, i = 16 W + li, as the
        // A operand of P U: element e of step i2 is m = 32 i2 + 16 (e / 4) +
        // 4 grp + e % 4 -- the accumulator layout of K_s Q_W^T, used as is
        bf16x8 ph[NT2], pl[NT2];
        const float g2i = sm.G2[b][16 * W + li];
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            float pf[8];
            #pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int s = 2 * i2 + half;
                if (s > W) {
                    #pragma unroll
                    for (int q = 0; q < 4; ++q) pf[4 * half + q] = 0.0f;
                    continue;
                }
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                #pragma unroll
                for (int kk = 0; kk < NKK; ++kk) {
                    const bf16x8 ko = s == W ? kw[kk]
                                             : *reinterpret_cast<const bf16x8*>(&kb[(16 * s + li) * KP + 32 * kk + 8 * grp]);
                    acc = mma(ko, __builtin_bit_cast(bf16x8, C.q[kk]), acc);
                }
                const f32x4 g2s = *reinterpret_cast<const f32x4*>(&sm.G2[b][16 * s + 4 * grp]);
                #pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bool keep = s < W || 4 * grp + q <= li;
                    pf[4 * half + q] = keep ? acc[q] * exp2f(g2i - g2s[q]) : 0.0f;
                }
            }
            split_n<8>(pf, ph[i2], pl[i2]);
        }
        lds_barrier();

        // ---- phase 2: U_W = T[W rows] R, and w U
        f32x4 ua = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int i2 = 0; i2 < NT2; ++i2) {
            const f32x4 ta = __builtin_bit_cast(f32x4, C.t[i2][0]);
            const f32x4 tc = __builtin_bit_cast(f32x4, C.t[i2][1]);
            const float tf[8] = {ta[0], ta[1], ta[2], ta[3], tc[0], tc[1], tc[2], tc[3]};
            bf16x8 th, tl;
            split_n<8>(tf, th, tl);
            const bf16x8 rh = *reinterpret_cast<const bf16x8*>(&sm.r[0][li * RP + 32 * i2 + 8 * grp]);
            const bf16x8 rl = *reinterpret_cast<const bf16x8*>(&sm.r[1][li * RP + 32 * i2 + 8 * grp]);
            ua = mma(th, rh, ua);
            ua = mma(th, rl, ua);
            ua = mma(tl, rh, ua);
        }
        const float g2l = sm.G2[b][CH - 1];
        {
            float uf[4], wf[4];
            #pragma unroll
            for (int q = 0; q < 4; ++q) {
                uf[q] = ua[q];
                wf[q] = ua[q] * exp2f(g2l - g2m[q]);
            }
            bf16x4 hi, lo;
            split_n<4>(uf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.u[0][li * RP + 16 * W + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.u[1][li * RP + 16 * W + 4 * grp]) = lo;
            split_n<4>(wf, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.wu[0][li * RP + 16 * W + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.wu[1][li * RP + 16 * W + 4 * grp]) = lo;
        }
        lds_barrier();

        // ---- phase 3: o_W = scale (gamma Q_W S + P U); S <- gamma_last S + K^T (w U)
        f32x4 oa;
        #pragma unroll
        for (int q = 0; q < 4; ++q) oa[q] = exp2f(g2m[q]) * qs[q];
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
                (uint32_t)((16 * W + 4 * grp + q) * x.o_row + ((int64_t)h * dv + j0 + li) * 4), 0, 0);
        const float gl = exp2f(g2l);
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d0 = 16 * (W * NDW + u);
            f32x4 acc;
            #pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] = gl * S[u][q];
            #pragma unroll
            for (int mm = 0; mm < 2; ++mm) {
                const int m0 = 32 * mm + 8 * grp;
                const bf16x8 kt = cat(tr4(kb, KP, m0, d0, li), tr4(kb, KP, m0 + 4, d0, li));
                const bf16x8 wh = *reinterpret_cast<const bf16x8*>(&sm.wu[0][li * RP + m0]);
                const bf16x8 wl = *reinterpret_cast<const bf16x8*>(&sm.wu[1][li * RP + m0]);
                acc = mma(kt, wh, acc);
                acc = mma(kt, wl, acc);
            }
            S[u] = acc;
        }
        stage(N, b ^ 1);
        publish_s();
        lds_barrier();
    };

    St A, B;
    load_chunk(A, 0);
    stage(A, 0);
    publish_s();
    lds_barrier();
    for (int64_t c = 0; c < x.n;) {
        step(c, A, B);
        if (++c >= x.n) break;
        step(c, B, A);
        ++c;
    }
    if (p.final_state) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            #pragma unroll
            for (int q = 0; q < 4; ++q) p.final_state[srow(u, q)] = S[u][q];
    }
}

template <int DK>
__global__ __launch_bounds__(64 * NW) void gdn_scan_kernel(const GdnParams p) {
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
    x.tid = tid;
    x.lane = tid & 63;
    x.li = x.lane & 15;
    x.grp = x.lane >> 4;
    x.T = p.T;
    x.n = (p.T + CH - 1) / CH;
    x.qk_row = (int64_t)x.H * DK * 2;
    x.v_row = (int64_t)x.H * x.dv * 2;
    x.o_row = (int64_t)x.H * x.dv * 4;

    switch (wave) {
        case 0: gdn_wave<DK, 0>(p, sm, x); break;
        case 1: gdn_wave<DK, 1>(p, sm, x); break;
        case 2: gdn_wave<DK, 2>(p, sm, x); break;
        default: gdn_wave<DK, 3>(p, sm, x); break;
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
    hipLaunchKernelGGL((gdn_scan_kernel<DK>), dim3((unsigned)(p.H * (p.dv / DVS))), dim3(64 * NW), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gdn(const GdnParams& p, hipStream_t stream) {
    if (p.dk == 128) return launch_t<128>(p, stream);
    if (p.dk == 64) return launch_t<64>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
