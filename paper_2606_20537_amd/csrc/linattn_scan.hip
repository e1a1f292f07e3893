// Chunked gated linear-attention prefill on gfx950 MFMA.
//
// Per head, S_t = exp(g_t) S_{t-1} + k_t^T v_t and o_t = scale * q_t S_t,
// evaluated chunk by chunk (paper §5: the prefill folds its recurrent state
// once per chunk of C tokens).  For chunk j with entering state S_j and
// inclusive in-chunk log-decay sums G_i:
//   o_i     = scale * (exp(G_i) q_i S_j + sum_{m<=i} exp(G_i - G_m)(q_i.k_m) v_m)
//   S_{j+1} = exp(G_last) S_j + sum_m exp(G_last - G_m) k_m^T v_m
//
// Work split: one workgroup per (head, 16-wide slice of the value columns).
// Column slices of S are independent: o[:, J] needs only S[:, J] and v[:, J],
// and the fold of S[:, J] needs only v[:, J].  The workgroup walks the chunks
// in order, so the arithmetic applied to chunk j depends only on (S_j, the
// chunk's inputs) -- never on the call's length, its first chunk or the grid.
// That is what makes restore-at-an-aligned-boundary-then-continue bitwise
// equal to one long prefill.
//
// Eight waves, two per SIMD, in two roles that overlap on every SIMD:
//   output waves 0-3: wave w owns rows 16w..16w+15 of the chunk and computes
//     A^T = K Q^T (causal tiles), P = A * decay, O^T = V^T P^T,
//     X^T = S_j^T Q^T and o = scale (exp(G) X + O);
//   state waves 4-7: stream the chunk two ahead from HBM into registers,
//     stage it in LDS, write the chunk-boundary states and fold the state
//     S^T = exp(G_last) S^T + (V w)^T K over their DK/64 tiles of 16 rows.
// Every product runs on v_mfma_f32_16x16x32_bf16 with fp32 accumulation,
// written transposed so that each lane ends with four consecutive value
// columns (16-byte stores).  Inputs are exact bf16 operands; fp32-derived
// operands (P, S_j, V w with w_m = exp(G_last - G_m)) are split hi + lo in
// bf16, which keeps them to ~2^-17 relative error, far inside the 2e-3 parity
// bar.  Scaling the 16-wide V slice by w instead of the dk-wide K keeps K
// exact and the split small.  fp32 inputs are split hi + lo on load and use
// three products per term.
//
// Decay: inside the chunk G is non-increasing for g <= 0.  Below the diagonal
// tile, exp(G_i - G_m) = exp(G_i - G_e) exp(G_e - G_m) with e the last token of
// m's 16-token block; both factors lie in (0, 1], come from per-chunk tables
// and never overflow.  The diagonal tile evaluates exp2 directly.
//
// LDS holds every tile row-major (K, Q, V, V w and the published S), written
// with 8- and 16-byte stores.  Operands whose contraction index runs along the
// rows (V^T, (V w)^T, S^T as A operands; K as the fold's B operand) are read
// with gfx950's transposing LDS load ds_read_b64_tr_b16: inside a 16-lane
// group, lane L addresses row k0 + L/4, columns 4(L%4)..+3, and lane n
// receives column n of rows k0..k0+3.  The contraction index may be permuted
// freely as long as both operands agree, which lets the accumulator of K Q^T
// serve directly as the B operand of V^T P^T.  HBM traffic goes through buffer
// resources: a scalar base per chunk, fixed per-lane offsets, and hardware
// range checks that read the ragged tail as zeros and drop stores past T.
// The one barrier per chunk orders LDS only and never waits for global stores.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int CH = 64;        // chunk length
constexpr int DVS = 16;       // value columns per workgroup
constexpr int NT = 512;       // threads per workgroup (8 waves)
constexpr int NS_T = 256;     // threads of the state role
constexpr int VP = DVS + 8;   // pitch (elements) of the [m][j] and [d][j] tiles
constexpr float LOG2E = 1.4426950408889634f;

__device__ inline f32x4 mma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Buffer resource over [base, base + nbytes) (raw, stride 0); accesses past
// nbytes read zeros / are dropped.
__device__ inline rsrc_t make_rsrc(const void* base, int64_t nbytes) {
    const int64_t n = nbytes < 0 ? 0 : (nbytes > 0x7ffffff0 ? 0x7ffffff0 : nbytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// Transposing LDS read of a row-major tile with `pitch` elements per row:
// lane n of each 16-lane group gets tile[k0 + 0..3][n0 + n].
__device__ inline bf16x4 tr4(const __bf16* tile, int pitch, int k0, int n0, int li) {
    const __bf16* p = tile + (k0 + (li >> 2)) * pitch + n0 + 4 * (li & 3);
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
    return __builtin_bit_cast(bf16x4, v);
}

__device__ inline bf16x8 cat(const bf16x4& a, const bf16x4& b) {
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP row shifts and
// row broadcasts (cross-lane ALU operations, no LDS round trip).  The
// association order is fixed, so the result is deterministic.
template <int CTRL, int ROW_MASK, bool BOUND_ZERO>
__device__ inline float dpp_f(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, ROW_MASK, 0xf,
                                                                 BOUND_ZERO));
}

__device__ inline float wave_inclusive_sum(float x) {
    x += dpp_f<0x111, 0xf, true>(x);   // row_shr:1
    x += dpp_f<0x112, 0xf, true>(x);   // row_shr:2
    x += dpp_f<0x114, 0xf, true>(x);   // row_shr:4
    x += dpp_f<0x118, 0xf, true>(x);   // row_shr:8  -> inclusive within rows of 16
    x += dpp_f<0x142, 0xa, false>(x);  // row_bcast:15 into rows 1 and 3
    x += dpp_f<0x143, 0xc, false>(x);  // row_bcast:31 into rows 2 and 3
    return x;
}

__device__ inline float lane_value(float x, int l) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), l));
}

// hi + lo split of fp32 values into bf16 (round to nearest even both times).
__device__ inline void split8(const float* f, bf16x8& hi, bf16x8& lo) {
    #pragma unroll
    for (int e = 0; e < 8; ++e) {
        const __bf16 h = (__bf16)f[e];
        hi[e] = h;
        lo[e] = (__bf16)(f[e] - (float)h);
    }
}

// Every member starts on a 16-byte boundary so that 16-byte LDS accesses
// compile to single ds_read_b128 / ds_write_b128 instructions.
template <int DK, bool F32>
struct alignas(16) Smem {
    static constexpr int KP = DK + 8;      // row pitch of K (elements)
    static constexpr int NL = F32 ? 2 : 1; // bf16 planes of the inputs: hi (and lo)
    alignas(16) __bf16 k[2][NL][CH * KP];  // K     [m][d]
    alignas(16) __bf16 v[2][NL][CH * VP];  // V     [m][j] (this slice)
    alignas(16) __bf16 vw[2][2][CH * VP];  // V w   [m][j], hi and lo planes
    alignas(16) __bf16 s[2][2][DK * VP];   // S_j   [d][j], hi and lo planes
    alignas(16) float G2[2][CH];           // G_t log2(e), G the inclusive log-decay sum
    alignas(16) float eG[2][CH];           // exp(G_t)
    alignas(16) float bm[2][CH];           // exp(G_e - G_m), e = last token of m's block
    alignas(16) float ai[2][CH][4];        // exp(G_i - G_e(M)) for 16-token blocks M below i's
};

// 8 consecutive input elements of one row (16 B of bf16 or 32 B of fp32).
template <bool F32>
struct Piece {
    u32x4 x[F32 ? 2 : 1];
};

template <bool F32>
__device__ inline void load_piece(Piece<F32>& p, rsrc_t r, uint32_t off) {
    p.x[0] = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    if (F32) p.x[F32 ? 1 : 0] = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, 0);
}

template <bool F32>
__device__ inline void piece_f32(const Piece<F32>& p, float* f) {
    if (F32) {
        const f32x4 a = __builtin_bit_cast(f32x4, p.x[0]);
        const f32x4 b = __builtin_bit_cast(f32x4, p.x[F32 ? 1 : 0]);
        #pragma unroll
        for (int e = 0; e < 4; ++e) { f[e] = a[e]; f[4 + e] = b[e]; }
    } else {
        const bf16x8 h = __builtin_bit_cast(bf16x8, p.x[0]);
        #pragma unroll
        for (int e = 0; e < 8; ++e) f[e] = (float)h[e];
    }
}

// A piece as bf16 hi (and lo, for fp32 inputs).
template <bool F32>
__device__ inline void split_piece(const Piece<F32>& p, bf16x8& hi, bf16x8& lo) {
    if (F32) {
        float f[8];
        piece_f32<F32>(p, f);
        split8(f, hi, lo);
    } else {
        hi = __builtin_bit_cast(bf16x8, p.x[0]);
        lo = bf16x8{};
    }
}

// Register staging of one chunk's global loads: K, V and g for the state
// role, the wave's own 16 rows of Q for an output wave.
template <bool F32, int PK>
struct Stage {
    Piece<F32> kp[PK];
    Piece<F32> vp;
    float g;
};

template <bool F32, int NKK>
struct QStage {
    Piece<F32> qp[NKK];
};

// Workgroup barrier for LDS traffic only.  Global stores of o and the states
// are never read back inside the kernel, so the barrier does not wait for
// them (a plain __syncthreads() would drain every outstanding global access).
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int DK, bool F32>
__global__ __launch_bounds__(NT) void linattn_scan_kernel(const ScanParams p) {
    using S_ = Smem<DK, F32>;
    constexpr int KP = S_::KP;
    constexpr int NL = S_::NL;
    constexpr int NKK = DK / 32;             // k-steps of 32 over dk
    constexpr int PK = (CH * DK / 8) / NS_T; // K pieces per state thread
    constexpr int NDW = DK / 64;             // state tiles (16 rows of d) per state wave
    constexpr int ES = F32 ? 4 : 2;          // input element size
    __shared__ S_ sm;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform
    const bool state_role = wave >= 4;
    const int wq = wave & 3;
    const int lane = tid & 63;
    const int li = lane & 15;
    const int grp = lane >> 4;
    const int st = tid - NS_T;  // state-role thread index (valid when state_role)

    // workgroup -> (head, slice); slices of one head share an XCD (and its L2)
    // when the grid allows it (workgroups go round-robin over 8 XCDs).
    const int H = p.H, dv = p.dv;
    const int NS = dv / DVS;
    const int N = H * NS;
    int logical = blockIdx.x;
    if ((N % 8) == 0 && ((N / 8) % NS) == 0) logical = (blockIdx.x % 8) * (N / 8) + blockIdx.x / 8;
    const int h = logical / NS;
    const int j0 = (logical % NS) * DVS;

    const int64_t T = p.T;
    const int64_t n_chunks = (T + CH - 1) / CH;
    const int64_t qk_row = (int64_t)H * DK * ES;  // bytes per token of q / k
    const int64_t v_row = (int64_t)H * dv * ES;   // bytes per token of v
    const int64_t o_row = (int64_t)H * dv * 4;    // bytes per token of o

    // ---- state (state role), as S^T tiles in accumulator layout: lane
    // (li, grp) of tile u holds S[d][j0 + 4 grp + r] with d = (wq*NDW + u)*16 + li.
    f32x4 S[NDW];
    #pragma unroll
    for (int u = 0; u < NDW; ++u) S[u] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (state_role && p.state_in) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = (wq * NDW + u) * 16 + li;
            S[u] = *reinterpret_cast<const f32x4*>(p.state_in + ((int64_t)h * DK + d) * dv + j0 + 4 * grp);
        }
    }

    using St = Stage<F32, PK>;

    // ---------------------------------------------------------- state role
    // Every global access of the state loop is issued unconditionally (chunks
    // past the end get an empty buffer range: loads read zeros, stores are
    // dropped), so the compiler's in-order memory counters stay exact and the
    // prefetch of chunk c + 2 is never drained while chunk c computes.
    auto load_chunk = [&](St& R, int64_t c) {
        const int64_t t0 = c * CH;
        const int64_t rows = T - t0;
        const rsrc_t rk = make_rsrc(static_cast<const char*>(p.k) + t0 * qk_row, rows * qk_row);
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = st + NS_T * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            load_piece<F32>(R.kp[u], rk, (uint32_t)(m * qk_row + ((int64_t)h * DK + d0) * ES));
        }
        // V slice: 128 pieces for state threads 0..127; threads 128..255 fetch
        // the same pieces (L2 hits) so that all state waves run one stream
        const rsrc_t rv = make_rsrc(static_cast<const char*>(p.v) + t0 * v_row, rows * v_row);
        const int vs = st & 127;
        load_piece<F32>(R.vp, rv, (uint32_t)((vs >> 1) * v_row + ((int64_t)h * dv + j0 + (vs & 1) * 8) * ES));
        const rsrc_t rg = make_rsrc(p.g + t0 * H, rows * H * 4);
        R.g = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, (uint32_t)((lane * H + h) * 4), 0, 0));
    };

    auto store_chunk = [&](const St& R, int b) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = st + NS_T * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            bf16x8 hi, lo;
            split_piece<F32>(R.kp[u], hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.k[b][0][m * KP + d0]) = hi;
            if (F32) *reinterpret_cast<bf16x8*>(&sm.k[b][NL - 1][m * KP + d0]) = lo;
        }
        // every state wave scans the chunk's log-gates: lane t holds G_t
        const float x = wave_inclusive_sum(R.g);
        const float glast = lane_value(x, 63);
        const float wl = __expf(glast - x);  // w_t = exp(G_last - G_t)
        const int vs = st & 127;
        const float wm = __shfl(wl, vs >> 1, 64);
        if (wave < 6) {  // V rows: raw (hi, lo) and V w (hi, lo)
            const int m = vs >> 1;
            const int jj = (vs & 1) * 8;
            float f[8];
            piece_f32<F32>(R.vp, f);
            bf16x8 hi, lo;
            split_piece<F32>(R.vp, hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.v[b][0][m * VP + jj]) = hi;
            if (F32) *reinterpret_cast<bf16x8*>(&sm.v[b][NL - 1][m * VP + jj]) = lo;
            #pragma unroll
            for (int e = 0; e < 8; ++e) f[e] *= wm;
            split8(f, hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.vw[b][0][m * VP + jj]) = hi;
            *reinterpret_cast<bf16x8*>(&sm.vw[b][1][m * VP + jj]) = lo;
        }
        if (wave == 4) {  // decay tables
            float ge[4];
            #pragma unroll
            for (int M = 0; M < 4; ++M) ge[M] = lane_value(x, 16 * M + 15);
            const int blk = lane >> 4;
            sm.G2[b][lane] = x * LOG2E;
            sm.eG[b][lane] = __expf(x);
            sm.bm[b][lane] = __expf(ge[blk] - x);
            f32x4 a;
            #pragma unroll
            for (int M = 0; M < 4; ++M) a[M] = (M < blk) ? __expf(x - ge[M]) : 0.0f;
            *reinterpret_cast<f32x4*>(&sm.ai[b][lane][0]) = a;
        }
    };

    // S_j split into bf16 hi/lo planes [d][j] for the next chunk's X^T.
    auto publish_state = [&](int b) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = (wq * NDW + u) * 16 + li;
            bf16x4 hi, lo;
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const __bf16 x = (__bf16)S[u][r];
                hi[r] = x;
                lo[r] = (__bf16)(S[u][r] - (float)x);
            }
            *reinterpret_cast<bf16x4*>(&sm.s[b][0][d * VP + 4 * grp]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.s[b][1][d * VP + 4 * grp]) = lo;
        }
    };

    // S^T = exp(G_last) S^T + (V w)^T K over this wave's tiles
    auto fold = [&](int b) {
        const float decay = sm.eG[b][CH - 1];
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            #pragma unroll
            for (int r = 0; r < 4; ++r) S[u][r] *= decay;
        }
        #pragma unroll
        for (int mm = 0; mm < 2; ++mm) {
            const int m0 = 32 * mm + 8 * grp;
            const bf16x8 wh = cat(tr4(sm.vw[b][0], VP, m0, 0, li), tr4(sm.vw[b][0], VP, m0 + 4, 0, li));
            const bf16x8 wlo = cat(tr4(sm.vw[b][1], VP, m0, 0, li), tr4(sm.vw[b][1], VP, m0 + 4, 0, li));
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                const int n0 = (wq * NDW + u) * 16;
                const bf16x8 kh = cat(tr4(sm.k[b][0], KP, m0, n0, li), tr4(sm.k[b][0], KP, m0 + 4, n0, li));
                S[u] = mma(wh, kh, S[u]);
                S[u] = mma(wlo, kh, S[u]);
                if (F32) {
                    const bf16x8 kl = cat(tr4(sm.k[b][NL - 1], KP, m0, n0, li),
                                          tr4(sm.k[b][NL - 1], KP, m0 + 4, n0, li));
                    S[u] = mma(wh, kl, S[u]);
                }
            }
        }
    };

    // --------------------------------------------------------- output role
    using QS = QStage<F32, NKK>;
    // this output wave's 16 rows of Q for chunk c, straight into registers
    auto load_q = [&](QS& Q, int64_t c) {
        const int64_t t0 = c * CH;
        const rsrc_t rq = make_rsrc(static_cast<const char*>(p.q) + t0 * qk_row, (T - t0) * qk_row);
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk)
            load_piece<F32>(Q.qp[kk], rq, (uint32_t)((16 * wq + li) * qk_row + ((int64_t)h * DK + 32 * kk + 8 * grp) * ES));
    };

    auto outputs = [&](int b, int64_t c, const QS& Q) {
        const int w = wq;
        const int i_row = 16 * w + li;
        bf16x8 qh[NKK], ql[NKK];
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) split_piece<F32>(Q.qp[kk], qh[kk], ql[kk]);
        // A^T = K Q^T for the causal m-blocks mb <= w (uniform branch); lane
        // (li, grp) of tile mb holds A^T[m = 16 mb + 4 grp + r][i = 16 w + li]
        f32x4 at[4];
        #pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            at[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (mb <= w) {
                bf16x8 a[NKK], al[NKK];
                #pragma unroll
                for (int kk = 0; kk < NKK; ++kk) {
                    const int off = (mb * 16 + li) * KP + 32 * kk + 8 * grp;
                    a[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[b][0][off]);
                    if (F32) al[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[b][NL - 1][off]);
                }
                #pragma unroll
                for (int kk = 0; kk < NKK; ++kk) {
                    at[mb] = mma(a[kk], qh[kk], at[mb]);
                    if (F32) {
                        at[mb] = mma(a[kk], ql[kk], at[mb]);
                        at[mb] = mma(al[kk], qh[kk], at[mb]);
                    }
                }
            }
        }
        // decay: factored tables below the diagonal tile, exp2 on it
        {
            const f32x4 ai = *reinterpret_cast<const f32x4*>(&sm.ai[b][i_row][0]);
            #pragma unroll
            for (int mb = 0; mb < 4; ++mb) {
                if (mb < w) {
                    const f32x4 bmv = *reinterpret_cast<const f32x4*>(&sm.bm[b][mb * 16 + 4 * grp]);
                    #pragma unroll
                    for (int r = 0; r < 4; ++r) at[mb][r] = (at[mb][r] * ai[mb]) * bmv[r];
                } else if (mb == w) {
                    const float gi = sm.G2[b][i_row];
                    const f32x4 gm = *reinterpret_cast<const f32x4*>(&sm.G2[b][mb * 16 + 4 * grp]);
                    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float pv = at[mb][r] * __builtin_amdgcn_exp2f(gi - gm[r]);
                        at[mb][r] = (4 * grp + r <= li) ? pv : 0.0f;
                    }
                }
            }
        }
        // O^T = V^T P^T, two m-blocks per MFMA; lane (li, grp) ends with
        // O[i = 16 w + li][j0 + 4 grp + r]
        f32x4 acc_o = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int pr = 0; pr < 2; ++pr) {
            if (2 * pr <= w) {
                float f[8];
                #pragma unroll
                for (int r = 0; r < 4; ++r) {
                    f[r] = at[2 * pr][r];
                    f[4 + r] = at[2 * pr + 1][r];
                }
                bf16x8 ph, pl;
                split8(f, ph, pl);
                const bf16x8 vh = cat(tr4(sm.v[b][0], VP, (2 * pr) * 16 + 4 * grp, 0, li),
                                      tr4(sm.v[b][0], VP, (2 * pr + 1) * 16 + 4 * grp, 0, li));
                acc_o = mma(vh, ph, acc_o);
                acc_o = mma(vh, pl, acc_o);
                if (F32) {
                    const bf16x8 vl = cat(tr4(sm.v[b][NL - 1], VP, (2 * pr) * 16 + 4 * grp, 0, li),
                                          tr4(sm.v[b][NL - 1], VP, (2 * pr + 1) * 16 + 4 * grp, 0, li));
                    acc_o = mma(vl, ph, acc_o);
                }
            }
        }
        // X^T = S_j^T Q^T from the published S planes, hi and lo products in
        // two independent accumulators
        f32x4 acc_x = {0.f, 0.f, 0.f, 0.f}, acc_xl = {0.f, 0.f, 0.f, 0.f};
        {
            bf16x8 sh[NKK], sl[NKK];
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                const int k0 = 32 * kk + 8 * grp;
                sh[kk] = cat(tr4(sm.s[b][0], VP, k0, 0, li), tr4(sm.s[b][0], VP, k0 + 4, 0, li));
                sl[kk] = cat(tr4(sm.s[b][1], VP, k0, 0, li), tr4(sm.s[b][1], VP, k0 + 4, 0, li));
            }
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                acc_x = mma(sh[kk], qh[kk], acc_x);
                acc_xl = mma(sl[kk], qh[kk], acc_xl);
                if (F32) acc_xl = mma(sh[kk], ql[kk], acc_xl);
            }
            acc_x += acc_xl;
        }
        // o row i = 16 w + li, columns j0 + 4 grp .. + 3: one 16-byte store;
        // rows past T fall outside the chunk's buffer range and are dropped
        {
            const int64_t t0 = c * CH;
            const rsrc_t ro = make_rsrc(reinterpret_cast<const char*>(p.o) + t0 * o_row, (T - t0) * o_row);
            const float eg = sm.eG[b][i_row];
            f32x4 val;
            #pragma unroll
            for (int r = 0; r < 4; ++r) val[r] = p.scale * (eg * acc_x[r] + acc_o[r]);
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, val), ro,
                                                   (uint32_t)(i_row * o_row + ((int64_t)h * dv + j0 + 4 * grp) * 4), 0, 0);
        }
    };

    // One loop per role; both run the same number of barriers.  The loops
    // advance two chunks per iteration so that the two register stages swap
    // roles without copies; a chunk index past the end does no visible work.
    // One loop per role; both run one barrier per chunk.  Each loop advances
    // three chunks per iteration so that three register stages rotate
    // without copies (loads run three chunks ahead); a chunk index past the
    // end issues only empty-range memory accesses and skips the barrier.
    if (state_role) {
        auto state_step = [&](int64_t c, St& Rfree, const St& Rnext) {
            const int b = (int)(c & 1);
            load_chunk(Rfree, c + 3);
            if (c + 1 < n_chunks) store_chunk(Rnext, b ^ 1);
            {
                const bool live = c < n_chunks && p.chunk_states != nullptr;
                const rsrc_t rc = make_rsrc(p.chunk_states + (live ? c : 0) * (int64_t)H * DK * dv,
                                            live ? (int64_t)H * DK * dv * 4 : 0);
                #pragma unroll
                for (int u = 0; u < NDW; ++u) {
                    const int d = (wq * NDW + u) * 16 + li;
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, S[u]), rc,
                                                           (uint32_t)((((int64_t)h * DK + d) * dv + j0 + 4 * grp) * 4), 0, 0);
                }
            }
            if (c < n_chunks) {
                fold(b);
                publish_state(b ^ 1);
                lds_barrier();
            }
        };
        St R0, R1, R2;
        load_chunk(R0, 0);
        load_chunk(R1, 1);
        load_chunk(R2, 2);
        store_chunk(R0, 0);
        publish_state(0);
        lds_barrier();
        for (int64_t c = 0; c < n_chunks; c += 3) {
            state_step(c, R0, R1);
            state_step(c + 1, R1, R2);
            state_step(c + 2, R2, R0);
        }
        if (p.final_state) {
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                const int d = (wq * NDW + u) * 16 + li;
                *reinterpret_cast<f32x4*>(p.final_state + ((int64_t)h * DK + d) * dv + j0 + 4 * grp) = S[u];
            }
        }
    } else {
        auto out_step = [&](int64_t c, QS& Q) {
            outputs((int)(c & 1), c, Q);  // past the end: reads stale LDS, stores nothing
            load_q(Q, c + 3);
            if (c < n_chunks) lds_barrier();
        };
        QS Q0, Q1, Q2;
        load_q(Q0, 0);
        load_q(Q1, 1);
        load_q(Q2, 2);
        lds_barrier();
        for (int64_t c = 0; c < n_chunks; c += 3) {
            out_step(c, Q0);
            out_step(c + 1, Q1);
            out_step(c + 2, Q2);
        }
    }
}

template <int DK, bool F32>
hipError_t launch_t(const ScanParams& p, hipStream_t stream) {
    const unsigned grid = (unsigned)(p.H * (p.dv / DVS));
    hipLaunchKernelGGL((linattn_scan_kernel<DK, F32>), dim3(grid), dim3(NT), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_linattn_scan(const ScanParams& p, hipStream_t stream) {
    // fp32 inputs keep hi and lo planes of K, Q and V in LDS; at dk = 128 that
    // exceeds the 160 KiB of LDS, so fp32 inputs are limited to dk = 64.
    if (p.dk == 128 && !p.in_f32) return launch_t<128, false>(p, stream);
    if (p.dk == 64) return p.in_f32 ? launch_t<64, true>(p, stream) : launch_t<64, false>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
