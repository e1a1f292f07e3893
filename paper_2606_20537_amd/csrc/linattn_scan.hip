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
// Four waves; wave w owns rows 16w..16w+15 of the chunk for the outputs and
// DK/64 of the DK/16 row tiles of the state.  Every product runs on
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation:
//   A^T = K Q^T          exact bf16 operands (inputs), causal tiles only
//   O  += P V            P = A * decay mask, split hi + lo in bf16
//   X   = Q S_j          S_j fp32, split hi + lo in bf16
//   S   = exp(G_last) S + (K * w)^T V   K * w split hi + lo in bf16
// The hi/lo split keeps fp32-derived operands to ~2^-17 relative error, far
// inside the 2e-3 parity bar, while inputs stay exact.  fp32 inputs (the tiny
// workload) are split hi + lo on load and use three products per term.
//
// Operand placement uses the fact that the contraction index may be permuted
// freely as long as both operands agree: the accumulator of K Q^T already
// holds, per lane, the P entries that P V needs as its A operand, and the
// state accumulator holds what Q S needs as its B operand once written to LDS
// as S^T.  K and V are staged in LDS (K row-major and transposed, V
// transposed); Q is read straight into registers.  Loads of chunk j+1 are
// issued before chunk j's math and written to the other LDS stage after it,
// with one barrier per chunk.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int CH = 64;        // chunk length
constexpr int DVS = 16;       // value columns per workgroup
constexpr int NT = 256;       // threads per workgroup (4 waves)
constexpr int MP = CH + 8;    // pitch (elements) of the transposed [x][m] tiles

__device__ inline f32x4 mma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

template <int DK, bool F32>
struct Smem {
    static constexpr int KP = DK + 8;      // row pitch of K and S^T (elements)
    static constexpr int NL = F32 ? 2 : 1; // bf16 planes: hi (and lo)
    __bf16 k[2][NL][CH * KP];    // K  [m][d]
    __bf16 kt[2][NL][DK * MP];   // K^T [d][m]
    __bf16 vt[2][NL][DVS * MP];  // V^T [j][m] of this slice
    float G[2][CH];              // inclusive cumulative log-decay
    float eG[2][CH];             // exp(G_i)
    float wL[2][CH];             // exp(G_last - G_m)
    __bf16 st[2][2][DVS * KP];   // S^T [j][d], hi and lo planes
};

// 8 consecutive input elements of one row (16 B of bf16 or 32 B of fp32).
template <bool F32>
struct Piece {
    u32x4 x[F32 ? 2 : 1];
};

template <bool F32>
__device__ inline void load_piece(Piece<F32>& p, const void* base, int64_t elem, bool valid) {
    if (F32) {
        const u32x4* s = reinterpret_cast<const u32x4*>(static_cast<const float*>(base) + elem);
        p.x[0] = valid ? s[0] : u32x4{0, 0, 0, 0};
        p.x[F32 ? 1 : 0] = valid ? s[1] : u32x4{0, 0, 0, 0};
    } else {
        const u32x4* s = reinterpret_cast<const u32x4*>(static_cast<const __bf16*>(base) + elem);
        p.x[0] = valid ? s[0] : u32x4{0, 0, 0, 0};
    }
}

// Split a piece into bf16 hi (and lo, for fp32 inputs) vectors.
template <bool F32>
__device__ inline void split_piece(const Piece<F32>& p, bf16x8& hi, bf16x8& lo) {
    if (F32) {
        const f32x4 a = __builtin_bit_cast(f32x4, p.x[0]);
        const f32x4 b = __builtin_bit_cast(f32x4, p.x[F32 ? 1 : 0]);
        float f[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
            const __bf16 h = (__bf16)f[e];
            hi[e] = h;
            lo[e] = (__bf16)(f[e] - (float)h);
        }
    } else {
        hi = __builtin_bit_cast(bf16x8, p.x[0]);
        lo = bf16x8{};
    }
}

__device__ inline void split8(const float* f, bf16x8& hi, bf16x8& lo) {
    #pragma unroll
    for (int e = 0; e < 8; ++e) {
        const __bf16 h = (__bf16)f[e];
        hi[e] = h;
        lo[e] = (__bf16)(f[e] - (float)h);
    }
}

template <int DK, bool F32>
__global__ __launch_bounds__(NT) void linattn_scan_kernel(const ScanParams p) {
    using S_ = Smem<DK, F32>;
    constexpr int KP = S_::KP;
    constexpr int NL = S_::NL;
    constexpr int NKK = DK / 32;           // k-steps of 32 over dk
    constexpr int PK = (CH * DK / 8) / NT; // K pieces per thread per chunk
    constexpr int NDW = DK / 64;           // state row tiles per wave
    __shared__ S_ sm;

    const int tid = threadIdx.x;
    const int w = tid >> 6;
    const int lane = tid & 63;
    const int li = lane & 15;
    const int grp = lane >> 4;

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

    // ---- state S[:, j0:j0+16] in accumulator layout: tile u covers rows
    // (w*NDW+u)*16 + 4*grp + r, column j0 + li.
    f32x4 S[NDW];
    #pragma unroll
    for (int u = 0; u < NDW; ++u) {
        #pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int d = (w * NDW + u) * 16 + 4 * grp + r;
            S[u][r] = p.state_in ? p.state_in[((int64_t)h * DK + d) * dv + j0 + li] : 0.0f;
        }
    }

    // ---- register staging of one chunk
    Piece<F32> kp[PK];
    Piece<F32> vp;
    Piece<F32> qp[NKK];
    float gval = 0.0f;

    auto load_chunk = [&](int64_t c) {
        const int64_t t0 = c * CH;
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = tid + NT * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            const int64_t t = t0 + m;
            load_piece<F32>(kp[u], p.k, (t * H + h) * DK + d0, t < T);
        }
        {
            const int m = (tid >> 1) & 63;
            const int jj = (tid & 1) * 8;
            const int64_t t = t0 + m;
            load_piece<F32>(vp, p.v, (t * H + h) * dv + j0 + jj, tid < 2 * CH && t < T);
        }
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const int64_t t = t0 + 16 * w + li;
            load_piece<F32>(qp[kk], p.q, (t * H + h) * DK + 32 * kk + 8 * grp, t < T);
        }
        if (w == 0) {
            const int64_t t = t0 + lane;
            gval = (t < T) ? p.g[t * H + h] : 0.0f;
        }
    };

    bf16x8 qh[NKK], ql[NKK];

    auto store_chunk = [&](int b) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = tid + NT * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            bf16x8 hi, lo;
            split_piece<F32>(kp[u], hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.k[b][0][m * KP + d0]) = hi;
            if (F32) *reinterpret_cast<bf16x8*>(&sm.k[b][NL - 1][m * KP + d0]) = lo;
            #pragma unroll
            for (int e = 0; e < 8; ++e) {
                sm.kt[b][0][(d0 + e) * MP + m] = hi[e];
                if (F32) sm.kt[b][NL - 1][(d0 + e) * MP + m] = lo[e];
            }
        }
        if (tid < 2 * CH) {
            const int m = (tid >> 1) & 63;
            const int jj = (tid & 1) * 8;
            bf16x8 hi, lo;
            split_piece<F32>(vp, hi, lo);
            #pragma unroll
            for (int e = 0; e < 8; ++e) {
                sm.vt[b][0][(jj + e) * MP + m] = hi[e];
                if (F32) sm.vt[b][NL - 1][(jj + e) * MP + m] = lo[e];
            }
        }
        if (w == 0) {
            float x = gval;
            #pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const float y = __shfl_up(x, off, 64);
                if (lane >= off) x += y;
            }
            const float glast = __shfl(x, 63, 64);
            sm.G[b][lane] = x;
            sm.eG[b][lane] = __expf(x);
            sm.wL[b][lane] = __expf(glast - x);
        }
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) split_piece<F32>(qp[kk], qh[kk], ql[kk]);
    };

    auto publish_state = [&](int b) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = (w * NDW + u) * 16 + 4 * grp;
            bf16x4 hi, lo;
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const __bf16 x = (__bf16)S[u][r];
                hi[r] = x;
                lo[r] = (__bf16)(S[u][r] - (float)x);
            }
            *reinterpret_cast<bf16x4*>(&sm.st[b][0][li * KP + d]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.st[b][1][li * KP + d]) = lo;
        }
    };

    if (n_chunks > 0) {
        load_chunk(0);
        store_chunk(0);
        publish_state(0);
    }
    __syncthreads();

    for (int64_t c = 0; c < n_chunks; ++c) {
        const int b = (int)(c & 1);
        const int64_t t0 = c * CH;
        if (c + 1 < n_chunks) load_chunk(c + 1);

        if (p.chunk_states) {
            float* cs = p.chunk_states + ((c * H + h) * DK) * (int64_t)dv + j0 + li;
            #pragma unroll
            for (int u = 0; u < NDW; ++u)
                #pragma unroll
                for (int r = 0; r < 4; ++r)
                    cs[(int64_t)((w * NDW + u) * 16 + 4 * grp + r) * dv] = S[u][r];
        }

        // ---- A^T = K Q^T for the causal tiles (m-block mb <= w)
        f32x4 at[4];
        #pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            at[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (mb <= w) {
                #pragma unroll
                for (int kk = 0; kk < NKK; ++kk) {
                    const int off = (mb * 16 + li) * KP + 32 * kk + 8 * grp;
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sm.k[b][0][off]);
                    at[mb] = mma(a, qh[kk], at[mb]);
                    if (F32) {
                        const bf16x8 al = *reinterpret_cast<const bf16x8*>(&sm.k[b][NL - 1][off]);
                        at[mb] = mma(a, ql[kk], at[mb]);
                        at[mb] = mma(al, qh[kk], at[mb]);
                    }
                }
            }
        }
        // ---- decay mask: P[i][m] = A[i][m] exp(G_i - G_m) for m <= i
        {
            const int i = 16 * w + li;
            const float Gi = sm.G[b][i];
            #pragma unroll
            for (int mb = 0; mb < 4; ++mb) {
                if (mb <= w) {
                    #pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int m = mb * 16 + 4 * grp + r;
                        at[mb][r] = (m <= i) ? at[mb][r] * __expf(Gi - sm.G[b][m]) : 0.0f;
                    }
                }
            }
        }
        // ---- O_intra = P V (pairs of m-blocks per MFMA)
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
                const int o0 = li * MP + (2 * pr) * 16 + 4 * grp;
                const int o1 = li * MP + (2 * pr + 1) * 16 + 4 * grp;
                bf16x8 vh;
                const bf16x4 va = *reinterpret_cast<const bf16x4*>(&sm.vt[b][0][o0]);
                const bf16x4 vb = *reinterpret_cast<const bf16x4*>(&sm.vt[b][0][o1]);
                #pragma unroll
                for (int e = 0; e < 4; ++e) { vh[e] = va[e]; vh[4 + e] = vb[e]; }
                acc_o = mma(ph, vh, acc_o);
                acc_o = mma(pl, vh, acc_o);
                if (F32) {
                    bf16x8 vl;
                    const bf16x4 la = *reinterpret_cast<const bf16x4*>(&sm.vt[b][NL - 1][o0]);
                    const bf16x4 lb = *reinterpret_cast<const bf16x4*>(&sm.vt[b][NL - 1][o1]);
                    #pragma unroll
                    for (int e = 0; e < 4; ++e) { vl[e] = la[e]; vl[4 + e] = lb[e]; }
                    acc_o = mma(ph, vl, acc_o);
                }
            }
        }
        // ---- X = Q S_j (S_j from the published S^T planes)
        f32x4 acc_x = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const int off = li * KP + 32 * kk + 8 * grp;
            const bf16x8 sh = *reinterpret_cast<const bf16x8*>(&sm.st[b][0][off]);
            const bf16x8 sl = *reinterpret_cast<const bf16x8*>(&sm.st[b][1][off]);
            acc_x = mma(qh[kk], sh, acc_x);
            acc_x = mma(qh[kk], sl, acc_x);
            if (F32) acc_x = mma(ql[kk], sh, acc_x);
        }
        // ---- outputs of rows 16w + 4grp + r
        #pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * w + 4 * grp + r;
            const int64_t t = t0 + i;
            if (t < T) {
                const float val = p.scale * (sm.eG[b][i] * acc_x[r] + acc_o[r]);
                p.o[(t * H + h) * (int64_t)dv + j0 + li] = val;
            }
        }
        // ---- state fold: S = exp(G_last) S + (K * wL)^T V
        {
            const float decay = sm.eG[b][CH - 1];
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                #pragma unroll
                for (int r = 0; r < 4; ++r) S[u][r] *= decay;
            }
            #pragma unroll
            for (int mm = 0; mm < 2; ++mm) {
                const int m0 = 32 * mm + 8 * grp;
                float wl[8];
                #pragma unroll
                for (int e = 0; e < 8; ++e) wl[e] = sm.wL[b][m0 + e];
                const bf16x8 vh = *reinterpret_cast<const bf16x8*>(&sm.vt[b][0][li * MP + m0]);
                bf16x8 vl;
                if (F32) vl = *reinterpret_cast<const bf16x8*>(&sm.vt[b][NL - 1][li * MP + m0]);
                #pragma unroll
                for (int u = 0; u < NDW; ++u) {
                    const int d = (w * NDW + u) * 16 + li;
                    const bf16x8 kh = *reinterpret_cast<const bf16x8*>(&sm.kt[b][0][d * MP + m0]);
                    float f[8];
                    if (F32) {
                        const bf16x8 kl = *reinterpret_cast<const bf16x8*>(&sm.kt[b][NL - 1][d * MP + m0]);
                        #pragma unroll
                        for (int e = 0; e < 8; ++e) f[e] = ((float)kh[e] + (float)kl[e]) * wl[e];
                    } else {
                        #pragma unroll
                        for (int e = 0; e < 8; ++e) f[e] = (float)kh[e] * wl[e];
                    }
                    bf16x8 ah, al;
                    split8(f, ah, al);
                    S[u] = mma(ah, vh, S[u]);
                    S[u] = mma(al, vh, S[u]);
                    if (F32) S[u] = mma(ah, vl, S[u]);
                }
            }
        }
        // ---- hand the new state and the next chunk to the other stage
        publish_state(b ^ 1);
        if (c + 1 < n_chunks) store_chunk(b ^ 1);
        __syncthreads();
    }

    if (p.final_state) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u)
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int d = (w * NDW + u) * 16 + 4 * grp + r;
                p.final_state[((int64_t)h * DK + d) * dv + j0 + li] = S[u][r];
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
    // fp32 inputs keep hi and lo planes of every staged tile; at dk = 128 that
    // exceeds the 160 KiB of LDS, so fp32 inputs are limited to dk = 64.
    if (p.dk == 128 && !p.in_f32) return launch_t<128, false>(p, stream);
    if (p.dk == 64) return p.in_f32 ? launch_t<64, true>(p, stream) : launch_t<64, false>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
