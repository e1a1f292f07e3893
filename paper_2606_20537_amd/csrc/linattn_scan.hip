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
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation, written transposed so that
// each lane ends with four consecutive value columns (16-byte stores):
//   A^T = K Q^T              exact bf16 operands (inputs)
//   O^T = V^T P^T            P = A * causal decay mask, split hi + lo in bf16
//   X^T = S_j^T Q^T          S_j fp32, split hi + lo in bf16
//   S^T = exp(G_last) S^T + (V w)^T K     w_m = exp(G_last - G_m) scales the
//                            16-wide V slice (not the dk-wide K), V w split
//                            hi + lo, K exact
// The hi/lo split keeps fp32-derived operands to ~2^-17 relative error, far
// inside the 2e-3 parity bar, while inputs stay exact.  fp32 inputs are split
// hi + lo on load and use three products per term.
//
// LDS holds every tile row-major (K, V, V w and the published S), written with
// 8- and 16-byte stores.  Operands whose contraction index runs along the rows
// (V^T, (V w)^T, S^T as A operands; K as the fold's B operand) are read with
// gfx950's transposing LDS load ds_read_b64_tr_b16: inside a 16-lane group,
// lane L addresses row k0 + L/4, columns 4(L%4)..+3, and lane n receives
// column n of rows k0..k0+3.  The contraction index may be permuted freely as
// long as both operands agree, which lets the accumulator of K Q^T serve
// directly as the B operand of V^T P^T.  Loads run two chunks ahead in
// registers and land in the other LDS stage after the current chunk's math;
// the one barrier per chunk orders LDS only and never waits for global stores.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int CH = 64;        // chunk length
constexpr int DVS = 16;       // value columns per workgroup
constexpr int NT = 256;       // threads per workgroup (4 waves)
constexpr int VP = DVS + 8;   // pitch (elements) of the [m][j] and [d][j] tiles

__device__ inline f32x4 mma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Transposing LDS read of a row-major tile with `pitch` elements per row:
// lane n of each 16-lane group gets tile[k0 + 0..3][n0 + n].
__device__ inline bf16x4 tr4(const __bf16* tile, int pitch, int k0, int n0, int li) {
    const __bf16* p = tile + (k0 + (li >> 2)) * pitch + n0 + 4 * (li & 3);
    const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
    return __builtin_bit_cast(bf16x4, v);
}

__device__ inline bf16x8 cat(const bf16x4& a, const bf16x4& b) {
    return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
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

template <int DK, bool F32>
struct Smem {
    static constexpr int KP = DK + 8;      // row pitch of K (elements)
    static constexpr int NL = F32 ? 2 : 1; // bf16 planes of the inputs: hi (and lo)
    __bf16 k[2][NL][CH * KP];    // K     [m][d]
    __bf16 v[2][NL][CH * VP];    // V     [m][j] (this slice)
    __bf16 vw[2][2][CH * VP];    // V w   [m][j], hi and lo planes
    float G[2][CH];              // inclusive cumulative log-decay
    float eG[2][CH];             // exp(G_i)
    __bf16 s[2][2][DK * VP];     // S_j   [d][j], hi and lo planes
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

// Register staging of one chunk's global loads.
template <bool F32, int PK, int NKK>
struct Stage {
    Piece<F32> kp[PK];
    Piece<F32> vp;
    Piece<F32> qp[NKK];
    float g;
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
    constexpr int NKK = DK / 32;           // k-steps of 32 over dk
    constexpr int PK = (CH * DK / 8) / NT; // K pieces per thread per chunk
    constexpr int NDW = DK / 64;           // state tiles (16 rows of d) per wave
    __shared__ S_ sm;

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, uniform
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

    // ---- state, as S^T tiles in accumulator layout: lane (li, grp) of tile u
    // holds S[d][j0 + 4 grp + r], r = 0..3, with d = (w*NDW + u)*16 + li.
    f32x4 S[NDW];
    #pragma unroll
    for (int u = 0; u < NDW; ++u) {
        const int d = (w * NDW + u) * 16 + li;
        S[u] = p.state_in ? *reinterpret_cast<const f32x4*>(p.state_in + ((int64_t)h * DK + d) * dv + j0 + 4 * grp)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
    }

    using St = Stage<F32, PK, NKK>;
    St R0, R1;
    bf16x8 qh[NKK], ql[NKK];

    auto load_chunk = [&](St& R, int64_t c) {
        const int64_t t0 = c * CH;
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = tid + NT * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            const int64_t t = t0 + m;
            load_piece<F32>(R.kp[u], p.k, (t * H + h) * DK + d0, t < T);
        }
        {
            const int m = (tid >> 1) & 63;
            const int jj = (tid & 1) * 8;
            const int64_t t = t0 + m;
            load_piece<F32>(R.vp, p.v, (t * H + h) * dv + j0 + jj, tid < 2 * CH && t < T);
        }
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            const int64_t t = t0 + 16 * w + li;
            load_piece<F32>(R.qp[kk], p.q, (t * H + h) * DK + 32 * kk + 8 * grp, t < T);
        }
        const int64_t tg = t0 + lane;
        R.g = (tg < T) ? p.g[tg * H + h] : 0.0f;
    };

    auto store_chunk = [&](const St& R, int b) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = tid + NT * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            bf16x8 hi, lo;
            split_piece<F32>(R.kp[u], hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.k[b][0][m * KP + d0]) = hi;
            if (F32) *reinterpret_cast<bf16x8*>(&sm.k[b][NL - 1][m * KP + d0]) = lo;
        }
        // every wave scans the chunk's log-gates (lane t holds G_t)
        float x = R.g;
        #pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const float y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        const float glast = __shfl(x, 63, 64);
        const float wl = __expf(glast - x);  // w_t = exp(G_last - G_t)
        if (w == 0) {
            sm.G[b][lane] = x;
            sm.eG[b][lane] = __expf(x);
        }
        if (tid < 2 * CH) {  // V rows: raw (hi, lo) and V w (hi, lo)
            const int m = (tid >> 1) & 63;
            const int jj = (tid & 1) * 8;
            const float wm = __shfl(wl, m, 64);
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
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) split_piece<F32>(R.qp[kk], qh[kk], ql[kk]);
    };

    // S_j split into bf16 hi/lo planes [d][j] for the next chunk's X^T.
    auto publish_state = [&](int b) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = (w * NDW + u) * 16 + li;
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

    auto chunk_body = [&](int64_t c, St& Rfree, const St& Rnext) {
        const int b = (int)(c & 1);
        const int64_t t0 = c * CH;
        if (c + 2 < n_chunks) load_chunk(Rfree, c + 2);

        if (p.chunk_states) {
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                const int d = (w * NDW + u) * 16 + li;
                *reinterpret_cast<f32x4*>(p.chunk_states + ((c * H + h) * DK + d) * (int64_t)dv + j0 + 4 * grp) = S[u];
            }
        }

        // ---- A^T = K Q^T, all four m-blocks; lane (li, grp) of tile mb holds
        // A^T[m = 16 mb + 4 grp + r][i = 16 w + li]
        f32x4 at[4];
        #pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            bf16x8 a[NKK], al[NKK];
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                const int off = (mb * 16 + li) * KP + 32 * kk + 8 * grp;
                a[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[b][0][off]);
                if (F32) al[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[b][NL - 1][off]);
            }
            at[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                at[mb] = mma(a[kk], qh[kk], at[mb]);
                if (F32) {
                    at[mb] = mma(a[kk], ql[kk], at[mb]);
                    at[mb] = mma(al[kk], qh[kk], at[mb]);
                }
            }
        }
        // ---- causal decay mask: P[i][m] = A[i][m] exp(G_i - G_m) for m <= i
        const int i_row = 16 * w + li;
        {
            const float Gi = sm.G[b][i_row];
            #pragma unroll
            for (int mb = 0; mb < 4; ++mb) {
                const f32x4 Gm = *reinterpret_cast<const f32x4*>(&sm.G[b][mb * 16 + 4 * grp]);
                #pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int m = mb * 16 + 4 * grp + r;
                    const float pv = at[mb][r] * __expf(Gi - Gm[r]);
                    at[mb][r] = (m <= i_row) ? pv : 0.0f;
                }
            }
        }
        // ---- O^T = V^T P^T, two m-blocks per MFMA; lane (li, grp) ends with
        // O[i = 16 w + li][j0 + 4 grp + r]
        f32x4 acc_o = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int pr = 0; pr < 2; ++pr) {
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
        // ---- X^T = S_j^T Q^T from the published S planes
        f32x4 acc_x = {0.f, 0.f, 0.f, 0.f};
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
                acc_x = mma(sl[kk], qh[kk], acc_x);
                if (F32) acc_x = mma(sh[kk], ql[kk], acc_x);
            }
        }
        // ---- o row i = 16 w + li, columns j0 + 4 grp .. + 3 (one 16-byte store)
        {
            const int64_t t = t0 + i_row;
            if (t < T) {
                const float eg = sm.eG[b][i_row];
                f32x4 val;
                #pragma unroll
                for (int r = 0; r < 4; ++r) val[r] = p.scale * (eg * acc_x[r] + acc_o[r]);
                *reinterpret_cast<f32x4*>(p.o + (t * H + h) * (int64_t)dv + j0 + 4 * grp) = val;
            }
        }
        // ---- state fold: S^T = exp(G_last) S^T + (V w)^T K
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
                const bf16x8 wh = cat(tr4(sm.vw[b][0], VP, m0, 0, li), tr4(sm.vw[b][0], VP, m0 + 4, 0, li));
                const bf16x8 wlo = cat(tr4(sm.vw[b][1], VP, m0, 0, li), tr4(sm.vw[b][1], VP, m0 + 4, 0, li));
                #pragma unroll
                for (int u = 0; u < NDW; ++u) {
                    const int n0 = (w * NDW + u) * 16;
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
        }
        // ---- hand the new state and the next chunk to the other stage
        publish_state(b ^ 1);
        if (c + 1 < n_chunks) store_chunk(Rnext, b ^ 1);
        lds_barrier();
    };

    if (n_chunks > 0) {
        load_chunk(R0, 0);
        if (n_chunks > 1) load_chunk(R1, 1);
        store_chunk(R0, 0);
        publish_state(0);
    }
    lds_barrier();

    // two chunks of loads in flight: chunk c + 2 is fetched while c computes
    for (int64_t c = 0; c < n_chunks; c += 2) {
        chunk_body(c, R0, R1);
        if (c + 1 < n_chunks) chunk_body(c + 1, R1, R0);
    }

    if (p.final_state) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d = (w * NDW + u) * 16 + li;
            *reinterpret_cast<f32x4*>(p.final_state + ((int64_t)h * DK + d) * dv + j0 + 4 * grp) = S[u];
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
    if (p.dk == 128) return p.in_f32 ? launch_t<128, true>(p, stream) : launch_t<128, false>(p, stream);
    if (p.dk == 64) return p.in_f32 ? launch_t<64, true>(p, stream) : launch_t<64, false>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
