// Chunked gated linear-attention prefill on gfx950 MFMA.
//
// Per head, S_t = exp(g_t) S_{t-1} + k_t^T v_t and o_t = scale * q_t S_t,
// evaluated chunk by chunk (paper §5: the prefill folds its recurrent state
// once per chunk of C tokens).  For chunk j with entering state S_j and
// inclusive in-chunk log-decay sums G_i:
//   o_i     = scale * (exp(G_i) q_i S_j + sum_{m<=i} exp(G_i - G_m)(q_i.k_m) v_m)
//   S_{j+1} = exp(G_last) S_j + D_j,  D_j = sum_m exp(G_last - G_m) k_m^T v_m
//
// Work split: one workgroup per (head, 16-wide slice of the value columns).
// Column slices of S are independent: o[:, J] needs only S[:, J] and v[:, J],
// and the fold of S[:, J] needs only v[:, J].  The workgroup walks the chunks
// in order, so the arithmetic applied to chunk j depends only on (S_j, the
// chunk's inputs) -- never on the call's length, its first chunk or the grid.
// That is what makes restore-at-an-aligned-boundary-then-continue bitwise
// equal to one long prefill.
//
// Only S_{j+1} = exp(G_last) S_j + D_j is a true recurrence; D_j, the
// intra-chunk scores and their decay do not depend on S.  The kernel is
// therefore a software pipeline over chunks with one LDS barrier per step;
// in step c:
//   state waves 4-7  issue the HBM loads of chunk c+4, stage chunk c+2 in LDS
//                    (K; wave 4 also V and V w; wave 5 writes the decay
//                    tables and fold weights of chunk c+3),
//                    start D_{c+1} on MFMA, write the chunk-boundary state
//                    S_c, then S_{c+1} = exp(G_last) S_c + D_c (one FMA per
//                    element) and publish S_{c+1} for step c+1;
//   output waves 0-3 start A^T_{c+1} = K_{c+1} Q_{c+1}^T (causal tiles) and
//                    finish chunk c: P = A^T * decay, O = P V, X = Q S_c,
//                    o = scale (exp(G) X + O).
// Wave w of the output role owns rows 16w..16w+15 of the chunk; each wave's
// role and row block are template parameters, so the causal tiling compiles
// to straight-line code the scheduler can interleave with the next chunk's
// products.  Stage buffers: K, V w and S by chunk parity, V and the tables by
// chunk mod 4, the register prefetch four chunks deep.
//
// Memory access.  Every 16-column slice of a head reads the head's full Q
// and K rows, so per chunk a workgroup asks L2 for ~380 cache lines, most of
// them also wanted by its sibling slices at the same moment.  With the
// measures below, memory latency is about a fifth of the time; the rest is
// the step period of the eight waves themselves (measured with every load
// and store emptied).  The measures: every load and store
// is coalesced (consecutive lanes touch consecutive bytes of a row); Q rows
// pass through a small per-wave LDS tile to reach operand layout; only one
// wave reads g and V; accumulators are laid out [row][value column] so that
// the 16 lanes of a group store 64 contiguous bytes of o or of a state row;
// and each slice prefetches its eighth of the head's lines into L2 ahead of
// the regular loads (see prefetch below).
//
// Every product runs on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.
// Inputs are exact bf16 operands; fp32-derived operands (P, S_j, V w with
// w_m = exp(G_last - G_m)) are split hi + lo in bf16, which keeps them to
// ~2^-17 relative error, far inside the 2e-3 parity bar.  Scaling the 16-wide
// V slice by w instead of the dk-wide K keeps K exact and the split small.
// fp32 inputs are split hi + lo on load and use three products per term.
//
// Decay: inside the chunk G is non-increasing for g <= 0.  Below the diagonal
// tile, exp(G_i - G_m) = exp(G_i - G_e) exp(G_e - G_m) with e the last token of
// m's 16-token block; both factors lie in (0, 1], come from per-chunk tables
// and never overflow.  The diagonal tile evaluates exp2 directly.
//
// LDS holds every tile row-major (K, V, V w, Q, and the published S as
// S^T), written with 8- and 16-byte stores.  Operands whose contraction index
// runs along the rows (K^T and V w for the fold, V for O) are read with
// gfx950's transposing LDS load ds_read_b64_tr_b16: inside a 16-lane group,
// lane L addresses row k0 + L/4, columns 4(L%4)..+3, and lane n receives
// column n of rows k0..k0+3.  The contraction index may be permuted freely as
// long as both operands agree, which lets the accumulator of K Q^T serve
// directly as the A operand of P V.  HBM traffic goes through buffer
// resources: a scalar base per chunk, fixed per-lane offsets, and hardware
// range checks that read the ragged tail as zeros and drop stores past T.
// The barrier orders LDS only and never waits for global stores.
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "internal.h"

namespace cap {
namespace {

using namespace dev;

constexpr int CH = 64;        // chunk length
constexpr int DVS = 16;       // value columns per workgroup
constexpr int NT = 512;       // threads per workgroup (8 waves)
constexpr int NS_T = 256;     // threads of the state role
constexpr int VP = DVS + 8;   // pitch (elements) of the [m][j] and [d][j] tiles

// Every member starts on a 16-byte boundary so that 16-byte LDS accesses
// compile to single ds_read_b128 / ds_write_b128 instructions.
template <int DK, bool F32>
struct alignas(16) Smem {
    // Row pitches (elements).  K rows are read 16 rows x 16 B at a time and
    // 4 rows x 32 B at a time (transposing reads): a pitch of 16 B times an
    // odd number whose 4-row windows do not overlap keeps both conflict-free
    // (304 B for dk = 128, 208 B for dk = 64).  S^T rows are read 16 x 16 B.
    static constexpr int KP = DK == 128 ? 152 : 104;
    static constexpr int SP = DK + 8;
    static constexpr int NL = F32 ? 2 : 1; // bf16 planes of the inputs: hi (and lo)
    alignas(16) __bf16 k[2][NL][CH * KP];  // K     [m][d]     by chunk parity
    alignas(16) __bf16 v[4][NL][CH * VP];  // V     [m][j]     by chunk mod 4
    alignas(16) __bf16 vw[2][2][CH * VP];  // V w   [m][j]     hi, lo; by chunk parity
    alignas(16) __bf16 s[2][2][DVS * SP];  // S_j^T [j][d]     hi, lo; by chunk parity
    alignas(16) __bf16 q[4][NL][16 * SP];  // Q     [i][d]     each output wave's 16 rows
    alignas(16) float G2[4][CH];           // G_t log2(e), G the inclusive log-decay sum
    alignas(16) float eG[4][CH];           // exp(G_t)
    alignas(16) float bm[4][CH];           // exp(G_e - G_m), e = last token of m's block
    alignas(16) float ai[4][CH][4];        // exp(G_i - G_e(M)) for 16-token blocks M below i's
    alignas(16) float w[4][CH];            // w_t = exp(G_last - G_t), the fold weights
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

// A piece as bf16 hi (and lo, for fp32 inputs).
template <bool F32>
__device__ inline void split_piece(const Piece<F32>& p, bf16x8& hi, bf16x8& lo) {
    if (F32) {
        const f32x4 a = __builtin_bit_cast(f32x4, p.x[0]);
        const f32x4 b = __builtin_bit_cast(f32x4, p.x[F32 ? 1 : 0]);
        float f[8];
        #pragma unroll
        for (int e = 0; e < 4; ++e) { f[e] = a[e]; f[4 + e] = b[e]; }
        split_n<8>(f, hi, lo);
    } else {
        hi = __builtin_bit_cast(bf16x8, p.x[0]);
        lo = bf16x8{};
    }
}

template <bool F32>
__device__ inline void piece_f32(const Piece<F32>& p, float* f) {
    if constexpr (F32) {
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

// Register staging of one chunk for the state role: its K pieces, and for
// the wave that owns the gates also its V slice and the log-gates of the
// next chunk.
template <bool F32, int PK>
struct Stage {
    Piece<F32> kp[PK];
    Piece<F32> vp[2];
    float g;
};

// Register staging of one chunk of Q rows for an output wave: 16-byte pieces
// in coalesced order (consecutive lanes read consecutive bytes of a row).
template <int NQI>
struct QStage {
    u32x4 qp[NQI];
};

// Per-workgroup constants shared by both roles.
struct Ctx {
    int h, j0, H, dv, lane, li, grp;
    int nfull, tail;               // full chunks, rows of the partial last one
    int64_t T, n;                  // tokens, chunks
    int64_t qk_row, v_row, o_row;  // bytes per token of q / k, v, o
};

// Valid rows of chunk c: CH up to the last full chunk, then the tail, then 0
// (chunks past the end).  32-bit arithmetic: the host bounds the number of
// chunks below 2^30, and a chunk's bytes of any tensor below 2^31.
__device__ inline uint32_t chunk_rows(const Ctx& x, int64_t c) {
    const int ci = (int)c;
    return ci < x.nfull ? (uint32_t)CH : (ci == x.nfull ? (uint32_t)x.tail : 0u);
}

// Both roles walk the chunks four steps per loop iteration (the register
// stages rotate without copies).  Every global access of a step is issued
// unconditionally (the chunk-state stores exist only in the instantiation
// that writes chunk states) -- chunks past the end get an empty buffer range: loads
// read zeros, stores are dropped -- so the compiler's in-order memory
// counters stay exact and the prefetch is never drained; a step past the end
// changes no state, writes only LDS buffers no live step reads, and skips
// the barrier.  Both roles run two barriers in the prologue and one per
// chunk; a call of at most one chunk takes a straight-line path through the
// same per-chunk code with a single barrier in both roles.

// ------------------------------------------------------------- state role
// Every state wave stages its share of K, folds and publishes its rows of
// S.  In addition the V wave (wave 4, VW) loads and stages V and V w and
// issues the cooperative L2 prefetch, and the gate wave (wave 5: wq == 1 of
// the plain instantiation, a wave-uniform branch) is the only wave that
// reads the gates -- 64 cache lines per chunk for 256 bytes, since g is
// token-major -- and writes the decay tables and the fold weights w one
// chunk ahead of the V wave, which reads its weights from LDS.  Waves 5-7
// share one instantiation: a separate one for the gate wave measured 10 %
// slower with the same arithmetic.
template <int DK, bool F32, bool ONE, bool CS, bool VW>
__device__ __forceinline__ void state_role(const ScanParams& p, Smem<DK, F32>& sm, const Ctx& x, int wq) {
    const bool GW = !VW && wq == 1;  // wave-uniform
    using S_ = Smem<DK, F32>;
    constexpr int KP = S_::KP;
    constexpr int NL = S_::NL;
    constexpr int ES = F32 ? 4 : 2;
    constexpr int PK = (CH * DK / 8) / NS_T;  // K pieces per state thread
    constexpr int NDW = DK / 64;              // state tiles (16 rows of d) per wave
    using St = Stage<F32, PK>;
    const int lane = x.lane, li = x.li, grp = x.grp, h = x.h, j0 = x.j0, H = x.H, dv = x.dv;
    const int st = 64 * wq + lane;

    // S tiles in accumulator layout: lane (li, grp) of tile u holds
    // S[d][j0 + li] for d = (wq*NDW + u)*16 + 4 grp + r, r = 0..3.  For each
    // r the 16 lanes of a group hold 64 contiguous bytes of a state row, so
    // state reads and writes coalesce.
    constexpr int SP = S_::SP;
    f32x4 S[NDW], D0[NDW], D1[NDW];
    auto srow = [&](int u, int r) -> int64_t {  // element offset of S[d][j0 + li] in a [H][dk][dv] state
        return ((int64_t)h * DK + (wq * NDW + u) * 16 + 4 * grp + r) * dv + j0 + li;
    };
    #pragma unroll
    for (int u = 0; u < NDW; ++u) {
        S[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        if (p.state_in) {
            #pragma unroll
            for (int r = 0; r < 4; ++r) S[u][r] = p.state_in[srow(u, r)];
        }
    }

    auto load_chunk = [&](St& R, int64_t c) {
        const int64_t t0 = c * CH;
        const uint32_t rows = chunk_rows(x, c);
        const rsrc_t rk = make_rsrc_u32(static_cast<const char*>(p.k) + t0 * x.qk_row, rows * (uint32_t)x.qk_row);
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = st + NS_T * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            load_piece<F32>(R.kp[u], rk, (uint32_t)(m * x.qk_row + ((int64_t)h * DK + d0) * ES));
        }
        if constexpr (VW) {
            // V slice (lane l: rows l/2 and 32 + l/2, columns 8 (l%2)..+7),
            // loaded by one wave only, so no two waves wait on the same lines
            const rsrc_t rv = make_rsrc_u32(static_cast<const char*>(p.v) + t0 * x.v_row, rows * (uint32_t)x.v_row);
            #pragma unroll
            for (int i = 0; i < 2; ++i)
                load_piece<F32>(R.vp[i], rv, (uint32_t)(((lane >> 1) + 32 * i) * x.v_row +
                                                        ((int64_t)h * dv + j0 + 8 * (lane & 1)) * ES));
        }
        if ((VW && ONE) || GW) {
            // the log-gates (lane t: token t): the gate wave's, and the V
            // wave's in a call of at most one chunk
            const rsrc_t rg = make_rsrc_u32(p.g + t0 * H, rows * (uint32_t)(H * 4));
            R.g = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, (uint32_t)((lane * H + h) * 4), 0, 0));
        }
    };

    // The gate wave's part for one chunk: the inclusive in-chunk sums of the
    // gates (lane t holds G_t), the decay tables the output waves read, and
    // the fold weights w_t = exp(G_last - G_t) for the V wave.
    auto gate_tables = [&](const St& R, int bq) {
        const float xs = wave_inclusive_sum(R.g);
        const float glast = lane_value(xs, 63);
        sm.w[bq][lane] = __expf(glast - xs);
        float ge[4];
        #pragma unroll
        for (int M = 0; M < 4; ++M) ge[M] = lane_value(xs, 16 * M + 15);
        const int blk = lane >> 4;
        sm.G2[bq][lane] = xs * LOG2E;
        sm.eG[bq][lane] = __expf(xs);
        sm.bm[bq][lane] = __expf(ge[blk] - xs);
        f32x4 a;
        #pragma unroll
        for (int M = 0; M < 4; ++M) a[M] = (M < blk) ? __expf(xs - ge[M]) : 0.0f;
        *reinterpret_cast<f32x4*>(&sm.ai[bq][lane][0]) = a;
    };

    // K rows of a chunk into LDS; the V wave also V and V w.
    auto stage = [&](St& R, int bk, int bq) {
        #pragma unroll
        for (int u = 0; u < PK; ++u) {
            const int pc = st + NS_T * u;
            const int m = pc / (DK / 8);
            const int d0 = (pc % (DK / 8)) * 8;
            bf16x8 hi, lo;
            split_piece<F32>(R.kp[u], hi, lo);
            *reinterpret_cast<bf16x8*>(&sm.k[bk][0][m * KP + d0]) = hi;
                if (F32) *reinterpret_cast<bf16x8*>(&sm.k[bk][NL - 1][m * KP + d0]) = lo;
        }
        if constexpr (VW) {
            // the V wave stages V and V w (lane l: rows l/2 and 32 + l/2,
            // columns 8 (l%2)..+7) with the weights the gate wave published
            // a step earlier; in a call of at most one chunk it computes
            // them itself, with the gate wave's instructions (same bits)
            float wl = 0.0f;
            if constexpr (ONE) {
                const float xs = wave_inclusive_sum(R.g);
                const float glast = lane_value(xs, 63);
                wl = __expf(glast - xs);
            }
            #pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int m = (lane >> 1) + 32 * i;
                const int jj = 8 * (lane & 1);
                const float wm = ONE ? __shfl(wl, m, 64) : sm.w[bq][m];
                float f[8];
                piece_f32<F32>(R.vp[i], f);
                bf16x8 hi, lo;
                split_piece<F32>(R.vp[i], hi, lo);
                *reinterpret_cast<bf16x8*>(&sm.v[bq][0][m * VP + jj]) = hi;
                if (F32) *reinterpret_cast<bf16x8*>(&sm.v[bq][NL - 1][m * VP + jj]) = lo;
                #pragma unroll
                for (int e = 0; e < 8; ++e) f[e] *= wm;
                split_n<8>(f, hi, lo);
                *reinterpret_cast<bf16x8*>(&sm.vw[bk][0][m * VP + jj]) = hi;
                *reinterpret_cast<bf16x8*>(&sm.vw[bk][1][m * VP + jj]) = lo;
            }
        }
    };

    // D = K^T (V w) over this wave's tiles of d, from zero
    auto fold_delta = [&](int bk, f32x4 (&D)[NDW]) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) D[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int mm = 0; mm < 2; ++mm) {
            const int m0 = 32 * mm + 8 * grp;
            const bf16x8 wh = cat(tr4(sm.vw[bk][0], VP, m0, 0, li), tr4(sm.vw[bk][0], VP, m0 + 4, 0, li));
            const bf16x8 wlo = cat(tr4(sm.vw[bk][1], VP, m0, 0, li), tr4(sm.vw[bk][1], VP, m0 + 4, 0, li));
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                const int n0 = (wq * NDW + u) * 16;
                const bf16x8 kh = cat(tr4(sm.k[bk][0], KP, m0, n0, li), tr4(sm.k[bk][0], KP, m0 + 4, n0, li));
                D[u] = mma(kh, wh, D[u]);
                D[u] = mma(kh, wlo, D[u]);
                if (F32) {
                    const bf16x8 kl = cat(tr4(sm.k[bk][NL - 1], KP, m0, n0, li),
                                          tr4(sm.k[bk][NL - 1], KP, m0 + 4, n0, li));
                    D[u] = mma(kl, wh, D[u]);
                }
            }
        }
    };

    // S split into bf16 hi/lo planes of S^T [j][d] for the output waves' X
    auto publish = [&](int bs) {
        #pragma unroll
        for (int u = 0; u < NDW; ++u) {
            const int d0 = (wq * NDW + u) * 16 + 4 * grp;
            float f[4] = {S[u][0], S[u][1], S[u][2], S[u][3]};
            bf16x4 hi, lo;
            split_n<4>(f, hi, lo);
            *reinterpret_cast<bf16x4*>(&sm.s[bs][0][li * SP + d0]) = hi;
            *reinterpret_cast<bf16x4*>(&sm.s[bs][1][li * SP + d0]) = lo;
        }
    };

    // Cooperative L2 prefetch.  The 16-column slices of a head all read the
    // head's full Q and K rows and share the 128-byte lines of V; fetched
    // at the same moment by every slice, each line costs every workgroup a
    // full HBM latency.  So the V wave of each slice touches its eighth
    // of the head's lines PREFETCH chunks ahead of the regular loads (rows
    // 8 s + i/2 of Q and K, line i%2; rows 16 (s%4) + i of V, line s/4), and
    // the other slices' loads then hit in L2.  The fetched value is only
    // consumed (as an asm operand, forcing nothing but the load's wait) two
    // steps later.
    constexpr int PREFETCH = 5;
    uint32_t pf[2] = {0u, 0u};
    auto prefetch = [&](int slot, int64_t c) {
        __asm__ volatile("" : : "v"(pf[slot]));
        const int64_t t0 = c * CH;
        const uint32_t rows = chunk_rows(x, c);
        const int s8 = (j0 / DVS) & 7;
        const int tsel = lane >> 4, i = lane & 15;
        const uint32_t qoff = (uint32_t)((8 * s8 + (i >> 1)) * x.qk_row + (int64_t)h * DK * ES + (i & 1) * 128);
        const uint32_t voff = (uint32_t)((16 * (s8 & 3) + i) * x.v_row + (int64_t)h * dv * ES + (s8 >> 2) * 128);
        const int64_t row_b = tsel == 2 ? x.v_row : x.qk_row;
        const void* base = tsel == 0 ? p.q : tsel == 1 ? p.k : p.v;
        const rsrc_t r = make_rsrc_u32(static_cast<const char*>(base) + t0 * row_b,
                                       tsel == 3 ? 0u : rows * (uint32_t)row_b);
        pf[slot] = __builtin_amdgcn_raw_buffer_load_b32(r, tsel == 2 ? voff : qoff, 0, 0);
    };

    // S_c as chunk state c (an empty buffer range when not wanted: the
    // one-chunk instance)
    auto store_state = [&](int64_t c, bool live) {
        const bool on = live && p.chunk_states != nullptr;
        const rsrc_t rc = make_rsrc_u32(p.chunk_states + (on ? c * (int64_t)H * DK * dv : 0),
                                        on ? (uint32_t)(H * DK * dv * 4) : 0u);
        #pragma unroll
        for (int t = 0; t < NDW; ++t) {
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float sv = S[t][r];  // (a bit_cast of the vector element itself reads element 0)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, sv), rc,
                                                      (uint32_t)(srow(t, r) * 4), 0, 0);
            }
        }
    };
    // S_{c+1} = exp(G_last of chunk c) S_c + D_c, tables of chunk c in buffer bq
    auto advance = [&](int bq, const f32x4 (&Dc)[NDW]) {
        const float gamma = sm.eG[bq][CH - 1];
        #pragma unroll
        for (int t = 0; t < NDW; ++t) {
            #pragma unroll
            for (int r = 0; r < 4; ++r) S[t][r] = __builtin_fmaf(gamma, S[t][r], Dc[t][r]);
        }
    };
    auto store_final = [&]() {
        if (p.final_state) {
            #pragma unroll
            for (int u = 0; u < NDW; ++u) {
                #pragma unroll
                for (int r = 0; r < 4; ++r) p.final_state[srow(u, r)] = S[u][r];
            }
        }
    };

    // step c: loads of c+4, staging of c+2 (the gate wave: tables of c+3,
    // from the registers Rg loaded a step earlier), D_{c+1}; S_c out;
    // S_{c+1} in
    auto step = [&](int64_t c, int u, St& Rc, St& Rs, const St& Rg, f32x4 (&Dn)[NDW], const f32x4 (&Dc)[NDW]) {
        if constexpr (VW) prefetch(u & 1, c + PREFETCH);
        load_chunk(Rc, c + 4);
        if (GW) gate_tables(Rg, (u + 3) & 3);
        stage(Rs, u & 1, (u + 2) & 3);
        fold_delta((u + 1) & 1, Dn);
        const bool live = c < x.n;
        if constexpr (CS) store_state(c, live);
        if (live) advance(u, Dc);
        publish((u + 1) & 1);
        if (live) lds_barrier();
    };

    if constexpr (ONE) {
        // At most one chunk (decode steps, short continuations): the same
        // per-chunk arithmetic in straight line, one barrier.
        St R0;
        load_chunk(R0, 0);
        if (GW) gate_tables(R0, 0);
        stage(R0, 0, 0);
        publish(0);
        lds_barrier();
        if (x.n == 1) {
            fold_delta(0, D0);
            store_state(0, true);
            advance(0, D0);
        }
        store_final();
        return;
    } else {

    St R0, R1, R2, R3;
    load_chunk(R0, 0);
    load_chunk(R1, 1);
    load_chunk(R2, 2);
    load_chunk(R3, 3);
    if (GW) {  // tables and weights of chunks 0-2 (step c writes those of c + 3)
        gate_tables(R0, 0);
        gate_tables(R1, 1);
        gate_tables(R2, 2);
    }
    lds_barrier();
    stage(R0, 0, 0);
    stage(R1, 1, 1);
    publish(0);
    lds_barrier();
    fold_delta(0, D0);
    lds_barrier();
    for (int64_t c = 0; c < x.n; c += 4) {
        step(c, 0, R0, R2, R3, D1, D0);
        step(c + 1, 1, R1, R3, R0, D0, D1);
        step(c + 2, 2, R2, R0, R1, D1, D0);
        step(c + 3, 3, R3, R1, R2, D0, D1);
    }
    store_final();
    if constexpr (VW) __asm__ volatile("" : : "v"(pf[0]), "v"(pf[1]));
    }
}

// ------------------------------------------------------------ output role
// Output wave W owns rows i = 16 W + li of every chunk.
template <int DK, bool F32, bool ONE, int W>
__device__ __forceinline__ void output_role(const ScanParams& p, Smem<DK, F32>& sm, const Ctx& x) {
    using S_ = Smem<DK, F32>;
    constexpr int KP = S_::KP;
    constexpr int SP = S_::SP;
    constexpr int NL = S_::NL;
    constexpr int ES = F32 ? 4 : 2;
    constexpr int NKK = DK / 32;  // k-steps of 32 over dk
    constexpr int PPR = DK * ES / 16;  // 16-byte pieces per Q row
    constexpr int RPI = 64 / PPR;      // Q rows per coalesced load
    constexpr int NQI = 16 / RPI;      // coalesced loads per 16 rows
    constexpr int EPP = 16 / ES;       // elements per piece
    using QS = QStage<NQI>;
    struct QOp {                       // Q rows as MFMA operands (hi, lo)
        bf16x8 h[NKK], l[NKK];
    };
    const int lane = x.lane, li = x.li, grp = x.grp, h = x.h, j0 = x.j0, dv = x.dv;
    const int i_row = 16 * W + li;

    // this wave's 16 rows of Q for chunk c, coalesced: load i, lane l reads
    // piece l % PPR of row RPI i + l / PPR
    auto load_q = [&](QS& Q, int64_t c) {
        const int64_t t0 = c * CH;
        const rsrc_t rq = make_rsrc_u32(static_cast<const char*>(p.q) + t0 * x.qk_row,
                                        chunk_rows(x, c) * (uint32_t)x.qk_row);
        #pragma unroll
        for (int i = 0; i < NQI; ++i)
            Q.qp[i] = __builtin_amdgcn_raw_buffer_load_b128(
                rq, (uint32_t)((16 * W + RPI * i + lane / PPR) * x.qk_row + (int64_t)h * DK * ES + (lane % PPR) * 16), 0, 0);
    };

    // through this wave's own LDS rows into operand layout (lane (li, grp)
    // gets row li, elements 32 kk + 8 grp..+7); the wave reads back only
    // what it wrote, so no barrier is involved
    auto q_operands = [&](const QS& Q, QOp& op) {
        #pragma unroll
        for (int i = 0; i < NQI; ++i) {
            const int row = RPI * i + lane / PPR;
            const int e0 = (lane % PPR) * EPP;
            if constexpr (F32) {
                const f32x4 a = __builtin_bit_cast(f32x4, Q.qp[i]);
                float f[4] = {a[0], a[1], a[2], a[3]};
                bf16x4 hi, lo;
                split_n<4>(f, hi, lo);
                *reinterpret_cast<bf16x4*>(&sm.q[W][0][row * SP + e0]) = hi;
                *reinterpret_cast<bf16x4*>(&sm.q[W][NL - 1][row * SP + e0]) = lo;
            } else {
                *reinterpret_cast<u32x4*>(&sm.q[W][0][row * SP + e0]) = Q.qp[i];
            }
        }
        #pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
            op.h[kk] = *reinterpret_cast<const bf16x8*>(&sm.q[W][0][li * SP + 32 * kk + 8 * grp]);
            op.l[kk] = F32 ? *reinterpret_cast<const bf16x8*>(&sm.q[W][NL - 1][li * SP + 32 * kk + 8 * grp]) : bf16x8{};
        }
    };

    // A^T = K Q^T for the causal m-blocks mb <= W; lane (li, grp) of tile mb
    // holds A^T[m = 16 mb + 4 grp + r][i = 16 W + li]
    auto scores = [&](const QOp& qo, int bk, f32x4 (&at)[4]) {
        const bf16x8* qh = qo.h;
        const bf16x8* ql = qo.l;
        #pragma unroll
        for (int mb = 0; mb <= W; ++mb) {
            bf16x8 a[NKK], al[NKK];
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                const int off = (mb * 16 + li) * KP + 32 * kk + 8 * grp;
                a[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[bk][0][off]);
                if (F32) al[kk] = *reinterpret_cast<const bf16x8*>(&sm.k[bk][NL - 1][off]);
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
    };

    // decay, O^T = V^T P^T, X^T = S_c^T Q^T and the o store of chunk c
    auto finish = [&](int64_t c, int u, const QOp& qo, f32x4 (&at)[4]) {
        const bf16x8* qh = qo.h;
        const bf16x8* ql = qo.l;
        // decay: factored tables below the diagonal tile, exp2 on it
        {
            const f32x4 ai = *reinterpret_cast<const f32x4*>(&sm.ai[u][i_row][0]);
            #pragma unroll
            for (int mb = 0; mb < W; ++mb) {
                const f32x4 bmv = *reinterpret_cast<const f32x4*>(&sm.bm[u][mb * 16 + 4 * grp]);
                #pragma unroll
                for (int r = 0; r < 4; ++r) at[mb][r] = (at[mb][r] * ai[mb]) * bmv[r];
            }
            const float gi = sm.G2[u][i_row];
            const f32x4 gm = *reinterpret_cast<const f32x4*>(&sm.G2[u][W * 16 + 4 * grp]);
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float pv = at[W][r] * __builtin_amdgcn_exp2f(gi - gm[r]);
                at[W][r] = (4 * grp + r <= li) ? pv : 0.0f;
            }
        }
        // O = P V, two m-blocks per MFMA (the score accumulators are P in
        // A-operand layout); lane (li, grp) ends with O[i = 16 W + 4 grp + r][j0 + li]
        f32x4 acc_o = {0.f, 0.f, 0.f, 0.f};
        #pragma unroll
        for (int pr = 0; 2 * pr <= W; ++pr) {
            float f[8];
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                f[r] = at[2 * pr][r];
                f[4 + r] = (2 * pr + 1 <= W) ? at[2 * pr + 1][r] : 0.0f;
            }
            bf16x8 ph, pl;
            split_n<8>(f, ph, pl);
            const bf16x8 vh = cat(tr4(sm.v[u][0], VP, (2 * pr) * 16 + 4 * grp, 0, li),
                                  tr4(sm.v[u][0], VP, (2 * pr + 1) * 16 + 4 * grp, 0, li));
            acc_o = mma(ph, vh, acc_o);
            acc_o = mma(pl, vh, acc_o);
            if (F32) {
                const bf16x8 vl = cat(tr4(sm.v[u][NL - 1], VP, (2 * pr) * 16 + 4 * grp, 0, li),
                                      tr4(sm.v[u][NL - 1], VP, (2 * pr + 1) * 16 + 4 * grp, 0, li));
                acc_o = mma(ph, vl, acc_o);
            }
        }
        // X = Q S_c from the published S^T planes, hi and lo products in two
        // independent accumulators
        f32x4 acc_x = {0.f, 0.f, 0.f, 0.f}, acc_xl = {0.f, 0.f, 0.f, 0.f};
        {
            const int bs = u & 1;
            bf16x8 sh[NKK], sl[NKK];
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                const int off = li * SP + 32 * kk + 8 * grp;
                sh[kk] = *reinterpret_cast<const bf16x8*>(&sm.s[bs][0][off]);
                sl[kk] = *reinterpret_cast<const bf16x8*>(&sm.s[bs][1][off]);
            }
            #pragma unroll
            for (int kk = 0; kk < NKK; ++kk) {
                acc_x = mma(qh[kk], sh[kk], acc_x);
                acc_xl = mma(qh[kk], sl[kk], acc_xl);
                if (F32) acc_xl = mma(ql[kk], sh[kk], acc_xl);
            }
            acc_x += acc_xl;
        }
        // o rows i = 16 W + 4 grp + r, column j0 + li: for each r the 16
        // lanes of a group store 64 contiguous bytes; rows past T fall outside
        // the chunk's buffer range and are dropped
        {
            const int64_t t0 = c * CH;
            const rsrc_t ro = make_rsrc_u32(reinterpret_cast<const char*>(p.o) + t0 * x.o_row,
                                            chunk_rows(x, c) * (uint32_t)x.o_row);
            const f32x4 eg = *reinterpret_cast<const f32x4*>(&sm.eG[u][16 * W + 4 * grp]);
            #pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float val = p.scale * (eg[r] * acc_x[r] + acc_o[r]);
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, val), ro,
                                                      (uint32_t)((16 * W + 4 * grp + r) * x.o_row + ((int64_t)h * dv + j0 + li) * 4),
                                                      0, 0);
            }
        }
    };

    // step c: Q operands and scores of chunk c+1, the rest of chunk c, then
    // the loads of Q for chunk c+4 into the freed register stage
    auto step = [&](int64_t c, int u, QS& Qc, const QS& Qn, const QOp& oc, QOp& on, f32x4 (&atc)[4],
                    f32x4 (&atn)[4]) {
        q_operands(Qn, on);
        scores(on, (u + 1) & 1, atn);
        finish(c, u, oc, atc);
        load_q(Qc, c + 4);
        if (c < x.n) lds_barrier();
    };

    QS Q0, Q1, Q2, Q3;
    QOp O0, O1;
    f32x4 A0[4], A1[4];
    if constexpr (ONE) {  // at most one chunk: straight line, one barrier
        load_q(Q0, 0);
        lds_barrier();
        if (x.n == 1) {
            q_operands(Q0, O0);
            scores(O0, 0, A0);
            finish(0, 0, O0, A0);
        }
        return;
    } else {
    load_q(Q0, 0);
    load_q(Q1, 1);
    load_q(Q2, 2);
    load_q(Q3, 3);
    lds_barrier();  // the gate wave's first tables
    lds_barrier();
    q_operands(Q0, O0);
    scores(O0, 0, A0);
    lds_barrier();
    for (int64_t c = 0; c < x.n; c += 4) {
        step(c, 0, Q0, Q1, O0, O1, A0, A1);
        step(c + 1, 1, Q1, Q2, O1, O0, A1, A0);
        step(c + 2, 2, Q2, Q3, O0, O1, A0, A1);
        step(c + 3, 3, Q3, Q0, O1, O0, A1, A0);
    }
    }
}

// ONE: the call holds at most one chunk.  CS: a multi-chunk call that
// stores the chunk states; without them the state waves issue no
// chunk-state stores at all (rather than stores to an empty range, whose
// address work costs the final-state-only call about 4 %).
template <int DK, bool F32, bool ONE, bool CS>
__global__ __launch_bounds__(NT) void linattn_scan_kernel(const ScanParams p) {
    __shared__ Smem<DK, F32> sm;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform

    // workgroup -> (head, slice); slices of one head share an XCD (and its L2)
    // when the grid allows it (workgroups go round-robin over 8 XCDs).
    Ctx x;
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
    constexpr int ES = F32 ? 4 : 2;
    x.qk_row = (int64_t)x.H * DK * ES;
    x.v_row = (int64_t)x.H * x.dv * ES;
    x.o_row = (int64_t)x.H * x.dv * 4;

    // Issue priority follows the step lengths: the V wave (4) and the gate
    // wave (5) have the longest steps of the eight, the output waves come
    // next, the two plain state waves finish first.
    if (wave == 4 || wave == 5) __builtin_amdgcn_s_setprio(3);
    if (wave < 4) __builtin_amdgcn_s_setprio(1);
    switch (wave) {
        case 0: output_role<DK, F32, ONE, 0>(p, sm, x); break;
        case 1: output_role<DK, F32, ONE, 1>(p, sm, x); break;
        case 2: output_role<DK, F32, ONE, 2>(p, sm, x); break;
        case 3: output_role<DK, F32, ONE, 3>(p, sm, x); break;
        case 4: state_role<DK, F32, ONE, CS, true>(p, sm, x, 0); break;
        default: state_role<DK, F32, ONE, CS, false>(p, sm, x, wave - 4); break;
    }
}

template <int DK, bool F32>
hipError_t launch_t(const ScanParams& p, hipStream_t stream) {
    const unsigned grid = (unsigned)(p.H * (p.dv / DVS));
    const void* fn = p.T <= CH ? reinterpret_cast<const void*>(&linattn_scan_kernel<DK, F32, true, true>)
                     : p.chunk_states ? reinterpret_cast<const void*>(&linattn_scan_kernel<DK, F32, false, true>)
                                      : reinterpret_cast<const void*>(&linattn_scan_kernel<DK, F32, false, false>);
    return launch_kernel(fn, dim3(grid), dim3(NT), p, stream);
}

}  // namespace

hipError_t launch_linattn_scan(const ScanParams& p, hipStream_t stream) {
    // fp32 inputs keep hi and lo planes of K and V in LDS; the scan supports
    // them at dk = 64.
    if (p.dk == 128 && !p.in_f32) return launch_t<128, false>(p, stream);
    if (p.dk == 64) return p.in_f32 ? launch_t<64, true>(p, stream) : launch_t<64, false>(p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
