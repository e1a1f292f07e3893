// One-token step of the gated delta rule on gfx950 (a decode step).  With a
// single token the chunked form (gdn_scan.hip) has A = 0 and T = I, so per
// head, with gamma = exp(g):
//   u   = beta (v - gamma k.S)               (1 x dv; k.S sums over the dk rows)
//   S'  = gamma S + k^T u
//   o   = scale (gamma q.S + (q.k) u)
// which is the token recurrence S' = gamma (I - beta k^T k) S + beta k^T v,
// o = scale q S' written out.  One launch on the vector ALU replaces the two
// launches of the chunked path; S' and o agree with that path to fp32
// rounding (its products run on MFMA with split operands).
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "internal.h"

namespace cap {
namespace {

using namespace dev;

constexpr int DVS = 16;  // value columns per workgroup

// Workgroup = (head, 16-column slice), 2 dk threads; thread t owns row
// d = t / 2, columns j0 + 8 (t % 2) .. +7 of the state (32 contiguous bytes).
// k.S and q.S are summed over the rows of a column half by lane shuffles
// within a wave and one LDS exchange between the waves.
template <int DK>
__global__ __launch_bounds__(2 * DK) void gdn_step_kernel(const GdnParams p) {
    constexpr int NW = 2 * DK / 64;  // waves
    __shared__ float part[NW][2][17];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // workgroup -> (head, slice); the slices of a head share an XCD (and its
    // L2), since neighbouring slices read the two halves of the same
    // 128-byte state lines (workgroups go round-robin over 8 XCDs)
    const int NS = p.dv / DVS;
    const int N = p.H * NS;
    int logical = blockIdx.x;
    if ((N % 8) == 0 && ((N / 8) % NS) == 0) logical = (blockIdx.x % 8) * (N / 8) + blockIdx.x / 8;
    const int h = logical / NS, j0 = (logical % NS) * DVS;
    const int d = tid >> 1, half = tid & 1, c0 = 8 * half;
    const int64_t sidx = ((int64_t)h * DK + d) * p.dv + j0 + c0;  // element of S[h][d][j0 + c0]

    const __bf16* q = static_cast<const __bf16*>(p.q);
    const __bf16* k = static_cast<const __bf16*>(p.k);
    const __bf16* v = static_cast<const __bf16*>(p.v);
    const float qd = (float)q[h * DK + d], kd = (float)k[h * DK + d];
    const bf16x8 vv = *reinterpret_cast<const bf16x8*>(v + (int64_t)h * p.dv + j0 + c0);
    const float gamma = __expf(p.g[h]), beta = p.beta[h];
    float S[8];
    if (p.state_in) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(p.state_in + sidx);
        const f32x4 b = *reinterpret_cast<const f32x4*>(p.state_in + sidx + 4);
        #pragma unroll
        for (int e = 0; e < 4; ++e) { S[e] = a[e]; S[4 + e] = b[e]; }
    } else {
        #pragma unroll
        for (int e = 0; e < 8; ++e) S[e] = 0.0f;
    }
    if (p.chunk_states) {  // the state entering the call's only chunk
        *reinterpret_cast<f32x4*>(p.chunk_states + sidx) = f32x4{S[0], S[1], S[2], S[3]};
        *reinterpret_cast<f32x4*>(p.chunk_states + sidx + 4) = f32x4{S[4], S[5], S[6], S[7]};
    }

    // partials of k.S (0..7), q.S (8..15) over this thread's row, and q.k (16)
    float x[17];
    #pragma unroll
    for (int e = 0; e < 8; ++e) { x[e] = kd * S[e]; x[8 + e] = qd * S[e]; }
    x[16] = qd * kd;
    #pragma unroll
    for (int off = 2; off < 64; off <<= 1)
        #pragma unroll
        for (int e = 0; e < 17; ++e) x[e] += __shfl_xor(x[e], off, 64);
    if (lane < 2)
        #pragma unroll
        for (int e = 0; e < 17; ++e) part[wave][lane][e] = x[e];
    __syncthreads();

    // u for this thread's 8 columns, then S' and (16 threads) o
    float u[8];
    #pragma unroll
    for (int e = 0; e < 8; ++e) {
        float ks = 0.0f;
        #pragma unroll
        for (int w = 0; w < NW; ++w) ks += part[w][half][e];
        u[e] = beta * ((float)vv[e] - gamma * ks);
    }
    if (p.final_state) {
        float Sn[8];
        #pragma unroll
        for (int e = 0; e < 8; ++e) Sn[e] = __builtin_fmaf(gamma, S[e], kd * u[e]);
        *reinterpret_cast<f32x4*>(p.final_state + sidx) = f32x4{Sn[0], Sn[1], Sn[2], Sn[3]};
        *reinterpret_cast<f32x4*>(p.final_state + sidx + 4) = f32x4{Sn[4], Sn[5], Sn[6], Sn[7]};
    }
    if (d == 0) {  // threads 0 and 1: the two column halves
        float qk = 0.0f;
        #pragma unroll
        for (int w = 0; w < NW; ++w) qk += part[w][0][16];
        float ov[8];
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
            float qs = 0.0f;
            #pragma unroll
            for (int w = 0; w < NW; ++w) qs += part[w][half][8 + e];
            ov[e] = p.scale * (gamma * qs + qk * u[e]);
        }
        float* o = p.o + (int64_t)h * p.dv + j0 + c0;
        *reinterpret_cast<f32x4*>(o) = f32x4{ov[0], ov[1], ov[2], ov[3]};
        *reinterpret_cast<f32x4*>(o + 4) = f32x4{ov[4], ov[5], ov[6], ov[7]};
    }
}

}  // namespace

hipError_t launch_gdn_step(const GdnParams& p, hipStream_t stream) {
    const unsigned grid = (unsigned)(p.H * (p.dv / DVS));
    if (p.T != 1) return hipErrorInvalidValue;
    if (p.dk == 128) return launch_kernel(reinterpret_cast<const void*>(&gdn_step_kernel<128>), dim3(grid), dim3(256), p, stream);
    if (p.dk == 64) return launch_kernel(reinterpret_cast<const void*>(&gdn_step_kernel<64>), dim3(grid), dim3(128), p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
