// One-token step of the gated linear-attention recurrence on gfx950 (a
// decode step): S' = exp(g) S + k^T v and o = scale (exp(g) q.S + (q.k) v),
// per head, the same recurrence the chunked prefill evaluates (paper §5).
#include <hip/hip_runtime.h>

#include "device_util.h"
#include "internal.h"

namespace cap {
namespace {

using namespace dev;

constexpr int DVS = 16;  // value columns per workgroup

// A call of exactly one bf16 token, on the vector ALU with no LDS staging
// and one barrier, so the step costs little more than the launch and one
// round trip to HBM.  S' is bit-identical to the chunked prefill's fold of a
// one-token chunk (linattn_scan.hip): there the fold product k_d v_j of two
// bf16 values is exact in fp32 and enters an accumulator that starts at +0,
// and the fold is one fma with exp(g) (a one-token decay sum is g itself);
// here the same three steps run on the vector ALU.  o takes another
// summation order than the chunked kernel's o (fp32 rounding only).
//
// Workgroup = (head, 16-column slice), 2 dk threads; thread t owns row
// d = t / 2, columns j0 + 8 (t % 2) .. +7 of the state: 32 contiguous bytes.
template <int DK>
__global__ __launch_bounds__(2 * DK) void linattn_step_kernel(const ScanParams p) {
    constexpr int NW = 2 * DK / 64;  // waves
    __shared__ float part[NW][2][9];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // workgroup -> (head, slice); the slices of a head share an XCD (and its
    // L2) when the grid allows it, since neighbouring slices read the two
    // halves of the same 128-byte state lines (workgroups go round-robin
    // over 8 XCDs)
    const int NS = p.dv / DVS;
    const int N = p.H * NS;
    int logical = blockIdx.x;
    if ((N % 8) == 0 && ((N / 8) % NS) == 0) logical = (blockIdx.x % 8) * (N / 8) + blockIdx.x / 8;
    const int h = logical / NS, j0 = (logical % NS) * DVS;
    const int d = tid >> 1, c0 = 8 * (tid & 1);
    const int64_t sidx = ((int64_t)h * DK + d) * p.dv + j0 + c0;  // element of S[h][d][j0 + c0]

    const __bf16* q = static_cast<const __bf16*>(p.q);
    const __bf16* k = static_cast<const __bf16*>(p.k);
    const float qd = (float)q[h * DK + d], kd = (float)k[h * DK + d];
    const bf16x8 vv = *reinterpret_cast<const bf16x8*>(static_cast<const __bf16*>(p.v) + (int64_t)h * p.dv + j0 + c0);
    const float gamma = __expf(p.g[h]);
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

    // per-thread partials of q.S (this row) and q.k, summed over the rows of
    // the same column half: lanes of equal parity in the wave, then the waves
    float xq[9];
    #pragma unroll
    for (int e = 0; e < 8; ++e) xq[e] = qd * S[e];
    xq[8] = qd * kd;
    #pragma unroll
    for (int off = 2; off < 64; off <<= 1)
        #pragma unroll
        for (int e = 0; e < 9; ++e) xq[e] += __shfl_xor(xq[e], off, 64);
    if (lane < 2)
        #pragma unroll
        for (int e = 0; e < 9; ++e) part[wave][lane][e] = xq[e];

    if (p.final_state) {
        float Sn[8];
        #pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float D = 0.0f + kd * (float)vv[e];
            Sn[e] = __builtin_fmaf(gamma, S[e], D);
        }
        *reinterpret_cast<f32x4*>(p.final_state + sidx) = f32x4{Sn[0], Sn[1], Sn[2], Sn[3]};
        *reinterpret_cast<f32x4*>(p.final_state + sidx + 4) = f32x4{Sn[4], Sn[5], Sn[6], Sn[7]};
    }
    __syncthreads();
    if (tid < DVS) {
        const int half = tid >> 3, e = tid & 7;
        float x = 0.0f, qk = 0.0f;
        #pragma unroll
        for (int w = 0; w < NW; ++w) {
            x += part[w][half][e];
            qk += part[w][0][8];
        }
        const float vj = (float)static_cast<const __bf16*>(p.v)[(int64_t)h * p.dv + j0 + tid];
        p.o[(int64_t)h * p.dv + j0 + tid] = p.scale * (gamma * x + qk * vj);
    }
}

}  // namespace

hipError_t launch_linattn_step(const ScanParams& p, hipStream_t stream) {
    const unsigned grid = (unsigned)(p.H * (p.dv / DVS));
    if (p.in_f32 || p.T != 1) return hipErrorInvalidValue;
    if (p.dk == 128)
        return launch_kernel(reinterpret_cast<const void*>(&linattn_step_kernel<128>), dim3(grid), dim3(256), p, stream);
    if (p.dk == 64)
        return launch_kernel(reinterpret_cast<const void*>(&linattn_step_kernel<64>), dim3(grid), dim3(128), p, stream);
    return hipErrorInvalidValue;
}

}  // namespace cap
