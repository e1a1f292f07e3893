// Device helpers shared by the chunked scans (linattn_scan.hip, gdn_scan.hip):
// gfx950 MFMA, buffer resources, transposing LDS reads, a DPP wave scan,
// hi/lo bf16 splitting and an LDS-only workgroup barrier.  Not part of the
// public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cap {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr float LOG2E = 1.4426950408889634f;

// D += A B on one 16x16x32 bf16 tile.  Lane l = 16 grp + li holds
// A[li][8 grp + e], B[8 grp + e][li] (e = 0..7) and D[4 grp + r][li] (r = 0..3).
__device__ inline f32x4 mma(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Buffer resource over [base, base + nbytes) (raw, stride 0); accesses past
// nbytes read zeros / are dropped.
__device__ inline rsrc_t make_rsrc(const void* base, int64_t nbytes) {
    const int64_t n = nbytes < 0 ? 0 : (nbytes > 0x7ffffff0 ? 0x7ffffff0 : nbytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// Buffer resource over [base, base + nbytes) for an nbytes the caller knows
// to be below 2^31 (no clamp: with wave-uniform arguments it is built on the
// scalar unit).
__device__ inline rsrc_t make_rsrc_u32(const void* base, uint32_t nbytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)nbytes, 0x00020000);
}

// Transposing LDS read of a row-major bf16 tile with `pitch` elements per
// row: lane n of each 16-lane group gets tile[k0 + 0..3][n0 + n].  k0 may
// differ between the four groups of a wave.
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

// hi + lo split of fp32 values into bf16 (round to nearest even both times):
// hi + lo carries ~16 significant bits, so a product of split operands
// (three MFMA terms, or two when one side is exact bf16) keeps ~2^-17
// relative error.
// Values go in pairs: one packed conversion gives both hi halves, which are
// widened back to fp32 with a shift and a mask (no second conversion).
template <int N, typename V>
__device__ inline void split_n(const float* f, V& hi, V& lo) {
    static_assert(N % 2 == 0, "pairs");
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    #pragma unroll
    for (int e = 0; e < N; e += 2) {
        const bf16x2 h = __builtin_convertvector((f32x2){f[e], f[e + 1]}, bf16x2);
        const uint32_t u = __builtin_bit_cast(uint32_t, h);
        const float h0 = __builtin_bit_cast(float, u << 16);
        const float h1 = __builtin_bit_cast(float, u & 0xFFFF0000u);
        const bf16x2 l = __builtin_convertvector((f32x2){f[e] - h0, f[e + 1] - h1}, bf16x2);
        hi[e] = h[0];
        hi[e + 1] = h[1];
        lo[e] = l[0];
        lo[e + 1] = l[1];
    }
}

// Workgroup barrier for LDS traffic only.  Global stores are never read back
// inside the scans, so the barrier does not wait for them (a plain
// __syncthreads() would drain every outstanding global access).
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace dev
}  // namespace cap
