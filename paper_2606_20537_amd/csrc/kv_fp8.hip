// FP8 KV region on gfx950: BF16 <-> OCP E4M3 conversion of KV rows.
//
// Paper §3 "Definition": the KV region may be held in FP8, which roughly
// halves the capsule; the BF16 working stage of the attention is not part of
// the capsule and, after a restore, is rebuilt lazily on the next read (§3
// cost model: restore copies bytes and rebinds, the stage follows on demand).
// Quantize writes appended rows into the FP8 region; dequantize rebuilds the
// BF16 stage for a range of rows.
//
// Format (OCP 8-bit floating point, E4M3): sign, 4 exponent bits with bias 7,
// 3 mantissa bits; subnormals m/8 * 2^-6; largest finite 448 (S.1111.110);
// S.1111.111 is NaN; there are no infinities.  Encoding rounds to nearest,
// ties to even, and saturates: |x| >= 448 and +-inf give +-448; NaN keeps its
// sign.  Both conversions are exact integer / power-of-two arithmetic, so the
// codes and the BF16 results are bit-identical to any implementation of the
// same definition.
//
// Streaming, HBM-bound: each thread converts groups of 16 elements (32 bytes
// of BF16 <-> 16 bytes of FP8) with 16-byte nontemporal loads and stores;
// one grid covers up to 64 segments (one per KV buffer), each block a run of
// 512 groups of one segment found by a binary search over the launch table.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint32_t f32_bits(float x) { return __builtin_bit_cast(uint32_t, x); }
__device__ inline float bits_f32(uint32_t u) { return __builtin_bit_cast(float, u); }

// fp32 -> E4M3 code (round to nearest even, saturating).
__device__ inline uint32_t e4m3_encode(float x) {
    const uint32_t u = f32_bits(x);
    const uint32_t sign = (u >> 24) & 0x80u;
    const uint32_t a = u & 0x7FFFFFFFu;
    if (a > 0x7F800000u) return sign | 0x7Fu;             // NaN
    if (a >= 0x43E00000u) return sign | 0x7Eu;            // |x| >= 448, inf: saturate
    if (a < 0x3C800000u) {                                // |x| < 2^-6: subnormal range
        // |x| * 2^9 is exact; rounding it to an integer (ties to even) gives
        // the subnormal mantissa, 8 meaning the smallest normal (code 0x08)
        return sign | (uint32_t)__builtin_rintf(bits_f32(a) * 512.0f);
    }
    // normal: keep 3 of the 23 mantissa bits, round to nearest even (a carry
    // into the exponent is the correct next binade); e = exponent - 127 + 7
    const uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
    const uint32_t e = (r >> 23) - 120u;
    return sign | (e << 3) | ((r >> 20) & 7u);
}

// E4M3 code -> fp32 (exact), NaN codes excluded by the caller.
__device__ inline float e4m3_decode(uint32_t c) {
    const uint32_t e = (c >> 3) & 15u, m = c & 7u;
    const float v = e == 0 ? (float)m * 0x1p-9f : bits_f32(((e + 120u) << 23) | (m << 20));
    return (c & 0x80u) ? -v : v;
}

// fp32 -> bf16 bits, round to nearest even (the conversion instruction).
__device__ inline uint32_t bf16_bits(float y) {
    return (uint32_t)__builtin_bit_cast(unsigned short, (__bf16)y);
}

__device__ inline uint32_t segment_of(const Fp8Params& p, uint32_t b) {
    uint32_t lo = 0, hi = p.n_seg - 1;  // last s with first_block[s] <= b
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (p.first_block[mid] <= b) lo = mid; else hi = mid - 1;
    }
    return lo;
}

template <bool QUANT>
__global__ __launch_bounds__(256) void fp8_kernel(const Fp8Params p) {
    const uint32_t s = __builtin_amdgcn_readfirstlane(segment_of(p, blockIdx.x));
    const uint64_t n = p.n_groups[s];
    const uint64_t g0 = (uint64_t)(blockIdx.x - p.first_block[s]) * kFp8GroupsPerBlock;
    const float mul = p.mul[s];
    constexpr int kU = kFp8GroupsPerBlock / 256;
    if (QUANT) {
        const u32x4* src = reinterpret_cast<const u32x4*>(p.src[s]);  // 2 vectors per group
        u32x4* dst = reinterpret_cast<u32x4*>(p.dst[s]);              // 1 vector per group
        u32x4 in[kU][2];
        #pragma unroll
        for (int u = 0; u < kU; ++u) {
            const uint64_t g = g0 + u * 256 + threadIdx.x;
            if (g < n) {
                in[u][0] = __builtin_nontemporal_load(src + 2 * g);
                in[u][1] = __builtin_nontemporal_load(src + 2 * g + 1);
            }
        }
        #pragma unroll
        for (int u = 0; u < kU; ++u) {
            const uint64_t g = g0 + u * 256 + threadIdx.x;
            if (g < n) {
                u32x4 out;
                #pragma unroll
                for (int w = 0; w < 4; ++w) {  // output word w = input elements 4w..4w+3
                    const u32x4& v = in[u][w >> 1];
                    const uint32_t lo = v[(w & 1) * 2], hi = v[(w & 1) * 2 + 1];
                    const uint32_t b0 = e4m3_encode(bits_f32(lo << 16) * mul);
                    const uint32_t b1 = e4m3_encode(bits_f32(lo & 0xFFFF0000u) * mul);
                    const uint32_t b2 = e4m3_encode(bits_f32(hi << 16) * mul);
                    const uint32_t b3 = e4m3_encode(bits_f32(hi & 0xFFFF0000u) * mul);
                    out[w] = b0 | (b1 << 8) | (b2 << 16) | (b3 << 24);
                }
                __builtin_nontemporal_store(out, dst + g);
            }
        }
    } else {
        const u32x4* src = reinterpret_cast<const u32x4*>(p.src[s]);  // 1 vector per group
        u32x4* dst = reinterpret_cast<u32x4*>(p.dst[s]);              // 2 vectors per group
        u32x4 in[kU];
        #pragma unroll
        for (int u = 0; u < kU; ++u) {
            const uint64_t g = g0 + u * 256 + threadIdx.x;
            if (g < n) in[u] = __builtin_nontemporal_load(src + g);
        }
        #pragma unroll
        for (int u = 0; u < kU; ++u) {
            const uint64_t g = g0 + u * 256 + threadIdx.x;
            if (g < n) {
                u32x4 out[2];
                #pragma unroll
                for (int e = 0; e < 16; e += 2) {
                    uint32_t h[2];
                    #pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        const uint32_t c = (in[u][(e + t) >> 2] >> (8 * ((e + t) & 3))) & 0xFFu;
                        h[t] = (c & 0x7Fu) == 0x7Fu ? ((c & 0x80u) ? 0xFFC0u : 0x7FC0u)
                                                    : bf16_bits(e4m3_decode(c) * mul);
                    }
                    out[e >> 3][(e >> 1) & 3] = h[0] | (h[1] << 16);
                }
                __builtin_nontemporal_store(out[0], dst + 2 * g);
                __builtin_nontemporal_store(out[1], dst + 2 * g + 1);
            }
        }
    }
}

}  // namespace

hipError_t launch_fp8(const Fp8Params& p, hipStream_t stream) {
    const uint32_t blocks = p.first_block[p.n_seg];
    if (blocks == 0) return hipSuccess;
    const void* fn = p.quantize ? reinterpret_cast<const void*>(&fp8_kernel<true>)
                                : reinterpret_cast<const void*>(&fp8_kernel<false>);
    return launch_kernel(fn, dim3(blocks), dim3(256), p, stream);
}

}  // namespace cap
