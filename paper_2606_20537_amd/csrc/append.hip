// Append of a suffix to a live buffer set on gfx950 (paper §3 Algorithm 1:
// after the capsule's bytes are copied back, the suffix is appended; §3
// "Definition": the full-attention KV region is positional, the convolution
// state is a fixed-size window of the latest inputs).
//
// One launch covers every buffer of the set that the append touches:
//   positional buffer: rows [position, position + n) <- the n new rows, a
//     plain copy cut into 16 KiB tiles (16-byte loads and stores, one tile
//     per block);
//   window (a fixed buffer with a source): the window becomes the last W
//     rows of (its rows, then the n new rows).  Source and destination
//     overlap (the window shifts in place), so one block reads every byte it
//     will write into registers, synchronises, then writes.
// The launch carries its table by value (no device-side descriptors), so a
// decode step enqueued inside a stream capture replays with no host work.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr uint32_t kWinVecPerThread = kAppendMaxWindow / 16 / kThreads;  // 16

__device__ inline uint32_t segment_of(const AppendParams& p, uint32_t b) {
    uint32_t lo = 0, hi = p.n_seg - 1;  // last s with first_block[s] <= b
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (p.first_block[mid] <= b) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ __launch_bounds__(kThreads) void append_kernel(const AppendParams p) {
    const uint32_t s = __builtin_amdgcn_readfirstlane(segment_of(p, blockIdx.x));
    const u32x4* src = reinterpret_cast<const u32x4*>(p.src[s]);
    u32x4* dst = reinterpret_cast<u32x4*>(p.dst[s]);
    const uint64_t nvec = p.bytes[s] / 16;
    const uint32_t wvec = p.win[s] / 16;
    if (wvec == 0) {
        // positional: vectors [t0, t0 + kAppendTile / 16) of the new rows
        const uint64_t t0 = (uint64_t)(blockIdx.x - p.first_block[s]) * (kAppendTile / 16);
        constexpr int kPer = kAppendTile / 16 / kThreads;  // 4
        u32x4 v[kPer];
        #pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const uint64_t i = t0 + u * kThreads + threadIdx.x;
            if (i < nvec) v[u] = src[i];
        }
        #pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const uint64_t i = t0 + u * kThreads + threadIdx.x;
            if (i < nvec) dst[i] = v[u];
        }
        return;
    }
    // window of wvec vectors: new[j] = (j + nvec < wvec) ? old[j + nvec] : src[j + nvec - wvec]
    u32x4 v[kWinVecPerThread];
    #pragma unroll
    for (uint32_t u = 0; u < kWinVecPerThread; ++u) {
        const uint64_t j = (uint64_t)u * kThreads + threadIdx.x;
        if (j < wvec) {
            const uint64_t k = j + nvec;
            v[u] = k < wvec ? dst[k] : src[k - wvec];
        }
    }
    __syncthreads();  // every read of the old window is done before any write
    #pragma unroll
    for (uint32_t u = 0; u < kWinVecPerThread; ++u) {
        const uint64_t j = (uint64_t)u * kThreads + threadIdx.x;
        if (j < wvec) dst[j] = v[u];
    }
}

}  // namespace

hipError_t launch_append(const AppendParams& p, hipStream_t stream) {
    const uint32_t blocks = p.first_block[p.n_seg];
    if (blocks == 0) return hipSuccess;
    return launch_kernel(reinterpret_cast<const void*>(&append_kernel), dim3(blocks), dim3(kThreads), p, stream);
}

}  // namespace cap
