// Descriptor-driven batched copy for capsule snapshot / restore / fork /
// gather-restore on gfx950.
//
// A capsule is the live buffer set valid at the aligned boundary P' (paper
// §3 Algorithm 1): buffers in set order, positional buffers contributing rows
// [0, P'), fixed buffers all their bytes.  The copy is HBM-bound (§3 Table
// "cost structure": restore is a bandwidth-bound copy of Theta(bytes)), so the
// kernel is built for bytes in flight, not arithmetic:
//   * each buffer's valid range is cut into tiles of kThreads x kUnroll
//     16-byte vectors that never cross a buffer boundary, one block per tile,
//     so inside a tile every thread addresses base + index with block-uniform
//     bases, and the kUnroll 16-byte loads of a thread are all issued before
//     its first store (global_load_dwordx4 / global_store_dwordx4, 1 KiB per
//     wave instruction);
//   * tile counts per buffer depend on the call's P', so each block turns the
//     set's static (a, b) table into capsule offsets and an exclusive prefix
//     sum of tile counts once, in LDS, and finds its tile's buffer by a
//     binary search in LDS;
//   * fork reads each vector once and stores it to every destination set;
//     gather gives each environment ("rep") its own source arena.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace cap {
namespace {

constexpr int kMaxSeg = 512;  // buffers per set

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte load / store, optionally non-temporal (streamed past the caches).
template <bool NT>
__device__ inline u32x4 ld16(const u32x4* p) {
    if (NT) return __builtin_nontemporal_load(p);
    return *p;
}

template <bool NT>
__device__ inline void st16(u32x4* p, const u32x4& v) {
    if (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

__device__ inline uint64_t seg_start(const SegEntry* t, uint32_t i, uint64_t P) {
    return (t[i].a + P * t[i].b) >> 4;  // in 16-byte vectors
}

// Last index i in [0, n] with a[i] <= x (a non-decreasing, a[0] = 0 <= x).
__device__ inline uint32_t last_le(const uint32_t* a, uint32_t n, uint32_t x) {
    uint32_t lo = 0, hi = n;
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (a[mid] <= x) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// kThreads threads of kUnroll 16-byte vectors each form one tile; kPtr
// destination pointers (buffers x destination sets) fit in LDS.
template <int kThreads, int kUnroll, bool NT_LD, bool NT_ST, int kPtr>
__global__ __launch_bounds__(kThreads) void capsule_copy_kernel(const CopyParams p) {
    constexpr uint32_t kTileVec = (uint32_t)kThreads * kUnroll;
    constexpr int kPer = (kMaxSeg + 1 + kThreads - 1) / kThreads;  // table entries per thread
    __shared__ uint64_t s_start[kMaxSeg + 1];  // capsule vector offset of buffer i
    __shared__ uint32_t s_tile[kMaxSeg + 1];   // first tile of buffer i
    __shared__ uint32_t s_wave[kThreads / 64];
    __shared__ uint64_t s_ptr[kPtr];           // live pointers of the current rep

    const uint32_t tid = threadIdx.x;
    const uint32_t lane = tid & 63, wave = tid >> 6;
    const uint32_t n = p.n_seg;

    // ---- per-call layout: starts and exclusive prefix sum of tile counts
    uint32_t cnt[kPer];
    uint32_t mine = 0;
    #pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const uint32_t i = tid * kPer + e;
        cnt[e] = 0;
        if (i <= n) {
            const uint64_t s0 = seg_start(p.layout, i, p.P);
            s_start[i] = s0;
            if (i < n) {
                const uint64_t len = seg_start(p.layout, i + 1, p.P) - s0;
                cnt[e] = (uint32_t)((len + kTileVec - 1) / kTileVec);
            }
        }
        mine += cnt[e];
    }
    uint32_t incl = mine;  // inclusive scan over the wave
    #pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off, 64);
        if (lane >= (uint32_t)off) incl += y;
    }
    if (lane == 63) s_wave[wave] = incl;
    __syncthreads();
    uint32_t before = incl - mine;
    for (uint32_t wv = 0; wv < wave; ++wv) before += s_wave[wv];
    #pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const uint32_t i = tid * kPer + e;
        if (i <= n) s_tile[i] = before;
        before += cnt[e];
    }
    __syncthreads();

    const uint32_t tiles_per_rep = s_tile[n];
    const uint64_t n_tiles = (uint64_t)tiles_per_rep * p.n_rep;
    const uint32_t n_dst = p.n_dst;
    int64_t cur_rep = -1;
    const u32x4* rep_src = nullptr;

    for (uint64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
        const uint32_t rep = (uint32_t)(t / tiles_per_rep);
        const uint32_t lt = (uint32_t)(t - (uint64_t)rep * tiles_per_rep);
        if ((int64_t)rep != cur_rep) {  // block-uniform
            __syncthreads();
            if (p.mode == kLiveToArena) {
                for (uint32_t i = tid; i < n; i += kThreads) s_ptr[i] = p.tabs[0][i].ptr;
            } else {
                for (uint32_t i = tid; i < n * n_dst; i += kThreads) {
                    const uint32_t d = i / n, s = i - d * n;
                    s_ptr[i] = p.tabs[rep * n_dst + d][s].ptr;
                }
                rep_src = reinterpret_cast<const u32x4*>(p.arena_in[rep]);
            }
            __syncthreads();
            cur_rep = (int64_t)rep;
        }

        const uint32_t seg = __builtin_amdgcn_readfirstlane(last_le(s_tile, n, lt));
        const uint64_t s0 = s_start[seg];
        const uint64_t len = s_start[seg + 1] - s0;
        const uint64_t off = (uint64_t)(lt - s_tile[seg]) * kTileVec;
        const uint64_t lim = len - off;  // vectors left in this buffer from the tile start
        u32x4 data[kUnroll];
        // Full tiles take a branch-free path; the last, partial tile of a
        // buffer clamps its load indices (so every load stays inside the
        // buffer) and predicates its stores.
        const bool full = lim >= kTileVec;
        const uint32_t last = (uint32_t)((full ? (uint64_t)kTileVec : lim) - 1);

        if (p.mode == kLiveToArena) {
            const u32x4* src = reinterpret_cast<const u32x4*>(s_ptr[seg]) + off;
            u32x4* dst = reinterpret_cast<u32x4*>(p.arena_out) + s0 + off;
            #pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const uint32_t i = u * kThreads + tid;
                data[u] = ld16<NT_LD>(src + (i < last ? i : last));
            }
            if (full) {
                #pragma unroll
                for (int u = 0; u < kUnroll; ++u) st16<NT_ST>(dst + u * kThreads + tid, data[u]);
            } else {
                #pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const uint32_t i = u * kThreads + tid;
                    if (i <= last) st16<NT_ST>(dst + i, data[u]);
                }
            }
        } else {
            const u32x4* src = rep_src + s0 + off;
            #pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const uint32_t i = u * kThreads + tid;
                data[u] = ld16<NT_LD>(src + (i < last ? i : last));
            }
            for (uint32_t d = 0; d < n_dst; ++d) {
                u32x4* dst = reinterpret_cast<u32x4*>(s_ptr[d * n + seg]) + off;
                if (full) {
                    #pragma unroll
                    for (int u = 0; u < kUnroll; ++u) st16<NT_ST>(dst + u * kThreads + tid, data[u]);
                } else {
                    #pragma unroll
                    for (int u = 0; u < kUnroll; ++u) {
                        const uint32_t i = u * kThreads + tid;
                        if (i <= last) st16<NT_ST>(dst + i, data[u]);
                    }
                }
            }
        }
    }
}

}  // namespace

namespace {

// tile shape of each verb (see launch_copy)
struct Shape {
    uint64_t threads, unroll, ptr;
};

Shape shape_of(const CopyParams& p) {
    if (p.n_dst > 1) return {512, 1, (uint64_t)kMaxPtrLds};
    return {256, 4, (uint64_t)kMaxSeg};
}

uint64_t tiles_of(const CopyParams& p) {
    const Shape s = shape_of(p);
    // one block per tile; every buffer adds at most one partial tile
    return (p.nvec / (s.threads * s.unroll) + p.n_seg) * p.n_rep;
}

template <int kThreads, int kUnroll, bool NT_LD, bool NT_ST, int kPtr>
hipError_t launch_t(const CopyParams& p, hipStream_t stream) {
    return launch_kernel(reinterpret_cast<const void*>(&capsule_copy_kernel<kThreads, kUnroll, NT_LD, NT_ST, kPtr>),
                         dim3((unsigned)tiles_of(p)), dim3(kThreads), p, stream);
}

}  // namespace

bool copy_params_ok(const CopyParams& p) {
    if (p.nvec == 0 || p.n_rep == 0) return true;
    if (p.n_seg > (uint32_t)kMaxSeg || (uint64_t)p.n_seg * p.n_dst > (uint64_t)kMaxPtrLds) return false;
    if ((uint64_t)p.n_seg * p.n_dst > shape_of(p).ptr) return false;
    return tiles_of(p) <= 0x7fffffffull;
}

hipError_t launch_copy(const CopyParams& p, int num_cus, hipStream_t stream) {
    (void)num_cus;
    if (p.nvec == 0 || p.n_rep == 0) return hipSuccess;
    if (!copy_params_ok(p)) return hipErrorInvalidValue;
    // Tile shapes chosen by measurement on MI355X:
    //  * snapshot / restore (882 MB capsule): 16 KiB tiles, loads and stores
    //    streamed past the caches;
    //  * fork, which stores every loaded vector several times: 8 KiB tiles of
    //    512 threads, streamed;
    //  * gather-restore: 16 KiB tiles with cached loads, so that a gallery
    //    small enough for the 256 MB Infinity Cache stays there across resets,
    //    and streamed stores, so that the environments' bytes do not evict it
    //    (-14 % per reset against cached stores).
    // Only fork keeps several destination pointer tables in LDS; the other
    // verbs size that table for one set, which leaves room for eight blocks
    // per CU.
    if (p.n_dst > 1) return launch_t<512, 1, true, true, kMaxPtrLds>(p, stream);
    if (p.n_rep > 1) return launch_t<256, 4, false, true, kMaxSeg>(p, stream);
    return launch_t<256, 4, true, true, kMaxSeg>(p, stream);
}

}  // namespace cap
