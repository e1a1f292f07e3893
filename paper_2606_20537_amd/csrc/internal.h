// Internal interface between the host ABI (capsule_host.cpp) and the HIP
// kernels (capsule_copy.hip, linattn_scan.hip, linattn_step.hip,
// gdn_scan.hip, gdn_step.hip, kv_fp8.hip, append.hip).  Not part of the
// public ABI.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "capsule.h"

namespace cap {

// Launch a kernel whose one argument is a parameter struct passed by value
// and return that launch's own status.  The library never calls
// hipGetLastError, so an error the caller left pending is neither read nor
// cleared by a launch.
template <class P>
inline hipError_t launch_kernel(const void* fn, dim3 grid, dim3 block, const P& p, hipStream_t stream) {
    void* args[] = {const_cast<P*>(&p)};
    return hipLaunchKernel(fn, grid, block, args, 0, stream);
}

// One entry of a live set's static device segment table.  For buffer i of a
// set, with the boundary P' chosen per call:
//   capsule byte offset of buffer i = a + P' * b
// where a sums the bytes of the fixed buffers before i and b sums the
// row_bytes of the positional buffers before i.  Entry n (one past the last
// buffer) carries the totals, so the capsule size is a[n] + P' * b[n] and
// buffer i occupies [a[i] + P' b[i], a[i+1] + P' b[i+1]).  All values are
// multiples of 16 bytes.
struct SegEntry {
    uint64_t ptr;  // live device address of buffer i (0 in entry n)
    uint64_t a;
    uint64_t b;
};

constexpr int kMaxRep = 64;   // sources (gather environments) per launch
constexpr int kMaxDst = 16;   // destinations per source (fork)
constexpr int kMaxPtrLds = 2048;  // live pointers one copy block holds in LDS

enum CopyMode : int { kLiveToArena = 0, kArenaToLive = 1 };

// Per-launch arguments of the copy kernel, passed by value.
//   kLiveToArena : rep 0 copies set `tabs[0]` -> arena_out.
//   kArenaToLive : rep r copies arena_in[r] -> n_dst destination sets
//                  tabs[r * n_dst + d] (fork: one rep, n_dst sets;
//                  gather: n_rep reps, one set each).
struct CopyParams {
    const SegEntry* layout;            // any table of the call (shared a, b)
    const SegEntry* tabs[kMaxRep];
    const uint8_t*  arena_in[kMaxRep];
    uint8_t*        arena_out;
    uint64_t        P;                 // aligned boundary
    uint64_t        nvec;              // capsule bytes / 16
    uint32_t        n_seg;
    uint32_t        n_dst;
    uint32_t        n_rep;
    int32_t         mode;
};

// Whether launch_copy accepts p (grid and LDS-table limits); a multi-launch
// call checks every launch with it before enqueueing the first one.
bool copy_params_ok(const CopyParams& p);
// Launch the descriptor-driven copy.  Returns hipSuccess or the launch error.
hipError_t launch_copy(const CopyParams& p, int num_cus, hipStream_t stream);

// Scan arguments after host validation (sizes as 64-bit, pointers raw).
struct ScanParams {
    const void*  q;
    const void*  k;
    const void*  v;
    const float* g;
    const float* state_in;
    float*       o;
    float*       chunk_states;
    float*       final_state;
    int64_t      T;
    int32_t      H, dk, dv;
    int32_t      in_f32;   // 1: q/k/v are fp32, 0: bf16
    float        scale;
};

// Host checks of a linattn_args (status codes as documented in capsule.h);
// on CAP_OK *out holds the launch parameters.
int validate_linattn(const linattn_args* a, ScanParams* out);

hipError_t launch_linattn_scan(const ScanParams& p, hipStream_t stream);
// T == 1, bf16 inputs (a decode step); same contract as launch_linattn_scan
hipError_t launch_linattn_step(const ScanParams& p, hipStream_t stream);

// Gated delta-rule prefill (bf16 q/k/v, fp32 gates, write strengths and
// state).  ws holds one record of kGdnWsRecord bytes per chunk of 64 tokens
// and head ([n_chunks][H]), written by the first launch and read by the
// scan: the causal blocks of the chunk's (I + A)^-1 as bf16 hi/lo MFMA
// operands (6 blocks x 2 KiB, in the scan's lane order), then G log2(e) (64
// fp32, inclusive in-chunk log-gate sums) and beta (64 fp32).
constexpr int64_t kGdnWsTBytes = 6 * 2048;
constexpr int64_t kGdnWsTabOff = kGdnWsTBytes;
constexpr int64_t kGdnWsRecord = kGdnWsTabOff + 2 * 64 * 4;

struct GdnParams {
    const void*  q;
    const void*  k;
    const void*  v;
    const float* g;
    const float* beta;
    const float* state_in;
    float*       o;
    float*       chunk_states;
    float*       final_state;
    uint8_t*     ws;
    int64_t      T;
    int32_t      H, dk, dv;
    float        scale;
};

// Host checks of a gdn_args; need_ws: the call reads args->workspace (a
// decode step does not).  On CAP_OK *out holds the launch parameters (ws =
// the caller's workspace, or NULL when need_ws is false).
int validate_gdn(const gdn_args* a, bool need_ws, GdnParams* out);

hipError_t launch_gdn(const GdnParams& p, hipStream_t stream);
// T == 1 (a decode step): one launch, no workspace use
hipError_t launch_gdn_step(const GdnParams& p, hipStream_t stream);

// FP8 (OCP E4M3) conversion of up to kFp8MaxSeg segments in one launch.
// Segment s converts n_groups[s] groups of 16 elements from src[s] to
// dst[s]; block b of the grid works on segment s with first_block[s] <= b <
// first_block[s + 1].  Quantize multiplies by mul[s] (1 / scale) before
// encoding; dequantize multiplies the decoded value by mul[s] (scale).
constexpr int kFp8MaxSeg = 64;
constexpr int kFp8GroupsPerBlock = 512;  // 256 threads x 2 groups of 16 elements

struct Fp8Params {
    uint64_t src[kFp8MaxSeg];
    uint64_t dst[kFp8MaxSeg];
    uint64_t n_groups[kFp8MaxSeg];
    uint32_t first_block[kFp8MaxSeg + 1];
    float    mul[kFp8MaxSeg];
    uint32_t n_seg;
    int32_t  quantize;  // 1: bf16 -> e4m3, 0: e4m3 -> bf16
};

hipError_t launch_fp8(const Fp8Params& p, hipStream_t stream);

// Append of a suffix of n tokens to a live set (one launch, up to
// kAppendMaxSeg buffers).  Segment s is either a positional copy of
// bytes[s] bytes from src[s] to dst[s] (tiles of kAppendTile bytes, several
// blocks), or, when win[s] != 0, a sliding window of win[s] bytes at dst[s]
// that takes the last win[s] bytes of (window, then the bytes[s] source
// bytes) in one block.  Block b works on segment s with first_block[s] <= b
// < first_block[s + 1].
constexpr int kAppendMaxSeg = 128;
constexpr uint32_t kAppendTile = 16384;        // bytes per positional block
constexpr uint32_t kAppendMaxWindow = 65536;   // bytes of one window

struct AppendParams {
    uint64_t src[kAppendMaxSeg];
    uint64_t dst[kAppendMaxSeg];
    uint64_t bytes[kAppendMaxSeg];
    uint32_t win[kAppendMaxSeg];
    uint32_t first_block[kAppendMaxSeg + 1];
    uint32_t n_seg;
};

hipError_t launch_append(const AppendParams& p, hipStream_t stream);

}  // namespace cap
