// Gated delta-rule prefill for callers that cannot allocate device memory
// (code under stream capture, tight serving loops): the same kernels as
// gdn_chunked_prefill, with the per-chunk workspace in a fixed array of
// device memory that the library owns instead of a caller workspace.
//
// The array holds two fp32 states of all heads (the hand-over between
// segments) and then as many per-(chunk, head) workspace records as fit.  A
// call whose chunks do not all fit runs as several segments of whole
// chunks, each a prepare launch and a scan launch, the state passing from
// one segment to the next through the two state slots.  A chunk's
// arithmetic depends only on (state entering it, its inputs), so a call cut
// into segments at chunk boundaries computes exactly what one call over all
// chunks computes (the aligned-continuation property of the scan).
#include <hip/hip_runtime.h>

#include <mutex>
#include <new>

#include "capsule.h"
#include "internal.h"

namespace {

constexpr uint64_t kScratchBytes = GDN_NOALLOC_SCRATCH_BYTES;

// Device scratch of this entry point: one copy per GPU the library runs on,
// held until the process ends.  Host code never uses this name as an
// address (on the host it is only a stand-in for the symbol); it uses the
// per-device address returned by hipGetSymbolAddress instead.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
uint8_t* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up

// Address of this device's scratch, looked up once per device with that
// device current.
int device_scratch(uint8_t** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CAP_E_HIP;
    if (dev < 0 || dev >= kMaxDevices) return CAP_E_UNSUPPORTED;
    std::lock_guard<std::mutex> guard(g_lock);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return CAP_E_HIP;
        g_scratch[dev] = static_cast<uint8_t*>(p);
    }
    *out = g_scratch[dev];
    return CAP_OK;
}

uint64_t round256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

int run(const gdn_args* a, void* stream) {
    if (!a) return CAP_E_INVAL;
    if (a->workspace || a->workspace_bytes) return CAP_E_INVAL;  // this variant takes no workspace
    cap::GdnParams p{};
    int rc = cap::validate_gdn(a, false, &p);
    if (rc != CAP_OK) return rc;
    const uint64_t H = (uint64_t)a->H, dk = (uint64_t)a->dk, dv = (uint64_t)a->dv;
    const uint64_t slot_bytes = round256(H * dk * dv * 4);
    const uint64_t chunk_rec = H * (uint64_t)cap::kGdnWsRecord;  // one chunk of all heads
    if (2 * slot_bytes + chunk_rec > kScratchBytes) return CAP_E_SIZE;
    if (a->T == 0 && !a->final_state) return CAP_OK;

    uint8_t* base = nullptr;
    rc = device_scratch(&base);
    if (rc != CAP_OK) return rc;
    float* slot[2] = {reinterpret_cast<float*>(base), reinterpret_cast<float*>(base + slot_bytes)};
    uint8_t* ws = base + 2 * slot_bytes;
    const hipStream_t s = static_cast<hipStream_t>(stream);

    const int64_t T = a->T;
    const int64_t n_chunks = (T + 63) / 64;
    const int64_t per_seg = (int64_t)((kScratchBytes - 2 * slot_bytes) / chunk_rec);
    if (n_chunks == 0) {  // T == 0: the final state is the entering state
        p.ws = ws;
        return cap::launch_gdn(p, s) == hipSuccess ? CAP_OK : CAP_E_HIP;
    }
    const char* q = static_cast<const char*>(a->q);
    const char* k = static_cast<const char*>(a->k);
    const char* v = static_cast<const char*>(a->v);
    int seg = 0;
    for (int64_t c0 = 0; c0 < n_chunks; c0 += per_seg, ++seg) {
        const int64_t c1 = c0 + per_seg < n_chunks ? c0 + per_seg : n_chunks;
        const bool last = c1 == n_chunks;
        const int64_t t0 = 64 * c0;
        const int64_t t1 = last ? T : 64 * c1;
        cap::GdnParams g = p;
        g.q = q + t0 * (int64_t)(H * dk * 2);
        g.k = k + t0 * (int64_t)(H * dk * 2);
        g.v = v + t0 * (int64_t)(H * dv * 2);
        g.g = a->g + t0 * (int64_t)H;
        g.beta = a->beta + t0 * (int64_t)H;
        g.o = a->o + t0 * (int64_t)(H * dv);
        g.chunk_states = a->chunk_states ? a->chunk_states + c0 * (int64_t)(H * dk * dv) : nullptr;
        g.state_in = seg == 0 ? a->state_in : slot[(seg - 1) & 1];
        g.final_state = last ? a->final_state : slot[seg & 1];
        g.T = t1 - t0;
        g.ws = ws;
        if (cap::launch_gdn(g, s) != hipSuccess) return CAP_E_HIP;
    }
    return CAP_OK;
}

}  // namespace

extern "C" int gdn_chunked_prefill_noalloc(const gdn_args* a, void* stream) {
    try {
        return run(a, stream);
    } catch (const std::bad_alloc&) {
        return CAP_E_NOMEM;
    } catch (...) {
        return CAP_E_INVAL;
    }
}
