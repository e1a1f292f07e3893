// Host side of the capsule C ABI: live sets, capsule headers, argument
// checks and kernel launches.  Every check runs before anything is enqueued,
// so an error return leaves device memory untouched (paper §4: the contract
// is mechanism only and reports errors as int status codes; §3 Algorithm 1:
// restore asserts the deployment digest before copying).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <atomic>
#include <memory>
#include <stdexcept>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>
#include <utility>
#include <vector>

#include "capsule.h"
#include "internal.h"

using cap::SegEntry;

struct BufInfo {
    std::string name;
    uint64_t ptr;
    uint64_t row_bytes;
    uint64_t rows;
    uint32_t kind;
};

// A BF16 working stage bound to an FP8 positional buffer of a set.
struct StageInfo {
    uint32_t buf;     // index of the FP8 buffer in the set
    uint64_t ptr;     // stage device address: rows x row_bytes bf16 elements
    float scale;
};

struct cap_set_s {
    std::vector<BufInfo> bufs;
    uint32_t chunk = 1;
    uint64_t deploy_key = 0;
    uint64_t position = 0;
    uint64_t max_position = 0;  // smallest positional capacity (UINT64_MAX if none)
    SegEntry* dtab = nullptr;   // n + 1 entries on the device
    int device = 0;
    int num_cus = 256;
    // FP8 working stages and their valid end: rows [0, stage_end) of every
    // bound stage are the dequantised FP8 rows.  `epoch` names the lineage of
    // the set's positional rows: it changes whenever rows the set already
    // held may be replaced (restore, fork, gather into the set, an append
    // below `high_water`, a rebinding); `high_water` is the end of the rows
    // written in this lineage.
    std::vector<StageInfo> stages;
    uint64_t stage_end = 0;
    uint64_t uid = 0;
    uint64_t epoch = 0;
    uint64_t high_water = 0;
};

struct cap_capsule_s {
    uint64_t P_requested = 0;
    uint64_t P_aligned = 0;
    uint64_t prefix_digest = 0;
    uint64_t deploy_key = 0;
    uint64_t bytes = 0;
    const void* arena = nullptr;
    uint64_t arena_bytes = 0;
    uint32_t tier = CAP_TIER_DEVICE;  // where the arena lives
    std::vector<uint64_t> row_bytes, rows;
    std::vector<uint32_t> kinds;
    // the FP8 stage's valid end at the snapshot (clipped to P'), and the
    // set and lineage it was recorded in
    uint64_t stage_end = 0;
    uint64_t set_uid = 0;
    uint64_t epoch = 0;
};

namespace {

// Every entry point runs its body through guarded(): a host allocation that
// fails (std::bad_alloc from a container, say) becomes CAP_E_NOMEM instead
// of an exception crossing the C boundary.
template <class F>
int guarded(F&& body) noexcept {
    try {
        return body();
    } catch (const std::bad_alloc&) {
        return CAP_E_NOMEM;
    } catch (const std::length_error&) {
        return CAP_E_NOMEM;
    } catch (...) {
        return CAP_E_INVAL;
    }
}

bool aligned16(uint64_t x) { return (x & 15u) == 0; }

// Process-wide counter for set identities and lineage epochs.
std::atomic<uint64_t> g_ids{1};
uint64_t next_id() { return g_ids.fetch_add(1, std::memory_order_relaxed); }

// The rows a set held may have been replaced: new lineage, stage valid over
// no rows unless `keep` says otherwise.
void new_lineage(cap_set_s* s, uint64_t keep_stage_end, uint64_t high_water) {
    s->stage_end = keep_stage_end;
    s->epoch = next_id();
    s->high_water = high_water;
}

uint64_t buf_bytes(uint64_t row_bytes, uint64_t rows, uint32_t kind, uint64_t P) {
    return kind == CAP_KIND_POSITIONAL ? P * row_bytes : row_bytes * rows;
}

// Shared checks of a buffer list.  need_ptr: device pointers must be set.
int check_bufs(const cap_buf* bufs, uint32_t n, uint32_t chunk, bool need_ptr) {
    if (!bufs || n == 0) return CAP_E_INVAL;
    if (n > CAP_MAX_BUFFERS) return CAP_E_UNSUPPORTED;
    if (chunk == 0) return CAP_E_INVAL;
    uint64_t total = 0;  // every byte count derived from the set stays below this sum
    for (uint32_t i = 0; i < n; ++i) {
        const cap_buf& b = bufs[i];
        if (b.kind != CAP_KIND_POSITIONAL && b.kind != CAP_KIND_FIXED) return CAP_E_UNSUPPORTED;
        if (b.reserved != 0) return CAP_E_INVAL;
        if (b.row_bytes == 0 || b.rows == 0) return CAP_E_INVAL;
        if (b.row_bytes > (UINT64_MAX / b.rows)) return CAP_E_SIZE;
        const uint64_t size = b.row_bytes * b.rows;
        if (size > UINT64_MAX - total) return CAP_E_SIZE;
        total += size;
        if (need_ptr && !b.dptr) return CAP_E_INVAL;
        if (need_ptr && (uint64_t)(uintptr_t)b.dptr > UINT64_MAX - size) return CAP_E_SIZE;  // range wraps
        if (!aligned16(b.row_bytes) || !aligned16((uint64_t)(uintptr_t)b.dptr)) return CAP_E_ALIGN;
    }
    // unique names (when given)
    std::vector<std::string> names;
    for (uint32_t i = 0; i < n; ++i)
        if (bufs[i].name) names.emplace_back(bufs[i].name);
    std::sort(names.begin(), names.end());
    if (std::adjacent_find(names.begin(), names.end()) != names.end()) return CAP_E_INVAL;
    if (need_ptr) {  // pairwise disjoint
        std::vector<std::pair<uint64_t, uint64_t>> r;
        for (uint32_t i = 0; i < n; ++i) {
            const uint64_t p = (uint64_t)(uintptr_t)bufs[i].dptr;
            r.emplace_back(p, p + bufs[i].row_bytes * bufs[i].rows);
        }
        std::sort(r.begin(), r.end());
        for (size_t i = 1; i < r.size(); ++i)
            if (r[i].first < r[i - 1].second) return CAP_E_INVAL;
    }
    return CAP_OK;
}

bool overlaps(uint64_t a0, uint64_t a1, uint64_t b0, uint64_t b1) { return a0 < b1 && b0 < a1; }

int current_device_matches(const cap_set_s* s) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CAP_E_HIP;
    return dev == s->device ? CAP_OK : CAP_E_INVAL;
}

bool same_layout(const cap_capsule_s* c, const cap_set_s* s) {
    if (c->kinds.size() != s->bufs.size()) return false;
    for (size_t i = 0; i < s->bufs.size(); ++i)
        if (c->row_bytes[i] != s->bufs[i].row_bytes || c->rows[i] != s->bufs[i].rows ||
            c->kinds[i] != s->bufs[i].kind)
            return false;
    return true;
}

// restore-side checks shared by restore, fork and gather (digest first).
int check_restore_target(const cap_capsule_s* c, const cap_set_s* s, uint64_t prefix_digest, bool check_prefix) {
    if (check_prefix && c->prefix_digest != prefix_digest) return CAP_E_DIGEST;
    if (c->deploy_key != s->deploy_key) return CAP_E_DIGEST;
    if (c->tier != CAP_TIER_DEVICE) return CAP_E_STATE;  // promote it first (capsule_move)
    if (!same_layout(c, s)) return CAP_E_SIZE;
    if (c->P_aligned > s->max_position) return CAP_E_SIZE;
    const uint64_t a0 = (uint64_t)(uintptr_t)c->arena, a1 = a0 + c->bytes;
    for (const BufInfo& b : s->bufs)
        if (overlaps(a0, a1, b.ptr, b.ptr + b.row_bytes * b.rows)) return CAP_E_INVAL;
    return CAP_OK;
}

int launch_status(hipError_t e) { return e == hipSuccess ? CAP_OK : CAP_E_HIP; }

// Live byte ranges of every buffer of the given sets must be pairwise
// disjoint (several destination sets of one fork or gather).
bool sets_disjoint(const cap_set* lives, uint32_t n) {
    std::vector<std::pair<uint64_t, uint64_t>> r;
    for (uint32_t i = 0; i < n; ++i)
        for (const BufInfo& b : lives[i]->bufs) r.emplace_back(b.ptr, b.ptr + b.row_bytes * b.rows);
    std::sort(r.begin(), r.end());
    for (size_t i = 1; i < r.size(); ++i)
        if (r[i].first < r[i - 1].second) return false;
    return true;
}

// Tier of an arena: memory of the current device, or page-locked host memory
// the device can address (hipHostMalloc).  Anything else -- pageable host
// memory, another device's memory, managed memory -- is rejected.
int arena_tier(const void* p, uint32_t* tier) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CAP_E_HIP;
    hipPointerAttribute_t a{};
    const hipError_t pending = hipPeekAtLastError();
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        // an unknown pointer makes the query report an error; clear it only
        // when no error was pending before the query, so an error the caller
        // left pending is never cleared
        if (pending == hipSuccess) (void)hipGetLastError();
        return CAP_E_INVAL;
    }
    if (a.isManaged) return CAP_E_UNSUPPORTED;
    if (a.type == hipMemoryTypeDevice && a.device == dev) { *tier = CAP_TIER_DEVICE; return CAP_OK; }
    if (a.type == hipMemoryTypeHost && a.devicePointer != nullptr) { *tier = CAP_TIER_HOST; return CAP_OK; }
    return CAP_E_INVAL;
}

}  // namespace

extern "C" {

const char* cap_status_string(int status) {
    switch (status) {
        case CAP_OK: return "ok";
        case CAP_E_INVAL: return "invalid argument";
        case CAP_E_SIZE: return "size or layout mismatch";
        case CAP_E_DIGEST: return "digest or deployment key mismatch";
        case CAP_E_UNSUPPORTED: return "unsupported kind, shape or dtype";
        case CAP_E_ALIGN: return "pointer or size not 16-byte aligned";
        case CAP_E_STATE: return "wrong state: set position is not the aligned boundary, or capsule not device-resident";
        case CAP_E_HIP: return "HIP runtime error";
        case CAP_E_NOMEM: return "host memory allocation failed";
        default: return "unknown status";
    }
}

uint64_t cap_align_boundary(uint64_t P, uint32_t chunk) {
    return chunk ? (P / chunk) * (uint64_t)chunk : 0;
}

int capsule_layout_bytes(const cap_buf* bufs, uint32_t n, uint32_t chunk, uint64_t P, uint64_t* bytes) {
    return guarded([&]() -> int {
        if (!bytes) return CAP_E_INVAL;
        const int rc = check_bufs(bufs, n, chunk, false);
        if (rc != CAP_OK) return rc;
        const uint64_t Pa = cap_align_boundary(P, chunk);
        uint64_t total = 0;
        for (uint32_t i = 0; i < n; ++i) {
            if (bufs[i].kind == CAP_KIND_POSITIONAL && Pa > bufs[i].rows) return CAP_E_SIZE;
            total += buf_bytes(bufs[i].row_bytes, bufs[i].rows, bufs[i].kind, Pa);
        }
        *bytes = total;
        return CAP_OK;
    });
}

int cap_set_create(const cap_buf* bufs, uint32_t n, uint32_t chunk, uint64_t deploy_key, cap_set* out) {
    if (!out) return CAP_E_INVAL;
    *out = nullptr;
    return guarded([&]() -> int {
        int rc = check_bufs(bufs, n, chunk, true);
        if (rc != CAP_OK) return rc;

        cap_set_s* s = new (std::nothrow) cap_set_s();
        if (!s) return CAP_E_NOMEM;
        std::unique_ptr<cap_set_s> own(s);
        s->chunk = chunk;
        s->deploy_key = deploy_key;
        s->max_position = UINT64_MAX;
        s->uid = next_id();
        s->epoch = next_id();
        std::vector<SegEntry> tab(n + 1);
        uint64_t a = 0, b = 0;
        for (uint32_t i = 0; i < n; ++i) {
            BufInfo bi{bufs[i].name ? bufs[i].name : std::string(), (uint64_t)(uintptr_t)bufs[i].dptr,
                       bufs[i].row_bytes, bufs[i].rows, bufs[i].kind};
            s->bufs.push_back(bi);
            tab[i] = SegEntry{bi.ptr, a, b};
            if (bi.kind == CAP_KIND_POSITIONAL) {
                b += bi.row_bytes;
                s->max_position = std::min(s->max_position, bi.rows);
            } else {
                a += bi.row_bytes * bi.rows;
            }
        }
        tab[n] = SegEntry{0, a, b};

        if (hipGetDevice(&s->device) != hipSuccess) return CAP_E_HIP;
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, s->device) == hipSuccess && cus > 0)
            s->num_cus = cus;
        void* d = nullptr;
        if (hipMalloc(&d, sizeof(SegEntry) * (n + 1)) != hipSuccess) return CAP_E_HIP;
        if (hipMemcpy(d, tab.data(), sizeof(SegEntry) * (n + 1), hipMemcpyHostToDevice) != hipSuccess) {
            (void)hipFree(d);
            return CAP_E_HIP;
        }
        s->dtab = static_cast<SegEntry*>(d);
        *out = own.release();
        return CAP_OK;
    });
}

int cap_set_destroy(cap_set set) {
    if (!set) return CAP_E_INVAL;
    if (set->dtab) (void)hipFree(set->dtab);
    delete set;
    return CAP_OK;
}

int cap_set_set_position(cap_set set, uint64_t position) {
    if (!set) return CAP_E_INVAL;
    if (position > set->max_position) return CAP_E_SIZE;
    set->position = position;
    return CAP_OK;
}

int cap_set_get_position(cap_set set, uint64_t* position) {
    if (!set || !position) return CAP_E_INVAL;
    *position = set->position;
    return CAP_OK;
}

int capsule_bytes(cap_set set, uint64_t P, uint64_t* bytes) {
    if (!set || !bytes) return CAP_E_INVAL;
    const uint64_t Pa = cap_align_boundary(P, set->chunk);
    if (Pa > set->max_position) return CAP_E_SIZE;
    uint64_t total = 0;
    for (const BufInfo& b : set->bufs) total += buf_bytes(b.row_bytes, b.rows, b.kind, Pa);
    *bytes = total;
    return CAP_OK;
}

int capsule_snapshot(cap_set live, uint64_t P, uint64_t prefix_digest, void* arena, uint64_t arena_bytes,
                     void* stream, cap_capsule* out) {
    if (!out) return CAP_E_INVAL;
    *out = nullptr;
    return guarded([&]() -> int {
        if (!live || !arena) return CAP_E_INVAL;
        if (!aligned16((uint64_t)(uintptr_t)arena)) return CAP_E_ALIGN;
        const uint64_t Pa = cap_align_boundary(P, live->chunk);
        if (Pa > live->max_position) return CAP_E_SIZE;
        if (live->position != Pa) return CAP_E_STATE;
        uint64_t bytes = 0;
        capsule_bytes(live, P, &bytes);
        if (arena_bytes < bytes) return CAP_E_SIZE;
        const uint64_t a0 = (uint64_t)(uintptr_t)arena, a1 = a0 + bytes;
        for (const BufInfo& b : live->bufs)
            if (overlaps(a0, a1, b.ptr, b.ptr + b.row_bytes * b.rows)) return CAP_E_INVAL;
        int rc = current_device_matches(live);
        if (rc != CAP_OK) return rc;
        uint32_t tier = CAP_TIER_DEVICE;
        rc = arena_tier(arena, &tier);
        if (rc != CAP_OK) return rc;

        cap_capsule_s* c = new (std::nothrow) cap_capsule_s();
        if (!c) return CAP_E_NOMEM;
        std::unique_ptr<cap_capsule_s> own(c);
        c->tier = tier;
        c->P_requested = P;
        c->P_aligned = Pa;
        c->prefix_digest = prefix_digest;
        c->deploy_key = live->deploy_key;
        c->bytes = bytes;
        c->arena = arena;
        c->arena_bytes = arena_bytes;
        for (const BufInfo& b : live->bufs) {
            c->row_bytes.push_back(b.row_bytes);
            c->rows.push_back(b.rows);
            c->kinds.push_back(b.kind);
        }
        c->stage_end = std::min(live->stage_end, Pa);
        c->set_uid = live->uid;
        c->epoch = live->epoch;

        cap::CopyParams p{};
        p.layout = live->dtab;
        p.tabs[0] = live->dtab;
        p.arena_out = static_cast<uint8_t*>(arena);
        p.P = Pa;
        p.nvec = bytes / 16;
        p.n_seg = (uint32_t)live->bufs.size();
        p.n_dst = 1;
        p.n_rep = 1;
        p.mode = cap::kLiveToArena;
        if (!cap::copy_params_ok(p)) return CAP_E_SIZE;
        rc = launch_status(cap::launch_copy(p, live->num_cus, static_cast<hipStream_t>(stream)));
        if (rc != CAP_OK) return rc;
        *out = own.release();
        return CAP_OK;
    });
}

int capsule_restore(cap_capsule cap, cap_set live, uint64_t prefix_digest, void* stream, uint64_t* P_restored) {
    return guarded([&]() -> int {
        if (!cap || !live) return CAP_E_INVAL;
        int rc = check_restore_target(cap, live, prefix_digest, true);
        if (rc != CAP_OK) return rc;
        rc = current_device_matches(live);
        if (rc != CAP_OK) return rc;
        cap::CopyParams p{};
        p.layout = live->dtab;
        p.tabs[0] = live->dtab;
        p.arena_in[0] = static_cast<const uint8_t*>(cap->arena);
        p.P = cap->P_aligned;
        p.nvec = cap->bytes / 16;
        p.n_seg = (uint32_t)live->bufs.size();
        p.n_dst = 1;
        p.n_rep = 1;
        p.mode = cap::kArenaToLive;
        if (!cap::copy_params_ok(p)) return CAP_E_SIZE;
        rc = launch_status(cap::launch_copy(p, live->num_cus, static_cast<hipStream_t>(stream)));
        if (rc != CAP_OK) return rc;
        live->position = cap->P_aligned;
        // re-bind the FP8 stage (nothing is converted here): in the set and
        // lineage the capsule was taken from, the stage rows below the
        // recorded end are still the dequantised capsule rows
        const bool same = cap->set_uid == live->uid && cap->epoch == live->epoch;
        new_lineage(live, same ? std::min(live->stage_end, cap->stage_end) : 0, cap->P_aligned);
        if (P_restored) *P_restored = cap->P_aligned;
        return CAP_OK;
    });
}

int capsule_fork(cap_capsule cap, const cap_set* lives, uint32_t n, uint64_t prefix_digest, void* stream) {
    return guarded([&]() -> int {
        if (!cap || !lives || n == 0) return CAP_E_INVAL;
        if (n > CAP_MAX_FORK) return CAP_E_UNSUPPORTED;
        for (uint32_t i = 0; i < n; ++i) {
            if (!lives[i]) return CAP_E_INVAL;
            for (uint32_t j = 0; j < i; ++j)
                if (lives[j] == lives[i]) return CAP_E_INVAL;
        }
        for (uint32_t i = 0; i < n; ++i) {
            const int rc = check_restore_target(cap, lives[i], prefix_digest, true);
            if (rc != CAP_OK) return rc;
            if (lives[i]->device != lives[0]->device) return CAP_E_INVAL;
        }
        if (!sets_disjoint(lives, n)) return CAP_E_INVAL;
        int rc = current_device_matches(lives[0]);
        if (rc != CAP_OK) return rc;
        // destinations per launch bounded by the kernel's LDS pointer table;
        // every launch's table is built and checked before the first launch
        const uint32_t n_seg = (uint32_t)lives[0]->bufs.size();
        const uint32_t per_launch = std::max<uint32_t>(1, std::min<uint32_t>(cap::kMaxDst, (uint32_t)cap::kMaxPtrLds / n_seg));
        std::vector<cap::CopyParams> launches;
        for (uint32_t first = 0; first < n; first += per_launch) {
            const uint32_t cnt = std::min(per_launch, n - first);
            cap::CopyParams p{};
            p.layout = lives[first]->dtab;
            for (uint32_t d = 0; d < cnt; ++d) p.tabs[d] = lives[first + d]->dtab;
            p.arena_in[0] = static_cast<const uint8_t*>(cap->arena);
            p.P = cap->P_aligned;
            p.nvec = cap->bytes / 16;
            p.n_seg = n_seg;
            p.n_dst = cnt;
            p.n_rep = 1;
            p.mode = cap::kArenaToLive;
            if (!cap::copy_params_ok(p)) return CAP_E_SIZE;
            launches.push_back(p);
        }
        for (const cap::CopyParams& p : launches) {
            rc = launch_status(cap::launch_copy(p, lives[0]->num_cus, static_cast<hipStream_t>(stream)));
            if (rc != CAP_OK) return rc;
        }
        for (uint32_t i = 0; i < n; ++i) {
            lives[i]->position = cap->P_aligned;
            new_lineage(lives[i], 0, cap->P_aligned);
        }
        return CAP_OK;
    });
}

int capsule_gather_restore(const cap_capsule* gallery, uint32_t n_gallery, const int32_t* ids,
                           const cap_set* lives, uint32_t n_env, void* stream) {
    return guarded([&]() -> int {
        if (!gallery || !ids || !lives || n_gallery == 0 || n_env == 0) return CAP_E_INVAL;
        if (n_gallery > CAP_MAX_GALLERY) return CAP_E_UNSUPPORTED;
        for (uint32_t gi = 0; gi < n_gallery; ++gi)
            if (!gallery[gi]) return CAP_E_INVAL;
        for (uint32_t e = 0; e < n_env; ++e) {
            if (!lives[e]) return CAP_E_INVAL;
            if (ids[e] < 0 || (uint32_t)ids[e] >= n_gallery) return CAP_E_INVAL;
        }
        {   // distinct environment sets
            std::vector<cap_set> v(lives, lives + n_env);
            std::sort(v.begin(), v.end());
            if (std::adjacent_find(v.begin(), v.end()) != v.end()) return CAP_E_INVAL;
        }
        const cap_capsule_s* c0 = gallery[0];
        for (uint32_t gi = 1; gi < n_gallery; ++gi) {
            const cap_capsule_s* c = gallery[gi];
            if (c->deploy_key != c0->deploy_key) return CAP_E_DIGEST;
            if (c->P_aligned != c0->P_aligned || c->bytes != c0->bytes || c->kinds != c0->kinds ||
                c->row_bytes != c0->row_bytes || c->rows != c0->rows)
                return CAP_E_SIZE;
        }
        for (uint32_t e = 0; e < n_env; ++e) {
            // every gallery arena is checked against every env set for overlap
            for (uint32_t gi = 0; gi < n_gallery; ++gi) {
                const int rc = check_restore_target(gallery[gi], lives[e], 0, false);
                if (rc != CAP_OK) return rc;
            }
            if (lives[e]->device != lives[0]->device) return CAP_E_INVAL;
        }
        // environments writing into shared bytes would race
        if (!sets_disjoint(lives, n_env)) return CAP_E_INVAL;
        int rc = current_device_matches(lives[0]);
        if (rc != CAP_OK) return rc;
        const uint32_t n_seg = (uint32_t)lives[0]->bufs.size();
        std::vector<cap::CopyParams> launches;
        for (uint32_t first = 0; first < n_env; first += cap::kMaxRep) {
            const uint32_t cnt = std::min<uint32_t>(cap::kMaxRep, n_env - first);
            cap::CopyParams p{};
            p.layout = lives[first]->dtab;
            for (uint32_t r = 0; r < cnt; ++r) {
                p.tabs[r] = lives[first + r]->dtab;
                p.arena_in[r] = static_cast<const uint8_t*>(gallery[ids[first + r]]->arena);
            }
            p.P = c0->P_aligned;
            p.nvec = c0->bytes / 16;
            p.n_seg = n_seg;
            p.n_dst = 1;
            p.n_rep = cnt;
            p.mode = cap::kArenaToLive;
            if (!cap::copy_params_ok(p)) return CAP_E_SIZE;
            launches.push_back(p);
        }
        for (const cap::CopyParams& p : launches) {
            rc = launch_status(cap::launch_copy(p, lives[0]->num_cus, static_cast<hipStream_t>(stream)));
            if (rc != CAP_OK) return rc;
        }
        for (uint32_t e = 0; e < n_env; ++e) {
            lives[e]->position = c0->P_aligned;
            new_lineage(lives[e], 0, c0->P_aligned);
        }
        return CAP_OK;
    });
}

int capsule_info(cap_capsule cap, uint64_t* P_aligned, uint64_t* bytes, uint64_t* prefix_digest,
                 uint64_t* deploy_key, const void** arena) {
    if (!cap) return CAP_E_INVAL;
    if (P_aligned) *P_aligned = cap->P_aligned;
    if (bytes) *bytes = cap->bytes;
    if (prefix_digest) *prefix_digest = cap->prefix_digest;
    if (deploy_key) *deploy_key = cap->deploy_key;
    if (arena) *arena = cap->arena;
    return CAP_OK;
}

int capsule_move(cap_capsule src, void* arena, uint64_t arena_bytes, void* stream, cap_capsule* out) {
    if (!out) return CAP_E_INVAL;
    *out = nullptr;
    return guarded([&]() -> int {
        if (!src || !arena) return CAP_E_INVAL;
        if (!aligned16((uint64_t)(uintptr_t)arena)) return CAP_E_ALIGN;
        if (arena_bytes < src->bytes) return CAP_E_SIZE;
        const uint64_t s0 = (uint64_t)(uintptr_t)src->arena, d0 = (uint64_t)(uintptr_t)arena;
        if (overlaps(s0, s0 + src->bytes, d0, d0 + src->bytes)) return CAP_E_INVAL;
        uint32_t tier = CAP_TIER_DEVICE;
        int rc = arena_tier(arena, &tier);
        if (rc != CAP_OK) return rc;
        cap_capsule_s* c = new (std::nothrow) cap_capsule_s(*src);
        if (!c) return CAP_E_NOMEM;
        std::unique_ptr<cap_capsule_s> own(c);
        c->arena = arena;
        c->arena_bytes = arena_bytes;
        c->tier = tier;
        if (src->bytes > 0 &&
            hipMemcpyAsync(arena, src->arena, src->bytes, hipMemcpyDefault, static_cast<hipStream_t>(stream)) != hipSuccess)
            return CAP_E_HIP;
        *out = own.release();
        return CAP_OK;
    });
}

int capsule_tier(cap_capsule cap, uint32_t* tier) {
    if (!cap || !tier) return CAP_E_INVAL;
    *tier = cap->tier;
    return CAP_OK;
}

int capsule_release(cap_capsule cap) {
    if (!cap) return CAP_E_INVAL;
    delete cap;
    return CAP_OK;
}

// ------------------------------------------------------------ append ----
int cap_set_append(cap_set live, const void* const* srcs, uint64_t n, void* stream) {
    return guarded([&]() -> int {
        if (!live || !srcs) return CAP_E_INVAL;
        const uint32_t nb = (uint32_t)live->bufs.size();
        std::vector<uint32_t> idx;
        for (uint32_t i = 0; i < nb; ++i) {
            if (!srcs[i]) continue;
            const BufInfo& b = live->bufs[i];
            if (!aligned16((uint64_t)(uintptr_t)srcs[i])) return CAP_E_ALIGN;
            if (n > UINT64_MAX / b.row_bytes) return CAP_E_SIZE;
            if (b.kind == CAP_KIND_POSITIONAL) {
                if (live->position > b.rows || n > b.rows - live->position) return CAP_E_SIZE;
            } else if (b.row_bytes * b.rows > cap::kAppendMaxWindow) {
                return CAP_E_UNSUPPORTED;
            }
            const uint64_t s0 = (uint64_t)(uintptr_t)srcs[i], s1 = s0 + n * b.row_bytes;
            for (const BufInfo& o : live->bufs)
                if (overlaps(s0, s1, o.ptr, o.ptr + o.row_bytes * o.rows)) return CAP_E_INVAL;
            idx.push_back(i);
        }
        int rc = current_device_matches(live);
        if (rc != CAP_OK) return rc;
        // every launch's table is built and checked before the first launch
        std::vector<cap::AppendParams> launches;
        if (n > 0) {
            for (size_t first = 0; first < idx.size(); first += cap::kAppendMaxSeg) {
                const size_t cnt = std::min<size_t>(cap::kAppendMaxSeg, idx.size() - first);
                cap::AppendParams p{};
                uint64_t blocks = 0;
                for (size_t k = 0; k < cnt; ++k) {
                    const BufInfo& b = live->bufs[idx[first + k]];
                    p.src[k] = (uint64_t)(uintptr_t)srcs[idx[first + k]];
                    p.bytes[k] = n * b.row_bytes;
                    p.first_block[k] = (uint32_t)blocks;
                    if (b.kind == CAP_KIND_POSITIONAL) {
                        p.dst[k] = b.ptr + live->position * b.row_bytes;
                        p.win[k] = 0;
                        blocks += (p.bytes[k] + cap::kAppendTile - 1) / cap::kAppendTile;
                    } else {
                        p.dst[k] = b.ptr;
                        p.win[k] = (uint32_t)(b.row_bytes * b.rows);
                        blocks += 1;
                    }
                    if (blocks > 0x7fffffffull) return CAP_E_SIZE;
                }
                p.first_block[cnt] = (uint32_t)blocks;
                p.n_seg = (uint32_t)cnt;
                launches.push_back(p);
            }
        }
        for (const cap::AppendParams& p : launches) {
            rc = launch_status(cap::launch_append(p, static_cast<hipStream_t>(stream)));
            if (rc != CAP_OK) return rc;
        }
        // rows below the high-water mark rewritten: a new lineage, and the
        // stage keeps only the rows below the append
        if (n > 0 && live->position < live->high_water)
            new_lineage(live, std::min(live->stage_end, live->position), live->high_water);
        live->position += n;
        live->high_water = live->position;
        return CAP_OK;
    });
}

// ------------------------------------------------------------ FP8 KV ----
static int fp8_convert(const kv_fp8_seg* segs, uint32_t n_seg, void* stream, bool quantize) {
    return guarded([&]() -> int {
        if (!segs || n_seg == 0) return CAP_E_INVAL;
        if (n_seg > KV_FP8_MAX_SEG) return CAP_E_UNSUPPORTED;
        const uint64_t src_es = quantize ? 2 : 1, dst_es = quantize ? 1 : 2;
        std::vector<std::pair<uint64_t, uint64_t>> dst_ranges;
        for (uint32_t i = 0; i < n_seg; ++i) {
            const kv_fp8_seg& g = segs[i];
            if (g.reserved != 0) return CAP_E_INVAL;
            if (!(g.scale > 0.0f) || !std::isfinite(g.scale)) return CAP_E_INVAL;
            if (g.n == 0) continue;
            if (!g.src || !g.dst) return CAP_E_INVAL;
            if ((g.n & 15u) != 0 || !aligned16((uint64_t)(uintptr_t)g.src) || !aligned16((uint64_t)(uintptr_t)g.dst))
                return CAP_E_ALIGN;
            if (g.n > (UINT64_MAX / 4)) return CAP_E_SIZE;
            const uint64_t s0 = (uint64_t)(uintptr_t)g.src, d0 = (uint64_t)(uintptr_t)g.dst;
            if (overlaps(s0, s0 + g.n * src_es, d0, d0 + g.n * dst_es)) return CAP_E_INVAL;
            dst_ranges.emplace_back(d0, d0 + g.n * dst_es);
        }
        std::sort(dst_ranges.begin(), dst_ranges.end());
        for (size_t i = 1; i < dst_ranges.size(); ++i)
            if (dst_ranges[i].first < dst_ranges[i - 1].second) return CAP_E_INVAL;
        cap::Fp8Params p{};
        uint64_t blocks = 0;
        for (uint32_t i = 0; i < n_seg; ++i) {
            const kv_fp8_seg& g = segs[i];
            p.src[i] = (uint64_t)(uintptr_t)g.src;
            p.dst[i] = (uint64_t)(uintptr_t)g.dst;
            p.n_groups[i] = g.n / 16;
            p.mul[i] = quantize ? 1.0f / g.scale : g.scale;
            p.first_block[i] = (uint32_t)blocks;
            blocks += (p.n_groups[i] + cap::kFp8GroupsPerBlock - 1) / cap::kFp8GroupsPerBlock;
            if (blocks > 0x7fffffffull) return CAP_E_SIZE;
        }
        p.first_block[n_seg] = (uint32_t)blocks;
        p.n_seg = n_seg;
        p.quantize = quantize ? 1 : 0;
        return launch_status(cap::launch_fp8(p, static_cast<hipStream_t>(stream)));
    });
}

int kv_fp8_quantize(const kv_fp8_seg* segs, uint32_t n_seg, void* stream) {
    return fp8_convert(segs, n_seg, stream, true);
}

int kv_fp8_dequantize(const kv_fp8_seg* segs, uint32_t n_seg, void* stream) {
    return fp8_convert(segs, n_seg, stream, false);
}

// ------------------------------------------------ FP8 working stage ----
int cap_set_bind_stage(cap_set set, uint32_t buffer, void* stage, float scale) {
    return guarded([&]() -> int {
        if (!set || !stage) return CAP_E_INVAL;
        if (buffer >= set->bufs.size()) return CAP_E_INVAL;
        if (!(scale > 0.0f) || !std::isfinite(scale)) return CAP_E_INVAL;
        const BufInfo& b = set->bufs[buffer];
        if (b.kind != CAP_KIND_POSITIONAL) return CAP_E_UNSUPPORTED;
        if (!aligned16((uint64_t)(uintptr_t)stage)) return CAP_E_ALIGN;
        const uint64_t s0 = (uint64_t)(uintptr_t)stage;
        if (b.rows * b.row_bytes > UINT64_MAX / 2) return CAP_E_SIZE;
        const uint64_t s1 = s0 + 2 * b.rows * b.row_bytes;
        for (const BufInfo& o : set->bufs)
            if (overlaps(s0, s1, o.ptr, o.ptr + o.row_bytes * o.rows)) return CAP_E_INVAL;
        bool replace = false;
        for (const StageInfo& t : set->stages) {
            if (t.buf == buffer) { replace = true; continue; }
            const BufInfo& tb = set->bufs[t.buf];
            if (overlaps(s0, s1, t.ptr, t.ptr + 2 * tb.rows * tb.row_bytes)) return CAP_E_INVAL;
        }
        if (!replace && set->stages.size() >= CAP_MAX_STAGES) return CAP_E_UNSUPPORTED;
        if (replace) {
            for (StageInfo& t : set->stages)
                if (t.buf == buffer) t = StageInfo{buffer, s0, scale};
        } else {
            set->stages.push_back(StageInfo{buffer, s0, scale});
        }
        new_lineage(set, 0, set->high_water);  // the bound stages hold nothing yet
        return CAP_OK;
    });
}

int cap_stage_acquire(cap_set set, uint64_t rows, void* stream, uint64_t* converted) {
    return guarded([&]() -> int {
        if (!set) return CAP_E_INVAL;
        if (set->stages.empty()) return CAP_E_STATE;
        if (rows > set->position) return CAP_E_SIZE;
        if (converted) *converted = 0;
        if (rows <= set->stage_end) return CAP_OK;
        int rc = current_device_matches(set);
        if (rc != CAP_OK) return rc;
        const uint64_t e0 = set->stage_end;
        std::vector<kv_fp8_seg> segs;
        for (const StageInfo& t : set->stages) {
            const BufInfo& b = set->bufs[t.buf];
            kv_fp8_seg g{};
            g.src = reinterpret_cast<const void*>(b.ptr + e0 * b.row_bytes);
            g.dst = reinterpret_cast<void*>(t.ptr + 2 * e0 * b.row_bytes);
            g.n = (rows - e0) * b.row_bytes;
            g.scale = t.scale;
            segs.push_back(g);
        }
        rc = fp8_convert(segs.data(), (uint32_t)segs.size(), stream, false);
        if (rc != CAP_OK) return rc;
        set->stage_end = rows;
        if (converted) *converted = rows - e0;
        return CAP_OK;
    });
}

int cap_stage_valid_end(cap_set set, uint64_t* end) {
    if (!set || !end) return CAP_E_INVAL;
    *end = set->stage_end;
    return CAP_OK;
}

int cap_stage_invalidate(cap_set set) {
    if (!set) return CAP_E_INVAL;
    new_lineage(set, 0, set->high_water);
    return CAP_OK;
}

int capsule_stage_end(cap_capsule cap, uint64_t* end) {
    if (!cap || !end) return CAP_E_INVAL;
    *end = cap->stage_end;
    return CAP_OK;
}

uint64_t capsule_digest_tokens(const int32_t* ids, uint64_t n) {
    uint64_t h = 0xcbf29ce484222325ULL;
    if (!ids) return h;
    for (uint64_t i = 0; i < n; ++i) {
        const uint32_t u = (uint32_t)ids[i];
        for (int byte = 0; byte < 4; ++byte) {
            h ^= (u >> (8 * byte)) & 0xFFu;
            h *= 0x100000001b3ULL;
        }
    }
    return h;
}

// ------------------------------------------------- linear-attention scan --
int linattn_chunked_prefill(const linattn_args* a, void* stream) {
    return guarded([&]() -> int {
        cap::ScanParams p{};
        const int rc = cap::validate_linattn(a, &p);
        if (rc != CAP_OK) return rc;
        if (a->T == 0 && !a->final_state) return CAP_OK;
        // every call, one token included, takes the chunked kernel, so that
        // a remainder re-prefilled after a restore reproduces what a longer
        // call computes for the same tokens
        return launch_status(cap::launch_linattn_scan(p, static_cast<hipStream_t>(stream)));
    });
}

int linattn_decode_step(const linattn_args* a, void* stream) {
    return guarded([&]() -> int {
        cap::ScanParams p{};
        const int rc = cap::validate_linattn(a, &p);
        if (rc != CAP_OK) return rc;
        if (a->T != 1) return CAP_E_UNSUPPORTED;
        // bf16 tokens take the vector-ALU step kernel; fp32 inputs the
        // chunked kernel's one-chunk instance
        if (p.in_f32) return launch_status(cap::launch_linattn_scan(p, static_cast<hipStream_t>(stream)));
        return launch_status(cap::launch_linattn_step(p, static_cast<hipStream_t>(stream)));
    });
}

// ---------------------------------------------------- delta-rule scan ----
uint64_t gdn_workspace_bytes(int64_t T, int32_t H, int32_t chunk) {
    if (T <= 0 || H < 1 || chunk != 64) return 0;
    const uint64_t n = ((uint64_t)T + 63) / 64;
    return n * (uint64_t)H * (uint64_t)cap::kGdnWsRecord;
}

int gdn_chunked_prefill(const gdn_args* a, void* stream) {
    return guarded([&]() -> int {
        cap::GdnParams p{};
        const int rc = cap::validate_gdn(a, true, &p);
        if (rc != CAP_OK) return rc;
        if (a->T == 0 && !a->final_state) return CAP_OK;
        // every call, one token included, takes the chunked path (see
        // linattn_chunked_prefill)
        return launch_status(cap::launch_gdn(p, static_cast<hipStream_t>(stream)));
    });
}

int gdn_decode_step(const gdn_args* a, void* stream) {
    return guarded([&]() -> int {
        cap::GdnParams p{};
        const int rc = cap::validate_gdn(a, false, &p);
        if (rc != CAP_OK) return rc;
        if (a->T != 1) return CAP_E_UNSUPPORTED;
        return launch_status(cap::launch_gdn_step(p, static_cast<hipStream_t>(stream)));
    });
}

}  // extern "C"

// ------------------------------------------------- argument validation ----
namespace cap {

int validate_linattn(const linattn_args* a, ScanParams* out) {
    if (!a) return CAP_E_INVAL;
    if (a->T < 0 || a->H < 1 || a->dk < 1 || a->dv < 1 || a->chunk < 1) return CAP_E_INVAL;
    if (a->in_dtype != CAP_DTYPE_BF16 && a->in_dtype != CAP_DTYPE_F32) return CAP_E_INVAL;
    if (a->chunk != 64 || (a->dk != 64 && a->dk != 128) || (a->dv % 16) != 0) return CAP_E_UNSUPPORTED;
    if (a->in_dtype == CAP_DTYPE_F32 && a->dk != 64) return CAP_E_UNSUPPORTED;
    if ((int64_t)a->H * (a->dv / 16) > 0x7fffffff) return CAP_E_UNSUPPORTED;
    // the kernels address one chunk of rows, and one state of all heads, with
    // 32-bit byte offsets, and count chunks in 32 bits
    {
        const uint64_t H = (uint64_t)a->H, dk = (uint64_t)a->dk, dv = (uint64_t)a->dv;
        if (64 * H * (dk > dv ? dk : dv) * 4 > 0x7fffffffull || H * dk * dv * 4 > 0x7fffffffull)
            return CAP_E_UNSUPPORTED;
    }
    if (a->T > ((int64_t)1 << 36)) return CAP_E_UNSUPPORTED;
    if (a->T > 0 && (!a->q || !a->k || !a->v || !a->g || !a->o)) return CAP_E_INVAL;
    const uint64_t ptrs[] = {(uint64_t)(uintptr_t)a->q, (uint64_t)(uintptr_t)a->k, (uint64_t)(uintptr_t)a->v,
                             (uint64_t)(uintptr_t)a->g, (uint64_t)(uintptr_t)a->state_in,
                             (uint64_t)(uintptr_t)a->o, (uint64_t)(uintptr_t)a->chunk_states,
                             (uint64_t)(uintptr_t)a->final_state};
    for (uint64_t p : ptrs)
        if (!aligned16(p)) return CAP_E_ALIGN;
    // outputs must not overlap inputs (final_state may alias state_in)
    const uint64_t T = (uint64_t)a->T, H = (uint64_t)a->H, dk = (uint64_t)a->dk, dv = (uint64_t)a->dv;
    const uint64_t es = a->in_dtype == CAP_DTYPE_F32 ? 4 : 2;
    const uint64_t nck = (T + 63) / 64;
    struct R { uint64_t p, n; };
    const R in[] = {{ptrs[0], T * H * dk * es}, {ptrs[1], T * H * dk * es}, {ptrs[2], T * H * dv * es},
                    {ptrs[3], T * H * 4}, {ptrs[4], H * dk * dv * 4}};
    const R outr[] = {{ptrs[5], T * H * dv * 4}, {ptrs[6], nck * H * dk * dv * 4}, {ptrs[7], H * dk * dv * 4}};
    for (int i = 0; i < 3; ++i) {
        if (!outr[i].p || !outr[i].n) continue;
        for (int j = 0; j < 5; ++j) {
            if (!in[j].p || !in[j].n) continue;
            if (i == 2 && j == 4 && outr[i].p == in[j].p) continue;  // in-place state update
            if (overlaps(outr[i].p, outr[i].p + outr[i].n, in[j].p, in[j].p + in[j].n)) return CAP_E_INVAL;
        }
        for (int j = 0; j < i; ++j) {
            if (!outr[j].p || !outr[j].n) continue;
            if (overlaps(outr[i].p, outr[i].p + outr[i].n, outr[j].p, outr[j].p + outr[j].n)) return CAP_E_INVAL;
        }
    }
    ScanParams& p = *out;
    p.q = a->q; p.k = a->k; p.v = a->v; p.g = a->g;
    p.state_in = a->state_in; p.o = a->o; p.chunk_states = a->chunk_states; p.final_state = a->final_state;
    p.T = a->T; p.H = a->H; p.dk = a->dk; p.dv = a->dv;
    p.in_f32 = a->in_dtype == CAP_DTYPE_F32 ? 1 : 0;
    p.scale = a->scale;
    return CAP_OK;
}

int validate_gdn(const gdn_args* a, bool need_ws, GdnParams* out) {
    if (!a) return CAP_E_INVAL;
    if (a->T < 0 || a->H < 1 || a->dk < 1 || a->dv < 1 || a->chunk < 1) return CAP_E_INVAL;
    if (a->in_dtype != CAP_DTYPE_BF16 && a->in_dtype != CAP_DTYPE_F32) return CAP_E_INVAL;
    if (a->in_dtype != CAP_DTYPE_BF16) return CAP_E_UNSUPPORTED;
    if (a->chunk != 64 || (a->dk != 64 && a->dk != 128) || (a->dv % 16) != 0) return CAP_E_UNSUPPORTED;
    // 32-bit offsets inside one chunk of q / k / v / o rows and inside one
    // state of all heads, and grid sizes
    const uint64_t T = (uint64_t)a->T, H = (uint64_t)a->H, dk = (uint64_t)a->dk, dv = (uint64_t)a->dv;
    const uint64_t nck = (T + 63) / 64;
    if (64 * H * (dk > dv ? dk : dv) * 4 > 0x7fffffffull || H * dk * dv * 4 > 0x7fffffffull)
        return CAP_E_UNSUPPORTED;
    if (H * (dv / 16) > 0x7fffffffull || nck * H > 0x7fffffffull) return CAP_E_UNSUPPORTED;
    if (a->T > 0 && (!a->q || !a->k || !a->v || !a->g || !a->beta || !a->o)) return CAP_E_INVAL;
    const uint64_t ws_need = need_ws ? gdn_workspace_bytes(a->T, a->H, a->chunk) : 0;
    if (need_ws && a->T > 0 && !a->workspace) return CAP_E_INVAL;
    if (need_ws && a->T > 0 && a->workspace_bytes < ws_need) return CAP_E_SIZE;
    const uint64_t ws_ptr = need_ws ? (uint64_t)(uintptr_t)a->workspace : 0;
    const uint64_t ptrs[] = {(uint64_t)(uintptr_t)a->q, (uint64_t)(uintptr_t)a->k, (uint64_t)(uintptr_t)a->v,
                             (uint64_t)(uintptr_t)a->g, (uint64_t)(uintptr_t)a->beta,
                             (uint64_t)(uintptr_t)a->state_in, (uint64_t)(uintptr_t)a->o,
                             (uint64_t)(uintptr_t)a->chunk_states, (uint64_t)(uintptr_t)a->final_state, ws_ptr};
    for (uint64_t p : ptrs)
        if (!aligned16(p)) return CAP_E_ALIGN;
    // outputs (and the workspace) must not overlap the inputs or each other;
    // final_state may alias state_in
    struct R { uint64_t p, n; };
    const R in[] = {{ptrs[0], T * H * dk * 2}, {ptrs[1], T * H * dk * 2}, {ptrs[2], T * H * dv * 2},
                    {ptrs[3], T * H * 4}, {ptrs[4], T * H * 4}, {ptrs[5], H * dk * dv * 4}};
    const R outr[] = {{ptrs[6], T * H * dv * 4}, {ptrs[7], nck * H * dk * dv * 4}, {ptrs[8], H * dk * dv * 4},
                      {ptrs[9], T > 0 ? ws_need : 0}};
    constexpr int NIN = sizeof(in) / sizeof(in[0]), NOUT = sizeof(outr) / sizeof(outr[0]);
    for (int i = 0; i < NOUT; ++i) {
        if (!outr[i].p || !outr[i].n) continue;
        for (int j = 0; j < NIN; ++j) {
            if (!in[j].p || !in[j].n) continue;
            if (i == 2 && j == 5 && outr[i].p == in[j].p) continue;  // in-place state update
            if (overlaps(outr[i].p, outr[i].p + outr[i].n, in[j].p, in[j].p + in[j].n)) return CAP_E_INVAL;
        }
        for (int j = 0; j < i; ++j) {
            if (!outr[j].p || !outr[j].n) continue;
            if (overlaps(outr[i].p, outr[i].p + outr[i].n, outr[j].p, outr[j].p + outr[j].n)) return CAP_E_INVAL;
        }
    }
    GdnParams& p = *out;
    p.q = a->q; p.k = a->k; p.v = a->v; p.g = a->g; p.beta = a->beta;
    p.state_in = a->state_in; p.o = a->o; p.chunk_states = a->chunk_states; p.final_state = a->final_state;
    p.ws = need_ws ? static_cast<uint8_t*>(a->workspace) : nullptr;
    p.T = a->T; p.H = a->H; p.dk = a->dk; p.dv = a->dv;
    p.scale = a->scale;
    return CAP_OK;
}

}  // namespace cap
