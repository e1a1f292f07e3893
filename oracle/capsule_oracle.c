/*
 * Capsule oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * Plain host memcpy semantics of the capsule verbs over host copies of the
 * live buffer set.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load it; it shares nothing with the device path.
 *
 * Paper: "Execution-State Capsules", §3 Algorithm 1 and the "Four verbs"
 * paragraph:
 *   snapshot(P): P' = floor(P / C) * C; the capsule bytes are a copy of the
 *                live buffer set as it is valid at P'.
 *   restore:     copy those bytes back into the live buffers (and rebind the
 *                boundary, i.e. the current position becomes P').
 *   fork(n):     n sessions, each a restore of the same capsule.
 *   rollback:    a restore of an earlier capsule of the same session.
 * §3 "Definition": the KV region is positional and valid over [0, P); the
 * recurrent / convolution state is fixed-size.
 *
 * Capsule byte format (the format both sides write independently): the
 * buffers of the set, in set order, concatenated; a positional buffer
 * contributes its first P' rows (rows are position-major), a fixed buffer
 * contributes all of its bytes.
 *
 * Token-prefix digest: the paper names a token-prefix digest in the boundary
 * descriptor (§3 Algorithm 1) without fixing the function; this oracle uses
 * 64-bit FNV-1a over the little-endian bytes of the int32 token ids.
 *
 * Parity status: pinned (published FNV-1a test vectors, the paper's capsule
 * size table slope, byte round trips, the alignment properties).
 */
#include <stdint.h>
#include <string.h>

enum { ORC_KIND_POSITIONAL = 0, ORC_KIND_FIXED = 1 };

/* Algorithm 1: chunk-align the boundary. */
uint64_t orc_align(uint64_t P, uint64_t C)
{
    return C ? (P / C) * C : 0;
}

static uint64_t buf_bytes(uint64_t row_bytes, uint64_t rows_total, uint32_t kind, uint64_t P_aligned)
{
    return kind == ORC_KIND_POSITIONAL ? P_aligned * row_bytes : row_bytes * rows_total;
}

/* Bytes of the capsule of this buffer set at the aligned boundary P'. */
uint64_t orc_capsule_bytes(uint32_t n, const uint64_t* row_bytes, const uint64_t* rows_total,
                           const uint32_t* kinds, uint64_t P_aligned)
{
    uint64_t total = 0;
    for (uint32_t i = 0; i < n; ++i)
        total += buf_bytes(row_bytes[i], rows_total[i], kinds[i], P_aligned);
    return total;
}

/* snapshot: live buffers -> arena, in set order. */
void orc_capsule_snapshot(uint32_t n, void* const* bufs, const uint64_t* row_bytes,
                          const uint64_t* rows_total, const uint32_t* kinds,
                          uint64_t P_aligned, void* arena)
{
    unsigned char* dst = (unsigned char*)arena;
    for (uint32_t i = 0; i < n; ++i) {
        const uint64_t nb = buf_bytes(row_bytes[i], rows_total[i], kinds[i], P_aligned);
        memcpy(dst, bufs[i], (size_t)nb);
        dst += nb;
    }
}

/* restore: arena -> live buffers, in set order. */
void orc_capsule_restore(uint32_t n, void* const* bufs, const uint64_t* row_bytes,
                         const uint64_t* rows_total, const uint32_t* kinds,
                         uint64_t P_aligned, const void* arena)
{
    const unsigned char* src = (const unsigned char*)arena;
    for (uint32_t i = 0; i < n; ++i) {
        const uint64_t nb = buf_bytes(row_bytes[i], rows_total[i], kinds[i], P_aligned);
        memcpy(bufs[i], src, (size_t)nb);
        src += nb;
    }
}

/* fork 1 -> n_sets: every destination set receives a restore of the same
   capsule.  sets is [n_sets][n] buffer pointers. */
void orc_capsule_fork(uint32_t n, uint32_t n_sets, void* const* sets, const uint64_t* row_bytes,
                      const uint64_t* rows_total, const uint32_t* kinds,
                      uint64_t P_aligned, const void* arena)
{
    for (uint32_t s = 0; s < n_sets; ++s)
        orc_capsule_restore(n, sets + (uint64_t)s * n, row_bytes, rows_total, kinds, P_aligned, arena);
}

/* gather-restore: environment e receives a restore of gallery[ids[e]].
   sets is [n_env][n] buffer pointers; gallery is [n_gallery] arenas.
   Returns 0, or -1 if an id is out of range (nothing is copied then). */
int orc_capsule_gather(uint32_t n, uint32_t n_env, void* const* sets, const uint64_t* row_bytes,
                       const uint64_t* rows_total, const uint32_t* kinds, uint64_t P_aligned,
                       uint32_t n_gallery, const void* const* gallery, const int32_t* ids)
{
    for (uint32_t e = 0; e < n_env; ++e)
        if (ids[e] < 0 || (uint32_t)ids[e] >= n_gallery) return -1;
    for (uint32_t e = 0; e < n_env; ++e)
        orc_capsule_restore(n, sets + (uint64_t)e * n, row_bytes, rows_total, kinds, P_aligned,
                            gallery[ids[e]]);
    return 0;
}

/* append of n tokens at `position` (§3 Algorithm 1 restore: after the copy
   the suffix is appended; §3 "Definition": the KV region is positional, the
   convolution state is a fixed-size window of the latest inputs).  For every
   buffer i with a source (srcs[i] != NULL, n rows of row_bytes[i] bytes):
     positional: rows [position, position + n) <- the n source rows
                 (-1 and nothing copied if position + n > rows_total[i]);
     fixed:      the buffer is a window of its rows_total rows holding the
                 latest rows of a history; it becomes the last rows_total rows
                 of (its current rows followed by the n source rows).
   Buffers without a source are untouched.  Returns 0 on success. */
int orc_set_append(uint32_t n_buf, void* const* bufs, const void* const* srcs, const uint64_t* row_bytes,
                   const uint64_t* rows_total, const uint32_t* kinds, uint64_t position, uint64_t n,
                   unsigned char* scratch)
{
    for (uint32_t i = 0; i < n_buf; ++i)
        if (srcs[i] && kinds[i] == ORC_KIND_POSITIONAL && position + n > rows_total[i]) return -1;
    for (uint32_t i = 0; i < n_buf; ++i) {
        if (!srcs[i] || n == 0) continue;
        const uint64_t rb = row_bytes[i];
        unsigned char* dst = (unsigned char*)bufs[i];
        if (kinds[i] == ORC_KIND_POSITIONAL) {
            memcpy(dst + position * rb, srcs[i], (size_t)(n * rb));
        } else {
            /* history = current window rows, then the new rows; keep its tail */
            const uint64_t W = rows_total[i];
            memcpy(scratch, dst, (size_t)(W * rb));
            memcpy(scratch + W * rb, srcs[i], (size_t)(n * rb));
            memcpy(dst, scratch + n * rb, (size_t)(W * rb));
        }
    }
    return 0;
}

/* 64-bit FNV-1a (offset basis 14695981039346656037, prime 1099511628211)
   over the little-endian bytes of n int32 token ids. */
uint64_t orc_digest_tokens(const int32_t* ids, uint64_t n)
{
    uint64_t h = 14695981039346656037ULL;
    for (uint64_t i = 0; i < n; ++i) {
        const uint32_t u = (uint32_t)ids[i];
        for (int b = 0; b < 4; ++b) {
            h ^= (u >> (8 * b)) & 0xFFu;
            h *= 1099511628211ULL;
        }
    }
    return h;
}

/* The same hash over raw bytes (used to pin the function against the
   published FNV-1a test vectors, which are defined over byte strings). */
uint64_t orc_digest_bytes(const unsigned char* p, uint64_t n)
{
    uint64_t h = 14695981039346656037ULL;
    for (uint64_t i = 0; i < n; ++i) {
        h ^= p[i];
        h *= 1099511628211ULL;
    }
    return h;
}
