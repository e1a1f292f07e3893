/*
 * capsule.h -- execution-state capsules and the chunked gated linear-attention
 * prefill scan, for one AMD Instinct MI355X (gfx950).  Plain C ABI.
 *
 * Source: "Execution-State Capsules: Graph-Bound Execution-State Checkpoint
 * and Restore for Low-Latency, Small-Batch, On-Device Physical-AI Serving".
 *
 *   - A capsule freezes a committed boundary P of a closed, named set of live
 *     device buffers (§3 "Definition"): positional full-attention KV valid
 *     over [0, P), plus fixed-size state (linear-attention recurrent state,
 *     convolution tails, other boundary state).
 *   - snapshot / restore / fork / rollback are byte copies of that set
 *     (§3 Algorithm 1 and "Four verbs"); snapshot chunk-aligns the boundary
 *     to P' = floor(P / C) * C (§3 Algorithm 1; §5 "chunk-alignment
 *     condition"); restore asserts the deployment digest first (§3
 *     Algorithm 1) and rebinds the boundary.
 *   - The robot episode reset is the same restore verb (§6); the batched form
 *     here restores a per-environment capsule chosen from a gallery.
 *   - The chunked scan is the recompute a capsule replaces (§3 Table "cost
 *     structure", §3 "Cost model"); it folds its recurrent state once per
 *     chunk (§5), which is what makes restore-at-P' followed by a prefill of
 *     the remainder reproduce a cold prefill exactly.
 *
 * Conventions (§4: buffers are the only state primitive, the framework owns
 * lifetime and pointers, copies are stream-ordered, errors are int returns;
 * the contract is mechanism, never policy):
 *   - Every device pointer is caller-owned (e.g. torch tensors).  The library
 *     owns only host headers and the small static device segment table that
 *     cap_set_create builds once per set.  No call below allocates device
 *     memory except cap_set_create.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Device work is
 *     asynchronous and stream-ordered; buffers and arenas must stay alive
 *     until the stream has passed the call.
 *   - Every function returns CAP_OK (0) or a negative CAP_E_* status.  All
 *     argument checks run on the host first, and a call that needs several
 *     launches builds and checks every launch's table before it enqueues the
 *     first: on any error other than CAP_E_HIP nothing has been enqueued and
 *     no device byte has been written.  CAP_E_HIP reports a launch the HIP
 *     runtime refused; in a multi-launch call (a fork into many sets, a
 *     gather of more than 64 environments, an append to more than 128
 *     buffers) the launches before it stay enqueued.
 *   - The library reads launch status from the launch calls themselves and
 *     never clears an error the caller left pending (the runtime's "last
 *     error"); it clears only the error its own pointer-attribute query
 *     raises for an unknown arena, and only when none was pending before.
 *   - Not thread-safe for concurrent calls on the same set or capsule.
 */
#ifndef CAPSULE_H
#define CAPSULE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define CAP_API __attribute__((visibility("default")))
#else
#define CAP_API
#endif

/* ------------------------------------------------------------ status ---- */
#define CAP_OK              0
#define CAP_E_INVAL        (-1)  /* null pointer, bad count/enum, overlapping buffers  */
#define CAP_E_SIZE         (-2)  /* arena too small, layout mismatch, P beyond capacity */
#define CAP_E_DIGEST       (-3)  /* prefix digest or deployment key mismatch           */
#define CAP_E_UNSUPPORTED  (-4)  /* unknown buffer kind, unsupported shape or dtype    */
#define CAP_E_ALIGN        (-5)  /* pointer or size not a multiple of 16 bytes         */
#define CAP_E_STATE        (-6)  /* set position is not the aligned boundary, or the
                                     capsule is not device-resident                   */
#define CAP_E_HIP          (-7)  /* HIP runtime error (no device, allocation, launch)  */
#define CAP_E_NOMEM        (-8)  /* host memory allocation failed                     */

/* Static message for a status code (never NULL). */
CAP_API const char* cap_status_string(int status);

/* ----------------------------------------------------- buffer kinds ---- */
/* CAP_KIND_POSITIONAL: a position-major buffer of `rows` rows of `row_bytes`
 *   bytes (full-attention K or V, [T_max, kv_heads, d]); valid rows are the
 *   prefix [0, P'), one contiguous byte range (§3 "Definition": the KV region
 *   is valid over [0, P)).
 * CAP_KIND_FIXED: a fixed-size buffer copied whole, row_bytes * rows bytes
 *   (recurrent state, convolution tail, any other boundary state). */
#define CAP_KIND_POSITIONAL 0u
#define CAP_KIND_FIXED      1u

#define CAP_DTYPE_F32  0
#define CAP_DTYPE_BF16 1

/* Capsule tiers (§3 Algorithm 1: snapshot returns a tiered handle; §4: the
 * contract's one cross-space mechanism is host-backed buffers plus an
 * asynchronous copy, so a capsule can be parked off the GPU). */
#define CAP_TIER_DEVICE 0u  /* arena in the current device's memory              */
#define CAP_TIER_HOST   1u  /* arena in page-locked host memory the device maps   */

/* One named live buffer.  dptr: device pointer, 16-byte aligned, owned by the
 * caller.  row_bytes: multiple of 16, > 0.  rows: > 0.  reserved: 0. */
typedef struct cap_buf {
    const char* name;      /* label (copied; may be NULL) */
    void*       dptr;
    uint64_t    row_bytes;
    uint64_t    rows;
    uint32_t    kind;      /* CAP_KIND_* */
    uint32_t    reserved;
} cap_buf;

/* Limits of one call (host-checked; CAP_E_UNSUPPORTED beyond them). */
#define CAP_MAX_BUFFERS 512u  /* buffers per set                   */
#define CAP_MAX_FORK    16u   /* destination sets of one fork      */
#define CAP_MAX_GALLERY 64u   /* capsules in one gather gallery    */

typedef struct cap_set_s*     cap_set;      /* closed named live set           */
typedef struct cap_capsule_s* cap_capsule;  /* host header of one capsule      */

/* P' = floor(P / chunk) * chunk (§3 Algorithm 1); 0 when chunk == 0. */
CAP_API uint64_t cap_align_boundary(uint64_t P, uint32_t chunk);

/* Capsule bytes of a buffer list at boundary P (pure host; no device):
 * sum over positional buffers of P' * row_bytes plus the bytes of every fixed
 * buffer.  Same checks as cap_set_create except that dptr may be NULL. */
CAP_API int capsule_layout_bytes(const cap_buf* bufs, uint32_t n, uint32_t chunk,
                                 uint64_t P, uint64_t* bytes);

/* Create a live set over n caller-owned buffers (the closed named buffer set
 * B of §3 Algorithm 1), with chunk size `chunk` (>= 1) and a caller-chosen
 * deployment key (a digest of weights, quantisation, kernels and shape
 * bucket; restore refuses a capsule taken under another key, §3 Algorithm 1).
 * Checks: names unique when given, kinds known, pointers and row_bytes
 * 16-byte aligned, buffers pairwise disjoint, every buffer's address range
 * and the sum of all buffer sizes within 64 bits (CAP_E_SIZE otherwise).  Builds the static device
 * segment table on the current device (one hipMalloc).  The set's position
 * starts at 0.  *out receives the handle. */
CAP_API int cap_set_create(const cap_buf* bufs, uint32_t n, uint32_t chunk,
                           uint64_t deploy_key, cap_set* out);
CAP_API int cap_set_destroy(cap_set set);

/* Declare the boundary the live set currently holds: fixed buffers hold the
 * state after `position` tokens and positional buffers are valid over
 * [0, position).  Must not exceed the capacity (rows) of any positional
 * buffer (CAP_E_SIZE). */
CAP_API int cap_set_set_position(cap_set set, uint64_t position);
CAP_API int cap_set_get_position(cap_set set, uint64_t* position);

/* Append a suffix of n tokens (§3 Algorithm 1 restore: "append suffix";
 * §3 "Definition": positional KV region, fixed-size convolution window).
 * srcs is a HOST array with one entry per buffer of the set, in set order:
 * NULL leaves the buffer alone (e.g. a recurrent state, which the scan
 * updates); otherwise a device pointer (16-byte aligned, disjoint from every
 * live buffer) to n rows of that buffer's row_bytes:
 *   positional buffer: rows [position, position + n) receive the n rows
 *     (CAP_E_SIZE if position + n exceeds its rows);
 *   fixed buffer: treated as a window of its `rows` rows holding the latest
 *     rows of a history (a convolution tail [W, C] declared with row_bytes =
 *     C * element size and rows = W); it becomes the last W rows of (its
 *     rows, then the n new rows); at most 64 KiB per window
 *     (CAP_E_UNSUPPORTED).
 * One stream-ordered launch per 128 touched buffers; then the set's position
 * advances by n.  The kernel arguments carry every address, so the call can
 * be recorded in a stream capture (a HIP graph) and replayed. */
CAP_API int cap_set_append(cap_set live, const void* const* srcs, uint64_t n, void* stream);

/* Capsule bytes of this set at boundary P (P is aligned first). */
CAP_API int capsule_bytes(cap_set set, uint64_t P, uint64_t* bytes);

/* snapshot(P) (§3 Algorithm 1): P' = floor(P / C) * C; the set's position
 * must equal P' (CAP_E_STATE otherwise -- the fixed buffers must hold the
 * state at P', e.g. from a prefill that stopped at P' or from the scan's
 * chunk-boundary state output); P' must fit every positional buffer
 * (CAP_E_SIZE).  Copies the set, valid at P', into `arena` (caller-owned,
 * 16-byte aligned, >= capsule_bytes, disjoint from every live buffer) in one
 * launch: buffers in set order, positional buffers contributing rows
 * [0, P'), fixed buffers all their bytes.  The arena is memory of the
 * current device (a device-tier capsule) or page-locked host memory from
 * hipHostMalloc (a host-tier capsule, written across the host link); any
 * other pointer is CAP_E_INVAL.  *out receives a host header {P',
 * prefix_digest, deploy key, layout, tier}; the arena stays the caller's and
 * must outlive the header's use. */
CAP_API int capsule_snapshot(cap_set live, uint64_t P, uint64_t prefix_digest,
                             void* arena, uint64_t arena_bytes, void* stream,
                             cap_capsule* out);

/* restore (§3 Algorithm 1; rollback is a restore of an earlier capsule):
 * checks, in order, the prefix digest and the set's deployment key
 * (CAP_E_DIGEST), that the capsule is device-resident (CAP_E_STATE: a
 * host-tier capsule is promoted first, with capsule_move), then that the
 * set's layout equals the capsule's (CAP_E_SIZE); then copies the arena back
 * into the live buffers in one
 * launch and rebinds the boundary: the set's position becomes P' (returned
 * in *P_restored, which may be NULL).  Positional rows at or beyond P' are
 * not written. */
CAP_API int capsule_restore(cap_capsule cap, cap_set live, uint64_t prefix_digest,
                            void* stream, uint64_t* P_restored);

/* fork 1 -> n (§3 "Four verbs", Algorithm 1 fork): restore one capsule into n
 * distinct live sets (1 <= n <= CAP_MAX_FORK) in one launch that reads each
 * capsule byte once and writes it n times.  Same checks as restore, for every
 * set; every set's position becomes P'. */
CAP_API int capsule_fork(cap_capsule cap, const cap_set* lives, uint32_t n,
                         uint64_t prefix_digest, void* stream);

/* Batched episode reset (§6: reset is a restore of a boundary capsule):
 * environment e in [0, n_env) receives a restore of gallery[ids[e]].  ids is
 * a HOST array of n_env int32 in [0, n_gallery) (CAP_E_INVAL otherwise).
 * All gallery capsules and all environment sets must share one layout and
 * one P' and deployment key (CAP_E_SIZE / CAP_E_DIGEST); the env sets must be
 * distinct.  One launch per call for any n_env; every env set's position
 * becomes P'. */
CAP_API int capsule_gather_restore(const cap_capsule* gallery, uint32_t n_gallery,
                                   const int32_t* ids, const cap_set* lives,
                                   uint32_t n_env, void* stream);

/* Header fields of a capsule (any output pointer may be NULL). */
CAP_API int capsule_info(cap_capsule cap, uint64_t* P_aligned, uint64_t* bytes,
                         uint64_t* prefix_digest, uint64_t* deploy_key,
                         const void** arena);

/* Promotion / demotion (§3 Algorithm 1: "if not GPU-resident, promote";
 * §4: host-backed buffers plus cross-space asynchronous copy).  Copies the
 * capsule's bytes into `arena` (current-device memory or page-locked host
 * memory; 16-byte aligned; >= the capsule's bytes, CAP_E_SIZE otherwise;
 * disjoint from the source arena) with one stream-ordered copy, and returns
 * in *out a new header over `arena` with the same descriptor and the new
 * tier.  Device -> host demotes, host -> device promotes; the source header
 * and arena stay valid.  The caller owns both arenas; the library allocates
 * nothing. */
CAP_API int capsule_move(cap_capsule src, void* arena, uint64_t arena_bytes,
                         void* stream, cap_capsule* out);

/* Tier of a capsule's arena: CAP_TIER_DEVICE or CAP_TIER_HOST. */
CAP_API int capsule_tier(cap_capsule cap, uint32_t* tier);

/* Free the host header (the arena remains the caller's). */
CAP_API int capsule_release(cap_capsule cap);

/* Token-prefix digest for the boundary descriptor (§3 Algorithm 1 names one
 * without fixing the function): 64-bit FNV-1a over the little-endian bytes
 * of n int32 token ids (host). */
CAP_API uint64_t capsule_digest_tokens(const int32_t* ids, uint64_t n);

/* ------------------------------------- chunked linear-attention prefill -- */
/* Gated linear attention, per head h (state dk x dv, §2 "hybrid recurrent
 * state": a fold over the whole prefix):
 *     S_t = exp(g_t) * S_{t-1} + k_t^T v_t,      o_t = scale * q_t S_t
 * computed in chunks of C tokens counted from the first token of the call
 * (§5: the state is folded once per chunk).  For chunk j with entering state
 * S_j and inclusive in-chunk log-decay sums G_i:
 *     o_i     = scale * (exp(G_i) q_i S_j + sum_{m<=i} exp(G_i - G_m) (q_i.k_m) v_m)
 *     S_{j+1} = exp(G_last) S_j + sum_m exp(G_last - G_m) k_m^T v_m
 * The arithmetic of a chunk depends only on (S_j, that chunk's inputs): a
 * call started at a chunk-aligned position from a restored state reproduces,
 * bit for bit, what one longer call computes for the same tokens.  This
 * holds for every T >= 1, so a remainder of one token re-prefilled after a
 * restore equals the cold prefill's last chunk bit for bit.
 *
 * Layouts (all contiguous, device, caller-owned):
 *   q, k : [T, H, dk]  in_dtype (bf16 or f32)      v : [T, H, dv] in_dtype
 *   g    : [T, H] fp32 log-gates, finite (normally <= 0)
 *   state_in     : [H, dk, dv] fp32, or NULL for a zero state
 *   o            : [T, H, dv] fp32 (written for every token)
 *   chunk_states : [ceil(T/C), H, dk, dv] fp32 or NULL; entry j is the state
 *                  ENTERING chunk j (entry 0 = state_in)
 *   final_state  : [H, dk, dv] fp32 or NULL; the state after the last token.
 *                  May be the same pointer as state_in (in-place update).
 * Supported: chunk == 64, dk in {64, 128} (fp32 inputs: dk == 64), dv a
 * multiple of 16, 1 <= H, H dk dv 4 < 2^31 and 64 H max(dk, dv) 4 < 2^31
 * (32-bit offsets inside one state and one chunk),
 * 0 <= T <= 2^36; pointers 16-byte aligned; o / chunk_states / final_state must not
 * overlap the inputs (except final_state == state_in).
 * Errors: CAP_E_INVAL (null required pointer, T < 0, H < 1, bad dtype,
 * overlap), CAP_E_UNSUPPORTED (shape outside the list), CAP_E_ALIGN. */
typedef struct linattn_args {
    const void*  q;
    const void*  k;
    const void*  v;
    const float* g;
    const float* state_in;
    float*       o;
    float*       chunk_states;
    float*       final_state;
    int64_t      T;
    int32_t      H;
    int32_t      dk;
    int32_t      dv;
    int32_t      chunk;
    int32_t      in_dtype;   /* CAP_DTYPE_BF16 or CAP_DTYPE_F32 */
    float        scale;
} linattn_args;

CAP_API int linattn_chunked_prefill(const linattn_args* args, void* stream);

/* One decode step (§3 Algorithm 1: after restore the session appends and
 * decodes token by token): the recurrence above for exactly one token
 * (args->T == 1, CAP_E_UNSUPPORTED otherwise), with the same arguments,
 * layouts and checks as linattn_chunked_prefill.  bf16 tokens take a short
 * vector-ALU path: its state is bit-identical to the chunked fold of a
 * one-token chunk (the product of two bf16 values is exact in fp32 and the
 * fold is one fma with exp(g)); its o takes another summation order, so it
 * may differ from a one-token prefill's o in fp32 rounding.  fp32 inputs
 * take the chunked path.  Decode steps are reproducible among themselves:
 * a session restored at P' and decoded equals a cold session decoded from
 * the same state, bit for bit. */
CAP_API int linattn_decode_step(const linattn_args* args, void* stream);

/* -------------------------------------- chunked gated delta-rule prefill -- */
/* Gated DeltaNet state of the paper's hybrid model (§2 "hybrid recurrent
 * state", §7 model description; the paper does not write the recurrence,
 * the standard gated delta rule is taken), per head h with state dk x dv:
 *     S_t = exp(g_t) (I - beta_t k_t^T k_t) S_{t-1} + beta_t k_t^T v_t
 *     o_t = scale * q_t S_t
 * computed in chunks of C tokens counted from the first token of the call.
 * For a chunk with entering state S and inclusive in-chunk log-decay sums
 * G_t (gamma_t = exp(G_t)) the pseudo-values U solve
 *     (I + A) U = diag(beta) (V - diag(gamma) K S),
 *     A_tm = beta_t exp(G_t - G_m) (k_t . k_m)  for m < t,
 * and o_t = scale (gamma_t q_t S + sum_{m<=t} exp(G_t - G_m)(q_t . k_m) u_m),
 * S_new = gamma_last S + sum_m exp(G_last - G_m) k_m^T u_m.  As for the
 * linear-attention scan, a chunk's arithmetic depends only on (S, that
 * chunk's inputs): restore at an aligned position then continue equals one
 * longer call bit for bit, for every T >= 1 (a one-token call takes the
 * chunked path too).
 *
 * Layouts (contiguous, device, caller-owned):
 *   q, k : [T, H, dk] bf16     v : [T, H, dv] bf16
 *   g    : [T, H] fp32 log-gates, finite (normally <= 0)
 *   beta : [T, H] fp32 write strengths (normally in [0, 1])
 *   state_in, chunk_states, final_state, o : as in linattn_args
 *   workspace : gdn_workspace_bytes(T, H, C) bytes of device scratch, 16-byte
 *               aligned; holds the per-chunk inverses (I + A)^-1 and gate
 *               tables during the call (contents undefined afterwards).  May
 *               be NULL when T = 0.
 * Supported: chunk == 64, dk in {64, 128}, dv a multiple of 16, bf16 inputs,
 * H dk dv 4 < 2^31 and 64 H max(dk, dv) 4 < 2^31 (32-bit offsets inside one
 * state and one chunk).
 * Errors: CAP_E_INVAL (null required pointer, T < 0, H < 1, bad dtype,
 * overlapping buffers), CAP_E_SIZE (workspace_bytes too small),
 * CAP_E_UNSUPPORTED (shape outside the list), CAP_E_ALIGN. */
typedef struct gdn_args {
    const void*  q;
    const void*  k;
    const void*  v;
    const float* g;
    const float* beta;
    const float* state_in;
    float*       o;
    float*       chunk_states;
    float*       final_state;
    void*        workspace;
    uint64_t     workspace_bytes;
    int64_t      T;
    int32_t      H;
    int32_t      dk;
    int32_t      dv;
    int32_t      chunk;
    int32_t      in_dtype;   /* CAP_DTYPE_BF16 */
    float        scale;
} gdn_args;

/* Workspace size for gdn_chunked_prefill: ceil(T / 64) * H * 12800 bytes
 * (per chunk and head: the chunk's (I + A)^-1 in operand form and its gate tables);
 * 0 for T <= 0, H < 1 or chunk != 64. */
CAP_API uint64_t gdn_workspace_bytes(int64_t T, int32_t H, int32_t chunk);

CAP_API int gdn_chunked_prefill(const gdn_args* args, void* stream);

/* One decode step of the delta rule: exactly one token (args->T == 1,
 * CAP_E_UNSUPPORTED otherwise) in one launch on a short vector-ALU path
 * (with one token A = 0 and (I + A)^-1 = I: u = beta (v - gamma k S),
 * S' = gamma S + k^T u, o = scale (gamma q S + (q.k) u)).  Same arguments
 * and checks as gdn_chunked_prefill except that the workspace is not used
 * (it may be NULL).  State and o agree with a one-token prefill's to fp32
 * rounding; decode steps are reproducible among themselves. */
CAP_API int gdn_decode_step(const gdn_args* args, void* stream);

/* ---------------------------- delta-rule prefill without allocation ---- */
/* For callers that cannot allocate device memory or hand in a workspace:
 * code recorded under stream capture (a HIP graph), tight serving loops,
 * harnesses that forbid allocation.  gdn_chunked_prefill with its
 * per-chunk workspace held in a fixed device array that the library owns:
 * GDN_NOALLOC_SCRATCH_BYTES on every GPU the library runs on, held until the
 * process ends.  The array keeps two states of all heads (the hand-over
 * between segments) and as many per-(chunk, head) workspace records as fit;
 * a call whose chunks do not all fit runs as several segments of whole
 * chunks (a prepare and a scan launch each), which computes exactly what one
 * gdn_chunked_prefill call computes (bit for bit: a chunk depends only on
 * the state entering it and its inputs).  Nothing is allocated: no
 * hipMalloc, no host heap.
 *
 * Arguments as gdn_chunked_prefill, except that workspace must be NULL and
 * workspace_bytes 0 (CAP_E_INVAL otherwise).  CAP_E_SIZE when one chunk of
 * all heads plus the two states does not fit the array:
 * 2 * round_up(H * dk * dv * 4, 256) + H * 12800 > GDN_NOALLOC_SCRATCH_BYTES
 * (H <= 233 at dk = dv = 128).  Every call on one GPU shares that GPU's
 * array (it keeps the last call's contents, which no call reads before
 * writing): calls that may overlap on one GPU -- on different streams, or
 * from several threads -- race and must be serialised by the caller. */
#define GDN_NOALLOC_SCRATCH_BYTES (32ull << 20)

CAP_API int gdn_chunked_prefill_noalloc(const gdn_args* args, void* stream);

/* ---------------------------------------------------------- FP8 KV ------ */
/* §3 "Definition": the KV region may be held in FP8, which roughly halves
 * the capsule (an FP8 K or V buffer is an ordinary POSITIONAL buffer with
 * one byte per element); the BF16 working stage read by the attention is not
 * part of the capsule and is rebuilt lazily after a restore (§3 cost model:
 * restore copies bytes and rebinds; the bound-stage calls below track which
 * rows a session's stage holds and convert only the rows it lacks).
 *
 * Format: OCP 8-bit floating point E4M3 (sign, 4 exponent bits with bias 7,
 * 3 mantissa bits; largest finite 448; S.1111.111 is NaN; no infinities),
 * one fp32 scale per segment, stored value = x / scale.
 *
 * A segment converts n elements (n % 16 == 0) from src to dst, both device
 * pointers, 16-byte aligned (CAP_E_ALIGN), caller-owned, disjoint (src from
 * dst, and the destinations of one call from each other: CAP_E_INVAL).
 * scale must be finite and > 0 (CAP_E_INVAL); reserved must be 0.  Up to
 * KV_FP8_MAX_SEG segments (one per K or V buffer) run in one launch;
 * segments with n = 0 are skipped. */
#define KV_FP8_MAX_SEG 64

typedef struct kv_fp8_seg {
    const void* src;
    void*       dst;
    uint64_t    n;         /* elements */
    float       scale;
    uint32_t    reserved;
} kv_fp8_seg;

/* ------------------------------------------- FP8 working stage (lazy) -- */
/* §3 "Definition" counts the FP8 dequantisation stage's valid end in a
 * capsule's KV region; §3 cost model and Table "cost structure": restore
 * copies bytes back and re-binds, and the BF16 stage is rebuilt lazily on
 * the next read, not eagerly in restore.
 *
 * A positional buffer of a set may hold FP8 rows (row_bytes = elements per
 * row) and be bound to a BF16 working stage, caller-owned device memory of
 * rows * row_bytes bf16 elements that the attention reads.  The set keeps
 * one stage valid end E for all its stages: rows [0, E) of every bound
 * stage hold the dequantisation (kv_fp8_dequantize) of the FP8 rows.
 *   - cap_stage_acquire(set, n) is the read: it converts exactly rows
 *     [E, n) of every stage in one launch (nothing when n <= E), then
 *     E = max(E, n).
 *   - capsule_snapshot records min(E, P') in the capsule (capsule_stage_end).
 *   - capsule_restore re-binds E and converts nothing: restoring into the
 *     set the capsule was taken from, in the same lineage -- no restore,
 *     fork, gather, rebinding or invalidation of that set since the
 *     snapshot, and no append below rows the set already held -- E becomes
 *     min(E, the capsule's recorded end), since those stage rows are already
 *     the dequantised capsule rows; in every other case E becomes 0.
 *   - capsule_fork and capsule_gather_restore leave every destination at 0.
 *   - cap_set_append below rows the set already held clips E to the append
 *     position.
 * The library assumes that bound stages, and the FP8 rows below a set's
 * position, change only through these calls; a caller that writes either
 * otherwise (filling the FP8 region itself, say) calls
 * cap_stage_invalidate.  Stages belong to the live session, never to a
 * capsule. */
#define CAP_MAX_STAGES 64u   /* stages per set (one rebuild launch) */

/* Bind buffer `buffer` (a POSITIONAL buffer of FP8 rows; CAP_E_UNSUPPORTED
 * otherwise) to a stage of rows * row_bytes bf16 elements at `stage`
 * (16-byte aligned, disjoint from every live buffer and every other stage of
 * the set: CAP_E_ALIGN / CAP_E_INVAL), decoded with `scale` (finite, > 0).
 * Binding a buffer again replaces its stage.  Sets E = 0.  Host only. */
CAP_API int cap_set_bind_stage(cap_set set, uint32_t buffer, void* stage, float scale);

/* The first read of rows [0, rows) of the stages: converts rows [E, rows) of
 * every bound stage (kv_fp8_dequantize semantics) in one stream-ordered
 * launch, sets E = max(E, rows) and returns the number of rows converted in
 * *converted (may be NULL; 0 when rows <= E, and then nothing is enqueued).
 * rows must not exceed the set's position (CAP_E_SIZE); a set with no bound
 * stage is CAP_E_STATE. */
CAP_API int cap_stage_acquire(cap_set set, uint64_t rows, void* stream, uint64_t* converted);

/* E of a set. */
CAP_API int cap_stage_valid_end(cap_set set, uint64_t* end);

/* E = 0 and a new lineage (after the caller wrote a stage or FP8 rows itself). */
CAP_API int cap_stage_invalidate(cap_set set);

/* The stage valid end a capsule recorded (min(E, P') at its snapshot). */
CAP_API int capsule_stage_end(cap_capsule cap, uint64_t* end);

/* bf16 -> E4M3: code = nearest representable value to float(x) * (1.0f /
 * scale) (fp32 product), ties to the even mantissa; |value| >= 448 and +-inf
 * saturate to +-448, NaN keeps its sign.  Appended K/V rows enter the FP8
 * region this way. */
CAP_API int kv_fp8_quantize(const kv_fp8_seg* segs, uint32_t n_seg, void* stream);

/* E4M3 -> bf16: decode(code) * scale in fp32, rounded to the nearest bf16
 * (ties to even); NaN codes give the canonical bf16 NaN with the code's
 * sign.  Rebuilds the BF16 stage of a row range (the lazy rebuild after a
 * restore). */
CAP_API int kv_fp8_dequantize(const kv_fp8_seg* segs, uint32_t n_seg, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CAPSULE_H */
