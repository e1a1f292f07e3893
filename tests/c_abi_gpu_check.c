/* A plain C99 program that drives the capsule C ABI on the GPU with device
 * memory from hipMalloc only (no PyTorch, no Python): a capsule round trip
 * over a three-buffer set, a refused restore, and the chunk-alignment
 * property of both scans (a prefill split at an aligned boundary equals one
 * call bit for bit, §5).  Each check prints "<name> ok" or "<name> FAIL
 * <detail>"; tests/test_c_abi.py runs it and reads the lines.  Any HIP or
 * library error ends the program with a nonzero status. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "capsule.h"

#define HIP(x)                                                                    \
    do {                                                                          \
        hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                   \
            printf("hip_error %d line %d\n", (int)e_, __LINE__);                  \
            exit(2);                                                              \
        }                                                                         \
    } while (0)
#define CAP(x)                                                                    \
    do {                                                                          \
        int s_ = (x);                                                             \
        if (s_ != CAP_OK) {                                                       \
            printf("cap_error %d line %d\n", s_, __LINE__);                       \
            exit(3);                                                              \
        }                                                                         \
    } while (0)

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {  /* xorshift64* */
    rng ^= rng >> 12; rng ^= rng << 25; rng ^= rng >> 27;
    return (uint32_t)((rng * 0x2545F4914F6CDD1Dull) >> 32);
}
static float next_unit(void) { return (float)(next_u32() >> 8) * (1.0f / 16777216.0f) * 2.0f - 1.0f; }
static uint16_t bf16_of(float f) { uint32_t u; memcpy(&u, &f, 4); return (uint16_t)(u >> 16); }

static void* dev_from(const void* host, size_t bytes) {
    void* d = NULL;
    HIP(hipMalloc(&d, bytes));
    HIP(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
    return d;
}

static int capsule_round_trip(void) {
    const uint64_t rows = 300, krb = 512, srb = 65536, vrb = 48;
    const size_t kb = rows * krb, sb = srb, vb = rows * vrb;
    uint8_t* hk = malloc(kb); uint8_t* hs = malloc(sb); uint8_t* hv = malloc(vb);
    uint8_t* back = malloc(kb > sb ? kb : sb);
    for (size_t i = 0; i < kb; ++i) hk[i] = (uint8_t)next_u32();
    for (size_t i = 0; i < sb; ++i) hs[i] = (uint8_t)next_u32();
    for (size_t i = 0; i < vb; ++i) hv[i] = (uint8_t)next_u32();
    void* dk = dev_from(hk, kb); void* ds = dev_from(hs, sb); void* dv = dev_from(hv, vb);
    cap_buf bufs[3];
    memset(bufs, 0, sizeof(bufs));
    bufs[0].name = "kv.k";  bufs[0].dptr = dk; bufs[0].row_bytes = krb; bufs[0].rows = rows; bufs[0].kind = CAP_KIND_POSITIONAL;
    bufs[1].name = "state"; bufs[1].dptr = ds; bufs[1].row_bytes = srb; bufs[1].rows = 1;    bufs[1].kind = CAP_KIND_FIXED;
    bufs[2].name = "kv.v";  bufs[2].dptr = dv; bufs[2].row_bytes = vrb; bufs[2].rows = rows; bufs[2].kind = CAP_KIND_POSITIONAL;
    cap_set set = NULL;
    CAP(cap_set_create(bufs, 3, 64, 77, &set));
    const uint64_t P = 130, Pa = 128;
    CAP(cap_set_set_position(set, Pa));
    uint64_t nbytes = 0;
    CAP(capsule_bytes(set, P, &nbytes));
    void* arena = NULL;
    HIP(hipMalloc(&arena, nbytes));
    cap_capsule c = NULL;
    CAP(capsule_snapshot(set, P, 4242, arena, nbytes, NULL, &c));
    HIP(hipMemset(dk, 0xFF, kb)); HIP(hipMemset(ds, 0xFF, sb)); HIP(hipMemset(dv, 0xFF, vb));
    uint64_t got_p = 0;
    const int refused = capsule_restore(c, set, 4243, NULL, &got_p);  /* wrong prefix digest */
    CAP(capsule_restore(c, set, 4242, NULL, &got_p));
    HIP(hipDeviceSynchronize());
    int ok = refused == CAP_E_DIGEST && got_p == Pa && nbytes == Pa * (krb + vrb) + srb;
    HIP(hipMemcpy(back, dk, kb, hipMemcpyDeviceToHost));
    ok = ok && memcmp(back, hk, Pa * krb) == 0;
    for (size_t i = Pa * krb; i < kb; ++i) ok = ok && back[i] == 0xFF;  /* rows past P' untouched */
    HIP(hipMemcpy(back, ds, sb, hipMemcpyDeviceToHost));
    ok = ok && memcmp(back, hs, sb) == 0;
    HIP(hipMemcpy(back, dv, vb, hipMemcpyDeviceToHost));
    ok = ok && memcmp(back, hv, Pa * vrb) == 0;
    for (size_t i = Pa * vrb; i < vb; ++i) ok = ok && back[i] == 0xFF;
    printf("capsule %s refused=%d P=%llu bytes=%llu\n", ok ? "ok" : "FAIL", refused, (unsigned long long)got_p,
           (unsigned long long)nbytes);
    CAP(capsule_release(c));
    CAP(cap_set_destroy(set));
    HIP(hipFree(arena)); HIP(hipFree(dk)); HIP(hipFree(ds)); HIP(hipFree(dv));
    free(hk); free(hs); free(hv); free(back);
    return ok;
}

/* one scan (gdn = 0: linear attention, 1: delta rule) over T tokens in one
 * call and split at the aligned boundary Pa; o and the final state must be
 * equal bit for bit */
static int split_equals_one_call(int gdn) {
    const int T = 300, H = 3, dk = 128, dv = 32, Pa = 128;
    const size_t nq = (size_t)T * H * dk, nv = (size_t)T * H * dv, ns = (size_t)H * dk * dv;
    uint16_t* hq = malloc(nq * 2); uint16_t* hk = malloc(nq * 2); uint16_t* hv = malloc(nv * 2);
    float* hg = malloc((size_t)T * H * 4); float* hb = malloc((size_t)T * H * 4);
    for (size_t i = 0; i < nq; ++i) { hq[i] = bf16_of(0.1f * next_unit()); hk[i] = bf16_of(0.1f * next_unit()); }
    for (size_t i = 0; i < nv; ++i) hv[i] = bf16_of(next_unit());
    for (int i = 0; i < T * H; ++i) { hg[i] = -0.05f * (1.0f + next_unit()); hb[i] = 0.5f + 0.4f * next_unit(); }
    void* q = dev_from(hq, nq * 2); void* k = dev_from(hk, nq * 2); void* v = dev_from(hv, nv * 2);
    float* g = dev_from(hg, (size_t)T * H * 4); float* beta = dev_from(hb, (size_t)T * H * 4);
    float *o1, *o2, *s1, *s2;
    HIP(hipMalloc((void**)&o1, nv * 4)); HIP(hipMalloc((void**)&o2, nv * 4));
    HIP(hipMalloc((void**)&s1, ns * 4)); HIP(hipMalloc((void**)&s2, ns * 4));
    void* ws = NULL;
    uint64_t wsb = 16;
    if (gdn) wsb = gdn_workspace_bytes(T, H, 64);
    HIP(hipMalloc(&ws, wsb));
    for (int part = 0; part < 3; ++part) {  /* 0: one call; 1: [0, Pa); 2: [Pa, T) */
        const int t0 = part == 2 ? Pa : 0, t1 = part == 1 ? Pa : T;
        float* o = (part == 0 ? o1 : o2) + (size_t)t0 * H * dv;
        float* st = part == 0 ? s1 : s2;
        const size_t qo = (size_t)t0 * H * dk * 2, vo = (size_t)t0 * H * dv * 2;
        if (gdn) {
            gdn_args a;
            memset(&a, 0, sizeof(a));
            a.q = (const char*)q + qo; a.k = (const char*)k + qo; a.v = (const char*)v + vo;
            a.g = g + (size_t)t0 * H; a.beta = beta + (size_t)t0 * H;
            a.state_in = part == 2 ? s2 : NULL; a.o = o; a.final_state = st;
            a.workspace = ws; a.workspace_bytes = wsb;
            a.T = t1 - t0; a.H = H; a.dk = dk; a.dv = dv; a.chunk = 64; a.in_dtype = CAP_DTYPE_BF16; a.scale = 1.0f;
            CAP(gdn_chunked_prefill(&a, NULL));
        } else {
            linattn_args a;
            memset(&a, 0, sizeof(a));
            a.q = (const char*)q + qo; a.k = (const char*)k + qo; a.v = (const char*)v + vo;
            a.g = g + (size_t)t0 * H;
            a.state_in = part == 2 ? s2 : NULL; a.o = o; a.final_state = st;
            a.T = t1 - t0; a.H = H; a.dk = dk; a.dv = dv; a.chunk = 64; a.in_dtype = CAP_DTYPE_BF16; a.scale = 1.0f;
            CAP(linattn_chunked_prefill(&a, NULL));
        }
    }
    HIP(hipDeviceSynchronize());
    float* a1 = malloc(nv * 4); float* a2 = malloc(nv * 4);
    HIP(hipMemcpy(a1, o1, nv * 4, hipMemcpyDeviceToHost)); HIP(hipMemcpy(a2, o2, nv * 4, hipMemcpyDeviceToHost));
    int ok = memcmp(a1, a2, nv * 4) == 0;
    double mx = 0.0;
    for (size_t i = 0; i < nv; ++i) { const double x = a1[i] < 0 ? -a1[i] : a1[i]; if (!(x <= 1e30)) ok = 0; if (x > mx) mx = x; }
    ok = ok && mx > 0.0;  /* finite and not all zero */
    float* b1 = malloc(ns * 4); float* b2 = malloc(ns * 4);
    HIP(hipMemcpy(b1, s1, ns * 4, hipMemcpyDeviceToHost)); HIP(hipMemcpy(b2, s2, ns * 4, hipMemcpyDeviceToHost));
    ok = ok && memcmp(b1, b2, ns * 4) == 0;
    printf("%s %s max|o|=%.4g\n", gdn ? "gdn_split" : "linattn_split", ok ? "ok" : "FAIL", mx);
    HIP(hipFree(q)); HIP(hipFree(k)); HIP(hipFree(v)); HIP(hipFree(g)); HIP(hipFree(beta));
    HIP(hipFree(o1)); HIP(hipFree(o2)); HIP(hipFree(s1)); HIP(hipFree(s2)); HIP(hipFree(ws));
    free(hq); free(hk); free(hv); free(hg); free(hb); free(a1); free(a2); free(b1); free(b2);
    return ok;
}

int main(void) {
    HIP(hipSetDevice(0));
    const int a = capsule_round_trip();
    const int b = split_equals_one_call(0);
    const int c = split_equals_one_call(1);
    printf("done %d\n", a && b && c);
    return a && b && c ? 0 : 1;
}
