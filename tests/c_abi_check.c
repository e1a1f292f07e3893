/* A plain C99 caller of the capsule C ABI (include/capsule.h), host-only
 * entry points: it proves that the header compiles as C and that the shared
 * library links and runs without any C++ or Python on the caller's side.
 * Prints one line per check; tests/test_c_abi.py builds, runs and reads it. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "capsule.h"

int main(void) {
    /* P' = floor(P / C) C (§3 Algorithm 1) */
    printf("align %llu %llu %llu\n", (unsigned long long)cap_align_boundary(130, 64),
           (unsigned long long)cap_align_boundary(64, 64), (unsigned long long)cap_align_boundary(5, 0));

    /* capsule bytes of a layout: positional rows [0, P') plus whole fixed buffers */
    cap_buf bufs[3];
    memset(bufs, 0, sizeof(bufs));
    bufs[0].name = "kv.k";  bufs[0].row_bytes = 512;   bufs[0].rows = 300; bufs[0].kind = CAP_KIND_POSITIONAL;
    bufs[1].name = "state"; bufs[1].row_bytes = 65536; bufs[1].rows = 1;   bufs[1].kind = CAP_KIND_FIXED;
    bufs[2].name = "kv.v";  bufs[2].row_bytes = 48;    bufs[2].rows = 300; bufs[2].kind = CAP_KIND_POSITIONAL;
    uint64_t bytes = 0;
    const int rc = capsule_layout_bytes(bufs, 3, 64, 200, &bytes);
    printf("layout %d %llu\n", rc, (unsigned long long)bytes);

    /* errors are status codes, never exceptions across the boundary */
    bufs[2].row_bytes = 40;
    printf("misaligned %d\n", capsule_layout_bytes(bufs, 3, 64, 200, &bytes));
    cap_set set = 0;
    printf("null_set %d\n", cap_set_create(NULL, 0, 64, 1, &set));
    printf("status %s\n", cap_status_string(CAP_E_SIZE));

    /* FNV-1a-64 of a token prefix */
    const int32_t ids[5] = {1, -2, 300000, 0, 2147483647};
    printf("digest %llu\n", (unsigned long long)capsule_digest_tokens(ids, 5));
    return 0;
}
