/* Plain C client of the C ABI (no HIP headers): checks that include/ws_attn.h
 * compiles as C and that the library answers version, status and
 * argument-validation queries.  Every attention call below fails validation
 * (NULL pointers or bad sizes), so nothing touches a device. */
#include <stdio.h>
#include <string.h>

#include "ws_attn.h"

static int fails = 0;
#define CHECK(cond)                                                     \
    do {                                                                \
        if (!(cond)) {                                                  \
            fprintf(stderr, "check failed: %s (line %d)\n", #cond, __LINE__); \
            ++fails;                                                    \
        }                                                               \
    } while (0)

int main(void) {
    CHECK(ws_abi_version() == WS_ABI_VERSION);
    CHECK(strcmp(ws_status_string(WS_OK), "WS_OK") == 0);
    CHECK(strcmp(ws_status_string(WS_ERR_OFFSETS), "WS_ERR_OFFSETS") == 0);

    ws_tensor4 none;
    memset(&none, 0, sizeof none);
    int32_t lens[1] = {0};
    /* no cache descriptor */
    CHECK(ws_kv_append(NULL, 1, lens, lens, 4, none, none, NULL) == WS_ERR_NULL);
    CHECK(ws_block_causal_attn_fwd(none, none, none, NULL, lens, lens, 1, 4, 2, 0.1f, 0, none, NULL,
                                   NULL, 0, NULL) == WS_ERR_NULL);
    CHECK(strlen(ws_last_error()) > 0);
    CHECK(ws_block_causal_attn_fwd_varlen(none, none, none, NULL, lens, lens, lens, lens, NULL, NULL, 1, 4, 2,
                                          0.1f, 0, none, NULL, NULL, 0, NULL) == WS_ERR_NULL);
    CHECK(ws_kv_append_varlen(NULL, 1, lens, lens, NULL, NULL, 4, none, none, NULL) == WS_ERR_NULL);
    /* negative sizes */
    int32_t offs[2] = {0, 8};
    CHECK(ws_block_causal_prefill(none, none, none, NULL, offs, offs, -1, 8, 1, 2, 1, 64, 0.1f, none,
                                  NULL, NULL) == WS_ERR_SHAPE);
    CHECK(ws_block_causal_prefill_bwd(none, none, none, none, none, NULL, offs, offs, NULL, NULL, 1, 8, 1,
                                      2, 1, 64, 0.1f, none, none, none, NULL, 0, NULL) == WS_ERR_NULL);
    /* nothing to do is fine */
    CHECK(ws_block_causal_prefill(none, none, none, NULL, offs, offs, 0, 8, 1, 2, 1, 64, 0.1f, none, NULL,
                                  NULL) == WS_OK);
    CHECK(ws_workspace_bytes(WS_OP_PREFILL_BWD, 1, 2, 1, 8, 8) > 0);
    CHECK(ws_workspace_bytes(WS_OP_PREFILL, 1, 2, 1, 8, 8) == 0);
    if (fails == 0) printf("c abi ok\n");
    return fails != 0;
}
