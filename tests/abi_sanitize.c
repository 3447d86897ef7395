/*
 * The library's host-side argument checks under the address and undefined-behaviour sanitizers
 * (test infrastructure; no GPU needed).
 *
 * tests/test_abi_sanitizers.py builds the library with both sanitizers on its host code (the
 * device code is built as usual; no kernel is launched) and links this program against it. Every call
 * below must return its documented status without touching memory it does not own: host-side
 * validation, size arithmetic near the int64 limits, overlap checks, status strings, and the
 * calls that reach the runtime and find no GPU. Prints "ok" and exits 0, or names the failed
 * check and exits 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "cc_join.h"

static int failures;

#define EXPECT(expr, want)                                                              \
    do {                                                                                \
        const long long got_ = (long long)(expr);                                       \
        if (got_ != (long long)(want)) {                                                \
            fprintf(stderr, "FAILED line %d: %s = %lld, want %lld\n", __LINE__, #expr, \
                    got_, (long long)(want));                                           \
            failures++;                                                                 \
        }                                                                               \
    } while (0)

#define P(x) ((void *)(uintptr_t)(x))   /* an address that is never dereferenced */

static cc_status sort_call(int32_t nv, uintptr_t off, uintptr_t kin, uintptr_t rin, int32_t rb,
                           int64_t tk, int64_t mk, uintptr_t kout, uintptr_t rout, uintptr_t w,
                           int64_t wb)
{
    return cc_sort_affinity(nv, P(off), P(kin), P(rin), rb, tk, mk, P(kout), P(rout), P(w), wb,
                            NULL);
}

int main(void)
{
    /* status strings, including an unknown code */
    EXPECT(strcmp(cc_status_string(CC_OK), "CC_OK"), 0);
    EXPECT(strcmp(cc_status_string(CC_ERR_STORE_FULL), "CC_ERR_STORE_FULL"), 0);
    EXPECT(strcmp(cc_status_string((cc_status)99), "CC_UNKNOWN_STATUS"), 0);
    EXPECT(cc_last_device_error(), 0);

    /* store creation: every rejected argument leaves the handle null */
    cc_store *h = (cc_store *)P(1234);
    const int64_t big = (int64_t)1 << 62;
    EXPECT(cc_store_create(NULL, 0, NULL, NULL, 16, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, -1, NULL, NULL, 16, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(h == NULL, 1);
    EXPECT(cc_store_create(&h, 4, P(8), P(8), 24, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, 4, P(8), P(8), 0, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, 4, P(8), P(8), (1 << 20) + 16, CC_SRC_HOST, NULL),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, 4, NULL, P(8), 16, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, 0, NULL, NULL, 16, 3, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, big, P(8), P(8), 16, CC_SRC_HOST, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create(&h, INT64_MAX, P(8), P(8), 1 << 20, CC_SRC_DEVICE, NULL),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(h == NULL, 1);
    EXPECT(cc_store_create_indexed(NULL, 10, 16, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create_indexed(&h, -1, 16, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create_indexed(&h, (int64_t)1 << 31, 16, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_create_indexed(&h, 10, 24, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(h == NULL, 1);

    /* a null store */
    int64_t n = 7;
    int32_t w = 7;
    EXPECT(cc_join(NULL, NULL, 0, NULL, 0, NULL, 16, NULL, NULL, 32, NULL, NULL),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_join_batched(NULL, 0, NULL, NULL, 0, NULL, NULL, 0, NULL, 16, NULL, 1, NULL, NULL,
                           32, NULL, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_join_batched_padded(NULL, 1, P(8), P(8), 1, P(8), P(8), 1, P(16), 16, NULL, 1,
                                  NULL, 4, P(16), 32, P(8), P(8), NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_info(NULL, &n, &w), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_layout(NULL, &w, &n), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_invalid_count(NULL, &n, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_reset_invalid_count(NULL, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_read(NULL, 0, 1, P(8), P(16), NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_upsert(NULL, 1, P(8), P(8), P(16), P(16), 1 << 20, &n, &n, NULL),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_resolve_ids(NULL, P(8), 1, P(8), NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_store_destroy(NULL), CC_OK);

    /* key validation */
    int64_t bad = 7;
    EXPECT(cc_validate_keys(NULL, NULL, 1, 0, NULL, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_validate_keys(NULL, NULL, 1, 0, &bad, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_validate_keys(P(8), NULL, 1, 5, &bad, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_validate_keys(P(12), P(16), 1, 5, &bad, NULL), CC_ERR_INVALID_ARGUMENT);
    EXPECT(cc_validate_keys(NULL, NULL, 0, 0, &bad, NULL), CC_OK);
    EXPECT(bad, -1);

    /* workspace sizes, including counts near the limits */
    EXPECT(cc_sort_workspace_bytes(0, 3), 0);
    EXPECT(cc_sort_workspace_bytes(-5, 3), 0);
    EXPECT(cc_sort_workspace_bytes(100, 0), 0);
    EXPECT(cc_sort_workspace_bytes(4097, 2) >= 2 * 16 * 4097 + 3 * 8, 1);
    EXPECT(cc_sort_workspace_bytes(((int64_t)1 << 32) - 1, INT32_MAX) > 0, 1);
    EXPECT(cc_upsert_workspace_bytes(0), 0);
    EXPECT(cc_upsert_workspace_bytes(-3), 0);
    EXPECT(cc_upsert_workspace_bytes(1000) >= 12 * 1000, 1);
    EXPECT(cc_upsert_workspace_bytes(INT64_MAX), 0);          /* beyond the batch limit */
    EXPECT(cc_upsert_workspace_bytes(((int64_t)1 << 30) + 1), 0);
    EXPECT(cc_sort_workspace_bytes((int64_t)1 << 32, 1), 0);  /* beyond the sort's limit */
    EXPECT(cc_sort_workspace_bytes(INT64_MAX, INT32_MAX), 0);

    /* sort: each rejected argument, and the calls with nothing to do */
    const int64_t ws = cc_sort_workspace_bytes(1000, 1);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 24, 1000, 0, 0x30000, 0x100000, 0x200000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, -1, 0, 0x30000, 0x100000, 0x200000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, (int64_t)1 << 32, 0, 0x30000, 0x100000,
                     0x200000, ws), CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, 1000, 0, 0x30000, 0x100000, 0x200000,
                     ws - 1), CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, 1000, 0, 0x2000, 0x100000, 0x200000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, 1000, 0, 0x30000, 0x10040, 0x200000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, 1000, 0, 0x30000, 0x100000, 0x30000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0x2000, 0x10000, 32, 1000, -1, 0x30000, 0x100000, 0x200000, ws),
           CC_ERR_INVALID_ARGUMENT);
    EXPECT(sort_call(1, 0x1000, 0, 0, 32, 0, 0, 0, 0, 0, 0), CC_OK);
    EXPECT(sort_call(0, 0, 0, 0, 32, 0, 0, 0, 0, 0, 0), CC_OK);

    /* valid arguments reach the runtime, which finds no GPU */
    const int64_t ids[2] = {1, 2};
    const unsigned char rows[32] = {0};
    const cc_status st = cc_store_create(&h, 2, ids, rows, 16, CC_SRC_HOST, NULL);
    EXPECT(st == CC_ERR_NOT_SUPPORTED || st == CC_ERR_DEVICE, 1);
    EXPECT(h == NULL, 1);

    if (failures)
        return 1;
    printf("ok\n");
    return 0;
}
