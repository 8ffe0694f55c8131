/* Drives the host side of the C ABI -- configuration checks, argument
 * checks, status strings, the profiling arrays and the test hooks -- for a
 * build whose host code runs under AddressSanitizer and
 * UndefinedBehaviorSanitizer.  Nothing here needs a GPU: every call fails
 * validation before any launch, or (ledger creation with a valid
 * configuration) fails or succeeds in the HIP runtime.  Exits non-zero on
 * an unexpected status. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "routerelay.h"

static int failures = 0;
#define EXPECT(cond)                                                          \
    do {                                                                      \
        if (!(cond)) {                                                        \
            fprintf(stderr, "line %d: %s (last error: %s)\n", __LINE__, #cond, \
                    rr_last_error());                                         \
            ++failures;                                                       \
        }                                                                     \
    } while (0)

static rr_config base(void)
{
    rr_config c;
    memset(&c, 0, sizeof(c));
    c.n_heads = 2; c.n_kv_heads = 1; c.n_q = 64; c.n_k = 64; c.d = 64;
    c.k = 8; c.m = 4; c.r = 4; c.dtype = RR_F32;
    return c;
}

int main(void)
{
    for (int s = -6; s <= 1; ++s) EXPECT(rr_status_string((rr_status)s) != NULL);
    EXPECT(rr_last_error() != NULL);

    rr_ledger *L = (rr_ledger *)0x1;
    EXPECT(rr_ledger_create(NULL, &L) == RR_ERR_INVALID && L == NULL);
    rr_config c = base();
    EXPECT(rr_ledger_create(&c, NULL) == RR_ERR_INVALID);

    /* invalid and unsupported configurations, on both the ledger and the
     * stateless path */
    struct { int field; int value; rr_status want; } cases[] = {
        {0, 0, RR_ERR_INVALID}, {1, 3, RR_ERR_INVALID}, {2, 0, RR_ERR_INVALID}, {3, 0, RR_ERR_INVALID},
        {4, 48, RR_ERR_UNSUPPORTED}, {5, 0, RR_ERR_INVALID}, {5, 65, RR_ERR_INVALID}, {6, -1, RR_ERR_INVALID},
        {7, -2, RR_ERR_INVALID}, {8, 7, RR_ERR_INVALID}, {9, 2, RR_ERR_INVALID}, {10, 9000, RR_ERR_UNSUPPORTED},
    };
    for (unsigned t = 0; t < sizeof(cases) / sizeof(cases[0]); ++t) {
        c = base();
        int32_t *f[] = {&c.n_heads, &c.n_kv_heads, &c.n_q, &c.n_k, &c.d, &c.k, &c.m, &c.r, &c.dtype, &c.causal};
        if (cases[t].field < 10) {
            *f[cases[t].field] = cases[t].value;
        } else {
            c.n_q = c.n_k = cases[t].value;
        }
        L = (rr_ledger *)0x1;
        EXPECT(rr_ledger_create(&c, &L) == cases[t].want && L == NULL);
        EXPECT(strlen(rr_last_error()) > 0);
        if (cases[t].field != 6 && cases[t].field != 7)
            EXPECT(rr_full_route(&c, (void *)0x1000, (void *)0x1000, (int32_t *)0x1000, NULL, NULL, NULL) ==
                   cases[t].want);
    }
    c = base();
    c.gamma = NAN;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_INVALID);
    c = base();
    c.options = 3;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_INVALID);
    c.options = 0x80;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_INVALID);
    c = base();
    c.causal = 1;
    c.n_q = 32;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_INVALID);
    c = base();
    c.n_q = c.n_k = 8192; c.d = 128; c.k = 32; c.m = 16; c.r = 16;
    c.options = RR_OPT_ONE_PASS_RELAY;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_UNSUPPORTED);
    c = base();
    c.n_heads = 1 << 20; c.n_kv_heads = 1; c.n_q = 8192; c.n_k = 8192;
    EXPECT(rr_ledger_create(&c, &L) == RR_ERR_UNSUPPORTED);

    /* NULL handles and pointers */
    EXPECT(rr_ledger_destroy(NULL) == RR_OK);
    EXPECT(rr_anchor_route(NULL, 0, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_relay_layer(NULL, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    c = base();
    EXPECT(rr_full_route(&c, NULL, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_full_route(NULL, NULL, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_ledger_routes(NULL) == NULL);
    EXPECT(rr_ledger_export(NULL, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_ledger_import(NULL, 0, NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_ledger_relay_stats(NULL, NULL, NULL, NULL, NULL) == RR_ERR_INVALID);
    EXPECT(rr_ledger_index_bytes(NULL) == 0);
    c = base();
    EXPECT(rr_ledger_index_bytes(&c) == (size_t)2 * 64 * 16 * 4);

    /* profiling arrays: a short length is refused without writing */
    double ms[RR_KERNEL_KINDS + 1];
    int64_t n[RR_KERNEL_KINDS + 1];
    for (int t = 0; t <= RR_KERNEL_KINDS; ++t) { ms[t] = -1.0; n[t] = -1; }
    EXPECT(rr_profile_start() == RR_OK);
    EXPECT(rr_profile_stop(ms, n, RR_KERNEL_KINDS - 1) == RR_ERR_INVALID);
    EXPECT(ms[0] == -1.0 && n[0] == -1);
    EXPECT(rr_profile_stop(ms, n, RR_KERNEL_KINDS) == RR_OK);
    EXPECT(ms[0] == 0.0 && n[RR_KERNEL_KINDS - 1] == 0 && n[RR_KERNEL_KINDS] == -1);
    EXPECT(rr_profile_stop(NULL, NULL, 0) == RR_OK);

    /* test hooks */
    EXPECT(rr_set_sweep_cap(-1) == RR_ERR_INVALID);
    EXPECT(rr_set_sweep_cap(0) == RR_OK);
    EXPECT(rr_unconverged_rows(NULL) == RR_ERR_INVALID);

    /* either side of the path: argument checks refuse these before any
     * launch (the pointers are never dereferenced) */
    void *fake = (void *)0x1000;
    EXPECT(rr_pool_chunks(NULL, 1, 64, 128, 8, RR_BF16, fake, NULL) == RR_ERR_INVALID);
    EXPECT(rr_pool_chunks(fake, 1, 64, 12, 8, RR_BF16, fake, NULL) == RR_ERR_INVALID);
    EXPECT(rr_pool_chunks(fake, 1, 64, 128, 0, RR_BF16, fake, NULL) == RR_ERR_INVALID);
    EXPECT(rr_expand_tokens(NULL, 1, 4, 8, 64, (int32_t *)fake, NULL) == RR_ERR_INVALID);
    EXPECT(rr_expand_tokens((const int32_t *)fake, 1, 70000, 70000, 64, (int32_t *)fake, NULL) == RR_ERR_INVALID);
    rr_attn_config ac;
    memset(&ac, 0, sizeof(ac));
    ac.n_heads = 4; ac.n_kv_heads = 2; ac.n_tokens = 512; ac.d = 128; ac.chunk = 64; ac.k = 4;
    ac.causal = 1; ac.dtype = RR_BF16;
    EXPECT(rr_sparse_attention(NULL, fake, fake, fake, (const int32_t *)fake, fake, NULL) == RR_ERR_INVALID);
    ac.d = 96;
    EXPECT(rr_sparse_attention(&ac, fake, fake, fake, (const int32_t *)fake, fake, NULL) == RR_ERR_UNSUPPORTED);
    ac.d = 128; ac.k = 300;
    EXPECT(rr_sparse_attention(&ac, fake, fake, fake, (const int32_t *)fake, fake, NULL) == RR_ERR_INVALID);
    ac.k = 4; ac.scale = NAN;
    EXPECT(rr_sparse_attention(&ac, fake, fake, fake, (const int32_t *)fake, fake, NULL) == RR_ERR_INVALID);

    /* a valid configuration: allocation fails cleanly without a GPU, or
     * succeeds and is released */
    c = base();
    L = NULL;
    rr_status st = rr_ledger_create(&c, &L);
    EXPECT((st == RR_OK) == (L != NULL));
    if (L) EXPECT(rr_ledger_destroy(L) == RR_OK);

    if (failures) return 1;
    printf("abi driver ok\n");
    return 0;
}
