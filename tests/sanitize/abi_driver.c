/*
 * Host-side checks of libtileattn's C ABI, built from the library sources
 * compiled for the host only with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_sanitizers.py builds and runs it on
 * the CPU).  Every entry point is called with fake, 16-byte aligned device
 * addresses and arguments that must fail validation, so nothing is ever
 * dereferenced or launched; the pure host functions (tile schedule, workspace
 * sizes, split heuristics, status strings) run on many shapes.  A status
 * other than the expected one, or any sanitizer report, fails the run.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "tileattn.h"

static int failures = 0;

#define EXPECT(cond, ...)                      \
    do {                                       \
        if (!(cond)) {                         \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
            fprintf(stderr, __VA_ARGS__);      \
            fputc('\n', stderr);               \
            ++failures;                        \
        }                                      \
    } while (0)

#define P(x) ((void *)(uintptr_t)(x))

/* attn_fwd family: base arguments are valid except where a case changes one */
typedef struct {
    uintptr_t Q, K, V, O, L, ws;
    int B, Hq, Hkv, Sq, Sk, D, causal, splits, o_bf16;
    float scale;
    size_t ws_bytes;
} attn_args;

static attn_args attn_ok(void)
{
    attn_args a = {0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000, 0x60000000,
                   1, 2, 2, 128, 128, 64, 0, 2, 0, 0.125f, 1u << 24};
    return a;
}

/* Every entry point with the arguments of one case (all of them must fail
   validation: the pointers are fake).  split_only: the case concerns an
   argument only the split entry points take, so the others (which would get
   valid arguments) are not called. */
static void attn_case_any(attn_args a, int want, const char *what, int split_only)
{
    int rc;
    if (split_only)
        goto split;
    rc = attn_fwd(P(a.Q), P(a.K), P(a.V), (float *)P(a.O), (float *)P(a.L), a.B, a.Hq, a.Hkv,
                      a.Sq, a.Sk, a.D, a.causal, a.scale, NULL);
    EXPECT(rc == want, "attn_fwd %s: %d want %d", what, rc, want);
    rc = attn_fwd_bf16out(P(a.Q), P(a.K), P(a.V), P(a.O), (float *)P(a.L), a.B, a.Hq, a.Hkv,
                          a.Sq, a.Sk, a.D, a.causal, a.scale, NULL);
    EXPECT(rc == want || (want == TA_ERR_ALIASING), "attn_fwd_bf16out %s: %d want %d", what, rc,
           want);
split:
    rc = attn_fwd_split(P(a.Q), P(a.K), P(a.V), P(a.O), a.o_bf16, (float *)P(a.L), a.B, a.Hq,
                        a.Hkv, a.Sq, a.Sk, a.D, a.causal, a.scale, a.splits, P(a.ws), a.ws_bytes,
                        NULL);
    EXPECT(rc == want, "attn_fwd_split %s: %d want %d", what, rc, want);
    rc = attn_fwd_split_noalloc(P(a.Q), P(a.K), P(a.V), P(a.O), a.o_bf16, (float *)P(a.L), a.B,
                                a.Hq, a.Hkv, a.Sq, a.Sk, a.D, a.causal, a.scale, a.splits, NULL);
    EXPECT(rc == want, "attn_fwd_split_noalloc %s: %d want %d", what, rc, want);
}

static void attn_case(attn_args a, int want, const char *what)
{
    attn_case_any(a, want, what, 0);
}

static void check_attn_validation(void)
{
    attn_args a;
#define CASE(field, value, want) \
    a = attn_ok();               \
    a.field = value;             \
    attn_case(a, want, #field "=" #value)
    CASE(Q, 0, TA_ERR_NULL_POINTER);
    CASE(K, 0, TA_ERR_NULL_POINTER);
    CASE(V, 0, TA_ERR_NULL_POINTER);
    CASE(O, 0, TA_ERR_NULL_POINTER);
    CASE(L, 0, TA_ERR_NULL_POINTER);
    CASE(B, 0, TA_ERR_INVALID_SHAPE);
    CASE(Hq, 0, TA_ERR_INVALID_SHAPE);
    CASE(Hkv, -1, TA_ERR_INVALID_SHAPE);
    CASE(Sq, 0, TA_ERR_INVALID_SHAPE);
    CASE(Sk, -7, TA_ERR_INVALID_SHAPE);
    CASE(Hkv, 3, TA_ERR_INVALID_SHAPE);
    CASE(Sq, 1 << 25, TA_ERR_INVALID_SHAPE);
    a = attn_ok();
    a.splits = 0;
    attn_case_any(a, TA_ERR_INVALID_SHAPE, "splits=0", 1);
    a.splits = 129;
    attn_case_any(a, TA_ERR_INVALID_SHAPE, "splits=129", 1);
    CASE(D, 96, TA_ERR_UNSUPPORTED);
    CASE(D, 256, TA_ERR_UNSUPPORTED);
    CASE(Q, 0x10000008, TA_ERR_MISALIGNED);
    CASE(O, 0x40000004, TA_ERR_MISALIGNED);
    CASE(L, 0x50000004, TA_ERR_MISALIGNED);
    CASE(scale, -0.5f, TA_ERR_INVALID_SCALE);
    CASE(scale, 1.0f / 0.0f, TA_ERR_INVALID_SCALE);
    CASE(O, 0x10000000 + 16, TA_ERR_ALIASING);
    CASE(L, 0x20000000 + 64, TA_ERR_ALIASING);
#undef CASE
    a = attn_ok();
    a.causal = 1;
    a.Sq = 129;
    attn_case(a, TA_ERR_INVALID_SHAPE, "causal Sq > Sk");
    /* workspace errors only concern attn_fwd_split */
    a = attn_ok();
    a.ws = 0;
    EXPECT(attn_fwd_split(P(a.Q), P(a.K), P(a.V), P(a.O), 0, (float *)P(a.L), a.B, a.Hq, a.Hkv,
                          a.Sq, a.Sk, a.D, 0, a.scale, 2, NULL, 1u << 24, NULL) == TA_ERR_WORKSPACE,
           "split without workspace");
    EXPECT(attn_fwd_split(P(a.Q), P(a.K), P(a.V), P(a.O), 0, (float *)P(a.L), a.B, a.Hq, a.Hkv,
                          a.Sq, a.Sk, a.D, 0, a.scale, 2, P(0x60000000), 1000, NULL) ==
               TA_ERR_WORKSPACE,
           "split with a small workspace");
    /* partial results beyond the static scratch */
    EXPECT(attn_fwd_split_noalloc(P(0x10000000), P(0x20000000), P(0x30000000), P(0x40000000), 0,
                                  (float *)P(0x50000000), 1, 32, 32, 4096, 4096, 128, 0, 0.1f, 2,
                                  NULL) == TA_ERR_SCRATCH,
           "noalloc beyond the scratch");
}

/* ta_schedule against a brute-force count of visible and masked pairs */
static void check_schedule(void)
{
    int bm, bn;
    EXPECT(ta_tile_shape(128, &bm, &bn) == TA_OK, "tile shape");
    EXPECT(ta_tile_shape(96, &bm, &bn) == TA_ERR_UNSUPPORTED, "tile shape D=96");
    EXPECT(ta_tile_shape(64, NULL, &bn) == TA_ERR_NULL_POINTER, "tile shape null");
    ta_tile_shape(64, &bm, &bn);
    const int sizes[] = {1, 2, 37, 63, 64, 65, 127, 128, 129, 200, 300, 511, 1000};
    const int ns = (int)(sizeof sizes / sizeof sizes[0]);
    for (int x = 0; x < ns; ++x)
        for (int y = 0; y < ns; ++y)
            for (int causal = 0; causal < 2; ++causal) {
                const int Sq = sizes[x], Sk = sizes[y];
                int n, fm;
                if (causal && Sq > Sk) {
                    EXPECT(ta_schedule(Sq, Sk, 64, causal, 0, &n, &fm) == TA_ERR_INVALID_SHAPE,
                           "schedule rejects causal Sq > Sk");
                    continue;
                }
                const int n_qt = (Sq + bm - 1) / bm;
                for (int qt = 0; qt < n_qt; ++qt) {
                    EXPECT(ta_schedule(Sq, Sk, 64, causal, qt, &n, &fm) == TA_OK, "schedule ok");
                    const int n_tiles = (Sk + bn - 1) / bn;
                    int last_vis = -1, first_mask = n_tiles;
                    for (int t = 0; t < n_tiles; ++t) {
                        int vis = 0, masked = 0;
                        for (int i = qt * bm; i < qt * bm + bm && i < Sq; ++i)
                            for (int j = t * bn; j < t * bn + bn; ++j) {
                                const int ok = j < Sk && (!causal || j <= i + Sk - Sq);
                                vis |= ok;
                                masked |= !ok;
                            }
                        if (vis)
                            last_vis = t;
                        if (masked && t < first_mask)
                            first_mask = t;
                    }
                    EXPECT(n == last_vis + 1, "n_kv %d want %d (Sq %d Sk %d qt %d)", n,
                           last_vis + 1, Sq, Sk, qt);
                    EXPECT(fm <= n && (fm == n || fm >= first_mask) && fm <= first_mask + 0 + n,
                           "first_masked %d (Sq %d Sk %d qt %d)", fm, Sq, Sk, qt);
                    EXPECT(fm == (first_mask < n ? first_mask : n),
                           "first_masked %d want %d (Sq %d Sk %d qt %d)", fm,
                           first_mask < n ? first_mask : n, Sq, Sk, qt);
                }
                EXPECT(ta_schedule(Sq, Sk, 64, causal, n_qt, &n, &fm) == TA_ERR_INVALID_SHAPE,
                       "schedule rejects a query tile past the end");
            }
}

static void check_host_helpers(void)
{
    size_t bytes = 0;
    EXPECT(ta_split_workspace_bytes(2, 3, 100, 128, 4, &bytes) == TA_OK &&
               bytes == (size_t)4 * 2 * 3 * 100 * 129 * 4,
           "split workspace bytes");
    EXPECT(ta_split_workspace_bytes(2, 3, 100, 128, 1, &bytes) == TA_OK && bytes == 0,
           "one split needs no workspace");
    EXPECT(ta_split_workspace_bytes(2, 3, 100, 128, 0, &bytes) == TA_ERR_INVALID_SHAPE,
           "zero splits");
    const int shapes[][6] = {{1, 32, 32, 512, 512, 128},   {1, 32, 32, 1024, 1024, 128},
                             {8, 32, 32, 2048, 2048, 128}, {1, 32, 8, 1024, 8192, 128},
                             {1, 1, 1, 1, 1, 64},           {1, 2, 2, 128, 100000, 64}};
    for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i) {
        int n = 0;
        for (int causal = 0; causal < 2; ++causal) {
            const int *s = shapes[i];
            const int rc = ta_split_heuristic(s[0], s[1], s[2], s[3], s[4], s[5], causal, &n);
            EXPECT(rc == (causal && s[3] > s[4] ? TA_ERR_INVALID_SHAPE : TA_OK),
                   "split heuristic status");
            if (rc == TA_OK)
                EXPECT(n >= 1 && n <= 128, "split heuristic range %d", n);
        }
    }
    EXPECT(mla_workspace_bytes(64, 128, 4, &bytes) == TA_OK &&
               bytes == (size_t)4 * 64 * 128 * 513 * 4,
           "mla workspace");
    int n = 0;
    EXPECT(mla_split_heuristic(64, 128, 1, 8192, &n) == TA_OK && n >= 1 && n <= 128,
           "mla heuristic");
    for (int s = 0; s < 12; ++s)
        EXPECT(ta_status_string((ta_status)s) && strlen(ta_status_string((ta_status)s)) > 0,
               "status string %d", s);
    EXPECT(ta_version() >= 400, "version");
}

static void check_other_validation(void)
{
    /* mla_decode */
    EXPECT(mla_decode(P(0x10000000), P(0x18000000), P(0x20000000), P(0x30000000),
                      (float *)P(0x40000000), (float *)P(0x50000000), 2, 128, 1, 256, 256, 64,
                      0.04f, 2, P(0x60000000), 1u << 24, NULL) == TA_ERR_UNSUPPORTED,
           "mla Dl");
    EXPECT(mla_decode(NULL, P(0x18000000), P(0x20000000), P(0x30000000), (float *)P(0x40000000),
                      (float *)P(0x50000000), 2, 128, 1, 256, 512, 64, 0.04f, 2, P(0x60000000),
                      1u << 24, NULL) == TA_ERR_NULL_POINTER,
           "mla null");
    EXPECT(mla_decode(P(0x10000000), P(0x18000000), P(0x20000000), P(0x30000000),
                      (float *)P(0x40000000), (float *)P(0x50000000), 2, 128, 1, 256, 512, 64,
                      0.04f, 2, NULL, 0, NULL) == TA_ERR_WORKSPACE,
           "mla workspace");
    /* gemm_bf16 */
    EXPECT(gemm_bf16(P(0x10000000), P(0x30000000), P(0x50000000), 0, 200, 256, 128, NULL) ==
               TA_ERR_UNSUPPORTED,
           "gemm M");
    EXPECT(gemm_bf16(P(0x10000000), P(0x30000000), P(0x10000000 + 1024), 0, 256, 256, 128,
                     NULL) == TA_ERR_ALIASING,
           "gemm aliasing");
    EXPECT(gemm_bf16(P(0x10000000), P(0x30000000), P(0x50000000), 0, 256, 65536, 16384, NULL) ==
               TA_ERR_INVALID_SHAPE,
           "gemm 32-bit offsets");
    /* SSD */
    EXPECT(ssd_chunk_scan(P(0x10000000), P(0x12000000), (const float *)P(0x20000000),
                          (const float *)P(0x13000000), (const float *)P(0x14000000),
                          (const float *)P(0x30000000), (const float *)P(0x15000000),
                          (float *)P(0x40000000), 1, 300, 4, 2, 128, 128, 256, NULL) ==
               TA_ERR_UNSUPPORTED,
           "ssd scan headdim");
    EXPECT(ssd_chunk_state(P(0x10000000), P(0x11000000), (const float *)P(0x13000000),
                           (const float *)P(0x14000000), (float *)P(0x11000000 + 4096), 1, 300,
                           4, 2, 64, 128, 256, NULL) == TA_ERR_ALIASING,
           "ssd state aliasing");
    EXPECT(ssd_bmm_chunk(P(0x12000000), P(0x11000000), NULL, 1, 300, 2, 128, 256, NULL) ==
               TA_ERR_NULL_POINTER,
           "ssd bmm null");
    EXPECT(ssd_state_passing((const float *)P(0x30000000), (const float *)P(0x13000000),
                             (const float *)P(0x14000000), (float *)P(0x30000000 + 1024), NULL, 1,
                             300, 4, 64, 128, 256, NULL) == TA_ERR_ALIASING,
           "ssd passing aliasing");
}

int main(void)
{
    check_attn_validation();
    check_schedule();
    check_host_helpers();
    check_other_validation();
    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("abi_driver: all checks passed\n");
    return 0;
}
