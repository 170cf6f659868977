/* Calls every entry point of include/mustafar.h whose validation is host-side,
 * with valid arguments (they run to their end: the launchers are stubs), with
 * each kind of invalid argument, and with extreme sizes (INT_MAX token counts,
 * huge batches, negative values), under AddressSanitizer and
 * UndefinedBehaviorSanitizer. Device pointers are fake aligned addresses that
 * nothing dereferences. Exits nonzero if a status differs from the expected
 * one; prints "abi harness ok" at the end. */
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "mustafar.h"

extern long mf_stub_launches;
static int failures = 0;

#define EXPECT(call, want)                                                              \
    do {                                                                                \
        const int got_ = (call);                                                        \
        if (got_ != (want)) {                                                           \
            fprintf(stderr, "%s:%d: %s -> %d, expected %d\n", __FILE__, __LINE__, #call, \
                    got_, (int)(want));                                                 \
            ++failures;                                                                 \
        }                                                                               \
    } while (0)

static void* P(uintptr_t a) { return (void*)a; }

static int init_cache(mustafar_ccache_t* c, int B, int H, int d, float s, int cap) {
    const int k = mustafar_keep_count(d, s);
    int64_t stride = mustafar_stream_capacity(d, k < 0 ? 0 : k, cap);
    if (stride < 8) stride = 8;
    stride = (stride + 7) / 8 * 8;
    return mustafar_ccache_init(c, P(0x100000), P(0x200000), P(0x300000), P(0x400000), B, H, d, s,
                                cap, stride);
}

int main(void) {
    mustafar_ccache_t K, V, G;
    /* sizes and counts */
    for (int d = -1; d <= 300; ++d)
        for (int s10 = -1; s10 <= 11; ++s10) {
            (void)mustafar_keep_count(d, s10 / 10.0f);
            (void)mustafar_token_max_elems(d, s10 * 12);
            (void)mustafar_stream_capacity(d, s10 * 12, INT_MAX);
            (void)mustafar_grouped_stream_capacity(d, s10 * 3, INT_MAX);
        }
    (void)mustafar_compress_workspace_bytes(INT_MAX, INT_MAX, INT_MAX);
    (void)mustafar_attn_workspace_bytes(INT_MAX, INT_MAX, 1, 256, INT_MAX, 0);
    (void)mustafar_attn_default_splits(INT_MAX, INT_MAX, 1, INT_MAX, MUSTAFAR_ATTN_SPARSE);
    /* kernel routes: every route steers the default splits, extreme sizes included */
    EXPECT(mustafar_attn_set_route(3), MUSTAFAR_EINVAL);
    EXPECT(mustafar_attn_set_route(-1), MUSTAFAR_EINVAL);
    for (int r = MUSTAFAR_ROUTE_DEFAULT; r <= MUSTAFAR_ROUTE_MATRIX_CORES; ++r) {
        EXPECT(mustafar_attn_set_route(r), MUSTAFAR_OK);
        EXPECT(mustafar_attn_route(), r);
        for (int g = 1; g <= 8; g *= 2) {
            (void)mustafar_attn_default_splits(INT_MAX, 8 * g, 8, INT_MAX, MUSTAFAR_ATTN_SPARSE);
            (void)mustafar_attn_default_splits(1, 8 * g, 8, 1, MUSTAFAR_ATTN_SPARSE);
            (void)mustafar_attn_workspace_bytes(INT_MAX, 8 * g, 8, 256, INT_MAX, 0);
        }
    }
    EXPECT(mustafar_attn_set_route(MUSTAFAR_ROUTE_DEFAULT), MUSTAFAR_OK);
    for (int st = -8; st <= 1; ++st) (void)strlen(mustafar_strerror(st));

    EXPECT(init_cache(&K, 2, 4, 128, 0.5f, 100), MUSTAFAR_OK);
    EXPECT(init_cache(&V, 2, 4, 128, 0.7f, 100), MUSTAFAR_OK);
    EXPECT(init_cache(&G, 2, 4, 128, 0.5f, INT_MAX), MUSTAFAR_EUNSUPPORTED); /* u32 offsets */
    EXPECT(mustafar_ccache_init(&G, P(0x100000), P(0x200000), P(0x300000), P(0x400000), 2, 4, 128, 0.7f,
                                96, 8), MUSTAFAR_EINVAL);  /* stride below the worst case */
    EXPECT(mustafar_ccache_init_grouped(&G, P(0x100000), P(0x200000), P(0x300000), P(0x400000), 2, 4,
                                        128, 0.7f, 96, mustafar_grouped_stream_capacity(128, 10, 96)),
           MUSTAFAR_OK);

    /* compression and appends */
    const size_t wsb = mustafar_compress_workspace_bytes(2, 4, 100);
    EXPECT(mustafar_prune_compress(&K, P(0x500000), 60, P(0x600000), wsb, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_prune_compress(&K, P(0x500000), 41, P(0x600000), wsb, NULL), MUSTAFAR_ECAPACITY);
    EXPECT(mustafar_prune_compress(&K, P(0x500000), INT_MAX, P(0x600000), wsb, NULL), MUSTAFAR_ECAPACITY);
    EXPECT(mustafar_prune_compress_bounded(&K, P(0x500000), 40, 0, P(0x600000), wsb, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_append(&K, P(0x500000), NULL), MUSTAFAR_ECAPACITY);
    K.n_tokens = 60;
    V.n_tokens = 60;
    EXPECT(mustafar_append_kv(&K, &V, P(0x500000), P(0x500040), NULL), MUSTAFAR_OK);
    EXPECT(mustafar_append_kv(&K, &K, P(0x500000), P(0x500040), NULL), MUSTAFAR_EINVAL);
    K.n_tokens = INT_MAX;   /* a corrupted descriptor is refused, not overflowed */
    EXPECT(mustafar_append(&K, P(0x500000), NULL), MUSTAFAR_EINVAL);
    K.n_tokens = 61;
    int32_t hk[4] = {64, 0, 32, 65};
    mustafar_prune_opts_t o = {MUSTAFAR_PRUNE_MAGNITUDE, hk, NULL};
    EXPECT(mustafar_prune_compress_ex(&K, P(0x500000), 4, &o, P(0x600000), wsb, NULL), MUSTAFAR_EINVAL);
    hk[3] = 1;
    EXPECT(mustafar_prune_compress_ex(&K, P(0x500000), 4, &o, P(0x600000), wsb, NULL), MUSTAFAR_OK);
    o.mode = MUSTAFAR_PRUNE_2_4;
    o.head_keep = NULL;
    EXPECT(mustafar_append_ex(&K, P(0x500000), &o, NULL), MUSTAFAR_OK);
    o.mode = MUSTAFAR_PRUNE_OUTPUT_AWARE;
    o.weights = (const float*)P(0x700000);
    EXPECT(mustafar_append_ex(&K, P(0x500000), &o, NULL), MUSTAFAR_OK);
    o.mode = MUSTAFAR_PRUNE_CHANNEL_OUTPUT_AWARE;
    EXPECT(mustafar_prune_compress_ex(&G, P(0x500000), 32, &o, P(0x600000), wsb, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_query_lookahead(P(0x500000), 2, 8, 4, INT_MAX, 128, 32, P(0x700000), NULL), MUSTAFAR_OK);
    EXPECT(mustafar_query_lookahead(P(0x500000), 2, 8, 3, 100, 128, 32, P(0x700000), NULL), MUSTAFAR_EINVAL);

    /* decode attention */
    K.n_tokens = V.n_tokens = 64;
    const size_t awb = mustafar_attn_workspace_bytes(2, 16, 4, 128, 64, 0);
    EXPECT(mustafar_sparse_decode_attn(P(0x500000), 2, 16, &K, &V, P(0x900000), P(0x980000), 32, 0.f,
                                       P(0x800000), 0, P(0xa00000), awb, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_sparse_decode_attn(P(0x500000), 2, 16, &K, &V, NULL, NULL, 0, 0.f, P(0x800000),
                                       INT_MAX, P(0xa00000), awb, NULL), MUSTAFAR_EINVAL);
    EXPECT(mustafar_sparse_decode_attn(P(0x500000), 2, 16, &K, &V, NULL, NULL, 0, 0.f, P(0x800000),
                                       -5, P(0xa00000), awb - 1, NULL), MUSTAFAR_EWORKSPACE);
    EXPECT(mustafar_sparse_decode_attn_static(P(0x500000), 2, 16, &K, &V, NULL, NULL, 0, 0.f,
                                              P(0x800000), 1 << 16, NULL), MUSTAFAR_ESCRATCH);
    EXPECT(mustafar_dense_decode_attn(P(0x500000), 2, 16, 4, P(0x900000), P(0x980000), INT_MAX, 128, 0.f,
                                      P(0x800000), 0, P(0xa00000), 64, NULL), MUSTAFAR_EINVAL);  /* > 2^30 */
    EXPECT(mustafar_dense_decode_attn(P(0x500000), 2, 16, 4, P(0x900000), P(0x980000), 1 << 30, 128, 0.f,
                                      P(0x800000), 0, P(0xa00000), 64, NULL), MUSTAFAR_EWORKSPACE);
    const size_t dwb = mustafar_attn_workspace_bytes(2, 16, 4, 128, 1000, 3);
    EXPECT(mustafar_dense_decode_attn(P(0x500000), 2, 16, 4, P(0x900000), P(0x980000), 1000, 128, 0.f,
                                      P(0x800000), 3, P(0xa00000), dwb, NULL), MUSTAFAR_OK);

    /* the window lifecycle */
    mustafar_window_t w;
    EXPECT(mustafar_window_init(&w, P(0xb00000), P(0xb80000), P(0xc00000), P(0xc00100), P(0xc00200), 2, 4,
                                128, 32, 0), MUSTAFAR_OK);
    mustafar_ccache_t Kw, Vw;
    EXPECT(init_cache(&Kw, 2, 4, 128, 0.5f, 200), MUSTAFAR_OK);
    EXPECT(init_cache(&Vw, 2, 4, 128, 0.7f, 200), MUSTAFAR_OK);
    const int32_t seq[2] = {100, 3};
    EXPECT(mustafar_window_prefill(&w, &Kw, &Vw, P(0x500000), P(0x580000), 100, seq, P(0x600000),
                                   mustafar_compress_workspace_bytes(1, 4, 100), NULL), MUSTAFAR_OK);
    for (int s = 0; s < 40; ++s) {
        EXPECT(mustafar_window_step(&w, &Kw, &Vw, P(0x500000), P(0x500400), P(0xc00300), NULL), MUSTAFAR_OK);
        EXPECT(mustafar_window_key_weights(P(0x500000), 2, 8, &w, P(0xc00300), (float*)P(0xd00000), NULL),
               MUSTAFAR_OK);
    }
    const size_t wab = mustafar_attn_workspace_bytes(2, 8, 4, 128, Kw.n_tokens, 0);
    EXPECT(mustafar_window_decode_attn(P(0x500000), 2, 8, &Kw, &Vw, &w, 0.f, P(0x800000), 0, P(0xa00000),
                                       wab, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_window_decode_attn_scores(P(0x500000), 2, 8, &Kw, &Vw, &w, NULL, (float*)P(0xd00000), 0.f,
                                              P(0x800000), 0, P(0xa00000), wab, NULL), MUSTAFAR_OK);
    EXPECT(mustafar_window_step_weighted(&w, &Kw, &Vw, P(0x500000), P(0x500400), NULL, (float*)P(0xd00000),
                                         NULL), MUSTAFAR_OK);
    mustafar_window_t wg;
    mustafar_ccache_t Kg;
    EXPECT(init_cache(&Kg, 2, 4, 128, 0.5f, 96), MUSTAFAR_OK);
    EXPECT(mustafar_ccache_init_grouped(&G, P(0x100000), P(0x200000), P(0x300000), P(0x400000), 2, 4,
                                        128, 0.7f, 96, mustafar_grouped_stream_capacity(128, 10, 96)),
           MUSTAFAR_OK);
    EXPECT(mustafar_window_init(&wg, P(0xb00000), P(0xb80000), P(0xc00000), P(0xc00100), P(0xc00200), 2, 4,
                                128, 64, 0), MUSTAFAR_OK);
    const int32_t gseq[2] = {70, 0};
    EXPECT(mustafar_window_prefill(&wg, &Kg, &G, P(0x500000), P(0x580000), 70, gseq, P(0x600000),
                                   mustafar_compress_workspace_bytes(1, 4, 70), NULL), MUSTAFAR_OK);
    for (int s = 0; s < 70; ++s) {
        const int st = mustafar_window_step_grouped(&wg, &Kg, &G, P(0x500000), P(0x500400), NULL,
                                                    (float*)P(0xd00000), NULL);
        if (st != MUSTAFAR_OK && st != MUSTAFAR_ECAPACITY) {
            fprintf(stderr, "grouped step %d -> %d\n", s, st);
            ++failures;
        }
    }
    if (failures) return 1;
    printf("abi harness ok (%ld launches stubbed)\n", mf_stub_launches);
    return 0;
}
