/* Drives every function of oracle/mustafar_oracle.c over random and edge-case
 * inputs (ties, +-0, subnormals, all kept counts, every head size) with buffers
 * of exactly the sizes the functions are documented to use, so that an
 * AddressSanitizer / UndefinedBehaviorSanitizer build catches any access out
 * of bounds or undefined operation. Prints "oracle harness ok" on success;
 * also checks decompress(compress(x)) against the kept values. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

double oracle_half_to_double(uint16_t h);
int oracle_keep_count(int d, float sparsity);
void oracle_prune_token(const uint16_t* x, int d, int k, uint8_t* keep);
void oracle_prune_token_24(const uint16_t* x, int d, uint8_t* keep);
void oracle_prune_token_scored(const uint16_t* x, const float* w, int d, int k, uint8_t* keep);
void oracle_prune_channel_group(const uint16_t* x, const float* w, int n, int d, int k, uint8_t* keep);
int oracle_encode_stream(const uint16_t* x, const uint8_t* keep_all, int n_tokens, int d,
                         uint64_t* bitmaps, uint32_t* offsets, uint16_t* values, int64_t values_cap,
                         uint32_t* stream_len);
int oracle_compress_stream(const uint16_t* x, int n_tokens, int d, int k, uint64_t* bitmaps,
                           uint32_t* offsets, uint16_t* values, int64_t values_cap, uint32_t* stream_len);
int oracle_decompress_stream(const uint64_t* bitmaps, const uint32_t* offsets, const uint16_t* values,
                             int n_tokens, int d, uint16_t* x_out);
int oracle_attention_probs(const uint16_t* q, int G, int d, const uint16_t* kc, int n_s,
                           const uint16_t* kl, int n_d, double scale, double* probs);
int oracle_decode_attention(const uint16_t* q, int G, int d, const uint16_t* kc, const uint16_t* vc,
                            int n_s, const uint16_t* kl, const uint16_t* vl, int n_d, double scale,
                            double* out);

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (uint32_t)(rng >> 11);
}

/* Finite fp16 bit patterns: normals, subnormals, +-0 and repeated magnitudes. */
static uint16_t rand_half(int ties) {
    const uint32_t r = next_u32();
    const uint16_t sign = (uint16_t)((r & 1u) << 15);
    if (ties) {
        static const uint16_t mags[] = {0x0000, 0x0001, 0x03ff, 0x3800, 0x3c00, 0x3c00, 0x4000};
        return (uint16_t)(sign | mags[(r >> 1) % 7]);
    }
    uint16_t exp = (uint16_t)((r >> 1) % 31); /* 0..30: never inf / nan */
    return (uint16_t)(sign | (exp << 10) | ((r >> 6) & 0x3ff));
}

static void* xmalloc(size_t n) {
    void* p = malloc(n ? n : 1);
    if (!p) { fprintf(stderr, "out of memory\n"); exit(2); }
    return p;
}

static int token_max_elems(int d, int k) {
    const int T = d / 64;
    const int nonempty = k < T ? k : T;
    const int m = (k + 7 * nonempty) / 8 * 8;
    return m < d ? m : d;
}

int main(void) {
    static const int dims[] = {64, 128, 256};
    for (int di = 0; di < 3; ++di) {
        const int d = dims[di], T = d / 64;
        for (int ties = 0; ties < 2; ++ties) {
            for (int k = 0; k <= d; k += (k < 8 || k > d - 8) ? 1 : 13) {
                const int n = 1 + (int)(next_u32() % 40);
                uint16_t* x = xmalloc(sizeof(uint16_t) * (size_t)n * d);
                for (int i = 0; i < n * d; ++i) x[i] = rand_half(ties);
                const int64_t cap = (int64_t)n * token_max_elems(d, k);
                uint64_t* bm = xmalloc(sizeof(uint64_t) * (size_t)n * T);
                uint32_t* off = xmalloc(sizeof(uint32_t) * (size_t)n * T);
                uint16_t* val = xmalloc(sizeof(uint16_t) * (size_t)(cap > 0 ? cap : 1));
                uint32_t len = 0;
                if (oracle_compress_stream(x, n, d, k, bm, off, val, cap, &len) != 0) {
                    fprintf(stderr, "compress failed d=%d k=%d\n", d, k);
                    return 1;
                }
                uint16_t* back = xmalloc(sizeof(uint16_t) * (size_t)n * d);
                if (oracle_decompress_stream(bm, off, val, n, d, back) != 0) return 1;
                uint8_t* keep = xmalloc((size_t)d);
                for (int j = 0; j < n; ++j) {
                    oracle_prune_token(x + (size_t)j * d, d, k, keep);
                    for (int c = 0; c < d; ++c) {
                        const uint16_t want = keep[c] ? x[(size_t)j * d + c] : 0;
                        if (back[(size_t)j * d + c] != want) {
                            fprintf(stderr, "round trip differs d=%d k=%d token %d channel %d\n", d, k, j, c);
                            return 1;
                        }
                    }
                }
                /* pruner variants and the encoder on their masks */
                uint8_t* keep_all = xmalloc((size_t)n * d);
                float* w = xmalloc(sizeof(float) * (size_t)n * d);
                for (int i = 0; i < n * d; ++i) w[i] = (float)(next_u32() % 1000) / 64.0f;
                for (int j = 0; j < n; ++j) {
                    if (j % 2) oracle_prune_token_24(x + (size_t)j * d, d, keep_all + (size_t)j * d);
                    else oracle_prune_token_scored(x + (size_t)j * d, w + (size_t)j * d, d, k, keep_all + (size_t)j * d);
                }
                const int64_t vcap = (int64_t)n * d;
                uint16_t* v2 = xmalloc(sizeof(uint16_t) * (size_t)vcap);
                if (oracle_encode_stream(x, keep_all, n, d, bm, off, v2, vcap, &len) != 0) return 1;
                /* per-channel groups (any group length, with and without weights) */
                const int kg = (int)(next_u32() % (unsigned)(n + 1));
                uint8_t* gkeep = xmalloc((size_t)n * d);
                oracle_prune_channel_group(x, NULL, n, d, kg, gkeep);
                oracle_prune_channel_group(x, w, n, d, kg, gkeep);
                /* attention: G query heads over the pruned tokens and a window */
                const int G = 1 << (next_u32() % 4), nd = (int)(next_u32() % 5);
                uint16_t* q = xmalloc(sizeof(uint16_t) * (size_t)G * d);
                for (int i = 0; i < G * d; ++i) q[i] = (uint16_t)(rand_half(0) & 0xbbff); /* |q| < 2 */
                uint16_t* kl = xmalloc(sizeof(uint16_t) * (size_t)(nd > 0 ? nd : 1) * d);
                for (int i = 0; i < nd * d; ++i) kl[i] = (uint16_t)(rand_half(0) & 0xbbff);
                double* probs = xmalloc(sizeof(double) * (size_t)G * (n + nd));
                double* out = xmalloc(sizeof(double) * (size_t)G * d);
                uint16_t* small = xmalloc(sizeof(uint16_t) * (size_t)n * d);
                for (int i = 0; i < n * d; ++i) small[i] = (uint16_t)(back[i] & 0xbbff);
                if (oracle_attention_probs(q, G, d, small, n, kl, nd, 0.0, probs) != 0) return 1;
                if (oracle_decode_attention(q, G, d, small, small, n, kl, kl, nd, 0.0, out) != 0) return 1;
                free(x); free(bm); free(off); free(val); free(back); free(keep); free(keep_all);
                free(w); free(v2); free(gkeep); free(q); free(kl); free(probs); free(out); free(small);
            }
        }
    }
    /* sparsity edge cases of the kept count, and every fp16 pattern's value */
    for (int i = 0; i <= 1000; ++i) (void)oracle_keep_count(128, (float)i / 1000.0f);
    (void)oracle_keep_count(0, 0.5f);
    (void)oracle_keep_count(128, -1.0f);
    double s = 0.0;
    for (uint32_t h = 0; h < 65536; ++h)
        if (((h >> 10) & 31u) != 31u) s += oracle_half_to_double((uint16_t)h);
    printf("oracle harness ok (%g)\n", s);
    return 0;
}
