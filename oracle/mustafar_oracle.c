/*
 * mustafar_oracle.c -- plain, slow CPU reference of MUSTAFAR's decode hot path
 * (arxiv 2505.22913): per-token magnitude pruning of the K/V caches, the
 * bitmap-based compressed format, and decode attention over a dense local
 * window plus the compressed caches.
 *
 * TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may load this library. It shares no code, header, table or
 * helper with the GPU library and never calls it.
 *
 * Every function works on ONE (batch, kv-head) stream; callers loop over
 * streams.  Floating point is done in IEEE double.  The fp16 inputs are decoded
 * from their bit patterns by the binary16 definition (no compiler half type).
 *
 * Readings of the paper taken where it is silent:
 *   R1 pruning unit = one token of one head (d channels)           (Sec. 2)
 *   R2 kept count   = d - floor(s*d + 1/2), clamped to [0, d]
 *   R3 ranking      = larger |x| first; equal |x| -> lower channel first
 *   R4 bitmap bit i of tile t of a token = channel 64t+i is KEPT    (Sec. 3)
 *   R5 tiles are 64 consecutive channels of one token; tiles of a stream are
 *      ordered token-major (token j, tile t) -> index j*T + t
 *   R6 per-tile offset = exclusive prefix sum, over the stream, of the
 *      tile's non-zero count rounded up to a multiple of 8, in fp16 elements;
 *      pad slots hold +0.0                                         (Sec. 4.3)
 *   R7 attention scale = 1/sqrt(d) unless the caller gives one; no causal
 *      mask; pruned elements are zeros, every token is in the softmax
 *                                                         (Algorithm 1)
 * Parity pins for every function live in tests/test_oracle_pins.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_TILE 64 /* channels per compressed tile (Sec. 3: 1x64 tiles) */
#define ORACLE_PAD 8   /* non-zeros padded to a multiple of 8 (Sec. 4.3)   */

/* binary16 bit pattern -> double.  sign(1) | exponent(5, bias 15) | fraction(10) */
double oracle_half_to_double(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24); /* subnormal: f * 2^-14 * 2^-10 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25); /* (1 + f/2^10) * 2^(e-15) */
    return sign ? -v : v;
}

/* R2: number of channels kept per token for target sparsity s. */
int oracle_keep_count(int d, float sparsity)
{
    double pruned = floor((double)sparsity * (double)d + 0.5);
    int k = d - (int)pruned;
    if (k < 0)
        k = 0;
    if (k > d)
        k = d;
    return k;
}

/* ---------------------------------------------------------------------------
 * Per-token magnitude pruning (Sec. 2; the method the paper settles on for
 * both caches): keep the k elements of largest magnitude of one token's
 * d-vector and zero the rest.
 * ------------------------------------------------------------------------- */
typedef struct {
    double mag;
    int idx;
} ranked_t;

/* R3: descending magnitude, ascending channel among equal magnitudes. */
static int rank_cmp(const void* pa, const void* pb)
{
    const ranked_t* a = (const ranked_t*)pa;
    const ranked_t* b = (const ranked_t*)pb;
    if (a->mag > b->mag)
        return -1;
    if (a->mag < b->mag)
        return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

/* keep[c] = 1 if channel c of token x (d fp16 values) survives pruning to k. */
void oracle_prune_token(const uint16_t* x, int d, int k, uint8_t* keep)
{
    ranked_t* r = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)(d > 0 ? d : 1));
    for (int c = 0; c < d; ++c) {
        r[c].mag = fabs(oracle_half_to_double(x[c]));
        r[c].idx = c;
    }
    qsort(r, (size_t)d, sizeof(ranked_t), rank_cmp);
    memset(keep, 0, (size_t)d);
    for (int i = 0; i < k && i < d; ++i)
        keep[r[i].idx] = 1;
    free(r);
}

/* ---------------------------------------------------------------------------
 * Pruner variants that keep the same format.
 * ------------------------------------------------------------------------- */

/* 2:4 semi-structured pruning of one token (Appendix B): in every group of 4
 * consecutive channels the 2 of largest magnitude are kept (R3 ties: lower
 * channel first). d must be a multiple of 4. */
void oracle_prune_token_24(const uint16_t* x, int d, uint8_t* keep)
{
    for (int g = 0; g + 4 <= d; g += 4) {
        ranked_t r[4];
        for (int i = 0; i < 4; ++i) {
            r[i].mag = fabs(oracle_half_to_double(x[g + i]));
            r[i].idx = g + i;
        }
        qsort(r, 4, sizeof(ranked_t), rank_cmp);
        for (int i = 0; i < 4; ++i)
            keep[r[i].idx] = i < 2;
    }
}

/* Output-aware pruning of one key token (Sec. 2): the score of channel c is
 * |x_c| * w_c with w the channel weights (the L1 sum of the query vectors that
 * will attend to the token); the k channels of largest score are kept, ties
 * to the lower channel. The score is the fp32 product of |x_c| (exact in fp32)
 * and w_c, rounded once: the selection is decided in the precision the GPU
 * decides it in. */
void oracle_prune_token_scored(const uint16_t* x, const float* w, int d, int k, uint8_t* keep)
{
    ranked_t* r = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)(d > 0 ? d : 1));
    for (int c = 0; c < d; ++c) {
        const float mag = (float)fabs(oracle_half_to_double(x[c]));
        const float score = mag * w[c];
        r[c].mag = (double)score;
        r[c].idx = c;
    }
    qsort(r, (size_t)d, sizeof(ranked_t), rank_cmp);
    memset(keep, 0, (size_t)d);
    for (int i = 0; i < k && i < d; ++i)
        keep[r[i].idx] = 1;
    free(r);
}

/* Per-channel pruning of one group of n consecutive tokens of a stream
 * (Sec. 2, value-cache study: every channel is pruned to the target sparsity
 * within groups of 32 tokens). For each channel c the k of the n tokens with
 * the largest key are kept; equal keys go to the lower token. The key is
 * |x_jc| in the magnitude form (w NULL); in the output-aware form it is the
 * fp32 product |x_jc| * w_j, rounded once, where w_j >= 0 is the attention
 * probability mass token j received (summed over its queries). The selection is
 * thus decided in the precision the GPU decides it in.
 * x, keep: [n][d]. */
void oracle_prune_channel_group(const uint16_t* x, const float* w, int n, int d, int k,
                                uint8_t* keep)
{
    ranked_t* r = (ranked_t*)malloc(sizeof(ranked_t) * (size_t)(n > 0 ? n : 1));
    for (int c = 0; c < d; ++c) {
        for (int j = 0; j < n; ++j) {
            const double mag = fabs(oracle_half_to_double(x[(int64_t)j * d + c]));
            if (w) {
                const float score = (float)mag * w[j];
                r[j].mag = (double)score;
            } else {
                r[j].mag = mag;
            }
            r[j].idx = j;
        }
        qsort(r, (size_t)n, sizeof(ranked_t), rank_cmp);
        for (int j = 0; j < n; ++j)
            keep[(int64_t)j * d + c] = 0;
        for (int i = 0; i < k && i < n; ++i)
            keep[(int64_t)r[i].idx * d + c] = 1;
    }
    free(r);
}

/* ---------------------------------------------------------------------------
 * Bitmap-based compressed format (Sec. 3; padding and offset overhead Sec. 4.3).
 * One stream = the tokens of one (batch, kv-head).  T = d/64 tiles per token.
 *   bitmaps[j*T+t] : 64-bit kept mask of channels 64t..64t+63 of token j
 *   offsets[j*T+t] : first fp16 element of that tile's packed non-zeros
 *   values[...]    : kept fp16 values in channel order, each tile zero-padded
 *                    to a multiple of 8 elements
 *   *stream_len    : total fp16 elements used by the stream
 * Returns 0, or -1 if d is not a multiple of 64, -2 if values_cap is too small.
 * ------------------------------------------------------------------------- */
/* The format of n_tokens tokens whose kept channels are given: keep_all
 * [n_tokens][d] (1 = kept). oracle_compress_stream is this after
 * oracle_prune_token; the pruner variants use it with their own masks. */
int oracle_encode_stream(const uint16_t* x, const uint8_t* keep_all, int n_tokens, int d,
                         uint64_t* bitmaps, uint32_t* offsets, uint16_t* values,
                         int64_t values_cap, uint32_t* stream_len)
{
    if (d <= 0 || d % ORACLE_TILE != 0)
        return -1;
    int T = d / ORACLE_TILE;
    int64_t pos = 0; /* running offset in fp16 elements */
    for (int j = 0; j < n_tokens; ++j) {
        const uint16_t* tok = x + (int64_t)j * d;
        const uint8_t* keep = keep_all + (int64_t)j * d;
        for (int t = 0; t < T; ++t) {
            uint64_t bm = 0;
            int count = 0;
            for (int i = 0; i < ORACLE_TILE; ++i)
                if (keep[t * ORACLE_TILE + i]) {
                    bm |= (uint64_t)1 << i;
                    ++count;
                }
            int padded = (count + ORACLE_PAD - 1) / ORACLE_PAD * ORACLE_PAD;
            if (pos + padded > values_cap)
                return -2;
            bitmaps[(int64_t)j * T + t] = bm;
            offsets[(int64_t)j * T + t] = (uint32_t)pos;
            int w = 0;
            for (int i = 0; i < ORACLE_TILE; ++i)
                if (keep[t * ORACLE_TILE + i])
                    values[pos + w++] = tok[t * ORACLE_TILE + i];
            for (; w < padded; ++w)
                values[pos + w] = 0x0000; /* R6: pad slots are +0.0 */
            pos += padded;
        }
    }
    *stream_len = (uint32_t)pos;
    return 0;
}

int oracle_compress_stream(const uint16_t* x, int n_tokens, int d, int k,
                           uint64_t* bitmaps, uint32_t* offsets, uint16_t* values,
                           int64_t values_cap, uint32_t* stream_len)
{
    if (d <= 0 || d % ORACLE_TILE != 0)
        return -1;
    uint8_t* keep = (uint8_t*)malloc((size_t)d * (size_t)(n_tokens > 0 ? n_tokens : 1));
    for (int j = 0; j < n_tokens; ++j)
        oracle_prune_token(x + (int64_t)j * d, d, k, keep + (int64_t)j * d);
    const int rc = oracle_encode_stream(x, keep, n_tokens, d, bitmaps, offsets, values, values_cap,
                                        stream_len);
    free(keep);
    return rc;
}

/* Inverse of the format: the zero-filled pruned cache, fp16 bits [n_tokens][d].
 * Element i of tile t is values[offset + (number of set bits below i)] when
 * bit i is set, else +0.0. */
int oracle_decompress_stream(const uint64_t* bitmaps, const uint32_t* offsets,
                             const uint16_t* values, int n_tokens, int d, uint16_t* x_out)
{
    if (d <= 0 || d % ORACLE_TILE != 0)
        return -1;
    int T = d / ORACLE_TILE;
    for (int j = 0; j < n_tokens; ++j)
        for (int t = 0; t < T; ++t) {
            uint64_t bm = bitmaps[(int64_t)j * T + t];
            uint32_t off = offsets[(int64_t)j * T + t];
            int seen = 0;
            for (int i = 0; i < ORACLE_TILE; ++i) {
                uint16_t v = 0x0000;
                if ((bm >> i) & 1)
                    v = values[off + seen++];
                x_out[(int64_t)j * d + t * ORACLE_TILE + i] = v;
            }
        }
    return 0;
}

/* The attention probabilities of Algorithm 1 for one kv-head: the softmax
 * over concat(S_C, S_L) of the scores scale * q_g . k_j, for each of the G
 * query heads. probs: [G][n_s + n_d] double. Output-aware per-channel value
 * pruning (Sec. 2) weighs value token j by the probability mass it receives. */
int oracle_attention_probs(const uint16_t* q, int G, int d, const uint16_t* kc, int n_s,
                           const uint16_t* kl, int n_d, double scale, double* probs)
{
    const int n_all = n_s + n_d; /* every token of concat(S_C, S_L) */
    if (n_all <= 0 || d <= 0 || G <= 0)
        return -1;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    for (int g = 0; g < G; ++g) {
        double* p = probs + (int64_t)g * n_all;
        for (int j = 0; j < n_all; ++j) {
            const uint16_t* kj = (j < n_s) ? kc + (int64_t)j * d : kl + (int64_t)(j - n_s) * d;
            double acc = 0.0;
            for (int c = 0; c < d; ++c)
                acc += oracle_half_to_double(q[(int64_t)g * d + c]) * oracle_half_to_double(kj[c]);
            p[j] = scale * acc;
        }
        double m = p[0];
        for (int j = 1; j < n_all; ++j)
            if (p[j] > m)
                m = p[j];
        double l = 0.0;
        for (int j = 0; j < n_all; ++j) {
            p[j] = exp(p[j] - m);
            l += p[j];
        }
        for (int j = 0; j < n_all; ++j)
            p[j] /= l;
    }
    return 0;
}

/* ---------------------------------------------------------------------------
 * Algorithm 1 (decode-phase attention with dense local and compressed caches)
 * for one kv-head and the G query heads that share it.
 *   q      : [G][d]        fp16 bits
 *   kc, vc : [n_s][d]      zero-filled pruned caches (from decompression)
 *   kl, vl : [n_d][d]      dense local window
 *   out    : [G][d]        double
 * Scores S = scale * q . k for the compressed tokens then the local ones
 * (concat(S_C, S_L)), softmax over all n_s + n_d scores, output
 * O = V_C S_C^T + V_L S_L^T.  scale <= 0 selects 1/sqrt(d).
 * ------------------------------------------------------------------------- */
int oracle_decode_attention(const uint16_t* q, int G, int d,
                            const uint16_t* kc, const uint16_t* vc, int n_s,
                            const uint16_t* kl, const uint16_t* vl, int n_d,
                            double scale, double* out)
{
    int n = n_s + n_d;
    if (n <= 0 || d <= 0 || G <= 0)
        return -1;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    double* s = (double*)malloc(sizeof(double) * (size_t)n);
    for (int g = 0; g < G; ++g) {
        const uint16_t* qg = q + (int64_t)g * d;
        /* scores of the compressed tokens, then of the local ones: concat(S_C, S_L) */
        for (int j = 0; j < n; ++j) {
            const uint16_t* kj = (j < n_s) ? kc + (int64_t)j * d : kl + (int64_t)(j - n_s) * d;
            double acc = 0.0;
            for (int c = 0; c < d; ++c)
                acc += oracle_half_to_double(qg[c]) * oracle_half_to_double(kj[c]);
            s[j] = scale * acc;
        }
        /* one softmax over the whole concatenation */
        double m = s[0];
        for (int j = 1; j < n; ++j)
            if (s[j] > m)
                m = s[j];
        double l = 0.0;
        for (int j = 0; j < n; ++j) {
            s[j] = exp(s[j] - m);
            l += s[j];
        }
        /* split back and O = V_C S_C^T + V_L S_L^T */
        for (int c = 0; c < d; ++c) {
            double o = 0.0;
            for (int j = 0; j < n; ++j) {
                const uint16_t* vj = (j < n_s) ? vc + (int64_t)j * d : vl + (int64_t)(j - n_s) * d;
                o += (s[j] / l) * oracle_half_to_double(vj[c]);
            }
            out[(int64_t)g * d + c] = o;
        }
    }
    free(s);
    return 0;
}
