/* Runs every oracle function on edge sizes and special values so that the
 * oracle, built with AddressSanitizer and UndefinedBehaviorSanitizer, is
 * checked for out-of-bounds accesses and undefined behaviour.  Each buffer
 * is allocated with exactly the size the oracle's contract gives it. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint16_t orc_bf16_rne(float f);
void orc_bf16_rne_array(const float *x, uint16_t *out, size_t n);
void orc_bf16_to_f32_array(const uint16_t *h, float *out, size_t n);
void orc_adam_step(float *p, float *m, float *v, const float *g, uint16_t *out, size_t n,
                   float lr, float b1, float b2, float eps, float wd, int64_t step, int adamw);
void orc_refresh(uint16_t *dst, const uint16_t *src, size_t count);
void orc_quantize_blockwise_i8(const uint16_t *x, size_t n, uint32_t block, int8_t *codes,
                               float *scales);
void orc_dequant_blockwise_i8(const int8_t *codes, const float *scales, size_t n, uint32_t block,
                              uint16_t *out);
void orc_dequant_gather_layer(const int8_t *const *codes, const float *const *scales,
                              uint32_t num_shards, size_t shard_elems, uint32_t block,
                              size_t layer_elems, uint16_t *out);
void orc_quantize_blockwise_i4(const float *x, size_t n, uint32_t block, uint8_t *codes,
                               float *scales);
void orc_unpack_i4(const uint8_t *codes, size_t n, int8_t *out);
void orc_dequant_reduce_i4(const uint8_t *const *codes, const float *const *scales,
                           uint32_t num_src, size_t n, uint32_t block, float scale_out, float *out);

static uint32_t rng_state = 12345u;
static uint32_t rnd(void)
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 17;
    rng_state ^= rng_state << 5;
    return rng_state;
}

static float rnd_value(void)
{
    uint32_t r = rnd();
    switch (r % 16) {
    case 0: return 0.0f;
    case 1: return INFINITY;
    case 2: return NAN;
    case 3: return 1e-40f;
    case 4: return -3e38f;
    default: return ((float)(int32_t)(r >> 8) / 8388608.0f) * 0.02f;
    }
}

static void *alloc(size_t bytes) { return malloc(bytes ? bytes : 1); }

int main(void)
{
    const size_t sizes[] = {0, 1, 2, 3, 7, 63, 64, 65, 255, 256, 257, 511, 4097};
    const uint32_t blocks[] = {64, 256, 4096};
    for (size_t si = 0; si < sizeof sizes / sizeof sizes[0]; si++) {
        const size_t n = sizes[si];
        float *f = alloc(n * 4), *p = alloc(n * 4), *m = alloc(n * 4), *v = alloc(n * 4);
        uint16_t *h = alloc(n * 2), *h2 = alloc(n * 2);
        for (size_t i = 0; i < n; i++) {
            f[i] = rnd_value();
            p[i] = rnd_value();
            m[i] = 0.0f;
            v[i] = 0.0f;
        }
        orc_bf16_rne_array(f, h, n);
        orc_bf16_to_f32_array(h, p, n);
        orc_adam_step(p, m, v, f, h2, n, 1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 3, 1);
        orc_adam_step(p, m, v, f, NULL, n, 1e-4f, 0.9f, 0.95f, 0.0f, 0.1f, 1, 0);
        orc_refresh(h2, h, n);
        for (size_t bi = 0; bi < sizeof blocks / sizeof blocks[0]; bi++) {
            const uint32_t B = blocks[bi];
            const size_t nb = (n + B - 1) / B;
            int8_t *c8 = alloc(n);
            float *sc = alloc(nb * 4);
            orc_quantize_blockwise_i8(h, n, B, c8, sc);
            orc_dequant_blockwise_i8(c8, sc, n, B, h2);
            const int8_t *cs[3] = {c8, c8, c8};
            const float *ss[3] = {sc, sc, sc};
            if (n) {
                uint16_t *lay = alloc(3 * n * 2);
                orc_dequant_gather_layer(cs, ss, 3, n, B, 3 * n, lay);
                orc_dequant_gather_layer(cs, ss, 3, n, B, 2 * n + 1, lay);
                free(lay);
            }
            uint8_t *c4 = alloc((n + 1) / 2);
            orc_quantize_blockwise_i4(f, n, B, c4, sc);
            int8_t *u = alloc(n);
            orc_unpack_i4(c4, n, u);
            const uint8_t *c4s[2] = {c4, c4};
            const float *s4s[2] = {sc, sc};
            orc_dequant_reduce_i4(c4s, s4s, 2, n, B, 0.5f, p);
            free(c8);
            free(sc);
            free(c4);
            free(u);
        }
        free(f);
        free(p);
        free(m);
        free(v);
        free(h);
        free(h2);
    }
    (void)orc_bf16_rne(1.0f);
    printf("sanitized oracle run ok\n");
    return 0;
}
