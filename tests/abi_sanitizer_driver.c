/*
 * The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
 * (CPU only): every entry point of zpp.h is called on its validation paths
 * and on size-0 calls, the host-side pointer and event arrays allocated with
 * exactly the length the call is told, so a read past num_shards, num_src or
 * num_wait is caught.  Every case returns before any HIP call (a validation
 * error, or a size-0 call with no events), so the device addresses below are
 * never dereferenced and no device is needed.
 *
 * The library's zpp_api.hip is linked with stand-ins for the kernel launchers
 * (tests/abi_launch_stubs.cpp) that count their calls: the count must stay 0.
 *
 * Test infrastructure: built and run by tests/test_abi_sanitized.py.  Prints
 * "sanitized abi run ok" and exits 0 on success.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "zpp.h"

static int failures = 0;

/* calls that reached a kernel launcher (tests/abi_launch_stubs.cpp) */
extern int zpp_test_launches;

#define EXPECT_STATUS(call, want)                                                              \
    do {                                                                                       \
        const zpp_status s_ = (call);                                                          \
        if (s_ != (want)) {                                                                    \
            printf("%s:%d: %s returned %d, expected %d\n", __FILE__, __LINE__, #call, (int)s_, \
                   (int)(want));                                                               \
            failures++;                                                                        \
        }                                                                                      \
    } while (0)

/* Device addresses that are only compared and range-checked: region k starts
 * at 16 GiB + k * 1 GiB, so regions of up to 1 GiB never overlap. */
static void *dev(unsigned k) { return (void *)(uintptr_t)((16ull << 30) + ((uint64_t)k << 30)); }
static void *dev_off(unsigned k, size_t bytes) { return (char *)dev(k) + bytes; }
static hipEvent_t fake_event(unsigned k) { return (hipEvent_t)(uintptr_t)(0x1000u + 0x100u * k); }

static void *xmalloc(size_t bytes)
{
    void *p = malloc(bytes);
    if (!p) {
        printf("out of host memory\n");
        exit(2);
    }
    return p;
}

static zpp_adam_hparams good_hp(void)
{
    zpp_adam_hparams hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1, 1};
    return hp;
}

static void check_adam(void)
{
    zpp_adam_hparams hp = good_hp();
    float *p = dev(0), *m = dev(1), *v = dev(2), *g = dev(3);
    uint16_t *o = dev(4);
    const size_t n = 1000;
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, 0, &hp, NULL), ZPP_OK);
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, n, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_adam_partition_step(NULL, m, v, g, o, n, &hp, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, SIZE_MAX, &hp, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_adam_partition_step(dev_off(0, 2), m, v, g, o, n, &hp, NULL), ZPP_EALIGN);
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, dev_off(0, 4 * n - 4), o, n, &hp, NULL),
                  ZPP_EOVERLAP);
    zpp_adam_hparams bad = hp;
    bad.step = 0;
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, n, &bad, NULL), ZPP_EINVAL);
    bad = hp;
    bad.beta1 = 1.0f;
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, n, &bad, NULL), ZPP_EINVAL);
    bad = hp;
    bad.lr = NAN;
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, n, &bad, NULL), ZPP_EINVAL);
    bad = hp;
    bad.eps = -1.0f;
    EXPECT_STATUS(zpp_adam_partition_step(p, m, v, g, o, n, &bad, NULL), ZPP_EINVAL);
}

static void check_fused(void)
{
    zpp_adam_hparams hp = good_hp();
    float *p = dev(0), *m = dev(1), *v = dev(2), *g = dev(3), *sc = dev(7);
    uint16_t *pr = dev(4), *se = dev(5);
    int8_t *c = dev(6);
    const size_t n = 1000;
    EXPECT_STATUS(zpp_adam_step_refresh_quantize(p, m, v, g, pr, se, c, sc, 0, 256, &hp, NULL,
                                                 NULL, NULL),
                  ZPP_OK);
    EXPECT_STATUS(zpp_adam_step_refresh_quantize(p, m, v, g, pr, se, c, sc, n, 100, &hp, NULL,
                                                 NULL, NULL),
                  ZPP_EINVAL);
    EXPECT_STATUS(zpp_adam_step_refresh_quantize(p, m, v, g, pr, dev_off(5, 1), c, sc, n, 256, &hp,
                                                 NULL, NULL, NULL),
                  ZPP_EALIGN);
    EXPECT_STATUS(zpp_adam_step_refresh_quantize(p, m, v, g, pr, se, (int8_t *)dev_off(7, 0), sc,
                                                 n, 256, &hp, NULL, NULL, NULL),
                  ZPP_EOVERLAP);
    EXPECT_STATUS(zpp_adam_step_refresh_quantize(p, m, v, g, pr, se, NULL, sc, n, 256, &hp, NULL,
                                                 NULL, NULL),
                  ZPP_EINVAL);
}

static void check_refresh_and_quantize(void)
{
    uint16_t *a = dev(0), *b = dev(1);
    EXPECT_STATUS(zpp_refresh_secondary(a, b, 0, NULL, NULL, NULL), ZPP_OK);
    EXPECT_STATUS(zpp_refresh_secondary(NULL, b, 16, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_refresh_secondary(a, dev_off(0, 30), 16, NULL, NULL, NULL), ZPP_EOVERLAP);
    EXPECT_STATUS(zpp_refresh_secondary(dev_off(0, 1), b, 16, NULL, NULL, NULL), ZPP_EALIGN);
    EXPECT_STATUS(zpp_refresh_secondary(a, b, SIZE_MAX / 8, NULL, NULL, NULL), ZPP_EINVAL);

    int8_t *c = dev(2);
    float *s = dev(3);
    EXPECT_STATUS(zpp_quantize_blockwise_i8(a, 0, 256, c, s, NULL, NULL, NULL), ZPP_OK);
    EXPECT_STATUS(zpp_quantize_blockwise_i8(a, 1000, 96, c, s, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_quantize_blockwise_i8(a, 1000, 8192, c, s, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_quantize_blockwise_i8(a, 1000, 256, c, dev_off(3, 2), NULL, NULL, NULL),
                  ZPP_EALIGN);
    EXPECT_STATUS(zpp_quantize_blockwise_i8(a, 1000, 256, (int8_t *)dev_off(0, 1000), s, NULL,
                                            NULL, NULL),
                  ZPP_EOVERLAP);

    uint16_t *sec = dev(6);
    EXPECT_STATUS(zpp_refresh_quantize_i8(sec, a, 0, 256, c, s, NULL, NULL, NULL), ZPP_OK);
    EXPECT_STATUS(zpp_refresh_quantize_i8(sec, a, 1000, 4160, c, s, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_refresh_quantize_i8(NULL, a, 1000, 256, c, s, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_refresh_quantize_i8(sec, a, 1000, 256, c, dev_off(3, 2), NULL, NULL, NULL),
                  ZPP_EALIGN);
    EXPECT_STATUS(zpp_refresh_quantize_i8(dev_off(0, 1000), a, 1000, 256, c, s, NULL, NULL, NULL),
                  ZPP_EOVERLAP);

    float *x = dev(4);
    uint8_t *c4 = dev(5);
    EXPECT_STATUS(zpp_quantize_blockwise_i4(x, 0, 256, c4, s, NULL, NULL, NULL), ZPP_OK);
    EXPECT_STATUS(zpp_quantize_blockwise_i4(x, 1000, 32, c4, s, NULL, NULL, NULL), ZPP_EINVAL);
    EXPECT_STATUS(zpp_quantize_blockwise_i4(dev_off(4, 1), 1000, 256, c4, s, NULL, NULL, NULL),
                  ZPP_EALIGN);
    EXPECT_STATUS(zpp_quantize_blockwise_i4(x, 1000, 256, (uint8_t *)dev_off(4, 3996), s, NULL,
                                            NULL, NULL),
                  ZPP_EOVERLAP);
}

static void check_gather(void)
{
    for (unsigned P = 1; P <= ZPP_MAX_SHARDS; P = P < 8 ? P + 1 : P * 2) {
        const size_t s = 4096;
        const int8_t **codes = xmalloc(P * sizeof *codes);
        const float **scales = xmalloc(P * sizeof *scales);
        for (unsigned j = 0; j < P; ++j) {
            codes[j] = dev_off(1, (size_t)j * 2 * s);
            scales[j] = dev_off(1, (size_t)j * 2 * s + s);
        }
        const unsigned W = P < 4 ? P : 4;
        hipEvent_t *waits = xmalloc(W * sizeof *waits);
        for (unsigned w = 0; w < W; ++w)
            waits[w] = fake_event(w);
        uint16_t *out = dev(0);
        /* size 0, no events: every shard pointer is read, nothing is enqueued */
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, 0, out, NULL, NULL, 0,
                                               NULL),
                      ZPP_OK);
        /* every event and every shard pointer is read before the missing output is found */
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s, NULL, NULL, waits,
                                               W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s + 1, out, NULL,
                                               NULL, 0, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, 0, 256, 0, out, NULL, NULL, 0,
                                               NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s,
                                               (uint16_t *)dev_off(1, 2 * s * (P - 1) + 2),
                                               NULL, NULL, 0, NULL),
                      ZPP_EOVERLAP);
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s, out, NULL, waits,
                                               ZPP_MAX_WAIT_EVENTS + 1, NULL),
                      ZPP_EINVAL);
        const float *keep = scales[P - 1];
        scales[P - 1] = dev_off(2, 2);
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s, out, NULL, NULL, 0,
                                               NULL),
                      ZPP_EALIGN);
        scales[P - 1] = keep;
        const int8_t *keep_c = codes[P - 1];
        codes[P - 1] = NULL;
        EXPECT_STATUS(zpp_dequant_gather_layer(codes, scales, P, s, 256, P * s, out, NULL, NULL, 0,
                                               NULL),
                      ZPP_EINVAL);
        codes[P - 1] = keep_c;
        free(codes);
        free(scales);
        free(waits);
    }
    EXPECT_STATUS(zpp_dequant_gather_layer(NULL, NULL, 0, 4096, 256, 0, dev(0), NULL, NULL, 0,
                                           NULL),
                  ZPP_EINVAL);
}

/* The int4 sources of the reduce and the two receive entries: P exact-length
 * arrays, source q's codes and scales in region 8 + q. */
struct Sources {
    const uint8_t **codes;
    const float **scales;
    hipEvent_t *waits;
    unsigned W;
};

static struct Sources make_sources(unsigned P, size_t n)
{
    struct Sources s;
    s.codes = xmalloc(P * sizeof *s.codes);
    s.scales = xmalloc(P * sizeof *s.scales);
    for (unsigned q = 0; q < P; ++q) {
        s.codes[q] = dev(8 + q % 8);
        s.scales[q] = dev_off(8 + q % 8, (n + 1) / 2 + 256);
    }
    s.W = P < 3 ? P : 3;
    s.waits = xmalloc(s.W * sizeof *s.waits);
    for (unsigned w = 0; w < s.W; ++w)
        s.waits[w] = fake_event(w);
    return s;
}

static void free_sources(struct Sources *s)
{
    free(s->codes);
    free(s->scales);
    free(s->waits);
}

static void check_qgz_receive(void)
{
    zpp_adam_hparams hp = good_hp();
    const size_t n = 1000;
    float *p = dev(0), *m = dev(1), *v = dev(2), *red = dev(3), *sc8 = dev(7);
    uint16_t *pr = dev(4), *se = dev(5);
    int8_t *c8 = dev(6);
    for (unsigned P = 1; P <= ZPP_MAX_SHARDS; P = P < 8 ? P + 1 : P * 2) {
        struct Sources s = make_sources(P, n);
        /* dequant-reduce */
        EXPECT_STATUS(zpp_dequant_reduce_i4(s.codes, s.scales, P, 0, 256, 0.5f, red, NULL, NULL, 0,
                                            NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_dequant_reduce_i4(s.codes, s.scales, P, n, 256, 0.5f, NULL, NULL,
                                            s.waits, s.W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_reduce_i4(s.codes, s.scales, P, n, 256, INFINITY, red, NULL,
                                            NULL, 0, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_reduce_i4(s.codes, s.scales, P, n, 256, 0.5f,
                                            (float *)dev_off(8 + (P - 1) % 8, 100), NULL, NULL, 0,
                                            NULL),
                      ZPP_EOVERLAP);
        /* the receive step */
        EXPECT_STATUS(zpp_qgz_receive_adam_step(p, m, v, s.codes, s.scales, P, 256, 0.5f, pr, 0,
                                                &hp, NULL, NULL, 0, NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_qgz_receive_adam_step(p, m, v, s.codes, s.scales, P, 256, 0.5f, NULL, n,
                                                &hp, NULL, s.waits, s.W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_adam_step(p, m, v, s.codes, s.scales, P, 256, 0.5f, pr, n,
                                                NULL, NULL, NULL, 0, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_adam_step((float *)dev_off(8 + (P - 1) % 8, 0), m, v,
                                                s.codes, s.scales, P, 256, 0.5f, pr, n, &hp, NULL,
                                                NULL, 0, NULL),
                      ZPP_EOVERLAP);
        /* the single receive pass */
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize(p, m, v, s.codes, s.scales, P, 256,
                                                            0.5f, pr, se, c8, sc8, 0, 256, &hp,
                                                            NULL, NULL, 0, NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize(p, m, v, s.codes, s.scales, P, 256,
                                                            0.5f, pr, se, NULL, sc8, n, 256, &hp,
                                                            NULL, s.waits, s.W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize(p, m, v, s.codes, s.scales, P, 48,
                                                            0.5f, pr, se, c8, sc8, n, 256, &hp,
                                                            NULL, NULL, 0, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize(
                          p, m, v, s.codes, s.scales, P, 256, 0.5f, pr, se, c8,
                          (float *)dev_off(8 + (P - 1) % 8, (n + 1) / 2 + 256), n, 256, &hp, NULL,
                          NULL, 0, NULL),
                      ZPP_EOVERLAP);
        free_sources(&s);
    }
    struct Sources s = make_sources(1, n);
    EXPECT_STATUS(zpp_dequant_reduce_i4(s.codes, s.scales, 0, n, 256, 0.5f, red, NULL, NULL, 0,
                                        NULL),
                  ZPP_EINVAL);
    EXPECT_STATUS(zpp_qgz_receive_adam_step(p, m, v, s.codes, s.scales, ZPP_MAX_SHARDS + 1, 256,
                                            0.5f, pr, n, &hp, NULL, NULL, 0, NULL),
                  ZPP_EINVAL);
    EXPECT_STATUS(zpp_qgz_receive_adam_step(p, m, v, NULL, s.scales, 1, 256, 0.5f, pr, n, &hp,
                                            NULL, NULL, 0, NULL),
                  ZPP_EINVAL);
    free_sources(&s);
}

static void check_interleaved(void)
{
    zpp_adam_hparams hp = good_hp();
    const size_t n = 1000;
    float *p = dev(0), *m = dev(1), *v = dev(2), *x = dev(3), *sc8 = dev(7), *is = dev(9);
    uint16_t *pr = dev(4), *se = dev(5);
    int8_t *c8 = dev(6);
    uint8_t *ic = dev(8);
    for (unsigned P = 1; P <= ZPP_MAX_SHARDS; P = P < 8 ? P + 1 : P * 2) {
        const unsigned W = P < 3 ? P : 3;
        hipEvent_t *waits = xmalloc(W * sizeof *waits);
        for (unsigned w = 0; w < W; ++w)
            waits[w] = fake_event(w);
        EXPECT_STATUS(zpp_quantize_blockwise_i4_interleaved(x, 0, 256, P - 1, P, ic, is, NULL, NULL,
                                                            NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_quantize_blockwise_i4_interleaved(x, n, 256, P, P, ic, is, NULL, NULL,
                                                            NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_quantize_blockwise_i4_interleaved(x, n, 256, 0, P, (uint8_t *)dev_off(3, 8),
                                                            is, NULL, NULL, NULL),
                      ZPP_EOVERLAP);
        EXPECT_STATUS(zpp_dequant_reduce_i4_interleaved(ic, is, P, 0, 256, 0.5f, NULL, NULL, NULL,
                                                        0, NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_dequant_reduce_i4_interleaved(ic, is, P, n, 256, 0.5f, NULL, NULL, waits,
                                                        W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_dequant_reduce_i4_interleaved(ic, is, P, n, 256, 0.5f,
                                                        (float *)dev_off(9, 0), NULL, NULL, 0,
                                                        NULL),
                      ZPP_EOVERLAP);
        EXPECT_STATUS(zpp_qgz_receive_adam_step_interleaved(p, m, v, ic, is, P, 256, 0.5f, pr, 0, &hp,
                                                            NULL, NULL, 0, NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_qgz_receive_adam_step_interleaved(p, m, v, ic, is, P, 256, 0.5f, NULL, n,
                                                            &hp, NULL, waits, W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_adam_step_interleaved(p, m, v, (uint8_t *)dev_off(0, 16), is,
                                                            P, 256, 0.5f, pr, n, &hp, NULL, NULL,
                                                            0, NULL),
                      ZPP_EOVERLAP);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize_interleaved(
                          p, m, v, ic, is, P, 256, 0.5f, pr, se, c8, sc8, 0, 256, &hp, NULL, NULL,
                          0, NULL),
                      ZPP_OK);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize_interleaved(
                          p, m, v, ic, is, P, 256, 0.5f, pr, se, NULL, sc8, n, 256, &hp, NULL,
                          waits, W, NULL),
                      ZPP_EINVAL);
        EXPECT_STATUS(zpp_qgz_receive_step_refresh_quantize_interleaved(
                          p, m, v, ic, (float *)dev_off(7, 0), P, 256, 0.5f, pr, se, c8, sc8, n,
                          256, &hp, NULL, NULL, 0, NULL),
                      ZPP_EOVERLAP);
        free(waits);
    }
    EXPECT_STATUS(zpp_qgz_receive_adam_step_interleaved(p, m, v, ic, is, 0, 256, 0.5f, pr, n, &hp,
                                                        NULL, NULL, 0, NULL),
                  ZPP_EINVAL);
    EXPECT_STATUS(zpp_qgz_receive_adam_step_interleaved(p, m, v, ic, is, 8, 256, 0.5f, pr,
                                                        SIZE_MAX / 16 / 8 + 1, &hp, NULL, NULL, 0,
                                                        NULL),
                  ZPP_EINVAL);
}

static void check_strings(void)
{
    const int all[] = {ZPP_OK, ZPP_EINVAL, ZPP_EALIGN, ZPP_EOVERLAP, ZPP_EHIP, 99, -1};
    for (size_t k = 0; k < sizeof all / sizeof all[0]; ++k) {
        const char *t = zpp_status_string(all[k]);
        if (!t || !*t) {
            printf("status %d has no string\n", all[k]);
            failures++;
        }
    }
    if (strcmp(zpp_status_string(99), "unknown status") != 0) {
        printf("status 99 is not reported as unknown\n");
        failures++;
    }
    (void)zpp_last_hip_error();
}

int main(void)
{
    check_adam();
    check_fused();
    check_refresh_and_quantize();
    check_gather();
    check_qgz_receive();
    check_interleaved();
    check_strings();
    if (zpp_test_launches) {
        printf("%d case(s) got past validation to a kernel launch\n", zpp_test_launches);
        failures++;
    }
    if (failures) {
        printf("sanitized abi run FAILED (%d checks)\n", failures);
        return 1;
    }
    printf("sanitized abi run ok\n");
    return 0;
}
