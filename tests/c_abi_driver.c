/*
 * The partition path driven from plain C through libzpp.so, with nothing but
 * the HIP runtime API around it: device buffers from hipMalloc, three
 * streams, caller-owned events, the four calls of one iteration in the order
 * of Algorithm 1 (Adam step -> refresh of the secondary copy -> qwZ
 * quantization -> dequantize-and-gather of the layer over P' shards), with
 * the gather ordered after the quantization by an event (the fix).  The
 * results are checked against the CPU oracle (liboracle.so), which runs the
 * same iteration on the same inputs on its own.  Then the qgZ receive fused
 * into the partition step (zpp_qgz_receive_adam_step) from int4 gradient
 * copies, against the dequantize-and-reduce followed by the step and against
 * the oracle, and the single receive pass that also writes the secondary
 * and its int8 quantization (zpp_qgz_receive_step_refresh_quantize) against
 * the same sequence and the oracle's quantization.  The same two receives
 * from one interleaved receive buffer (the int4 copies block by block, as
 * include/zpp.h lays them out), each copy written into its slots by
 * zpp_quantize_blockwise_i4_interleaved.  Also checks a few
 * validation errors of the ABI.
 *
 * Test infrastructure: built by the repository's build step, run by
 * tests/test_gpu_c_abi.py.  Prints "c abi ok" and exits 0 on success.
 *
 * Usage: c_abi_driver [n]    (n: elements of the rank partition)
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "zpp.h"

/* the oracle's C entry points (oracle/zpp_oracle.c) */
uint16_t orc_bf16_rne(float f);
void orc_adam_step(float *p, float *m, float *v, const float *g, uint16_t *out, size_t n,
                   float lr, float beta1, float beta2, float eps, float wd, int64_t step,
                   int adamw);
void orc_quantize_blockwise_i8(const uint16_t *x, size_t n, uint32_t block, int8_t *codes,
                               float *scales);
void orc_dequant_gather_layer(const int8_t *const *shard_codes, const float *const *shard_scales,
                              uint32_t num_shards, size_t shard_elems, uint32_t block,
                              size_t layer_elems, uint16_t *out);
void orc_quantize_blockwise_i4(const float *x, size_t n, uint32_t block, uint8_t *codes,
                               float *scales);
void orc_dequant_reduce_i4(const uint8_t *const *src_codes, const float *const *src_scales,
                           uint32_t num_src, size_t n, uint32_t block, float scale_out,
                           float *out);

#define B 256u
#define P2 4u

static int failures = 0;

#define HIP_OK(call)                                                                     \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess) {                                                          \
            fprintf(stderr, "%s:%d: %s -> %s\n", __FILE__, __LINE__, #call,              \
                    hipGetErrorString(e_));                                              \
            exit(2);                                                                     \
        }                                                                                \
    } while (0)

#define EXPECT(cond, ...)                                                                \
    do {                                                                                 \
        if (!(cond)) {                                                                   \
            fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__);                         \
            fprintf(stderr, __VA_ARGS__);                                                \
            fprintf(stderr, "\n");                                                       \
            failures++;                                                                  \
        }                                                                                \
    } while (0)

/* splitmix64: a counter-based generator for the synthetic inputs */
static uint64_t mix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* normal draws by Box-Muller from two uniform draws in (0, 1) */
static void fill_normal(float *x, size_t n, double std, uint64_t seed)
{
    const double two_pi = 6.283185307179586;
    for (size_t i = 0; i < n; i++) {
        const double u1 = ((double)(mix64(seed ^ (2 * i)) >> 11) + 0.5) * 0x1p-53;
        const double u2 = ((double)(mix64(seed ^ (2 * i + 1)) >> 11) + 0.5) * 0x1p-53;
        x[i] = (float)(std * sqrt(-2.0 * log(u1)) * cos(two_pi * u2));
    }
}

static void *dev_alloc(size_t bytes)
{
    void *p = NULL;
    HIP_OK(hipMalloc(&p, bytes ? bytes : 1));
    return p;
}

static double rel_err(double got, double ref, double floor_)
{
    if (got == ref)
        return 0.0;
    const double d = fabs(ref) > floor_ ? fabs(ref) : floor_;
    return fabs(got - ref) / d;
}

#define NSRC 4u

/* The qgZ receive fused into the partition step, from plain C: NSRC int4
 * copies of a gradient (quantized by the oracle, as the senders would),
 * uploaded on their own stream; the fused call waits on the upload's event.
 * Its state must equal, bit for bit, that of the dequantize-and-reduce
 * followed by the partition step, and match the oracle's. */
static void check_receive(size_t n, const float *p0, const zpp_adam_hparams *hp)
{
    const size_t nb = (n + B - 1) / B, nbytes = (n + 1) / 2;
    const float scale_out = 1.0f / NSRC;
    float *x = malloc(n * 4);
    const size_t half = B / 2, il_bytes = nb * NSRC * half, il_count = nb * NSRC;
    uint8_t *hil_c = calloc(il_bytes, 1);
    float *hil_s = calloc(il_count, 4);
    uint8_t *dil_c = dev_alloc(il_bytes);
    float *dil_s = dev_alloc(il_count * 4);
    float *dx[NSRC];
    uint8_t *hc[NSRC];
    float *hs[NSRC];
    const uint8_t *dc[NSRC];
    const float *ds[NSRC];
    hipStream_t up, st;
    HIP_OK(hipStreamCreateWithFlags(&up, hipStreamNonBlocking));
    HIP_OK(hipStreamCreateWithFlags(&st, hipStreamNonBlocking));
    for (unsigned q = 0; q < NSRC; q++) {
        fill_normal(x, n, 1e-3, 200 + q);
        hc[q] = malloc(nbytes);
        hs[q] = malloc(nb * 4);
        orc_quantize_blockwise_i4(x, n, B, hc[q], hs[q]);
        /* the interleaved layout built on the host from the oracle's copy */
        for (size_t k = 0; k < nb; k++) {
            const size_t len = nbytes - k * half < half ? nbytes - k * half : half;
            memcpy(hil_c + (k * NSRC + q) * half, hc[q] + k * half, len);
            hil_s[k * NSRC + q] = hs[q][k];
        }
        dx[q] = dev_alloc(n * 4);
        HIP_OK(hipMemcpy(dx[q], x, n * 4, hipMemcpyHostToDevice));
        uint8_t *c = dev_alloc(nbytes);
        float *sc = dev_alloc(nb * 4);
        HIP_OK(hipMemcpyAsync(c, hc[q], nbytes, hipMemcpyHostToDevice, up));
        HIP_OK(hipMemcpyAsync(sc, hs[q], nb * 4, hipMemcpyHostToDevice, up));
        dc[q] = c;
        ds[q] = sc;
    }
    hipEvent_t uploaded, done;
    HIP_OK(hipEventCreateWithFlags(&uploaded, hipEventDisableTiming));
    HIP_OK(hipEventCreateWithFlags(&done, hipEventDisableTiming));
    /* each copy quantized on the device into its slots of one interleaved buffer */
    HIP_OK(hipMemsetAsync(dil_c, 0, il_bytes, up));
    for (unsigned q = 0; q < NSRC; q++)
        EXPECT(zpp_quantize_blockwise_i4_interleaved(dx[q], n, B, q, NSRC, dil_c, dil_s, up, NULL,
                                                     NULL) == ZPP_OK,
               "interleaved int4 quantization of source %u", q);
    HIP_OK(hipEventRecord(uploaded, up));
    /* state 0: reduce then step; 1: the receive step; 2: the single pass;
     * 3 and 4: the same two from the interleaved buffer */
    float *d[5][3];
    uint16_t *dprim[5];
    for (int k = 0; k < 5; k++) {
        for (int a = 0; a < 3; a++) {
            d[k][a] = dev_alloc(n * 4);
            if (a == 0)
                HIP_OK(hipMemcpy(d[k][a], p0, n * 4, hipMemcpyHostToDevice));
            else
                HIP_OK(hipMemset(d[k][a], 0, n * 4));
        }
        dprim[k] = dev_alloc(n * 2);
    }
    float *dgrad = dev_alloc(n * 4), *dgrad_il = dev_alloc(n * 4);
    uint16_t *dsec = dev_alloc(n * 2);
    int8_t *dq8 = dev_alloc(n);
    float *ds8 = dev_alloc(nb * 4);
    uint16_t *dsec_il = dev_alloc(n * 2);
    int8_t *dq8_il = dev_alloc(n);
    float *ds8_il = dev_alloc(nb * 4);
    HIP_OK(hipDeviceSynchronize());
    /* the two-call sequence, then the fused call, both ordered after the upload */
    EXPECT(zpp_dequant_reduce_i4(dc, ds, NSRC, n, B, scale_out, dgrad, st, &uploaded, 1, NULL) ==
               ZPP_OK,
           "dequant-reduce");
    EXPECT(zpp_adam_partition_step(d[0][0], d[0][1], d[0][2], dgrad, dprim[0], n, hp, st) ==
               ZPP_OK,
           "adam from the reduced gradient");
    EXPECT(zpp_qgz_receive_adam_step(d[1][0], d[1][1], d[1][2], dc, ds, NSRC, B, scale_out,
                                     dprim[1], n, hp, st, &uploaded, 1, NULL) == ZPP_OK,
           "fused receive step");
    EXPECT(zpp_qgz_receive_step_refresh_quantize(d[2][0], d[2][1], d[2][2], dc, ds, NSRC, B,
                                                 scale_out, dprim[2], dsec, dq8, ds8, n, B, hp,
                                                 st, &uploaded, 1, NULL) == ZPP_OK,
           "single receive pass");
    EXPECT(zpp_dequant_reduce_i4_interleaved(dil_c, dil_s, NSRC, n, B, scale_out, dgrad_il, st,
                                             &uploaded, 1, NULL) == ZPP_OK,
           "dequant-reduce from the interleaved buffer");
    EXPECT(zpp_qgz_receive_adam_step_interleaved(d[3][0], d[3][1], d[3][2], dil_c, dil_s, NSRC,
                                                 B, scale_out, dprim[3], n, hp, st, &uploaded, 1,
                                                 NULL) == ZPP_OK,
           "receive step from the interleaved buffer");
    EXPECT(zpp_qgz_receive_step_refresh_quantize_interleaved(
               d[4][0], d[4][1], d[4][2], dil_c, dil_s, NSRC, B, scale_out, dprim[4], dsec_il,
               dq8_il, ds8_il, n, B, hp, st, &uploaded, 1, done) == ZPP_OK,
           "single receive pass from the interleaved buffer");
    HIP_OK(hipEventSynchronize(done));
    float *h[5][3], *hg = malloc(n * 4), *rg = malloc(n * 4), *hs8 = malloc(nb * 4),
          *rs8 = malloc(nb * 4);
    uint16_t *hp16[5], *hsec = malloc(n * 2), *hsec_il = malloc(n * 2);
    int8_t *hq8 = malloc(n), *rq8 = malloc(n), *hq8_il = malloc(n);
    float *hs8_il = malloc(nb * 4);
    uint8_t *gil_c = malloc(il_bytes);
    float *gil_s = malloc(il_count * 4);
    HIP_OK(hipMemcpy(gil_c, dil_c, il_bytes, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gil_s, dil_s, il_count * 4, hipMemcpyDeviceToHost));
    EXPECT(memcmp(gil_c, hil_c, il_bytes) == 0, "interleaved codes differ from the oracle's");
    EXPECT(memcmp(gil_s, hil_s, il_count * 4) == 0, "interleaved scales differ from the oracle's");
    HIP_OK(hipMemcpy(hsec_il, dsec_il, n * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hq8_il, dq8_il, n, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hs8_il, ds8_il, nb * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hsec, dsec, n * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hq8, dq8, n, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(hs8, ds8, nb * 4, hipMemcpyDeviceToHost));
    for (int k = 0; k < 5; k++) {
        for (int a = 0; a < 3; a++) {
            h[k][a] = malloc(n * 4);
            HIP_OK(hipMemcpy(h[k][a], d[k][a], n * 4, hipMemcpyDeviceToHost));
        }
        hp16[k] = malloc(n * 2);
        HIP_OK(hipMemcpy(hp16[k], dprim[k], n * 2, hipMemcpyDeviceToHost));
    }
    HIP_OK(hipMemcpy(hg, dgrad, n * 4, hipMemcpyDeviceToHost));
    float *hg_il = malloc(n * 4);
    HIP_OK(hipMemcpy(hg_il, dgrad_il, n * 4, hipMemcpyDeviceToHost));
    EXPECT(memcmp(hg_il, hg, n * 4) == 0, "interleaved dequant-reduce differs");
    for (int k = 1; k < 5; k++) {
        for (int a = 0; a < 3; a++)
            EXPECT(memcmp(h[0][a], h[k][a], n * 4) == 0, "receive %d: state array %d differs", k,
                   a);
        EXPECT(memcmp(hp16[0], hp16[k], n * 2) == 0, "receive %d: primary differs", k);
    }
    EXPECT(memcmp(hsec, hp16[0], n * 2) == 0, "single receive pass: secondary differs");
    EXPECT(memcmp(hsec_il, hp16[0], n * 2) == 0, "interleaved single pass: secondary differs");
    EXPECT(memcmp(hq8_il, hq8, n) == 0, "interleaved single pass: codes differ");
    EXPECT(memcmp(hs8_il, hs8, nb * 4) == 0, "interleaved single pass: scales differ");
    orc_quantize_blockwise_i8(hp16[0], n, B, rq8, rs8);
    EXPECT(memcmp(hq8, rq8, n) == 0, "single receive pass: codes differ from the oracle's");
    EXPECT(memcmp(hs8, rs8, nb * 4) == 0, "single receive pass: scales differ from the oracle's");
    orc_dequant_reduce_i4((const uint8_t *const *)hc, (const float *const *)hs, NSRC, n, B,
                          scale_out, rg);
    EXPECT(memcmp(hg, rg, n * 4) == 0, "reduced gradient differs from the oracle's");
    float *rp = malloc(n * 4), *rm = calloc(n, 4), *rv = calloc(n, 4);
    uint16_t *rprim = malloc(n * 2);
    memcpy(rp, p0, n * 4);
    orc_adam_step(rp, rm, rv, rg, rprim, n, hp->lr, hp->beta1, hp->beta2, hp->eps,
                  hp->weight_decay, hp->step, hp->adamw);
    double ep = 0, e;
    for (size_t i = 0; i < n; i++)
        if ((e = rel_err(h[1][0][i], rp[i], hp->lr)) > ep) ep = e;
    EXPECT(ep <= 1e-5, "fused receive master rel err %g", ep);
    printf("qgz receive step and single pass: %u sources, separate or interleaved, "
           "bit-identical to reduce + step, codes and scales equal to the oracle's, "
           "master rel err %.3g\n",
           NSRC, ep);
    HIP_OK(hipStreamDestroy(up));
    HIP_OK(hipStreamDestroy(st));
}

static void check_validation(void)
{
    zpp_adam_hparams hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1, 1};
    float *p = (float *)dev_alloc(64 * sizeof(float));
    uint16_t *h = (uint16_t *)dev_alloc(64 * sizeof(uint16_t));
    EXPECT(zpp_adam_partition_step(NULL, p, p, p, h, 16, &hp, NULL) == ZPP_EINVAL,
           "NULL master accepted");
    EXPECT(zpp_adam_partition_step(p, p + 16, p + 32, p + 48, h, 16, NULL, NULL) == ZPP_EINVAL,
           "NULL hparams accepted");
    EXPECT(zpp_adam_partition_step(p, p + 16, p + 32, p + 48, (uint16_t *)((char *)h + 1), 16,
                                   &hp, NULL) == ZPP_EALIGN,
           "odd bf16 pointer accepted");
    EXPECT(zpp_refresh_secondary(h, h + 8, 16, NULL, NULL, NULL) == ZPP_EOVERLAP,
           "overlapping refresh accepted");
    hp.step = 0;
    EXPECT(zpp_adam_partition_step(p, p + 16, p + 32, p + 48, h, 16, &hp, NULL) == ZPP_EINVAL,
           "step 0 accepted");
    EXPECT(zpp_quantize_blockwise_i8(h, 16, 100, (int8_t *)p, p + 32, NULL, NULL, NULL) ==
               ZPP_EINVAL,
           "block 100 accepted");
    EXPECT(zpp_refresh_secondary(h, h + 32, 0, NULL, NULL, NULL) == ZPP_OK,
           "empty refresh rejected");
    EXPECT(strlen(zpp_status_string(ZPP_EOVERLAP)) > 0, "no status string");
    HIP_OK(hipDeviceSynchronize());
    HIP_OK(hipFree(p));
    HIP_OK(hipFree(h));
}

int main(int argc, char **argv)
{
    const size_t n = argc > 1 ? (size_t)strtoull(argv[1], NULL, 10) : ((size_t)1 << 20) + 4096;
    const size_t s = n / B * B;                 /* shard of the layer: the first s codes */
    const size_t N = P2 * s - 777;              /* the layer ends inside the last shard */
    const size_t nb = (n + B - 1) / B;
    const zpp_adam_hparams hp = {1e-4f, 0.9f, 0.95f, 1e-8f, 0.1f, 1, 1};
    if (n < B || N <= (P2 - 1) * s) {
        fprintf(stderr, "n too small\n");
        return 2;
    }
    printf("c abi driver: n=%zu shard=%zu layer=%zu P'=%u\n", n, s, N, P2);
    fflush(stdout);

    /* host inputs */
    float *p = malloc(n * 4), *g = malloc(n * 4);
    fill_normal(p, n, 0.02, 11);
    fill_normal(g, n, 1e-3, 12);
    int8_t *peer_codes[P2];
    float *peer_scales[P2];
    float *wf = malloc(s * 4);
    uint16_t *wb = malloc(s * 2);
    for (unsigned j = 1; j < P2; j++) {
        fill_normal(wf, s, 0.02, 100 + j);
        for (size_t i = 0; i < s; i++)
            wb[i] = orc_bf16_rne(wf[i]);
        peer_codes[j] = malloc(s);
        peer_scales[j] = malloc(s / B * 4);
        orc_quantize_blockwise_i8(wb, s, B, peer_codes[j], peer_scales[j]);
    }

    /* device state */
    float *dp = dev_alloc(n * 4), *dm = dev_alloc(n * 4), *dv = dev_alloc(n * 4);
    float *dg = dev_alloc(n * 4);
    uint16_t *dprim = dev_alloc(n * 2), *dsec = dev_alloc(n * 2), *dout = dev_alloc(N * 2);
    int8_t *dcodes = dev_alloc(n);
    float *dscales = dev_alloc(nb * 4);
    const int8_t *gc[P2];
    const float *gs[P2];
    gc[0] = dcodes;
    gs[0] = dscales;
    for (unsigned j = 1; j < P2; j++) {
        int8_t *c = dev_alloc(s);
        float *sc = dev_alloc(s / B * 4);
        HIP_OK(hipMemcpy(c, peer_codes[j], s, hipMemcpyHostToDevice));
        HIP_OK(hipMemcpy(sc, peer_scales[j], s / B * 4, hipMemcpyHostToDevice));
        gc[j] = c;
        gs[j] = sc;
    }
    HIP_OK(hipMemcpy(dp, p, n * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dg, g, n * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemset(dm, 0, n * 4));
    HIP_OK(hipMemset(dv, 0, n * 4));
    HIP_OK(hipMemset(dsec, 0xFF, n * 2)); /* NaN poison: a stale read would show */
    HIP_OK(hipDeviceSynchronize());

    hipStream_t compute, copy, comm;
    HIP_OK(hipStreamCreateWithFlags(&compute, hipStreamNonBlocking));
    HIP_OK(hipStreamCreateWithFlags(&copy, hipStreamNonBlocking));
    HIP_OK(hipStreamCreateWithFlags(&comm, hipStreamNonBlocking));
    hipEvent_t ev_primary, ev_refresh, ev_quant, ev_gather;
    HIP_OK(hipEventCreateWithFlags(&ev_primary, hipEventDisableTiming));
    HIP_OK(hipEventCreateWithFlags(&ev_refresh, hipEventDisableTiming));
    HIP_OK(hipEventCreateWithFlags(&ev_quant, hipEventDisableTiming));
    HIP_OK(hipEventCreateWithFlags(&ev_gather, hipEventDisableTiming));

    /* one iteration: compute -> copy -> comm, ordered by events only */
    EXPECT(zpp_adam_partition_step(dp, dm, dv, dg, dprim, n, &hp, compute) == ZPP_OK, "adam");
    HIP_OK(hipEventRecord(ev_primary, compute));
    EXPECT(zpp_refresh_secondary(dsec, dprim, n, copy, ev_primary, ev_refresh) == ZPP_OK,
           "refresh");
    EXPECT(zpp_quantize_blockwise_i8(dsec, n, B, dcodes, dscales, copy, NULL, ev_quant) == ZPP_OK,
           "quantize");
    EXPECT(zpp_dequant_gather_layer(gc, gs, P2, s, B, N, dout, comm, &ev_quant, 1, ev_gather) ==
               ZPP_OK,
           "gather");
    HIP_OK(hipEventSynchronize(ev_gather));
    HIP_OK(hipDeviceSynchronize());

    float *rp = malloc(n * 4), *rm = calloc(n, 4), *rv = calloc(n, 4);
    uint16_t *rprim = malloc(n * 2), *gprim = malloc(n * 2), *gsec = malloc(n * 2);
    float *gp = malloc(n * 4), *gm = malloc(n * 4), *gv = malloc(n * 4);
    int8_t *gcodes = malloc(n), *rcodes = malloc(n);
    float *gscales = malloc(nb * 4), *rscales = malloc(nb * 4);
    uint16_t *gout = malloc(N * 2), *rout = malloc(N * 2);
    HIP_OK(hipMemcpy(gp, dp, n * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gm, dm, n * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gv, dv, n * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gprim, dprim, n * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gsec, dsec, n * 2, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gcodes, dcodes, n, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gscales, dscales, nb * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(gout, dout, N * 2, hipMemcpyDeviceToHost));

    /* the oracle's iteration, from the same inputs, on its own results only */
    memcpy(rp, p, n * 4);
    orc_adam_step(rp, rm, rv, g, rprim, n, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay,
                  hp.step, hp.adamw);
    orc_quantize_blockwise_i8(rprim, n, B, rcodes, rscales);
    const int8_t *rc[P2];
    const float *rs[P2];
    rc[0] = rcodes;
    rs[0] = rscales;
    for (unsigned j = 1; j < P2; j++) {
        rc[j] = peer_codes[j];
        rs[j] = peer_scales[j];
    }
    orc_dequant_gather_layer(rc, rs, P2, s, B, N, rout);

    /* Adam: fp32 state within 1e-5 relative (the master against max(|p|, lr));
     * the bf16 primary is the exact rounding of the kernel's master and within
     * one bf16 ulp of the oracle's */
    double ep = 0, em = 0, ev = 0;
    int ulp = 0, exact = 1;
    for (size_t i = 0; i < n; i++) {
        double e;
        if ((e = rel_err(gp[i], rp[i], hp.lr)) > ep) ep = e;
        if ((e = rel_err(gm[i], rm[i], 1e-30)) > em) em = e;
        if ((e = rel_err(gv[i], rv[i], 1e-30)) > ev) ev = e;
        const int d = abs((int)(int16_t)gprim[i] - (int)(int16_t)rprim[i]);
        if (d > ulp) ulp = d;
        if (gprim[i] != orc_bf16_rne(gp[i])) exact = 0;
    }
    EXPECT(ep <= 1e-5 && em <= 1e-5 && ev <= 1e-5, "adam rel err p %g m %g v %g", ep, em, ev);
    EXPECT(ulp <= 1, "bf16 primary off by %d ulp", ulp);
    EXPECT(exact, "primary is not the bf16 rounding of the master");
    EXPECT(memcmp(gsec, gprim, n * 2) == 0, "secondary is not a bit copy of the primary");

    /* quantization and gather: bit-exact in every block whose primary agrees
     * with the oracle's (the primaries may differ by one ulp at a few elements) */
    size_t same = 0, lo_same = 0;
    for (size_t k = 0; k < nb; k++) {
        const size_t a = k * B, e = a + B < n ? a + B : n;
        if (memcmp(gprim + a, rprim + a, (e - a) * 2) != 0)
            continue;
        same++;
        EXPECT(memcmp(gcodes + a, rcodes + a, e - a) == 0, "codes of block %zu", k);
        EXPECT(memcmp(gscales + k, rscales + k, 4) == 0, "scale of block %zu", k);
        if (e <= s) {
            lo_same++;
            EXPECT(memcmp(gout + a, rout + a, (e - a) * 2) == 0, "local gather block %zu", k);
        }
    }
    EXPECT(same * 100 >= nb * 99, "only %zu of %zu blocks agree", same, nb);
    EXPECT(memcmp(gout + s, rout + s, (N - s) * 2) == 0, "gather of the peer shards");

    /* the refresh and the quantization as one pass over the same primary:
     * the same secondary, codes and scales as the two calls, bit for bit */
    {
        uint16_t *dsec2 = dev_alloc(n * 2);
        int8_t *dcodes2 = dev_alloc(n);
        float *dscales2 = dev_alloc(nb * 4);
        uint16_t *gsec2 = malloc(n * 2);
        int8_t *gcodes2 = malloc(n);
        float *gscales2 = malloc(nb * 4);
        EXPECT(zpp_refresh_quantize_i8(dsec2, dprim, n, B, dcodes2, dscales2, copy, ev_gather,
                                       ev_quant) == ZPP_OK,
               "refresh + quantize");
        HIP_OK(hipEventSynchronize(ev_quant));
        HIP_OK(hipMemcpy(gsec2, dsec2, n * 2, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(gcodes2, dcodes2, n, hipMemcpyDeviceToHost));
        HIP_OK(hipMemcpy(gscales2, dscales2, nb * 4, hipMemcpyDeviceToHost));
        EXPECT(memcmp(gsec2, gsec, n * 2) == 0, "one-pass secondary");
        EXPECT(memcmp(gcodes2, gcodes, n) == 0, "one-pass codes");
        EXPECT(memcmp(gscales2, gscales, nb * 4) == 0, "one-pass scales");
        free(gsec2);
        free(gcodes2);
        free(gscales2);
        HIP_OK(hipFree(dsec2));
        HIP_OK(hipFree(dcodes2));
        HIP_OK(hipFree(dscales2));
    }

    check_receive(n, p, &hp);
    check_validation();

    printf("adam rel err p %.3g m %.3g v %.3g, bf16 %d ulp, %zu/%zu blocks bit-exact "
           "(%zu in the local shard)\n", ep, em, ev, ulp, same, nb, lo_same);
    if (failures) {
        printf("c abi FAILED (%d checks)\n", failures);
        return 1;
    }
    printf("c abi ok\n");
    return 0;
}
