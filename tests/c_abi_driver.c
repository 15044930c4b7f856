/*
 * The partition path driven from plain C through libzpp.so, with nothing but
 * the HIP runtime API around it: device buffers from hipMalloc, three
 * streams, caller-owned events, the four calls of one iteration in the order
 * of Algorithm 1 (Adam step -> refresh of the secondary copy -> qwZ
 * quantization -> dequantize-and-gather of the layer over P' shards), with
 * the gather ordered after the quantization by an event (the fix).  The
 * results are checked against the CPU oracle (liboracle.so), which runs the
 * same iteration on the same inputs on its own.  Also checks a few
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
