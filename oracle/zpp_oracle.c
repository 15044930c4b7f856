/*
 * Plain CPU oracle for the one-rank partition path of the modified ZeRO++ hpZ
 * scheme (arXiv 2407.01614).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * definition that the HIP kernels are checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark may load it; the
 * product path never does.  It shares no source, header, helper or constant
 * with the HIP library.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math, no FTZ/DAZ,
 * default round-to-nearest), so every float operation below is one IEEE
 * binary32 (or binary64) operation in program order.
 *
 * Every loop is scalar and walks the data once in index order; nothing is
 * blocked, fused or reordered beyond what each definition states.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* bf16 <-> fp32.  The paper fixes no precision; the primary and secondary   */
/* weight copies are taken as bf16 and the master weights as fp32.           */
/* ------------------------------------------------------------------------ */

/* Round a binary32 value to bfloat16 (8-bit significand) with IEEE
 * round-to-nearest, ties-to-even.  The 16 discarded low bits are compared
 * with one half of the last kept place: above half rounds up, below half
 * rounds down, exactly half rounds to the even neighbour.  A carry out of the
 * significand moves into the exponent, which is also how a value above the
 * largest finite bf16 becomes infinity.  NaN becomes the canonical quiet NaN
 * 0x7FC0 (sign dropped).  Parity pinned against a library conversion. */
uint16_t orc_bf16_rne(float f)
{
    uint32_t bits;
    memcpy(&bits, &f, sizeof bits);
    if (f != f)
        return 0x7FC0u;
    uint32_t kept = bits >> 16;
    uint32_t dropped = bits & 0xFFFFu;
    int round_up;
    if (dropped > 0x8000u)
        round_up = 1;
    else if (dropped < 0x8000u)
        round_up = 0;
    else
        round_up = (int)(kept & 1u); /* exact tie: go to the even neighbour */
    return (uint16_t)(kept + (uint32_t)round_up);
}

/* bf16 to binary32 is exact: the 16 bits become the high half. */
float orc_bf16_to_f32(uint16_t h)
{
    uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return f;
}

void orc_bf16_rne_array(const float *x, uint16_t *out, size_t n)
{
    for (size_t i = 0; i < n; i++)
        out[i] = orc_bf16_rne(x[i]);
}

void orc_bf16_to_f32_array(const uint16_t *h, float *out, size_t n)
{
    for (size_t i = 0; i < n; i++)
        out[i] = orc_bf16_to_f32(h[i]);
}

/* ------------------------------------------------------------------------ */
/* Partition step: the optimizer.step() that closes every iteration of       */
/* Algorithm 1, applied to the rank's ZeRO partition (the optimizer states   */
/* are sharded over the data-parallel ranks, Background section).  The paper */
/* does not name the optimizer; this is Adam (Kingma & Ba, Algorithm 1) with */
/* decoupled weight decay (Loshchilov & Hutter), or with the L2 term added   */
/* to the gradient when adamw == 0.                                          */
/*                                                                          */
/* Arithmetic is binary64 from the binary32 inputs and hyperparameters; the  */
/* new state is rounded to binary32 once per step, because that is what is   */
/* stored.  The emitted primary weight is the bf16 rounding of the stored    */
/* binary32 master weight.                                                   */
/* ------------------------------------------------------------------------ */
void orc_adam_step(float *p, float *m, float *v, const float *g, uint16_t *out, size_t n,
                   float lr_f, float beta1_f, float beta2_f, float eps_f, float wd_f,
                   int64_t step, int adamw)
{
    const double lr = lr_f, b1 = beta1_f, b2 = beta2_f, eps = eps_f, wd = wd_f;
    /* bias corrections for 1-based step t */
    const double bc1 = 1.0 - pow(b1, (double)step);
    const double bc2 = 1.0 - pow(b2, (double)step);
    for (size_t i = 0; i < n; i++) {
        double theta = p[i];
        double grad = g[i];
        double mom1 = m[i];
        double mom2 = v[i];
        if (adamw)
            theta = theta - lr * wd * theta; /* decoupled decay on the old weight */
        else
            grad = grad + wd * theta; /* L2 penalty folded into the gradient */
        mom1 = b1 * mom1 + (1.0 - b1) * grad;
        mom2 = b2 * mom2 + (1.0 - b2) * grad * grad;
        const double mhat = mom1 / bc1;
        const double vhat = mom2 / bc2;
        theta = theta - lr * mhat / (sqrt(vhat) + eps);
        p[i] = (float)theta;
        m[i] = (float)mom1;
        v[i] = (float)mom2;
        if (out)
            out[i] = orc_bf16_rne(p[i]);
    }
}

/* ------------------------------------------------------------------------ */
/* Secondary refresh: the asynchronous device-to-device copy that fills the  */
/* secondary partition after a layer's forward pass (Algorithm 1; Eq. 1 and  */
/* the text after it: the local rank's weights are copied out of the full    */
/* parameter tensor).  A bit copy: NaN payloads are kept as they are.        */
/* ------------------------------------------------------------------------ */
void orc_refresh(uint16_t *dst, const uint16_t *src, size_t count)
{
    for (size_t i = 0; i < count; i++)
        dst[i] = src[i];
}

/*
 * qwZ: weights are quantized before the AllGather (Background section).  The
 * paper gives no format; the one taken here is symmetric absmax int8 over
 * blocks of `block` consecutive elements of one shard, one binary32 scale per
 * block, codes in [-127, 127].  All decisions are taken in binary32, the
 * precision the kernels use:
 *   block holds a non-finite value -> scale = NaN (0x7FC00000), codes 0;
 *   absmax a == 0                  -> scale = 0, codes 0;
 *   otherwise scale = RN(a / 127) and inv = RN(127 / a), and code =
 *   rint(x * inv) (ties to even), clamped to [-127, 127].  When a < 2^-100
 *   both x and a are first multiplied by 2^64 (exact) so that 127 / a cannot
 *   overflow; the codes then stay invariant under scaling of the block by any
 *   power of two.  The last block of a shard may be short.
 */
static const uint32_t ORC_SCALE_NAN_BITS = 0x7FC00000u;

void orc_quantize_blockwise_i8(const uint16_t *x, size_t n, uint32_t block, int8_t *codes,
                               float *scales)
{
    if (block == 0)
        return;
    const size_t nblocks = (n + block - 1) / block;
    for (size_t k = 0; k < nblocks; k++) {
        const size_t lo = k * (size_t)block;
        const size_t hi = (lo + block < n) ? lo + block : n;
        int nonfinite = 0;
        float a = 0.0f;
        for (size_t i = lo; i < hi; i++) {
            const float xi = orc_bf16_to_f32(x[i]);
            if (!isfinite(xi))
                nonfinite = 1;
            else if (fabsf(xi) > a)
                a = fabsf(xi);
        }
        if (nonfinite) {
            float qnan;
            memcpy(&qnan, &ORC_SCALE_NAN_BITS, sizeof qnan);
            scales[k] = qnan;
            for (size_t i = lo; i < hi; i++)
                codes[i] = 0;
            continue;
        }
        if (a == 0.0f) {
            scales[k] = 0.0f;
            for (size_t i = lo; i < hi; i++)
                codes[i] = 0;
            continue;
        }
        scales[k] = a / 127.0f;
        float pre = 1.0f;
        if (a < 0x1p-100f)
            pre = 0x1p64f;
        const float inv = 127.0f / (a * pre);
        for (size_t i = lo; i < hi; i++) {
            const float y = (orc_bf16_to_f32(x[i]) * pre) * inv;
            float q = rintf(y);
            if (q > 127.0f)
                q = 127.0f;
            if (q < -127.0f)
                q = -127.0f;
            codes[i] = (int8_t)q;
        }
    }
}

/* Dequantize one shard: y = bf16_rne(float(code) * scale), one binary32
 * multiply then one rounding to bf16 (no fused step). */
void orc_dequant_blockwise_i8(const int8_t *codes, const float *scales, size_t n, uint32_t block,
                              uint16_t *out)
{
    for (size_t i = 0; i < n; i++) {
        const float prod = (float)codes[i] * scales[i / block];
        out[i] = orc_bf16_rne(prod);
    }
}

/* ------------------------------------------------------------------------ */
/* Backward-pass AllGather(L_k, P') of Algorithm 1 over the node-local       */
/* secondary shards, with the qwZ dequantization: the full layer is the      */
/* in-order concatenation of the P' dequantized shards, each shard_elems     */
/* long, cut at layer_elems (the zero padding of the last shard is dropped). */
/* shard_codes / shard_scales are arrays of num_shards pointers.             */
/* ------------------------------------------------------------------------ */
void orc_dequant_gather_layer(const int8_t *const *shard_codes, const float *const *shard_scales,
                              uint32_t num_shards, size_t shard_elems, uint32_t block,
                              size_t layer_elems, uint16_t *out)
{
    for (uint32_t j = 0; j < num_shards; j++) {
        for (size_t i = 0; i < shard_elems; i++) {
            const size_t o = (size_t)j * shard_elems + i;
            if (o >= layer_elems)
                return;
            const float prod = (float)shard_codes[j][i] * shard_scales[j][i / block];
            out[o] = orc_bf16_rne(prod);
        }
    }
}

/*
 * qgZ: gradients are quantized before the exchange that replaces the
 * ReduceScatter (Background section; Algorithm 1, backward loop, where an
 * INT4 all-to-all takes the ReduceScatter's place).  The paper gives no
 * format; the one taken here is symmetric absmax int4 over blocks of `block`
 * consecutive binary32 gradient values of one destination partition, one
 * binary32 scale per block, codes in [-7, 7], all decisions in binary32:
 *   block holds a non-finite value -> scale = NaN (0x7FC00000), codes 0;
 *   absmax a == 0                  -> scale = 0, codes 0;
 *   otherwise scale = RN(a / 7), inv = RN(7 / a), code = rint(x * inv)
 *   (ties to even), clamped to [-7, 7]; when a < 2^-100 both x and a are
 *   first multiplied by 2^64 (exact).
 * Codes are packed two per byte, element 2i in the low nibble and 2i+1 in the
 * high nibble, as 4-bit two's complement; an odd tail leaves the last high
 * nibble 0.
 */
void orc_quantize_blockwise_i4(const float *x, size_t n, uint32_t block, uint8_t *codes,
                               float *scales)
{
    if (block == 0)
        return;
    for (size_t b = 0; b < (n + 1) / 2; b++)
        codes[b] = 0;
    const size_t nblocks = (n + block - 1) / block;
    for (size_t k = 0; k < nblocks; k++) {
        const size_t lo = k * (size_t)block;
        const size_t hi = (lo + block < n) ? lo + block : n;
        int nonfinite = 0;
        float a = 0.0f;
        for (size_t i = lo; i < hi; i++) {
            if (!isfinite(x[i]))
                nonfinite = 1;
            else if (fabsf(x[i]) > a)
                a = fabsf(x[i]);
        }
        if (nonfinite) {
            float qnan;
            memcpy(&qnan, &ORC_SCALE_NAN_BITS, sizeof qnan);
            scales[k] = qnan;
            continue; /* codes stay 0 */
        }
        if (a == 0.0f) {
            scales[k] = 0.0f;
            continue;
        }
        scales[k] = a / 7.0f;
        float pre = 1.0f;
        if (a < 0x1p-100f)
            pre = 0x1p64f;
        const float inv = 7.0f / (a * pre);
        for (size_t i = lo; i < hi; i++) {
            float q = rintf((x[i] * pre) * inv);
            if (q > 7.0f)
                q = 7.0f;
            if (q < -7.0f)
                q = -7.0f;
            const uint8_t nib = (uint8_t)((int)q & 0xF);
            if (i % 2 == 0)
                codes[i / 2] |= nib;
            else
                codes[i / 2] |= (uint8_t)(nib << 4);
        }
    }
}

/* The signed value of 4-bit code i of a packed array. */
static int orc_i4_code(const uint8_t *codes, size_t i)
{
    const int nib = (i % 2 == 0) ? (codes[i / 2] & 0xF) : (codes[i / 2] >> 4);
    return nib >= 8 ? nib - 16 : nib;
}

void orc_unpack_i4(const uint8_t *codes, size_t n, int8_t *out)
{
    for (size_t i = 0; i < n; i++)
        out[i] = (int8_t)orc_i4_code(codes, i);
}

/* The receiving side of the qgZ exchange for one destination partition:
 * num_src quantized copies of the same n-element partition (one from each
 * sending rank, in rank order) are dequantized and summed,
 *     acc = 0;  acc = fma(code_q[i], scale_q[i / block], acc) for q = 0..num_src-1
 *     out[i] = acc * scale_out
 * each fma a single rounding, the final product one more; scale_out is 1
 * for a sum or 1/P for the data-parallel mean. */
void orc_dequant_reduce_i4(const uint8_t *const *src_codes, const float *const *src_scales,
                           uint32_t num_src, size_t n, uint32_t block, float scale_out,
                           float *out)
{
    for (size_t i = 0; i < n; i++) {
        float acc = 0.0f;
        for (uint32_t q = 0; q < num_src; q++)
            acc = fmaf((float)orc_i4_code(src_codes[q], i), src_scales[q][i / block], acc);
        out[i] = acc * scale_out;
    }
}
