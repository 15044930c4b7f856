// Dequant-gather: the local half of the backward AllGather(L, P') over the
// node-local secondary shards (Algorithm 1, backward branch), with the qwZ
// dequantization fused in.  1 B + 4/B B read, 2 B written per element.
//
// The shard pointers travel by value in the kernel arguments; blockIdx.y picks
// the shard, so the pointer is a uniform (scalar) load.
//
// Row kernel (blocks that are powers of two): a one-wave workgroup takes one
// row of 512 consecutive elements of a shard; lane l turns the 8 codes
// [8 l, 8 l + 8) of the row (one 8-byte load) into 8 bf16 (one 16-byte
// store), about three VALU operations per element.  The row's max(1, 512/B)
// scales are the same for the whole wave, so they are read by scalar loads
// (through the scalar cache, beside the vector loads of the codes rather than
// among them), and whether every one of them takes the fast dequantization is
// one scalar branch.  Measured at the Llama-2-13B layer: 143.7-144.8 us
// against 148.4-149.7 us for two-wave workgroups of two rows per wave reading
// the scales by vector loads (the vector kernel below); more rows per wave or
// more waves per workgroup were slower (148.8-152.4 us), and an access
// pattern of the same loads and stores with no scales and no arithmetic
// takes 139 us.
//
// Vector kernel (any other multiple of 64 as the block): a lane's scale is
// a vector load at its own block index (shared by the lanes of a block,
// served from cache); two-wave workgroups with two rows per wave, at most 12
// workgroups per CU.
#include "zpp_device.h"
#include "zpp_launch.h"

#ifndef ZPP_GATHER_UNROLL
#define ZPP_GATHER_UNROLL 2
#endif
#ifndef ZPP_GATHER_THREADS
#define ZPP_GATHER_THREADS 128
#endif
#ifndef ZPP_GATHER_RESIDENCY
#define ZPP_GATHER_RESIDENCY 12
#endif
#ifndef ZPP_GATHER_MAX_GRID_X
#define ZPP_GATHER_MAX_GRID_X (1u << 20)
#endif
// the row kernel takes shards of up to this many rows (one workgroup each);
// longer shards (beyond 2^40 elements) go to the grid-stride vector kernel
#ifndef ZPP_GATHER_ROW_MAX_GRID_X
#define ZPP_GATHER_ROW_MAX_GRID_X 0x7FFFFFFFu
#endif

namespace zpp {
namespace {

constexpr int kGatherThreads = ZPP_GATHER_THREADS;

struct GatherArgs {
    GatherShards shards;
    uint16_t *out;
    size_t shard_elems;
    size_t layer_elems;
    BlockDiv block;
};

__device__ __forceinline__ float code_f32(uint32_t w, int byte) {
    return (float)(int)(int8_t)(uint8_t)(w >> (8 * byte));
}

// Scales in [2^-100, 2^100]: every product code * s is zero or a normal
// float, and -128 * s is exact.  For such scales the product is formed as
// fma(u, s, -128 s) with u = code + 128 taken straight from the byte by the
// unsigned byte converts; u*s - 128*s equals code*s exactly, so the single
// rounding of the fma is the rounding of code * s.  The pair is then rounded
// to bf16 (nearest even) by the packed convert.
__device__ __forceinline__ bool fast_scale(float s) {
    return s >= 0x1p-100f && s <= 0x1p100f;
}

__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
    const bf16x2 v = __builtin_convertvector((f32x2){lo, hi}, bf16x2);
    return __builtin_bit_cast(uint32_t, v);
}

// 4 codes (one word, biased by 0x80 per byte) -> 2 words of packed bf16
__device__ __forceinline__ u32x2 dequant_word_fast(uint32_t biased, float s, float c) {
    const float x0 = __builtin_fmaf((float)(biased & 0xFFu), s, c);
    const float x1 = __builtin_fmaf((float)((biased >> 8) & 0xFFu), s, c);
    const float x2 = __builtin_fmaf((float)((biased >> 16) & 0xFFu), s, c);
    const float x3 = __builtin_fmaf((float)(biased >> 24), s, c);
    return u32x2{bf16x2_rne(x0, x1), bf16x2_rne(x2, x3)};
}

// Any scale (zero, negative, tiny, huge, Inf, NaN): one rounded product and
// the integer RNE of bf16_rne_bits, NaN made canonical.
__device__ __forceinline__ u32x2 dequant_word_any(uint32_t w, float s) {
    u32x2 r;
    r.x = pack_bf16x2(code_f32(w, 0) * s, code_f32(w, 1) * s);
    r.y = pack_bf16x2(code_f32(w, 2) * s, code_f32(w, 3) * s);
    return r;
}

// A row is one wave-wide pass: 64 lanes x 8 consecutive codes = 512 output
// elements, read as one contiguous 512-byte load and written as one
// contiguous 1 KiB store.  A tile is U rows per wave.
template <int U>
__global__ __launch_bounds__(kGatherThreads) void gather_vec_kernel(GatherArgs a) {
    constexpr size_t kRow = (size_t)kGatherThreads * 8;  // elements per row of the workgroup
    constexpr size_t kTile = kRow * U;
    const uint32_t j = blockIdx.y;
    const size_t lo = (size_t)j * a.shard_elems;
    if (lo >= a.layer_elems)
        return;
    const size_t rest = a.layer_elems - lo;
    const size_t valid = rest < a.shard_elems ? rest : a.shard_elems;
    const int8_t *__restrict__ codes = a.shards.codes[j];
    const float *__restrict__ scales = a.shards.scales[j];
    uint16_t *__restrict__ out = a.out + lo;
    const size_t ntiles = (valid + kTile - 1) / kTile;
    for (size_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
        const size_t base = t * kTile + (size_t)threadIdx.x * 8;
        if ((t + 1) * kTile <= valid) {
            u32x2 c[U];
            float s[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kRow;
                c[u] = ld_nt(reinterpret_cast<const u32x2 *>(codes + i));
                s[u] = scales[block_of(a.block, i)];
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i = base + (size_t)u * kRow;
                u32x2 r0, r1;
                if (fast_scale(s[u])) {
                    const float cb = -128.0f * s[u];
                    r0 = dequant_word_fast(c[u].x ^ 0x80808080u, s[u], cb);
                    r1 = dequant_word_fast(c[u].y ^ 0x80808080u, s[u], cb);
                } else {
                    r0 = dequant_word_any(c[u].x, s[u]);
                    r1 = dequant_word_any(c[u].y, s[u]);
                }
                st_nt(reinterpret_cast<u32x4 *>(out + i), u32x4{r0.x, r0.y, r1.x, r1.y});
            }
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const size_t i0 = base + (size_t)u * kRow;
                for (size_t i = i0; i < i0 + 8 && i < valid; ++i) {
                    const float x = (float)codes[i] * scales[block_of(a.block, i)];
                    out[i] = (uint16_t)bf16_rne_bits(x);
                }
            }
        }
    }
}


// One row of 512 elements per one-wave workgroup, one workgroup per row (a
// one-shot grid: no loop, so the scale loads come before any store and the
// compiler keeps them scalar).  B is a power of two: the row holds
// kBlocks = max(1, 512 / B) whole blocks, or lies inside one.
template <int B>
__global__ __launch_bounds__(kWave) void gather_row_kernel(GatherArgs a) {
    constexpr int kBlocks = B >= 512 ? 1 : 512 / B;
    constexpr int kLanesPerBlock = B >= 512 ? kWave : B / 8;
    const uint32_t j = blockIdx.y;  // every shard of the grid holds layer elements
    const size_t lo = (size_t)j * a.shard_elems;
    const size_t rest = a.layer_elems - lo;
    const size_t valid = rest < a.shard_elems ? rest : a.shard_elems;
    const int8_t *__restrict__ codes = a.shards.codes[j];
    const float *__restrict__ scales = a.shards.scales[j];
    uint16_t *__restrict__ out = a.out + lo;
    const uint32_t lane = threadIdx.x;
    const size_t r = blockIdx.x;
    const size_t i = r * 512 + (size_t)lane * 8;
    if ((r + 1) * 512 <= valid) {
        const u32x2 c = ld_nt(reinterpret_cast<const u32x2 *>(codes + i));
        // the row's scales: uniform indices, scalar loads
        const size_t k0 = r * 512 / B;
        float sv[kBlocks];
        bool fast = true;
#pragma unroll
        for (int q = 0; q < kBlocks; ++q) {
            sv[q] = scales[k0 + q];
            fast = fast && fast_scale(sv[q]);
        }
        float s = sv[0];
#pragma unroll
        for (int q = 1; q < kBlocks; ++q)
            s = (lane / kLanesPerBlock == (uint32_t)q) ? sv[q] : s;
        u32x2 r0, r1;
        if (fast) {
            const float cb = -128.0f * s;
            r0 = dequant_word_fast(c.x ^ 0x80808080u, s, cb);
            r1 = dequant_word_fast(c.y ^ 0x80808080u, s, cb);
        } else {
            r0 = dequant_word_any(c.x, s);
            r1 = dequant_word_any(c.y, s);
        }
        st_nt(reinterpret_cast<u32x4 *>(out + i), u32x4{r0.x, r0.y, r1.x, r1.y});
    } else {
        for (size_t e = i; e < i + 8 && e < valid; ++e) {
            const float x = (float)codes[e] * scales[e / B];
            out[e] = (uint16_t)bf16_rne_bits(x);
        }
    }
}

template <int B>
void launch_rows(const GatherArgs &a, unsigned rows, unsigned shards, hipStream_t stream) {
    hipLaunchKernelGGL((gather_row_kernel<B>), dim3(rows, shards), dim3(kWave), 0, stream, a);
}

// Any shard length and alignment: one output element per thread.
__global__ __launch_bounds__(kThreads) void gather_scalar_kernel(GatherArgs a) {
    const uint32_t j = blockIdx.y;
    const size_t lo = (size_t)j * a.shard_elems;
    if (lo >= a.layer_elems)
        return;
    const size_t rest = a.layer_elems - lo;
    const size_t valid = rest < a.shard_elems ? rest : a.shard_elems;
    const int8_t *codes = a.shards.codes[j];
    const float *scales = a.shards.scales[j];
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < valid; i += stride) {
        const float x = (float)codes[i] * scales[block_of(a.block, i)];
        a.out[lo + i] = (uint16_t)bf16_rne_bits(x);
    }
}

}  // namespace

hipError_t launch_gather(const GatherShards &shards, uint32_t num_shards, size_t shard_elems,
                         uint32_t block, size_t layer_elems, uint16_t *out, bool vector_path,
                         hipStream_t stream) {
    GatherArgs a;
    a.shards = shards;
    a.out = out;
    a.shard_elems = shard_elems;
    a.layer_elems = layer_elems;
    a.block = make_block_div(block);
    const size_t per_shard = shard_elems < layer_elems ? shard_elems : layer_elems;
    const size_t nrows = (per_shard + 511) / 512;
    if (vector_path && (block & (block - 1)) == 0 && nrows <= ZPP_GATHER_ROW_MAX_GRID_X) {
        // only the shards that hold layer elements
        const unsigned gy = (unsigned)((layer_elems + shard_elems - 1) / shard_elems);
        const unsigned gx = (unsigned)nrows;
        switch (block) {
        case 64: launch_rows<64>(a, gx, gy, stream); break;
        case 128: launch_rows<128>(a, gx, gy, stream); break;
        case 256: launch_rows<256>(a, gx, gy, stream); break;
        case 512: launch_rows<512>(a, gx, gy, stream); break;
        case 1024: launch_rows<1024>(a, gx, gy, stream); break;
        case 2048: launch_rows<2048>(a, gx, gy, stream); break;
        default: launch_rows<4096>(a, gx, gy, stream); break;
        }
    } else if (vector_path) {
        constexpr size_t kTile = (size_t)kGatherThreads * 8 * ZPP_GATHER_UNROLL;
        const size_t tiles = (per_shard + kTile - 1) / kTile;
        const unsigned gx =
            (unsigned)(tiles < ZPP_GATHER_MAX_GRID_X ? tiles : ZPP_GATHER_MAX_GRID_X);
        hipLaunchKernelGGL((gather_vec_kernel<ZPP_GATHER_UNROLL>), dim3(gx, num_shards),
                           dim3(kGatherThreads), residency_lds(ZPP_GATHER_RESIDENCY), stream, a);
    } else {
        const size_t blocks = (per_shard + kThreads - 1) / kThreads;
        const unsigned gx = (unsigned)(blocks < (1u << 20) ? blocks : (1u << 20));
        hipLaunchKernelGGL(gather_scalar_kernel, dim3(gx, num_shards), dim3(kThreads), 0,
                           stream, a);
    }
    return hipGetLastError();
}

}  // namespace zpp
