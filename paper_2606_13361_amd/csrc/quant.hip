// quant.hip -- the int8 KV artifact: per-tensor symmetric quantization of the
// cached rows [0, L) of a bf16 layer cache (paper, Section "Quantizing the
// artifact: size vs. exactness").
//
//   s = max|x| / 127 over the whole tensor (1 for an all-zero tensor)
//   code = clamp(round-half-even(x / s), -127, 127)
// both divisions correctly rounded fp32.  Four launches: clear the two maxima,
// reduce max|K| and max|V| (float bits of non-negative values order like
// unsigned integers, so an atomic max is exact and order-free), write the
// codes in the artifact layout, turn the maxima into scales.
//
// Artifact layout (head_dim 128, P = capacity rounded up to 32):
//   kq [Hkv][P][128]: code of K[g][j][d] at row byte 64*((d>>3)&1) + 8*(d>>4) + (d&7)
//   vq [Hkv][P/32][128][32]: code of V[g][32b+k][d] at ((g*P/32+b)*128+d)*32 + pos(k),
//      pos(k) = 16*((k>>2)&1) + 8*(k>>4) + 4*((k>>3)&1) + (k&3)
#include "kvr_internal.hpp"

namespace kvr {
namespace {

constexpr int D = 128;
constexpr int QMAX = 127;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__global__ void q8_clear_kernel(float *scales) {
    if (threadIdx.x < 2) scales[threadIdx.x] = 0.f;
}

// blockIdx.y: 0 = K, 1 = V.  Each thread scans 16-byte chunks (8 values) of rows [0, L).
__global__ __launch_bounds__(256) void q8_absmax_kernel(const QuantParams p) {
    const uint16_t *src = (const uint16_t *)(blockIdx.y == 0 ? p.kc : p.vc);
    const int64_t chunks = (int64_t)p.n_kv_heads * p.L * (D / 8);
    float m = 0.f;
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < chunks; c += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = c / (D / 8);                 // (g, j) with j < L
        const int64_t g = row / p.L, j = row % p.L;
        const u32x4 v = *(const u32x4 *)(src + (g * p.cap + j) * D + 8 * (c % (D / 8)));
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            m = fmaxf(m, fabsf(bf16_to_f32((uint16_t)(v[q] & 0xffff))));
            m = fmaxf(m, fabsf(bf16_to_f32((uint16_t)(v[q] >> 16))));
        }
    }
    // wave max, then one atomic per wave
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
    if ((threadIdx.x & 63) == 0 && m > 0.f) atomicMax((unsigned int *)&p.scales[blockIdx.y], __float_as_uint(m));
}

__device__ __forceinline__ float scale_from_max(float m) { return m > 0.f ? __fdiv_rn(m, (float)QMAX) : 1.f; }

__device__ __forceinline__ uint32_t code(float x, float s) {
    const float q = fminf(fmaxf(rintf(__fdiv_rn(x, s)), -(float)QMAX), (float)QMAX);
    return (uint32_t)(int32_t)q & 0xffu;
}

// One block per (kv head g, 32-key block b): stages the 32 K and V rows in LDS
// (rows >= L read as zero), then each thread writes one 16-byte chunk of the
// K codes and one of the V codes.
__global__ __launch_bounds__(256) void q8_quant_kernel(const QuantParams p) {
    __shared__ uint16_t kt[32][D + 8];
    __shared__ uint16_t vt[32][D + 8];
    const int g = blockIdx.x % p.n_kv_heads;
    const int b = blockIdx.x / p.n_kv_heads;
    const int tid = threadIdx.x;
    const float sk = scale_from_max(p.scales[0]);
    const float sv = scale_from_max(p.scales[1]);
    for (int i = tid; i < 32 * (D / 8); i += 256) {
        const int k = i / (D / 8), c = i % (D / 8);
        const int64_t j = (int64_t)b * 32 + k;
        u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
        if (j < p.L) {
            kv = *(const u32x4 *)((const uint16_t *)p.kc + ((int64_t)g * p.cap + j) * D + 8 * c);
            vv = *(const u32x4 *)((const uint16_t *)p.vc + ((int64_t)g * p.cap + j) * D + 8 * c);
        }
        *(u32x4 *)&kt[k][8 * c] = kv;
        *(u32x4 *)&vt[k][8 * c] = vv;
    }
    __syncthreads();
    const int64_t P = p.padded;
    // K: row k, output chunk c (bytes 16c .. 16c+15) = grp c>>2, head-dim steps 2(c&3), 2(c&3)+1
    {
        const int k = tid >> 3, c = tid & 7;
        const int grp = c >> 2, ks0 = 2 * (c & 3);
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t x = 0;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int pos = 4 * q + e4;                       // 0..15 within the chunk
                const int d = 16 * (ks0 + (pos >> 3)) + 8 * grp + (pos & 7);
                x |= code(bf16_to_f32(kt[k][d]), sk) << (8 * e4);
            }
            w[q] = x;
        }
        const int64_t j = (int64_t)b * 32 + k;
        *(u32x4 *)((unsigned char *)p.kq + ((int64_t)g * P + j) * D + 16 * c) = (u32x4){w[0], w[1], w[2], w[3]};
    }
    // V: head-dim row d, output chunk h (positions 16h .. 16h+15 of the 32 keys' slots)
    {
        const int d = tid >> 1, h = tid & 1;
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t x = 0;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
                const int pos = 16 * h + 4 * q + e4;              // 0..31
                // invert pos(k): pos = 16*grp + 8*kk + e, key = 16*kk + 8*(e>>2) + 4*grp + (e&3)
                const int grp = pos >> 4, kk = (pos >> 3) & 1, e = pos & 7;
                const int key = 16 * kk + 8 * (e >> 2) + 4 * grp + (e & 3);
                x |= code(bf16_to_f32(vt[key][d]), sv) << (8 * e4);
            }
            w[q] = x;
        }
        *(u32x4 *)((unsigned char *)p.vq + (((int64_t)g * (P / 32) + b) * D + d) * 32 + 16 * h) =
            (u32x4){w[0], w[1], w[2], w[3]};
    }
}

__global__ void q8_finalize_kernel(float *scales) {
    if (threadIdx.x < 2) scales[threadIdx.x] = scale_from_max(scales[threadIdx.x]);
}

}  // namespace

hipError_t launch_quantize(const QuantParams &p, hipStream_t s) {
    hipLaunchKernelGGL(q8_clear_kernel, dim3(1), dim3(64), 0, s, p.scales);
    const int64_t chunks = (int64_t)p.n_kv_heads * p.L * (D / 8);
    int blocks = (int)((chunks + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(q8_absmax_kernel, dim3(blocks, 2), dim3(256), 0, s, p);
    const int64_t nb = (p.L + 31) / 32;
    hipLaunchKernelGGL(q8_quant_kernel, dim3((unsigned)(nb * p.n_kv_heads)), dim3(256), 0, s, p);
    hipLaunchKernelGGL(q8_finalize_kernel, dim3(1), dim3(64), 0, s, p.scales);
    return hipGetLastError();
}

}  // namespace kvr
