// layer.hip -- libkvr_model: the decoder layer around libkvr's attention
// (include/kvr_model.h).  Normalizations, the per-head q/k normalization with
// the rotary embedding, the gated activation and the one-row products of a
// one-token step are kernels of this file; the matrix products of more rows
// go to hipBLASLt; the attention is libkvr's public entry points.
#include <hipblaslt/hipblaslt.h>
#include <math.h>
#include <string.h>

#include <map>
#include <tuple>

#include "attn_common.hpp"
#include "kvr_model.h"

namespace kvr {
namespace model {
namespace {

using namespace dev;

constexpr int NT = 256;

__device__ __forceinline__ float block_sum(float v, float *red) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) t += red[i];
    return t;
}

// One workgroup per row: sum of squares in fp32, then x * rsqrt(mean + eps) * w,
// rounded once.  Rows of n elements, 8 per 16-byte chunk.
template <class E>
__global__ __launch_bounds__(NT) void rmsnorm_kernel(const uint16_t *x, const uint16_t *w, uint16_t *y, int n,
                                                     float eps) {
    __shared__ float red[NT / 64];
    const int64_t row = blockIdx.x;
    const uint16_t *xr = x + row * n;
    float ss = 0.f;
    for (int c = threadIdx.x; c < n / 8; c += NT) {
        const u32x4 v = *(const u32x4 *)(xr + 8 * c);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float a = E::lo(v[i]), b = E::hi(v[i]);
            ss = __builtin_fmaf(a, a, ss);
            ss = __builtin_fmaf(b, b, ss);
        }
    }
    const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)n + eps);
    uint16_t *yr = y + row * n;
    for (int c = threadIdx.x; c < n / 8; c += NT) {
        const u32x4 v = *(const u32x4 *)(xr + 8 * c);
        const u32x4 g = *(const u32x4 *)(w + 8 * c);
        u32x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i)
            o[i] = E::pack2(E::lo(v[i]) * inv * E::lo(g[i]), E::hi(v[i]) * inv * E::hi(g[i]));
        *(u32x4 *)(yr + 8 * c) = o;
    }
}

// One wave per (token, head) of the fused q|k|v rows.  Lane l holds dims l and
// l + D/2 (the rotary pair), so the normalization needs one wave reduction and
// the rotation none.  q and k heads: rmsnorm * weight, then the rotation at
// position pos0 + token, one rounding; v heads are copied.  Outputs go to
// token-major q/k/v rows and, when kc is set, the k and v rows also to cache
// rows pos0 + token.
struct QkParams {
    const uint16_t *qkv;           // [T][(Hq + 2 Hkv) D]
    const uint16_t *qn, *kn;       // [D]
    const float *cs;               // RoPE table [n_pos][D/2][2]
    uint16_t *q, *k, *v;           // [T][H][D]
    uint16_t *kc, *vc;             // [Hkv][cap][D] or null
    int64_t T, pos0, cap;
    int32_t Hq, Hkv;
    float eps;
};

template <class E, int D>
__global__ __launch_bounds__(NT) void qk_norm_rope_kernel(const QkParams p) {
    const int lane = threadIdx.x & 63;
    const int64_t item = (int64_t)blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
    const int H = p.Hq + 2 * p.Hkv;
    if (item >= p.T * H) return;                      // whole waves leave together
    const int64_t t = item / H;
    const int hh = (int)(item % H);
    const int64_t pos = p.pos0 + t;
    const bool act = lane < D / 2;
    const uint16_t *src = p.qkv + (t * H + hh) * D;
    float x1 = act ? E::lo((uint32_t)src[lane]) : 0.f;
    float x2 = act ? E::lo((uint32_t)src[lane + D / 2]) : 0.f;
    auto put = [&](uint16_t *dst, float a, float b) {
        const uint32_t pk = E::pack2(a, b);
        dst[lane] = (uint16_t)(pk & 0xffffu);
        dst[lane + D / 2] = (uint16_t)(pk >> 16);
    };
    if (hh >= p.Hq + p.Hkv) {                         // value head: copy
        const int g = hh - p.Hq - p.Hkv;
        if (act) {
            put(p.v + (t * p.Hkv + g) * D, x1, x2);
            if (p.vc) put(p.vc + ((int64_t)g * p.cap + pos) * D, x1, x2);
        }
        return;
    }
    float ss = x1 * x1 + x2 * x2;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    const float inv = 1.0f / sqrtf(ss / (float)D + p.eps);
    const bool is_q = hh < p.Hq;
    const uint16_t *nw = is_q ? p.qn : p.kn;
    if (!act) return;
    const float n1 = x1 * inv * E::lo((uint32_t)nw[lane]);
    const float n2 = x2 * inv * E::lo((uint32_t)nw[lane + D / 2]);
    const float2 csv = *(const float2 *)(p.cs + pos * D + 2 * lane);
    float y1, y2;
    rope_rot(n1, n2, csv.x, csv.y, y1, y2);
    if (is_q) {
        put(p.q + (t * p.Hq + hh) * D, y1, y2);
    } else {
        const int g = hh - p.Hq;
        put(p.k + (t * p.Hkv + g) * D, y1, y2);
        if (p.kc) put(p.kc + ((int64_t)g * p.cap + pos) * D, y1, y2);
    }
}

// silu(g) = g / (1 + e^-g) with the hardware exponential (2^x) and reciprocal
// (each within about an ulp of fp32): the product with the up row is rounded to
// the element format, far coarser.  Large -g gives 2^x = inf, rcp = 0, silu = -0.
// One definition for the multi-row kernel and the one-row prologue, so a
// continuation step and a prefill give the same activation bits.
__device__ __forceinline__ float silu(float g) {
    return g * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(g * -1.4426950408889634f));
}

// act[t][i] = silu(gu[t][i]) * gu[t][I + i], 8 elements per thread.
template <class E>
__global__ __launch_bounds__(NT) void silu_mul_kernel(const uint16_t *gu, uint16_t *act, int64_t T, int I) {
    const int64_t per_row = I / 8;
    const int64_t n = T * per_row;
    for (int64_t idx = (int64_t)blockIdx.x * NT + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * NT) {
        const int64_t t = idx / per_row;
        const int c = (int)(idx % per_row);
        const u32x4 g = *(const u32x4 *)(gu + t * 2 * I + 8 * c);
        const u32x4 u = *(const u32x4 *)(gu + t * 2 * I + I + 8 * c);
        u32x4 o;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float g0 = E::lo(g[i]), g1 = E::hi(g[i]);
            o[i] = E::pack2(silu(g0) * E::lo(u[i]), silu(g1) * E::hi(u[i]));
        }
        *(u32x4 *)(act + t * I + 8 * c) = o;
    }
}

// ---------------------------------------------------------------- one row
// y[n] = sum_k x'[k] w[n][k] (+ y[n]) for a single row x: the weights are
// streamed once from HBM, 16-byte loads coalesced along k, which bounds the
// one-token step; a matrix-core product has nothing to reuse here.  x' is
// built once per workgroup in LDS by the prologue:
//   kPlain  x' = x
//   kNorm   x' = round(rmsnorm(x) * ln)           (the layer's input norms)
//   kSilu   x' = round(silu(x[k]) * x[K + k])     (x = the gate|up row)
// so the norm and the activation need no launch of their own.
enum { kPlain = 0, kNorm = 1, kSilu = 2 };
constexpr int kGemvMaxK = 16384;

struct GemvParams {
    const uint16_t *x;     // [K] (kSilu: [2K])
    const uint16_t *w;     // [N][K]
    const uint16_t *ln;    // [K] (kNorm)
    uint16_t *y;           // [N]
    int64_t N;
    int32_t K;
    int32_t beta;          // 1: add into y
    float eps;
};

constexpr int GT = 512;            // threads of a one-row-product workgroup
constexpr int kGemvMaxGrid = 512;  // workgroups: two per compute unit

// x' of a one-row product into LDS (see above), by all NTH threads of the workgroup
template <class E, int PRO, int NTH>
__device__ __forceinline__ void build_x(const GemvParams &p, uint16_t *xs, float *red, int tid) {
    constexpr int NW = NTH / 64;
    const int KC = p.K / 8;
    const int wave = tid >> 6, lane = tid & 63;
    (void)wave; (void)lane;
    if (PRO == kNorm) {
        float ss = 0.f;
        for (int c = tid; c < KC; c += NTH) {
            const u32x4 v = *(const u32x4 *)(p.x + 8 * c);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float a = E::lo(v[i]), b = E::hi(v[i]);
                ss = __builtin_fmaf(a, a, ss);
                ss = __builtin_fmaf(b, b, ss);
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
        if (lane == 0) red[wave] = ss;
        __syncthreads();
        float tot = 0.f;
#pragma unroll
        for (int i = 0; i < NW; ++i) tot += red[i];
        const float inv = 1.0f / sqrtf(tot / (float)p.K + p.eps);
        for (int c = tid; c < KC; c += NTH) {
            const u32x4 v = *(const u32x4 *)(p.x + 8 * c);
            const u32x4 g = *(const u32x4 *)(p.ln + 8 * c);
            u32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                o[i] = E::pack2(E::lo(v[i]) * inv * E::lo(g[i]), E::hi(v[i]) * inv * E::hi(g[i]));
            *(u32x4 *)(xs + 8 * c) = o;
        }
    } else if (PRO == kSilu) {
        for (int c = tid; c < KC; c += NTH) {
            const u32x4 g = *(const u32x4 *)(p.x + 8 * c);
            const u32x4 u = *(const u32x4 *)(p.x + p.K + 8 * c);
            u32x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float g0 = E::lo(g[i]), g1 = E::hi(g[i]);
                o[i] = E::pack2(silu(g0) * E::lo(u[i]), silu(g1) * E::hi(u[i]));
            }
            *(u32x4 *)(xs + 8 * c) = o;
        }
    } else {
        for (int c = tid; c < KC; c += NTH) *(u32x4 *)(xs + 8 * c) = *(const u32x4 *)(p.x + 8 * c);
    }
}

// PAIR (RW = 2): the weights hold 2N rows, gate rows 0..N-1 then up rows
// N..2N-1; a wave takes the pair (n, N + n) and stores act[n] =
// silu(g) * u with g and u rounded to the element format first, as the
// multi-row path rounds them before silu_mul_kernel.
template <class E, int PRO, int RW, int PAIR = 0>
__global__ __launch_bounds__(GT) void gemv_kernel(const GemvParams p) {
    static_assert(!PAIR || RW == 2, "a pair is two rows");
    __shared__ __attribute__((aligned(16))) uint16_t xs[kGemvMaxK];
    __shared__ float red[GT / 64];
    constexpr int U = RW == 1 ? 8 : 4;                   // k-steps per block of loads
    constexpr int NW = GT / 64;
    constexpr int RPW = PAIR ? 1 : RW;                   // outputs per wave and step
    const int tid = threadIdx.x;
    const int KC = p.K / 8;
    const int wave = tid >> 6, lane = tid & 63;
    const int steps = (KC + 63) / 64;
    // wave w of workgroup b takes row groups (b * NW + w) * RPW, then every
    // grid-stride after it: each workgroup builds x' once for all its rows
    const int64_t stride = (int64_t)gridDim.x * NW * RPW;
    int64_t n0 = ((int64_t)blockIdx.x * NW + wave) * RPW;
    u32x4 wv[U][RW];
    // Every load is issued, from a clamped (valid) address: without branches
    // the compiler counts the loads in flight and waits only for the block it
    // uses.  Chunks past K and rows past N are loaded and never used.
    auto load_block = [&](int64_t nb, int s0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = min(lane + 64 * (s0 + u), KC - 1);
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const int64_t row = PAIR ? (nb < p.N ? nb : p.N - 1) + r * p.N
                                         : (nb + r < p.N ? nb + r : p.N - 1);
                wv[u][r] = *(const u32x4 *)(p.w + row * p.K + 8 * c);
            }
        }
    };
    // the first weights do not depend on x: in flight while the prologue runs
    load_block(n0, 0);

    build_x<E, PRO, GT>(p, xs, red, tid);
    __syncthreads();

    for (; n0 < p.N; n0 += stride) {
        const int rows = p.N - n0 < RPW ? (int)(p.N - n0) : RPW;
        float acc[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) acc[r] = 0.f;
        for (int s0 = 0; s0 < steps; s0 += U) {
            u32x4 cur[U][RW];
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int r = 0; r < RW; ++r) cur[u][r] = wv[u][r];
            // the next block streams in meanwhile: of this row group, or the
            // first of the next one
            if (s0 + U < steps) load_block(n0, s0 + U);
            else load_block(n0 + stride, 0);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int c = lane + 64 * (s0 + u);
                if (c < KC) {
                    const u32x4 xv = *(const u32x4 *)(xs + 8 * c);
#pragma unroll
                    for (int r = 0; r < RW; ++r)
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            acc[r] = __builtin_fmaf(E::lo(cur[u][r][i]), E::lo(xv[i]), acc[r]);
                            acc[r] = __builtin_fmaf(E::hi(cur[u][r][i]), E::hi(xv[i]), acc[r]);
                        }
                }
            }
        }
#pragma unroll
        for (int r = 0; r < RW; ++r)
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) acc[r] += __shfl_xor(acc[r], o);
        if constexpr (PAIR) {
            if (lane == 0) {
                const float g = E::lo(E::pack2(acc[0], 0.f)), u = E::lo(E::pack2(acc[1], 0.f));
                p.y[n0] = (uint16_t)(E::pack2(silu(g) * u, 0.f) & 0xffffu);
            }
        } else if (lane < rows) {
            float v = acc[0];
#pragma unroll
            for (int r = 1; r < RW; ++r)
                if (lane == r) v = acc[r];
            if (p.beta) v += E::lo((uint32_t)p.y[n0 + lane]);
            p.y[n0 + lane] = (uint16_t)(E::pack2(v, 0.f) & 0xffffu);
        }
    }
}

// One output row per wave, its whole weight row in one block of U 16-byte
// loads per lane (U * 64 * 8 >= K), issued right after the prologue's reads of
// x: every weight byte of the product is requested at once, for outputs of up to
// kGemv1MaxRows rows (the layer's QKV, O and down products).  The grid-stride
// kernel above pipelines blocks of 8 and serves the wide products.
constexpr int64_t kGemv1MaxRows = 8192;
constexpr int64_t kGemv1Cus = 256;    // compute units of the part (MI355X)
constexpr int kGemv1MaxSteps = 19;   // K = 9728 (the Qwen3-4B MLP width) exactly

template <class E, int PRO, int U, int NWV>
__global__ __launch_bounds__(64 * NWV) void gemv1_kernel(const GemvParams p) {
    constexpr int NTH = 64 * NWV;
    __shared__ __attribute__((aligned(16))) uint16_t xs[kGemvMaxK];
    __shared__ float red[NWV];
    const int tid = threadIdx.x;
    const int KC = p.K / 8;
    const int wave = tid >> 6, lane = tid & 63;
    const int64_t n = (int64_t)blockIdx.x * NWV + wave;
    const int64_t row = n < p.N ? n : p.N - 1;       // past N: loaded, never stored
    // x' first: a wave's loads complete in issue order, so the prologue's reads
    // of x issued behind the weights would wait for all of them.  A plain x is
    // read into registers, the weights requested, and x stored to LDS after.
    constexpr int XR = (64 * U + NTH - 1) / NTH;     // x chunks per thread (K <= 512 U)
    u32x4 xr[XR];
    if constexpr (PRO == kPlain) {
#pragma unroll
        for (int i = 0; i < XR; ++i) xr[i] = *(const u32x4 *)(p.x + 8 * min(tid + NTH * i, KC - 1));
    } else {
        build_x<E, PRO, NTH>(p, xs, red, tid);
    }
    u32x4 wv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int c = min(lane + 64 * u, KC - 1);    // past K: loaded, never used
        wv[u] = *(const u32x4 *)(p.w + row * p.K + 8 * c);
    }
    if constexpr (PRO == kPlain) {
#pragma unroll
        for (int i = 0; i < XR; ++i)
            if (tid + NTH * i < KC) *(u32x4 *)(xs + 8 * (tid + NTH * i)) = xr[i];
    }
    __syncthreads();
    float acc = 0.f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int c = lane + 64 * u;
        if (c < KC) {
            const u32x4 xv = *(const u32x4 *)(xs + 8 * c);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                acc = __builtin_fmaf(E::lo(wv[u][i]), E::lo(xv[i]), acc);
                acc = __builtin_fmaf(E::hi(wv[u][i]), E::hi(xv[i]), acc);
            }
        }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0 && n < p.N) {
        float v = acc;
        if (p.beta) v += E::lo((uint32_t)p.y[n]);
        p.y[n] = (uint16_t)(E::pack2(v, 0.f) & 0xffffu);
    }
}

int grid_of(int64_t threads) {
    const int64_t b = (threads + NT - 1) / NT;
    return (int)(b < 16384 ? (b > 0 ? b : 1) : 16384);
}

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }
bool is16(int32_t dt) { return dt == KVR_BF16 || dt == KVR_F16; }
size_t up256(size_t b) { return (b + 255) / 256 * 256; }

// ---------------------------------------------------------------- products
struct Blas {
    hipblasLtHandle_t h = nullptr;
    // (rows, n_in, n_out, beta != 0, dtype) -> algorithm
    std::map<std::tuple<int64_t, int32_t, int32_t, int, int32_t>, hipblasLtMatmulAlgo_t> algos;
};

struct Gemm {
    hipblasLtMatmulDesc_t op = nullptr;
    hipblasLtMatrixLayout_t a = nullptr, b = nullptr, c = nullptr;
    ~Gemm() {
        if (a) hipblasLtMatrixLayoutDestroy(a);
        if (b) hipblasLtMatrixLayoutDestroy(b);
        if (c) hipblasLtMatrixLayoutDestroy(c);
        if (op) hipblasLtMatmulDescDestroy(op);
    }
};

int gemv(int32_t dtype, int pro, const void *x, const void *ln, float eps, const void *w, int32_t K, int64_t N,
         int beta, void *y, hipStream_t s);

// y = x w^T (+ y): in column-major terms y^T [n_out x rows] = w^T [n_out x n_in]
// (w stored as an n_in x n_out column-major matrix, transposed) times
// x^T [n_in x rows].
int linear(Blas *bl, int32_t dtype, const void *x, const void *w, int64_t rows, int32_t n_in, int32_t n_out,
           float beta, void *y, void *ws, size_t ws_bytes, hipStream_t s) {
    if (rows == 1 && n_in <= kGemvMaxK)
        return gemv(dtype, kPlain, x, nullptr, 0.f, w, n_in, n_out, beta != 0.f ? 1 : 0, y, s);
    const hipDataType ty = dtype == KVR_F16 ? HIP_R_16F : HIP_R_16BF;
    Gemm g;
    if (hipblasLtMatmulDescCreate(&g.op, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS)
        return KVR_ERR_DEVICE;
    const int32_t ta = HIPBLAS_OP_T, tb = HIPBLAS_OP_N;
    hipblasLtMatmulDescSetAttribute(g.op, HIPBLASLT_MATMUL_DESC_TRANSA, &ta, sizeof ta);
    hipblasLtMatmulDescSetAttribute(g.op, HIPBLASLT_MATMUL_DESC_TRANSB, &tb, sizeof tb);
    if (hipblasLtMatrixLayoutCreate(&g.a, ty, n_in, n_out, n_in) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&g.b, ty, n_in, rows, n_in) != HIPBLAS_STATUS_SUCCESS ||
        hipblasLtMatrixLayoutCreate(&g.c, ty, n_out, rows, n_out) != HIPBLAS_STATUS_SUCCESS)
        return KVR_ERR_DEVICE;
    const auto key = std::make_tuple(rows, n_in, n_out, beta != 0.f ? 1 : 0, dtype);
    auto it = bl->algos.find(key);
    if (it == bl->algos.end()) {
        hipblasLtMatmulPreference_t pref;
        if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) return KVR_ERR_DEVICE;
        const uint64_t wsb = KVR_BLAS_WORKSPACE_BYTES;
        hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsb, sizeof wsb);
        hipblasLtMatmulHeuristicResult_t res;
        int n = 0;
        const hipblasStatus_t st =
            hipblasLtMatmulAlgoGetHeuristic(bl->h, g.op, g.a, g.b, g.c, g.c, pref, 1, &res, &n);
        hipblasLtMatmulPreferenceDestroy(pref);
        if (st != HIPBLAS_STATUS_SUCCESS || n < 1) return KVR_ERR_DEVICE;
        it = bl->algos.emplace(key, res.algo).first;
    }
    const float alpha = 1.f;
    const hipblasStatus_t st = hipblasLtMatmul(bl->h, g.op, &alpha, w, g.a, x, g.b, &beta, y, g.c, y, g.c,
                                               &it->second, ws, ws_bytes, s);
    return st == HIPBLAS_STATUS_SUCCESS ? KVR_OK : KVR_ERR_DEVICE;
}

// One-row product: up to kGemv1MaxRows outputs with rows of at most
// kGemv1MaxSteps loads per lane, one row per wave and all loads at once;
// otherwise at most kGemvMaxGrid workgroups of GT threads, one row per wave and
// step (two for outputs of 65536 rows and more).
int gemv(int32_t dtype, int pro, const void *x, const void *ln, float eps, const void *w, int32_t K, int64_t N,
         int beta, void *y, hipStream_t s) {
    GemvParams g;
    g.x = (const uint16_t *)x;
    g.w = (const uint16_t *)w;
    g.ln = (const uint16_t *)ln;
    g.y = (uint16_t *)y;
    g.N = N;
    g.K = K;
    g.beta = beta;
    g.eps = eps;
    const int steps = (K / 8 + 63) / 64;
    if (N <= kGemv1MaxRows && steps <= kGemv1MaxSteps) {
        // waves per workgroup: the fewest rows on the busiest CU (kGemv1Cus
        // compute units, one workgroup each per round), ties to the larger
        // workgroup (fewer prologues): 2560 rows -> 10 waves, 6144 -> 12
        int nwv = 8;
        int64_t best = -1;
        for (const int c : {8, 10, 12, 16}) {
            const int64_t wgs = (N + c - 1) / c;
            const int64_t busiest = (wgs + kGemv1Cus - 1) / kGemv1Cus * c;
            if (best < 0 || busiest <= best) { best = busiest; nwv = c; }
        }
        const dim3 grid1((unsigned)((N + nwv - 1) / nwv));
#define KVR_GEMV1_W(E_, P_, U_, W_) hipLaunchKernelGGL((gemv1_kernel<E_, P_, U_, W_>), grid1, dim3(64 * W_), 0, s, g)
#define KVR_GEMV1(E_, P_, U_) do { if (nwv == 10) KVR_GEMV1_W(E_, P_, U_, 10); else if (nwv == 12) KVR_GEMV1_W(E_, P_, U_, 12); \
                                   else if (nwv == 16) KVR_GEMV1_W(E_, P_, U_, 16); else KVR_GEMV1_W(E_, P_, U_, 8); } while (0)
#define KVR_GEMV1_U(E_, P_) do { if (steps <= 5) KVR_GEMV1(E_, P_, 5); else if (steps <= 8) KVR_GEMV1(E_, P_, 8); \
                                 else KVR_GEMV1(E_, P_, kGemv1MaxSteps); } while (0)
#define KVR_GEMV1_PRO(E_) do { if (pro == kNorm) KVR_GEMV1_U(E_, kNorm); else if (pro == kSilu) KVR_GEMV1_U(E_, kSilu); \
                               else KVR_GEMV1_U(E_, kPlain); } while (0)
        if (dtype == KVR_F16) KVR_GEMV1_PRO(F16);
        else KVR_GEMV1_PRO(Bf16);
#undef KVR_GEMV1_PRO
#undef KVR_GEMV1_U
#undef KVR_GEMV1
#undef KVR_GEMV1_W
        return hipGetLastError() == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
    }
    const int rw = N >= 65536 ? 2 : 1;
    const int64_t groups = (N + rw * (GT / 64) - 1) / (rw * (GT / 64));
    const dim3 grid((unsigned)(groups < kGemvMaxGrid ? groups : kGemvMaxGrid));
#define KVR_GEMV(E_, P_, R_) hipLaunchKernelGGL((gemv_kernel<E_, P_, R_>), grid, dim3(GT), 0, s, g)
#define KVR_GEMV_RW(E_, P_) do { if (rw == 2) KVR_GEMV(E_, P_, 2); else KVR_GEMV(E_, P_, 1); } while (0)
#define KVR_GEMV_PRO(E_) do { if (pro == kNorm) KVR_GEMV_RW(E_, kNorm); else if (pro == kSilu) KVR_GEMV_RW(E_, kSilu); \
                              else KVR_GEMV_RW(E_, kPlain); } while (0)
    if (dtype == KVR_F16) KVR_GEMV_PRO(F16);
    else KVR_GEMV_PRO(Bf16);
#undef KVR_GEMV_PRO
#undef KVR_GEMV_RW
#undef KVR_GEMV
    return hipGetLastError() == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
}

// act[n] = silu(x' wg[n]) * (x' wg[I + n]) for one row x, x' = rmsnorm(x) * ln:
// the gate and up products of the one-token step, paired in each wave.
int gemv_gate_up(int32_t dtype, const void *x, const void *ln, float eps, const void *w, int32_t K, int64_t I,
                 void *act, hipStream_t s) {
    GemvParams g;
    g.x = (const uint16_t *)x;
    g.w = (const uint16_t *)w;
    g.ln = (const uint16_t *)ln;
    g.y = (uint16_t *)act;
    g.N = I;
    g.K = K;
    g.beta = 0;
    g.eps = eps;
    const int64_t groups = (I + GT / 64 - 1) / (GT / 64);
    const dim3 grid((unsigned)(groups < kGemvMaxGrid ? groups : kGemvMaxGrid));
    if (dtype == KVR_F16) hipLaunchKernelGGL((gemv_kernel<F16, kNorm, 2, 1>), grid, dim3(GT), 0, s, g);
    else hipLaunchKernelGGL((gemv_kernel<Bf16, kNorm, 2, 1>), grid, dim3(GT), 0, s, g);
    return hipGetLastError() == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
}

int check_shape(const kvr_desc *d, const kvr_layer_shape *sh) {
    if (!d || !sh) return KVR_ERR_NULL;
    if (!is16(d->dtype)) return KVR_ERR_DTYPE;
    if (d->n_q_heads <= 0 || d->n_kv_heads <= 0 || d->n_q_heads % d->n_kv_heads) return KVR_ERR_SHAPE;
    if (d->head_dim != 64 && d->head_dim != 128) return KVR_ERR_SHAPE;
    if (sh->hidden <= 0 || sh->hidden % 8 || sh->hidden > 65536) return KVR_ERR_SHAPE;
    if (sh->intermediate <= 0 || sh->intermediate % 8 || sh->intermediate > 262144) return KVR_ERR_SHAPE;
    if (!(sh->eps >= 0.f) || isinf(sh->eps) || sh->reserved != 0) return KVR_ERR_SHAPE;
    return KVR_OK;
}

struct LayerWs {
    size_t xn, qkv, q, k, v, att, gu, act, split, blas, total;
};

LayerWs layer_ws(const kvr_desc *d, const kvr_layer_shape *sh, int64_t T, int64_t Lmax) {
    LayerWs w;
    const size_t e = 2, Hq = d->n_q_heads, Hkv = d->n_kv_heads, D = d->head_dim;
    size_t o = 0;
    auto take = [&](size_t b) { const size_t at = o; o += up256(b); return at; };
    w.xn = take((size_t)T * sh->hidden * e);
    w.qkv = take((size_t)T * (Hq + 2 * Hkv) * D * e);
    w.q = take((size_t)T * Hq * D * e);
    w.k = take((size_t)T * Hkv * D * e);
    w.v = take((size_t)T * Hkv * D * e);
    w.att = take((size_t)T * Hq * D * e);
    w.gu = take((size_t)T * 2 * sh->intermediate * e);
    w.act = take((size_t)T * sh->intermediate * e);
    const size_t sb = kvr_workspace_bytes(d, Lmax, T, 1);
    w.split = take(sb == (size_t)-1 ? 0 : sb);
    w.blas = take(KVR_BLAS_WORKSPACE_BYTES);
    w.total = o;
    return w;
}

}  // namespace
}  // namespace model
}  // namespace kvr

using namespace kvr::model;

extern "C" {

int kvr_model_abi_version(void) { return KVR_MODEL_ABI_VERSION; }

int kvr_blas_create(void **blas) {
    if (!blas) return KVR_ERR_NULL;
    Blas *b = new Blas();
    if (hipblasLtCreate(&b->h) != HIPBLAS_STATUS_SUCCESS) {
        delete b;
        *blas = nullptr;
        return KVR_ERR_DEVICE;
    }
    *blas = b;
    return KVR_OK;
}

int kvr_blas_destroy(void *blas) {
    if (!blas) return KVR_ERR_NULL;
    Blas *b = (Blas *)blas;
    if (b->h) hipblasLtDestroy(b->h);
    delete b;
    return KVR_OK;
}

int kvr_linear(void *blas, int32_t dtype, const void *x, const void *w, int64_t rows, int32_t n_in, int32_t n_out,
               float beta, void *y, void *ws, size_t ws_bytes, void *stream) {
    if (!is16(dtype)) return KVR_ERR_DTYPE;
    if (rows < 0 || rows > ((int64_t)1 << 30) || n_in <= 0 || n_out <= 0 || n_in % 8 || n_out % 8)
        return KVR_ERR_SHAPE;
    if (beta != 0.f && beta != 1.f) return KVR_ERR_SHAPE;
    if (rows == 0) return KVR_OK;
    if (!blas || !x || !w || !y || !ws) return KVR_ERR_NULL;
    if (ws_bytes < KVR_BLAS_WORKSPACE_BYTES) return KVR_ERR_WORKSPACE;
    if (!aligned16(x) || !aligned16(w) || !aligned16(y) || !aligned16(ws)) return KVR_ERR_ALIGN;
    return linear((Blas *)blas, dtype, x, w, rows, n_in, n_out, beta, y, ws, ws_bytes, (hipStream_t)stream);
}

int kvr_rmsnorm(int32_t dtype, const void *x, const void *w, int64_t rows, int32_t n, float eps, void *y,
                void *stream) {
    if (!is16(dtype)) return KVR_ERR_DTYPE;
    if (rows < 0 || rows > 0x7fffffff || n <= 0 || n % 8 || n > 65536 || !(eps >= 0.f) || isinf(eps))
        return KVR_ERR_SHAPE;
    if (rows == 0) return KVR_OK;
    if (!x || !w || !y) return KVR_ERR_NULL;
    if (!aligned16(x) || !aligned16(w) || !aligned16(y)) return KVR_ERR_ALIGN;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == KVR_F16)
        hipLaunchKernelGGL(rmsnorm_kernel<F16>, dim3((unsigned)rows), dim3(NT), 0, s, (const uint16_t *)x,
                           (const uint16_t *)w, (uint16_t *)y, n, eps);
    else
        hipLaunchKernelGGL(rmsnorm_kernel<Bf16>, dim3((unsigned)rows), dim3(NT), 0, s, (const uint16_t *)x,
                           (const uint16_t *)w, (uint16_t *)y, n, eps);
    return hipGetLastError() == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
}

size_t kvr_layer_workspace_bytes(const kvr_desc *desc, const kvr_layer_shape *shape, int64_t T,
                                 int64_t L_prefix_max) {
    if (check_shape(desc, shape) != KVR_OK || T < 0 || L_prefix_max < 0) return (size_t)-1;
    return layer_ws(desc, shape, T, L_prefix_max).total;
}

int kvr_layer_forward(const kvr_desc *desc, const kvr_layer_shape *shape, const kvr_layer_weights *w,
                      const kvr_rope *rope, void *blas, void *h, int64_t T, int64_t L_prefix, void *kcache,
                      void *vcache, void *ws, size_t ws_bytes, void *stream) {
    int st = check_shape(desc, shape);
    if (st) return st;
    if (T < 0 || T > ((int64_t)1 << 24) || L_prefix < 0) return KVR_ERR_SHAPE;
    // one wave per (token, head) of the q/k/v rows: the grid must fit 32 bits
    if (T * (desc->n_q_heads + 2 * (int64_t)desc->n_kv_heads) > 0x7fffffffLL) return KVR_ERR_SHAPE;
    if (L_prefix + T > desc->capacity) return KVR_ERR_CAPACITY;
    if (T == 0) return KVR_OK;
    if (!w || !rope || !blas || !h || !kcache || !vcache || !ws) return KVR_ERR_NULL;
    if (!w->ln1 || !w->wqkv || !w->q_norm || !w->k_norm || !w->wo || !w->ln2 || !w->wgu || !w->wd || !rope->cos_sin)
        return KVR_ERR_NULL;
    if (rope->n_pos < L_prefix + T) return KVR_ERR_POSITION;
    const LayerWs lw = layer_ws(desc, shape, T, L_prefix);
    if (ws_bytes < lw.total) return KVR_ERR_WORKSPACE;
    const void *ptrs[] = {w->ln1, w->wqkv, w->q_norm, w->k_norm, w->wo, w->ln2, w->wgu, w->wd,
                          rope->cos_sin, h, kcache, vcache, ws};
    for (const void *p : ptrs)
        if (!aligned16(p)) return KVR_ERR_ALIGN;

    hipStream_t s = (hipStream_t)stream;
    unsigned char *b = (unsigned char *)ws;
    Blas *bl = (Blas *)blas;
    const int32_t dt = desc->dtype;
    const int Hq = desc->n_q_heads, Hkv = desc->n_kv_heads, D = desc->head_dim;
    const int H = shape->hidden, I = shape->intermediate;
    const int Wq = (Hq + 2 * Hkv) * D;
    void *blws = b + lw.blas;

    // one token: the one-row products with the norms and the activation in
    // their prologues; more tokens: separate norm / activation kernels and
    // hipBLASLt products
    const bool one = T == 1 && H <= kGemvMaxK && I <= kGemvMaxK && Hq * D <= kGemvMaxK;

    // attention block
    if (one) {
        if ((st = gemv(dt, kNorm, h, w->ln1, shape->eps, w->wqkv, H, Wq, 0, b + lw.qkv, s))) return st;
    } else {
        if ((st = kvr_rmsnorm(dt, h, w->ln1, T, H, shape->eps, b + lw.xn, stream))) return st;
        if ((st = linear(bl, dt, b + lw.xn, w->wqkv, T, H, Wq, 0.f, b + lw.qkv, blws, KVR_BLAS_WORKSPACE_BYTES, s)))
            return st;
    }
    QkParams qp;
    qp.qkv = (const uint16_t *)(b + lw.qkv);
    qp.qn = (const uint16_t *)w->q_norm;
    qp.kn = (const uint16_t *)w->k_norm;
    qp.cs = rope->cos_sin;
    qp.q = (uint16_t *)(b + lw.q);
    qp.k = (uint16_t *)(b + lw.k);
    qp.v = (uint16_t *)(b + lw.v);
    // a prefill writes its own cache rows inside the attention kernel
    qp.kc = L_prefix > 0 ? (uint16_t *)kcache : nullptr;
    qp.vc = L_prefix > 0 ? (uint16_t *)vcache : nullptr;
    qp.T = T;
    qp.pos0 = L_prefix;
    qp.cap = desc->capacity;
    qp.Hq = Hq;
    qp.Hkv = Hkv;
    qp.eps = shape->eps;
    const int64_t waves = T * (Hq + 2 * Hkv);
    const dim3 qg((unsigned)((waves + NT / 64 - 1) / (NT / 64)));
    if (dt == KVR_F16) {
        if (D == 128) hipLaunchKernelGGL((qk_norm_rope_kernel<F16, 128>), qg, dim3(NT), 0, s, qp);
        else hipLaunchKernelGGL((qk_norm_rope_kernel<F16, 64>), qg, dim3(NT), 0, s, qp);
    } else {
        if (D == 128) hipLaunchKernelGGL((qk_norm_rope_kernel<Bf16, 128>), qg, dim3(NT), 0, s, qp);
        else hipLaunchKernelGGL((qk_norm_rope_kernel<Bf16, 64>), qg, dim3(NT), 0, s, qp);
    }
    if (hipGetLastError() != hipSuccess) return KVR_ERR_DEVICE;
    if (L_prefix == 0)
        st = kvr_prefill(desc, b + lw.q, b + lw.k, b + lw.v, T, b + lw.att, kcache, vcache, stream);
    else
        st = kvr_continue(desc, b + lw.q, b + lw.k, b + lw.v, kcache, vcache, L_prefix, T, b + lw.att,
                          b + lw.split, lw.blas - lw.split, stream);
    if (st) return st;
    if ((st = linear(bl, dt, b + lw.att, w->wo, T, Hq * D, H, 1.f, h, blws, KVR_BLAS_WORKSPACE_BYTES, s)))
        return st;
    // MLP block
    if (one) {
        if ((st = gemv_gate_up(dt, h, w->ln2, shape->eps, w->wgu, H, I, b + lw.act, s))) return st;
        return gemv(dt, kPlain, b + lw.act, nullptr, 0.f, w->wd, I, H, 1, h, s);
    }
    if ((st = kvr_rmsnorm(dt, h, w->ln2, T, H, shape->eps, b + lw.xn, stream))) return st;
    if ((st = linear(bl, dt, b + lw.xn, w->wgu, T, H, 2 * I, 0.f, b + lw.gu, blws, KVR_BLAS_WORKSPACE_BYTES, s)))
        return st;
    if (dt == KVR_F16)
        hipLaunchKernelGGL(silu_mul_kernel<F16>, dim3(grid_of(T * (I / 8))), dim3(NT), 0, s,
                           (const uint16_t *)(b + lw.gu), (uint16_t *)(b + lw.act), T, I);
    else
        hipLaunchKernelGGL(silu_mul_kernel<Bf16>, dim3(grid_of(T * (I / 8))), dim3(NT), 0, s,
                           (const uint16_t *)(b + lw.gu), (uint16_t *)(b + lw.act), T, I);
    if (hipGetLastError() != hipSuccess) return KVR_ERR_DEVICE;
    return linear(bl, dt, b + lw.act, w->wd, T, I, H, 1.f, h, blws, KVR_BLAS_WORKSPACE_BYTES, s);
}

}  // extern "C"
