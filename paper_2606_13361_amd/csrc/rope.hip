// rope.hip -- rotary position embedding: the cos/sin table and the pre-pass
// that rotates key rows (and, for continuations, query rows) once, before the
// attention kernels read them.
//
// The paper's exactness condition on positions (Section "Consuming an
// artifact"): a continuation's tokens sit at positions L, L+1, ... where L is
// the artifact's length, so their rotation matches a pass from scratch.  The
// pre-pass takes every row's position from the call (pos0 plus the row's
// index within its segment); the cache holds rotated keys.
//
// Keys are rotated here rather than inside the attention kernels because
// every key row is read by many workgroups (all query tiles of its kv head):
// rotating it once costs one pass over K, rotating it on every read would
// cost one per workgroup.  Query rows of prefill and many readers are rotated
// in registers by the attention kernels themselves (each row is read once).
#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int RT = 256;

__device__ __forceinline__ int64_t row_position(const RopeParams &p, int64_t t) {
    int lo = 0, hi = p.n_seg - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (p.seg_tok0[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return p.pos0 + t - p.seg_tok0[lo];
}

// cos and sin of p * theta_i, theta_i = base^(-2i/d): the angle and both
// functions in fp64, rounded once to fp32.
__global__ __launch_bounds__(RT) void rope_table_kernel(float *cs, int half, double base, int64_t n) {
    for (int64_t idx = (int64_t)blockIdx.x * RT + threadIdx.x; idx < n; idx += (int64_t)gridDim.x * RT) {
        const int64_t pos = idx / half;
        const int i = (int)(idx % half);
        const double theta = pow(base, -(double)(2 * i) / (double)(2 * half));
        const double a = (double)pos * theta;
        float2 v;
        v.x = (float)cos(a);
        v.y = (float)sin(a);
        *(float2 *)(cs + 2 * idx) = v;
    }
}

// One thread per (row, chunk c): dims 8c..8c+7 and their partners d/2 + 8c...
template <class E, int D>
__global__ __launch_bounds__(RT) void rope16_kernel(const RopeParams p) {
    const RopeJob &J = blockIdx.y ? p.job[1] : p.job[0];
    constexpr int CH = D / 16;
    const int64_t total = p.n_tok * J.n_heads * CH;
    for (int64_t idx = (int64_t)blockIdx.x * RT + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * RT) {
        const int c = (int)(idx % CH);
        const int64_t row = idx / CH;
        const int h = (int)(row % J.n_heads);
        const int64_t t = row / J.n_heads;
        const int64_t pos = row_position(p, t);
        const uint16_t *xr = (const uint16_t *)J.x + row * D;
        u32x4 lo = *(const u32x4 *)(xr + 8 * c);
        u32x4 hi = *(const u32x4 *)(xr + D / 2 + 8 * c);
        rope_rot8<E>(lo, hi, p.cs + pos * D + 16 * c);
        if (J.y) {
            uint16_t *yr = (uint16_t *)J.y + row * D;
            *(u32x4 *)(yr + 8 * c) = lo;
            *(u32x4 *)(yr + D / 2 + 8 * c) = hi;
        }
        const int64_t crow = ((int64_t)h * p.cap + pos) * D;
        if (J.cache) {
            uint16_t *cr = (uint16_t *)J.cache + crow;
            *(u32x4 *)(cr + 8 * c) = lo;
            *(u32x4 *)(cr + D / 2 + 8 * c) = hi;
        }
        if (J.v) {
            const uint16_t *vr = (const uint16_t *)J.v + row * D;
            uint16_t *vcr = (uint16_t *)J.vcache + crow;
            *(u32x4 *)(vcr + 8 * c) = *(const u32x4 *)(vr + 8 * c);
            *(u32x4 *)(vcr + D / 2 + 8 * c) = *(const u32x4 *)(vr + D / 2 + 8 * c);
        }
    }
}

// fp32 rows: the same rotation without rounding.
template <int D>
__global__ __launch_bounds__(RT) void rope32_kernel(const RopeParams p) {
    const RopeJob &J = blockIdx.y ? p.job[1] : p.job[0];
    constexpr int CH = D / 8;      // 4 dims and their partners per thread
    const int64_t total = p.n_tok * J.n_heads * CH;
    for (int64_t idx = (int64_t)blockIdx.x * RT + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * RT) {
        const int c = (int)(idx % CH);
        const int64_t row = idx / CH;
        const int h = (int)(row % J.n_heads);
        const int64_t t = row / J.n_heads;
        const int64_t pos = row_position(p, t);
        const float *xr = (const float *)J.x + row * D;
        const float4 a = *(const float4 *)(xr + 4 * c);
        const float4 b = *(const float4 *)(xr + D / 2 + 4 * c);
        const float4 *cs = (const float4 *)(p.cs + pos * D + 8 * c);
        const float4 c01 = cs[0], c23 = cs[1];
        float4 ya, yb;
        rope_rot(a.x, b.x, c01.x, c01.y, ya.x, yb.x);
        rope_rot(a.y, b.y, c01.z, c01.w, ya.y, yb.y);
        rope_rot(a.z, b.z, c23.x, c23.y, ya.z, yb.z);
        rope_rot(a.w, b.w, c23.z, c23.w, ya.w, yb.w);
        if (J.y) {
            float *yr = (float *)J.y + row * D;
            *(float4 *)(yr + 4 * c) = ya;
            *(float4 *)(yr + D / 2 + 4 * c) = yb;
        }
        const int64_t crow = ((int64_t)h * p.cap + pos) * D;
        if (J.cache) {
            float *cr = (float *)J.cache + crow;
            *(float4 *)(cr + 4 * c) = ya;
            *(float4 *)(cr + D / 2 + 4 * c) = yb;
        }
        if (J.v) {
            const float *vr = (const float *)J.v + row * D;
            float *vcr = (float *)J.vcache + crow;
            *(float4 *)(vcr + 4 * c) = *(const float4 *)(vr + 4 * c);
            *(float4 *)(vcr + D / 2 + 4 * c) = *(const float4 *)(vr + D / 2 + 4 * c);
        }
    }
}

int grid_for(int64_t threads) {
    const int64_t b = (threads + RT - 1) / RT;
    return (int)(b < 8192 ? (b > 0 ? b : 1) : 8192);
}

template <int D>
hipError_t launch_d(const RopeParams &p, int elt, hipStream_t s) {
    int64_t most = 0;
    for (int j = 0; j < p.n_jobs; ++j) {
        const int64_t n = p.n_tok * p.job[j].n_heads;
        most = n > most ? n : most;
    }
    const int per_row = elt == 1 ? D / 8 : D / 16;
    const dim3 grid(grid_for(most * per_row), p.n_jobs);
    if (elt == 1)
        hipLaunchKernelGGL(rope32_kernel<D>, grid, dim3(RT), 0, s, p);
    else if (elt == 2)
        hipLaunchKernelGGL((rope16_kernel<F16, D>), grid, dim3(RT), 0, s, p);
    else
        hipLaunchKernelGGL((rope16_kernel<Bf16, D>), grid, dim3(RT), 0, s, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_rope(const RopeParams &p, int head_dim, int elt, hipStream_t s) {
    if (p.n_tok <= 0 || p.n_jobs <= 0) return hipSuccess;
    return head_dim == 128 ? launch_d<128>(p, elt, s) : launch_d<64>(p, elt, s);
}

hipError_t launch_rope_table(float *cs, int head_dim, double base, int64_t n_pos, hipStream_t s) {
    const int half = head_dim / 2;
    const int64_t n = n_pos * half;
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(rope_table_kernel, dim3(grid_for(n)), dim3(RT), 0, s, cs, half, base, n);
    return hipGetLastError();
}

}  // namespace kvr
