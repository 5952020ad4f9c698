// append.hip -- cache write: rows [L_cur, L_cur+S) of every kv head receive
// the new K/V rows bit for bit (the cache update of a decode step, and the
// cache fill of a prefill).  Pure 16-byte copies: a K/V row of head_dim
// elements is row_chunks 16-byte chunks; one lane moves one chunk of K and
// the same chunk of V.
#include "kvr_internal.hpp"

namespace kvr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void append_kernel(const AppendParams p) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t per_row = p.row_chunks;
    const int64_t total = p.S * p.n_kv_heads * per_row;
    if (idx >= total) return;
    const int64_t c = idx % per_row;
    const int64_t src_row = idx / per_row;          // t * n_kv_heads + g
    const int64_t t = src_row / p.n_kv_heads;
    const int64_t g = src_row % p.n_kv_heads;
    const int64_t dst_row = g * p.cap + p.L_cur + t;
    const u32x4 *ks = (const u32x4 *)p.k + src_row * per_row + c;
    const u32x4 *vs = (const u32x4 *)p.v + src_row * per_row + c;
    u32x4 *kd = (u32x4 *)p.kc + dst_row * per_row + c;
    u32x4 *vd = (u32x4 *)p.vc + dst_row * per_row + c;
    *kd = *ks;
    *vd = *vs;
}

}  // namespace

hipError_t launch_append(const AppendParams &p, hipStream_t s) {
    const int64_t total = p.S * p.n_kv_heads * p.row_chunks;
    const int64_t grid = (total + 255) / 256;
    hipLaunchKernelGGL(append_kernel, dim3((unsigned)grid), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace kvr
