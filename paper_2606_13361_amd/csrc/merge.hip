// merge.hip -- combine the per-split partial results of a split continuation
// (16-bit outputs: bf16 or fp16 as the descriptor says)
// (fixed split order, so the result is reproducible bit for bit):
//   M = max_s m_s,  w_s = 2^(m_s - M),  out = sum_s w_s O_s / sum_s w_s l_s
// which is the log-sum-exp merge of partial softmax sums.
//
// One lane per 4 consecutive head-dim values of one row: a 64-lane
// workgroup covers 64 / (D/4) rows of one kv head (2 at D = 128, 4 at
// D = 64), so the partials of a continuation are read by many compute units
// at once.  The lanes of a row first build the split weights together --
// lane k takes splits k, k + D/4, ...; the row maximum and l come from xor
// butterflies inside the row's lanes (same bits in every lane); the weights
// go through LDS -- then every lane streams its 16 bytes of every split with
// 16 loads in flight.  Block b serves kv head b % Hkv, the same residue the
// attention kernel gives the head's blocks, so with 8 kv heads the partials
// are read on the XCD whose L2 took them.
#include <type_traits>

#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int MERGE_THREADS = 64;
constexpr int MERGE_BATCH = 16;   // split loads in flight per lane (more than 32 splits)

template <int D, class E>
__global__ __launch_bounds__(MERGE_THREADS) void merge_bf16_kernel(const MergeParams p) {
    constexpr int CPR = D / 4;                 // lanes per row
    constexpr int RPW = MERGE_THREADS / CPR;   // rows per workgroup
    __shared__ float wts[RPW][kMaxSplits + 1];
    const int tid = threadIdx.x;
    const int rr = tid / CPR;
    const int part = tid % CPR;
    const int g = blockIdx.x % p.n_kv_heads;
    const int r0 = (blockIdx.x / p.n_kv_heads) * RPW;
    const int r = r0 + rr;
    const bool valid = r < p.rows;
    const int64_t per_split = (int64_t)p.n_kv_heads * p.rows;
    const float *ml = p.ws + (int64_t)p.nsplit * per_split * D;
    const int64_t row = (int64_t)g * p.rows + (valid ? r : r0);   // rows past the end read row r0
    const float *src = p.ws + row * D + 4 * part;
    const int64_t sstride = per_split * D;
    auto store_row = [&](const float4 &acc, float l) {
        const float il = l > 0.f ? 1.f / l : 0.f;
        const int tok = r / p.group;
        const int head = g * p.group + r % p.group;
        uint16_t *out = (uint16_t *)p.out + ((int64_t)tok * p.n_q_heads + head) * D + 4 * part;
        u32x2 v;
        v[0] = E::pack2(acc.x * il, acc.y * il);
        v[1] = E::pack2(acc.z * il, acc.w * il);
        *(u32x2 *)out = v;
    };

    // up to 16 or 32 splits: every split's (m, l) and partial row at once, one
    // memory round trip; each lane reads all of its row's records itself (the
    // row's lanes read the same addresses), no LDS and no shuffles.  Indices
    // past nsplit re-read the last split and get weight 0.
    auto one_trip = [&](auto ns_tag) {
        constexpr int NS = decltype(ns_tag)::value;
        float4 o[NS];
        float2 ml2[NS];
#pragma unroll
        for (int k = 0; k < NS; ++k) o[k] = *(const float4 *)(src + min(k, p.nsplit - 1) * sstride);
#pragma unroll
        for (int k = 0; k < NS; ++k) ml2[k] = *(const float2 *)(ml + (min(k, p.nsplit - 1) * per_split + row) * 2);
        __builtin_amdgcn_sched_barrier(0);   // every load issued before any use
        float M = -INFINITY;
#pragma unroll
        for (int k = 0; k < NS; ++k) M = fmaxf(M, ml2[k].x);
        float l = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int k = 0; k < NS; ++k) {
            const float w = k < p.nsplit ? __builtin_amdgcn_exp2f(ml2[k].x - M) : 0.f;
            l = __builtin_fmaf(w, ml2[k].y, l);
            acc.x = __builtin_fmaf(w, o[k].x, acc.x);
            acc.y = __builtin_fmaf(w, o[k].y, acc.y);
            acc.z = __builtin_fmaf(w, o[k].z, acc.z);
            acc.w = __builtin_fmaf(w, o[k].w, acc.w);
        }
        if (valid) store_row(acc, l);
    };
    if (p.nsplit <= 16) {
        one_trip(std::integral_constant<int, 16>{});
        return;
    }
    if (p.nsplit <= 32) {
        one_trip(std::integral_constant<int, 32>{});
        return;
    }

    // the first MERGE_BATCH splits' partial rows do not depend on the
    // weights: their loads go out before the (m, l) round trip (split indices
    // past nsplit re-read the last split and are never used)
    float4 o0[MERGE_BATCH];
#pragma unroll
    for (int k = 0; k < MERGE_BATCH; ++k) o0[k] = *(const float4 *)(src + min(k, p.nsplit - 1) * sstride);

    float M = -INFINITY;
    for (int s = part; s < p.nsplit; s += CPR) M = fmaxf(M, ml[(s * per_split + row) * 2]);
#pragma unroll
    for (int x = 1; x < CPR; x <<= 1) M = fmaxf(M, __shfl_xor(M, x));
    float l = 0.f;
    for (int s = part; s < p.nsplit; s += CPR) {
        const float2 v = *(const float2 *)(ml + (s * per_split + row) * 2);
        const float w = __builtin_amdgcn_exp2f(v.x - M);
        wts[rr][s] = w;
        l = __builtin_fmaf(w, v.y, l);
    }
#pragma unroll
    for (int x = 1; x < CPR; x <<= 1) l += __shfl_xor(l, x);
    __syncthreads();
    if (!valid) return;

    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    const int n0 = p.nsplit < MERGE_BATCH ? p.nsplit : MERGE_BATCH;
#pragma unroll
    for (int k = 0; k < MERGE_BATCH; ++k) {
        if (k < n0) {
            const float w = wts[rr][k];
            acc.x = __builtin_fmaf(w, o0[k].x, acc.x);
            acc.y = __builtin_fmaf(w, o0[k].y, acc.y);
            acc.z = __builtin_fmaf(w, o0[k].z, acc.z);
            acc.w = __builtin_fmaf(w, o0[k].w, acc.w);
        }
    }
    int s = n0;
    for (; s + MERGE_BATCH <= p.nsplit; s += MERGE_BATCH) {
        float4 o[MERGE_BATCH];
#pragma unroll
        for (int k = 0; k < MERGE_BATCH; ++k) o[k] = *(const float4 *)(src + (s + k) * sstride);
#pragma unroll
        for (int k = 0; k < MERGE_BATCH; ++k) {
            const float w = wts[rr][s + k];
            acc.x = __builtin_fmaf(w, o[k].x, acc.x);
            acc.y = __builtin_fmaf(w, o[k].y, acc.y);
            acc.z = __builtin_fmaf(w, o[k].z, acc.z);
            acc.w = __builtin_fmaf(w, o[k].w, acc.w);
        }
    }
    for (; s < p.nsplit; ++s) {
        const float4 o = *(const float4 *)(src + s * sstride);
        const float w = wts[rr][s];
        acc.x = __builtin_fmaf(w, o.x, acc.x);
        acc.y = __builtin_fmaf(w, o.y, acc.y);
        acc.z = __builtin_fmaf(w, o.z, acc.z);
        acc.w = __builtin_fmaf(w, o.w, acc.w);
    }
    store_row(acc, l);
}

}  // namespace

hipError_t launch_merge_bf16(const MergeParams &p, int head_dim, bool f16, hipStream_t s) {
    const int rpw = MERGE_THREADS / (head_dim / 4);
    const int grid = (p.rows + rpw - 1) / rpw * p.n_kv_heads;
    if (head_dim == 128) {
        if (f16) hipLaunchKernelGGL((merge_bf16_kernel<128, F16>), dim3(grid), dim3(MERGE_THREADS), 0, s, p);
        else hipLaunchKernelGGL((merge_bf16_kernel<128, Bf16>), dim3(grid), dim3(MERGE_THREADS), 0, s, p);
    } else {
        if (f16) hipLaunchKernelGGL((merge_bf16_kernel<64, F16>), dim3(grid), dim3(MERGE_THREADS), 0, s, p);
        else hipLaunchKernelGGL((merge_bf16_kernel<64, Bf16>), dim3(grid), dim3(MERGE_THREADS), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace kvr
