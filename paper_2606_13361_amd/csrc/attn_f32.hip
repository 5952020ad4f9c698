// attn_f32.hip -- the fp32 member of the attention family: the same rows,
// segments and causal offset as the bf16 kernel, computed entirely in fp32 on
// the vector ALUs (no reduced-precision matrix instructions), for inputs whose
// tolerance is 1e-5.
//
// Workgroup: 64 query rows x 4 lanes per row; each lane owns a quarter of the
// head dim of its row (q and the output accumulator live in registers).  Key
// tiles of 32 rows are staged in LDS and read by every row of the workgroup.
#include "attn_common.hpp"

namespace kvr {
namespace {

using dev::rope_rot;

constexpr int ROWS = kRowsF32;
constexpr int LANES_PER_ROW = 4;
constexpr int THREADS = ROWS * LANES_PER_ROW;
constexpr int KT = 32;   // keys per LDS tile

__device__ __forceinline__ int find_segment_f32(const AttnParams &p, int tile) {
    int lo = 0, hi = p.n_seg - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (p.seg_tile0[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    return lo;
}

template <int D>
__global__ __launch_bounds__(THREADS) void attn_f32_kernel(const AttnParams p) {
    constexpr int DQ = D / LANES_PER_ROW;   // head-dim slice per lane
    __shared__ __attribute__((aligned(16))) float ks[KT][D];
    __shared__ __attribute__((aligned(16))) float vs[KT][D];

    const int tid = threadIdx.x;
    const int part = tid % LANES_PER_ROW;

    int b = blockIdx.x;
    const int g = b % p.n_kv_heads;
    b /= p.n_kv_heads;
    const int tile_lin = p.reverse ? (p.tiles_total - 1 - b) : b;
    const int seg = find_segment_f32(p, tile_lin);
    const int rt = tile_lin - p.seg_tile0[seg];
    const int tok0 = p.seg_tok0[seg];
    const int n_tok = p.seg_tok0[seg + 1] - tok0;
    const int G = p.group;
    const int R = G * n_tok;
    const int row0 = rt * ROWS;
    const int row_last = min(row0 + ROWS, R) - 1;
    const int64_t npre = p.n_prefix;

    const int r = row0 + tid / LANES_PER_ROW;
    const bool valid = r < R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int64_t pos = valid ? npre + tok : -1;
    const int64_t ke = npre + row_last / G + 1;

    float q[DQ], o[DQ];
    {
        const float *qrow = (const float *)p.q + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D + part * DQ;
#pragma unroll
        for (int c = 0; c < DQ; ++c) {
            q[c] = valid ? qrow[c] : 0.f;
            o[c] = 0.f;
        }
        // RoPE (prefill, readers): dim i < D/2 of the row pairs with dim
        // i + D/2, which the lane two over (part + 2) holds
        if (p.rope) {
            const int half = part & 1;              // which DQ-slice of the pair index
            const bool upper = part >= 2;
            const float *cs = p.rope + (valid ? pos : 0) * D + 2 * half * DQ;
#pragma unroll
            for (int c = 0; c < DQ; ++c) {
                const float other = __shfl_xor(q[c], 2);
                float y1, y2;
                if (upper) rope_rot(other, q[c], cs[2 * c], cs[2 * c + 1], y1, y2);
                else rope_rot(q[c], other, cs[2 * c], cs[2 * c + 1], y1, y2);
                if (valid) q[c] = upper ? y2 : y1;
            }
        }
    }
    float m_run = -INFINITY, l_run = 0.f;
    const float scale = p.scale;

    const float *kc = (const float *)p.kc + (int64_t)g * p.cap * D;
    const float *vc = (const float *)p.vc + (int64_t)g * p.cap * D;
    const int64_t nstride = p.new_tok_stride;
    const float *kn = (const float *)p.kn + (int64_t)tok0 * nstride + p.new_head_stride * g;
    const float *vn = (const float *)p.vn + (int64_t)tok0 * nstride + p.new_head_stride * g;

    for (int64_t k0 = 0; k0 < ke; k0 += KT) {
        // stage KT key rows: float4 chunks, D/4 per row
        for (int idx = tid; idx < KT * (D / 4); idx += THREADS) {
            const int kr = idx / (D / 4);
            const int c4 = idx % (D / 4);
            const int64_t key = k0 + kr;
            float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
            if (key < ke) {
                const float *ksrc = key < npre ? kc + key * D : kn + (key - npre) * nstride;
                const float *vsrc = key < npre ? vc + key * D : vn + (key - npre) * nstride;
                kv = *(const float4 *)(ksrc + 4 * c4);
                vv = *(const float4 *)(vsrc + 4 * c4);
            }
            *(float4 *)&ks[kr][4 * c4] = kv;
            *(float4 *)&vs[kr][4 * c4] = vv;
        }
        __syncthreads();

        float s[KT];
        float mx = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < KT; ++kk) {
            float acc = 0.f;
#pragma unroll
            for (int c = 0; c < DQ; ++c) acc = __builtin_fmaf(q[c], ks[kk][part * DQ + c], acc);
            // the four lanes of a row hold the four quarter sums; all end with the same total
            acc += __shfl_xor(acc, 1);
            acc += __shfl_xor(acc, 2);
            const int64_t key = k0 + kk;
            s[kk] = key <= pos ? acc * scale : -INFINITY;
            mx = fmaxf(mx, s[kk]);
        }
        const float m_new = fmaxf(m_run, mx);
        if (m_new != -INFINITY) {
            const float alpha = expf(m_run - m_new);   // 0 on the first visible tile
            l_run *= alpha;
#pragma unroll
            for (int c = 0; c < DQ; ++c) o[c] *= alpha;
#pragma unroll
            for (int kk = 0; kk < KT; ++kk) {
                const float w = expf(s[kk] - m_new);
                l_run += w;
#pragma unroll
                for (int c = 0; c < DQ; ++c) o[c] = __builtin_fmaf(w, vs[kk][part * DQ + c], o[c]);
            }
            m_run = m_new;
        }
        __syncthreads();
    }

    if (!valid) return;
    const float inv = 1.f / l_run;
    float *orow = (float *)p.out + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D + part * DQ;
#pragma unroll
    for (int c = 0; c < DQ; c += 4)
        *(float4 *)(orow + c) = make_float4(o[c] * inv, o[c + 1] * inv, o[c + 2] * inv, o[c + 3] * inv);
}

}  // namespace

hipError_t launch_attn_f32(const AttnParams &p, int head_dim, int grid, hipStream_t s) {
    if (head_dim == 128)
        hipLaunchKernelGGL(attn_f32_kernel<128>, dim3(grid), dim3(THREADS), 0, s, p);
    else
        hipLaunchKernelGGL(attn_f32_kernel<64>, dim3(grid), dim3(THREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace kvr
