// attn_bf16.hip -- causal grouped-query attention with a query offset, bf16
// in, fp32 accumulate, for gfx950 (MI355X).  One kernel serves the three
// modes of the library:
//   prefill        keys are the new rows only, row tiles visited longest first;
//   continue       keys are the cached prefix plus the new rows, the prefix is
//                  split across workgroups and merged afterwards (split-K);
//   many readers   one shared prefix, one segment of rows per reader.
//
// Per workgroup: 4 waves x 32 query rows = 128 rows of one kv head; every
// wave reads the same K/V tile from LDS (GQA sharing: the 4 query heads of a
// group read each cached row once per workgroup).
//
// Per 64-key tile and wave, on MFMA v_mfma_f32_32x32x16_bf16:
//   S^T[key][row] = K Q^T      (K rows from LDS, Q^T held in registers)
//   online softmax on S^T: a lane owns one query row (column) and 16 keys of
//   each 32-key sub-tile, so the row max / sum need only one cross-lane step
//   O^T[d][row] += V^T P^T     (V^T from LDS, P^T straight from the S^T
//                               accumulator registers, rounded to bf16)
// Working on the transposed products keeps P in the registers the score
// MFMA left it in: no LDS round trip for P.
#include "kvr_internal.hpp"

namespace kvr {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int BN = kKeyTile;     // keys per tile
constexpr int ROWS = kRowsBf16;  // rows per workgroup
constexpr int THREADS = 256;

template <int D>
struct Tile {
    static constexpr int CH = D / 8;                  // 16-byte chunks per K/V row
    static constexpr int KPT = BN * CH / THREADS;     // keys each thread stages (4 or 2)
    static constexpr int K_PITCH = D * 2 + 16;        // LDS bytes per K row (pad: no bank conflicts)
    static constexpr int V_PITCH = BN * 2 + 8;        // LDS bytes per V^T row (one head-dim index)
    static constexpr int K_BYTES = BN * K_PITCH;
    static constexpr int V_BYTES = D * V_PITCH;
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static constexpr int KSTEPS = D / 16;             // MFMA k-steps over the head dim
    static constexpr int DBLK = D / 32;               // 32-row blocks of O^T
    static_assert(KPT * THREADS == BN * CH, "tile staging must cover the tile");
};

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    // v_cvt_pk_bf16_f32: round to nearest even
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    bf16x2 v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Locate the segment (reader) that owns a linear row-tile index.
__device__ __forceinline__ int find_segment(const AttnParams &p, int tile) {
    int lo = 0, hi = p.n_seg - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (p.seg_tile0[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    return lo;
}

template <int D>
__global__ __launch_bounds__(THREADS) void attn_bf16_kernel(const AttnParams p) {
    using T = Tile<D>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * T::STAGE];

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int j = lane & 31;      // query row (MFMA column) owned by this lane
    const int grp = lane >> 5;    // which half of each key quad-set this lane holds

    // ---- which work item: kv head fastest (consecutive workgroups land on
    // different XCDs, so each XCD keeps one head's K/V in its L2)
    int b = blockIdx.x;
    const int g = b % p.n_kv_heads;
    b /= p.n_kv_heads;
    const int split = b % p.nsplit;
    b /= p.nsplit;
    const int tile_lin = p.reverse ? (p.tiles_total - 1 - b) : b;
    const int seg = find_segment(p, tile_lin);
    const int rt = tile_lin - p.seg_tile0[seg];
    const int tok0 = p.seg_tok0[seg];
    const int n_tok = p.seg_tok0[seg + 1] - tok0;
    const int G = p.group;
    const int R = G * n_tok;                       // rows of this segment for head g
    const int row0 = rt * ROWS;                    // first row of the workgroup
    const int row_last = min(row0 + ROWS, R) - 1;  // last valid row of the workgroup
    const int64_t npre = p.n_prefix;
    const int D_ = D;

    // ---- this lane's query row
    const int r = row0 + wave * 32 + j;
    const bool valid = r < R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int64_t pos = valid ? npre + tok : -1;   // absolute position; -1 sees nothing

    // ---- key range of this workgroup
    const int64_t k_all = npre + row_last / G + 1;   // keys any row of the workgroup may see
    int64_t kb = 0, ke = k_all;
    if (p.nsplit > 1) {
        kb = (int64_t)split * p.chunk;
        ke = (split == p.nsplit - 1) ? k_all : min(kb + p.chunk, npre);
    }
    // rows of this wave see every key below k_full (no mask needed there)
    const int wrow0 = row0 + wave * 32;
    const bool wave_active = wrow0 < R;
    const int64_t k_full = wave_active ? npre + wrow0 / G + 1 : 0;

    // ---- Q^T fragments (MFMA B operand): column j, head-dim slots 16*ks + 8*grp + 0..7
    u32x4 qf[T::KSTEPS];
    {
        const __bf16 *qrow = (const __bf16 *)p.q + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D_;
#pragma unroll
        for (int ks = 0; ks < T::KSTEPS; ++ks) {
            qf[ks] = valid ? *(const u32x4 *)(qrow + 16 * ks + 8 * grp) : (u32x4){0, 0, 0, 0};
        }
    }

    // ---- staging map: thread -> (16-byte chunk c of the head dim, KPT consecutive keys)
    const int sc = tid % T::CH;
    const int skq = tid / T::CH;
    const __bf16 *kc = (const __bf16 *)p.kc + (int64_t)g * p.cap * D_ + 8 * sc;
    const __bf16 *vc = (const __bf16 *)p.vc + (int64_t)g * p.cap * D_ + 8 * sc;
    const int64_t nstride = (int64_t)p.n_kv_heads * D_;
    const __bf16 *kn = (const __bf16 *)p.kn + (int64_t)tok0 * nstride + (int64_t)g * D_ + 8 * sc;
    const __bf16 *vn = (const __bf16 *)p.vn + (int64_t)tok0 * nstride + (int64_t)g * D_ + 8 * sc;

    u32x4 kreg[T::KPT], vreg[T::KPT];
    auto gload = [&](int64_t k0) {
#pragma unroll
        for (int i = 0; i < T::KPT; ++i) {
            const int64_t key = k0 + skq * T::KPT + i;
            if (key < ke) {
                const __bf16 *ks_ = key < npre ? kc + key * D_ : kn + (key - npre) * nstride;
                const __bf16 *vs_ = key < npre ? vc + key * D_ : vn + (key - npre) * nstride;
                kreg[i] = *(const u32x4 *)ks_;
                vreg[i] = *(const u32x4 *)vs_;
            } else {
                kreg[i] = (u32x4){0, 0, 0, 0};
                vreg[i] = (u32x4){0, 0, 0, 0};
            }
        }
    };
    auto swrite = [&](int stage) {
        unsigned char *ks_ = smem + stage * T::STAGE;
        unsigned char *vs_ = ks_ + T::K_BYTES;
#pragma unroll
        for (int i = 0; i < T::KPT; ++i)
            *(u32x4 *)(ks_ + (skq * T::KPT + i) * T::K_PITCH + 16 * sc) = kreg[i];
        // V^T: for each of the 8 head-dim indices of the chunk, KPT consecutive keys
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int d = 8 * sc + e;
            unsigned char *dst = vs_ + d * T::V_PITCH + skq * T::KPT * 2;
            const int w = e >> 1;
            if constexpr (T::KPT == 4) {
                uint32_t a0 = vreg[0][w], a1 = vreg[1][w], a2 = vreg[2][w], a3 = vreg[3][w];
                u32x2 o;
                if (e & 1) {
                    o[0] = (a0 >> 16) | (a1 & 0xffff0000u);
                    o[1] = (a2 >> 16) | (a3 & 0xffff0000u);
                } else {
                    o[0] = (a0 & 0xffffu) | (a1 << 16);
                    o[1] = (a2 & 0xffffu) | (a3 << 16);
                }
                *(u32x2 *)dst = o;
            } else {
                uint32_t a0 = vreg[0][w], a1 = vreg[1][w];
                uint32_t o = (e & 1) ? ((a0 >> 16) | (a1 & 0xffff0000u)) : ((a0 & 0xffffu) | (a1 << 16));
                *(uint32_t *)dst = o;
            }
        }
    };

    // ---- running softmax state of this lane's row (log2 domain, scaled)
    float m_run = -1e30f;
    float l_run = 0.f;
    f32x16 o_acc[T::DBLK];
#pragma unroll
    for (int mt = 0; mt < T::DBLK; ++mt)
        for (int i = 0; i < 16; ++i) o_acc[mt][i] = 0.f;
    const float c2 = p.scale_log2;

    const int ntiles = ke > kb ? (int)((ke - kb + BN - 1) / BN) : 0;
    if (ntiles > 0) {
        gload(kb);
        swrite(0);
    }
    __syncthreads();

    for (int it = 0; it < ntiles; ++it) {
        const int64_t k0 = kb + (int64_t)it * BN;
        const int cur = it & 1;
        const bool more = it + 1 < ntiles;
        if (more) gload(k0 + BN);   // next tile's global loads overlap this tile's math

        if (wave_active) {
            const unsigned char *ks_ = smem + cur * T::STAGE;
            const unsigned char *vs_ = ks_ + T::K_BYTES;

            // S^T for the two 32-key sub-tiles
            f32x16 s[2];
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                for (int i = 0; i < 16; ++i) s[st][i] = 0.f;
#pragma unroll
                for (int ks = 0; ks < T::KSTEPS; ++ks) {
                    u32x4 a = *(const u32x4 *)(ks_ + (32 * st + j) * T::K_PITCH + (16 * ks + 8 * grp) * 2);
                    s[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(qf[ks]), s[st], 0, 0, 0);
                }
            }
            // causal mask: key k0 + 32*st + 8*(i/4) + 4*grp + i%4 is visible iff <= pos
            if (k0 + BN > k_full) {
#pragma unroll
                for (int st = 0; st < 2; ++st)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int64_t key = k0 + 32 * st + 8 * (i >> 2) + 4 * grp + (i & 3);
                        if (key > pos) s[st][i] = -INFINITY;
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[st][i]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx * c2);
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
            m_run = m_new;
            if (__ballot(alpha != 1.f)) {
#pragma unroll
                for (int mt = 0; mt < T::DBLK; ++mt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) o_acc[mt][i] *= alpha;
            }
            float lsum = 0.f;
            u32x4 pf[2][2];   // P^T as bf16, [sub-tile][16-key half]
#pragma unroll
            for (int st = 0; st < 2; ++st) {
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i], c2, -m_new));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i + 1], c2, -m_new));
                    lsum += p0 + p1;
                    pf[st][i >> 3][(i & 7) >> 1] = pack_bf16x2(p0, p1);
                }
            }
            l_run = l_run * alpha + lsum;

            // O^T += V^T P^T; P^T slot e of half kk is key 32*st + 16*kk + 8*(e/4) + 4*grp + e%4
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int kk = 0; kk < 2; ++kk) {
                    const int kbase = 32 * st + 16 * kk + 4 * grp;
#pragma unroll
                    for (int mt = 0; mt < T::DBLK; ++mt) {
                        const unsigned char *vrow = vs_ + (32 * mt + j) * T::V_PITCH;
                        u32x2 lo = *(const u32x2 *)(vrow + kbase * 2);
                        u32x2 hi = *(const u32x2 *)(vrow + (kbase + 8) * 2);
                        u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
                        o_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(pf[st][kk]),
                                                                           o_acc[mt], 0, 0, 0);
                    }
                }
        }
        if (more) swrite(cur ^ 1);
        __syncthreads();
    }

    // ---- epilogue
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!valid) return;
    if (p.nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        __bf16 *orow = (__bf16 *)p.out + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D_;
#pragma unroll
        for (int mt = 0; mt < T::DBLK; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int d = 32 * mt + 8 * q4 + 4 * grp;
                u32x2 v;
                v[0] = pack_bf16x2(o_acc[mt][4 * q4 + 0] * inv, o_acc[mt][4 * q4 + 1] * inv);
                v[1] = pack_bf16x2(o_acc[mt][4 * q4 + 2] * inv, o_acc[mt][4 * q4 + 3] * inv);
                *(u32x2 *)(orow + d) = v;
            }
    } else {
        const int64_t prow = ((int64_t)split * p.n_kv_heads + g) * p.rows_total + r;
        float *po = p.ws + prow * D_;
#pragma unroll
        for (int mt = 0; mt < T::DBLK; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int d = 32 * mt + 8 * q4 + 4 * grp;
                float4 v = make_float4(o_acc[mt][4 * q4], o_acc[mt][4 * q4 + 1], o_acc[mt][4 * q4 + 2],
                                       o_acc[mt][4 * q4 + 3]);
                *(float4 *)(po + d) = v;
            }
        if (grp == 0) {
            float *pml = p.ws + (int64_t)p.nsplit * p.n_kv_heads * p.rows_total * D_ + prow * 2;
            *(float2 *)pml = make_float2(m_run, l_tot);
        }
    }
}

// Combine the per-split partial results of every row (fixed split order, so
// the result is reproducible bit for bit):
//   M = max_s m_s,  w_s = 2^(m_s - M),  out = sum_s w_s O_s / sum_s w_s l_s
template <int D>
__global__ __launch_bounds__(256) void merge_bf16_kernel(const MergeParams p) {
    constexpr int RPB = 256 / D;   // rows per block
    const int r_in = threadIdx.x / D;
    const int d = threadIdx.x % D;
    const int64_t gr = (int64_t)blockIdx.x * RPB + r_in;   // over n_kv_heads * rows
    if (gr >= (int64_t)p.n_kv_heads * p.rows) return;
    const int g = (int)(gr / p.rows);
    const int r = (int)(gr % p.rows);
    const int64_t per_split = (int64_t)p.n_kv_heads * p.rows;
    const float *ml = p.ws + (int64_t)p.nsplit * per_split * D;
    float M = -INFINITY;
    for (int s = 0; s < p.nsplit; ++s) M = fmaxf(M, ml[(s * per_split + gr) * 2]);
    float acc = 0.f, l = 0.f;
    for (int s = 0; s < p.nsplit; ++s) {
        const float w = __builtin_amdgcn_exp2f(ml[(s * per_split + gr) * 2] - M);
        l += w * ml[(s * per_split + gr) * 2 + 1];
        acc += w * p.ws[(s * per_split + gr) * D + d];
    }
    const int tok = r / p.group;
    const int head = g * p.group + r % p.group;
    __bf16 *o = (__bf16 *)p.out + ((int64_t)tok * p.n_q_heads + head) * D + d;
    *o = (__bf16)(l > 0.f ? acc / l : 0.f);
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams &p, int head_dim, int grid, hipStream_t s) {
    if (head_dim == 128)
        hipLaunchKernelGGL(attn_bf16_kernel<128>, dim3(grid), dim3(THREADS), 0, s, p);
    else
        hipLaunchKernelGGL(attn_bf16_kernel<64>, dim3(grid), dim3(THREADS), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_merge_bf16(const MergeParams &p, int head_dim, hipStream_t s) {
    const int64_t rows = (int64_t)p.n_kv_heads * p.rows;
    if (head_dim == 128) {
        const int grid = (int)((rows + 1) / 2);
        hipLaunchKernelGGL(merge_bf16_kernel<128>, dim3(grid), dim3(256), 0, s, p);
    } else {
        const int grid = (int)((rows + 3) / 4);
        hipLaunchKernelGGL(merge_bf16_kernel<64>, dim3(grid), dim3(256), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace kvr
