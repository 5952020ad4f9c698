// attn_rows.hip -- continuation over a long cached prefix (the HBM-bound
// mode), bf16, head_dim 128, for up to 96 query rows per kv head (G*S <= 96:
// decode steps and short continuations).
//
// A workgroup (4 waves, one per SIMD) owns one key range [kb, ke) of one kv
// head; the host splits the prefix across workgroups so that about one
// workgroup runs per CU, and the merge kernel combines the splits.  Inside the
// workgroup the waves split the QUERY ROWS (about R/4 each, one MFMA column
// tile), not the keys: the 64-key stages of the range stream through one ring
// of NS stages shared by the four waves (direct-to-LDS loads, each wave moving
// a quarter of every stage), and every wave runs every stage for its own rows
// (two 32-key sub-tiles: two independent score chains per stage).
// So nothing is merged inside the workgroup (each wave stores its rows' split
// partial, or its final rows), and the suffix's own keys (the last split) are
// one more stage for the whole workgroup rather than one more stage for one
// wave.  One barrier per stage: after it, stage t is in LDS (each wave first
// waited for its own loads) and stage t-1 is no longer read, so its slot is
// refilled with stage t+NS-1.
//
// LDS layout as in the other members: 256-byte K/V rows with the 16-byte
// chunk c of row r in slot c ^ swz(r) (conflict-free K reads and transposing
// V reads); the query rows the same way, read once into registers.
#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int D = 128;
constexpr int ROWB = D * 2;                  // 256 bytes per K/V row
constexpr int SKEYS = 64;                    // keys per stage
constexpr int HALF = SKEYS * ROWB;           // 16 KB: K (or V) of one stage
constexpr int STAGE = 2 * HALF;              // 32 KB
constexpr int NS = 4;                        // ring stages: 128 KB
constexpr int RING = NS * STAGE;
constexpr int QW = 24;                       // query rows per wave (R <= 96)
constexpr int LDS_BYTES = RING + 4 * QW * ROWB;   // + 24 KB of Q
constexpr int SL = 8;                        // 1 KB loads per wave per stage
constexpr int RTHREADS = 256;
static_assert(4 * QW == kContMaxRows, "four waves hold every row");

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }

// s_waitcnt for "every load of this wave but those of its last k stages has landed"
__device__ __forceinline__ void wait_stages(int k) {
    switch (k) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<SL>(); break;
        default: wait_vmcnt<2 * SL>(); break;
    }
}
static_assert(NS - 2 <= 2, "wait_stages covers at most two stages in flight");

__global__ __launch_bounds__(RTHREADS) void attn_rows_kernel(const AttnParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int lane = tid & 63;
    const int j = lane & 31;
    const int grp = lane >> 5;

    // ---- key range: split-K across workgroups, kv head fastest (XCD locality)
    const int g = blockIdx.x % p.n_kv_heads;
    const int split = blockIdx.x / p.n_kv_heads;
    const int G = p.group;
    const int S = p.seg_tok0[1];
    const int R = G * S;                            // <= 96
    const int64_t npre = p.n_prefix;
    const int64_t k_all = npre + S;
    int64_t kb = 0, ke = k_all;
    if (p.nsplit > 1) {
        kb = (int64_t)split * p.chunk;
        ke = split == p.nsplit - 1 ? k_all : min(kb + p.chunk, npre);
    }
    const int nst = (int)((ke - kb + SKEYS - 1) / SKEYS);   // >= 1
    const int64_t cache_end = ke < npre ? ke : npre;

    // ---- rows: wave w holds rows rw*w .. rw*w + rw - 1 (token-major (token, head)
    // pairs of kv head g); MFMA column j is row rw*w + j
    const int rw = (R + 3) / 4;
    const int r = rw * wave + j;
    const bool valid = j < rw && r < R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int64_t pos = valid ? npre + tok : -1;

    // ---- load map: wave w moves K rows 16w..16w+15 and V rows 16w..16w+15 of a
    // stage, 4 rows per instruction; lane -> row 16w + 4i + lane/16, LDS slot
    // lane%16, global chunk slot ^ swz(row)
    const int64_t nstride_b = (int64_t)p.n_kv_heads * ROWB;
    const uint64_t kc_a = (uint64_t)(uintptr_t)p.kc + (uint64_t)g * p.cap * ROWB;
    const uint64_t vc_a = (uint64_t)(uintptr_t)p.vc + (uint64_t)g * p.cap * ROWB;
    const uint64_t kn_a = (uint64_t)(uintptr_t)p.kn + (uint64_t)g * ROWB;
    const uint64_t vn_a = (uint64_t)(uintptr_t)p.vn + (uint64_t)g * ROWB;
    int lrow[4];
    uint32_t lchunk[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        lrow[i] = 16 * wave + 4 * i + (lane >> 4);
        lchunk[i] = 16u * (uint32_t)((lane & 15) ^ swz(lrow[i]));
    }
    auto load_stage = [&](int t) {
        const int64_t key0 = kb + (int64_t)t * SKEYS;
        unsigned char *kd = smem + (t % NS) * STAGE + 16 * wave * ROWB;
        unsigned char *vd = kd + HALF;
        if (key0 + SKEYS <= cache_end) {            // every row cached
            const uint64_t kb_ = kc_a + (uint64_t)key0 * ROWB, vb_ = vc_a + (uint64_t)key0 * ROWB;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t off = (uint32_t)lrow[i] * ROWB + lchunk[i];
                dma16_s(kb_, off, kd + 1024 * i);
                dma16_s(vb_, off, vd + 1024 * i);
            }
        } else if (key0 >= npre && key0 + SKEYS <= ke) {   // every row new
            const uint64_t nrow = (uint64_t)(key0 - npre) * nstride_b;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t off = (uint32_t)lrow[i] * (uint32_t)nstride_b + lchunk[i];
                dma16_s(kn_a + nrow, off, kd + 1024 * i);
                dma16_s(vn_a + nrow, off, vd + 1024 * i);
            }
        } else {
            // prefix/new boundary or ragged end: per-row source; rows past ke
            // repeat row ke-1 (beyond every row's bound, masked)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t key = min(key0 + lrow[i], ke - 1);
                const bool c = key < npre;
                const uint64_t off = (uint64_t)(c ? key : key - npre) * (c ? (uint64_t)ROWB : (uint64_t)nstride_b);
                const uint64_t sel = 0 - (uint64_t)c;   // base select by mask
                dma16((const void *)(((kc_a & sel) | (kn_a & ~sel)) + off + lchunk[i]), kd + 1024 * i);
                dma16((const void *)(((vc_a & sel) | (vn_a & ~sel)) + off + lchunk[i]), vd + 1024 * i);
            }
        }
    };

    // ---- read maps (per lane, loop invariant), as in the other members
    uint32_t ka[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) ka[ks] = (uint32_t)j * ROWB + 16u * (uint32_t)((2 * ks + grp) ^ swz(j));
    const int l16 = lane & 15;
    const int g16 = lane >> 4;
    uint32_t va[2][D / 32];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt) {
            const int row = 8 * h + 4 * (g16 >> 1) + (l16 >> 2);
            const int chunk = (32 * mt + 16 * (g16 & 1) + 4 * (l16 & 3)) / 8;
            va[h][mt] = (uint32_t)row * ROWB + 16u * (uint32_t)(chunk ^ swz(row)) + 8u * (uint32_t)(l16 & 1);
        }

    // ---- prologue: this wave's query rows into LDS (swizzled like K; rows past
    // R repeat row R-1, never stored), then the first NS-1 stages; Q is older
    // than every stage in the wave's load queue
    unsigned char *qlds = smem + RING + wave * QW * ROWB;
    {
        const uint64_t q_a = (uint64_t)(uintptr_t)p.q + (uint64_t)g * G * ROWB;
        const uint64_t qtok_b = (uint64_t)p.n_q_heads * ROWB;
        const int nq = (rw + 3) / 4;                 // <= 6
        for (int i = 0; i < nq; ++i) {
            const int row = 4 * i + (lane >> 4);     // local row
            const int rr = min(rw * wave + row, R - 1);
            const uint64_t src = q_a + (uint64_t)(rr / G) * qtok_b + (uint64_t)(rr % G) * ROWB +
                                 16u * (uint32_t)((lane & 15) ^ swz(row));
            dma16((const void *)src, qlds + 4 * i * ROWB);
        }
    }
    const int pro = min(NS - 1, nst);
    for (int t = 0; t < pro; ++t) load_stage(t);
    wait_stages(pro - 1);                            // Q and stage 0 landed
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    u32x4 qf[D / 16];
    {
        const int row = min(j, QW - 1);
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
            const u32x4 v = *(const u32x4 *)(qlds + row * ROWB + 16 * ((2 * ks + grp) ^ swz(row)));
            qf[ks] = valid ? v : (u32x4){0, 0, 0, 0};
        }
    }

    RowState<D> rs;
    rs.zero();
    const float c2 = p.scale_log2;
    for (int t = 0; t < nst; ++t) {
        if (t > 0) {
            wait_stages(min(t + NS - 2, nst - 1) - t);   // this wave's loads of stage t landed
            __builtin_amdgcn_s_barrier();                // everyone's; stage t-1 is free
            asm volatile("" ::: "memory");
        }
        if (t + NS - 1 < nst) load_stage(t + NS - 1);   // into stage t-1's slot
        const int64_t key0 = kb + (int64_t)t * SKEYS;
        const unsigned char *ks_ = smem + (t % NS) * STAGE;
        const unsigned char *vs_ = ks_ + HALF;
        // keys past a row's position (the suffix's own keys) or past ke (ragged end)
        const bool mask = key0 + SKEYS > cache_end;
        const int64_t vis = min(pos, ke - 1) - key0;
        const int lim = (int)max((int64_t)-1, min(vis, (int64_t)SKEYS));
        tile_step<D, 2>(
            rs, qf, [&](int st, int ks) { return ks_ + ka[ks] + 32 * st * ROWB; },
            [&](int st, int kk, int h, int mt) { return vs_ + (32 * st + 16 * kk) * ROWB + va[h][mt]; }, mask, lim,
            c2, grp);
    }

    // ---- this wave's rows: final bf16 rows, or the split partial
    const float l_tot = pair_sum(rs.l);
    if (!valid) return;
    if (p.nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        __bf16 *orow = (__bf16 *)p.out + ((int64_t)tok * p.n_q_heads + head) * D;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                u32x2 v;
                v[0] = pack_bf16x2(rs.o[mt][4 * q4] * inv, rs.o[mt][4 * q4 + 1] * inv);
                v[1] = pack_bf16x2(rs.o[mt][4 * q4 + 2] * inv, rs.o[mt][4 * q4 + 3] * inv);
                *(u32x2 *)(orow + 32 * mt + 8 * q4 + 4 * grp) = v;
            }
    } else {
        const int64_t prow = ((int64_t)split * p.n_kv_heads + g) * p.rows_total + r;
        float *po = p.ws + prow * D;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                *(float4 *)(po + 32 * mt + 8 * q4 + 4 * grp) =
                    make_float4(rs.o[mt][4 * q4], rs.o[mt][4 * q4 + 1], rs.o[mt][4 * q4 + 2], rs.o[mt][4 * q4 + 3]);
        if (grp == 0) {
            float *pml = p.ws + (int64_t)p.nsplit * p.n_kv_heads * p.rows_total * D + prow * 2;
            *(float2 *)pml = make_float2(rs.m, l_tot);
        }
    }
}

}  // namespace

hipError_t launch_attn_rows(const AttnParams &p, int grid, hipStream_t s) {
    hipLaunchKernelGGL(attn_rows_kernel, dim3(grid), dim3(RTHREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace kvr
