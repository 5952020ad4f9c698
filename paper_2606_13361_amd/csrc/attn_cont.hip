// attn_cont.hip -- continuation over a long cached prefix (the HBM-bound
// mode), bf16, head_dim 128, for up to 96 query rows per kv head (G*S <= 96:
// decode steps and short continuations).
//
// Split-K inside the workgroup: each of the 4 waves owns ALL query rows of
// the workgroup (1..3 MFMA column tiles of 32) and a quarter of the keys --
// 32-key stages w, w+4, w+8, ... of the workgroup's key range.  A wave
// streams its stages through its own 2-slot LDS ring with direct-to-LDS loads
// (global_load_lds_dwordx4) and waits only on its own loads, so there is no
// workgroup barrier in the key loop.  Within a stage every K fragment and
// every V^T fragment read from LDS feeds all column tiles (1..3 independent
// MFMA accumulation chains).  At the end the 4 waves' (m, l, O) are merged in
// LDS (max, rescale, two-round tree add, fixed order) and wave 0 writes the
// workgroup's split partial -- or the output when there is no split.
//
// LDS tile layout as in the streamed kernel: 256-byte rows, 16-byte chunk c of
// row r in slot c ^ swz(r), conflict-free for the K reads and the
// transposing V reads.
#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int D = 128;
constexpr int ROWB = D * 2;                  // 256 bytes per K/V row
constexpr int SKEYS = 32;                    // keys per stage
constexpr int HALF = SKEYS * ROWB;           // 8 KB: K (or V) of one stage
constexpr int STAGE = 2 * HALF;              // 16 KB
constexpr int NSW = 2;                       // ring slots per wave
constexpr int LOADS = STAGE / 1024;          // 16 wave-wide 1 KB loads per stage
constexpr int RING = NSW * STAGE;            // 32 KB per wave
constexpr int RINGS = 4 * RING;              // 128 KB
constexpr int QROWS = 96;                    // query rows held in LDS
constexpr int LDS_BYTES = RINGS + QROWS * ROWB;   // + 24 KB of Q

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }


template <int NCT>
__global__ __launch_bounds__(THREADS) void attn_cont_kernel(const AttnParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int lane = tid & 63;
    const int j = lane & 31;
    const int grp = lane >> 5;

    const int g = blockIdx.x % p.n_kv_heads;
    const int split = blockIdx.x / p.n_kv_heads;
    const int G = p.group;
    const int S = p.seg_tok0[1];
    const int R = G * S;                            // <= 32 * NCT
    const int64_t npre = p.n_prefix;
    const int64_t k_all = npre + S;
    int64_t kb = 0, ke = k_all;
    if (p.nsplit > 1) {
        kb = (int64_t)split * p.chunk;
        ke = (split == p.nsplit - 1) ? k_all : min(kb + p.chunk, npre);
    }

    // ---- rows: column tile c, lane column j -> row 32*c + j
    int64_t pos[NCT];
    bool valid[NCT];
    int tok[NCT], head[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
        const int r = 32 * c + j;
        valid[c] = r < R;
        tok[c] = valid[c] ? r / G : 0;
        head[c] = g * G + (valid[c] ? r % G : 0);
        pos[c] = valid[c] ? npre + tok[c] : -1;
    }
    // Q rows of all column tiles into LDS once (swizzled like K; rows past R are zero),
    // shared by the 4 waves; Q^T fragments are read from there for every stage
    unsigned char *qlds = smem + RINGS;
    for (int idx = tid; idx < 32 * NCT * 16; idx += THREADS) {
        const int row = idx >> 4, chunk = idx & 15;
        u32x4 v = {0, 0, 0, 0};
        if (row < R) {
            const __bf16 *qrow =
                (const __bf16 *)p.q + ((int64_t)(row / G) * p.n_q_heads + g * G + row % G) * D;
            v = *(const u32x4 *)(qrow + 8 * chunk);
        }
        *(u32x4 *)(qlds + row * ROWB + 16 * (chunk ^ swz(row))) = v;
    }
    __syncthreads();

    // ---- this wave's stages and its load map (instruction i moves rows 4*i + lane/16)
    const int nst = ke > kb ? (int)((ke - kb + SKEYS - 1) / SKEYS) : 0;
    const int my_n = nst > wave ? (nst - wave + 3) / 4 : 0;
    const int64_t nstride_b = (int64_t)p.n_kv_heads * ROWB;
    const unsigned char *kc0 = (const unsigned char *)p.kc + (int64_t)g * p.cap * ROWB;
    const unsigned char *vc0 = (const unsigned char *)p.vc + (int64_t)g * p.cap * ROWB;
    const unsigned char *kn0 = (const unsigned char *)p.kn + (int64_t)g * ROWB;
    const unsigned char *vn0 = (const unsigned char *)p.vn + (int64_t)g * ROWB;
    uint32_t lchunk[8], off_c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int row = 4 * i + (lane >> 4);
        lchunk[i] = 16u * (uint32_t)((lane & 15) ^ swz(row));
        off_c[i] = (uint32_t)row * ROWB + lchunk[i];
    }
    const int64_t cache_end = ke < npre ? ke : npre;
    // addresses as integers: no pointer selects, nothing left in private memory
    const uint64_t kc_a = (uint64_t)(uintptr_t)kc0, vc_a = (uint64_t)(uintptr_t)vc0;
    const uint64_t kn_a = (uint64_t)(uintptr_t)kn0, vn_a = (uint64_t)(uintptr_t)vn0;
    const uint32_t ring_lds = (uint32_t)(wave * RING);
    auto load_stage = [=](int t) {
        const int64_t key0 = kb + (int64_t)(wave + 4 * t) * SKEYS;
        const unsigned char *kd = smem + ring_lds + (t % NSW) * STAGE;
        const unsigned char *vd = kd + HALF;
        if (key0 + SKEYS <= cache_end) {
            const uint64_t kb_ = kc_a + (uint64_t)key0 * ROWB, vb_ = vc_a + (uint64_t)key0 * ROWB;
#pragma unroll
            for (int i = 0; i < 8; ++i) dma16((const void *)(kb_ + off_c[i]), kd + 1024 * i);
#pragma unroll
            for (int i = 0; i < 8; ++i) dma16((const void *)(vb_ + off_c[i]), vd + 1024 * i);
        } else {
            // prefix/new boundary, new rows or a ragged end: per-row source;
            // rows past ke clamp to a valid row (beyond every causal bound, masked)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int64_t key = key0 + 4 * i + (lane >> 4);
                const int64_t kk = key < ke ? key : ke - 1;
                const bool in_cache = kk < npre;
                const uint64_t off = in_cache ? (uint64_t)kk * ROWB : (uint64_t)(kk - npre) * (uint64_t)nstride_b;
                const uint64_t kbase = in_cache ? kc_a : kn_a;
                const uint64_t vbase = in_cache ? vc_a : vn_a;
                dma16((const void *)(kbase + off + lchunk[i]), kd + 1024 * i);
                dma16((const void *)(vbase + off + lchunk[i]), vd + 1024 * i);
            }
        }
    };

    // ---- read maps (per lane, loop invariant); see the streamed kernel
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

    RowState<D> rs[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) rs[c].zero();
    const float c2 = p.scale_log2;

    if (my_n > 0) load_stage(0);
    for (int t = 0; t < my_n; ++t) {
        asm volatile("" ::: "memory");
        if (t + 1 < my_n) {
            load_stage(t + 1);          // its slot held stage t-1, consumed last iteration
            wait_vmcnt<LOADS>();        // stage t landed, stage t+1 in flight
        } else {
            wait_vmcnt<0>();
        }
        asm volatile("" ::: "memory");
        const int64_t key0 = kb + (int64_t)(wave + 4 * t) * SKEYS;
        const unsigned char *ks_ = smem + ring_lds + (t % NSW) * STAGE;
        const unsigned char *vs_ = ks_ + HALF;

        // S^T for every column tile: each K fragment feeds NCT chains
        f32x16 s[NCT];
#pragma unroll
        for (int c = 0; c < NCT; ++c)
#pragma unroll
            for (int i = 0; i < 16; ++i) s[c][i] = 0.f;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
            const u32x4 a = *(const u32x4 *)(ks_ + ka[ks]);
#pragma unroll
            for (int c = 0; c < NCT; ++c) {
                // Q row 32*c + j has the same swizzle as row j
                const u32x4 b = *(const u32x4 *)(qlds + 32 * c * ROWB + ka[ks]);
                s[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), s[c], 0, 0, 0);
            }
        }
        u32x4 pf[NCT][2];
#pragma unroll
        for (int c = 0; c < NCT; ++c) {
            // causal mask: only stages reaching past the first continuation row's position
            if (key0 + SKEYS > npre + 1) {
                const int64_t lim64 = pos[c] - key0;
                const int lim = lim64 < -1 ? -1 : (lim64 > SKEYS ? SKEYS : (int)lim64);
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int o = 8 * (i >> 2) + 4 * grp + (i & 3);
                    if (o > lim) s[c][i] = -INFINITY;
                }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[c][i]);
            mx = pair_max(mx) * c2;
            const bool need = mx > rs[c].m + kRescaleSlack;
            if (__ballot(need)) {
                const float m_new = need ? mx : rs[c].m;
                const float alpha = __builtin_amdgcn_exp2f(rs[c].m - m_new);
                rs[c].m = m_new;
                rs[c].l *= alpha;
#pragma unroll
                for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) rs[c].o[mt][i] *= alpha;
            }
            float lsum = 0.f;
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[c][i], c2, -rs[c].m));
                const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[c][i + 1], c2, -rs[c].m));
                const uint32_t pk = pack_bf16x2(p0, p1);
                lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk), kOnes, lsum, false);
                pf[c][i >> 3][(i & 7) >> 1] = pk;
            }
            rs[c].l += lsum;
        }
        // O^T += V^T P^T: each V^T fragment feeds NCT chains
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt) {
                const unsigned char *va0 = vs_ + va[0][mt] + 16 * kk * ROWB;
                const unsigned char *va1 = vs_ + va[1][mt] + 16 * kk * ROWB;
                const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)va0);
                const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)va1);
                const u32x2 lo2 = __builtin_bit_cast(u32x2, lo);
                const u32x2 hi2 = __builtin_bit_cast(u32x2, hi);
                const u32x4 a = {lo2[0], lo2[1], hi2[0], hi2[1]};
#pragma unroll
                for (int c = 0; c < NCT; ++c)
                    rs[c].o[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(pf[c][kk]),
                                                                         rs[c].o[mt], 0, 0, 0);
            }
    }

    // ---- merge the 4 waves (fixed order): M = max_w m_w, scale by 2^(m_w - M), tree-add
    float *obuf = (float *)smem;                                // 2 x [NCT*64 regs][64 lanes]
    float *lbuf = obuf + 2 * NCT * 64 * 64;                     // 2 x [NCT][64]
    float *mbuf = lbuf + 2 * NCT * 64;                          // [4][NCT][32]
    __syncthreads();                                            // every wave is done with its ring
    if (grp == 0) {
#pragma unroll
        for (int c = 0; c < NCT; ++c) mbuf[(wave * NCT + c) * 32 + j] = rs[c].m;
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
        float M = mbuf[(0 * NCT + c) * 32 + j];
#pragma unroll
        for (int w = 1; w < 4; ++w) M = fmaxf(M, mbuf[(w * NCT + c) * 32 + j]);
        const float alpha = __builtin_amdgcn_exp2f(rs[c].m - M);
        rs[c].m = M;
        rs[c].l *= alpha;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int i = 0; i < 16; ++i) rs[c].o[mt][i] *= alpha;
    }
    auto put = [&](int slot) {
#pragma unroll
        for (int c = 0; c < NCT; ++c) {
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    obuf[((slot * NCT + c) * 64 + mt * 16 + i) * 64 + lane] = rs[c].o[mt][i];
            lbuf[(slot * NCT + c) * 64 + lane] = rs[c].l;
        }
    };
    auto add = [&](int slot) {
#pragma unroll
        for (int c = 0; c < NCT; ++c) {
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
                for (int i = 0; i < 16; ++i)
                    rs[c].o[mt][i] += obuf[((slot * NCT + c) * 64 + mt * 16 + i) * 64 + lane];
            rs[c].l += lbuf[(slot * NCT + c) * 64 + lane];
        }
    };
    if (wave >= 2) put(wave - 2);     // round 1: waves 2, 3 -> slots 0, 1
    __syncthreads();
    if (wave < 2) add(wave);          // wave 0 += wave 2, wave 1 += wave 3
    __syncthreads();
    if (wave == 1) put(0);            // round 2: wave 1 -> slot 0
    __syncthreads();
    if (wave != 0) return;
    add(0);                           // wave 0 holds the workgroup's result

    Work w{};
    w.g = g;
    w.split = split;
    w.tok0 = 0;
#pragma unroll
    for (int c = 0; c < NCT; ++c) epilogue<D, kModeContinue>(p, w, rs[c], 32 * c + j, valid[c], tok[c], head[c], grp);
}

}  // namespace

hipError_t launch_attn_cont(const AttnParams &p, int ncol_tiles, int grid, hipStream_t s) {
    switch (ncol_tiles) {
        case 1: hipLaunchKernelGGL(attn_cont_kernel<1>, dim3(grid), dim3(THREADS), 0, s, p); break;
        case 2: hipLaunchKernelGGL(attn_cont_kernel<2>, dim3(grid), dim3(THREADS), 0, s, p); break;
        default: hipLaunchKernelGGL(attn_cont_kernel<3>, dim3(grid), dim3(THREADS), 0, s, p); break;
    }
    return hipGetLastError();
}

}  // namespace kvr
