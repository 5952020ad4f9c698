// attn_rows.hip -- continuation over a long cached prefix (the HBM-bound
// mode), bf16, head_dim 128, for 33..96 query rows per kv head (short
// continuations, G*S <= 96) when each workgroup's key range is short (the
// host routes one-tile decode steps and long ranges to the keys-split kernel).
//
// A workgroup owns one key range [kb, ke) of one kv head; the host splits the
// prefix across workgroups so that about one workgroup runs per CU, and the
// merge kernel combines the splits.  The 32-key stages of the range stream
// through one ring of NS stages shared by the whole workgroup (direct-to-LDS
// loads, each wave moving an eighth of every stage).
//
// Eight waves, two per SIMD.  Wave w holds the query rows of row group w % 4
// (about R/4 rows, one MFMA column tile) and runs the stages of parity w / 4:
// the two waves sharing a SIMD hold the same rows and take alternate stages,
// so one's matrix products overlap the other's softmax.  Each iteration
// covers two stages behind one barrier (after it both are in LDS -- each wave
// first waited for its own loads -- and the two stages of the previous
// iteration are free, so their slots are refilled).  At the end the two waves
// of a row group combine their (m, l, O) through LDS; the suffix's own keys
// (last split) are one more stage, not one more stage per wave.
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
constexpr int SKEYS = 32;                    // keys per stage
constexpr int HALF = SKEYS * ROWB;           // 8 KB: K (or V) of one stage
constexpr int STAGE = 2 * HALF;              // 16 KB
constexpr int NS = 8;                        // ring stages: 128 KB (four iterations)
constexpr int RING = NS * STAGE;
constexpr int QW = 24;                       // query rows per row group (R <= 96)
constexpr int LDS_BYTES = RING + 4 * QW * ROWB;   // + 24 KB of Q
constexpr int SL = 2;                        // 1 KB loads per wave per stage
constexpr int RTHREADS = 512;
static_assert(4 * QW == kContMaxRows, "four row groups hold every row");
// pair exchange after the loop: (O, m, l) of 64 lanes per row group
constexpr int XCH_FLOATS = 16 * 4 + 2;
static_assert(4 * 64 * XCH_FLOATS * 4 <= RING, "exchange buffer exceeds the ring");

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }

// s_waitcnt for "every load of this wave but those of its last k stages has landed"
__device__ __forceinline__ void wait_stages(int k) {
    switch (k) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<SL>(); break;
        case 2: wait_vmcnt<2 * SL>(); break;
        case 3: wait_vmcnt<3 * SL>(); break;
        case 4: wait_vmcnt<4 * SL>(); break;
        case 5: wait_vmcnt<5 * SL>(); break;
        default: wait_vmcnt<6 * SL>(); break;
    }
}
static_assert(NS - 2 <= 6, "wait_stages covers at most six stages in flight");

template <class E>
__global__ __launch_bounds__(RTHREADS) void attn_rows_kernel(const AttnParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int rg = wave & 3;                                     // row group
    const int par = wave >> 2;                                   // stage parity
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

    // ---- rows: row group rg holds rows rw*rg .. rw*rg + rw - 1 (token-major
    // (token, head) pairs of kv head g); MFMA column j is row rw*rg + j
    const int rw = (R + 3) / 4;
    const int r = rw * rg + j;
    const bool valid = j < rw && r < R;
    const float inv_g = __builtin_amdgcn_rcpf((float)G);   // within 1 ulp: enough for div_small

    // ---- load map: wave w moves K rows 4w..4w+3 and V rows 4w..4w+3 of a stage,
    // one instruction each; lane -> row 4w + lane/16, LDS slot lane%16, global
    // chunk slot ^ swz(row)
    const int64_t nstride_b = (int64_t)p.n_kv_heads * ROWB;
    const uint64_t kc_a = (uint64_t)(uintptr_t)p.kc + (uint64_t)g * p.cap * ROWB;
    const uint64_t vc_a = (uint64_t)(uintptr_t)p.vc + (uint64_t)g * p.cap * ROWB;
    const uint64_t kn_a = (uint64_t)(uintptr_t)p.kn + (uint64_t)g * ROWB;
    const uint64_t vn_a = (uint64_t)(uintptr_t)p.vn + (uint64_t)g * ROWB;
    const int lrow = 4 * wave + (lane >> 4);
    const uint32_t lchunk = 16u * (uint32_t)((lane & 15) ^ swz(lrow));
    auto load_stage = [&](int t) {
        const int64_t key0 = kb + (int64_t)t * SKEYS;
        unsigned char *kd = smem + (t % NS) * STAGE + 4 * wave * ROWB;
        unsigned char *vd = kd + HALF;
        if (key0 + SKEYS <= cache_end) {            // every row cached
            const uint32_t off = (uint32_t)lrow * ROWB + lchunk;
            dma16_s(kc_a + (uint64_t)key0 * ROWB, off, kd);
            dma16_s(vc_a + (uint64_t)key0 * ROWB, off, vd);
        } else if (key0 >= npre && key0 + SKEYS <= ke) {   // every row new
            const uint64_t nrow = (uint64_t)(key0 - npre) * nstride_b;
            const uint32_t off = (uint32_t)lrow * (uint32_t)nstride_b + lchunk;
            dma16_s(kn_a + nrow, off, kd);
            dma16_s(vn_a + nrow, off, vd);
        } else {
            // prefix/new boundary or ragged end: per-row source; rows past ke
            // repeat row ke-1 (beyond every row's bound, masked)
            const int64_t key = min(key0 + lrow, ke - 1);
            const bool c = key < npre;
            const uint64_t off = (uint64_t)(c ? key : key - npre) * (c ? (uint64_t)ROWB : (uint64_t)nstride_b);
            const uint64_t sel = 0 - (uint64_t)c;   // base select by mask
            dma16((const void *)(((kc_a & sel) | (kn_a & ~sel)) + off + lchunk), kd);
            dma16((const void *)(((vc_a & sel) | (vn_a & ~sel)) + off + lchunk), vd);
        }
    };

    // ---- prologue: the row groups' query rows into LDS (the stage-parity-0 wave
    // of each group moves them; swizzled like K; rows past R repeat row R-1,
    // never stored), then the first NS-2 stages (three iterations); Q is older
    // than every stage in the loading wave's queue
    const unsigned char *qlds = smem + RING + rg * QW * ROWB;
    if (par == 0) {
        const uint64_t q_a = (uint64_t)(uintptr_t)p.q + (uint64_t)g * G * ROWB;
        const uint64_t qtok_b = (uint64_t)p.n_q_heads * ROWB;
        const int nq = (rw + 3) / 4;                 // <= 6
        for (int i = 0; i < nq; ++i) {
            const int row = 4 * i + (lane >> 4);     // local row
            const int rr = min(rw * rg + row, R - 1);
            const int tk = div_small(rr, inv_g);
            const uint64_t src = q_a + (uint64_t)tk * qtok_b + (uint64_t)(rr - tk * G) * ROWB +
                                 16u * (uint32_t)((lane & 15) ^ swz(row));
            dma16((const void *)src, qlds + 4 * i * ROWB);
        }
    }
    const int pro = min(NS - 2, nst);
    for (int t = 0; t < pro; ++t) load_stage(t);

    // ---- built while the first loads are in flight: the row's token and
    // head, and the read maps
    const int tk = div_small(r, inv_g);
    const int tok = valid ? tk : 0;
    const int head = g * G + (valid ? r - tk * G : 0);
    const int64_t pos = valid ? npre + tok : -1;
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

    wait_stages(max(pro - 2, 0));                    // Q and stages 0, 1 landed
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

    // One 32-key stage for this wave's rows.  Every fragment of the stage is
    // read from LDS first (K for the scores, V^T for the product), so the
    // reads' latency overlaps the score products and the softmax; the scores
    // come from two independent accumulation chains (even / odd head-dim
    // steps).  Softmax as in the two-group kernel: weights against the current
    // reference m first, the row maximum only when some lane's weights sum
    // above 2^kRescaleSlack or above kSignificance of its mass so far (the
    // first stage always, on flat rows the next two or three).
    auto stage_step = [&](const unsigned char *ks_, const unsigned char *vs_, bool mask, int lim) {
        u32x4 kf[D / 16], vf[8];
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) kf[ks] = *(const u32x4 *)(ks_ + ka[ks]);
#pragma unroll
        for (int idx = 0; idx < 8; ++idx) {           // (kk, mt)
            const int kk = idx >> 2, mt = idx & 3;
            const unsigned char *b = vs_ + 16 * kk * ROWB;
            const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(b + va[0][mt]));
            const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(b + va[1][mt]));
            const u32x2 lo2 = __builtin_bit_cast(u32x2, lo);
            const u32x2 hi2 = __builtin_bit_cast(u32x2, hi);
            vf[idx] = (u32x4){lo2[0], lo2[1], hi2[0], hi2[1]};
        }
        f32x16 sa, sb;
#pragma unroll
        for (int i = 0; i < 16; ++i) sa[i] = sb[i] = 0.f;
#pragma unroll
        for (int ks = 0; ks < D / 16; ks += 2) {
            sa = E::mfma(kf[ks], qf[ks], sa);
            sb = E::mfma(kf[ks + 1], qf[ks + 1], sb);
        }
        float sv[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) sv[i] = sa[i] + sb[i];
        if (mask) {
            // key offset 8*(i/4) + 4*grp + i%4 is visible iff <= lim
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (8 * (i >> 2) + 4 * grp + (i & 3) > lim) sv[i] = -INFINITY;
        }
        u32x4 pf[2];
        auto exps = [&]() {
            float ls[2] = {0.f, 0.f};
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i], c2, -rs.m));
                const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i + 1], c2, -rs.m));
                pf[i >> 3][(i & 7) >> 1] = E::pack2(p0, p1);
                ls[(i >> 1) & 1] += p0 + p1;
            }
            return ls[0] + ls[1];
        };
        float part = exps();
        if (__ballot(!(part <= kSlackSum) || part > kSignificance * (rs.l + part))) {
            float mx = sv[0];
#pragma unroll
            for (int i = 1; i < 16; ++i) mx = fmaxf(mx, sv[i]);
            mx = pair_max(mx) * c2;
            const float pmax = __builtin_amdgcn_exp2f(mx - rs.m);
            const bool sig = mx > rs.m && pmax > kSignificance * pair_sum(rs.l + part);
            const bool need = mx > rs.m + (sig ? 0.f : kRescaleSlack);
            if (__ballot(need)) {
                move_reference(rs, need ? mx : rs.m);
                part = exps();
            }
        }
        rs.l += part;
#pragma unroll
        for (int idx = 0; idx < 8; ++idx) {
            const int kk = idx >> 2, mt = idx & 3;
            rs.o[mt] = E::mfma(vf[idx], pf[kk], rs.o[mt]);
        }
    };

    const int nit = (nst + 1) / 2;
    for (int u = 0; u < nit; ++u) {
        const int t0 = 2 * u;                        // this iteration's stages: t0, t0 + 1
        if (u > 0) {
            // loads issued so far: stages up to min(t0 + 5, nst - 1); stages t0, t0+1 must have landed
            wait_stages(max(min(t0 + NS - 3, nst - 1) - (t0 + 1), 0));
            __builtin_amdgcn_s_barrier();            // everyone's; the previous iteration's stages are free
            asm volatile("" ::: "memory");
        }
        // refill the previous iteration's slots with stages t0 + 6, t0 + 7
        if (t0 + NS - 2 < nst) load_stage(t0 + NS - 2);
        if (t0 + NS - 1 < nst) load_stage(t0 + NS - 1);
        const int t = t0 + par;
        if (t < nst) {
            const int64_t key0 = kb + (int64_t)t * SKEYS;
            const unsigned char *ks_ = smem + (t % NS) * STAGE;
            const unsigned char *vs_ = ks_ + HALF;
            // keys past a row's position (the suffix's own keys) or past ke (ragged end)
            const bool mask = key0 + SKEYS > cache_end;
            const int64_t vis = min(pos, ke - 1) - key0;
            const int lim = (int)max((int64_t)-1, min(vis, (int64_t)SKEYS));
            stage_step(ks_, vs_, mask, lim);
        }
    }

    // ---- the two waves of a row group combine (m, l, O): parity 1 posts its
    // state, parity 0 scales both to the larger m and adds (in that order)
    wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();                    // the ring is no longer read
    asm volatile("" ::: "memory");
    float4 *xo = (float4 *)smem + rg * 16 * 64;                  // [16][64 lanes] float4
    float *xml = (float *)smem + 4 * 16 * 64 * 4 + rg * 2 * 64;  // m then l, [64 lanes] each
    if (par == 1) {
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                xo[(4 * mt + q4) * 64 + lane] = make_float4(rs.o[mt][4 * q4], rs.o[mt][4 * q4 + 1],
                                                            rs.o[mt][4 * q4 + 2], rs.o[mt][4 * q4 + 3]);
        xml[lane] = rs.m;
        xml[64 + lane] = rs.l;
    }
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (par == 1) {
        // the waves of parity 1 are done: they store the cache update, if any
        if (p.kc_app && split == p.nsplit - 1) append_new_rows<ROWB>(p, g, S, tid - 256, 256);
        return;
    }
    {
        const float m1 = xml[lane], l1 = xml[64 + lane];
        const float M = fmaxf(rs.m, m1);
        const float a0 = __builtin_amdgcn_exp2f(rs.m - M), a1 = __builtin_amdgcn_exp2f(m1 - M);
        rs.m = M;
        rs.l = a0 * rs.l + a1 * l1;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const float4 v = xo[(4 * mt + q4) * 64 + lane];
                rs.o[mt][4 * q4] = a0 * rs.o[mt][4 * q4] + a1 * v.x;
                rs.o[mt][4 * q4 + 1] = a0 * rs.o[mt][4 * q4 + 1] + a1 * v.y;
                rs.o[mt][4 * q4 + 2] = a0 * rs.o[mt][4 * q4 + 2] + a1 * v.z;
                rs.o[mt][4 * q4 + 3] = a0 * rs.o[mt][4 * q4 + 3] + a1 * v.w;
            }
    }

    // ---- the row group's rows: final bf16 rows, or the split partial
    const float l_tot = pair_sum(rs.l);
    if (!valid) return;
    if (p.nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        uint16_t *orow = (uint16_t *)p.out + ((int64_t)tok * p.n_q_heads + head) * D;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                u32x2 v;
                v[0] = E::pack2(rs.o[mt][4 * q4] * inv, rs.o[mt][4 * q4 + 1] * inv);
                v[1] = E::pack2(rs.o[mt][4 * q4 + 2] * inv, rs.o[mt][4 * q4 + 3] * inv);
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

hipError_t launch_attn_rows(const AttnParams &p, bool f16, int grid, hipStream_t s) {
    if (f16) hipLaunchKernelGGL(attn_rows_kernel<F16>, dim3(grid), dim3(RTHREADS), 0, s, p);
    else hipLaunchKernelGGL(attn_rows_kernel<Bf16>, dim3(grid), dim3(RTHREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace kvr
