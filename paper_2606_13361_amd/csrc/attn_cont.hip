// attn_cont.hip -- continuation over a long cached prefix (the HBM-bound
// mode), bf16, head_dim 128, for up to 96 query rows per kv head (G*S <= 96:
// decode steps and short continuations; the row-split kernel takes 33..96
// rows over short key ranges per workgroup), and over the int8 artifact.
//
// Split-K inside the workgroup: each of the 4 waves owns ALL query rows of
// the workgroup (1..3 MFMA column tiles of 32) and a quarter of the keys --
// 32-key stages w, w+4, w+8, ... of the workgroup's key range.  A wave
// streams its stages through its own 2-slot LDS ring with direct-to-LDS loads
// (global_load_lds_dwordx4) and waits only on its own loads, so there is no
// workgroup barrier in the key loop.  Within a stage every K fragment and
// every V^T fragment read from LDS feeds all column tiles (1..3 independent
// MFMA accumulation chains).  The query rows reach LDS by the same direct
// loads, issued together with each wave's first K/V stage.
//
// Merge with a single barrier: every wave posts its (m, l) and the three
// head-dim quarters of O it does not own; wave w then owns quarter w, sums the
// four contributions scaled to the common maximum in a fixed order, and
// stores that quarter of the workgroup's split partial -- or of the output
// when there is no split.
//
// LDS tile layout as in the two-group kernel: 256-byte rows, 16-byte chunk c of
// row r in slot c ^ swz(r), conflict-free for the K reads and the
// transposing V reads.
#include <type_traits>

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

// merge buffers, reusing the rings and Q: O quarters [4 owners][3 sources][NCT][4][64 lanes]
// as float4, then m and l [4 waves][NCT][64 lanes]
template <int NCT> constexpr int obuf_bytes() { return 12 * NCT * 4 * 64 * 16; }
template <int NCT> constexpr int merge_bytes() { return obuf_bytes<NCT>() + 2 * 4 * NCT * 64 * 4; }
static_assert(merge_bytes<3>() <= LDS_BYTES, "merge buffers exceed the LDS allocation");

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }


// Head-dim quarter MT of every column tile: the four waves' contributions,
// each scaled by 2^(m_w - M) with M the largest m_w, summed in wave order
// 0..3 (the owner's own quarter comes from its registers, the others from
// LDS), then stored -- bf16 output rows when there is no split, else the
// split partial O quarter and, from the owner of quarter 0, (M, l).
template <class E, int NCT, int MT>
__device__ __forceinline__ void finish_quarter(const AttnParams &p, const RowState<D> (&rs)[NCT],
                                               const float4 *obuf, const float *lbuf, const float *mbuf,
                                               const bool (&valid)[NCT], const int (&tok)[NCT],
                                               const int (&head)[NCT], int g, int split, int lane) {
    const int j = lane & 31;
    const int grp = lane >> 5;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
        float mw[4], alpha[4];
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            mw[w] = mbuf[(w * NCT + c) * 64 + lane];
            M = fmaxf(M, mw[w]);
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) alpha[w] = __builtin_amdgcn_exp2f(mw[w] - M);
        float l = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) l = __builtin_fmaf(alpha[w], lbuf[(w * NCT + c) * 64 + lane], l);
        const float l_tot = pair_sum(l);
        float acc[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[i] = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            float x[16];
            if (w == MT) {
#pragma unroll
                for (int i = 0; i < 16; ++i) x[i] = rs[c].o[MT][i];
            } else {
                const int slot = 3 * MT + (w > MT ? w - 1 : w);
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const float4 v = obuf[((slot * NCT + c) * 4 + q4) * 64 + lane];
                    x[4 * q4] = v.x;
                    x[4 * q4 + 1] = v.y;
                    x[4 * q4 + 2] = v.z;
                    x[4 * q4 + 3] = v.w;
                }
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i] = __builtin_fmaf(alpha[w], x[i], acc[i]);
        }
        if (!valid[c]) continue;
        const int r = 32 * c + j;
        if (p.nsplit == 1) {
            const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
            uint16_t *orow = (uint16_t *)p.out + ((int64_t)tok[c] * p.n_q_heads + head[c]) * D;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                u32x2 v;
                v[0] = E::pack2(acc[4 * q4] * inv, acc[4 * q4 + 1] * inv);
                v[1] = E::pack2(acc[4 * q4 + 2] * inv, acc[4 * q4 + 3] * inv);
                *(u32x2 *)(orow + 32 * MT + 8 * q4 + 4 * grp) = v;
            }
        } else {
            const int64_t prow = ((int64_t)split * p.n_kv_heads + g) * p.rows_total + r;
            float *po = p.ws + prow * D;
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                *(float4 *)(po + 32 * MT + 8 * q4 + 4 * grp) =
                    make_float4(acc[4 * q4], acc[4 * q4 + 1], acc[4 * q4 + 2], acc[4 * q4 + 3]);
            if (MT == 0 && grp == 0) {
                float *pml = p.ws + (int64_t)p.nsplit * p.n_kv_heads * p.rows_total * D + prow * 2;
                *(float2 *)pml = make_float2(M, l_tot);
            }
        }
    }
}

// int8 artifact stages: 32 keys of K codes (32 rows x 128 B) at the slot
// start, the 32-key block of V codes (128 head-dim rows x 32 B) at +HALF.
// 16-byte chunk c of K row r sits in slot c ^ swzk(r), chunk h of V row d in
// slot h ^ swzv(d): the 16-lane groups of the fragment reads below then touch
// 16 distinct bank groups.
__device__ __forceinline__ int swzk(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int swzv(int d) { return (d >> 3) & 1; }
constexpr int LOADS_Q8 = 8;                  // direct loads per int8 stage (4 K + 4 V)

// 16 int8 codes -> two MFMA operands of 8 bf16 each (exact: |code| <= 127)
__device__ __forceinline__ void codes_to_bf16(const u32x4 w, u32x4 &lo, u32x4 &hi) {
    uint32_t o[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int32_t x = (int32_t)w[q];
        const float f0 = (float)((x << 24) >> 24), f1 = (float)((x << 16) >> 24);
        const float f2 = (float)((x << 8) >> 24), f3 = (float)(x >> 24);
        o[2 * q] = pack_bf16x2(f0, f1);
        o[2 * q + 1] = pack_bf16x2(f2, f3);
    }
    lo = (u32x4){o[0], o[1], o[2], o[3]};
    hi = (u32x4){o[4], o[5], o[6], o[7]};
}

// Q8 = false: cache and new rows are bf16.  Q8 = true: the cached rows come
// from the int8 artifact (kq/vq codes, scales s_K, s_V): scores of cached keys
// are scaled by s_K inside the softmax exponent, the cached part of O by s_V
// before the first new key (or at the end); the new rows stay bf16.  Cached
// and new keys then never share a stage.
template <int NCT, bool Q8, class E>
__global__ __launch_bounds__(THREADS) void attn_cont_kernel(const AttnParams p) {
    static_assert(!Q8 || std::is_same<E, Bf16>::value, "the int8 artifact is a bf16 model's");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[LDS_BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int lane = tid & 63;
    const int j = lane & 31;
    const int grp = lane >> 5;

    const int g = blockIdx.x % p.n_kv_heads;
    const int split = blockIdx.x / p.n_kv_heads;
    const int G = p.group;
    const float inv_g = __builtin_amdgcn_rcpf((float)G);   // within 1 ulp: enough for div_small
    const int S = p.seg_tok0[1];
    const int R = G * S;                            // <= 32 * NCT
    const int64_t npre = p.n_prefix;
    const int64_t k_all = npre + S;
    const bool last_split = split == p.nsplit - 1;
    int64_t kb = 0, ke = k_all;
    if (p.nsplit > 1) {
        kb = (int64_t)split * p.chunk;
        ke = last_split ? k_all : min(kb + p.chunk, npre);
    }

    // ---- stages.  bf16: 32-key stages over [kb, ke).  Q8: n_cst stages of cached
    // keys [kb, ce) (the last one may reach past npre: masked), then the new rows'
    // stages (last split only).  Wave w takes stages w, w+4, ...
    const int64_t ce = ke < npre ? ke : npre;
    const int n_cst = Q8 ? (ce > kb ? (int)((ce - kb + SKEYS - 1) / SKEYS) : 0) : 0;
    const int nst = Q8 ? n_cst + ((p.nsplit == 1 || last_split) ? (S + SKEYS - 1) / SKEYS : 0)
                       : (ke > kb ? (int)((ke - kb + SKEYS - 1) / SKEYS) : 0);
    // The split holding the new rows has one stage more than the others, and one
    // wave would run it after everyone else's last stage.  When the new rows fit in
    // that last stage, it is loaded in the prologue into wave 3's second slot
    // (first used by wave 3's stage 1) and run before the loop by waves 0 .. NCT-1,
    // one column tile each; the loop then runs the other nst - 1 stages.
    const bool sfx_split = !Q8 && (p.nsplit == 1 || last_split) && nst >= 2 &&
                           kb + (int64_t)SKEYS * (nst - 1) <= npre;
    const int nmain = sfx_split ? nst - 1 : nst;
    const int my_n = nmain > wave ? (nmain - wave + 3) / 4 : 0;
    auto is_q8 = [&](int t) { return Q8 && wave + 4 * t < n_cst; };

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
    // int8 load maps: K instruction i moves rows 8i + lane/8, V instruction i head-dim
    // rows 32i + lane/2
    uint32_t offk[4], offv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = 8 * i + (lane >> 3);
        offk[i] = (uint32_t)row * D + 16u * (uint32_t)((lane & 7) ^ swzk(row));
        const int d = 32 * i + (lane >> 1);
        offv[i] = (uint32_t)d * 32 + 16u * (uint32_t)((lane & 1) ^ swzv(d));
    }
    const int64_t padded = (p.cap + 31) / 32 * 32;
    const uint64_t kq_a = (uint64_t)(uintptr_t)p.kc + (uint64_t)g * padded * D;   // Q8: artifact
    const uint64_t vq_a = (uint64_t)(uintptr_t)p.vc + (uint64_t)g * padded * D;
    const int64_t cache_end = ce;
    // addresses as integers: no pointer selects, nothing left in private memory
    const uint64_t kc_a = (uint64_t)(uintptr_t)kc0, vc_a = (uint64_t)(uintptr_t)vc0;
    const uint64_t kn_a = (uint64_t)(uintptr_t)kn0, vn_a = (uint64_t)(uintptr_t)vn0;
    const uint32_t ring_lds = (uint32_t)(wave * RING);
    auto load_stage_to = [=](int i_st, const unsigned char *kd) {
        const unsigned char *vd = kd + HALF;
        if (Q8 && i_st < n_cst) {
            const int64_t key0 = kb + (int64_t)i_st * SKEYS;                   // a multiple of 32
            const uint64_t kb_ = kq_a + (uint64_t)key0 * D, vb_ = vq_a + (uint64_t)key0 * D;
#pragma unroll
            for (int i = 0; i < 4; ++i) dma16_s(kb_, offk[i], kd + 1024 * i);
#pragma unroll
            for (int i = 0; i < 4; ++i) dma16_s(vb_, offv[i], vd + 1024 * i);
            return;
        }
        // bf16 keys: key0 is absolute (bf16 path) or npre + the new row index (Q8)
        const int64_t key0 = Q8 ? npre + (int64_t)(i_st - n_cst) * SKEYS : kb + (int64_t)i_st * SKEYS;
        if (!Q8 && key0 + SKEYS <= cache_end) {
            const uint64_t kb_ = kc_a + (uint64_t)key0 * ROWB, vb_ = vc_a + (uint64_t)key0 * ROWB;
#pragma unroll
            for (int i = 0; i < 8; ++i) dma16_s(kb_, off_c[i], kd + 1024 * i);
#pragma unroll
            for (int i = 0; i < 8; ++i) dma16_s(vb_, off_c[i], vd + 1024 * i);
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
    auto load_stage = [=](int t) { load_stage_to(wave + 4 * t, smem + ring_lds + (t % NSW) * STAGE); };
    const unsigned char *sfx_lds = smem + 3 * RING + STAGE;   // the split suffix stage: wave 3's slot 1

    // ---- read maps (per lane, loop invariant): K fragments and transposing V reads of the swizzled rows
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
    float c2q = c2, s_v = 1.f;
    if (Q8) {
        c2q = c2 * p.qscale[0];
        s_v = p.qscale[1];
    }

    // Q rows of all column tiles into LDS (swizzled like K, rows past R repeat
    // row R-1: their columns are computed and never stored), then this wave's
    // first stage; Q is older than the stage in the wave's load queue
    const unsigned char *qlds = smem + RINGS;
    {
        const uint64_t q_a = (uint64_t)(uintptr_t)p.q + (uint64_t)g * G * ROWB;
        const uint64_t qtok_b = (uint64_t)p.n_q_heads * ROWB;
#pragma unroll
        for (int i = 0; i < 2 * NCT; ++i) {
            const int base = 4 * (2 * NCT * wave + i);
            const int row = base + (lane >> 4);
            const int rr = row < R ? row : R - 1;
            const int tk = div_small(rr, inv_g);
            const uint64_t src = q_a + (uint64_t)tk * qtok_b + (uint64_t)(rr - tk * G) * ROWB +
                                 16u * (uint32_t)((lane & 15) ^ swz(row));
            dma16((const void *)src, qlds + base * ROWB);
        }
    }
    if (sfx_split && wave == 3) load_stage_to(nst - 1, sfx_lds);
    if (my_n > 0) load_stage(0);

    // ---- rows: column tile c, lane column j -> row 32*c + j (computed while
    // the first loads are in flight)
    int64_t pos[NCT];
    bool valid[NCT];
    int tok[NCT], head[NCT];
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
        const int r = 32 * c + j;
        valid[c] = r < R;
        const int tk = div_small(r, inv_g);
        tok[c] = valid[c] ? tk : 0;
        head[c] = g * G + (valid[c] ? r - tk * G : 0);
        pos[c] = valid[c] ? npre + tok[c] : -1;
    }

    if (my_n > 0) {
        if (is_q8(0)) wait_vmcnt<LOADS_Q8>();
        else wait_vmcnt<LOADS>();
    } else {
        wait_vmcnt<0>();
    }
    __builtin_amdgcn_s_barrier();       // all of Q (and the split suffix stage) is in LDS
    asm volatile("" ::: "memory");

    bool o_scaled = !Q8;                // Q8: cached part of O still in code units of V
    auto scale_o = [&]() {
#pragma unroll
        for (int c = 0; c < NCT; ++c)
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
                for (int i = 0; i < 16; ++i) rs[c].o[mt][i] *= s_v;
        o_scaled = true;
    };

    // one stage; the kind (int8 codes or bf16 rows) is a compile-time tag, so the
    // int8 stages and the bf16 stages run in loops of their own
    // the arithmetic of one stage for the column tiles in CM (a bit mask)
    auto compute = [&](auto kind, auto cm, const unsigned char *ks_, const unsigned char *vs_,
                       int64_t key0) {
        constexpr bool q8 = decltype(kind)::value;
        constexpr int CM = decltype(cm)::value;
        // S^T for every column tile: each K fragment feeds NCT chains
        f32x16 s[NCT];
#pragma unroll
        for (int c = 0; c < NCT; ++c)
#pragma unroll
            for (int i = 0; i < 16; ++i) s[c][i] = 0.f;   // unused tiles: dead code
        if constexpr (q8) {
            // lane (j, grp): codes of row j, head-dim steps 2 pr and 2 pr + 1
#pragma unroll
            for (int pr = 0; pr < 4; ++pr) {
                const u32x4 w = *(const u32x4 *)(ks_ + j * D + 16 * ((4 * grp + pr) ^ swzk(j)));
                u32x4 a0, a1;
                codes_to_bf16(w, a0, a1);
#pragma unroll
                for (int c = 0; c < NCT; ++c) {
                    if (!((CM >> c) & 1)) continue;
                    const u32x4 b0 = *(const u32x4 *)(qlds + 32 * c * ROWB + ka[2 * pr]);
                    const u32x4 b1 = *(const u32x4 *)(qlds + 32 * c * ROWB + ka[2 * pr + 1]);
                    s[c] = E::mfma(a0, b0, s[c]);
                    s[c] = E::mfma(a1, b1, s[c]);
                }
            }
        } else {
#pragma unroll
            for (int ks = 0; ks < D / 16; ++ks) {
                const u32x4 a = *(const u32x4 *)(ks_ + ka[ks]);
#pragma unroll
                for (int c = 0; c < NCT; ++c) {
                    if (!((CM >> c) & 1)) continue;
                    // Q row 32*c + j has the same swizzle as row j
                    const u32x4 b = *(const u32x4 *)(qlds + 32 * c * ROWB + ka[ks]);
                    s[c] = E::mfma(a, b, s[c]);
                }
            }
        }
        const float c2s = q8 ? c2q : c2;
        u32x4 pf[NCT][2];
#pragma unroll
        for (int c = 0; c < NCT; ++c) {
            if (!((CM >> c) & 1)) continue;
            // mask: keys past a row's causal bound (new rows) or past the cached
            // prefix (an int8 stage reaching beyond npre)
            if (key0 + SKEYS > npre + 1 || (q8 && key0 + SKEYS > npre)) {
                const int64_t lim64 = (q8 ? npre - 1 : pos[c]) - key0;
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
            mx = pair_max(mx) * c2s;
            // the first stage, or p could exceed 2^kRescaleSlack
            const bool need = mx > rs[c].m + kRescaleSlack;
            if (__ballot(need)) move_reference(rs[c], need ? mx : rs[c].m);
            auto exps = [&]() {
                float lsum = 0.f;
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[c][i], c2s, -rs[c].m));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[c][i + 1], c2s, -rs[c].m));
                    const uint32_t pk = E::pack2(p0, p1);
                    lsum += p0 + p1;
                    pf[c][i >> 3][(i & 7) >> 1] = pk;
                }
                return lsum;
            };
            float lsum = exps();
            // a new maximum whose weight exceeds kSignificance of the row's
            // mass: reference to that maximum, exactly (the lane test holds
            // in the lane that has the key)
            if (__ballot(mx > rs[c].m && lsum > kSignificance * (rs[c].l + lsum))) {
                const float pmax = __builtin_amdgcn_exp2f(mx - rs[c].m);
                const bool mv = mx > rs[c].m && pmax > kSignificance * pair_sum(rs[c].l + lsum);
                if (__ballot(mv)) {
                    move_reference(rs[c], mv ? mx : rs[c].m);
                    lsum = exps();
                }
            }
            rs[c].l += lsum;
        }
        // O^T += V^T P^T: each V^T fragment feeds NCT chains
        if constexpr (q8) {
            // lane (j, grp): codes of head-dim row 32 mt + j, key slots of half kk = 0 and 1
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt) {
                const int d = 32 * mt + j;
                const u32x4 w = *(const u32x4 *)(vs_ + d * 32 + 16 * (grp ^ swzv(d)));
                u32x4 a0, a1;
                codes_to_bf16(w, a0, a1);
#pragma unroll
                for (int c = 0; c < NCT; ++c) {
                    if (!((CM >> c) & 1)) continue;
                    rs[c].o[mt] = E::mfma(a0, pf[c][0], rs[c].o[mt]);
                    rs[c].o[mt] = E::mfma(a1, pf[c][1], rs[c].o[mt]);
                }
            }
        } else {
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
                        if ((CM >> c) & 1) rs[c].o[mt] = E::mfma(a, pf[c][kk], rs[c].o[mt]);
                }
        }
    };
    auto stage = [&](auto kind, int t) {
        constexpr bool q8 = decltype(kind)::value;
        asm volatile("" ::: "memory");
        if (t + 1 < my_n) {
            load_stage(t + 1);          // its slot held stage t-1, consumed last iteration
            if (is_q8(t + 1)) wait_vmcnt<LOADS_Q8>();   // stage t landed, stage t+1 in flight
            else wait_vmcnt<LOADS>();
        } else {
            wait_vmcnt<0>();
        }
        asm volatile("" ::: "memory");
        const int i_st = wave + 4 * t;
        // absolute key of the stage's first row
        const int64_t key0 = Q8 ? (q8 ? kb + (int64_t)i_st * SKEYS : npre + (int64_t)(i_st - n_cst) * SKEYS)
                                : kb + (int64_t)i_st * SKEYS;
        const unsigned char *ks_ = smem + ring_lds + (t % NSW) * STAGE;
        const unsigned char *vs_ = ks_ + HALF;
        if constexpr (Q8 && !q8) {
            if (!o_scaled) scale_o();
        }
        compute(kind, std::integral_constant<int, (1 << NCT) - 1>{}, ks_, vs_, key0);
    };

    // the split suffix stage, one column tile per wave (waves 0 .. NCT-1), then a
    // barrier: after it wave 3 may refill its second slot
    if (sfx_split) {
        const int64_t key0 = kb + (int64_t)SKEYS * (nst - 1);
        if (wave == 0) compute(std::false_type{}, std::integral_constant<int, 1>{}, sfx_lds, sfx_lds + HALF, key0);
        if constexpr (NCT > 1) {
            if (wave == 1) compute(std::false_type{}, std::integral_constant<int, 2>{}, sfx_lds, sfx_lds + HALF, key0);
        }
        if constexpr (NCT > 2) {
            if (wave == 2) compute(std::false_type{}, std::integral_constant<int, 4>{}, sfx_lds, sfx_lds + HALF, key0);
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    }
    int t = 0;
    if constexpr (Q8) {
        for (; t < my_n && is_q8(t); ++t) stage(std::true_type{}, t);
    }
    for (; t < my_n; ++t) stage(std::false_type{}, t);
    if (Q8 && !o_scaled) scale_o();

    // ---- merge: post (m, l) and the non-owned O quarters, one barrier, then
    // wave w finishes head-dim quarter w
    __syncthreads();                    // every wave is done with its ring and with Q
    float4 *obuf = (float4 *)smem;
    float *lbuf = (float *)(smem + obuf_bytes<NCT>());
    float *mbuf = lbuf + 4 * NCT * 64;
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
        mbuf[(wave * NCT + c) * 64 + lane] = rs[c].m;
        lbuf[(wave * NCT + c) * 64 + lane] = rs[c].l;
    }
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt) {
        if (mt == wave) continue;
        const int slot = 3 * mt + (wave > mt ? wave - 1 : wave);
#pragma unroll
        for (int c = 0; c < NCT; ++c)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                obuf[((slot * NCT + c) * 4 + q4) * 64 + lane] =
                    make_float4(rs[c].o[mt][4 * q4], rs[c].o[mt][4 * q4 + 1], rs[c].o[mt][4 * q4 + 2],
                                rs[c].o[mt][4 * q4 + 3]);
    }
    __syncthreads();
    switch (wave) {
        case 0: finish_quarter<E, NCT, 0>(p, rs, obuf, lbuf, mbuf, valid, tok, head, g, split, lane); break;
        case 1: finish_quarter<E, NCT, 1>(p, rs, obuf, lbuf, mbuf, valid, tok, head, g, split, lane); break;
        case 2: finish_quarter<E, NCT, 2>(p, rs, obuf, lbuf, mbuf, valid, tok, head, g, split, lane); break;
        default: finish_quarter<E, NCT, 3>(p, rs, obuf, lbuf, mbuf, valid, tok, head, g, split, lane); break;
    }
    if (!Q8 && p.kc_app && (p.nsplit == 1 || last_split)) append_new_rows<ROWB>(p, g, S, tid, THREADS);
}

}  // namespace

template <bool Q8, class E>
void launch_nct(const AttnParams &p, int ncol_tiles, int grid, hipStream_t s) {
    switch (ncol_tiles) {
        case 1: hipLaunchKernelGGL((attn_cont_kernel<1, Q8, E>), dim3(grid), dim3(THREADS), 0, s, p); break;
        case 2: hipLaunchKernelGGL((attn_cont_kernel<2, Q8, E>), dim3(grid), dim3(THREADS), 0, s, p); break;
        default: hipLaunchKernelGGL((attn_cont_kernel<3, Q8, E>), dim3(grid), dim3(THREADS), 0, s, p); break;
    }
}

hipError_t launch_attn_cont(const AttnParams &p, int ncol_tiles, bool q8, bool f16, int grid, hipStream_t s) {
    if (q8) launch_nct<true, Bf16>(p, ncol_tiles, grid, s);
    else if (f16) launch_nct<false, F16>(p, ncol_tiles, grid, s);
    else launch_nct<false, Bf16>(p, ncol_tiles, grid, s);
    return hipGetLastError();
}

}  // namespace kvr
