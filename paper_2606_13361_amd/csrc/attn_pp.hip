// attn_pp.hip -- prefill and many readers, bf16, head_dim 128: the two-group
// ("ping-pong") member of the attention family.
//
// A workgroup is 8 waves, 2 per SIMD, holding 256 query rows of one kv head
// (32 rows per wave, GQA-packed as everywhere in the family).  Waves 0-3 form
// group A, waves 4-7 group B; the two waves sharing a SIMD belong to
// different groups.  Per 64-key tile t a group runs two steps:
//   GEMM(t)  O += V_{t-1} P_{t-1}  and  S_t = K_t Q^T     (32 MFMAs)
//   SOFT(t)  mask, row max, rescale, P_t = exp2(...)        (VALU)
// and the groups are offset by one step: while A runs GEMM(t), B runs
// SOFT(t-1); while A runs SOFT(t), B runs GEMM(t).  Every step ends at a
// workgroup barrier, so each SIMD always has one wave feeding the matrix core
// and one wave on the vector ALU.  The wave in its GEMM step runs at raised
// wave priority (s_setprio), so its MFMAs are not starved by the other
// wave's vector stream; without it the older wave slot wins and the phases
// where the younger wave multiplies run about 40 % longer.
//
// K/V tiles reach LDS by direct loads (global_load_lds_dwordx4) into a ring
// of 4 stages of 32 KB: tile t is issued four steps before its first use and
// its stage is refilled only after both groups have read it.  Rows are
// unpadded 256-byte rows with the 16-byte chunk c of row r in slot
// c ^ swz(r) (conflict-free K reads and transposing V reads).
//
// The workgroup holding the first query row of a token also copies that
// token's K/V rows into the cache, from the tiles still in LDS after its
// attention work; output rows leave through LDS as full 256-byte rows.
#include <type_traits>

#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int D = 128;
constexpr int ROWB = D * 2;               // 256 bytes per K/V row
constexpr int KEYS = 64;                  // keys per tile
constexpr int TILE = KEYS * ROWB;         // 16 KB: K (or V) of one tile
constexpr int STAGE = 2 * TILE;           // 32 KB
constexpr int NS = 4;                     // ring stages: 128 KB of LDS
constexpr int PP_THREADS = 512;
constexpr int PP_LOADS = 4;               // direct loads per wave per tile (2 K + 2 V)
static_assert(kSlackSum == (float)(1 << (int)kRescaleSlack), "slack sum must match the rescale slack");

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }

// the four loads of a step: K and V bases (uniform), the lanes' offsets for row
// groups 0 and 1, the LDS destination
struct TileSrc {
    uint64_t kb, vb;
    uint32_t o0, o1;
    int lds;          // LDS byte offset of load 0
    int on;           // 1: the loads run; 0: they run with no lane enabled
};

template <int MODE, class E>
__global__ __launch_bounds__(PP_THREADS) void attn_pp_kernel(const AttnParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[NS * STAGE];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int gw = wave >> 2;                                    // group: 0 = A, 1 = B
    const int lane = tid & 63;
    const int j = lane & 31;
    const int grp = lane >> 5;

    // ---- work: kv head fastest (XCD locality); prefill row tiles longest first.
    // Keys are the cached prefix [0, npre) (readers) followed by own rows from
    // token tok0 on; prefill has no prefix.
    //
    // Readers: the rows of all readers of the launch are packed (G rows per
    // token, token-major) and cut into tiles of kRowsPP rows regardless of
    // where a reader ends, since every reader sees the same prefix.  A tile's
    // own keys start at the first token of the reader that holds its first row
    // (tok0); a row of a later reader in the tile must not see the own keys
    // before its reader's first token, keys [npre, lo) in its frame.  Tiles
    // from tail_tile0 on run as nsplit workgroups each, over equal shares of
    // the tile's key tiles, and leave fp32 partials for the merge kernel.
    const int G = p.group;
    const int g = blockIdx.x % p.n_kv_heads;
    const int bh = blockIdx.x / p.n_kv_heads;
    int tile_lin, split = 0, nsplit = 1, tok0, R, row0, seg0 = 0;
    if constexpr (MODE == kModePrefill) {
        tile_lin = p.tiles_total - 1 - bh;
        tok0 = 0;
        R = G * p.seg_tok0[1];
        row0 = tile_lin * kRowsPP;
    } else {
        if (bh < p.tail_tile0) {
            tile_lin = bh;
        } else {
            nsplit = p.nsplit;
            split = (bh - p.tail_tile0) % nsplit;
            tile_lin = p.tail_tile0 + (bh - p.tail_tile0) / nsplit;
        }
        const int T0 = p.seg_tok0[0];
        const int prow0 = tile_lin * kRowsPP;                 // packed row of the launch
        seg0 = segment_of_token(p, T0 + prow0 / G, 0);
        tok0 = p.seg_tok0[seg0];
        R = G * (p.seg_tok0[p.n_seg] - tok0);
        row0 = prow0 - G * (tok0 - T0);
    }
    const int row_last = min(row0 + kRowsPP, R) - 1;
    const int npre = MODE == kModePrefill ? 0 : (int)p.n_prefix;
    const int ke = npre + row_last / G + 1;                       // keys any row here may see
    const int ntiles = (ke + KEYS - 1) / KEYS;
    // this workgroup's key tiles [tb, te)
    const int tb = MODE == kModePrefill ? 0 : split * ntiles / nsplit;
    const int te = MODE == kModePrefill ? ntiles : (split + 1) * ntiles / nsplit;

    // rows 32*slot .. +31 of the tile, slot 2*(wave & 3) + group: a partial tile
    // keeps both waves of a SIMD busy as long as it can
    const int wrow0 = row0 + 32 * (2 * (wave & 3) + gw);
    const int r = wrow0 + j;
    const bool valid = r < R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int pos = valid ? npre + tok : -1;
    const bool wave_active = wrow0 < R;
    const int k_full = wave_active ? npre + wrow0 / G + 1 : 0;   // keys every row of this wave sees
    // readers: the row's hole [npre, lo) (empty for rows of the tile's first
    // reader), the wave's largest lo, and the row's own position for RoPE
    int lo = npre, hole_end = npre;
    if constexpr (MODE == kModeReaders) {
        // the readers that start inside the tile, by a uniform scan (scalar
        // loads; none for a tile inside one reader): the lane keeps the last
        // start at or before its token
        const int t_abs = tok0 + tok;
        const int t_last = tok0 + row_last / G;
        int lo_tok = tok0;
        for (int k = seg0 + 1; k < p.n_seg && p.seg_tok0[k] <= t_last; ++k)
            lo_tok = t_abs >= p.seg_tok0[k] ? p.seg_tok0[k] : lo_tok;
        lo = valid ? npre + (lo_tok - tok0) : npre;
        // rows (and their readers) increase with the lane: the wave's largest lo
        // is its last valid row's
        if (wave_active) hole_end = __builtin_amdgcn_readlane(lo, min(31, R - 1 - wrow0));
    }
    const int rope_pos = pos - (lo - npre);

    u32x4 qf[D / 16];
    {
        const uint16_t *qrow = (const uint16_t *)p.q + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
            qf[ks] = valid ? *(const u32x4 *)(qrow + 16 * ks + 8 * grp) : (u32x4){0, 0, 0, 0};
        // RoPE: the row is rotated once, at its own position
        if (p.rope && valid) rope_q_frag<E, D>(qf, p.rope + (int64_t)rope_pos * D, grp);
    }

    // ---- load map: wave w moves K rows 8w..8w+7 and V rows 8w..8w+7 of a tile,
    // 4 rows per instruction; lane -> row 8w + 4i + lane/16, LDS slot lane%16,
    // global chunk slot ^ swz(row)
    const int64_t nstride_b = p.new_tok_stride * 2;
    const uint64_t nhead_b = (uint64_t)p.new_head_stride * 2 * g;
    // new rows of this segment (key npre + i is row tok0 + i), cached rows of head g
    const uint64_t kn_a = (uint64_t)(uintptr_t)p.kn + (uint64_t)tok0 * nstride_b + nhead_b;
    const uint64_t vn_a = (uint64_t)(uintptr_t)p.vn + (uint64_t)tok0 * nstride_b + nhead_b;
    const uint64_t kc_a = (uint64_t)(uintptr_t)p.kc + (uint64_t)g * p.cap * ROWB;
    const uint64_t vc_a = (uint64_t)(uintptr_t)p.vc + (uint64_t)g * p.cap * ROWB;
    int lrow[2];
    uint32_t lchunk[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        lrow[i] = 8 * wave + 4 * i + (lane >> 4);
        lchunk[i] = 16u * (uint32_t)((lane & 15) ^ swz(lrow[i]));
    }
    // A tile whose 64 rows are all cached or all new is "fast": its loads are
    // the saddr form (one uniform base per tensor, a per-lane row offset),
    // issued from inside a step as straight-line code.  Any other tile (the
    // prefix/new boundary, the ragged end) is loaded row by row, before the step.
    auto tile_fast = [&](int t) {
        const int k0 = t * KEYS;
        return k0 + KEYS <= npre || (k0 >= npre && k0 + KEYS <= ke);
    };
    auto load_rows = [&](int t) {
        // per-row source; rows past ke repeat row ke-1 (beyond every causal
        // bound, masked)
        const int lds0 = (t % NS) * STAGE + 8 * wave * ROWB;
#pragma unroll
        for (int q = 0; q < PP_LOADS; ++q) {
            const int i = q & 1;
            const uint64_t nbase = (q >> 1) ? vn_a : kn_a;
            const uint64_t cbase = (q >> 1) ? vc_a : kc_a;
            const int key = min(t * KEYS + lrow[i], ke - 1);
            const bool c = key < npre;
            const uint64_t off = (uint64_t)(c ? key : key - npre) * (c ? (uint64_t)ROWB : (uint64_t)nstride_b);
            const uint64_t sel = 0 - (uint64_t)c;               // base select by mask
            dma16((const void *)(((cbase & sel) | (nbase & ~sel)) + off + lchunk[i]),
                  smem + lds0 + (q >> 1) * TILE + 1024 * i);
        }
    };
    // The four loads a step issues (load q: K row groups 0, 1, then V row groups
    // 0, 1).  For a fast tile dt they are its loads; otherwise (no tile left, or
    // a tile loaded row by row just before) the same four instructions run with
    // no lane enabled, so every step's loads are branch-free.  Every choice here
    // is wave-uniform.
    auto plan = [&](int dt) {
        const bool fast = dt >= 0 && tile_fast(dt);
        if (dt >= 0 && !fast) load_rows(dt);
        const int k0 = dt * KEYS;
        const bool cached = k0 + KEYS <= npre;
        const uint64_t nrow = (uint64_t)(k0 - npre) * nstride_b;
        const uint64_t row0_k = npre > 0 ? kc_a : kn_a;
        TileSrc f;
        f.kb = fast ? (cached ? kc_a + (uint64_t)k0 * ROWB : kn_a + nrow) : row0_k;
        f.vb = fast ? (cached ? vc_a + (uint64_t)k0 * ROWB : vn_a + nrow) : row0_k;
        const uint32_t stride = fast ? (cached ? (uint32_t)ROWB : (uint32_t)nstride_b) : 0u;
        f.o0 = (uint32_t)lrow[0] * stride + lchunk[0];
        f.o1 = (uint32_t)lrow[1] * stride + lchunk[1];
        f.lds = fast ? (dt % NS) * STAGE + 8 * wave * ROWB : 0;
        f.on = fast ? 1 : 0;
        return f;
    };
    auto dma_fast = [&](const TileSrc &f, int q) {
        dma16_s_if((q >> 1) ? f.vb : f.kb, (q & 1) ? f.o1 : f.o0, smem + f.lds + (q >> 1) * TILE + 1024 * (q & 1), f.on);
    };
    auto load_tile = [&](int t) {
        const TileSrc f = plan(t);
#pragma unroll
        for (int q = 0; q < PP_LOADS; ++q) dma_fast(f, q);
    };

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

    RowState<D> rs;
    rs.zero();
    const float c2 = p.scale_log2;
    f32x16 s[2];            // S_t^T of the two 32-key sub-tiles (GEMM(t) -> SOFT(t))
    u32x4 pf[2][2];         // P_t^T as bf16 (SOFT(t) -> GEMM(t+1))
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int i = 0; i < 16; ++i) s[st][i] = 0.f;
        pf[st][0] = pf[st][1] = (u32x4){0, 0, 0, 0};
    }

    // GEMM(t): O += V_{t-1} P_{t-1} (t > tb), S_t = K_t Q^T (t < te), as 8
    // chunks of 2 S and 2 PV MFMAs; chunk c+1's LDS fragments are read while
    // chunk c's MFMAs run, and nothing moves across chunks (bounded registers)
    auto kfrag = [&](const unsigned char *ks_, int st, int ks) {
        return *(const u32x4 *)(ks_ + ka[ks] + 32 * st * ROWB);
    };
    auto vfrag = [&](const unsigned char *vs_, int idx) {   // PV product idx = (st, kk, mt)
        const int st = idx >> 3, kk = (idx >> 2) & 1, mt = idx & 3;
        const unsigned char *b = vs_ + (32 * st + 16 * kk) * ROWB;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(b + va[0][mt]));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(b + va[1][mt]));
        const u32x2 lo2 = __builtin_bit_cast(u32x2, lo);
        const u32x2 hi2 = __builtin_bit_cast(u32x2, hi);
        return (u32x4){lo2[0], lo2[1], hi2[0], hi2[1]};
    };
    auto pv = [&](const u32x4 &a, int idx) {
        const int st = idx >> 3, kk = (idx >> 2) & 1, mt = idx & 3;
        rs.o[mt] = E::mfma(a, pf[st][kk], rs.o[mt]);
    };
    auto sm = [&](const u32x4 &a, int st, int ks) {
        s[st] = E::mfma(a, qf[ks], s[st]);
    };
    auto s_zero = [&]() {
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int i = 0; i < 16; ++i) s[st][i] = 0.f;
    };
    auto gemm_s = [&](int t) {            // S only (first tile)
        const unsigned char *ks_ = smem + (t % NS) * STAGE;
        s_zero();
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
#pragma unroll
            for (int st = 0; st < 2; ++st) sm(kfrag(ks_, st, ks), st, ks);
    };
    auto gemm_pv = [&](int t) {           // PV only (after the last tile)
        const unsigned char *vs_ = smem + ((t + NS - 1) % NS) * STAGE + TILE;
#pragma unroll
        for (int idx = 0; idx < 16; ++idx) pv(vfrag(vs_, idx), idx);
    };
    auto gemm = [&](auto with_loads, int t, const TileSrc &f) {   // both; with_loads: the
                                                                   // step's loads between chunks
        const unsigned char *ks_ = smem + (t % NS) * STAGE;
        const unsigned char *vs_ = smem + ((t + NS - 1) % NS) * STAGE + TILE;
        s_zero();
        u32x4 k0 = kfrag(ks_, 0, 0), k1 = kfrag(ks_, 1, 0), v0 = vfrag(vs_, 0), v1 = vfrag(vs_, 1);
#pragma unroll
        for (int c = 0; c < 8; ++c) {
            u32x4 nk0, nk1, nv0, nv1;
            if (c + 1 < 8) {
                nk0 = kfrag(ks_, 0, c + 1);
                nk1 = kfrag(ks_, 1, c + 1);
                nv0 = vfrag(vs_, 2 * c + 2);
                nv1 = vfrag(vs_, 2 * c + 3);
            }
            sm(k0, 0, c);
            pv(v0, 2 * c);
            sm(k1, 1, c);
            pv(v1, 2 * c + 1);
            if constexpr (decltype(with_loads)::value) {
                if (c & 1) dma_fast(f, c >> 1);
            }
            __builtin_amdgcn_sched_barrier(0);
            if (c + 1 < 8) {
                k0 = nk0; k1 = nk1; v0 = nv0; v1 = nv1;
            }
        }
    };
    // SOFT(t): causal mask, row max, lazy rescale of (O, l), P_t = 2^(S c2 - m)
    auto soft = [&](auto with_loads, int t, const TileSrc &f) {   // with_loads: the step's
                                                                   // loads among the exps
        const int k0 = t * KEYS;
        const bool in_hole = MODE == kModeReaders && k0 < hole_end && k0 + KEYS > npre;
        if (k0 + KEYS > k_full || in_hole) {
            const int lim = max(-1, min(pos - k0, KEYS));
            // the hole [npre, lo) as tile offsets [h0, h0 + hn): one unsigned compare
            const int h0 = npre - k0;
            const unsigned hn = (unsigned)(lo - npre);
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int o = 32 * st + 8 * (i >> 2) + 4 * grp + (i & 3);
                    const bool dead = (o > lim) | ((unsigned)(o - h0) < hn);   // no short circuit: selects, not branches
                    s[st][i] = dead ? -INFINITY : s[st][i];
                }
        }
        // P against the current reference m first; the row maximum is needed
        // only when some lane's weights sum above 2^kRescaleSlack (then one of
        // them may exceed it) or above kSignificance of its mass so far (then
        // one of them may be a significant new maximum) -- the first tile
        // (m = -1e30) always, on flat rows the next two or three
        auto exps = [&](auto loads) {
            float lsum[4] = {0.f, 0.f, 0.f, 0.f};   // four independent partial sums
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i], c2, -rs.m));
                    const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i + 1], c2, -rs.m));
                    const uint32_t pk = E::pack2(p0, p1);
                    // row sums with plain fp32 adds: a v_dot2 would queue behind the
                    // other wave's MFMAs on the matrix pipe and stall this wave
                    float &acc = lsum[(i >> 1) & 3];
                    acc += p0 + p1;
                    pf[st][i >> 3][(i & 7) >> 1] = pk;
                    if constexpr (decltype(loads)::value) {
                        if ((i & 7) == 6) dma_fast(f, 2 * st + (i >> 3));
                    }
                }
            return (lsum[0] + lsum[1]) + (lsum[2] + lsum[3]);
        };
        float part = exps(with_loads);
        if (__ballot(!(part <= kSlackSum) || part > kSignificance * (rs.l + part))) {
            // row max as a tree (5 dependent levels)
            float v[32];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                v[i] = s[0][i];
                v[16 + i] = s[1][i];
            }
#pragma unroll
            for (int w = 16; w >= 1; w >>= 1)
#pragma unroll
                for (int i = 0; i < w; ++i) v[i] = fmaxf(v[i], v[i + w]);
            const float mx = pair_max(v[0]) * c2;
            const float pmax = __builtin_amdgcn_exp2f(mx - rs.m);
            const bool sig = mx > rs.m && pmax > kSignificance * pair_sum(rs.l + part);
            const bool need = mx > rs.m + (sig ? 0.f : kRescaleSlack);
            if (__ballot(need)) {
                move_reference(rs, need ? mx : rs.m);
                part = exps(std::false_type{});
            }
        }
        rs.l += part;
    };

    // ---- steps, over key tiles [tb, te), phases counted from tb.  Phase 2u
    // starts once tile tb+u has landed (each wave waits for its own loads, then
    // the barrier); during phase 2u every wave issues its loads of tile tb+u+2,
    // spread through its step, into the stage that held tile tb+u-2 (last read
    // in phase 2u-1).  Group A: GEMM(t) in phase 2u, SOFT(t) in phase 2u+1;
    // group B one phase later.  Both run 2n + 2 phases, n = te - tb.
    const int n = te - tb;
    auto sync = [&](int phi) {
        __builtin_amdgcn_sched_barrier(0);
        if ((phi & 1) == 0) {
            if ((phi >> 1) + 1 < n) wait_vmcnt<PP_LOADS>();   // this tile landed, the next may still fly
            else wait_vmcnt<0>();
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        } else {
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    load_tile(tb);
    if (n > 1) load_tile(tb + 1);
    // One use of the Q fragments here, on every path: the compiler puts its wait
    // for their loads (which also covers the first two tiles, issued after them)
    // at this point, and none in the loops below -- otherwise a path that
    // reaches a loop without having used them makes it wait for every load in
    // flight at the first product of each step.
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) asm volatile("" ::"v"(qf[ks]));
    const bool act = wave_active;
    auto next = [&](int t) { return t + 2 < te ? t + 2 : -1; };   // tile issued in tile t's GEMM phase
    if (gw == 0) {
        sync(0);
        if (act) { __builtin_amdgcn_s_setprio(1); gemm_s(tb); __builtin_amdgcn_s_setprio(0); }
        if (next(tb) >= 0) load_tile(next(tb));
        sync(1);
        if (act) soft(std::false_type{}, tb, TileSrc{});
        for (int t = tb + 1; t < te; ++t) {
            sync(2 * (t - tb));
            const TileSrc f = plan(next(t));
            if (act) {
                __builtin_amdgcn_s_setprio(1);
                gemm(std::true_type{}, t, f);
                __builtin_amdgcn_s_setprio(0);
            } else {
#pragma unroll
                for (int q = 0; q < PP_LOADS; ++q) dma_fast(f, q);
            }
            sync(2 * (t - tb) + 1);
            if (act) soft(std::false_type{}, t, TileSrc{});
        }
        sync(2 * n);
        if (act) { __builtin_amdgcn_s_setprio(1); gemm_pv(te); __builtin_amdgcn_s_setprio(0); }
        sync(2 * n + 1);
    } else {
        sync(0);
        if (next(tb) >= 0) load_tile(next(tb));
        sync(1);
        if (act) { __builtin_amdgcn_s_setprio(1); gemm_s(tb); __builtin_amdgcn_s_setprio(0); }
        for (int t = tb + 1; t < te; ++t) {
            sync(2 * (t - tb));
            const TileSrc f = plan(next(t));
            if (act) {
                soft(std::true_type{}, t - 1, f);
            } else {
#pragma unroll
                for (int q = 0; q < PP_LOADS; ++q) dma_fast(f, q);
            }
            sync(2 * (t - tb) + 1);
            if (act) {
                __builtin_amdgcn_s_setprio(1);
                gemm(std::false_type{}, t, TileSrc{});
                __builtin_amdgcn_s_setprio(0);
            }
        }
        sync(2 * n);
        if (act) soft(std::false_type{}, te - 1, TileSrc{});
        sync(2 * n + 1);
        if (act) { __builtin_amdgcn_s_setprio(1); gemm_pv(te); __builtin_amdgcn_s_setprio(0); }
    }

    // ---- epilogue.  Every tile has landed and the ring is only read from here
    // on.  Prefill: group A, idle while group B runs its last PV product, copies
    // the cache rows of the tokens whose first query row is in this workgroup out
    // of the ring: those tokens are the workgroup's last keys (at most 256/G + 1
    // of them, aligned so that they lie within the last four tiles).  Four LDS
    // reads go out before their four stores.
    if constexpr (MODE == kModePrefill) if (p.kc_out && gw == 0) {
        const int own_lo = (row0 + G - 1) / G;
        const int own_hi = row_last / G;               // inclusive, = ke - 1
        const int n_copy = own_hi >= own_lo ? (own_hi - own_lo + 1) * 32 : 0;
        unsigned char *kc = (unsigned char *)p.kc_out + ((int64_t)g * p.cap) * ROWB;
        unsigned char *vc = (unsigned char *)p.vc_out + ((int64_t)g * p.cap) * ROWB;
        constexpr int A_THREADS = PP_THREADS / 2;
        for (int base = tid; base < n_copy; base += 4 * A_THREADS) {
            u32x4 v[4];
            u32x4 *dp[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int idx = min(base + u * A_THREADS, n_copy - 1);   // past the end: re-read, not stored
                const int tk = own_lo + (idx >> 5);
                const int half = (idx >> 4) & 1;             // 0: K row, 1: V row
                const int c = idx & 15;
                const int r = tk & (KEYS - 1);
                v[u] = *(const u32x4 *)(smem + ((tk / KEYS) % NS) * STAGE + half * TILE + r * ROWB + 16 * (c ^ swz(r)));
                dp[u] = (u32x4 *)((half ? vc : kc) + (int64_t)tk * ROWB + 16 * c);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (base + u * A_THREADS < n_copy) *dp[u] = v[u];
        }
    }
    // Readers, a split tile: each row's unnormalised O and its (m, l) go to the
    // workspace for the merge kernel, straight from registers (records numbered
    // from the first row of tile tail_tile0, split-major as the merge reads them).
    if constexpr (MODE == kModeReaders) if (nsplit > 1) {
        const float l_row = pair_sum(rs.l);
        if (valid) {
            const int64_t rows_m = p.rows_total;
            const int64_t mr = (int64_t)G * (tok0 - p.seg_tok0[0]) - (int64_t)p.tail_tile0 * kRowsPP + r;
            const int64_t rec = ((int64_t)split * p.n_kv_heads + g) * rows_m + mr;
            float *orow = p.ws + rec * D;
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4)
                    *(float4 *)(orow + 32 * mt + 8 * q4 + 4 * grp) =
                        make_float4(rs.o[mt][4 * q4], rs.o[mt][4 * q4 + 1], rs.o[mt][4 * q4 + 2], rs.o[mt][4 * q4 + 3]);
            if (grp == 0)
                *(float2 *)(p.ws + (int64_t)nsplit * p.n_kv_heads * rows_m * D + rec * 2) = make_float2(rs.m, l_row);
        }
        return;
    }
    // after this barrier no wave reads the ring any more
    __syncthreads();

    // output rows through LDS: the wave's 32 rows in bf16 (pitch OPITCH), then 16
    // bytes per lane, 4 rows (one token's 4 heads for G = 4: 1 KB) per store
    constexpr int OPITCH = ROWB + 16;
    const float l_tot = pair_sum(rs.l);
    if (wave_active) {
        unsigned char *ob = smem + wave * 32 * OPITCH;
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                u32x2 v;
                v[0] = E::pack2(rs.o[mt][4 * q4] * inv, rs.o[mt][4 * q4 + 1] * inv);
                v[1] = E::pack2(rs.o[mt][4 * q4 + 2] * inv, rs.o[mt][4 * q4 + 3] * inv);
                *(u32x2 *)(ob + j * OPITCH + 2 * (32 * mt + 8 * q4 + 4 * grp)) = v;
            }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // this wave's rows are in LDS
        // all eight LDS reads before the stores
        u32x4 v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = *(const u32x4 *)(ob + (4 * i + (lane >> 4)) * OPITCH + 16 * (lane & 15));
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int rw = wrow0 + 4 * i + (lane >> 4);
            if (rw < R) {
                uint16_t *orow = (uint16_t *)p.out + ((int64_t)(tok0 + rw / G) * p.n_q_heads + g * G + rw % G) * D;
                *(u32x4 *)(orow + 8 * (lane & 15)) = v[i];
            }
        }
    }
}

}  // namespace

hipError_t launch_attn_pp(const AttnParams &p, int mode, bool f16, int grid, hipStream_t s) {
    if (mode == kModePrefill) {
        if (f16) hipLaunchKernelGGL((attn_pp_kernel<kModePrefill, F16>), dim3(grid), dim3(PP_THREADS), 0, s, p);
        else hipLaunchKernelGGL((attn_pp_kernel<kModePrefill, Bf16>), dim3(grid), dim3(PP_THREADS), 0, s, p);
    } else {
        if (f16) hipLaunchKernelGGL((attn_pp_kernel<kModeReaders, F16>), dim3(grid), dim3(PP_THREADS), 0, s, p);
        else hipLaunchKernelGGL((attn_pp_kernel<kModeReaders, Bf16>), dim3(grid), dim3(PP_THREADS), 0, s, p);
    }
    return hipGetLastError();
}

}  // namespace kvr
