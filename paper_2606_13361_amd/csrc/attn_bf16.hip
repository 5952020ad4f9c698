// attn_bf16.hip -- causal grouped-query attention with a query offset, bf16
// in, fp32 accumulate, for gfx950 (MI355X): the register-staged member of the
// kernel family.  It serves every mode at head_dim 64 and continuations of
// more than 96 query rows per kv head at head_dim 128; prefill and many
// readers at head_dim 128 run on the two-group kernel (attn_pp.hip), shorter
// continuations on attn_rows.hip / attn_cont.hip.  The per-tile arithmetic is
// shared (attn_common.hpp).
//
//   prefill   keys are the new rows only, row tiles visited longest first, and
//             the workgroup owning a token also writes its K/V row into the
//             cache from the registers it staged (one launch does both)
//   continue  cached prefix + new rows, prefix split across workgroups
//   readers   shared prefix + each reader's own rows
//
// Per workgroup: 4 waves x 32 query rows = 128 rows of one kv head; every
// wave reads the same K/V tile from LDS (GQA sharing).  Tiles of 64 keys are
// staged global -> registers -> LDS, double buffered: the next tile's global
// loads are issued before the current tile's math.  K rows are padded to a
// 16-byte multiple + 16 (conflict-free 16-byte reads), V rows by 64 bytes
// (conflict-free transposing reads).
#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

template <int D>
struct Tile {
    static constexpr int CH = D / 8;                  // 16-byte chunks per K/V row
    static constexpr int RPP = THREADS / CH;          // rows staged per pass
    static constexpr int KPT = BN / RPP;              // passes (rows per thread): 4 or 2
    static constexpr int K_PITCH = D * 2 + 16;        // LDS bytes per K row
    static constexpr int V_PITCH = D * 2 + 64;        // LDS bytes per V row
    static constexpr int K_BYTES = BN * K_PITCH;
    static constexpr int V_BYTES = BN * V_PITCH;
    static constexpr int STAGE = K_BYTES + V_BYTES;
    static_assert(KPT * RPP == BN, "tile staging must cover the tile");
};

template <int D, int MODE, class E>
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_bf16_kernel(const AttnParams p) {
    using T = Tile<D>;
    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * T::STAGE];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int lane = tid & 63;
    const int j = lane & 31;      // query row (MFMA column) owned by this lane
    const int grp = lane >> 5;    // which half of each key quad-set this lane holds

    const Work w = decode_work<MODE>(p);
    const int G = w.G;
    const int row0 = w.row0;
    const int64_t npre = w.npre, kb = w.kb, ke = w.ke;
    const int g = w.g;
    const int tok0 = w.tok0;

    // ---- this lane's query row
    const int r = row0 + wave * 32 + j;
    const bool valid = r < w.R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int64_t pos = valid ? npre + tok : -1;   // absolute position; -1 sees nothing
    // rows of this wave see every key below k_full (no mask needed there)
    const int wrow0 = row0 + wave * 32;
    const bool wave_active = wrow0 < w.R;
    const int64_t k_full = wave_active ? npre + wrow0 / G + 1 : 0;

    // ---- Q^T fragments (MFMA B operand): column j, head-dim slots 16*ks + 8*grp + 0..7
    u32x4 qf[D / 16];
    {
        const uint16_t *qrow = (const uint16_t *)p.q + ((int64_t)(tok0 + tok) * p.n_q_heads + head) * D;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
            qf[ks] = valid ? *(const u32x4 *)(qrow + 16 * ks + 8 * grp) : (u32x4){0, 0, 0, 0};
        // RoPE (prefill, readers): the row is rotated once, at its own position
        if (p.rope && valid) rope_q_frag<E, D>(qf, p.rope + pos * D, grp);
    }

    // ---- staging map: thread -> 16-byte chunk sc of rows srow + RPP * i
    const int sc = tid % T::CH;
    const int srow = tid / T::CH;
    const uint16_t *kc = (const uint16_t *)p.kc + (int64_t)g * p.cap * D + 8 * sc;
    const uint16_t *vc = (const uint16_t *)p.vc + (int64_t)g * p.cap * D + 8 * sc;
    const int64_t nstride = p.new_tok_stride;
    const int64_t nhead = p.new_head_stride * g;
    const uint16_t *kn = (const uint16_t *)p.kn + (int64_t)tok0 * nstride + nhead + 8 * sc;
    const uint16_t *vn = (const uint16_t *)p.vn + (int64_t)tok0 * nstride + nhead + 8 * sc;
    uint16_t *kco = (uint16_t *)p.kc_out + (int64_t)g * p.cap * D + 8 * sc;   // prefill: cache rows out
    uint16_t *vco = (uint16_t *)p.vc_out + (int64_t)g * p.cap * D + 8 * sc;

    u32x4 kreg[T::KPT], vreg[T::KPT];
    // Interior tiles (all 64 rows from one source, none past ke, no cache row
    // to store) load with one uniform base address per tile and fixed
    // per-thread byte offsets.  Only the tiles at the prefix/new boundary, at
    // the end of the range or holding this workgroup's own prefill tokens take
    // the general path, where rows past ke are clamped to a valid row (they lie
    // beyond every row's causal bound, so they are masked and never count).
    // 32-bit byte offsets per pass: interior tiles load through a buffer
    // resource (uniform base in SGPRs) plus these per-lane offsets
    uint32_t coff[T::KPT], noff[T::KPT];
#pragma unroll
    for (int i = 0; i < T::KPT; ++i) {
        coff[i] = (uint32_t)((srow + T::RPP * i) * D * 2 + 16 * sc);
        noff[i] = (uint32_t)((srow + T::RPP * i) * nstride * 2 + 16 * sc);
    }
    const int64_t cache_end = ke < npre ? ke : npre;   // keys [.., cache_end) come from the cache
    int64_t own_lo = 0, own_hi = -1;                   // prefill tokens whose cache row this WG stores
    if (MODE == kModePrefill && p.kc_out) {
        own_lo = (row0 + G - 1) / G;
        own_hi = (row0 + ROWS - 1) / G;
    }
    const unsigned char *kc0 = (const unsigned char *)p.kc + (int64_t)g * p.cap * D * 2;
    const unsigned char *vc0 = (const unsigned char *)p.vc + (int64_t)g * p.cap * D * 2;
    const unsigned char *kn0 = (const unsigned char *)p.kn + ((int64_t)tok0 * nstride + nhead) * 2;
    const unsigned char *vn0 = (const unsigned char *)p.vn + ((int64_t)tok0 * nstride + nhead) * 2;
    auto gload = [&](int64_t k0) {
        const bool own = MODE == kModePrefill && k0 <= own_hi && k0 + BN > own_lo;
        if (k0 + BN <= cache_end) {
            const auto rk = buf_rsrc(kc0 + k0 * D * 2), rv = buf_rsrc(vc0 + k0 * D * 2);
#pragma unroll
            for (int i = 0; i < T::KPT; ++i) {
                kreg[i] = buf_load16(rk, coff[i]);
                vreg[i] = buf_load16(rv, coff[i]);
            }
        } else if (k0 >= npre && k0 + BN <= ke && !own) {
            const auto rk = buf_rsrc(kn0 + (k0 - npre) * nstride * 2), rv = buf_rsrc(vn0 + (k0 - npre) * nstride * 2);
#pragma unroll
            for (int i = 0; i < T::KPT; ++i) {
                kreg[i] = buf_load16(rk, noff[i]);
                vreg[i] = buf_load16(rv, noff[i]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < T::KPT; ++i) {
                const int64_t key = k0 + srow + T::RPP * i;
                const int64_t kk = key < ke ? key : ke - 1;
                const bool in_cache = kk < npre;
                const int64_t off = in_cache ? kk * D : (kk - npre) * nstride;
                const uint16_t *kbase = in_cache ? kc : kn;
                const uint16_t *vbase = in_cache ? vc : vn;
                kreg[i] = *(const u32x4 *)(kbase + off);
                vreg[i] = *(const u32x4 *)(vbase + off);
                if constexpr (MODE == kModePrefill) {
                    // the workgroup holding the first query row of token `key` stores its cache row
                    if (key >= own_lo && key <= own_hi && key < ke) {
                        *(u32x4 *)(kco + key * D) = kreg[i];
                        *(u32x4 *)(vco + key * D) = vreg[i];
                    }
                }
            }
        }
    };
    auto swrite = [&](int stage) {
        unsigned char *ks_ = smem + stage * T::STAGE;
        unsigned char *vs_ = ks_ + T::K_BYTES;
#pragma unroll
        for (int i = 0; i < T::KPT; ++i) {
            *(u32x4 *)(ks_ + (srow + T::RPP * i) * T::K_PITCH + 16 * sc) = kreg[i];
            *(u32x4 *)(vs_ + (srow + T::RPP * i) * T::V_PITCH + 16 * sc) = vreg[i];
        }
    };

    // Transposing V read: in each 16-lane group, lane i addresses
    // V[key KB + i/4][d D0 + 4*(i%4) .. +3] and receives column d = D0 + i over
    // the 4 keys KB..KB+3 -- the V^T MFMA operand slots of keys 4*grp + 0..3.
    const int l16 = lane & 15;
    const int g16 = lane >> 4;
    const uint32_t v_lane = (4 * (g16 >> 1) + (l16 >> 2)) * T::V_PITCH + (16 * (g16 & 1) + 4 * (l16 & 3)) * 2;
    const uint32_t k_lane = j * T::K_PITCH + 16 * grp;

    RowState<D> rs;
    rs.zero();
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
            const bool mask = k0 + BN > k_full;
            const int64_t lim64 = pos - k0;
            const int lim = lim64 < -1 ? -1 : (lim64 > BN ? BN : (int)lim64);
            tile_step<E, D>(
                rs, qf,
                [&](int st, int ks) { return ks_ + k_lane + 32 * st * T::K_PITCH + 32 * ks; },
                [&](int st, int kk, int h, int mt) {
                    return vs_ + v_lane + (32 * st + 16 * kk + 8 * h) * T::V_PITCH + 64 * mt;
                },
                mask, lim, c2, grp);
        }
        if (more) swrite(cur ^ 1);
        __syncthreads();
    }
    epilogue<E, D, MODE>(p, w, rs, r, valid, tok, head, grp);
}

template <int D, class E>
hipError_t launch_d(const AttnParams &p, int mode, int grid, hipStream_t s) {
    switch (mode) {
        case kModePrefill:
            hipLaunchKernelGGL((attn_bf16_kernel<D, kModePrefill, E>), dim3(grid), dim3(THREADS), 0, s, p);
            break;
        case kModeContinue:
            hipLaunchKernelGGL((attn_bf16_kernel<D, kModeContinue, E>), dim3(grid), dim3(THREADS), 0, s, p);
            break;
        default:
            hipLaunchKernelGGL((attn_bf16_kernel<D, kModeReaders, E>), dim3(grid), dim3(THREADS), 0, s, p);
            break;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams &p, int head_dim, int mode, bool f16, int grid, hipStream_t s) {
    if (f16) return head_dim == 128 ? launch_d<128, F16>(p, mode, grid, s) : launch_d<64, F16>(p, mode, grid, s);
    return head_dim == 128 ? launch_d<128, Bf16>(p, mode, grid, s) : launch_d<64, Bf16>(p, mode, grid, s);
}


}  // namespace kvr
