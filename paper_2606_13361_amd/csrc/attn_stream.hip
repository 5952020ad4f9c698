// attn_stream.hip -- the streamed member of the bf16 attention family, for
// many readers of one long cached prefix, head_dim 128.
//
// K/V tiles go from global memory straight into LDS (global_load_lds_dwordx4,
// no registers on the way), NSTAGE tiles deep: NSTAGE-1 tiles are in flight
// while one is computed, which is what keeps enough bytes moving per CU to
// stream a cache from HBM.  Waits are explicit (s_waitcnt vmcnt for this
// wave's own loads, then s_barrier for everybody's), so the loads of later
// tiles stay in flight across the barrier.
//
// LDS layout: a 64-key tile of K (and of V) is 64 rows of 256 bytes, no
// padding; the 16-byte chunk c of row r sits in slot c ^ swz(r) with
// swz(r) = ((r >> 2) & 3) | ((r & 3) << 2), which makes both the 16-byte K
// reads (16 rows, one chunk) and the transposing V reads (4 rows x 16 bytes
// per lane group) touch every bank once.
//
// The per-tile arithmetic is the shared tile_step (attn_common.hpp).
#include "attn_common.hpp"

namespace kvr {
namespace {

using namespace dev;

constexpr int D = 128;
constexpr int ROW_BYTES = D * 2;                        // 256
constexpr int ROWS_PER_LOAD = 64 * 16 / ROW_BYTES;      // one wave instruction moves 4 rows

// NSUB 32-key sub-tiles per pipeline stage
template <int NSUB>
struct Stage {
    static constexpr int KEYS = 32 * NSUB;
    static constexpr int TILE_BYTES = KEYS * ROW_BYTES;                    // K (or V) of one stage
    static constexpr int BYTES = 2 * TILE_BYTES;
    static constexpr int LOADS = 2 * TILE_BYTES / (THREADS * 16);          // per thread per stage (K + V)
    static constexpr int LOADS_PER_WAVE = TILE_BYTES / (4 * 64 * 16);      // K (or V) instructions per wave
    static constexpr int ROWS_PER_WAVE = KEYS / 4;
};

__device__ __forceinline__ int swz(int row) { return ((row >> 2) & 3) | ((row & 3) << 2); }


template <int NSTAGE, int NSUB, int MODE>
__device__ __forceinline__ void stream_body(const AttnParams &p) {
    using SG = Stage<NSUB>;
    constexpr int KEYS = SG::KEYS;
    constexpr int NL = SG::LOADS_PER_WAVE;
    static_assert(NSTAGE >= 2 && NSTAGE <= 4, "pipeline depth");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[NSTAGE * SG::BYTES];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
    const int lane = tid & 63;
    const int j = lane & 31;
    const int grp = lane >> 5;

    const Work w = decode_work<MODE>(p);
    const int G = w.G;
    const int g = w.g;
    const int64_t npre = w.npre, kb = w.kb, ke = w.ke;

    const int r = w.row0 + wave * 32 + j;
    const bool valid = r < w.R;
    const int tok = valid ? r / G : 0;
    const int head = g * G + (valid ? r % G : 0);
    const int64_t pos = valid ? npre + tok : -1;
    const int wrow0 = w.row0 + wave * 32;
    const bool wave_active = wrow0 < w.R;
    const int64_t k_full = wave_active ? npre + wrow0 / G + 1 : 0;

    u32x4 qf[D / 16];
    {
        const __bf16 *qrow = (const __bf16 *)p.q + ((int64_t)(w.tok0 + tok) * p.n_q_heads + head) * D;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
            qf[ks] = valid ? *(const u32x4 *)(qrow + 16 * ks + 8 * grp) : (u32x4){0, 0, 0, 0};
    }

    // ---- load map: wave `wave`, instruction i covers stage rows RPW*wave + 4*i + 0..3;
    // lane -> row RPW*wave + 4*i + lane/16, LDS slot lane%16 (fixed by the
    // instruction), fetching the global chunk slot ^ swz(row)
    const int64_t nstride_b = (int64_t)p.n_kv_heads * D * 2;   // bytes between new rows
    const unsigned char *kc0 = (const unsigned char *)p.kc + (int64_t)g * p.cap * ROW_BYTES;
    const unsigned char *vc0 = (const unsigned char *)p.vc + (int64_t)g * p.cap * ROW_BYTES;
    const unsigned char *kn0 = (const unsigned char *)p.kn + (int64_t)w.tok0 * nstride_b + (int64_t)g * ROW_BYTES;
    const unsigned char *vn0 = (const unsigned char *)p.vn + (int64_t)w.tok0 * nstride_b + (int64_t)g * ROW_BYTES;
    int lrow[NL];
    uint32_t lchunk[NL], off_c[NL], off_n[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
        lrow[i] = SG::ROWS_PER_WAVE * wave + ROWS_PER_LOAD * i + (lane >> 4);
        lchunk[i] = 16u * (uint32_t)((lane & 15) ^ swz(lrow[i]));
        off_c[i] = (uint32_t)lrow[i] * ROW_BYTES + lchunk[i];
        off_n[i] = (uint32_t)(lrow[i] * nstride_b) + lchunk[i];
    }
    const int64_t cache_end = ke < npre ? ke : npre;
    // addresses as integers: no pointer selects, nothing left in private memory
    const uint64_t kc_a = (uint64_t)(uintptr_t)kc0, vc_a = (uint64_t)(uintptr_t)vc0;
    const uint64_t kn_a = (uint64_t)(uintptr_t)kn0, vn_a = (uint64_t)(uintptr_t)vn0;
    const uint32_t wave_lds = (uint32_t)(SG::ROWS_PER_WAVE * wave * ROW_BYTES);
    auto load_tile = [=](int64_t k0, int stage) {
        const unsigned char *kd = smem + stage * SG::BYTES + wave_lds;
        const unsigned char *vd = kd + SG::TILE_BYTES;
        if (k0 + KEYS <= cache_end) {                     // all rows cached
            const uint64_t kb_ = kc_a + (uint64_t)k0 * ROW_BYTES, vb_ = vc_a + (uint64_t)k0 * ROW_BYTES;
#pragma unroll
            for (int i = 0; i < NL; ++i) dma16_s(kb_, off_c[i], kd + 1024 * i);
#pragma unroll
            for (int i = 0; i < NL; ++i) dma16_s(vb_, off_c[i], vd + 1024 * i);
        } else if (k0 >= npre && k0 + KEYS <= ke) {       // all rows new
            const uint64_t kb_ = kn_a + (uint64_t)(k0 - npre) * (uint64_t)nstride_b;
            const uint64_t vb_ = vn_a + (uint64_t)(k0 - npre) * (uint64_t)nstride_b;
#pragma unroll
            for (int i = 0; i < NL; ++i) dma16_s(kb_, off_n[i], kd + 1024 * i);
#pragma unroll
            for (int i = 0; i < NL; ++i) dma16_s(vb_, off_n[i], vd + 1024 * i);
        } else {
            // mixed or ragged stage: rows past ke clamp to a valid row (beyond every
            // row's causal bound, masked, never counted)
#pragma unroll
            for (int i = 0; i < NL; ++i) {
                const int64_t key = k0 + lrow[i];
                const int64_t kk = key < ke ? key : ke - 1;
                const bool in_cache = kk < npre;
                const uint64_t off = in_cache ? (uint64_t)kk * ROW_BYTES : (uint64_t)(kk - npre) * (uint64_t)nstride_b;
                // base select by mask (a plain select of the two uniform bases was
                // lowered through private memory)
                const uint64_t sel = 0 - (uint64_t)in_cache;
                const uint64_t kbase = (kc_a & sel) | (kn_a & ~sel);
                const uint64_t vbase = (vc_a & sel) | (vn_a & ~sel);
                dma16((const void *)(kbase + off + lchunk[i]), kd + 1024 * i);
                dma16((const void *)(vbase + off + lchunk[i]), vd + 1024 * i);
            }
        }
    };

    // ---- read maps (per lane, loop invariant)
    // K: row 32*st + j, chunk 2*ks + grp -> slot (2*ks + grp) ^ swz(j)  (st does not change swz)
    uint32_t ka[D / 16];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) ka[ks] = (uint32_t)j * ROW_BYTES + 16u * (uint32_t)((2 * ks + grp) ^ swz(j));
    // V (transposing read): lane i of 16-lane group g16 reads row KB + i/4 at head-dim
    // D0 + 4*(i%4): chunk (D0 + 4*(i%4)) / 8, half (i%4) & 1, with
    // KB = 32*st + 16*kk + 8*h + 4*(g16/2) and D0 = 32*mt + 16*(g16&1)
    const int l16 = lane & 15;
    const int g16 = lane >> 4;
    uint32_t va[2][D / 32];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt) {
            const int row = 8 * h + 4 * (g16 >> 1) + (l16 >> 2);      // + 32*st + 16*kk (keeps swz)
            const int dcol = 32 * mt + 16 * (g16 & 1) + 4 * (l16 & 3);
            const int chunk = dcol / 8;
            va[h][mt] = (uint32_t)row * ROW_BYTES + 16u * (uint32_t)(chunk ^ swz(row)) + 8u * (uint32_t)(l16 & 1);
        }

    RowState<D> rs;
    rs.zero();
    const float c2 = p.scale_log2;
    const int ntiles = ke > kb ? (int)((ke - kb + KEYS - 1) / KEYS) : 0;
    constexpr int PF = NSTAGE - 1;   // stages in flight while one is computed

#pragma unroll
    for (int s = 0; s < PF; ++s)
        if (s < ntiles) load_tile(kb + (int64_t)s * KEYS, s);

    for (int it = 0; it < ntiles; ++it) {
        // this wave's loads of stage `it` are done once at most `ahead` later stages' remain
        const int ahead = min(PF - 1, ntiles - 1 - it);
        asm volatile("" ::: "memory");
        if (ahead >= 2) wait_vmcnt<2 * SG::LOADS>();
        else if (ahead == 1) wait_vmcnt<SG::LOADS>();
        else wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();          // ... and everybody's; the stage refilled next was read last iteration
        asm volatile("" ::: "memory");
        if (it + PF < ntiles) load_tile(kb + (int64_t)(it + PF) * KEYS, (it + PF) % NSTAGE);

        if (wave_active) {
            const int64_t k0 = kb + (int64_t)it * KEYS;
            const unsigned char *ks_ = smem + (it % NSTAGE) * SG::BYTES;
            const unsigned char *vs_ = ks_ + SG::TILE_BYTES;
            const bool mask = k0 + KEYS > k_full;
            const int64_t lim64 = pos - k0;
            const int lim = lim64 < -1 ? -1 : (lim64 > KEYS ? KEYS : (int)lim64);
            tile_step<D, NSUB>(
                rs, qf, [&](int st, int ks) { return ks_ + ka[ks] + 32 * st * ROW_BYTES; },
                [&](int st, int kk, int h, int mt) { return vs_ + va[h][mt] + (32 * st + 16 * kk) * ROW_BYTES; },
                mask, lim, c2, grp);
        }
    }
    epilogue<D, MODE>(p, w, rs, r, valid, tok, head, grp);
}

// many readers: two workgroups per CU, so registers must fit two waves per SIMD
__global__ __launch_bounds__(THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
void attn_stream_readers_kernel(const AttnParams p) {
    stream_body<kStreamStagesReaders, kStreamSubReaders, kModeReaders>(p);
}

}  // namespace

hipError_t launch_attn_stream_readers(const AttnParams &p, int grid, hipStream_t s) {
    hipLaunchKernelGGL(attn_stream_readers_kernel, dim3(grid), dim3(THREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace kvr
