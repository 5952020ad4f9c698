// attn_common.hpp -- device pieces shared by the 16-bit attention kernels
// (attn_bf16.hip, attn_pp.hip, attn_rows.hip, attn_cont.hip, merge.hip):
// element formats, work-item decoding, the per-tile MFMA / online-softmax
// step, the direct-to-LDS loads and the epilogue.
//
// Notation of one 64-key tile and one wave (32 query rows = MFMA columns):
//   S^T[key][row] = K Q^T              v_mfma_f32_32x32x16_bf16, K from LDS,
//                                      Q^T fragments held in registers
//   online softmax in the log2 domain  a lane owns one query row and 16 keys
//                                      of each 32-key sub-tile; lanes l and
//                                      l^32 hold the two halves of a row
//   O^T[d][row] += V^T P^T             V^T through the transposing LDS read,
//                                      P^T = the score accumulator, rounded
//                                      to bf16 in registers
// The MFMA k-slots of P^T and V^T only have to name the same key: slot e of
// 16-key half kk of sub-tile st is key 32*st + 16*kk + 8*(e/4) + 4*grp + e%4,
// which is where the score accumulator left it.
#pragma once

#include "kvr_internal.hpp"

namespace kvr {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int BN = kKeyTile;     // keys per tile
constexpr int ROWS = kRowsBf16;  // query rows per workgroup (4 waves x 32)
constexpr int THREADS = 256;
// The running row maximum is only moved when a tile's maximum exceeds it by
// more than this (log2 units): p = 2^(s - m) then stays below 2^8, which bf16
// P and fp32 sums hold as well as p <= 1, and the O rescale is skipped for
// almost every tile.
constexpr float kRescaleSlack = 8.f;
// A lane's weights of one tile summing to at most 2^kRescaleSlack are each at
// most that: the test that lets a tile skip the row maximum.
constexpr float kSlackSum = 256.f;
// A tile whose largest weight (against the current reference) exceeds this
// share of the row's mass so far (running sum plus the tile) is
// "significant": if it also holds a new row maximum, the reference moves to
// that maximum exactly, so that weight is 2^0 = 1, which the 16-bit P operand
// holds without rounding.  Every weight that is rounded then holds at most a
// quarter of its row's final mass, or lies below the reference (as with a
// plain running maximum), so a dominant key of a peaky row never is.  On flat
// rows no key comes near that share after the first tile.
constexpr float kSignificance = 0.25f;

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    // v_cvt_pk_bf16_f32: round to nearest even
    bf16x2 v;
    v[0] = (__bf16)lo;
    v[1] = (__bf16)hi;
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// The two 16-bit element formats of the MFMA path (the descriptor's dtype):
// the matrix product on 8 elements per lane, and the round-to-nearest-even
// packing used for P and for the output rows.
struct Bf16 {
    __device__ static __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
    }
    __device__ static __forceinline__ uint32_t pack2(float lo, float hi) { return pack_bf16x2(lo, hi); }
    // the two elements of a packed word, widened exactly
    __device__ static __forceinline__ float lo(uint32_t w) { return __uint_as_float(w << 16); }
    __device__ static __forceinline__ float hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
};
struct F16 {
    __device__ static __forceinline__ f32x16 mfma(u32x4 a, u32x4 b, f32x16 c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c,
                                                      0, 0, 0);
    }
    __device__ static __forceinline__ uint32_t pack2(float lo, float hi) {
        f16x2 v;
        v[0] = (_Float16)lo;
        v[1] = (_Float16)hi;
        return __builtin_bit_cast(uint32_t, v);
    }
    __device__ static __forceinline__ float lo(uint32_t w) { return (float)__builtin_bit_cast(f16x2, w)[0]; }
    __device__ static __forceinline__ float hi(uint32_t w) { return (float)__builtin_bit_cast(f16x2, w)[1]; }
};

// The cache update of a continuation, done by one workgroup per kv head after
// its attention work: the S new K and V rows of kv head g (token-major inputs)
// into cache rows [n_prefix, n_prefix + S), 16-byte chunks spread over the
// calling threads.  The attention reads cache rows [0, n_prefix) only, so the
// stores never meet a read of the same launch.
template <int ROWB>
__device__ __forceinline__ void append_new_rows(const AttnParams &p, int g, int S, int tid, int nthreads) {
    constexpr int CH = ROWB / 16;
    const int64_t nstride = (int64_t)p.n_kv_heads * ROWB;
    for (int i = tid; i < 2 * S * CH; i += nthreads) {
        const int half = i / (S * CH);                 // 0: K, 1: V
        const int rem = i - half * S * CH;
        const int t = rem / CH, c = rem - t * CH;
        const unsigned char *src = (const unsigned char *)(half ? p.vn : p.kn) + t * nstride + g * ROWB + 16 * c;
        unsigned char *dst = (unsigned char *)(half ? p.vc_app : p.kc_app) +
                             ((int64_t)g * p.cap + p.n_prefix + t) * ROWB + 16 * c;
        *(u32x4 *)dst = *(const u32x4 *)src;
    }
}

// Rotary position embedding of one pair (x1, x2) = (x[i], x[i + d/2]) by the
// angle whose cosine and sine are c and s (rotary embedding of Su et al. in
// the half-split pairing).  Written with explicit fused multiply-adds so that
// every kernel that rotates a row (the key pre-pass, the in-register query
// rotation) produces the same bits.
__device__ __forceinline__ void rope_rot(float x1, float x2, float c, float s, float &y1, float &y2) {
    y1 = __builtin_fmaf(x1, c, -(x2 * s));
    y2 = __builtin_fmaf(x2, c, x1 * s);
}

// Rotate 8 + 8 packed elements: lo holds dims i0..i0+7, hi dims i0+d/2..; cs
// points at the table entries (cos, sin) of dims i0..i0+7 at the row's position.
template <class E>
__device__ __forceinline__ void rope_rot8(u32x4 &lo, u32x4 &hi, const float *cs) {
    const float4 *c4 = (const float4 *)cs;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const float4 t = c4[w];        // (cos, sin) of dims 2w and 2w + 1
        float a1, a2, b1, b2;
        rope_rot(E::lo(lo[w]), E::lo(hi[w]), t.x, t.y, a1, a2);
        rope_rot(E::hi(lo[w]), E::hi(hi[w]), t.z, t.w, b1, b2);
        lo[w] = E::pack2(a1, b1);
        hi[w] = E::pack2(a2, b2);
    }
}

// Query fragments in the matrix-core operand layout (qf[ks] holds dims
// 16 ks + 8 grp .. +7 of the lane's row): the partner of dim i < d/2 is in
// qf[ks + d/32] of the same lane, so the rotation needs no data exchange.
// cs_row: the table row of the lane's position, (cos, sin) for dims 0..d/2-1.
template <class E, int D>
__device__ __forceinline__ void rope_q_frag(u32x4 (&qf)[D / 16], const float *cs_row, int grp) {
#pragma unroll
    for (int ks = 0; ks < D / 32; ++ks) rope_rot8<E>(qf[ks], qf[ks + D / 32], cs_row + 2 * (16 * ks + 8 * grp));
}

// Lanes l and l^32 hold the two halves of one query row.  v_permlane32_swap
// exchanges the upper half of its first operand with the lower half of its
// second; with both operands x the two results are {x[l], x[l^32]} in some
// order, so their max / sum is the row's (and the same bits in both lanes).
__device__ __forceinline__ float pair_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}


// r / G for the small row indices of a continuation workgroup (0 <= r < 128,
// 1 <= G <= 128) from inv_g = 1/G in fp32 (within a few ulp): (r + 1/2) / G
// lies at least 1/(2G) from an integer, far beyond the relative error of a
// few 2^-24 of the product, so the truncation is exact -- one multiply
// instead of an integer division.
__device__ __forceinline__ int div_small(int r, float inv_g) { return (int)(((float)r + 0.5f) * inv_g); }

// Locate the segment (reader) that owns a linear row-tile index.
__device__ __forceinline__ int find_segment(const AttnParams &p, int tile) {
    int lo = 0, hi = p.n_seg - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (p.seg_tile0[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// The segment (reader) that holds packed token t: the last of segments
// [first, n_seg) whose first token is at most t (segments are non-empty, so
// their first tokens increase).
__device__ __forceinline__ int segment_of_token(const AttnParams &p, int t, int first) {
    int lo = first, hi = p.n_seg - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (p.seg_tok0[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// What one workgroup computes: 128 rows (token-major (token, head) pairs of
// kv head g) of one segment, over keys [kb, ke).
struct Work {
    int g, split, seg, tok0, n_tok, G, R, row0, row_last;
    int64_t npre, kb, ke;
};

template <int MODE>
__device__ __forceinline__ Work decode_work(const AttnParams &p) {
    Work w;
    int b = blockIdx.x;
    // kv head fastest: consecutive workgroups land on different XCDs, so each
    // XCD keeps one head's K/V rows in its L2
    w.g = b % p.n_kv_heads;
    b /= p.n_kv_heads;
    w.split = b % p.nsplit;
    b /= p.nsplit;
    const int tile_lin = MODE == kModePrefill ? (p.tiles_total - 1 - b) : b;   // longest rows first
    w.seg = MODE == kModeReaders ? find_segment(p, tile_lin) : 0;
    const int rt = tile_lin - p.seg_tile0[w.seg];
    w.tok0 = p.seg_tok0[w.seg];
    w.n_tok = p.seg_tok0[w.seg + 1] - w.tok0;
    w.G = p.group;
    w.R = w.G * w.n_tok;
    w.row0 = rt * ROWS;
    w.row_last = min(w.row0 + ROWS, w.R) - 1;
    w.npre = MODE == kModePrefill ? 0 : p.n_prefix;
    const int64_t k_all = w.npre + w.row_last / w.G + 1;   // keys any row of the workgroup may see
    w.kb = 0;
    w.ke = k_all;
    if (MODE == kModeContinue && p.nsplit > 1) {
        w.kb = (int64_t)w.split * p.chunk;
        w.ke = (w.split == p.nsplit - 1) ? k_all : min(w.kb + p.chunk, w.npre);
    }
    return w;
}

// Running softmax state of one lane's query row (log2 domain, scaled).
template <int D>
struct RowState {
    f32x16 o[D / 32];
    float m = -1e30f;
    float l = 0.f;
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[mt][i] = 0.f;
    }
};

// Move the reference of a lane's row to m_new (>= the current one): (O, l)
// are rescaled by 2^(m - m_new).
template <int D>
__device__ __forceinline__ void move_reference(RowState<D> &rs, float m_new) {
    const float alpha = __builtin_amdgcn_exp2f(rs.m - m_new);
    rs.m = m_new;
    rs.l *= alpha;
#pragma unroll
    for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
        for (int i = 0; i < 16; ++i) rs.o[mt][i] *= alpha;
}

// Direct-to-LDS load of 16 bytes per lane: lane l's bytes land at LDS byte
// lds + 16*l (lds is wave-uniform).  Issued as inline asm so the compiler does
// not treat it as an LDS write it must wait for before every later LDS read
// (it cannot tell pipeline stages apart and would drain all loads in flight);
// the kernels wait for their own stages explicitly with wait_vmcnt, and order
// these loads against the LDS reads of the slot they refill with compiler
// fences (asm volatile statements keep their order among themselves).
// m0 is named as clobbered: these kernels use it for nothing else (no LDS
// DMA of the compiler's own, no indirect register indexing, no messages).
__device__ __forceinline__ void dma16(const void *src, const void *lds_dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src) : "m0");
}
// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset (the instruction's saddr form): no per-lane address arithmetic.
__device__ __forceinline__ void dma16_s(uint64_t base, uint32_t off, const void *lds_dst) {
    const uint32_t lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds), "v"(off), "s"(base) : "m0");
}

// dma16_s for one instruction under the exec mask when `on` is nonzero, and
// with no lane enabled (nothing loaded, nothing written) when it is zero; `on`
// must be wave-uniform.  exec is restored inside the statement.
__device__ __forceinline__ void dma16_s_if(uint64_t base, uint32_t off, const void *lds_dst, int on) {
    const uint32_t lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)lds_dst;
    const int on_s = __builtin_amdgcn_readfirstlane(on);
    uint64_t saved, m;
    asm volatile("s_mov_b32 m0, %2\n\t"
                 "s_cmp_lg_u32 %5, 0\n\t"
                 "s_cselect_b64 %1, -1, 0\n\t"
                 "s_and_saveexec_b64 %0, %1\n\t"
                 "global_load_lds_dwordx4 %3, %4\n\t"
                 "s_mov_b64 exec, %0"
                 : "=&s"(saved), "=&s"(m)
                 : "s"(lds), "v"(off), "s"(base), "s"(on_s)
                 : "m0", "scc");
}

// 16-byte load through a buffer resource: the 64-bit base lives in SGPRs
// (one per tile, built with scalar arithmetic) and each lane supplies a
// 32-bit byte offset, so interior tiles need no per-lane address arithmetic.
// Raw buffer, stride 0, range 2^31 - 1 bytes (every offset used is far
// below); dword 3 = 0x00020000 is the gfx9-family format word (32-bit data).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
}

// s_waitcnt with vmcnt = N and the other counters left alone (gfx9 encoding:
// vmcnt[3:0] bits 3:0, expcnt bits 6:4, lgkmcnt bits 11:8, vmcnt[5:4] bits 15:14).
// Vector memory loads complete in issue order, so vmcnt(N) means every load
// but the last N issued has landed.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
    asm volatile("" ::: "memory");
}

// One tile of 32 * NSUB keys for one wave.
//   kaddr(st, ks)         LDS byte address of this lane's K fragment (row 32*st + j,
//                         head-dim slots 16*ks + 8*grp .. +7)
//   vaddr(st, kk, h, mt)  LDS byte address this lane passes to the transposing
//                         read for keys 32*st + 16*kk + 8*h + 4*(g16/2) .. +3
//   lim                   keys with tile offset > lim are masked (only if mask)
template <class E, int D, int NSUB = 2, class KA, class VA>
__device__ __forceinline__ void tile_step(RowState<D> &rs, const u32x4 (&qf)[D / 16], KA kaddr, VA vaddr,
                                          bool mask, int lim, float c2, int grp) {
    f32x16 s[NSUB];
#pragma unroll
    for (int st = 0; st < NSUB; ++st)
#pragma unroll
        for (int i = 0; i < 16; ++i) s[st][i] = 0.f;
    // K fragments one head-dim step ahead of the MFMAs that consume them, the
    // NSUB accumulation chains interleaved
    u32x4 a[2][NSUB];
#pragma unroll
    for (int st = 0; st < NSUB; ++st) a[0][st] = *(const u32x4 *)kaddr(st, 0);
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
        if (ks + 1 < D / 16) {
#pragma unroll
            for (int st = 0; st < NSUB; ++st) a[(ks + 1) & 1][st] = *(const u32x4 *)kaddr(st, ks + 1);
        }
#pragma unroll
        for (int st = 0; st < NSUB; ++st)
            s[st] = E::mfma(a[ks & 1][st], qf[ks], s[st]);
    }
    // causal mask: tile key offset 32*st + 8*(i/4) + 4*grp + i%4 is visible iff <= lim
    if (mask) {
#pragma unroll
        for (int st = 0; st < NSUB; ++st)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int o = 32 * st + 8 * (i >> 2) + 4 * grp + (i & 3);
                if (o > lim) s[st][i] = -INFINITY;
            }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < NSUB; ++st)
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[st][i]);
    mx = pair_max(mx) * c2;
    // lazy rescale: move the reference when p could exceed 2^kRescaleSlack
    // (the first tile always)
    const bool need = mx > rs.m + kRescaleSlack;
    if (__ballot(need)) move_reference(rs, need ? mx : rs.m);
    u32x4 pf[NSUB][2];   // P^T as bf16, [sub-tile][16-key half]
    auto exps = [&]() {
        float lsum = 0.f;
#pragma unroll
        for (int st = 0; st < NSUB; ++st) {
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i], c2, -rs.m));
                const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[st][i + 1], c2, -rs.m));
                const uint32_t pk = E::pack2(p0, p1);
                // row sum in fp32 adds (a v_dot2 would wait behind MFMAs on the matrix pipe)
                lsum += p0 + p1;
                pf[st][i >> 3][(i & 7) >> 1] = pk;
            }
        }
        return lsum;
    };
    float lsum = exps();
    // a new maximum whose weight exceeds kSignificance of the row's mass:
    // reference to that maximum, exactly.  The lane test (the lane's weights
    // above that share of its own mass) holds in the lane that has the key.
    if (__ballot(mx > rs.m && lsum > kSignificance * (rs.l + lsum))) {
        const float pmax = __builtin_amdgcn_exp2f(mx - rs.m);
        const bool mv = mx > rs.m && pmax > kSignificance * pair_sum(rs.l + lsum);
        if (__ballot(mv)) {
            move_reference(rs, mv ? mx : rs.m);
            lsum = exps();
        }
    }
    rs.l += lsum;
#pragma unroll
    for (int st = 0; st < NSUB; ++st)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int mt = 0; mt < D / 32; ++mt) {
                const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)vaddr(st, kk, 0, mt));
                const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)vaddr(st, kk, 1, mt));
                const u32x2 lo2 = __builtin_bit_cast(u32x2, lo);
                const u32x2 hi2 = __builtin_bit_cast(u32x2, hi);
                const u32x4 a = {lo2[0], lo2[1], hi2[0], hi2[1]};
                rs.o[mt] = E::mfma(a, pf[st][kk], rs.o[mt]);
            }
}

// Final output (normalised, bf16) or split partial (unnormalised O, m, l).
template <class E, int D, int MODE>
__device__ __forceinline__ void epilogue(const AttnParams &p, const Work &w, const RowState<D> &rs, int r,
                                         bool valid, int tok, int head, int grp) {
    const float l_tot = pair_sum(rs.l);
    if (!valid) return;
    if (MODE != kModeContinue || p.nsplit == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        uint16_t *orow = (uint16_t *)p.out + ((int64_t)(w.tok0 + tok) * p.n_q_heads + head) * D;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int d = 32 * mt + 8 * q4 + 4 * grp;
                u32x2 v;
                v[0] = E::pack2(rs.o[mt][4 * q4 + 0] * inv, rs.o[mt][4 * q4 + 1] * inv);
                v[1] = E::pack2(rs.o[mt][4 * q4 + 2] * inv, rs.o[mt][4 * q4 + 3] * inv);
                *(u32x2 *)(orow + d) = v;
            }
    } else {
        const int64_t prow = ((int64_t)w.split * p.n_kv_heads + w.g) * p.rows_total + r;
        float *po = p.ws + prow * D;
#pragma unroll
        for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int d = 32 * mt + 8 * q4 + 4 * grp;
                *(float4 *)(po + d) = make_float4(rs.o[mt][4 * q4], rs.o[mt][4 * q4 + 1], rs.o[mt][4 * q4 + 2],
                                                  rs.o[mt][4 * q4 + 3]);
            }
        if (grp == 0) {
            float *pml = p.ws + (int64_t)p.nsplit * p.n_kv_heads * p.rows_total * D + prow * 2;
            *(float2 *)pml = make_float2(rs.m, l_tot);
        }
    }
}

}  // namespace dev
}  // namespace kvr
