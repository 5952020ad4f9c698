// kvr_api.hip -- host side of libkvr: argument validation, work planning
// (row tiles, key splits, workspace), and kernel launches on the caller's
// stream.  Validation runs before any HIP call, so every error path can be
// exercised on a machine without a GPU.
#include <math.h>
#include <string.h>

#include <mutex>

#include "kvr.h"
#include "kvr_internal.hpp"

namespace kvr {
namespace {

constexpr int64_t kMaxTokens = (int64_t)1 << 30;   // rows of Q per call; keeps int32 row math safe
constexpr int64_t kMaxKeys = (int64_t)1 << 40;
// Split heuristic for the continuation: aim for this many workgroups on the
// 256-CU part (two per CU for both kernels), never split the prefix below
// this many keys per workgroup.
constexpr int64_t kTargetWorkgroupsStaged = 512;
constexpr int64_t kTargetWorkgroupsCont = 256;   // split-K-in-workgroup kernel: one per CU (155 KB of LDS)
constexpr int64_t kMinSplitKeys = 256;
// longest key range per workgroup for which the row-split continuation is used
constexpr int64_t kRowsSplitMaxKeys = 640;
// Many readers on the two-group kernel (one 128 KB workgroup per CU): tiles
// past the last full round of workgroups are split over the keys, into at
// most this many splits of at least kReaderMinSplitTiles key tiles each.
// Costs in units of one whole workgroup, whose time is about kReaderTileUs per
// key tile: a split workgroup takes 1/ns of it plus kReaderSplitFixed (its own
// query rows, first tiles and epilogue); a split launch adds the merge launch,
// kReaderMergeCost, and the fp32 partials written and read back at about
// kPartialBytesPerUs.
constexpr int64_t kCus = 256;
constexpr int64_t kReaderMaxSplits = 16;
constexpr int64_t kReaderMinSplitTiles = 4;
constexpr double kReaderSplitFixed = 0.07;
constexpr double kReaderMergeCost = 0.04;
constexpr double kReaderTileUs = 2.0;
constexpr double kPartialBytesPerUs = 5.0e6;

// bf16 and fp16 share the 16-bit MFMA path; f16() picks the element format
bool is16(const kvr_desc *d) { return d->dtype == KVR_BF16 || d->dtype == KVR_F16; }
bool f16(const kvr_desc *d) { return d->dtype == KVR_F16; }

// Continuations of at most kContMaxRows query rows per kv head (decode steps,
// short suffixes) at bf16 / head_dim 128 use the kernel whose waves split the keys.
bool use_cont(const kvr_desc *d, int64_t S) {
    return is16(d) && d->head_dim == 128 && (int64_t)(d->n_q_heads / d->n_kv_heads) * S <= kContMaxRows;
}

// Prefill and many readers at bf16 / head_dim 128 use the two-group kernel.
bool use_pp(const kvr_desc *d) { return is16(d) && d->head_dim == 128; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

int check_desc(const kvr_desc *d) {
    if (!d) return KVR_ERR_NULL;
    if (d->dtype != KVR_BF16 && d->dtype != KVR_F32 && d->dtype != KVR_F16) return KVR_ERR_DTYPE;
    if (d->n_q_heads <= 0 || d->n_kv_heads <= 0 || d->n_q_heads % d->n_kv_heads != 0) return KVR_ERR_SHAPE;
    if (d->n_q_heads > 4096) return KVR_ERR_SHAPE;
    if (d->head_dim != 64 && d->head_dim != 128) return KVR_ERR_SHAPE;
    if (d->capacity < 0 || d->capacity > kMaxKeys) return KVR_ERR_SHAPE;
    if (d->reserved != 0) return KVR_ERR_SHAPE;
    if (isnan(d->scale) || isinf(d->scale)) return KVR_ERR_SHAPE;
    return KVR_OK;
}

float eff_scale(const kvr_desc *d) { return d->scale > 0.f ? d->scale : 1.f / sqrtf((float)d->head_dim); }

int elt_bytes(const kvr_desc *d) { return is16(d) ? 2 : 4; }

int rows_per_tile(const kvr_desc *d) { return is16(d) ? kRowsBf16 : kRowsF32; }

struct Split {
    int32_t nsplit;
    int64_t chunk;
    size_t ws_bytes;
};

// Key split of a single continuation: enough workgroups to cover the chip,
// every split a whole number of key tiles.  A pure function of the shape.
Split plan_split(const kvr_desc *d, int64_t L_prefix, int64_t S) {
    Split s{1, 0, 0};
    if (!is16(d) || L_prefix <= 0 || S <= 0) return s;
    const int64_t G = d->n_q_heads / d->n_kv_heads;
    const int64_t rows = G * S;
    const int64_t tiles = (rows + kRowsBf16 - 1) / kRowsBf16;
    const int64_t base = tiles * d->n_kv_heads;
    const int64_t target = use_cont(d, S) ? kTargetWorkgroupsCont : kTargetWorkgroupsStaged;
    if (base >= target) return s;
    int64_t want = (target + base - 1) / base;
    const int64_t most = (L_prefix + kMinSplitKeys - 1) / kMinSplitKeys;
    if (want > most) want = most;
    if (want > kMaxSplits) want = kMaxSplits;
    if (want <= 1) return s;
    int64_t chunk = (L_prefix + want - 1) / want;
    chunk = (chunk + kKeyTile - 1) / kKeyTile * kKeyTile;
    int64_t n = (L_prefix + chunk - 1) / chunk;
    // A prefix up to 32 - S keys past a multiple of want x 128 keys (a decode
    // chain just past a round length) would round every chunk above up by 64 keys,
    // and two of the four waves of the keys-split kernel would run one stage more.
    // Instead: want chunks of a multiple of 128 keys, the last one taking the
    // remainder; its few extra keys share the stage of the new rows, which that
    // kernel runs across its waves.  Every wave then runs the same stage count.
    if (use_cont(d, S) && S <= 32) {
        const int64_t c2 = L_prefix / want / 128 * 128;
        if (c2 >= kMinSplitKeys && L_prefix - want * c2 + S <= 32) {
            chunk = c2;
            n = want;
        }
    }
    if (n <= 1) return s;
    s.nsplit = (int32_t)n;
    s.chunk = chunk;
    // sized by the requested split count (n <= want): non-decreasing in
    // L_prefix, so one workspace serves every shorter prefix of a decode chain
    s.ws_bytes = (size_t)want * d->n_kv_heads * rows * (d->head_dim + 2) * sizeof(float);
    return s;
}

// Many readers (n >= 2) on the two-group kernel, one launch (n <= kMaxSegments):
// the rows of all readers are packed into tiles of kRowsPP rows, tiles per kv
// head = ceil(G total_S / kRowsPP).  The workgroups run in rounds of kCus (one
// per CU); the tiles of a last, partial round would leave CUs idle, so each
// of them runs as nsplit workgroups over equal shares of its key tiles,
// followed by the merge of their partials, nsplit chosen by the cost of the
// rounds the split workgroups take.  A pure function of the shape,
// non-decreasing in L_prefix.
struct ReaderPlan {
    int64_t tiles, tail0, nsplit, rows_tail;
    size_t ws_bytes;
};
ReaderPlan plan_readers(const kvr_desc *d, int64_t L_prefix, int64_t total_S, int32_t n) {
    const int64_t G = d->n_q_heads / d->n_kv_heads;
    ReaderPlan r{0, 0, 1, 0, 0};
    r.tiles = (G * total_S + kRowsPP - 1) / kRowsPP;
    r.tail0 = r.tiles;
    // partial-tile records are whole tokens only when G divides the tile
    if (!use_pp(d) || n < 2 || n > kMaxSegments || kRowsPP % G != 0 || r.tiles == 0) return r;
    const int64_t per_round = kCus / d->n_kv_heads;
    if (per_round < 1) return r;
    const int64_t tail = r.tiles % per_round;
    if (tail == 0) return r;
    const int64_t tail_wg = tail * d->n_kv_heads;
    const int64_t rows_tail = G * total_S - (r.tiles - tail) * kRowsPP;
    const int64_t by_keys = L_prefix / (kReaderMinSplitTiles * kKeyTile);
    // one whole workgroup: the prefix's key tiles and a few of its own
    const double wg_us = kReaderTileUs * (double)(L_prefix / kKeyTile + 2);
    const double rec_bytes = (double)d->n_kv_heads * (double)rows_tail * (d->head_dim + 2) * sizeof(float);
    int64_t ns = 1;
    double best = 1.0 + kReaderSplitFixed;   // the tail as whole workgroups: one round
    for (int64_t k = 2; k <= kReaderMaxSplits && k <= by_keys; ++k) {
        const int64_t rounds = (tail_wg * k + kCus - 1) / kCus;
        const double traffic = 2.0 * (double)k * rec_bytes / kPartialBytesPerUs / wg_us;
        const double c = (double)rounds * (1.0 / (double)k + kReaderSplitFixed) + kReaderMergeCost + traffic;
        if (c < best - 1e-9) {
            best = c;
            ns = k;
        }
    }
    if (ns < 2) return r;
    r.nsplit = ns;
    r.tail0 = r.tiles - tail;
    r.rows_tail = rows_tail;
    r.ws_bytes = (size_t)ns * d->n_kv_heads * r.rows_tail * (d->head_dim + 2) * sizeof(float);
    return r;
}

int to_status(hipError_t e) { return e == hipSuccess ? KVR_OK : KVR_ERR_DEVICE; }

void fill_common(AttnParams &p, const kvr_desc *d) {
    memset(&p, 0, sizeof p);
    p.n_q_heads = d->n_q_heads;
    p.n_kv_heads = d->n_kv_heads;
    p.group = d->n_q_heads / d->n_kv_heads;
    p.scale = eff_scale(d);
    p.scale_log2 = p.scale * 1.4426950408889634f;
    p.cap = d->capacity;
    p.nsplit = 1;
    p.new_tok_stride = (int64_t)d->n_kv_heads * d->head_dim;
    p.new_head_stride = d->head_dim;
}

// RoPE table argument of a call that rotates positions [0, n_pos_needed)
int check_rope(const kvr_rope *r, int64_t n_pos_needed) {
    if (!r || !r->cos_sin) return KVR_ERR_NULL;
    if (r->n_pos < 0 || r->n_pos < n_pos_needed) return KVR_ERR_POSITION;
    if (!aligned16(r->cos_sin)) return KVR_ERR_ALIGN;
    return KVR_OK;
}

size_t align256(size_t b) { return (b + 255) / 256 * 256; }

// Workspace of the RoPE continuations: the plain split partials (of a single
// continuation, or of the many readers' split tiles), then the rotated query
// rows (single continuation only), then the rotated key rows.
struct RopeWs {
    size_t split, q_off, k_off, total;
};
RopeWs rope_ws(const kvr_desc *d, int64_t L_prefix, int64_t total_S, int32_t n) {
    RopeWs w{0, 0, 0, 0};
    const size_t row = (size_t)d->head_dim * elt_bytes(d);
    if (n <= 1) {
        w.split = align256(plan_split(d, L_prefix, total_S).ws_bytes);
        w.q_off = w.split;
        w.k_off = w.q_off + align256((size_t)total_S * d->n_q_heads * row);
    } else {
        w.split = align256(plan_readers(d, L_prefix, total_S, n).ws_bytes);
        w.q_off = w.k_off = w.split;
    }
    w.total = w.k_off + align256((size_t)total_S * d->n_kv_heads * row);
    return w;
}

// One pre-pass job over a single segment of n_tok rows at positions pos0..
RopeParams rope_params(const kvr_desc *d, const kvr_rope *r, int64_t n_tok, int64_t pos0) {
    RopeParams rp;
    memset(&rp, 0, sizeof rp);
    rp.cs = r->cos_sin;
    rp.n_tok = n_tok;
    rp.cap = d->capacity;
    rp.pos0 = pos0;
    rp.n_seg = 1;
    rp.seg_tok0[0] = 0;
    rp.seg_tok0[1] = (int32_t)(n_tok < 0x7fffffff ? n_tok : 0x7fffffff);
    return rp;
}

// One segment: rows of tokens [0, n_tok).
int append_impl(const kvr_desc *d, const void *Ks, const void *Vs, int64_t S, void *kc, void *vc,
                int64_t L_cur, hipStream_t stream) {
    AppendParams a;
    a.k = Ks; a.v = Vs; a.kc = kc; a.vc = vc;
    a.S = S; a.L_cur = L_cur; a.cap = d->capacity;
    a.n_kv_heads = d->n_kv_heads;
    a.row_chunks = d->head_dim * elt_bytes(d) / 16;
    return to_status(launch_append(a, stream));
}

// mode kModePrefill: kc/vc are the caches to fill (bf16: in the attention
// kernel itself); kModeContinue: kc/vc are the cached prefix (read only).
// qscale != NULL: continuation over the int8 artifact (kc/vc are its codes).
// rope != NULL (prefill): rotate the query rows in registers, and read the
// already rotated keys and the values back from kc/vc instead of K/V (the
// RoPE pre-pass wrote them there); the kernel then writes no cache rows.
int launch_single(const kvr_desc *d, int mode, const void *Q, const void *K, const void *V, void *kc,
                  void *vc, int64_t n_prefix, int64_t n_tok, void *out, const Split &sp, void *ws,
                  hipStream_t stream, const float *qscale = nullptr, const float *rope = nullptr,
                  bool append = false) {
    AttnParams p;
    fill_common(p, d);
    p.q = Q; p.kn = K; p.vn = V; p.out = out;
    const bool reverse = mode == kModePrefill;
    const bool keys_in_cache = mode == kModePrefill && rope != nullptr;
    if (keys_in_cache) {
        p.rope = rope;
        p.kn = kc;
        p.vn = vc;
        p.new_tok_stride = d->head_dim;
        p.new_head_stride = d->capacity * d->head_dim;
    } else if (mode == kModePrefill) {
        p.kc_out = kc;
        p.vc_out = vc;
    } else {
        p.kc = kc;
        p.vc = vc;
    }
    p.ws = (float *)ws;
    p.qscale = qscale;
    p.n_prefix = n_prefix;
    p.nsplit = sp.nsplit;
    p.chunk = sp.chunk;
    const int64_t G = p.group;
    const int64_t rows = G * n_tok;
    if (rows > 0x7fffffff) return KVR_ERR_SHAPE;   // row indices are 32-bit on the device
    const int rpt = rows_per_tile(d);
    const int64_t tiles = (rows + rpt - 1) / rpt;
    p.n_seg = 1;
    p.reverse = reverse ? 1 : 0;
    p.tiles_total = (int32_t)tiles;
    p.rows_total = (int32_t)rows;
    p.seg_tok0[0] = 0;
    p.seg_tok0[1] = (int32_t)n_tok;
    p.seg_tile0[0] = 0;
    p.seg_tile0[1] = (int32_t)tiles;
    const int64_t grid = tiles * p.nsplit * p.n_kv_heads;
    if (grid <= 0) return KVR_OK;
    if (grid > 0x7fffffff) return KVR_ERR_SHAPE;
    hipError_t e;
    if (mode == kModeContinue && use_cont(d, n_tok)) {
        // The row split removes the in-workgroup merge and the suffix stage
        // that one wave alone would run, but spends about a third more matrix
        // and softmax work per key (24 of 32 MFMA columns, every wave on every
        // stage): it pays for short key ranges per workgroup and more than 32
        // rows.  Decode steps (one column tile), long ranges and the int8
        // artifact use the kernel whose waves split the keys.
        const int nct = (int)((rows + 31) / 32);
        const int64_t keys_per_wg = p.nsplit > 1 ? p.chunk : n_prefix + n_tok;
        if (append) {            // both kernels store the new rows themselves
            p.kc_app = kc;
            p.vc_app = vc;
            append = false;
        }
        if (qscale || nct == 1 || keys_per_wg > kRowsSplitMaxKeys)
            e = launch_attn_cont(p, nct, qscale != nullptr, f16(d), (int)grid, stream);
        else
            e = launch_attn_rows(p, f16(d), (int)grid, stream);
    } else if (mode == kModePrefill && use_pp(d)) {
        const int64_t pp_tiles = (rows + kRowsPP - 1) / kRowsPP;
        p.tiles_total = (int32_t)pp_tiles;
        e = launch_attn_pp(p, kModePrefill, f16(d), (int)(pp_tiles * p.n_kv_heads), stream);
    } else if (is16(d)) {
        e = launch_attn_bf16(p, d->head_dim, mode, f16(d), (int)grid, stream);
    } else {
        if (mode == kModePrefill && !keys_in_cache) {   // the fp32 kernel does not write the cache itself
            const int st = append_impl(d, K, V, n_tok, kc, vc, 0, stream);
            if (st) return st;
        }
        e = launch_attn_f32(p, d->head_dim, (int)grid, stream);
    }
    if (e != hipSuccess) return KVR_ERR_DEVICE;
    if (append) {                // the other kernels: the cache update as its own launch
        const int st = append_impl(d, K, V, n_tok, kc, vc, n_prefix, stream);
        if (st) return st;
    }
    if (p.nsplit > 1) {
        MergeParams m;
        m.ws = p.ws; m.out = out; m.nsplit = p.nsplit; m.n_q_heads = p.n_q_heads;
        m.n_kv_heads = p.n_kv_heads; m.group = p.group; m.rows = (int32_t)rows;
        e = launch_merge_bf16(m, d->head_dim, f16(d), stream);
        if (e != hipSuccess) return KVR_ERR_DEVICE;
    }
    return KVR_OK;
}


// Validation shared by both batched entry points; *total receives cu[n] and
// *longest the longest reader.  Returns KVR_OK with *total == 0 for no work.
int check_batched(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, const int32_t *cu,
                  int32_t n, const void *kcache, const void *vcache, int64_t L_prefix, void *out,
                  int64_t *total, int64_t *longest) {
    *total = 0;
    *longest = 0;
    int st = check_desc(desc);
    if (st) return st;
    if (n < 0 || L_prefix < 0 || L_prefix > kMaxKeys) return KVR_ERR_SHAPE;
    if (L_prefix > desc->capacity) return KVR_ERR_CAPACITY;
    if (n == 0) return KVR_OK;
    if (!cu) return KVR_ERR_NULL;
    if (cu[0] != 0) return KVR_ERR_SHAPE;
    for (int32_t i = 0; i < n; ++i)
        if (cu[i + 1] < cu[i]) return KVR_ERR_SHAPE;
    if ((int64_t)cu[n] > kMaxTokens) return KVR_ERR_SHAPE;
    const int64_t G = desc->n_q_heads / desc->n_kv_heads;
    for (int32_t i = 0; i < n; ++i) {
        const int64_t len = cu[i + 1] - cu[i];
        if (G * len > 0x7fffffff) return KVR_ERR_SHAPE;
        if (len > *longest) *longest = len;
    }
    // the two-group kernel packs the rows of a launch's readers: row indices
    // of a whole launch group must fit 32 bits there
    if (use_pp(desc))
        for (int32_t first = 0; first < n; first += kMaxSegments) {
            const int32_t last = (n - first) < kMaxSegments ? n : first + kMaxSegments;
            if (G * ((int64_t)cu[last] - cu[first]) > 0x7fffffff) return KVR_ERR_SHAPE;
        }
    if (cu[n] == 0) return KVR_OK;
    if (!Qs || !Ks || !Vs || !out) return KVR_ERR_NULL;
    if (L_prefix > 0 && (!kcache || !vcache)) return KVR_ERR_NULL;
    if (!aligned16(Qs) || !aligned16(Ks) || !aligned16(Vs) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache))
        return KVR_ERR_ALIGN;
    *total = cu[n];
    return KVR_OK;
}

// rope != NULL: the query rows are rotated in registers (Ks already rotated).
// ws: the split partials of plan_readers (unused when it does not split).
int batched_impl(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, const int32_t *cu,
                 int32_t n, const void *kcache, const void *vcache, int64_t L_prefix, void *out,
                 const float *rope, void *ws, void *stream) {
    const int64_t G = desc->n_q_heads / desc->n_kv_heads;
    const bool pp = use_pp(desc);
    const int rpt = pp ? kRowsPP : rows_per_tile(desc);
    for (int32_t first = 0; first < n; first += kMaxSegments) {
        const int32_t cnt = (n - first) < kMaxSegments ? (n - first) : kMaxSegments;
        AttnParams p;
        fill_common(p, desc);
        p.q = Qs; p.kn = Ks; p.vn = Vs; p.kc = kcache; p.vc = vcache; p.out = out;
        p.rope = rope;
        p.n_prefix = L_prefix;
        p.reverse = 0;
        int32_t tiles = 0, seg = 0;
        for (int32_t i = 0; i < cnt; ++i) {
            const int64_t len = cu[first + i + 1] - cu[first + i];
            if (len == 0) continue;   // an empty reader has no rows
            p.seg_tok0[seg] = cu[first + i];
            p.seg_tok0[seg + 1] = cu[first + i + 1];
            p.seg_tile0[seg] = tiles;
            tiles += (int32_t)((G * len + rpt - 1) / rpt);
            ++seg;
        }
        if (seg == 0) continue;
        p.seg_tile0[seg] = tiles;
        p.n_seg = seg;
        p.rows_total = 0;
        hipError_t e;
        if (pp) {
            // packed tiles; one launch (n <= kMaxSegments) may split its last round
            const int64_t n_tok = (int64_t)p.seg_tok0[seg] - p.seg_tok0[0];
            const ReaderPlan rp = n <= kMaxSegments ? plan_readers(desc, L_prefix, n_tok, n)
                                                    : plan_readers(desc, 0, n_tok, 0);
            p.tiles_total = (int32_t)rp.tiles;
            p.tail_tile0 = (int32_t)rp.tail0;
            p.nsplit = (int32_t)rp.nsplit;
            p.rows_total = (int32_t)rp.rows_tail;
            p.ws = (float *)ws;
            const int64_t grid = (rp.tail0 + (rp.tiles - rp.tail0) * rp.nsplit) * p.n_kv_heads;
            e = launch_attn_pp(p, kModeReaders, f16(desc), (int)grid, (hipStream_t)stream);
            if (e == hipSuccess && rp.nsplit > 1) {
                MergeParams mp;
                mp.ws = (const float *)ws;
                mp.out = (unsigned char *)out +
                         ((int64_t)p.seg_tok0[0] + rp.tail0 * kRowsPP / G) * desc->n_q_heads * desc->head_dim *
                             elt_bytes(desc);
                mp.nsplit = (int32_t)rp.nsplit;
                mp.n_q_heads = desc->n_q_heads;
                mp.n_kv_heads = desc->n_kv_heads;
                mp.group = (int32_t)G;
                mp.rows = (int32_t)rp.rows_tail;
                e = launch_merge_bf16(mp, desc->head_dim, f16(desc), (hipStream_t)stream);
            }
        } else {
            p.tiles_total = tiles;
            const int64_t grid = (int64_t)tiles * p.n_kv_heads;
            e = is16(desc) ? launch_attn_bf16(p, desc->head_dim, kModeReaders, f16(desc), (int)grid,
                                              (hipStream_t)stream)
                           : launch_attn_f32(p, desc->head_dim, (int)grid, (hipStream_t)stream);
        }
        if (e != hipSuccess) return KVR_ERR_DEVICE;
    }
    return KVR_OK;
}

// Host and device checks shared by kvr_continue and kvr_continue_noalloc
// (everything but the workspace).
int check_continue(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, const void *kcache,
                   const void *vcache, int64_t L_prefix, int64_t S, void *out) {
    int st = check_desc(desc);
    if (st) return st;
    if (L_prefix < 0 || S < 0 || S > kMaxTokens || L_prefix > kMaxKeys) return KVR_ERR_SHAPE;
    if (L_prefix > desc->capacity) return KVR_ERR_CAPACITY;
    if (S == 0) return KVR_OK;
    if (!Qs || !Ks || !Vs || !out) return KVR_ERR_NULL;
    if (L_prefix > 0 && (!kcache || !vcache)) return KVR_ERR_NULL;
    if (!aligned16(Qs) || !aligned16(Ks) || !aligned16(Vs) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache))
        return KVR_ERR_ALIGN;
    return KVR_OK;
}

}  // namespace
}  // namespace kvr

// The split partials of kvr_continue_noalloc: a fixed buffer, one copy per
// device, held until the process ends.  Host code uses the device address
// that hipGetSymbolAddress returns for the current device, never this name
// (on the host it only stands in for the symbol).
static __device__ __align__(256) unsigned char scratch[KVR_NOALLOC_SCRATCH_BYTES];

namespace kvr {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];

// Device address of `scratch` on device dev, looked up once per device with
// that device current (the caller's current device is restored).
int scratch_on(int dev, void **ptr) {
    if (dev < 0 || dev >= kMaxDevices) return KVR_ERR_DEVICE;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        int cur = -1;
        if (hipGetDevice(&cur) != hipSuccess) return KVR_ERR_DEVICE;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return KVR_ERR_DEVICE;
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (cur != dev && hipSetDevice(cur) != hipSuccess) return KVR_ERR_DEVICE;
        if (e != hipSuccess || !p) return KVR_ERR_DEVICE;
        g_scratch[dev] = p;
    }
    *ptr = g_scratch[dev];
    return KVR_OK;
}

// the device a stream belongs to (the current device for the null stream)
int stream_device(hipStream_t stream, int *dev) {
    if (!stream) return hipGetDevice(dev) == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
    hipDevice_t d;
    if (hipStreamGetDevice(stream, &d) != hipSuccess) return KVR_ERR_DEVICE;
    *dev = (int)d;
    return KVR_OK;
}

}  // namespace
}  // namespace kvr

using namespace kvr;

extern "C" {

int kvr_abi_version(void) { return KVR_ABI_VERSION; }

const char *kvr_strerror(int status) {
    switch (status) {
        case KVR_OK: return "ok";
        case KVR_ERR_NULL: return "a required pointer is NULL";
        case KVR_ERR_SHAPE: return "invalid heads, head_dim, length or cu_seqlens";
        case KVR_ERR_DTYPE: return "unsupported element type";
        case KVR_ERR_CAPACITY: return "cache rows exceed the descriptor's capacity";
        case KVR_ERR_WORKSPACE: return "workspace smaller than kvr_workspace_bytes()";
        case KVR_ERR_ALIGN: return "device pointer not 16-byte aligned";
        case KVR_ERR_DEVICE: return "HIP call or kernel launch failed";
        case KVR_ERR_MISMATCH: return "artifact metadata does not match the running model (model id, dtype or shape)";
        case KVR_ERR_POSITION: return "RoPE table lacks a position the call rotates, or invalid table arguments";
        case KVR_ERR_TOO_LARGE: return "the call needs more than the no-allocation entry point's fixed scratch buffer";
        default: return "unknown kvr status";
    }
}

size_t kvr_workspace_bytes(const kvr_desc *desc, int64_t L_prefix, int64_t total_S, int32_t n) {
    if (check_desc(desc) != KVR_OK || L_prefix < 0 || total_S < 0 || n < 0) return (size_t)-1;
    if (n >= 2) return plan_readers(desc, L_prefix, total_S, n).ws_bytes;   // many readers
    return plan_split(desc, L_prefix, total_S).ws_bytes;
}

int kvr_prefill(const kvr_desc *desc, const void *Q, const void *K, const void *V, int64_t L, void *out,
                void *kcache, void *vcache, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (L < 0 || L > kMaxTokens) return KVR_ERR_SHAPE;
    if (L > desc->capacity) return KVR_ERR_CAPACITY;
    if (L == 0) return KVR_OK;
    if (!Q || !K || !V || !out || !kcache || !vcache) return KVR_ERR_NULL;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache))
        return KVR_ERR_ALIGN;
    Split none{1, 0, 0};
    return launch_single(desc, kModePrefill, Q, K, V, kcache, vcache, 0, L, out, none, nullptr,
                         (hipStream_t)stream);
}

int kvr_continue(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, const void *kcache,
                 const void *vcache, int64_t L_prefix, int64_t S, void *out, void *ws, size_t ws_bytes,
                 void *stream) {
    int st = check_continue(desc, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out);
    if (st || S == 0) return st;
    const Split sp = plan_split(desc, L_prefix, S);
    if (ws_bytes < sp.ws_bytes) return KVR_ERR_WORKSPACE;
    if (sp.ws_bytes > 0 && !ws) return KVR_ERR_NULL;
    if (!aligned16(ws)) return KVR_ERR_ALIGN;
    return launch_single(desc, kModeContinue, Qs, Ks, Vs, (void *)kcache, (void *)vcache, L_prefix, S, out,
                         sp, ws, (hipStream_t)stream);
}

int kvr_continue_noalloc(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                         const void *kcache, const void *vcache, int64_t L_prefix, int64_t S, void *out,
                         void *stream) {
    int st = check_continue(desc, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out);
    if (st || S == 0) return st;
    const Split sp = plan_split(desc, L_prefix, S);
    if (sp.ws_bytes > KVR_NOALLOC_SCRATCH_BYTES) return KVR_ERR_TOO_LARGE;
    void *ws = nullptr;
    if (sp.ws_bytes > 0) {
        int dev = -1;
        st = stream_device((hipStream_t)stream, &dev);
        if (st) return st;
        st = scratch_on(dev, &ws);
        if (st) return st;
    }
    return launch_single(desc, kModeContinue, Qs, Ks, Vs, (void *)kcache, (void *)vcache, L_prefix, S, out,
                         sp, ws, (hipStream_t)stream);
}

int kvr_continue_append(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, void *kcache,
                        void *vcache, int64_t L_prefix, int64_t S, void *out, void *ws, size_t ws_bytes,
                        void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (L_prefix < 0 || S < 0 || S > kMaxTokens || L_prefix > kMaxKeys) return KVR_ERR_SHAPE;
    if (L_prefix + S > desc->capacity) return KVR_ERR_CAPACITY;
    if (S == 0) return KVR_OK;
    if (!Qs || !Ks || !Vs || !out || !kcache || !vcache) return KVR_ERR_NULL;
    const Split sp = plan_split(desc, L_prefix, S);
    if (ws_bytes < sp.ws_bytes) return KVR_ERR_WORKSPACE;
    if (sp.ws_bytes > 0 && !ws) return KVR_ERR_NULL;
    if (!aligned16(Qs) || !aligned16(Ks) || !aligned16(Vs) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache) || !aligned16(ws))
        return KVR_ERR_ALIGN;
    return launch_single(desc, kModeContinue, Qs, Ks, Vs, kcache, vcache, L_prefix, S, out, sp, ws,
                         (hipStream_t)stream, nullptr, nullptr, true);
}

size_t kvr_q8_bytes(const kvr_desc *desc) {
    if (check_desc(desc) != KVR_OK) return (size_t)-1;
    const int64_t padded = (desc->capacity + 31) / 32 * 32;
    return (size_t)desc->n_kv_heads * (size_t)padded * (size_t)desc->head_dim;
}

int kvr_quantize_cache(const kvr_desc *desc, const void *kcache, const void *vcache, int64_t L, void *kq,
                       void *vq, float *scales, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (desc->dtype != KVR_BF16) return KVR_ERR_DTYPE;
    if (desc->head_dim != 128) return KVR_ERR_SHAPE;
    if (L < 0 || L > kMaxKeys) return KVR_ERR_SHAPE;
    if (L > desc->capacity) return KVR_ERR_CAPACITY;
    if (L == 0) return KVR_OK;
    if (!kcache || !vcache || !kq || !vq || !scales) return KVR_ERR_NULL;
    if (!aligned16(kcache) || !aligned16(vcache) || !aligned16(kq) || !aligned16(vq) || ((uintptr_t)scales & 3u))
        return KVR_ERR_ALIGN;
    QuantParams q;
    q.kc = kcache; q.vc = vcache; q.kq = kq; q.vq = vq; q.scales = scales;
    q.L = L; q.cap = desc->capacity; q.padded = (desc->capacity + 31) / 32 * 32;
    q.n_kv_heads = desc->n_kv_heads;
    return launch_quantize(q, (hipStream_t)stream) == hipSuccess ? KVR_OK : KVR_ERR_DEVICE;
}

int kvr_continue_q8(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs, const void *kq,
                    const void *vq, const float *scales, int64_t L_prefix, int64_t S, void *out, void *ws,
                    size_t ws_bytes, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (desc->dtype != KVR_BF16) return KVR_ERR_DTYPE;
    if (L_prefix < 0 || S < 0 || S > kMaxTokens || L_prefix > kMaxKeys) return KVR_ERR_SHAPE;
    if (desc->head_dim != 128 || !use_cont(desc, S)) return KVR_ERR_SHAPE;
    if (L_prefix > desc->capacity) return KVR_ERR_CAPACITY;
    if (S == 0) return KVR_OK;
    if (!Qs || !Ks || !Vs || !out) return KVR_ERR_NULL;
    if (L_prefix > 0 && (!kq || !vq || !scales)) return KVR_ERR_NULL;
    const Split sp = plan_split(desc, L_prefix, S);
    if (ws_bytes < sp.ws_bytes) return KVR_ERR_WORKSPACE;
    if (sp.ws_bytes > 0 && !ws) return KVR_ERR_NULL;
    if (!aligned16(Qs) || !aligned16(Ks) || !aligned16(Vs) || !aligned16(out) || !aligned16(kq) ||
        !aligned16(vq) || !aligned16(ws) || ((uintptr_t)scales & 3u))
        return KVR_ERR_ALIGN;
    // without a prefix there is nothing quantized: a plain continuation
    if (L_prefix == 0)
        return launch_single(desc, kModeContinue, Qs, Ks, Vs, nullptr, nullptr, 0, S, out, sp, ws,
                             (hipStream_t)stream);
    return launch_single(desc, kModeContinue, Qs, Ks, Vs, (void *)kq, (void *)vq, L_prefix, S, out, sp, ws,
                         (hipStream_t)stream, scales);
}

int kvr_continue_batched(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                         const int32_t *cu, int32_t n, const void *kcache, const void *vcache,
                         int64_t L_prefix, void *out, void *ws, size_t ws_bytes, void *stream) {
    int64_t total, longest;
    const int st = check_batched(desc, Qs, Ks, Vs, cu, n, kcache, vcache, L_prefix, out, &total, &longest);
    if (st || total == 0) return st;
    const size_t need = plan_readers(desc, L_prefix, total, n).ws_bytes;
    if (ws_bytes < need) return KVR_ERR_WORKSPACE;
    if (need > 0 && !ws) return KVR_ERR_NULL;
    if (!aligned16(ws)) return KVR_ERR_ALIGN;
    return batched_impl(desc, Qs, Ks, Vs, cu, n, kcache, vcache, L_prefix, out, nullptr, ws, stream);
}

int kvr_cache_append(const kvr_desc *desc, const void *Ks, const void *Vs, int64_t S, void *kcache,
                     void *vcache, int64_t L_cur, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (S < 0 || L_cur < 0 || S > kMaxTokens || L_cur > kMaxKeys) return KVR_ERR_SHAPE;
    if (L_cur + S > desc->capacity) return KVR_ERR_CAPACITY;
    if (S == 0) return KVR_OK;
    if (!Ks || !Vs || !kcache || !vcache) return KVR_ERR_NULL;
    if (!aligned16(Ks) || !aligned16(Vs) || !aligned16(kcache) || !aligned16(vcache)) return KVR_ERR_ALIGN;
    return append_impl(desc, Ks, Vs, S, kcache, vcache, L_cur, (hipStream_t)stream);
}

int kvr_rope_table(int32_t head_dim, double base, int64_t n_pos, float *cos_sin, void *stream) {
    if (head_dim != 64 && head_dim != 128) return KVR_ERR_SHAPE;
    if (!(base > 0.0) || isinf(base) || n_pos < 0 || n_pos > kMaxKeys) return KVR_ERR_POSITION;
    if (n_pos == 0) return KVR_OK;
    if (!cos_sin) return KVR_ERR_NULL;
    if (!aligned16(cos_sin)) return KVR_ERR_ALIGN;
    return to_status(launch_rope_table(cos_sin, head_dim, base, n_pos, (hipStream_t)stream));
}

int kvr_rope_apply(const kvr_desc *desc, const kvr_rope *rope, const void *x, int64_t n_tok, int32_t n_heads,
                   int64_t pos0, void *y, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (n_tok < 0 || n_tok > kMaxTokens || n_heads <= 0 || n_heads > 4096) return KVR_ERR_SHAPE;
    if (pos0 < 0 || pos0 > kMaxKeys) return KVR_ERR_POSITION;
    if (n_tok == 0) return KVR_OK;
    if (!x || !y) return KVR_ERR_NULL;
    if ((st = check_rope(rope, pos0 + n_tok))) return st;
    if (!aligned16(x) || !aligned16(y)) return KVR_ERR_ALIGN;
    RopeParams rp = rope_params(desc, rope, n_tok, pos0);
    rp.n_jobs = 1;
    rp.job[0].x = x;
    rp.job[0].y = y;
    rp.job[0].n_heads = n_heads;
    return to_status(launch_rope(rp, desc->head_dim, desc->dtype, (hipStream_t)stream));
}

int kvr_prefill_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Q, const void *K, const void *V,
                     int64_t L, void *out, void *kcache, void *vcache, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (L < 0 || L > kMaxTokens) return KVR_ERR_SHAPE;
    if (L > desc->capacity) return KVR_ERR_CAPACITY;
    if (L == 0) return KVR_OK;
    if (!Q || !K || !V || !out || !kcache || !vcache) return KVR_ERR_NULL;
    if ((st = check_rope(rope, L))) return st;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache))
        return KVR_ERR_ALIGN;
    // rotated keys and the values into cache rows [0, L), then attention over them
    RopeParams rp = rope_params(desc, rope, L, 0);
    rp.n_jobs = 1;
    rp.job[0].x = K;
    rp.job[0].cache = kcache;
    rp.job[0].v = V;
    rp.job[0].vcache = vcache;
    rp.job[0].n_heads = desc->n_kv_heads;
    if (launch_rope(rp, desc->head_dim, desc->dtype, (hipStream_t)stream) != hipSuccess) return KVR_ERR_DEVICE;
    Split none{1, 0, 0};
    return launch_single(desc, kModePrefill, Q, nullptr, nullptr, kcache, vcache, 0, L, out, none, nullptr,
                         (hipStream_t)stream, nullptr, rope->cos_sin);
}

size_t kvr_workspace_bytes_rope(const kvr_desc *desc, int64_t L_prefix, int64_t total_S, int32_t n) {
    if (check_desc(desc) != KVR_OK || L_prefix < 0 || total_S < 0 || n < 0) return (size_t)-1;
    return rope_ws(desc, L_prefix, total_S, n).total;
}

int kvr_continue_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Qs, const void *Ks, const void *Vs,
                      void *kcache, void *vcache, int64_t L_prefix, int64_t S, int32_t append, void *out, void *ws,
                      size_t ws_bytes, void *stream) {
    int st = check_desc(desc);
    if (st) return st;
    if (L_prefix < 0 || S < 0 || S > kMaxTokens || L_prefix > kMaxKeys) return KVR_ERR_SHAPE;
    if (L_prefix > desc->capacity) return KVR_ERR_CAPACITY;
    if (append && L_prefix + S > desc->capacity) return KVR_ERR_CAPACITY;
    if (S == 0) return KVR_OK;
    if (!Qs || !Ks || !Vs || !out || !ws) return KVR_ERR_NULL;
    if ((L_prefix > 0 || append) && (!kcache || !vcache)) return KVR_ERR_NULL;
    if ((st = check_rope(rope, L_prefix + S))) return st;
    const RopeWs w = rope_ws(desc, L_prefix, S, 1);
    if (ws_bytes < w.total) return KVR_ERR_WORKSPACE;
    if (!aligned16(Qs) || !aligned16(Ks) || !aligned16(Vs) || !aligned16(out) || !aligned16(kcache) ||
        !aligned16(vcache) || !aligned16(ws))
        return KVR_ERR_ALIGN;
    unsigned char *wsb = (unsigned char *)ws;
    // the rows at positions L_prefix..: queries and keys rotated into the
    // workspace, and with append the rotated keys and the values into the cache
    RopeParams rp = rope_params(desc, rope, S, L_prefix);
    rp.n_jobs = 2;
    rp.job[0].x = Qs;
    rp.job[0].y = wsb + w.q_off;
    rp.job[0].n_heads = desc->n_q_heads;
    rp.job[1].x = Ks;
    rp.job[1].y = wsb + w.k_off;
    rp.job[1].n_heads = desc->n_kv_heads;
    if (append) {
        rp.job[1].cache = kcache;
        rp.job[1].v = Vs;
        rp.job[1].vcache = vcache;
    }
    if (launch_rope(rp, desc->head_dim, desc->dtype, (hipStream_t)stream) != hipSuccess) return KVR_ERR_DEVICE;
    const Split sp = plan_split(desc, L_prefix, S);
    return launch_single(desc, kModeContinue, wsb + w.q_off, wsb + w.k_off, Vs, kcache, vcache, L_prefix, S, out,
                         sp, ws, (hipStream_t)stream);
}

int kvr_continue_batched_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Qs, const void *Ks,
                              const void *Vs, const int32_t *cu, int32_t n, const void *kcache, const void *vcache,
                              int64_t L_prefix, void *out, void *ws, size_t ws_bytes, void *stream) {
    int64_t total, longest;
    int st = check_batched(desc, Qs, Ks, Vs, cu, n, kcache, vcache, L_prefix, out, &total, &longest);
    if (st || total == 0) return st;
    if ((st = check_rope(rope, L_prefix + longest))) return st;
    const RopeWs w = rope_ws(desc, L_prefix, total, n < 2 ? 2 : n);
    if (!ws) return KVR_ERR_NULL;
    if (ws_bytes < w.total) return KVR_ERR_WORKSPACE;
    if (!aligned16(ws)) return KVR_ERR_ALIGN;
    // each reader's keys rotated at L_prefix + (row within the reader), in
    // groups of at most kMaxSegments readers (the pre-pass's segment table)
    const size_t row_b = (size_t)desc->n_kv_heads * desc->head_dim * elt_bytes(desc);
    unsigned char *kr = (unsigned char *)ws + w.k_off;
    for (int32_t first = 0; first < n; first += kMaxSegments) {
        const int32_t cnt = (n - first) < kMaxSegments ? (n - first) : kMaxSegments;
        const int64_t t0 = cu[first];
        const int64_t nt = cu[first + cnt] - t0;
        if (nt == 0) continue;
        RopeParams rp = rope_params(desc, rope, nt, L_prefix);
        rp.n_seg = cnt;
        for (int32_t i = 0; i <= cnt; ++i) rp.seg_tok0[i] = (int32_t)(cu[first + i] - t0);
        rp.n_jobs = 1;
        rp.job[0].x = (const unsigned char *)Ks + (size_t)t0 * row_b;
        rp.job[0].y = kr + (size_t)t0 * row_b;
        rp.job[0].n_heads = desc->n_kv_heads;
        if (launch_rope(rp, desc->head_dim, desc->dtype, (hipStream_t)stream) != hipSuccess) return KVR_ERR_DEVICE;
    }
    return batched_impl(desc, Qs, kr, Vs, cu, n, kcache, vcache, L_prefix, out, rope->cos_sin, ws, stream);
}

}  // extern "C"
