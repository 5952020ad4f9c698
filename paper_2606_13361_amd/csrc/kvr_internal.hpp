// kvr_internal.hpp -- launch parameters shared by the host entry points and
// the gfx950 kernels of libkvr.  Not part of the public ABI (include/kvr.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvr {

// Readers handled by one launch of the attention kernel; kvr_continue_batched
// issues one launch per group of this many readers.
constexpr int kMaxSegments = 128;

// Query rows are (token, head) pairs packed token-major: for kv head g with
// group size G, row r of a segment is token r / G, query head g*G + r % G.
// That keeps every row of a workgroup on the same K/V rows.
struct AttnParams {
    const void *q;   // [tokens][n_q_heads][D]
    const void *kn;  // new keys   [tokens][n_kv_heads][D]
    const void *vn;  // new values [tokens][n_kv_heads][D]
    const void *kc;  // cached keys   [n_kv_heads][cap][D]
    const void *vc;  // cached values [n_kv_heads][cap][D]
    void *out;       // [tokens][n_q_heads][D]
    void *kc_out;    // prefill: cache the new K rows go to [n_kv_heads][cap][D]
    void *vc_out;
    float *ws;       // split partials: O [nsplit][Hkv][rows][D], then (m, l) [nsplit][Hkv][rows][2]
    const float *qscale;   // int8 artifact continuation: {s_K, s_V} (kc/vc then point at the codes)
    // RoPE table [pos][D/2] of (cos, sin), or null.  Set for prefill and many
    // readers only: those kernels rotate each query row in registers at its
    // position n_prefix + token (continuations get their rows rotated by the
    // pre-pass instead).
    const float *rope;
    // Element strides of kn/vn: token and kv head.  Token-major new rows have
    // (n_kv_heads * D, D); prefill with RoPE reads its rotated rows back from
    // the cache, (D, cap * D).  Honoured by the prefill / readers kernels.
    int64_t new_tok_stride, new_head_stride;
    // Continuation with the cache update: the workgroup that reads the new
    // rows of a kv head last (the last split) also stores them into rows
    // [n_prefix, n_prefix + S) of these caches; null: no update.  Honoured by
    // the keys-split and row-split continuation kernels.
    void *kc_app, *vc_app;
    int64_t cap;
    int64_t n_prefix;  // cached keys, positions [0, n_prefix); every query row sees them all
    int64_t chunk;     // prefix keys per split, a multiple of the key tile
    int32_t n_q_heads, n_kv_heads, group;
    int32_t nsplit;
    float scale;        // softmax scale
    float scale_log2;   // scale * log2(e)
    int32_t n_seg;      // segments (independent readers); 1 for prefill / continue
    int32_t reverse;    // fp32 path: visit row tiles last-first (longest causal rows first)
    int32_t tiles_total;
    int32_t rows_total;  // rows per kv head of the split partials (from the first split row)
    // many readers on the two-group kernel: row tiles from this one on run as
    // nsplit key splits each (tiles_total: none)
    int32_t tail_tile0;
    int32_t seg_tok0[kMaxSegments + 1];   // packed token offset of each segment (cu_seqlens)
    int32_t seg_tile0[kMaxSegments + 1];  // first row tile of each segment (prefix sums; not used
                                          // by the two-group kernel, whose reader tiles are packed)
};

struct AppendParams {
    const void *k;  // [S][n_kv_heads][D]
    const void *v;
    void *kc;       // [n_kv_heads][cap][D]
    void *vc;
    int64_t S, L_cur, cap;
    int32_t n_kv_heads;
    int32_t row_chunks;  // 16-byte chunks per row (D * elt / 16)
};

// Quantization of cache rows [0, L) into the int8 artifact (layouts in kvr.h)
struct QuantParams {
    const void *kc;   // bf16 [n_kv_heads][cap][128]
    const void *vc;
    void *kq;         // int8 artifact, padded rows per head
    void *vq;
    float *scales;    // [2]: maxima while the kernels run, then {s_K, s_V}
    int64_t L, cap, padded;
    int32_t n_kv_heads;
};

struct MergeParams {
    const float *ws;
    void *out;
    int32_t nsplit, n_q_heads, n_kv_heads, group, rows;
};

enum { kModePrefill = 0, kModeContinue = 1, kModeReaders = 2 };

// bf16 path (MFMA), D in {64, 128}
// (the 16-bit MFMA path: f16 selects fp16 elements, else bf16)
hipError_t launch_attn_bf16(const AttnParams &p, int head_dim, int mode, bool f16, int grid, hipStream_t s);
hipError_t launch_merge_bf16(const MergeParams &p, int head_dim, bool f16, hipStream_t s);
// bf16 prefill and many readers at D = 128: two groups of 4 waves alternate
// matrix and softmax steps
constexpr int kRowsPP = 256;   // query rows per workgroup (8 waves x 32)
hipError_t launch_attn_pp(const AttnParams &p, int mode, bool f16, int grid, hipStream_t s);
// bf16 continuation for G*S <= 96 rows (D = 128).  33..96 rows: the waves of
// a workgroup split the rows and share one ring of key stages; up to 32 rows
// (decode steps) and the int8 artifact: the waves split the keys
constexpr int kContMaxRows = 96;
hipError_t launch_attn_rows(const AttnParams &p, bool f16, int grid, hipStream_t s);
hipError_t launch_attn_cont(const AttnParams &p, int ncol_tiles, bool q8, bool f16, int grid, hipStream_t s);
// int8 artifact
hipError_t launch_quantize(const QuantParams &p, hipStream_t s);
// fp32 path (VALU), D in {64, 128}
hipError_t launch_attn_f32(const AttnParams &p, int head_dim, int grid, hipStream_t s);
// cache write
hipError_t launch_append(const AppendParams &p, hipStream_t s);

// RoPE pre-pass: rotate token-major rows [n_tok][n_heads][D] at their
// positions into token-major rows (y) and/or cache rows (cache, row = the
// position), and copy value rows into a cache unchanged.
struct RopeJob {
    const void *x;       // rows to rotate, [n_tok][n_heads][D]
    void *y;             // rotated rows, token-major (may equal x), or null
    void *cache;         // rotated rows into [n_heads][cap][D] at row = position, or null
    const void *v;       // rows copied unrotated into vcache at row = position, or null
    void *vcache;
    int32_t n_heads;
};
struct RopeParams {
    RopeJob job[2];
    const float *cs;     // [n_pos][D/2] (cos, sin)
    int64_t n_tok, cap;
    int64_t pos0;        // token t of segment s sits at pos0 + t - seg_tok0[s]
    int32_t n_jobs;
    int32_t n_seg;
    int32_t seg_tok0[kMaxSegments + 1];
};
// elt: 0 bf16, 1 fp32, 2 fp16 (kvr_dtype)
hipError_t launch_rope(const RopeParams &p, int head_dim, int elt, hipStream_t s);
hipError_t launch_rope_table(float *cs, int head_dim, double base, int64_t n_pos, hipStream_t s);

// row-tile geometry of the two paths
constexpr int kRowsBf16 = 128;  // query rows per workgroup, bf16 path
constexpr int kRowsF32 = 64;    // query rows per workgroup, fp32 path
constexpr int kKeyTile = 64;    // keys per tile (split chunks are multiples of it)
constexpr int kMaxSplits = 256; // key splits of one continuation (merge kernel LDS table)

}  // namespace kvr
