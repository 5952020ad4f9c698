// Drives the host side of libkvr (kvr_api.hip, artifact.hip: argument
// validation, split planning, workspace layouts, artifact headers) under
// AddressSanitizer and UndefinedBehaviorSanitizer, without a GPU.  The kernel
// launchers are replaced by stubs that count their calls and fail, so a call
// with valid arguments ends in KVR_ERR_DEVICE without touching a device; a
// rejected call must reach no launcher at all.  Device pointers are fake
// aligned integers and are never dereferenced on the host.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "kvr.h"
#include "kvr_internal.hpp"

static int g_launches = 0;
static int64_t g_nsplit = -1, g_chunk = -1;   // the split plan the last continuation launch got
static int g_pp_bad = 0;                       // many-readers launches whose plan broke an invariant
static int g_pp_split = 0, g_pp_whole = 0;     // many-readers launches checked: split last round or not
static int64_t g_pp_grid = -1, g_pp_tail0 = -1, g_pp_rows = -1;

namespace kvr {
hipError_t launch_attn_bf16(const AttnParams &, int, int, bool, int, hipStream_t) { ++g_launches; return hipErrorUnknown; }
hipError_t launch_merge_bf16(const MergeParams &, int, bool, hipStream_t) { ++g_launches; return hipErrorUnknown; }
// many readers on the two-group kernel: the packed plan must cover its tiles
// with whole workgroups (split tiles ns times), and split partial rows must
// number the rows from the first split tile to the end of the launch
hipError_t launch_attn_pp(const AttnParams &p, int mode, bool, int grid, hipStream_t) {
    ++g_launches;
    if (mode == kModeReaders) {
        const int64_t ns = p.nsplit, tiles = p.tiles_total, t0 = p.tail_tile0;
        const int64_t rows = (int64_t)p.group * ((int64_t)p.seg_tok0[p.n_seg] - p.seg_tok0[0]);
        bool ok = ns >= 1 && ns <= 16 && t0 >= 0 && t0 <= tiles && tiles == (rows + kRowsPP - 1) / kRowsPP &&
                  (int64_t)grid == (t0 + (tiles - t0) * ns) * p.n_kv_heads;
        if (ns > 1) ok = ok && t0 < tiles && p.ws && p.rows_total == rows - t0 * kRowsPP && kRowsPP % p.group == 0;
        else ok = ok && t0 == tiles;
        if (!ok) ++g_pp_bad;
        ++(ns > 1 ? g_pp_split : g_pp_whole);
        g_pp_grid = grid; g_pp_tail0 = t0; g_pp_rows = p.rows_total;
    }
    return hipErrorUnknown;
}
hipError_t launch_attn_rows(const AttnParams &p, bool, int, hipStream_t) {
    ++g_launches; g_nsplit = p.nsplit; g_chunk = p.chunk; return hipErrorUnknown;
}
hipError_t launch_attn_cont(const AttnParams &p, int, bool, bool, int, hipStream_t) {
    ++g_launches; g_nsplit = p.nsplit; g_chunk = p.chunk; return hipErrorUnknown;
}
hipError_t launch_quantize(const QuantParams &, hipStream_t) { ++g_launches; return hipErrorUnknown; }
hipError_t launch_attn_f32(const AttnParams &, int, int, hipStream_t) { ++g_launches; return hipErrorUnknown; }
hipError_t launch_append(const AppendParams &, hipStream_t) { ++g_launches; return hipErrorUnknown; }
hipError_t launch_rope(const RopeParams &, int, int, hipStream_t) { ++g_launches; return hipErrorUnknown; }
hipError_t launch_rope_table(float *, int, double, int64_t, hipStream_t) { ++g_launches; return hipErrorUnknown; }
}  // namespace kvr

static void *const A = (void *)(uintptr_t)0x10000;    // 16-byte aligned fake device pointer
static void *const MIS = (void *)(uintptr_t)0x10008;  // 8-byte aligned only
static const float *const AF = (const float *)A;
static int fails = 0;

#define EXPECT(expr, want)                                                                              \
    do {                                                                                                \
        const int before_ = g_launches;                                                                 \
        const int got_ = (int)(expr);                                                                   \
        if (got_ != (want)) {                                                                           \
            fprintf(stderr, "line %d: %s = %d, want %d\n", __LINE__, #expr, got_, (int)(want));       \
            ++fails;                                                                                    \
        }                                                                                               \
        if ((want) != KVR_OK && (want) != KVR_ERR_DEVICE && g_launches != before_) {                    \
            fprintf(stderr, "line %d: %s launched after a rejection\n", __LINE__, #expr);              \
            ++fails;                                                                                    \
        }                                                                                               \
    } while (0)

static kvr_desc desc(int hq = 32, int hkv = 8, int d = 128, int dt = KVR_BF16, int64_t cap = 4096) {
    kvr_desc x;
    memset(&x, 0, sizeof x);
    x.n_q_heads = hq; x.n_kv_heads = hkv; x.head_dim = d; x.dtype = dt; x.capacity = cap; x.scale = 0.f;
    return x;
}

static uint64_t rng = 0x2545f4914f6cdd1dull;
static uint64_t next() { rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17; return rng; }
static int64_t pick(const int64_t *v, int n) { return v[next() % (uint64_t)n]; }

static void fixed_cases() {
    kvr_desc d = desc();
    const size_t big = (size_t)1 << 40;
    // descriptors
    EXPECT(kvr_prefill(nullptr, A, A, A, 4, A, A, A, nullptr), KVR_ERR_NULL);
    kvr_desc bad = desc(); bad.dtype = 7;
    EXPECT(kvr_prefill(&bad, A, A, A, 4, A, A, A, nullptr), KVR_ERR_DTYPE);
    bad = desc(); bad.n_q_heads = 30;
    EXPECT(kvr_continue(&bad, A, A, A, A, A, 8, 4, A, A, big, nullptr), KVR_ERR_SHAPE);
    bad = desc(); bad.head_dim = 96;
    EXPECT(kvr_cache_append(&bad, A, A, 4, A, A, 0, nullptr), KVR_ERR_SHAPE);
    bad = desc(); bad.reserved = 1;
    EXPECT(kvr_prefill(&bad, A, A, A, 4, A, A, A, nullptr), KVR_ERR_SHAPE);
    bad = desc(); bad.scale = NAN;
    EXPECT(kvr_prefill(&bad, A, A, A, 4, A, A, A, nullptr), KVR_ERR_SHAPE);
    bad = desc(); bad.capacity = -1;
    EXPECT(kvr_prefill(&bad, A, A, A, 4, A, A, A, nullptr), KVR_ERR_SHAPE);
    // lengths, capacity, pointers, alignment
    EXPECT(kvr_prefill(&d, A, A, A, -1, A, A, A, nullptr), KVR_ERR_SHAPE);
    EXPECT(kvr_prefill(&d, A, A, A, 4097, A, A, A, nullptr), KVR_ERR_CAPACITY);
    EXPECT(kvr_prefill(&d, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr, nullptr), KVR_OK);
    EXPECT(kvr_prefill(&d, MIS, A, A, 4, A, A, A, nullptr), KVR_ERR_ALIGN);
    EXPECT(kvr_prefill(&d, A, A, A, 4, A, nullptr, A, nullptr), KVR_ERR_NULL);
    EXPECT(kvr_continue(&d, A, A, A, A, A, -1, 4, A, A, big, nullptr), KVR_ERR_SHAPE);
    EXPECT(kvr_continue(&d, A, A, A, A, A, 4097, 4, A, A, big, nullptr), KVR_ERR_CAPACITY);
    EXPECT(kvr_continue(&d, nullptr, nullptr, nullptr, A, A, 8, 0, nullptr, nullptr, 0, nullptr), KVR_OK);
    const size_t need = kvr_workspace_bytes(&d, 4096, 24, 1);
    EXPECT(need > 0, 1);
    EXPECT(kvr_continue(&d, A, A, A, A, A, 4096, 24, A, A, need - 1, nullptr), KVR_ERR_WORKSPACE);
    EXPECT(kvr_continue(&d, A, A, A, A, A, 4096, 24, A, nullptr, need, nullptr), KVR_ERR_NULL);
    EXPECT(kvr_continue(&d, A, A, A, A, A, 4096, 24, A, MIS, need, nullptr), KVR_ERR_ALIGN);
    EXPECT(kvr_continue(&d, A, A, A, A, A, 4096, 24, A, A, need, nullptr), KVR_ERR_DEVICE);   // reaches a stub
    EXPECT(kvr_continue_append(&d, A, A, A, A, A, 4090, 24, A, A, big, nullptr), KVR_ERR_CAPACITY);
    EXPECT(kvr_cache_append(&d, A, A, 10, A, A, 4090, nullptr), KVR_ERR_CAPACITY);
    EXPECT(kvr_cache_append(&d, A, A, -1, A, A, 0, nullptr), KVR_ERR_SHAPE);
    // readers: cu_seqlens checks
    const int32_t cu_ok[4] = {0, 5, 5, 12}, cu_dec[3] = {0, 7, 3}, cu_first[3] = {2, 4, 6};
    EXPECT(kvr_continue_batched(&d, A, A, A, cu_dec, 2, A, A, 100, A, A, big, nullptr), KVR_ERR_SHAPE);
    EXPECT(kvr_continue_batched(&d, A, A, A, cu_first, 2, A, A, 100, A, A, big, nullptr), KVR_ERR_SHAPE);
    EXPECT(kvr_continue_batched(&d, A, A, A, nullptr, 3, A, A, 100, A, A, big, nullptr), KVR_ERR_NULL);
    EXPECT(kvr_continue_batched(&d, A, A, A, cu_ok, 3, A, A, 5000, A, A, big, nullptr), KVR_ERR_CAPACITY);
    EXPECT(kvr_continue_batched(&d, A, A, A, cu_ok, 3, A, A, 100, A, A, big, nullptr), KVR_ERR_DEVICE);
    {
        // 64 readers, 8424 tokens over 3774: 132 tiles per kv head, the last 4 split 8 ways
        std::vector<int32_t> cu64(65, 0);
        const int step[4] = {120, 140, 131, 135};
        for (int i = 1; i <= 64; ++i) cu64[i] = cu64[i - 1] + step[i % 4];
        cu64[64] = 8424;
        kvr_desc dr = desc(32, 8, 128, KVR_BF16, 4096);
        const size_t wsr = kvr_workspace_bytes(&dr, 3774, 8424, 64);
        EXPECT(wsr == (size_t)8 * 8 * 928 * 130 * 4, 1);
        EXPECT(kvr_continue_batched(&dr, A, A, A, cu64.data(), 64, A, A, 3774, A, A, wsr - 1, nullptr),
               KVR_ERR_WORKSPACE);
        EXPECT(kvr_continue_batched(&dr, A, A, A, cu64.data(), 64, A, A, 3774, A, A, wsr, nullptr), KVR_ERR_DEVICE);
        EXPECT(g_pp_grid == (128 + 4 * 8) * 8 * 1 && g_pp_tail0 == 128 && g_pp_rows == 928, 1);
    }
    // int8 artifact
    kvr_desc f32 = desc(32, 8, 128, KVR_F32);
    EXPECT(kvr_quantize_cache(&f32, A, A, 10, A, A, (float *)A, nullptr), KVR_ERR_DTYPE);
    EXPECT(kvr_continue_q8(&d, A, A, A, A, A, nullptr, 100, 4, A, A, big, nullptr), KVR_ERR_NULL);
    // RoPE
    kvr_rope r;
    r.cos_sin = AF; r.n_pos = 64;
    EXPECT(kvr_rope_table(96, 1e6, 10, (float *)A, nullptr), KVR_ERR_SHAPE);
    EXPECT(kvr_rope_table(128, -1.0, 10, (float *)A, nullptr), KVR_ERR_POSITION);
    EXPECT(kvr_prefill_rope(&d, &r, A, A, A, 65, A, A, A, nullptr), KVR_ERR_POSITION);
    EXPECT(kvr_continue_rope(&d, &r, A, A, A, A, A, 60, 8, 1, A, A, big, nullptr), KVR_ERR_POSITION);
    EXPECT(kvr_continue_rope(&d, nullptr, A, A, A, A, A, 60, 4, 1, A, A, big, nullptr), KVR_ERR_NULL);
    EXPECT(kvr_continue_batched_rope(&d, &r, A, A, A, cu_ok, 3, A, A, 60, A, A, big, nullptr), KVR_ERR_POSITION);
    EXPECT(kvr_rope_apply(&d, &r, A, 4, 0, 0, A, nullptr), KVR_ERR_SHAPE);
    // artifact: header round trip with L = 0 (no copies), then every corrupted field
    std::vector<unsigned char> host(KVR_ARTIFACT_HEADER_BYTES + 64);
    const void *kcs[2] = {A, A};
    void *kcd[2] = {A, A};
    int64_t L_out = -5;
    EXPECT(kvr_artifact_save(&d, "qwen3-4b", 2, 0, kcs, kcs, host.data(), host.size(), nullptr), KVR_OK);
    EXPECT(kvr_artifact_load(&d, "qwen3-4b", 2, host.data(), host.size(), kcd, kcd, &L_out, nullptr), KVR_OK);
    EXPECT(L_out == 0, 1);
    EXPECT(kvr_artifact_load(&d, "qwen3-8b", 2, host.data(), host.size(), kcd, kcd, &L_out, nullptr),
           KVR_ERR_MISMATCH);
    EXPECT(kvr_artifact_load(&d, "qwen3-4b", 3, host.data(), host.size(), kcd, kcd, &L_out, nullptr),
           KVR_ERR_MISMATCH);
    EXPECT(kvr_artifact_load(&d, "qwen3-4b", 2, host.data(), KVR_ARTIFACT_HEADER_BYTES - 1, kcd, kcd, &L_out,
                             nullptr),
           KVR_ERR_WORKSPACE);
    char long_id[200];
    memset(long_id, 'x', sizeof long_id - 1);
    long_id[sizeof long_id - 1] = 0;
    EXPECT(kvr_artifact_save(&d, long_id, 2, 0, kcs, kcs, host.data(), host.size(), nullptr), KVR_ERR_SHAPE);
    for (size_t off = 0; off < KVR_ARTIFACT_HEADER_BYTES; ++off) {
        std::vector<unsigned char> h2(host);
        h2[off] ^= 0x5a;
        const int st = kvr_artifact_load(&d, "qwen3-4b", 2, h2.data(), h2.size(), kcd, kcd, &L_out, nullptr);
        // the reserved tail of the header is ignored; every other byte is checked
        if (st != KVR_OK && st != KVR_ERR_MISMATCH && st != KVR_ERR_CAPACITY && st != KVR_ERR_WORKSPACE) {
            fprintf(stderr, "corrupted header byte %zu: status %d\n", off, st);
            ++fails;
        }
    }
}

// Random descriptors, lengths and reader tables through every entry point:
// whatever the status, the sanitizers watch the host arithmetic.
static void fuzz() {
    const int heads[] = {1, 2, 3, 4, 8, 16, 32, 64, 4096, 5000, 0, -3};
    const int dims[] = {64, 128, 96, 0};
    const int64_t caps[] = {0, 1, 64, 4096, 40000, 1LL << 20, (int64_t)1 << 31, -1};
    const int64_t lens[] = {0, 1, 2, 31, 32, 33, 63, 64, 65, 96, 255, 3774, 32768, 1LL << 20, (int64_t)1 << 31,
                            (int64_t)1 << 40, -1, -7};
    for (int it = 0; it < 20000; ++it) {
        kvr_desc d = desc();
        d.n_kv_heads = heads[next() % 12];
        d.n_q_heads = d.n_kv_heads * (int)(1 + next() % 8);
        if (next() % 8 == 0) d.n_q_heads = heads[next() % 12];
        d.head_dim = dims[next() % 4];
        d.dtype = (int)(next() % 4);
        d.capacity = pick(caps, 8);
        const int64_t Lp = pick(lens, 18), S = pick(lens, 18);
        const int32_t n = (int32_t)(next() % 140);
        std::vector<int32_t> cu(n + 1);
        cu[0] = 0;
        for (int32_t i = 1; i <= n; ++i) cu[i] = cu[i - 1] + (int32_t)(next() % 300);
        if (n > 0 && next() % 16 == 0) cu[next() % (n + 1)] = -(int32_t)(next() % 5);
        const size_t ws = kvr_workspace_bytes(&d, Lp, S, 1);
        const size_t wsn = kvr_workspace_bytes(&d, Lp, n > 0 ? cu[n] : 0, n);
        const size_t wsr = kvr_workspace_bytes_rope(&d, Lp, S, 1);
        const size_t wsrn = kvr_workspace_bytes_rope(&d, Lp, n > 0 ? cu[n] : 0, n);
        const size_t big = (size_t)1 << 50;
        kvr_rope r;
        r.cos_sin = AF;
        r.n_pos = pick(lens, 18);
        (void)kvr_prefill(&d, A, A, A, Lp, A, A, A, nullptr);
        (void)kvr_continue(&d, A, A, A, A, A, Lp, S, A, A, next() % 2 ? ws : big, nullptr);
        (void)kvr_continue_append(&d, A, A, A, A, A, Lp, S, A, A, ws, nullptr);
        (void)kvr_continue_batched(&d, A, A, A, cu.data(), n, A, A, Lp, A, A, wsn, nullptr);
        (void)kvr_cache_append(&d, A, A, S, A, A, Lp, nullptr);
        (void)kvr_q8_bytes(&d);
        (void)kvr_quantize_cache(&d, A, A, Lp, A, A, (float *)A, nullptr);
        (void)kvr_continue_q8(&d, A, A, A, A, A, AF, Lp, S, A, A, ws, nullptr);
        (void)kvr_prefill_rope(&d, &r, A, A, A, Lp, A, A, A, nullptr);
        (void)kvr_continue_rope(&d, &r, A, A, A, A, A, Lp, S, (int32_t)(next() % 2), A, A, wsr, nullptr);
        (void)kvr_continue_batched_rope(&d, &r, A, A, A, cu.data(), n, A, A, Lp, A, A, wsrn, nullptr);
        (void)kvr_rope_apply(&d, &r, A, S, (int32_t)(next() % 40) - 2, Lp, A, nullptr);
        (void)kvr_artifact_bytes(&d, (int32_t)(next() % 40) - 2, Lp);
    }
}

// The split plan of the continuation, as the kernels receive it: splits of
// whole 64-key tiles, no more splits than 256-key pieces of the prefix, the
// last one non-empty and
// ending at the prefix end -- or, for a prefix at most 32 - S keys past a
// multiple of the split count x 128 keys, chunks of a multiple of 128 keys
// whose last split also takes the few remaining keys.
static void split_plans() {
    const int64_t cap = 40200;
    kvr_desc e = desc(32, 8, 128, KVR_BF16, cap);
    void *P = (void *)(uintptr_t)0x100000;
    const int64_t lens[] = {256, 300, 1000, 3774, 4096, 8191, 16384, 16387, 16400, 32768, 32769, 32775,
                            32790, 32799, 32800, 32900, 40000};
    const int64_t sfx[] = {1, 2, 8, 12, 24, 31, 32, 33, 64, 96};
    int planned = 0;
    for (int64_t L : lens)
        for (int64_t S : sfx) {
            if (L + S > cap) continue;
            const size_t ws = kvr_workspace_bytes(&e, L, S, 1);
            g_nsplit = g_chunk = -1;
            const int st = kvr_continue(&e, P, P, P, P, P, L, S, P, P, ws, nullptr);
            if (st != KVR_ERR_DEVICE) { fprintf(stderr, "plan L=%ld S=%ld: status %d\n", (long)L, (long)S, st); ++fails; continue; }
            if (g_nsplit <= 1) continue;
            ++planned;
            const int64_t n = g_nsplit, c = g_chunk;
            const bool tiles = c % 64 == 0 && n <= (L + 255) / 256 && (n - 1) * c < L;
            const bool covers = n * c >= L || (c % 128 == 0 && L - n * c + S <= 32);
            if (!tiles || !covers) {
                fprintf(stderr, "plan L=%ld S=%ld: %ld splits of %ld keys\n", (long)L, (long)S, (long)n, (long)c);
                ++fails;
            }
        }
    if (planned < 50) { fprintf(stderr, "only %d split plans checked\n", planned); ++fails; }
}

int main() {
    if (kvr_abi_version() != KVR_ABI_VERSION) {
        fprintf(stderr, "ABI version mismatch\n");
        return 1;
    }
    for (int s = -1; s < 12; ++s)
        if (!kvr_strerror(s) || !kvr_strerror(s)[0]) ++fails;
    fixed_cases();
    split_plans();
    fuzz();
    if (g_pp_bad) {
        fprintf(stderr, "%d many-readers launches broke a plan invariant\n", g_pp_bad);
        ++fails;
    }
    if (g_pp_split < 20 || g_pp_whole < 20) {
        fprintf(stderr, "only %d split and %d whole many-readers plans checked\n", g_pp_split, g_pp_whole);
        ++fails;
    }
    if (fails) {
        fprintf(stderr, "%d checks failed\n", fails);
        return 1;
    }
    printf("host driver: all checks passed (%d stub launches; many-readers plans: %d split, %d whole)\n", g_launches,
           g_pp_split, g_pp_whole);
    return 0;
}
