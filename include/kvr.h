/*
 * kvr.h -- C ABI of libkvr: prefill and prefix-reuse continuation attention
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation (paper, Section "Method"): a decoder layer's causal
 * grouped-query attention in two modes of one computation.
 *
 *   prefill   -- L tokens attend causally to each other and their K/V rows
 *                are written into the layer's cache (Alg. 1: the publisher's
 *                one-time forward pass that produces the KV artifact).
 *   continue  -- S new tokens at positions L_prefix .. L_prefix+S-1 attend to
 *                the cached rows 0 .. L_prefix-1 and causally to their own
 *                keys (Alg. 2: positions continue from the artifact's length
 *                and the mask spans the whole cached context).  Claim 1 of the
 *                paper: row i of a continuation equals row L_prefix+i of a
 *                prefill of the concatenation, since cached entries of a causal
 *                prefix never depend on later tokens.
 *
 *   For query row at absolute position p, head h, kv head g = h / G with
 *   G = n_q_heads / n_kv_heads, keys j = 0..p:
 *       out = sum_j softmax_j(scale * q . k_j) v_j
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library
 *     never allocates, frees or retains device memory and keeps no state
 *     between calls (every call is thread-safe) -- except
 *     kvr_continue_noalloc, which keeps its split partials in a fixed buffer
 *     inside the library (see there).
 *   - Layouts are dense row-major:
 *         Q, out            [tokens][n_q_heads][head_dim]
 *         K, V (new rows)   [tokens][n_kv_heads][head_dim]
 *         kcache, vcache    [n_kv_heads][capacity][head_dim]
 *     Elements are bf16 (KVR_BF16), fp16 (KVR_F16, the paper's precision) or
 *     fp32 (KVR_F32) as the descriptor says; 16-bit inputs accumulate in fp32,
 *     the attention weights enter the second product in the input format, and
 *     16-bit outputs are rounded to nearest-even.
 *   - Every call validates all arguments on the host, synchronously, before
 *     any HIP call; on an error nothing is launched and a kvr_status != 0 is
 *     returned.  On success the work is enqueued on `stream` (a hipStream_t;
 *     NULL is the default stream) and the call returns at once.
 *   - Device pointers must be 16-byte aligned (KVR_ERR_ALIGN otherwise).
 *   - Zero-length work (L == 0, S == 0, n == 0) is a successful no-op.
 *   - For a fixed shape and device the results are bitwise reproducible:
 *     the key split and the order of every reduction are fixed.
 */
#ifndef KVR_H
#define KVR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVR_ABI_VERSION 4

typedef enum {
    KVR_OK = 0,
    KVR_ERR_NULL = 1,      /* a required pointer is NULL                          */
    KVR_ERR_SHAPE = 2,     /* heads, head_dim, lengths or cu_seqlens invalid        */
    KVR_ERR_DTYPE = 3,     /* unsupported element type                             */
    KVR_ERR_CAPACITY = 4,  /* the cache rows addressed exceed the capacity         */
    KVR_ERR_WORKSPACE = 5, /* workspace smaller than kvr_workspace_bytes()         */
    KVR_ERR_ALIGN = 6,     /* a device pointer is not 16-byte aligned              */
    KVR_ERR_DEVICE = 7,    /* a HIP call or kernel launch failed                   */
    KVR_ERR_MISMATCH = 8,  /* an artifact's metadata does not match (model, dtype,
                              heads, head_dim, layers) or its header is not valid  */
    KVR_ERR_POSITION = 9,  /* a RoPE table without an entry for a position the call
                              rotates, or invalid table arguments                  */
    KVR_ERR_TOO_LARGE = 10 /* the call needs more scratch memory than the fixed
                              buffer of kvr_continue_noalloc holds                 */
} kvr_status;

typedef enum { KVR_BF16 = 0, KVR_F32 = 1, KVR_F16 = 2 } kvr_dtype;

/*
 * Layer descriptor.  The paper's artifact metadata (model id, dtype, length;
 * Section "Producing an artifact") must match between producer and consumer;
 * at this level that is the element type and the head geometry, which every
 * call checks.
 *   n_q_heads, n_kv_heads  > 0 and n_q_heads % n_kv_heads == 0
 *   head_dim               64 or 128
 *   dtype                  a kvr_dtype
 *   scale                  softmax scale; <= 0 selects 1/sqrt(head_dim)
 *   capacity               rows per kv head in kcache/vcache (>= 0)
 */
typedef struct {
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t dtype;
    float scale;
    int32_t reserved; /* must be 0 */
    int64_t capacity;
} kvr_desc;

/*
 * Full causal prefill of L tokens (Alg. 1, attention part).
 *   Q [L][Hq][d], K/V [L][Hkv][d] in; out [L][Hq][d] out.
 *   Writes kcache/vcache rows [0, L) of every kv head (exact copies of K/V);
 *   rows >= L are not touched.  Needs L <= capacity (KVR_ERR_CAPACITY).
 *   out must not alias Q, K or V.
 */
int kvr_prefill(const kvr_desc *desc, const void *Q, const void *K, const void *V, int64_t L,
                void *out, void *kcache, void *vcache, void *stream);

/*
 * Continuation of S tokens over a cached prefix (Alg. 2, one forward call).
 *   Qs [S][Hq][d] at positions L_prefix..L_prefix+S-1; Ks/Vs [S][Hkv][d] are
 *   their own keys and values; kcache/vcache rows [0, L_prefix) are the
 *   cached prefix and are only read (many readers may share one cache).
 *   out [S][Hq][d].  Needs L_prefix <= capacity.  L_prefix == 0 gives a
 *   prefill of the S tokens (the caches may then be NULL).
 *   ws: device workspace of at least kvr_workspace_bytes(desc, L_prefix, S, 1)
 *   bytes (may be NULL when that is 0); it holds per-split partial results.
 */
int kvr_continue(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                 const void *kcache, const void *vcache, int64_t L_prefix, int64_t S,
                 void *out, void *ws, size_t ws_bytes, void *stream);

/*
 * kvr_continue without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Arguments, layouts, results and errors are those of
 * kvr_continue; the result is bit-identical to it.
 *   The split partials go to a buffer of KVR_NOALLOC_SCRATCH_BYTES inside the
 *   library, one per device, held from the first call on that device until the
 *   process ends.  A call whose plan needs more (kvr_workspace_bytes(desc,
 *   L_prefix, S, 1) > KVR_NOALLOC_SCRATCH_BYTES) returns KVR_ERR_TOO_LARGE and
 *   launches nothing; every decode step and the 24-token continuation of a
 *   32-query / 8-kv-head / 128-wide layer fit.  The call allocates nothing;
 *   its first call on a device looks the buffer up (KVR_ERR_DEVICE if that
 *   fails).  Every call on a device shares that device's buffer: calls that
 *   may overlap on one device (different streams, threads) race and must be
 *   ordered by the caller.  Nothing in the buffer needs clearing between calls.
 */
#define KVR_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int kvr_continue_noalloc(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                         const void *kcache, const void *vcache, int64_t L_prefix, int64_t S,
                         void *out, void *stream);

/*
 * Many independent continuations of one shared cached prefix (the paper's
 * N readers of one document), in one call.
 *   Reader r owns packed rows [cu[r], cu[r+1]) of Qs/Ks/Vs/out, which sit at
 *   positions L_prefix .. L_prefix + (cu[r+1]-cu[r]) - 1 and see the shared
 *   prefix plus their own rows causally, never another reader's rows.
 *   cu_seqlens_host: HOST array of n+1 int32, cu[0] == 0, non-decreasing.
 *   ws: device workspace of at least kvr_workspace_bytes(desc, L_prefix,
 *   cu[n], n) bytes (16-byte aligned; may be NULL when that is 0).  At bf16 /
 *   fp16 and head_dim 128, for 2..128 readers, the call may split the row
 *   tiles of its last partial round of workgroups over the prefix keys and
 *   merge them through ws.  KVR_ERR_WORKSPACE if ws_bytes is smaller.
 */
int kvr_continue_batched(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                         const int32_t *cu_seqlens_host, int32_t n, const void *kcache,
                         const void *vcache, int64_t L_prefix, void *out, void *ws,
                         size_t ws_bytes, void *stream);

/*
 * kvr_continue followed by the cache update of its tokens (Alg. 2's forward
 * call and cache update; a decode step when S == 1): out as kvr_continue
 * computes it over cache rows [0, L_prefix), and cache rows
 * [L_prefix, L_prefix + S) receive Ks/Vs unchanged, exactly as
 * kvr_cache_append(desc, Ks, Vs, S, kcache, vcache, L_prefix) writes them.
 * Needs L_prefix + S <= capacity.  For 16-bit continuations at head_dim 128
 * with (n_q_heads / n_kv_heads) * S <= 96 the attention kernel stores the
 * rows itself (one launch fewer); other shapes issue the update after it.
 * ws as for kvr_continue.
 */
int kvr_continue_append(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                        void *kcache, void *vcache, int64_t L_prefix, int64_t S, void *out,
                        void *ws, size_t ws_bytes, void *stream);

/*
 * Cache write: rows [L_cur, L_cur+S) of each kv head receive Ks/Vs
 * [S][Hkv][d] unchanged (Alg. 2's cache update after a decode step).
 * Needs 0 <= L_cur and L_cur + S <= capacity.  Other rows are untouched.
 */
int kvr_cache_append(const kvr_desc *desc, const void *Ks, const void *Vs, int64_t S,
                     void *kcache, void *vcache, int64_t L_cur, void *stream);

/*
 * The int8 KV artifact (paper, Section "Quantizing the artifact: size vs.
 * exactness": the context KV stored at per-tensor symmetric int8, half the
 * bytes of the 16-bit artifact, no longer token-exact).
 *   One scale per tensor: s_K = max|K| / 127 over every kv head and cached row
 *   [0, L) (fp32, correctly rounded; 1 for an all-zero tensor), likewise s_V.
 *   Code of x: clamp(round-half-even(x / s), -127, 127), the quotient in fp32.
 *   Layouts (bytes; P = capacity rounded up to a multiple of 32, head_dim 128):
 *     kq  [n_kv_heads][P][128]: row j of kv head g holds the code of K[g][j][d]
 *         at byte 64 * ((d >> 3) & 1) + 8 * (d >> 4) + (d & 7) of the row
 *     vq  [n_kv_heads][P / 32][128][32]: the code of V[g][32 b + k][d] is byte
 *         ((g * (P / 32) + b) * 128 + d) * 32 + pos(k), with
 *         pos(k) = 16 * ((k >> 2) & 1) + 8 * (k >> 4) + 4 * ((k >> 3) & 1) + (k & 3)
 *     scales  float[2] = {s_K, s_V} in device memory
 *   These are the operand orders of the continuation kernel's matrix products,
 *   so it reads every code with plain 16-byte loads.  The artifact is read
 *   only; a decode chain continues over it and keeps its new rows in bf16.
 */

/* Bytes of kq (and of vq) for this descriptor; (size_t)-1 if it is invalid. */
size_t kvr_q8_bytes(const kvr_desc *desc);

/*
 * Quantize cache rows [0, L) of every kv head (bf16 kcache/vcache) into the
 * int8 artifact: writes kq/vq rows [0, L) plus the zero codes up to the next
 * multiple of 32, and scales.  Needs bf16 (KVR_ERR_DTYPE), head_dim 128
 * (KVR_ERR_SHAPE), L <= capacity.  kq and vq hold kvr_q8_bytes(desc) bytes
 * each and are 16-byte aligned; scales needs 4-byte alignment.  Runs four
 * small kernels on `stream` (scales first hold the maxima).
 */
int kvr_quantize_cache(const kvr_desc *desc, const void *kcache, const void *vcache, int64_t L,
                       void *kq, void *vq, float *scales, void *stream);

/*
 * Continuation of S tokens over the int8 artifact: kvr_continue with the
 * cached rows [0, L_prefix) replaced by their dequantized values code * s;
 * the new tokens' Ks/Vs stay bf16.  The artifact must come from
 * kvr_quantize_cache with the same descriptor and some L >= L_prefix.
 * Supported: bf16, head_dim 128 and (n_q_heads / n_kv_heads) * S <= 96
 * (decode steps and short continuations); KVR_ERR_SHAPE otherwise.
 * ws as for kvr_continue (kvr_workspace_bytes(desc, L_prefix, S, 1)).
 */
int kvr_continue_q8(const kvr_desc *desc, const void *Qs, const void *Ks, const void *Vs,
                    const void *kq, const void *vq, const float *scales, int64_t L_prefix,
                    int64_t S, void *out, void *ws, size_t ws_bytes, void *stream);

/*
 * The KV artifact on the host (paper, Alg. 1 SaveKV and Alg. 2
 * GenerateFromKV): the per-layer cached K/V rows [0, L) serialized with
 * metadata m = (model id, dtype, L); the consumer rejects an artifact made for
 * another (model, dtype).  Layout, little-endian:
 *   header, KVR_ARTIFACT_HEADER_BYTES bytes:
 *     char     magic[8]         "KVRART01"
 *     uint32   version          1
 *     uint32   header_bytes     256
 *     char     model_id[128]    NUL-terminated, NUL-padded
 *     int32    dtype, n_layers, n_kv_heads, head_dim
 *     int64    length           L, cached rows per kv head
 *     uint64   payload_bytes    2 * n_layers * n_kv_heads * L * head_dim * element bytes
 *     80 bytes of zero
 *   payload: for layer 0, 1, ...: K rows [n_kv_heads][L][head_dim], then V rows
 *   likewise (the cache rows [0, L) of each kv head, packed).
 * The copies run on `stream` (device <-> host, one strided copy per layer and
 * tensor); host memory from hipHostMalloc (or torch pin_memory) makes them
 * asynchronous at full link speed, pageable memory works but serializes.
 */
#define KVR_ARTIFACT_HEADER_BYTES 256

/* Bytes of an artifact of n_layers layers and L rows; (size_t)-1 if invalid. */
size_t kvr_artifact_bytes(const kvr_desc *desc, int32_t n_layers, int64_t L);

/*
 * Serialize cache rows [0, L) of n_layers layers into host memory `host`
 * (host_bytes >= kvr_artifact_bytes, else KVR_ERR_WORKSPACE).  kcaches and
 * vcaches are HOST arrays of n_layers device pointers to [n_kv_heads][capacity]
 * [head_dim] caches.  The header is written before the call returns; the rows
 * are copied on `stream` (synchronize before reading them).  model_id: at most
 * 127 bytes (KVR_ERR_SHAPE otherwise).
 */
int kvr_artifact_save(const kvr_desc *desc, const char *model_id, int32_t n_layers, int64_t L,
                      const void *const *kcaches, const void *const *vcaches, void *host,
                      size_t host_bytes, void *stream);

/*
 * Load an artifact from host memory into the caches of n_layers layers (rows
 * [0, L); other rows untouched) after checking its header against the running
 * model: magic and version, model_id, dtype, n_kv_heads, head_dim, n_layers
 * (KVR_ERR_MISMATCH on any difference), L <= capacity (KVR_ERR_CAPACITY),
 * payload within host_bytes (KVR_ERR_WORKSPACE).  The checks run on the host
 * before any copy; *L_out receives L (Alg. 2: the continuation starts at m.L).
 */
int kvr_artifact_load(const kvr_desc *desc, const char *model_id, int32_t n_layers, const void *host,
                      size_t host_bytes, void *const *kcaches, void *const *vcaches, int64_t *L_out,
                      void *stream);

/*
 * Rotary position embedding with the position offset (paper, Section
 * "Consuming an artifact": the continuation's tokens take positions L, L+1,
 * ... after an artifact of length L, so that the positional encoding, e.g.
 * RoPE, agrees with a pass from scratch).  The rotary embedding of Su et al.
 * in the half-split pairing of the Qwen family: pair i in [0, d/2) of a head
 * row is (x[i], x[i + d/2]); at position p it turns by the angle p * theta_i,
 * theta_i = base^(-2 i / d):
 *     y[i]       = x[i] cos - x[i + d/2] sin
 *     y[i + d/2] = x[i + d/2] cos + x[i] sin
 * Queries and keys are rotated, values are not, and the cache holds rotated
 * keys (as the model's cache does).  The rotation runs in fp32 from the
 * table's fp32 cos/sin and rounds once to the element format (16-bit: to
 * nearest even); every entry point rotates a given row at a given position to
 * the same bits.
 *
 * The table: float [n_pos][head_dim / 2][2] = (cos, sin) of p * theta_i in
 * device memory (16-byte aligned), made by kvr_rope_table.  An entry point
 * that rotates positions up to P needs n_pos > P (KVR_ERR_POSITION).
 */
typedef struct {
    const float *cos_sin; /* device table [n_pos][head_dim / 2][2]            */
    int64_t n_pos;        /* positions 0 .. n_pos - 1 it holds                  */
} kvr_rope;

/*
 * Fill cos_sin [n_pos][head_dim / 2][2] for the given base on `stream`: the
 * angle p * theta_i and its cosine and sine in fp64, each rounded once to
 * fp32.  head_dim 64 or 128 (KVR_ERR_SHAPE), base finite and > 0, n_pos >= 0
 * (KVR_ERR_POSITION); cos_sin 16-byte aligned.
 */
int kvr_rope_table(int32_t head_dim, double base, int64_t n_pos, float *cos_sin, void *stream);

/*
 * Rotate rows x [n_tok][n_heads][head_dim] (element type and head_dim from
 * desc) at positions pos0 .. pos0 + n_tok - 1 into y (same layout; y == x
 * rotates in place, other overlaps are not allowed).  n_heads > 0.  For
 * callers that compose the other entry points themselves, e.g. rotated keys
 * for kvr_cache_append or rotated Q/K for kvr_continue_q8.
 */
int kvr_rope_apply(const kvr_desc *desc, const kvr_rope *rope, const void *x, int64_t n_tok,
                   int32_t n_heads, int64_t pos0, void *y, void *stream);

/*
 * kvr_prefill with RoPE: Q and K arrive unrotated, token t sits at position t.
 * A pre-pass writes the rotated K rows and the V rows into kcache/vcache rows
 * [0, L); the attention kernel reads the keys back from the cache and rotates
 * each query row in registers.  Needs rope->n_pos >= L.
 */
int kvr_prefill_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Q, const void *K,
                     const void *V, int64_t L, void *out, void *kcache, void *vcache, void *stream);

/*
 * kvr_continue with RoPE (Alg. 2): Qs and Ks arrive unrotated and are rotated
 * at positions L_prefix .. L_prefix + S - 1; kcache rows [0, L_prefix) hold
 * rotated keys (from kvr_prefill_rope, an earlier call with append, or
 * kvr_rope_apply + kvr_cache_append).  append != 0 also writes the rotated Ks
 * and the Vs into cache rows [L_prefix, L_prefix + S) (a decode step in one
 * call; needs L_prefix + S <= capacity); append == 0 leaves the cache
 * untouched.  The rotated Qs/Ks rows go through ws:
 * ws_bytes >= kvr_workspace_bytes_rope(desc, L_prefix, S, 1).
 * Needs rope->n_pos >= L_prefix + S.
 */
int kvr_continue_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Qs, const void *Ks,
                      const void *Vs, void *kcache, void *vcache, int64_t L_prefix, int64_t S,
                      int32_t append, void *out, void *ws, size_t ws_bytes, void *stream);

/*
 * kvr_continue_batched with RoPE: reader r's rows [cu[r], cu[r+1]) sit at
 * positions L_prefix .. L_prefix + (cu[r+1] - cu[r]) - 1.  Their rotated keys
 * go through ws (kvr_workspace_bytes_rope(desc, L_prefix, cu[n], n) bytes);
 * query rows are rotated in registers.  The shared cache is only read.
 * Needs rope->n_pos >= L_prefix + the longest reader.
 */
int kvr_continue_batched_rope(const kvr_desc *desc, const kvr_rope *rope, const void *Qs,
                              const void *Ks, const void *Vs, const int32_t *cu_seqlens_host,
                              int32_t n, const void *kcache, const void *vcache, int64_t L_prefix,
                              void *out, void *ws, size_t ws_bytes, void *stream);

/*
 * Workspace bytes of kvr_continue_rope (n <= 1, total_S = S) and
 * kvr_continue_batched_rope (n >= 2, total_S = cu[n]): the plain
 * continuation's workspace plus room for the rotated rows.  Non-decreasing in
 * L_prefix for a fixed total_S; (size_t)-1 for an invalid descriptor.
 */
size_t kvr_workspace_bytes_rope(const kvr_desc *desc, int64_t L_prefix, int64_t total_S, int32_t n);

/*
 * Workspace bytes a continuation needs: n <= 1 for kvr_continue with
 * total_S = S, n >= 2 for kvr_continue_batched with total_S = cu[n].
 * A pure function of its arguments (no device query); returns 0 when no
 * workspace is needed and (size_t)-1 for an invalid descriptor.  For a fixed
 * S it never decreases with L_prefix: a workspace sized for the longest
 * prefix serves every shorter one (e.g. all steps of a decode chain).
 */
size_t kvr_workspace_bytes(const kvr_desc *desc, int64_t L_prefix, int64_t total_S, int32_t n);

/* Static text for a kvr_status value. */
const char *kvr_strerror(int status);

/* KVR_ABI_VERSION of the loaded library. */
int kvr_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVR_H */
