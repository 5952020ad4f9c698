/*
 * kvr_model.h -- C ABI of libkvr_model: the decoder layer around the
 * attention of libkvr, so that whole-model prefill and continuation costs
 * (the paper's Table 1: a full prefill of an L-token context against one
 * continuation step over the resident cache) can be measured.
 *
 * The layer (a reading: the paper names Qwen3-4B, 36 layers, 8 KV heads of
 * width 128, and no layer formula; this is the published Qwen3 decoder layer):
 *
 *     x  = rmsnorm(h) * ln1
 *     [q | k | v] = x Wqkv^T
 *     q_h = rope(rmsnorm(q_h) * q_norm),  k_h = rope(rmsnorm(k_h) * k_norm)   (per head)
 *     h  = h + attention(q, k, v) Wo^T
 *     x  = rmsnorm(h) * ln2
 *     [g | u] = x Wgu^T
 *     h  = h + (silu(g) * u) Wd^T
 *
 * rmsnorm(x) = x / sqrt(mean(x^2) + eps), silu(x) = x / (1 + e^-x).  Token t
 * of a call sits at position L_prefix + t (Alg. 2: positions continue from the
 * artifact's length); rope is the rotation of kvr_rope_apply; attention is
 * kvr_prefill (L_prefix == 0) or kvr_continue over cache rows [0, L_prefix).
 *
 * Conventions: as in kvr.h (device pointers owned by the caller, validation on
 * the host before any launch, work enqueued on `stream`, 16-byte alignment).
 * Elements are bf16 or fp16 (desc->dtype); every activation is held in that
 * format between operations and computed in fp32.  Weights are row-major
 * [out][in] (the layout of a linear layer's weight).  Matrix products of more
 * than one token run on hipBLASLt (fp32 accumulation); a one-token step's
 * products, and every other operation, are this library's kernels (fp32
 * accumulation; the step's RMSNorms and SiLU gate run inside its products).
 */
#ifndef KVR_MODEL_H
#define KVR_MODEL_H

#include <stddef.h>
#include <stdint.h>

#include "kvr.h"

#ifdef __cplusplus
extern "C" {
#endif

#define KVR_MODEL_ABI_VERSION 1

/* Widths of the layer beyond the attention geometry of kvr_desc. */
typedef struct {
    int32_t hidden;       /* model width, a multiple of 8, <= 65536          */
    int32_t intermediate; /* MLP width, a multiple of 8, <= 262144           */
    float eps;            /* RMSNorm epsilon, >= 0                           */
    int32_t reserved;     /* must be 0                                       */
} kvr_layer_shape;

/* One layer's weights (device pointers, element type of the descriptor). */
typedef struct {
    const void *ln1;    /* [hidden]                                        */
    const void *wqkv;   /* [(n_q_heads + 2 n_kv_heads) head_dim][hidden]:
                           the q heads' rows, then k, then v               */
    const void *q_norm; /* [head_dim]                                      */
    const void *k_norm; /* [head_dim]                                      */
    const void *wo;     /* [hidden][n_q_heads head_dim]                    */
    const void *ln2;    /* [hidden]                                        */
    const void *wgu;    /* [2 intermediate][hidden]: gate rows, then up    */
    const void *wd;     /* [hidden][intermediate]                          */
} kvr_layer_weights;

/*
 * A matrix-product context: a hipBLASLt handle and the algorithms chosen for
 * the shapes seen so far.  Owned by the caller; use it from one thread at a
 * time.  The first product of a new shape queries the library's heuristics
 * on the host (do that before capturing a HIP graph).
 */
int kvr_blas_create(void **blas);
int kvr_blas_destroy(void *blas);

/* hipBLASLt workspace bytes every product of this library may use. */
#define KVR_BLAS_WORKSPACE_BYTES ((size_t)32 << 20)

/*
 * y[rows][n_out] = x[rows][n_in] w[n_out][n_in]^T + beta * y, accumulated in
 * fp32 and rounded once to the element type (beta 0 or 1; with beta 1, y is
 * read and written in place).  ws: at least KVR_BLAS_WORKSPACE_BYTES.
 */
int kvr_linear(void *blas, int32_t dtype, const void *x, const void *w, int64_t rows, int32_t n_in,
               int32_t n_out, float beta, void *y, void *ws, size_t ws_bytes, void *stream);

/* y[rows][n] = rmsnorm(x[rows][n]) * w[n]; n a multiple of 8, <= 65536. */
int kvr_rmsnorm(int32_t dtype, const void *x, const void *w, int64_t rows, int32_t n, float eps, void *y,
                void *stream);

/* Workspace bytes of kvr_layer_forward for T tokens and prefixes up to
 * L_prefix_max ((size_t)-1 for invalid arguments). */
size_t kvr_layer_workspace_bytes(const kvr_desc *desc, const kvr_layer_shape *shape, int64_t T,
                                 int64_t L_prefix_max);

/*
 * One decoder layer over T tokens at positions L_prefix .. L_prefix + T - 1.
 *   h [T][hidden]: the residual stream, updated in place.
 *   kcache/vcache: rows [0, L_prefix) are read; the tokens' rotated keys and
 *   values are written into rows [L_prefix, L_prefix + T) (needs
 *   L_prefix + T <= capacity).
 *   rope: table with n_pos >= L_prefix + T.
 *   ws: kvr_layer_workspace_bytes(desc, shape, T, L) bytes for some L >= L_prefix.
 * bf16 / fp16 only (KVR_ERR_DTYPE), head_dim 64 or 128.
 */
int kvr_layer_forward(const kvr_desc *desc, const kvr_layer_shape *shape, const kvr_layer_weights *w,
                      const kvr_rope *rope, void *blas, void *h, int64_t T, int64_t L_prefix, void *kcache,
                      void *vcache, void *ws, size_t ws_bytes, void *stream);

/* KVR_MODEL_ABI_VERSION of the loaded library. */
int kvr_model_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVR_MODEL_H */
