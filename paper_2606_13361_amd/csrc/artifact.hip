// artifact.hip -- the KV artifact on the host: serialize the cached K/V rows
// of every layer with the metadata m = (model id, dtype, L) and load them back
// after checking that metadata against the running model (paper, Alg. 1
// SaveKV and Alg. 2 GenerateFromKV; Section "Producing an artifact": an
// artifact is valid only for the (model, dtype) it was made with).
//
// Host code only: the header is built and checked on the host; the rows move
// with one strided hipMemcpy2DAsync per layer and tensor (the kv heads' rows
// [0, L) are the "rows" of the 2-D copy, the cache capacity its source or
// destination pitch).  Layout in include/kvr.h.
#include <string.h>

#include "kvr.h"
#include "kvr_internal.hpp"

namespace kvr {
namespace {

constexpr char kMagic[8] = {'K', 'V', 'R', 'A', 'R', 'T', '0', '1'};
constexpr uint32_t kVersion = 1;
constexpr int kModelIdBytes = 128;

struct ArtifactHeader {
    char magic[8];
    uint32_t version;
    uint32_t header_bytes;
    char model_id[kModelIdBytes];
    int32_t dtype, n_layers, n_kv_heads, head_dim;
    int64_t length;
    uint64_t payload_bytes;
    uint8_t reserved[80];
};
static_assert(sizeof(ArtifactHeader) == KVR_ARTIFACT_HEADER_BYTES, "artifact header layout");

int valid_desc(const kvr_desc *d) {
    if (!d) return KVR_ERR_NULL;
    if (d->dtype != KVR_BF16 && d->dtype != KVR_F32 && d->dtype != KVR_F16) return KVR_ERR_DTYPE;
    if (d->n_q_heads <= 0 || d->n_kv_heads <= 0 || d->n_q_heads % d->n_kv_heads != 0) return KVR_ERR_SHAPE;
    if (d->head_dim != 64 && d->head_dim != 128) return KVR_ERR_SHAPE;
    if (d->capacity < 0 || d->reserved != 0) return KVR_ERR_SHAPE;
    return KVR_OK;
}

size_t elt(const kvr_desc *d) { return d->dtype == KVR_F32 ? 4 : 2; }

// bytes of one layer's K (or V) rows [0, L)
size_t tensor_bytes(const kvr_desc *d, int64_t L) { return (size_t)d->n_kv_heads * (size_t)L * d->head_dim * elt(d); }

int model_id_len(const char *model_id) {
    if (!model_id) return -1;
    const size_t n = strnlen(model_id, kModelIdBytes);
    return n < (size_t)kModelIdBytes ? (int)n : -1;
}

}  // namespace
}  // namespace kvr

using namespace kvr;

extern "C" {

size_t kvr_artifact_bytes(const kvr_desc *desc, int32_t n_layers, int64_t L) {
    if (valid_desc(desc) != KVR_OK || n_layers <= 0 || L < 0) return (size_t)-1;
    return KVR_ARTIFACT_HEADER_BYTES + 2 * (size_t)n_layers * tensor_bytes(desc, L);
}

int kvr_artifact_save(const kvr_desc *desc, const char *model_id, int32_t n_layers, int64_t L,
                      const void *const *kcaches, const void *const *vcaches, void *host, size_t host_bytes,
                      void *stream) {
    int st = valid_desc(desc);
    if (st) return st;
    if (n_layers <= 0 || L < 0) return KVR_ERR_SHAPE;
    if (L > desc->capacity) return KVR_ERR_CAPACITY;
    if (!model_id || !kcaches || !vcaches || !host) return KVR_ERR_NULL;
    const int idn = model_id_len(model_id);
    if (idn < 0) return KVR_ERR_SHAPE;
    if (host_bytes < kvr_artifact_bytes(desc, n_layers, L)) return KVR_ERR_WORKSPACE;
    if (L > 0)
        for (int32_t l = 0; l < n_layers; ++l)
            if (!kcaches[l] || !vcaches[l]) return KVR_ERR_NULL;

    ArtifactHeader h;
    memset(&h, 0, sizeof h);
    memcpy(h.magic, kMagic, sizeof h.magic);
    h.version = kVersion;
    h.header_bytes = KVR_ARTIFACT_HEADER_BYTES;
    memcpy(h.model_id, model_id, (size_t)idn);
    h.dtype = desc->dtype;
    h.n_layers = n_layers;
    h.n_kv_heads = desc->n_kv_heads;
    h.head_dim = desc->head_dim;
    h.length = L;
    h.payload_bytes = 2 * (uint64_t)n_layers * tensor_bytes(desc, L);
    memcpy(host, &h, sizeof h);
    if (L == 0) return KVR_OK;

    const size_t row = (size_t)L * desc->head_dim * elt(desc);            // one kv head's rows
    const size_t pitch = (size_t)desc->capacity * desc->head_dim * elt(desc);
    unsigned char *dst = (unsigned char *)host + KVR_ARTIFACT_HEADER_BYTES;
    for (int32_t l = 0; l < n_layers; ++l) {
        for (int t = 0; t < 2; ++t) {
            const void *src = t == 0 ? kcaches[l] : vcaches[l];
            if (hipMemcpy2DAsync(dst, row, src, pitch, row, desc->n_kv_heads, hipMemcpyDeviceToHost,
                                 (hipStream_t)stream) != hipSuccess)
                return KVR_ERR_DEVICE;
            dst += row * desc->n_kv_heads;
        }
    }
    return KVR_OK;
}

int kvr_artifact_load(const kvr_desc *desc, const char *model_id, int32_t n_layers, const void *host,
                      size_t host_bytes, void *const *kcaches, void *const *vcaches, int64_t *L_out, void *stream) {
    int st = valid_desc(desc);
    if (st) return st;
    if (n_layers <= 0) return KVR_ERR_SHAPE;
    if (!model_id || !host || !kcaches || !vcaches || !L_out) return KVR_ERR_NULL;
    const int idn = model_id_len(model_id);
    if (idn < 0) return KVR_ERR_SHAPE;
    if (host_bytes < KVR_ARTIFACT_HEADER_BYTES) return KVR_ERR_WORKSPACE;
    ArtifactHeader h;
    memcpy(&h, host, sizeof h);
    // Alg. 2: the artifact must come from the running (model, dtype) and shape
    if (memcmp(h.magic, kMagic, sizeof h.magic) != 0 || h.version != kVersion ||
        h.header_bytes != KVR_ARTIFACT_HEADER_BYTES)
        return KVR_ERR_MISMATCH;
    if (strnlen(h.model_id, kModelIdBytes) != (size_t)idn || memcmp(h.model_id, model_id, (size_t)idn) != 0)
        return KVR_ERR_MISMATCH;
    if (h.dtype != desc->dtype || h.n_kv_heads != desc->n_kv_heads || h.head_dim != desc->head_dim ||
        h.n_layers != n_layers)
        return KVR_ERR_MISMATCH;
    if (h.length < 0 || h.payload_bytes != 2 * (uint64_t)n_layers * tensor_bytes(desc, h.length))
        return KVR_ERR_MISMATCH;
    if (h.length > desc->capacity) return KVR_ERR_CAPACITY;
    if (host_bytes < KVR_ARTIFACT_HEADER_BYTES + h.payload_bytes) return KVR_ERR_WORKSPACE;
    const int64_t L = h.length;
    if (L > 0)
        for (int32_t l = 0; l < n_layers; ++l)
            if (!kcaches[l] || !vcaches[l]) return KVR_ERR_NULL;
    *L_out = L;
    if (L == 0) return KVR_OK;

    const size_t row = (size_t)L * desc->head_dim * elt(desc);
    const size_t pitch = (size_t)desc->capacity * desc->head_dim * elt(desc);
    const unsigned char *src = (const unsigned char *)host + KVR_ARTIFACT_HEADER_BYTES;
    for (int32_t l = 0; l < n_layers; ++l) {
        for (int t = 0; t < 2; ++t) {
            void *dst = t == 0 ? kcaches[l] : vcaches[l];
            if (hipMemcpy2DAsync(dst, pitch, src, row, row, desc->n_kv_heads, hipMemcpyHostToDevice,
                                 (hipStream_t)stream) != hipSuccess)
                return KVR_ERR_DEVICE;
            src += row * desc->n_kv_heads;
        }
    }
    return KVR_OK;
}

}  // extern "C"
