// C entry points for single-layer calls: argument validation, then launch.
// Nothing is enqueued unless every check passes.
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace oc {

static thread_local std::string g_err;

void set_error(const std::string &msg) { g_err = msg; }
void clear_error() { g_err.clear(); }
int fail(int status, const std::string &msg) {
    g_err = msg;
    return status;
}
int hip_fail(hipError_t e, const char *what) {
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return OC_EHIP;
}

int check_copy_pieces(int64_t pieces, const char *what) {
    if (pieces > OC_MAX_GRID_ITEMS)
        return fail(OC_ERANGE, std::string(what) + ": more than 2^32 16-byte pieces in one launch");
    return OC_OK;
}

static int check_layout(const oc_layout &l) {
    if (l.num_layers < 1 || l.num_q_heads < 1 || l.num_kv_heads < 1 || l.head_dim < 1 || l.page_size < 1 ||
        l.chunk_tokens < 1 || l.num_pages < 1)
        return fail(OC_EINVAL, "layout fields must be positive");
    if (l.num_q_heads % l.num_kv_heads != 0) return fail(OC_ESHAPE, "num_q_heads must be a multiple of num_kv_heads");
    if (l.head_dim % 8 != 0) return fail(OC_ESHAPE, "head_dim must be a multiple of 8");
    if (l.page_size % 8 != 0) return fail(OC_ESHAPE, "page_size must be a multiple of 8");
    return OC_OK;
}

static int check_table(const oc_block_table *bt, const oc_layout &l) {
    if (!bt) return fail(OC_EINVAL, "block_table is NULL");
    if (bt->num_tokens < 0 || bt->num_entries < 0) return fail(OC_EINVAL, "negative block table size");
    const int64_t need = (bt->num_tokens + l.page_size - 1) / l.page_size;
    if (bt->num_entries < need) return fail(OC_ERANGE, "block table shorter than the prefix needs");
    if (need > 0 && !bt->pages) return fail(OC_EINVAL, "block table pages pointer is NULL");
    if (need > l.num_pages) return fail(OC_ERANGE, "prefix needs more pages than the pool has");
    return OC_OK;
}

static IngestArgs ingest_args(const oc_kv_pool *pool, const oc_block_table *bt, int32_t layer,
                              const void *staging) {
    const oc_layout &l = pool->layout;
    IngestArgs a{};
    const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
    uint16_t *base = static_cast<uint16_t *>(pool->base);
    a.staging = static_cast<const uint16_t *>(staging);
    a.pool_k = base + ((int64_t)layer * 2 + 0) * l.num_pages * block;
    a.pool_v = base + ((int64_t)layer * 2 + 1) * l.num_pages * block;
    a.pages = bt->pages;
    a.num_tokens = bt->num_tokens;
    a.G = l.chunk_tokens;
    a.n_kv = l.num_kv_heads;
    a.d = l.head_dim;
    a.Ps = l.page_size;
    return a;
}

IngestArgs chunks_ingest_args(const oc_kv_pool *pool, const oc_block_table *bt, const void *objects,
                              int64_t first_chunk, int64_t num_chunks) {
    const oc_layout &l = pool->layout;
    IngestArgs a = ingest_args(pool, bt, 0, objects);
    const int64_t slice = 2LL * l.chunk_tokens * l.num_kv_heads * l.head_dim;   // elements of S
    const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
    a.num_tokens = num_chunks * l.chunk_tokens;
    a.token0 = first_chunk * l.chunk_tokens;
    a.chunk_stride = (int64_t)l.num_layers * slice;
    a.n_layers = l.num_layers;
    a.layer_step_staging = slice;
    a.layer_step_pool = 2 * l.num_pages * block;
    return a;
}

AppendArgs append_args(const oc_kv_pool *pool, const oc_block_table *bt, int32_t layer, const void *k_new,
                       const void *v_new, int64_t suffix_tokens) {
    const oc_layout &l = pool->layout;
    const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
    uint16_t *base = static_cast<uint16_t *>(pool->base);
    AppendArgs a{};
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.pool_k = base + ((int64_t)layer * 2 + 0) * l.num_pages * block;
    a.pool_v = base + ((int64_t)layer * 2 + 1) * l.num_pages * block;
    a.pages = bt->pages;
    a.num_tokens = suffix_tokens;
    a.token0 = bt->num_tokens;
    a.n_kv = l.num_kv_heads;
    a.d = l.head_dim;
    a.Ps = l.page_size;
    return a;
}

// the table must also hold pages for suffix_tokens tokens behind the prefix
int check_append_table(const oc_block_table *bt, const oc_layout &l, int64_t suffix_tokens) {
    const int64_t need = (bt->num_tokens + suffix_tokens + l.page_size - 1) / l.page_size;
    if (bt->num_entries < need)
        return fail(OC_ERANGE, "block table needs " + std::to_string(need) +
                                   " entries to hold the suffix behind the prefix");
    if (need > l.num_pages) return fail(OC_ERANGE, "prefix and suffix need more pages than the pool has");
    if (need > 0 && !bt->pages) return fail(OC_EINVAL, "block table pages pointer is NULL");
    return OC_OK;
}

static int check_staging_shape(const oc_layout &l, const oc_block_table *bt, int64_t num_chunks,
                               int64_t slice_bytes) {
    const int64_t S = 2LL * l.chunk_tokens * l.num_kv_heads * l.head_dim * 2;
    if (num_chunks < 0) return fail(OC_EINVAL, "negative num_chunks");
    if (slice_bytes != S)
        return fail(OC_ESHAPE, "per_layer_chunk_bytes must equal 2*G*n_kv*d*2 = " + std::to_string(S));
    if (num_chunks * l.chunk_tokens != bt->num_tokens)
        return fail(OC_ESHAPE, "num_chunks * chunk_tokens must equal the block table's num_tokens");
    return OC_OK;
}

static int check_attention_layout(const oc_layout &l) {
    int rc = check_layout(l);
    if (rc) return rc;
    if (l.head_dim != 64 && l.head_dim != 128) return fail(OC_ESHAPE, "attention supports head_dim 64 or 128");
    if (l.page_size != 16) return fail(OC_ESHAPE, "attention supports page_size 16");
    return OC_OK;
}

int check_attention_args(const oc_layout &l, int64_t Tp, int64_t Ts) {
    int rc = check_attention_layout(l);
    return rc ? rc : check_attention_shape(l, Tp, Ts);
}

// ---- workspace of the allocation-free attention entry point ----------------
// The split partials of oc_suffix_prefill_layer_noalloc live in this array;
// every GPU the library runs on holds its own copy until the process ends.
// Host code never passes the array's name to a kernel (on the host it stands
// for no device address): it takes the device address that
// hipGetSymbolAddress reports, once per device, and uses only that.
static __device__ __align__(256) unsigned char scratch[OC_NOALLOC_WORKSPACE_BYTES];

constexpr int kMaxScratchDevices = 64;
static std::once_flag g_scratch_once[kMaxScratchDevices];
static void *g_scratch_ptr[kMaxScratchDevices];
static hipError_t g_scratch_status[kMaxScratchDevices];

// device address of `scratch` on the current device
static int scratch_on_current_device(void **ptr) {
    int dev = 0;
    OC_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxScratchDevices) return fail(OC_EINVAL, "device index beyond the library's table");
    std::call_once(g_scratch_once[dev], [dev] {
        void *p = nullptr;
        g_scratch_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = p;
    });
    if (g_scratch_status[dev] != hipSuccess) return hip_fail(g_scratch_status[dev], "hipGetSymbolAddress(scratch)");
    if (!g_scratch_ptr[dev]) return fail(OC_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    *ptr = g_scratch_ptr[dev];
    return OC_OK;
}

}  // namespace oc

using namespace oc;

extern "C" {

int oc_abi_version(void) { return OC_ABI_VERSION; }

const char *oc_last_error(void) { return g_err.c_str(); }

static int block_table_check_body(const int32_t *host_pages, int64_t num_entries, int64_t num_tokens, int64_t num_pages,
                                  int32_t page_size) {
    clear_error();
    if (page_size < 1 || num_tokens < 0 || num_entries < 0 || num_pages < 1)
        return fail(OC_EINVAL, "bad sizes");
    const int64_t need = (num_tokens + page_size - 1) / page_size;
    if (num_entries < need) return fail(OC_ERANGE, "block table shorter than the prefix needs");
    if (need > 0 && !host_pages) return fail(OC_EINVAL, "pages is NULL");
    for (int64_t i = 0; i < need; ++i) {
        const int64_t p = host_pages[i];
        if (p < 0 || p >= num_pages) return fail(OC_ERANGE, "page id " + std::to_string(p) + " out of range");
    }
    // repeats: sorted, equal ids are neighbours (memory follows the table,
    // not the pool)
    std::vector<int32_t> ids(host_pages, host_pages + need);
    std::sort(ids.begin(), ids.end());
    for (size_t i = 1; i < ids.size(); ++i)
        if (ids[i] == ids[i - 1]) return fail(OC_ERANGE, "page id " + std::to_string(ids[i]) + " repeats");
    return OC_OK;
}

int oc_block_table_check(const int32_t *host_pages, int64_t num_entries, int64_t num_tokens, int64_t num_pages,
                         int32_t page_size) {
    return guarded([&] { return block_table_check_body(host_pages, num_entries, num_tokens, num_pages, page_size); });
}

static int kv_layer_ingest_body(const oc_staging *staging, const oc_block_table *block_table, oc_kv_pool *kv_pool,
                                int32_t layer, void *stream) {
    clear_error();
    if (!staging || !kv_pool) return fail(OC_EINVAL, "staging and kv_pool must not be NULL");
    int rc = check_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    if (layer < 0 || layer >= l.num_layers) return fail(OC_ERANGE, "layer out of range");
    if ((rc = check_staging_shape(l, block_table, staging->num_chunks, staging->per_layer_chunk_bytes))) return rc;
    if ((rc = check_copy_pieces(block_table->num_tokens * 2 * l.num_kv_heads * (l.head_dim / 8), "layer payload")))
        return rc;
    if (block_table->num_tokens == 0) return OC_OK;
    if (!staging->data || !kv_pool->base) return fail(OC_EINVAL, "NULL data or pool base");
    if (!aligned(staging->data, 16) || !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "staging data and pool base must be 16-byte aligned");
    IngestArgs a = ingest_args(kv_pool, block_table, layer, staging->data);
    const int64_t n_pages = (block_table->num_tokens + l.page_size - 1) / l.page_size;
    OC_HIP(launch_ingest(a, n_pages, static_cast<hipStream_t>(stream), false));
    return OC_OK;
}

int oc_kv_layer_ingest(const oc_staging *staging, const oc_block_table *block_table, oc_kv_pool *kv_pool,
                       int32_t layer, void *stream) {
    return guarded([&] { return kv_layer_ingest_body(staging, block_table, kv_pool, layer, stream); });
}

static int kv_chunks_ingest_body(const oc_staging *objects, int64_t first_chunk, const oc_block_table *block_table,
                                 oc_kv_pool *kv_pool, void *stream) {
    clear_error();
    if (!objects || !kv_pool) return fail(OC_EINVAL, "objects and kv_pool must not be NULL");
    int rc = check_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    const int64_t S = 2LL * l.chunk_tokens * l.num_kv_heads * l.head_dim * 2;
    if (objects->per_layer_chunk_bytes != S)
        return fail(OC_ESHAPE, "per_layer_chunk_bytes must equal 2*G*n_kv*d*2 = " + std::to_string(S));
    if (first_chunk < 0 || objects->num_chunks < 0) return fail(OC_EINVAL, "negative first_chunk or num_chunks");
    if ((first_chunk + objects->num_chunks) * l.chunk_tokens > block_table->num_tokens)
        return fail(OC_ERANGE, "chunks past the end of the block table's prefix");
    if ((rc = check_copy_pieces(objects->num_chunks * l.chunk_tokens * 2 * l.num_kv_heads * (l.head_dim / 8),
                                "chunk objects of one layer")))
        return rc;
    if (objects->num_chunks == 0) return OC_OK;
    if (!objects->data || !kv_pool->base) return fail(OC_EINVAL, "NULL data or pool base");
    if (!aligned(objects->data, 16) || !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "object data and pool base must be 16-byte aligned");
    IngestArgs a = chunks_ingest_args(kv_pool, block_table, objects->data, first_chunk, objects->num_chunks);
    OC_HIP(launch_chunks_ingest(a, static_cast<hipStream_t>(stream)));
    return OC_OK;
}

int oc_kv_chunks_ingest(const oc_staging *objects, int64_t first_chunk, const oc_block_table *block_table,
                        oc_kv_pool *kv_pool, void *stream) {
    return guarded([&] { return kv_chunks_ingest_body(objects, first_chunk, block_table, kv_pool, stream); });
}

static int kv_layer_gather_body(const oc_block_table *block_table, const oc_kv_pool *kv_pool, int32_t layer,
                                void *staging_out, int64_t num_chunks, int64_t per_layer_chunk_bytes, void *stream) {
    clear_error();
    if (!kv_pool) return fail(OC_EINVAL, "kv_pool must not be NULL");
    int rc = check_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    if (layer < 0 || layer >= l.num_layers) return fail(OC_ERANGE, "layer out of range");
    if ((rc = check_staging_shape(l, block_table, num_chunks, per_layer_chunk_bytes))) return rc;
    if ((rc = check_copy_pieces(block_table->num_tokens * 2 * l.num_kv_heads * (l.head_dim / 8), "layer payload")))
        return rc;
    if (block_table->num_tokens == 0) return OC_OK;
    if (!staging_out || !kv_pool->base) return fail(OC_EINVAL, "NULL staging_out or pool base");
    if (!aligned(staging_out, 16) || !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "staging and pool base must be 16-byte aligned");
    IngestArgs a = ingest_args(kv_pool, block_table, layer, nullptr);
    OC_HIP(launch_gather(a, static_cast<uint16_t *>(staging_out), static_cast<hipStream_t>(stream)));
    return OC_OK;
}

int oc_kv_layer_gather(const oc_block_table *block_table, const oc_kv_pool *kv_pool, int32_t layer,
                       void *staging_out, int64_t num_chunks, int64_t per_layer_chunk_bytes, void *stream) {
    return guarded([&] {
        return kv_layer_gather_body(block_table, kv_pool, layer, staging_out, num_chunks, per_layer_chunk_bytes,
                                    stream);
    });
}

static int kv_chunks_gather_body(const oc_block_table *block_table, const oc_kv_pool *kv_pool, int64_t first_chunk,
                                 int64_t num_chunks, void *objects_out, void *stream) {
    clear_error();
    if (!kv_pool) return fail(OC_EINVAL, "kv_pool must not be NULL");
    int rc = check_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    if (first_chunk < 0 || num_chunks < 0) return fail(OC_EINVAL, "negative first_chunk or num_chunks");
    if ((first_chunk + num_chunks) * l.chunk_tokens > block_table->num_tokens)
        return fail(OC_ERANGE, "chunks past the end of the block table's tokens");
    if ((rc = check_copy_pieces(num_chunks * l.chunk_tokens * 2 * l.num_kv_heads * (l.head_dim / 8),
                                "chunk objects of one layer")))
        return rc;
    if (num_chunks == 0) return OC_OK;
    if (!objects_out || !kv_pool->base) return fail(OC_EINVAL, "NULL objects_out or pool base");
    if (!aligned(objects_out, 16) || !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "objects_out and pool base must be 16-byte aligned");
    IngestArgs a = chunks_ingest_args(kv_pool, block_table, nullptr, first_chunk, num_chunks);
    OC_HIP(launch_gather(a, static_cast<uint16_t *>(objects_out), static_cast<hipStream_t>(stream)));
    return OC_OK;
}

int oc_kv_chunks_gather(const oc_block_table *block_table, const oc_kv_pool *kv_pool, int64_t first_chunk,
                        int64_t num_chunks, void *objects_out, void *stream) {
    return guarded([&] {
        return kv_chunks_gather_body(block_table, kv_pool, first_chunk, num_chunks, objects_out, stream);
    });
}

static int rest_of_layer_body(const void *attn_out, int64_t tokens, const oc_layout *layout,
                              const oc_layer_weights *weights, int32_t layer, const oc_layer_buffers *buffers,
                              void *stream) {
    clear_error();
    if (!layout) return fail(OC_EINVAL, "layout is NULL");
    int rc = check_layout(*layout);
    if (rc) return rc;
    if ((rc = check_layer_weights(*layout, weights))) return rc;
    if (layer < 0 || layer >= layout->num_layers) return fail(OC_ERANGE, "layer out of range");
    if (tokens < 0) return fail(OC_EINVAL, "negative tokens");
    if (tokens > INT32_MAX / 2) return fail(OC_ERANGE, "too many tokens");
    if (tokens == 0) return OC_OK;
    if (!attn_out) return fail(OC_EINVAL, "attn_out is NULL");
    if (!aligned(attn_out, 16)) return fail(OC_EALIGN, "attn_out must be 16-byte aligned");
    if ((rc = check_layer_buffers(buffers))) return rc;
    LayerArgs a = layer_args(*layout, *weights, layer, attn_out, tokens, *buffers);
    return launch_rest_of_layer(a, static_cast<hipStream_t>(stream));
}

int oc_rest_of_layer(const void *attn_out, int64_t tokens, const oc_layout *layout, const oc_layer_weights *weights,
                     int32_t layer, const oc_layer_buffers *buffers, void *stream) {
    return guarded([&] { return rest_of_layer_body(attn_out, tokens, layout, weights, layer, buffers, stream); });
}

static int kv_suffix_append_body(const void *k_new, const void *v_new, int64_t suffix_tokens,
                                 const oc_block_table *block_table, oc_kv_pool *kv_pool, int32_t layer, void *stream) {
    clear_error();
    if (!kv_pool) return fail(OC_EINVAL, "kv_pool must not be NULL");
    int rc = check_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    if (layer < 0 || layer >= l.num_layers) return fail(OC_ERANGE, "layer out of range");
    if (suffix_tokens < 0) return fail(OC_EINVAL, "negative suffix_tokens");
    if ((rc = check_append_table(block_table, l, suffix_tokens))) return rc;
    if ((rc = check_copy_pieces(suffix_tokens * l.num_kv_heads * (l.head_dim / 8), "suffix K/V"))) return rc;
    if (suffix_tokens == 0) return OC_OK;
    if (!k_new || !v_new || !kv_pool->base) return fail(OC_EINVAL, "NULL k_new, v_new or pool base");
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "k_new, v_new and pool base must be 16-byte aligned");
    AppendArgs a = append_args(kv_pool, block_table, layer, k_new, v_new, suffix_tokens);
    OC_HIP(launch_append(a, static_cast<hipStream_t>(stream)));
    return OC_OK;
}

int oc_kv_suffix_append(const void *k_new, const void *v_new, int64_t suffix_tokens,
                        const oc_block_table *block_table, oc_kv_pool *kv_pool, int32_t layer, void *stream) {
    return guarded([&] {
        return kv_suffix_append_body(k_new, v_new, suffix_tokens, block_table, kv_pool, layer, stream);
    });
}

size_t oc_attention_workspace_bytes(const oc_layout *layout, int64_t prefix_tokens, int64_t suffix_tokens) {
    clear_error();
    if (!layout) {
        fail(OC_EINVAL, "layout is NULL");
        return 0;
    }
    if (check_attention_args(*layout, prefix_tokens, suffix_tokens)) return 0;
    AttnPlan p;
    plan_attention(*layout, prefix_tokens, suffix_tokens, &p);
    return p.total;
}

}  // extern "C"

namespace oc {

// Checks of one layer's attention call apart from its workspace; on OC_OK
// `plan` holds the launch plan.
static int check_attention_call(const void *q, const void *k_new, const void *v_new, int64_t suffix_tokens,
                                const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer,
                                void *out, AttnPlan *plan) {
    if (!kv_pool) return fail(OC_EINVAL, "kv_pool must not be NULL");
    int rc = check_attention_layout(kv_pool->layout);
    if (rc) return rc;
    const oc_layout &l = kv_pool->layout;
    if ((rc = check_table(block_table, l))) return rc;
    if (layer < 0 || layer >= l.num_layers) return fail(OC_ERANGE, "layer out of range");
    if (suffix_tokens < 1) return fail(OC_EINVAL, "suffix_tokens must be >= 1");
    if ((rc = check_attention_shape(l, block_table->num_tokens, suffix_tokens))) return rc;
    if (!q || !k_new || !v_new || !out) return fail(OC_EINVAL, "NULL tensor");
    if (block_table->num_tokens > 0 && !kv_pool->base) return fail(OC_EINVAL, "NULL pool base");
    if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(out, 16) ||
        !aligned(kv_pool->base, 16))
        return fail(OC_EALIGN, "q, k_new, v_new, out and pool base must be 16-byte aligned");
    plan_attention(l, block_table->num_tokens, suffix_tokens, plan);
    return OC_OK;
}

static int enqueue_attention(const AttnPlan &p, const void *q, const void *k_new, const void *v_new,
                             const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer, void *out,
                             void *workspace, hipStream_t stream) {
    const oc_layout &l = kv_pool->layout;
    AttnArgs a{};
    const int64_t block = (int64_t)l.num_kv_heads * l.page_size * l.head_dim;
    const uint16_t *base = static_cast<const uint16_t *>(kv_pool->base);
    a.q = static_cast<const uint16_t *>(q);
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.pool_k = base + ((int64_t)layer * 2 + 0) * l.num_pages * block;
    a.pool_v = base + ((int64_t)layer * 2 + 1) * l.num_pages * block;
    a.pages = block_table->pages;
    a.out = static_cast<uint16_t *>(out);
    a.ws = static_cast<unsigned char *>(workspace);
    OC_HIP(launch_attention(p, a, stream));
    return OC_OK;
}

}  // namespace oc

extern "C" {

static int suffix_prefill_layer_body(const void *q, const void *k_new, const void *v_new, int64_t suffix_tokens,
                                     const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer, void *out,
                                     void *workspace, size_t workspace_bytes, void *stream) {
    clear_error();
    AttnPlan p;
    int rc = check_attention_call(q, k_new, v_new, suffix_tokens, kv_pool, block_table, layer, out, &p);
    if (rc) return rc;
    if (!workspace) return fail(OC_EINVAL, "NULL workspace");
    if (!aligned(workspace, 256)) return fail(OC_EALIGN, "workspace must be 256-byte aligned");
    if (workspace_bytes < p.total)
        return fail(OC_EINVAL, "workspace too small: need " + std::to_string(p.total) + " bytes");
    return enqueue_attention(p, q, k_new, v_new, kv_pool, block_table, layer, out, workspace,
                             static_cast<hipStream_t>(stream));
}

int oc_suffix_prefill_layer(const void *q, const void *k_new, const void *v_new, int64_t suffix_tokens,
                            const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer, void *out,
                            void *workspace, size_t workspace_bytes, void *stream) {
    return guarded([&] {
        return suffix_prefill_layer_body(q, k_new, v_new, suffix_tokens, kv_pool, block_table, layer, out, workspace,
                                         workspace_bytes, stream);
    });
}

static int suffix_prefill_layer_noalloc_body(const void *q, const void *k_new, const void *v_new, int64_t suffix_tokens,
                                             const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer,
                                             void *out, void *stream) {
    clear_error();
    AttnPlan p;
    int rc = check_attention_call(q, k_new, v_new, suffix_tokens, kv_pool, block_table, layer, out, &p);
    if (rc) return rc;
    if (p.total > OC_NOALLOC_WORKSPACE_BYTES)
        return fail(OC_ERANGE, "this shape needs " + std::to_string(p.total) +
                                   " bytes of workspace; the static workspace holds " +
                                   std::to_string((size_t)OC_NOALLOC_WORKSPACE_BYTES));
    void *ws = nullptr;
    if ((rc = scratch_on_current_device(&ws))) return rc;
    return enqueue_attention(p, q, k_new, v_new, kv_pool, block_table, layer, out, ws,
                             static_cast<hipStream_t>(stream));
}

int oc_suffix_prefill_layer_noalloc(const void *q, const void *k_new, const void *v_new, int64_t suffix_tokens,
                                    const oc_kv_pool *kv_pool, const oc_block_table *block_table, int32_t layer,
                                    void *out, void *stream) {
    return guarded([&] {
        return suffix_prefill_layer_noalloc_body(q, k_new, v_new, suffix_tokens, kv_pool, block_table, layer, out,
                                                 stream);
    });
}

}  // extern "C"
