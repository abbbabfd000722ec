// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <new>
#include <stdexcept>
#include <string>
#include <system_error>

#include "objectcache.h"

namespace oc {

// thread-local error message behind oc_last_error()
void set_error(const std::string &msg);
void clear_error();
int fail(int status, const std::string &msg);
int hip_fail(hipError_t e, const char *what);

// The body of a C entry point, run so that no C++ exception leaves the
// library: host memory that cannot be allocated, or a thread that cannot be
// started, becomes OC_ENOMEM with a message.
template <class F>
int guarded(F &&body) noexcept {
    const char *why;
    try {
        return body();
    } catch (const std::bad_alloc &) {
        why = "out of host memory";
    } catch (const std::length_error &) {
        why = "out of host memory";
    } catch (const std::system_error &) {
        why = "could not start a host thread";
    } catch (...) {
        why = "unexpected C++ exception";
    }
    try {
        set_error(why);
    } catch (...) {
    }
    return OC_ENOMEM;
}

#define OC_HIP(call)                                 \
    do {                                             \
        hipError_t e_ = (call);                      \
        if (e_ != hipSuccess) return oc::hip_fail(e_, #call); \
    } while (0)

inline bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// A dispatch counts the work-items of each grid dimension in 32 bits
// (workgroups x workgroup size).  The copy kernels number their 16-byte
// pieces along x, one per work-item; OC_OK or OC_ERANGE.
constexpr int64_t OC_MAX_GRID_ITEMS = 0xFFFFFFFFLL - 1023;
int check_copy_pieces(int64_t pieces, const char *what);

// ---- ingest / gather ------------------------------------------------------
struct IngestArgs {
    const uint16_t *staging;   // chunk slices [N][2][G][n_kv][d], chunk_stride apart
    uint16_t *pool_k;          // pool + ((layer*2+0)*P) * n_kv * Ps * d
    uint16_t *pool_v;          // pool + ((layer*2+1)*P) * n_kv * Ps * d
    const int32_t *pages;
    int64_t num_tokens;        // tokens in the staging (N * G)
    int32_t G, n_kv, d, Ps;
    // optional (0 = one layer payload): elements from one chunk's slice to the
    // next (a layer payload: 2*G*n_kv*d; whole chunk objects: L times that),
    // the first staged token's index in the prefix, and for whole chunk
    // objects the layer count with the per-layer steps in staging and pool
    int64_t chunk_stride, token0;
    int32_t n_layers;
    int64_t layer_step_staging, layer_step_pool;
    // filled by the launcher
    int64_t region;            // pool_v - pool_k, elements
    int32_t d8, lg_d8, lg_ps, lg_nkv, lg_g;
};
// beside_compute: launched to run next to the attention kernel (more bytes in
// flight per thread) rather than alone on the GPU
hipError_t launch_ingest(IngestArgs a, int64_t n_pages_used, hipStream_t s, bool beside_compute);
// every layer of whole chunk objects (n_layers, layer steps and token0 set)
hipError_t launch_chunks_ingest(IngestArgs a, hipStream_t s);
// arguments for chunks first_chunk .. first_chunk+num_chunks-1 of a request,
// stored back to back as whole objects at `objects`
IngestArgs chunks_ingest_args(const oc_kv_pool *pool, const oc_block_table *bt, const void *objects,
                              int64_t first_chunk, int64_t num_chunks);
// the inverse direction, pool -> `out` laid out as the staging would be (a
// layer payload, or whole chunk objects with n_layers and the steps set)
hipError_t launch_gather(IngestArgs a, uint16_t *out, hipStream_t s);

// ---- suffix append -------------------------------------------------------------
struct AppendArgs {
    const uint16_t *k_new, *v_new;   // [num_tokens][n_kv][d] each
    uint16_t *pool_k, *pool_v;       // the layer's K and V regions
    const int32_t *pages;
    int64_t num_tokens, token0;      // suffix tokens, the first one's logical position
    int32_t n_kv, d, Ps;
    // filled by the launcher
    int64_t region;
    int32_t d8;
};
hipError_t launch_append(AppendArgs a, hipStream_t s);
// OC_OK when bt also holds pages for suffix_tokens tokens behind its prefix
int check_append_table(const oc_block_table *bt, const oc_layout &l, int64_t suffix_tokens);
// arguments for appending `suffix_tokens` tokens of `layer` behind bt->num_tokens
AppendArgs append_args(const oc_kv_pool *pool, const oc_block_table *bt, int32_t layer, const void *k_new,
                       const void *v_new, int64_t suffix_tokens);

// ---- rest-of-layer compute window ---------------------------------------------
struct LayerArgs {
    int64_t T, H, F, NQKV;                           // tokens, n_q*d, ffn_dim, (n_q+2n_kv)*d
    const uint16_t *attn_out;                        // [T][H]
    const uint16_t *w_o, *w_gu, *w_down, *w_qkv;    // this layer's weights, [K][N] row-major
    uint16_t *o, *gu, *act, *h, *qkv;                // outputs of the chain's stages
};
// enqueues O, gate|up, SiLU gating, down and QKV on `s`; an oc_status
int launch_rest_of_layer(const LayerArgs &a, hipStream_t s);
LayerArgs layer_args(const oc_layout &l, const oc_layer_weights &w, int32_t layer, const void *attn_out,
                     int64_t tokens, const oc_layer_buffers &b);
int check_layer_weights(const oc_layout &l, const oc_layer_weights *w);
int check_layer_buffers(const oc_layer_buffers *b);
// bytes of one buffer set for `tokens` rows, and each stage's offset in it
size_t layer_buffer_bytes(const oc_layout &l, int32_t ffn_dim, int64_t tokens, size_t off[5]);
// drop the GEMM library's state bound to a stream about to be destroyed
void forget_blas_stream(hipStream_t s);

// ---- emulated compute window ---------------------------------------------------
// holds stream `s` for `seconds` (at most OC_MAX_WINDOW_S, checked by callers)
hipError_t launch_compute_window(double seconds, hipStream_t s);
constexpr double OC_MAX_WINDOW_S = 10.0;

// ---- attention --------------------------------------------------------------
struct AttnPlan {
    int64_t Tp, Ts;
    int32_t nq, nkv, grp, d;
    int64_t rows;              // Ts * grp rows per KV head
    int32_t m_tiles;           // row tiles per KV head
    int32_t n_split;           // key-range splits
    int64_t n_pre_pages;       // ceil(Tp / 16)
    int64_t n_suf_pages;       // ceil(Ts / 16)
    int64_t n_blocks;          // key blocks of 64 keys over prefix then suffix pages
    int64_t blocks_per_split;
    // workspace carve-up (byte offsets): split partials
    size_t off_o, off_ml, total;
};
int plan_attention(const oc_layout &lay, int64_t Tp, int64_t Ts, AttnPlan *plan);
// Shapes the attention kernels can index: the layout (head_dim 64 or 128,
// page_size 16; OC_ESHAPE otherwise) and the 32-bit limits of their
// arithmetic (OC_ERANGE): suffix K/V byte offsets, key positions, rows and
// the grids of both kernels.
int check_attention_shape(const oc_layout &lay, int64_t Tp, int64_t Ts);
// check_attention_shape after the layout's own checks (positive fields, GQA
// head ratio, alignment multiples)
int check_attention_args(const oc_layout &lay, int64_t Tp, int64_t Ts);
// workgroups of the attention launch of one plan
int64_t attention_grid(const AttnPlan &p);
// at most this many workgroups in one attention launch (all its requests)
int64_t attention_max_grid();
// LDS one attention workgroup holds at this head_dim (0: not supported)
size_t attention_lds_bytes(int head_dim);
// LDS of one compute unit on gfx950
constexpr size_t CU_LDS_BYTES = 160 * 1024;
// one launch for up to MAX_ATTN_BATCH requests of one layer: keys are split
// so that every workgroup gets about the same number of key blocks
constexpr int MAX_ATTN_BATCH = 16;
int plan_attention_batch(const oc_layout &lay, const int64_t *Tp, const int64_t *Ts, int n, AttnPlan *plans);

struct AttnArgs {
    const uint16_t *q, *k_new, *v_new;
    const uint16_t *pool_k, *pool_v;   // layer bases as in IngestArgs
    const int32_t *pages;
    uint16_t *out;
    unsigned char *ws;
};
hipError_t launch_attention(const AttnPlan &p, const AttnArgs &a, hipStream_t s);
// all plans from one plan_attention_batch call, same layout
hipError_t launch_attention_batch(const AttnPlan *plans, const AttnArgs *args, int n, hipStream_t s);

}  // namespace oc
