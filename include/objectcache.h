/*
 * objectcache.h -- C ABI of the MI355X layerwise prefix-KV library.
 *
 * A reused prefix KV cache arrives one layer at a time as a single contiguous,
 * layer-major payload (the storage server's per-layer aggregation of all
 * matched chunk objects, Section 3.3 of the ObjectCache paper).  This library
 * unpacks each layer payload into a paged KV pool through a block table and
 * runs the suffix-prefill GQA attention of that layer over the cached prefix
 * plus the new suffix tokens, while the next layer is still landing
 * (layerwise prefetch, Section 3.5, eq. (3)).
 *
 * Conventions for every entry point:
 *   - Element type is bfloat16 (2 bytes) for K, V, Q and outputs; the paper's
 *     eq. (1) uses p = 2 bytes per element.
 *   - Device pointers are HIP device memory owned by the caller; they must
 *     stay valid until the stream the call was enqueued on is synchronised.
 *     Host pointers are read during the call only, except where stated.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Single-layer calls are asynchronous on that stream.
 *   - Return value: OC_OK (0) or a negative oc_status.  Arguments are fully
 *     validated before anything is launched; on error nothing is enqueued and
 *     oc_last_error() returns a message (thread-local, valid until the next
 *     call on the same thread).  No C++ exception crosses this boundary.
 *   - The library never allocates device memory inside the single-layer
 *     calls; scratch space is the caller's `workspace` (or, for
 *     oc_suffix_prefill_layer_noalloc, a static device array).
 *   - Lengths are validated against the kernels' 32-bit index arithmetic as
 *     well: a shape whose offsets, rows or grid would not fit is OC_ERANGE.
 */
#ifndef OBJECTCACHE_H
#define OBJECTCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OC_ABI_VERSION 6

typedef enum {
    OC_OK = 0,
    OC_EINVAL = -1,    /* null pointer, bad enum, negative size            */
    OC_ESHAPE = -2,    /* shapes disagree (S != 2*G*n_kv*d*2, n_q % n_kv)  */
    OC_EALIGN = -3,    /* pointer not 16-byte aligned                      */
    OC_ERANGE = -4,    /* layer or page index out of range, table too short */
    OC_EHIP = -5,      /* the HIP runtime reported an error                */
    OC_ETIMEOUT = -6,  /* a layer did not arrive within the timeout        */
    OC_ENOMEM = -7,    /* host/pinned/device allocation failed (contexts)  */
    OC_EABORT = -8,    /* the producer stopped before delivering a layer   */
    OC_ESHORT = -9     /* a delivered payload is shorter than the layer    */
} oc_status;

/* Model and paging layout (Section 2.1, eq. (1); Table "ObjectCache request
 * descriptor" fields num_layers L and chunk_tokens G).  The per-layer chunk
 * slice is S = 2 * G * n_kv * d * 2 bytes. */
typedef struct {
    int32_t num_layers;     /* L                                              */
    int32_t num_q_heads;    /* n_q, a multiple of n_kv (GQA)                  */
    int32_t num_kv_heads;   /* n_kv                                           */
    int32_t head_dim;       /* d, 64 or 128                                   */
    int32_t page_size;      /* tokens per pool page, a multiple of 8          */
    int32_t chunk_tokens;   /* G, tokens per stored chunk                     */
    int64_t num_pages;      /* P, pages in the pool                           */
} oc_layout;

/* Paged KV pool, device memory of L*2*P*n_kv*page_size*d bfloat16 values laid
 * out [L][2][P][n_kv][page_size][d]: per layer the K region then the V
 * region; each (page, head) block holds its slots in order, one d-element
 * row per slot, for K and V alike.  16-byte aligned. */
typedef struct {
    void *base;
    oc_layout layout;
} oc_kv_pool;

/* Block table of one request: device int32 page ids.  Logical prefix token T
 * lives in page pages[T / page_size] at slot T % page_size.  num_tokens is the
 * cached prefix length; num_entries >= ceil(num_tokens / page_size).  Page ids
 * must be distinct and in [0, P); the kernels trust them (validate with
 * oc_block_table_check when the table is not trusted). */
typedef struct {
    const int32_t *pages;
    int64_t num_entries;
    int64_t num_tokens;
} oc_block_table;

/* One layer's staging payload in device memory (the "client buffer" of the
 * layerwise GET): the concatenation, in prefix order, of the layer slice of
 * each of num_chunks chunk objects.  Each slice is KV_L2TD (Section 3.3):
 * the K matrix then the V matrix, each [G tokens][n_kv heads][d].
 * per_layer_chunk_bytes is S. */
typedef struct {
    const void *data;
    int64_t num_chunks;
    int64_t per_layer_chunk_bytes;
} oc_staging;

/* Library version (OC_ABI_VERSION) */
int oc_abi_version(void);

/* Message for the last failing call on this thread ("" if none). */
const char *oc_last_error(void);

/* Host-side check of a block table held in HOST memory: every entry needed
 * for num_tokens tokens is in [0, P) and no page repeats.  Returns OC_OK or
 * OC_ERANGE. */
int oc_block_table_check(const int32_t *host_pages, int64_t num_entries, int64_t num_tokens,
                         int64_t num_pages, int32_t page_size);

/* Layer ingest (unpack + scatter): copy every K and V row of the staging
 * payload of `layer` into the pool pages named by the block table.
 * Requirements: S == 2*G*n_kv*d*2, num_chunks*G == block_table->num_tokens,
 * 0 <= layer < L, data/base 16-byte aligned.  Bytes are copied exactly (NaN
 * and denormal patterns included); pool slots past the prefix are not
 * written.  Asynchronous on `stream`. */
int oc_kv_layer_ingest(const oc_staging *staging, const oc_block_table *block_table,
                       oc_kv_pool *kv_pool, int32_t layer, void *stream);

/* Chunkwise ingest (the delivery mode of eq. (2) below the threshold, where
 * whole chunk objects arrive instead of layer payloads): scatter every layer
 * of num_chunks consecutive chunk objects of a request into the pool.
 * objects->data holds the objects back to back as stored (each L*S bytes:
 * layer 0's KV_L2TD slice, then layer 1's, ...); they are chunks
 * first_chunk .. first_chunk+num_chunks-1 of the request's prefix, so their
 * tokens are first_chunk*G .. and the block table must cover them
 * (block_table->num_tokens >= (first_chunk+num_chunks)*G).  The pool result
 * equals oc_kv_layer_ingest of every layer payload.  Same alignment and
 * shape requirements as oc_kv_layer_ingest; asynchronous on `stream`. */
int oc_kv_chunks_ingest(const oc_staging *objects, int64_t first_chunk, const oc_block_table *block_table,
                        oc_kv_pool *kv_pool, void *stream);

/* Inverse of the ingest: read the prefix of `layer` out of the pool into a
 * staging-layout device buffer (the layout a chunk object's layer slice has;
 * the write-back direction).  Same requirements as oc_kv_layer_ingest. */
int oc_kv_layer_gather(const oc_block_table *block_table, const oc_kv_pool *kv_pool,
                       int32_t layer, void *staging_out, int64_t num_chunks,
                       int64_t per_layer_chunk_bytes, void *stream);

/* Offload gather (the write-back of chunks to object storage, Section 3
 * opening, and the inverse of oc_kv_chunks_ingest): rebuild chunk objects
 * first_chunk .. first_chunk+num_chunks-1 of a request from the pool, every
 * layer.  objects_out (device, 16-byte aligned, caller-owned) receives them
 * back to back, each L*S bytes in KV_L2TD order (layer 0's slice, then layer
 * 1's, ...).  Their tokens must lie inside the table:
 * (first_chunk+num_chunks)*G <= block_table->num_tokens -- to offload chunks
 * that hold suffix tokens appended with oc_kv_suffix_append, pass a table
 * whose num_tokens counts them.  num_chunks == 0 is not an error.
 * Asynchronous on `stream`. */
int oc_kv_chunks_gather(const oc_block_table *block_table, const oc_kv_pool *kv_pool, int64_t first_chunk,
                        int64_t num_chunks, void *objects_out, void *stream);

/* Suffix append (the prefill node materialising the full KV state, Section 3
 * opening): write one layer's suffix K and V (device [suffix_tokens][n_kv][d]
 * bfloat16 each, 16-byte aligned) into the pool behind the prefix: token i
 * goes to logical position T_p + i (T_p = block_table->num_tokens), i.e. page
 * pages[(T_p+i) / page_size], slot (T_p+i) % page_size.  The table must hold
 * ceil((T_p+suffix_tokens)/page_size) entries.  Prefix slots are not
 * touched.  suffix_tokens == 0 is not an error.  Asynchronous on `stream`. */
int oc_kv_suffix_append(const void *k_new, const void *v_new, int64_t suffix_tokens,
                        const oc_block_table *block_table, oc_kv_pool *kv_pool, int32_t layer, void *stream);

/* Bytes of device workspace oc_suffix_prefill_layer needs for these lengths
 * (at least 256; 0 means the layout or lengths are not supported). */
size_t oc_attention_workspace_bytes(const oc_layout *layout, int64_t prefix_tokens,
                                    int64_t suffix_tokens);

/* Suffix-prefill GQA attention of one layer (the compute the miss tokens
 * expose per layer, Section 3.5):
 *   out[i][h][:] = sum_j softmax_j(q[i][h].k_j[g] / sqrt(d)) v_j[g],
 *   g = h / (n_q / n_kv), j over the prefix tokens 0..T_p-1 read from the pool
 *   through the block table (T_p = block_table->num_tokens), then the suffix
 *   tokens 0..i from k_new/v_new (causal within the suffix).
 * q, out: device [suffix_tokens][n_q][d]; k_new, v_new: device
 * [suffix_tokens][n_kv][d]; bfloat16, 16-byte aligned.  Scores and
 * accumulation are fp32; out is rounded to bfloat16 (nearest even).
 * workspace: device, at least oc_attention_workspace_bytes(), 256-byte
 * aligned.  suffix_tokens >= 1.  Asynchronous on `stream`.  The kernel's
 * wavefronts raise their issue priority (s_setprio 1, 2 in the matrix
 * phases), so kernels at the default priority that share its compute units,
 * such as the pipeline's ingest, issue after it. */
int oc_suffix_prefill_layer(const void *q, const void *k_new, const void *v_new,
                            int64_t suffix_tokens, const oc_kv_pool *kv_pool,
                            const oc_block_table *block_table, int32_t layer, void *out,
                            void *workspace, size_t workspace_bytes, void *stream);

/* Bytes of the static device workspace behind oc_suffix_prefill_layer_noalloc.
 * Every shape oc_suffix_prefill_layer accepts needs at most about 64.9 MiB of
 * workspace (fewer than 512 (row tile, key split) pairs of 130 KiB each at
 * head_dim 128), so this holds the workspace of every accepted shape. */
#define OC_NOALLOC_WORKSPACE_BYTES ((size_t)65 << 20)

/* oc_suffix_prefill_layer for callers that cannot allocate device memory or
 * pass a workspace: code under stream capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Same arguments (less the workspace), same checks,
 * same kernels and bit-identical output.  The split partials go to a static
 * device array of OC_NOALLOC_WORKSPACE_BYTES that every GPU the library runs
 * on holds from its first call there until the process ends; the call
 * allocates nothing.  It runs on the calling thread's current device, and
 * `stream` must belong to it.  Calls on one GPU share that array: two calls
 * whose kernels overlap in time (on different streams, or from different
 * threads without ordering) race and corrupt each other's output; calls in
 * order on one stream are safe.  Nothing in the array needs to start at zero
 * (every partial the merge reads is first written by the same call), and it
 * keeps the last call's partials.  A shape whose workspace exceeds
 * OC_NOALLOC_WORKSPACE_BYTES is OC_ERANGE (none of the accepted shapes does).
 * Asynchronous on `stream`. */
int oc_suffix_prefill_layer_noalloc(const void *q, const void *k_new, const void *v_new,
                                    int64_t suffix_tokens, const oc_kv_pool *kv_pool,
                                    const oc_block_table *block_table, int32_t layer, void *out,
                                    void *stream);

/* Rest-of-layer compute window (the C_l of eq. (3): the compute the miss
 * tokens expose per layer, Section 3.5; every layer runs the same
 * projections and feed-forward network, Section 3.6).  A Llama-style layer
 * around the attention, on T suffix tokens, bf16 with fp32 accumulation:
 *   o    = attn_out . W_o           [T][H]        H = n_q * d
 *   gu   = o . W_gate_up            [T][2F]       gate columns, then up columns
 *   act  = silu(gate) * up          [T][F]        silu(x) = x / (1 + e^-x), fp32
 *   h    = act . W_down             [T][H]
 *   qkv  = h . W_qkv                [T][(n_q + 2 n_kv) d]   the next layer's projection
 * Each stage is rounded to bf16 (nearest even).  Norms, residuals and biases
 * are left out.  The GEMMs run in rocBLAS, the gating in a kernel of this
 * library.  Weights are device bf16, [K][N] row-major (input features by
 * output features), one matrix per layer back to back, 16-byte aligned;
 * caller-owned and only read. */
typedef struct {
    int32_t ffn_dim;           /* F, a multiple of 8                                     */
    const void *w_o;           /* [L][H][H]                                              */
    const void *w_gate_up;     /* [L][H][2F]                                             */
    const void *w_down;        /* [L][F][H]                                              */
    const void *w_qkv;         /* [L][H][(n_q + 2 n_kv) d]                               */
} oc_layer_weights;

/* Device outputs of the chain's stages for T rows (caller-owned, 16-byte
 * aligned, shapes as above). */
typedef struct {
    void *o;
    void *gate_up;
    void *act;
    void *h;
    void *qkv;
} oc_layer_buffers;

/* The chain above for one layer; attn_out is device bf16 [tokens][H] (the
 * attention output, as oc_suffix_prefill_layer writes it).  tokens == 0 is
 * not an error.  Asynchronous on `stream`; the first call on a stream
 * creates the GEMM library's handle for it (which may allocate). */
int oc_rest_of_layer(const void *attn_out, int64_t tokens, const oc_layout *layout,
                     const oc_layer_weights *weights, int32_t layer, const oc_layer_buffers *buffers,
                     void *stream);

/* ---------------------------------------------------------------------------
 * Layerwise pipeline (Section 3.5, eq. (3)): for every layer, the payload
 * lands (host producer -> pinned slot -> DMA into an HBM slot), is ingested
 * into the pool, and the layer's attention runs on a second stream as soon
 * as that layer is in; layer l+1 lands and is ingested while layer l
 * computes.  The producer stands in for the storage server's layerwise GET:
 * it assembles each layer payload from the chunk objects in prefix order
 * (appendix pseudocode "layerwise GET"), paced to a byte rate, and signals
 * layer-ready.  With several requests sharing one rate (OC_ALLOC_FIFO),
 * layers are delivered layer-major, request-minor (round-robin); with an
 * allocation policy each request gets its own rate, fixed from its admission
 * until its deliveries end: requests that arrive at the start share one
 * scheduling epoch, later ones are admitted at later boundaries with the
 * budget then free (oc_epoch_schedule), and the producer dispatches the
 * admitted requests' payload pieces by weighted deficit round robin
 * (Section 3.6 and its appendix pseudocode).
 * A request delivered chunkwise (eq. (2)) instead receives its whole chunk
 * objects in prefix order, as many per staging slot as fit; each group is
 * landed and ingested with oc_kv_chunks_ingest, and its L layers' attention
 * runs once the last group is in.  Chunkwise requests are delivered before
 * the layerwise ones share the rate; they take OC_ALLOC_FIFO only (the
 * allocation policies schedule layerwise requests, Section 3.4).
 * ------------------------------------------------------------------------- */

/* Per-request bandwidth under a shared cap (Section 3.6; the baselines of the
 * multi-tenant evaluation).  Request i moves s_i bytes per layer and has a
 * compute window of c_i seconds per layer; r*_i = s_i / c_i is its zero-stall
 * rate (eq. (4)). */
typedef enum {
    OC_ALLOC_FIFO = 0,          /* no per-request rates: one shared stream            */
    OC_ALLOC_EQUAL = 1,         /* B / n each                                           */
    OC_ALLOC_KV_PROP = 2,       /* proportional to s_i                                  */
    OC_ALLOC_BW_PROP = 3,       /* proportional to r*_i                                 */
    OC_ALLOC_STALL_OPT = 4,     /* eqs. (5)-(6): min sum s_i/r_i, sum r_i = B, r_i <= r*_i */
    OC_ALLOC_CAL_STALL_OPT = 5  /* eq. (7): the same with r_i <= r*_i + margin          */
} oc_alloc_policy;

/* Host-only: rates_out[i] (bytes/s) for n requests under budget B (bytes/s).
 * layer_bytes[i] = s_i > 0; layer_compute_s[i] = c_i > 0 (needed by BW_PROP,
 * STALL_OPT, CAL_STALL_OPT; may be NULL otherwise); margin = delta >= 0 (used by
 * CAL_STALL_OPT).  Stall-opt policies leave budget unassigned when every
 * request's cap fits.  Returns OC_OK, or OC_EINVAL for bad input or
 * OC_ALLOC_FIFO.  Arrays are caller-owned; nothing is retained. */
int oc_bandwidth_allocate(int32_t policy, int32_t n, const double *layer_bytes,
                          const double *layer_compute_s, double budget_bytes_per_s,
                          double margin_bytes_per_s, double *rates_out);

/* Host-only: the scheduling epochs of Section 3.6 for requests that arrive
 * over time.  Request i arrives at arrival_s[i] (seconds, >= 0) and moves
 * num_layers payloads of layer_bytes[i].  At each epoch boundary the requests
 * that have arrived and wait are admitted together; they share, under
 * `policy` (as oc_bandwidth_allocate), the budget the admitted requests still
 * in flight do not hold.  An admitted request keeps its rate until its
 * deliveries end (admission + num_layers * layer_bytes[i] / rate); the rate it
 * then releases goes to requests admitted at a later boundary, never to one
 * already in flight.  Boundaries are the multiples of epoch_s (> 0), or, with
 * epoch_s == 0, every arrival and every end of a delivery.  Outputs:
 * rates_out[i] (bytes/s) and admit_s_out[i] (the boundary at which request i
 * was admitted).  Same argument rules as oc_bandwidth_allocate, plus
 * num_layers >= 1, finite arrival_s >= 0 and epoch_s >= 0; OC_EINVAL
 * otherwise.  Arrays are caller-owned; nothing is retained. */
int oc_epoch_schedule(int32_t policy, int32_t n, const double *layer_bytes, const double *layer_compute_s,
                      int32_t num_layers, const double *arrival_s, double budget_bytes_per_s,
                      double margin_bytes_per_s, double epoch_s, double *rates_out, double *admit_s_out);

typedef enum {
    OC_MODE_HBM_RESIDENT = 0,  /* pool already holds the prefix: attention only          */
    OC_MODE_DEVICE_STAGED = 1, /* payloads already in HBM: ingest + attention, 2 streams  */
    OC_MODE_PRODUCER = 2       /* host producer -> pinned -> HBM -> ingest -> attention   */
} oc_mode;

typedef enum {
    OC_FAULT_NONE = 0,
    OC_FAULT_STALL = 1,        /* producer stops delivering at fault_layer (tests timeouts) */
    OC_FAULT_ABORT = 2,        /* producer gives up at fault_layer (tests error paths)      */
    OC_FAULT_SHORT_WRITE = 3   /* producer's payload for fault_layer ends half a chunk slice
                                  early (a torn object read); tests the length check        */
} oc_fault;

/* Delivery of a request's cached prefix (eq. (2), Section 3.4).  The
 * storage layout is always chunkwise; the delivery order is the choice. */
typedef enum {
    OC_DELIVERY_LAYERWISE = 0, /* per-layer payloads; layer l computes while l+1 lands  */
    OC_DELIVERY_CHUNKWISE = 1, /* whole chunk objects in prefix order; compute starts
                                  after the last one is in (the chunkwise baseline)      */
    OC_DELIVERY_AUTO = 2       /* eq. (2) per request: chunkwise when W = N*L*S is
                                  below theta_bytes, layerwise otherwise                 */
} oc_delivery;

typedef struct {
    int32_t mode;              /* oc_mode                                                  */
    double rate_bytes_per_s;   /* producer pacing; 0 = as fast as memcpy goes              */
    int64_t piece_bytes;       /* pacing/copy granularity (default 1 MiB when 0)           */
    int32_t slots;             /* pinned and HBM staging slots (>= 2; default 3 when 0)    */
    int32_t producer_threads;  /* memcpy threads (default 4 when 0)                        */
    int32_t timeout_ms;        /* wait limit per layer (default 60000 when 0)              */
    int32_t fault;             /* oc_fault, test injection                                 */
    int32_t fault_layer;       /* layer at which the fault triggers                        */
    int32_t alloc_policy;      /* oc_alloc_policy (PRODUCER mode); budget = rate_bytes_per_s */
    double margin_bytes_per_s; /* delta of OC_ALLOC_CAL_STALL_OPT                          */
    int32_t delivery;          /* oc_delivery, PRODUCER mode only (other modes: layerwise) */
    double theta_bytes;        /* Theta of OC_DELIVERY_AUTO                                */
    int32_t emulate_compute;   /* nonzero: each request computes on a stream of its own,
                                  and after each layer's attention that stream is held
                                  for the request's layer_compute_s -- a stand-in for the
                                  rest of the model's per-layer compute, so eq. (3)'s
                                  window C_l can be set; windows of different requests
                                  overlap (at most 10 s per layer) as long as their
                                  streams get hardware queues of their own
                                  (GPU_MAX_HW_QUEUES >= requests + 2)                      */
    int32_t append_suffix;     /* nonzero: after each layer's attention, append that
                                  layer's suffix K/V into the pool behind the prefix
                                  (oc_kv_suffix_append), so the run leaves the full KV
                                  state; every block table must then hold
                                  ceil((T_p+T_s)/page_size) entries                       */
    int32_t attention_per_request;
                               /* nonzero: one attention launch per request and layer,
                                  planned as oc_suffix_prefill_layer plans it.  Otherwise,
                                  when 2..16 requests are all delivered layer-major on one
                                  schedule (no allocation policy, no chunkwise request, no
                                  emulated windows), each layer's attention is one launch
                                  over all of them after their ingests, with key splits
                                  planned for all their row tiles together               */
    const oc_layer_weights *layer_weights;
                               /* non-NULL: after each layer's attention (and append), run
                                  oc_rest_of_layer on the attention output, on the same
                                  stream, so each layer's window C_l is the whole layer's
                                  compute; the struct is copied at context creation, the
                                  weights must outlive the context                        */
    double epoch_s;            /* with an allocation policy: scheduling epoch length for
                                  requests with arrival_s > 0 (oc_epoch_schedule); 0 = an
                                  epoch begins at every arrival and end of a delivery    */
} oc_pipeline_opts;

/* One request.  Device arrays are [L][...] stacks of the per-layer tensors. */
typedef struct {
    int64_t prefix_tokens;                /* T_p = num_chunks * G                          */
    int64_t suffix_tokens;                /* T_s >= 1                                      */
    const oc_block_table *block_table;    /* device table covering T_p                     */
    const void *const *chunk_objects;     /* PRODUCER: host, num_chunks objects, each L*S
                                             bytes (KV_L2TD, all layers); read during run   */
    const void *device_payload;           /* DEVICE_STAGED: device, L payloads of T_p*b
                                             bytes back to back (b = 2*n_kv*d*2)           */
    const void *q;                        /* device [L][T_s][n_q][d]                       */
    const void *k_new;                    /* device [L][T_s][n_kv][d]                      */
    const void *v_new;                    /* device [L][T_s][n_kv][d]                      */
    void *out;                            /* device [L][T_s][n_q][d]                       */
    double layer_compute_s;               /* c_i for the allocation policies (seconds per
                                             layer), and the emulated window with
                                             emulate_compute; otherwise ignored             */
    double arrival_s;                     /* seconds after the run starts at which the
                                             request arrives; > 0 only with an allocation
                                             policy (its rate and admission then follow
                                             oc_epoch_schedule)                             */
} oc_request;

/* Per-request timings (milliseconds from the start of the run, all on one
 * clock).  Arrays, when non-NULL, are caller-owned with num_layers entries.
 * For a request delivered chunkwise, produced/landed/ingested of every layer
 * are those of its last chunk group (the time every layer became usable). */
typedef struct {
    double ttft_ms;            /* arrival -> this request's last layer done        */
    double *produced_ms;       /* host: layer payload fully in its pinned slot     */
    double *landed_ms;         /* device: payload in HBM (layer-ready)             */
    double *ingested_ms;       /* device: ingest kernel finished                   */
    double *done_ms;           /* device: attention finished                       */
    double rate_bytes_per_s;   /* the request's allocated rate (0 under FIFO)      */
    int32_t delivery;          /* the delivery the request got (oc_delivery)       */
    double admitted_ms;        /* the epoch boundary at which the request was
                                  admitted (its deliveries are paced from there)  */
} oc_request_stats;

/* Create a context on `device` for one pool.  Allocates the streams, events,
 * the attention workspace for up to max_prefix_tokens / max_suffix_tokens
 * and, in PRODUCER mode, the pinned and HBM staging rings (`slots` slots
 * each, a slot holding the largest layer payload, max_prefix_tokens * b
 * bytes, or one whole chunk object if that is larger and the delivery may be
 * chunkwise), and keeps them until oc_context_destroy.  The staging ring is
 * touched once before the call returns (every pinned page written by the
 * host, every slot copied to HBM once), so that the first run does not pay
 * for the first use of fresh pinned memory; this takes about 0.1 s for a
 * ring of 3 x 256 MiB.  The pool stays caller-owned.  An
 * absent device is OC_EINVAL.  Context calls make `device` current while they
 * run and give the caller its current device back. */
int oc_context_create(int device, const oc_kv_pool *kv_pool, const oc_pipeline_opts *opts,
                      int64_t max_prefix_tokens, int64_t max_suffix_tokens, void **ctx);

/* Run the pipeline over n_reqs requests for all L layers; synchronous.
 * A context serves one run at a time; runs on different contexts may
 * overlap, from different host threads (each context has its own streams,
 * staging and producer threads).
 * stats (optional) has n_reqs entries.  On OC_ETIMEOUT / OC_EABORT the run is
 * stopped, all enqueued GPU work is drained and the context stays usable.
 * Once the producer completes a payload, the byte count it reports is
 * checked against the layer's size (prefix_tokens * 2 * n_kv * d * 2, or the
 * chunk group's objects): a short payload is never ingested (its leading
 * pieces may have been copied to the HBM staging slot); the run stops with
 * OC_ESHORT, drained, the context usable.  Layers ingested before it stay in
 * the pool.  With OC_ALLOC_FIFO and a rate cap, a layer payload is copied to
 * HBM in spans (an eighth of the layer, at least 8 MiB) as its leading bytes
 * complete; the ingest waits for the whole layer.  With the library built
 * against roctx, each run and each layer's enqueue on the driver thread is a
 * named range ("oc_pipeline_run", "layer <l> req <r>"), and the producer
 * marks each payload it completes ("ready layer <l> req <r>"), so a
 * rocprofv3 --marker-trace timeline shows delivery against the kernels.
 * The run's GPU work starts after all work enqueued so far on the device's
 * null (legacy default) stream; work on other streams that writes the pool,
 * tables or tensors of reqs must be complete before the call. */
int oc_pipeline_run(void *ctx, const oc_request *reqs, int32_t n_reqs, oc_request_stats *stats);

/* Time of the whole last run (ms, start -> last layer of the last request). */
double oc_pipeline_last_ms(void *ctx);

void oc_context_destroy(void *ctx);

#ifdef __cplusplus
}
#endif
#endif /* OBJECTCACHE_H */
