/*
 * CPU oracle for the layerwise prefix-KV path.  TEST INFRASTRUCTURE ONLY:
 * tests, the smoke check and the benchmark's CPU-baseline leg may call it;
 * the product path never does.  It shares no code with the GPU library.
 *
 * Plain, slow, obviously correct:
 *   - layer assembly: the storage-server readout of one layer across all
 *     matched chunk objects, in prefix order (Section 3.3, "Server-Side Layer
 *     Aggregation", and the layerwise-GET pseudocode in the appendix);
 *   - KV_L2TD decoding: a chunk object stores its layers back to back, each
 *     layer as the K matrix then the V matrix, each matrix token-major with the
 *     hidden dimension (head-major, then head dim) innermost (Section 3.3,
 *     KV_L2TD in Section 3.3; per-layer slice size S of eq. (1));
 *   - paged-pool scatter and gather, one element at a time, through the block
 *     table (the vLLM paged substrate the serving node builds on), and the
 *     write path: the suffix's K/V appended behind the prefix, and whole
 *     chunk objects rebuilt from the pool for offload;
 *   - suffix-prefill GQA attention in float64 over the logical, un-paged keys:
 *     softmax of scaled dot products, each suffix token seeing every cached
 *     prefix token and the suffix tokens up to itself.
 *
 * bfloat16 values travel as uint16 bit patterns and are widened exactly.
 * Pool layout (a design choice; the paper leaves the paged layout to the
 * serving engine):  pool[L][2][P][n_kv][Ps][d] -- for each layer, K then V;
 * each (page, head) block holds its page's slots in order, one d-element row
 * per slot, for K and V alike.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- layer assembly: B_l = concat_j chunk_j[l*S, (l+1)*S) ---------------- */
void oco_assemble_layer(const void *const *chunks, int64_t n_chunks, int64_t slice_bytes,
                        int32_t layer, void *out) {
    unsigned char *dst = (unsigned char *)out;
    for (int64_t j = 0; j < n_chunks; ++j) {
        const unsigned char *obj = (const unsigned char *)chunks[j];
        const unsigned char *src = obj + (int64_t)layer * slice_bytes;
        for (int64_t b = 0; b < slice_bytes; ++b) dst[j * slice_bytes + b] = src[b];
    }
}

/* ---- KV_L2TD element address inside one chunk object ---------------------
 * element (layer l, matrix m in {0=K,1=V}, token t < G, head h, dim e) */
static int64_t l2td_index(int32_t l, int32_t m, int32_t t, int32_t h, int32_t e,
                          int32_t G, int32_t n_kv, int32_t d) {
    int64_t D = (int64_t)n_kv * d;                   /* hidden width of one row */
    return (((int64_t)l * 2 + m) * G + t) * D + (int64_t)h * d + e;
}

/* Logical prefix K and V of one layer, [T][n_kv][d], decoded from chunk objects. */
void oco_logical_kv(const uint16_t *const *chunks, int64_t n_chunks, int32_t G, int32_t n_kv,
                    int32_t d, int32_t layer, uint16_t *k_out, uint16_t *v_out) {
    for (int64_t j = 0; j < n_chunks; ++j)
        for (int32_t t = 0; t < G; ++t)
            for (int32_t h = 0; h < n_kv; ++h)
                for (int32_t e = 0; e < d; ++e) {
                    int64_t T = j * G + t;
                    int64_t o = (T * n_kv + h) * d + e;
                    k_out[o] = chunks[j][l2td_index(layer, 0, t, h, e, G, n_kv, d)];
                    v_out[o] = chunks[j][l2td_index(layer, 1, t, h, e, G, n_kv, d)];
                }
}

/* ---- paged pool addressing ------------------------------------------------ */
static int64_t pool_index(int32_t l, int32_t m, int64_t page, int32_t h, int32_t slot, int32_t e,
                          int64_t P, int32_t n_kv, int32_t Ps, int32_t d) {
    int64_t block = (((int64_t)l * 2 + m) * P + page) * n_kv + h;
    return (block * Ps + slot) * (int64_t)d + e;       /* [slot][dim] for K and V */
}

/* Scatter one layer's staging payload (concatenated layer slices of n_chunks
 * chunk objects, prefix order) into the pool.  Token T = j*G + t of the prefix
 * lands in page table[T / Ps], slot T % Ps.  Returns 0, or -1 when a table
 * entry is outside [0, P). */
static int ingest_chunk_range(const uint16_t *staging, int64_t j0, int64_t j1, int32_t G, int32_t n_kv,
                              int32_t d, int32_t Ps, const int32_t *table, int64_t table_len, uint16_t *pool,
                              int64_t P, int32_t layer) {
    int64_t slice = 2LL * G * n_kv * d;
    for (int64_t j = j0; j < j1; ++j)
        for (int32_t m = 0; m < 2; ++m)
            for (int32_t t = 0; t < G; ++t)
                for (int32_t h = 0; h < n_kv; ++h)
                    for (int32_t e = 0; e < d; ++e) {
                        int64_t T = j * G + t;
                        int64_t q = T / Ps;
                        if (q >= table_len) return -1;
                        int64_t page = table[q];
                        if (page < 0 || page >= P) return -1;
                        int64_t src = j * slice + l2td_index(0, m, t, h, e, G, n_kv, d);
                        pool[pool_index(layer, m, page, h, (int32_t)(T % Ps), e, P, n_kv, Ps, d)] =
                            staging[src];
                    }
    return 0;
}

int oco_ingest_layer(const uint16_t *staging, int64_t n_chunks, int32_t G, int32_t n_kv, int32_t d,
                     int32_t Ps, const int32_t *table, int64_t table_len, uint16_t *pool, int64_t P,
                     int32_t layer) {
    return ingest_chunk_range(staging, 0, n_chunks, G, n_kv, d, Ps, table, table_len, pool, P, layer);
}

/* The same scatter with the chunks divided into `threads` contiguous ranges,
 * one thread each.  Chunks write distinct pool elements as long as the page
 * ids are distinct (the block table's contract), so the result equals
 * oco_ingest_layer's.  Returns -2 when a thread could not be started (its
 * range is then not copied). */
struct ingest_job {
    const uint16_t *staging;
    int64_t j0, j1;
    int32_t G, n_kv, d, Ps, layer;
    const int32_t *table;
    int64_t table_len, P;
    uint16_t *pool;
    int rc;
};

static void *ingest_worker(void *arg) {
    struct ingest_job *J = (struct ingest_job *)arg;
    J->rc = ingest_chunk_range(J->staging, J->j0, J->j1, J->G, J->n_kv, J->d, J->Ps, J->table, J->table_len,
                               J->pool, J->P, J->layer);
    return NULL;
}

int oco_ingest_layer_mt(const uint16_t *staging, int64_t n_chunks, int32_t G, int32_t n_kv, int32_t d,
                        int32_t Ps, const int32_t *table, int64_t table_len, uint16_t *pool, int64_t P,
                        int32_t layer, int32_t threads) {
    if (threads < 1) threads = 1;
    if (threads > 256) threads = 256;
    if (threads > n_chunks) threads = n_chunks > 0 ? (int32_t)n_chunks : 1;
    struct ingest_job jobs[256];
    pthread_t tid[256];
    for (int32_t i = 0; i < threads; ++i) {
        struct ingest_job J = {staging, n_chunks * i / threads, n_chunks * (i + 1) / threads, G, n_kv, d, Ps,
                               layer, table, table_len, P, pool, 0};
        jobs[i] = J;
    }
    char started[256] = {0};
    for (int32_t i = 1; i < threads; ++i) started[i] = pthread_create(&tid[i], NULL, ingest_worker, &jobs[i]) == 0;
    ingest_worker(&jobs[0]);
    int rc = jobs[0].rc;
    for (int32_t i = 1; i < threads; ++i) {
        if (!started[i]) {   /* its chunks were not copied */
            rc = -2;
            continue;
        }
        pthread_join(tid[i], NULL);
        if (jobs[i].rc != 0) rc = jobs[i].rc;
    }
    return rc;
}

/* Inverse of the scatter: read the layer back out of the pool into the
 * staging layout. */
int oco_gather_layer(const uint16_t *pool, int64_t P, int32_t layer, const int32_t *table,
                     int64_t table_len, int64_t n_chunks, int32_t G, int32_t n_kv, int32_t d,
                     int32_t Ps, uint16_t *staging) {
    int64_t slice = 2LL * G * n_kv * d;
    for (int64_t j = 0; j < n_chunks; ++j)
        for (int32_t m = 0; m < 2; ++m)
            for (int32_t t = 0; t < G; ++t)
                for (int32_t h = 0; h < n_kv; ++h)
                    for (int32_t e = 0; e < d; ++e) {
                        int64_t T = j * G + t;
                        int64_t q = T / Ps;
                        if (q >= table_len) return -1;
                        int64_t page = table[q];
                        if (page < 0 || page >= P) return -1;
                        staging[j * slice + l2td_index(0, m, t, h, e, G, n_kv, d)] =
                            pool[pool_index(layer, m, page, h, (int32_t)(T % Ps), e, P, n_kv, Ps, d)];
                    }
    return 0;
}

/* Suffix append (the prefill node materialising the full KV state, Section 3
 * opening): suffix token i of one layer, K and V given dense [T_s][n_kv][d],
 * is written to logical position T = token0 + i, i.e. page table[T / Ps],
 * slot T % Ps -- the same paging rule as the prefix.  Returns 0, or -1 when a
 * table entry is missing or outside [0, P). */
int oco_append_suffix(const uint16_t *k_new, const uint16_t *v_new, int64_t Ts, int32_t n_kv, int32_t d,
                      int32_t Ps, const int32_t *table, int64_t table_len, int64_t token0, uint16_t *pool,
                      int64_t P, int32_t layer) {
    for (int32_t m = 0; m < 2; ++m)
        for (int64_t i = 0; i < Ts; ++i)
            for (int32_t h = 0; h < n_kv; ++h)
                for (int32_t e = 0; e < d; ++e) {
                    int64_t T = token0 + i;
                    int64_t q = T / Ps;
                    if (q >= table_len) return -1;
                    int64_t page = table[q];
                    if (page < 0 || page >= P) return -1;
                    const uint16_t *src = m == 0 ? k_new : v_new;
                    pool[pool_index(layer, m, page, h, (int32_t)(T % Ps), e, P, n_kv, Ps, d)] =
                        src[(i * n_kv + h) * d + e];
                }
    return 0;
}

/* Offload (write-back of newly produced chunks, Section 3 opening): rebuild
 * chunk objects first_chunk .. first_chunk+n_chunks-1 from the pool, every
 * layer, in KV_L2TD order; object j is written at objects + j*L*2*G*n_kv*d.
 * Returns 0, or -1 when a table entry is missing or outside [0, P). */
int oco_gather_chunks(const uint16_t *pool, int64_t P, int32_t L, const int32_t *table, int64_t table_len,
                      int64_t first_chunk, int64_t n_chunks, int32_t G, int32_t n_kv, int32_t d, int32_t Ps,
                      uint16_t *objects) {
    int64_t obj_elems = (int64_t)L * 2 * G * n_kv * d;
    for (int64_t j = 0; j < n_chunks; ++j)
        for (int32_t l = 0; l < L; ++l)
            for (int32_t m = 0; m < 2; ++m)
                for (int32_t t = 0; t < G; ++t)
                    for (int32_t h = 0; h < n_kv; ++h)
                        for (int32_t e = 0; e < d; ++e) {
                            int64_t T = (first_chunk + j) * G + t;
                            int64_t q = T / Ps;
                            if (q >= table_len) return -1;
                            int64_t page = table[q];
                            if (page < 0 || page >= P) return -1;
                            objects[j * obj_elems + l2td_index(l, m, t, h, e, G, n_kv, d)] =
                                pool[pool_index(l, m, page, h, (int32_t)(T % Ps), e, P, n_kv, Ps, d)];
                        }
    return 0;
}

/* ---- attention -------------------------------------------------------------- */
static double bf16(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

typedef struct {
    const uint16_t *q, *kp, *vp, *kn, *vn;
    int64_t Tp, Ts;
    int32_t nq, nkv, d;
    const int64_t *rows;       /* suffix token indices to compute */
    int64_t n_rows;
    double *out;               /* [n_rows][nq][d] */
    int64_t next;              /* work counter (row*nq + head) */
    int failed;                /* a worker could not allocate its score row */
    pthread_mutex_t mu;
} attn_job;

/* One (suffix token i, query head h): o = sum_j w_j v_j / sum_j w_j with
 * w_j = exp(s_j - max s), s_j = q.k_j / sqrt(d), j over prefix keys 0..Tp-1
 * and suffix keys 0..i; query head h reads KV head h / (nq / nkv). */
static void attn_row(const attn_job *J, int64_t r, int32_t h, double *score) {
    int64_t i = J->rows[r];
    int32_t grp = J->nq / J->nkv, g = h / grp, d = J->d;
    const uint16_t *q = J->q + (i * J->nq + h) * d;
    int64_t n_keys = J->Tp + i + 1;
    double inv = 1.0 / sqrt((double)d);
    double m = -INFINITY;
    for (int64_t j = 0; j < n_keys; ++j) {
        const uint16_t *k = j < J->Tp ? J->kp + (j * J->nkv + g) * d
                                      : J->kn + ((j - J->Tp) * J->nkv + g) * d;
        double s = 0.0;
        for (int32_t e = 0; e < d; ++e) s += bf16(q[e]) * bf16(k[e]);
        s *= inv;
        score[j] = s;
        if (s > m) m = s;
    }
    double *o = J->out + (r * J->nq + h) * d;
    for (int32_t e = 0; e < d; ++e) o[e] = 0.0;
    double den = 0.0;
    for (int64_t j = 0; j < n_keys; ++j) {
        double w = exp(score[j] - m);
        const uint16_t *v = j < J->Tp ? J->vp + (j * J->nkv + g) * d
                                      : J->vn + ((j - J->Tp) * J->nkv + g) * d;
        den += w;
        for (int32_t e = 0; e < d; ++e) o[e] += w * bf16(v[e]);
    }
    for (int32_t e = 0; e < d; ++e) o[e] /= den;
}

static void *attn_worker(void *arg) {
    attn_job *J = (attn_job *)arg;
    double *score = (double *)malloc(sizeof(double) * (size_t)(J->Tp + J->Ts + 1));
    if (!score) {
        pthread_mutex_lock(&J->mu);
        J->failed = 1;
        pthread_mutex_unlock(&J->mu);
        return NULL;
    }
    int64_t total = J->n_rows * J->nq;
    for (;;) {
        pthread_mutex_lock(&J->mu);
        int64_t w = J->next++;
        pthread_mutex_unlock(&J->mu);
        if (w >= total) break;
        attn_row(J, w / J->nq, (int32_t)(w % J->nq), score);
    }
    free(score);
    return NULL;
}

/* q [Ts][nq][d], k_prefix/v_prefix [Tp][nkv][d] (logical, un-paged),
 * k_new/v_new [Ts][nkv][d], all bfloat16 bits.  Computes the listed suffix
 * rows (rows == NULL: all Ts rows) into out [n_rows][nq][d] float64.
 * Returns 0, -1 on bad arguments, -2 when memory runs out. */
int oco_attention(const uint16_t *q, const uint16_t *k_prefix, const uint16_t *v_prefix,
                  const uint16_t *k_new, const uint16_t *v_new, int64_t Tp, int64_t Ts, int32_t nq,
                  int32_t nkv, int32_t d, const int64_t *rows, int64_t n_rows, double *out,
                  int32_t threads) {
    if (nkv <= 0 || nq % nkv != 0 || d <= 0 || Ts < 0 || Tp < 0) return -1;
    int64_t *all = NULL;
    if (!rows) {
        all = (int64_t *)malloc(sizeof(int64_t) * (size_t)(Ts > 0 ? Ts : 1));
        if (!all) return -2;
        for (int64_t i = 0; i < Ts; ++i) all[i] = i;
        rows = all;
        n_rows = Ts;
    }
    for (int64_t r = 0; r < n_rows; ++r)
        if (rows[r] < 0 || rows[r] >= Ts) { free(all); return -1; }
    attn_job J;
    memset(&J, 0, sizeof J);
    J.q = q; J.kp = k_prefix; J.vp = v_prefix; J.kn = k_new; J.vn = v_new;
    J.Tp = Tp; J.Ts = Ts; J.nq = nq; J.nkv = nkv; J.d = d;
    J.rows = rows; J.n_rows = n_rows; J.out = out;
    pthread_mutex_init(&J.mu, NULL);
    if (threads < 1) threads = 1;
    if (threads > 256) threads = 256;
    pthread_t th[256];
    int started = 0;
    for (int t = 0; t < threads; ++t)
        if (pthread_create(&th[t], NULL, attn_worker, &J) == 0) ++started;
    if (started == 0) attn_worker(&J);
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    pthread_mutex_destroy(&J.mu);
    free(all);
    return J.failed ? -2 : 0;
}
