// Layer ingest: unpack one layer payload (concatenated KV_L2TD layer slices
// of the matched chunk objects, Section 3.3) and scatter it into the paged
// pool through the block table.
//
// Both sides keep one head's d-element row per token, so the scatter is a
// copy of 16-byte pieces with remapped addresses: the payload holds the rows
// of a chunk token-major ([K|V][token][head][dim]), the pool holds them per
// (page, head) block ([slot][dim]).  Two launch shapes:
//  - alone on the GPU (the single-layer entry point, the first layer of a
//    run): one piece per thread in payload order, so every wavefront reads
//    1 KiB of the payload contiguously and writes four 256-byte rows, and
//    many short wavefronts keep the most bytes in flight;
//  - beside the attention kernel of an earlier layer, where two ingest
//    wavefronts per SIMD run at the lowest issue priority: a thread takes
//    8 slots x one 16-byte column of one (page, head) block and moves its K
//    rows, then its V rows (8 loads in flight, one page lookup per 256 bytes
//    moved, a shift decode of the thread's block and column).
// The gather (pool -> payload or whole chunk objects, the offload direction)
// numbers pieces the same way, reversed.  The suffix append writes the new
// tokens' K/V rows behind the prefix through the same block table.
#include "common.hpp"

namespace oc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// 8 slots x one 16-byte column of one (page, head) block, K then V.  With
// POW2 (d/8, page size, KV heads and a chunk size of at least 8 all powers of
// two) the decode is shifts and masks and the 8 tokens sit in one chunk.
// Every group of 8 slots lies wholly inside or wholly past the prefix when
// the chunk size is a multiple of 8; only other chunk sizes reach the
// per-token bounds checks.
template <bool POW2>
__global__ __launch_bounds__(kThreads, 8) void kv_ingest_rows_kernel(IngestArgs a, int64_t n_rows8) {
    const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (u >= n_rows8) return;
    const int d = a.d, G = a.G, nkv = a.n_kv;
    int c, s8, h;
    int64_t q, T0;
    if (POW2) {
        const int lg_s8 = a.lg_ps - 3;                   // page_size / 8 groups per page
        c = (int)(u & (a.d8 - 1));
        s8 = (int)((u >> a.lg_d8) & ((1 << lg_s8) - 1));
        h = (int)((u >> (a.lg_d8 + lg_s8)) & (nkv - 1));
        q = u >> (a.lg_d8 + lg_s8 + a.lg_nkv);
        T0 = (q << a.lg_ps) + s8 * 8;
    } else {
        c = (int)(u % a.d8);
        int64_t rest = u / a.d8;
        s8 = (int)(rest % (a.Ps / 8));
        rest /= a.Ps / 8;
        h = (int)(rest % nkv);
        q = rest / nkv;
        T0 = q * a.Ps + s8 * 8;                          // first token of the 8
    }
    const int64_t left = a.num_tokens - T0;
    if (left <= 0) return;                               // slots past the prefix
    const int64_t D = (int64_t)nkv * d;
    const int64_t page = a.pages[q];
    uint16_t *kdst = a.pool_k + ((page * nkv + h) * a.Ps + s8 * 8) * (int64_t)d + c * 8;
    const int64_t col = (int64_t)h * d + c * 8;
    const int64_t vstep = (int64_t)G * D;                // K row -> V row of a token
    // non-temporal: the payload is read once and the pool rows are not read
    // again until that layer's attention, so keep both out of the L2 that the
    // running attention uses for its K/V tiles
    u32x4 r[8];
    if (POW2 || (G % 8 == 0)) {
        // the 8 tokens sit in one chunk, one payload row apart, all inside
        // the prefix (it is a whole number of chunks)
        const int64_t j = POW2 ? T0 >> a.lg_g : T0 / G;
        const uint16_t *src = a.staging + j * a.chunk_stride + (T0 - j * G) * D + col;
#pragma unroll
        for (int kv = 0; kv < 2; ++kv) {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                r[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src + kv * vstep + i * D));
#pragma unroll
            for (int i = 0; i < 8; ++i)
                __builtin_nontemporal_store(r[i], reinterpret_cast<u32x4 *>(kdst + kv * a.region + i * d));
        }
        return;
    }
    // chunk sizes that are not a multiple of 8: the 8 tokens may span two
    // chunks and run past the prefix
    const int valid = left < 8 ? (int)left : 8;
    int64_t src[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t T = T0 + i, j = T / G;
        src[i] = j * a.chunk_stride + (T - j * G) * D + col;
    }
#pragma unroll
    for (int kv = 0; kv < 2; ++kv) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (i < valid)
                r[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.staging + src[i] + kv * vstep));
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (i < valid) __builtin_nontemporal_store(r[i], reinterpret_cast<u32x4 *>(kdst + kv * a.region + i * d));
    }
}

// Piece e of a payload numbered in payload order ([chunk][K|V][token][head]
// [16-byte column]) -> its element offsets in the staging (from `staging`)
// and in the pool (from `pool_k`), both including the layer step of
// blockIdx.y.  With POW2 every divisor (d/8, KV heads, chunk size, page size)
// is a power of two and the decode is shifts and masks.
template <bool POW2>
__device__ inline void src_order_piece(const IngestArgs &a, int64_t e, int64_t &stage, int64_t &pool) {
    const int64_t slice_pieces = 2LL * a.G * a.n_kv * a.d8;   // 16-byte pieces per chunk slice
    int c, h, t, kv;
    int64_t j;
    if (POW2) {
        c = (int)(e & (a.d8 - 1));
        h = (int)((e >> a.lg_d8) & (a.n_kv - 1));
        t = (int)((e >> (a.lg_d8 + a.lg_nkv)) & (a.G - 1));
        kv = (int)((e >> (a.lg_d8 + a.lg_nkv + a.lg_g)) & 1);
        j = e >> (a.lg_d8 + a.lg_nkv + a.lg_g + 1);
    } else {
        int64_t r = e / a.d8;
        c = (int)(e - r * a.d8);
        int64_t r2 = r / a.n_kv;
        h = (int)(r - r2 * a.n_kv);
        int64_t r3 = r2 / a.G;
        t = (int)(r2 - r3 * a.G);
        j = r3 >> 1;
        kv = (int)(r3 & 1);
    }
    const int64_t T = a.token0 + j * a.G + t;
    int64_t q, slot;
    if (POW2) {
        q = T >> a.lg_ps;
        slot = T & (a.Ps - 1);
    } else {
        q = T / a.Ps;
        slot = T - q * a.Ps;
    }
    const int64_t page = a.pages[q];
    stage = blockIdx.y * a.layer_step_staging + j * a.chunk_stride + (e - j * slice_pieces) * 8;
    pool = blockIdx.y * a.layer_step_pool + kv * a.region + ((page * a.n_kv + h) * a.Ps + slot) * (int64_t)a.d +
           c * 8;
}

// Ingest, one 16-byte piece per thread in payload order: every wavefront
// reads 1 KiB of the payload contiguously and writes 256-byte rows into the
// (page, head) blocks.  Many short wavefronts keep the most bytes in flight.
// Every byte is read once and written once, so both sides bypass the L2's
// normal retention (non-temporal): about 2.5 % faster alone than plain
// accesses at the 8b-64k layer.
// For whole chunk objects blockIdx.y is the layer.
template <bool POW2>
__global__ __launch_bounds__(kThreads) void kv_ingest_src_kernel(IngestArgs a, int64_t n_pieces) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= n_pieces) return;
    int64_t stage, pool;
    src_order_piece<POW2>(a, e, stage, pool);
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.staging + stage));
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(a.pool_k + pool));
}

// Gather (pool -> layer payload or whole chunk objects, the offload
// direction): the same numbering, so every wavefront writes 1 KiB of the
// output contiguously and reads 256-byte pool rows; non-temporal on both
// sides like the ingest (about 7 % faster than plain accesses over the
// chunk objects of the 64K prefix).
template <bool POW2>
__global__ __launch_bounds__(kThreads) void kv_gather_src_kernel(IngestArgs a, uint16_t *out, int64_t n_pieces) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= n_pieces) return;
    int64_t stage, pool;
    src_order_piece<POW2>(a, e, stage, pool);
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(a.pool_k + pool));
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(out + stage));
}

// Suffix append: token i of k_new / v_new ([T_s][n_kv][d]; blockIdx.y picks
// K or V) goes to logical position token0 + i through the block table.
__global__ __launch_bounds__(kThreads) void kv_append_kernel(AppendArgs a, int64_t n_pieces) {
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= n_pieces) return;
    const int kv = (int)blockIdx.y;
    const int64_t r = e / a.d8;
    const int c = (int)(e - r * a.d8);
    const int64_t i = r / a.n_kv;
    const int h = (int)(r - i * a.n_kv);
    const int64_t T = a.token0 + i;
    const int64_t q = T / a.Ps, slot = T - q * a.Ps;
    const int64_t page = a.pages[q];
    const uint16_t *src = (kv ? a.v_new : a.k_new) + e * 8;
    uint16_t *dst = a.pool_k + kv * a.region + ((page * a.n_kv + h) * a.Ps + slot) * (int64_t)a.d + c * 8;
    *reinterpret_cast<u32x4 *>(dst) = *reinterpret_cast<const u32x4 *>(src);
}

static bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
static int lg(int64_t x) {
    int r = 0;
    while ((1LL << r) < x) ++r;
    return r;
}

// Fills the derived fields and the defaults of a single layer payload;
// returns whether the shift decode applies.
static bool prepare(IngestArgs &a) {
    if (a.chunk_stride == 0) a.chunk_stride = 2LL * a.G * a.n_kv * a.d;
    if (a.n_layers == 0) a.n_layers = 1;
    a.d8 = a.d / 8;
    a.region = (int64_t)(a.pool_v - a.pool_k);
    const bool p2 = pow2(a.d8) && pow2(a.Ps) && pow2(a.n_kv) && pow2(a.G);
    a.lg_d8 = lg(a.d8);
    a.lg_ps = lg(a.Ps);
    a.lg_nkv = lg(a.n_kv);
    a.lg_g = lg(a.G);
    return p2;
}

hipError_t launch_ingest(IngestArgs a, int64_t n_pages_used, hipStream_t s, bool beside_compute) {
    if (n_pages_used == 0) return hipSuccess;
    const bool p2 = prepare(a);
    if (beside_compute && a.token0 == 0) {
        const int64_t n = n_pages_used * a.n_kv * (a.Ps / 8) * a.d8;
        const dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
        // Each workgroup reserves half the LDS an attention workgroup leaves
        // free (the kernel itself uses none), so that at most two ingest
        // workgroups, two wavefronts per SIMD, share a CU with the attention;
        // registers alone would admit three.  With the attention's wavefronts
        // issuing ahead of the ingest's, that is the count that moves the
        // most bytes without lengthening the attention beside it.
        const size_t attn = attention_lds_bytes(a.d);
        const size_t lds = attn > 0 && attn < CU_LDS_BYTES ? (CU_LDS_BYTES - attn) / 2 : 0;
        if (p2 && a.Ps >= 8 && a.G >= 8)
            hipLaunchKernelGGL(kv_ingest_rows_kernel<true>, grid, dim3(kThreads), lds, s, a, n);
        else
            hipLaunchKernelGGL(kv_ingest_rows_kernel<false>, grid, dim3(kThreads), lds, s, a, n);
    } else {
        const int64_t n = a.num_tokens * 2 * a.n_kv * a.d8;   // 16-byte pieces of the payload
        const dim3 grid((unsigned)((n + kThreads - 1) / kThreads));
        if (p2) hipLaunchKernelGGL(kv_ingest_src_kernel<true>, grid, dim3(kThreads), 0, s, a, n);
        else hipLaunchKernelGGL(kv_ingest_src_kernel<false>, grid, dim3(kThreads), 0, s, a, n);
    }
    return hipGetLastError();
}

hipError_t launch_chunks_ingest(IngestArgs a, hipStream_t s) {
    if (a.num_tokens == 0) return hipSuccess;
    const bool p2 = prepare(a);
    const int64_t n = a.num_tokens * 2 * a.n_kv * a.d8;   // 16-byte pieces of one layer
    const dim3 grid((unsigned)((n + kThreads - 1) / kThreads), (unsigned)a.n_layers);
    if (p2) hipLaunchKernelGGL(kv_ingest_src_kernel<true>, grid, dim3(kThreads), 0, s, a, n);
    else hipLaunchKernelGGL(kv_ingest_src_kernel<false>, grid, dim3(kThreads), 0, s, a, n);
    return hipGetLastError();
}

hipError_t launch_gather(IngestArgs a, uint16_t *out, hipStream_t s) {
    if (a.num_tokens == 0) return hipSuccess;
    const bool p2 = prepare(a);
    const int64_t n = a.num_tokens * 2 * a.n_kv * a.d8;   // 16-byte pieces of one layer
    const dim3 grid((unsigned)((n + kThreads - 1) / kThreads), (unsigned)a.n_layers);
    if (p2) hipLaunchKernelGGL(kv_gather_src_kernel<true>, grid, dim3(kThreads), 0, s, a, out, n);
    else hipLaunchKernelGGL(kv_gather_src_kernel<false>, grid, dim3(kThreads), 0, s, a, out, n);
    return hipGetLastError();
}

hipError_t launch_append(AppendArgs a, hipStream_t s) {
    if (a.num_tokens == 0) return hipSuccess;
    a.d8 = a.d / 8;
    a.region = (int64_t)(a.pool_v - a.pool_k);
    const int64_t n = a.num_tokens * a.n_kv * a.d8;        // 16-byte pieces of K (and of V)
    const dim3 grid((unsigned)((n + kThreads - 1) / kThreads), 2);
    hipLaunchKernelGGL(kv_append_kernel, grid, dim3(kThreads), 0, s, a, n);
    return hipGetLastError();
}

}  // namespace oc
