// Layer ingest: unpack one layer payload (concatenated KV_L2TD layer slices
// of the matched chunk objects, Section 3.3) and scatter it into the paged
// pool through the block table.
//
// One thread moves one 8-token x 8-dim block of one head: eight 16-byte
// rows of K and eight of V.  K rows keep their [slot][dim] order; V rows are
// transposed in registers (16-bit lane permutes) and leave as eight 16-byte
// runs of the pool's [dim][slot] V block.  Neighbouring threads take
// neighbouring 8-dim groups, so every load and K store is a contiguous
// 256-byte run per (token, head) across 16 lanes.  No LDS and little index
// arithmetic: the kernel is pure HBM traffic and stays small enough (<= 64
// VGPRs) to run beside the attention kernel of the previous layer.
#include "common.hpp"

namespace oc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// Column k of an 8x8 block of 16-bit elements whose row i is in[i]
// (8 elements, two per dword).
__device__ inline u32x4 column8(const u32x4 (&in)[8], int k) {
    const int w = k >> 1;
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t a = in[2 * j][w], b = in[2 * j + 1][w];
        o[j] = (k & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
    }
    return u32x4{o[0], o[1], o[2], o[3]};
}

struct Unit {
    int64_t q;      // block-table index (page of the prefix)
    int h, s8, e8;  // head, 8-slot group, 8-dim group
};

__device__ inline Unit unit_of(int64_t u, int d8, int s8n, int nkv) {
    Unit r;
    r.e8 = (int)(u % d8);
    int64_t rest = u / d8;
    r.s8 = (int)(rest % s8n);
    rest /= s8n;
    r.h = (int)(rest % nkv);
    r.q = rest / nkv;
    return r;
}

__global__ __launch_bounds__(kThreads, 8) void kv_ingest_kernel(IngestArgs a, int64_t n_units) {
    const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (u >= n_units) return;
    const int d = a.d, Ps = a.Ps, G = a.G, nkv = a.n_kv;
    const Unit w = unit_of(u, d >> 3, Ps >> 3, nkv);
    const int64_t D = (int64_t)nkv * d;
    const int64_t T0 = w.q * Ps + w.s8 * 8;                  // first token of the unit
    const int64_t rest = a.num_tokens - T0;
    const int valid = rest < 8 ? (int)rest : 8;              // tokens of the unit inside the prefix
    const int64_t page = a.pages[w.q];
    // G is a multiple of 8, so the unit's 8 tokens sit in one chunk
    const int64_t j = T0 / G, t0 = T0 - j * G;
    const uint16_t *src = a.staging + (j * 2 * G + t0) * D + (int64_t)w.h * d + w.e8 * 8;
    const int64_t blk = (page * nkv + w.h) * (int64_t)Ps * d;  // (page, head) block

    u32x4 r[8];
    // K: rows straight to [slot][dim]
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (i < valid) r[i] = *reinterpret_cast<const u32x4 *>(src + i * D);
    uint16_t *kdst = a.pool_k + blk + (int64_t)(w.s8 * 8) * d + w.e8 * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (i < valid) *reinterpret_cast<u32x4 *>(kdst + i * d) = r[i];

    // V: rows in, transposed, out as [dim][slot]
    const uint16_t *vsrc = src + (int64_t)G * D;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        r[i] = i < valid ? *reinterpret_cast<const u32x4 *>(vsrc + i * D) : u32x4{0, 0, 0, 0};
    // each column leaves as soon as it is formed, freeing its source dwords
    uint16_t *vdst = a.pool_v + blk + (int64_t)(w.e8 * 8) * Ps + w.s8 * 8;
    if (valid == 8) {
#pragma unroll
        for (int k = 0; k < 8; ++k) *reinterpret_cast<u32x4 *>(vdst + k * Ps) = column8(r, k);
    } else {
        // last, partial page: write only the slots that hold prefix tokens
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const u32x4 ck = column8(r, k);
            uint16_t v[8];
            __builtin_memcpy(v, &ck, 16);
            for (int i = 0; i < valid; ++i) vdst[k * Ps + i] = v[i];
        }
    }
}

// Inverse: pool pages back into the staging layout (same units, transposes reversed).
__global__ __launch_bounds__(kThreads, 8) void kv_gather_kernel(IngestArgs a, uint16_t *staging, int64_t n_units) {
    const int64_t u = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (u >= n_units) return;
    const int d = a.d, Ps = a.Ps, G = a.G, nkv = a.n_kv;
    const Unit w = unit_of(u, d >> 3, Ps >> 3, nkv);
    const int64_t D = (int64_t)nkv * d;
    const int64_t T0 = w.q * Ps + w.s8 * 8;
    const int64_t rest = a.num_tokens - T0;
    const int valid = rest < 8 ? (int)rest : 8;
    const int64_t page = a.pages[w.q];
    const int64_t j = T0 / G, t0 = T0 - j * G;
    uint16_t *dst = staging + (j * 2 * G + t0) * D + (int64_t)w.h * d + w.e8 * 8;
    const int64_t blk = (page * nkv + w.h) * (int64_t)Ps * d;

    u32x4 r[8];
    const uint16_t *ksrc = a.pool_k + blk + (int64_t)(w.s8 * 8) * d + w.e8 * 8;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (i < valid) r[i] = *reinterpret_cast<const u32x4 *>(ksrc + i * d);
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (i < valid) *reinterpret_cast<u32x4 *>(dst + i * D) = r[i];

    const uint16_t *vsrc = a.pool_v + blk + (int64_t)(w.e8 * 8) * Ps + w.s8 * 8;
    if (valid == 8) {
#pragma unroll
        for (int k = 0; k < 8; ++k) r[k] = *reinterpret_cast<const u32x4 *>(vsrc + k * Ps);
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            uint16_t v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            for (int i = 0; i < valid; ++i) v[i] = vsrc[k * Ps + i];
            __builtin_memcpy(&r[k], v, 16);
        }
    }
    uint16_t *vdst = dst + (int64_t)G * D;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        if (i < valid) *reinterpret_cast<u32x4 *>(vdst + i * D) = column8(r, i);
}

static int64_t n_units(const IngestArgs &a, int64_t n_pages_used) {
    return n_pages_used * a.n_kv * (a.d / 8) * (a.Ps / 8);
}

hipError_t launch_ingest(const IngestArgs &a, int64_t n_pages_used, hipStream_t s) {
    if (n_pages_used == 0) return hipSuccess;
    const int64_t n = n_units(a, n_pages_used);
    hipLaunchKernelGGL(kv_ingest_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, s, a, n);
    return hipGetLastError();
}

hipError_t launch_gather(const IngestArgs &a, uint16_t *staging_out, int64_t n_pages_used, hipStream_t s) {
    if (n_pages_used == 0) return hipSuccess;
    const int64_t n = n_units(a, n_pages_used);
    hipLaunchKernelGGL(kv_gather_kernel, dim3((unsigned)((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, s, a,
                       staging_out, n);
    return hipGetLastError();
}

}  // namespace oc
