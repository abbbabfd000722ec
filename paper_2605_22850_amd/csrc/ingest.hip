// Layer ingest: unpack one layer payload (concatenated KV_L2TD layer slices
// of the matched chunk objects, Section 3.3) and scatter it into the paged
// pool through the block table.
//
// One workgroup moves one pool page for a group of KV heads.  K rows keep
// their [slot][dim] order and go straight from registers to HBM in 16-byte
// vectors.  V rows are staged through LDS and leave transposed ([dim][slot]
// per page), so the attention later reads eight consecutive keys of one
// dimension as one 16-byte vector.  Both the staging reads and the pool
// writes are contiguous 16-byte vectors across the wavefront.
#include "common.hpp"

namespace oc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kBatch = 8;        // 16-byte vectors in flight per thread

__device__ inline u32x4 pack8(const uint16_t *v) {
    u32x4 r;
    r.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
    r.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
    r.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
    r.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
    return r;
}

__global__ __launch_bounds__(kThreads) void kv_ingest_kernel(IngestArgs a) {
    extern __shared__ __align__(16) uint16_t lds[];
    const int H = a.heads_per_block, h0 = blockIdx.y * H;
    const int d = a.d, Ps = a.Ps, G = a.G, nkv = a.n_kv;
    const int64_t D = (int64_t)nkv * d;
    const int64_t qi = blockIdx.x;                         // index into the block table
    const int64_t page = a.pages[qi];
    const int64_t T0 = qi * Ps;
    const int64_t rest = a.num_tokens - T0;
    const int valid = rest < Ps ? (int)rest : Ps;          // slots of this page holding prefix tokens
    const int d8 = d >> 3;
    const int row_pieces = H * d8;
    const int n_pieces = Ps * row_pieces;
    const int lds_row = H * d + 8;                         // padded row: spreads the transposed reads over banks

    for (int base = 0; base < n_pieces; base += kBatch * kThreads) {
        u32x4 kr[kBatch], vr[kBatch];
        int64_t kdst[kBatch];
        int ldst[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int p = base + u * kThreads + (int)threadIdx.x;
            kdst[u] = -1;
            if (p < n_pieces) {
                const int s = p / row_pieces;
                const int rem = p - s * row_pieces;
                const int hh = rem / d8;
                const int e8 = rem - hh * d8;
                if (s < valid) {
                    const int64_t T = T0 + s;
                    const int64_t j = T / G;
                    const int64_t t = T - j * G;
                    const uint16_t *src = a.staging + j * 2 * G * D + t * D + (int64_t)(h0 + hh) * d + e8 * 8;
                    kr[u] = *reinterpret_cast<const u32x4 *>(src);
                    vr[u] = *reinterpret_cast<const u32x4 *>(src + (int64_t)G * D);
                    kdst[u] = ((page * nkv + h0 + hh) * Ps + s) * (int64_t)d + e8 * 8;
                    ldst[u] = s * lds_row + hh * d + e8 * 8;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            if (kdst[u] >= 0) {
                *reinterpret_cast<u32x4 *>(a.pool_k + kdst[u]) = kr[u];
                *reinterpret_cast<u32x4 *>(lds + ldst[u]) = vr[u];
            }
        }
    }
    __syncthreads();

    // V leaves as [dim][slot]; one output vector = 8 consecutive slots of one dim
    const int s8n = Ps >> 3;
    const int n_out = H * d * s8n;
    for (int o = threadIdx.x; o < n_out; o += kThreads) {
        const int hh = o / (d * s8n);
        const int rem = o - hh * d * s8n;
        const int e = rem / s8n;
        const int sb = (rem - e * s8n) * 8;
        if (sb >= valid) continue;
        uint16_t *dv = a.pool_v + ((page * nkv + h0 + hh) * (int64_t)d + e) * Ps + sb;
        const uint16_t *col = lds + sb * lds_row + hh * d + e;
        if (sb + 8 <= valid) {
            uint16_t v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = col[i * lds_row];
            *reinterpret_cast<u32x4 *>(dv) = pack8(v);
        } else {
            for (int i = 0; sb + i < valid; ++i) dv[i] = col[i * lds_row];
        }
    }
}

// Inverse: pool pages back into the staging layout.
__global__ __launch_bounds__(kThreads) void kv_gather_kernel(IngestArgs a, uint16_t *staging) {
    extern __shared__ __align__(16) uint16_t lds[];
    const int H = a.heads_per_block, h0 = blockIdx.y * H;
    const int d = a.d, Ps = a.Ps, G = a.G, nkv = a.n_kv;
    const int64_t D = (int64_t)nkv * d;
    const int64_t qi = blockIdx.x;
    const int64_t page = a.pages[qi];
    const int64_t T0 = qi * Ps;
    const int64_t rest = a.num_tokens - T0;
    const int valid = rest < Ps ? (int)rest : Ps;
    const int d8 = d >> 3;
    const int lds_row = H * d + 8;

    // V pages ([dim][slot]) into LDS rows [slot][head*d + dim]
    const int s8n = Ps >> 3;
    const int n_in = H * d * s8n;
    for (int o = threadIdx.x; o < n_in; o += kThreads) {
        const int hh = o / (d * s8n);
        const int rem = o - hh * d * s8n;
        const int e = rem / s8n;
        const int sb = (rem - e * s8n) * 8;
        if (sb >= valid) continue;
        const uint16_t *sv = a.pool_v + ((page * nkv + h0 + hh) * (int64_t)d + e) * Ps + sb;
        uint16_t *col = lds + sb * lds_row + hh * d + e;
        const int n = valid - sb < 8 ? valid - sb : 8;
        for (int i = 0; i < n; ++i) col[i * lds_row] = sv[i];
    }
    __syncthreads();

    const int row_pieces = H * d8;
    const int n_pieces = Ps * row_pieces;
    for (int p = threadIdx.x; p < n_pieces; p += kThreads) {
        const int s = p / row_pieces;
        const int rem = p - s * row_pieces;
        const int hh = rem / d8;
        const int e8 = rem - hh * d8;
        if (s >= valid) continue;
        const int64_t T = T0 + s;
        const int64_t j = T / G;
        const int64_t t = T - j * G;
        uint16_t *dst = staging + j * 2 * G * D + t * D + (int64_t)(h0 + hh) * d + e8 * 8;
        const uint16_t *kp = a.pool_k + ((page * nkv + h0 + hh) * Ps + s) * (int64_t)d + e8 * 8;
        *reinterpret_cast<u32x4 *>(dst) = *reinterpret_cast<const u32x4 *>(kp);
        *reinterpret_cast<u32x4 *>(dst + (int64_t)G * D) =
            *reinterpret_cast<const u32x4 *>(lds + s * lds_row + hh * d + e8 * 8);
    }
}

int ingest_heads_per_block(int n_kv, int d, int Ps) {
    // largest divisor of n_kv whose V page fits a 64 KiB LDS stage
    for (int h = n_kv; h >= 1; --h) {
        if (n_kv % h) continue;
        if ((size_t)Ps * (h * d + 8) * 2 <= 65536) return h;
    }
    return 0;
}

static size_t lds_bytes(const IngestArgs &a) { return (size_t)a.Ps * (a.heads_per_block * a.d + 8) * 2; }

hipError_t launch_ingest(const IngestArgs &a, int64_t n_pages_used, hipStream_t s) {
    if (n_pages_used == 0) return hipSuccess;
    dim3 grid((unsigned)n_pages_used, (unsigned)(a.n_kv / a.heads_per_block));
    hipLaunchKernelGGL(kv_ingest_kernel, grid, dim3(kThreads), lds_bytes(a), s, a);
    return hipGetLastError();
}

hipError_t launch_gather(const IngestArgs &a, uint16_t *staging_out, int64_t n_pages_used, hipStream_t s) {
    if (n_pages_used == 0) return hipSuccess;
    dim3 grid((unsigned)n_pages_used, (unsigned)(a.n_kv / a.heads_per_block));
    hipLaunchKernelGGL(kv_gather_kernel, grid, dim3(kThreads), lds_bytes(a), s, a, staging_out);
    return hipGetLastError();
}

}  // namespace oc
