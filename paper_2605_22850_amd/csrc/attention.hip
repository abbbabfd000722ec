// Suffix-prefill GQA attention over a paged cached prefix plus the new
// suffix tokens (the per-layer compute C_l of eq. (3)).
//
// Work split: for each KV head g, the query rows are the (suffix token,
// query head of g's group) pairs, token-major, so one 32-row MFMA column
// block shares tokens across the group's heads (GQA packing).  A workgroup
// (4 wavefronts x 32 rows) owns a 128-row tile and one contiguous range of
// 64-key blocks; key ranges are split over workgroups (split-KV) so long
// prefixes fill the chip, and a combine kernel merges the splits by their
// log-sum-exp.  Workgroups that share (KV head, split) -- and therefore read
// the same K/V pages -- are launched onto the same XCD back to back so their
// re-reads hit that XCD's L2.
//
// Per 64-key block: the workgroup stages K ([key][dim]) and V ([dim][key],
// as the pool stores it) into LDS, each wavefront computes S^T = K Q^T with
// bf16 MFMA 32x32x16 (fp32 accumulate), updates the online softmax in
// registers (each lane owns one query column; the two half-waves combine
// their maxima), converts P to bf16 and accumulates O^T += V^T P.  Rows of
// the K tile are fed to the MFMA in an order that leaves each half-wave
// holding eight consecutive keys of P per MFMA step, which matches eight
// consecutive keys of one V row in LDS: both operands load as 16-byte vectors.
#include <math.h>

#include "common.hpp"

namespace oc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

constexpr int PAGE = 16;          // tokens per pool page (attention requires page_size 16)
constexpr int KB = 64;            // keys per block = 4 pages
constexpr int WAVES = 4;
constexpr int QW = 32;            // query rows per wavefront
constexpr int TILE_ROWS = WAVES * QW;
constexpr int THREADS = WAVES * 64;
constexpr int TARGET_WGS = 512;   // two workgroups per CU on 256 CUs

struct KParams {
    const uint16_t *q;
    const uint16_t *pool_k, *pool_v;
    const int32_t *pages;
    const uint16_t *ks, *vs;      // suffix pages packed like pool pages
    float *o_part, *ml_part;
    uint16_t *out;
    int64_t Tp, Ts, rows, rows_pad, n_pre_pages, n_suf_pages, n_blocks, blocks_per_split;
    int nq, nkv, grp, m_tiles, n_split, n_groups;
    float scale_log2;
};

// ---------------------------------------------------------------------------
// suffix K/V into page-shaped blocks (K [slot][dim], V [dim][slot]), zero past Ts
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void suffix_pack_kernel(const uint16_t *__restrict__ k_new,
                                                          const uint16_t *__restrict__ v_new,
                                                          uint16_t *__restrict__ ks, uint16_t *__restrict__ vs,
                                                          int64_t Ts, int nkv, int d) {
    const int64_t u = blockIdx.x;
    const int h = blockIdx.y;
    const int n = PAGE * d;
    for (int idx = threadIdx.x; idx < n; idx += 256) {
        int s = idx / d, e = idx - s * d;
        int64_t T = u * PAGE + s;
        ks[((u * nkv + h) * PAGE + s) * d + e] = T < Ts ? k_new[(T * nkv + h) * d + e] : (uint16_t)0;
        int e2 = idx / PAGE, s2 = idx - e2 * PAGE;
        int64_t T2 = u * PAGE + s2;
        vs[((u * nkv + h) * d + e2) * PAGE + s2] = T2 < Ts ? v_new[(T2 * nkv + h) * d + e2] : (uint16_t)0;
    }
}

__device__ inline float wave_partner(float x) { return __shfl_xor(x, 32); }

// tile row r of a 32-key MFMA tile reads physical key perm(r): bits 2 and 3 swapped
__device__ inline int key_perm(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

template <int D>
__global__ __launch_bounds__(THREADS) void attn_fwd_kernel(KParams p) {
    constexpr int KS = D + 8;      // padded LDS row of K (elements)
    constexpr int VS = KB + 8;     // padded LDS row of V
    constexpr int D8 = D / 8;
    constexpr int PIECES = PAGE * D8;            // 16-byte pieces per page block
    constexpr int PPT = 4 * PIECES / THREADS;    // pieces per thread per tile
    static_assert(PPT >= 1 && (4 * PIECES) % THREADS == 0, "tile does not divide over the workgroup");
    __shared__ __align__(16) uint16_t sk[KB * KS];
    __shared__ __align__(16) uint16_t sv[D * VS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 31, half = lane >> 5;

    // XCD-aware decode: workgroup w runs on XCD w % 8; all row tiles of one
    // (KV head, split) group get consecutive slots on the same XCD
    const int w = blockIdx.x;
    const int xcd = w & 7, local = w >> 3;
    const int gamma = (local / p.m_tiles) * 8 + xcd;
    if (gamma >= p.n_groups) return;
    const int mt = local % p.m_tiles;
    const int g = gamma / p.n_split, split = gamma - g * p.n_split;

    const int64_t row = (int64_t)mt * TILE_ROWS + wave * QW + col;
    const bool row_ok = row < p.rows;
    const int64_t tok = row_ok ? row / p.grp : 0;
    const int head = g * p.grp + (row_ok ? (int)(row % p.grp) : 0);

    bf16x8 qop[D / 16];
    {
        const uint16_t *qr = p.q + (tok * p.nq + head) * D + half * 8;
#pragma unroll
        for (int ds = 0; ds < D / 16; ++ds) {
            u32x4 v = row_ok ? *reinterpret_cast<const u32x4 *>(qr + ds * 16) : u32x4{0, 0, 0, 0};
            qop[ds] = __builtin_bit_cast(bf16x8, v);
        }
    }

    int64_t b0 = (int64_t)split * p.blocks_per_split;
    int64_t b1 = b0 + p.blocks_per_split;
    if (b1 > p.n_blocks) b1 = p.n_blocks;
    {   // causal clip: no row of this tile sees suffix keys past its last token
        int64_t row_hi = ((int64_t)mt + 1) * TILE_ROWS - 1;
        if (row_hi > p.rows - 1) row_hi = p.rows - 1;
        const int64_t last_page = p.n_pre_pages + (row_hi / p.grp) / PAGE;
        if (b1 > last_page / 4 + 1) b1 = last_page / 4 + 1;
    }
    const int64_t full_pre_pages = p.Tp / PAGE;

    f32x16 oacc[D / 32];
#pragma unroll
    for (int et = 0; et < D / 32; ++et) oacc[et] = f32x16{};
    float m_run = -__builtin_inff(), l_run = 0.f;

    u32x4 kreg[PPT], vreg[PPT];
    auto load_block = [&](int64_t b) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int piece = u * THREADS + tid;
            const int pg = piece / PIECES, within = piece - pg * PIECES;
            const int64_t v = b * 4 + pg;
            const uint16_t *kb = nullptr, *vb = nullptr;
            if (v < p.n_pre_pages) {
                const int64_t page = p.pages[v];
                kb = p.pool_k + (page * p.nkv + g) * (int64_t)(PAGE * D);
                vb = p.pool_v + (page * p.nkv + g) * (int64_t)(PAGE * D);
            } else if (v - p.n_pre_pages < p.n_suf_pages) {
                const int64_t su = v - p.n_pre_pages;
                kb = p.ks + (su * p.nkv + g) * (int64_t)(PAGE * D);
                vb = p.vs + (su * p.nkv + g) * (int64_t)(PAGE * D);
            }
            if (kb) {
                kreg[u] = *reinterpret_cast<const u32x4 *>(kb + within * 8);
                vreg[u] = *reinterpret_cast<const u32x4 *>(vb + within * 8);
            } else {
                kreg[u] = u32x4{0, 0, 0, 0};
                vreg[u] = u32x4{0, 0, 0, 0};
            }
        }
    };
    auto store_block = [&](int64_t b) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int piece = u * THREADS + tid;
            const int pg = piece / PIECES, within = piece - pg * PIECES;
            const int s = within / D8, e8 = within - s * D8;          // K block [slot][dim]
            *reinterpret_cast<u32x4 *>(&sk[(pg * PAGE + s) * KS + e8 * 8]) = kreg[u];
            const int e = within >> 1, sh = within & 1;                // V block [dim][slot]
            u32x4 vv = vreg[u];
            const int64_t v = b * 4 + pg;
            if (v == full_pre_pages && v < p.n_pre_pages) {
                // last, partial prefix page: slots past Tp may hold anything;
                // zero them so masked keys contribute exactly nothing
                const int valid = (int)(p.Tp - v * PAGE) - sh * 8;
                uint16_t t[8];
                __builtin_memcpy(t, &vv, 16);
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    if (i >= valid) t[i] = 0;
                __builtin_memcpy(&vv, t, 16);
            }
            *reinterpret_cast<u32x4 *>(&sv[e * VS + pg * PAGE + sh * 8]) = vv;
        }
    };

    const int krow_base = key_perm(col);
    if (b0 < b1) {
        load_block(b0);
        store_block(b0);
        __syncthreads();
    }
    for (int64_t b = b0; b < b1; ++b) {
        const bool more = b + 1 < b1;
        if (more) load_block(b + 1);

        // S^T = K Q^T for two 32-key tiles
        f32x16 sacc[2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            sacc[kt] = f32x16{};
            const uint16_t *kr = &sk[(kt * 32 + krow_base) * KS + half * 8];
#pragma unroll
            for (int ds = 0; ds < D / 16; ++ds) {
                bf16x8 a = *reinterpret_cast<const bf16x8 *>(kr + ds * 16);
                sacc[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qop[ds], sacc[kt], 0, 0, 0);
            }
        }

        // mask keys past the prefix end or past this row's own suffix token
        if ((b + 1) * 4 > full_pre_pages) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int kin = kt * 32 + (i < 8 ? 8 * half + i : 16 + 8 * half + (i - 8));
                    const int64_t v = b * 4 + (kin >> 4);
                    const int64_t slot = kin & 15;
                    bool ok;
                    if (v < p.n_pre_pages) ok = v * PAGE + slot < p.Tp;
                    else ok = (v - p.n_pre_pages) * PAGE + slot <= tok;
                    if (!ok) sacc[kt][i] = -__builtin_inff();
                }
            }
        }

        float mx = -__builtin_inff();
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kt][i]);
        mx = fmaxf(mx, wave_partner(mx));
        const float m_new = fmaxf(m_run, mx * p.scale_log2);
        const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        m_run = m_new;

        float lsum = 0.f;
        bf16x8 pop[2][2];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                f32x8 pv;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const float e = __builtin_amdgcn_exp2f(fmaf(sacc[kt][hf * 8 + i], p.scale_log2, -m_use));
                    lsum += e;
                    pv[i] = e;
                }
                pop[kt][hf] = __builtin_convertvector(pv, bf16x8);
            }
        }
        l_run = l_run * alpha + lsum;

        // O^T += V^T P
#pragma unroll
        for (int et = 0; et < D / 32; ++et) {
            oacc[et] *= alpha;
            const uint16_t *vr = &sv[(et * 32 + col) * VS + half * 8];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int hf = 0; hf < 2; ++hf) {
                    bf16x8 a = *reinterpret_cast<const bf16x8 *>(vr + kt * 32 + hf * 16);
                    oacc[et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pop[kt][hf], oacc[et], 0, 0, 0);
                }
        }

        __syncthreads();
        if (more) {
            store_block(b + 1);
            __syncthreads();
        }
    }

    const float l_tot = l_run + wave_partner(l_run);
    if (!row_ok) return;
    if (p.n_split == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        uint16_t *orow = p.out + (tok * p.nq + head) * D;
#pragma unroll
        for (int et = 0; et < D / 32; ++et)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                f32x4 o4 = {oacc[et][vq * 4 + 0] * inv, oacc[et][vq * 4 + 1] * inv, oacc[et][vq * 4 + 2] * inv,
                            oacc[et][vq * 4 + 3] * inv};
                typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
                bf16x4 b4 = __builtin_convertvector(o4, bf16x4);
                *reinterpret_cast<bf16x4 *>(orow + et * 32 + vq * 8 + half * 4) = b4;
            }
    } else {
        const int64_t prow = ((int64_t)split * p.nkv + g) * p.rows_pad + row;
        float *orow = p.o_part + prow * D;
#pragma unroll
        for (int et = 0; et < D / 32; ++et)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                f32x4 o4 = {oacc[et][vq * 4 + 0], oacc[et][vq * 4 + 1], oacc[et][vq * 4 + 2], oacc[et][vq * 4 + 3]};
                *reinterpret_cast<f32x4 *>(orow + et * 32 + vq * 8 + half * 4) = o4;
            }
        if (half == 0) {
            p.ml_part[prow * 2 + 0] = m_run;
            p.ml_part[prow * 2 + 1] = l_tot;
        }
    }
}

// Merge the splits of each row: weights 2^(m_s - M), normalised by the
// matching sum of l_s; bf16 out.
template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(KParams p) {
    constexpr int TPR = D / 4;                 // threads per row, 4 floats each
    constexpr int RPB = 256 / TPR;             // rows per block
    const int64_t gr = (int64_t)blockIdx.x * RPB + threadIdx.x / TPR;   // over nkv * rows
    const int c4 = threadIdx.x % TPR;
    if (gr >= (int64_t)p.nkv * p.rows) return;
    const int g = (int)(gr / p.rows);
    const int64_t row = gr - (int64_t)g * p.rows;
    float M = -__builtin_inff();
    for (int s = 0; s < p.n_split; ++s)
        M = fmaxf(M, p.ml_part[(((int64_t)s * p.nkv + g) * p.rows_pad + row) * 2]);
    const float Mu = M == -__builtin_inff() ? 0.f : M;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float L = 0.f;
    for (int s = 0; s < p.n_split; ++s) {
        const int64_t prow = ((int64_t)s * p.nkv + g) * p.rows_pad + row;
        const float w = __builtin_amdgcn_exp2f(p.ml_part[prow * 2] - Mu);
        L += w * p.ml_part[prow * 2 + 1];
        f32x4 o = *reinterpret_cast<const f32x4 *>(p.o_part + prow * D + c4 * 4);
        acc += w * o;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int64_t tok = row / p.grp;
    const int head = g * p.grp + (int)(row % p.grp);
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 b4 = __builtin_convertvector(acc * inv, bf16x4);
    *reinterpret_cast<bf16x4 *>(p.out + (tok * p.nq + head) * D + c4 * 4) = b4;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int plan_attention(const oc_layout &lay, int64_t Tp, int64_t Ts, AttnPlan *pl) {
    AttnPlan p{};
    p.Tp = Tp;
    p.Ts = Ts;
    p.nq = lay.num_q_heads;
    p.nkv = lay.num_kv_heads;
    p.grp = p.nq / p.nkv;
    p.d = lay.head_dim;
    p.rows = Ts * p.grp;
    p.m_tiles = (int)((p.rows + TILE_ROWS - 1) / TILE_ROWS);
    p.n_pre_pages = (Tp + PAGE - 1) / PAGE;
    p.n_suf_pages = (Ts + PAGE - 1) / PAGE;
    p.n_blocks = (p.n_pre_pages + p.n_suf_pages + 3) / 4;
    int64_t tiles = (int64_t)p.nkv * p.m_tiles;
    int64_t ns = (TARGET_WGS + tiles - 1) / tiles;
    if (ns > p.n_blocks) ns = p.n_blocks;
    if (ns < 1) ns = 1;
    p.blocks_per_split = (p.n_blocks + ns - 1) / ns;
    p.n_split = (int)((p.n_blocks + p.blocks_per_split - 1) / p.blocks_per_split);
    const int64_t rows_pad = (int64_t)p.m_tiles * TILE_ROWS;
    size_t off = 0;
    p.off_ks = off;
    off = round_up(off + (size_t)p.n_suf_pages * p.nkv * PAGE * p.d * 2, 256);
    p.off_vs = off;
    off = round_up(off + (size_t)p.n_suf_pages * p.nkv * PAGE * p.d * 2, 256);
    p.off_o = off;
    if (p.n_split > 1) off = round_up(off + (size_t)p.n_split * p.nkv * rows_pad * p.d * 4, 256);
    p.off_ml = off;
    if (p.n_split > 1) off = round_up(off + (size_t)p.n_split * p.nkv * rows_pad * 2 * 4, 256);
    p.total = off;
    *pl = p;
    return OC_OK;
}

template <int D>
static hipError_t launch_d(const AttnPlan &pl, const AttnArgs &a, hipStream_t s) {
    KParams p{};
    p.q = a.q;
    p.pool_k = a.pool_k;
    p.pool_v = a.pool_v;
    p.pages = a.pages;
    p.ks = reinterpret_cast<const uint16_t *>(a.ws + pl.off_ks);
    p.vs = reinterpret_cast<const uint16_t *>(a.ws + pl.off_vs);
    p.o_part = reinterpret_cast<float *>(a.ws + pl.off_o);
    p.ml_part = reinterpret_cast<float *>(a.ws + pl.off_ml);
    p.out = a.out;
    p.Tp = pl.Tp;
    p.Ts = pl.Ts;
    p.rows = pl.rows;
    p.rows_pad = (int64_t)pl.m_tiles * TILE_ROWS;
    p.n_pre_pages = pl.n_pre_pages;
    p.n_suf_pages = pl.n_suf_pages;
    p.n_blocks = pl.n_blocks;
    p.blocks_per_split = pl.blocks_per_split;
    p.nq = pl.nq;
    p.nkv = pl.nkv;
    p.grp = pl.grp;
    p.m_tiles = pl.m_tiles;
    p.n_split = pl.n_split;
    p.n_groups = pl.nkv * pl.n_split;
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));

    hipLaunchKernelGGL(suffix_pack_kernel, dim3((unsigned)pl.n_suf_pages, (unsigned)pl.nkv), dim3(256), 0, s,
                       a.k_new, a.v_new, const_cast<uint16_t *>(p.ks), const_cast<uint16_t *>(p.vs), pl.Ts,
                       pl.nkv, D);
    const int64_t groups_per_xcd = (p.n_groups + 7) / 8;
    const int64_t grid = 8 * groups_per_xcd * pl.m_tiles;
    hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3((unsigned)grid), dim3(THREADS), 0, s, p);
    if (pl.n_split > 1) {
        constexpr int RPB = 256 / (D / 4);
        const int64_t nrows = (int64_t)pl.nkv * pl.rows;
        hipLaunchKernelGGL(attn_combine_kernel<D>, dim3((unsigned)((nrows + RPB - 1) / RPB)), dim3(256), 0, s, p);
    }
    return hipGetLastError();
}

hipError_t launch_attention(const AttnPlan &pl, const AttnArgs &a, hipStream_t s) {
    if (pl.d == 128) return launch_d<128>(pl, a, s);
    return launch_d<64>(pl, a, s);
}

}  // namespace oc
