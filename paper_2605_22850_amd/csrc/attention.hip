// Suffix-prefill GQA attention over a paged cached prefix plus the new
// suffix tokens (the per-layer compute C_l of eq. (3)).
//
// Work split: for each KV head g the query rows are the (suffix token, query
// head of g's group) pairs, token-major, so one 32-row MFMA block shares
// tokens across the group's heads (GQA packing).  A workgroup of 8
// wavefronts owns 8 x 32 rows and one contiguous range of 64-key blocks; key
// ranges are split over workgroups (split-KV) so long prefixes fill the chip,
// and a combine kernel merges the splits by log-sum-exp.  Workgroups that read
// the same K/V pages (same KV head and split) are dispatched back to back onto
// the same XCD, so their re-reads hit that XCD's L2.
//
// Per 64-key block: the K and V rows of four pages ([slot][dim] pool blocks,
// or for the suffix the k_new / v_new rows themselves) are copied straight
// into token-major LDS tiles by the global->LDS load path, three blocks in
// flight, one barrier per block.  The tiles' 16-byte columns are XOR-swizzled
// by row so the operand reads are free of bank conflicts.  Each wavefront
// computes S^T = K Q^T for its 32 queries with bf16 MFMA 32x32x16 (fp32
// accumulate), runs the online softmax with one query column per lane (the
// two half-waves combine their maxima with a lane swap; the running maximum
// is only raised -- and O rescaled -- when a block's maximum exceeds it by more
// than 2^8), converts P to bf16 and accumulates O^T += V^T P.  The V^T operand
// (eight consecutive keys of one dimension per lane) comes from two
// transposing LDS reads of the token-major V tile.  The K tile's rows are fed
// to the MFMA in an order (bits 2 and 3 of the row swapped) that leaves each
// half-wave holding eight consecutive keys of P, matching those eight keys of
// the V operand.
#include <math.h>

#include <algorithm>
#include <mutex>

#include "common.hpp"

namespace oc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int PAGE = 16;          // tokens per pool page (attention requires page_size 16)
constexpr int KB = 64;            // keys per block = 4 pages
constexpr int WAVES = 8;          // two per SIMD: one's softmax overlaps the other's MFMAs
constexpr int QB = 1;             // 32-row query blocks per wavefront
constexpr int WAVE_ROWS = 32 * QB;
constexpr int TILE_ROWS = WAVES * WAVE_ROWS;
constexpr int THREADS = WAVES * 64;
constexpr int TARGET_WGS = 256;   // one workgroup per CU
constexpr int kMaxDevices = 64;   // devices a process may launch on
#ifndef OC_BATCH_ROUNDS
#define OC_BATCH_ROUNDS 2
#endif
constexpr int BATCH_ROUNDS = OC_BATCH_ROUNDS;   // workgroups per CU a batched launch may queue
constexpr float RESCALE_SLACK = 8.0f;   // log2 units the running max may lag
#ifndef OC_LOOKAHEAD
#define OC_LOOKAHEAD 4
#endif
constexpr int LOOKAHEAD = OC_LOOKAHEAD;   // MFMAs an operand read runs ahead of its use

struct KParams {
    const uint16_t *q;
    const uint16_t *pool_k, *pool_v;
    const int32_t *pages;
    const uint16_t *k_new, *v_new;   // suffix rows [Ts][nkv][D]
    float *o_part, *ml_part;
    uint16_t *out;
    int64_t Tp, Ts, rows, rows_pad, n_pre_pages, n_suf_pages, n_blocks, blocks_per_split;
    int nq, nkv, grp, m_tiles, n_split, n_groups;
    float scale_log2;
};

// One launch serves up to MAX_ATTN_BATCH requests of one layer: workgroup w
// belongs to the last request whose first workgroup it has reached (and a
// block of the split merge, likewise, to the last whose first block it has
// reached; a request without splits has none).
struct KBatch {
    int32_t n;
    int32_t first_wg[MAX_ATTN_BATCH];
    int32_t first_cb[MAX_ATTN_BATCH];
    KParams req[MAX_ATTN_BATCH];
};

// value of the lane 32 positions away (the other half of the wavefront)
__device__ inline float half_swap_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float half_swap_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier that waits only for this wavefront's LDS operations.
// (__syncthreads() would also wait for every outstanding global load, which
// would stall the register prefetch of the block after next.)
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// tile row r of a 32-key MFMA tile reads physical key perm(r): bits 2 and 3 swapped
__device__ inline int key_perm(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// LDS element offset of 16-byte column c of K tile row r (D/8 columns per row)
template <int D>
__device__ inline int k_lds(int r, int c) {
    constexpr int NS = D / 8;
    return r * D + ((c ^ (r & (NS - 1))) << 3);
}

// XOR applied to the 16-byte column index of V tile row r.  The transposing
// reads of the PV operand take 4 dims x 4 keys per 16-lane group, from rows
// that differ in their low key bits; this spreads those rows over all banks.
template <int D>
__device__ inline int v_swz(int r) {
    if constexpr (D == 128) return 4 * (r & 3);
    else return 4 * ((r >> 1) & 1);
}

typedef __attribute__((address_space(3))) void *lds_ptr_t;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// one 16-byte global -> LDS copy per lane from `base` (wave-uniform) plus the
// lane's byte offset; the wavefront's 64 lanes fill 1 KiB of LDS starting at
// `lds_chunk`, lane i at byte 16*i.  Issued as inline
// assembly on purpose: the compiler treats every outstanding global->LDS copy
// as a possible writer of any LDS address, and would make each operand read
// of the current tile wait (vmcnt(0)) for the copies of the blocks still in
// flight, which serialises the prefetch.  The kernel orders these copies
// itself: wait_vmcnt before the per-block barrier, which is the only point
// where a tile becomes readable, and a buffer is refilled only after every
// wavefront has passed the barrier that follows its last read.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is written here and read by nothing else in these kernels
__device__ inline void dma16(const void *base, uint32_t lane_off, uint16_t *lds_chunk) {
    const uint32_t m0 = (uint32_t)(uintptr_t)(lds_ptr_t)lds_chunk;   // LDS byte address, wave-uniform
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(lane_off), "s"(base), "s"(m0)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ inline void wait_vmcnt() {
    static_assert(N == 0 || N == 2 || N == 4, "unexpected count");
    if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else if constexpr (N == 2) asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
}

// Per-wavefront running state of the online softmax for its 32 query rows.
template <int D>
struct WaveState {
    f32x16 o[D / 32];    // O^T: 32 dims x 32 rows per tile, fp32
    f32x16 s[2];         // scores of the current block, one 32-key half each
    bf16x8 p[2][2];      // P of the last softmaxed block as the PV operand: [half][8-key group]
    float m, l;          // running maximum (log2 units) and sum of this lane's row
};

// Matrix phase of a wavefront: O^T += V^T P for the previous block (PV:
// 16 MFMAs at d = 128, each V^T fragment from two transposing LDS reads),
// then S^T = K Q^T for the current block (S: 16 MFMAs, K fragments from the
// swizzled tile, the two 32-key halves alternating so that consecutive MFMAs
// are independent).  Written as one flat sequence whose operand reads run
// LOOKAHEAD MFMAs ahead (with PV, the first LOOKAHEAD come preloaded, see
// prefetch_vt); a scheduling fence after every MFMA keeps that order (left
// alone, the compiler hoists every read to the top and runs out of VGPRs).
// V^T fragment n of a PV pass (n = 8-key group * D/32 + dim tile)
template <int D>
__device__ __forceinline__ bf16x8 load_vt(const uint16_t *V, const int (&voff)[D / 32], int n) {
    constexpr int NET = D / 32;
    const int et = n % NET, g4 = n / NET;     // g4 = 2*half + key group
    const uint16_t *vp = V + voff[et] + ((g4 >> 1) * 32 + (g4 & 1) * 16) * D;
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)vp);
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(vp + 4 * D));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// The first LOOKAHEAD V^T fragments of a PV pass, read ahead of the barrier
// that opens the matrix phase (the V tile of the previous block is already
// readable there), so the phase starts without waiting on LDS.
template <int D>
__device__ __forceinline__ void prefetch_vt(const uint16_t *V, const int (&voff)[D / 32], bf16x8 (&pre)[LOOKAHEAD]) {
#pragma unroll
    for (int n = 0; n < LOOKAHEAD; ++n) pre[n] = load_vt<D>(V, voff, n);
}

template <int D, bool PV, bool S>
__device__ __forceinline__ void matrix_phase(WaveState<D> &w, const uint16_t *V, const int (&voff)[D / 32],
                                             const uint16_t *K, const bf16x8 (&qop)[D / 16], int krow, int half,
                                             const bf16x8 (&pre)[LOOKAHEAD]) {
    constexpr int NET = D / 32, NDS = D / 16;
    constexpr int NPV = PV ? 4 * NET : 0;
    constexpr int N = NPV + (S ? 2 * NDS : 0);
    static_assert(!PV || NPV >= LOOKAHEAD, "prefetched fragments must all be V^T fragments");
    auto load = [&](int n) -> bf16x8 {
        if (n < NPV) return load_vt<D>(V, voff, n);
        const int n2 = n - NPV, ds = n2 >> 1, kt = n2 & 1;
        return *reinterpret_cast<const bf16x8 *>(&K[k_lds<D>(kt * 32 + krow, ds * 2 + half)]);
    };
    bf16x8 f[N];
    // the wavefront in its matrix phase issues ahead of its SIMD partner's
    // softmax: the MFMA pipe is the longer of the two (about 3 % per layer)
    __builtin_amdgcn_s_setprio(2);
#pragma unroll
    for (int n = 0; n < LOOKAHEAD && n < N; ++n) f[n] = PV ? pre[n] : load(n);
#pragma unroll
    for (int n = 0; n < N; ++n) {
        if (n + LOOKAHEAD < N) f[n + LOOKAHEAD] = load(n + LOOKAHEAD);
        if (n < NPV) {
            const int et = n % NET, g4 = n / NET;
            w.o[et] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[n], w.p[g4 >> 1][g4 & 1], w.o[et], 0, 0, 0);
        } else {
            const int n2 = n - NPV, ds = n2 >> 1, kt = n2 & 1;
            w.s[kt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[n], qop[ds], ds == 0 ? f32x16{} : w.s[kt], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    __builtin_amdgcn_s_setprio(1);
}

// Softmax phase of a wavefront for one block: the block maximum (one lane
// swap between the half-waves), the lazy raise of the running maximum (O and
// l rescaled only when the block maximum exceeds it by more than
// 2^RESCALE_SLACK), then P = 2^(s*scale*log2(e) - m) as bf16 and the row sums
// of that rounded P.
template <int D>
__device__ __forceinline__ void softmax_phase(WaveState<D> &w, float scale_log2) {
    float mx[2] = {-__builtin_inff(), -__builtin_inff()};   // two partial maxima
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int i2 = 0; i2 < 16; ++i2) mx[i2 & 1] = fmaxf(mx[i2 & 1], w.s[kt][i2]);
    const float mblk = half_swap_max(fmaxf(mx[0], mx[1])) * scale_log2;
    if (__any(mblk > w.m + RESCALE_SLACK)) {
        const float m_new = fmaxf(w.m, mblk);
        const float alpha = __builtin_amdgcn_exp2f(w.m - (m_new == -__builtin_inff() ? 0.f : m_new));
        w.m = m_new;
        w.l *= alpha;
#pragma unroll
        for (int et = 0; et < D / 32; ++et) w.o[et] *= alpha;
    }
    const float m_use = w.m == -__builtin_inff() ? 0.f : w.m;
    // row sums of the rounded P (the values the PV product uses), two bf16
    // pairs per dot instruction, two partial sums
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const bf16x2 ones = {(__bf16)1.f, (__bf16)1.f};
    float lsum[2] = {0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            f32x8 pv;
#pragma unroll
            for (int i2 = 0; i2 < 8; ++i2)
                pv[i2] = __builtin_amdgcn_exp2f(fmaf(w.s[kt][hf * 8 + i2], scale_log2, -m_use));
            const bf16x8 pp = __builtin_convertvector(pv, bf16x8);
            w.p[kt][hf] = pp;
            lsum[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pp, pp, 0, 1), ones, lsum[0], false);
            lsum[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pp, pp, 2, 3), ones, lsum[1], false);
            lsum[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pp, pp, 4, 5), ones, lsum[0], false);
            lsum[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pp, pp, 6, 7), ones, lsum[1], false);
        }
    w.l += lsum[0] + lsum[1];
}

template <int D>
__global__ __launch_bounds__(THREADS) void attn_fwd_kernel(KBatch batch) {
    // read the request's parameters straight from the kernel-argument segment
    // (scalar loads at a uniform offset; indexing the by-value copy would
    // place it in scratch memory)
    typedef const __attribute__((address_space(4))) KBatch *kbatch_ptr;
    // every wavefront issues ahead of the ingest wavefronts that may share
    // its SIMD (they keep the lowest priority); the matrix phase goes one
    // level higher still
    __builtin_amdgcn_s_setprio(1);
    const kbatch_ptr bp = (kbatch_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    int req = 0;
    for (int i = 1; i < bp->n; ++i) req += (int)blockIdx.x >= bp->first_wg[i];
    const __attribute__((address_space(4))) KParams &p = bp->req[req];
    const int wg = (int)blockIdx.x - bp->first_wg[req];
    // Every parameter is read once into a register here: read through `p`
    // inside the loop, each use would be reloaded from the argument segment
    // after every inline-assembly statement (they clobber memory), each reload
    // a scalar load that the next LDS wait must also wait for.  Token, page,
    // block and row counts fit 32 bits (the host limits prefix + suffix to
    // 2^30 tokens and rows to 2^30).
    const int m_tiles = p.m_tiles, n_groups = p.n_groups, n_split = p.n_split;
    const int grp = p.grp, nq = p.nq, nkv = p.nkv;
    const int rows = (int)p.rows, Tp = (int)p.Tp, Ts = (int)p.Ts, n_pre_pages = (int)p.n_pre_pages;
    const int n_blocks = (int)p.n_blocks, blocks_per_split = (int)p.blocks_per_split;
    const int64_t rows_pad = p.rows_pad;
    const float scale_log2 = p.scale_log2;
    const uint16_t *const q_in = p.q;
    const uint16_t *const pool_k = p.pool_k, *const pool_v = p.pool_v;
    const uint16_t *const k_new = p.k_new, *const v_new = p.v_new;
    uint16_t *const out_ptr = p.out;
    float *const o_part = p.o_part, *const ml_part = p.ml_part;
    const __attribute__((address_space(4))) int32_t *pages_c =
        (const __attribute__((address_space(4))) int32_t *)p.pages;
    constexpr int TILE = KB * D;                   // elements of one K (or V) tile
    constexpr int CHUNKS = TILE * 2 / 1024;        // 1 KiB DMA chunks per tile
    constexpr int CPW = CHUNKS / WAVES;            // chunks per wavefront per tile
    constexpr int KROWS = 512 / D;                 // K rows per chunk
    constexpr int CPP = D / 32;                    // chunks per page (K and V alike)
    constexpr int NDMA = 2 * CPW;                  // DMA instructions per wavefront per block
    // buffers: the current block, the previous one (its V is read in this
    // block's phase B), and two blocks whose copies are in flight
    constexpr int NBUF = 4;
    static_assert(CPW >= 1 && CHUNKS % WAVES == 0, "tile does not divide");
    extern __shared__ __align__(1024) uint16_t lds[];   // [NBUF][K tile, V tile]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31, half = lane >> 5;

    // XCD-aware decode: workgroup w runs on XCD w % 8; all row tiles of one
    // (KV head, split) group get consecutive slots on the same XCD, the last
    // row tile first: under the causal mask later rows see more suffix keys,
    // and dispatching the longest tiles first keeps them out of the tail
    const int xcd = wg & 7, local = wg >> 3;
    const int gamma = (local / m_tiles) * 8 + xcd;
    if (gamma >= n_groups) return;
    const int mt = m_tiles - 1 - local % m_tiles;
    const int g = gamma / n_split, split = gamma - g * n_split;

    const int row = mt * TILE_ROWS + wave * WAVE_ROWS + col;
    const bool row_ok = row < rows;
    const int tok = row_ok ? row / grp : 0;
    bf16x8 qop[D / 16];
    {
        const int head = g * grp + (row_ok ? row % grp : 0);
        const uint16_t *qr = q_in + ((int64_t)tok * nq + head) * D + half * 8;
#pragma unroll
        for (int ds = 0; ds < D / 16; ++ds) {
            u32x4 v = row_ok ? *reinterpret_cast<const u32x4 *>(qr + ds * 16) : u32x4{0, 0, 0, 0};
            qop[ds] = __builtin_bit_cast(bf16x8, v);
        }
    }

    const int b0 = split * blocks_per_split;
    int b1 = b0 + blocks_per_split;
    if (b1 > n_blocks) b1 = n_blocks;
    {   // causal clip: no row of this tile sees suffix keys past its last token
        int row_hi = (mt + 1) * TILE_ROWS - 1;
        if (row_hi > rows - 1) row_hi = rows - 1;
        const int last_page = n_pre_pages + (row_hi / grp) / PAGE;
        if (b1 > last_page / 4 + 1) b1 = last_page / 4 + 1;
    }
    const int full_pre_pages = Tp / PAGE;
    const int64_t head_block = (int64_t)PAGE * D;      // elements of one (page, head) block

    // ---- global -> LDS copy of one 64-key block (4 pages) ----
    // Both tiles are token-major ([key][dim]) with 16-byte columns XOR-swizzled
    // by key row (K for the S reads, V for the transposing PV reads); each
    // lane fetches the global piece that belongs at its fixed LDS position.
    // Every 1 KiB chunk comes from a single page; a wavefront copies CPW
    // chunks of each tile.  The base pointers stay in registers, and the page
    // ids of a block are loaded (scalar loads through the constant address
    // space) one block ahead of its copy, so no copy waits on a lookup.
    auto load_pids = [&](int b, int32_t (&pid)[CPW]) {
#pragma unroll
        for (int u = 0; u < CPW; ++u) {
            const int v = b * 4 + (u * WAVES + wave) / CPP;
            pid[u] = v < n_pre_pages ? pages_c[v] : 0;
        }
    };
    // per-lane parts of the copy addresses (bytes), fixed for the whole loop:
    // chunk u of a wavefront covers key rows rr[u] + [0, KROWS) of its page
    uint32_t klane[CPW], vlane[CPW];
    int rr[CPW];
#pragma unroll
    for (int u = 0; u < CPW; ++u) {
        const unsigned q = (unsigned)(u * WAVES + wave);
        const int r = (int)(q % CPP) * KROWS + lane / (D / 8);   // key row within the page
        const int ck = (lane % (D / 8)) ^ (r & (D / 8 - 1));
        const int cv = (lane % (D / 8)) ^ v_swz<D>(r);
        rr[u] = r;
        klane[u] = (uint32_t)(r * D + ck * 8) * 2;
        vlane[u] = (uint32_t)(r * D + cv * 8) * 2;
    }
    auto issue_block = [&](int b, int buf, const int32_t (&pid)[CPW]) {
        uint16_t *kt_lds = lds + buf * 2 * TILE;
        uint16_t *vt_lds = kt_lds + TILE;
#pragma unroll
        for (int u = 0; u < CPW; ++u) {
            const int q = u * WAVES + wave;                   // chunk index, uniform per wavefront
            const int v = b * 4 + q / CPP;                    // page of the key sequence
            if (v < n_pre_pages) {
                const int64_t blk = ((int64_t)pid[u] * nkv + g) * head_block;
                dma16(pool_k + blk, klane[u], kt_lds + q * 512);
                dma16(pool_v + blk, vlane[u], vt_lds + q * 512);
            } else {
                // suffix token; rows past the last one repeat it (finite, and masked)
                int T = (v - n_pre_pages) * PAGE + rr[u];
                if (T > Ts - 1) T = Ts - 1;
                // below 2^31: the host limits T_s * n_kv * d * 2 bytes
                const uint32_t rw = ((uint32_t)(T * nkv + g) * D - (uint32_t)rr[u] * D) * 2;
                dma16(k_new, rw + klane[u], kt_lds + q * 512);
                dma16(v_new, rw + vlane[u], vt_lds + q * 512);
            }
        }
    };

    WaveState<D> w;
#pragma unroll
    for (int et = 0; et < D / 32; ++et) w.o[et] = f32x16{};
    w.m = -__builtin_inff();
    w.l = 0.f;
    const int krow = key_perm(col);
    // Transposing V reads: in each 16-lane group, source lane 4j+q names the
    // four dims [4q, 4q+4) of key row j; output lane i then holds dim i of
    // the four rows.  Group k covers dims 16*(k%2) + [0,16) and keys
    // 8*(k/2) + [0,4) of the 16-key slice (the second read adds 4 rows).
    int voff[D / 32];
    {
        const int k16 = lane >> 4, j = (lane >> 2) & 3, q4 = lane & 3;
        const int key = 8 * (k16 >> 1) + j;
#pragma unroll
        for (int et = 0; et < D / 32; ++et) {
            const int dim = et * 32 + 16 * (k16 & 1) + 4 * q4;
            voff[et] = key * D + (((dim >> 3) ^ v_swz<D>(key)) << 3) + (dim & 7);
        }
    }

    // Mask of one block: keys [0, pe) of the block are prefix keys, suffix
    // keys start at ps, and a row sees suffix key k (block position) when
    // k - ps <= its token.  Branch-free bitwise select of the score or -inf
    // (a short-circuit form was compiled into divergent branches that
    // dropped the kept value).
    // (The limits are shifted by this half-wave's key offset so that each
    // comparison is against a constant: no per-lane key index stays live.)
    auto mask_block = [&](int b) {
        const int sh = 8 * half;
        const int pe = Tp - b * KB - sh;
        const int ps = n_pre_pages * PAGE - b * KB - sh;
        const int lim = tok + ps;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int i2 = 0; i2 < 16; ++i2) {
                const int kin = kt * 32 + (i2 < 8 ? i2 : 8 + i2);   // key in the block, less 8*half
                const uint32_t keep = 0u - (uint32_t)((kin < pe) | ((kin >= ps) & (kin <= lim)));
                w.s[kt][i2] = __uint_as_float((__float_as_uint(w.s[kt][i2]) & keep) | (0xff800000u & ~keep));
            }
    };
    // Q operands are in registers before the key loop starts (a wait the
    // compiler sees, so it places none of its own inside the loop)
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    const int nb = b1 > b0 ? b1 - b0 : 0;
    int32_t pid[CPW];
    if (nb > 0) {
        load_pids(b0, pid);
        issue_block(b0, 0, pid);
    }
    if (nb > 1) {
        load_pids(b0 + 1, pid);
        issue_block(b0 + 1, 1, pid);
    }
    if (nb > 2) load_pids(b0 + 2, pid);
    // Ping-pong schedule.  Each wavefront alternates a matrix phase (PV of
    // block j-1, S of block j) and a softmax phase (block j); wavefronts 4-7
    // (the second wavefront of every SIMD) run the same sequence one phase
    // later than wavefronts 0-3, so on every SIMD one wavefront's MFMAs run
    // beside the other's softmax.  A workgroup barrier ends every phase.
    // Block j's tile becomes readable at phase 2j: its copies were started
    // at phase 2j-4 and each wavefront waits for its own before the barrier;
    // the copy of block j+2 then goes into the buffer of block j-2, whose
    // last reads (wavefronts 4-7's PV of block j-2) ended with phase 2j-1.
    const bool first = (wave >> 2) == 0;
    auto tile_k = [&](int j) -> const uint16_t * { return lds + (j % NBUF) * 2 * TILE; };
    auto tile_v = [&](int j) -> const uint16_t * { return lds + (j % NBUF) * 2 * TILE + TILE; };
    // phase 2j: block j's tile becomes readable, block j+2's copy starts
    auto open_block = [&](int j) {
        if (j + 1 < nb) wait_vmcnt<NDMA>();
        else wait_vmcnt<0>();
        lds_barrier();
        if (j + 2 < nb) issue_block(b0 + j + 2, (j + 2) % NBUF, pid);
        if (j + 3 < nb) load_pids(b0 + j + 3, pid);
        const int b = b0 + j;
        if (j < nb && (b + 1) * 4 > full_pre_pages && b * 4 <= full_pre_pages && full_pre_pages < n_pre_pages) {
            // last, partial prefix page: its slots past Tp may hold anything;
            // zero them so masked keys contribute exactly nothing (the V
            // tile is first read after the next barrier)
            uint16_t *V = lds + (j % NBUF) * 2 * TILE + TILE;
            const int pg = full_pre_pages - b * 4, k0 = Tp % PAGE;
            for (int idx = tid; idx < D * (PAGE - k0); idx += THREADS) V[(pg * PAGE + k0) * D + idx] = 0;
        }
    };
    // A block needs the mask only if it holds slots of the prefix's partial
    // last page, or suffix keys that some row of this wavefront does not see
    // yet (the wavefront's rows start at token tok_min).
    const int tok_min = (mt * TILE_ROWS + wave * WAVE_ROWS) / grp;
    auto softmax_block = [&](int j) {
        const int b = b0 + j;
        if ((b + 1) * 4 > full_pre_pages) {
            const int ps = n_pre_pages * PAGE - b * KB, pe = Tp - b * KB;
            const bool partial_prefix = ps > 0 && pe < (ps < KB ? ps : KB);
            const bool unseen_suffix = ps < KB && KB - 1 - ps > tok_min;
            if (partial_prefix || unseen_suffix) mask_block(b);
        }
        softmax_phase<D>(w, scale_log2);
    };
    // Each group runs its own copy of the loop (one straight path each, so
    // the accumulators keep their registers); both execute the same barriers.
    if (nb > 0) {
        bf16x8 pre[LOOKAHEAD];
        if (first) {
            open_block(0);
            matrix_phase<D, false, true>(w, nullptr, voff, tile_k(0), qop, krow, half, pre);
            lds_barrier();
            softmax_block(0);
            for (int j = 1; j < nb; ++j) {
                prefetch_vt<D>(tile_v(j - 1), voff, pre);
                open_block(j);
                matrix_phase<D, true, true>(w, tile_v(j - 1), voff, tile_k(j), qop, krow, half, pre);
                lds_barrier();
                softmax_block(j);
            }
            prefetch_vt<D>(tile_v(nb - 1), voff, pre);
            open_block(nb);
            matrix_phase<D, true, false>(w, tile_v(nb - 1), voff, nullptr, qop, krow, half, pre);
            lds_barrier();
        } else {
            open_block(0);
            lds_barrier();
            matrix_phase<D, false, true>(w, nullptr, voff, tile_k(0), qop, krow, half, pre);
            for (int j = 1; j < nb; ++j) {
                open_block(j);
                softmax_block(j - 1);
                prefetch_vt<D>(tile_v(j - 1), voff, pre);
                lds_barrier();
                matrix_phase<D, true, true>(w, tile_v(j - 1), voff, tile_k(j), qop, krow, half, pre);
            }
            open_block(nb);
            softmax_block(nb - 1);
            prefetch_vt<D>(tile_v(nb - 1), voff, pre);
            lds_barrier();
            matrix_phase<D, true, false>(w, tile_v(nb - 1), voff, nullptr, qop, krow, half, pre);
        }
    }

    const float l_tot = half_swap_sum(w.l);
    if (!row_ok) return;
    if (n_split == 1) {
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        const int head = g * grp + row % grp;
        uint16_t *orow = out_ptr + ((int64_t)tok * nq + head) * D;
#pragma unroll
        for (int et = 0; et < D / 32; ++et)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                f32x4 o4 = {w.o[et][vq * 4 + 0], w.o[et][vq * 4 + 1], w.o[et][vq * 4 + 2], w.o[et][vq * 4 + 3]};
                *reinterpret_cast<bf16x4 *>(orow + et * 32 + vq * 8 + half * 4) = __builtin_convertvector(o4 * inv, bf16x4);
            }
    } else {
        const int64_t prow = ((int64_t)split * nkv + g) * rows_pad + row;
        float *orow = o_part + prow * D;
#pragma unroll
        for (int et = 0; et < D / 32; ++et)
#pragma unroll
            for (int vq = 0; vq < 4; ++vq) {
                f32x4 o4 = {w.o[et][vq * 4 + 0], w.o[et][vq * 4 + 1], w.o[et][vq * 4 + 2], w.o[et][vq * 4 + 3]};
                *reinterpret_cast<f32x4 *>(orow + et * 32 + vq * 8 + half * 4) = o4;
            }
        if (half == 0) {
            ml_part[prow * 2 + 0] = w.m;
            ml_part[prow * 2 + 1] = l_tot;
        }
    }
}

template <int D>
constexpr size_t attn_lds_bytes() { return (size_t)4 * 2 * KB * D * 2; }

// Merge the splits of each row: weights 2^(m_s - M), normalised by the
// matching sum of l_s; bf16 out.  Block `blk` of a request's merge covers
// RPB of its (KV head, row) pairs.
template <int D>
__device__ __forceinline__ void combine_block(const float *ml_part, const float *o_part, uint16_t *out, int nkv,
                                              int64_t rows, int64_t rows_pad, int n_split, int grp, int nq,
                                              int64_t blk) {
    constexpr int TPR = D / 4;                 // threads per row, 4 floats each
    constexpr int RPB = 256 / TPR;             // rows per block
    const int64_t gr = blk * RPB + threadIdx.x / TPR;   // over nkv * rows
    const int c4 = threadIdx.x % TPR;
    if (gr >= (int64_t)nkv * rows) return;
    const int g = (int)(gr / rows);
    const int64_t row = gr - (int64_t)g * rows;
    // One pass over the splits, eight at a time: a group's (m, l) pairs and
    // partial rows are independent loads issued together, so the merge waits
    // on memory once per group rather than once for the maxima and again
    // for the sums; the running maximum rescales what earlier groups added.
    const int64_t split_stride = (int64_t)nkv * rows_pad;
    const int64_t prow0 = (int64_t)g * rows_pad + row;
    constexpr int GS = 8;
    float M = -__builtin_inff(), L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int s0 = 0; s0 < n_split; s0 += GS) {
        float2 ml[GS];
        f32x4 o[GS];
#pragma unroll
        for (int i = 0; i < GS; ++i) {
            if (s0 + i < n_split) {
                const int64_t prow = prow0 + (int64_t)(s0 + i) * split_stride;
                ml[i] = *reinterpret_cast<const float2 *>(ml_part + prow * 2);
                o[i] = *reinterpret_cast<const f32x4 *>(o_part + prow * D + c4 * 4);
            }
        }
        float Mg = M;
#pragma unroll
        for (int i = 0; i < GS; ++i)
            if (s0 + i < n_split) Mg = fmaxf(Mg, ml[i].x);
        const float Mu = Mg == -__builtin_inff() ? 0.f : Mg;
        const float r = __builtin_amdgcn_exp2f(M - Mu);     // 0 while nothing has been added
        L *= r;
        acc *= r;
#pragma unroll
        for (int i = 0; i < GS; ++i) {
            if (s0 + i < n_split) {
                const float w = __builtin_amdgcn_exp2f(ml[i].x - Mu);
                L += w * ml[i].y;
                acc += w * o[i];
            }
        }
        M = Mg;
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int64_t tok = row / grp;
    const int head = g * grp + (int)(row % grp);
    *reinterpret_cast<bf16x4 *>(out + (tok * nq + head) * D + c4 * 4) = __builtin_convertvector(acc * inv, bf16x4);
}

// The merge of one request, with its parameters alone as the kernel
// arguments (a lone request's launch stays short).
template <int D>
__global__ __launch_bounds__(256) void attn_combine_kernel(KParams p) {
    combine_block<D>(p.ml_part, p.o_part, p.out, p.nkv, p.rows, p.rows_pad, p.n_split, p.grp, p.nq, blockIdx.x);
}

// The merges of every request of a batch that has splits, in one launch.
template <int D>
__global__ __launch_bounds__(256) void attn_combine_batch_kernel(KBatch batch) {
    // parameters straight from the kernel-argument segment, as in the
    // attention kernel
    typedef const __attribute__((address_space(4))) KBatch *kbatch_ptr;
    const kbatch_ptr bp = (kbatch_ptr)__builtin_amdgcn_kernarg_segment_ptr();
    int req = 0;
    for (int i = 1; i < bp->n; ++i) req += (int)blockIdx.x >= bp->first_cb[i];
    const __attribute__((address_space(4))) KParams &p = bp->req[req];
    combine_block<D>(p.ml_part, p.o_part, p.out, p.nkv, p.rows, p.rows_pad, p.n_split, p.grp, p.nq,
                     (int64_t)blockIdx.x - bp->first_cb[req]);
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Tiles and key blocks of one request; the split count is set apart.
static AttnPlan plan_shape(const oc_layout &lay, int64_t Tp, int64_t Ts) {
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
    return p;
}

// Split the keys into ns ranges, then size the workspace.
static void plan_splits(AttnPlan &p, int64_t ns) {
    if (ns > p.n_blocks) ns = p.n_blocks;
    if (ns < 1) ns = 1;
    p.blocks_per_split = (p.n_blocks + ns - 1) / ns;
    p.n_split = (int)((p.n_blocks + p.blocks_per_split - 1) / p.blocks_per_split);
    const int64_t rows_pad = (int64_t)p.m_tiles * TILE_ROWS;
    size_t off = 0;
    p.off_o = off;
    if (p.n_split > 1) off = round_up(off + (size_t)p.n_split * p.nkv * rows_pad * p.d * 4, 256);
    p.off_ml = off;
    if (p.n_split > 1) off = round_up(off + (size_t)p.n_split * p.nkv * rows_pad * 2 * 4, 256);
    p.total = off > 256 ? off : 256;   // never 0: a size of 0 reports an unsupported shape
}

// One request alone: split the keys so that its row tiles fill the CUs.
int plan_attention(const oc_layout &lay, int64_t Tp, int64_t Ts, AttnPlan *pl) {
    AttnPlan p = plan_shape(lay, Tp, Ts);
    const int64_t tiles = (int64_t)p.nkv * p.m_tiles;
    plan_splits(p, (TARGET_WGS + tiles - 1) / tiles);
    *pl = p;
    return OC_OK;
}

// Several requests in one launch: every workgroup gets at most `budget` key
// blocks, the smallest budget that keeps the launch within BATCH_ROUNDS
// workgroups per CU (or one range per tile, if there are more tiles), so the
// dispatcher can even out long and short prefixes as CUs free up.
int plan_attention_batch(const oc_layout &lay, const int64_t *Tp, const int64_t *Ts, int n, AttnPlan *plans) {
    int64_t tiles = 0, work = 0, longest = 1;
    for (int i = 0; i < n; ++i) {
        plans[i] = plan_shape(lay, Tp[i], Ts[i]);
        const int64_t t = (int64_t)plans[i].nkv * plans[i].m_tiles;
        tiles += t;
        work += t * plans[i].n_blocks;
        longest = std::max<int64_t>(longest, plans[i].n_blocks);
    }
    auto wgs_for = [&](int64_t budget) {
        int64_t w = 0;
        for (int i = 0; i < n; ++i)
            w += (int64_t)plans[i].nkv * plans[i].m_tiles * ((plans[i].n_blocks + budget - 1) / budget);
        return w;
    };
    const int64_t cap = std::max<int64_t>((int64_t)TARGET_WGS * BATCH_ROUNDS, tiles);
    int64_t budget = std::max<int64_t>(1, (work + cap - 1) / cap);
    while (budget < longest && wgs_for(budget) > cap) ++budget;
    for (int i = 0; i < n; ++i) plan_splits(plans[i], (plans[i].n_blocks + budget - 1) / budget);
    return OC_OK;
}

int64_t attention_grid(const AttnPlan &p) { return 8 * (((int64_t)p.nkv * p.n_split + 7) / 8) * p.m_tiles; }

// a dispatch holds at most 2^32 - 1 work-items along x
int64_t attention_max_grid() { return OC_MAX_GRID_ITEMS / THREADS; }

size_t attention_lds_bytes(int head_dim) {
    return head_dim == 64 ? attn_lds_bytes<64>() : head_dim == 128 ? attn_lds_bytes<128>() : 0;
}

int check_attention_shape(const oc_layout &l, int64_t Tp, int64_t Ts) {
    if (l.head_dim != 64 && l.head_dim != 128) return fail(OC_ESHAPE, "attention supports head_dim 64 or 128");
    if (l.page_size != PAGE) return fail(OC_ESHAPE, "attention supports page_size 16");
    if (Tp < 0 || Ts < 1) return fail(OC_EINVAL, "attention needs prefix_tokens >= 0 and suffix_tokens >= 1");
    // the suffix rows are copied to LDS with 32-bit byte offsets from k_new / v_new
    if (Ts * l.num_kv_heads * l.head_dim * 2 > INT32_MAX)
        return fail(OC_ERANGE, "suffix K/V of more than 2^31 bytes (suffix_tokens * n_kv * d * 2)");
    // key positions, query rows and their tokens are 32-bit in the kernels
    if (Tp + Ts > (int64_t)1 << 30) return fail(OC_ERANGE, "prefix + suffix tokens exceed 2^30");
    const int64_t grp = l.num_q_heads / l.num_kv_heads;
    if (Ts * grp > (int64_t)1 << 30) return fail(OC_ERANGE, "suffix_tokens * (n_q / n_kv) exceeds 2^30");
    AttnPlan p;
    plan_attention(l, Tp, Ts, &p);
    if (attention_grid(p) > attention_max_grid())
        return fail(OC_ERANGE, "attention grid of more than " + std::to_string(attention_max_grid()) + " workgroups");
    // the split merge runs d/4 work-items per (KV head, row)
    if ((int64_t)p.nkv * p.rows * (p.d / 4) > OC_MAX_GRID_ITEMS)
        return fail(OC_ERANGE, "split merge grid exceeds 2^32 work-items");
    return OC_OK;
}

template <int D>
static KParams make_params(const AttnPlan &pl, const AttnArgs &a) {
    KParams p{};
    p.q = a.q;
    p.pool_k = a.pool_k;
    p.pool_v = a.pool_v;
    p.pages = a.pages;
    p.k_new = a.k_new;
    p.v_new = a.v_new;
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
    return p;
}

template <int D>
static hipError_t launch_d(const AttnPlan *pl, const AttnArgs *a, int n, hipStream_t s) {
    // requests with the longest workgroups first: the dispatcher then fills
    // the tail of the launch with short ones
    int order[MAX_ATTN_BATCH];
    for (int i = 0; i < n; ++i) order[i] = i;
    std::stable_sort(order, order + n, [&](int x, int y) { return pl[x].blocks_per_split > pl[y].blocks_per_split; });
    KBatch batch{};
    batch.n = n;
    int64_t grid = 0;
    for (int k = 0; k < n; ++k) {
        const int i = order[k];
        batch.req[k] = make_params<D>(pl[i], a[i]);
        batch.first_wg[k] = (int32_t)grid;
        grid += 8 * ((batch.req[k].n_groups + 7) / 8) * (int64_t)pl[i].m_tiles;
    }
    if (grid > attention_max_grid()) return hipErrorInvalidConfiguration;
    // the kernel's dynamic LDS above the default limit, set once per device
    // (any thread may make the first launch on a device)
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    static std::once_flag lds_once[kMaxDevices];
    static hipError_t lds_status[kMaxDevices];
    std::call_once(lds_once[dev], [dev] {
        lds_status[dev] = hipFuncSetAttribute(reinterpret_cast<const void *>(&attn_fwd_kernel<D>),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)attn_lds_bytes<D>());
    });
    if (lds_status[dev] != hipSuccess) return lds_status[dev];
    if (grid > 0) hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3((unsigned)grid), dim3(THREADS), attn_lds_bytes<D>(), s, batch);
    // the split merge of every request that has splits, in one launch
    constexpr int RPB = 256 / (D / 4);
    int64_t cblocks[MAX_ATTN_BATCH], ctotal = 0;
    for (int k = 0; k < n; ++k) {
        cblocks[k] = batch.req[k].n_split > 1 ? ((int64_t)batch.req[k].nkv * batch.req[k].rows + RPB - 1) / RPB : 0;
        batch.first_cb[k] = (int32_t)std::min<int64_t>(ctotal, INT32_MAX);
        ctotal += cblocks[k];
    }
    const int with_splits = (int)std::count_if(cblocks, cblocks + n, [](int64_t c) { return c > 0; });
    if (with_splits > 1 && ctotal * 256 <= OC_MAX_GRID_ITEMS) {
        hipLaunchKernelGGL(attn_combine_batch_kernel<D>, dim3((unsigned)ctotal), dim3(256), 0, s, batch);
    } else {
        // one request with splits, or too many rows for one dispatch: one
        // merge per request (each fits, as the shape checks require)
        for (int k = 0; k < n; ++k)
            if (cblocks[k])
                hipLaunchKernelGGL(attn_combine_kernel<D>, dim3((unsigned)cblocks[k]), dim3(256), 0, s,
                                   batch.req[k]);
    }
    return hipGetLastError();
}

hipError_t launch_attention(const AttnPlan &pl, const AttnArgs &a, hipStream_t s) {
    if (pl.d == 128) return launch_d<128>(&pl, &a, 1, s);
    return launch_d<64>(&pl, &a, 1, s);
}

hipError_t launch_attention_batch(const AttnPlan *pl, const AttnArgs *a, int n, hipStream_t s) {
    if (n < 1 || n > MAX_ATTN_BATCH) return hipErrorInvalidValue;
    if (pl[0].d == 128) return launch_d<128>(pl, a, n, s);
    return launch_d<64>(pl, a, n, s);
}

}  // namespace oc
