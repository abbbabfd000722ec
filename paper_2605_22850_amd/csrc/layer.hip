// Rest-of-layer compute window: what a transformer layer runs on the miss
// tokens besides the attention (the C_l of eq. (3); every layer has the same
// projections and feed-forward network, Section 3.6).  Four bf16 GEMMs with
// fp32 accumulation (O, gate|up, down, next layer's QKV) go to rocBLAS; the
// SiLU gating between them is a kernel of its own.
#include <rocblas/rocblas.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <utility>

#include "common.hpp"

namespace oc {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));

// act[t][c] = silu(gu[t][c]) * gu[t][F + c], 8 columns per thread, fp32 math,
// rounded to bf16 (nearest even).
__global__ __launch_bounds__(256) void silu_mul_kernel(const uint16_t *gu, uint16_t *act, int64_t F8, int64_t n) {
    const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (e >= n) return;
    const int64_t t = e / F8, c = e - t * F8;
    const uint16_t *grow = gu + t * 16 * F8 + c * 8;
    const u32x4 gb = *reinterpret_cast<const u32x4 *>(grow);
    const u32x4 ub = *reinterpret_cast<const u32x4 *>(grow + 8 * F8);
    f32x8 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float g0 = __uint_as_float(gb[i] << 16), g1 = __uint_as_float(gb[i] & 0xFFFF0000u);
        const float u0 = __uint_as_float(ub[i] << 16), u1 = __uint_as_float(ub[i] & 0xFFFF0000u);
        r[2 * i] = g0 / (1.f + __expf(-g0)) * u0;
        r[2 * i + 1] = g1 / (1.f + __expf(-g1)) * u1;
    }
    *reinterpret_cast<u32x4 *>(act + t * 8 * F8 + c * 8) = __builtin_bit_cast(u32x4, __builtin_convertvector(r, bf16x8));
}

// One rocBLAS handle per (device, stream): a handle's workspace must not be
// shared by GEMMs running on different streams.  Handles live until the
// process ends, or until forget_blas_stream() for streams the library owns.
static std::mutex g_blas_mu;
static std::map<std::pair<int, hipStream_t>, rocblas_handle> g_blas;

static int blas_for(hipStream_t s, rocblas_handle *out) {
    int dev = 0;
    OC_HIP(hipGetDevice(&dev));
    auto key = std::make_pair(dev, s);
    auto it = g_blas.find(key);
    if (it == g_blas.end()) {
        rocblas_handle h = nullptr;
        if (rocblas_create_handle(&h) != rocblas_status_success) return fail(OC_EHIP, "rocblas_create_handle failed");
        it = g_blas.emplace(key, h).first;
    }
    if (rocblas_set_stream(it->second, s) != rocblas_status_success) return fail(OC_EHIP, "rocblas_set_stream failed");
    *out = it->second;
    return OC_OK;
}

void forget_blas_stream(hipStream_t s) {
    std::lock_guard<std::mutex> g(g_blas_mu);
    for (auto it = g_blas.begin(); it != g_blas.end();) {
        if (it->first.second == s) {
            rocblas_destroy_handle(it->second);
            it = g_blas.erase(it);
        } else {
            ++it;
        }
    }
}

// Y[M][N] = X[M][K] . W[K][N], all row-major bf16: column-major rocBLAS sees
// Y^T = W^T . X^T with no transposes.
static int gemm(rocblas_handle h, const uint16_t *X, const uint16_t *W, uint16_t *Y, int64_t M, int64_t K, int64_t N) {
    const float alpha = 1.f, beta = 0.f;
    rocblas_status st = rocblas_gemm_ex(h, rocblas_operation_none, rocblas_operation_none, (rocblas_int)N,
                                        (rocblas_int)M, (rocblas_int)K, &alpha, W, rocblas_datatype_bf16_r,
                                        (rocblas_int)N, X, rocblas_datatype_bf16_r, (rocblas_int)K, &beta, Y,
                                        rocblas_datatype_bf16_r, (rocblas_int)N, Y, rocblas_datatype_bf16_r,
                                        (rocblas_int)N, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
    if (st != rocblas_status_success)
        return fail(OC_EHIP, std::string("rocblas_gemm_ex: ") + rocblas_status_to_string(st));
    return OC_OK;
}

// Rows are independent, so long inputs go through the chain in row blocks
// that keep every matrix handed to the GEMM library under 1 GiB.
int launch_rest_of_layer(const LayerArgs &a, hipStream_t s) {
    if (a.T == 0) return OC_OK;
    std::lock_guard<std::mutex> g(g_blas_mu);
    rocblas_handle h = nullptr;
    int rc = blas_for(s, &h);
    if (rc) return rc;
    const int64_t widest = std::max(std::max(2 * a.F, a.H), a.NQKV);
    const int64_t rb = std::max<int64_t>(1, (INT64_C(1) << 29) / widest);
    for (int64_t r0 = 0; r0 < a.T; r0 += rb) {
        const int64_t m = std::min(rb, a.T - r0);
        const uint16_t *x = a.attn_out + r0 * a.H;
        uint16_t *o = a.o + r0 * a.H, *gu = a.gu + r0 * 2 * a.F, *act = a.act + r0 * a.F;
        uint16_t *hh = a.h + r0 * a.H, *qkv = a.qkv + r0 * a.NQKV;
        if ((rc = gemm(h, x, a.w_o, o, m, a.H, a.H))) return rc;
        if ((rc = gemm(h, o, a.w_gu, gu, m, a.H, 2 * a.F))) return rc;
        const int64_t n = m * (a.F / 8);
        hipLaunchKernelGGL(silu_mul_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, gu, act,
                           (int64_t)(a.F / 8), n);
        OC_HIP(hipGetLastError());
        if ((rc = gemm(h, act, a.w_down, hh, m, a.F, a.H))) return rc;
        if ((rc = gemm(h, hh, a.w_qkv, qkv, m, a.H, a.NQKV))) return rc;
    }
    return OC_OK;
}

LayerArgs layer_args(const oc_layout &l, const oc_layer_weights &w, int32_t layer, const void *attn_out,
                     int64_t tokens, const oc_layer_buffers &b) {
    LayerArgs a{};
    a.T = tokens;
    a.H = (int64_t)l.num_q_heads * l.head_dim;
    a.F = w.ffn_dim;
    a.NQKV = (int64_t)(l.num_q_heads + 2 * l.num_kv_heads) * l.head_dim;
    a.attn_out = static_cast<const uint16_t *>(attn_out);
    a.w_o = static_cast<const uint16_t *>(w.w_o) + layer * a.H * a.H;
    a.w_gu = static_cast<const uint16_t *>(w.w_gate_up) + layer * a.H * 2 * a.F;
    a.w_down = static_cast<const uint16_t *>(w.w_down) + layer * a.F * a.H;
    a.w_qkv = static_cast<const uint16_t *>(w.w_qkv) + layer * a.H * a.NQKV;
    a.o = static_cast<uint16_t *>(b.o);
    a.gu = static_cast<uint16_t *>(b.gate_up);
    a.act = static_cast<uint16_t *>(b.act);
    a.h = static_cast<uint16_t *>(b.h);
    a.qkv = static_cast<uint16_t *>(b.qkv);
    return a;
}

int check_layer_weights(const oc_layout &l, const oc_layer_weights *w) {
    if (!w) return fail(OC_EINVAL, "layer weights are NULL");
    if (w->ffn_dim < 8 || w->ffn_dim % 8) return fail(OC_ESHAPE, "ffn_dim must be a positive multiple of 8");
    if (!w->w_o || !w->w_gate_up || !w->w_down || !w->w_qkv) return fail(OC_EINVAL, "NULL layer weight");
    if (!aligned(w->w_o, 16) || !aligned(w->w_gate_up, 16) || !aligned(w->w_down, 16) || !aligned(w->w_qkv, 16))
        return fail(OC_EALIGN, "layer weights must be 16-byte aligned");
    const int64_t H = (int64_t)l.num_q_heads * l.head_dim;
    if (H * 2 * w->ffn_dim > INT32_MAX || (int64_t)(l.num_q_heads + 2 * l.num_kv_heads) * l.head_dim > INT32_MAX)
        return fail(OC_ERANGE, "layer too wide");
    return OC_OK;
}

int check_layer_buffers(const oc_layer_buffers *b) {
    if (!b) return fail(OC_EINVAL, "layer buffers are NULL");
    if (!b->o || !b->gate_up || !b->act || !b->h || !b->qkv) return fail(OC_EINVAL, "NULL layer buffer");
    if (!aligned(b->o, 16) || !aligned(b->gate_up, 16) || !aligned(b->act, 16) || !aligned(b->h, 16) ||
        !aligned(b->qkv, 16))
        return fail(OC_EALIGN, "layer buffers must be 16-byte aligned");
    return OC_OK;
}

size_t layer_buffer_bytes(const oc_layout &l, int32_t ffn_dim, int64_t tokens, size_t off[5]) {
    const int64_t H = (int64_t)l.num_q_heads * l.head_dim;
    const int64_t NQKV = (int64_t)(l.num_q_heads + 2 * l.num_kv_heads) * l.head_dim;
    const int64_t cols[5] = {H, 2LL * ffn_dim, ffn_dim, H, NQKV};
    size_t total = 0;
    for (int i = 0; i < 5; ++i) {
        off[i] = total;
        total += ((size_t)tokens * cols[i] * 2 + 255) / 256 * 256;
    }
    return total;
}

}  // namespace oc
