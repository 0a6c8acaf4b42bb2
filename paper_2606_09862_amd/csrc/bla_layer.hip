// A whole BLA layer (the operator between its projections): the queries, keys and values
// are linear projections of the hidden states (the attention layer of Sec. 2.1, which BLA
// replaces the softmax of), the heads run the operator of Sec. 3.1 (bla_forward), and an
// output projection mixes the heads back into the model width.
//
//   qkv = x W_qkv        x [B*L, D], W_qkv [D, 3D]   (hipBLASLt, bf16 in, float32 accumulation)
//   o = BLA(q, k, v)     q, k, v read in place from qkv, viewed as [B, L, 3, H, d], and o
//                        written in place as [B, L, H, d] (the operator's strided form)
//   y = o W_o            W_o [D, D]                   (hipBLASLt)
//
// The two products are plain dense GEMMs, so they go to the vendor library; the operator
// runs in this library's kernels and reads and writes the GEMMs' row-major tensors
// directly, so no head split or merge pass touches memory.
#include <stdint.h>
#include <string.h>

#include <mutex>

#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include "bla.h"
#include "bla_device.h"
#include "bla_plan.h"

namespace bla {
namespace {

constexpr size_t kLayerAlign = 256;
constexpr size_t kGemmWorkspace = size_t(32) << 20;  // hipBLASLt scratch inside the caller's workspace

size_t lalign(size_t x) { return (x + kLayerAlign - 1) / kLayerAlign * kLayerAlign; }

// One hipBLASLt handle per device, created on first use and kept for the process.  Creation
// is serialised, so threads that reach a device's first call together share one handle.
hipblasLtHandle_t gemm_handle()
{
    static std::mutex mu;
    static hipblasLtHandle_t handles[64] = {nullptr};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
    std::lock_guard<std::mutex> lk(mu);
    if (!handles[dev] && hipblasLtCreate(&handles[dev]) != HIPBLAS_STATUS_SUCCESS) handles[dev] = nullptr;
    return handles[dev];
}

// Row-major Y [m, n] = X [m, k] W [k, n] in bf16 with float32 accumulation.  In hipBLASLt's
// column-major terms this is Y^T = W^T X^T with no transposes: A = W (n x k, ld n),
// B = X (k x m, ld k), C = D = Y (n x m, ld n).
bool gemm_rowmajor(const bf16* X, const bf16* W, bf16* Y, long long m, long long n, long long k, void* ws,
                   size_t ws_bytes, hipStream_t s)
{
    hipblasLtHandle_t h = gemm_handle();
    if (!h) return false;
    hipblasLtMatmulDesc_t desc = nullptr;
    hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
    hipblasLtMatmulPreference_t pref = nullptr;
    bool ok = false;
    do {
        if (hipblasLtMatmulDescCreate(&desc, HIPBLAS_COMPUTE_32F, HIP_R_32F) != HIPBLAS_STATUS_SUCCESS) break;
        const int32_t opn = HIPBLAS_OP_N;
        if (hipblasLtMatmulDescSetAttribute(desc, HIPBLASLT_MATMUL_DESC_TRANSA, &opn, sizeof(opn)) != HIPBLAS_STATUS_SUCCESS ||
            hipblasLtMatmulDescSetAttribute(desc, HIPBLASLT_MATMUL_DESC_TRANSB, &opn, sizeof(opn)) != HIPBLAS_STATUS_SUCCESS)
            break;
        if (hipblasLtMatrixLayoutCreate(&la, HIP_R_16BF, n, k, n) != HIPBLAS_STATUS_SUCCESS) break;
        if (hipblasLtMatrixLayoutCreate(&lb, HIP_R_16BF, k, m, k) != HIPBLAS_STATUS_SUCCESS) break;
        if (hipblasLtMatrixLayoutCreate(&lc, HIP_R_16BF, n, m, n) != HIPBLAS_STATUS_SUCCESS) break;
        if (hipblasLtMatmulPreferenceCreate(&pref) != HIPBLAS_STATUS_SUCCESS) break;
        const uint64_t wsz = ws_bytes;
        if (hipblasLtMatmulPreferenceSetAttribute(pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &wsz,
                                                  sizeof(wsz)) != HIPBLAS_STATUS_SUCCESS)
            break;
        hipblasLtMatmulHeuristicResult_t res[1];
        int cnt = 0;
        if (hipblasLtMatmulAlgoGetHeuristic(h, desc, la, lb, lc, lc, pref, 1, res, &cnt) != HIPBLAS_STATUS_SUCCESS ||
            cnt < 1)
            break;
        const float alpha = 1.f, beta = 0.f;
        ok = hipblasLtMatmul(h, desc, &alpha, W, la, X, lb, &beta, Y, lc, Y, lc, &res[0].algo, ws, ws_bytes, s) ==
             HIPBLAS_STATUS_SUCCESS;
    } while (false);
    if (pref) hipblasLtMatmulPreferenceDestroy(pref);
    if (lc) hipblasLtMatrixLayoutDestroy(lc);
    if (lb) hipblasLtMatrixLayoutDestroy(lb);
    if (la) hipblasLtMatrixLayoutDestroy(la);
    if (desc) hipblasLtMatmulDescDestroy(desc);
    return ok;
}

struct LayerPlan {
    size_t off_qkv, off_o, off_fwd, off_gemm, total;
    size_t fwd_bytes;
};

bla_status layer_plan(const bla_params* p, LayerPlan* lp)
{
    if (!p) return BLA_ERR_INVALID_ARG;
    if (p->io_dtype != BLA_BF16) return BLA_ERR_UNSUPPORTED;
    const bla_status st = bla_supported(p);
    if (st != BLA_OK) return st;
    const size_t tok = (size_t)p->B * p->L, D = (size_t)p->H * p->d_k;
    lp->fwd_bytes = bla_workspace_size(p);
    size_t off = 0;
    lp->off_qkv = off; off = lalign(off + tok * 3 * D * 2);  // [B, L, 3, H, d]
    lp->off_o = off;   off = lalign(off + tok * D * 2);      // [B, L, H, d]
    lp->off_fwd = off; off = lalign(off + lp->fwd_bytes);
    lp->off_gemm = off; off = lalign(off + kGemmWorkspace);
    lp->total = off;
    return BLA_OK;
}

}  // namespace
}  // namespace bla

using namespace bla;

extern "C" {

size_t bla_layer_workspace_size(const bla_params* p)
{
    LayerPlan lp;
    if (layer_plan(p, &lp) != BLA_OK) return 0;
    return lp.total;
}

static bla_status layer_impl(const bla_params* p, const double* T, const void* x, const void* w_qkv,
                             const void* w_o, const float* state_k_in, const float* state_v_in, void* y,
                             float* state_k_out, float* state_v_out, void* workspace, size_t workspace_bytes,
                             void* stream, void* const* events)
{
    LayerPlan lp;
    bla_status st = layer_plan(p, &lp);
    if (st != BLA_OK) return st;
    if (p->d_k != p->d_v) return BLA_ERR_UNSUPPORTED;
    const long long tok = (long long)p->B * p->L, D = (long long)p->H * p->d_k;
    if (tok == 0 || p->H == 0) return bla_forward(p, T, nullptr, nullptr, nullptr, state_k_in, state_v_in, nullptr,
                                                  state_k_out, state_v_out, workspace, workspace_bytes, stream);
    auto a16 = [](const void* ptr) { return ((uintptr_t)ptr & 15u) == 0; };
    if (!x || !w_qkv || !w_o || !y || !a16(x) || !a16(w_qkv) || !a16(w_o) || !a16(y)) return BLA_ERR_INVALID_ARG;
    if (!workspace || workspace_bytes < lp.total || !a16(workspace)) return BLA_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    auto mark = [&](int i) -> bool {
        return !events || !events[i] || hipEventRecord((hipEvent_t)events[i], s) == hipSuccess;
    };
    bf16* qkv = (bf16*)(ws + lp.off_qkv);
    bf16* o = (bf16*)(ws + lp.off_o);
    void* gws = ws + lp.off_gemm;
    const long long L = p->L, d = p->d_k;
    const long long in_strides[3] = {L * 3 * D, d, 3 * D};  // [B, L, 3, H, d]
    const long long out_strides[3] = {L * D, d, D};         // [B, L, H, d]

    if (!mark(0)) return BLA_ERR_HIP;
    if (!gemm_rowmajor((const bf16*)x, (const bf16*)w_qkv, qkv, tok, 3 * D, D, gws, kGemmWorkspace, s))
        return BLA_ERR_HIP;
    if (!mark(1)) return BLA_ERR_HIP;
    st = forward_strided(p, T, qkv, qkv + D, qkv + 2 * D, in_strides, state_k_in, state_v_in, o, out_strides,
                         state_k_out, state_v_out, ws + lp.off_fwd, lp.fwd_bytes, stream, nullptr);
    if (st != BLA_OK) return st;
    if (!mark(2)) return BLA_ERR_HIP;
    if (!gemm_rowmajor(o, (const bf16*)w_o, (bf16*)y, tok, D, D, gws, kGemmWorkspace, s)) return BLA_ERR_HIP;
    if (!mark(3)) return BLA_ERR_HIP;
    return BLA_OK;
}

bla_status bla_layer_forward(const bla_params* p, const double* T, const void* x, const void* w_qkv, const void* w_o,
                             const float* state_k_in, const float* state_v_in, void* y, float* state_k_out,
                             float* state_v_out, void* workspace, size_t workspace_bytes, void* stream)
{
    return layer_impl(p, T, x, w_qkv, w_o, state_k_in, state_v_in, y, state_k_out, state_v_out, workspace,
                      workspace_bytes, stream, nullptr);
}

bla_status bla_layer_forward_timed(const bla_params* p, const double* T, const void* x, const void* w_qkv,
                                   const void* w_o, const float* state_k_in, const float* state_v_in, void* y,
                                   float* state_k_out, float* state_v_out, void* workspace, size_t workspace_bytes,
                                   void* stream, void* const* events)
{
    return layer_impl(p, T, x, w_qkv, w_o, state_k_in, state_v_in, y, state_k_out, state_v_out, workspace,
                      workspace_bytes, stream, events);
}

}  // extern "C"
