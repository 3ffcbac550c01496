// C ABI of libqe: argument validation, workspace checks and launch sequencing.
// Every argument error is detected on the host before anything is enqueued.
#include <cmath>
#include <mutex>

#include "qe_internal.h"

using namespace qe;

namespace {

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

bool bad_bits(int bits) { return bits < 1 || bits > 8; }
bool bad_block(int block) { return !(block == 0 || block == 16 || block == 32 || block == 64 || block == 128); }

// Shapes must be positive and small enough that q*p and p*p index in int64.
bool bad_dims(int64_t q, int64_t p)
{
    return q <= 0 || p <= 0 || q > (int64_t(1) << 31) || p > (int64_t(1) << 31);
}

__global__ void status_clear_kernel(int* status)
{
    if (threadIdx.x == 0) *status = 0;
}

// A fill kernel rather than a memset node, so that calls stay capturable.
qe_status clear_status(void* ws, hipStream_t s)
{
    hipLaunchKernelGGL(status_clear_kernel, dim3(1), dim3(64), 0, s, static_cast<int*>(ws));
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status cd_arg_error(const float* W, const float* Sigma, const float* scale, const float* zero,
                       const float* W_hat, const uint8_t* codes, const float* R, int64_t q,
                       int64_t p, int bits, int sweeps, int block, uint32_t flags)
{
    if (!W || !Sigma || !scale || !zero || !W_hat || !codes || !R) return QE_ERR_ARG;
    if (bad_dims(q, p) || bad_bits(bits) || bad_block(block) || sweeps < 0) return QE_ERR_ARG;
    if (flags & ~(QE_INIT_FROM_W | QE_R_VALID | QE_CODES_VALID | QE_RELAX_MASK | QE_CD_FP32 |
                  QE_CD_DENSE | QE_DEBUG_CHECKS | QE_OBJ_IN))
        return QE_ERR_ARG;
    return QE_OK;
}

// QE_OBJ_IN reads obj[0]: it needs obj, and means nothing after QE_INIT_FROM_W
// (the objective of What = W is 0).
bool bad_obj_in(uint32_t flags, const double* obj)
{
    return (flags & QE_OBJ_IN) && (!obj || (flags & QE_INIT_FROM_W));
}

// ---- scratch of qe_cd_sweep_noalloc
// One copy per GPU, held until the process ends.  In host code `scratch` only
// names the symbol; its device address comes from hipGetSymbolAddress, taken
// once per device with that device current.
static __device__ __align__(256) unsigned char scratch[QE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

qe_status scratch_on_stream(hipStream_t s, void** out)
{
    int dev = 0;
    if (s) {
        if (hipStreamGetDevice(s, &dev) != hipSuccess) return QE_ERR_HIP;
    } else if (hipGetDevice(&dev) != hipSuccess) {
        return QE_ERR_HIP;
    }
    if (dev < 0 || dev >= kMaxDevices) return QE_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        int cur = 0;
        if (hipGetDevice(&cur) != hipSuccess) return QE_ERR_HIP;
        if (cur != dev && hipSetDevice(dev) != hipSuccess) return QE_ERR_HIP;
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev && hipSetDevice(cur) != hipSuccess) return QE_ERR_HIP;
        if (e != hipSuccess || !ptr) return QE_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return QE_OK;
}

__global__ void status_copy_kernel(const int* from, int* to)
{
    if (threadIdx.x == 0) *to = *from;
}

}  // namespace

extern "C" {

const char* qe_status_string(qe_status s)
{
    switch (s) {
        case QE_OK: return "ok";
        case QE_ERR_ARG: return "invalid argument";
        case QE_ERR_DIAG: return "Sigma has a non-positive or non-finite diagonal entry";
        case QE_ERR_SCALE: return "grid scale non-positive or non-finite";
        case QE_ERR_WORKSPACE: return "workspace missing or too small";
        case QE_ERR_HIP: return "HIP runtime error";
        case QE_ERR_UNSUPPORTED: return "unsupported request";
        case QE_ERR_TOO_LARGE: return "request needs more than the fixed scratch of qe_cd_sweep_noalloc";
        case QE_ERR_NONFINITE: return "an input holds a NaN or an infinity";
        default: return "unknown status";
    }
}

int qe_version(void) { return 1; }

qe_status qe_sync_status(void* ws, void* stream)
{
    if (!ws) return QE_ERR_ARG;
    hipStream_t s = as_stream(stream);
    int code = 0;
    if (hipMemcpyAsync(&code, ws, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess)
        return QE_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return QE_ERR_HIP;
    if (code != 0 && clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    if (code != 0 && hipStreamSynchronize(s) != hipSuccess) return QE_ERR_HIP;
    return code;
}

// ------------------------------------------------------------------ Gram
size_t qe_gram_workspace_size(int64_t p, int64_t n)
{
    if (p <= 0 || n <= 0) return kStatusBytes;
    return gram_ws_bytes(p, n);
}

qe_status qe_gram(const float* X, int64_t p, int64_t n, int layout, float* Sigma, int accumulate,
                  float damp, void* ws, size_t ws_bytes, void* stream)
{
    if (!X || !Sigma || p <= 0 || n <= 0 || p > (int64_t(1) << 31)) return QE_ERR_ARG;
    const int base_layout = layout & ~(QE_GRAM_FP32 | QE_GRAM_BF16X3);
    if (base_layout != QE_LAYOUT_PN && base_layout != QE_LAYOUT_NP) return QE_ERR_ARG;
    if ((layout & QE_GRAM_FP32) && (layout & QE_GRAM_BF16X3)) return QE_ERR_ARG;
    if (!(damp >= 0.f) || !std::isfinite(damp)) return QE_ERR_ARG;
    if (!ws || ws_bytes < gram_ws_bytes(p, n)) return QE_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    return launch_gram(X, p, n, layout, Sigma, accumulate ? 1 : 0, damp, ws, s);
}

// ------------------------------------------------------------------ grid
qe_status qe_grid_minmax(const float* W, const float* H, int64_t q, int64_t p, int bits,
                         float* scale, float* zero, void* stream)
{
    if (!W || !scale || !zero || bad_dims(q, p) || bad_bits(bits)) return QE_ERR_ARG;
    return launch_grid_minmax(W, H, q, p, bits, scale, zero, as_stream(stream));
}

// ------------------------------------------------------------------ CD
size_t qe_cd_workspace_size(int64_t q, int64_t p, int block)
{
    if (bad_dims(q, p) || bad_block(block)) return 0;
    return cd_ws_bytes(q, p, block);
}

qe_status qe_cd_sweep(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                      const float* scale, const float* zero, float* W_hat, uint8_t* codes,
                      float* R, int sweeps, int block, uint32_t flags, double* obj, void* ws,
                      size_t ws_bytes, void* stream)
{
    const qe_status bad = cd_arg_error(W, Sigma, scale, zero, W_hat, codes, R, q, p, bits, sweeps,
                                       block, flags);
    if (bad != QE_OK) return bad;
    if (bad_obj_in(flags, obj)) return QE_ERR_ARG;
    if (!ws || ws_bytes < cd_ws_bytes(q, p, block)) return QE_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    return launch_cd(W, Sigma, q, p, bits, scale, zero, W_hat, codes, R, nullptr, sweeps, block,
                     flags, obj, 1, (flags & QE_OBJ_IN) ? obj : nullptr, ws, s);
}

qe_status qe_cd_sweep_noalloc(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                              const float* scale, const float* zero, float* W_hat,
                              uint8_t* codes, float* R, int sweeps, int block, uint32_t flags,
                              double* obj, int* status, void* stream)
{
    const qe_status bad = cd_arg_error(W, Sigma, scale, zero, W_hat, codes, R, q, p, bits, sweeps,
                                       block, flags);
    if (bad != QE_OK) return bad;
    if (bad_obj_in(flags, obj)) return QE_ERR_ARG;
    if (cd_ws_bytes(q, p, block) > QE_NOALLOC_SCRATCH_BYTES) return QE_ERR_TOO_LARGE;
    hipStream_t s = as_stream(stream);
    void* ws = nullptr;
    qe_status st = scratch_on_stream(s, &ws);
    if (st != QE_OK) return st;
    // the previous call's status word is still there
    if (clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    st = launch_cd(W, Sigma, q, p, bits, scale, zero, W_hat, codes, R, nullptr, sweeps, block,
                   flags, obj, 1, (flags & QE_OBJ_IN) ? obj : nullptr, ws, s);
    if (st != QE_OK) return st;
    if (status) {
        hipLaunchKernelGGL(status_copy_kernel, dim3(1), dim3(64), 0, s,
                           static_cast<const int*>(ws), status);
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    return QE_OK;
}

// ------------------------------------------------------------------ outlier-aware CD
size_t qe_outlier_workspace_size(int64_t q, int64_t p, int block, int64_t s)
{
    if (bad_dims(q, p) || bad_block(block) || s < 0 || s > q * p) return 0;
    return outlier_ws_bytes(q, p, block, s);
}

qe_status qe_cd_outlier_sweep(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                              const float* scale, const float* zero, float* W_hat,
                              uint8_t* codes, float* H, float* E, int64_t s, float lambda_max,
                              int64_t* support, int64_t* support_nnz, int sweeps, int block,
                              uint32_t flags, double* obj, void* ws, size_t ws_bytes,
                              void* stream)
{
    if (!W || !Sigma || !scale || !zero || !W_hat || !codes || !H || !E || !support_nnz)
        return QE_ERR_ARG;
    if (bad_dims(q, p) || bad_bits(bits) || bad_block(block) || sweeps < 0) return QE_ERR_ARG;
    if (s < 0 || s > q * p || (s > 0 && !support)) return QE_ERR_ARG;
    if (!(lambda_max > 0.f) || !std::isfinite(lambda_max)) return QE_ERR_ARG;
    if (flags & ~(QE_INIT_FROM_W | QE_R_VALID | QE_CODES_VALID | QE_OUTLIER_COLUMNS | QE_CD_FP32 |
                  QE_CD_DENSE | QE_DEBUG_CHECKS))
        return QE_ERR_ARG;
    if (!ws || ws_bytes < outlier_ws_bytes(q, p, block, s)) return QE_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (clear_status(ws, st) != QE_OK) return QE_ERR_HIP;
    return launch_outlier(W, Sigma, q, p, bits, scale, zero, W_hat, codes, H, E, s, lambda_max,
                          support, support_nnz, sweeps, block, flags, obj, ws, st);
}

// ------------------------------------------------------------------ P_s
size_t qe_topk_workspace_size(int64_t count, int64_t s)
{
    if (count < 0 || s < 0) return 0;
    return topk_ws_bytes(count, s);
}

qe_status qe_topk_abs(const float* V, int64_t count, int64_t s, float* out, int64_t* support,
                      int64_t* nnz, void* ws, size_t ws_bytes, void* stream)
{
    if (!V || !out || !nnz || count <= 0 || s < 0 || s > count || (s > 0 && !support))
        return QE_ERR_ARG;
    if (!ws || ws_bytes < topk_ws_bytes(count, s)) return QE_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (clear_status(ws, st) != QE_OK) return QE_ERR_HIP;
    return launch_topk(V, count, s, out, support, nnz, ws, st);
}

size_t qe_topk_columns_workspace_size(int64_t q, int64_t p)
{
    if (bad_dims(q, p)) return 0;
    return topk_columns_ws_bytes(q, p);
}

qe_status qe_topk_columns(const float* V, int64_t q, int64_t p, int64_t c, float* out,
                          int64_t* columns, int64_t* support, int64_t* nnz, void* ws,
                          size_t ws_bytes, void* stream)
{
    if (!V || !out || !nnz || bad_dims(q, p) || c < 0 || c > p || (c > 0 && !support))
        return QE_ERR_ARG;
    if (!ws || ws_bytes < topk_columns_ws_bytes(q, p)) return QE_ERR_WORKSPACE;
    hipStream_t st = as_stream(stream);
    if (clear_status(ws, st) != QE_OK) return QE_ERR_HIP;
    return launch_topk_columns(V, q, p, c, out, columns, support, nnz, ws, st);
}

// ------------------------------------------------------------------ export
int64_t qe_packed_row_bytes(int64_t p, int bits)
{
    if (p < 0 || bad_bits(bits)) return 0;
    return packed_row_bytes(p, bits);
}

qe_status qe_pack_codes(const uint8_t* codes, int64_t q, int64_t p, int bits, uint8_t* packed,
                        void* stream)
{
    if (!codes || !packed || bad_dims(q, p) || bad_bits(bits)) return QE_ERR_ARG;
    return launch_pack_codes(codes, q, p, bits, packed, as_stream(stream));
}

qe_status qe_outliers_csr(const float* H, int64_t q, int64_t p, const int64_t* support,
                          const int64_t* nnz, int64_t cap, int64_t* rowptr, int32_t* cols,
                          float* vals, void* stream)
{
    if (!H || !nnz || !rowptr || bad_dims(q, p) || cap < 0) return QE_ERR_ARG;
    if (cap > 0 && (!support || !cols || !vals)) return QE_ERR_ARG;
    return launch_outliers_csr(H, q, p, support, nnz, cap, rowptr, cols, vals, as_stream(stream));
}

// ------------------------------------------------------------------ objective
size_t qe_objective_workspace_size(int64_t q, int64_t p)
{
    if (bad_dims(q, p)) return 0;
    return objective_ws_bytes(q, p);
}

qe_status qe_objective(const float* W, const float* W_hat, const float* H, const float* Sigma,
                       int64_t q, int64_t p, double* out, void* ws, size_t ws_bytes, void* stream)
{
    if (!W || !W_hat || !Sigma || !out || bad_dims(q, p)) return QE_ERR_ARG;
    if (!ws || ws_bytes < objective_ws_bytes(q, p)) return QE_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    return launch_objective(W, W_hat, H, Sigma, q, p, out, ws, s);
}

// ------------------------------------------------------------------ lambda_max
size_t qe_lambda_workspace_size(int64_t p)
{
    if (p <= 0) return 0;
    return lambda_ws_bytes(p);
}

qe_status qe_lambda_max(const float* Sigma, int64_t p, int max_iters, float tol,
                        float* lambda_out, void* ws, size_t ws_bytes, void* stream)
{
    if (!Sigma || !lambda_out || p <= 0 || max_iters < 1 || !(tol >= 0.f)) return QE_ERR_ARG;
    if (!ws || ws_bytes < lambda_ws_bytes(p)) return QE_ERR_WORKSPACE;
    hipStream_t s = as_stream(stream);
    if (clear_status(ws, s) != QE_OK) return QE_ERR_HIP;
    return launch_lambda(Sigma, p, max_iters, tol, lambda_out, ws, s);
}

}  // extern "C"
