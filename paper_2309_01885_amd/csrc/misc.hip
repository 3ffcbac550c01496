// Grid, exact objective and lambda_max kernels (gfx950).
#include <algorithm>
#include <cmath>

#include "nt_x3.h"
#include "qe_internal.h"

namespace qe {

// ---------------------------------------------------------------- grid
// Per-row asymmetric min/max grid (Sec. 2.1: uniformly spaced levels per output
// channel; the paper does not print the formula, see qe.h): one workgroup per
// row, min/max reductions (exact in any order), then the scale and zero point
// in fp32.  Entries with H != 0 are excluded (outlier-aware grid, Sec. 4.3).
__global__ __launch_bounds__(256) void grid_minmax_kernel(const float* __restrict__ W,
                                                          const float* __restrict__ H, int64_t p,
                                                          float maxq, float* scale, float* zero)
{
    __shared__ float slo[256], shi[256];
    const int64_t i = blockIdx.x;
    float lo = 0.f, hi = 0.f;
    for (int64_t j = threadIdx.x; j < p; j += blockDim.x) {
        if (H && H[i * p + j] != 0.f) continue;
        const float w = W[i * p + j];
        lo = fminf(lo, w);
        hi = fmaxf(hi, w);
    }
    slo[threadIdx.x] = lo;
    shi[threadIdx.x] = hi;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) {
            slo[threadIdx.x] = fminf(slo[threadIdx.x], slo[threadIdx.x + s]);
            shi[threadIdx.x] = fmaxf(shi[threadIdx.x], shi[threadIdx.x + s]);
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        lo = slo[0];
        hi = shi[0];
        if (lo == 0.f && hi == 0.f) {
            lo = -1.f;
            hi = 1.f;
        }
        const float s = (hi - lo) / maxq;
        scale[i] = s;
        zero[i] = rintf(-lo / s);
    }
}

// ---------------------------------------------------------------- input checks
// Any NaN or infinity among `count` floats sets QE_ERR_NONFINITE.
__global__ __launch_bounds__(256) void nonfinite_scan_kernel(const float* __restrict__ a,
                                                             int64_t count, int vec4, int* status)
{
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    // exponent field all ones: infinity or NaN
    auto bad = [](float x) { return (int)((__float_as_uint(x) & 0x7f800000u) == 0x7f800000u); };
    int found = 0;
    int64_t tail = 0;
    if (vec4) {
        const f32x4* a4 = reinterpret_cast<const f32x4*>(a);
        const int64_t n4 = count / 4;
        for (int64_t e = tid; e < n4; e += G) {
            const f32x4 v = a4[e];
            found |= bad(v[0]) | bad(v[1]) | bad(v[2]) | bad(v[3]);
        }
        tail = n4 * 4;
    }
    for (int64_t e = tail + tid; e < count; e += G) found |= bad(a[e]);
    if (found) set_status(status, QE_ERR_NONFINITE);
}

qe_status launch_nonfinite_scan(const float* a, int64_t count, int* status, hipStream_t s)
{
    if (!a || count <= 0) return QE_OK;
    const int64_t wgs = std::min<int64_t>(2048, std::max<int64_t>(1, cdiv(count / 4, 256)));
    hipLaunchKernelGGL(nonfinite_scan_kernel, dim3((unsigned)wgs), dim3(256), 0, s, a, count,
                       aligned16(a) ? 1 : 0, status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status launch_grid_minmax(const float* W, const float* H, int64_t q, int64_t p, int bits,
                             float* scale, float* zero, hipStream_t s)
{
    if (q == 0) return QE_OK;
    hipLaunchKernelGGL(grid_minmax_kernel, dim3((unsigned)q), dim3(256), 0, s, W, H, p,
                       (float)((1 << bits) - 1), scale, zero);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

// ---------------------------------------------------------------- exact objective
// <A, A Sigma> for A = P1 + P2 - P3 (P2, P3 nullable), fused: each 128 x 128
// tile of A Sigma is formed on matrix cores and immediately dotted with the
// matching tile of A in fp64; per-tile partials are summed in a fixed order.
__global__ __launch_bounds__(256, 2) void quad_form_kernel(const float* p1, const float* p2,
                                                        const float* p3, const float* Sigma,
                                                        int64_t q, int64_t p, double* partial,
                                                        int vec4, const int* status)
{
    if (failed(status)) return;
    __shared__ __attribute__((aligned(16))) float lds[kNTLdsFloats];
    __shared__ double sh[256];
    const int64_t tn_count = cdiv(p, kTile);
    const int64_t row0 = (blockIdx.x / tn_count) * kTile, col0 = (blockIdx.x % tn_count) * kTile;
    f32x16 acc[2][2];
    zero_acc(acc);
    // (D Sigma) tile on the bf16 matrix cores with the exact three-way split
    const X3Comp A{p1, p2, p3, p, q, p};
    const X3Row B{Sigma, p, p, p};
    uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
    if (vec4 && row0 + kTile <= q && col0 + kTile <= p && p % (2 * kX3KC) == 0)
        nt_tile_x3_full(A, row0, B, col0, p, l32, acc);
    else
        nt_tile_x3_edge(A, row0, B, col0, p, l32, acc);
    double d = 0.0;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t r = row0 + acc_row(mi, v), c = col0 + acc_col(ni);
                if (r < q && c < p) {
                    const int64_t e = r * p + c;
                    float a = p2 ? p1[e] + p2[e] : p1[e];
                    if (p3) a = a - p3[e];
                    d += (double)a * (double)acc[mi][ni][v];
                }
            }
    const double s = block_sum_f64(d, sh);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// The same on 256 x 256 tiles of eight waves (nt_tile_x3_wide: operand reads
// pipelined through three LDS stage buffers), for q and p multiples of 256 and
// aligned rows.  Tiles are dealt to the 8 XCDs in contiguous ranges (the
// hardware places workgroup b on XCD b % 8) of a banded order (bands of 4 tile
// rows, column-major inside a band), so that the 32 workgroups an XCD holds
// at a time share 4 row panels of A and 8 of Sigma in its L2.
// A = P1 (+ P2) (- P3) with the present terms fixed at compile time, so that
// the loads in flight hold only the operands that exist.
template <bool P2, bool P3>
struct X3CompT {
    const float *p1, *p2, *p3;
    int64_t ld;
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t off = (row0 + (t >> 1)) * ld + k0 + 8 * (t & 1);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4 v = *reinterpret_cast<const f32x4*>(p1 + off + 4 * h);
            if constexpr (P2) v = v + *reinterpret_cast<const f32x4*>(p2 + off + 4 * h);
            if constexpr (P3) v = v - *reinterpret_cast<const f32x4*>(p3 + off + 4 * h);
            st.v[h] = v;
        }
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const { x3_store_row8(op, st); }
};

template <bool P2, bool P3>
__global__ __launch_bounds__(512, 1) void quad_form_wide_kernel(const float* p1, const float* p2,
                                                             const float* p3,
                                                             const float* Sigma, int64_t q,
                                                             int64_t p, double* partial,
                                                             const int* status)
{
    if (failed(status)) return;
    __shared__ __attribute__((aligned(16))) uint32_t lds[kX3wLdsDw];
    __shared__ double sh[512];
    const int64_t tm_count = q / 256, tn_count = p / 256, tiles = tm_count * tn_count;
    const int64_t per = cdiv(tiles, 8);
    const int64_t item = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= tiles) return;                    // uniform: the whole workgroup leaves
    const int64_t b0 = (item / (4 * tn_count)) * 4;
    const int64_t bh = min((int64_t)4, tm_count - b0);
    const int64_t u = item - b0 * tn_count;
    const int64_t row0 = (b0 + u % bh) * 256, col0 = (u / bh) * 256;
    f32x16 acc[2][4];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mi][ni][v] = 0.f;
    const X3CompT<P2, P3> A{p1, p2, p3, p};
    const X3Row B{Sigma, p, p, p};
    nt_tile_x3_wide(A, row0, B, col0, p, lds, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    double d = 0.0;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t r = row0 + wm * 64 + 32 * mi + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                const int64_t c = col0 + wn * 128 + 32 * ni + (lane & 31);
                const int64_t e = r * p + c;
                float a = p1[e];
                if constexpr (P2) a = a + p2[e];
                if constexpr (P3) a = a - p3[e];
                d += (double)a * (double)acc[mi][ni][v];
            }
    sh[threadIdx.x] = d;
    __syncthreads();
    for (int st = 256; st > 0; st >>= 1) {
        if ((int)threadIdx.x < st) sh[threadIdx.x] += sh[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[item] = sh[0];
}

__global__ __launch_bounds__(256) void sum_tiles_kernel(const double* partial, int64_t n,
                                                        double* out, const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double acc = 0.0;
    for (int64_t e = threadIdx.x; e < n; e += blockDim.x) acc += partial[e];
    const double s = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) *out = s;
}

size_t objective_ws_bytes(int64_t q, int64_t p)
{
    const int64_t tiles = cdiv(q, kTile) * cdiv(p, kTile);
    return kStatusBytes + 2 * align256(sizeof(double) * tiles);
}

qe_status launch_objective(const float* W, const float* Wh, const float* H, const float* Sigma,
                           int64_t q, int64_t p, double* out, void* ws, hipStream_t s)
{
    int* status = static_cast<int*>(ws);
    Ws w(ws);
    const int64_t tiles = cdiv(q, kTile) * cdiv(p, kTile);
    double* part0 = w.take<double>(tiles);
    double* part1 = w.take<double>(tiles);
    const bool vec4 = aligned16(W) && aligned16(Wh) && aligned16(Sigma) && (!H || aligned16(H)) &&
                      p % 4 == 0;
    if (vec4 && q % 256 == 0 && p % 256 == 0) {
        // 256 x 256 tiles: q p / 65536 partials (fewer than the 128 x 128 count)
        const int64_t wt = (q / 256) * (p / 256);
        const dim3 grid((unsigned)(8 * cdiv(wt, 8)));
        if (H)
            hipLaunchKernelGGL((quad_form_wide_kernel<true, true>), grid, dim3(512), 0, s, Wh, H,
                               W, Sigma, q, p, part0, status);
        else
            hipLaunchKernelGGL((quad_form_wide_kernel<false, true>), grid, dim3(512), 0, s, Wh,
                               H, W, Sigma, q, p, part0, status);
        hipLaunchKernelGGL(sum_tiles_kernel, dim3(1), dim3(256), 0, s, part0, wt, out, status);
        hipLaunchKernelGGL((quad_form_wide_kernel<false, false>), grid, dim3(512), 0, s, W,
                           (const float*)nullptr, (const float*)nullptr, Sigma, q, p, part1,
                           status);
        hipLaunchKernelGGL(sum_tiles_kernel, dim3(1), dim3(256), 0, s, part1, wt, out + 1, status);
        return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
    }
    // D = What + H - W
    hipLaunchKernelGGL(quad_form_kernel, dim3((unsigned)tiles), dim3(256), 0, s, Wh, H, W, Sigma,
                       q, p, part0, vec4 ? 1 : 0, status);
    hipLaunchKernelGGL(sum_tiles_kernel, dim3(1), dim3(256), 0, s, part0, tiles, out, status);
    // W itself
    hipLaunchKernelGGL(quad_form_kernel, dim3((unsigned)tiles), dim3(256), 0, s, W,
                       (const float*)nullptr, (const float*)nullptr, Sigma, q, p, part1,
                       vec4 ? 1 : 0, status);
    hipLaunchKernelGGL(sum_tiles_kernel, dim3(1), dim3(256), 0, s, part1, tiles, out + 1, status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

// ---------------------------------------------------------------- lambda_max
// Power method (Sec. 4.3): v_k = y_{k-1} / ||y_{k-1}|| (v_0 = 1/sqrt(p)),
// y_k = Sigma v_k, lambda_k = v_k . y_k (Rayleigh quotient of the unit v_k).
// One kernel per iteration: every workgroup first forms 1/||y_{k-1}|| from the
// previous iteration's per-workgroup partials (same fixed-order sum in every
// workgroup), then 8 rows of y_k (two per wavefront, processed together so
// that each float4 of y_{k-1} serves two rows of Sigma; fp64 dot products
// against y_{k-1} itself, the normalisation applied once per row), and writes
// its partials of ||y_k||^2 and v_k . y_k.  Workgroup 0 also records
// lambda_{k-1}.  Sigma is read once per iteration: the kernel is bound by
// that stream (HBM or, for Sigma within the die-level cache, that cache).
constexpr int kSymvRows = 8;
constexpr int kLambdaCheck = 32;   // iterations per host check (the stop is still per iteration)

// Sums the per-workgroup partials (|Sv|^2, v'Sv, |v|^2) of one iteration.
__device__ inline void sum_partials3(const double* part, int n, double* sh, double& yy,
                                     double& vy, double& vv)
{
    double a = 0.0, b = 0.0, c = 0.0;
    for (int e = threadIdx.x; e < n; e += blockDim.x) {
        a += part[3 * e];
        b += part[3 * e + 1];
        c += part[3 * e + 2];
    }
    yy = block_sum_f64(a, sh);
    vy = block_sum_f64(b, sh);
    vv = block_sum_f64(c, sh);
}

// Quotient rho = v'Sv / v'v and squared inclusion radius |Sv - rho v|^2 / |v|^2
// (= (|Sv|^2 - (v'Sv)^2 / v'v) / v'v) of one iteration, into lam_hist.
__device__ inline void put_hist(double* lam_hist, int slot, double yy, double vy, double vv)
{
    lam_hist[2 * slot] = vv > 0.0 ? vy / vv : 0.0;
    lam_hist[2 * slot + 1] = vv > 0.0 ? fmax(0.0, yy - vy * vy / vv) / vv : 0.0;
}

// One power iteration y = Sigma v with v = yprev / |S v_prev| (the first: all
// ones / sqrt(p)); the products and the partial sums are fp64, y is stored in
// fp32 for the next iteration.
__global__ __launch_bounds__(256) void power_step_kernel(const float* __restrict__ Sigma,
                                                         int64_t p, const float* __restrict__ yprev,
                                                         const double* __restrict__ pprev,
                                                         int first, int vec4, float* y,
                                                         double* part, double* lam_hist, int slot)
{
    __shared__ double sh[256];
    __shared__ double wpart[4][3];
    const int nwg = (int)gridDim.x;
    // v_k = yprev * inv (the first iteration: yprev taken as all ones)
    double inv;
    if (first) {
        inv = 1.0 / sqrt((double)p);
    } else {
        double yy, vy, vv;
        sum_partials3(pprev, nwg, sh, yy, vy, vv);
        inv = yy > 0.0 ? 1.0 / sqrt(yy) : 0.0;
        if (blockIdx.x == 0 && threadIdx.x == 0 && slot > 0) put_hist(lam_hist, slot - 1, yy, vy, vv);
    }
    auto wj = [&](int64_t j) -> float { return first ? 1.f : yprev[j]; };
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int RW = kSymvRows / 4;            // rows per wavefront
    const int64_t r0 = (int64_t)blockIdx.x * kSymvRows + wave * RW;
    const float* srow[RW];
    bool ok[RW];
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
        ok[rr] = r0 + rr < p;
        srow[rr] = Sigma + (ok[rr] ? r0 + rr : 0) * p;
    }
    double acc[RW];
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) acc[rr] = 0.0;
    int64_t tail = 0;
    if (vec4) {
        const int64_t n4 = p / 4;
#pragma unroll 4
        for (int64_t f = lane; f < n4; f += 64) {
            const f32x4 wv = first ? f32x4{1.f, 1.f, 1.f, 1.f}
                                   : *reinterpret_cast<const f32x4*>(yprev + 4 * f);
#pragma unroll
            for (int rr = 0; rr < RW; ++rr) {
                const f32x4 sv = *reinterpret_cast<const f32x4*>(srow[rr] + 4 * f);
#pragma unroll
                for (int u = 0; u < 4; ++u) acc[rr] += (double)sv[u] * (double)wv[u];
            }
        }
        tail = 4 * n4;
    }
    for (int64_t j = tail + lane; j < p; j += 64) {
        const double wv = (double)wj(j);
#pragma unroll
        for (int rr = 0; rr < RW; ++rr) acc[rr] += (double)srow[rr][j] * wv;
    }
    double pyy = 0.0, pvy = 0.0, pvv = 0.0;
#pragma unroll
    for (int rr = 0; rr < RW; ++rr) {
        double a = acc[rr];
        for (int off = 32; off > 0; off >>= 1) a += __shfl_xor(a, off, 64);
        if (!ok[rr]) continue;
        const double yd = a * inv;               // (S v)_r in fp64
        if (lane == 0) y[r0 + rr] = (float)yd;
        const double vr = (double)wj(r0 + rr) * inv;
        pyy += yd * yd;
        pvy += vr * yd;
        pvv += vr * vr;
    }
    if (lane == 0) {
        wpart[wave][0] = pyy;
        wpart[wave][1] = pvy;
        wpart[wave][2] = pvv;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int c = 0; c < 3; ++c)
            part[3 * blockIdx.x + c] = ((wpart[0][c] + wpart[1][c]) + wpart[2][c]) + wpart[3][c];
    }
}

// Quotient and radius of the last iteration of a batch.
__global__ __launch_bounds__(256) void power_last_kernel(const double* part, int nwg,
                                                         double* lam_hist, int slot)
{
    __shared__ double sh[256];
    double yy, vy, vv;
    sum_partials3(part, nwg, sh, yy, vy, vv);
    if (threadIdx.x == 0) put_hist(lam_hist, slot, yy, vy, vv);
}

size_t lambda_ws_bytes(int64_t p)
{
    const int64_t nwg = cdiv(p, kSymvRows);
    return kStatusBytes + 2 * align256(sizeof(float) * p) +
           2 * align256(sizeof(double) * 3 * nwg) + align256(sizeof(double) * 2 * kLambdaCheck);
}

qe_status launch_lambda(const float* Sigma, int64_t p, int max_iters, float tol, float* out,
                        void* ws, hipStream_t s)
{
    Ws w(ws);
    const int64_t nwg = cdiv(p, kSymvRows);
    float* y[2] = {w.take<float>(p), w.take<float>(p)};
    double* part[2] = {w.take<double>(3 * nwg), w.take<double>(3 * nwg)};
    double* hist = w.take<double>(2 * kLambdaCheck);      // (rho, radius^2) per iteration
    const int vec4 = (aligned16(Sigma) && p % 4 == 0) ? 1 : 0;
    double last = 0.0, prev = 0.0, last_r2 = 0.0;
    int it = 0, cur = 0;
    while (it < max_iters) {
        const int batch = std::min(kLambdaCheck, max_iters - it);
        for (int b = 0; b < batch; ++b) {
            const int nxt = cur ^ 1;
            hipLaunchKernelGGL(power_step_kernel, dim3((unsigned)nwg), dim3(256), 0, s, Sigma, p,
                               y[cur], part[cur], it + b == 0 ? 1 : 0, vec4, y[nxt], part[nxt],
                               hist, b);
            cur = nxt;
        }
        hipLaunchKernelGGL(power_last_kernel, dim3(1), dim3(256), 0, s, part[cur], (int)nwg, hist,
                           batch - 1);
        it += batch;
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
        double h[2 * kLambdaCheck];
        if (hipMemcpyAsync(h, hist, sizeof(double) * 2 * batch, hipMemcpyDeviceToHost, s) !=
            hipSuccess)
            return QE_ERR_HIP;
        if (hipStreamSynchronize(s) != hipSuccess) return QE_ERR_HIP;
        // the first iteration of the batch whose quotient moved by <= tol relative
        bool done = false;
        for (int b = 0; b < batch && !done; ++b) {
            prev = last;
            last = h[2 * b];
            last_r2 = h[2 * b + 1];
            done = it - batch + b > 0 && last > 0.0 && fabs(last - prev) <= (double)tol * last;
        }
        if (done) break;
    }
    // Upper bound: for v and rho = v'Sv / v'v some eigenvalue of the symmetric
    // Sigma lies within |Sv - rho v| / |v| of rho, and v approximates the
    // leading eigenvector, so rho plus that radius bounds lambda_max from
    // above.  Both come from fp64 sums of the fp64 product S v; a relative
    // 2^-30 covers their rounding, and the result is rounded up to fp32.  The
    // IHT step 1 / (2 lambda) then stays within the Lipschitz bound of Lemma 3.
    const double bound = (last + sqrt(last_r2)) * (1.0 + 0x1p-30);
    float f = (float)bound;
    if ((double)f < bound) f = std::nextafter(f, INFINITY);
    *out = f;
    return QE_OK;
}

}  // namespace qe
