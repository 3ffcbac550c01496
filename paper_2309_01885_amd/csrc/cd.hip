// Blocked cyclic coordinate descent of QuantEase on gfx950.
//
// State: What (q x p), codes (q x p, uint8) and the residual R = (What - W) Sigma.
// Lemma 1 (Sec. 4.2) in residual form: for column j and every row i,
//     beta = What_ij - R_ij / Sigma_jj,   What_ij <- q_i(beta),
// and the rank-1 identity of Sec. 4.2 (both halves fused, as the paper's
// acceleration note suggests) keeps R exact:  R += delta_{:,j} Sigma_{j,:}.
//
// Columns are taken in blocks J of width B.  One launch ("step") of
// cd_step_kernel does two independent jobs on disjoint data:
//  * panel workgroups (16 rows each) run the B column updates of block J in
//    order.  Each row is spread over 16 lanes (one DPP row); lane g holds the
//    block columns g, g + 16, ... in registers.  The owner lane of column j
//    computes the new code, broadcasts delta with DPP row_newbcast, and every
//    lane applies delta * Sigma_{j, its columns} from an LDS copy of
//    Sigma_{J,J}.  Before that, the panel adds the previous block's update to
//    its own columns (R_{:,J} += Delta_prev Sigma_{Jprev,J}) and writes R_{:,J}.
//  * GEMM workgroups apply the previous block's update to every other
//    column: R_{:,~J} += Delta_prev Sigma_{Jprev,~J}, an fp32 matrix-core GEMM
//    with K = B (Sigma symmetric, so Sigma_{Jprev,c} is row c of Sigma).
// The panel of block J therefore overlaps the wide GEMM of the block before
// it.  After the last block, a GEMM-only step leaves R = (What - W) Sigma exact.
#include <utility>

#include "qe_internal.h"

namespace qe {

// ---------------------------------------------------------------- setup kernels
__global__ void diag_prep_kernel(const float* __restrict__ Sigma, int64_t p, float* inv_d,
                                 int* status)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= p) return;
    const float d = Sigma[j * p + j];
    if (!(d > 0.f) || !isfinite(d)) {
        set_status(status, QE_ERR_DIAG);
        inv_d[j] = 0.f;
    } else {
        inv_d[j] = 1.0f / d;
    }
}

__global__ void grid_prep_kernel(const float* __restrict__ scale, const float* __restrict__ zero,
                                 int64_t q, float* inv_s, int* status)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= q) return;
    const float s = scale[i], z = zero[i];
    if (!(s > 0.f) || !isfinite(s) || !isfinite(z)) {
        set_status(status, QE_ERR_SCALE);
        inv_s[i] = 0.f;
    } else {
        inv_s[i] = 1.0f / s;
    }
}

// What = W - H (H may be null), R = 0 (Sec. 4.1 / Sec. 5.3 initialisation).
__global__ void init_from_w_kernel(const float* __restrict__ W, const float* __restrict__ H,
                                   float* Wh, float* R, int64_t count, const int* status)
{
    if (failed(status)) return;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x) {
        Wh[e] = H ? W[e] - H[e] : W[e];
        R[e] = 0.f;
    }
}

// R = (What + H - W) Sigma over all 128 x 128 tiles (warm start from any What).
__global__ __launch_bounds__(256) void residual_init_kernel(const float* Wh, const float* H,
                                                            const float* W, const float* Sigma,
                                                            int64_t q, int64_t p, float* R,
                                                            int vec4, const int* status)
{
    if (failed(status)) return;
    __shared__ __attribute__((aligned(16))) float lds[kNTLdsFloats];
    const int64_t tn_count = cdiv(p, kTile);
    const int64_t row0 = (blockIdx.x / tn_count) * kTile, col0 = (blockIdx.x % tn_count) * kTile;
    f32x16 acc[2][2];
    zero_acc(acc);
    const CompOp A{Wh, H, W, p, q, p, vec4 != 0};
    const RowOp B{Sigma, p, p, p, vec4 != 0};
    nt_tile(A, row0, B, col0, p, lds, acc);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t r = row0 + acc_row(mi, v), c = col0 + acc_col(ni);
                if (r < q && c < p) R[r * p + c] = acc[mi][ni][v];
            }
}

// ---------------------------------------------------------------- objective from R
// f = <What + H - W, R> in fp64: fixed grid, fixed per-thread order, fixed tree.

__global__ __launch_bounds__(256) void obj_partial_kernel(const float* __restrict__ W,
                                                          const float* __restrict__ Wh,
                                                          const float* __restrict__ H,
                                                          const float* __restrict__ R,
                                                          int64_t count, double* partial,
                                                          const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double acc = 0.0;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x) {
        float d = Wh[e] - W[e];
        if (H) d = (Wh[e] + H[e]) - W[e];
        acc += (double)d * (double)R[e];
    }
    const double s = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void sum_partials_kernel(const double* partial, int n,
                                                           double* out, const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double acc = 0.0;
    for (int e = threadIdx.x; e < n; e += blockDim.x) acc += partial[e];
    const double s = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) *out = s;
}

// ---------------------------------------------------------------- the step kernel
struct StepArgs {
    float* R;
    float* Wh;
    uint8_t* codes;
    const float* Sigma;
    const float* inv_d;
    const float* scale;
    const float* zero;
    const float* inv_s;
    float* dcur;          // q x B: this block's column deltas (panel output)
    const float* dprev;   // q x B: previous block's deltas (applied in this step)
    int64_t q, p;
    int64_t blk;          // first column of the panel block, or -1 (GEMM-only step)
    int64_t prev_blk;     // first column of the previous block, or -1 (panel-only step)
    int cur_w, prev_w;    // widths of the two blocks (<= B)
    float maxq;
    int codes_valid;      // current codes may be kept on an exact tie (Sec. 4.3)
    int n_panel;          // workgroups [0, n_panel) run the panel
    int64_t tiles_n;      // GEMM column tiles
    int sig_vec4;
    const int* status;
};

template <int SLOTS>
struct PanelState {
    float L[SLOTS];     // residual of the lane's block columns (local copy of R_{i,J})
    float w[SLOTS];     // What_{i,J}
    float cd[SLOTS];    // codes as floats
    float dl[SLOTS];    // delta of the columns this lane owns
    float invd[SLOTS];  // 1 / Sigma_jj
};

// Broadcast lane O of every 16-lane DPP row to the whole row.
template <int O>
__device__ __forceinline__ float row_bcast(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x150 + O, 0xF, 0xF,
                                                      false));
}

// One column update (column J of the block) for all 16 rows of the workgroup.
template <int SLOTS, int J>
__device__ __forceinline__ void panel_step(PanelState<SLOTS>& st, const float* sS, int g,
                                           int width, float s, float z, float inv_s,
                                           float maxq, bool cvalid)
{
    constexpr int B = 16 * SLOTS;
    constexpr int M = J / 16, O = J % 16;
    if (J >= width) return;                          // uniform across the workgroup
    // Lemma 1: unconstrained minimiser, then its position t on the grid
    const float beta = fmaf(-st.L[M], st.invd[M], st.w[M]);
    const float t = fmaf(beta, inv_s, z);
    // nearest level (half to even), clamped to the finite grid
    float k = fminf(fmaxf(rintf(t), 0.f), maxq);
    // modified CD: an equally near current level is kept
    if (cvalid && fabsf(t - st.cd[M]) <= fabsf(t - k)) k = st.cd[M];
    const float wn = s * (k - z);
    const float delta = wn - st.w[M];
    const float db = row_bcast<O>(delta);
    if (g == O) {
        st.w[M] = wn;
        st.cd[M] = k;
        st.dl[M] = delta;
    }
    // rank-1 update restricted to the block: L_{i,c} += delta_i Sigma_{j,c}
    const float* srow = sS + J * B + g * SLOTS;
    if constexpr (SLOTS % 4 == 0) {
#pragma unroll
        for (int q4 = 0; q4 < SLOTS / 4; ++q4) {
            const f32x4 sv = *reinterpret_cast<const f32x4*>(srow + 4 * q4);
#pragma unroll
            for (int u = 0; u < 4; ++u) st.L[4 * q4 + u] = fmaf(db, sv[u], st.L[4 * q4 + u]);
        }
    } else {
#pragma unroll
        for (int mm = 0; mm < SLOTS; ++mm) st.L[mm] = fmaf(db, srow[mm], st.L[mm]);
    }
}

template <int SLOTS, int... Js>
__device__ __forceinline__ void panel_run(std::integer_sequence<int, Js...>,
                                          PanelState<SLOTS>& st, const float* sS, int g,
                                          int width, float s, float z, float inv_s, float maxq,
                                          bool cvalid)
{
    (panel_step<SLOTS, Js>(st, sS, g, width, s, z, inv_s, maxq, cvalid), ...);
}

// Stages Sigma[r0 + k][c0 + c] (k < kw, c < cw; else 0) into LDS with the
// column permutation used by the panel: column c = 16 m + g sits at g * SLOTS + m.
template <int SLOTS>
__device__ inline void stage_sigma_block(const float* __restrict__ Sigma, int64_t p, int64_t r0,
                                         int kw, int64_t c0, int cw, float* sS)
{
    constexpr int B = 16 * SLOTS;
    for (int e = threadIdx.x; e < B * B; e += blockDim.x) {
        const int k = e / B, c = e % B;
        float v = 0.f;
        if (k < kw && c < cw) v = Sigma[(r0 + k) * p + c0 + c];
        sS[k * B + (c & 15) * SLOTS + (c >> 4)] = v;
    }
}

template <int SLOTS>
__device__ void panel_role(const StepArgs& a, float* lds)
{
    constexpr int B = 16 * SLOTS;
    float* sS = lds;            // B x B
    float* sD = lds + B * B;    // 16 x B: previous deltas of this workgroup's rows
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane & 15;
    const int lrow = wave * 4 + (lane >> 4);
    const int64_t i0 = (int64_t)blockIdx.x * 16;
    const int64_t i = i0 + lrow;
    const bool rowok = i < a.q;
    const int width = a.cur_w;
    const int64_t p = a.p;

    PanelState<SLOTS> st;
#pragma unroll
    for (int m = 0; m < SLOTS; ++m) {
        const int c = 16 * m + g;
        const bool ok = rowok && c < width;
        const int64_t idx = i * p + a.blk + c;
        st.L[m] = ok ? a.R[idx] : 0.f;
        st.w[m] = ok ? a.Wh[idx] : 0.f;
        st.cd[m] = ok ? (float)a.codes[idx] : 0.f;
        st.invd[m] = c < width ? a.inv_d[a.blk + c] : 0.f;
        st.dl[m] = 0.f;
    }
    const float s = rowok ? a.scale[i] : 1.f;
    const float z = rowok ? a.zero[i] : 0.f;
    const float inv_s = rowok ? a.inv_s[i] : 1.f;

    if (a.prev_blk >= 0) {
        // look-ahead: R_{i,J} += Delta_prev_{i,:} Sigma_{Jprev, J}
        const int pw = a.prev_w;
        stage_sigma_block<SLOTS>(a.Sigma, p, a.prev_blk, pw, a.blk, width, sS);
        for (int e = threadIdx.x; e < 16 * B; e += blockDim.x) {
            const int64_t ii = i0 + e / B;
            sD[e] = ii < a.q ? a.dprev[ii * B + (e % B)] : 0.f;
        }
        __syncthreads();
        for (int k = 0; k < pw; ++k) {
            const float dk = sD[lrow * B + k];
#pragma unroll
            for (int m = 0; m < SLOTS; ++m) st.L[m] = fmaf(dk, sS[k * B + g * SLOTS + m], st.L[m]);
        }
#pragma unroll
        for (int m = 0; m < SLOTS; ++m) {
            const int c = 16 * m + g;
            if (rowok && c < width) a.R[i * p + a.blk + c] = st.L[m];
        }
        __syncthreads();
    }

    stage_sigma_block<SLOTS>(a.Sigma, p, a.blk, width, a.blk, width, sS);
    __syncthreads();
    panel_run<SLOTS>(std::make_integer_sequence<int, B>{}, st, sS, g, width, s, z, inv_s,
                     a.maxq, a.codes_valid != 0);

#pragma unroll
    for (int m = 0; m < SLOTS; ++m) {
        const int c = 16 * m + g;
        if (rowok && c < width) {
            a.Wh[i * p + a.blk + c] = st.w[m];
            a.codes[i * p + a.blk + c] = (uint8_t)st.cd[m];
        }
        if (rowok) a.dcur[i * B + c] = st.dl[m];
    }
}

template <int SLOTS>
__device__ void gemm_role(const StepArgs& a, float* lds, int64_t t)
{
    constexpr int B = 16 * SLOTS;
    const int64_t tm = t / a.tiles_n, tn = t % a.tiles_n;
    const int64_t row0 = tm * kTile, col0 = tn * kTile;
    const int64_t ex0 = a.blk, ex1 = a.blk >= 0 ? a.blk + a.cur_w : -1;
    if (a.blk >= 0 && col0 >= ex0 && min(col0 + kTile, a.p) <= ex1) return;   // all in J
    f32x16 acc[2][2];
    zero_acc(acc);
    const RowOp A{a.dprev, B, a.q, a.prev_w, true};
    const RowOp Bo{a.Sigma + a.prev_blk, a.p, a.p, a.prev_w, a.sig_vec4 != 0};
    nt_tile(A, row0, Bo, col0, a.prev_w, lds, acc);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t r = row0 + acc_row(mi, v), c = col0 + acc_col(ni);
                if (r < a.q && c < a.p && !(c >= ex0 && c < ex1))
                    a.R[r * a.p + c] += acc[mi][ni][v];
            }
}

template <int SLOTS>
constexpr int step_lds_floats()
{
    return (16 * SLOTS) * (16 * SLOTS) + 16 * (16 * SLOTS) > kNTLdsFloats
               ? (16 * SLOTS) * (16 * SLOTS) + 16 * (16 * SLOTS)
               : kNTLdsFloats;
}

template <int SLOTS>
__global__ __launch_bounds__(256) void cd_step_kernel(StepArgs a)
{
    if (failed(a.status)) return;
    __shared__ __attribute__((aligned(16))) float lds[step_lds_floats<SLOTS>()];
    if ((int)blockIdx.x < a.n_panel)
        panel_role<SLOTS>(a, lds);
    else
        gemm_role<SLOTS>(a, lds, (int64_t)blockIdx.x - a.n_panel);
}

// ---------------------------------------------------------------- host side
static int block_width(int block) { return block == 0 ? 128 : block; }

size_t cd_ws_bytes(int64_t q, int64_t p, int block)
{
    const int B = block_width(block);
    size_t b = kStatusBytes;
    b += align256(sizeof(float) * p);               // inv_d
    b += align256(sizeof(float) * q);               // inv_s
    b += 2 * align256(sizeof(float) * q * B);       // delta double buffer
    b += align256(sizeof(double) * kObjBlocks);     // objective partials
    return b;
}

// <What + H - W, R> into *out (fp64, deterministic); `part` holds kObjBlocks doubles.
qe_status launch_residual_dot(const float* W, const float* Wh, const float* H, const float* R,
                              int64_t count, double* out, double* part, const int* status,
                              hipStream_t s)
{
    hipLaunchKernelGGL(obj_partial_kernel, dim3(kObjBlocks), dim3(256), 0, s, W, Wh, H, R, count,
                       part, status);
    hipLaunchKernelGGL(sum_partials_kernel, dim3(1), dim3(256), 0, s, part, kObjBlocks, out,
                       status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

template <int SLOTS>
static qe_status launch_steps(StepArgs base, float* d0, float* d1, int64_t nb, int64_t q,
                              int64_t p, hipStream_t s)
{
    constexpr int B = 16 * SLOTS;
    const int64_t panel_wgs = cdiv(q, 16);
    const int64_t tiles_m = cdiv(q, kTile), tiles_n = cdiv(p, kTile);
    for (int64_t k = 0; k <= nb; ++k) {
        StepArgs a = base;
        a.blk = k < nb ? k * B : -1;
        a.cur_w = k < nb ? (int)std::min<int64_t>(B, p - k * B) : 0;
        a.prev_blk = k > 0 ? (k - 1) * B : -1;
        a.prev_w = k > 0 ? (int)std::min<int64_t>(B, p - (k - 1) * B) : 0;
        a.dcur = (k & 1) ? d1 : d0;
        a.dprev = (k & 1) ? d0 : d1;
        a.n_panel = k < nb ? (int)panel_wgs : 0;
        a.tiles_n = tiles_n;
        const int64_t gemm_wgs = k > 0 ? tiles_m * tiles_n : 0;
        const int64_t grid = a.n_panel + gemm_wgs;
        hipLaunchKernelGGL(cd_step_kernel<SLOTS>, dim3((unsigned)grid), dim3(256), 0, s, a);
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    return QE_OK;
}

qe_status launch_cd(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                    const float* scale, const float* zero, float* Wh, uint8_t* codes, float* R,
                    const float* H, int sweeps, int block, uint32_t flags, double* obj,
                    int obj_stride, void* ws, hipStream_t s)
{
    const int B = block_width(block);
    int* status = static_cast<int*>(ws);
    Ws w(ws);
    float* inv_d = w.take<float>(p);
    float* inv_s = w.take<float>(q);
    float* d0 = w.take<float>((size_t)q * B);
    float* d1 = w.take<float>((size_t)q * B);
    double* part = w.take<double>(kObjBlocks);

    hipLaunchKernelGGL(diag_prep_kernel, dim3((unsigned)cdiv(p, 256)), dim3(256), 0, s, Sigma, p,
                       inv_d, status);
    hipLaunchKernelGGL(grid_prep_kernel, dim3((unsigned)cdiv(q, 256)), dim3(256), 0, s, scale,
                       zero, q, inv_s, status);
    const bool vec4 = aligned16(Sigma) && aligned16(W) && aligned16(Wh) && (p % 4 == 0) &&
                      (!H || aligned16(H));
    if (flags & QE_INIT_FROM_W) {
        hipLaunchKernelGGL(init_from_w_kernel, dim3(2048), dim3(256), 0, s, W, H, Wh, R, q * p,
                           status);
    } else if (!(flags & QE_R_VALID)) {
        const int64_t tiles = cdiv(q, kTile) * cdiv(p, kTile);
        hipLaunchKernelGGL(residual_init_kernel, dim3((unsigned)tiles), dim3(256), 0, s, Wh, H, W,
                           Sigma, q, p, R, vec4 ? 1 : 0, status);
    }
    if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;

    StepArgs base{};
    base.R = R;
    base.Wh = Wh;
    base.codes = codes;
    base.Sigma = Sigma;
    base.inv_d = inv_d;
    base.scale = scale;
    base.zero = zero;
    base.inv_s = inv_s;
    base.q = q;
    base.p = p;
    base.maxq = (float)((1 << bits) - 1);
    base.sig_vec4 = (aligned16(Sigma) && p % 4 == 0) ? 1 : 0;
    base.status = status;
    const bool codes_valid0 = (flags & QE_CODES_VALID) && !(flags & QE_INIT_FROM_W);
    const int64_t nb = cdiv(p, B);
    for (int sw = 0; sw < sweeps; ++sw) {
        base.codes_valid = (sw > 0 || codes_valid0) ? 1 : 0;
        qe_status st;
        switch (B) {
            case 16: st = launch_steps<1>(base, d0, d1, nb, q, p, s); break;
            case 32: st = launch_steps<2>(base, d0, d1, nb, q, p, s); break;
            case 64: st = launch_steps<4>(base, d0, d1, nb, q, p, s); break;
            default: st = launch_steps<8>(base, d0, d1, nb, q, p, s); break;
        }
        if (st != QE_OK) return st;
        if (obj) {
            st = launch_residual_dot(W, Wh, H, R, q * p, obj + (size_t)sw * obj_stride, part,
                                     status, s);
            if (st != QE_OK) return st;
        }
    }
    return QE_OK;
}

}  // namespace qe
