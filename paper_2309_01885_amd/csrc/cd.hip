// Blocked cyclic coordinate descent of QuantEase on gfx950.
//
// State: What (q x p), codes (q x p, uint8) and the residual R = (What - W) Sigma.
// Lemma 1 (Sec. 3.2) in residual form: for column j and every row i,
//     beta = What_ij - R_ij / Sigma_jj,   What_ij <- q_i(beta),
// and the rank-1 identity of Sec. 3.2 (both halves fused, as the paper's
// acceleration note suggests) keeps R exact:  R += delta_{:,j} Sigma_{j,:}.
//
// Columns are taken in blocks J of width B (the panel width), grouped into
// super-blocks of S = m * B columns.  One launch ("step") of cd_step_kernel
// does two independent jobs on disjoint data:
//  * panel workgroups (16 rows each) run the m blocks of super-block t in
//    order.  Each row is spread over 16 lanes (one DPP row); lane g holds the
//    block columns g, g + 16, ... in registers.  The owner lane of column j
//    computes the new code, broadcasts delta with DPP row_newbcast, and every
//    lane applies delta * Sigma_{j, its columns} from an LDS copy of
//    Sigma_{J,J}.  Before a block starts, the panel adds to its columns the
//    deltas of super-block t-1 (written back to R) and of the earlier blocks
//    of super-block t (kept local).
//  * GEMM workgroups apply the deltas of super-block t-1 to every column
//    outside super-block t: R_{:,c} += Delta_{t-1} Sigma_{SB(t-1), c}, an fp32
//    matrix-core GEMM with K = S (Sigma symmetric, so Sigma_{SB(t-1), c} is a
//    stretch of row c).
// The panels of super-block t therefore overlap the wide GEMM of super-block
// t-1; after the last one a GEMM-only step leaves R = (What - W) Sigma exact.
#include <utility>

#include "nt_x3.h"
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

// What = W - H (H may be null), R = 0 (Sec. 3.1 / Sec. 4.3 initialisation).
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
__global__ __launch_bounds__(256, 2) void residual_init_kernel(const float* Wh, const float* H,
                                                            const float* W, const float* Sigma,
                                                            int64_t q, int64_t p, float* R,
                                                            int vec4, int fp32, const int* status)
{
    if (failed(status)) return;
    __shared__ __attribute__((aligned(16))) float lds[kNTLdsFloats];
    const int64_t tn_count = cdiv(p, kTile);
    const int64_t row0 = (blockIdx.x / tn_count) * kTile, col0 = (blockIdx.x % tn_count) * kTile;
    f32x16 acc[2][2];
    zero_acc(acc);
    if (fp32) {
        const CompOp A{Wh, H, W, p, q, p, vec4 != 0};
        const RowOp B{Sigma, p, p, p, vec4 != 0};
        nt_tile(A, row0, B, col0, p, lds, acc);
    } else {
        // split bf16 products (nt_x3.h)
        const X3Comp A{Wh, H, W, p, q, p};
        const X3Row B{Sigma, p, p, p};
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
        if (vec4 && row0 + kTile <= q && col0 + kTile <= p && p % (2 * kX3KC) == 0)
            nt_tile_x3_full(A, row0, B, col0, p, l32, acc);
        else
            nt_tile_x3_edge(A, row0, B, col0, p, l32, acc);
    }
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
                                                          int64_t count, int vec4, double* partial,
                                                          const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double acc = 0.0;
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t tail = 0;
    if (vec4) {
        const int64_t n4 = count / 4;
        const f32x4* W4 = reinterpret_cast<const f32x4*>(W);
        const f32x4* Wh4 = reinterpret_cast<const f32x4*>(Wh);
        const f32x4* H4 = reinterpret_cast<const f32x4*>(H);
        const f32x4* R4 = reinterpret_cast<const f32x4*>(R);
#pragma unroll 2
        for (int64_t e = tid; e < n4; e += G) {
            const f32x4 w = W4[e], wh = Wh4[e], r = R4[e];
            f32x4 d = wh - w;
            if (H) d = (wh + H4[e]) - w;
#pragma unroll
            for (int u = 0; u < 4; ++u) acc += (double)d[u] * (double)r[u];
        }
        tail = n4 * 4;
    }
    for (int64_t e = tail + tid; e < count; e += G) {
        float d = Wh[e] - W[e];
        if (H) d = (Wh[e] + H[e]) - W[e];
        acc += (double)d * (double)R[e];
    }
    const double s = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) partial[blockIdx.x] = s;
}

// *out = (*prev, or 0 without prev) + the n partials, in a fixed order (out may
// equal prev).
__global__ __launch_bounds__(256) void sum_partials_kernel(const double* partial, int n,
                                                           const double* prev, double* out,
                                                           const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double acc = 0.0;
    for (int e = threadIdx.x; e < n; e += blockDim.x) acc += partial[e];
    const double s = block_sum_f64(acc, sh);
    if (threadIdx.x == 0) *out = (prev ? *prev : 0.0) + s;
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
    float* dcur;          // q x S: deltas of the current super-block (panel output)
    const float* dprev;   // q x S: deltas of the previous super-block (applied here)
    int64_t q, p;
    int64_t sb;           // first column of the current super-block, or -1 (GEMM-only step)
    int64_t psb;          // first column of the previous super-block, or -1 (panel-only step)
    int sbw, psbw;        // their widths (<= S)
    int S;                // super-block width = row stride of dcur / dprev
    float maxq;
    int codes_valid;      // current codes may be kept on an exact tie (Sec. 3.3)
    int relax;            // write beta unquantized (relaxed sweep, Sec. 3.2)
    int intd;             // deltas as code differences k_new - k_old (see launch_cd)
    int fp32;             // GEMM role on the fp32 matrix cores (else the split bf16 ones)
    int dense;            // no sparse block update (every tile on the matrix cores)
    int n_panel;          // workgroups [0, n_panel) run the panel
    int64_t tiles_n;      // GEMM column tiles
    int sig_vec4;
    int r_vec4;           // R allows aligned 16-byte row access
    int* nzcur;           // q: nonzero code differences of each row in the current super-block
    const int* nzprev;    // q: the same for the previous super-block (code differences only)
    double* fpart;        // per panel wave: the objective change of this sweep's moves so far
    int fobj;             // accumulate fpart (the per-sweep objective is wanted)
    int ffirst;           // first launch of a sweep: fpart is written, not added to
    const int* status;
};

// Per lane, slot m holds block column 16 m + g.  Quantized sweeps keep What
// fixed during the block and track codes: the new What and the deltas follow
// from the final codes after the block.
template <int SLOTS>
struct PanelState {
    float L[SLOTS];     // residual of the lane's block columns (local copy of R_{i,J})
    float w[SLOTS];     // What_{i,J} (relaxed sweeps: updated as the block runs)
    float u[SLOTS];     // quantized: 1 / (Sigma_jj s_i); relaxed: 1 / Sigma_jj
    float v[SLOTS];     // quantized: What_ij / s_i + z_i (the code itself with code
                        // differences); relaxed: delta of owned columns
    float k[SLOTS];     // quantized: code of the column (NaN while none is valid)
    float Ls;           // L of the current 16-column group's slot at the group's start
    float fl;           // the row's objective change over the block (this lane's share)
    float srow[3][SLOTS];   // Sigma rows J, J+1, J+2 (lane's columns), fetched ahead
};

// Broadcast lane O of every 16-lane DPP row to the whole row.
template <int O>
__device__ __forceinline__ float row_bcast(float v)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + O, 0xF, 0xF, false));
}

// Fetches this lane's entries of Sigma row `row` of the block, from slot FIRST
// on (earlier slots are no longer needed): single floats up to the next float4
// boundary, then float4 granules.  Loading only live slots matters: a register
// loaded but dead may be reused at once, which makes the fetch wait.
template <int SLOTS, int FIRST = 0>
__device__ __forceinline__ void load_srow(float (&dst)[SLOTS], const float* sS, int row, int g)
{
    const float* src = sS + row * (16 * SLOTS) + g * SLOTS;
    if constexpr (SLOTS % 4 == 0) {
        constexpr int A = (FIRST + 3) / 4 * 4;
#pragma unroll
        for (int m = FIRST; m < A; ++m) dst[m] = src[m];
#pragma unroll
        for (int q4 = A / 4; q4 < SLOTS / 4; ++q4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(src + 4 * q4);
#pragma unroll
            for (int u = 0; u < 4; ++u) dst[4 * q4 + u] = v[u];
        }
    } else {
#pragma unroll
        for (int m = 0; m < SLOTS; ++m) dst[m] = src[m];
    }
}

// Objective change of the moves delta_G of one 16-column group G, from the
// residual R0 at the group's start: summed over the group's coordinate steps,
// delta (2 R_ij + delta Sigma_jj) = 2 <delta_G, R0_G> + delta_G^T Sigma_GG
// delta_G = <delta_G, R0_G + R1_G>, where R1 = R0 + Sigma_GG delta_G is the
// slot's residual once the group is done (every lane's slot M column receives
// all 16 moves of group M).  With code differences the lane's share is in
// units of s_i.
template <int SLOTS, int M, bool RELAX, bool INTD>
__device__ __forceinline__ void group_objective(PanelState<SLOTS>& st, int g, int width, float s,
                                                float z)
{
    float d;
    if constexpr (RELAX)
        d = st.v[M];
    else if constexpr (INTD)
        d = st.k[M] - st.v[M];
    else
        d = fmaf(s, st.k[M] - z, -st.w[M]);
    if (16 * M + g < width) st.fl = fmaf(d, st.Ls + st.L[M], st.fl);
}

// One column update (column J of the block) for all 16 rows of the workgroup.
// FULL blocks (width == B) carry no per-column test.  The Sigma row of column
// J + 2 is fetched from LDS while column J's dependent chain runs.
template <int SLOTS, int J, bool FULL, bool RELAX, bool INTD>
__device__ __forceinline__ void panel_step(PanelState<SLOTS>& st, const float* sS, int g,
                                           int width, float s, float z, float maxq)
{
    constexpr int B = 16 * SLOTS;
    constexpr int M = J / 16, O = J % 16;
    if constexpr (O == 0) st.Ls = st.L[M];
    if (!FULL && J >= width) {                       // uniform across the workgroup
        if constexpr (O == 15) group_objective<SLOTS, M, RELAX, INTD>(st, g, width, s, z);
        return;
    }
    if constexpr (J + 2 < B) load_srow<SLOTS, (J + 2) / 16>(st.srow[(J + 2) % 3], sS, J + 2, g);
    // keep the fetch here: the scheduler would otherwise sink it next to its use
    __builtin_amdgcn_sched_barrier(0);
    const float w = st.w[M];
    const bool own = g == O;
    float delta;
    if constexpr (RELAX) {
        // relaxed sweep: the unconstrained minimiser of Lemma 1 itself
        const float beta = fmaf(-st.L[M], st.u[M], w);
        delta = beta - w;
        st.w[M] = own ? beta : w;
        st.v[M] = own ? delta : st.v[M];
    } else {
        // Lemma 1's minimiser on the grid axis: t = beta / s + z with
        // beta = What_ij - R_ij / Sigma_jj
        const float t = fmaf(-st.L[M], st.u[M], st.v[M]);
        // nearest level (half to even), clamped to the finite grid
        const float kn = __builtin_amdgcn_fmed3f(rintf(t), 0.f, maxq);
        // modified CD: a valid, equally near current level is kept (NaN never is)
        const float kc = st.k[M];
        const float k = fabsf(t - kc) <= fabsf(t - kn) ? kc : kn;
        if constexpr (INTD)
            delta = s * (k - kc);                    // What on the grid: s (k_new - k_old)
        else
            delta = fmaf(s, k - z, -w);              // s (k - z) - What_ij
        st.k[M] = own ? k : kc;
    }
    const float db = row_bcast<O>(delta);
    // rank-1 update restricted to the block: L_{i,c} += delta_i Sigma_{j,c}.
    // Slot mm holds columns 16 mm + g; slots below M are finished this block.
#pragma unroll
    for (int mm = M; mm < SLOTS; ++mm) st.L[mm] = fmaf(db, st.srow[J % 3][mm], st.L[mm]);
    if constexpr (O == 15) group_objective<SLOTS, M, RELAX, INTD>(st, g, width, s, z);
}

template <int SLOTS, bool FULL, bool RELAX, bool INTD, int... Js>
__device__ __forceinline__ void panel_run(std::integer_sequence<int, Js...>,
                                          PanelState<SLOTS>& st, const float* sS, int g,
                                          int width, float s, float z, float maxq)
{
    load_srow<SLOTS>(st.srow[0], sS, 0, g);
    if constexpr (16 * SLOTS > 1) load_srow<SLOTS>(st.srow[1], sS, 1, g);
    (panel_step<SLOTS, Js, FULL, RELAX, INTD>(st, sS, g, width, s, z, maxq), ...);
}

// Stages Sigma[r0 + k][c0 + c] (k < kw, c < cw; else 0) into LDS with the
// column permutation used by the panel: column c = 16 m + g sits at g * SLOTS + m.
// Full blocks issue all their loads before the first LDS store, so the global
// latency is paid once per block.
template <int SLOTS>
__device__ __forceinline__ void stage_sigma_block(const float* __restrict__ Sigma, int64_t p,
                                                  int64_t r0, int kw, int64_t c0, int cw,
                                                  bool vec4, float* sS)
{
    constexpr int B = 16 * SLOTS;
    constexpr int Q = B / 4;                     // float4 per row
    constexpr int PER = (B * Q + 255) / 256;     // float4 per thread
    if constexpr (SLOTS % 4 == 0) {
        if (kw == B && cw == B) {
            // thread t takes (row k, lane g) pairs: the lane's SLOTS columns
            // g, g + 16, ... of row k, read as single floats (16 lanes of a
            // wave cover 64 contiguous bytes of a row), written as float4
            // runs of the panel layout (a quarter of the LDS store
            // instructions of element-wise stores)
            constexpr int PPT = B * 16 / 256;    // pairs per thread
            float v[PPT][SLOTS];
#pragma unroll
            for (int u = 0; u < PPT; ++u) {
                const int pi = threadIdx.x + 256 * u;
                const int k = pi >> 4, g = pi & 15;
                const float* src = Sigma + (r0 + k) * p + c0 + g;
#pragma unroll
                for (int m = 0; m < SLOTS; ++m) v[u][m] = src[16 * m];
            }
#pragma unroll
            for (int u = 0; u < PPT; ++u) {
                const int pi = threadIdx.x + 256 * u;
                const int k = pi >> 4, g = pi & 15;
#pragma unroll
                for (int m4 = 0; m4 < SLOTS / 4; ++m4)
                    *reinterpret_cast<f32x4*>(sS + k * B + g * SLOTS + 4 * m4) =
                        f32x4{v[u][4 * m4], v[u][4 * m4 + 1], v[u][4 * m4 + 2], v[u][4 * m4 + 3]};
            }
            return;
        }
    }
    if (vec4 && kw == B && cw == B) {
        f32x4 v[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int f = threadIdx.x + 256 * u;
            if (f < B * Q)
                v[u] = *reinterpret_cast<const f32x4*>(Sigma + (r0 + f / Q) * p + c0 + 4 * (f % Q));
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            const int f = threadIdx.x + 256 * u;
            if (f >= B * Q) continue;
            const int k = f / Q, cb = 4 * (f % Q);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int cc = cb + e;
                sS[k * B + (cc & 15) * SLOTS + (cc >> 4)] = v[u][e];
            }
        }
        return;
    }
    for (int e = threadIdx.x; e < B * B; e += blockDim.x) {
        const int k = e / B, cc = e % B;
        float x = 0.f;
        if (k < kw && cc < cw) x = Sigma[(r0 + k) * p + c0 + cc];
        sS[k * B + (cc & 15) * SLOTS + (cc >> 4)] = x;
    }
}

// L_{i,J} += dscale_i D_{i, k0..k0+kw} Sigma_{r0..r0+kw, J} for the workgroup's
// 16 rows (kw <= B), with D a q x S row-major delta buffer and dscale the row's
// grid step when D holds code differences (else 1).
//
// B >= 64: on matrix cores (v_mfma_f32_16x16x4f32, 16 x 16 output tiles; wave
// w owns block columns [B/4 w, B/4 (w+1))).  A = the 16 delta rows, fetched as
// float4 straight into registers; B = Sigma_{r0+k, j0+c}, staged in LDS
// transposed (k contiguous) from rows j0+c of Sigma, which are the same
// numbers by symmetry.  Both operands use the same k order inside each group
// of 16 (lane half h covers k = 4h .. 4h+3), which leaves the sum unchanged.
// The 16 x B result passes through LDS into the panel's register layout.
// B < 64: a VALU loop over k with Sigma staged in the panel layout.

constexpr int kTStride = 128 + 4;   // transposed-Sigma LDS row stride (floats)

template <int SLOTS>
__device__ __forceinline__ void add_block_update(PanelState<SLOTS>& st, const StepArgs& a,
                                                 const float* D, int64_t k0, int kw, int64_t r0,
                                                 int64_t j0, int width, int64_t i0, int lrow,
                                                 int g, float* lds, float dscale)
{
    constexpr int B = 16 * SLOTS;
    if constexpr (SLOTS >= 4) {
        constexpr int CPW = B / 4;               // block columns per wave
        constexpr int T = CPW / 16;              // 16-column MFMA tiles per wave
        constexpr int KG = B / 16;               // k groups of 16
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        const int r = lane & 15, h = lane >> 4;
        float* sT = lds;                         // B columns x kTStride
        __syncthreads();                         // LDS free
        // Sigma staged transposed: sT[c][k] = Sigma[j0 + c][r0 + k]
        constexpr int PER = B * (B / 4) / 256;  // float4 per thread
        constexpr int HALF = PER >= 8 ? PER / 2 : PER;   // in flight at once (register budget)
        if (kw == B && width == B && a.sig_vec4) {
#pragma unroll
            for (int u0 = 0; u0 < PER; u0 += HALF) {
                f32x4 v[HALF];
#pragma unroll
                for (int u = 0; u < HALF; ++u) {
                    const int f = threadIdx.x + 256 * (u0 + u);
                    v[u] = *reinterpret_cast<const f32x4*>(a.Sigma + (j0 + f / (B / 4)) * a.p +
                                                           r0 + 4 * (f % (B / 4)));
                }
#pragma unroll
                for (int u = 0; u < HALF; ++u) {
                    const int f = threadIdx.x + 256 * (u0 + u);
                    *reinterpret_cast<f32x4*>(sT + (f / (B / 4)) * kTStride + 4 * (f % (B / 4))) =
                        v[u];
                }
            }
        } else {
            for (int e = threadIdx.x; e < B * B; e += blockDim.x) {
                const int cc = e / B, k = e % B;
                sT[cc * kTStride + k] =
                    (cc < width && k < kw) ? a.Sigma[(j0 + cc) * a.p + r0 + k] : 0.f;
            }
        }
        // A fragments: row i0 + r, k = 16 kg + 4h .. +3 (fetched after the Sigma
        // loads retire, to keep both sets from being live at once)
        f32x4 av[KG];
        const int64_t ia = i0 + r;
        const bool full = kw == B && i0 + 16 <= a.q;
#pragma unroll
        for (int kg = 0; kg < KG; ++kg) {
            const int kk = 16 * kg + 4 * h;
            if (full) {
                av[kg] = *reinterpret_cast<const f32x4*>(D + ia * a.S + k0 + kk);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    av[kg][u] = (ia < a.q && kk + u < kw) ? D[ia * a.S + k0 + kk + u] : 0.f;
            }
        }
        __syncthreads();
        f32x4 acc[T];
#pragma unroll
        for (int t = 0; t < T; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kg = 0; kg < KG; ++kg) {
#pragma unroll
            for (int t = 0; t < T; ++t) {
                const f32x4 bv = *reinterpret_cast<const f32x4*>(
                    sT + (CPW * wave + 16 * t + r) * kTStride + 16 * kg + 4 * h);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[kg][u], bv[u], acc[t], 0, 0, 0);
            }
        }
        __syncthreads();                         // sT consumed; reuse as the result tile
        float* sC = lds;                         // 16 x B
        // 16 x 16 output: lane holds rows 4 (lane / 16) + v, column lane % 16
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v) sC[(4 * h + v) * B + CPW * wave + 16 * t + r] = acc[t][v];
        __syncthreads();
#pragma unroll
        for (int m = 0; m < SLOTS; ++m) st.L[m] = fmaf(dscale, sC[lrow * B + 16 * m + g], st.L[m]);
    } else {
        float* sS = lds;            // B x B
        float* sD = lds + B * B;    // 16 x B
        __syncthreads();            // staging buffers free
        stage_sigma_block<SLOTS>(a.Sigma, a.p, r0, kw, j0, width, a.sig_vec4 != 0, sS);
        for (int e = threadIdx.x; e < 16 * B; e += blockDim.x) {
            const int rr = e / B, k = e % B;
            const int64_t ii = i0 + rr;
            sD[e] = (ii < a.q && k < kw) ? D[ii * a.S + k0 + k] : 0.f;
        }
        __syncthreads();
        for (int k = 0; k < kw; ++k) {
            const float dk = dscale * sD[lrow * B + k];
#pragma unroll
            for (int m = 0; m < SLOTS; ++m) st.L[m] = fmaf(dk, sS[k * B + g * SLOTS + m], st.L[m]);
        }
    }
}

// Look-ahead of a super-block: R_{I,SB(t)} += dscale_i D_{I,SB(t-1)} Sigma_{SB(t-1),SB(t)}
// for the workgroup's 16 rows I, before its panels start (D: the deltas of the
// previous super-block, q x S; dscale: the row's grid step when D holds code
// differences, else 1).  One 16 x 256 x 256 product on the fp32 matrix cores
// (v_mfma_f32_16x16x4f32; wave w owns output columns [64 w, 64 w + 64)), with
// Sigma's block staged through LDS in K chunks of 64 -- read as rows of the
// current super-block, the same numbers by symmetry, transposed so that k is
// contiguous -- and the next chunk (Sigma and the delta fragments) loaded into
// registers while the current chunk's matrix-core work runs.  The result is
// added to R in the panel's own lane layout (lane g of row lrow: columns
// 16 m + g), so that the panels' later loads of R are the same lanes' reads
// of their own writes.
constexpr int kLaK = 64;                  // K per staged chunk
constexpr int kLaStride = kLaK + 4;       // LDS row stride (floats) of a staged chunk
constexpr int kLaCols = 256;              // super-block columns covered
constexpr int kLaUStride = kLaCols + 4;   // LDS row stride of the 16 x 256 result

template <bool FULL>
__device__ __forceinline__ void la_fetch(const StepArgs& a, int64_t i0, int kc, f32x4 (&v)[16],
                                         f32x4 (&av)[4])
{
    const int lane = threadIdx.x & 63;
    const int r = lane & 15, h = lane >> 4;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int c = f >> 4, kq = f & 15;
        const int64_t base = (a.sb + c) * a.p + a.psb + kc + 4 * kq;
        if constexpr (FULL) {
            v[u] = *reinterpret_cast<const f32x4*>(a.Sigma + base);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[u][e] = (c < a.sbw && kc + 4 * kq + e < a.psbw) ? a.Sigma[base + e] : 0.f;
        }
    }
    const int64_t ia = i0 + r;
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
        const int k = kc + 16 * kg + 4 * h;
        if constexpr (FULL) {
            av[kg] = *reinterpret_cast<const f32x4*>(a.dprev + ia * a.S + k);
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e)
                av[kg][e] = (ia < a.q && k + e < a.psbw) ? a.dprev[ia * a.S + k + e] : 0.f;
        }
    }
}

template <bool FULL>
__device__ __forceinline__ void lookahead_k(const StepArgs& a, float* lds, int64_t i0,
                                            f32x4 (&acc)[4])
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, h = lane >> 4;
    f32x4 v[16], av[4], avn[4];
    la_fetch<FULL>(a, i0, 0, v, avn);
    for (int kc = 0; kc < a.psbw; kc += kLaK) {
        __syncthreads();                         // the previous chunk's reads are done
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const int f = threadIdx.x + 256 * u;
            *reinterpret_cast<f32x4*>(lds + (f >> 4) * kLaStride + 4 * (f & 15)) = v[u];
        }
#pragma unroll
        for (int kg = 0; kg < 4; ++kg) av[kg] = avn[kg];
        __syncthreads();
        if (kc + kLaK < a.psbw) la_fetch<FULL>(a, i0, kc + kLaK, v, avn);   // in flight below
#pragma unroll
        for (int kg = 0; kg < 4; ++kg)
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const f32x4 bv = *reinterpret_cast<const f32x4*>(
                    lds + (64 * wave + 16 * t + r) * kLaStride + 16 * kg + 4 * h);
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[kg][u], bv[u], acc[t], 0, 0, 0);
            }
    }
}

__device__ __forceinline__ void lookahead(const StepArgs& a, float* lds, int64_t i0, int lrow,
                                          int g, bool rowok, float dscale)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, h = lane >> 4;
    f32x4 acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (a.sig_vec4 && a.sbw == kLaCols && a.psbw % kLaK == 0 && i0 + 16 <= a.q)
        lookahead_k<true>(a, lds, i0, acc);
    else
        lookahead_k<false>(a, lds, i0, acc);
    __syncthreads();                             // the last chunk's reads are done
    float* sU = lds;                             // 16 x 256 result
    // 16 x 16 output: lane holds rows 4 (lane / 16) + v, column lane % 16
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int v = 0; v < 4; ++v) sU[(4 * h + v) * kLaUStride + 64 * wave + 16 * t + r] = acc[t][v];
    __syncthreads();
    if (!rowok) return;
    const int64_t i = i0 + lrow;
#pragma unroll
    for (int m = 0; m < kLaCols / 16; ++m) {
        const int c = 16 * m + g;
        if (c < a.sbw) {
            float* rp = a.R + i * a.p + a.sb + c;
            *rp = fmaf(dscale, sU[lrow * kLaUStride + c], *rp);
        }
    }
}

// The look-ahead when the workgroup's rows changed few codes in the previous
// super-block (code differences; each row at most kLaNz): the row's nonzero
// D_ik, listed in LDS through ballots over its 16 lanes, are applied to the
// lane's own columns of this super-block (c = 16 m + g, the layout of the
// dense look-ahead and of the panels' later R loads) as fp32 FMAs, kLaGroup
// of them per round of Sigma loads; rows without one are left as they are.
// cnt: the row's count.  Uses the first 16 * kLaNz int2 of LDS, wave-locally.
constexpr int kLaNz = 8;
constexpr int kLaGroup = 4;

__device__ __forceinline__ void lookahead_sparse(const StepArgs& a, float* lds, int64_t i0,
                                                 int lrow, int g, bool rowok, float dscale,
                                                 int cnt)
{
    const int lane = threadIdx.x & 63;
    int2* ent = reinterpret_cast<int2*>(lds) + lrow * kLaNz;
    const int64_t i = i0 + lrow;
    // the row's D over the previous super-block: lane g holds k = 64 w + 4 g + c
    float dv[4][4];
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int k = 64 * w + 4 * g + c;
            dv[w][c] = (cnt > 0 && k < a.psbw) ? a.dprev[i * a.S + k] : 0.f;
        }
    const int shift = 16 * (lane >> 4);
    const uint32_t below = (1u << g) - 1u;
    int base = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const bool on = dv[w][c] != 0.f;
            const uint32_t rb = (uint32_t)(__ballot(on) >> shift) & 0xffffu;
            if (on) {
                const int pos = base + __popc(rb & below);
                if (pos < kLaNz) ent[pos] = make_int2(64 * w + 4 * g + c, __float_as_int(dv[w][c]));
            }
            base += __popc(rb);
        }
    if (!rowok || cnt == 0) return;
    float acc[kLaCols / 16];
#pragma unroll
    for (int m = 0; m < kLaCols / 16; ++m) acc[m] = 0.f;
    for (int n0 = 0; n0 < cnt; n0 += kLaGroup) {
        float dn[kLaGroup], sv[kLaGroup][kLaCols / 16];
#pragma unroll
        for (int n = 0; n < kLaGroup; ++n) {
            dn[n] = 0.f;
#pragma unroll
            for (int m = 0; m < kLaCols / 16; ++m) sv[n][m] = 0.f;
            if (n0 + n >= cnt) continue;
            const int2 en = ent[n0 + n];
            dn[n] = __int_as_float(en.y);
            const float* srow = a.Sigma + (a.psb + en.x) * a.p + a.sb;
#pragma unroll
            for (int m = 0; m < kLaCols / 16; ++m)
                if (16 * m + g < a.sbw) sv[n][m] = srow[16 * m + g];
        }
#pragma unroll
        for (int n = 0; n < kLaGroup; ++n)
#pragma unroll
            for (int m = 0; m < kLaCols / 16; ++m) acc[m] = fmaf(dn[n], sv[n][m], acc[m]);
    }
#pragma unroll
    for (int m = 0; m < kLaCols / 16; ++m) {
        const int c = 16 * m + g;
        if (c < a.sbw) {
            float* rp = a.R + i * a.p + a.sb + c;
            *rp = fmaf(dscale, acc[m], *rp);
        }
    }
}

template <int SLOTS>
__device__ __forceinline__ void panel_role(const StepArgs& a, float* lds)
{
    constexpr int B = 16 * SLOTS;
    float* sS = lds;            // B x B: Sigma_{J,J} in the panel layout
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane & 15;
    const int lrow = wave * 4 + (lane >> 4);
    const int64_t i0 = (int64_t)blockIdx.x * 16;
    const int64_t i = i0 + lrow;
    const bool rowok = i < a.q;
    const int64_t p = a.p;
    const float s = rowok ? a.scale[i] : 1.f;
    const float z = rowok ? a.zero[i] : 0.f;
    const float inv_s = rowok ? a.inv_s[i] : 1.f;
    const int nsub = (int)cdiv(a.sbw, B);
    const float dscale = a.intd ? s : 1.f;
    float fl = 0.f;        // this lane's share of its row's objective change (launch)
    int nz = 0;            // this lane's nonzero code differences (launch)
    // (1) look-ahead: the previous super-block's deltas on this one's columns
    //     (written to R: this launch's GEMM leaves these columns out)
    if (a.psb >= 0) {
        if (a.intd && !a.dense) {
            const int cnt = rowok ? a.nzprev[i] : 0;
            if (__syncthreads_and(cnt <= kLaNz))
                lookahead_sparse(a, lds, i0, lrow, g, rowok, dscale, cnt);
            else
                lookahead(a, lds, i0, lrow, g, rowok, dscale);
        } else {
            lookahead(a, lds, i0, lrow, g, rowok, dscale);
        }
    }

    for (int sub = 0; sub < nsub; ++sub) {
        const int64_t j0 = a.sb + (int64_t)sub * B;
        const int width = (int)min((int64_t)B, a.sb + a.sbw - j0);
        PanelState<SLOTS> st;
        st.fl = 0.f;
        const bool cvalid = a.codes_valid != 0;
#pragma unroll
        for (int m = 0; m < SLOTS; ++m) {
            const int c = 16 * m + g;
            const bool ok = rowok && c < width;
            const int64_t idx = i * p + j0 + c;
            st.L[m] = ok ? a.R[idx] : 0.f;
            st.w[m] = ok ? a.Wh[idx] : 0.f;
            const float invd = c < width ? a.inv_d[j0 + c] : 0.f;
            if (a.relax) {
                st.u[m] = invd;
                st.v[m] = 0.f;
            } else {
                st.u[m] = invd * inv_s;
                st.v[m] = fmaf(st.w[m], inv_s, z);
                // the current code is recovered exactly from What (|k - z| <= 255
                // keeps the rounding error far below 1/2)
                st.k[m] = cvalid ? rintf(st.v[m]) : __builtin_nanf("");
                // with code differences t is taken from the code itself: What's
                // exact level s (k - z) over s, plus z, is k
                if (a.intd) st.v[m] = st.k[m];
            }
        }
        // (2) earlier blocks of this super-block (this workgroup's own rows; not
        //     written to R: the next launch's GEMM applies the whole super-block)
        for (int sp = 0; sp < sub; ++sp)
            add_block_update<SLOTS>(st, a, a.dcur, (int64_t)sp * B, B, a.sb + (int64_t)sp * B, j0,
                                    width, i0, lrow, g, lds, dscale);
        // (3) the B column updates in order
        __syncthreads();
        stage_sigma_block<SLOTS>(a.Sigma, p, j0, width, j0, width, a.sig_vec4 != 0, sS);
        __syncthreads();
        constexpr auto cols = std::make_integer_sequence<int, B>{};
        if (a.relax)
            panel_run<SLOTS, false, true, false>(cols, st, sS, g, width, s, z, a.maxq);
        else if (a.intd && width == B)
            panel_run<SLOTS, true, false, true>(cols, st, sS, g, width, s, z, a.maxq);
        else if (a.intd)
            panel_run<SLOTS, false, false, true>(cols, st, sS, g, width, s, z, a.maxq);
        else if (width == B)
            panel_run<SLOTS, true, false, false>(cols, st, sS, g, width, s, z, a.maxq);
        else
            panel_run<SLOTS, false, false, false>(cols, st, sS, g, width, s, z, a.maxq);
#pragma unroll
        for (int m = 0; m < SLOTS; ++m) {
            const int c = 16 * m + g;
            float d;
            if (a.relax) {
                d = st.v[m];
                if (rowok && c < width) a.Wh[i * p + j0 + c] = st.w[m];
            } else {
                // the same delta the column's step broadcast (as a code
                // difference: the GEMM and the look-ahead scale it by s)
                if (a.intd)
                    d = c < width ? st.k[m] - st.v[m] : 0.f;
                else
                    d = c < width ? fmaf(s, st.k[m] - z, -st.w[m]) : 0.f;
                if (rowok && c < width) {
                    a.Wh[i * p + j0 + c] = s * (st.k[m] - z);
                    a.codes[i * p + j0 + c] = (uint8_t)st.k[m];
                }
            }
            if (rowok) a.dcur[i * a.S + (int64_t)sub * B + c] = d;
            nz += d != 0.f;
        }
        fl += st.fl;
        if (a.intd && sub == nsub - 1) {
            // the row's count over its 16 lanes, for the next launch's block update
#pragma unroll
            for (int o = 8; o > 0; o >>= 1) nz += __shfl_xor(nz, o, 16);
            if (g == 0 && rowok) a.nzcur[i] = nz;
        }
        // This block's deltas are read back only by this workgroup (its next
        // blocks), after the __syncthreads() that opens add_block_update: a
        // workgroup-scope release/acquire.  A device-scope fence here would
        // write back and invalidate L2 under the concurrent GEMM tiles.
    }
    if (a.fobj) {
        // one fp64 partial per wave (4 rows), added to across the sweep's
        // launches in stream order: a fixed summation order, no atomics
        double fsum = rowok ? (double)(fl * dscale) : 0.0;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) fsum += __shfl_xor(fsum, o, 64);
        if (lane == 0) {
            double* slot = a.fpart + (((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6);
            *slot = a.ffirst ? fsum : *slot + fsum;
        }
    }
}

// R's tile is read only after the K loop (through an LDS-staged, float4-wide
// read-modify-write): holding it across the loop would cost 64 registers and
// the second workgroup per CU, which matters more than hiding its latency.
// A tile takes the sparse path when at most kSparseRows of its rows changed a
// code in the previous super-block, none of them more than kSparseRowNz
// codes.  A wave takes its rows kSpPass at a time, with the loads of each
// phase of those rows in flight together: two memory round trips per pass,
// plus one per further kSpGroup nonzeros of its busiest row (a dense tile
// costs a whole K loop).
constexpr int kSparseRows = 64;
constexpr int kSparseRowNz = 32;
constexpr int kSpPass = 8;
constexpr int kSpGroup = 4;

// Block update of a tile whose rows hold few nonzero code differences (late
// sweeps, where most codes are kept and their differences are exact zeros):
// R_ic += s_i sum_k D_ik Sigma_kc over the nonzero D_ik only, in increasing
// k, as fp32 FMAs.  Rows without a nonzero difference are left as they are
// (their update is 0).  The active rows are listed in LDS with their counts;
// wave w takes list entries w, w + 4, ..., lane l holding columns 2l and
// 2l + 1.  Per pass of kSpPass rows: the D rows (lane l: k = l + 64 e) and R
// segments are loaded; each row's nonzeros are written, in k order, to the
// wave's LDS area (positions from the ballots); then all their Sigma
// segments are loaded, then R is updated.  nz: this thread's row count
// (threads < 128).
__device__ __forceinline__ void gemm_sparse(const StepArgs& a, int* li, int nz, int active,
                                            int64_t row0, int64_t col0, int64_t ex0, int64_t ex1)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int* cnt = li;                                   // 2: active rows among tile rows 0-63, 64-127
    int* list = li + 2;                              // kSparseRows tile row offsets, ascending
    int* lcount = list + kSparseRows;                // their counts
    int2* ent = reinterpret_cast<int2*>(lcount + kSparseRows) +
                wave * kSpPass * kSparseRowNz;       // this wave's (k, d) entries
    uint64_t b = 0;
    if (wave < 2) {
        b = __ballot(nz > 0);
        if (lane == 0) cnt[wave] = __popcll(b);
    }
    __syncthreads();
    if (wave < 2 && nz > 0) {
        const int j = (wave == 1 ? cnt[0] : 0) + (int)__popcll(b & ((1ull << lane) - 1ull));
        list[j] = (int)threadIdx.x;
        lcount[j] = nz;
    }
    __syncthreads();

    const uint64_t below = (1ull << lane) - 1ull;
    const int64_t c0 = col0 + 2 * lane;
    const bool ok0 = c0 < a.p && !(c0 >= ex0 && c0 < ex1);
    const bool ok1 = c0 + 1 < a.p && !(c0 + 1 >= ex0 && c0 + 1 < ex1);
    const bool pair = a.sig_vec4 && a.r_vec4 && c0 + 1 < a.p;   // 8-byte aligned pairs
    for (int j0 = wave; j0 < active; j0 += 4 * kSpPass) {
        int64_t ir[kSpPass];
        int cn[kSpPass];
        float dv[kSpPass][4], r0v[kSpPass], r1v[kSpPass];
#pragma unroll
        for (int u = 0; u < kSpPass; ++u) {
            const int j = j0 + 4 * u;
            ir[u] = j < active ? row0 + list[j] : -1;    // uniform
            cn[u] = j < active ? lcount[j] : 0;
            r0v[u] = r1v[u] = 0.f;
#pragma unroll
            for (int e = 0; e < 4; ++e) dv[u][e] = 0.f;
            if (ir[u] < 0) continue;
            const float* drow = a.dprev + ir[u] * a.S;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k = lane + 64 * e;
                if (k < a.psbw) dv[u][e] = drow[k];
            }
            const float* rrow = a.R + ir[u] * a.p;
            if (pair) {
                const f32x2 v = *reinterpret_cast<const f32x2*>(rrow + c0);
                r0v[u] = v[0];
                r1v[u] = v[1];
            } else {
                if (c0 < a.p) r0v[u] = rrow[c0];
                if (c0 + 1 < a.p) r1v[u] = rrow[c0 + 1];
            }
        }
        // each row's nonzeros, in increasing k, to the wave's LDS area
#pragma unroll
        for (int u = 0; u < kSpPass; ++u) {
            if (ir[u] < 0) continue;
            int base = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool on = dv[u][e] != 0.f;
                const uint64_t m = __ballot(on);
                if (on)
                    ent[u * kSparseRowNz + base + (int)__popcll(m & below)] =
                        make_int2(lane + 64 * e, __float_as_int(dv[u][e]));
                base += (int)__popcll(m);
            }
        }
        // Sigma segments of kSpGroup nonzeros per row at a time, all rows at once
        int cmax = 0;
#pragma unroll
        for (int u = 0; u < kSpPass; ++u) cmax = max(cmax, cn[u]);
        float acc0[kSpPass], acc1[kSpPass];
#pragma unroll
        for (int u = 0; u < kSpPass; ++u) acc0[u] = acc1[u] = 0.f;
        for (int n0 = 0; n0 < cmax; n0 += kSpGroup) {
            float dn[kSpPass][kSpGroup], s0[kSpPass][kSpGroup], s1[kSpPass][kSpGroup];
#pragma unroll
            for (int u = 0; u < kSpPass; ++u)
#pragma unroll
                for (int n = 0; n < kSpGroup; ++n) {
                    dn[u][n] = s0[u][n] = s1[u][n] = 0.f;
                    if (n0 + n >= cn[u]) continue;       // uniform
                    const int2 en = ent[u * kSparseRowNz + n0 + n];
                    dn[u][n] = __int_as_float(en.y);
                    const float* srow = a.Sigma + (a.psb + en.x) * a.p;
                    if (pair) {
                        const f32x2 sv = *reinterpret_cast<const f32x2*>(srow + c0);
                        s0[u][n] = sv[0];
                        s1[u][n] = sv[1];
                    } else {
                        if (c0 < a.p) s0[u][n] = srow[c0];
                        if (c0 + 1 < a.p) s1[u][n] = srow[c0 + 1];
                    }
                }
#pragma unroll
            for (int u = 0; u < kSpPass; ++u)
#pragma unroll
                for (int n = 0; n < kSpGroup; ++n) {
                    acc0[u] = fmaf(dn[u][n], s0[u][n], acc0[u]);
                    acc1[u] = fmaf(dn[u][n], s1[u][n], acc1[u]);
                }
        }
#pragma unroll
        for (int u = 0; u < kSpPass; ++u) {
            if (ir[u] < 0) continue;
            const float si = a.scale[ir[u]];
            float* rrow = a.R + ir[u] * a.p;
            if (ok0) rrow[c0] = fmaf(si, acc0[u], r0v[u]);
            if (ok1) rrow[c0 + 1] = fmaf(si, acc1[u], r1v[u]);
        }
    }
}

__device__ __forceinline__ void gemm_role(const StepArgs& a, float* lds, int64_t t)
{
    const int64_t tm = t / a.tiles_n, tn = t % a.tiles_n;
    const int64_t row0 = tm * kTile, col0 = tn * kTile;
    const int64_t ex0 = a.sb >= 0 ? a.sb : 0, ex1 = a.sb >= 0 ? a.sb + a.sbw : 0;
    if (a.sb >= 0 && col0 >= ex0 && min(col0 + kTile, a.p) <= ex1) return;   // all excluded
    if (a.intd && !a.dense) {
        // rows of the tile that changed a code in the previous super-block
        int nz = 0;
        if (threadIdx.x < kTile && row0 + threadIdx.x < a.q) nz = a.nzprev[row0 + threadIdx.x];
        const int active = __syncthreads_count(nz > 0);
        const int heavy = __syncthreads_count(nz > kSparseRowNz);
        if (active <= kSparseRows && heavy == 0) {
            gemm_sparse(a, reinterpret_cast<int*>(lds), nz, active, row0, col0, ex0, ex1);
            return;
        }
    }
    f32x16 acc[2][2];
    zero_acc(acc);
    if (a.fp32) {
        const RowOp A{a.dprev, a.S, a.q, a.psbw, true};
        const RowOp Bo{a.Sigma + a.psb, a.p, a.p, a.psbw, a.sig_vec4 != 0};
        nt_tile(A, row0, Bo, col0, a.psbw, lds, acc);
    } else {
        // split bf16 products (nt_x3.h); Delta rows are 16-byte aligned (stride S)
        const XRowQ<256, 3> Bo{a.Sigma + a.psb, a.p, a.p, a.psbw};
        uint32_t* l32 = reinterpret_cast<uint32_t*>(lds);
        const bool full =
            a.sig_vec4 && row0 + kTile <= a.q && col0 + kTile <= a.p && a.psbw % (2 * kX3KC) == 0;
        if (a.intd) {
            // code differences are exact in bf16: three exact products with Sigma's planes
            const XRowQ<256, 1> A{a.dprev, a.S, a.q, a.psbw};
            if (full)
                nt_tile_x3_full<true, 3>(A, row0, Bo, col0, a.psbw, l32, acc);
            else
                nt_tile_x3_edge<3>(A, row0, Bo, col0, a.psbw, l32, acc);
        } else {
            const XRowQ<256, 3> A{a.dprev, a.S, a.q, a.psbw};
            if (full)
                nt_tile_x3_full(A, row0, Bo, col0, a.psbw, l32, acc);
            else
                nt_tile_x3_edge(A, row0, Bo, col0, a.psbw, l32, acc);
        }
    }
    // R's tile is fetched before the accumulators pass through LDS, which
    // hides part of its latency
    TileRM rv;
    tile_load_rm(a.R, a.p, a.q, a.p, row0, col0, a.r_vec4 != 0, rv);
    acc_to_lds(acc, lds);                                // the K loop ended with a barrier
    __syncthreads();
    // code differences: R += s_i (D Sigma)_i
    tile_add_store_rm(a.R, a.p, a.q, a.p, row0, col0, a.r_vec4 != 0, rv, lds, ex0, ex1,
                      a.intd ? a.scale : nullptr);
}

template <int SLOTS>
constexpr int step_lds_floats()
{
    return (16 * SLOTS) * (16 * SLOTS) + 16 * (16 * SLOTS) > kNTLdsFloats
               ? (16 * SLOTS) * (16 * SLOTS) + 16 * (16 * SLOTS)
               : kNTLdsFloats;
}

template <int SLOTS>
__global__ __launch_bounds__(256, 2) void cd_step_kernel(StepArgs a)
{
    if (failed(a.status)) return;
    static_assert(step_lds_floats<SLOTS>() >= kLaCols * kLaStride, "look-ahead staging fits");
    __shared__ __attribute__((aligned(16))) float lds[step_lds_floats<SLOTS>()];
    if ((int)blockIdx.x < a.n_panel)
        panel_role<SLOTS>(a, lds);
    else
        gemm_role(a, lds, (int64_t)blockIdx.x - a.n_panel);
}

// ---------------------------------------------------------------- host side
static int block_width(int block) { return block == 0 ? 128 : block; }

// Super-block width = the GEMM's K per launch (a multiple of the panel width).
static int super_width(int B) { return B >= 256 ? B : 256; }

size_t cd_ws_bytes(int64_t q, int64_t p, int block)
{
    const int S = super_width(block_width(block));
    size_t b = kStatusBytes;
    b += align256(sizeof(float) * p);               // inv_d
    b += align256(sizeof(float) * q);               // inv_s
    b += 2 * align256(sizeof(float) * q * S);       // delta double buffer
    b += 2 * align256(sizeof(int) * q);             // nonzero-difference counts, double buffer
    b += align256(sizeof(double) * kObjBlocks);     // objective partials
    b += align256(sizeof(double) * 4 * cdiv(q, 16)); // per panel wave: objective change
    b += align256(sizeof(double));                  // objective of the incoming state
    return b;
}

// <What + H - W, R> into *out (fp64, deterministic); `part` holds kObjBlocks doubles.
qe_status launch_residual_dot(const float* W, const float* Wh, const float* H, const float* R,
                              int64_t count, double* out, double* part, const int* status,
                              hipStream_t s)
{
    const int vec4 = aligned16(W) && aligned16(Wh) && aligned16(R) && (!H || aligned16(H));
    hipLaunchKernelGGL(obj_partial_kernel, dim3(kObjBlocks), dim3(256), 0, s, W, Wh, H, R, count,
                       vec4, part, status);
    hipLaunchKernelGGL(sum_partials_kernel, dim3(1), dim3(256), 0, s, part, kObjBlocks,
                       (const double*)nullptr, out, status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

template <int SLOTS>
static qe_status launch_steps(StepArgs base, float* d0, float* d1, int* nz0, int* nz1,
                              int64_t q, int64_t p, hipStream_t s)
{
    const int S = base.S;
    const int64_t nsb = cdiv(p, S);
    const int64_t panel_wgs = cdiv(q, 16);
    const int64_t tiles_m = cdiv(q, kTile), tiles_n = cdiv(p, kTile);
    for (int64_t t = 0; t <= nsb; ++t) {
        StepArgs a = base;
        a.sb = t < nsb ? t * S : -1;
        a.sbw = t < nsb ? (int)std::min<int64_t>(S, p - t * S) : 0;
        a.psb = t > 0 ? (t - 1) * S : -1;
        a.psbw = t > 0 ? (int)std::min<int64_t>(S, p - (t - 1) * S) : 0;
        a.ffirst = t == 0;
        a.dcur = (t & 1) ? d1 : d0;
        a.dprev = (t & 1) ? d0 : d1;
        a.nzcur = (t & 1) ? nz1 : nz0;
        a.nzprev = (t & 1) ? nz0 : nz1;
        a.n_panel = t < nsb ? (int)panel_wgs : 0;
        a.tiles_n = tiles_n;
        const int64_t gemm_wgs = t > 0 ? tiles_m * tiles_n : 0;
        const int64_t grid = a.n_panel + gemm_wgs;
        hipLaunchKernelGGL(cd_step_kernel<SLOTS>, dim3((unsigned)grid), dim3(256), 0, s, a);
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    return QE_OK;
}

qe_status launch_cd(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                    const float* scale, const float* zero, float* Wh, uint8_t* codes, float* R,
                    const float* H, int sweeps, int block, uint32_t flags, double* obj,
                    int obj_stride, const double* f_in, void* ws, hipStream_t s)
{
    const int B = block_width(block);
    const int S = super_width(B);
    int* status = static_cast<int*>(ws);
    Ws w(ws);
    float* inv_d = w.take<float>(p);
    float* inv_s = w.take<float>(q);
    float* d0 = w.take<float>((size_t)q * S);
    float* d1 = w.take<float>((size_t)q * S);
    int* nz0 = w.take<int>(q);
    int* nz1 = w.take<int>(q);
    double* part = w.take<double>(kObjBlocks);
    const int n_fpart = (int)(4 * cdiv(q, 16));
    double* fpart = w.take<double>(n_fpart);
    double* fstart = w.take<double>(1);

    if (flags & QE_DEBUG_CHECKS) {
        // every input of the call (the footnote to Lemma 1: checks before the sweeps)
        const float* inputs[6] = {W, Sigma, scale, zero,
                                  (flags & QE_INIT_FROM_W) ? nullptr : Wh,
                                  (flags & QE_R_VALID) ? R : nullptr};
        const int64_t counts[6] = {q * p, p * p, q, q, q * p, q * p};
        for (int k = 0; k < 6; ++k)
            if (launch_nonfinite_scan(inputs[k], counts[k], status, s) != QE_OK) return QE_ERR_HIP;
        if (launch_nonfinite_scan(H, q * p, status, s) != QE_OK) return QE_ERR_HIP;
    }
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
                           Sigma, q, p, R, vec4 ? 1 : 0, (flags & QE_CD_FP32) ? 1 : 0, status);
    }
    if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    // The per-sweep objective is the incoming one plus the exact change of
    // the sweep's coordinate moves, which the panel sums as it goes.  The
    // incoming value: given (f_in), 0 after QE_INIT_FROM_W (What [+ H] = W),
    // else one pass over R.
    const double* f_prev = f_in;
    if (obj && !f_in && !(flags & QE_INIT_FROM_W)) {
        const qe_status st = launch_residual_dot(W, Wh, H, R, q * p, fstart, part, status, s);
        if (st != QE_OK) return st;
        f_prev = fstart;
    }

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
    base.S = S;
    base.maxq = (float)((1 << bits) - 1);
    base.sig_vec4 = (aligned16(Sigma) && p % 4 == 0) ? 1 : 0;
    base.r_vec4 = (aligned16(R) && p % 4 == 0) ? 1 : 0;
    base.fp32 = (flags & QE_CD_FP32) ? 1 : 0;
    base.dense = (flags & QE_CD_DENSE) ? 1 : 0;
    base.fpart = fpart;
    base.fobj = obj ? 1 : 0;
    base.status = status;
    const bool codes_valid0 = (flags & QE_CODES_VALID) && !(flags & QE_INIT_FROM_W);
    const int period = (int)((flags & QE_RELAX_MASK) >> 8);
    bool prev_relaxed = false;
    for (int sw = 0; sw < sweeps; ++sw) {
        const int k = sw + 1;
        base.relax = (period > 0 && k % period == 0 && k != sweeps) ? 1 : 0;
        base.codes_valid = ((sw > 0 || codes_valid0) && !prev_relaxed) ? 1 : 0;
        // A quantized sweep that starts with every What_ij on its grid level
        // moves coordinates only between levels: delta = s_i (k_new - k_old).
        // The deltas are then handed on as the code differences (exact small
        // integers, a single bf16 plane) and the row's s_i is applied after
        // the product: R += s_i (D Sigma).  R then follows the exact levels
        // s (k - z) rather than their fp32 roundings.
        base.intd = (base.codes_valid && !base.relax) ? 1 : 0;
        prev_relaxed = base.relax != 0;
        qe_status st;
        switch (B) {
            case 16: st = launch_steps<1>(base, d0, d1, nz0, nz1, q, p, s); break;
            case 32: st = launch_steps<2>(base, d0, d1, nz0, nz1, q, p, s); break;
            case 64: st = launch_steps<4>(base, d0, d1, nz0, nz1, q, p, s); break;
            default: st = launch_steps<8>(base, d0, d1, nz0, nz1, q, p, s); break;
        }
        if (st != QE_OK) return st;
        if (obj) {
            double* out = obj + (size_t)sw * obj_stride;
            hipLaunchKernelGGL(sum_partials_kernel, dim3(1), dim3(256), 0, s, fpart, n_fpart,
                               f_prev, out, status);
            if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
            f_prev = out;
        }
    }
    return QE_OK;
}

}  // namespace qe
