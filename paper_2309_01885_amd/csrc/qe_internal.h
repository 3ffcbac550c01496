// Internal declarations of libqe (gfx950 / CDNA4).  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "qe.h"

namespace qe {

// ---------------------------------------------------------------- constants
constexpr int kTile = 128;            // square output tile of the NT matrix-core kernels
constexpr int kKC = 32;               // K chunk staged through LDS per pipeline stage
constexpr int kLdsStride = kKC + 4;   // padded LDS row (floats)
constexpr size_t kStatusBytes = 256;  // status word region at the head of every workspace
constexpr int kNTLdsFloats = 2 * 2 * kTile * kLdsStride;  // double-buffered A and B chunks
constexpr int kObjBlocks = 1024;      // workgroups of the fp64 residual dot product

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Device status word (first int of every workspace).  Set with a vector
// atomic; read at kernel entry so that later kernels of a failed call are no-ops.
__device__ inline void set_status(int* status, int code) { atomicCAS(status, 0, code); }
__device__ inline bool failed(const int* status) { return *status != 0; }

// ---------------------------------------------------------------- NT tile GEMM
// C[128 x 128] (+)= A[128 x K] * B[128 x K]^T on fp32 matrix cores.
// An operand supplies element (r, k) of a 128 x 32 chunk; out-of-range
// elements read as 0.  Four waves in a 2 x 2 arrangement; each wave owns a
// 64 x 64 quarter as 2 x 2 tiles of v_mfma_f32_32x32x2f32.
//
// K permutation: the sum over k is order-free, so inside each group of 8 the
// lane half h = lane / 32 covers k = 8t + 4h + u for MFMA step u = 0..3.  A and
// B use the same map, so every lane fetches its 4 k-values as one 16-byte
// LDS read.

// Staging registers for one 128 x 32 chunk of one operand (256 threads x 4 float4).
struct Stage { f32x4 v[4]; };

// Stores a chunk staged in the k-contiguous order (thread t holds rows
// t/8 + 32m, k = 4 (t % 8) .. +3).
__device__ inline void store_rowmajor(float* lds, const Stage& st)
{
    const int t = threadIdx.x;
    const int kq = (t & 7) * 4;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int r = (t >> 3) + 32 * m;
        *reinterpret_cast<f32x4*>(lds + r * kLdsStride + kq) = st.v[m];
    }
}

// Row-major operand: element (r, k) at base[r * ld + k].
// Chunks fully inside the matrix take a branch-free path (the test is uniform
// across the workgroup); edge chunks fall back to guarded element loads.
struct RowOp {
    const float* base;
    int64_t ld, rows, kvalid;
    bool vec4;   // base and ld allow aligned 16-byte loads
    __device__ inline void load(int64_t row0, int64_t k0, Stage& st) const
    {
        const int t = threadIdx.x;
        const int kq = (t & 7) * 4;
        if (vec4 && row0 + kTile <= rows && k0 + kKC <= kvalid) {
            const float* src = base + (row0 + (t >> 3)) * ld + k0 + kq;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                st.v[m] = *reinterpret_cast<const f32x4*>(src + (int64_t)(32 * m) * ld);
            return;
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t gr = row0 + (t >> 3) + 32 * m;
            const int64_t gk = k0 + kq;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (gr < rows) {
                const float* src = base + gr * ld + gk;
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (gk + u < kvalid) v[u] = src[u];
            }
            st.v[m] = v;
        }
    }
    __device__ inline void store(float* lds, const Stage& st) const { store_rowmajor(lds, st); }
};

// Row-major composite operand P1 + P2 - P3 (P2, P3 may be null), e.g. What + H - W.
struct CompOp {
    const float *p1, *p2, *p3;
    int64_t ld, rows, kvalid;
    bool vec4;
    __device__ inline void load(int64_t row0, int64_t k0, Stage& st) const
    {
        const int t = threadIdx.x;
        const int kq = (t & 7) * 4;
        if (vec4 && row0 + kTile <= rows && k0 + kKC <= kvalid) {
            const int64_t off0 = (row0 + (t >> 3)) * ld + k0 + kq;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int64_t off = off0 + (int64_t)(32 * m) * ld;
                f32x4 v = *reinterpret_cast<const f32x4*>(p1 + off);
                if (p2) v = v + *reinterpret_cast<const f32x4*>(p2 + off);
                if (p3) v = v - *reinterpret_cast<const f32x4*>(p3 + off);
                st.v[m] = v;
            }
            return;
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t gr = row0 + (t >> 3) + 32 * m;
            const int64_t gk = k0 + kq;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (gr < rows) {
                const int64_t off = gr * ld + gk;
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (gk + u < kvalid) {
                        float x = p1[off + u];
                        if (p2) x = x + p2[off + u];
                        if (p3) x = x - p3[off + u];
                        v[u] = x;
                    }
            }
            st.v[m] = v;
        }
    }
    __device__ inline void store(float* lds, const Stage& st) const { store_rowmajor(lds, st); }
};

// Transposed operand: element (r, k) at base[k * ld + r] (token-major X).
// Each thread fetches 4 consecutive rows of one k and scatters them into the
// k-contiguous LDS layout.
struct ColOp {
    const float* base;
    int64_t ld, rows, kvalid;
    bool vec4;
    __device__ inline void load(int64_t row0, int64_t k0, Stage& st) const
    {
        const int t = threadIdx.x;
        const int rq = (t & 31) * 4;
        if (vec4 && row0 + kTile <= rows && k0 + kKC <= kvalid) {
            const float* src = base + (k0 + (t >> 5)) * ld + row0 + rq;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                st.v[m] = *reinterpret_cast<const f32x4*>(src + (int64_t)(8 * m) * ld);
            return;
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int64_t gk = k0 + (t >> 5) + 8 * m;
            const int64_t gr = row0 + rq;
            f32x4 v = {0.f, 0.f, 0.f, 0.f};
            if (gk < kvalid) {
                const float* src = base + gk * ld + gr;
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (gr + u < rows) v[u] = src[u];
            }
            st.v[m] = v;
        }
    }
    __device__ inline void store(float* lds, const Stage& st) const
    {
        const int t = threadIdx.x;
        const int rq = (t & 31) * 4;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int kk = (t >> 5) + 8 * m;
#pragma unroll
            for (int u = 0; u < 4; ++u) lds[(rq + u) * kLdsStride + kk] = st.v[m][u];
        }
    }
};

// acc[mi][ni] += A(wave rows mi) * B(wave cols ni)^T over one staged chunk.
__device__ inline void mfma_chunk(const float* ldsA, const float* ldsB, f32x16 (&acc)[2][2])
{
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int r = lane & 31, h = lane >> 5;
#pragma unroll
    for (int t = 0; t < kKC / 8; ++t) {
        const int ko = 8 * t + 4 * h;
        f32x4 a0 = *reinterpret_cast<const f32x4*>(ldsA + (wm * 64 + r) * kLdsStride + ko);
        f32x4 a1 = *reinterpret_cast<const f32x4*>(ldsA + (wm * 64 + 32 + r) * kLdsStride + ko);
        f32x4 b0 = *reinterpret_cast<const f32x4*>(ldsB + (wn * 64 + r) * kLdsStride + ko);
        f32x4 b1 = *reinterpret_cast<const f32x4*>(ldsB + (wn * 64 + 32 + r) * kLdsStride + ko);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[u], b0[u], acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[u], b1[u], acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[u], b0[u], acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[u], b1[u], acc[1][1], 0, 0, 0);
        }
    }
}

// Row / column (within the 128 x 128 tile) of accumulator element v of
// sub-tile (mi, ni) held by this lane: the 32 x 32 output of
// v_mfma_f32_32x32x2f32 puts column lane % 32 in every lane and rows
// 8 * (v / 4) + 4 * (lane / 32) + v % 4.
__device__ inline int acc_row(int mi, int v)
{
    const int lane = threadIdx.x & 63;
    const int wm = (threadIdx.x >> 6) >> 1;
    return wm * 64 + mi * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}
__device__ inline int acc_col(int ni)
{
    const int lane = threadIdx.x & 63;
    const int wn = (threadIdx.x >> 6) & 1;
    return wn * 64 + ni * 32 + (lane & 31);
}

// Loads the 128 x 128 tile at (row0, col0) of a row-major matrix (ld floats
// per row) in accumulator layout; elements outside rows x cols read as 0.
__device__ inline void tile_load(const float* M, int64_t ld, int64_t rows, int64_t cols,
                                 int64_t row0, int64_t col0, f32x16 (&v)[2][2])
{
    if (row0 + kTile <= rows && col0 + kTile <= cols) {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    v[mi][ni][e] = M[(row0 + acc_row(mi, e)) * ld + col0 + acc_col(ni)];
        return;
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t r = row0 + acc_row(mi, e), c = col0 + acc_col(ni);
                v[mi][ni][e] = (r < rows && c < cols) ? M[r * ld + c] : 0.f;
            }
}

// Stores v to the tile at (row0, col0), skipping elements outside rows x cols
// and columns in [ex0, ex1).
__device__ inline void tile_store(float* M, int64_t ld, int64_t rows, int64_t cols, int64_t row0,
                                  int64_t col0, const f32x16 (&v)[2][2], int64_t ex0 = 0,
                                  int64_t ex1 = 0)
{
    if (row0 + kTile <= rows && col0 + kTile <= cols && (ex1 <= col0 || ex0 >= col0 + kTile)) {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    M[(row0 + acc_row(mi, e)) * ld + col0 + acc_col(ni)] = v[mi][ni][e];
        return;
    }
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t r = row0 + acc_row(mi, e), c = col0 + acc_col(ni);
                if (r < rows && c < cols && !(c >= ex0 && c < ex1)) M[r * ld + c] = v[mi][ni][e];
            }
}

// Row-major view of a 128 x 128 tile for a 256-thread workgroup: thread t owns
// the float4 at row (t >> 5) + 8 j, columns 4 (t & 31) .. +3, for j = 0..15.
// One base address per thread keeps a prefetched tile cheap in registers.
struct TileRM { f32x4 v[16]; };

__device__ inline void tile_load_rm(const float* M, int64_t ld, int64_t rows, int64_t cols,
                                    int64_t row0, int64_t col0, bool vec4, TileRM& T)
{
    const int t = threadIdx.x;
    const int64_t r0 = row0 + (t >> 5), c0 = col0 + 4 * (t & 31);
    if (vec4 && row0 + kTile <= rows && col0 + kTile <= cols) {
        const float* base = M + r0 * ld + c0;
#pragma unroll
        for (int j = 0; j < 16; ++j) T.v[j] = *reinterpret_cast<const f32x4*>(base + 8 * j * ld);
        return;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int64_t r = r0 + 8 * j;
#pragma unroll
        for (int u = 0; u < 4; ++u) T.v[j][u] = (r < rows && c0 + u < cols) ? M[r * ld + c0 + u] : 0.f;
    }
}

// Writes T + (the accumulator tile staged in LDS by acc_to_lds) to M, skipping
// elements outside rows x cols and columns in [ex0, ex1).  rowscale (nullable,
// indexed by M's row) multiplies each accumulator row first, in one fused
// multiply-add; without it the sum is T + acc.
constexpr int kAccStride = kTile + 4;
__device__ inline void tile_add_store_rm(float* M, int64_t ld, int64_t rows, int64_t cols,
                                         int64_t row0, int64_t col0, bool vec4, const TileRM& T,
                                         const float* accLds, int64_t ex0 = 0, int64_t ex1 = 0,
                                         const float* rowscale = nullptr)
{
    const int t = threadIdx.x;
    const int lr = t >> 5, lc = 4 * (t & 31);
    const int64_t r0 = row0 + lr, c0 = col0 + lc;
    if (vec4 && row0 + kTile <= rows && col0 + kTile <= cols &&
        (ex1 <= col0 || ex0 >= col0 + kTile)) {
        float* base = M + r0 * ld + c0;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const f32x4 a = *reinterpret_cast<const f32x4*>(accLds + (lr + 8 * j) * kAccStride + lc);
            if (rowscale) {
                const float sc = rowscale[r0 + 8 * j];
                f32x4 o;
#pragma unroll
                for (int u = 0; u < 4; ++u) o[u] = fmaf(sc, a[u], T.v[j][u]);
                *reinterpret_cast<f32x4*>(base + 8 * j * ld) = o;
            } else {
                *reinterpret_cast<f32x4*>(base + 8 * j * ld) = T.v[j] + a;
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        const int64_t r = r0 + 8 * j;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int64_t c = c0 + u;
            if (r < rows && c < cols && !(c >= ex0 && c < ex1)) {
                const float a = accLds[(lr + 8 * j) * kAccStride + lc + u];
                M[r * ld + c] = rowscale ? fmaf(rowscale[r], a, T.v[j][u]) : T.v[j][u] + a;
            }
        }
    }
}

// Stages the accumulators into LDS as a row-major 128 x 128 tile (row stride
// kAccStride); needs kTile * kAccStride floats.  Caller synchronises after.
__device__ inline void acc_to_lds(const f32x16 (&acc)[2][2], float* lds)
{
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int e = 0; e < 16; ++e) lds[acc_row(mi, e) * kAccStride + acc_col(ni)] = acc[mi][ni][e];
}

// Double-buffered K loop: acc += A[row0a.., 0..K) * B[row0b.., 0..K)^T.
// `lds` must hold kNTLdsFloats floats.  Ends with a barrier.  The loop is
// unrolled by two so that both buffer addresses are compile-time offsets of
// the LDS array (a runtime-selected buffer pointer degrades to flat accesses,
// which wait on the outstanding global prefetch).
template <class OA, class OB>
__device__ inline void nt_tile(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                               int64_t K, float* lds, f32x16 (&acc)[2][2])
{
    float* const la0 = lds;
    float* const la1 = lds + kTile * kLdsStride;
    float* const lb0 = lds + 2 * kTile * kLdsStride;
    float* const lb1 = lds + 3 * kTile * kLdsStride;
    const int64_t nch = cdiv(K, kKC);
    Stage sa, sb;
    A.load(row0a, 0, sa);
    B.load(row0b, 0, sb);
    A.store(la0, sa);
    B.store(lb0, sb);
    __syncthreads();
    for (int64_t c = 0; c < nch; c += 2) {
        // chunk c in buffer 0, prefetch c + 1 into buffer 1
        bool more = c + 1 < nch;
        if (more) {
            A.load(row0a, (c + 1) * kKC, sa);
            B.load(row0b, (c + 1) * kKC, sb);
        }
        mfma_chunk(la0, lb0, acc);
        if (more) {
            A.store(la1, sa);
            B.store(lb1, sb);
        }
        __syncthreads();
        if (!more) break;
        // chunk c + 1 in buffer 1, prefetch c + 2 into buffer 0
        more = c + 2 < nch;
        if (more) {
            A.load(row0a, (c + 2) * kKC, sa);
            B.load(row0b, (c + 2) * kKC, sb);
        }
        mfma_chunk(la1, lb1, acc);
        if (more) {
            A.store(la0, sa);
            B.store(lb0, sb);
        }
        __syncthreads();
    }
}

__device__ inline void zero_acc(f32x16 (&acc)[2][2])
{
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// ---------------------------------------------------------------- reductions
// Deterministic fp64 sum over a 256-thread block (fixed tree); every thread gets it.
__device__ inline double block_sum_f64(double v, double* sh /* >= 256 */)
{
    sh[threadIdx.x] = v;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
        __syncthreads();
    }
    double r = sh[0];
    __syncthreads();
    return r;
}

// ---------------------------------------------------------------- host helpers
// Bump allocator over a caller workspace; the first kStatusBytes hold the status word.
struct Ws {
    char* base;
    size_t off;
    explicit Ws(void* p) : base(static_cast<char*>(p)), off(kStatusBytes) {}
    template <typename T>
    T* take(size_t count)
    {
        T* r = reinterpret_cast<T*>(base + off);
        off = align256(off + count * sizeof(T));
        return r;
    }
};

// Launch helpers implemented in the kernel translation units (host side).
size_t gram_ws_bytes(int64_t p, int64_t n);
qe_status launch_gram(const float* X, int64_t p, int64_t n, int layout, float* Sigma,
                      int accumulate, float damp, void* ws, hipStream_t s);
qe_status launch_grid_minmax(const float* W, const float* H, int64_t q, int64_t p, int bits,
                             float* scale, float* zero, hipStream_t s);
qe_status launch_nonfinite_scan(const float* a, int64_t count, int* status, hipStream_t s);
size_t objective_ws_bytes(int64_t q, int64_t p);
qe_status launch_objective(const float* W, const float* Wh, const float* H, const float* Sigma,
                           int64_t q, int64_t p, double* out, void* ws, hipStream_t s);
size_t cd_ws_bytes(int64_t q, int64_t p, int block);
qe_status launch_cd(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                    const float* scale, const float* zero, float* Wh, uint8_t* codes, float* R,
                    const float* H, int sweeps, int block, uint32_t flags, double* obj,
                    int obj_stride, const double* f_in, void* ws, hipStream_t s);
qe_status launch_residual_dot(const float* W, const float* Wh, const float* H, const float* R,
                              int64_t count, double* out, double* part, const int* status,
                              hipStream_t s);
size_t topk_ws_bytes(int64_t count, int64_t s);
qe_status launch_topk(const float* V, int64_t count, int64_t s, float* out, int64_t* support,
                      int64_t* nnz, void* ws, hipStream_t st);
size_t topk_columns_ws_bytes(int64_t q, int64_t p);
qe_status launch_topk_columns(const float* V, int64_t q, int64_t p, int64_t c, float* out,
                              int64_t* columns, int64_t* support, int64_t* nnz, void* ws,
                              hipStream_t st);
size_t outlier_ws_bytes(int64_t q, int64_t p, int block, int64_t s);
qe_status launch_outlier(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                         const float* scale, const float* zero, float* Wh, uint8_t* codes,
                         float* H, float* E, int64_t s, float lambda, int64_t* support,
                         int64_t* support_nnz, int sweeps, int block, uint32_t flags,
                         double* obj, void* ws, hipStream_t st);
int64_t packed_row_bytes(int64_t p, int bits);
qe_status launch_pack_codes(const uint8_t* codes, int64_t q, int64_t p, int bits,
                            uint8_t* packed, hipStream_t s);
qe_status launch_outliers_csr(const float* H, int64_t q, int64_t p, const int64_t* support,
                              const int64_t* nnz, int64_t cap, int64_t* rowptr, int32_t* cols,
                              float* vals, hipStream_t s);
size_t lambda_ws_bytes(int64_t p);
qe_status launch_lambda(const float* Sigma, int64_t p, int max_iters, float tol, float* out,
                        void* ws, hipStream_t s);

}  // namespace qe
