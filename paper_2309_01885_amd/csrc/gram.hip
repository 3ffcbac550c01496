// Gram matrix Sigma = X X^T on the matrix cores of gfx950.
//
// Products: by default, on the 256 x 256 tiles, on the fp16 matrix cores with
// every channel scaled by a power of two and split into two fp16 values, three
// products kept per fp32 product (gram_x3w_kernel with F2, see nt_f2.h); on
// the other tiles, or with QE_GRAM_BF16X3, on the bf16 matrix cores with every
// fp32 operand split exactly into three bf16 values and six products kept
// (gram_x3_kernel and gram_x3w_kernel, see nt_x3.h); with QE_GRAM_FP32 on the
// fp32 matrix cores (gram_kernel).  All share the work split and the
// reductions below.
//
// Lemma 1 (Sec. 3.2) needs X only through Sigma, a p x p statistic whose size
// does not grow with the token count n.  Work split: 128 x 128 tiles of the
// upper triangle (ti <= tj) x token splits of at most kSplitTokensMax tokens,
// their count chosen to fill the last round of workgroups (gram_splits).
// Each workgroup sums its split in the fp32 matrix-core accumulators (a
// running sum of at most 32768 products), writes the partial tile to the
// workspace, and a finalize kernel adds the splits in a fixed order in fp64.
// When the split partials would not fit the workspace budget (very large p),
// one workgroup per tile sums all tokens with a two-level accumulator (inner
// sums of 512 tokens added into a second fp32 accumulator) and writes Sigma
// directly.  The lower triangle is
// written as an exact mirror through an LDS transpose.
#include "nt_f2.h"
#include "nt_x3.h"
#include "qe_internal.h"

namespace qe {

constexpr int kInnerChunks = 16;          // two-level mode: 16 x 32 = 512 tokens per inner sum
constexpr int64_t kSplitTokensMax = 32768;  // longest single fp32 running sum allowed
constexpr size_t kSplitBudget = size_t(2) << 30;   // bytes of split partials allowed
constexpr int kTileFloats = kTile * kTile;
constexpr int kTStride = kTile + 1;       // LDS transpose tile row stride

__device__ inline void tri_index(int64_t t, int64_t nt, int64_t& ti, int64_t& tj)
{
    // row ti of the upper triangle starts at ti * nt - ti * (ti - 1) / 2
    const double b = 2.0 * nt + 1.0;
    int64_t r = (int64_t)((b - sqrt(b * b - 8.0 * (double)t)) * 0.5);
    if (r < 0) r = 0;
    auto start = [nt](int64_t i) { return i * nt - i * (i - 1) / 2; };
    while (r > 0 && start(r) > t) --r;
    while (r + 1 < nt && start(r + 1) <= t) ++r;
    ti = r;
    tj = r + (t - start(r));
}

__device__ inline int64_t tri_row_start(int64_t i, int64_t nt) { return i * nt - i * (i - 1) / 2; }

// Tile t of the upper triangle in banded order: bands of 8 tile rows, each
// band ordered by tile column, so that consecutive tiles share their row
// panels (and, within a band, their column panel).
__device__ inline void band_index(int64_t t, int64_t nt, int64_t& ti, int64_t& tj)
{
    int64_t r, c;
    tri_index(t, nt, r, c);
    const int64_t b0 = (r / 8) * 8;
    const int64_t bh = min((int64_t)8, nt - b0);
    const int64_t u = t - tri_row_start(b0, nt);
    const int64_t tri = bh * (bh + 1) / 2;
    if (u < tri) {
        int64_t m = (int64_t)((sqrt(8.0 * (double)u + 1.0) - 1.0) * 0.5);
        while (m > 0 && m * (m + 1) / 2 > u) --m;
        while ((m + 1) * (m + 2) / 2 <= u) ++m;
        tj = b0 + m;
        ti = b0 + (u - m * (m + 1) / 2);
    } else {
        const int64_t v = u - tri;
        tj = b0 + bh + v / bh;
        ti = b0 + v % bh;
    }
}

// Writes rows [r0, r0 + nr) of the 128 x 128 tile (held in LDS as rows
// 0 .. nr-1, row stride kTStride) to Sigma's upper block (ti, tj) and their
// mirror in block (tj, ti).  On a diagonal tile only the entries with
// row <= col are taken and the rest mirrored, so Sigma is exactly symmetric.
// With `accumulate`, the old upper value is added first.
__device__ void write_symmetric(float* tileLds, int64_t ti, int64_t tj, float* Sigma, int64_t p,
                                int accumulate, int r0, int nr)
{
    const int64_t a0 = ti * kTile + r0, b0 = tj * kTile;
    const bool diag = ti == tj;
    for (int e = threadIdx.x; e < nr * kTile; e += blockDim.x) {
        const int r = e / kTile, c = e % kTile;
        const int64_t a = a0 + r, b = b0 + c;
        if (a < p && b < p && (!diag || r0 + r <= c)) {
            float v = tileLds[r * kTStride + c];
            if (accumulate) v += Sigma[a * p + b];
            Sigma[a * p + b] = v;
            tileLds[r * kTStride + c] = v;
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < nr * kTile; e += blockDim.x) {
        const int c = e / nr, r = e % nr;            // consecutive threads: consecutive a
        const int64_t a = a0 + r, b = b0 + c;
        if (a < p && b < p && (!diag || r0 + r < c)) Sigma[b * p + a] = tileLds[r * kTStride + c];
    }
}

template <bool TRANS, bool TWO_LEVEL>
__global__ __launch_bounds__(256, TWO_LEVEL ? 1 : 2) void gram_kernel(
    const float* __restrict__ X, int64_t p, int64_t n, int64_t nt, int64_t split_len,
    float* __restrict__ out, int accumulate, int x_vec4, const int* status)
{
    if (failed(status)) return;
    __shared__ __attribute__((aligned(16))) float lds[kNTLdsFloats];
    int64_t ti, tj;
    tri_index(blockIdx.x, nt, ti, tj);
    const int64_t k0 = (int64_t)blockIdx.y * split_len;
    const int64_t k1 = min(n, k0 + split_len);

    f32x16 acc[2][2];
    auto run = [&](int64_t kb, int64_t ke) {
        if (TRANS) {
            // X is n x p: element (channel r, token k) at X[k * p + r]
            const ColOp op{X + kb * p, p, p, ke - kb, x_vec4 != 0};
            nt_tile(op, ti * kTile, op, tj * kTile, ke - kb, lds, acc);
        } else {
            const RowOp op{X + kb, n, p, ke - kb, x_vec4 != 0};
            nt_tile(op, ti * kTile, op, tj * kTile, ke - kb, lds, acc);
        }
    };
    if constexpr (TWO_LEVEL) {
        f32x16 outer[2][2];
        zero_acc(outer);
        const int64_t inner = (int64_t)kInnerChunks * kKC;
        for (int64_t kb = k0; kb < k1; kb += inner) {
            zero_acc(acc);
            run(kb, min(k1, kb + inner));
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b) outer[a][b] += acc[a][b];
        }
        float* tl = lds;   // reuse the pipeline LDS (nt_tile ended with a barrier)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    tl[acc_row(mi, v) * kTStride + acc_col(ni)] = outer[mi][ni][v];
        __syncthreads();
        write_symmetric(tl, ti, tj, out, p, accumulate, 0, kTile);
    } else {
        zero_acc(acc);
        run(k0, k1);
        float* dst = out + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * kTileFloats;
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[acc_row(mi, v) * kTile + acc_col(ni)] = acc[mi][ni][v];
    }
}

// The same work on the bf16 matrix cores with the exact three-way split of
// each fp32 operand (six bf16 products per fp32 product, fp32 accumulation).
// Work items (tile, split) are dealt to the 8 XCDs in contiguous ranges (the
// hardware places workgroup b on XCD b % 8), split-major and in banded tile
// order inside a split, so the workgroups resident on one XCD at a time share
// their X panels through that XCD's L2.
// FULL launches (every 128-row panel inside X, every K range a multiple of
// 32, aligned rows) take the unguarded two-stage-prefetch loop; any other
// shape takes the guarded loop for every tile.
template <bool TRANS, bool TWO_LEVEL, bool FULL>
__global__ __launch_bounds__(256, TWO_LEVEL ? 1 : 2) void gram_x3_kernel(
    const float* __restrict__ X, int64_t p, int64_t n, int64_t nt, int64_t tiles,
    int64_t splits, int64_t split_len, float* __restrict__ out, int accumulate, const int* status)
{
    if (failed(status)) return;
    // the two-level mode also stages the finished 128 x kTStride tile here
    constexpr int kLds = TWO_LEVEL && kTile * kTStride > kX3LdsDw ? kTile * kTStride : kX3LdsDw;
    __shared__ __attribute__((aligned(16))) uint32_t lds[kLds];
    const int64_t items = tiles * splits;
    const int64_t per = cdiv(items, 8);
    const int64_t item = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= items) return;                    // uniform: the whole workgroup leaves
    const int64_t sp = item / tiles;
    int64_t ti, tj;
    band_index(item % tiles, nt, ti, tj);
    const int64_t k0 = sp * split_len;
    const int64_t k1 = min(n, k0 + split_len);

    f32x16 acc[2][2];
    auto run = [&](int64_t kb, int64_t ke) {
        const int64_t K = ke - kb;
        if constexpr (TRANS) {
            const X3Col op{X + kb * p, p, p, K};
            if constexpr (FULL) nt_tile_x3_full<true>(op, ti * kTile, op, tj * kTile, K, lds, acc);
            else nt_tile_x3_edge(op, ti * kTile, op, tj * kTile, K, lds, acc);
        } else {
            const X3Row op{X + kb, n, p, K};
            if constexpr (FULL) nt_tile_x3_full<true>(op, ti * kTile, op, tj * kTile, K, lds, acc);
            else nt_tile_x3_edge(op, ti * kTile, op, tj * kTile, K, lds, acc);
        }
    };
    float* tl = reinterpret_cast<float*>(lds);
    if constexpr (TWO_LEVEL) {
        f32x16 outer[2][2];
        zero_acc(outer);
        const int64_t inner = (int64_t)kInnerChunks * kKC;
        for (int64_t kb = k0; kb < k1; kb += inner) {
            zero_acc(acc);
            run(kb, min(k1, kb + inner));
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b) outer[a][b] += acc[a][b];
        }
        // the K loop ended with a barrier: the stage area is free
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    tl[acc_row(mi, v) * kTStride + acc_col(ni)] = outer[mi][ni][v];
        __syncthreads();
        write_symmetric(tl, ti, tj, out, p, accumulate, 0, kTile);
    } else {
        zero_acc(acc);
        run(k0, k1);
        const int64_t slot = tri_row_start(ti, nt) + (tj - ti);
        float* dst = out + (sp * tiles + slot) * kTileFloats;
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    dst[acc_row(mi, v) * kTile + acc_col(ni)] = acc[mi][ni][v];
    }
}

// Split mode on 256 x 256 tiles: one workgroup of eight waves per CU, each
// wave a 64 x 128 block, so that every staged operand value feeds twice the
// matrix-core work of the 128 x 128 tile (half the split work, LDS traffic
// and L2 traffic per product), with the operand reads pipelined through three
// LDS stage buffers (nt_tile_x3_wide).  Used when every 256-row panel lies
// inside X (p a multiple of 256, aligned rows, token ranges multiples of 32),
// in either layout (channel-major rows through X3Row, token-major through
// X3Col).  Each wave's 64 x 128 block lies in one 128 x 128 tile of the
// upper triangle, so the partials use the same slots as gram_x3_kernel and
// the same finalize.
constexpr int kWide = 256;

__device__ inline void band_index_wide(int64_t t, int64_t nt, int64_t& ti, int64_t& tj)
{
    // bands of 4 tile rows: about the 32 workgroups an XCD holds at a time
    int64_t r, c;
    tri_index(t, nt, r, c);
    const int64_t b0 = (r / 4) * 4;
    const int64_t bh = min((int64_t)4, nt - b0);
    const int64_t u = t - tri_row_start(b0, nt);
    const int64_t tri = bh * (bh + 1) / 2;
    if (u < tri) {
        int64_t m = (int64_t)((sqrt(8.0 * (double)u + 1.0) - 1.0) * 0.5);
        while (m > 0 && m * (m + 1) / 2 > u) --m;
        while ((m + 1) * (m + 2) / 2 <= u) ++m;
        tj = b0 + m;
        ti = b0 + (u - m * (m + 1) / 2);
    } else {
        const int64_t v = u - tri;
        tj = b0 + bh + v / bh;
        ti = b0 + v % bh;
    }
}

// DIRECT: one token range per launch (n <= kSplitTokensMax, a single fp32
// running sum), written to Sigma itself (with accumulate) through the same
// LDS-transposed symmetric writes as the two-level mode, 128 x 128 quadrant
// by quadrant; the large-p replacement of the two-level mode for streamed
// token chunks.
//
// F2: the two-way fp16 split of nt_f2.h, channel i scaled by 2^chexp[i] on the
// way in and every sum scaled back by 2^-(chexp[i] + chexp[j]) on the way out
// (exact); otherwise the three-way bf16 split of nt_x3.h (chexp unused).
template <bool DIRECT, bool TRANS, bool F2>
__global__ __launch_bounds__(512, 1) void gram_x3w_kernel(
    const float* __restrict__ X, int64_t p, int64_t n, int64_t ntw, int64_t tiles_w, int64_t nt,
    int64_t tiles, int64_t splits, int64_t split_len, float* __restrict__ out, int accumulate,
    const int* __restrict__ chexp, const int* status)
{
    if (failed(status)) return;
    // the direct mode also stages a finished 128 x kTStride quadrant here
    static_assert(kTile * kTStride <= 3 * kF2BufDw && kTile * kTStride <= kX3wLdsDw, "quadrant fits");
    __shared__ __attribute__((aligned(16))) uint32_t lds[F2 ? (TRANS ? 4 : 3) * kF2BufDw : kX3wLdsDw];
    const int64_t items = tiles_w * splits;
    const int64_t per = cdiv(items, 8);
    const int64_t item = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= items) return;                    // uniform: the whole workgroup leaves
    const int64_t sp = item / tiles_w;
    int64_t ti, tj;
    band_index_wide(item % tiles_w, ntw, ti, tj);
    const int64_t k0 = sp * split_len;
    const int64_t K = min(n, k0 + split_len) - k0;
    f32x16 acc[2][4];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mi][ni][v] = 0.f;
    if constexpr (F2 && TRANS) {
        // X is n x p; this thread stages channel t / 2 of both panels (eight
        // tokens, buffer loads); four stage buffers
        const int r = threadIdx.x >> 1;
        const F2ColB A{X + k0 * p, p, ldexpf(1.f, chexp[ti * kWide + r])};
        const F2ColB B{X + k0 * p, p, ldexpf(1.f, chexp[tj * kWide + r])};
        nt_tile_f2_wide<4>(A, ti * kWide, B, tj * kWide, K, lds, acc);
    } else if constexpr (F2) {
        // this thread stages channels t / 4 and t / 4 + 128 of both panels
        // (four tokens each); three stage buffers, which keep the loop free of
        // register spills
        const int r = threadIdx.x >> 2;
        const F2RowQ A{X + k0, n, {ldexpf(1.f, chexp[ti * kWide + r]),
                                   ldexpf(1.f, chexp[ti * kWide + r + 128])}};
        const F2RowQ B{X + k0, n, {ldexpf(1.f, chexp[tj * kWide + r]),
                                   ldexpf(1.f, chexp[tj * kWide + r + 128])}};
        nt_tile_f2_wide<3>(A, ti * kWide, B, tj * kWide, K, lds, acc);
    } else if constexpr (TRANS) {
        // X is n x p: element (channel r, token k) at X[k * p + r]
        const X3Col op{X + k0 * p, p, 0, K};
        nt_tile_x3_wide(op, ti * kWide, op, tj * kWide, K, lds, acc);
    } else {
        const X3Row op{X + k0, n, 0, K};
        nt_tile_x3_wide(op, ti * kWide, op, tj * kWide, K, lds, acc);
    }
    // wave (wm, wn): rows 64 wm .. of the tile, columns 128 wn ..
    const int wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t qi = 2 * ti + wm / 2, qj = 2 * tj + wn;
    const int lane = threadIdx.x & 63;
    const int r0 = (wm & 1) * 64;
    if constexpr (F2) {
        int ec[4];
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) ec[ni] = chexp[tj * kWide + wn * 128 + 32 * ni + (lane & 31)];
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int er = chexp[ti * kWide + wm * 64 + 32 * mi + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)];
#pragma unroll
                for (int ni = 0; ni < 4; ++ni) acc[mi][ni][v] = ldexpf(acc[mi][ni][v], -(er + ec[ni]));
            }
    }
    if constexpr (DIRECT) {
        // the K loop ended with a barrier: its LDS holds a 128 x kTStride tile
        float* tl = reinterpret_cast<float*>(lds);
#pragma unroll 1
        for (int quad = 0; quad < 4; ++quad) {
            const int a = quad >> 1, b = quad & 1;          // rows 128 a.., columns 128 b..
            const int64_t gi = 2 * ti + a, gj = 2 * tj + b;
            if (gi > gj) continue;                           // uniform across the workgroup
            if (wm / 2 == a && wn == b) {
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            tl[(r0 + 32 * mi + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * kTStride +
                               32 * ni + (lane & 31)] = acc[mi][ni][v];
            }
            __syncthreads();
            write_symmetric(tl, gi, gj, out, p, accumulate, 0, kTile);
            __syncthreads();
        }
        return;
    }
    if (qi > qj) return;                          // below the diagonal of a diagonal tile
    float* dst = out + (sp * tiles + tri_row_start(qi, nt) + (qj - qi)) * kTileFloats;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                dst[(r0 + 32 * mi + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * kTile + 32 * ni +
                    (lane & 31)] = acc[mi][ni][v];
}

// Adds the split partial tiles in fixed split order (fp64) and writes Sigma.
// Workgroup (tile, quarter): rows [32 quarter, 32 quarter + 32) of the tile,
// one float4 column group per thread and pass, all splits in flight.
constexpr int kFinRows = 32;

__global__ __launch_bounds__(256) void gram_finalize_kernel(const float* __restrict__ parts,
                                                            int64_t ntiles, int splits,
                                                            int64_t nt, float* Sigma, int64_t p,
                                                            int accumulate, const int* status)
{
    if (failed(status)) return;
    __shared__ float tl[kFinRows * kTStride];
    int64_t ti, tj;
    tri_index(blockIdx.x, nt, ti, tj);
    const int r0 = (int)blockIdx.y * kFinRows;
    const float* src0 = parts + (int64_t)blockIdx.x * kTileFloats + r0 * kTile;
    const int64_t sstride = ntiles * kTileFloats;
#pragma unroll
    for (int u = 0; u < kFinRows * kTile / 4 / 256; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int r = f / (kTile / 4), c = 4 * (f % (kTile / 4));
        const float* src = src0 + r * kTile + c;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
#pragma unroll 4
        for (int sp = 0; sp < splits; ++sp) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(src + sp * sstride);
            s0 += (double)v[0];
            s1 += (double)v[1];
            s2 += (double)v[2];
            s3 += (double)v[3];
        }
        float* d = tl + r * kTStride + c;
        d[0] = (float)s0;
        d[1] = (float)s1;
        d[2] = (float)s2;
        d[3] = (float)s3;
    }
    __syncthreads();
    write_symmetric(tl, ti, tj, Sigma, p, accumulate, r0, kFinRows);
}

// Sigma_jj += damp * mean_j(Sigma_jj): one workgroup, fp64 mean.
__global__ __launch_bounds__(256) void damp_kernel(float* Sigma, int64_t p, float damp,
                                                   const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    double s = 0.0;
    for (int64_t j = threadIdx.x; j < p; j += blockDim.x) s += (double)Sigma[j * p + j];
    const double total = block_sum_f64(s, sh);
    const float add = (float)((double)damp * (total / (double)p));
    for (int64_t j = threadIdx.x; j < p; j += blockDim.x) Sigma[j * p + j] += add;
}

// Channel exponents of the fp16 split: e with the channel's largest |x| times
// 2^e in [2^14, 2^15) (frexp: amax = f 2^ex, f in [1/2, 1)), at most 127 (2^e
// a normal float; e >= -113 holds for any finite amax); 0 for an all-zero or
// non-finite channel (a non-finite value reaches Sigma as in fp32).
__device__ inline int chan_exp(float amax)
{
    if (!(amax > 0.f) || !isfinite(amax)) return 0;
    int ex;
    (void)frexpf(amax, &ex);
    return min(15 - ex, 127);
}

__device__ inline float absmax4(float m, f32x4 v)
{
    return fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
}

// Channel-major X (p x n): one workgroup per channel.
__global__ __launch_bounds__(256) void chan_exp_pn_kernel(const float* __restrict__ X, int64_t n,
                                                          int x_vec4, int* __restrict__ chexp,
                                                          const int* status)
{
    if (failed(status)) return;
    __shared__ float sh[4];
    const float* row = X + (int64_t)blockIdx.x * n;
    float m = 0.f;
    if (x_vec4) {
        // n % 4 == 0 and 16-byte aligned rows
        const f32x4* r4 = reinterpret_cast<const f32x4*>(row);
#pragma unroll 4
        for (int64_t i = threadIdx.x; i < n / 4; i += 256) m = absmax4(m, r4[i]);
    } else {
        for (int64_t i = threadIdx.x; i < n; i += 256) m = fmaxf(m, fabsf(row[i]));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) chexp[blockIdx.x] = chan_exp(fmaxf(fmaxf(sh[0], sh[1]), fmaxf(sh[2], sh[3])));
}

// Token-major X (n x p): workgroup (column block of 1024, token slice y) takes
// the tokens y, y + slices, ... of its columns (4 per thread) and writes
// their largest |x| to part[y * p + column]; chan_exp_np_kernel reduces.
__global__ __launch_bounds__(256) void chan_absmax_np_kernel(const float* __restrict__ X, int64_t p,
                                                             int64_t n, int x_vec4,
                                                             float* __restrict__ part,
                                                             const int* status)
{
    if (failed(status)) return;
    const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (c >= p) return;
    const int64_t slices = gridDim.y;
    f32x4 m = {0.f, 0.f, 0.f, 0.f};
    if (x_vec4) {
        // p % 4 == 0 and 16-byte aligned token rows: the 4 columns are inside X
        float a = 0.f, b = 0.f, cc = 0.f, d = 0.f;
#pragma unroll 8
        for (int64_t t = blockIdx.y; t < n; t += slices) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(X + t * p + c);
            a = fmaxf(a, fabsf(v[0]));
            b = fmaxf(b, fabsf(v[1]));
            cc = fmaxf(cc, fabsf(v[2]));
            d = fmaxf(d, fabsf(v[3]));
        }
        m = f32x4{a, b, cc, d};
    } else {
        for (int64_t t = blockIdx.y; t < n; t += slices)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (c + u < p) m[u] = fmaxf(m[u], fabsf(X[t * p + c + u]));
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
        if (c + u < p) part[blockIdx.y * p + c + u] = m[u];
}

__global__ __launch_bounds__(256) void chan_exp_np_kernel(const float* __restrict__ part, int64_t p,
                                                          int slices, int* __restrict__ chexp,
                                                          const int* status)
{
    if (failed(status)) return;
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j >= p) return;
    float m = 0.f;
#pragma unroll 8
    for (int y = 0; y < slices; ++y) m = fmaxf(m, part[y * p + j]);
    chexp[j] = chan_exp(m);
}

// Token slices of chan_absmax_np_kernel: about 2048 workgroups, at least 256
// tokens a slice, at most 512 slices (the partials then hold at most 8 MB).
static int64_t chan_slices(int64_t p, int64_t n)
{
    return std::max<int64_t>(
        1, std::min<int64_t>(std::min<int64_t>(512, 2048 / cdiv(p, 1024)), cdiv(n, 256)));
}

// Workspace of the channel exponents: p ints and the token-major partials.
static size_t chan_ws_bytes(int64_t p, int64_t n)
{
    return align256((size_t)p * sizeof(int)) +
           align256((size_t)chan_slices(p, n) * p * sizeof(float));
}

// Number of token splits, or 0 for the two-level direct mode.
//
// The tile kernels hold one workgroup per slot (256 slots for the 256 x 256
// tiles at one workgroup per CU, 512 for the 128 x 128 tiles at two, on the 256
// CUs of the MI355X), so a launch of items = tiles x splits workgroups of
// ceil(n / splits) tokens takes ceil(items / slots) rounds.  The count chosen
// minimises, in units of one workgroup's time per token, rounds x (tokens per
// split + a fixed cost per workgroup) + the finalize's reads of the partials,
// over the counts whose splits hold at most kSplitTokensMax tokens and whose
// partials fit kSplitBudget; ties keep the fewer splits.  Depends only on (p, n).
constexpr int64_t kGramSlotsWide = 256, kGramSlotsNarrow = 512;
constexpr double kGramWgCostTokens = 32.0;        // prologue, pipeline fill, partial-tile store
constexpr double kGramFinalizeTokensPerTile = 0.11;   // one 64 KB partial tile read in finalize

static int64_t gram_splits(int64_t p, int64_t n)
{
    const int64_t nt = cdiv(p, kTile);
    const int64_t tiles = nt * (nt + 1) / 2;
    const bool wide = p % kWide == 0;
    const int64_t items = wide ? (p / kWide) * (p / kWide + 1) / 2 : tiles;
    const int64_t slots = wide ? kGramSlotsWide : kGramSlotsNarrow;
    const int64_t s_min = cdiv(n, kSplitTokensMax);
    const int64_t s_max = std::min<int64_t>(
        (int64_t)(kSplitBudget / ((size_t)tiles * kTileFloats * sizeof(float))), cdiv(n, kKC));
    if (s_min > s_max) return 0;
    int64_t best = s_min;
    double best_cost = 0.0;
    for (int64_t sp = s_min; sp <= s_max; ++sp) {
        const int64_t len = cdiv(cdiv(n, sp), kKC) * kKC;
        const int64_t used = cdiv(n, len);
        const double cost = (double)cdiv(items * used, slots) * ((double)len + kGramWgCostTokens) +
                            kGramFinalizeTokensPerTile * (double)(used * tiles);
        if (sp == s_min || cost < best_cost) {
            best = sp;
            best_cost = cost;
        }
    }
    return best;
}

static size_t gram_ws_one(int64_t p, int64_t n)
{
    const int64_t nt = cdiv(p, kTile);
    const int64_t tiles = nt * (nt + 1) / 2;
    const int64_t splits = gram_splits(p, n);
    return kStatusBytes + align256((size_t)splits * tiles * kTileFloats * sizeof(float)) +
           chan_ws_bytes(p, n);
}

// Token-major X with a token count that is not a multiple of 32 is taken as
// an aligned part on the 256 x 256 tiles and a short tail (launch_gram).
constexpr int64_t kTokAlign = 2 * kX3KC;

size_t gram_ws_bytes(int64_t p, int64_t n)
{
    size_t b = gram_ws_one(p, n);
    if (n > kTokAlign && n % kTokAlign != 0)
        b = std::max(b, std::max(gram_ws_one(p, n - n % kTokAlign), gram_ws_one(p, n % kTokAlign)));
    return b;
}

static qe_status launch_gram_one(const float* X, int64_t p, int64_t n, int layout, float* Sigma,
                                 int accumulate, float damp, void* ws, hipStream_t s);

qe_status launch_gram(const float* X, int64_t p, int64_t n, int layout, float* Sigma,
                      int accumulate, float damp, void* ws, hipStream_t s)
{
    const bool trans = (layout & ~(QE_GRAM_FP32 | QE_GRAM_BF16X3)) == QE_LAYOUT_NP;
    if (trans && !(layout & QE_GRAM_FP32) && p % kWide == 0 && n > kTokAlign &&
        n % kTokAlign != 0) {
        // token rows are contiguous: the tail is X's last n % 32 token rows
        const int64_t tail = n % kTokAlign, main = n - tail;
        const qe_status st = launch_gram_one(X, p, main, layout, Sigma, accumulate, 0.f, ws, s);
        if (st != QE_OK) return st;
        return launch_gram_one(X + main * p, p, tail, layout, Sigma, 1, damp, ws, s);
    }
    return launch_gram_one(X, p, n, layout, Sigma, accumulate, damp, ws, s);
}

static qe_status launch_gram_one(const float* X, int64_t p, int64_t n, int layout, float* Sigma,
                                 int accumulate, float damp, void* ws, hipStream_t s)
{
    int* status = static_cast<int*>(ws);
    const int64_t nt = cdiv(p, kTile);
    const int64_t tiles = nt * (nt + 1) / 2;
    const int64_t splits = gram_splits(p, n);
    const bool fp32 = (layout & QE_GRAM_FP32) != 0;
    // the fp16 split (its token-major loader's buffer offsets are 32-bit)
    const bool f2 = (layout & QE_GRAM_BF16X3) == 0 && p <= (int64_t(1) << 24);
    const bool trans = (layout & ~(QE_GRAM_FP32 | QE_GRAM_BF16X3)) == QE_LAYOUT_NP;
    // 16-byte loads need an aligned base and a row stride that keeps them aligned
    const int x_vec4 = aligned16(X) && ((trans ? p : n) % 4 == 0);
    // split length: a multiple of the K chunk, at most kSplitTokensMax
    const int64_t split_len = splits == 0 ? n : cdiv(cdiv(n, splits), kKC) * kKC;
    const int64_t used = splits == 0 ? 1 : cdiv(n, split_len);
    float* parts = reinterpret_cast<float*>(static_cast<char*>(ws) + kStatusBytes);
    float* dst = splits == 0 ? Sigma : parts;
    // channel exponents (fp16 split) after the split partials
    char* const chws = static_cast<char*>(ws) + kStatusBytes +
                       align256((size_t)splits * tiles * kTileFloats * sizeof(float));
    int* const chexp = reinterpret_cast<int*>(chws);
    float* const chpart = reinterpret_cast<float*>(chws + align256((size_t)p * sizeof(int)));
    if (fp32) {
        dim3 grid((unsigned)tiles, (unsigned)used);
        if (splits == 0) {
            if (trans)
                hipLaunchKernelGGL((gram_kernel<true, true>), grid, dim3(256), 0, s, X, p, n, nt,
                                   n, Sigma, accumulate, x_vec4, status);
            else
                hipLaunchKernelGGL((gram_kernel<false, true>), grid, dim3(256), 0, s, X, p, n, nt,
                                   n, Sigma, accumulate, x_vec4, status);
        } else {
            if (trans)
                hipLaunchKernelGGL((gram_kernel<true, false>), grid, dim3(256), 0, s, X, p, n, nt,
                                   split_len, parts, accumulate, x_vec4, status);
            else
                hipLaunchKernelGGL((gram_kernel<false, false>), grid, dim3(256), 0, s, X, p, n,
                                   nt, split_len, parts, accumulate, x_vec4, status);
        }
    } else {
        const unsigned grid = (unsigned)(8 * cdiv(tiles * used, 8));
        // every panel inside X, every K range a multiple of 32 (split_len is)
        const bool full = x_vec4 && p % kTile == 0 && n % (2 * kX3KC) == 0;
#define QE_GRAM_X3(T, L, F)                                                                     \
    hipLaunchKernelGGL((gram_x3_kernel<T, L, F>), dim3(grid), dim3(256), 0, s, X, p, n, nt, tiles, \
                       used, split_len, dst, accumulate, status)
        const bool two = splits == 0;
        if (full && p % kWide == 0 && (!two || n <= kSplitTokensMax)) {
            const int64_t ntw = p / kWide;
            const int64_t tiles_w = ntw * (ntw + 1) / 2;
            const dim3 grid((unsigned)(8 * cdiv(tiles_w * used, 8)));
            if (f2) {
                if (trans) {
                    const int64_t sl = chan_slices(p, n);
                    hipLaunchKernelGGL(chan_absmax_np_kernel,
                                       dim3((unsigned)cdiv(p, 1024), (unsigned)sl), dim3(256), 0, s,
                                       X, p, n, x_vec4, chpart, status);
                    hipLaunchKernelGGL(chan_exp_np_kernel, dim3((unsigned)cdiv(p, 256)), dim3(256),
                                       0, s, chpart, p, (int)sl, chexp, status);
                } else {
                    hipLaunchKernelGGL(chan_exp_pn_kernel, dim3((unsigned)p), dim3(256), 0, s, X, n,
                                       x_vec4, chexp, status);
                }
                if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
            }
#define QE_GRAM_X3W(D, T, F, SPLITS, LEN, OUT)                                                  \
    hipLaunchKernelGGL((gram_x3w_kernel<D, T, F>), grid, dim3(512), 0, s, X, p, n, ntw, tiles_w,   \
                       nt, tiles, SPLITS, LEN, OUT, accumulate, chexp, status)
            if (f2) {
                if (two && trans) QE_GRAM_X3W(true, true, true, (int64_t)1, n, Sigma);
                else if (two) QE_GRAM_X3W(true, false, true, (int64_t)1, n, Sigma);
                else if (trans) QE_GRAM_X3W(false, true, true, used, split_len, parts);
                else QE_GRAM_X3W(false, false, true, used, split_len, parts);
            } else {
                if (two && trans) QE_GRAM_X3W(true, true, false, (int64_t)1, n, Sigma);
                else if (two) QE_GRAM_X3W(true, false, false, (int64_t)1, n, Sigma);
                else if (trans) QE_GRAM_X3W(false, true, false, used, split_len, parts);
                else QE_GRAM_X3W(false, false, false, used, split_len, parts);
            }
#undef QE_GRAM_X3W
        } else if (trans) {
            if (two) { if (full) QE_GRAM_X3(true, true, true); else QE_GRAM_X3(true, true, false); }
            else { if (full) QE_GRAM_X3(true, false, true); else QE_GRAM_X3(true, false, false); }
        } else {
            if (two) { if (full) QE_GRAM_X3(false, true, true); else QE_GRAM_X3(false, true, false); }
            else { if (full) QE_GRAM_X3(false, false, true); else QE_GRAM_X3(false, false, false); }
        }
#undef QE_GRAM_X3
    }
    if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    if (splits != 0) {
        hipLaunchKernelGGL(gram_finalize_kernel, dim3((unsigned)tiles, kTile / kFinRows), dim3(256),
                           0, s, parts, tiles, (int)used, nt, Sigma, p, accumulate, status);
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    if (damp > 0.f) {
        hipLaunchKernelGGL(damp_kernel, dim3(1), dim3(256), 0, s, Sigma, p, damp, status);
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    return QE_OK;
}

}  // namespace qe
