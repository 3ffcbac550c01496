// Outlier-aware QuantEase (Sec. 4) on gfx950: P_s by radix select, the IHT
// step and the sparse residual update.
//
// P_s (Sec. 4.3) keeps the s entries of largest |v|.  |v| of an fp32 value is
// ordered exactly like its bit pattern with the sign cleared, so the s-th
// largest key tau is found by a 3-pass radix select (digits of 11, 11 and 10
// bits; per-workgroup LDS histograms merged with integer atomics, so counts
// are exact and order-free).  Selected: every key > tau, plus the first
// (s - #{key > tau}) keys == tau in linear-index order; tau == 0 selects no
// zeros.  Compaction keeps index order (per-workgroup counts, a scan, then
// wavefront ballots inside each workgroup), so the support comes out sorted.
//
// IHT step (Sec. 4.3, Lemma 3): V = H - E / lambda_max, H+ = P_s(V), then
// E += (H+ - H) Sigma.  The old and new supports are merged into one list
// sorted by linear index (an entry in both carries new - old); the sparse
// product walks each row's stretch of that list in ascending index.
#include <utility>

#include "qe_internal.h"

namespace qe {

constexpr int kSelWgs = 1024;     // workgroups of the histogram / compaction passes
constexpr int kHistBins = 2048;

struct SelState {
    int64_t k_rem;     // rank (1-based, from the top) still to locate inside the prefix class
    int64_t cnt_gt;    // keys strictly above the prefix class
    int64_t need_eq;   // last pass: keys equal to tau to admit
    int64_t nnz;       // selected count
    uint32_t prefix;   // digits chosen so far
    uint32_t tau;
};

__device__ inline uint32_t abs_key(float v) { return __float_as_uint(v) & 0x7fffffffu; }

__global__ void sel_init_kernel(SelState* st, int64_t k, uint32_t* hist, const int* status)
{
    if (failed(status)) return;
    if (threadIdx.x == 0) {
        st->k_rem = k;
        st->cnt_gt = 0;
        st->need_eq = 0;
        st->nnz = 0;
        st->prefix = 0;
        st->tau = 0;
    }
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x) hist[b] = 0u;
}

// Histogram of digit (key >> shift) & dmask over the keys whose higher bits
// (key >> (shift + dbits)) equal the current prefix (pass 0: all keys).
__device__ inline void hist_key(uint32_t* h, uint32_t key, uint32_t prefix, int shift, int hs,
                                uint32_t dmask, bool first)
{
    if (first || (key >> hs) == prefix) atomicAdd(&h[(key >> shift) & dmask], 1u);
}

__global__ __launch_bounds__(256) void sel_hist_kernel(const float* __restrict__ V, int64_t count,
                                                       int shift, int dbits, int first,
                                                       int vec4, const SelState* st,
                                                       uint32_t* hist, const int* status)
{
    if (failed(status)) return;
    __shared__ uint32_t h[kHistBins];
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x) h[b] = 0u;
    __syncthreads();
    const uint32_t prefix = first ? 0u : st->prefix;
    const uint32_t dmask = (1u << dbits) - 1u;
    const int hs = shift + dbits;
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t tail = 0;
    if (vec4) {
        const int64_t n4 = count / 4;
        const f32x4* V4 = reinterpret_cast<const f32x4*>(V);
#pragma unroll 4
        for (int64_t e = tid; e < n4; e += G) {
            const f32x4 v = V4[e];
#pragma unroll
            for (int u = 0; u < 4; ++u) hist_key(h, abs_key(v[u]), prefix, shift, hs, dmask, first);
        }
        tail = n4 * 4;
    }
    for (int64_t e = tail + tid; e < count; e += G)
        hist_key(h, abs_key(V[e]), prefix, shift, hs, dmask, first);
    __syncthreads();
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x)
        if (h[b]) atomicAdd(&hist[b], h[b]);
}

// Finds the digit holding the k_rem-th largest key of the prefix class,
// extends the prefix, and clears the histogram for the next pass.
__global__ __launch_bounds__(256) void sel_pick_kernel(SelState* st, uint32_t* hist, int dbits,
                                                       int last, const int* status)
{
    if (failed(status)) return;
    __shared__ int64_t part[256];
    __shared__ int64_t above[256];
    const int nb = 1 << dbits;
    const int per = nb / 256;            // bins per thread (8 or 4)
    const int t = threadIdx.x;
    // thread t owns bins [nb - (t+1)*per, nb - t*per): thread 0 the top bins
    const int hi = nb - t * per, lo = hi - per;
    int64_t c = 0;
    for (int b = lo; b < hi; ++b) c += hist[b];
    part[t] = c;
    __syncthreads();
    if (t == 0) {
        int64_t run = 0;
        for (int u = 0; u < 256; ++u) {
            above[u] = run;
            run += part[u];
        }
    }
    __syncthreads();
    const int64_t k = st->k_rem;
    const int64_t a0 = above[t];
    if (a0 < k && k <= a0 + part[t]) {
        int64_t run = a0;
        for (int b = hi - 1; b >= lo; --b) {
            const int64_t hb = hist[b];
            if (k <= run + hb) {
                st->cnt_gt += run;
                st->k_rem = k - run;
                st->prefix = (st->prefix << dbits) | (uint32_t)b;
                if (last) {
                    st->tau = st->prefix;
                    st->need_eq = st->prefix == 0u ? 0 : k - run;
                }
                break;
            }
            run += hb;
        }
    }
    __syncthreads();
    for (int b = t; b < kHistBins; b += blockDim.x) hist[b] = 0u;
}

// Per-workgroup counts of keys > tau and keys == tau over contiguous chunks.
__global__ __launch_bounds__(256) void sel_count_kernel(const float* __restrict__ V, int64_t count,
                                                        int64_t chunk, const SelState* st,
                                                        int64_t* cnt, const int* status)
{
    if (failed(status)) return;
    __shared__ double sh[256];
    const uint32_t tau = st->tau;
    const bool want_eq = st->need_eq > 0;
    const int64_t e0 = (int64_t)blockIdx.x * chunk, e1 = min(count, e0 + chunk);
    int64_t gt = 0, eq = 0;
    for (int64_t e = e0 + threadIdx.x; e < e1; e += blockDim.x) {
        const uint32_t key = abs_key(V[e]);
        gt += key > tau;
        eq += want_eq && key == tau;
    }
    const double g = block_sum_f64((double)gt, sh);
    const double q = block_sum_f64((double)eq, sh);
    if (threadIdx.x == 0) {
        cnt[2 * blockIdx.x] = (int64_t)g;
        cnt[2 * blockIdx.x + 1] = (int64_t)q;
    }
}

// Output offset and admitted tie count of every workgroup.  Ties are admitted
// greedily in workgroup order: with exclusive prefix sums GT_w, EQ_w and
// need = #ties to admit, workgroup w admits min(eq_w, max(0, need - EQ_w))
// ties and writes from GT_w + min(EQ_w, need).  One 256-thread workgroup,
// kSelWgs / 256 counts per thread, exact int64 scans.
constexpr int kScanPer = kSelWgs / 256;

__global__ __launch_bounds__(256) void sel_scan_kernel(const int64_t* cnt, int64_t cap,
                                                       SelState* st, int64_t* off, int64_t* adm,
                                                       int64_t* nnz_out, const int* status)
{
    if (failed(status)) return;
    __shared__ int64_t sg[256], se[256];
    const int t = threadIdx.x;
    int64_t g[kScanPer], q[kScanPer], lg = 0, le = 0;
#pragma unroll
    for (int u = 0; u < kScanPer; ++u) {
        g[u] = cnt[2 * (t * kScanPer + u)];
        q[u] = cnt[2 * (t * kScanPer + u) + 1];
        lg += g[u];
        le += q[u];
    }
    sg[t] = lg;
    se[t] = le;
    __syncthreads();
    // inclusive Hillis-Steele scan over the 256 thread totals
    for (int d = 1; d < 256; d <<= 1) {
        const int64_t ag = t >= d ? sg[t - d] : 0, ae = t >= d ? se[t - d] : 0;
        __syncthreads();
        sg[t] += ag;
        se[t] += ae;
        __syncthreads();
    }
    const int64_t need = st->need_eq;
    int64_t pg = sg[t] - lg, pe = se[t] - le;   // exclusive prefixes of this thread's first count
#pragma unroll
    for (int u = 0; u < kScanPer; ++u) {
        const int w = t * kScanPer + u;
        const int64_t room = need - pe > 0 ? need - pe : 0;
        off[w] = pg + (pe < need ? pe : need);
        adm[w] = q[u] < room ? q[u] : room;
        pg += g[u];
        pe += q[u];
    }
    if (t == 255) {
        int64_t pos = sg[255] + (se[255] < need ? se[255] : need);
        if (pos > cap) pos = cap;   // never more than k <= cap by construction; guards the buffers
        st->nnz = pos;
        if (nnz_out) *nnz_out = pos;
    }
}

// Writes the selected indices (ascending) and values, and the dense P_s(V).
__global__ __launch_bounds__(256) void sel_write_kernel(const float* __restrict__ V, int64_t count,
                                                        int64_t chunk, const SelState* st,
                                                        const int64_t* off, const int64_t* adm,
                                                        int64_t cap, int64_t* idx_out,
                                                        float* val_out, float* dense_out,
                                                        const int* status)
{
    if (failed(status)) return;
    __shared__ int wsel[4], weq[4];
    const uint32_t tau = st->tau;
    const bool want_eq = st->need_eq > 0;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t e0 = (int64_t)blockIdx.x * chunk, e1 = min(count, e0 + chunk);
    int64_t pos = off[blockIdx.x];
    int64_t eq_seen = 0;
    const int64_t eq_admit = adm[blockIdx.x];
    for (int64_t base = e0; base < e1; base += blockDim.x) {
        const int64_t e = base + threadIdx.x;
        const bool in = e < e1;
        const float v = in ? V[e] : 0.f;
        const uint32_t key = abs_key(v);
        const bool is_gt = in && key > tau;
        const bool is_eq = in && want_eq && key == tau;
        // rank of this tie among the workgroup's ties so far
        const uint64_t meq = __ballot(is_eq);
        if (lane == 0) weq[wave] = __popcll(meq);
        __syncthreads();
        int eq_before = __popcll(meq & below);
        for (int w = 0; w < wave; ++w) eq_before += weq[w];
        int eq_tile = weq[0] + weq[1] + weq[2] + weq[3];
        const bool sel = (is_gt || (is_eq && eq_seen + eq_before < eq_admit));
        const uint64_t msel = __ballot(sel);
        if (lane == 0) wsel[wave] = __popcll(msel);
        __syncthreads();
        int sel_before = __popcll(msel & below);
        for (int w = 0; w < wave; ++w) sel_before += wsel[w];
        const int sel_tile = wsel[0] + wsel[1] + wsel[2] + wsel[3];
        if (sel && pos + sel_before < cap) {
            idx_out[pos + sel_before] = e;
            if (val_out) val_out[pos + sel_before] = v;
        }
        if (in && dense_out) dense_out[e] = sel ? v : 0.f;
        pos += sel_tile;
        eq_seen += eq_tile;
        __syncthreads();
    }
}

// Radix select + compaction over `count` values.  idx/val receive the
// support (val may be null); dense (may be null) receives P_s(V).  With
// `hist0_done`, the first-digit histogram was already accumulated into
// `hist` (by the kernel that produced V) after sel_init_kernel cleared it.
static void select_init(SelState* st, int64_t k, uint32_t* hist, const int* status, hipStream_t hs)
{
    hipLaunchKernelGGL(sel_init_kernel, dim3(1), dim3(256), 0, hs, st, k, hist, status);
}

static qe_status run_select(const float* V, int64_t count, int64_t s, SelState* st,
                            uint32_t* hist, int64_t* cnt, int64_t* off, int64_t* adm,
                            int64_t* idx, float* val, float* dense, int64_t* nnz_out,
                            const int* status, hipStream_t hs, bool hist0_done = false)
{
    const int64_t k = s < count ? s : count;
    if (!hist0_done) select_init(st, k, hist, status, hs);
    const int shifts[3] = {21, 10, 0};
    const int bits[3] = {11, 11, 10};
    const int hist_wgs = (int)std::min<int64_t>(kSelWgs, std::max<int64_t>(1, cdiv(count, 1024)));
    const int vec4 = aligned16(V) ? 1 : 0;
    for (int pass = 0; pass < 3; ++pass) {
        if (pass > 0 || !hist0_done)
            hipLaunchKernelGGL(sel_hist_kernel, dim3(hist_wgs), dim3(256), 0, hs, V, count,
                               shifts[pass], bits[pass], pass == 0 ? 1 : 0, vec4, st, hist,
                               status);
        hipLaunchKernelGGL(sel_pick_kernel, dim3(1), dim3(256), 0, hs, st, hist, bits[pass],
                           pass == 2 ? 1 : 0, status);
    }
    const int64_t chunk = cdiv(count, kSelWgs);
    hipLaunchKernelGGL(sel_count_kernel, dim3(kSelWgs), dim3(256), 0, hs, V, count, chunk, st, cnt,
                       status);
    hipLaunchKernelGGL(sel_scan_kernel, dim3(1), dim3(256), 0, hs, cnt, k, st, off, adm, nnz_out,
                       status);
    hipLaunchKernelGGL(sel_write_kernel, dim3(kSelWgs), dim3(256), 0, hs, V, count, chunk, st, off,
                       adm, k, idx, val, dense, status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

struct SelBufs {
    SelState* st;
    uint32_t* hist;
    int64_t* cnt;
    int64_t* off;
    int64_t* adm;
};

static SelBufs take_sel(Ws& w)
{
    SelBufs b;
    b.st = w.take<SelState>(1);
    b.hist = w.take<uint32_t>(kHistBins);
    b.cnt = w.take<int64_t>(2 * kSelWgs);
    b.off = w.take<int64_t>(kSelWgs);
    b.adm = w.take<int64_t>(kSelWgs);
    return b;
}

static size_t sel_bytes()
{
    return align256(sizeof(SelState)) + align256(sizeof(uint32_t) * kHistBins) +
           align256(sizeof(int64_t) * 2 * kSelWgs) + 2 * align256(sizeof(int64_t) * kSelWgs);
}

__global__ void set_i64_kernel(int64_t* p, int64_t v)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) *p = v;
}

__global__ void fill_f32_kernel(float* p, int64_t n, float v)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x)
        p[e] = v;
}

size_t topk_ws_bytes(int64_t, int64_t) { return kStatusBytes + sel_bytes(); }

qe_status launch_topk(const float* V, int64_t count, int64_t s, float* out, int64_t* support,
                      int64_t* nnz, void* ws, hipStream_t hs)
{
    const int* status = static_cast<const int*>(ws);
    if (s == 0 || count == 0) {
        hipLaunchKernelGGL(set_i64_kernel, dim3(1), dim3(64), 0, hs, nnz, (int64_t)0);
        if (count > 0)
            hipLaunchKernelGGL(fill_f32_kernel, dim3(1024), dim3(256), 0, hs, out, count, 0.f);
        return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
    }
    Ws w(ws);
    SelBufs b = take_sel(w);
    return run_select(V, count, s, b.st, b.hist, b.cnt, b.off, b.adm, support, nullptr, out, nnz,
                      status, hs);
}

// ---------------------------------------------------------------- IHT step
// V = H - E / lambda (Sec. 4.3: eta = 1 / (2 lambda_max), gradient 2E), and
// the first-digit histogram of |V| for the radix select in the same pass.
__global__ __launch_bounds__(256) void iht_target_kernel(const float* __restrict__ H,
                                                         const float* __restrict__ E,
                                                         float lambda, float* V, int64_t n,
                                                         int vec4, uint32_t* hist,
                                                         const int* status)
{
    if (failed(status)) return;
    __shared__ uint32_t h[kHistBins];
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x) h[b] = 0u;
    __syncthreads();
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t tail = 0;
    if (vec4) {
        const int64_t n4 = n / 4;
        const f32x4* H4 = reinterpret_cast<const f32x4*>(H);
        const f32x4* E4 = reinterpret_cast<const f32x4*>(E);
        f32x4* V4 = reinterpret_cast<f32x4*>(V);
#pragma unroll 2
        for (int64_t e = tid; e < n4; e += G) {
            const f32x4 hv = H4[e], ev = E4[e];
            f32x4 v;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                v[u] = hv[u] - ev[u] / lambda;
                if (hist) atomicAdd(&h[abs_key(v[u]) >> 21], 1u);
            }
            V4[e] = v;
        }
        tail = n4 * 4;
    }
    for (int64_t e = tail + tid; e < n; e += G) {
        const float v = H[e] - E[e] / lambda;
        if (hist) atomicAdd(&h[abs_key(v) >> 21], 1u);
        V[e] = v;
    }
    if (!hist) return;
    __syncthreads();
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x)
        if (h[b]) atomicAdd(&hist[b], h[b]);
}

// rowptr[i] = first list position whose linear index is >= i * p (i = 0..q).
__global__ void rowptr_kernel(const int64_t* idx, const int64_t* nnz_p, int64_t q, int64_t p,
                              int64_t* rowptr, const int* status)
{
    if (failed(status)) return;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i > q) return;
    const int64_t key = i * p;
    int64_t lo = 0, hi = *nnz_p;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (idx[mid] < key) lo = mid + 1; else hi = mid;
    }
    rowptr[i] = lo;
}

// val[e] = H[idx[e]] for the caller-provided support.
// A caller-provided support is trusted only as far as the buffers allow: its
// size is clamped to the capacity and out-of-range indices read as 0.
__global__ void gather_kernel(const float* H, const int64_t* idx, int64_t* nnz_p, int64_t cap,
                              int64_t count, float* val, const int* status)
{
    if (failed(status)) return;
    int64_t n = *nnz_p;
    if (n < 0) n = 0;
    if (n > cap) n = cap;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = idx[e];
        val[e] = (k >= 0 && k < count) ? H[k] : 0.f;
    }
    __syncthreads();
    if (blockIdx.x == 0 && threadIdx.x == 0) *nnz_p = n;
}

// Merges the old support (values negated) and the new support into one list
// sorted by linear index, an old entry before a new one with the same index.
// Each entry finds its place by one binary search in the other list.
// Entries [cap, 2 cap) of the thread range stand for the new list.
__device__ inline int64_t count_below(const int64_t* a, int64_t n, int64_t key, bool inclusive)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (a[mid] < key || (inclusive && a[mid] == key)) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(256) void merge_supports_kernel(
    const int64_t* __restrict__ oidx, const float* __restrict__ oval, const int64_t* on_p,
    const int64_t* __restrict__ nidx, const float* __restrict__ nval, const int64_t* nn_p,
    int64_t cap, int64_t* midx, float* mval, int64_t* mcount, const int* status)
{
    if (failed(status)) return;
    const int64_t no = min(max(*on_p, (int64_t)0), cap), nn = min(max(*nn_p, (int64_t)0), cap);
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e == 0) *mcount = no + nn;
    if (e < cap) {
        if (e >= no) return;
        const int64_t k = oidx[e];
        const int64_t pos = e + count_below(nidx, nn, k, false);
        midx[pos] = k;
        mval[pos] = -oval[e];
    } else if (e < 2 * cap) {
        const int64_t b = e - cap;
        if (b >= nn) return;
        const int64_t k = nidx[b];
        const int64_t pos = b + count_below(oidx, no, k, true);
        midx[pos] = k;
        mval[pos] = nval[b];
    }
}

// E_i += sum_k (Hnew_ik - Hold_ik) Sigma_k,:  from the merged list, in
// ascending k per row (a deterministic order).  Workgroup = 16 rows x 128
// columns: lanes 16 r .. 16 r + 15 (one DPP row) own row r; lane g holds
// columns 4 g .. 4 g + 3 and 64 + 4 g .. 64 + 4 g + 3 of the block, so that the
// 16 lanes of each 16-byte load cover whole cache lines of a Sigma row.
// A batch of 16 list entries is fetched one per lane; the first entry of an
// (old, new) pair carries new - old, its partner 0.  Entries are then taken
// in order, broadcast with DPP, and each lane applies one Sigma row segment.
// Workgroups are handed out column block by column block per XCD (8 XCDs
// take workgroups round-robin), so a 2 MB column slice of Sigma is shared in
// each XCD's L2 by all row tiles.  Indices outside row i are ignored.
constexpr int kSpRows = 16;
constexpr int kSpCols = 128;

template <int O>
__device__ __forceinline__ int row_bcast_i(int v)
{
    return __builtin_amdgcn_mov_dpp(v, 0x150 + O, 0xF, 0xF, false);
}
template <int O>
__device__ __forceinline__ float row_bcast_f(float v)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x150 + O, 0xF, 0xF, false));
}

// One batch: the 16 broadcast entries' Sigma segments are fetched first (a
// row whose entry carries 0 issues no load: its lanes are masked off), then
// applied in list order.
template <int... Us>
__device__ __forceinline__ void spmm_batch(std::integer_sequence<int, Us...>, float (&acc)[8],
                                           float dd, int col, const float* Sigma, int64_t p,
                                           int64_t c0, bool full)
{
    constexpr int N = sizeof...(Us);
    const float du[N] = {row_bcast_f<Us>(dd)...};
    const int cu[N] = {row_bcast_i<Us>(col)...};
    f32x4 sa[N], sb[N];
#pragma unroll
    for (int u = 0; u < N; ++u) {
        sa[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        sb[u] = sa[u];
        if (du[u] != 0.f) {
            const float* src = Sigma + (int64_t)cu[u] * p + c0;
            if (full) {
                sa[u] = *reinterpret_cast<const f32x4*>(src);
                sb[u] = *reinterpret_cast<const f32x4*>(src + kSpCols / 2);
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sa[u][e] = c0 + e < p ? src[e] : 0.f;
                    sb[u][e] = c0 + kSpCols / 2 + e < p ? src[kSpCols / 2 + e] : 0.f;
                }
            }
        }
    }
#pragma unroll
    for (int u = 0; u < N; ++u) {
        if (du[u] != 0.f) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[e] = fmaf(du[u], sa[u][e], acc[e]);
                acc[4 + e] = fmaf(du[u], sb[u][e], acc[4 + e]);
            }
        }
    }
}

__global__ __launch_bounds__(256) void spmm_delta_kernel(const int64_t* __restrict__ midx,
                                                         const float* __restrict__ mval,
                                                         const int64_t* __restrict__ mrp,
                                                         const float* __restrict__ Sigma,
                                                         int64_t q, int64_t p, int64_t n_rt,
                                                         int64_t n_cb, int vec4, float* E,
                                                         const int* status)
{
    if (failed(status)) return;
    const int64_t work = n_rt * n_cb;
    const int64_t per = cdiv(work, 8);
    const int64_t w = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (w >= work) return;
    const int64_t cb = w / n_rt, rt = w % n_rt;
    const int r = threadIdx.x >> 4, g = threadIdx.x & 15;
    const int64_t i = rt * kSpRows + r;
    const int64_t c0 = cb * kSpCols + 4 * g;
    const bool rowok = i < q;
    const int64_t m0 = rowok ? mrp[i] : 0, m1 = rowok ? mrp[i + 1] : 0;
    const int64_t len = m1 > m0 ? m1 - m0 : 0;
    int64_t wl = len;   // longest stretch among the wave's four rows (wave-uniform)
#pragma unroll
    for (int off = 16; off < 64; off <<= 1) {
        const int64_t o = __shfl_xor(wl, off, 64);
        wl = o > wl ? o : wl;
    }
    if (wl == 0) return;
    const bool full = vec4 && cb * kSpCols + kSpCols <= p;
    float* erow = E + i * p + c0;
    // acc[e]: column c0 + e (e < 4) or c0 + 64 + e - 4
    auto coff = [](int e) { return e < 4 ? e : kSpCols / 2 - 4 + e; };
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = (len > 0 && c0 + coff(e) < p) ? erow[coff(e)] : 0.f;
    const int64_t rlo = i * p, rhi = rlo + p;
    // lane g's entry of the batch at `base`: (delta, Sigma row), 0 if none
    auto fetch = [&](int64_t base, float& dd, int& col) {
        const int64_t m = m0 + base + g;
        dd = 0.f;
        col = 0;
        if (m < m1) {
            const int64_t k = midx[m];
            const float d0 = mval[m];
            const int64_t kp = m > m0 ? midx[m - 1] : -1;
            int64_t kn = -1;
            float d1 = 0.f;
            if (m + 1 < m1) {
                kn = midx[m + 1];
                d1 = mval[m + 1];
            }
            const float d = kn == k ? d0 + d1 : d0;
            if (kp != k && d != 0.f && k >= rlo && k < rhi) {
                dd = d;
                col = (int)(k - rlo);
            }
        }
    };
    float dd, dn = 0.f;
    int col, cn = 0;
    fetch(0, dd, col);
    for (int64_t base = 0; base < wl; base += 16) {
        if (base + 16 < wl) fetch(base + 16, dn, cn);   // next batch in flight
        // entries past a row's stretch carry 0
        spmm_batch(std::make_integer_sequence<int, 8>{}, acc, dd, col, Sigma, p, c0, full);
        spmm_batch(std::integer_sequence<int, 8, 9, 10, 11, 12, 13, 14, 15>{}, acc, dd, col, Sigma,
                   p, c0, full);
        dd = dn;
        col = cn;
    }
    if (len > 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (c0 + coff(e) < p) erow[coff(e)] = acc[e];
    }
}

// ---------------------------------------------------------------- structured projection
// "Structured Outliers" (Sec. 4.3): keep the floor(s / q) whole columns of V
// with the largest l2 norm.  Key of column j: sum_i V_ij^2 in fp64 (row
// chunks summed in a fixed order), rounded to fp32; the columns are then
// chosen by the radix select above (ties: lower column first; all-zero
// columns never kept), and the kept columns are expanded into the dense
// result and the ascending list of their entries.
constexpr int kColChunkRows = 256;

__global__ __launch_bounds__(256) void colnorm_partial_kernel(const float* __restrict__ V,
                                                              int64_t q, int64_t p,
                                                              double* part, const int* status)
{
    if (failed(status)) return;
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= p) return;
    const int64_t r0 = (int64_t)blockIdx.y * kColChunkRows;
    const int64_t r1 = min(q, r0 + kColChunkRows);
    double acc = 0.0;
    for (int64_t i = r0; i < r1; ++i) {
        const double v = (double)V[i * p + c];
        acc += v * v;
    }
    part[(int64_t)blockIdx.y * p + c] = acc;
}

__global__ __launch_bounds__(256) void colnorm_key_kernel(const double* __restrict__ part,
                                                          int nchunks, int64_t p, float* key,
                                                          uint8_t* mask, const int* status)
{
    if (failed(status)) return;
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= p) return;
    double acc = 0.0;
    for (int k = 0; k < nchunks; ++k) acc += part[(int64_t)k * p + c];
    key[c] = (float)acc;
    mask[c] = 0;
}

__global__ void colmask_kernel(const int64_t* cols, const int64_t* ncols_p, int64_t p,
                               uint8_t* mask, const int* status)
{
    if (failed(status)) return;
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= *ncols_p) return;
    const int64_t c = cols[k];
    if (c >= 0 && c < p) mask[c] = 1;
}

// dense result, and (idx, val) of every entry of the kept columns, ascending
__global__ __launch_bounds__(256) void colexpand_kernel(const float* __restrict__ V, int64_t q,
                                                        int64_t p, const uint8_t* __restrict__ mask,
                                                        const int64_t* __restrict__ cols,
                                                        const int64_t* ncols_p, int64_t cap,
                                                        float* dense, int64_t* idx, float* val,
                                                        int64_t* nnz, const int* status)
{
    if (failed(status)) return;
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (dense)
        for (int64_t i = blockIdx.x; i < q; i += gridDim.x)
            for (int64_t c = threadIdx.x; c < p; c += blockDim.x)
                dense[i * p + c] = mask[c] ? V[i * p + c] : 0.f;
    const int64_t nc = *ncols_p;
    const int64_t total = nc > 0 ? min(q * nc, cap) : 0;
    for (int64_t e = tid; e < total; e += G) {
        const int64_t i = e / nc, c = cols[e % nc];
        idx[e] = i * p + c;
        if (val) val[e] = V[i * p + c];
    }
    if (tid == 0 && nnz) *nnz = total;
}

struct ColBufs {
    double* part;
    float* key;
    uint8_t* mask;
    int64_t* cols;
    int64_t* ncols;
};

static size_t col_bytes(int64_t q, int64_t p)
{
    const int64_t nch = cdiv(q, kColChunkRows);
    return align256(sizeof(double) * nch * p) + align256(sizeof(float) * p) + align256(p) +
           align256(sizeof(int64_t) * p) + align256(sizeof(int64_t));
}

static ColBufs take_col(Ws& w, int64_t q, int64_t p)
{
    ColBufs b;
    b.part = w.take<double>(cdiv(q, kColChunkRows) * p);
    b.key = w.take<float>(p);
    b.mask = w.take<uint8_t>(p);
    b.cols = w.take<int64_t>(p);
    b.ncols = w.take<int64_t>(1);
    return b;
}

// columns: the kept column list (ascending, device) may be b.cols itself
static qe_status run_select_columns(const float* V, int64_t q, int64_t p, int64_t c,
                                    const SelBufs& sb, const ColBufs& cb, float* dense,
                                    int64_t* idx, float* val, int64_t* nnz, int64_t cap,
                                    const int* status, hipStream_t hs)
{
    const int nch = (int)cdiv(q, kColChunkRows);
    hipLaunchKernelGGL(colnorm_partial_kernel, dim3((unsigned)cdiv(p, 256), (unsigned)nch),
                       dim3(256), 0, hs, V, q, p, cb.part, status);
    hipLaunchKernelGGL(colnorm_key_kernel, dim3((unsigned)cdiv(p, 256)), dim3(256), 0, hs,
                       cb.part, nch, p, cb.key, cb.mask, status);
    if (c > 0) {
        const qe_status st = run_select(cb.key, p, c, sb.st, sb.hist, sb.cnt, sb.off, sb.adm,
                                        cb.cols, nullptr, nullptr, cb.ncols, status, hs);
        if (st != QE_OK) return st;
    } else {
        hipLaunchKernelGGL(set_i64_kernel, dim3(1), dim3(64), 0, hs, cb.ncols, (int64_t)0);
    }
    hipLaunchKernelGGL(colmask_kernel, dim3((unsigned)cdiv(p, 256)), dim3(256), 0, hs, cb.cols,
                       cb.ncols, p, cb.mask, status);
    hipLaunchKernelGGL(colexpand_kernel, dim3(2048), dim3(256), 0, hs, V, q, p, cb.mask, cb.cols,
                       cb.ncols, cap, dense, idx, val, nnz, status);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

size_t topk_columns_ws_bytes(int64_t q, int64_t p) { return kStatusBytes + sel_bytes() + col_bytes(q, p); }

qe_status launch_topk_columns(const float* V, int64_t q, int64_t p, int64_t c, float* out,
                              int64_t* columns, int64_t* support, int64_t* nnz, void* ws,
                              hipStream_t hs)
{
    const int* status = static_cast<const int*>(ws);
    Ws w(ws);
    SelBufs sb = take_sel(w);
    ColBufs cb = take_col(w, q, p);
    const qe_status st = run_select_columns(V, q, p, c, sb, cb, out, support, nullptr, nnz,
                                            q * c, status, hs);
    if (st != QE_OK) return st;
    if (columns && c > 0 &&
        hipMemcpyAsync(columns, cb.cols, sizeof(int64_t) * c, hipMemcpyDeviceToDevice, hs) !=
            hipSuccess)
        return QE_ERR_HIP;
    return QE_OK;
}

size_t outlier_ws_bytes(int64_t q, int64_t p, int block, int64_t s)
{
    const int64_t cap = s > 0 ? s : 1;
    size_t b = cd_ws_bytes(q, p, block);
    b += align256(sizeof(float) * q * p);                         // V
    b += sel_bytes();
    b += 2 * (align256(sizeof(int64_t) * cap) + align256(sizeof(float) * cap));  // two supports
    b += align256(sizeof(int64_t) * 2 * cap) + align256(sizeof(float) * 2 * cap);  // merged list
    b += align256(sizeof(int64_t) * (q + 1));                     // its row pointers
    b += 3 * align256(sizeof(int64_t));                           // list sizes
    b += align256(sizeof(double) * kObjBlocks);                   // objective partials
    b += col_bytes(q, p);                                         // structured projection
    return b;
}

qe_status launch_outlier(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                         const float* scale, const float* zero, float* Wh, uint8_t* codes,
                         float* H, float* E, int64_t s, float lambda, int64_t* support,
                         int64_t* support_nnz, int sweeps, int block, uint32_t flags,
                         double* obj, void* ws, hipStream_t hs)
{
    const int* status = static_cast<const int*>(ws);
    const int64_t n = q * p;
    const int64_t cap = s > 0 ? s : 1;
    Ws w(ws);
    w.off = cd_ws_bytes(q, p, block);
    float* V = w.take<float>(n);
    SelBufs sb = take_sel(w);
    int64_t* idx[2] = {w.take<int64_t>(cap), nullptr};
    float* val[2] = {w.take<float>(cap), nullptr};
    idx[1] = w.take<int64_t>(cap);
    val[1] = w.take<float>(cap);
    int64_t* midx = w.take<int64_t>(2 * cap);
    float* mval = w.take<float>(2 * cap);
    int64_t* mrp = w.take<int64_t>(q + 1);
    int64_t* cnt[2] = {w.take<int64_t>(1), w.take<int64_t>(1)};
    int64_t* mcount = w.take<int64_t>(1);
    double* opart = w.take<double>(kObjBlocks);
    ColBufs cb = take_col(w, q, p);
    const bool columns = (flags & QE_OUTLIER_COLUMNS) != 0;
    const int vec4 = (aligned16(H) && aligned16(E) && aligned16(V)) ? 1 : 0;
    const int sig_vec4 = (aligned16(Sigma) && p % 4 == 0) ? 1 : 0;
    const int64_t n_rt = cdiv(q, kSpRows), n_cb = cdiv(p, kSpCols);
    const int64_t sp_grid = 8 * cdiv(n_rt * n_cb, 8);

    // current support = the caller's (e.g. P_s(W) for the initialisation)
    if (hipMemcpyAsync(cnt[0], support_nnz, sizeof(int64_t), hipMemcpyDeviceToDevice, hs) !=
        hipSuccess)
        return QE_ERR_HIP;
    if (s > 0) {
        if (hipMemcpyAsync(idx[0], support, sizeof(int64_t) * s, hipMemcpyDeviceToDevice, hs) !=
            hipSuccess)
            return QE_ERR_HIP;
        hipLaunchKernelGGL(gather_kernel, dim3(256), dim3(256), 0, hs, H, idx[0], cnt[0], cap, n,
                           val[0], status);
    }
    int cur = 0;
    for (int it = 0; it < sweeps; ++it) {
        const uint32_t f = it == 0 ? (flags & ~QE_OUTLIER_COLUMNS)
                                   : (QE_R_VALID | QE_CODES_VALID |
                                      (flags & (QE_CD_FP32 | QE_CD_DENSE)));
        // the CD sweep's objective builds on g after the previous IHT step
        qe_status st = launch_cd(W, Sigma, q, p, bits, scale, zero, Wh, codes, E, H, 1, block, f,
                                 obj ? obj + 2 * it : nullptr, 2,
                                 obj && it > 0 ? obj + 2 * it - 1 : nullptr, ws, hs);
        if (st != QE_OK) return st;
        if (s > 0) {
            const int nxt = cur ^ 1;
            if (columns) {
                hipLaunchKernelGGL(iht_target_kernel, dim3(2048), dim3(256), 0, hs, H, E, lambda,
                                   V, n, vec4, (uint32_t*)nullptr, status);
                st = run_select_columns(V, q, p, s / q, sb, cb, H, idx[nxt], val[nxt], cnt[nxt],
                                        cap, status, hs);
            } else {
                select_init(sb.st, s < n ? s : n, sb.hist, status, hs);
                hipLaunchKernelGGL(iht_target_kernel, dim3(2048), dim3(256), 0, hs, H, E, lambda,
                                   V, n, vec4, sb.hist, status);
                st = run_select(V, n, s, sb.st, sb.hist, sb.cnt, sb.off, sb.adm, idx[nxt],
                                val[nxt], H, cnt[nxt], status, hs, true);
            }
            if (st != QE_OK) return st;
            hipLaunchKernelGGL(merge_supports_kernel, dim3((unsigned)cdiv(2 * cap, 256)),
                               dim3(256), 0, hs, idx[cur], val[cur], cnt[cur], idx[nxt], val[nxt],
                               cnt[nxt], cap, midx, mval, mcount, status);
            hipLaunchKernelGGL(rowptr_kernel, dim3((unsigned)cdiv(q + 1, 256)), dim3(256), 0, hs,
                               midx, mcount, q, p, mrp, status);
            hipLaunchKernelGGL(spmm_delta_kernel, dim3((unsigned)sp_grid), dim3(256), 0, hs, midx,
                               mval, mrp, Sigma, q, p, n_rt, n_cb, sig_vec4, E, status);
            cur = nxt;
        }
        if (obj) {
            // g after the IHT step: <What + H - W, E>
            st = launch_residual_dot(W, Wh, H, E, n, obj + 2 * it + 1, opart, status, hs);
            if (st != QE_OK) return st;
        }
        if (hipGetLastError() != hipSuccess) return QE_ERR_HIP;
    }
    if (s > 0) {
        if (hipMemcpyAsync(support, idx[cur], sizeof(int64_t) * s, hipMemcpyDeviceToDevice, hs) !=
            hipSuccess)
            return QE_ERR_HIP;
    }
    if (hipMemcpyAsync(support_nnz, cnt[cur], sizeof(int64_t), hipMemcpyDeviceToDevice, hs) !=
        hipSuccess)
        return QE_ERR_HIP;
    return QE_OK;
}

}  // namespace qe
