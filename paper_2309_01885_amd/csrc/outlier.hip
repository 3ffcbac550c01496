// Outlier-aware QuantEase (Sec. 5) on gfx950: P_s by radix select, the IHT
// step and the sparse residual update.
//
// P_s (Sec. 5.3) keeps the s entries of largest |v|.  |v| of an fp32 value is
// ordered exactly like its bit pattern with the sign cleared, so the s-th
// largest key tau is found by a 3-pass radix select (digits of 11, 11 and 10
// bits; per-workgroup LDS histograms merged with integer atomics, so counts
// are exact and order-free).  Selected: every key > tau, plus the first
// (s - #{key > tau}) keys == tau in linear-index order; tau == 0 selects no
// zeros.  Compaction keeps index order (per-workgroup counts, a scan, then
// wavefront ballots inside each workgroup), so the support comes out sorted.
//
// IHT step (Sec. 5.3, Lemma 3): V = H - E / lambda_max, H+ = P_s(V), then
// E += (H+ - H) Sigma, gathered per row from the old and new supports.
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
__global__ __launch_bounds__(256) void sel_hist_kernel(const float* __restrict__ V, int64_t count,
                                                       int shift, int dbits, int first,
                                                       const SelState* st, uint32_t* hist,
                                                       const int* status)
{
    if (failed(status)) return;
    __shared__ uint32_t h[kHistBins];
    for (int b = threadIdx.x; b < kHistBins; b += blockDim.x) h[b] = 0u;
    __syncthreads();
    const uint32_t prefix = st->prefix;
    const uint32_t dmask = (1u << dbits) - 1u;
    const int hs = shift + dbits;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < count;
         e += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t key = abs_key(V[e]);
        if (!first && (key >> hs) != prefix) continue;
        atomicAdd(&h[(key >> shift) & dmask], 1u);
    }
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

// Output offset and admitted tie count of every workgroup (sequential scan).
__global__ void sel_scan_kernel(const int64_t* cnt, int nw, int64_t cap, SelState* st,
                                int64_t* off, int64_t* adm, int64_t* nnz_out, const int* status)
{
    if (failed(status)) return;
    if (threadIdx.x != 0) return;
    int64_t need = st->need_eq, pos = 0;
    for (int w = 0; w < nw; ++w) {
        const int64_t take = need < cnt[2 * w + 1] ? need : cnt[2 * w + 1];
        off[w] = pos;
        adm[w] = take;
        pos += cnt[2 * w] + take;
        need -= take;
    }
    if (pos > cap) pos = cap;   // never more than k <= cap by construction; guards the buffers
    st->nnz = pos;
    if (nnz_out) *nnz_out = pos;
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
// support (val may be null); dense (may be null) receives P_s(V).
static qe_status run_select(const float* V, int64_t count, int64_t s, SelState* st,
                            uint32_t* hist, int64_t* cnt, int64_t* off, int64_t* adm,
                            int64_t* idx, float* val, float* dense, int64_t* nnz_out,
                            const int* status, hipStream_t hs)
{
    const int64_t k = s < count ? s : count;
    hipLaunchKernelGGL(sel_init_kernel, dim3(1), dim3(256), 0, hs, st, k, hist, status);
    const int shifts[3] = {21, 10, 0};
    const int bits[3] = {11, 11, 10};
    const int hist_wgs = (int)std::min<int64_t>(kSelWgs, std::max<int64_t>(1, cdiv(count, 256)));
    for (int pass = 0; pass < 3; ++pass) {
        hipLaunchKernelGGL(sel_hist_kernel, dim3(hist_wgs), dim3(256), 0, hs, V, count,
                           shifts[pass], bits[pass], pass == 0 ? 1 : 0, st, hist, status);
        hipLaunchKernelGGL(sel_pick_kernel, dim3(1), dim3(256), 0, hs, st, hist, bits[pass],
                           pass == 2 ? 1 : 0, status);
    }
    const int64_t chunk = cdiv(count, kSelWgs);
    hipLaunchKernelGGL(sel_count_kernel, dim3(kSelWgs), dim3(256), 0, hs, V, count, chunk, st, cnt,
                       status);
    hipLaunchKernelGGL(sel_scan_kernel, dim3(1), dim3(64), 0, hs, cnt, kSelWgs, k, st, off, adm,
                       nnz_out, status);
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
// V = H - E / lambda (Sec. 5.3: eta = 1 / (2 lambda_max), gradient 2E).
__global__ void iht_target_kernel(const float* __restrict__ H, const float* __restrict__ E,
                                  float lambda, float* V, int64_t n, const int* status)
{
    if (failed(status)) return;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x)
        V[e] = H[e] - E[e] / lambda;
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

// E_i += sum_k (Hnew_ik - Hold_ik) Sigma_k,:  over the union of the two sorted
// supports of row i, in ascending k (a deterministic order).  One workgroup
// per row; columns in register chunks of 256 x kSpmmPer.
constexpr int kSpmmPer = 16;

__global__ __launch_bounds__(256) void spmm_delta_kernel(
    const int64_t* __restrict__ oidx, const float* __restrict__ oval, const int64_t* __restrict__ orp,
    const int64_t* __restrict__ nidx, const float* __restrict__ nval, const int64_t* __restrict__ nrp,
    const float* __restrict__ Sigma, int64_t p, float* E, const int* status)
{
    if (failed(status)) return;
    const int64_t i = blockIdx.x;
    const int64_t o0 = orp[i], o1 = orp[i + 1], n0 = nrp[i], n1 = nrp[i + 1];
    if (o0 == o1 && n0 == n1) return;
    const int64_t big = INT64_MAX;
    for (int64_t cbase = 0; cbase < p; cbase += 256 * kSpmmPer) {
        float acc[kSpmmPer];
#pragma unroll
        for (int u = 0; u < kSpmmPer; ++u) {
            const int64_t c = cbase + u * 256 + threadIdx.x;
            acc[u] = c < p ? E[i * p + c] : 0.f;
        }
        int64_t a = o0, b = n0;
        while (a < o1 || b < n1) {
            const int64_t ka = a < o1 ? oidx[a] : big;
            const int64_t kb = b < n1 ? nidx[b] : big;
            int64_t k;
            float d;
            if (ka < kb) {
                k = ka;
                d = -oval[a++];
            } else if (kb < ka) {
                k = kb;
                d = nval[b++];
            } else {
                k = ka;
                d = nval[b++] - oval[a++];
            }
            if (d == 0.f || k < i * p || k >= (i + 1) * p) continue;
            const float* srow = Sigma + (k - i * p) * p;
#pragma unroll
            for (int u = 0; u < kSpmmPer; ++u) {
                const int64_t c = cbase + u * 256 + threadIdx.x;
                if (c < p) acc[u] = fmaf(d, srow[c], acc[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < kSpmmPer; ++u) {
            const int64_t c = cbase + u * 256 + threadIdx.x;
            if (c < p) E[i * p + c] = acc[u];
        }
    }
}

size_t outlier_ws_bytes(int64_t q, int64_t p, int block, int64_t s)
{
    const int64_t cap = s > 0 ? s : 1;
    size_t b = cd_ws_bytes(q, p, block);
    b += align256(sizeof(float) * q * p);                         // V
    b += sel_bytes();
    b += 2 * (align256(sizeof(int64_t) * cap) + align256(sizeof(float) * cap));  // two supports
    b += 2 * align256(sizeof(int64_t) * (q + 1));                 // row pointers
    b += 2 * align256(sizeof(int64_t));                           // their sizes
    b += align256(sizeof(double) * kObjBlocks);                   // objective partials
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
    int64_t* rp[2] = {w.take<int64_t>(q + 1), w.take<int64_t>(q + 1)};
    int64_t* cnt[2] = {w.take<int64_t>(1), w.take<int64_t>(1)};
    double* opart = w.take<double>(kObjBlocks);

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
        const uint32_t f = it == 0 ? flags : (QE_R_VALID | QE_CODES_VALID);
        qe_status st = launch_cd(W, Sigma, q, p, bits, scale, zero, Wh, codes, E, H, 1, block, f,
                                 obj ? obj + 2 * it : nullptr, 2, ws, hs);
        if (st != QE_OK) return st;
        if (s > 0) {
            const int nxt = cur ^ 1;
            hipLaunchKernelGGL(iht_target_kernel, dim3(2048), dim3(256), 0, hs, H, E, lambda, V, n,
                               status);
            st = run_select(V, n, s, sb.st, sb.hist, sb.cnt, sb.off, sb.adm, idx[nxt], val[nxt], H,
                            cnt[nxt], status, hs);
            if (st != QE_OK) return st;
            hipLaunchKernelGGL(rowptr_kernel, dim3((unsigned)cdiv(q + 1, 256)), dim3(256), 0, hs,
                               idx[cur], cnt[cur], q, p, rp[cur], status);
            hipLaunchKernelGGL(rowptr_kernel, dim3((unsigned)cdiv(q + 1, 256)), dim3(256), 0, hs,
                               idx[nxt], cnt[nxt], q, p, rp[nxt], status);
            hipLaunchKernelGGL(spmm_delta_kernel, dim3((unsigned)q), dim3(256), 0, hs, idx[cur],
                               val[cur], rp[cur], idx[nxt], val[nxt], rp[nxt], Sigma, p, E,
                               status);
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
