// Export of a quantized layer for serving: bit-packed codes and the outliers
// in CSR form.  The paper leaves serving kernels out of scope (Sec. 4.3,
// "Structured Outliers"); the layouts are this library's (see qe.h).
#include "qe_internal.h"

namespace qe {

// One thread per output byte: byte b of row i holds bit positions
// [8 b, 8 b + 8) of the row's stream, code j occupying [j bits, (j+1) bits).
__global__ __launch_bounds__(256) void pack_codes_kernel(const uint8_t* __restrict__ codes,
                                                         int64_t q, int64_t p, int bits,
                                                         int64_t row_bytes, uint8_t* packed)
{
    const int64_t total = q * row_bytes;
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / row_bytes, b = e % row_bytes;
        const int64_t bit0 = 8 * b;
        const uint32_t mask = (1u << bits) - 1u;
        uint32_t out = 0;
        for (int64_t j = bit0 / bits; j < p && j * bits < bit0 + 8; ++j) {
            const uint32_t c = codes[i * p + j] & mask;
            const int64_t sh = j * bits - bit0;          // may be negative for the first code
            out |= sh >= 0 ? (c << sh) : (c >> (-sh));
        }
        packed[e] = (uint8_t)(out & 0xffu);
    }
}

// CSR of the support entries (ascending linear indices) of H.
__global__ __launch_bounds__(256) void csr_kernel(const float* __restrict__ H,
                                                  const int64_t* __restrict__ support,
                                                  const int64_t* nnz_p, int64_t cap, int64_t q,
                                                  int64_t p, int64_t* rowptr, int32_t* cols,
                                                  float* vals)
{
    int64_t n = *nnz_p;
    n = n < 0 ? 0 : (n > cap ? cap : n);
    const int64_t G = (int64_t)gridDim.x * blockDim.x;
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    for (int64_t e = tid; e < n; e += G) {
        int64_t k = support[e];
        k = k < 0 ? 0 : (k >= q * p ? q * p - 1 : k);
        cols[e] = (int32_t)(k % p);
        vals[e] = H[k];
    }
    for (int64_t i = tid; i <= q; i += G) {
        const int64_t key = i * p;
        int64_t lo = 0, hi = n;
        while (lo < hi) {
            const int64_t mid = (lo + hi) >> 1;
            if (support[mid] < key) lo = mid + 1; else hi = mid;
        }
        rowptr[i] = lo;
    }
}

int64_t packed_row_bytes(int64_t p, int bits) { return (p * bits + 7) / 8; }

qe_status launch_pack_codes(const uint8_t* codes, int64_t q, int64_t p, int bits,
                            uint8_t* packed, hipStream_t s)
{
    const int64_t rb = packed_row_bytes(p, bits);
    const int64_t total = q * rb;
    if (total == 0) return QE_OK;
    const unsigned grid = (unsigned)std::min<int64_t>(4096, cdiv(total, 256));
    hipLaunchKernelGGL(pack_codes_kernel, dim3(grid), dim3(256), 0, s, codes, q, p, bits, rb,
                       packed);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

qe_status launch_outliers_csr(const float* H, int64_t q, int64_t p, const int64_t* support,
                              const int64_t* nnz, int64_t cap, int64_t* rowptr, int32_t* cols,
                              float* vals, hipStream_t s)
{
    const unsigned grid = (unsigned)std::min<int64_t>(1024, std::max<int64_t>(1, cdiv(cap, 256)));
    hipLaunchKernelGGL(csr_kernel, dim3(grid), dim3(256), 0, s, H, support, nnz, cap, q, p,
                       rowptr, cols, vals);
    return hipGetLastError() == hipSuccess ? QE_OK : QE_ERR_HIP;
}

}  // namespace qe
