/*
 * qe.h -- C ABI of the MI355X (gfx950) QuantEase hot-path library, libqe.so.
 *
 * QuantEase (arXiv 2309.01885) quantizes one linear layer at a time by
 * minimising f(What) = ||W X - What X||_F^2 over a per-output-channel uniform
 * b-bit grid (Sec. 2.1, problem (1)), with cyclic coordinate descent (Sec. 3)
 * and, optionally, a sparse full-precision outlier matrix H chosen by
 * iterative hard thresholding (Sec. 4).
 *
 * Conventions shared by every entry point:
 *  - Matrices are dense, row-major, contiguous fp32 in DEVICE memory (HBM)
 *    unless stated otherwise: W, What, R/E, H are q x p (q output channels,
 *    p input channels); Sigma is p x p and symmetric; X is p x n or n x p.
 *  - The library never allocates or frees caller memory.  Scratch space comes
 *    from the caller as a device workspace `ws` of at least the size returned
 *    by the matching *_workspace_size query; the first 256 bytes of every
 *    workspace hold a device status word.
 *  - All work is enqueued on `stream` (a hipStream_t; NULL = the default
 *    stream) and is asynchronous.  Host-detectable argument errors return
 *    immediately with nothing enqueued.  Data-dependent errors (a
 *    non-positive diagonal entry of Sigma, a non-finite or non-positive grid
 *    scale) are written to the workspace status word, the remaining kernels
 *    of that call become no-ops, and qe_sync_status() reports them.
 *  - Results are bitwise deterministic for a fixed shape, block width and
 *    flag set (no floating-point atomics anywhere).
 *  - Concurrent calls on different streams need disjoint workspaces and
 *    outputs.
 */
#ifndef QE_H
#define QE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int qe_status;

#define QE_OK              0
#define QE_ERR_ARG         1  /* null pointer, bad size, bits outside [1, 8], ... */
#define QE_ERR_DIAG        2  /* some Sigma_jj <= 0 or not finite (Lemma 1 assumes Sigma_jj > 0) */
#define QE_ERR_SCALE       3  /* some grid scale <= 0 or not finite */
#define QE_ERR_WORKSPACE   4  /* workspace null or smaller than the size query */
#define QE_ERR_HIP         5  /* a HIP runtime call failed */
#define QE_ERR_UNSUPPORTED 6  /* a valid request this library does not implement */
#define QE_ERR_TOO_LARGE   7  /* qe_cd_sweep_noalloc: the sizes need more than its fixed scratch */
#define QE_ERR_NONFINITE   8  /* QE_DEBUG_CHECKS found a NaN or infinity in an input */

/* Layouts of X for qe_gram, optionally or-ed with one of QE_GRAM_FP32 and
 * QE_GRAM_BF16X3 (both at once is QE_ERR_ARG). */
#define QE_LAYOUT_PN 0        /* X is p x n: each channel's n tokens contiguous */
#define QE_LAYOUT_NP 1        /* X is n x p: each token's p channels contiguous */
#define QE_GRAM_FP32 0x100    /* products on the fp32 matrix cores instead of split ones */
#define QE_GRAM_BF16X3 0x200  /* the three-way bf16 split everywhere (no fp16 split) */

/* Flags for qe_cd_sweep / qe_cd_outlier_sweep. */
#define QE_INIT_FROM_W 0x1u   /* start from What = W (Sec. 3.1) or What = W - H (Sec. 4.3);
                                 R (or E) is set to 0; codes are not yet valid */
#define QE_R_VALID     0x2u   /* R (or E) already holds (What [+ H] - W) Sigma: resume */
#define QE_CODES_VALID 0x4u   /* codes hold What's grid codes: the keep-current tie rule of the
                                 modified CD (Sec. 3.3) applies from the first sweep */
/* Relaxed sweeps (Sec. 3.2, "Initialization": some iterations skip the
 * quantization).  With period k in [1, 255], sweeps k, 2k, ... of a call
 * (counted from 1) write the unconstrained minimiser beta of Lemma 1 instead
 * of q_i(beta); the last sweep of a call is never relaxed.  After a relaxed
 * sweep What is off the grid, so the next sweep starts with codes invalid;
 * codes are left as they were during a relaxed sweep. */
#define QE_RELAX_PERIOD(k) ((((uint32_t)(k)) & 0xffu) << 8)
#define QE_RELAX_MASK      0xff00u
/* qe_cd_outlier_sweep only: structured outliers ("Structured Outliers",
 * Sec. 4.3): the projection keeps the floor(s / q) whole columns of largest
 * l2 norm instead of the s largest entries (see qe_topk_columns). */
#define QE_OUTLIER_COLUMNS 0x10u
/* Block-update and residual products on the fp32 matrix cores instead of the
 * default exact three-way bf16 split (the split is described at qe_gram). */
#define QE_CD_FP32 0x20u
/* Checks before the sweeps (the paper asks for checks on the inputs before
 * QuantEase runs, footnote to Lemma 1): every input of the call -- W, Sigma,
 * scale, zero, What unless QE_INIT_FROM_W, R (or E) with QE_R_VALID, and H in
 * the outlier-aware call -- is scanned for NaN and infinity, which sets
 * QE_ERR_NONFINITE (reported by qe_sync_status; the rest of the call does
 * nothing).  One extra read of those arrays (about 30 us at 4096 x 4096).
 * Without the flag only Sigma's diagonal and the grid are checked. */
#define QE_DEBUG_CHECKS 0x40u
/* Every block update on the matrix cores.  By default, from the second sweep
 * on (codes valid), a 128 x 128 tile of the block update whose rows changed
 * few codes in the super-block just finished (at most 64 rows, each at most 32
 * codes) applies only those nonzero code differences, as fp32 FMAs; its
 * other rows' update is exactly 0 and is skipped.  Both forms give R up to
 * fp32 rounding; with this flag R's rounding does not depend on how many
 * codes moved. */
#define QE_CD_DENSE 0x10000u
/* qe_cd_sweep only: obj[0] holds, on entry, the objective f of the incoming
 * What and R (e.g. the last value of the previous call), so that chained
 * calls report f without a pass over R.  Needs obj; not with QE_INIT_FROM_W
 * (QE_ERR_ARG). */
#define QE_OBJ_IN 0x80u

/* Human-readable name of a status code (static string). */
const char* qe_status_string(qe_status s);

/* Library ABI version (increases on any signature change). */
int qe_version(void);

/* Synchronises `stream`, then returns the status word of workspace `ws`
 * (QE_OK if no kernel reported a data error).  Also clears the word. */
qe_status qe_sync_status(void* ws, void* stream);

/* ------------------------------------------------------------------------
 * Gram matrix.  Lemma 1 (Sec. 3.2) works with Sigma = X X^T, whose size is
 * independent of the token count n (Sec. 3.2, "Memory Footprint").
 *   Sigma (+)= X X^T; then, if damp > 0, Sigma_jj += damp * mean_j(Sigma_jj).
 * X: p x n (QE_LAYOUT_PN) or n x p (QE_LAYOUT_NP), fp32, device.
 * Sigma: p x p fp32, device; overwritten (accumulate = 0) or added to
 * (accumulate = 1, for token chunks streamed through several calls; pass
 * damp = 0 on all but the last).  The result is exactly symmetric.
 * Products, by default: when p is a multiple of 256 (at most 2^24), X's rows
 * are 16-byte aligned, n is a multiple of 32 (token-major X: all but its last
 * n % 32 tokens) and either the split partials fit the workspace or
 * n <= 32768 (at very large p, stream longer token ranges in chunks of at
 * most 32768), each channel i is first scaled by 2^e_i (exact; its largest |x|
 * lands in [2^14, 2^15), a pass over X; e_i at most 127) and each scaled value
 * y is split into two fp16 values
 * (h = fp16(y), m = fp16(y - h)); y_i y_j is formed from the three products
 * h h, h m, m h on the fp16 matrix cores, every product exact in fp32, and
 * the sums are scaled back by 2^-(e_i + e_j).  The dropped terms are below
 * 3 * 2^-22 |y_i y_j| (plus 2^-39 of the channels' largest values for the
 * smallest ones).  Otherwise, or with QE_GRAM_BF16X3, each fp32 value x is
 * split exactly into three bf16 values (h = bf16(x), m = bf16(x - h),
 * l = x - h - m) and x_i x_j is formed from the six products h h, h m, m h,
 * h l, m m, l h on the bf16 matrix cores; the dropped terms are below
 * 2^-23 |x_i x_j| (one fp32 rounding).  With QE_GRAM_FP32 the products run
 * on the fp32 matrix cores.  Accumulation: fp32 over short token chunks,
 * chunk sums added in fp32, split partial sums reduced in fp64.
 * ------------------------------------------------------------------------ */
size_t qe_gram_workspace_size(int64_t p, int64_t n);
qe_status qe_gram(const float* X, int64_t p, int64_t n, int layout, float* Sigma,
                  int accumulate, float damp, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Per-row uniform grid Q_i = { scale_i (k - zero_i) : k = 0 .. 2^bits - 1 }
 * (Sec. 2.1: uniformly spaced levels per output channel).  Asymmetric min/max
 * reading: lo = min(0, min_j W_ij), hi = max(0, max_j W_ij), an all-zero row
 * uses [-1, 1]; scale = (hi - lo) / (2^bits - 1), zero = rint(-lo / scale),
 * all in fp32.  Entries with H_ij != 0 are excluded (outlier-aware grid,
 * Sec. 4.3); H may be NULL.
 * W, H: q x p device.  scale, zero: q floats each, device, written.
 * ------------------------------------------------------------------------ */
qe_status qe_grid_minmax(const float* W, const float* H, int64_t q, int64_t p, int bits,
                         float* scale, float* zero, void* stream);

/* ------------------------------------------------------------------------
 * Blocked cyclic coordinate descent (Sec. 3; Lemma 1; the rank-1 identity of
 * Sec. 3.2; Algorithm "QuantEase").
 * Residual form: R = (What - W) Sigma.  For each column j in order, for all
 * rows i at once:  beta = What_ij - R_ij / Sigma_jj;  What_ij <- q_i(beta)
 * (nearest grid level, half to even, a valid equally-near current level is
 * kept, Sec. 3.3);  R += (What_new - What_old)_{:,j} Sigma_{j,:}.
 * Columns are processed in blocks of `block` (0 = 128; one of 16, 32, 64,
 * 128): inside a block the rank-1 updates touch only the block's columns;
 * the accumulated block update is then applied to every column as one
 * matrix-core GEMM.  The result equals the column-by-column algorithm up to
 * floating-point rounding.
 *
 * W:      q x p, device, read (only for R initialisation and the objective).
 * Sigma:  p x p, device, symmetric with Sigma_jj > 0 (else QE_ERR_DIAG).
 * scale, zero: q floats, device (e.g. from qe_grid_minmax); bits in [1, 8].
 * W_hat:  q x p, device, in/out.  codes: q x p uint8, device, in/out.
 * R:      q x p, device, in/out: (What - W) Sigma on exit.
 * sweeps: >= 0 full passes over the columns.
 * flags:  QE_INIT_FROM_W | QE_R_VALID | QE_CODES_VALID | QE_RELAX_PERIOD(k)
 *         | QE_CD_FP32 | QE_CD_DENSE | QE_DEBUG_CHECKS | QE_OBJ_IN.
 *         Without QE_INIT_FROM_W and without QE_R_VALID, R is first
 *         computed as (What - W) Sigma (warm start from any What, Sec. 3.1).
 * obj:    NULL, or device array of `sweeps` doubles receiving
 *         f_k = <What - W, R> = ||(W - What) X||_F^2 after sweep k, formed
 *         as the incoming f plus the exact change of each coordinate move
 *         (Lemma 1's one-dimensional quadratic: delta (2 R_ij + delta
 *         Sigma_jj)), summed in fp64 while the sweep runs, in a fixed order.
 *         The incoming f is 0 with QE_INIT_FROM_W, obj[0] with QE_OBJ_IN,
 *         else one pass <What - W, R> at the start of the call.
 * ------------------------------------------------------------------------ */
size_t qe_cd_workspace_size(int64_t q, int64_t p, int block);
qe_status qe_cd_sweep(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                      const float* scale, const float* zero, float* W_hat, uint8_t* codes,
                      float* R, int sweeps, int block, uint32_t flags, double* obj,
                      void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * qe_cd_sweep without allocation or workspace, for callers that cannot
 * allocate device memory: code under stream/graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Arguments and results as for
 * qe_cd_sweep, except:
 *  - the scratch (the status word, 1/Sigma_jj, 1/scale, the two delta
 *    buffers of q x max(256, block) floats, fp64 partial sums) lives in a
 *    library-owned device array of QE_NOALLOC_SCRATCH_BYTES per GPU, held
 *    until the process ends; the call needs qe_cd_workspace_size(q, p, block)
 *    bytes of it and returns QE_ERR_TOO_LARGE, with nothing enqueued, when
 *    that is more (q up to about 30000 rows at the default block);
 *  - status: NULL, or a device int that receives, in stream order at the
 *    end of the call, the call's data-error status (QE_OK, QE_ERR_DIAG,
 *    QE_ERR_SCALE), as qe_sync_status would report it;
 *  - every call on one GPU uses that GPU's one scratch array: calls that
 *    overlap on one GPU (different streams, host threads) race and must be
 *    serialised by the caller.  Each call clears what it needs cleared.
 * No hipMalloc, hipFree or allocating routine is called; the scratch's
 * device address is looked up once per GPU, on the first call there.
 * ------------------------------------------------------------------------ */
#define QE_NOALLOC_SCRATCH_BYTES (64u << 20)
qe_status qe_cd_sweep_noalloc(const float* W, const float* Sigma, int64_t q, int64_t p, int bits,
                              const float* scale, const float* zero, float* W_hat,
                              uint8_t* codes, float* R, int sweeps, int block, uint32_t flags,
                              double* obj, int* status, void* stream);

/* ------------------------------------------------------------------------
 * Outlier-aware QuantEase (Sec. 4, Algorithm "Outlier-Aware QuantEase").
 * Per iteration: one CD sweep on What with H fixed (linear term from
 * W - H, residual E = (What + H - W) Sigma), then one iterative-hard-
 * thresholding step  H <- P_s(H - eta grad_H g),  grad_H g = 2E,
 * eta = 1 / (2 lambda_max), i.e. V = H - E / lambda_max (fp32); P_s keeps
 * the s entries of largest |V| (ties: lower linear index i*p + j; zeros are
 * never kept); then E += (H_new - H_old) Sigma.
 *
 * H:        q x p dense, device, in/out.
 * E:        q x p, device, in/out (the residual).
 * support:  device int64 array of capacity s, in/out: ascending linear
 *           indices of H's nonzeros.  support_nnz: device int64, in/out.
 * s:        outlier budget, 0 <= s <= q*p.  lambda_max > 0 (qe_lambda_max).
 * flags:    QE_INIT_FROM_W: What = W - H (H and support as given, e.g. from
 *           qe_topk_abs on W, Sec. 4.3 initialisation), E = 0.
 *           QE_R_VALID: E already valid.  QE_CODES_VALID as above.
 *           QE_OUTLIER_COLUMNS: structured outliers (whole columns); start
 *           from qe_topk_columns on W.
 *           Without QE_INIT_FROM_W / QE_R_VALID, E = (What + H - W) Sigma.
 *           QE_CD_FP32, QE_CD_DENSE and QE_DEBUG_CHECKS as for qe_cd_sweep.
 * obj:      NULL or device array of 2*sweeps doubles: obj[2k] = g after the
 *           CD sweep of iteration k (g after the previous IHT step, or at
 *           the start, plus the exact change of the sweep's moves, as for
 *           qe_cd_sweep), obj[2k+1] = g after its IHT step (<What + H - W, E>).
 * scale/zero: the outlier-aware grid (qe_grid_minmax with H excluded).
 * ------------------------------------------------------------------------ */
size_t qe_outlier_workspace_size(int64_t q, int64_t p, int block, int64_t s);
qe_status qe_cd_outlier_sweep(const float* W, const float* Sigma, int64_t q, int64_t p,
                              int bits, const float* scale, const float* zero, float* W_hat,
                              uint8_t* codes, float* H, float* E, int64_t s, float lambda_max,
                              int64_t* support, int64_t* support_nnz, int sweeps, int block,
                              uint32_t flags, double* obj, void* ws, size_t ws_bytes,
                              void* stream);

/* ------------------------------------------------------------------------
 * P_s of Sec. 4.3 on a dense array: keep the s entries largest in absolute
 * value (ties: lower index first; exact zeros never kept).
 * V: `count` floats, device.  out: `count` floats, device: P_s(V).
 * support: device int64[s]: kept indices, ascending.  nnz: device int64.
 * ------------------------------------------------------------------------ */
size_t qe_topk_workspace_size(int64_t count, int64_t s);
qe_status qe_topk_abs(const float* V, int64_t count, int64_t s, float* out, int64_t* support,
                      int64_t* nnz, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Structured projection ("Structured Outliers", Sec. 4.3): keep the c whole
 * columns of the q x p matrix V with the largest l2 norm, zero elsewhere.
 * Selection key of column j: sum_i V_ij^2 accumulated in fp64, rounded to
 * fp32; ties go to the lower column; all-zero columns are never kept.
 * out: q x p floats, device.  columns: NULL or device int64[c]: the kept
 * columns, ascending.  support: device int64[q * c]: linear indices of every
 * entry of the kept columns, ascending (the support format of
 * qe_cd_outlier_sweep).  nnz: device int64: number of support entries
 * (q x number of kept columns).
 * ------------------------------------------------------------------------ */
size_t qe_topk_columns_workspace_size(int64_t q, int64_t p);
qe_status qe_topk_columns(const float* V, int64_t q, int64_t p, int64_t c, float* out,
                          int64_t* columns, int64_t* support, int64_t* nnz, void* ws,
                          size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Exact objective and its normaliser (Sec. 2.1 problem (1); Sec. 3.4 relative
 * calibration error), recomputed from scratch, independent of R:
 *   out[0] = <D, D Sigma> = ||(What + H - W) X||_F^2,  D = What + H - W,
 *   out[1] = <W, W Sigma> = ||W X||_F^2.
 * The products D Sigma use the exact three-way bf16 split (see qe_gram);
 * <D, D Sigma> is summed in fp64.  H may be NULL.  out: device, 2 doubles.
 * ------------------------------------------------------------------------ */
size_t qe_objective_workspace_size(int64_t q, int64_t p);
qe_status qe_objective(const float* W, const float* W_hat, const float* H, const float* Sigma,
                       int64_t q, int64_t p, double* out, void* ws, size_t ws_bytes,
                       void* stream);

/* ------------------------------------------------------------------------
 * lambda_max(Sigma) by the power method (Sec. 4.3: matrix-vector products
 * only, O(p^2) per iteration), returned as an upper bound, since the IHT step
 * 1 / (2 lambda) of Lemma 3 needs lambda >= lambda_max.  Start vector
 * 1/sqrt(p); iterate v_k = S v_{k-1} / |S v_{k-1}|, quotient
 * rho_k = v_k' S v_k / v_k' v_k.  The iteration used is the first whose
 * quotient changed by at most tol (relative) from the previous one, else
 * iteration max_iters; the result is rho + |S v - rho v| / |v| of that
 * iteration (an eigenvalue lies within that radius of rho; v approximates the
 * leading eigenvector), from fp64 sums, widened by a relative 2^-30 and
 * rounded up to fp32.
 * Synchronises `stream` every 32 iterations.
 * lambda_out: HOST float.
 * ------------------------------------------------------------------------ */
size_t qe_lambda_workspace_size(int64_t p);
qe_status qe_lambda_max(const float* Sigma, int64_t p, int max_iters, float tol,
                        float* lambda_out, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Export for serving.  The paper leaves serving kernels out of scope
 * (Sec. 4.3, "Structured Outliers"); these layouts are this library's.
 *
 * qe_pack_codes: each row of the q x p codes (device uint8, values < 2^bits,
 * bits in [1, 8]) becomes one little-endian bit stream of
 * qe_packed_row_bytes(p, bits) bytes (device, out): code j occupies bits
 * [j*bits, (j+1)*bits), bytes are filled from their least significant bit,
 * rows start on a byte boundary.  Higher code bits are ignored.
 *
 * qe_outliers_csr: the support entries of H (q x p, device) as CSR:
 * support = ascending linear indices (device int64, capacity cap), nnz =
 * device int64 count (clamped to [0, cap]); rowptr: device int64[q + 1],
 * cols: device int32[cap], vals: device float[cap] (out).  Out-of-range
 * indices are clamped into the matrix.
 * ------------------------------------------------------------------------ */
int64_t qe_packed_row_bytes(int64_t p, int bits);
qe_status qe_pack_codes(const uint8_t* codes, int64_t q, int64_t p, int bits, uint8_t* packed,
                        void* stream);
qe_status qe_outliers_csr(const float* H, int64_t q, int64_t p, const int64_t* support,
                          const int64_t* nnz, int64_t cap, int64_t* rowptr, int32_t* cols,
                          float* vals, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QE_H */
