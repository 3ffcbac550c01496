// fp32 Gram products on the fp16 matrix cores of gfx950 (two-way split of
// power-of-two-scaled channels), on the 256 x 256 tile of eight waves.
//
// Channel i of X is scaled by 2^e_i, exactly, with e_i chosen so that the
// channel's largest |x| lands in [2^14, 2^15) (a pre-pass over X; e_i is
// capped at 127 so that 2^e_i is a normal float, which leaves a channel whose
// largest |x| is below 2^-112 under 2^14 after scaling).  Every
// scaled value y then splits into two fp16 values,
//     h = fp16(y),  m = fp16(y - h),
// with round-to-nearest-even conversions: y - h is exact in fp32 and at most
// 2^-11 |y|, and the remainder y - h - m is at most 2^-22 |y| (at most 2^-25,
// i.e. 2^-39 of the channel's largest value, where y - h is below fp16's
// normal range).  The product of two fp16 values is exact in fp32, and
//     y_i y_j = h_i h_j + (h_i m_j + m_i h_j) + E,
// where the dropped part E (m_i m_j and the products with the remainders) is
// below 3 * 2^-22 |y_i y_j| with random signs.  The three kept products run
// as v_mfma_f32_32x32x16_f16 with fp32 accumulation, half the matrix-core
// work of the six-product bf16 split (nt_x3.h); the tile's sums are scaled
// back by 2^-(e_i + e_j), exactly, before they leave the kernel.
//
// Pipeline as nt_tile_x3_wide: wave (wm, wn) owns rows wm * 64 + 32 mi and
// columns wn * 128 + 32 ni of the tile, K in stages of 16 through three or
// four LDS stage buffers (one barrier per stage, or per two), global loads
// three stages ahead.
// Per operand and stage the LDS holds 256 rows of 16 dwords: four 16-byte
// slots (plane 2 p + half, each 8 k values of one plane) whose order is
// permuted by row bits 1 to 3, so that any 4, 8 or 16 consecutive lanes of an
// operand read (consecutive rows, one slot) or of a staging write (row pairs,
// both halves of one plane) touch distinct 16-byte bank groups: conflict-free
// whether the 16-byte accesses are served 4, 8 or 16 lanes at a time.
#pragma once

#include <utility>

#include "nt_x3.h"

namespace qe {

constexpr int kF2RowDw = 16;                      // h, m: 8 dwords each
constexpr int kF2OpDw = 256 * kF2RowDw;           // one operand of one stage
constexpr int kF2BufDw = 2 * kF2OpDw;             // A and B of one stage

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// Slot permutation of a row (b_k: row bit k): bit 1 = b2 ^ b1, bit 0 = b3 ^ b1.
__device__ inline int f2_perm(int row)
{
    const int b1 = (row >> 1) & 1;
    return ((((row >> 2) & 1) ^ b1) << 1) | (((row >> 3) & 1) ^ b1);
}

// Dword offset of (row, half, plane) inside one operand's stage area.
__device__ inline int f2_addr(int row, int half, int plane)
{
    return row * kF2RowDw + 4 * ((2 * plane + half) ^ f2_perm(row));
}

// Scales a stage held as thread t (row t / 2, k = 8 (t % 2) .. +7) by the
// power of two sc, splits it and stores one 16-byte half of each plane.  The
// remainder x sc - h is one fused multiply-add with the fp16 h as its addend
// (v_fma_mix_f32): exact, and the same value as (x sc) - h.
__device__ inline void f2_store_row8(uint32_t* op, const X3Stage& st, float sc)
{
    const int t = threadIdx.x;
    u32x4 h, m;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const float x0 = st.v[u >> 1][2 * (u & 1)], x1 = st.v[u >> 1][2 * (u & 1) + 1];
        const f16x2 hh = __builtin_convertvector((f32x2){x0 * sc, x1 * sc}, f16x2);
        const f16x2 mm = __builtin_convertvector(
            (f32x2){fmaf(x0, sc, -(float)hh[0]), fmaf(x1, sc, -(float)hh[1])}, f16x2);
        h[u] = __builtin_bit_cast(uint32_t, hh);
        m[u] = __builtin_bit_cast(uint32_t, mm);
    }
    *reinterpret_cast<u32x4*>(op + f2_addr(t >> 1, t & 1, 0)) = h;
    *reinterpret_cast<u32x4*>(op + f2_addr(t >> 1, t & 1, 1)) = m;
}

// Channel-major operand staged by four lanes per row (512 threads): thread t
// holds rows t / 4 and t / 4 + 128 at k = 4 (t % 4) .. +3, so that each 16-byte
// load instruction of a wave covers 16 rows of 64 contiguous bytes (half the
// cache lines of two lanes per row); sc[h] = 2^e of its two rows.  The planes
// go to LDS as 8-byte pieces (dwords 2 (k % 2) .. +1 of the slot of half
// k / 2), which keep the slot layout's reads and writes conflict-free.
struct F2RowQ {
    const float* base;
    int64_t ld;
    float sc[2];
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const float* src = base + (row0 + (t >> 2)) * ld + k0 + 4 * (t & 3);
        st.v[0] = *reinterpret_cast<const f32x4*>(src);
        st.v[1] = *reinterpret_cast<const f32x4*>(src + 128 * ld);
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int kq = t & 3;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = (t >> 2) + 128 * h;
            u32x2 hp, mp;
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const float x0 = st.v[h][2 * u], x1 = st.v[h][2 * u + 1];
                const f16x2 hh = __builtin_convertvector((f32x2){x0 * sc[h], x1 * sc[h]}, f16x2);
                const f16x2 mm = __builtin_convertvector(
                    (f32x2){fmaf(x0, sc[h], -(float)hh[0]), fmaf(x1, sc[h], -(float)hh[1])}, f16x2);
                hp[u] = __builtin_bit_cast(uint32_t, hh);
                mp[u] = __builtin_bit_cast(uint32_t, mm);
            }
            *reinterpret_cast<u32x2*>(op + f2_addr(r, kq >> 1, 0) + 2 * (kq & 1)) = hp;
            *reinterpret_cast<u32x2*>(op + f2_addr(r, kq >> 1, 1) + 2 * (kq & 1)) = mp;
        }
    }
};

// Token-major operand with X3Col's staging (thread t: channel t / 2 at eight
// tokens), read through a buffer descriptor per stage: one 32-bit offset per
// thread and the token steps as scalar offsets, instead of eight 64-bit
// addresses.  base = the launch's first token row, ld = p; the descriptor
// covers the stage's 16 token rows (reads outside it return 0).
struct F2ColB {
    const float* base;
    int64_t ld;
    float sc;
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float*>(base + k0 * ld), 0, (int)(16 * ld * 4), 0x00020000);
        const int vo = (int)((8 * (t & 1) * ld + row0 + (t >> 1)) * 4);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            st.v[u >> 2][u & 3] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rs, vo, (int)(u * ld * 4), 0));
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const { f2_store_row8(op, st, sc); }
};

__device__ __forceinline__ f16x8 f2_frag(const uint32_t* p)
{
    return __builtin_bit_cast(f16x8, *reinterpret_cast<const u32x4*>(p));
}

// One 32-column block ni of one stage: products mh, hm, hh (A planes m, h, h),
// two MFMAs (mi = 0, 1) each.
__device__ __forceinline__ void f2w_block(const f16x8 (&a)[2][2], const f16x8 (&b)[2],
                                          f32x16 (&acc)[2][4], int ni)
{
    constexpr int PA[3] = {1, 0, 0};
    constexpr int PB[3] = {0, 1, 0};
#pragma unroll
    for (int q = 0; q < 3; ++q)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[mi][PA[q]], b[PB[q]],
                                                                 acc[mi][ni], 0, 0, 0);
}

// Stage c: multiplies the fragments of `cur` (fa and fb[0] arrive holding A
// and B block 0), splits and writes stage c + 2 from (ga, gb) to `wr`, loads
// stage kload into (la, lb), and leaves fa and fb[0] holding the fragments of
// `nxt` (stage c + 1).  offa[pl] / offb[pl]: this lane's plane-pl fragment of
// row block 0 (further blocks of 32 rows keep the slot permutation).
template <bool SYNC, class OA, class OB>
__device__ __forceinline__ void f2w_stage(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                          int64_t kload, const uint32_t* cur, const uint32_t* nxt,
                                          uint32_t* wr, X3Stage& ga, X3Stage& gb, X3Stage& la,
                                          X3Stage& lb, const int (&offa)[2], const int (&offb)[2],
                                          f16x8 (&fa)[2][2], f16x8 (&fb)[2][2], f32x16 (&acc)[2][4])
{
    constexpr int BLK = 32 * kF2RowDw;
    // group 0: global loads, B block 1 reads, split of A (stage c + 2)
    A.load_full(row0a, kload, la);
    B.load_full(row0b, kload, lb);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) fb[1][pl] = f2_frag(cur + offb[pl] + 1 * BLK);
    f2w_block(fa, fb[0], acc, 0);
    A.store(wr, ga);
    __builtin_amdgcn_sched_barrier(0);
    // group 1: B block 2 reads, split of B
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) fb[0][pl] = f2_frag(cur + offb[pl] + 2 * BLK);
    f2w_block(fa, fb[1], acc, 1);
    B.store(wr + kF2OpDw, gb);
    __builtin_amdgcn_sched_barrier(0);
    // group 2: B block 3 reads; with SYNC, the barrier makes the stages written
    // so far visible and ends the reads of the stages multiplied so far
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) fb[1][pl] = f2_frag(cur + offb[pl] + 3 * BLK);
    f2w_block(fa, fb[0], acc, 2);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (SYNC) __syncthreads();
    // group 3: next stage's B block 0 and A fragments, each after its last use
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) fb[0][pl] = f2_frag(nxt + offb[pl]);
    {
        constexpr int PA[3] = {1, 0, 0};
        constexpr int PB[3] = {0, 1, 0};
#pragma unroll
        for (int q = 0; q < 3; ++q) {
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
                acc[mi][3] = __builtin_amdgcn_mfma_f32_32x32x16_f16(fa[mi][PA[q]], fb[1][PB[q]],
                                                                    acc[mi][3], 0, 0, 0);
            if (q == 0 || q == 2) {
                const int pl = PA[q];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) fa[mi][pl] = f2_frag(nxt + offa[pl] + mi * BLK);
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);
}

// Stage s = c + R (c a multiple of the unroll, a multiple of 2 and 3): stage
// s lives in LDS buffer s % NBUF and in register set s % 3; the set that held
// stage s + 1 takes stage s + 4 (a load past the last stage re-reads the last
// stage: in bounds, and it lands in a buffer no stage reads).  Stage s writes
// stage s + 2 into buffer (s + 2) % NBUF.  With three buffers every stage
// ends its reads with a barrier.  With four, only the odd stages do: a stage
// reads its own buffer and (after its third block) the next one's; the next
// stage's buffer was written two stages earlier, before an odd stage's barrier,
// and the buffer a stage writes was last read two stages earlier, before one.
template <int R, int NBUF, class OA, class OB>
__device__ __forceinline__ void f2w_stage_r(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                            int64_t c, int64_t nst, uint32_t* lds,
                                            X3Stage (&ga)[3], X3Stage (&gb)[3],
                                            const int (&offa)[2], const int (&offb)[2],
                                            f16x8 (&fa)[2][2], f16x8 (&fb)[2][2],
                                            f32x16 (&acc)[2][4])
{
    f2w_stage<NBUF == 3 || (R & 1)>(
        A, row0a, B, row0b, min(c + R + 4, nst - 1) * kX3KC, lds + (R % NBUF) * kF2BufDw,
        lds + ((R + 1) % NBUF) * kF2BufDw, lds + ((R + 2) % NBUF) * kF2BufDw, ga[(R + 2) % 3],
        gb[(R + 2) % 3], ga[(R + 1) % 3], gb[(R + 1) % 3], offa, offb, fa, fb, acc);
}

template <int NBUF, class OA, class OB, int... R>
__device__ __forceinline__ void f2w_stages(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                           int64_t c, int64_t nst, uint32_t* lds,
                                           X3Stage (&ga)[3], X3Stage (&gb)[3],
                                           const int (&offa)[2], const int (&offb)[2],
                                           f16x8 (&fa)[2][2], f16x8 (&fb)[2][2],
                                           f32x16 (&acc)[2][4], bool guarded,
                                           std::integer_sequence<int, R...>)
{
    ((!guarded || c + R < nst
          ? f2w_stage_r<R, NBUF>(A, row0a, B, row0b, c, nst, lds, ga, gb, offa, offb, fa, fb, acc)
          : void()),
     ...);
}

// acc += A[row0a.., 0..K) B[row0b.., 0..K)^T (scaled values) on the 256 x 256
// tile of 512 threads; K a positive multiple of 32, every 256-row panel
// inside the matrix, aligned rows.  `lds` holds NBUF * kF2BufDw dwords.  Ends
// with a barrier.
template <int NBUF, class OA, class OB>
__device__ __forceinline__ void nt_tile_f2_wide(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                                int64_t K, uint32_t* lds, f32x16 (&acc)[2][4])
{
    static_assert(NBUF == 3 || NBUF == 4, "three or four stage buffers");
    constexpr int U = NBUF == 3 ? 3 : 12;          // stages per loop trip
    const int64_t nst = K / kX3KC;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int ra = wm * 64 + (lane & 31), rb = wn * 128 + (lane & 31);
    const int offa[2] = {f2_addr(ra, lane >> 5, 0), f2_addr(ra, lane >> 5, 1)};
    const int offb[2] = {kF2OpDw + f2_addr(rb, lane >> 5, 0), kF2OpDw + f2_addr(rb, lane >> 5, 1)};
    X3Stage ga[3], gb[3];
    A.load_full(row0a, 0, ga[0]);
    B.load_full(row0b, 0, gb[0]);
    A.load_full(row0a, kX3KC, ga[1]);
    B.load_full(row0b, kX3KC, gb[1]);
    A.store(lds, ga[0]);
    B.store(lds + kF2OpDw, gb[0]);
    A.load_full(row0a, min<int64_t>(2, nst - 1) * kX3KC, ga[2]);
    B.load_full(row0b, min<int64_t>(2, nst - 1) * kX3KC, gb[2]);
    A.load_full(row0a, min<int64_t>(3, nst - 1) * kX3KC, ga[0]);
    B.load_full(row0b, min<int64_t>(3, nst - 1) * kX3KC, gb[0]);
    A.store(lds + kF2BufDw, ga[1]);
    B.store(lds + kF2BufDw + kF2OpDw, gb[1]);
    __syncthreads();
    f16x8 fa[2][2], fb[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int pl = 0; pl < 2; ++pl) fa[mi][pl] = f2_frag(lds + offa[pl] + mi * 32 * kF2RowDw);
#pragma unroll
    for (int pl = 0; pl < 2; ++pl) fb[0][pl] = f2_frag(lds + offb[pl]);
    constexpr auto all = std::make_integer_sequence<int, U>{};
    int64_t c = 0;
    for (; c + U <= nst; c += U)
        f2w_stages<NBUF>(A, row0a, B, row0b, c, nst, lds, ga, gb, offa, offb, fa, fb, acc, false, all);
    if (c < nst)
        f2w_stages<NBUF>(A, row0a, B, row0b, c, nst, lds, ga, gb, offa, offb, fa, fb, acc, true,
                         std::make_integer_sequence<int, U - 1>{});
    __syncthreads();
}

}  // namespace qe
