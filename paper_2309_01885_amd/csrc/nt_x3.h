// fp32 NT tile products on the bf16 matrix cores of gfx950 (three-way split).
//
// Every fp32 operand x is split exactly into three bf16 values,
//     h = bf16(x),  m = bf16(x - h),  l = x - h - m     (x = h + m + l),
// with round-to-nearest-even conversions: x - h and (x - h) - m are exact
// (Sterbenz), |m| <= 2^-8 |x| and l has at most 8 significant bits, so it is a
// bf16 value.  The product of two bf16 values is exact in fp32, and
//     a b = ha hb + (ha mb + ma hb) + (ha lb + ma mb + la hb) + E,
// where the dropped part E = ma lb + la mb + la lb is below 2^-23 |a b| with a
// random sign, the size of one fp32 rounding.  The six kept products run as
// v_mfma_f32_32x32x16_bf16 with fp32 accumulation: six bf16 passes take 6/16
// of the fp32 matrix-core time of the same tile.
//
// Tile geometry as the fp32 NT tile: C[128 x 128] (+)= A[128 x K] B[128 x K]^T,
// four waves in 2 x 2, each wave a 64 x 64 quarter of 2 x 2 32 x 32 blocks.
// K runs in stages of 16 through a double-buffered LDS area.  Per operand and
// stage the LDS holds 128 rows of 24 dwords: the h, m and l planes of the
// row's 16 values, 8 dwords (two 16-byte halves of 8 values) each.  The half
// index is XOR-ed with bit 3 of the row, which keeps both the 16-byte operand
// reads (16 consecutive rows, one half) and the staging writes (8 rows, both
// halves) free of LDS bank conflicts.  Lane l of a wave reads row l % 32 of a
// block and half l / 32 for both A and B, so the k order inside a stage is the
// same on both sides.
#pragma once

#include "qe_internal.h"

namespace qe {

constexpr int kX3KC = 16;                        // K per stage
constexpr int kX3RowDw = 24;                     // h, m, l: 8 dwords each
constexpr int kX3OpDw = kTile * kX3RowDw;        // one operand of one stage
constexpr int kX3LdsDw = 4 * kX3OpDw;            // A and B, double buffered: 49,152 bytes

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Dword offset of (row, half, plane) inside one operand's stage area.
__device__ inline int x3_addr(int row, int half, int plane)
{
    return row * kX3RowDw + 8 * plane + 4 * (half ^ ((row >> 3) & 1));
}

// Two floats (a: low half, b: high half) as three packed bf16 pairs h, m, l.
struct X3Pair { uint32_t h, m, l; };
__device__ inline X3Pair split3(float a, float b)
{
    X3Pair r;
    r.h = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
    const float ra = a - __uint_as_float(r.h << 16);
    const float rb = b - __uint_as_float(r.h & 0xffff0000u);
    r.m = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){ra, rb}, bf16x2));
    const float la = ra - __uint_as_float(r.m << 16);
    const float lb = rb - __uint_as_float(r.m & 0xffff0000u);
    r.l = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){la, lb}, bf16x2));
    return r;
}

// Staging registers of one operand for one stage (8 floats per thread).
struct X3Stage { f32x4 v[2]; };

// Splits and stores a stage held as thread t: row t / 2, k = 8 (t % 2) .. +7
// (one 16-byte half of each plane).
__device__ inline void x3_store_row8(uint32_t* op, const X3Stage& st)
{
    const int t = threadIdx.x;
    u32x4 h, m, l;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const X3Pair q = split3(st.v[u >> 1][2 * (u & 1)], st.v[u >> 1][2 * (u & 1) + 1]);
        h[u] = q.h;
        m[u] = q.m;
        l[u] = q.l;
    }
    *reinterpret_cast<u32x4*>(op + x3_addr(t >> 1, t & 1, 0)) = h;
    *reinterpret_cast<u32x4*>(op + x3_addr(t >> 1, t & 1, 1)) = m;
    *reinterpret_cast<u32x4*>(op + x3_addr(t >> 1, t & 1, 2)) = l;
}

// Row-major operand, element (r, k) at base[r * ld + k], staged as above.
struct X3Row {
    const float* base;
    int64_t ld, rows, kvalid;
    // whole stage inside the matrix, 16-byte aligned rows
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const float* src = base + (row0 + (t >> 1)) * ld + k0 + 8 * (t & 1);
        st.v[0] = *reinterpret_cast<const f32x4*>(src);
        st.v[1] = *reinterpret_cast<const f32x4*>(src + 4);
    }
    // any stage: elements outside rows x kvalid read as 0
    __device__ inline void load(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t r = row0 + (t >> 1);
        const int64_t k = k0 + 8 * (t & 1);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            st.v[u >> 2][u & 3] = (r < rows && k + u < kvalid) ? base[r * ld + k + u] : 0.f;
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const { x3_store_row8(op, st); }
};

// Row-major operand whose values are exact in bf16 (e.g. small integers: the
// code differences of the CD block update), staged as its h plane only; it
// pairs with the three planes of the other operand (x3_mfma_stage<3>).
struct X1Row : X3Row {
    __device__ inline void store(uint32_t* op, const X3Stage& st) const
    {
        const int t = threadIdx.x;
        u32x4 h;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            h[u] = __builtin_bit_cast(uint32_t, __builtin_convertvector(
                (f32x2){st.v[u >> 1][2 * (u & 1)], st.v[u >> 1][2 * (u & 1) + 1]}, bf16x2));
        *reinterpret_cast<u32x4*>(op + x3_addr(t >> 1, t & 1, 0)) = h;
    }
};

// Row-major operand staged by four lanes per row: with NT threads, thread t
// holds rows t / 4 and t / 4 + NT / 4 at k = 4 (t % 4) .. +3, so that each
// 16-byte load instruction of a wave covers 16 rows of 64 contiguous bytes
// (half as many cache lines per instruction as two lanes per row).  NT / 2
// rows per stage; PLANES = 3 stores h, m and l, PLANES = 1 only h (values
// exact in bf16, such as the code differences of the CD block update).
template <int NT, int PLANES>
struct XRowQ {
    const float* base;
    int64_t ld, rows, kvalid;
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const float* src = base + (row0 + (t >> 2)) * ld + k0 + 4 * (t & 3);
        st.v[0] = *reinterpret_cast<const f32x4*>(src);
        st.v[1] = *reinterpret_cast<const f32x4*>(src + (NT / 4) * ld);
    }
    __device__ inline void load(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t k = k0 + 4 * (t & 3);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int64_t r = row0 + (t >> 2) + h * (NT / 4);
#pragma unroll
            for (int u = 0; u < 4; ++u)
                st.v[h][u] = (r < rows && k + u < kvalid) ? base[r * ld + k + u] : 0.f;
        }
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int kq = t & 3;                    // half kq / 2, dwords 2 (kq % 2) .. +1 of it
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int o = x3_addr((t >> 2) + h * (NT / 4), kq >> 1, 0) + 2 * (kq & 1);
            if constexpr (PLANES == 3) {
                const X3Pair q0 = split3(st.v[h][0], st.v[h][1]);
                const X3Pair q1 = split3(st.v[h][2], st.v[h][3]);
                *reinterpret_cast<u32x2*>(op + o) = u32x2{q0.h, q1.h};
                *reinterpret_cast<u32x2*>(op + o + 8) = u32x2{q0.m, q1.m};
                *reinterpret_cast<u32x2*>(op + o + 16) = u32x2{q0.l, q1.l};
            } else {
                const uint32_t h0 = __builtin_bit_cast(
                    uint32_t, __builtin_convertvector((f32x2){st.v[h][0], st.v[h][1]}, bf16x2));
                const uint32_t h1 = __builtin_bit_cast(
                    uint32_t, __builtin_convertvector((f32x2){st.v[h][2], st.v[h][3]}, bf16x2));
                *reinterpret_cast<u32x2*>(op + o) = u32x2{h0, h1};
            }
        }
    }
};

// Row-major composite operand P1 + P2 - P3 (P2, P3 may be null), e.g.
// What + H - W, staged as X3Row.
struct X3Comp {
    const float *p1, *p2, *p3;
    int64_t ld, rows, kvalid;
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t off = (row0 + (t >> 1)) * ld + k0 + 8 * (t & 1);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4 v = *reinterpret_cast<const f32x4*>(p1 + off + 4 * h);
            if (p2) v = v + *reinterpret_cast<const f32x4*>(p2 + off + 4 * h);
            if (p3) v = v - *reinterpret_cast<const f32x4*>(p3 + off + 4 * h);
            st.v[h] = v;
        }
    }
    __device__ inline void load(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t r = row0 + (t >> 1);
        const int64_t k = k0 + 8 * (t & 1);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            float x = 0.f;
            if (r < rows && k + u < kvalid) {
                const int64_t e = r * ld + k + u;
                x = p1[e];
                if (p2) x = x + p2[e];
                if (p3) x = x - p3[e];
            }
            st.v[u >> 2][u & 3] = x;
        }
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const { x3_store_row8(op, st); }
};

// Transposed operand, element (r, k) at base[k * ld + r] (token-major X),
// for any thread count NT (NT / 2 rows per stage): thread t stages row t / 2
// at k = 8 (t % 2) .. +7, one value per token, so that each 4-byte load
// instruction of a wave covers 32 consecutive rows at two tokens (two whole
// 128-byte lines), and the stage goes to LDS exactly as a row-major one
// (x3_store_row8: 16-byte pieces, consecutive lanes on consecutive pieces of
// a row pair, no bank conflicts).
struct X3Col {
    const float* base;
    int64_t ld, rows, kvalid;
    // whole stage inside the matrix
    __device__ inline void load_full(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const float* src = base + (k0 + 8 * (t & 1)) * ld + row0 + (t >> 1);
#pragma unroll
        for (int u = 0; u < 8; ++u) st.v[u >> 2][u & 3] = src[u * ld];
    }
    // any stage: elements outside rows x kvalid read as 0
    __device__ inline void load(int64_t row0, int64_t k0, X3Stage& st) const
    {
        const int t = threadIdx.x;
        const int64_t r = row0 + (t >> 1);
        const int64_t k = k0 + 8 * (t & 1);
#pragma unroll
        for (int u = 0; u < 8; ++u)
            st.v[u >> 2][u & 3] = (r < rows && k + u < kvalid) ? base[(k + u) * ld + r] : 0.f;
    }
    __device__ inline void store(uint32_t* op, const X3Stage& st) const { x3_store_row8(op, st); }
};

// acc[mi][ni] += A(wave rows mi) B(wave cols ni)^T over one staged K = 16 of
// the 128 x 128 tile: waves form a 2 x 2 grid, wave (wm, wn) owns rows
// wm * 64 + 32 mi and columns wn * 64 + 32 ni (mi, ni < 2).  NP = 6: both
// operands split in three (the six kept products); NP = 3: A exact in bf16
// (its h plane only), B split in three, all three products exact.
template <int NP = 6>
__device__ __forceinline__ void x3_mfma_stage(const uint32_t* sA, const uint32_t* sB,
                                              f32x16 (&acc)[2][2])
{
    static_assert(NP == 6 || NP == 3, "six or three products");
    constexpr int NA = NP == 6 ? 3 : 1;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int r = lane & 31, half = lane >> 5;
    // small terms first
    constexpr int PA[6] = {2, 1, 0, 1, 0, 0};
    constexpr int PB[6] = {0, 1, 2, 0, 1, 0};
    constexpr int QA[3] = {0, 0, 0};
    constexpr int QB[3] = {2, 1, 0};
    bf16x8 a[2][NA], b[2][3];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int pl = 0; pl < NA; ++pl)
            a[i][pl] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(sA + x3_addr(wm * 64 + i * 32 + r, half, pl)));
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int pl = 0; pl < 3; ++pl)
            b[i][pl] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(sB + x3_addr(wn * 64 + i * 32 + r, half, pl)));
    // the four accumulators interleave so that no MFMA waits on the one just issued
#pragma unroll
    for (int q = 0; q < NP; ++q)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 2; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    a[mi][NP == 6 ? PA[q] : QA[q % 3] % NA], b[ni][NP == 6 ? PB[q] : QB[q % 3]],
                    acc[mi][ni], 0, 0, 0);
}

// LDS store instructions of one operand's stage: the four-lanes-per-row
// loaders store 8-byte pieces (two per plane), the others 16-byte ones.
template <class O> struct X3Writes { static constexpr int value = 3; };
template <> struct X3Writes<X1Row> { static constexpr int value = 1; };
template <int NT, int PL> struct X3Writes<XRowQ<NT, PL>> { static constexpr int value = 2 * PL; };
template <class O> constexpr int x3_writes() { return X3Writes<O>::value; }

// Instruction order of one stage when INTERLEAVE is set: the operand reads,
// then the MFMAs, each followed by a few VALU instructions of the next stage's
// split, then the LDS writes, so that the split runs while the matrix cores
// work.
template <int NP = 6, int WRITES = (NP == 6 ? 6 : 4)>
__device__ __forceinline__ void x3_interleave()
{
    // operand reads: A's planes (three, or one with NP = 3) and B's three, per
    // 32-row block; MFMAs 4 NP; LDS writes of the next stage (the operands'
    // store instructions)
    constexpr int reads = NP == 6 ? 12 : 8, writes = WRITES;
    __builtin_amdgcn_sched_group_barrier(0x100, reads, 0);         // DS reads
#pragma unroll
    for (int i = 0; i < 4 * NP; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);         // MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);         // VALU
    }
    __builtin_amdgcn_sched_group_barrier(0x200, writes, 0);        // DS writes
}

// acc += A[row0a.., 0..K) B[row0b.., 0..K)^T on the 128 x 128 tile of 256
// threads for operands whose 128-row panels lie inside the matrix, with K a
// positive multiple of 32 and aligned rows.  Global loads run two stages ahead
// of the matrix cores; every load is unconditional so that the wait before a
// stage's LDS store leaves the next stage's loads in flight.  `lds` holds
// kX3LdsDw dwords.  Ends with a barrier.  INTERLEAVE pays off in long K loops
// (the Gram), not in the CD block update.
template <bool INTERLEAVE = false, int NP = 6, class OA, class OB>
__device__ __forceinline__ void nt_tile_x3_full(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                       int64_t K, uint32_t* lds, f32x16 (&acc)[2][2])
{
    constexpr int OPDW = kX3OpDw;
    uint32_t* const a0 = lds;
    uint32_t* const b0 = lds + OPDW;
    uint32_t* const a1 = lds + 2 * OPDW;
    uint32_t* const b1 = lds + 3 * OPDW;
    const int64_t nst = K / kX3KC;
    X3Stage ra0, rb0, ra1, rb1;
    A.load_full(row0a, 0, ra0);
    B.load_full(row0b, 0, rb0);
    A.load_full(row0a, kX3KC, ra1);
    B.load_full(row0b, kX3KC, rb1);
    A.store(a0, ra0);
    B.store(b0, rb0);
    __syncthreads();
    for (int64_t c = 0; c + 2 < nst; c += 2) {
        // LDS 0: stage c; registers 1: stage c + 1; registers 0 take stage c + 2
        A.load_full(row0a, (c + 2) * kX3KC, ra0);
        B.load_full(row0b, (c + 2) * kX3KC, rb0);
        __builtin_amdgcn_sched_barrier(0);
        x3_mfma_stage<NP>(a0, b0, acc);
        if constexpr (!INTERLEAVE) __builtin_amdgcn_sched_barrier(0);
        A.store(a1, ra1);
        B.store(b1, rb1);
        if constexpr (INTERLEAVE) x3_interleave<NP, x3_writes<OA>() + x3_writes<OB>()>();
        __syncthreads();
        // LDS 1: stage c + 1; registers 0: stage c + 2; registers 1 take stage c + 3
        A.load_full(row0a, (c + 3) * kX3KC, ra1);
        B.load_full(row0b, (c + 3) * kX3KC, rb1);
        __builtin_amdgcn_sched_barrier(0);
        x3_mfma_stage<NP>(a1, b1, acc);
        if constexpr (!INTERLEAVE) __builtin_amdgcn_sched_barrier(0);
        A.store(a0, ra0);
        B.store(b0, rb0);
        if constexpr (INTERLEAVE) x3_interleave<NP, x3_writes<OA>() + x3_writes<OB>()>();
        __syncthreads();
    }
    x3_mfma_stage<NP>(a0, b0, acc);
    A.store(a1, ra1);
    B.store(b1, rb1);
    __syncthreads();
    x3_mfma_stage<NP>(a1, b1, acc);
    __syncthreads();
}

// Any shape: guarded loads (out-of-range elements read as 0), one stage of
// prefetch.  Ends with a barrier.
template <int NP = 6, class OA, class OB>
__device__ __forceinline__ void nt_tile_x3_edge(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                       int64_t K, uint32_t* lds, f32x16 (&acc)[2][2])
{
    uint32_t* const a0 = lds;
    uint32_t* const b0 = lds + kX3OpDw;
    uint32_t* const a1 = lds + 2 * kX3OpDw;
    uint32_t* const b1 = lds + 3 * kX3OpDw;
    const int64_t nst = cdiv(K, kX3KC);
    X3Stage sa, sb;
    A.load(row0a, 0, sa);
    B.load(row0b, 0, sb);
    A.store(a0, sa);
    B.store(b0, sb);
    __syncthreads();
    for (int64_t c = 0; c < nst; c += 2) {
        bool more = c + 1 < nst;
        if (more) {
            A.load(row0a, (c + 1) * kX3KC, sa);
            B.load(row0b, (c + 1) * kX3KC, sb);
        }
        x3_mfma_stage<NP>(a0, b0, acc);
        if (more) {
            A.store(a1, sa);
            B.store(b1, sb);
        }
        __syncthreads();
        if (!more) break;
        more = c + 2 < nst;
        if (more) {
            A.load(row0a, (c + 2) * kX3KC, sa);
            B.load(row0b, (c + 2) * kX3KC, sb);
        }
        x3_mfma_stage<NP>(a1, b1, acc);
        if (more) {
            A.store(a0, sa);
            B.store(b0, sb);
        }
        __syncthreads();
    }
}

// 256 x 256 tile of eight waves (wave (wm, wn) owns rows wm * 64 + 32 mi,
// mi < 2, and columns wn * 128 + 32 ni, ni < 4): every staged value feeds
// twice the matrix-core work of the 128 x 128 tile.  Three LDS stage buffers
// let each wave read the next stage's operand fragments while the current
// stage's MFMAs run: B fragments one 32-column block ahead, A fragments right
// after their last use in the stage's final block.  One barrier per stage,
// placed after the stage's LDS writes and its last reads of the current
// buffer.  Global loads run three stages ahead of the matrix cores (four
// register stages would not fit beside the 128 accumulators).
constexpr int kX3wOpDw = 256 * kX3RowDw;          // one operand of one stage
constexpr int kX3wBufDw = 2 * kX3wOpDw;           // A and B of one stage
constexpr int kX3wLdsDw = 3 * kX3wBufDw;          // three stages: 147,456 bytes

__device__ __forceinline__ bf16x8 x3w_frag(const uint32_t* p)
{
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// One 32-column block ni of one stage: products lh, mh, mm, hh, hm, hl (A
// planes l, m, m, h, h, h), two MFMAs (mi = 0, 1) each.
__device__ __forceinline__ void x3w_block(const bf16x8 (&a)[2][3], const bf16x8 (&b)[3],
                                          f32x16 (&acc)[2][4], int ni)
{
    constexpr int PA[6] = {2, 1, 1, 0, 0, 0};
    constexpr int PB[6] = {0, 0, 1, 0, 1, 2};
#pragma unroll
    for (int q = 0; q < 6; ++q)
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi][PA[q]], b[PB[q]],
                                                                  acc[mi][ni], 0, 0, 0);
}

// Stage c of the 256 x 256 tile: multiplies the fragments of `cur` (fa and
// fb[0] arrive holding A and B block 0), splits and writes stage c + 2 from
// (ga, gb) to `wr`, loads stage kload into (la, lb), and leaves fa and fb[0]
// holding the fragments of `nxt` (stage c + 1).
template <class OA, class OB>
__device__ __forceinline__ void x3w_stage(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                          int64_t kload, const uint32_t* cur, const uint32_t* nxt,
                                          uint32_t* wr, X3Stage& ga, X3Stage& gb, X3Stage& la, X3Stage& lb,
                                          int offa, int offb, bf16x8 (&fa)[2][3], bf16x8 (&fb)[2][3],
                                          f32x16 (&acc)[2][4])
{
    // group 0: global loads, B block 1 reads, split of A (stage c + 2)
    A.load_full(row0a, kload, la);
    B.load_full(row0b, kload, lb);
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) fb[1][pl] = x3w_frag(cur + offb + 1 * 32 * kX3RowDw + 8 * pl);
    x3w_block(fa, fb[0], acc, 0);
    A.store(wr, ga);
    __builtin_amdgcn_sched_group_barrier(0x020, 4, 0);     // VMEM reads
    __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);     // DS reads
#pragma unroll
    for (int i = 0; i < 12; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x200, 3, 0);     // DS writes
    __builtin_amdgcn_sched_barrier(0);
    // group 1: B block 2 reads, split of B
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) fb[0][pl] = x3w_frag(cur + offb + 2 * 32 * kX3RowDw + 8 * pl);
    x3w_block(fa, fb[1], acc, 1);
    B.store(wr + kX3wOpDw, gb);
    __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x200, 3, 0);
    __builtin_amdgcn_sched_barrier(0);
    // group 2: B block 3 reads; the barrier makes stage c + 2 visible and ends
    // this stage's reads of `cur`
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) fb[1][pl] = x3w_frag(cur + offb + 3 * 32 * kX3RowDw + 8 * pl);
    x3w_block(fa, fb[0], acc, 2);
    __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 12, 0);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    // group 3: next stage's B block 0 and A fragments, each after its last use
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) fb[0][pl] = x3w_frag(nxt + offb + 8 * pl);
    {
        constexpr int PA[6] = {2, 1, 1, 0, 0, 0};
        constexpr int PB[6] = {0, 0, 1, 0, 1, 2};
#pragma unroll
        for (int q = 0; q < 6; ++q) {
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
                acc[mi][3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[mi][PA[q]], fb[1][PB[q]], acc[mi][3], 0, 0, 0);
            if (q == 0 || q == 2 || q == 5) {
                const int pl = PA[q];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) fa[mi][pl] = x3w_frag(nxt + offa + mi * 32 * kX3RowDw + 8 * pl);
            }
        }
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_barrier(0);
}

// Stage c with c % 3 == R: stage s lives in LDS buffer s % 3 and in
// register set s % 3; the set that held stage c + 1 takes stage c + 4 (a
// load past the last stage re-reads the last stage: in bounds, and it lands
// in a buffer no stage reads).
template <int R, class OA, class OB>
__device__ __forceinline__ void x3w_stage3(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                           int64_t c, int64_t nst, uint32_t* lds, X3Stage (&ga)[3],
                                           X3Stage (&gb)[3], int offa, int offb, bf16x8 (&fa)[2][3],
                                           bf16x8 (&fb)[2][3], f32x16 (&acc)[2][4])
{
    x3w_stage(A, row0a, B, row0b, min(c + 4, nst - 1) * kX3KC, lds + R * kX3wBufDw,
              lds + ((R + 1) % 3) * kX3wBufDw, lds + ((R + 2) % 3) * kX3wBufDw, ga[(R + 2) % 3],
              gb[(R + 2) % 3], ga[(R + 1) % 3], gb[(R + 1) % 3], offa, offb, fa, fb, acc);
}

// acc += A[row0a.., 0..K) B[row0b.., 0..K)^T on the 256 x 256 tile of 512
// threads; K a positive multiple of 32, every 256-row panel inside the matrix,
// aligned rows.  `lds` holds kX3wLdsDw dwords.  Ends with a barrier.
template <class OA, class OB>
__device__ __forceinline__ void nt_tile_x3_wide(const OA& A, int64_t row0a, const OB& B, int64_t row0b,
                                                int64_t K, uint32_t* lds, f32x16 (&acc)[2][4])
{
    const int64_t nst = K / kX3KC;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int offa = x3_addr(wm * 64 + (lane & 31), lane >> 5, 0);
    const int offb = kX3wOpDw + x3_addr(wn * 128 + (lane & 31), lane >> 5, 0);
    X3Stage ga[3], gb[3];
    A.load_full(row0a, 0, ga[0]);
    B.load_full(row0b, 0, gb[0]);
    A.load_full(row0a, kX3KC, ga[1]);
    B.load_full(row0b, kX3KC, gb[1]);
    A.store(lds, ga[0]);
    B.store(lds + kX3wOpDw, gb[0]);
    A.load_full(row0a, min<int64_t>(2, nst - 1) * kX3KC, ga[2]);
    B.load_full(row0b, min<int64_t>(2, nst - 1) * kX3KC, gb[2]);
    A.load_full(row0a, min<int64_t>(3, nst - 1) * kX3KC, ga[0]);
    B.load_full(row0b, min<int64_t>(3, nst - 1) * kX3KC, gb[0]);
    A.store(lds + kX3wBufDw, ga[1]);
    B.store(lds + kX3wBufDw + kX3wOpDw, gb[1]);
    __syncthreads();
    bf16x8 fa[2][3], fb[2][3];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int pl = 0; pl < 3; ++pl) fa[mi][pl] = x3w_frag(lds + offa + mi * 32 * kX3RowDw + 8 * pl);
#pragma unroll
    for (int pl = 0; pl < 3; ++pl) fb[0][pl] = x3w_frag(lds + offb + 8 * pl);
    int64_t c = 0;
    for (; c + 3 <= nst; c += 3) {
        x3w_stage3<0>(A, row0a, B, row0b, c, nst, lds, ga, gb, offa, offb, fa, fb, acc);
        x3w_stage3<1>(A, row0a, B, row0b, c + 1, nst, lds, ga, gb, offa, offb, fa, fb, acc);
        x3w_stage3<2>(A, row0a, B, row0b, c + 2, nst, lds, ga, gb, offa, offb, fa, fb, acc);
    }
    if (c < nst) x3w_stage3<0>(A, row0a, B, row0b, c, nst, lds, ga, gb, offa, offb, fa, fb, acc);
    if (c + 1 < nst) x3w_stage3<1>(A, row0a, B, row0b, c + 1, nst, lds, ga, gb, offa, offb, fa, fb, acc);
    __syncthreads();
}
}  // namespace qe
