// One ALS half-sweep on gfx950 (MI355X): C ABI of include/als.h plus its kernels.
//
// Per row u of a CSR matrix (eq. 2 of the paper; Algorithm 1's Get_Hermitian_X then
// Batch_Solve):  A_u = sum theta_v theta_v^T + lambda n_u I,  b_u = sum r_uv theta_v,
// x_u = A_u^{-1} b_u.
//
// Design (one wave = one worker):
//   k_plan          integer partition of the rows (and of long rows' entries) into chunks of a
//                   cost axis: W large chunks, then 8W small ones (see als_plan in als.h); no
//                   host synchronisation needed.
//   k_herm_solve    persistent waves claim chunks in order and walk their row pieces; gather
//                   theta_v for four entries at a time straight into MFMA operand registers
//                   (lane = 16*k + column, so each group of 16 lanes reads 64 contiguous bytes of
//                   one theta_v), with the rating appended as column f, and accumulate the upper
//                   block-triangle of the augmented Gram matrix [A b; b^T c] with
//                   v_mfma_f32_16x16x4_f32 (the mostly-padding last block column with 4x4x1
//                   16-block MFMAs when it fits whole quads).  Rows that end in the chunk are
//                   regularised and solved in registers by a blocked Cholesky: per 16-column
//                   block, the 16 x 16 diagonal tile is factored and inverted with lane
//                   broadcasts, and the panel and trailing updates are again 16x16x4 MFMAs; the
//                   forward substitution rides along as the augmented column; the back
//                   substitution is a short blocked pass.
//   k_reduce_*      rows cut by chunk boundaries: sum the chunks' partial accumulators in chunk
//                   order (fixed, so results are reproducible), then the same solve.
//   k_rmse_rows     residuals per stored entry through the same gather pipeline, x_u held in
//                   registers per row piece; fp64 partial sums in a fixed order.
//
// Register layout of the accumulators (the 16x16 MFMA C/D layout): tile (I,J), I <= J, lane l,
// element r holds M[16 I + 4 (l >> 4) + r][16 J + (l & 15)] of the augmented matrix M, whose
// column f is b (and M[f][f] = sum r^2, unused).  NB = f/16 + 1 column blocks cover f + 1.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <climits>
#include <cstring>
#include <mutex>
#include <new>

#include "als.h"

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWave = 64;
constexpr int kMaxNB = ALS_F_MAX / 16 + 1;      // 9 column blocks of 16 cover f + 1 <= 129
constexpr int kSnap = 256;                      // partition cut grid (entries)
constexpr int kCostPerEntry = 16;               // c_nnz
constexpr int kTailDiv = 8;                     // the small chunks cover floor(T / 8) of the cost
constexpr int kSmallPerWave = 8;                // small chunks per wave
constexpr int chunks_of(int waves) { return waves * (1 + kSmallPerWave); }
constexpr int kMaxWavesPerCU = 32;
constexpr int kRmseWavesPerCU = 32;                // RMSE: up to 8 waves per SIMD (occupancy)
constexpr int kTransposeWavesPerCU = 8;            // CSR -> CSC: row blocks per CU (at most)

constexpr int ntiles(int nb) { return nb * (nb + 1) / 2; }
// the quad form with a theta quad (f = 16 (NB - 1) + 4) exists for NB whose f is in range
template <int NB>
constexpr bool kQuad2 = 16 * (NB - 1) + 4 <= ALS_F_MAX;
// upper block-triangle, row-major: tile (I, J) with I <= J
constexpr int tu(int nb, int I, int J) { return I * nb - I * (I - 1) / 2 + (J - I); }
// floats per partial-accumulator slot: tiles, 4 per lane
constexpr int slot_floats(int nb) { return ntiles(nb) * 4 * kWave; }

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// acc + a' * b, where a' is `a` taken from lane N of the lane's 16-lane row (DPP row_newbcast:N),
// in one v_fmac.  A DPP source needs two wait states after its last VALU write; the caller keeps
// them (volatile, so the statements stay in source order and the caller can count).  `a` may be
// the value of `acc` itself: as an operand of its own, a copy the register allocator makes for
// the tied accumulator never becomes the DPP source.
template <int N>
__device__ __forceinline__ float fmac_bcast(float acc, float a, float b) {
    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:%3 row_mask:0xf bank_mask:0xf"
                 : "+v"(acc)
                 : "v"(a), "v"(b), "n"(N));
    return acc;
}
// Two wait states (for a DPP read of a register a VALU op wrote just before).
__device__ __forceinline__ void dpp_settle() { asm volatile("s_nop 1"); }

// -1.0 in the lanes whose bit is set in the 64-bit lane mask, else 0 (one v_cndmask; the mask
// is a constant in scalar registers).
__device__ __forceinline__ float lane_select_minus_one(uint64_t mask) {
    float r;
    asm("v_cndmask_b32_e64 %0, 0, -1.0, %1" : "=v"(r) : "s"(mask));
    return r;
}

// Sum over the 16 lanes of a DPP row (lanes 16g..16g+15), returned to all 16 lanes with the
// same bits: swap neighbours, swap pairs (quad_perm), then mirror within 8 and within 16.
__device__ __forceinline__ float row_sum16(float v) {
    v += dpp_f<0xB1>(v);    // quad_perm [1,0,3,2]
    v += dpp_f<0x4E>(v);    // quad_perm [2,3,0,1]
    v += dpp_f<0x141>(v);   // row_half_mirror
    v += dpp_f<0x140>(v);   // row_mirror
    return v;
}

// Sums over the 16 lanes of a DPP row of v[0..3], transposed: lane c of the row returns the sum
// of v[c & 3] (each sum lands in four lanes, added in different orders).  Pairs of values trade
// halves between neighbours (xor 1), then between pairs (xor 2), so every lane keeps adding one
// value; rotations by 4 and 8 finish the sum.  11 VALU ops against 16 for four plain row sums.
__device__ __forceinline__ float row_sum16_t(f4 v) {
    float v0 = v[0], v1 = v[1], v2 = v[2], v3 = v[3], t0, t1;
    asm volatile(
        "v_cndmask_b32_e64 %[t0], %[v1], %[v0], %[odd]\n\t"    // odd ? v0 : v1 (sent)
        "v_cndmask_b32_e64 %[t1], %[v3], %[v2], %[odd]\n\t"    // odd ? v2 : v3 (sent)
        "v_cndmask_b32_e64 %[v0], %[v0], %[v1], %[odd]\n\t"    // odd ? v1 : v0 (kept)
        "v_cndmask_b32_e64 %[v2], %[v2], %[v3], %[odd]\n\t"    // odd ? v3 : v2 (kept)
        "v_add_f32_dpp %[v0], %[t0], %[v0] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_add_f32_dpp %[v2], %[t1], %[v2] quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
        "v_cndmask_b32_e64 %[t0], %[v2], %[v0], %[two]\n\t"    // two ? v0 : v2 (sent)
        "v_cndmask_b32_e64 %[v0], %[v0], %[v2], %[two]\n\t"    // two ? v2 : v0 (kept)
        "s_nop 0\n\t"
        "v_add_f32_dpp %[v0], %[t0], %[v0] quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_add_f32_dpp %[v0], %[v0], %[v0] row_ror:4 row_mask:0xf bank_mask:0xf\n\t"
        "s_nop 1\n\t"
        "v_add_f32_dpp %[v0], %[v0], %[v0] row_ror:8 row_mask:0xf bank_mask:0xf"
        : [t0] "=&v"(t0), [t1] "=&v"(t1), [v0] "+v"(v0), [v1] "+v"(v1), [v2] "+v"(v2),
          [v3] "+v"(v3)
        : [odd] "s"(0xAAAAAAAAAAAAAAAAull), [two] "s"(0xCCCCCCCCCCCCCCCCull));
    return v0;
}

// ------------------------------------------------------------------------------- plan ----

// Cost prefix P(u) = c_nnz rowptr[u] + c_row u, T = P(m).  C chunks: W large ones cover
// T1 = T - T2 and C - W small ones the tail T2 = floor(T / kTailDiv) (T2 = 0 when C = W);
// boundary b sits at s_b = floor(T1 b / W) for b <= W, T1 + floor(T2 (b - W) / (C - W)) beyond.
// Thread 0 also resets the chunk counter the persistent waves claim chunks from.
__global__ void k_plan(const int64_t* __restrict__ rowptr, int64_t m, int W, int C, int64_t c_nnz,
                       int64_t c_row, int64_t q, int64_t* __restrict__ bounds,
                       unsigned* __restrict__ chunk_ctr) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b == 0 && chunk_ctr) *chunk_ctr = 0u;
    if (b > C) return;
    const int64_t T = c_nnz * rowptr[m] + c_row * m;
    const int64_t T2 = C > W ? T / kTailDiv : 0, T1 = T - T2;
    int64_t s;   // floor(X b / D) as Q b + floor(R b / D), without 128-bit products
    if (b <= W) {
        s = T1 / W * b + (T1 % W) * b / W;
    } else {
        const int64_t D = C - W, e = b - W;
        s = T1 + T2 / D * e + (T2 % D) * e / D;
    }
    int64_t lo = 0, hi = m;                  // largest u in [0, m] with P(u) <= s
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (c_nnz * rowptr[mid] + c_row * mid <= s) lo = mid; else hi = mid - 1;
    }
    const int64_t u = lo;
    int64_t kk = 0;
    if (u < m) {
        const int64_t nu = rowptr[u + 1] - rowptr[u];
        const int64_t over = s - (c_nnz * rowptr[u] + c_row * u) - c_row;
        int64_t raw = over <= 0 ? 0 : (over + c_nnz - 1) / c_nnz;
        if (raw > nu) raw = nu;
        kk = (raw + q / 2) / q * q;
        if (kk > 0 && kk + q / 2 > nu) kk = nu;
    }
    bounds[2 * b] = u;
    bounds[2 * b + 1] = kk;
}

// --------------------------------------------------------------------- Gram + RHS --------

// Gather pipeline: the gathers of step s + kDepth are issued before step s runs, so every gather
// has kDepth steps of matrix work of this wave to hide behind.  Steps run in unrolled groups of
// kGroup = kDepth + 1 with as many operand buffers; at sub-step J the step kDepth ahead goes into
// the buffer whose step ran at sub-step J - 1, so the buffers rotate by renaming, never by copying
// registers that are loading.  Each entry's gather word and rating come in batches of 48 entries
// (12 steps) through a two-slot LDS ring (entry p of the piece sits at p mod 96): batch k+1 is
// loaded (one entry per lane) at the top of batch k's first group and stored at the top of its
// second group, before the first gather that reads it (which needs kDepth <= 5) and after the
// last one that read the slot's previous batch, so any register carried around the loop only
// ever waits on a load older than the gathers in flight.
constexpr int kDepth = 3;
constexpr int kGroup = kDepth + 1;
constexpr int kBatch = 48;
constexpr int kBatchGroups = kBatch / 4 / kGroup;
constexpr int kRing = 2 * kBatch;
static_assert(kBatchGroups * kGroup * 4 == kBatch && kBatchGroups >= 2 && 2 * kDepth <= 11,
              "pipeline depth must divide the batch and stay within one group of lookahead");

// The last block column NB-1 holds f - 16 (NB-1) theta columns and the rating, the rest of it
// padding.  In the quad form (P > 0: the theta columns fill P-1 whole column quads and the
// rating is column 4 (P-1) of the block) the 16x16 tiles cover only the block columns J < NB-1.
// The theta columns of the last block are accumulated by v_mfma_f32_4x4x1_16b_f32 (16 blocks of
// 4x4, lane 4b + i of the A operand holds row i of block b, so block b = 4e + qq is entry slot e,
// row quad qq of an operand block exactly as gathered): q[I][p], lane 4b + j, register i holds
// the slot-e part of M[16 I + 4 qq + i][16 (NB-1) + 4 p + j], with the second operand w[p]
// holding column 4p + j of the entry's last block in every quad.  The rating column needs one
// value per row, so it is a plain FMA per lane: b[I] at lane (e, c) holds the slot-e part of
// M[16 I + c][f] (the lane's own operand times its slot's rating).
template <int NB, int P>
struct QuadAcc {
    f4 q[NB][P > 1 ? P - 1 : 1];   // used for P > 1
    float b[NB];
};
template <int NB>
struct QuadAcc<NB, 0> {};

template <int NB, int P>
__device__ __forceinline__ void mfma_step(const float (&v)[NB], const float (&w)[P > 0 ? P : 1],
                                          float r, f4 (&acc)[ntiles(NB)], QuadAcc<NB, P>& qa) {
    constexpr int JT = P > 0 ? NB - 1 : NB;   // block columns covered by 16x16 tiles
#pragma unroll
    for (int I = 0; I < JT; ++I)
#pragma unroll
        for (int J = I; J < JT; ++J)
            acc[tu(NB, I, J)] =
                __builtin_amdgcn_mfma_f32_16x16x4f32(v[I], v[J], acc[tu(NB, I, J)], 0, 0, 0);
    if constexpr (P > 0) {
#pragma unroll
        for (int I = 0; I < NB; ++I)
#pragma unroll
            for (int p = 0; p + 1 < P; ++p)
                qa.q[I][p] = __builtin_amdgcn_mfma_f32_4x4x1f32(v[I], w[p], qa.q[I][p], 0, 0, 0);
#pragma unroll
        for (int I = 0; I < NB; ++I) qa.b[I] = __builtin_fmaf(v[I], r, qa.b[I]);
    }
}

// The quad accumulators into standard tiles acc[tu(NB, I, NB-1)]: the tile's lane (g, c),
// register r needs M[16 I + 4 g + r][16 (NB-1) + c] = the sum over entry slots e = 0..3, in that
// order, of q[I][c / 4] at lane 16 e + 4 g + (c & 3), register r, for the theta columns, and of
// b[I] at lane 16 e + 4 g + r for the rating column; columns past it stay 0.  One LDS exchange
// for both.  scratch: (P - 1) NB 64 vectors then NB 64 floats, 16-byte aligned.
template <int NB, int P>
constexpr int quad_scratch_bytes() {
    return (P - 1) * NB * kWave * 16 + NB * kWave * 4;
}
template <int NB, int P>
__device__ __forceinline__ void quad_to_tiles(const QuadAcc<NB, P>& qa, f4 (&acc)[ntiles(NB)],
                                              void* scratch, int lane) {
    const int g = lane >> 4, c = lane & 15;
    f4* sq = reinterpret_cast<f4*>(scratch);
    float* sb = reinterpret_cast<float*>(sq + (P - 1) * NB * kWave);
#pragma unroll
    for (int p = 0; p + 1 < P; ++p)
#pragma unroll
        for (int I = 0; I < NB; ++I) sq[(p * NB + I) * kWave + lane] = qa.q[I][p];
#pragma unroll
    for (int I = 0; I < NB; ++I) sb[I * kWave + lane] = qa.b[I];
    __syncthreads();
#pragma unroll
    for (int I = 0; I < NB; ++I) acc[tu(NB, I, NB - 1)] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p + 1 < P; ++p) {
        if ((c >> 2) == p) {
            const int src = 4 * g + (c & 3);
#pragma unroll
            for (int I = 0; I < NB; ++I) {
                const f4* s = sq + (p * NB + I) * kWave + src;
                acc[tu(NB, I, NB - 1)] = ((s[0] + s[16]) + s[32]) + s[48];
            }
        }
    }
    if (c == 4 * (P - 1)) {
#pragma unroll
        for (int I = 0; I < NB; ++I) {
            const f4* s = reinterpret_cast<const f4*>(sb + I * kWave + 4 * g);   // slot e: s[4e]
            acc[tu(NB, I, NB - 1)] = ((s[0] + s[4]) + s[8]) + s[12];
        }
    }
    __syncthreads();
}

// The theta gather of one step, as MFMA operands: lane (g, c) of block I reads
// theta_{v_g}[16 I + c], and the lane of column f takes the rating.  Three forms (the second
// template argument):
//   kFormBuffer, for theta below 2 GiB: raw buffer loads against a descriptor that bounds
//     theta.  The gather word of an entry is its byte offset 4 f v; an entry past the piece's end
//     gets the buffer size, and the lanes of padding columns add the size to their offset, so
//     those loads return 0 by the hardware's range check and nothing is masked in the loop.
//   kFormGlobal, for any size: 64-bit global loads; the gather word is the row's address (a row
//     of zeros past the piece's end), and padding lanes read a column of their block's cache
//     line whose value is then replaced (see Gather<NB, kFormGlobal, P>).
//   kFormStaged, a design alternative kept for the ablation: the rows go through LDS.
// All issue their loads unconditionally, so they stay in flight across earlier matrix ops.
constexpr int kFormGlobal = 0, kFormBuffer = 1, kFormStaged = 2;

// One entry of the index ring: the entry's gather word (a byte offset or a row address, as the
// gather form defines it) and its rating.
template <class W>
struct RingEntryT {
    W e;
    float r;
};

template <int NB, int BUF, int P = 0>
struct Gather;

template <int NB, int P>
struct Gather<NB, kFormBuffer, P> {
    using Entry = RingEntryT<int>;
    static constexpr int kBuf = NB + (P > 1 ? P - 1 : 0);   // operand values per step
    __amdgpu_buffer_rsrc_t rs;
    unsigned fbytes, size, lo, llast;
    bool jr, jq;
    // quad form: quads 0..P-2 hold theta columns 16 (NB-1) + 4p + (lane & 3) (all below f), and
    // quad P-1 holds only the rating, in its first column (f = 16 (NB-1) + 4 (P-1))
    unsigned lw[P > 1 ? P - 1 : 1];
    __device__ __forceinline__ Gather(const float* theta, int64_t n, int f, int c,
                                      float* = nullptr) {
        fbytes = 4u * (unsigned)f;
        size = (unsigned)n * fbytes;
        rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(theta), 0, (int)size,
                                               0x00020000);
        lo = 4u * (unsigned)c;
        const int jlast = 16 * (NB - 1) + c;
        llast = jlast < f ? 4u * (unsigned)jlast : size;
        jr = jlast == f;
        jq = (c & 3) == 0;
#pragma unroll
        for (int p = 0; p < (P > 1 ? P - 1 : 1); ++p)
            lw[p] = 4u * (unsigned)(16 * (NB - 1) + 4 * p + (c & 3));
    }
    __device__ __forceinline__ int word(int col, bool valid) const {
        return valid ? (int)((unsigned)col * fbytes) : (int)size;
    }
    __device__ __forceinline__ void issue(int e, float (&v)[kBuf]) const {
        const unsigned base = (unsigned)e + lo;
#pragma unroll
        for (int I = 0; I < NB - 1; ++I)
            v[I] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rs, base + 64u * I, 0, 0));
        v[NB - 1] = __builtin_bit_cast(
            float, __builtin_amdgcn_raw_buffer_load_b32(rs, (unsigned)e + llast, 0, 0));
#pragma unroll
        for (int p = 0; p + 1 < P; ++p)
            v[NB + p] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rs, (unsigned)e + lw[p], 0, 0));
    }
    __device__ __forceinline__ void operands(const float (&B)[kBuf], float r, bool,
                                             float (&v)[NB], float (&w)[P > 0 ? P : 1]) const {
#pragma unroll
        for (int I = 0; I < NB - 1; ++I) v[I] = B[I];
        v[NB - 1] = jr ? r : B[NB - 1];
        if constexpr (P > 0) {
#pragma unroll
            for (int p = 0; p + 1 < P; ++p) w[p] = B[NB + p];
            w[P - 1] = jq ? r : 0.f;
        }
    }
};

// A row of zeros, read in place of theta_v by the 64-bit gather for entries past a piece's end.
__device__ float g_zero_row[16 * kMaxNB];

// Gather<NB, kFormGlobal, P>, for any size of theta: 64-bit global loads.  The gather word of an
// entry is its row's address (g_zero_row past the piece's end, so such entries gather zeros);
// lane (g, c) reads block I < NB-1 at that address + 4 (16 I + c), with 64 I as the
// instruction's immediate offset.  In the last block a padding lane reads a column of the cache
// line the block's real lanes read -- its first column, or column f - 1 when it has none -- and
// the value is replaced (by the rating in column f, else by 0); the quad operands read their
// columns 16 (NB-1) + 4 p + (c & 3) as in the buffer form.
template <int NB, int P>
struct Gather<NB, kFormGlobal, P> {
    using Entry = RingEntryT<uint64_t>;
    static constexpr int kBuf = NB + (P > 1 ? P - 1 : 0);
    typedef const __attribute__((address_space(1))) float* gptr;
    uint64_t base, zero;
    unsigned fbytes, lo, llast;
    bool jpad, jr, jq;
    unsigned lw[P > 1 ? P - 1 : 1];
    __device__ __forceinline__ Gather(const float* theta, int64_t, int f, int c,
                                      float* = nullptr) {
        base = (uint64_t)theta;
        zero = (uint64_t)g_zero_row;
        fbytes = 4u * (unsigned)f;
        lo = 4u * (unsigned)c;
        const int jlast = 16 * (NB - 1) + c;
        jpad = jlast >= f;
        const int jsame = 16 * (NB - 1) < f ? 16 * (NB - 1) : f - 1;
        llast = 4u * (unsigned)(jpad ? jsame : jlast);
        jr = jlast == f;
        jq = (c & 3) == 0;
#pragma unroll
        for (int p = 0; p < (P > 1 ? P - 1 : 1); ++p)
            lw[p] = 4u * (unsigned)(16 * (NB - 1) + 4 * p + (c & 3));
    }
    __device__ __forceinline__ uint64_t word(int col, bool valid) const {
        return valid ? base + (uint64_t)(unsigned)col * fbytes : zero;
    }
    __device__ __forceinline__ void issue(uint64_t e, float (&v)[kBuf]) const {
        const gptr pl = (gptr)(e + lo);
#pragma unroll
        for (int I = 0; I < NB - 1; ++I) v[I] = pl[16 * I];
        v[NB - 1] = *(gptr)(e + llast);
#pragma unroll
        for (int p = 0; p + 1 < P; ++p) v[NB + p] = *(gptr)(e + lw[p]);
    }
    __device__ __forceinline__ void operands(const float (&B)[kBuf], float r, bool,
                                             float (&v)[NB], float (&w)[P > 0 ? P : 1]) const {
#pragma unroll
        for (int I = 0; I < NB - 1; ++I) v[I] = B[I];
        v[NB - 1] = jpad ? (jr ? r : 0.f) : B[NB - 1];
        if constexpr (P > 0) {
#pragma unroll
            for (int p = 0; p + 1 < P; ++p) w[p] = B[NB + p];
            w[P - 1] = jq ? r : 0.f;
        }
    }
};

// Gather<NB, kFormStaged>: a design alternative (for the ablation of the gather; theta below
// 2 GiB, f a multiple of 4): the step's four theta rows are read row by row with two 16-byte
// loads per lane -- lane (g, c) reads bytes 16 c and 256 + 16 c of row g, the rating lane's
// bytes included -- written to a per-wave LDS buffer of four rows of 16 NB floats (zero past
// the loaded columns), and the MFMA operands are read back from it (lane (g, c) of block I:
// row g, column 16 I + c).  Past the piece's end and past a row's 4 f bytes the loads are out of
// range and return zeros, as in the buffer form.
constexpr int stage_floats(int nb) { return 4 * 16 * nb; }

template <int NB>
struct Gather<NB, kFormStaged, 0> {
    using Entry = RingEntryT<int>;
    static constexpr int kBuf = 8;
    __amdgpu_buffer_rsrc_t rs;
    unsigned fbytes, size, o0, o1;
    int lane;
    bool jr;
    float* stage;
    __device__ __forceinline__ Gather(const float* theta, int64_t n, int f, int c, float* st) {
        fbytes = 4u * (unsigned)f;
        size = (unsigned)n * fbytes;
        rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(theta), 0, (int)size,
                                               0x00020000);
        o0 = 16u * c < fbytes ? 16u * c : size;
        o1 = 256u + 16u * c < fbytes ? 256u + 16u * c : size;
        jr = 16 * (NB - 1) + c == f;
        lane = (int)(threadIdx.x & 63);
        stage = st;
    }
    __device__ __forceinline__ int word(int col, bool valid) const {
        return valid ? (int)((unsigned)col * fbytes) : (int)size;
    }
    __device__ __forceinline__ void issue(int e, float (&v)[kBuf]) const {
        const f4 a = __builtin_bit_cast(
            f4, __builtin_amdgcn_raw_buffer_load_b128(rs, (unsigned)e + o0, 0, 0));
        const f4 b = __builtin_bit_cast(
            f4, __builtin_amdgcn_raw_buffer_load_b128(rs, (unsigned)e + o1, 0, 0));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v[j] = a[j];
            v[4 + j] = b[j];
        }
    }
    __device__ __forceinline__ void operands(const float (&B)[kBuf], float r, bool,
                                             float (&v)[NB], float (&)[1]) const {
        const int g = lane >> 4, c = lane & 15;
        float* row = stage + g * 16 * NB;
        if (4 * c + 4 <= 16 * NB)
            *reinterpret_cast<f4*>(row + 4 * c) = f4{B[0], B[1], B[2], B[3]};
        if (64 + 4 * c + 4 <= 16 * NB)
            *reinterpret_cast<f4*>(row + 64 + 4 * c) = f4{B[4], B[5], B[6], B[7]};
        __syncthreads();
#pragma unroll
        for (int I = 0; I < NB; ++I) v[I] = row[16 * I + c];
        if (jr) v[NB - 1] = r;
        __syncthreads();   // the next step rewrites the rows
    }
};

// Entry `first + lane` of the piece starting at kbeg (lanes below kBatch; past the end: the
// invalid gather word and rating 0).
template <class G>
__device__ __forceinline__ typename G::Entry load_entry(const G& gat,
                                                        const int32_t* __restrict__ colidx,
                                                        const float* __restrict__ vals,
                                                        int64_t kbeg, int64_t total,
                                                        int64_t first, int lane) {
    const bool valid = lane < kBatch && first + lane < total;
    int col = 0;
    float rv = 0.f;
    if (valid) {
        col = colidx[kbeg + first + lane];
        rv = vals[kbeg + first + lane];
    }
    return typename G::Entry{gat.word(col, valid), rv};
}

// The first two index batches of a row piece, loaded ahead of time into registers.
template <class G>
struct RowIndex {
    typename G::Entry q0, q1;
};

// The gather pipeline's in-flight state: operand values and ratings of the steps in flight
// (b[0..kDepth-1] at the top of a group; b[kDepth] is the extra buffer of the rotation).
template <int NBUF>
struct Inflight {
    float b[kGroup][NBUF];
    float r[kGroup];
};

template <class G>
__device__ __forceinline__ void gram_prefetch(const G& gat, const int32_t* __restrict__ colidx,
                                              const float* __restrict__ vals, int64_t kbeg,
                                              int64_t kend, int lane, RowIndex<G>& ix) {
    ix.q0 = load_entry(gat, colidx, vals, kbeg, kend - kbeg, 0, lane);
    ix.q1 = load_entry(gat, colidx, vals, kbeg, kend - kbeg, kBatch, lane);
}

// Put a piece's first two batches into ring slots 0 and 1 (the ring must be idle) and issue
// the gathers of its first kDepth steps.
template <class G>
__device__ __forceinline__ void gram_stage(const G& gat, const RowIndex<G>& ix,
                                           typename G::Entry* ring, int lane,
                                           Inflight<G::kBuf>& in) {
    const int g = lane >> 4;
    if (lane < kBatch) {
        ring[lane] = ix.q0;
        ring[kBatch + lane] = ix.q1;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
        const typename G::Entry q = ring[4 * j + g];
        in.r[j] = q.r;
        gat.issue(q.e, in.b[j]);
    }
}

// Sub-steps J..kGroup-1 of a group: run step s0 + J from buffer J (a step past the piece's end
// adds nothing) after issuing step s0 + J + kDepth into buffer (J + kDepth) mod kGroup (free: its
// step ran at sub-step J - 1).
template <int J, class G, class Body>
__device__ __forceinline__ void pipe_substeps(const G& gat, const typename G::Entry* ring, int rq,
                                              int s0, int total, int g, Inflight<G::kBuf>& in,
                                              Body& body) {
    if constexpr (J < kGroup) {
        constexpr int JN = (J + kDepth) % kGroup;
        body.take(in.b[J], in.r[J], 4 * (s0 + J) + g < total);
        __builtin_amdgcn_sched_barrier(0);
        int pos = rq + 4 * J;
        if (pos >= kRing) pos -= kRing;
        const typename G::Entry e = ring[pos + g];
        in.r[JN] = e.r;
        gat.issue(e.e, in.b[JN]);
        body.template run<J>();
        pipe_substeps<J + 1>(gat, ring, rq, s0, total, g, in, body);
    }
}

// Run entries [kbeg, kend) of one row piece through the gather pipeline, starting from the state
// gram_stage left in the ring and in `in`.  Per step the body takes the step's operands
// (body.take(B, r, ok): B the loaded values, r the rating, ok whether the step's entry lies in the
// piece), then -- after the gather kDepth steps ahead has been issued -- runs the step
// (body.run<J>(), J the step's place in its group of kGroup; the loop always runs whole groups:
// stopping inside the last group costs more, as a branch per step or as a second copy of the
// group, than the steps of zeros it would skip).
// ring: this wave's LDS ring of kRing entries.  Returns with the ring idle.
template <class G, class Body>
__device__ __forceinline__ void pipe_loop(const G& gat, const int32_t* __restrict__ colidx,
                                          const float* __restrict__ vals, int64_t kbeg,
                                          int64_t kend, typename G::Entry* ring, int lane,
                                          Inflight<G::kBuf>& in, Body& body) {
    const int g = lane >> 4;
    // a row has fewer than 2^31 entries (its columns are distinct int32 indices)
    const int total = (int)(kend - kbeg);
    const int nsteps = (total + 3) >> 2;
    const int ngroups = (nsteps + kGroup - 1) / kGroup;
    typename G::Entry nq{};
    int qb = 0, k = 0;       // group's position in its batch; batch of the group's steps
    int rq = 4 * kDepth;     // ring position of the first step issued in the group
    for (int q = 0; q < ngroups; ++q) {
        if constexpr (Body::kParts) {
            // at every part boundary the body folds its accumulators away (see GramBody)
            if (q > 0 && (q & body.part_mask) == 0) body.flush(q == body.part_mask + 1);
        }
        // batch k+1 goes into the ring at the top of group 1, one group after its load was
        // issued at the top of group 0 (the store comes first in program order, so its wait
        // never covers the gathers issued after the load)
        if (qb == 1 && k > 0) {
            if (lane < kBatch) ring[((k + 1) & 1) * kBatch + lane] = nq;
            __syncthreads();
        }
        if (qb == 0 && k > 0)
            nq = load_entry(gat, colidx, vals, kbeg, total, (int64_t)(k + 1) * kBatch, lane);
        pipe_substeps<0>(gat, ring, rq, q * kGroup, total, g, in, body);
        rq += 4 * kGroup;
        if (rq >= kRing) rq -= kRing;
        if (++qb == kBatchGroups) {
            qb = 0;
            ++k;
        }
    }
    __syncthreads();   // the ring is refilled by the next piece
}

// A piece longer than a part (kPart entries by default; a power of two times the 16 entries of a
// pipeline group) runs in parts (the last one shorter): each part's Gram is accumulated in
// registers from zero, and the parts' sums are added in order into the wave's own
// partial-accumulator slot in the workspace, the second level of a two-level sum, so that no fp32
// running sum spans more than a part (a column of tens of millions of ratings otherwise
// accumulates over a million entries in one register chain).  After the last part the slot is
// added into the registers and the piece goes on as one accumulator.
constexpr int64_t kPart = 1 << 16;
constexpr int kEntriesPerGroup = 4 * kGroup;

// A partial-accumulator slot: tile t of lane l at f4 index 64 t + l (16 contiguous bytes per
// lane, 1 KiB per tile).
template <int NB>
__device__ __forceinline__ void store_slot(const f4 (&acc)[ntiles(NB)], float* __restrict__ slot,
                                           int lane) {
    f4* s = reinterpret_cast<f4*>(slot);
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) s[t * kWave + lane] = acc[t];
}

// acc += slot.  All loads are issued before the first add (a dependent load-add chain would
// leave one load in flight at a time).
template <int NB>
__device__ __forceinline__ void add_slot(f4 (&acc)[ntiles(NB)], const float* __restrict__ slot,
                                         int lane) {
    const f4* s = reinterpret_cast<const f4*>(slot);
    f4 v[ntiles(NB)];
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) v[t] = s[t * kWave + lane];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) acc[t] += v[t];
}

// slot += acc, four tiles at a time (the temporaries stay at 16 registers beside the
// accumulators).
template <int NB>
__device__ __forceinline__ void fold_into_slot(const f4 (&acc)[ntiles(NB)],
                                               float* __restrict__ slot, int lane) {
    f4* s = reinterpret_cast<f4*>(slot);
#pragma unroll
    for (int t0 = 0; t0 < ntiles(NB); t0 += 4) {
        f4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (t0 + j < ntiles(NB)) v[j] = s[(t0 + j) * kWave + lane];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (t0 + j < ntiles(NB)) s[(t0 + j) * kWave + lane] = v[j] + acc[t0 + j];
        __builtin_amdgcn_sched_barrier(0);
    }
}

// acc += slot, four tiles at a time.
template <int NB>
__device__ __forceinline__ void add_slot_in_fours(f4 (&acc)[ntiles(NB)],
                                                  const float* __restrict__ slot, int lane) {
    const f4* s = reinterpret_cast<const f4*>(slot);
#pragma unroll
    for (int t0 = 0; t0 < ntiles(NB); t0 += 4) {
        f4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (t0 + j < ntiles(NB)) v[j] = s[(t0 + j) * kWave + lane];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (t0 + j < ntiles(NB)) acc[t0 + j] += v[j];
        __builtin_amdgcn_sched_barrier(0);
    }
}

// The Gram body: accumulate the upper block-triangle of the augmented Gram matrix into acc
// (and the quad accumulators of the last block column).  Every kPartGroups groups the pipeline
// calls flush(): the accumulators so far (the quad ones turned into tiles) are stored into, or
// added to, the wave's slot, and start again from zero.
template <int NB, int P>
__device__ __forceinline__ void zero_quads(QuadAcc<NB, P>& qa) {
    if constexpr (P > 0) {
#pragma unroll
        for (int I = 0; I < NB; ++I) {
#pragma unroll
            for (int p = 0; p + 1 < P; ++p) qa.q[I][p] = f4{0.f, 0.f, 0.f, 0.f};
            qa.b[I] = 0.f;
        }
    }
}

template <int NB, int P, class G, bool PARTS>
struct GramBody {
    static constexpr bool kParts = PARTS;
    int part_mask;        // groups per part - 1 (a power of two - 1)
    const G& gat;
    f4 (&acc)[ntiles(NB)];
    QuadAcc<NB, P>& qa;
    void* quad_scratch;   // LDS for the quad exchange
    float* wslot;         // the wave's slot
    int lane;
    float v[NB], w[P > 0 ? P : 1], r;
    __device__ __forceinline__ void take(const float (&B)[G::kBuf], float rr, bool ok) {
        gat.operands(B, rr, ok, v, w);
        r = rr;   // quad form only (buffer gather: an entry past the end has rating 0)
    }
    template <int J>
    __device__ __forceinline__ void run() { mfma_step<NB, P>(v, w, r, acc, qa); }
    __device__ __forceinline__ void flush(bool first) {
        if constexpr (P > 0) quad_to_tiles<NB, P>(qa, acc, quad_scratch, lane);
        if (first) store_slot<NB>(acc, wslot, lane);
        else fold_into_slot<NB>(acc, wslot, lane);
#pragma unroll
        for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
        zero_quads<NB, P>(qa);
    }
};

template <int NB, int P, bool PARTS, class G>
__device__ __forceinline__ void gram_loop(const G& gat, const int32_t* __restrict__ colidx,
                                          const float* __restrict__ vals, int64_t kbeg,
                                          int64_t kend, f4 (&acc)[ntiles(NB)],
                                          QuadAcc<NB, P>& qa, typename G::Entry* ring, int lane,
                                          Inflight<G::kBuf>& in, void* quad_scratch,
                                          float* wslot, int part_mask) {
    GramBody<NB, P, G, PARTS> body{part_mask, gat, acc, qa, quad_scratch, wslot, lane, {}, {},
                                   0.f};
    pipe_loop(gat, colidx, vals, kbeg, kend, ring, lane, in, body);
}

// The gather stage made visible (test and debug support): for one row, the operands the Gram's
// MFMAs would receive -- the same Gather form, index ring and pipeline as k_herm_solve -- are
// written out per entry instead of multiplied.  Entry k's record has 16 (NB + 3) floats: block I
// of the MFMA operand at 16 I + c (lane c of the entry's 16-lane group), the quad operands w[p] at
// 16 (NB + p) + c (quad form only; untouched otherwise), and the rating the body uses at
// 16 (NB + 2) + c.
template <int NB>
constexpr int dump_floats() { return 16 * (NB + 3); }

template <int NB, int P, class G>
struct DumpBody {
    static constexpr bool kParts = false;
    const G& gat;
    float* __restrict__ out;
    int64_t limit;   // entries that fit in out
    int total, lane, step;
    float v[NB], w[P > 0 ? P : 1], r;
    __device__ __forceinline__ void take(const float (&B)[G::kBuf], float rr, bool ok) {
        gat.operands(B, rr, ok, v, w);
        r = rr;
    }
    template <int J>
    __device__ __forceinline__ void run() {
        const int g = lane >> 4, c = lane & 15;
        const int64_t k = 4 * (int64_t)step + g;
        if (k < total && k < limit) {
            float* rec = out + k * dump_floats<NB>();
#pragma unroll
            for (int I = 0; I < NB; ++I) rec[16 * I + c] = v[I];
            if constexpr (P > 0) {
#pragma unroll
                for (int p = 0; p < P; ++p) rec[16 * (NB + p) + c] = w[p];
            }
            rec[16 * (NB + 2) + c] = r;
        }
        ++step;
    }
};

template <int NB, int BUF, int P>
__global__ __launch_bounds__(kWave) void k_gather_dump(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, const float* __restrict__ theta, int64_t n, int f, int64_t u,
    float* __restrict__ out, int64_t limit) {
    using G = Gather<NB, BUF, P>;
    __shared__ typename G::Entry ring[kRing];
    __shared__ __attribute__((aligned(16))) float stage[BUF == kFormStaged ? stage_floats(NB) : 4];
    const int lane = threadIdx.x;
    if constexpr (BUF == kFormStaged) {
        for (int i = lane; i < stage_floats(NB); i += kWave) stage[i] = 0.f;
        __syncthreads();
    }
    const G gat(theta, n, f, lane & 15, stage);
    const int64_t kbeg = rowptr[u], kend = rowptr[u + 1];
    RowIndex<G> ix;
    Inflight<G::kBuf> in;
    gram_prefetch(gat, colidx, vals, kbeg, kend, lane, ix);
    gram_stage(gat, ix, ring, lane, in);
    DumpBody<NB, P, G> body{gat, out, limit, (int)(kend - kbeg), lane, 0, {}, {}, 0.f};
    pipe_loop(gat, colidx, vals, kbeg, kend, ring, lane, in, body);
}

// ------------------------------------------------------------------ solve in registers ---

// LDS scratch of one wave for the solve.
template <int NB>
struct SolveLds {
    float W[NB][256];   // -W_K = -L_KK^{-1} per block, column-major: W[K][16 j + i] = -W_K[i][j]
    float T[256];       // a diagonal tile, row-major
    float y[16 * NB];   // forward-substitution result (row f of the augmented factor)
    float x[16 * NB];   // solution, zero past f
    float z[16];
};

// Registers of factor_tile (see there).
struct FactorRegs {
    float tr[4], wr[4], to[4], wo[4];   // to/wo[0] unused
};

// Pivot kk = 4 B + P of factor_tile.  The next pivot waits on this one's readlane, s, s^2, the
// product for the next row and that row's update, so the next row (P + 1) is updated first.
// One transcendental per pivot (s = piv^{-1/2}; 1/piv = s^2).
template <int B, int P, bool kFull>
__device__ __forceinline__ void factor_pivot(FactorRegs& R, bool live, int& pmin, int& pmax,
                                             float* ystore) {
    constexpr int kk = 4 * B + P;
    // the pivot T[kk][kk] = -N[kk][kk]: lane kk's value with the sign bit flipped (scalar)
    int pb = __builtin_amdgcn_readlane(__builtin_bit_cast(int, R.tr[P]), kk) ^ 0x80000000;
    pb = live ? pb : 0x3F800000;   // 1.0f
    pmin = min(pmin, pb);
    pmax = max(pmax, pb);
    asm volatile("" : "+s"(pmin), "+s"(pmax));   // fold in now, in scalar registers
    const float s = live ? __builtin_amdgcn_rsqf(__builtin_bit_cast(float, pb)) : 0.f;
    const float s2 = s * s;   // 1 / piv
    const float at = s2 * R.tr[P];          // N[kk][c] / piv
    const float aw = s2 * R.wr[P];          // (-W)[kk][c] / piv
    if (ystore) ystore[kk] = -s * R.tr[P];  // L[nlast][kk] = s T[kk][nlast]
    R.wr[P] *= s;                           // row kk of -W is final
    // Order: row P + 1 (W, then T: the W update reads T's column kk before the T update changes
    // it), then the other rows' W updates, then their T updates.  A DPP read of a T register then
    // sits at least n - 1 instructions after the previous pivot's write of it (n row updates
    // here); a block's first pivot always waits (its sources were loaded or carried over the
    // block's branch).
    // (without the later rows, kFull = false, every pivot waits)
    constexpr int n = (3 - P) + (3 - B);
    if constexpr (P == 0 || n < 3 || !kFull) dpp_settle();
    if constexpr (P < 3) {
        R.wr[P + 1] = fmac_bcast<kk>(R.wr[P + 1], R.tr[P + 1], aw);
        R.tr[P + 1] = fmac_bcast<kk>(R.tr[P + 1], R.tr[P + 1], at);
    }
#pragma unroll
    for (int j = P + 2; j < 4; ++j) R.wr[j] = fmac_bcast<kk>(R.wr[j], R.tr[j], aw);
    if constexpr (kFull) {
#pragma unroll
        for (int bb = B + 1; bb < 4; ++bb) R.wo[bb] = fmac_bcast<kk>(R.wo[bb], R.to[bb], aw);
    }
#pragma unroll
    for (int j = P + 2; j < 4; ++j) R.tr[j] = fmac_bcast<kk>(R.tr[j], R.tr[j], at);
    if constexpr (kFull) {
#pragma unroll
        for (int bb = B + 1; bb < 4; ++bb) R.to[bb] = fmac_bcast<kk>(R.to[bb], R.to[bb], at);
    }
}

// Factor and invert the symmetric 16 x 16 diagonal tile T, staged negated in S.T (row-major:
// N = -T, as the accumulator tiles hold it), right-looking: pivot kk = T[kk][kk] scales row kk of
// W = L_KK^{-1} (built from the identity) by s = piv^{-1/2} and then takes
// T[i][c] -= T[i][kk] T[kk][c] / piv and W[i][c] -= T[i][kk] W[kk][c] / piv for every later row i.
// The registers hold N and -W, for which the same steps read N[i][c] += N[i][kk] N[kk][c] / piv
// and (-W)[i][c] += N[i][kk] (-W)[kk][c] / piv; -W goes to S.W, as the panel and the back
// substitution use it.  Lane (g, c) holds column c.  The rows of the current 4-row block b sit in every group
// (tr, wr: rows 4b + j); a later row 4b' + g is held by group g alone (to, wo[b']), so each
// group updates a quarter of them.  Either way the multiplier T[i][kk] is the row's own register
// in lane kk (DPP row_newbcast:kk), and N[kk][c] / piv, (-W)[kk][c] / piv are the lane's own (the
// current block is replicated).  Between blocks the groups trade the next block's rows through
// LDS.  Columns left of the pivot are not needed again; they go to zero as the elimination
// proceeds instead of being masked.  npiv real pivots: a block with none is skipped (last block
// only) and a pivot past npiv inside a block runs with s = 0, so it adds nothing (a branch per
// pivot would make the register allocator copy DPP sources right before their reads); rows of W
// past npiv stay as the updates left them (the identity in the padding, zero for a pivot skipped
// inside a block).  In the last block the row nlast is the augmented b row, whose L entries are y
// (written to S.y).  pmin/pmax track the pivots' bit patterns: every pivot was positive and
// finite (not NaN, not +inf) iff pmin > 0 and pmax < the bits of +inf.
// kFull = false: the tile has at most 4 real rows (the last block when f - 16 (NB - 1) <= 4).
// Then the rows past the first block are neither pivots nor needed (the b row's L entries come
// from the pivot rows' column nlast), so only block 0 is factored and rows 4..15 of -W are
// written as zeros (the back substitution multiplies them by zeros).
template <int NB, bool kFull, int B = 0>
__device__ __forceinline__ void factor_blocks(SolveLds<NB>& S, FactorRegs& R, int K, int npiv,
                                              float* ystore, int& pmin, int& pmax, int lane) {
    const int g = lane >> 4, c = lane & 15;
    if (4 * B < npiv) {
        factor_pivot<B, 0, kFull>(R, 4 * B + 0 < npiv, pmin, pmax, ystore);
        factor_pivot<B, 1, kFull>(R, 4 * B + 1 < npiv, pmin, pmax, ystore);
        factor_pivot<B, 2, kFull>(R, 4 * B + 2 < npiv, pmin, pmax, ystore);
        factor_pivot<B, 3, kFull>(R, 4 * B + 3 < npiv, pmin, pmax, ystore);
    }
    if constexpr (!kFull) {
        const f4 z = f4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<f4*>(&S.W[K][c * 16 + 4 * g]) =
            g == 0 ? f4{R.wr[0], R.wr[1], R.wr[2], R.wr[3]} : z;
        return;
    }
    if (g == 0)
        *reinterpret_cast<f4*>(&S.W[K][c * 16 + 4 * B]) = f4{R.wr[0], R.wr[1], R.wr[2], R.wr[3]};
    if constexpr (B < 3) {
        // rows 4(B+1) + j: group j's to/wo[B+1] -> every group's tr/wr[j].  The staged tile is
        // in registers now; its LDS holds the exchange.
        float* X = S.T;
        __syncthreads();
        *reinterpret_cast<float2*>(&X[c * 8 + 2 * g]) = float2{R.to[B + 1], R.wo[B + 1]};
        __syncthreads();
        const f4 u0 = *reinterpret_cast<const f4*>(&X[c * 8]);
        const f4 u1 = *reinterpret_cast<const f4*>(&X[c * 8 + 4]);
        R.tr[0] = u0[0]; R.wr[0] = u0[1]; R.tr[1] = u0[2]; R.wr[1] = u0[3];
        R.tr[2] = u1[0]; R.wr[2] = u1[1]; R.tr[3] = u1[2]; R.wr[3] = u1[3];
        factor_blocks<NB, kFull, B + 1>(S, R, K, npiv, ystore, pmin, pmax, lane);
    }
}

template <int NB, bool kFull>
__device__ __forceinline__ void factor_tile(SolveLds<NB>& S, int K, int npiv, int nlast,
                                            int& pmin, int& pmax, int lane) {
    const int g = lane >> 4, c = lane & 15;
    FactorRegs R;
#pragma unroll
    for (int j = 0; j < 4; ++j) R.tr[j] = S.T[c * 16 + j];
    // -identity: row j in lanes c == j; row 4b' + g in lanes 16 g + 4 b' + g
#pragma unroll
    for (int j = 0; j < 4; ++j) R.wr[j] = lane_select_minus_one(0x0001000100010001ull << j);
    R.to[0] = R.wo[0] = 0.f;
    if constexpr (kFull) {
#pragma unroll
        for (int bb = 1; bb < 4; ++bb) R.to[bb] = S.T[c * 16 + 4 * bb + g];
#pragma unroll
        for (int bb = 1; bb < 4; ++bb)
            R.wo[bb] = lane_select_minus_one(0x0008000400020001ull << (4 * bb));
    } else {
#pragma unroll
        for (int bb = 1; bb < 4; ++bb) R.to[bb] = R.wo[bb] = 0.f;
    }
    float* ystore = ((K == NB - 1) && lane == nlast) ? &S.y[16 * K] : nullptr;
    factor_blocks<NB, kFull>(S, R, K, npiv, ystore, pmin, pmax, lane);
}

// Block K's acc-indexed steps, one instantiation per K (the block loop runs at run time so the
// factor code above exists once):
// The tiles not yet factored hold the Schur complement negated (-U), so that the trailing update
// is a plain multiply-accumulate.
//   stage: diagonal tile -U_KK = acc, less lambda n_u on its diagonal (real columns only),
//          -> S.T, so that lane c can read row (= column) c;
//   panel: D_I = W_K U_{K,I} = L_IK^T for I > K (stored positive); y_K from the augmented
//          column; trailing update -U_{J,I} += D_J^T D_I for K < J <= I.  Each product is four
//          16x16x4 MFMAs over the permuted contraction index p = 4g + s, under which lane (g, c)
//          element s of a C-layout tile is both the A operand (of its transpose) and the B
//          operand;
//   matvec: sum_{I>K} D_{K,I}[4g + r][c] x[16 I + c] per lane (summed over c by the caller).
template <int NB, int K>
struct Block {
    static __device__ __forceinline__ void stage(const f4 (&acc)[ntiles(NB)], SolveLds<NB>& S,
                                                 float lam_n, int nlast, int lane) {
        const int g = lane >> 4, c = lane & 15;
        f4 t = acc[tu(NB, K, K)];
        // the diagonal is element r of lanes c == 4g + r
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (c == 4 * g + r && (K < NB - 1 || c < nlast)) t[r] -= lam_n;
        *reinterpret_cast<f4*>(&S.T[c * 16 + 4 * g]) = t;
    }
    static __device__ __forceinline__ void panel(f4 (&acc)[ntiles(NB)], SolveLds<NB>& S,
                                                 int nlast, int lane) {
        if constexpr (K < NB - 1) {
            const int g = lane >> 4, c = lane & 15;
            f4 wop;   // element s: -W_K[c][4g + s] (the tiles hold -U)
#pragma unroll
            for (int s = 0; s < 4; ++s) wop[s] = S.W[K][(4 * g + s) * 16 + c];
#pragma unroll
            for (int I = K + 1; I < NB; ++I) {
                f4 d = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    d = __builtin_amdgcn_mfma_f32_16x16x4f32(wop[s], acc[tu(NB, K, I)][s], d,
                                                             0, 0, 0);
                acc[tu(NB, K, I)] = d;
            }
            if (c == nlast)   // y_K: the augmented column of the last panel tile
                *reinterpret_cast<f4*>(&S.y[16 * K + 4 * g]) = acc[tu(NB, K, NB - 1)];
#pragma unroll
            for (int J = K + 1; J < NB; ++J)
#pragma unroll
                for (int I = J; I < NB; ++I)
#pragma unroll
                    for (int s = 0; s < 4; ++s)
                        acc[tu(NB, J, I)] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            acc[tu(NB, K, J)][s], acc[tu(NB, K, I)][s], acc[tu(NB, J, I)], 0,
                            0, 0);
        }
    }
    static __device__ __forceinline__ f4 matvec(const f4 (&acc)[ntiles(NB)],
                                                const SolveLds<NB>& S, int lane) {
        const int c = lane & 15;
        f4 part = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int I = K + 1; I < NB; ++I) part += acc[tu(NB, K, I)] * S.x[16 * I + c];
        return part;
    }
};

// run-time K -> Block<NB, K>.  Each case ends in its own empty asm statement so that the
// optimiser cannot merge the cases into one access with a run-time tile index (which would move
// the accumulator tiles out of registers).
template <int K>
__device__ __forceinline__ void case_marker() {
    asm volatile("; als block case %0" ::"n"(K));
}
template <int NB, int K = 0>
__device__ __forceinline__ void stage_diag(int k, const f4 (&acc)[ntiles(NB)], SolveLds<NB>& S,
                                           float lam_n, int nlast, int lane) {
    if (k == K) {
        Block<NB, K>::stage(acc, S, lam_n, nlast, lane);
        case_marker<K>();
    } else if constexpr (K + 1 < NB) {
        stage_diag<NB, K + 1>(k, acc, S, lam_n, nlast, lane);
    }
}
template <int NB, int K = 0>
__device__ __forceinline__ void panel_update(int k, f4 (&acc)[ntiles(NB)], SolveLds<NB>& S,
                                             int nlast, int lane) {
    if (k == K) {
        Block<NB, K>::panel(acc, S, nlast, lane);
        case_marker<K>();
    } else if constexpr (K + 1 < NB - 1) {
        panel_update<NB, K + 1>(k, acc, S, nlast, lane);
    }
}
template <int NB, int K = 0>
__device__ __forceinline__ f4 back_matvec(int k, const f4 (&acc)[ntiles(NB)],
                                          const SolveLds<NB>& S, int lane) {
    if (k == K) {
        const f4 r = Block<NB, K>::matvec(acc, S, lane);
        case_marker<K>();
        return r;
    }
    if constexpr (K + 1 < NB) return back_matvec<NB, K + 1>(k, acc, S, lane);
    return f4{0.f, 0.f, 0.f, 0.f};
}

// Regularise and solve, in place on the accumulator tiles (upper block-triangle of the
// augmented matrix M = [A b; b^T .]).  Blocked right-looking Cholesky over the 16-column blocks:
// factor and invert the diagonal tile (factor_tile), then panel and trailing update by MFMA
// (Block::panel).  The augmented column carries b through the same updates, so its entries
// become y = L^{-1} b.  Back substitution x_K = W_K^T (y_K - sum_{I>K} D_{K,I} x_I) runs last
// block first.  Only real pivots (rows < f) are factored; the last block's padding is the
// identity.  Returns false if a pivot was not positive; leaves the solution in S.x (zero past
// f).
template <int NB>
__device__ __forceinline__ bool solve_core(f4 (&acc)[ntiles(NB)], int f, float lam_n,
                                           SolveLds<NB>& S, int lane) {
    const int g = lane >> 4, c = lane & 15;
    const int nlast = f - 16 * (NB - 1);   // real columns of the last block; b is its column nlast
    // -M: the factorisation below keeps unfactored tiles negated (the regularisation joins each
    // diagonal tile as it is staged)
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) acc[t] = -acc[t];

    int pmin = 0x7FFFFFFF, pmax = 0;
    // unrolled: with a run-time block loop every block's results had to be copied back into the
    // loop-carried registers (about 110 register-pair moves per row)
#pragma unroll
    for (int K = 0; K < NB; ++K) {
        stage_diag<NB>(K, acc, S, lam_n, nlast, lane);
        __syncthreads();
        if (K == NB - 1 && nlast <= 4)
            factor_tile<NB, false>(S, K, nlast, nlast, pmin, pmax, lane);
        else
            factor_tile<NB, true>(S, K, (K < NB - 1) ? 16 : nlast, nlast, pmin, pmax, lane);
        __syncthreads();
        panel_update<NB>(K, acc, S, nlast, lane);
    }
    const bool ok = pmin > 0 && pmax < 0x7F800000;   // every pivot positive and finite
    // back substitution, last block first; x is zero past f (b column and padding).  Lane
    // (g, c < 4) finishes entry kk = 4g + c of the block (the transposed row sums put it there);
    // with -W_K in S.W, it works with -z.
    for (int j = lane; j < 16 * NB; j += kWave) S.x[j] = 0.f;
    __syncthreads();
    const int kq = 4 * g + (c & 3);
#pragma unroll
    for (int K = NB - 1; K >= 0; --K) {
        const bool real = K < NB - 1 || kq < nlast;
        const float part = row_sum16_t(back_matvec<NB>(K, acc, S, lane));
        const float nz = real ? part - S.y[16 * K + kq] : 0.f;   // -z[kq]
        if (c < 4) S.z[kq] = nz;
        __syncthreads();
        const float zc = S.z[c];
        f4 xs;
#pragma unroll
        for (int s = 0; s < 4; ++s) xs[s] = S.W[K][(4 * g + s) * 16 + c] * zc;
        const float xv = row_sum16_t(xs);
        if (c < 4) S.x[16 * K + kq] = real ? xv : 0.f;
        __syncthreads();
    }
    return ok;
}

// solve_core, then x_u (f floats, NaN if a pivot was not positive) to xrow.
template <int NB>
__device__ __forceinline__ bool solve_row(f4 (&acc)[ntiles(NB)], int f, float lam_n,
                                          SolveLds<NB>& S, float* __restrict__ xrow, int lane) {
    const bool ok = solve_core<NB>(acc, f, lam_n, S, lane);
    for (int j = lane; j < f; j += kWave) xrow[j] = ok ? S.x[j] : __builtin_nanf("");
    return ok;
}

template <int NB>
__device__ __forceinline__ void write_zero_row(float* __restrict__ xrow, int f, int lane) {
    for (int j = lane; j < f; j += kWave) xrow[j] = 0.f;
}

// ------------------------------------------------------------------------ kernels --------

// Persistent waves claim chunks in order from a counter; chunk c covers the entries from
// bounds[c] to bounds[c+1].  Whole rows are solved here; the piece of a row cut at the start of
// the chunk goes to slot 2c, the piece cut at its end to slot 2c+1, so what is stored where does
// not depend on which wave ran the chunk.  Rows are software-pipelined: the next piece's index
// batches load while this piece's Gram runs, and its first theta gathers are in flight while
// this piece is solved.
struct Piece {
    int64_t u, beg, end;   // row, entry range [beg, end)
    bool whole;            // the chunk holds the whole row
};

template <int NB, int BUF, int P, bool PARTS>
__global__ __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(NB <= 8 ? 2 : 1)))
void k_herm_solve(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, const float* __restrict__ theta, int64_t m, int64_t n,
    int f, float lambda, int C, const int64_t* __restrict__ bounds, float* __restrict__ x_out,
    float* __restrict__ slots, float* __restrict__ wave_slots, int part_mask, int64_t c_row,
    unsigned long long* __restrict__ nonspd, unsigned* __restrict__ chunk_ctr) {
    // Both instantiations (with and without parts) are launched; the one that does not match
    // this call returns at once.  A piece lies within a chunk and within a row: a chunk holds at
    // most ceil(T1 / W) cost units (c_nnz per entry) plus the snapping of its two cut offsets,
    // and a row at most n entries (its columns are distinct).
    {
        const int64_t T = kCostPerEntry * rowptr[m] + c_row * m;
        int64_t longest = (T / (int64_t)gridDim.x + 1) / kCostPerEntry + 2 * kSnap + 1;
        if (longest > n) longest = n;
        if ((longest > (int64_t)kEntriesPerGroup * (part_mask + 1)) != PARTS) return;
    }
    using G = Gather<NB, BUF, P>;
    __shared__ __attribute__((aligned(16))) SolveLds<NB> lds;
    __shared__ typename G::Entry ring[kRing];
    __shared__ __attribute__((aligned(16))) float stage[BUF == kFormStaged ? stage_floats(NB) : 4];
    const int lane = threadIdx.x;
    if constexpr (BUF == kFormStaged) {
        for (int i = lane; i < stage_floats(NB); i += kWave) stage[i] = 0.f;
        __syncthreads();
    }
    const Gather<NB, BUF, P> gat(theta, n, f, lane & 15, stage);
    float* __restrict__ wslot = wave_slots + (size_t)blockIdx.x * slot_floats(NB);
    // No lane-0-only region in the claim loop: every lane takes part in the claim (lane 0 adds
    // one, the others zero), and the wave's count of non-SPD rows stays in a register until the
    // loop has ended (a lane-0 region at each end of a loop body can be joined across the back
    // edge, leaving lanes 1..63 in a loop of their own).
    unsigned bad = 0;
    for (;;) {
        const unsigned got = atomicAdd(chunk_ctr, lane == 0 ? 1u : 0u);
        const int c = __builtin_amdgcn_readfirstlane((int)got);
        if (c >= C) break;
        const int64_t u0 = bounds[2 * c], k0 = bounds[2 * c + 1];
        const int64_t u1 = bounds[2 * c + 2], k1 = bounds[2 * c + 3];
        // the first piece with entries at or after row u; empty rows on the way get x_u = 0
        auto next_piece = [&](int64_t u, Piece& p) -> bool {
            for (; u <= u1 && u < m; ++u) {
                const int64_t rs = rowptr[u], nu = rowptr[u + 1] - rs;
                const int64_t ka = (u == u0) ? k0 : 0;
                int64_t kb = nu;
                if (u == u1) {
                    if (k1 == 0) return false;
                    kb = k1;
                }
                if (nu == 0) {
                    write_zero_row<NB>(x_out + (size_t)u * f, f, lane);
                    continue;
                }
                if (ka >= kb) continue;
                p = Piece{u, rs + ka, rs + kb, ka == 0 && kb == nu};
                return true;
            }
            return false;
        };
        Piece cur;
        if (!next_piece(u0, cur)) continue;
        RowIndex<G> ix;
        Inflight<G::kBuf> in;
        gram_prefetch(gat, colidx, vals, cur.beg, cur.end, lane, ix);
        gram_stage(gat, ix, ring, lane, in);
        for (;;) {
            Piece nxt;
            const bool more = next_piece(cur.u + 1, nxt);
            if (more) gram_prefetch(gat, colidx, vals, nxt.beg, nxt.end, lane, ix);
            f4 acc[ntiles(NB)];
#pragma unroll
            for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
            QuadAcc<NB, P> qa;
            zero_quads<NB, P>(qa);
            gram_loop<NB, P, PARTS>(gat, colidx, vals, cur.beg, cur.end, acc, qa, ring, lane,
                                    in, &lds, wslot, part_mask);
            if (more) gram_stage(gat, ix, ring, lane, in);
            if constexpr (P > 0) {
                static_assert(quad_scratch_bytes<NB, P>() <= sizeof(SolveLds<NB>),
                              "the quad exchange reuses the solve's LDS");
                quad_to_tiles<NB, P>(qa, acc, &lds, lane);
            }
            // a piece longer than a part: its earlier parts' sum is in the wave's slot
            if constexpr (PARTS) {
                if (cur.end - cur.beg > (int64_t)kEntriesPerGroup * (part_mask + 1))
                    add_slot_in_fours<NB>(acc, wslot, lane);
            }
            // the solve is a latency-bound chain; raised priority lets it win issue slots over
            // the other wave's independent Gram MFMAs, which then fill the solve's gaps
            __builtin_amdgcn_s_setprio(2);
            if (cur.whole) {
                const int64_t nu = cur.end - cur.beg;
                const float lam_n = (float)((double)lambda * (double)nu);
                if (!solve_row<NB>(acc, f, lam_n, lds, x_out + (size_t)cur.u * f, lane)) ++bad;
            } else {
                const int which = (cur.u == u0) ? 0 : 1;
                store_slot<NB>(acc, slots + (size_t)(2 * c + which) * slot_floats(NB), lane);
            }
            __builtin_amdgcn_s_setprio(0);
            if (!more) break;
            cur = nxt;
        }
    }
    bad = __builtin_amdgcn_readfirstlane(bad);
    if (bad) atomicAdd(nonspd, lane == 0 ? (unsigned long long)bad : 0ull);
}

// Rows cut by chunk boundaries.  Row u's pieces are: the first, held by chunk b_first - 1 (as
// that chunk's first piece if it started in row u, else as its last), then the piece starting at
// each boundary b_first..b_last that cuts u, in slot 2b (empty, and unwritten, when several
// boundaries snapped to one cut point).  The boundaries cutting one row are consecutive, so both
// ends are found by binary search over the sorted bounds.  A row with more than kPieceGroup
// boundary pieces is summed in two passes: every kPieceGroup-th boundary leads a group and sums
// the group's pieces, in chunk order, into its own slot; then the row's first boundary adds the
// first piece and the group sums, in order, and solves.  The order is fixed, so the result does
// not depend on timing.
constexpr int kPieceGroup = 16;

__device__ __forceinline__ bool cuts_row(const int64_t* __restrict__ rowptr, int64_t m,
                                         const int64_t* __restrict__ bounds, int b) {
    const int64_t u = bounds[2 * b], k = bounds[2 * b + 1];
    return u < m && k > 0 && k < rowptr[u + 1] - rowptr[u];
}

// First and last boundary in [1, C-1] that cut row u, given that boundary b does.  Boundaries
// with row u and an offset strictly inside it form one run around b (bounds are sorted by (row,
// offset): one of row u at offset 0 precedes the run, one at n_u follows it).  Most runs hold one
// or two boundaries, so each end is found by galloping out from b (steps 1, 2, 4, ...) and then
// bisecting the last step: a few dependent loads for a short run instead of a bisection of all C.
__device__ __forceinline__ void cut_range(const int64_t* __restrict__ rowptr, int64_t m,
                                          const int64_t* __restrict__ bounds, int C, int b,
                                          int64_t u, int& b_first, int& b_last) {
    const auto in_run = [&](int x) { return bounds[2 * x] == u && cuts_row(rowptr, m, bounds, x); };
    int in = b, out = 0;   // in the run / below it (0: no boundary below the range)
    for (int d = 1;; d <<= 1) {
        const int x = b - d;
        if (x < 1) break;
        if (!in_run(x)) {
            out = x;
            break;
        }
        in = x;
    }
    while (in - out > 1) {
        const int mid = (in + out) >> 1;
        if (in_run(mid)) in = mid; else out = mid;
    }
    b_first = in;
    in = b;
    out = C;               // above the run (C: no boundary above the range)
    for (int d = 1;; d <<= 1) {
        const int x = b + d;
        if (x > C - 1) break;
        if (!in_run(x)) {
            out = x;
            break;
        }
        in = x;
    }
    while (out - in > 1) {
        const int mid = (in + out) >> 1;
        if (in_run(mid)) in = mid; else out = mid;
    }
    b_last = in;
}

// Add the non-empty boundary pieces of row u for boundaries bb in [from, to] into acc.
template <int NB>
__device__ __forceinline__ void add_pieces(f4 (&acc)[ntiles(NB)], const int64_t* __restrict__ bounds,
                                           const float* __restrict__ slots, int from, int to,
                                           int b_last, int64_t nu, int lane) {
    for (int bb = from; bb <= to; ++bb) {
        // the piece of chunk bb runs to the next boundary in the row, or to the row's end
        const int64_t piece_end = bb < b_last ? bounds[2 * (bb + 1) + 1] : nu;
        if (bounds[2 * bb + 1] < piece_end)
            add_slot<NB>(acc, slots + (size_t)(2 * bb) * slot_floats(NB), lane);
    }
}

// Pass 1: one wave per internal boundary (the loop also serves smaller grids); group leaders of
// long cut rows sum their group.
template <int NB>
__global__ __launch_bounds__(kWave) void k_reduce_groups(
    const int64_t* __restrict__ rowptr, int64_t m, int C, const int64_t* __restrict__ bounds,
    float* __restrict__ slots) {
    const int lane = threadIdx.x;
    for (int b = blockIdx.x + 1; b < C; b += gridDim.x) {
        if (!cuts_row(rowptr, m, bounds, b)) continue;
        const int64_t u = bounds[2 * b];
        int b_first, b_last;
        cut_range(rowptr, m, bounds, C, b, u, b_first, b_last);
        if (b_last - b_first + 1 <= kPieceGroup || (b - b_first) % kPieceGroup != 0) continue;
        f4 acc[ntiles(NB)];
#pragma unroll
        for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
        const int to = b + kPieceGroup - 1 < b_last ? b + kPieceGroup - 1 : b_last;
        add_pieces<NB>(acc, bounds, slots, b, to, b_last, rowptr[u + 1] - rowptr[u], lane);
        store_slot<NB>(acc, slots + (size_t)(2 * b) * slot_floats(NB), lane);
    }
}

// Pass 2: one wave per internal boundary (the loop also serves smaller grids); the first
// boundary that cuts a row sums its pieces (or its group sums) and solves it.
template <int NB>
__device__ __forceinline__ void reduce_row(const int64_t* __restrict__ rowptr, int64_t m, int C,
                                           int f, float lambda, const int64_t* __restrict__ bounds,
                                           float* __restrict__ x_out,
                                           const float* __restrict__ slots, unsigned& bad,
                                           SolveLds<NB>& lds, int b, int lane) {
    if (!cuts_row(rowptr, m, bounds, b)) return;
    const int64_t u = bounds[2 * b];
    if (b > 1 && cuts_row(rowptr, m, bounds, b - 1) && bounds[2 * (b - 1)] == u)
        return;   // not the first cut
    int b_first, b_last;
    cut_range(rowptr, m, bounds, C, b, u, b_first, b_last);
    f4 acc[ntiles(NB)];
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
    // chunk b-1 holds the row's first piece: as its first piece if it started in row u
    // (then at entry 0), else as its last piece
    const int first_slot = (bounds[2 * (b - 1)] == u) ? 2 * (b - 1) : 2 * (b - 1) + 1;
    add_slot<NB>(acc, slots + (size_t)first_slot * slot_floats(NB), lane);
    const int64_t nu = rowptr[u + 1] - rowptr[u];
    if (b_last - b_first + 1 <= kPieceGroup) {
        add_pieces<NB>(acc, bounds, slots, b, b_last, b_last, nu, lane);
    } else {
        for (int g = b; g <= b_last; g += kPieceGroup)
            add_slot<NB>(acc, slots + (size_t)(2 * g) * slot_floats(NB), lane);
    }
    const float lam_n = (float)((double)lambda * (double)nu);
    if (!solve_row<NB>(acc, f, lam_n, lds, x_out + (size_t)u * f, lane)) ++bad;
}

template <int NB>
__global__ __launch_bounds__(kWave) void k_reduce_solve(
    const int64_t* __restrict__ rowptr, int64_t m, int C, int f, float lambda,
    const int64_t* __restrict__ bounds, float* __restrict__ x_out,
    const float* __restrict__ slots, unsigned long long* __restrict__ nonspd) {
    __shared__ __attribute__((aligned(16))) SolveLds<NB> lds;
    const int lane = threadIdx.x;
    unsigned bad = 0;   // non-SPD rows of this wave, added once after the loop
    for (int b = blockIdx.x + 1; b < C; b += gridDim.x)
        reduce_row<NB>(rowptr, m, C, f, lambda, bounds, x_out, slots, bad, lds, b, lane);
    bad = __builtin_amdgcn_readfirstlane(bad);
    if (bad) atomicAdd(nonspd, lane == 0 ? (unsigned long long)bad : 0ull);
}

// RMSE body: per step, entry slot g's residual r - x_u . theta_v in fp32 (the dot product over
// the slot's 16 lanes by DPP row sums); the squares of a group's kGroup steps are summed in fp32
// (at most kGroup terms per lane) and that sum is added in fp64 by the slot's first lane at the
// group's last step.  An entry past the piece's end gathers zeros and rating 0, so its residual
// is 0.  x_u sits in registers: lane (g, c) holds x_u[16 I + c] (0 past f, which also cancels the
// rating that the gather puts in column f).
template <int NB, class G>
struct RmseBody {
    static constexpr bool kParts = false;
    const G& gat;
    const float (&xr)[NB];
    double& acc;
    bool lead;
    float v[NB], w[1], r;
    float sq;   // this group's squares so far
    __device__ __forceinline__ void take(const float (&B)[G::kBuf], float rr, bool ok) {
        gat.operands(B, rr, ok, v, w);
        r = ok ? rr : 0.f;
    }
    template <int J>
    __device__ __forceinline__ void run() {
        float d = 0.f;
#pragma unroll
        for (int I = 0; I < NB; ++I) d = __builtin_fmaf(v[I], xr[I], d);
        d = row_sum16(d);
        const float e = r - d;
        sq = (J == 0) ? e * e : __builtin_fmaf(e, e, sq);
        if constexpr (J == kGroup - 1) acc += lead ? (double)sq : 0.0;
    }
};

// RMSE partials: the entries are cut into C equal chunks, chunk w = [nnz w / C, nnz (w+1) / C);
// persistent waves claim chunks in order from a counter and walk each row piece by row piece
// through the gather pipeline (the next piece's index batches load during the current piece;
// x_u is loaded once per piece).  Chunk w's fp64 sum goes to partial[w], so the result does not
// depend on how many waves run or which wave took which chunk: the kernel may run at any width,
// e.g. one wave per SIMD beside a half-sweep.  NB = f / 16 + 1 (the gather's block count).
template <int NB, bool BUF>
__global__ __launch_bounds__(kWave) void k_rmse_rows(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, int64_t m, int64_t n, int f, const float* __restrict__ x,
    const float* __restrict__ theta, int C, double* __restrict__ partial,
    unsigned* __restrict__ claim) {
    using G = Gather<NB, BUF ? kFormBuffer : kFormGlobal, 0>;
    __shared__ typename G::Entry ring[kRing];
    const int lane = threadIdx.x, c = lane & 15;
    const int64_t nnz = rowptr[m];
    // No lane-0-only region in this loop: every lane takes part in the claim (lane 0 adds one,
    // the others zero) and every lane stores the wave's sum.  (Two lane-0 regions at the ends of
    // the loop body were joined across the back edge by the compiler, leaving lanes 1..63 in a
    // loop of their own that read a stale chunk number.)
    for (;;) {
        const unsigned got = atomicAdd(claim, lane == 0 ? 1u : 0u);
        const int w = __builtin_amdgcn_readfirstlane((int)got);
        if (w >= C) break;
        const int64_t kb = nnz / C * w + (nnz % C) * w / C;
        const int64_t ke = nnz / C * (w + 1) + (nnz % C) * (w + 1) / C;
        double acc = 0.0;
        if (kb < ke) {
            int64_t lo = 0, hi = m - 1;   // row of entry kb: largest u < m with rowptr[u] <= kb
            while (lo < hi) {
                const int64_t mid = (lo + hi + 1) >> 1;
                if (rowptr[mid] <= kb) lo = mid; else hi = mid - 1;
            }
            int64_t u = lo;
            int64_t pb = kb, pe = rowptr[u + 1] < ke ? rowptr[u + 1] : ke;
            const G gat(theta, n, f, c);
            RowIndex<G> ix;
            Inflight<G::kBuf> in;
            gram_prefetch(gat, colidx, vals, pb, pe, lane, ix);
            gram_stage(gat, ix, ring, lane, in);
            for (;;) {
                int64_t un = u + 1;   // the next row with entries in the range
                while (un < m && rowptr[un] < ke && rowptr[un + 1] == rowptr[un]) ++un;
                const bool more = un < m && rowptr[un] < ke;
                int64_t nb0 = 0, nb1 = 0;
                if (more) {
                    nb0 = rowptr[un];
                    nb1 = rowptr[un + 1] < ke ? rowptr[un + 1] : ke;
                    gram_prefetch(gat, colidx, vals, nb0, nb1, lane, ix);
                }
                float xr[NB];
#pragma unroll
                for (int I = 0; I < NB; ++I) {
                    const int j = 16 * I + c;
                    xr[I] = j < f ? x[(size_t)u * (size_t)f + j] : 0.f;
                }
                RmseBody<NB, G> body{gat, xr, acc, c == 0, {}, {}, 0.f, 0.f};
                pipe_loop(gat, colidx, vals, pb, pe, ring, lane, in, body);
                if (!more) break;
                gram_stage(gat, ix, ring, lane, in);
                u = un;
                pb = nb0;
                pe = nb1;
            }
        }
        // only the 16-lane groups' first lanes hold sums: the full butterfly leaves the wave's
        // total in every lane
        for (int o = 1; o < kWave; o <<= 1) acc += __shfl_xor(acc, o);
        partial[w] = acc;
    }
}

__global__ __launch_bounds__(kWave) void k_rmse_final(const int64_t* __restrict__ rowptr,
                                                      int64_t m, int W,
                                                      const double* __restrict__ partial,
                                                      double* __restrict__ out) {
    const int lane = threadIdx.x;
    double s = 0.0;
    for (int i = lane; i < W; i += kWave) s += partial[i];
    for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) {
        const int64_t nnz = rowptr[m];
        out[0] = nnz > 0 ? sqrt(s / (double)nnz) : 0.0;
    }
}

__global__ void k_reset_counter(unsigned long long* p) { *p = 0ull; }

// ------------------------------------------------------------------ CSR -> CSC -----------

// The transpose R -> R^T that the update-Theta half-sweep reads (eq. 3 is the same method on
// the columns of R).  Stable: within a column the entries keep the order of their rows.
// The rows are cut into R row blocks of about nnz / R entries each (whole rows; block b holds
// rows [tr_row_begin(b), tr_row_begin(b+1))).  cnt[b][v] counts block b's entries in column v;
// a prefix over b turns it into the offset of block b's first entry within column v, and one
// wave per block then walks its rows in order, so every column receives its rows ascending.
// Entries whose column lies outside [0, n) are skipped by every pass (the contract leaves them
// undefined; skipping keeps every access in bounds).

// First row of row block b: the smallest u with rowptr[u] >= floor(b nnz / R) (binary search).
__device__ __forceinline__ int64_t tr_row_begin(const int64_t* __restrict__ rowptr, int64_t m,
                                                int R, int b) {
    const int64_t nnz = rowptr[m];
    // floor(nnz b / R) without overflow: nnz = q R + r, r b < R^2
    const int64_t target = (nnz / R) * b + ((nnz % R) * b) / R;
    int64_t lo = 0, hi = m;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (rowptr[mid] < target) lo = mid + 1; else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(256) void k_tr_zero(int32_t* __restrict__ p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * 256)
        p[i] = 0;
}

// cnt[b][v] += 1 for every entry of row block b (one workgroup per block; the order of the
// increments does not matter).
__global__ __launch_bounds__(256) void k_tr_count(const int64_t* __restrict__ rowptr,
                                                  const int32_t* __restrict__ colidx, int64_t m,
                                                  int64_t n, int R, int32_t* __restrict__ cnt) {
    const int b = blockIdx.x;
    const int64_t k0 = rowptr[tr_row_begin(rowptr, m, R, b)];
    const int64_t k1 = rowptr[tr_row_begin(rowptr, m, R, b + 1)];
    int32_t* row = cnt + (size_t)b * (size_t)n;
    for (int64_t k = k0 + threadIdx.x; k < k1; k += 256) {
        const int32_t v = colidx[k];
        if (v >= 0 && v < n) atomicAdd(&row[v], 1);
    }
}

// Per column v (one thread each): cnt[b][v] <- the sum over b' < b, and colptr[v] <- the
// column's total (scanned over v afterwards).
__global__ __launch_bounds__(256) void k_tr_colscan(int64_t n, int R, int32_t* __restrict__ cnt,
                                                    int64_t* __restrict__ colptr) {
    const int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (v >= n) return;
    int32_t run = 0;
    for (int b = 0; b < R; ++b) {
        int32_t* c = cnt + (size_t)b * (size_t)n + v;
        const int32_t t = *c;
        *c = run;
        run += t;
    }
    colptr[v] = run;
}

// Exclusive scan of a[0, len) in place, a[len] <- the total: tile sums (kScanTile elements per
// workgroup), a scan of the tile sums by one workgroup, then each tile scanned with its offset.
constexpr int kScanPer = 16;
constexpr int kScanTile = 256 * kScanPer;

// Exclusive scan of one value per thread over a workgroup of 256 (4 waves); returns the prefix
// and sets *total.
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t x, int64_t* sh, int64_t* total) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    int64_t inc = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int64_t y = __shfl_up(inc, o);
        if (lane >= o) inc += y;
    }
    if (lane == 63) sh[w] = inc;
    __syncthreads();
    int64_t base = 0;
    for (int i = 0; i < w; ++i) base += sh[i];
    *total = sh[0] + sh[1] + sh[2] + sh[3];
    __syncthreads();
    return base + inc - x;
}

__global__ __launch_bounds__(256) void k_scan_sums(const int64_t* __restrict__ a, int64_t len,
                                                   int64_t* __restrict__ sums) {
    __shared__ int64_t sh[4];
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    int64_t x = 0;
    for (int j = 0; j < kScanPer; ++j) {
        const int64_t i = base + (int64_t)threadIdx.x * kScanPer + j;
        if (i < len) x += a[i];
    }
    int64_t total;
    (void)block_exclusive_scan(x, sh, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(256) void k_scan_top(int64_t* __restrict__ sums, int64_t tiles,
                                                  int64_t* __restrict__ a, int64_t len) {
    __shared__ int64_t sh[4];
    int64_t carry = 0;
    for (int64_t c = 0; c < tiles; c += 256) {
        const int64_t i = c + threadIdx.x;
        const int64_t x = i < tiles ? sums[i] : 0;
        int64_t total;
        const int64_t ex = block_exclusive_scan(x, sh, &total);
        if (i < tiles) sums[i] = carry + ex;
        carry += total;
    }
    if (threadIdx.x == 0) a[len] = carry;
}

__global__ __launch_bounds__(256) void k_scan_apply(int64_t* __restrict__ a, int64_t len,
                                                    const int64_t* __restrict__ sums) {
    __shared__ int64_t sh[4];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanPer;
    int64_t v[kScanPer];
    int64_t x = 0;
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        v[j] = base + j < len ? a[base + j] : 0;
        x += v[j];
    }
    int64_t total;
    int64_t run = sums[blockIdx.x] + block_exclusive_scan(x, sh, &total);
#pragma unroll
    for (int j = 0; j < kScanPer; ++j) {
        if (base + j < len) a[base + j] = run;
        run += v[j];
    }
}

// LDS forms of the count and the scatter, for n <= kTrLdsCols: the block's per-column counters
// (cursors) live in the workgroup's LDS.  Counting: one workgroup of 256 per row block adds its
// entries into LDS and writes the n counts out.  Scatter: one wave per row block loads
// colptr[v] + cnt[b][v] into LDS and walks its rows in order; a wave's LDS atomics are performed
// in issue order, so a column's entries again arrive in row order.
constexpr int kTrLdsCols = 40960;   // 160 KB of int32 counters

__global__ __launch_bounds__(256) void k_tr_count_lds(const int64_t* __restrict__ rowptr,
                                                      const int32_t* __restrict__ colidx,
                                                      int64_t m, int n, int R,
                                                      int32_t* __restrict__ cnt) {
    extern __shared__ int32_t lcnt[];
    const int b = blockIdx.x;
    for (int v = threadIdx.x; v < n; v += 256) lcnt[v] = 0;
    __syncthreads();
    const int64_t k0 = rowptr[tr_row_begin(rowptr, m, R, b)];
    const int64_t k1 = rowptr[tr_row_begin(rowptr, m, R, b + 1)];
    for (int64_t k = k0 + threadIdx.x; k < k1; k += 256) {
        const int32_t v = colidx[k];
        if (v >= 0 && v < n) atomicAdd(&lcnt[v], 1);
    }
    __syncthreads();
    int32_t* row = cnt + (size_t)b * (size_t)n;
    for (int v = threadIdx.x; v < n; v += 256) row[v] = lcnt[v];
}

__global__ __launch_bounds__(kWave) void k_tr_scatter_lds(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, int64_t m, int n, int R, const int32_t* __restrict__ cnt,
    const int64_t* __restrict__ colptr, int32_t* __restrict__ rowidx,
    float* __restrict__ vals_t) {
    // cur[v]: where this block's next entry of column v goes -- its absolute position when
    // nnz < 2^31 (then no colptr read per entry), else its position within column v's run
    extern __shared__ int32_t cur[];
    const int b = blockIdx.x, lane = threadIdx.x;
    const bool absolute = rowptr[m] <= (int64_t)INT32_MAX;
    const int32_t* row = cnt + (size_t)b * (size_t)n;
    for (int v = lane; v < n; v += kWave)
        cur[v] = absolute ? (int32_t)(colptr[v] + row[v]) : row[v];
    __syncthreads();
    const int64_t u0 = tr_row_begin(rowptr, m, R, b), u1 = tr_row_begin(rowptr, m, R, b + 1);
    // chunks of up to 64 entries of one row, in order; the next chunk's column indices and
    // ratings load while this one is placed (a chunk never spans two rows, so the lanes of one
    // LDS atomic never share a column)
    int64_t u = u0, ks = 0, ke = 0;
    auto next_chunk = [&](int64_t& cu, int64_t& cs, int64_t& ce) {
        if (cs + kWave < ce) {
            cs += kWave;
            return;
        }
        for (++cu; cu < u1; ++cu) {
            cs = rowptr[cu];
            ce = rowptr[cu + 1];
            if (cs < ce) return;
        }
    };
    u = u0 - 1;
    next_chunk(u, ks, ke);   // the first chunk (ks + kWave >= ke = 0 starts the row walk)
    int32_t v = -1;
    float r = 0.f;
    if (u < u1 && ks + lane < ke) {
        v = colidx[ks + lane];
        r = vals[ks + lane];
    }
    while (u < u1) {
        int64_t nu = u, ns = ks, ne = ke;
        next_chunk(nu, ns, ne);
        int32_t nv = -1;
        float nr = 0.f;
        if (nu < u1 && ns + lane < ne) {
            nv = colidx[ns + lane];
            nr = vals[ns + lane];
        }
        if (ks + lane < ke && v >= 0 && v < n) {
            const int32_t at = atomicAdd(&cur[v], 1);
            const int64_t pos = absolute ? (int64_t)at : colptr[v] + at;
            rowidx[pos] = (int32_t)u;
            vals_t[pos] = r;
        }
        u = nu;
        ks = ns;
        ke = ne;
        v = nv;
        r = nr;
    }
}

// One wave per row block, its rows in order: each entry goes to colptr[v] + cnt[b][v], which
// then moves on by one.  The columns of one row are distinct, so the lanes of a row never share
// a counter; the fence after each row orders its counter updates before the next row's.
__global__ __launch_bounds__(kWave) void k_tr_scatter(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, int64_t m, int64_t n, int R, int32_t* __restrict__ cnt,
    const int64_t* __restrict__ colptr, int32_t* __restrict__ rowidx,
    float* __restrict__ vals_t) {
    const int b = blockIdx.x, lane = threadIdx.x;
    const int64_t u0 = tr_row_begin(rowptr, m, R, b), u1 = tr_row_begin(rowptr, m, R, b + 1);
    int32_t* row = cnt + (size_t)b * (size_t)n;
    for (int64_t u = u0; u < u1; ++u) {
        const int64_t k1 = rowptr[u + 1];
        for (int64_t k = rowptr[u] + lane; k < k1; k += kWave) {
            const int32_t v = colidx[k];
            if (v >= 0 && v < n) {
                const int32_t at = atomicAdd(&row[v], 1);
                const int64_t pos = colptr[v] + at;
                rowidx[pos] = (int32_t)u;
                vals_t[pos] = vals[k];
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    }
}

// --------------------------------------------------------------------- host side ---------

struct Layout {
    size_t status, bounds, rmse, slots, wave_slots, total;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// waves[nb] = W for f in (16 (nb-1), 16 nb]; the slot region holds 2 C partial accumulators,
// C = chunks_of(W), and the wave-slot region one more per wave (the second summation level of
// long pieces)
Layout make_layout(const int* waves, int nb_max, int cus) {
    int c_cap = 1;
    size_t slot_bytes = 0, wave_bytes = 0;
    for (int nb = 1; nb <= nb_max; ++nb) {
        const int C = chunks_of(waves[nb]);
        if (C > c_cap) c_cap = C;
        const size_t sb = sizeof(float) * (size_t)slot_floats(nb) * 2 * (size_t)C;
        if (sb > slot_bytes) slot_bytes = sb;
        const size_t wb = sizeof(float) * (size_t)slot_floats(nb) * (size_t)waves[nb];
        if (wb > wave_bytes) wave_bytes = wb;
    }
    Layout L;
    size_t off = 0;
    L.status = off; off = align256(off + 256);   // non-SPD counter at 0, chunk counters at 64, 128
    L.bounds = off; off = align256(off + sizeof(int64_t) * 2 * (size_t)(c_cap + 1));
    L.rmse = off;   off = align256(off + sizeof(double) * (size_t)cus * kRmseWavesPerCU);
    L.slots = off;  off = align256(off + slot_bytes);
    L.wave_slots = off; off = align256(off + wave_bytes);
    L.total = off;
    return L;
}

// Resident waves per CU of both gather forms (the partition is shared, so every wave of either
// form is resident at once).
template <int NB>
int occupancy_waves(int cus, int* waves) {
    int blocks = 1 << 30;
    const void* forms[] = {(const void*)k_herm_solve<NB, kFormBuffer, 0, false>,
                           (const void*)k_herm_solve<NB, kFormBuffer, 1, false>,
                           kQuad2<NB> ? (const void*)k_herm_solve<NB, kFormBuffer,
                                                                  kQuad2<NB> ? 2 : 1, false>
                                      : nullptr,
                           (const void*)k_herm_solve<NB, kFormGlobal, 0, false>,
                           (const void*)k_herm_solve<NB, kFormGlobal, 1, false>,
                           kQuad2<NB> ? (const void*)k_herm_solve<NB, kFormGlobal,
                                                                  kQuad2<NB> ? 2 : 1, false>
                                      : nullptr,
                           (const void*)k_herm_solve<NB, kFormBuffer, 0, true>,
                           (const void*)k_herm_solve<NB, kFormBuffer, 1, true>,
                           kQuad2<NB> ? (const void*)k_herm_solve<NB, kFormBuffer,
                                                                  kQuad2<NB> ? 2 : 1, true>
                                      : nullptr,
                           (const void*)k_herm_solve<NB, kFormGlobal, 0, true>,
                           (const void*)k_herm_solve<NB, kFormGlobal, 1, true>,
                           kQuad2<NB> ? (const void*)k_herm_solve<NB, kFormGlobal,
                                                                  kQuad2<NB> ? 2 : 1, true>
                                      : nullptr};
    for (const void* k : forms) {
        if (!k) continue;
        int b = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, k, kWave, 0) != hipSuccess) return -1;
        if (b < blocks) blocks = b;
    }
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxWavesPerCU) blocks = kMaxWavesPerCU;
    const char* env = getenv("ALS_WAVES_PER_CU");
    if (env && atoi(env) > 0) blocks = atoi(env) < blocks ? atoi(env) : blocks;
    *waves = blocks * cus;
    return 0;
}

// Launch the RMSE partials kernel over C = cus * kRmseWavesPerCU chunks (the partials buffer
// holds that many) with as many resident waves as fit, at most `cap_per_cu` per CU if that is
// positive; the claim counter is reset first, on the same stream.
template <int NB, bool BUF>
hipError_t rmse_rows_launch(int cus, int cap_per_cu, hipStream_t st, const int64_t* rowptr,
                            const int32_t* colidx, const float* vals, int64_t m, int64_t n,
                            int f, const float* x, const float* theta, double* part,
                            unsigned* claim, int C) {
    int b = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &b, (const void*)k_rmse_rows<NB, BUF>, kWave, 0);
    if (e != hipSuccess) return e;
    b = b < 1 ? 1 : (b > kRmseWavesPerCU ? kRmseWavesPerCU : b);
    if (cap_per_cu > 0 && b > cap_per_cu) b = cap_per_cu;
    hipLaunchKernelGGL(k_reset_counter, dim3(1), dim3(1), 0, st, (unsigned long long*)claim);
    hipLaunchKernelGGL((k_rmse_rows<NB, BUF>), dim3(cus * b), dim3(kWave), 0, st, rowptr,
                       colidx, vals, m, n, f, x, theta, C, part, claim);
    return hipGetLastError();
}

int waves_for_nb(int nb, int cus, int* w) {
    switch (nb) {
        case 1: return occupancy_waves<1>(cus, w);
        case 2: return occupancy_waves<2>(cus, w);
        case 3: return occupancy_waves<3>(cus, w);
        case 4: return occupancy_waves<4>(cus, w);
        case 5: return occupancy_waves<5>(cus, w);
        case 6: return occupancy_waves<6>(cus, w);
        case 7: return occupancy_waves<7>(cus, w);
        case 8: return occupancy_waves<8>(cus, w);
        case 9: return occupancy_waves<9>(cus, w);
        default: return -1;
    }
}

template <int NB>
int staged_occupancy(int cus, int* waves) {
    int b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &b, (const void*)k_herm_solve<NB, kFormStaged, 0, true>, kWave, 0) != hipSuccess)
        return -1;
    int b2 = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &b2, (const void*)k_herm_solve<NB, kFormStaged, 0, false>, kWave, 0) != hipSuccess)
        return -1;
    if (b2 < b) b = b2;
    if (b < 1) b = 1;
    if (b > kMaxWavesPerCU) b = kMaxWavesPerCU;
    *waves = b * cus;
    return 0;
}

int staged_waves_for_nb(int nb, int cus, int* w) {
    switch (nb) {
        case 1: return staged_occupancy<1>(cus, w);
        case 2: return staged_occupancy<2>(cus, w);
        case 3: return staged_occupancy<3>(cus, w);
        case 4: return staged_occupancy<4>(cus, w);
        case 5: return staged_occupancy<5>(cus, w);
        case 6: return staged_occupancy<6>(cus, w);
        case 7: return staged_occupancy<7>(cus, w);
        case 8: return staged_occupancy<8>(cus, w);
        case 9: return staged_occupancy<9>(cus, w);
        default: return -1;
    }
}

int nb_of(int f) { return f / 16 + 1; }   // blocks of 16 covering the augmented f + 1

// Solve cost of one row in c_nnz units: per 16-column block about 2,500 cycles of factor and
// inverse on the vector ALU plus the panel and trailing-update MFMAs (32 cycles each); the
// vector part overlaps other waves' matrix work, so half of the total is charged.  Tunable
// through ALS_ROW_COST (entries per row).
int64_t row_cost(int f) {
    const char* env = getenv("ALS_ROW_COST");
    if (env && atoll(env) > 0) return atoll(env) * kCostPerEntry;
    const int nb = nb_of(f);
    const double mfma_cycles_per_entry = 8.0 * ntiles(nb);
    double mfmas = 0;
    for (int K = 0; K < nb; ++K) mfmas += 4.0 * ((nb - K - 1) + (nb - K - 1) * (nb - K) / 2.0);
    const double solve_cycles = 2500.0 * nb + 32.0 * mfmas;
    double entries = 0.5 * solve_cycles / mfma_cycles_per_entry;
    if (entries < 1.0) entries = 1.0;
    return (int64_t)(entries * kCostPerEntry);
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

struct als_ctx {
    int device;
    int cus;
    int f_max;
    int nb_max;
    int w_cap;
    int waves[kMaxNB + 1];
    unsigned char* ws;
    size_t ws_bytes;
    Layout lay;
    int last_hip;
    hipEvent_t* prof_ev;   // 4 events per profiled half-sweep, or null
    int prof_cap;
    int prof_count;
    bool global_gather;    // use the 64-bit-load gather for every size (ALS_GATHER=global)
    bool staged_gather;    // stage theta through LDS (ALS_GATHER=lds; ablation)
    bool tile_last_block;  // 16x16 tiles for the last block column always (ALS_LAST_BLOCK=tiles)
    int rmse_waves_per_simd;   // cap on resident RMSE waves per SIMD (0 = as many as fit)
    int part_groups;           // pipeline groups per part of a long piece (a power of two)
    size_t lds_per_block;      // the device's LDS bytes per workgroup
};

namespace {

int fail_hip(als_ctx* ctx, hipError_t e) {
    if (ctx) ctx->last_hip = (int)e;
    return ALS_ERR_HIP;
}

struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        ok = (prev == dev) || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

int query_device(int device, int f_max, int* cus, int* waves, int* w_cap,
                 size_t* lds_per_block = nullptr) {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return ALS_ERR_DEVICE;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) return ALS_ERR_DEVICE;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return ALS_ERR_DEVICE;
    *cus = prop.multiProcessorCount;
    if (lds_per_block) *lds_per_block = prop.sharedMemPerBlock;
    DeviceGuard guard(device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    *w_cap = 1;
    for (int nb = 1; nb <= nb_of(f_max); ++nb) {
        if (waves_for_nb(nb, *cus, &waves[nb]) != 0) return ALS_ERR_HIP;
        if (waves[nb] > *w_cap) *w_cap = waves[nb];
    }
    return ALS_OK;
}

// theta sizes (bytes) served by the buffer-load gather: offsets past the end, plus a padding
// lane's offset, must stay below 2^32
constexpr uint64_t kBufferGatherMax = 0x7FFFF000ull;

// The staged gather (an ablation form) reads whole 16-byte groups of a row through one buffer
// descriptor.
bool staged_supported(int64_t n, int f) {
    return f % 4 == 0 && (uint64_t)n * (uint64_t)f * sizeof(float) <= kBufferGatherMax;
}

struct HermArgs {
    const int64_t* rowptr;
    const int32_t* colidx;
    const float* vals;
    const float* theta;
    int64_t m, n;
    int f;
    float lambda;
    int C;
    const int64_t* bounds;
    float* x;
    float* slots;
    float* wslots;
    int part_mask;
    int64_t c_row;
    unsigned long long* nonspd;
    unsigned* chunk_ctr;
};

// Both instantiations; the kernels pick the one that runs from rowptr[m] on the device (no
// host synchronisation), the other returns at once.
template <int NB, int BUF, int P>
void launch_herm(int W, hipStream_t st, const HermArgs& a) {
    hipLaunchKernelGGL((k_herm_solve<NB, BUF, P, false>), dim3(W), dim3(kWave), 0, st,
                       a.rowptr, a.colidx, a.vals, a.theta, a.m, a.n, a.f, a.lambda, a.C,
                       a.bounds, a.x, a.slots, a.wslots, a.part_mask, a.c_row, a.nonspd,
                       a.chunk_ctr);
    hipLaunchKernelGGL((k_herm_solve<NB, BUF, P, true>), dim3(W), dim3(kWave), 0, st,
                       a.rowptr, a.colidx, a.vals, a.theta, a.m, a.n, a.f, a.lambda, a.C,
                       a.bounds, a.x, a.slots, a.wslots, a.part_mask, a.c_row, a.nonspd,
                       a.chunk_ctr);
}

template <int NB>
void launch_sweep(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                  int64_t m, int64_t n, int f, float lambda, const float* theta, float* x,
                  hipStream_t st, int W) {
    int64_t* bounds = (int64_t*)(ctx->ws + ctx->lay.bounds);
    float* slots = (float*)(ctx->ws + ctx->lay.slots);
    float* wslots = (float*)(ctx->ws + ctx->lay.wave_slots);
    const int part_mask = ctx->part_groups - 1;
    auto* nonspd = (unsigned long long*)(ctx->ws + ctx->lay.status);
    auto* chunk_ctr = (unsigned*)(ctx->ws + ctx->lay.status + 64);
    const int C = chunks_of(W);
    hipEvent_t* ev = nullptr;
    if (ctx->prof_ev && ctx->prof_count < ctx->prof_cap) ev = ctx->prof_ev + 4 * ctx->prof_count++;
    if (ev) (void)hipEventRecord(ev[0], st);
    hipLaunchKernelGGL(k_plan, dim3((C + 1 + 63) / 64), dim3(64), 0, st, rowptr, m, W, C,
                       (int64_t)kCostPerEntry, row_cost(f), (int64_t)kSnap, bounds, chunk_ctr);
    if (ev) (void)hipEventRecord(ev[1], st);
    // the quad form of the last block column: when its theta columns fill whole quads (none or
    // one) and the rating starts a quad of its own
    const int f_last = f - 16 * (NB - 1);
    const int quads =
        (!ctx->tile_last_block && (f_last == 0 || f_last == 4)) ? f_last / 4 + 1 : 0;
    const HermArgs a{rowptr, colidx, vals, theta, m, n, f, lambda, C, bounds, x, slots, wslots,
                     part_mask, row_cost(f), nonspd, chunk_ctr};
    if (ctx->staged_gather) {   // f % 4 == 0 and theta below 2 GiB (checked by the caller)
        launch_herm<NB, kFormStaged, 0>(W, st, a);
    } else if (!ctx->global_gather &&
               (uint64_t)n * (uint64_t)f * sizeof(float) <= kBufferGatherMax) {
        if (quads == 1) {
            launch_herm<NB, kFormBuffer, 1>(W, st, a);
        } else if (quads == 2) {
            if constexpr (kQuad2<NB>) launch_herm<NB, kFormBuffer, 2>(W, st, a);
        } else {
            launch_herm<NB, kFormBuffer, 0>(W, st, a);
        }
    } else {
        if (quads == 1) {
            launch_herm<NB, kFormGlobal, 1>(W, st, a);
        } else if (quads == 2) {
            if constexpr (kQuad2<NB>) launch_herm<NB, kFormGlobal, 2>(W, st, a);
        } else {
            launch_herm<NB, kFormGlobal, 0>(W, st, a);
        }
    }
    if (ev) (void)hipEventRecord(ev[2], st);
    if (C > 1) {
        // one wave per boundary: the rows' solves run side by side
        hipLaunchKernelGGL(k_reduce_groups<NB>, dim3(C - 1), dim3(kWave), 0, st, rowptr, m, C,
                           bounds, slots);
        hipLaunchKernelGGL(k_reduce_solve<NB>, dim3(C - 1), dim3(kWave), 0, st, rowptr, m, C, f,
                           lambda, bounds, x, slots, nonspd);
    }
    if (ev) (void)hipEventRecord(ev[3], st);
}

// The gather form k_herm_solve would use for this call (buffer loads or 64-bit loads; quad form or
// tiles for the last block column), run by k_gather_dump on row u.
template <int NB>
void launch_dump(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                 int64_t n, int f, const float* theta, int64_t u, float* out, int64_t limit,
                 hipStream_t st) {
    const int f_last = f - 16 * (NB - 1);
    const int quads =
        (!ctx->tile_last_block && (f_last == 0 || f_last == 4)) ? f_last / 4 + 1 : 0;
    if (ctx->staged_gather) {
        hipLaunchKernelGGL((k_gather_dump<NB, kFormStaged, 0>), dim3(1), dim3(kWave), 0, st,
                           rowptr, colidx, vals, theta, n, f, u, out, limit);
    } else if (!ctx->global_gather &&
               (uint64_t)n * (uint64_t)f * sizeof(float) <= kBufferGatherMax) {
        if (quads == 1)
            hipLaunchKernelGGL((k_gather_dump<NB, kFormBuffer, 1>), dim3(1), dim3(kWave), 0, st, rowptr,
                               colidx, vals, theta, n, f, u, out, limit);
        else if (quads == 2) {
            if constexpr (kQuad2<NB>)
                hipLaunchKernelGGL((k_gather_dump<NB, kFormBuffer, 2>), dim3(1), dim3(kWave), 0, st,
                                   rowptr, colidx, vals, theta, n, f, u, out, limit);
        } else
            hipLaunchKernelGGL((k_gather_dump<NB, kFormBuffer, 0>), dim3(1), dim3(kWave), 0, st, rowptr,
                               colidx, vals, theta, n, f, u, out, limit);
    } else {
        if (quads == 1)
            hipLaunchKernelGGL((k_gather_dump<NB, kFormGlobal, 1>), dim3(1), dim3(kWave), 0, st,
                               rowptr, colidx, vals, theta, n, f, u, out, limit);
        else if (quads == 2) {
            if constexpr (kQuad2<NB>)
                hipLaunchKernelGGL((k_gather_dump<NB, kFormGlobal, 2>), dim3(1), dim3(kWave), 0,
                                   st, rowptr, colidx, vals, theta, n, f, u, out, limit);
        } else
            hipLaunchKernelGGL((k_gather_dump<NB, kFormGlobal, 0>), dim3(1), dim3(kWave), 0, st,
                               rowptr, colidx, vals, theta, n, f, u, out, limit);
    }
}

// ---------------------------------------------------------- fixed scratch (no workspace) ---

// als_rmse_noalloc's scratch: the claim counter (at 0) and one fp64 partial per RMSE chunk (at
// 256), for devices of up to kNoAllocMaxCUs compute units.  Each device holds its own copy of
// the array; host code reaches a device's copy only through the address hipGetSymbolAddress
// returns with that device current (the array's name is a host-side stand-in).
constexpr int kNoAllocMaxCUs = 320;
constexpr size_t kNoAllocPartials = 256;
constexpr size_t kNoAllocScratchBytes =
    kNoAllocPartials + sizeof(double) * (size_t)kNoAllocMaxCUs * kRmseWavesPerCU;
constexpr int kNoAllocMaxDevices = 64;

struct NoAllocDevice {
    std::once_flag once;
    int rc = ALS_ERR_DEVICE;
    unsigned char* ptr = nullptr;   // this device's copy of the scratch array
    int cus = 0;
};
NoAllocDevice g_noalloc[kNoAllocMaxDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

// Once per device, with that device current: its compute units and the device address of its
// copy of `scratch`.  Called by als_init and by the first als_rmse_noalloc on a device.
int noalloc_setup(int device) {
    if (device < 0 || device >= kNoAllocMaxDevices) return ALS_ERR_DEVICE;
    NoAllocDevice& d = g_noalloc[device];
    std::call_once(d.once, [&d, device]() {
        int n = 0;
        if (hipGetDeviceCount(&n) != hipSuccess || device >= n) return;
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, device) != hipSuccess) return;
        if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return;
        DeviceGuard guard(device);
        if (!guard.ok) return;
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
            d.rc = ALS_ERR_HIP;
            return;
        }
        d.ptr = (unsigned char*)ptr;
        d.cus = prop.multiProcessorCount;
        d.rc = ALS_OK;
    });
    return d.rc;
}

int rmse_check(const int64_t* rowptr, const int32_t* colidx, const float* vals, int64_t m,
               int64_t n, int32_t f, const float* x, const float* theta, const double* rmse_out) {
    if (f < 1 || f > ALS_F_MAX) return ALS_ERR_UNSUPPORTED_F;
    if (m < 0 || n < 0 || !rowptr || !rmse_out) return ALS_ERR_INVALID_ARG;
    if (m > 0 && (!x || (n > 0 && (!colidx || !vals || !theta)))) return ALS_ERR_INVALID_ARG;
    if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(vals, 4) || !aligned(x, 4) ||
        !aligned(theta, 4) || !aligned(rmse_out, 8))
        return ALS_ERR_ALIGN;
    return ALS_OK;
}

// The RMSE's two kernels on `st`: partials over C = cus * kRmseWavesPerCU fixed chunks (at most
// cap_per_cu resident waves per CU if positive), then their fixed-order sum.  part holds C
// doubles; claim is the chunk counter (reset here by a kernel).
hipError_t rmse_launch(int cus, int cap_per_cu, bool force_global, hipStream_t st,
                       const int64_t* rowptr, const int32_t* colidx, const float* vals, int64_t m,
                       int64_t n, int f, const float* x, const float* theta, double* part,
                       unsigned* claim, double* rmse_out) {
    const int C = cus * kRmseWavesPerCU;
    if (m > 0) {
        const bool buf =
            !force_global && (uint64_t)n * (uint64_t)f * sizeof(float) <= kBufferGatherMax;
        hipError_t le = hipSuccess;
#define ALS_RMSE_ARGS cus, cap_per_cu, st, rowptr, colidx, vals, m, n, f, x, theta, part, claim, C
        switch (f / 16 + 1) {
#define ALS_RMSE_CASE(NB)                                                           \
            case NB:                                                                \
                le = buf ? rmse_rows_launch<NB, true>(ALS_RMSE_ARGS)                \
                         : rmse_rows_launch<NB, false>(ALS_RMSE_ARGS);              \
                break;
            ALS_RMSE_CASE(1) ALS_RMSE_CASE(2) ALS_RMSE_CASE(3) ALS_RMSE_CASE(4) ALS_RMSE_CASE(5)
            ALS_RMSE_CASE(6) ALS_RMSE_CASE(7) ALS_RMSE_CASE(8) ALS_RMSE_CASE(9)
#undef ALS_RMSE_CASE
#undef ALS_RMSE_ARGS
            default: return hipErrorInvalidValue;
        }
        if (le != hipSuccess) return le;
    }
    hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(kWave), 0, st, rowptr, m, m > 0 ? C : 0, part,
                       rmse_out);
    return hipGetLastError();
}

void profile_free(als_ctx* ctx) {
    if (!ctx->prof_ev) return;
    for (int i = 0; i < 4 * ctx->prof_cap; ++i) (void)hipEventDestroy(ctx->prof_ev[i]);
    delete[] ctx->prof_ev;
    ctx->prof_ev = nullptr;
    ctx->prof_cap = ctx->prof_count = 0;
}

}  // namespace

extern "C" {

size_t als_workspace_bytes(int device, int32_t f_max) {
    if (f_max < 1 || f_max > ALS_F_MAX) return 0;
    int cus = 0, w_cap = 0, waves[kMaxNB + 1] = {0};
    if (query_device(device, f_max, &cus, waves, &w_cap) != ALS_OK) return 0;
    return make_layout(waves, nb_of(f_max), cus).total;
}

int als_init(als_ctx** out, int device, void* workspace, size_t workspace_bytes, int32_t f_max) {
    if (!out) return ALS_ERR_INVALID_ARG;
    *out = nullptr;
    if (f_max < 1 || f_max > ALS_F_MAX) return ALS_ERR_UNSUPPORTED_F;
    if (!workspace) return ALS_ERR_WORKSPACE;
    if (!aligned(workspace, 256)) return ALS_ERR_ALIGN;
    als_ctx* ctx = new (std::nothrow) als_ctx();
    if (!ctx) return ALS_ERR_INVALID_ARG;
    int rc = query_device(device, f_max, &ctx->cus, ctx->waves, &ctx->w_cap,
                          &ctx->lds_per_block);
    if (rc != ALS_OK) { delete ctx; return rc; }
    ctx->device = device;
    ctx->f_max = f_max;
    {
        const char* g = getenv("ALS_GATHER");
        ctx->global_gather = g && strcmp(g, "global") == 0;
        ctx->staged_gather = g && strcmp(g, "lds") == 0;
        const char* t = getenv("ALS_LAST_BLOCK");
        ctx->tile_last_block = t && strcmp(t, "tiles") == 0;
        // part length in entries: kPart, or ALS_PART_ENTRIES rounded down to a power of two
        // times the entries of a pipeline group (at least one group)
        int64_t part = kPart;
        const char* pe = getenv("ALS_PART_ENTRIES");
        if (pe && atoll(pe) > 0) part = atoll(pe);
        int groups = 1;
        while ((int64_t)kEntriesPerGroup * groups * 2 <= part && groups < (1 << 24)) groups *= 2;
        ctx->part_groups = groups;
    }
    ctx->nb_max = nb_of(f_max);
    if (int su = noalloc_setup(device); su != ALS_OK) { delete ctx; return su; }
    if (ctx->staged_gather) {   // the staged form's residency bounds the partition's W
        DeviceGuard g2(device);
        for (int nb = 1; nb <= ctx->nb_max; ++nb) {
            int w = 0;
            if (staged_waves_for_nb(nb, ctx->cus, &w) != 0) { delete ctx; return ALS_ERR_HIP; }
            if (w < ctx->waves[nb]) ctx->waves[nb] = w;
        }
    }
    ctx->lay = make_layout(ctx->waves, ctx->nb_max, ctx->cus);
    if (workspace_bytes < ctx->lay.total) { delete ctx; return ALS_ERR_WORKSPACE; }
    ctx->ws = (unsigned char*)workspace;
    ctx->ws_bytes = workspace_bytes;
    DeviceGuard guard(device);
    hipLaunchKernelGGL(k_reset_counter, dim3(1), dim3(1), 0, nullptr,
                       (unsigned long long*)(ctx->ws + ctx->lay.status));
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) { delete ctx; return ALS_ERR_HIP; }
    *out = ctx;
    return ALS_OK;
}

int als_destroy(als_ctx* ctx) {
    if (ctx) {
        DeviceGuard guard(ctx->device);
        profile_free(ctx);
    }
    delete ctx;
    return ALS_OK;
}

int als_profile_begin(als_ctx* ctx, int32_t capacity) {
    if (!ctx || capacity < 1) return ALS_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    profile_free(ctx);
    ctx->prof_ev = new (std::nothrow) hipEvent_t[4 * (size_t)capacity];
    if (!ctx->prof_ev) return ALS_ERR_INVALID_ARG;
    for (int i = 0; i < 4 * capacity; ++i) {
        hipError_t e = hipEventCreate(&ctx->prof_ev[i]);
        if (e != hipSuccess) {
            for (int j = 0; j < i; ++j) (void)hipEventDestroy(ctx->prof_ev[j]);
            delete[] ctx->prof_ev;
            ctx->prof_ev = nullptr;
            return fail_hip(ctx, e);
        }
    }
    ctx->prof_cap = capacity;
    ctx->prof_count = 0;
    return ALS_OK;
}

int als_profile_end(als_ctx* ctx, float* ms_out, int32_t capacity, int32_t* count_out) {
    if (!ctx || !count_out || (capacity > 0 && !ms_out)) return ALS_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    *count_out = 0;
    if (!ctx->prof_ev) return ALS_OK;
    const int cnt = ctx->prof_count < capacity ? ctx->prof_count : capacity;
    int rc = ALS_OK;
    if (ctx->prof_count > 0) {
        hipError_t e = hipEventSynchronize(ctx->prof_ev[4 * (ctx->prof_count - 1) + 3]);
        if (e != hipSuccess) rc = fail_hip(ctx, e);
    }
    for (int i = 0; i < cnt && rc == ALS_OK; ++i)
        for (int k = 0; k < 3; ++k) {
            float ms = 0.f;
            hipError_t e = hipEventElapsedTime(&ms, ctx->prof_ev[4 * i + k], ctx->prof_ev[4 * i + k + 1]);
            if (e != hipSuccess) { rc = fail_hip(ctx, e); break; }
            ms_out[3 * i + k] = ms;
        }
    *count_out = cnt;
    profile_free(ctx);
    return rc;
}

int als_half_sweep(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                   int64_t m, int64_t n, int32_t f, float lambda, const float* theta_in,
                   float* x_out, void* stream) {
    if (!ctx) return ALS_ERR_INVALID_ARG;
    if (f < 1 || f > ctx->f_max) return ALS_ERR_UNSUPPORTED_F;
    if (m < 0 || n < 0 || !(lambda >= 0.f) || !std::isfinite(lambda)) return ALS_ERR_INVALID_ARG;
    if (m == 0) return ALS_OK;
    if (!rowptr || !x_out || (n > 0 && (!colidx || !vals || !theta_in))) return ALS_ERR_INVALID_ARG;
    if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(vals, 4) ||
        !aligned(theta_in, 4) || !aligned(x_out, 4))
        return ALS_ERR_ALIGN;
    if (theta_in && n > 0) {
        const char* t0 = (const char*)theta_in;
        const char* t1 = t0 + sizeof(float) * (size_t)n * (size_t)f;
        const char* x0 = (const char*)x_out;
        const char* x1 = x0 + sizeof(float) * (size_t)m * (size_t)f;
        if (t0 < x1 && x0 < t1) return ALS_ERR_ALIAS;
    }
    if (ctx->staged_gather && !staged_supported(n, f)) return ALS_ERR_UNSUPPORTED_F;
    const int nb = nb_of(f);
    const int W = ctx->waves[nb];
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    switch (nb) {
        case 1: launch_sweep<1>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 2: launch_sweep<2>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 3: launch_sweep<3>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 4: launch_sweep<4>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 5: launch_sweep<5>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 6: launch_sweep<6>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 7: launch_sweep<7>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 8: launch_sweep<8>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        case 9: launch_sweep<9>(ctx, rowptr, colidx, vals, m, n, f, lambda, theta_in, x_out, st, W); break;
        default: return ALS_ERR_UNSUPPORTED_F;
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_rmse(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
             int64_t m, int64_t n, int32_t f, const float* x, const float* theta,
             double* rmse_out, void* stream) {
    if (!ctx) return ALS_ERR_INVALID_ARG;
    const int rc = rmse_check(rowptr, colidx, vals, m, n, f, x, theta, rmse_out);
    if (rc != ALS_OK) return rc;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipError_t e = rmse_launch(ctx->cus, 4 * ctx->rmse_waves_per_simd, ctx->global_gather,
                               (hipStream_t)stream, rowptr, colidx, vals, m, n, f, x, theta,
                               (double*)(ctx->ws + ctx->lay.rmse),
                               (unsigned*)(ctx->ws + ctx->lay.status + 128), rmse_out);
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_rmse_noalloc(int device, const int64_t* rowptr, const int32_t* colidx,
                     const float* vals, int64_t m, int64_t n, int32_t f, const float* x,
                     const float* theta, double* rmse_out, void* stream) {
    const int rc = rmse_check(rowptr, colidx, vals, m, n, f, x, theta, rmse_out);
    if (rc != ALS_OK) return rc;
    const int su = noalloc_setup(device);
    if (su != ALS_OK) return su;
    const NoAllocDevice& d = g_noalloc[device];
    // the partials of the device's fixed chunk count must fit the fixed array
    if (kNoAllocPartials + sizeof(double) * (size_t)d.cus * kRmseWavesPerCU > kNoAllocScratchBytes)
        return ALS_ERR_WORKSPACE;
    DeviceGuard guard(device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipError_t e = rmse_launch(d.cus, 0, false, (hipStream_t)stream, rowptr, colidx, vals, m, n,
                               f, x, theta, (double*)(d.ptr + kNoAllocPartials),
                               (unsigned*)d.ptr, rmse_out);
    return e == hipSuccess ? ALS_OK : ALS_ERR_HIP;
}

int als_status(als_ctx* ctx, void* stream, int64_t* nonspd_rows) {
    if (!ctx || !nonspd_rows) return ALS_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    unsigned long long host = 0;
    auto* dev = (unsigned long long*)(ctx->ws + ctx->lay.status);
    hipError_t e = hipMemcpyAsync(&host, dev, sizeof host, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(ctx, e);
    hipLaunchKernelGGL(k_reset_counter, dim3(1), dim3(1), 0, st, dev);
    e = hipGetLastError();
    if (e != hipSuccess) return fail_hip(ctx, e);
    *nonspd_rows = (int64_t)host;
    return ALS_OK;
}

int als_plan(als_ctx* ctx, const int64_t* rowptr, int64_t m, int32_t f, int64_t* bounds_out,
             int64_t capacity, int64_t* params_out, void* stream) {
    if (!ctx || !rowptr || !bounds_out || !params_out || m < 0) return ALS_ERR_INVALID_ARG;
    if (f < 1 || f > ctx->f_max) return ALS_ERR_UNSUPPORTED_F;
    if (!aligned(rowptr, 8) || !aligned(bounds_out, 8)) return ALS_ERR_ALIGN;
    const int W = ctx->waves[nb_of(f)];
    const int C = chunks_of(W);
    params_out[0] = C;
    params_out[1] = kCostPerEntry;
    params_out[2] = row_cost(f);
    params_out[3] = kSnap;
    params_out[4] = W;
    params_out[5] = kTailDiv;
    if (capacity < C + 1) return ALS_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipLaunchKernelGGL(k_plan, dim3((C + 1 + 63) / 64), dim3(64), 0, (hipStream_t)stream, rowptr,
                       m, W, C, (int64_t)kCostPerEntry, row_cost(f), (int64_t)kSnap, bounds_out,
                       nullptr);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_csr_to_csc(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                   int64_t m, int64_t n, int64_t* colptr, int32_t* rowidx, float* vals_t,
                   void* stream) {
    if (!ctx || !rowptr || !colptr || m < 0 || n < 0 || m > INT32_MAX) return ALS_ERR_INVALID_ARG;
    if (m > 0 && n > 0 && (!colidx || !vals || !rowidx || !vals_t)) return ALS_ERR_INVALID_ARG;
    if (!aligned(rowptr, 8) || !aligned(colptr, 8) || !aligned(colidx, 4) || !aligned(vals, 4) ||
        !aligned(rowidx, 4) || !aligned(vals_t, 4))
        return ALS_ERR_ALIGN;
    // scratch: everything past the status block (no half-sweep runs meanwhile on this context)
    const size_t tiles = (size_t)(n + kScanTile - 1) / kScanTile;
    const size_t sums_bytes = align256(sizeof(int64_t) * (tiles + 1));
    const size_t avail = ctx->ws_bytes - ctx->lay.bounds;
    if (avail < sums_bytes + sizeof(int32_t) * (size_t)(n > 0 ? n : 1)) return ALS_ERR_WORKSPACE;
    int64_t R = n > 0 ? (int64_t)((avail - sums_bytes) / (sizeof(int32_t) * (size_t)n)) : 1;
    const int64_t r_cap = (int64_t)ctx->cus * kTransposeWavesPerCU;
    if (R > r_cap) R = r_cap;
    if (R > m) R = m;
    if (R < 1) R = 1;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    int64_t* sums = (int64_t*)(ctx->ws + ctx->lay.bounds);
    int32_t* cnt = (int32_t*)(ctx->ws + ctx->lay.bounds + sums_bytes);
    const int64_t cells = R * n;
    if (cells > 0) {
        const int64_t zb = (cells + 255) / 256;
        hipLaunchKernelGGL(k_tr_zero, dim3((unsigned)(zb < 65536 ? zb : 65536)), dim3(256), 0, st,
                           cnt, cells);
    }
    // LDS counters when one row block's fit in a workgroup's LDS
    const size_t lds_bytes = sizeof(int32_t) * (size_t)(n > 0 ? n : 1);
    bool lds = n <= kTrLdsCols && lds_bytes <= ctx->lds_per_block;
    if (lds && m > 0 && n > 0) {
        hipError_t ea = hipFuncSetAttribute((const void*)k_tr_count_lds,
                                            hipFuncAttributeMaxDynamicSharedMemorySize,
                                            (int)lds_bytes);
        if (ea == hipSuccess)
            ea = hipFuncSetAttribute((const void*)k_tr_scatter_lds,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
        if (ea != hipSuccess) return fail_hip(ctx, ea);
    }
    if (m > 0 && n > 0) {
        if (lds)
            hipLaunchKernelGGL(k_tr_count_lds, dim3((unsigned)R), dim3(256),
                               sizeof(int32_t) * (size_t)n, st, rowptr, colidx, m, (int)n, (int)R,
                               cnt);
        else
            hipLaunchKernelGGL(k_tr_count, dim3((unsigned)R), dim3(256), 0, st, rowptr, colidx,
                               m, n, (int)R, cnt);
    }
    if (n > 0)
        hipLaunchKernelGGL(k_tr_colscan, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, n,
                           (int)R, cnt, colptr);
    if (n > 0)
        hipLaunchKernelGGL(k_scan_sums, dim3((unsigned)tiles), dim3(256), 0, st, colptr, n, sums);
    hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(256), 0, st, sums, (int64_t)tiles, colptr, n);
    if (n > 0)
        hipLaunchKernelGGL(k_scan_apply, dim3((unsigned)tiles), dim3(256), 0, st, colptr, n, sums);
    if (m > 0 && n > 0) {
        if (lds)
            hipLaunchKernelGGL(k_tr_scatter_lds, dim3((unsigned)R), dim3(kWave),
                               sizeof(int32_t) * (size_t)n, st, rowptr, colidx, vals, m, (int)n,
                               (int)R, cnt, colptr, rowidx, vals_t);
        else
            hipLaunchKernelGGL(k_tr_scatter, dim3((unsigned)R), dim3(kWave), 0, st, rowptr,
                               colidx, vals, m, n, (int)R, cnt, colptr, rowidx, vals_t);
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_gather_dump(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx,
                    const float* vals, int64_t m, int64_t n, int32_t f, const float* theta,
                    int64_t u, float* out, int64_t capacity, void* stream) {
    if (!ctx) return ALS_ERR_INVALID_ARG;
    if (f < 1 || f > ctx->f_max) return ALS_ERR_UNSUPPORTED_F;
    if (m < 1 || n < 0 || u < 0 || u >= m || capacity < 0 || !rowptr || !out)
        return ALS_ERR_INVALID_ARG;
    if (n > 0 && (!colidx || !vals || !theta)) return ALS_ERR_INVALID_ARG;
    if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(vals, 4) || !aligned(theta, 4) ||
        !aligned(out, 4))
        return ALS_ERR_ALIGN;
    if (ctx->staged_gather && !staged_supported(n, f)) return ALS_ERR_UNSUPPORTED_F;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    const int nb = nb_of(f);
    const int64_t limit = capacity / (16 * (nb + 3));
    switch (nb) {
#define ALS_DUMP_CASE(NB)                                                                     \
        case NB:                                                                              \
            launch_dump<NB>(ctx, rowptr, colidx, vals, n, f, theta, u, out, limit, st);       \
            break;
        ALS_DUMP_CASE(1) ALS_DUMP_CASE(2) ALS_DUMP_CASE(3) ALS_DUMP_CASE(4) ALS_DUMP_CASE(5)
        ALS_DUMP_CASE(6) ALS_DUMP_CASE(7) ALS_DUMP_CASE(8) ALS_DUMP_CASE(9)
#undef ALS_DUMP_CASE
        default: return ALS_ERR_UNSUPPORTED_F;
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_rmse_waves(als_ctx* ctx, int32_t waves_per_simd) {
    if (!ctx || waves_per_simd < 0 || waves_per_simd > kRmseWavesPerCU / 4)
        return ALS_ERR_INVALID_ARG;
    ctx->rmse_waves_per_simd = waves_per_simd;
    return ALS_OK;
}

int als_last_hip_error(const als_ctx* ctx) { return ctx ? ctx->last_hip : 0; }

const char* als_strerror(int status) {
    switch (status) {
        case ALS_OK: return "ok";
        case ALS_ERR_INVALID_ARG: return "invalid argument";
        case ALS_ERR_UNSUPPORTED_F: return "f outside the supported range";
        case ALS_ERR_WORKSPACE: return "workspace missing or too small";
        case ALS_ERR_ALIGN: return "pointer not naturally aligned";
        case ALS_ERR_HIP: return "HIP runtime error";
        case ALS_ERR_ALIAS: return "theta_in and x_out overlap";
        case ALS_ERR_DEVICE: return "invalid or unsupported device";
        default: return "unknown status";
    }
}

}  // extern "C"
