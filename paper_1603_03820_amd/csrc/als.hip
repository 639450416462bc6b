// One ALS half-sweep on gfx950 (MI355X): C ABI of include/als.h plus its kernels.
//
// Per row u of a CSR matrix (eq. 2 of the paper; Algorithm 1's Get_Hermitian_X then
// Batch_Solve):  A_u = sum theta_v theta_v^T + lambda n_u I,  b_u = sum r_uv theta_v,
// x_u = A_u^{-1} b_u.
//
// Design (one wave = one worker):
//   k_plan          integer partition of rows (and of long rows' entries) into W equal shares
//                   of a cost axis (see als_plan in als.h); no host synchronisation needed.
//   k_herm_solve    per wave: walk its share row by row; gather theta_v for four entries at a
//                   time straight into MFMA operand registers (lane = 16*k + column, so each
//                   group of 16 lanes reads 64 contiguous bytes of one theta_v), accumulate the
//                   lower block-triangle of the Gram matrix with v_mfma_f32_16x16x4_f32 and b_u
//                   with VALU FMAs; rows that end in the share are regularised, factored
//                   (Cholesky, folded forward substitution) and back-substituted in registers,
//                   with a 16*NB-float LDS column buffer as the only broadcast medium.
//   k_reduce_solve  rows cut by share boundaries: sum the per-wave partial accumulators in
//                   wave order (fixed, so results are reproducible), then the same solve.
//   k_rmse_*        residuals per stored entry, fp64 partial sums in a fixed order.
//
// Register layout of the accumulators (the 16x16 MFMA C/D layout): tile (I,J), J <= I, lane l,
// element r holds A[16 I + 4 (l >> 4) + r][16 J + (l & 15)].  The b accumulator of lane l holds
// partial sums of b[16 J + (l & 15)] over the entries its 16-lane group saw.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <new>

#include "als.h"

typedef float f4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kWave = 64;
constexpr int kMaxNB = (ALS_F_MAX + 15) / 16;   // 8 column blocks of 16
constexpr int kSnap = 256;                      // partition cut grid (entries)
constexpr int kCostPerEntry = 16;               // c_nnz
constexpr int kMaxWavesPerCU = 32;

constexpr int ntiles(int nb) { return nb * (nb + 1) / 2; }
constexpr int tix(int I, int J) { return I * (I + 1) / 2 + J; }   // J <= I
// floats per partial-accumulator slot: tiles (4 per lane) + b (1 per block per lane)
constexpr int slot_floats(int nb) { return (ntiles(nb) * 4 + nb) * kWave; }
constexpr int lds_floats(int nb) { return 2 * (16 * nb + 4); }

__device__ __forceinline__ float readlane_f(float v, int lane) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

__device__ __forceinline__ float pick4(const f4 v, int r) {
    return r == 0 ? v[0] : (r == 1 ? v[1] : (r == 2 ? v[2] : v[3]));
}

// ------------------------------------------------------------------------------- plan ----

// Cost prefix P(u) = c_nnz rowptr[u] + c_row u; boundary b at s_b = floor(T b / W).
__global__ void k_plan(const int64_t* __restrict__ rowptr, int64_t m, int W, int64_t c_nnz,
                       int64_t c_row, int64_t q, int64_t* __restrict__ bounds) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b > W) return;
    const int64_t T = c_nnz * rowptr[m] + c_row * m;
    const int64_t Q = T / W, R = T % W;
    const int64_t s = Q * b + (R * b) / W;   // == floor(T b / W) without 128-bit products
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

// theta values of one 4-entry step, as MFMA operands: lane (g, c) holds theta_{v_g}[16 I + c]
template <int NB>
__device__ __forceinline__ void load_step(const float* __restrict__ theta, int f, int col,
                                          bool ok, int c, float (&v)[NB]) {
    const float* tp = theta + (size_t)(unsigned)col * (size_t)f;
#pragma unroll
    for (int I = 0; I < NB; ++I) {
        const int j = 16 * I + c;
        float t = 0.f;
        if (ok && (I < NB - 1 || j < f)) t = tp[j];
        v[I] = t;
    }
}

// Accumulate entries [kbeg, kend) of one row into acc (lower block-triangle Gram) and bacc.
template <int NB>
__device__ __forceinline__ void gram_accumulate(const int32_t* __restrict__ colidx,
                                                const float* __restrict__ vals,
                                                const float* __restrict__ theta, int f,
                                                int64_t kbeg, int64_t kend,
                                                f4 (&acc)[ntiles(NB)], float (&bacc)[NB],
                                                int lane) {
    if (kbeg >= kend) return;
    const int g = lane >> 4, c = lane & 15;
    // 64 entries (16 steps) of indices per batch, one per lane; next batch prefetched
    int64_t base = kbeg;
    int col_b = 0;
    float rv_b = 0.f;
    if (base + lane < kend) { col_b = colidx[base + lane]; rv_b = vals[base + lane]; }
    int cnt = (int)((kend - base) < 64 ? (kend - base) : 64);
    float vn[NB];
    float rn;
    {
        const int cs = __shfl(col_b, g);
        rn = __shfl(rv_b, g);
        const bool ok = g < cnt;
        if (!ok) rn = 0.f;
        load_step<NB>(theta, f, cs, ok, c, vn);
    }
    while (true) {
        const int64_t nbase = base + 64;
        int col_n = 0;
        float rv_n = 0.f;
        if (nbase + lane < kend) { col_n = colidx[nbase + lane]; rv_n = vals[nbase + lane]; }
        const int ncnt = nbase < kend ? (int)((kend - nbase) < 64 ? (kend - nbase) : 64) : 0;
        const int nsteps = (cnt + 3) >> 2;
        for (int s = 0; s < nsteps; ++s) {
            float v[NB];
#pragma unroll
            for (int I = 0; I < NB; ++I) v[I] = vn[I];
            const float r = rn;
            // issue the next step's gathers before this step's matrix ops
            if (s + 1 < nsteps) {
                const int src = 4 * (s + 1) + g;
                const int cs = __shfl(col_b, src);
                rn = __shfl(rv_b, src);
                const bool ok = src < cnt;
                if (!ok) rn = 0.f;
                load_step<NB>(theta, f, cs, ok, c, vn);
            } else if (ncnt > 0) {
                const int cs = __shfl(col_n, g);
                rn = __shfl(rv_n, g);
                const bool ok = g < ncnt;
                if (!ok) rn = 0.f;
                load_step<NB>(theta, f, cs, ok, c, vn);
            }
#pragma unroll
            for (int I = 0; I < NB; ++I) bacc[I] += r * v[I];
#pragma unroll
            for (int I = 0; I < NB; ++I)
#pragma unroll
                for (int J = 0; J <= I; ++J)
                    acc[tix(I, J)] =
                        __builtin_amdgcn_mfma_f32_16x16x4f32(v[I], v[J], acc[tix(I, J)], 0, 0, 0);
        }
        if (ncnt == 0) break;
        base = nbase;
        col_b = col_n;
        rv_b = rv_n;
        cnt = ncnt;
    }
}

// ------------------------------------------------------------------ solve in registers ---

// Regularise, factor A = L L^T in place (right-looking, one column per step), fold the forward
// substitution L y = b into the factorisation, back-substitute L^T x = y, write x_u.
// buf: this wave's LDS, lds_floats(NB) floats.
template <int NB>
__device__ __forceinline__ void solve_row(f4 (&acc)[ntiles(NB)], float (&bacc)[NB], int f,
                                          float lam_n, float* buf, float* __restrict__ xrow,
                                          unsigned long long* __restrict__ nonspd, int lane) {
    const int g = lane >> 4, c = lane & 15;
    constexpr int BS = 16 * NB + 4;
    constexpr int PIV = 16 * NB;
    float bcol[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) {   // sum b over the four 16-lane groups
        float t = bacc[I];
        t += __shfl_xor(t, 16);
        t += __shfl_xor(t, 32);
        bcol[I] = t;
    }
#pragma unroll
    for (int I = 0; I < NB; ++I)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            if (c == 4 * g + r && 16 * I + c < f) acc[tix(I, I)][r] += lam_n;

    bool ok = true;
#pragma unroll
    for (int K = 0; K < NB; ++K) {
        const int kn = (f - 16 * K) < 16 ? (f - 16 * K) : 16;
        for (int kc = 0; kc < kn; ++kc) {
            const int k = 16 * K + kc;
            float* b = buf + (k & 1) * BS;
            if (c == kc) {   // the four lanes holding column k publish it (rows <= k as 0)
#pragma unroll
                for (int I = K; I < NB; ++I) {
                    const f4 v = acc[tix(I, K)];
                    const int i0 = 16 * I + 4 * g;
                    f4 w;
#pragma unroll
                    for (int r = 0; r < 4; ++r) w[r] = (i0 + r > k) ? v[r] : 0.f;
                    *reinterpret_cast<f4*>(b + i0) = w;
                    if (I == K) {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (i0 + r == k) b[PIV] = v[r];
                    }
                }
            }
            __syncthreads();
            const float d = b[PIV];
            ok = ok && (d > 0.f);
            const float s = 1.0f / sqrtf(d);
            const float yk = readlane_f(bcol[K], kc) * s;
            f4 colv[NB];
            float colj[NB];
#pragma unroll
            for (int I = K; I < NB; ++I) {
                colv[I] = *reinterpret_cast<const f4*>(b + 16 * I + 4 * g) * s;
                colj[I] = b[16 * I + c] * s;
            }
#pragma unroll
            for (int I = K; I < NB; ++I)
#pragma unroll
                for (int J = K; J <= I; ++J) acc[tix(I, J)] -= colv[I] * colj[J];
#pragma unroll
            for (int J = K; J < NB; ++J) bcol[J] -= colj[J] * yk;
            if (c == kc) {
#pragma unroll
                for (int I = K; I < NB; ++I) {
                    const int i0 = 16 * I + 4 * g;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        if (i0 + r > k) acc[tix(I, K)][r] = colv[I][r];
                        else if (i0 + r == k) acc[tix(I, K)][r] = d * s;
                    }
                }
                bcol[K] = yk;
            }
        }
    }
    // back substitution L^T x = y, y held in bcol (column layout)
    float xcol[NB];
#pragma unroll
    for (int J = 0; J < NB; ++J) xcol[J] = 0.f;
#pragma unroll
    for (int J = NB - 1; J >= 0; --J) {
        const int jn = (f - 16 * J) < 16 ? (f - 16 * J) : 16;
        for (int jc = jn - 1; jc >= 0; --jc) {
            const int j = 16 * J + jc;
            float* b = buf + (j & 1) * BS;
            if (g == (jc >> 2)) {   // row j of L: lanes of group jc/4, element jc%4
#pragma unroll
                for (int I = 0; I <= J; ++I) {
                    const int i = 16 * I + c;
                    const float v = pick4(acc[tix(J, I)], jc & 3);
                    b[i] = (i <= j) ? v : 0.f;
                }
            }
            __syncthreads();
            const float xj = readlane_f(bcol[J], jc) / b[j];
#pragma unroll
            for (int I = 0; I <= J; ++I) {
                const float lji = b[16 * I + c];
                if (16 * I + c < j) bcol[I] -= lji * xj;
            }
            if (c == jc) xcol[J] = xj;
        }
    }
    if (g == 0) {
#pragma unroll
        for (int J = 0; J < NB; ++J)
            if (16 * J + c < f) xrow[16 * J + c] = ok ? xcol[J] : __builtin_nanf("");
    }
    if (!ok && lane == 0) atomicAdd(nonspd, 1ull);
}

template <int NB>
__device__ __forceinline__ void write_zero_row(float* __restrict__ xrow, int f, int lane) {
    for (int j = lane; j < f; j += kWave) xrow[j] = 0.f;
}

template <int NB>
__device__ __forceinline__ void store_slot(const f4 (&acc)[ntiles(NB)], const float (&bacc)[NB],
                                           float* __restrict__ slot, int lane) {
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) slot[(t * 4 + r) * kWave + lane] = acc[t][r];
#pragma unroll
    for (int I = 0; I < NB; ++I) slot[(ntiles(NB) * 4 + I) * kWave + lane] = bacc[I];
}

template <int NB>
__device__ __forceinline__ void add_slot(f4 (&acc)[ntiles(NB)], float (&bacc)[NB],
                                         const float* __restrict__ slot, int lane) {
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[t][r] += slot[(t * 4 + r) * kWave + lane];
#pragma unroll
    for (int I = 0; I < NB; ++I) bacc[I] += slot[(ntiles(NB) * 4 + I) * kWave + lane];
}

// ------------------------------------------------------------------------ kernels --------

// Wave w: entries from bounds[w] to bounds[w+1].  Whole rows are solved here; the piece of a
// row cut at the start of the share goes to slot 2w, the piece cut at its end to slot 2w+1.
template <int NB>
__global__ __launch_bounds__(kWave) void k_herm_solve(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, const float* __restrict__ theta, int64_t m, int f,
    float lambda, const int64_t* __restrict__ bounds, float* __restrict__ x_out,
    float* __restrict__ slots, unsigned long long* __restrict__ nonspd) {
    __shared__ __attribute__((aligned(16))) float buf[lds_floats(NB)];
    const int lane = threadIdx.x;
    const int w = blockIdx.x;
    const int64_t u0 = bounds[2 * w], k0 = bounds[2 * w + 1];
    const int64_t u1 = bounds[2 * w + 2], k1 = bounds[2 * w + 3];
    for (int64_t u = u0; u <= u1 && u < m; ++u) {
        const int64_t rs = rowptr[u], nu = rowptr[u + 1] - rs;
        const int64_t ka = (u == u0) ? k0 : 0;
        int64_t kb = nu;
        if (u == u1) {
            if (k1 == 0) break;
            kb = k1;
        }
        if (nu == 0) {                       // empty row: x_u = 0
            write_zero_row<NB>(x_out + (size_t)u * f, f, lane);
            continue;
        }
        if (ka >= kb) continue;              // nothing of this row in the share
        f4 acc[ntiles(NB)];
        float bacc[NB];
#pragma unroll
        for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int I = 0; I < NB; ++I) bacc[I] = 0.f;
        gram_accumulate<NB>(colidx, vals, theta, f, rs + ka, rs + kb, acc, bacc, lane);
        if (ka == 0 && kb == nu) {
            const float lam_n = (float)((double)lambda * (double)nu);
            solve_row<NB>(acc, bacc, f, lam_n, buf, x_out + (size_t)u * f, nonspd, lane);
        } else {
            const int which = (u == u0) ? 0 : 1;
            store_slot<NB>(acc, bacc, slots + (size_t)(2 * w + which) * slot_floats(NB), lane);
        }
    }
}

// One wave per internal boundary b (1..W-1); the first boundary that cuts a row sums that
// row's pieces -- wave b-1's, then b, b+1, ... -- and solves it.
template <int NB>
__global__ __launch_bounds__(kWave) void k_reduce_solve(
    const int64_t* __restrict__ rowptr, int64_t m, int W, int f, float lambda,
    const int64_t* __restrict__ bounds, float* __restrict__ x_out,
    const float* __restrict__ slots, unsigned long long* __restrict__ nonspd) {
    __shared__ __attribute__((aligned(16))) float buf[lds_floats(NB)];
    const int lane = threadIdx.x;
    const int b = blockIdx.x + 1;
    if (b >= W) return;
    auto cuts = [&](int bb) -> bool {   // boundary bb lies strictly inside its row
        const int64_t u = bounds[2 * bb], k = bounds[2 * bb + 1];
        return u < m && k > 0 && k < rowptr[u + 1] - rowptr[u];
    };
    if (!cuts(b)) return;
    const int64_t u = bounds[2 * b];
    if (b > 1 && cuts(b - 1) && bounds[2 * (b - 1)] == u) return;   // not the first cut
    f4 acc[ntiles(NB)];
    float bacc[NB];
#pragma unroll
    for (int t = 0; t < ntiles(NB); ++t) acc[t] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int I = 0; I < NB; ++I) bacc[I] = 0.f;
    // wave b-1 holds the row's first piece: as its first piece if it started in row u
    // (then at entry 0), else as its last piece
    const int first_slot = (bounds[2 * (b - 1)] == u) ? 2 * (b - 1) : 2 * (b - 1) + 1;
    add_slot<NB>(acc, bacc, slots + (size_t)first_slot * slot_floats(NB), lane);
    const int64_t nu = rowptr[u + 1] - rowptr[u];
    for (int bb = b;; ++bb) {   // waves b, b+1, ... start inside row u: their first piece
        const bool more = bb + 1 < W && cuts(bb + 1) && bounds[2 * (bb + 1)] == u;
        // several boundaries can snap to one cut point; the waves between them hold an empty
        // piece of row u and wrote no slot
        const int64_t piece_end = more ? bounds[2 * (bb + 1) + 1] : nu;
        if (bounds[2 * bb + 1] < piece_end)
            add_slot<NB>(acc, bacc, slots + (size_t)(2 * bb) * slot_floats(NB), lane);
        if (!more) break;
    }
    const float lam_n = (float)((double)lambda * (double)nu);
    solve_row<NB>(acc, bacc, f, lam_n, buf, x_out + (size_t)u * f, nonspd, lane);
}

// RMSE: wave w covers entries [nnz w / W, nnz (w+1) / W); each 16-lane group takes one entry
// per step.  Partial sums in fp64, one per wave.
__global__ __launch_bounds__(kWave) void k_rmse_partial(
    const int64_t* __restrict__ rowptr, const int32_t* __restrict__ colidx,
    const float* __restrict__ vals, int64_t m, int f, const float* __restrict__ x,
    const float* __restrict__ theta, int W, double* __restrict__ partial) {
    const int lane = threadIdx.x, g = lane >> 4, c = lane & 15;
    const int w = blockIdx.x;
    const int64_t nnz = rowptr[m];
    const int64_t kb = nnz / W * w + (nnz % W) * w / W;
    const int64_t ke = nnz / W * (w + 1) + (nnz % W) * (w + 1) / W;
    double acc = 0.0;
    if (kb < ke) {
        int64_t lo = 0, hi = m - 1;   // row of entry kb: largest u < m with rowptr[u] <= kb
        while (lo < hi) {
            const int64_t mid = (lo + hi + 1) >> 1;
            if (rowptr[mid] <= kb) lo = mid; else hi = mid - 1;
        }
        int64_t u = lo;
        for (int64_t k = kb + g; k - g < ke; k += 4) {
            const bool ok = k < ke;
            float part = 0.f;
            float r = 0.f;
            if (ok) {
                while (rowptr[u + 1] <= k) ++u;
                const float* tp = theta + (size_t)(unsigned)colidx[k] * f;
                const float* xp = x + (size_t)u * f;
                for (int j = c; j < f; j += 16) part += tp[j] * xp[j];
                r = vals[k];
            }
            part += __shfl_xor(part, 8);
            part += __shfl_xor(part, 4);
            part += __shfl_xor(part, 2);
            part += __shfl_xor(part, 1);
            if (ok && c == 0) {
                const double e = (double)(r - part);
                acc += e * e;
            }
        }
    }
    acc += __shfl_xor(acc, 16);
    acc += __shfl_xor(acc, 32);
    if (lane == 0) partial[w] = acc;
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

// --------------------------------------------------------------------- host side ---------

struct Layout {
    size_t status, bounds, rmse, slots, total;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// waves[nb] = W for f in (16 (nb-1), 16 nb]; the slot region holds 2 W partial accumulators
Layout make_layout(const int* waves, int nb_max) {
    int w_cap = 1;
    size_t slot_bytes = 0;
    for (int nb = 1; nb <= nb_max; ++nb) {
        if (waves[nb] > w_cap) w_cap = waves[nb];
        const size_t sb = sizeof(float) * (size_t)slot_floats(nb) * 2 * (size_t)waves[nb];
        if (sb > slot_bytes) slot_bytes = sb;
    }
    Layout L;
    size_t off = 0;
    L.status = off; off = align256(off + 256);
    L.bounds = off; off = align256(off + sizeof(int64_t) * 2 * (size_t)(w_cap + 1));
    L.rmse = off;   off = align256(off + sizeof(double) * (size_t)w_cap);
    L.slots = off;  off = align256(off + slot_bytes);
    L.total = off;
    return L;
}

template <int NB>
int occupancy_waves(int cus, int* waves) {
    int blocks = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_herm_solve<NB>, kWave, 0);
    if (e != hipSuccess) return -1;
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxWavesPerCU) blocks = kMaxWavesPerCU;
    const char* env = getenv("ALS_WAVES_PER_CU");
    if (env && atoi(env) > 0) blocks = atoi(env) < blocks ? atoi(env) : blocks;
    *waves = blocks * cus;
    return 0;
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
        default: return -1;
    }
}

int nb_of(int f) { return (f + 15) / 16; }

// Solve cost of one row in c_nnz units: the Cholesky runs on the vector ALU while other waves
// keep the matrix cores busy, so it is charged at a fraction of its latency.  Tunable through
// ALS_ROW_COST (entries per row).
int64_t row_cost(int f) {
    const char* env = getenv("ALS_ROW_COST");
    if (env && atoll(env) > 0) return atoll(env) * kCostPerEntry;
    const int nb = nb_of(f);
    const double mfma_cycles_per_entry = 8.0 * ntiles(nb);
    const double chol_cycles = 16.0 * 4.0 * 4.0 * [&] {
        double t = 0;
        for (int K = 0; K < nb; ++K) t += (nb - K) * (nb - K + 1) / 2.0;
        return t;
    }() + 60.0 * f;
    double entries = 0.5 * chol_cycles / mfma_cycles_per_entry;
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

int query_device(int device, int f_max, int* cus, int* waves, int* w_cap) {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || device < 0 || device >= n) return ALS_ERR_DEVICE;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) != hipSuccess) return ALS_ERR_DEVICE;
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) return ALS_ERR_DEVICE;
    *cus = prop.multiProcessorCount;
    DeviceGuard guard(device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    *w_cap = 1;
    for (int nb = 1; nb <= nb_of(f_max); ++nb) {
        if (waves_for_nb(nb, *cus, &waves[nb]) != 0) return ALS_ERR_HIP;
        if (waves[nb] > *w_cap) *w_cap = waves[nb];
    }
    return ALS_OK;
}

template <int NB>
void launch_sweep(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                  int64_t m, int f, float lambda, const float* theta, float* x, hipStream_t st,
                  int W) {
    int64_t* bounds = (int64_t*)(ctx->ws + ctx->lay.bounds);
    float* slots = (float*)(ctx->ws + ctx->lay.slots);
    auto* nonspd = (unsigned long long*)(ctx->ws + ctx->lay.status);
    hipEvent_t* ev = nullptr;
    if (ctx->prof_ev && ctx->prof_count < ctx->prof_cap) ev = ctx->prof_ev + 4 * ctx->prof_count++;
    if (ev) (void)hipEventRecord(ev[0], st);
    hipLaunchKernelGGL(k_plan, dim3((W + 1 + 63) / 64), dim3(64), 0, st, rowptr, m, W,
                       (int64_t)kCostPerEntry, row_cost(f), (int64_t)kSnap, bounds);
    if (ev) (void)hipEventRecord(ev[1], st);
    hipLaunchKernelGGL(k_herm_solve<NB>, dim3(W), dim3(kWave), 0, st, rowptr, colidx, vals,
                       theta, m, f, lambda, bounds, x, slots, nonspd);
    if (ev) (void)hipEventRecord(ev[2], st);
    if (W > 1)
        hipLaunchKernelGGL(k_reduce_solve<NB>, dim3(W - 1), dim3(kWave), 0, st, rowptr, m, W, f,
                           lambda, bounds, x, slots, nonspd);
    if (ev) (void)hipEventRecord(ev[3], st);
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
    return make_layout(waves, nb_of(f_max)).total;
}

int als_init(als_ctx** out, int device, void* workspace, size_t workspace_bytes, int32_t f_max) {
    if (!out) return ALS_ERR_INVALID_ARG;
    *out = nullptr;
    if (f_max < 1 || f_max > ALS_F_MAX) return ALS_ERR_UNSUPPORTED_F;
    if (!workspace) return ALS_ERR_WORKSPACE;
    if (!aligned(workspace, 256)) return ALS_ERR_ALIGN;
    als_ctx* ctx = new (std::nothrow) als_ctx();
    if (!ctx) return ALS_ERR_INVALID_ARG;
    int rc = query_device(device, f_max, &ctx->cus, ctx->waves, &ctx->w_cap);
    if (rc != ALS_OK) { delete ctx; return rc; }
    ctx->device = device;
    ctx->f_max = f_max;
    ctx->nb_max = nb_of(f_max);
    ctx->lay = make_layout(ctx->waves, ctx->nb_max);
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
    const int nb = nb_of(f);
    const int W = ctx->waves[nb];
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    switch (nb) {
        case 1: launch_sweep<1>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 2: launch_sweep<2>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 3: launch_sweep<3>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 4: launch_sweep<4>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 5: launch_sweep<5>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 6: launch_sweep<6>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 7: launch_sweep<7>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        case 8: launch_sweep<8>(ctx, rowptr, colidx, vals, m, f, lambda, theta_in, x_out, st, W); break;
        default: return ALS_ERR_UNSUPPORTED_F;
    }
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
}

int als_rmse(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
             int64_t m, int64_t n, int32_t f, const float* x, const float* theta,
             double* rmse_out, void* stream) {
    if (!ctx) return ALS_ERR_INVALID_ARG;
    if (f < 1 || f > ALS_F_MAX) return ALS_ERR_UNSUPPORTED_F;
    if (m < 0 || n < 0 || !rowptr || !rmse_out) return ALS_ERR_INVALID_ARG;
    if (m > 0 && (!x || (n > 0 && (!colidx || !vals || !theta)))) return ALS_ERR_INVALID_ARG;
    if (!aligned(rowptr, 8) || !aligned(colidx, 4) || !aligned(vals, 4) || !aligned(x, 4) ||
        !aligned(theta, 4) || !aligned(rmse_out, 8))
        return ALS_ERR_ALIGN;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipStream_t st = (hipStream_t)stream;
    const int W = ctx->w_cap;
    double* part = (double*)(ctx->ws + ctx->lay.rmse);
    if (m > 0)
        hipLaunchKernelGGL(k_rmse_partial, dim3(W), dim3(kWave), 0, st, rowptr, colidx, vals, m,
                           f, x, theta, W, part);
    hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(kWave), 0, st, rowptr, m, m > 0 ? W : 0, part,
                       rmse_out);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
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
    params_out[0] = W;
    params_out[1] = kCostPerEntry;
    params_out[2] = row_cost(f);
    params_out[3] = kSnap;
    if (capacity < W + 1) return ALS_ERR_INVALID_ARG;
    DeviceGuard guard(ctx->device);
    if (!guard.ok) return ALS_ERR_DEVICE;
    hipLaunchKernelGGL(k_plan, dim3((W + 1 + 63) / 64), dim3(64), 0, (hipStream_t)stream, rowptr,
                       m, W, (int64_t)kCostPerEntry, row_cost(f), (int64_t)kSnap, bounds_out);
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? ALS_OK : fail_hip(ctx, e);
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
