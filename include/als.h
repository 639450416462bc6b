/*
 * als.h -- one ALS half-sweep on an AMD Instinct MI355X (gfx950).
 *
 * The operation is the update-X step of alternating least squares for the weighted-lambda
 * cost function (eq. 1) of Tan, Cao and Fong, "Faster and Cheaper: Parallelizing Large-Scale
 * Matrix Factorization on GPUs" (HPDC'16): for every row u of the sparse m x n rating matrix R,
 *
 *     A_u = sum over stored (u,v) of (theta_v theta_v^T + lambda I)  =  G_u + lambda n_u I
 *     b_u = Theta^T R_u*^T  =  sum over stored (u,v) of r_uv theta_v
 *     x_u = A_u^{-1} b_u                                         (eq. 2, Algorithm 1)
 *
 * The update-Theta step (eq. 3) is the same call on the transposed matrix (CSC of R) with the
 * roles of X and Theta exchanged.
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers on the context's device, owned by the caller.
 *     The library never allocates or frees device memory; its only scratch is the workspace
 *     handed to als_init.
 *   - Sparse matrices are CSR: rowptr int64[m+1] (rowptr[0] = 0, non-decreasing, rowptr[m] =
 *     nnz), colidx int32[nnz] (0 <= colidx < n, no repeated column within a row), vals
 *     fp32[nnz].  Every stored entry counts as a rating, whatever its value.
 *   - Factor matrices are dense row-major fp32: Theta is n x f (theta_v contiguous, i.e. the
 *     bytes of the paper's f x n Theta^T stored column-major), X is m x f.
 *   - Pointers must be naturally aligned (8 bytes for int64, 4 bytes for int32/fp32), else
 *     ALS_ERR_ALIGN.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Argument checks happen before the
 *     call returns; all device work is queued on `stream` without a host synchronisation, so
 *     inputs must stay valid until the stream has passed the call.
 *   - Index ranges are not validated on the device; out-of-range colidx is undefined.
 *   - No C++ exception crosses this interface.  Status codes are below; after ALS_ERR_HIP the
 *     HIP error code is available from als_last_hip_error.
 *   - A context serves one device and must not be used from two host threads at once; calls
 *     queued on different streams of one context must not overlap in time (they share the
 *     workspace).
 */
#ifndef ALS_H
#define ALS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ALS_OK = 0,
    ALS_ERR_INVALID_ARG = -1,   /* null pointer, negative size, lambda < 0 or not finite   */
    ALS_ERR_UNSUPPORTED_F = -2, /* f outside [1, ALS_F_MAX]                                 */
    ALS_ERR_WORKSPACE = -3,     /* workspace missing or smaller than als_workspace_bytes    */
    ALS_ERR_ALIGN = -4,         /* a pointer is not naturally aligned                        */
    ALS_ERR_HIP = -5,           /* a HIP runtime call failed (see als_last_hip_error)        */
    ALS_ERR_ALIAS = -6,         /* theta_in and x_out overlap                                */
    ALS_ERR_DEVICE = -7         /* device index invalid or not a gfx950 device               */
};

#define ALS_F_MAX 128

typedef struct als_ctx als_ctx;

/* Bytes of device workspace a context on `device` needs for every f <= f_max.  Returns 0 if
   the device cannot be queried or f_max is outside [1, ALS_F_MAX].  The size depends on the
   device's compute-unit count and f_max only (not on m, n or nnz); it is dominated by two
   partial-accumulator slots per work chunk (about 1.4 GB on a 256-CU MI355X at f_max = 128). */
size_t als_workspace_bytes(int device, int32_t f_max);

/* Create a context on `device` using the caller's device workspace (at least
   als_workspace_bytes(device, f_max) bytes, 256-byte aligned; owned by the caller, who keeps
   it alive until als_destroy).  f_max bounds the f of later calls.
   Two environment variables, read here, select design alternatives of the same computation
   (for tests and ablation; results agree within the parity tolerance):
     ALS_GATHER=global      gather theta/x with 64-bit global loads at every size (otherwise
                            bounded buffer loads whenever the factor is below 2 GiB);
     ALS_LAST_BLOCK=tiles   accumulate the last block column with 16x16x4 tiles even when its
                            quad form applies (f = 0 or 4 mod 16).
   A third sets the part length of long pieces (tests; the default is 65,536 entries):
     ALS_PART_ENTRIES=k     a row piece longer than k entries (rounded down to 16 times a power
                            of two) is accumulated in parts of that length, whose sums are added
                            in order in a per-wave slot of the workspace (a two-level sum: no
                            fp32 running sum spans more than one part). */
int als_init(als_ctx** ctx, int device, void* workspace, size_t workspace_bytes, int32_t f_max);

/* Release the context (not the workspace).  Does not synchronise. */
int als_destroy(als_ctx* ctx);

/*
 * One half-sweep (eq. 2; Algorithm 1, Get_Hermitian_X then Batch_Solve):
 *   x_out[u] = (sum_v theta_v theta_v^T + lambda n_u I)^{-1} sum_v r_uv theta_v
 * for every row u in [0, m), v over the stored columns of row u, theta_v = theta_in[v].
 *   rowptr, colidx, vals : CSR of the m x n matrix (see conventions)
 *   theta_in             : n x f, read only; must not overlap x_out
 *   x_out                : m x f, every row is written
 *   lambda               : >= 0 and finite
 * Rows with no stored entry get x_u = 0 (the paper does not define them; J does not depend
 * on such an x_u).  A row whose A_u is not numerically positive definite (possible only when
 * lambda = 0 or through overflow: a Cholesky pivot that is not positive, is NaN or is +inf)
 * gets NaN in x_u and is counted in the device counter that als_status reports.  The result
 * does not depend on the stream, on earlier calls or on timing: the summation order is fixed.
 */
int als_half_sweep(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx,
                   const float* vals, int64_t m, int64_t n, int32_t f, float lambda,
                   const float* theta_in, float* x_out, void* stream);

/*
 * Training root-mean-square error over the stored entries (the evaluation metric of the
 * paper's experiments, on the training set):
 *   *rmse_out = sqrt( sum over stored (u,v) of (r_uv - x_u . theta_v)^2 / nnz )
 * Residuals in fp32.  The squares of an entry slot's four consecutive pipeline steps (at most
 * four terms) are summed in fp32; those group sums are accumulated in fp64 per fixed chunk of
 * entries, and the chunk sums are added in fp64 in a fixed order.  rmse_out is a DEVICE
 * double; 0 when nnz = 0.
 */
int als_rmse(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
             int64_t m, int64_t n, int32_t f, const float* x, const float* theta,
             double* rmse_out, void* stream);

/* Width of later als_rmse calls on this context: at most `waves_per_simd` resident waves per
   SIMD (1..8), or as many as fit (0, the default).  The entries are always cut into the same
   fixed chunks, claimed by the running waves in order, and summed per chunk in a fixed order,
   so the result does not depend on the width.  A narrow RMSE can run beside a half-sweep of
   another context (its own workspace) on another stream: at f <= 112 the half-sweep leaves
   room for one RMSE wave per SIMD.  ALS_ERR_INVALID_ARG outside 0..8. */
int als_rmse_waves(als_ctx* ctx, int32_t waves_per_simd);

/*
 * For callers that cannot allocate device memory or hold a workspace (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the training RMSE of
 * als_rmse, the same kernels, chunks and summation order (so the same value as als_rmse at its
 * default width), on `device` without a context.  Its scratch -- the chunk counter and one fp64
 * partial per chunk, 256 + 8 x 32 x (compute units) bytes -- is a fixed array of the library
 * of 82,176 bytes (devices of up to 320 compute units; a larger device gets ALS_ERR_WORKSPACE),
 * one copy per device, held until the process ends.  The call allocates nothing: no hipMalloc,
 * no hipFree, no allocating library routine.  Set-up (the device query and the array's device
 * address) runs once per device, in als_init on that device or else in the first call; later
 * calls only check arguments and queue three kernels on `stream` (the counter is cleared by a
 * kernel, not a memset).  Every call on one device shares that device's array: calls that
 * overlap in time on one device -- on different streams or from different host threads --
 * race and give undefined results; the caller orders them.  Arguments, layout and errors as
 * als_rmse; ALS_ERR_DEVICE if `device` is invalid or not a gfx950 device.
 */
int als_rmse_noalloc(int device, const int64_t* rowptr, const int32_t* colidx,
                     const float* vals, int64_t m, int64_t n, int32_t f, const float* x,
                     const float* theta, double* rmse_out, void* stream);

/* Synchronise `stream`, then return (and reset to 0) the number of rows found not positive
   definite by half-sweeps since the previous call. */
int als_status(als_ctx* ctx, void* stream, int64_t* nonspd_rows);

/*
 * The work partition a half-sweep with this f would use (integer work, exposed so it can be
 * checked bit for bit).  Each row u costs c_row + c_nnz n_u units on a cost axis with prefix
 * P(u) = c_nnz rowptr[u] + c_row u, T = P(m).  The axis is cut into C chunks: W large chunks
 * (W = the device's resident waves for this f) cover T1 = T - T2 and C - W small chunks cover
 * T2 = floor(T / tail_div).  Boundary b sits at s_b = floor(T1 b / W) for b <= W and at
 * T1 + floor(T2 (b - W) / (C - W)) for b > W: in row u_b, the largest u with P(u) <= s_b, at
 * entry offset k_b = ceil((s_b - P(u_b) - c_row) / c_nnz) clamped to [0, n_u], rounded to the
 * nearest multiple of q and, if not 0, moved to n_u when fewer than q/2 entries would remain.
 * Chunk c takes the entries from (u_c, k_c) up to (u_{c+1}, k_{c+1}); the waves claim chunks in
 * order from a counter, so the large chunks go first and the small ones even out the finish.  A
 * row cut by a boundary is finished by a second pass that sums its pieces in chunk order, so the
 * result does not depend on which wave ran which chunk.
 *   bounds_out : DEVICE int64[2 (C+1)], (u_b, k_b) pairs; capacity in pairs (>= C + 1, else
 *                ALS_ERR_INVALID_ARG after params_out is filled, so a first call with
 *                capacity 0 learns C)
 *   params_out : HOST int64[6] = {C, c_nnz, c_row, q, W, tail_div}
 */
int als_plan(als_ctx* ctx, const int64_t* rowptr, int64_t m, int32_t f, int64_t* bounds_out,
             int64_t capacity, int64_t* params_out, void* stream);

/*
 * Test and debug support: the gather stage of the half-sweep (Algorithm 1's read of the theta_v
 * of a row's rated columns) for row u, made visible.  The same gather form, index pipeline and
 * operand layout as als_half_sweep with this context and f run over row u, and instead of the
 * matrix products they write what each entry's operands hold.  With NB = f / 16 + 1, entry k
 * of the row (k < n_u) gets a record of 16 (NB + 3) floats at out + k 16 (NB + 3):
 *   [16 I + c]        block I of the MFMA operand, lane c: theta_v[16 I + c] for 16 I + c < f,
 *                     the rating r at 16 I + c == f, 0 beyond (I < NB);
 *   [16 (NB + p) + c] the quad-form operand w[p], when the last block column runs in quad form
 *                     (p < P): theta_v[16 (NB - 1) + 4 p + (c & 3)] for the theta quads, and for
 *                     the rating quad r at (c & 3) == 0, else 0 (untouched otherwise);
 *   [16 (NB + 2) + c] the rating r (every c).
 * Records past capacity (in floats) are not written.  Bit-exact against theta and vals.
 */
int als_gather_dump(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx,
                    const float* vals, int64_t m, int64_t n, int32_t f, const float* theta,
                    int64_t u, float* out, int64_t capacity, void* stream);

/*
 * Measurement support (not part of the method).  After als_profile_begin, each of the next
 * `capacity` half-sweeps records HIP events on its own stream around its three kernels (plan,
 * herm_solve, reduce_solve).  als_profile_end synchronises on the last event, writes
 * ms_out[3 i + 0..2] (HOST, capacity x 3 floats) for half-sweep i in call order, sets
 * *count_out, and stops recording.
 */
int als_profile_begin(als_ctx* ctx, int32_t capacity);
int als_profile_end(als_ctx* ctx, float* ms_out, int32_t capacity, int32_t* count_out);

/*
 * The transpose R -> R^T as CSC (equivalently the CSR of R^T): the input of the update-Theta
 * half-sweep, which applies eq. 2 to the columns of R (eq. 3).  Stable: the entries of a column
 * appear in ascending row order (for a valid CSR, the order of their positions in colidx),
 * with their ratings carried along, so the result is unique and the same on every run.
 *   rowptr, colidx, vals : CSR of the m x n matrix (see conventions); m <= INT32_MAX
 *   colptr               : DEVICE int64[n+1], written: colptr[0] = 0, colptr[n] = nnz
 *   rowidx, vals_t       : DEVICE int32[nnz], fp32[nnz], written: the row index and rating of
 *                          each entry, column by column
 * colidx, vals, rowidx and vals_t must not be null when m > 0 and n > 0 (ALS_ERR_INVALID_ARG).
 * Outputs must not overlap the inputs.  Scratch is the context's workspace (past its status
 * block): it holds one int32 counter per column for each of R row blocks, with R chosen to fit
 * (at most 8 per compute unit, at least 1); if even one block does not fit (about 4 n bytes),
 * ALS_ERR_WORKSPACE.  Entries with a column outside [0, n) are skipped (not validated otherwise;
 * colptr[n] then counts only the others).  Queued on `stream`; it shares the workspace with the
 * other calls of the context, so it must not overlap them in time.
 */
int als_csr_to_csc(als_ctx* ctx, const int64_t* rowptr, const int32_t* colidx, const float* vals,
                   int64_t m, int64_t n, int64_t* colptr, int32_t* rowidx, float* vals_t,
                   void* stream);

/* HIP error code of the most recent ALS_ERR_HIP on this context (0 if none). */
int als_last_hip_error(const als_ctx* ctx);

/* Static description of a status code. */
const char* als_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* ALS_H */
