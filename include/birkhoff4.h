/*
 * birkhoff4.h -- batched 4x4 Birkhoff projection on AMD Instinct MI355X (gfx950).
 *
 * The forward pass projects exp(H[b]) onto the Birkhoff polytope of doubly
 * stochastic 4x4 matrices in the KL geometry (eq. birkhoff_projection), by
 * Newton's method on the reduced 3-dimensional entropic-OT dual (Sec. 3.1-3.2,
 * eq. min_fx, eq. grad_hess; cost M = -H, eta = 1, a = b = 1). The backward pass
 * maps dL/dP to dL/dH by implicit differentiation through the optimality
 * conditions (Sec. 4, eq. derivative, with the sign flip for H = -M), reading
 * only P and dP: no iterates or Hessians are stored.
 *
 * Conventions shared by every entry point
 *   - All array arguments are DEVICE pointers on the current HIP device; the
 *     caller owns them. The library never allocates, frees or synchronises.
 *   - Work is enqueued on `stream` (0 = the null stream) and the call returns
 *     at once; errors found on the host are returned before anything is queued.
 *   - 4x4 arrays are [B][4][4] row-major and contiguous: element (b,i,j) is at
 *     16*b + 4*i + j. `dual` is [B][8] = (alpha_1..alpha_4, beta_1..beta_4) with
 *     beta_4 = 0, so that log P_ij - H_ij = alpha_i + beta_j.
 *   - Every array must be 16-byte aligned, and no output may overlap another
 *     argument (in-place use is not supported).
 *   - B = 0 is a no-op returning BIRKHOFF4_OK.
 *   - Numerical outcomes are not errors: a matrix that does not reach `tol`
 *     within `max_iter` iterations returns its last accepted (row-stochastic)
 *     iterate; a matrix with a NaN or infinite entry returns NaN in all its
 *     outputs. The _ex variants report both cases per matrix.
 */
#ifndef BIRKHOFF4_H
#define BIRKHOFF4_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
    BIRKHOFF4_OK = 0,
    BIRKHOFF4_ERR_NULL = -1,      /* a required pointer is NULL while B > 0 */
    BIRKHOFF4_ERR_SIZE = -2,      /* B < 0, or too large for the index type */
    BIRKHOFF4_ERR_TOL = -3,       /* tol < 0 or NaN */
    BIRKHOFF4_ERR_MAX_ITER = -4,  /* max_iter < 0 or > 10000 */
    BIRKHOFF4_ERR_DTYPE = -5,     /* unknown storage dtype code */
    BIRKHOFF4_ERR_ALIGN = -6,     /* an array is not 16-byte aligned */
    BIRKHOFF4_ERR_OVERLAP = -7,   /* an output overlaps another argument */
    BIRKHOFF4_ERR_STEPS = -8,     /* Sinkhorn step count out of range */
    BIRKHOFF4_ERR_DEVICE = -9,    /* HIP device query failed */
    BIRKHOFF4_ERR_LAUNCH = -10,   /* kernel launch failed (hipGetLastError) */
    BIRKHOFF4_ERR_VARIANT = -11,  /* unknown forward variant */
    BIRKHOFF4_ERR_ETA = -12,      /* eta not positive and finite */
    BIRKHOFF4_ERR_CHANNELS = -13  /* stream width C negative or not a whole number of 16-byte chunks */
};

/* Forward kernel variants (birkhoff4_fwd_ex2). Both compute the same projection to the
 * same tolerance; they differ in how problems map to lanes, so iterates and step counts may
 * differ at the rounding level. */
enum {
    BIRKHOFF4_AUTO = 0,       /* LATENCY for B <= 32768, else THROUGHPUT */
    BIRKHOFF4_THROUGHPUT = 1, /* one problem per lane, with lane-level refill */
    BIRKHOFF4_LATENCY = 2     /* four lanes per problem (one row each), no refill */
};

/* Storage dtypes for inputs (outputs are always fp32; compute is always fp32). */
enum {
    BIRKHOFF4_F32 = 0,
    BIRKHOFF4_BF16 = 1
};

/* Per-matrix status codes written to `iters` by birkhoff4_fwd_ex (values >= 0
 * are the number of Newton trial steps taken, see below). */
enum {
    BIRKHOFF4_NOT_CONVERGED = -1, /* max_iter trial steps did not reach tol */
    BIRKHOFF4_NON_FINITE = -2     /* the input matrix had a NaN or infinite entry */
};

/* Forward projection, fp32 input.
 *
 * H     [B][4][4] fp32 logits (the paper's residual logits, R = -M).
 * P     [B][4][4] fp32 output: the projection, rows summing to one by
 *       construction and every column sum within `tol` of one on return.
 * dual  [B][8] fp32 output, or NULL to skip it: alpha*(beta*) (eq. alpha_opt)
 *       and beta* with beta_4 = 0 (Sec. 3.1 gauge).
 * tol   stopping tolerance on max_j |sum_i P_ij - 1| (the paper uses 1e-6);
 *       tol = 0 stops a matrix only when its fp32 column sums are exactly one,
 *       so in practice most run for max_iter trial steps.
 * max_iter  maximum number of Newton trial steps per matrix, 0..10000 (each is one
 *       evaluation of the dual at a trial point: a damped Newton step, or a
 *       backtracking of it with a larger Levenberg-Marquardt shift). 0 returns T at the initial point, which is the
 *       row softmax of H after the columns are centred (beta_j^(0) = mean of
 *       column 4 minus mean of column j). A step moves the column
 *       potentials apart by at most 8 (natural-log units), so logits whose
 *       solution lies far from the centred start need more: at H ~ N(0, s^2)
 *       64 steps converge every matrix up to s = 100 and leave up to 30 % at
 *       s = 500-1000, where 1000 steps converge them all.
 *   Range: finite logits up to about 5e37 in magnitude are handled; larger
 *       ones can overflow the fp32 scaling by log2(e) and are then reported
 *       like a non-finite input.
 */
int birkhoff4_fwd(const float* H, float* P, float* dual, int64_t B, float tol,
                  int max_iter, hipStream_t stream);

/* Backward (vector-Jacobian product), fp32 upstream gradient.
 *
 * P     [B][4][4] fp32: the projection returned by the forward pass (T*).
 * dual  accepted for symmetry with the forward pass and not read (the 4x4
 *       backward needs only T* and G, Sec. 4.2); may be NULL.
 * dP    [B][4][4] fp32: dL/dP (the paper's G).
 * dH    [B][4][4] fp32 output: dL/dH = -D of eq. derivative, with Delta taken as
 *       the Hessian of the reduced dual at P. Rows and columns of dH sum to zero.
 */
int birkhoff4_bwd(const float* P, const float* dual, const float* dP, float* dH,
                  int64_t B, hipStream_t stream);

/* Forward projection with a storage dtype for H and per-matrix diagnostics.
 * h_dtype is BIRKHOFF4_F32 or BIRKHOFF4_BF16 (H then holds B*16 bf16 values,
 * widened exactly to fp32). iters is NULL or an int32 [B] output receiving the
 * number of trial steps taken, or BIRKHOFF4_NOT_CONVERGED / BIRKHOFF4_NON_FINITE.
 * Other arguments as in birkhoff4_fwd. */
int birkhoff4_fwd_ex(const void* H, int h_dtype, float* P, float* dual, int32_t* iters,
                     int64_t B, float tol, int max_iter, hipStream_t stream);

/* Forward with an explicit kernel variant (BIRKHOFF4_AUTO, _THROUGHPUT or _LATENCY); other
 * arguments as in birkhoff4_fwd_ex, which is this call with BIRKHOFF4_AUTO. The latency
 * variant splits each problem's row-wise work over four lanes (the paper's Sec. 3.3 also
 * spreads one matrix over several lanes), which shortens the serial chain of a Newton step
 * for batches too small to fill the GPU; returns BIRKHOFF4_ERR_VARIANT for other values. */
int birkhoff4_fwd_ex2(const void* H, int h_dtype, float* P, float* dual, int32_t* iters,
                      int64_t B, float tol, int max_iter, int variant, hipStream_t stream);

/* Backward with a storage dtype for dP (BIRKHOFF4_F32 or BIRKHOFF4_BF16). */
int birkhoff4_bwd_ex(const float* P, const void* dP, int dp_dtype, float* dH, int64_t B,
                     hipStream_t stream);

/* Saved-Hessian variant (Sec. 4.2: at the solution the Hessian of the reduced dual equals
 * the Delta of eq. derivative, so the forward's Hessian can be kept for the backward).
 * birkhoff4_fwd_hess is birkhoff4_fwd_ex (one problem per lane, any B) that also writes,
 * per matrix, the six column weights W_jk = sum_i P_ij P_ik of its output P, whose
 * Laplacian grounded at column 4 is that Hessian: hess [B][8] fp32 =
 * (W_12, W_13, W_14, W_23, W_24, W_34, 0, 0), 32 bytes per matrix, caller-owned, 16-byte
 * aligned, not overlapping the other arrays; dual and iters may be NULL.
 * birkhoff4_bwd_hess is birkhoff4_bwd_ex taking those weights instead of recomputing them
 * from P. Both return the codes of the calls they extend; hess NULL gives
 * BIRKHOFF4_ERR_NULL. This trades 32 bytes of writes and of reads per matrix for the six
 * weight sums of the backward; the default pair above does not use it. */
int birkhoff4_fwd_hess(const void* H, int h_dtype, float* P, float* dual, float* hess, int32_t* iters,
                       int64_t B, float tol, int max_iter, hipStream_t stream);
int birkhoff4_bwd_hess(const float* P, const float* hess, const void* dP, int dp_dtype, float* dH,
                       int64_t B, hipStream_t stream);

/* Baseline: n_steps iterations of Sinkhorn-Knopp (eq. sinkhorn_knopp) from
 * v^(0) = 1 on A = exp(H) (each row shifted by its maximum, which leaves every
 * iterate diag(u) A diag(v) unchanged); P = diag(u^(n)) A diag(v^(n)), whose
 * columns sum to one. 1 <= n_steps <= 48. Denominators are clamped at the
 * smallest normal fp32 so that underflowed rows and columns stay finite. */
int birkhoff4_sk_fwd(const void* H, int h_dtype, float* P, int64_t B, int n_steps,
                     hipStream_t stream);

/* Baseline backward: the exact gradient of the n_steps Sinkhorn-Knopp map at H,
 * applied to dP (reverse mode through the unrolled iterations, recomputed from
 * H in registers; nothing is stored between the passes). */
int birkhoff4_sk_bwd(const void* H, int h_dtype, const void* dP, int dp_dtype, float* dH,
                     int64_t B, int n_steps, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * n = 8 (the mHC layer with eight streams, Sec. 3.1): the same projection and
 * gradient for 8 x 8 matrices, by Newton on the 7-dimensional reduced dual with the
 * general gradient and Hessian (eq. grad_hess with a = b = 1, eta = 1) and the general
 * implicit backward (eq. derivative). Return codes, dtypes and status words as above.
 *
 * H     [B][8][8] (h_dtype fp32 or bf16), row-major, device memory.
 * P     [B][8][8] fp32 output: rows and columns sum to one within tol.
 * dual  NULL or [B][16] fp32 output: (alpha_1..alpha_8, beta_1..beta_7, beta_8 = 0),
 *       natural-log units, log P_ij = H_ij + alpha_i + beta_j.
 * iters NULL or int32 [B] output: trial steps taken, BIRKHOFF4_NOT_CONVERGED or
 *       BIRKHOFF4_NON_FINITE (that matrix's P and dual are then NaN).
 * tol, max_iter as in birkhoff4_fwd. Buffers must not overlap; 16-byte alignment.
 * Asynchronous on `stream`; nothing is allocated. */
int birkhoff8_fwd(const void* H, int h_dtype, float* P, float* dual, int32_t* iters,
                  int64_t B, float tol, int max_iter, hipStream_t stream);

/* Backward for n = 8: dH [B][8][8] fp32 = dL/dH from P (the forward's output) and
 * dP [B][8][8] (dp_dtype fp32 or bf16), eq. derivative with Delta the Hessian of the
 * reduced dual at P. Rows and columns of dH sum to zero. dH must not overlap P or dP. */
int birkhoff8_bwd(const float* P, const void* dP, int dp_dtype, float* dH, int64_t B,
                  hipStream_t stream);

/* ---------------------------------------------------------------------------
 * General entropic OT for 4 x 4 (eq. entropic, Sec. 2.3): for each b,
 *   T = argmin over { T >= 0, T 1 = a, T^T 1 = b } of <T, M> - eta h(T),
 * h(T) = -sum T_ij (log T_ij - 1), by the same Newton iteration on the reduced dual
 * (eq. min_fx with the general eq. grad_hess); the Birkhoff projection is the case
 * M = -H, a = b = 1, eta = 1.
 *
 * M     [B][4][4] fp32 cost, row-major.
 * a, b  [B][4] fp32 marginals: positive, sum(a[b]) = sum(b[b]) for each b (when the
 *       sums differ there is no solution and the status is BIRKHOFF4_NOT_CONVERGED).
 * eta   regulariser > 0 (BIRKHOFF4_ERR_ETA otherwise).
 * T     [B][4][4] fp32 output: rows sum to a exactly up to rounding, columns to b
 *       within tol: |c_j - b_j| <= tol max(1, sum(a) / n, b_j) for every column (n = 4
 *       here): absolute for unit-sized marginals, relative above, where the fp32 resolution
 *       of the column sums grows with the masses; for a = b = 1 this is the Birkhoff test.
 *       The last column, whose potential is fixed, may in addition differ by
 *       |sum a - sum b| as computed in fp32, since fp32 marginals rarely have equal sums.
 * dual  NULL or [B][8] fp32 output: (alpha_1..4, beta_1..3, beta_4 = 0) in the units of
 *       M, with T_ij = exp((alpha_i + beta_j - M_ij) / eta) (eq. dual).
 * iters NULL or int32 [B]: trial steps taken, BIRKHOFF4_NOT_CONVERGED, or
 *       BIRKHOFF4_NON_FINITE for a NaN, infinite or non-positive input (T, dual NaN).
 * tol, max_iter, alignment, overlap rules and asynchrony as in birkhoff4_fwd. */
int birkhoff4_ot_fwd(const float* M, const float* a, const float* b, float eta, float* T,
                     float* dual, int32_t* iters, int64_t B, float tol, int max_iter,
                     hipStream_t stream);

/* Backward of birkhoff4_ot_fwd (eq. derivative): dM [B][4][4] fp32 = dL/dM from the
 * solution T, the row marginals a [B][4] and dT = dL/dT [B][4][4] fp32, with Delta the
 * Hessian of the reduced dual at T. Rows and columns of dM sum to zero. dM must not
 * overlap the inputs. */
int birkhoff4_ot_bwd(const float* T, const float* a, const float* dT, float eta, float* dM,
                     int64_t B, hipStream_t stream);

/* General entropic OT for 8 x 8 problems: birkhoff4_ot_fwd / birkhoff4_ot_bwd with n = m = 8
 * (eq. entropic, eq. grad_hess, eq. derivative). M, T, dT, dM are [B][8][8] fp32 (256 bytes per
 * problem), a and b [B][8] fp32, dual [B][16] = (alpha_1..8, beta_1..7, beta_8 = 0) with
 * T_ij = exp((alpha_i + beta_j - M_ij) / eta); iters as for birkhoff8_fwd. Arguments, return
 * codes, status words and ownership as for the 4 x 4 calls. */
int birkhoff8_ot_fwd(const float* M, const float* a, const float* b, float eta, float* T, float* dual,
                     int32_t* iters, int64_t B, float tol, int max_iter, hipStream_t stream);
int birkhoff8_ot_bwd(const float* T, const float* a, const float* dT, float eta, float* dM, int64_t B,
                     hipStream_t stream);

/* Residual mixing of the mHC layer (Sec. 2.1): each token's n = 4 streams are mixed by its
 * projected matrix, Y = P X with P = proj(exp(H)), the term H^res x_l of the layer's update.
 *
 * H      [B][4][4] logits, h_dtype F32 or BF16 (as in birkhoff4_fwd_ex).
 * X      [B][4][C] streams of each token, row-major (stream i of token b starts at element
 *        (4 b + i) C), x_dtype F32 or BF16; NULL allowed when C = 0.
 * Y      [B][4][C] output in x_dtype: Y_i = sum_j P_ij X_j per token, accumulated in fp32;
 *        bf16 results are rounded to nearest even.
 * P      [B][4][4] fp32 output: the projection, exactly what birkhoff4_fwd_ex would write
 *        for H (the default forward variant); the backward needs it.
 * dual, iters  NULL or outputs as in birkhoff4_fwd_ex.
 * C      channels per stream, >= 0, a multiple of 8 for BF16 streams or 4 for F32
 *        (BIRKHOFF4_ERR_CHANNELS otherwise): every row is whole 16-byte chunks.
 * tol, max_iter as in birkhoff4_fwd. Y must not overlap any input or P, dual or iters; P,
 * dual and iters must not overlap X. Every check is made before anything is queued. */
int birkhoff4_mix_fwd(const void* H, int h_dtype, const void* X, int x_dtype, void* Y, float* P, float* dual,
                      int32_t* iters, int64_t B, int64_t C, float tol, int max_iter, hipStream_t stream);

/* Backward of birkhoff4_mix_fwd: from P (its output), the streams X and dY = dL/dY
 * ([B][4][C], both in x_dtype), writes dX = dL/dX = P^T dY per token ([B][4][C] in x_dtype,
 * fp32 accumulation, bf16 rounded to nearest even) and dH = dL/dH ([B][4][4] fp32): the
 * projection's backward (eq. derivative, as in birkhoff4_bwd) applied to
 * dP_ij = sum_c dY_i[c] X_j[c]. One pass over X and dY. Outputs must not overlap each other
 * or any input. Return codes as for birkhoff4_mix_fwd. */
int birkhoff4_mix_bwd(const float* P, const void* X, const void* dY, int x_dtype, void* dX, float* dH, int64_t B,
                      int64_t C, hipStream_t stream);

/* Residual mixing with n = 8 streams per token: birkhoff4_mix_fwd / birkhoff4_mix_bwd with the
 * 8 x 8 projection (birkhoff8_fwd / birkhoff8_bwd). H and P are [B][8][8], X, Y, dY, dX are
 * [B][8][C] (stream i of token b starts at element (8 b + i) C), dual [B][16] and iters as for
 * birkhoff8_fwd, dH [B][8][8] fp32. Arguments, dtypes, the rule for C, return codes and overlap
 * rules as for the 4 x 4 calls. */
int birkhoff8_mix_fwd(const void* H, int h_dtype, const void* X, int x_dtype, void* Y, float* P, float* dual,
                      int32_t* iters, int64_t B, int64_t C, float tol, int max_iter, hipStream_t stream);
int birkhoff8_mix_bwd(const float* P, const void* X, const void* dY, int x_dtype, void* dX, float* dH, int64_t B,
                      int64_t C, hipStream_t stream);

/* Human-readable text for a return code (static storage). */
const char* birkhoff4_strerror(int code);

/* Library version: major * 10000 + minor * 100 + patch. */
int birkhoff4_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BIRKHOFF4_H */
