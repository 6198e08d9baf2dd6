// birkhoff4.hip -- batched 4x4 Birkhoff projection for gfx950 (MI355X).
//
// Forward: Newton's method on the reduced 3-dimensional entropic-OT dual
// (Sec. 3.1-3.2: eq. min_fx, eq. grad_hess, eq. tij_stable, eq. c_g), with cost
// M = -H, eta = 1, a = b = 1. Backward: implicit differentiation (Sec. 4,
// eq. derivative) from P and dP only. Baseline: n-step Sinkhorn-Knopp
// (eq. sinkhorn_knopp) and its reverse-mode gradient.
//
// Mapping: one 4x4 problem per lane; all per-problem state lives in VGPRs. No
// MFMA (the only products are six 4-long dot products per matrix), no global
// atomics. Loads and stores are 16-byte vector accesses. The implicit kernel
// streams wave-contiguous pieces with non-temporal hints and transposes them
// through LDS; the Newton kernel uses LDS for its ring of initialised problems, for
// staging its outputs and for the batch counter its waves share; it writes P
// non-temporally and the 32-byte dual records through L2, where neighbouring records
// that finish close in time merge into whole lines.
//
// Forward numerics (fp32; exponents in log2 units so that v_exp_f32 applies directly;
// the library is compiled with fp32 denormals flushed to zero):
//  * state is the row softmax T at the current point, with the row normalisers a and
//    column potentials beta (log2 T = H log2(e) + beta - a 1^T). A trial that moves the
//    potentials by s multiplies column j by 2^(s_j) and renormalises the rows: three
//    exponentials per trial instead of sixteen, and entries keep full relative precision
//    whatever |beta| is (a beta-only state recomputed from H cannot tune the column sums
//    below ~1e-5 once |beta| reaches hundreds). Entries that fall below the smallest
//    normal float flush to zero and are re-derived from H once the accumulated column
//    shifts could have brought them within reach of fp32 resolution;
//  * Hessian of the reduced dual = Laplacian of the column graph with weights
//    W_jk = sum_i T_ij T_ik (rows of T sum to one), grounded at column 4; the
//    Newton system is solved by elimination with pivots formed as sums of these
//    positive weights, plus a Levenberg-Marquardt shift max(1e-3 max_j |g_j|, 5e-8)
//    that keeps directions finite when weights underflow and keeps gradient
//    components at the fp32 rounding floor from driving huge steps;
//  * step: spread of the column shifts max_j d_j - min_j d_j (with d_4 = 0) capped at 8
//    (natural-log units), Armijo backtracking on the
//    reduced dual f, with a gradient-norm test once f no longer resolves the
//    decrease; each backtrack halves the step and multiplies the shift by 16
//    (re-solving with the saved weights), and the trial step doubles while full
//    steps keep descending strongly;
//  * initial point beta_j = mean_i H_i4 - mean_i H_ij (column centring), evaluated in the
//    log domain;
//  * stop when max over the four columns of |c_j - 1| <= tol.
//
// Work distribution: each workgroup owns a contiguous range of problems, cut into
// batches of 64 that its waves claim through an LDS counter. A wave initialises a batch
// with one problem per lane at full width: the initial point, its column sums and, for
// problems not already converged there, the column weights and gradient. Problems that
// are finished at the initial point are written out at once; the others are compacted
// into a per-wave LDS ring. Every lane then runs Newton trials on its own problem, and a
// lane whose problem finishes writes it out and takes the next problem from the ring at
// once, so a wave pays the mean number of trials, not the maximum over its 64 lanes.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <tuple>
#include <type_traits>

#include "birkhoff4.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kCap2 = 8.0f * kLog2e;  // step cap in log2 units
constexpr float kLM = 1e-3f;            // Levenberg-Marquardt coefficient
// Floor of the shift: column sums are rounded to ~2e-7 in fp32, so a gradient at that
// level is noise; with the floor it can move a weakly coupled column by a few nats at
// most instead of swamping the step that the real residual needs.
constexpr float kLMFloor = 5e-8f;
constexpr float kArmijo = 1e-4f;
constexpr float kFNoise = 4e-6f;        // |delta f| below this is rounding noise
constexpr int kMaxExpandLog2 = 4;      // initial trial step <= 16
constexpr float kMaxShift = 1e18f;      // keeps the escalated shift finite
constexpr float kTiny = 1e-30f;
// Backward pivots at or below this are treated as disconnected nodes (potential 0):
// v_rcp_f32 of a denormal is infinite, and such a node's entries of dH carry
// factors of T that are far below fp32 resolution anyway.
constexpr float kPivMin = 1e-30f;
constexpr float kFltMin = 1.17549435e-38f;
constexpr int kMaxSkSteps = 48;   // sk_bwd keeps (n+1) x 4 floats per lane in LDS
constexpr int kSkRegSteps = 20;   // step count whose backward keeps the iterates in VGPRs
constexpr int kMaxIterCap = 10000;
// Batches up to this size take the four-lanes-per-problem forward by default.
constexpr int64_t kLatencyMaxB = int64_t(1) << 15;
constexpr int64_t kMaxGrid = int64_t(1) << 24;  // blocks of a streaming launch
constexpr int kFwdBlock = 1024;  // one workgroup per CU: 16 waves, 4 per SIMD
constexpr int kFwdWaves = kFwdBlock / 64;
// Ring slot of the forward kernel, in v4f: a problem's state at its initial point.
constexpr int kSlot = 9;
// Accumulated spread of column shifts (log2 units) after which entries that flushed to
// zero are re-derived from H: such an entry was below 2^-126 when it flushed and has grown
// by at most this much (plus one trial's spread, <= 2 step caps) since, so it is still
// below 2^-43 when it is re-derived.
constexpr float kReviveBits = 60.0f;

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// ---------------------------------------------------------------------------
// Loads and stores of one 4x4 problem (row-major, 64 B fp32 / 32 B bf16)
// ---------------------------------------------------------------------------
__device__ __forceinline__ void load16_f32(const float* base, int64_t b, float v[16]) {
    const v4f* p = reinterpret_cast<const v4f*>(base) + 4 * b;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const v4f r = *(p + q);
        v[4 * q + 0] = r.x;
        v[4 * q + 1] = r.y;
        v[4 * q + 2] = r.z;
        v[4 * q + 3] = r.w;
    }
}

__device__ __forceinline__ void load16_bf16(const uint16_t* base, int64_t b, float v[16]) {
    const v4u* p = reinterpret_cast<const v4u*>(base) + 2 * b;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const v4u r = *(p + q);
        const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[8 * q + 2 * k + 0] = __uint_as_float(w[k] << 16);
            v[8 * q + 2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
    }
}

template <int DT>
__device__ __forceinline__ void load16(const void* base, int64_t b, float v[16]) {
    if constexpr (DT == BIRKHOFF4_BF16)
        load16_bf16(static_cast<const uint16_t*>(base), b, v);
    else
        load16_f32(static_cast<const float*>(base), b, v);
}

// Raw storage words of one problem (8 for bf16, 16 for fp32), kept undecoded in the
// prefetch ring and moved between lanes with ds_bpermute.
template <int DT>
struct RawWords {
    static constexpr int n = (DT == BIRKHOFF4_BF16) ? 8 : 16;
};

template <int DT>
__device__ __forceinline__ void load_raw(const void* base, int64_t b, uint32_t w[RawWords<DT>::n]) {
    const v4u* p = reinterpret_cast<const v4u*>(base) + (RawWords<DT>::n / 4) * b;
#pragma unroll
    for (int q = 0; q < RawWords<DT>::n / 4; ++q) {
        const v4u r = p[q];
        w[4 * q + 0] = r.x;
        w[4 * q + 1] = r.y;
        w[4 * q + 2] = r.z;
        w[4 * q + 3] = r.w;
    }
}

template <int DT>
__device__ __forceinline__ void decode_raw(const uint32_t w[RawWords<DT>::n], float h[16]) {
    if constexpr (DT == BIRKHOFF4_BF16) {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            h[2 * k + 0] = __uint_as_float(w[k] << 16);
            h[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k) h[k] = __uint_as_float(w[k]);
    }
}

__device__ __forceinline__ void store16(float* base, int64_t b, const float v[16]) {
    v4f* p = reinterpret_cast<v4f*>(base) + 4 * b;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const v4f r = {v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]};
        *(p + q) = r;
    }
}

// ---------------------------------------------------------------------------
// Forward
// ---------------------------------------------------------------------------

// Column-graph weights W_jk = sum_i T_ij T_ik (the p_jk of Sec. 3.2 extended to
// column 4). With unit row sums the Hessian of the reduced dual is the Laplacian
// of this graph grounded at column 4: h_jk = -W_jk, h_jj = sum_{k != j} W_jk.
struct Weights {
    float w01, w02, w03, w12, w13, w23;
};

__device__ __forceinline__ Weights column_weights(const float T[16]) {
    Weights W = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float t0 = T[4 * i], t1 = T[4 * i + 1], t2 = T[4 * i + 2], t3 = T[4 * i + 3];
        W.w01 = __builtin_fmaf(t0, t1, W.w01);
        W.w02 = __builtin_fmaf(t0, t2, W.w02);
        W.w03 = __builtin_fmaf(t0, t3, W.w03);
        W.w12 = __builtin_fmaf(t1, t2, W.w12);
        W.w13 = __builtin_fmaf(t1, t3, W.w13);
        W.w23 = __builtin_fmaf(t2, t3, W.w23);
    }
    return W;
}

// Newton direction in log2 units: d = -log2(e) (Lap(W) + lam I)^{-1} g.
// Elimination of nodes 0, 1, 2 in turn; every pivot is a sum of non-negative
// conductances (lam acts as an extra conductance to the ground).
__device__ __forceinline__ void newton_solve(const Weights& W, float g0, float g1, float g2, float lam,
                                             float& d0, float& d1, float& d2) {
    float r0 = -kLog2e * g0, r1 = -kLog2e * g1, r2 = -kLog2e * g2;
    float q0 = W.w03 + lam, q1 = W.w13 + lam, q2 = W.w23 + lam;  // conductance to ground
    const float i0 = rcp(__builtin_fmaxf(W.w01 + W.w02 + q0, kTiny));
    const float f1 = W.w01 * i0, f2 = W.w02 * i0;
    const float a12 = __builtin_fmaf(f1, W.w02, W.w12);
    q1 = __builtin_fmaf(f1, q0, q1);
    q2 = __builtin_fmaf(f2, q0, q2);
    r1 = __builtin_fmaf(f1, r0, r1);
    r2 = __builtin_fmaf(f2, r0, r2);
    const float i1 = rcp(__builtin_fmaxf(a12 + q1, kTiny));
    const float f2b = a12 * i1;
    q2 = __builtin_fmaf(f2b, q1, q2);
    r2 = __builtin_fmaf(f2b, r1, r2);
    d2 = r2 * rcp(__builtin_fmaxf(q2, kTiny));
    d1 = __builtin_fmaf(a12, d2, r1) * i1;
    d0 = __builtin_fmaf(W.w01, d1, __builtin_fmaf(W.w02, d2, r0)) * i0;
}

// Spread max_j v_j - min_j v_j of a column shift (v_4 = 0). It bounds how far any entry
// of the row-normalised T can move, in log2 units, when the column potentials move by v.
__device__ __forceinline__ float spread(float v0, float v1, float v2) {
    return __builtin_fmaxf(__builtin_fmaxf(v0, v1), __builtin_fmaxf(v2, 0.f)) -
           __builtin_fminf(__builtin_fminf(v0, v1), __builtin_fminf(v2, 0.f));
}

// Trial evaluation, eq. tij_stable in product form. T is the row softmax at the current
// point; moving the column potentials by s (log2 units, s_4 = 0) multiplies column j by
// 2^(s_j), and each row is renormalised. T becomes the trial's row softmax, l the log2 of
// the row sums (the change of the row normalisers) and g the column sums minus one
// (eq. c_g, all four columns). Products that fall below the smallest normal float flush
// to zero; such entries are re-derived from H when they could matter again.
__device__ __forceinline__ void evaluate(float T[16], float s0, float s1, float s2, float l[4], float g[4]) {
    const float S0 = ex2(s0), S1 = ex2(s1), S2 = ex2(s2);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float e0 = T[4 * i + 0] * S0;
        const float e1 = T[4 * i + 1] * S1;
        const float e2 = T[4 * i + 2] * S2;
        const float e3 = T[4 * i + 3];
        const float sum = (e0 + e1) + (e2 + e3);
        const float r = rcp(sum);
        l[i] = lg2(sum);
        T[4 * i + 0] = e0 * r;
        T[4 * i + 1] = e1 * r;
        T[4 * i + 2] = e2 * r;
        T[4 * i + 3] = e3 * r;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
        g[j] = ((T[j] + T[4 + j]) + (T[8 + j] + T[12 + j])) - 1.0f;
}

// Initial point of one problem from its raw words: beta^(0)_j = mean_i H_i4 - mean_i H_ij
// (column centring), T = row softmax of H + 1 beta^T evaluated in the log domain with the
// row maxima subtracted (eq. tij_stable), a = log2 of the row normalisers of
// H log2(e) + beta, g = column sums - 1. A NaN or infinite entry makes the column-mean
// sum NaN or infinite and poisons T, a and beta with NaN (a finite sum that overflows
// needs entries near FLT_MAX, where exp overflows anyway).
template <int DT>
__device__ __forceinline__ void init_problem(const uint32_t w[RawWords<DT>::n], float T[16], float a[4],
                                             float& b0, float& b1, float& b2, float g[4]) {
    float h[16];
    decode_raw<DT>(w, h);
    float cm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cm[j] = 0.25f * kLog2e * ((h[j] + h[4 + j]) + (h[8 + j] + h[12 + j]));
    const float hs = (cm[0] + cm[1]) + (cm[2] + cm[3]);
    const float poison = hs - hs;  // 0, or NaN for a non-finite input
    b0 = cm[3] - cm[0] + poison;
    b1 = cm[3] - cm[1] + poison;
    b2 = cm[3] - cm[2] + poison;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float u0 = __builtin_fmaf(h[4 * i + 0], kLog2e, b0);
        const float u1 = __builtin_fmaf(h[4 * i + 1], kLog2e, b1);
        const float u2 = __builtin_fmaf(h[4 * i + 2], kLog2e, b2);
        const float u3 = __builtin_fmaf(h[4 * i + 3], kLog2e, poison);
        const float m = __builtin_fmaxf(__builtin_fmaxf(u0, u1), __builtin_fmaxf(u2, u3)) + poison;
        const float e0 = ex2(u0 - m), e1 = ex2(u1 - m), e2 = ex2(u2 - m), e3 = ex2(u3 - m);
        const float sum = (e0 + e1) + (e2 + e3);
        const float r = rcp(sum);
        T[4 * i + 0] = e0 * r;
        T[4 * i + 1] = e1 * r;
        T[4 * i + 2] = e2 * r;
        T[4 * i + 3] = e3 * r;
        a[i] = m + lg2(sum);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
        g[j] = ((T[j] + T[4 + j]) + (T[8 + j] + T[12 + j])) - 1.0f;
}

// Output of one problem: P = T, dual = (alpha*(beta), beta) in natural-log units with
// beta_4 = 0 (NaN for a poisoned input), the status word, and (saved-Hessian variant) the
// column weights of P.
template <bool WRITE_DUAL, bool WRITE_ITERS, bool WRITE_HESS>
__device__ __forceinline__ void store_output(float* __restrict__ P, float* __restrict__ dual,
                                             int32_t* __restrict__ iters, float* __restrict__ hess, int64_t gi,
                                             const float T[16], const float a[4], float b0, float b1, float b2,
                                             int status) {
    store16(P, gi, T);
    if constexpr (WRITE_HESS) {
        const Weights W = column_weights(T);
        v4f* hp = reinterpret_cast<v4f*>(hess) + 2 * gi;
        hp[0] = v4f{W.w01, W.w02, W.w03, W.w12};
        hp[1] = v4f{W.w13, W.w23, 0.f, 0.f};
    }
    if constexpr (WRITE_DUAL) {
        v4f* dp = reinterpret_cast<v4f*>(dual) + 2 * gi;
        dp[0] = v4f{-a[0] * kLn2, -a[1] * kLn2, -a[2] * kLn2, -a[3] * kLn2};
        dp[1] = v4f{b0 * kLn2, b1 * kLn2, b2 * kLn2, b0 * 0.f};
    }
    if constexpr (WRITE_ITERS) iters[gi] = status;
}

template <int DT, bool WRITE_DUAL, bool WRITE_ITERS, bool WRITE_HESS>
__global__ __launch_bounds__(kFwdBlock) void newton_fwd_kernel(const void* __restrict__ H,
                                                                float* __restrict__ P,
                                                                float* __restrict__ dual,
                                                                int32_t* __restrict__ iters,
                                                                float* __restrict__ hess, int64_t B,
                                                                int64_t chunk, float tol, int max_iter) {
    constexpr int NW = RawWords<DT>::n;
    const int lane = threadIdx.x & 63;
    // the wave index is uniform across the wave: keep the range bookkeeping in SGPRs
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    // Per-wave ring of 64 slots of kSlot v4f. A slot first holds a problem that is
    // initialised and not finished at its initial point: T rows (v4f 0..3), a (4),
    // beta_1..3 and the problem's offset (5), the column weights and gradient at the
    // initial point (6..8). The lane that takes it leaves the output of its previous
    // problem in its place: P rows (0..3), dual (4..5), (offset or -1, status) (6), and in
    // the saved-Hessian variant the column weights of P (7..8).
    __shared__ v4f ring_all[kFwdWaves][64 * kSlot];
    __shared__ int32_t next_batch;  // next unclaimed batch of the block's range
    v4f* const ring = ring_all[wv];
    // The block owns problems lo .. hi - 1, in batches of 64 consecutive problems. Its
    // waves share them through an LDS counter: a wave that the SIMD arbiter favours
    // simply takes more batches, so all waves of a CU finish within about one batch.
    const int64_t lo = static_cast<int64_t>(blockIdx.x) * chunk;
    if (lo >= B) return;  // uniform across the block
    const int64_t hi = (lo + chunk < B) ? lo + chunk : B;
    const int32_t nrel = static_cast<int32_t>(hi - lo);
    const int32_t nbatch = (nrel + 63) >> 6;
    if (threadIdx.x == 0) next_batch = kFwdWaves;  // wave w starts on batch w
    __syncthreads();
    if (wv >= nbatch) return;  // uniform across the wave
    auto claim = [&]() -> int32_t {
        int32_t v = 0;
        if (lane == 0) v = atomicAdd(&next_batch, 1);
        return __builtin_amdgcn_readfirstlane(v);
    };
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

    // Raw words of the batch to initialise next (one problem per lane), loaded one batch
    // ahead with whole-wave loads.
    uint32_t raw[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) raw[q] = 0u;
    int32_t nxt = wv;
    if ((nxt << 6) + lane < nrel) load_raw<DT>(H, lo + (nxt << 6) + lane, raw);
    int nfresh = 0;  // ring slots [icur, nfresh) hold problems not yet taken
    int icur = 0;

    // Per-problem state of this lane. T is the current point (row softmax); a, beta its
    // row normalisers and column potentials (log2 units, so log2 T = H log2(e) + beta - a).
    bool active = false;   // working on a problem
    bool want = true;      // needs a problem
    bool has_out = false;  // holds the finished output of its last problem
    int status = 0;        // status word of that output
    int32_t rel = 0;       // problem offset from lo
    float T[16], a[4], b0 = 0.f, b1 = 0.f, b2 = 0.f;
#pragma unroll
    for (int q = 0; q < 16; ++q) T[q] = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = 0.f;
    Weights Wa = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};  // column weights at the accepted point
    float ga0 = 0.f, ga1 = 0.f, ga2 = 0.f;        // gradient at the accepted point
    float lam = 0.f;                              // Levenberg-Marquardt shift
    float gn2 = 0.f;                              // |g|^2 at the accepted point
    float t = 1.f;                                // trial step along the Newton direction
    float o0 = 0.f, o1 = 0.f, o2 = 0.f;           // current point minus accepted point
    float fofs = 0.f;                             // f(current) - f(accepted), log2 units
    float gsum = 0.f;                             // column-shift spreads since the last re-derivation
    // bits 0-15: trial steps taken; bits 16-18: log2 of the initial trial step
    int cnt = 0;

    // Write out the outputs left in ring slots h0 .. h0 + n - 1, 16 problems at a time: 4
    // lanes per P (one 64-byte row block each), 2 per dual, 1 per status, so that a store
    // instruction writes whole 64-byte pieces. A slot whose offset is negative holds no
    // output. Each pass reads its slots' offsets and data before it branches on them.
    auto flush = [&](int h0, int n) {
        for (int h = 0; h < n; h += 16) {
            const int m = (n - h < 16) ? n - h : 16;
            const int ep = lane >> 2, ed = lane >> 1;
            const v4f* sp = ring + (h0 + h + (ep < m ? ep : 0)) * kSlot;
            const v4f* sd = ring + (h0 + h + (ed < m ? ed : 0)) * kSlot;
            const v4f* si = ring + (h0 + h + (lane < m ? lane : 0)) * kSlot;
            const int32_t ip = __float_as_int(sp[6].x);
            const v4f pv = sp[lane & 3];
            int32_t id = -1;
            v4f dv = {0.f, 0.f, 0.f, 0.f}, hv = {0.f, 0.f, 0.f, 0.f};
            if constexpr (WRITE_DUAL || WRITE_HESS) id = __float_as_int(sd[6].x);
            if constexpr (WRITE_DUAL) dv = sd[4 + (lane & 1)];
            if constexpr (WRITE_HESS) hv = sd[7 + (lane & 1)];
            int32_t ii = -1, st = 0;
            if constexpr (WRITE_ITERS) {
                const v4f sv = si[6];
                ii = __float_as_int(sv.x);
                st = __float_as_int(sv.y);
            }
            // P bypasses L2 retention (non-temporal): the partial dual lines then stay in
            // L2 long enough to merge with their neighbours' halves
            if (ep < m && ip >= 0) __builtin_nontemporal_store(pv, reinterpret_cast<v4f*>(P) + 4 * (lo + ip) + (lane & 3));
            if constexpr (WRITE_DUAL)
                if (ed < m && id >= 0) reinterpret_cast<v4f*>(dual)[2 * (lo + id) + (lane & 1)] = dv;
            if constexpr (WRITE_HESS)
                if (ed < m && id >= 0) reinterpret_cast<v4f*>(hess)[2 * (lo + id) + (lane & 1)] = hv;
            if constexpr (WRITE_ITERS)
                if (lane < m && ii >= 0) iters[lo + ii] = st;
        }
    };

    // Leave the output of this lane's finished problem in ring slot `slot`.
    auto stage_output = [&](int slot, const float To[16], const float ao[4], float c0, float c1, float c2,
                            int32_t idx, int st) {
        v4f* sl = ring + slot * kSlot;
        sl[0] = v4f{To[0], To[1], To[2], To[3]};
        sl[1] = v4f{To[4], To[5], To[6], To[7]};
        sl[2] = v4f{To[8], To[9], To[10], To[11]};
        sl[3] = v4f{To[12], To[13], To[14], To[15]};
        if constexpr (WRITE_DUAL) {
            sl[4] = v4f{-ao[0] * kLn2, -ao[1] * kLn2, -ao[2] * kLn2, -ao[3] * kLn2};
            sl[5] = v4f{c0 * kLn2, c1 * kLn2, c2 * kLn2, c0 * 0.f};  // beta_4 = 0, NaN if poisoned
        }
        sl[6] = v4f{__int_as_float(idx), __int_as_float(st), 0.f, 0.f};
        if constexpr (WRITE_HESS) {
            const Weights W = column_weights(To);
            sl[7] = v4f{W.w01, W.w02, W.w03, W.w12};
            sl[8] = v4f{W.w13, W.w23, 0.f, 0.f};
        }
    };

    // Initialise the batch whose raw words are loaded, one problem per lane with the whole
    // wave. Every global store of the kernel is issued here (or after the last batch), right
    // after the wait for the batch's words and before the next batch's words are requested:
    // memory operations retire in order, so that wait never covers a store younger than one
    // batch period. The outputs left in the ring are written out first. Then the problems
    // that are not finished at their initial point are compacted into ring slots
    // 0 .. nfresh - 1 with their column weights and gradient, and those that are (converged,
    // non-finite, or max_iter = 0) are staged right after them and written out.
    auto init_batch = [&]() {
        // Take the batch's words into use here (the compiler waits for them before these
        // empty statements), and keep every store below after them.
#pragma unroll
        for (int q = 0; q < NW; ++q) asm volatile("" : "+v"(raw[q])::"memory");
        const int32_t r = (nxt << 6) + lane;
        float Ti[16], ai[4], c0, c1, c2, g[4];
        init_problem<DT>(raw, Ti, ai, c0, c1, c2, g);
        flush(0, nfresh);
        const float gmax = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(g[0]), __builtin_fabsf(g[1])),
                                           __builtin_fmaxf(__builtin_fabsf(g[2]), __builtin_fabsf(g[3])));
        const bool nonfinite = __builtin_isnan(c0);  // beta is NaN exactly for poisoned inputs
        const bool conv = gmax <= tol;
        const bool valid = r < nrel;
        const bool done = valid && (conv || nonfinite || max_iter == 0);
        const bool fresh = valid && !done;
        const uint64_t fm = __ballot(fresh), dm = __ballot(done);
        const int nf = __popcll(fm);
        if (fresh) {
            v4f* sl = ring + __popcll(fm & below) * kSlot;
            const Weights W = column_weights(Ti);
            sl[0] = v4f{Ti[0], Ti[1], Ti[2], Ti[3]};
            sl[1] = v4f{Ti[4], Ti[5], Ti[6], Ti[7]};
            sl[2] = v4f{Ti[8], Ti[9], Ti[10], Ti[11]};
            sl[3] = v4f{Ti[12], Ti[13], Ti[14], Ti[15]};
            sl[4] = v4f{ai[0], ai[1], ai[2], ai[3]};
            sl[5] = v4f{c0, c1, c2, __int_as_float(r)};
            sl[6] = v4f{W.w01, W.w02, W.w03, W.w12};
            sl[7] = v4f{W.w13, W.w23, g[0], g[1]};
            sl[8] = v4f{g[2], __builtin_fmaxf(kLM * gmax, kLMFloor),
                        g[0] * g[0] + g[1] * g[1] + g[2] * g[2] + g[3] * g[3], 0.f};
        }
        if (done)
            stage_output(nf + __popcll(dm & below), Ti, ai, c0, c1, c2, r,
                         nonfinite ? BIRKHOFF4_NON_FINITE : (conv ? 0 : BIRKHOFF4_NOT_CONVERGED));
        flush(nf, __popcll(dm));
        nfresh = nf;
        icur = 0;
        nxt = claim();
        if (nxt < nbatch && (nxt << 6) + lane < nrel) load_raw<DT>(H, lo + (nxt << 6) + lane, raw);
    };

    for (;;) {
        if (active) {
            // Newton direction at the accepted point, with the step capped so that no two
            // columns move apart by more than the cap (gauge-symmetric)
            float d0, d1, d2;
            newton_solve(Wa, ga0, ga1, ga2, lam, d0, d1, d2);
            t = __builtin_fminf(t, kCap2 * rcp(__builtin_fmaxf(spread(d0, d1, d2), kTiny)));
            // trial point: accepted point + t d, reached from the current point
            const float s0 = __builtin_fmaf(t, d0, -o0), s1 = __builtin_fmaf(t, d1, -o1),
                        s2 = __builtin_fmaf(t, d2, -o2);
            float l[4], g[4];
            evaluate(T, s0, s1, s2, l, g);
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] += l[i];
            b0 += s0;
            b1 += s1;
            b2 += s2;
            o0 += s0;
            o1 += s1;
            o2 += s2;
            // f(trial) - f(accepted) = f(current) - f(accepted) + row-wise change (log2 units)
            const float df = fofs + ((l[0] + l[1]) + (l[2] + l[3])) - ((s0 + s1) + s2);
            fofs = df;
            gsum += spread(s0, s1, s2);
            ++cnt;
            const float gmax = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(g[0]), __builtin_fabsf(g[1])),
                                               __builtin_fmaxf(__builtin_fabsf(g[2]), __builtin_fabsf(g[3])));
            const float gn2t = g[0] * g[0] + g[1] * g[1] + g[2] * g[2] + g[3] * g[3];
            // directional derivative of f along d at the accepted point (log2 units)
            const float slope = ga0 * d0 + ga1 * d1 + ga2 * d2;
            const bool accept = (df <= kArmijo * t * slope) || (__builtin_fabsf(df) < kFNoise && gn2t < gn2);
            const int evals = cnt & 0xffff;
            const bool conv = accept && gmax <= tol;
            if (!conv && evals < max_iter) {
                // Entries that underflowed to zero can grow by at most the accumulated spread;
                // before that could bring one within reach of fp32 resolution, re-derive every
                // zero entry from H at the current point (they stay zero while still tiny).
                if (gsum >= kReviveBits) {
                    gsum = 0.f;
                    float tmin = T[0];
#pragma unroll
                    for (int q = 1; q < 16; ++q) tmin = __builtin_fminf(tmin, T[q]);
                    if (tmin == 0.f) {
                        float h[16];
                        load16<DT>(H, lo + rel, h);
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float bj[4] = {b0, b1, b2, 0.f};
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                if (T[4 * i + j] == 0.f)
                                    T[4 * i + j] = ex2(__builtin_fmaf(h[4 * i + j], kLog2e, bj[j]) - a[i]);
                        }
                    }
                }
                if (accept) {
                    const float dd = g[0] * d0 + g[1] * d1 + g[2] * d2;
                    const int ts = cnt >> 16;  // the trial step doubles while full steps
                    const bool grow = t >= 0.999f * __builtin_ldexpf(1.f, ts) && dd < 0.25f * slope;
                    cnt = evals | ((grow ? (ts < kMaxExpandLog2 ? ts + 1 : ts) : 0) << 16);
                    fofs = 0.f;
                    o0 = o1 = o2 = 0.f;
                    gn2 = gn2t;
                    Wa = column_weights(T);
                    ga0 = g[0];
                    ga1 = g[1];
                    ga2 = g[2];
                    lam = __builtin_fmaxf(kLM * gmax, kLMFloor);
                    t = __builtin_ldexpf(1.f, cnt >> 16);
                } else {
                    // backtrack: halve the step and raise the Levenberg-Marquardt shift, so a
                    // direction spoiled by rounding in weakly coupled modes is replaced
                    t *= 0.5f;
                    cnt = evals;
                    lam = __builtin_fminf(16.f * lam, kMaxShift);
                }
            } else {
                if (!accept) {
                    // max_iter reached on a rejected trial: return to the accepted point
                    evaluate(T, -o0, -o1, -o2, l, g);
#pragma unroll
                    for (int i = 0; i < 4; ++i) a[i] += l[i];
                    b0 -= o0;
                    b1 -= o1;
                    b2 -= o2;
                }
                status = conv ? evals : BIRKHOFF4_NOT_CONVERGED;
                active = false;
                want = true;
                has_out = true;
            }
        }
        // Hand-off: every lane that wants a problem takes the next one of the ring and
        // leaves its finished output in the slot; batches are initialised as the ring runs out.
        uint64_t wm = __ballot(want);
        while (wm != 0) {
            const int k = __popcll(wm);
            const int rank = __popcll(wm & below);
            const int avail = nfresh - icur;
            if (want && rank < avail) {
                const v4f* sl = ring + (icur + rank) * kSlot;
                const v4f r0 = sl[0], r1 = sl[1], r2 = sl[2], r3 = sl[3], av = sl[4], bv = sl[5],
                          w0 = sl[6], w1 = sl[7], w2 = sl[8];
                stage_output(icur + rank, T, a, b0, b1, b2, has_out ? rel : -1, status);
                T[0] = r0.x; T[1] = r0.y; T[2] = r0.z; T[3] = r0.w;
                T[4] = r1.x; T[5] = r1.y; T[6] = r1.z; T[7] = r1.w;
                T[8] = r2.x; T[9] = r2.y; T[10] = r2.z; T[11] = r2.w;
                T[12] = r3.x; T[13] = r3.y; T[14] = r3.z; T[15] = r3.w;
                a[0] = av.x; a[1] = av.y; a[2] = av.z; a[3] = av.w;
                b0 = bv.x; b1 = bv.y; b2 = bv.z;
                rel = __float_as_int(bv.w);
                Wa = Weights{w0.x, w0.y, w0.z, w0.w, w1.x, w1.y};
                ga0 = w1.z; ga1 = w1.w; ga2 = w2.x;
                lam = w2.y;
                gn2 = w2.z;
                t = 1.f;
                o0 = o1 = o2 = 0.f;
                fofs = gsum = 0.f;
                cnt = 0;
                active = true;
                want = false;
                has_out = false;
            }
            if (k <= avail) {
                icur += k;
                break;
            }
            icur = nfresh;
            if (nxt >= nbatch) {
                // nothing left to initialise: lanes still holding an output write it and idle
                if (has_out)
                    store_output<WRITE_DUAL, WRITE_ITERS, WRITE_HESS>(P, dual, iters, hess, lo + rel, T, a, b0, b1,
                                                                      b2, status);
                has_out = false;
                want = false;
                break;
            }
            init_batch();
            wm = __ballot(want);
        }
        if (__ballot(active) == 0) break;
    }
    flush(0, icur);
}

// ---------------------------------------------------------------------------
// Forward, latency variant: four lanes per problem
// ---------------------------------------------------------------------------
// For small batches the one-problem-per-lane kernel is bound by the serial chain of one
// Newton trial (~300 dependent instructions) times the slowest problem's trial count. Here
// the four lanes of a quad hold one row each: the row-wise work of a trial is split four
// ways, column sums and column weights are butterfly sums over the quad (DPP quad_perm, so
// every lane of the quad gets bit-identical results), and the 3x3 solve and step control
// run redundantly in the four lanes. There is no refill: a wave covers 16 problems and
// runs until its slowest one is done, which is what a small batch pays anyway.

// Sum over the four lanes of a quad, in the association ((x0 + x1) + (x2 + x3)); all four
// lanes receive the same value. Contraction is off here: fused into a product computed by the
// caller, the first add would become fma(own factors, partner's rounded product), which
// differs between partner lanes, and the quad's replicated step control would split.
__device__ __forceinline__ float qsum(float x) {
#pragma clang fp contract(off)
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, true));  // (1,0,3,2)
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, true));  // (2,3,0,1)
    return x;
}

// The value held by lane k of the quad, in every lane of the quad.
template <int K>
__device__ __forceinline__ float qget(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), K | (K << 2) | (K << 4) | (K << 6), 0xF, 0xF, true));
}

// Row q of problem b (4 values).
template <int DT>
__device__ __forceinline__ void load_row(const void* base, int64_t b, int q, float h[4]) {
    if constexpr (DT == BIRKHOFF4_BF16) {
        const uint32_t* p = static_cast<const uint32_t*>(base) + 8 * b + 2 * q;
        const uint2 w = *reinterpret_cast<const uint2*>(p);
        h[0] = __uint_as_float(w.x << 16);
        h[1] = __uint_as_float(w.x & 0xffff0000u);
        h[2] = __uint_as_float(w.y << 16);
        h[3] = __uint_as_float(w.y & 0xffff0000u);
    } else {
        const v4f r = reinterpret_cast<const v4f*>(base)[4 * b + q];
        h[0] = r.x; h[1] = r.y; h[2] = r.z; h[3] = r.w;
    }
}

template <int DT, bool WRITE_DUAL, bool WRITE_ITERS>
__global__ __launch_bounds__(256) void newton_fwd_quad_kernel(const void* __restrict__ H,
                                                               float* __restrict__ P,
                                                               float* __restrict__ dual,
                                                               int32_t* __restrict__ iters, int64_t B,
                                                               float tol, int max_iter) {
    const int64_t gt = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t b = gt >> 2;       // this quad's problem
    const int q = threadIdx.x & 3;   // this lane's row
    const bool valid = b < B;        // uniform across the quad
    // Initial point (column centring), eq. tij_stable in the log domain, as in init_problem.
    float h[4] = {0.f, 0.f, 0.f, 0.f};
    if (valid) load_row<DT>(H, b, q, h);
    float cm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cm[j] = 0.25f * kLog2e * qsum(h[j]);
    const float hs = (cm[0] + cm[1]) + (cm[2] + cm[3]);
    const float poison = hs - hs;  // 0, or NaN for a non-finite input anywhere in the matrix
    float b0 = cm[3] - cm[0] + poison, b1 = cm[3] - cm[1] + poison, b2 = cm[3] - cm[2] + poison;
    float T[4], a;
    {
        const float u0 = __builtin_fmaf(h[0], kLog2e, b0), u1 = __builtin_fmaf(h[1], kLog2e, b1),
                    u2 = __builtin_fmaf(h[2], kLog2e, b2), u3 = __builtin_fmaf(h[3], kLog2e, poison);
        const float m = __builtin_fmaxf(__builtin_fmaxf(u0, u1), __builtin_fmaxf(u2, u3)) + poison;
        const float e0 = ex2(u0 - m), e1 = ex2(u1 - m), e2 = ex2(u2 - m), e3 = ex2(u3 - m);
        const float sum = (e0 + e1) + (e2 + e3);
        const float r = rcp(sum);
        T[0] = e0 * r; T[1] = e1 * r; T[2] = e2 * r; T[3] = e3 * r;
        a = m + lg2(sum);
    }
    float g[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) g[j] = qsum(T[j]) - 1.0f;
    auto gmax_of = [](const float gg[4]) {
        return __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(gg[0]), __builtin_fabsf(gg[1])),
                               __builtin_fmaxf(__builtin_fabsf(gg[2]), __builtin_fabsf(gg[3])));
    };
    auto weights = [&]() {
        return Weights{qsum(T[0] * T[1]), qsum(T[0] * T[2]), qsum(T[0] * T[3]),
                       qsum(T[1] * T[2]), qsum(T[1] * T[3]), qsum(T[2] * T[3])};
    };
    float gmax = gmax_of(g);
    const bool nonfinite = __builtin_isnan(b0);
    bool active = valid && !(gmax <= tol) && !nonfinite && max_iter > 0;
    int status = nonfinite ? BIRKHOFF4_NON_FINITE : (gmax <= tol ? 0 : BIRKHOFF4_NOT_CONVERGED);
    Weights Wa = weights();
    float ga0 = g[0], ga1 = g[1], ga2 = g[2];
    float lam = __builtin_fmaxf(kLM * gmax, kLMFloor);
    float gn2 = g[0] * g[0] + g[1] * g[1] + g[2] * g[2] + g[3] * g[3];
    float t = 1.f, o0 = 0.f, o1 = 0.f, o2 = 0.f, fofs = 0.f, gsum = 0.f;
    int cnt = 0;
    while (__ballot(active)) {
        if (active) {
            float d0, d1, d2;
            newton_solve(Wa, ga0, ga1, ga2, lam, d0, d1, d2);
            t = __builtin_fminf(t, kCap2 * rcp(__builtin_fmaxf(spread(d0, d1, d2), kTiny)));
            const float s0 = __builtin_fmaf(t, d0, -o0), s1 = __builtin_fmaf(t, d1, -o1),
                        s2 = __builtin_fmaf(t, d2, -o2);
            // trial evaluation of this lane's row (product form, as evaluate())
            const float e0 = T[0] * ex2(s0), e1 = T[1] * ex2(s1), e2 = T[2] * ex2(s2), e3 = T[3];
            const float sum = (e0 + e1) + (e2 + e3);
            const float r = rcp(sum);
            const float l = lg2(sum);
            T[0] = e0 * r; T[1] = e1 * r; T[2] = e2 * r; T[3] = e3 * r;
            float gt4[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) gt4[j] = qsum(T[j]) - 1.0f;
            a += l;
            b0 += s0; b1 += s1; b2 += s2;
            o0 += s0; o1 += s1; o2 += s2;
            const float df = fofs + qsum(l) - ((s0 + s1) + s2);
            fofs = df;
            gsum += spread(s0, s1, s2);
            ++cnt;
            const float gm = gmax_of(gt4);
            const float gn2t = gt4[0] * gt4[0] + gt4[1] * gt4[1] + gt4[2] * gt4[2] + gt4[3] * gt4[3];
            const float slope = ga0 * d0 + ga1 * d1 + ga2 * d2;
            const bool accept = (df <= kArmijo * t * slope) || (__builtin_fabsf(df) < kFNoise && gn2t < gn2);
            const int evals = cnt & 0xffff;
            const bool conv = accept && gm <= tol;
            if (!conv && evals < max_iter) {
                if (gsum >= kReviveBits) {  // flushed entries: re-derive from H (per lane)
                    gsum = 0.f;
                    const float bj[4] = {b0, b1, b2, 0.f};
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        if (T[j] == 0.f) T[j] = ex2(__builtin_fmaf(h[j], kLog2e, bj[j]) - a);
                }
                if (accept) {
                    const float dd = gt4[0] * d0 + gt4[1] * d1 + gt4[2] * d2;
                    const int ts = cnt >> 16;
                    const bool grow = t >= 0.999f * __builtin_ldexpf(1.f, ts) && dd < 0.25f * slope;
                    cnt = evals | ((grow ? (ts < kMaxExpandLog2 ? ts + 1 : ts) : 0) << 16);
                    fofs = 0.f;
                    o0 = o1 = o2 = 0.f;
                    gn2 = gn2t;
                    Wa = weights();
                    ga0 = gt4[0]; ga1 = gt4[1]; ga2 = gt4[2];
                    lam = __builtin_fmaxf(kLM * gm, kLMFloor);
                    t = __builtin_ldexpf(1.f, cnt >> 16);
                } else {
                    t *= 0.5f;
                    cnt = evals;
                    lam = __builtin_fminf(16.f * lam, kMaxShift);
                }
            } else {
                if (!accept) {  // max_iter reached on a rejected trial: back to the accepted point
                    const float f0 = T[0] * ex2(-o0), f1 = T[1] * ex2(-o1), f2 = T[2] * ex2(-o2), f3 = T[3];
                    const float s = (f0 + f1) + (f2 + f3);
                    const float rr = rcp(s);
                    T[0] = f0 * rr; T[1] = f1 * rr; T[2] = f2 * rr; T[3] = f3 * rr;
                    a += lg2(s);
                    b0 -= o0; b1 -= o1; b2 -= o2;
                }
                status = conv ? evals : BIRKHOFF4_NOT_CONVERGED;
                active = false;
            }
        }
    }
    // outputs: lane q writes row q of P; lanes 0 and 1 write the dual record; lane 0 the status
    if (valid) {
        reinterpret_cast<v4f*>(P)[4 * b + q] = v4f{T[0], T[1], T[2], T[3]};
        const float al0 = qget<0>(a), al1 = qget<1>(a), al2 = qget<2>(a), al3 = qget<3>(a);
        if constexpr (WRITE_DUAL) {
            v4f* dp = reinterpret_cast<v4f*>(dual) + 2 * b;
            if (q == 0) dp[0] = v4f{-al0 * kLn2, -al1 * kLn2, -al2 * kLn2, -al3 * kLn2};
            if (q == 1) dp[1] = v4f{b0 * kLn2, b1 * kLn2, b2 * kLn2, b0 * 0.f};
        }
        if constexpr (WRITE_ITERS)
            if (q == 0) iters[b] = status;
    }
}

// ---------------------------------------------------------------------------
// Backward (Sec. 4.2)
// ---------------------------------------------------------------------------
// dH for one problem from T (= P) and G (= dP): -D of eq. derivative, Sec. 4.2. With
// GIVEN_W the column weights come from the forward (the Hessian at the solution, which is
// the Delta of eq. derivative: the saved-Hessian reading of Sec. 4.2) instead of from T.
template <bool GIVEN_W = false>
__device__ __forceinline__ void implicit_vjp(const float T[16], const float G[16], float out[16],
                                             const float* Wg = nullptr) {
    // W_jk = sum_i T_ij T_ik; F_jk = sum_i T_ij T_ik (G_ij - G_ik): the right-hand
    // side mu_c,j - sum_i T_ij mu_r,i of eq. derivative is sum_{k != j} F_jk.
    float W01 = 0.f, W02 = 0.f, W03 = 0.f, W12 = 0.f, W13 = 0.f, W23 = 0.f;
    float F01 = 0.f, F02 = 0.f, F03 = 0.f, F12 = 0.f, F13 = 0.f, F23 = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float t0 = T[4 * i], t1 = T[4 * i + 1], t2 = T[4 * i + 2], t3 = T[4 * i + 3];
        const float g0 = G[4 * i], g1 = G[4 * i + 1], g2 = G[4 * i + 2], g3 = G[4 * i + 3];
        float p;
        p = t0 * t1; if constexpr (!GIVEN_W) W01 += p; F01 = __builtin_fmaf(p, g0 - g1, F01);
        p = t0 * t2; if constexpr (!GIVEN_W) W02 += p; F02 = __builtin_fmaf(p, g0 - g2, F02);
        p = t0 * t3; if constexpr (!GIVEN_W) W03 += p; F03 = __builtin_fmaf(p, g0 - g3, F03);
        p = t1 * t2; if constexpr (!GIVEN_W) W12 += p; F12 = __builtin_fmaf(p, g1 - g2, F12);
        p = t1 * t3; if constexpr (!GIVEN_W) W13 += p; F13 = __builtin_fmaf(p, g1 - g3, F13);
        p = t2 * t3; if constexpr (!GIVEN_W) W23 += p; F23 = __builtin_fmaf(p, g2 - g3, F23);
    }
    if constexpr (GIVEN_W) {
        W01 = Wg[0]; W02 = Wg[1]; W03 = Wg[2]; W12 = Wg[3]; W13 = Wg[4]; W23 = Wg[5];
    }
    // Delta w = rhs, Delta = Hessian at T (Laplacian of W grounded at column 4).
    // Eliminating a node joins its neighbours j,k by W_jp W_pk / piv and moves its
    // flows onto the same edges, F_jk += (W_pk F_jp + W_jp F_pk) / piv, so every
    // right-hand side stays a sum of antisymmetric edge flows. Each product is formed
    // as (W_jp / piv) times a weight or flow: the ratio is at most one, so a product
    // underflows only when its result does (two tiny weights multiplied first could
    // flush to zero while the flows they pair with survive).
    const float piv0 = W01 + W02 + W03;
    const float i0 = piv0 > kPivMin ? rcp(piv0) : 0.f;
    const float f1 = W01 * i0, f2 = W02 * i0, f3 = W03 * i0;
    const float W12b = __builtin_fmaf(f1, W02, W12);
    const float W13b = __builtin_fmaf(f1, W03, W13);
    const float W23b = __builtin_fmaf(f2, W03, W23);
    const float F12b = __builtin_fmaf(f1, F02, __builtin_fmaf(-f2, F01, F12));
    const float F13b = __builtin_fmaf(f1, F03, __builtin_fmaf(-f3, F01, F13));
    const float F23b = __builtin_fmaf(f2, F03, __builtin_fmaf(-f3, F02, F23));
    const float piv1 = W12b + W13b;
    const float i1 = piv1 > kPivMin ? rcp(piv1) : 0.f;
    const float g2 = W12b * i1, g3 = W13b * i1;
    const float W23c = __builtin_fmaf(g2, W13b, W23b);
    const float F23c = __builtin_fmaf(g2, F13b, __builtin_fmaf(-g3, F12b, F23b));
    const float w2 = W23c > kPivMin ? F23c * rcp(W23c) : 0.f;
    const float w1 = __builtin_fmaf(W12b, w2, F12b + F13b) * i1;
    const float w0 = __builtin_fmaf(W01, w1, __builtin_fmaf(W02, w2, (F01 + F02) + F03)) * i0;
    // dH = -D: dH_ij = T_ij (psi_ij - sum_k T_ik psi_ik), psi = G - 1 w^T, w_4 = 0
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float s0 = G[4 * i] - w0, s1 = G[4 * i + 1] - w1, s2 = G[4 * i + 2] - w2,
                    s3 = G[4 * i + 3];
        const float avg = __builtin_fmaf(T[4 * i], s0,
                          __builtin_fmaf(T[4 * i + 1], s1,
                          __builtin_fmaf(T[4 * i + 2], s2, T[4 * i + 3] * s3)));
        out[4 * i + 0] = T[4 * i + 0] * (s0 - avg);
        out[4 * i + 1] = T[4 * i + 1] * (s1 - avg);
        out[4 * i + 2] = T[4 * i + 2] * (s2 - avg);
        out[4 * i + 3] = T[4 * i + 3] * (s3 - avg);
    }
}

// One 64-problem chunk per wave: P, dP and dH move between HBM and registers in
// wave-contiguous 16-byte pieces (each load or store instruction covers 1 KB of
// consecutive problems), transposed through a per-wave LDS buffer to one problem per
// lane. Per-lane 64-byte records (four 16-byte accesses at a 64-byte stride) stream at
// about half the rate. Every byte is touched once, so all accesses carry the
// non-temporal hint (measured 11 % faster on MI355X than default caching).
constexpr int kBwdBlock = 256;
constexpr int kBwdWaves = kBwdBlock / 64;
constexpr int kBwdStride = 5;  // v4f per problem in the LDS buffer (4 rows + 1 pad: no bank conflicts on reads)

template <int DT, bool HESS = false>
__global__ __launch_bounds__(kBwdBlock) void implicit_bwd_kernel(const float* __restrict__ P,
                                                                  const void* __restrict__ dP,
                                                                  float* __restrict__ dH, int64_t B,
                                                                  const float* __restrict__ hess) {
    __shared__ v4f buf_all[kBwdWaves][64 * kBwdStride];
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    v4f* const buf = buf_all[wv];
    const v4f* P4 = reinterpret_cast<const v4f*>(P);
    v4f* dH4 = reinterpret_cast<v4f*>(dH);
    // slot of the 16-byte piece this lane moves in a coalesced access q: problem 16 q + lane / 4, row lane % 4
    const int cpos = (lane >> 2) * kBwdStride + (lane & 3);
    const int64_t nchunk = (B + 63) / 64;
    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kBwdWaves + wv; c < nchunk;
         c += static_cast<int64_t>(gridDim.x) * kBwdWaves) {
        const int64_t base = c * 64;
        const int n = (B - base < 64) ? static_cast<int>(B - base) : 64;  // problems in this chunk
        // issue every load of the chunk first
        v4f pc[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = 64 * q + lane;  // 16-byte piece within the chunk
            pc[q] = k < 4 * n ? __builtin_nontemporal_load(P4 + 4 * base + k) : v4f{0.f, 0.f, 0.f, 0.f};
        }
        constexpr int NG = (DT == BIRKHOFF4_BF16) ? 2 : 4;  // 16-byte pieces of dP per lane
        constexpr int GP = (DT == BIRKHOFF4_BF16) ? 2 : 4;  // 16-byte pieces per problem
        v4u gc[NG];
        const v4u* G4 = reinterpret_cast<const v4u*>(dP);
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int k = 64 * q + lane;
            gc[q] = k < GP * n ? __builtin_nontemporal_load(G4 + GP * base + k) : v4u{0u, 0u, 0u, 0u};
        }
        [[maybe_unused]] v4f hc[2];  // saved column weights (saved-Hessian variant), two pieces per problem
        if constexpr (HESS) {
            const v4f* W4 = reinterpret_cast<const v4f*>(hess);
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int k = 64 * q + lane;
                hc[q] = k < 2 * n ? __builtin_nontemporal_load(W4 + 2 * base + k) : v4f{0.f, 0.f, 0.f, 0.f};
            }
        }
        // P: pieces to one problem per lane
#pragma unroll
        for (int q = 0; q < 4; ++q) buf[16 * q * kBwdStride + cpos] = pc[q];
        __builtin_amdgcn_wave_barrier();
        float T[16], G[16];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const v4f t = buf[lane * kBwdStride + r];
            T[4 * r + 0] = t.x; T[4 * r + 1] = t.y; T[4 * r + 2] = t.z; T[4 * r + 3] = t.w;
        }
        __builtin_amdgcn_wave_barrier();
        // dP: the same, GP pieces per problem
        v4u* bufu = reinterpret_cast<v4u*>(buf);
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int k = 64 * q + lane;
            bufu[(k / GP) * kBwdStride + (k % GP)] = gc[q];
        }
        __builtin_amdgcn_wave_barrier();
        {
            uint32_t w[4 * GP];
#pragma unroll
            for (int r = 0; r < GP; ++r) {
                const v4u u = bufu[lane * kBwdStride + r];
                w[4 * r + 0] = u.x; w[4 * r + 1] = u.y; w[4 * r + 2] = u.z; w[4 * r + 3] = u.w;
            }
            decode_raw<DT>(w, G);
        }
        __builtin_amdgcn_wave_barrier();
        float out[16];
        if constexpr (HESS) {
            // saved column weights: two 16-byte pieces per problem, through the same buffer
#pragma unroll
            for (int q = 0; q < 2; ++q) {
                const int k = 64 * q + lane;
                buf[(k >> 1) * kBwdStride + (k & 1)] = hc[q];
            }
            __builtin_amdgcn_wave_barrier();
            const v4f w0 = buf[lane * kBwdStride], w1 = buf[lane * kBwdStride + 1];
            __builtin_amdgcn_wave_barrier();
            const float Wg[6] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y};
            implicit_vjp<true>(T, G, out, Wg);
        } else {
            implicit_vjp(T, G, out);
        }
        // dH: one problem per lane to pieces
#pragma unroll
        for (int r = 0; r < 4; ++r)
            buf[lane * kBwdStride + r] = v4f{out[4 * r], out[4 * r + 1], out[4 * r + 2], out[4 * r + 3]};
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = 64 * q + lane;
            const v4f o = buf[16 * q * kBwdStride + cpos];
            if (k < 4 * n) __builtin_nontemporal_store(o, dH4 + 4 * base + k);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// Residual mixing of the mHC layer (Sec. 2.1): the streams of a token are mixed by its
// projected matrix, x <- H^res x
// ---------------------------------------------------------------------------
// A token carries n = 4 (or 8) streams of C channels, [B][n][C] row-major. The forward
// writes Y_i = sum_j P_ij X_j; the backward writes dX_j = sum_i P_ij dY_i and forms
// dP_ij = sum_c dY_i[c] X_j[c], from which dH follows as in the projection's backward. A
// wave works on one token at a time (with n = 8, the four waves of a block on the same
// token): P is uniform over the wave (scalar loads) and the lanes stream 16-byte chunks of
// the rows, so that each load or store instruction covers 1 KB of one row. Every stream
// byte is touched once: non-temporal loads and stores.
constexpr int kMixBlock = 256;
constexpr int kMixWaves = kMixBlock / 64;
constexpr int kMixPerCu = 8;  // blocks per CU the grid is sized for

template <int DX>
struct MixChunk {  // channels in one 16-byte chunk of a row
    static constexpr int E = (DX == BIRKHOFF4_BF16) ? 8 : 4;
};

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

template <int DX>
__device__ __forceinline__ void unpack_chunk(const v4u w, float v[MixChunk<DX>::E]) {
    const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if constexpr (DX == BIRKHOFF4_BF16) {
            v[2 * k + 0] = __uint_as_float(u[k] << 16);
            v[2 * k + 1] = __uint_as_float(u[k] & 0xffff0000u);
        } else {
            v[k] = __uint_as_float(u[k]);
        }
    }
}

// bf16 outputs are rounded to nearest even (the hardware conversion).
template <int DX>
__device__ __forceinline__ v4u pack_chunk(const float v[MixChunk<DX>::E]) {
    uint32_t u[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if constexpr (DX == BIRKHOFF4_BF16)
            u[k] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{v[2 * k], v[2 * k + 1]}), bf16x2));
        else
            u[k] = __float_as_uint(v[k]);
    }
    return v4u{u[0], u[1], u[2], u[3]};
}

// Channels of 32-bit word w of a chunk: two for bf16, one for fp32.
template <int DX>
__device__ __forceinline__ void unpack_word(const v4u c, int w, float v[MixChunk<DX>::E / 4]) {
    const uint32_t u = w == 0 ? c.x : w == 1 ? c.y : w == 2 ? c.z : c.w;
    if constexpr (DX == BIRKHOFF4_BF16) {
        v[0] = __uint_as_float(u << 16);
        v[1] = __uint_as_float(u & 0xffff0000u);
    } else {
        v[0] = __uint_as_float(u);
    }
}

// out_i = sum_j m_ij in_j over the E channels of one chunk of each of the N rows (TRANS:
// m_ji, the transpose, read in place), one 32-bit word of the chunk at a time so that only
// that word's channels are unpacked at once.
template <int DX, int N, bool TRANS = false>
__device__ __forceinline__ void mix_chunk(const float m[N * N], const v4u in[N], v4u out[N]) {
    constexpr int EW = MixChunk<DX>::E / 4;
    uint32_t o[N][4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        float x[N][EW];
#pragma unroll
        for (int j = 0; j < N; ++j) unpack_word<DX>(in[j], w, x[j]);
#pragma unroll
        for (int i = 0; i < N; ++i) {
            float y[EW];
#pragma unroll
            for (int e = 0; e < EW; ++e) {
                y[e] = m[TRANS ? i : N * i] * x[0][e];
#pragma unroll
                for (int j = 1; j < N; ++j) y[e] = __builtin_fmaf(m[TRANS ? N * j + i : N * i + j], x[j][e], y[e]);
            }
            if constexpr (DX == BIRKHOFF4_BF16)
                o[i][w] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{y[0], y[1]}), bf16x2));
            else
                o[i][w] = __float_as_uint(y[0]);
        }
    }
#pragma unroll
    for (int i = 0; i < N; ++i) out[i] = v4u{o[i][0], o[i][1], o[i][2], o[i][3]};
}

// P of token t (N x N), uniform over the wave.
template <int N>
__device__ __forceinline__ void load_token_matrix(const float* __restrict__ P, int64_t t, float p[N * N]) {
    const float* pt = P + N * N * t;
#pragma unroll
    for (int q = 0; q < N * N; ++q) p[q] = pt[q];
}

// A wave walks the items (t, c0) of its tokens: lane l handles chunk c0 + l of each of the
// N rows. With one wave per token (WPT = 1) c0 = 0, 64, 128, ... < nc; with WPT waves per
// token, wave s of the token takes c0 = 64 s, 64 (s + WPT), ..., so that the token's waves
// stream adjacent kilobytes of each row together. (Eight rows per token are sixteen or
// twenty-four separate streams per wave; measured on a plain copy of this pattern, HBM
// delivers about 10% more when four waves share a token's rows than when one wave walks
// them alone. In the 8-stream backward two or eight waves per token measured 5-8% slower
// than four. Four rows stream best one token per wave.) The next item's loads are issued
// before the current item is mixed and stored (loads and stores retire in order, so a
// wait for loads issued after a store would also wait for that store), into the other of
// two buffers so that no register copy waits for them. Lanes past the end of a row take
// its last chunk: they load, mix and store the same bytes as that chunk's own lane, so
// every memory instruction is issued by the whole wave and the waits count exactly.
// A block of kMixWaves waves takes kMixWaves tokens at a time (WPT = 1); with WPT > 1 the
// block is the WPT waves of one token.
constexpr int kMix8Wpt = 4;  // waves per token of the n = 8 kernels

template <int WPT>
struct MixWalk {  // a wave's first token and chunk, and the strides of its walk
    static constexpr int kTokensPerBlock = WPT == 1 ? kMixWaves : 1;
    static constexpr int kBlockThreads = WPT == 1 ? kMixBlock : 64 * WPT;
    static constexpr int64_t kStep = 64 * WPT;
    static __device__ __forceinline__ int wave() {
        return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    }
    static __device__ __forceinline__ int64_t first_token() {
        return static_cast<int64_t>(blockIdx.x) * kTokensPerBlock + (WPT == 1 ? wave() : 0);
    }
    static __device__ __forceinline__ int64_t first_chunk() { return 64 * (wave() % WPT); }
    static __device__ __forceinline__ int64_t token_stride() {
        return static_cast<int64_t>(gridDim.x) * kTokensPerBlock;
    }
};

template <int DX, int N, int WPT = 1>
__global__ __launch_bounds__(kMixBlock) void mix_fwd_kernel(const float* __restrict__ P,
                                                             const v4u* __restrict__ X, v4u* __restrict__ Y,
                                                             int64_t B, int64_t nc) {
    using W = MixWalk<WPT>;
    const int lane = threadIdx.x & 63;
    const int64_t stride = W::token_stride();
    const int64_t cfirst = W::first_chunk();
    int64_t t = W::first_token();
    if (t >= B || cfirst >= nc) return;  // uniform over the wave; nc >= 1 here
    int64_t c0 = cfirst;
    auto offset = [&](int64_t tt, int64_t cc0) {
        const int64_t cc = cc0 + lane;
        return N * nc * tt + (cc < nc ? cc : nc - 1);
    };
    auto load_item = [&](int64_t off, v4u v[N]) {
#pragma unroll
        for (int j = 0; j < N; ++j) v[j] = __builtin_nontemporal_load(X + off + j * nc);
    };
    float p[N * N];
    load_token_matrix<N>(P, t, p);
    // mix the item in `cur` while the next one (or, after the last, this one again) loads
    // into `nxt`
    auto step = [&](const v4u cur[N], v4u nxt[N]) {
        int64_t tn = t, cn = c0 + W::kStep;
        if (cn >= nc) {
            cn = cfirst;
            tn = t + stride;
        }
        const bool more = tn < B;
        load_item(more ? offset(tn, cn) : offset(t, c0), nxt);
        __builtin_amdgcn_sched_barrier(0);  // keep the prefetch ahead of the waits for `cur`
        v4u out[N];
        mix_chunk<DX, N>(p, cur, out);
        const int64_t off = offset(t, c0);
#pragma unroll
        for (int i = 0; i < N; ++i) __builtin_nontemporal_store(out[i], Y + off + i * nc);
        if (more && tn != t) load_token_matrix<N>(P, tn, p);
        t = tn;
        c0 = cn;
    };
    // The first step is peeled and the rest run as a counted loop of two steps: each step's
    // loads are then used unconditionally by the next one (so they stay where they are
    // issued), and every path into a step leaves the same loads and stores in flight (so the
    // wait for `cur` does not cover the previous step's stores).
    const int64_t items = ((B - t + stride - 1) / stride) * ((nc - cfirst + W::kStep - 1) / W::kStep);
    v4u a[N], b[N];
    load_item(offset(t, cfirst), a);
    step(a, b);
    int64_t k = 1;
    for (; k + 2 <= items; k += 2) {
        step(b, a);
        step(a, b);
    }
    if (k < items) step(b, a);
}

// Sum over the 64 lanes of the wave of each of v[0..15]; every lane receives all sixteen
// sums. Halving exchange: at lane mask m a lane keeps the half of its values selected by
// its bit m and adds its partner's copy of that half, so after masks 32, 16, 8, 4 lane L
// holds value (L >> 2) & 15 summed over the lanes that share its two low bits; two more
// exchanges complete the sums (17 shuffles instead of 96).
// The same exchange for 64 values: after masks 32 .. 1 lane L holds the wave's sum of
// value L (63 shuffles). Each step writes a new array of half the size, so that every value
// stays in a register.
template <int M>
__device__ __forceinline__ void halve_step(const float (&v)[2 * M], float (&h)[M], int lane) {
    const bool hi = (lane & M) != 0;
#pragma unroll
    for (int k = 0; k < M; ++k) {
        const float send = hi ? v[k] : v[k + M];
        const float keep = hi ? v[k + M] : v[k];
        h[k] = keep + __shfl_xor(send, M);
    }
}

__device__ __forceinline__ float wave_sum64_own(const float (&v)[64], int lane) {
    float a[32], b[16], c[8], d[4], e[2], f[1];
    halve_step<32>(v, a, lane);
    halve_step<16>(a, b, lane);
    halve_step<8>(b, c, lane);
    halve_step<4>(c, d, lane);
    halve_step<2>(d, e, lane);
    halve_step<1>(e, f, lane);
    return f[0];
}

__device__ __forceinline__ void wave_sum16(float v[16], int lane, float s[16]) {
#pragma unroll
    for (int step = 0; step < 4; ++step) {
        const int m = 32 >> step, n = 8 >> step;
        const bool hi = (lane & m) != 0;
#pragma unroll
        for (int k = 0; k < n; ++k) {
            const float send = hi ? v[k] : v[k + n];
            const float keep = hi ? v[k + n] : v[k];
            v[k] = keep + __shfl_xor(send, m);
        }
    }
    float r = v[0];
    r += __shfl_xor(r, 1);
    r += __shfl_xor(r, 2);
#pragma unroll
    for (int q = 0; q < 16; ++q) s[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(r), 4 * q));
}

// The same walk; a token's dP is summed over the wave when its last item is done, while
// the next item's loads are in flight. Lanes past the end of a row zero their X words, so
// that the chunk they repeat adds nothing to dP. With several waves per token (n = 8 only,
// all the block's waves on one token at a time) each wave leaves its sums in LDS and the
// block's first wave adds them in wave order, so the result does not depend on timing.
// That takes a barrier per token, which every wave must reach equally often: each wave
// needs at least one item per token, nc >= 64 WPT (the launcher's condition).
template <int DX, int N, int WPT = 1>
__global__ __launch_bounds__(kMixBlock) void mix_bwd_kernel(const float* __restrict__ P,
                                                             const v4u* __restrict__ X,
                                                             const v4u* __restrict__ dY, v4u* __restrict__ dX,
                                                             float* __restrict__ dH, int64_t B, int64_t nc) {
    static_assert(WPT == 1 || (N == 8 && 64 * WPT <= kMixBlock), "several waves per token: n = 8 only");
    using W = MixWalk<WPT>;
    constexpr int E = MixChunk<DX>::E;
    const int lane = threadIdx.x & 63;
    const int64_t stride = W::token_stride();
    const int64_t cfirst = W::first_chunk();
    int64_t t = W::first_token();
    if (t >= B) return;  // uniform over the block when WPT > 1
    // per-wave sums of the token's dP (WPT > 1), two buffers by token parity: a wave writes
    // buffer q for token k + 2 only after the barrier of token k + 1, which the first wave
    // reaches after it has read buffer q for token k
    __shared__ float part[WPT > 1 ? 2 * WPT * 64 : 1];
    int parity = 0;
    constexpr int NN = N * N;
    float p[NN], acc[NN];  // acc: this lane's part of dP_ij = sum_c dY_i[c] X_j[c]
    auto token_matrix = [&](int64_t tt) { load_token_matrix<N>(P, tt, p); };
    // dH of token t from the lanes' partial dP (uniform branch: every lane takes part)
    // (n = 8: dP itself, lane L writing entry L, for the 8 x 8 backward to take over)
    auto finish_token = [&]() {
        if constexpr (N == 4) {
            float G[16], out[16];
            wave_sum16(acc, lane, G);
            implicit_vjp(p, G, out);
            if (lane < 4) {
                const v4f row = lane == 0 ? v4f{out[0], out[1], out[2], out[3]}
                              : lane == 1 ? v4f{out[4], out[5], out[6], out[7]}
                              : lane == 2 ? v4f{out[8], out[9], out[10], out[11]}
                                          : v4f{out[12], out[13], out[14], out[15]};
                reinterpret_cast<v4f*>(dH)[4 * t + lane] = row;
            }
        } else if constexpr (WPT == 1) {
            dH[64 * t + lane] = wave_sum64_own(acc, lane);
        } else {
            float* buf = part + parity * (WPT * 64);
            const int w = W::wave();
            buf[64 * w + lane] = wave_sum64_own(acc, lane);
            // LDS-only fences: the next item's global loads stay in flight across the barrier
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
            if (w == 0) {
                float sum = buf[lane];
#pragma unroll
                for (int q = 1; q < WPT; ++q) sum += buf[64 * q + lane];
                dH[64 * t + lane] = sum;
            }
            parity ^= 1;
        }
#pragma unroll
        for (int q = 0; q < NN; ++q) acc[q] = 0.f;
    };
#pragma unroll
    for (int q = 0; q < NN; ++q) acc[q] = 0.f;
    token_matrix(t);
    if (nc == 0) {  // no channels: dP = 0 (uniform)
        for (;;) {
            finish_token();
            t += stride;
            if (t >= B) return;
            token_matrix(t);
        }
    }
    int64_t c0 = cfirst;
    auto offset = [&](int64_t tt, int64_t cc0) {
        const int64_t cc = cc0 + lane;
        return N * nc * tt + (cc < nc ? cc : nc - 1);
    };
    auto load_item = [&](int64_t off, v4u x[N], v4u g[N]) {
#pragma unroll
        for (int j = 0; j < N; ++j) {
            x[j] = __builtin_nontemporal_load(X + off + j * nc);
            g[j] = __builtin_nontemporal_load(dY + off + j * nc);
        }
    };
    // dX of the item in (xc, gc) and its part of dP
    auto process = [&](const v4u xc[N], const v4u gc[N]) {
        v4u o[N];
        mix_chunk<DX, N, true>(p, gc, o);
        const int64_t off = offset(t, c0);
#pragma unroll
        for (int j = 0; j < N; ++j) __builtin_nontemporal_store(o[j], dX + off + j * nc);
        const bool own = c0 + lane < nc;
        constexpr int EW = E / 4;
#pragma unroll
        for (int w = 0; w < 4; ++w) {  // one 32-bit word of the chunk at a time
            if constexpr (DX == BIRKHOFF4_BF16) {
                // two channels per word: bf16 dot products accumulated in fp32 (the products
                // of two bf16 values are exact in fp32), on the packed words as loaded
                uint32_t xw[N], gw[N];
#pragma unroll
                for (int j = 0; j < N; ++j) {
                    const v4u xj = own ? xc[j] : v4u{0u, 0u, 0u, 0u};
                    xw[j] = w == 0 ? xj.x : w == 1 ? xj.y : w == 2 ? xj.z : xj.w;
                    gw[j] = w == 0 ? gc[j].x : w == 1 ? gc[j].y : w == 2 ? gc[j].z : gc[j].w;
                }
#pragma unroll
                for (int i = 0; i < N; ++i)
#pragma unroll
                    for (int j = 0; j < N; ++j)
                        acc[N * i + j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, gw[i]),
                                                                          __builtin_bit_cast(bf16x2, xw[j]),
                                                                          acc[N * i + j], false);
            } else {
                float xv[N][EW], gv[N][EW];
#pragma unroll
                for (int j = 0; j < N; ++j) {
                    unpack_word<DX>(own ? xc[j] : v4u{0u, 0u, 0u, 0u}, w, xv[j]);
                    unpack_word<DX>(gc[j], w, gv[j]);
                }
#pragma unroll
                for (int i = 0; i < N; ++i)
#pragma unroll
                    for (int j = 0; j < N; ++j)
#pragma unroll
                        for (int e = 0; e < EW; ++e)
                            acc[N * i + j] = __builtin_fmaf(gv[i][e], xv[j][e], acc[N * i + j]);
            }
        }
    };
    const int64_t items = ((B - t + stride - 1) / stride) * ((nc - cfirst + W::kStep - 1) / W::kStep);
    // process the item in (xc, gc) while the next one loads into (xn, gn)
    auto step = [&](const v4u xc[N], const v4u gc[N], v4u xn[N], v4u gn[N]) {
        int64_t tn = t, cn = c0 + W::kStep;
        if (cn >= nc) {
            cn = cfirst;
            tn = t + stride;
        }
        const bool more = tn < B;
        load_item(more ? offset(tn, cn) : offset(t, c0), xn, gn);
        __builtin_amdgcn_sched_barrier(0);
        process(xc, gc);
        if (tn != t) {
            finish_token();
            if (more) token_matrix(tn);
        }
        t = tn;
        c0 = cn;
    };
    // peeled first step and counted loop of two, as in the forward
    v4u xa[N], ga[N], xb[N], gb[N];
    load_item(offset(t, c0), xa, ga);
    step(xa, ga, xb, gb);
    int64_t k = 1;
    for (; k + 2 <= items; k += 2) {
        step(xb, gb, xa, ga);
        step(xa, ga, xb, gb);
    }
    if (k < items) step(xb, gb, xa, ga);
}

// ---------------------------------------------------------------------------
// Sinkhorn-Knopp baseline (eq. sinkhorn_knopp), one problem per lane
// ---------------------------------------------------------------------------
__device__ __forceinline__ void sk_kernel_matrix(const float h[16], float A[16]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float m = __builtin_fmaxf(__builtin_fmaxf(h[4 * i], h[4 * i + 1]),
                                        __builtin_fmaxf(h[4 * i + 2], h[4 * i + 3]));
#pragma unroll
        for (int j = 0; j < 4; ++j) A[4 * i + j] = ex2((h[4 * i + j] - m) * kLog2e);
    }
}

// u = 1 / max(A v, FLT_MIN), v = 1 / max(A^T u, FLT_MIN)
__device__ __forceinline__ void sk_u(const float A[16], const float v[4], float u[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
        u[i] = rcp(__builtin_fmaxf(__builtin_fmaf(A[4 * i], v[0], __builtin_fmaf(A[4 * i + 1], v[1],
                   __builtin_fmaf(A[4 * i + 2], v[2], A[4 * i + 3] * v[3]))), kFltMin));
}
__device__ __forceinline__ void sk_v(const float A[16], const float u[4], float v[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        v[j] = rcp(__builtin_fmaxf(__builtin_fmaf(A[j], u[0], __builtin_fmaf(A[4 + j], u[1],
                   __builtin_fmaf(A[8 + j], u[2], A[12 + j] * u[3]))), kFltMin));
}

template <int DT>
__global__ __launch_bounds__(256) void sk_fwd_kernel(const void* __restrict__ H, float* __restrict__ P,
                                                      int64_t B, int n_steps) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; b < B; b += stride) {
        float h[16], A[16], u[4], v[4] = {1.f, 1.f, 1.f, 1.f};
        load16<DT>(H, b, h);
        sk_kernel_matrix(h, A);
        for (int k = 0; k < n_steps; ++k) {
            sk_u(A, v, u);
            sk_v(A, u, v);
        }
        float out[16];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) out[4 * i + j] = u[i] * A[4 * i + j] * v[j];
        store16(P, b, out);
    }
}

// Adjoints of P = diag(u) A diag(v) for dL/dP = G: A-bar = G o u v^T, u-bar, v-bar.
__device__ __forceinline__ void sk_adjoint_init(const float A[16], const float G[16], const float u[4],
                                                const float v[4], float Ab[16], float ub[4], float vb[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) ub[i] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) vb[j] = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float gg = G[4 * i + j];
            Ab[4 * i + j] = gg * u[i] * v[j];
            ub[i] = __builtin_fmaf(gg * A[4 * i + j], v[j], ub[i]);
            vb[j] = __builtin_fmaf(gg * u[i], A[4 * i + j], vb[j]);
        }
}

// One step back through u^(k) = 1 / max(A v^(k-1), FLT_MIN), v^(k) = 1 / max(A^T u^(k),
// FLT_MIN): u^(k) is recomputed from v^(k-1); on entry vb holds dL/dv^(k) and ub the
// direct part of dL/du^(k) (zero before the last step's), on exit vb holds dL/dv^(k-1),
// ub is cleared and A-bar has gathered both steps' terms. A clamped denominator
// contributes no gradient.
__device__ __forceinline__ void sk_reverse(const float A[16], const float vk[4], const float vp[4], float Ab[16],
                                           float ub[4], float vb[4]) {
    float uk[4];
    sk_u(A, vp, uk);
    float bb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float den = __builtin_fmaf(A[j], uk[0], __builtin_fmaf(A[4 + j], uk[1],
                          __builtin_fmaf(A[8 + j], uk[2], A[12 + j] * uk[3])));
        bb[j] = den >= kFltMin ? -vb[j] * vk[j] * vk[j] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            ub[i] = __builtin_fmaf(A[4 * i + j], bb[j], ub[i]);
            Ab[4 * i + j] = __builtin_fmaf(uk[i], bb[j], Ab[4 * i + j]);
        }
    float ab[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float den = __builtin_fmaf(A[4 * i], vp[0], __builtin_fmaf(A[4 * i + 1], vp[1],
                          __builtin_fmaf(A[4 * i + 2], vp[2], A[4 * i + 3] * vp[3])));
        ab[i] = den >= kFltMin ? -ub[i] * uk[i] * uk[i] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) vb[j] = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            vb[j] = __builtin_fmaf(A[4 * i + j], ab[i], vb[j]);
            Ab[4 * i + j] = __builtin_fmaf(ab[i], vp[j], Ab[4 * i + j]);
        }
#pragma unroll
    for (int i = 0; i < 4; ++i) ub[i] = 0.f;
}

// Reverse mode through the n-step map, any n: the iterates v^(k) are kept in LDS (one
// 64-lane block, [k][component][lane] so that lanes hit distinct banks).
template <int DT, int DG>
__global__ __launch_bounds__(64) void sk_bwd_kernel(const void* __restrict__ H,
                                                     const void* __restrict__ dP,
                                                     float* __restrict__ dH, int64_t B, int n_steps) {
    extern __shared__ float vbuf[];  // [(n_steps + 1) * 4][64]
    const int lane = threadIdx.x;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + lane; b < B; b += stride) {
        float h[16], G[16], A[16], u[4], v[4] = {1.f, 1.f, 1.f, 1.f};
        load16<DT>(H, b, h);
        load16<DG>(dP, b, G);
        sk_kernel_matrix(h, A);
#pragma unroll
        for (int j = 0; j < 4; ++j) vbuf[j * 64 + lane] = 1.f;
        for (int k = 1; k <= n_steps; ++k) {
            sk_u(A, v, u);
            sk_v(A, u, v);
#pragma unroll
            for (int j = 0; j < 4; ++j) vbuf[(4 * k + j) * 64 + lane] = v[j];
        }
        float Ab[16], ub[4], vb[4];
        sk_adjoint_init(A, G, u, v, Ab, ub, vb);
        for (int k = n_steps; k >= 1; --k) {
            float vk[4], vp[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                vk[j] = vbuf[(4 * k + j) * 64 + lane];
                vp[j] = vbuf[(4 * (k - 1) + j) * 64 + lane];
            }
            sk_reverse(A, vk, vp, Ab, ub, vb);
        }
        float out[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) out[q] = Ab[q] * A[q];
        store16(dH, b, out);
    }
}

// The same for a step count fixed at compile time: the iterates stay in VGPRs (the
// loops are unrolled), so occupancy is set by registers, not by the LDS the iterates
// would take. Same arithmetic in the same order as the LDS kernel.
template <int DT, int DG, int NS>
__global__ __launch_bounds__(256, 3) void sk_bwd_reg_kernel(const void* __restrict__ H,
                                                          const void* __restrict__ dP,
                                                          float* __restrict__ dH, int64_t B) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
    for (int64_t b = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; b < B; b += stride) {
        float h[16], G[16], A[16], u[4], vs[NS + 1][4];
        load16<DT>(H, b, h);
        sk_kernel_matrix(h, A);
#pragma unroll
        for (int j = 0; j < 4; ++j) vs[0][j] = 1.f;
#pragma unroll
        for (int k = 1; k <= NS; ++k) {
            sk_u(A, vs[k - 1], u);
            sk_v(A, u, vs[k]);
        }
        load16<DG>(dP, b, G);  // needed from here on only
        float Ab[16], ub[4], vb[4];
        sk_adjoint_init(A, G, u, vs[NS], Ab, ub, vb);
        // Each reverse step recomputes u^(k) from v^(k-1); tying the step's inputs to the
        // adjoint it receives keeps that work in its own step (hoisted ahead, or shared with
        // the forward steps, it would keep ~20 values per step live at once).
#pragma unroll
        for (int k = NS; k >= 1; --k) {
            float vk[4] = {vs[k][0], vs[k][1], vs[k][2], vs[k][3]};
            float vp[4] = {vs[k - 1][0], vs[k - 1][1], vs[k - 1][2], vs[k - 1][3]};
            asm volatile("" : "+v"(vk[0]), "+v"(vk[1]), "+v"(vk[2]), "+v"(vk[3]), "+v"(vp[0]), "+v"(vp[1]),
                              "+v"(vp[2]), "+v"(vp[3]) : "v"(vb[0]), "v"(vb[1]), "v"(vb[2]), "v"(vb[3]));
            sk_reverse(A, vk, vp, Ab, ub, vb);
        }
        float out[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) out[q] = Ab[q] * A[q];
        store16(dH, b, out);
    }
}

// ---------------------------------------------------------------------------
// n = 8 (Sec. 3.1 and eq. grad_hess / eq. derivative with n = m = 8): one problem per
// lane. The forward is the 4 x 4 kernel's iteration written for 7 free potentials (the
// row-softmax state in product form, trial steps capped in spread, Armijo with the
// rounding-noise test, Levenberg-Marquardt shift, re-derivation of flushed entries). A
// wave takes every nwv-th batch of 32 problems (nwv the resident waves of the grid); it
// initialises a batch with all its lanes (two lanes per problem) into an LDS ring, and a
// lane whose problem finishes takes the next one from the ring at once. The Newton system is the column Laplacian with 28 weights,
// grounded at column 8 and solved by subtraction-free elimination of nodes 1..7.
// ---------------------------------------------------------------------------
constexpr int kB8Block = 256;
constexpr int kB8Waves = kB8Block / 64;
constexpr int kB8Ring = 32;  // problems per initialisation batch (= ring slots per wave)
constexpr int kB8Slot = 23;  // v4f per ring slot (22 used; odd, so that slots start in different banks)
constexpr int kB8SlotOT = 27;  // the same with the two marginals (26 used)

// Index of the weight of column pair (j, k), j < k < 8, in a packed array of 28.
__host__ __device__ constexpr int pw8(int j, int k) { return j * 8 - (j * (j + 1)) / 2 + (k - j - 1); }

// Row i (8 values) of problem b of an [B][8][8] array stored as fp32 or bf16.
template <int DT>
__device__ __forceinline__ void load_row8(const void* base, int64_t b, int i, float h[8]) {
    if constexpr (DT == BIRKHOFF4_BF16) {
        const v4u r = reinterpret_cast<const v4u*>(base)[8 * b + i];
        const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            h[2 * k] = __uint_as_float(w[k] << 16);
            h[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
        }
    } else {
        const v4f* p = reinterpret_cast<const v4f*>(base) + 16 * b + 2 * i;
        const v4f r0 = p[0], r1 = p[1];
        h[0] = r0.x; h[1] = r0.y; h[2] = r0.z; h[3] = r0.w;
        h[4] = r1.x; h[5] = r1.y; h[6] = r1.z; h[7] = r1.w;
    }
}

__device__ __forceinline__ float sum8(const float v[8]) {
    return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// Column sum j of T minus one (eq. c_g).
__device__ __forceinline__ float colgrad8(const float T[64], int j) {
    return (((T[j] + T[8 + j]) + (T[16 + j] + T[24 + j])) + ((T[32 + j] + T[40 + j]) + (T[48 + j] + T[56 + j]))) - 1.0f;
}

// W_jk = sum_i T_ij T_ik for the 28 column pairs.
__device__ __forceinline__ void weights8(const float T[64], float W[28]) {
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int k = j + 1; k < 8; ++k) {
            float s = T[j] * T[k];
#pragma unroll
            for (int i = 1; i < 8; ++i) s = __builtin_fmaf(T[8 * i + j], T[8 * i + k], s);
            W[pw8(j, k)] = s;
        }
}

// W_jk = sum_i w_i T_ij T_ik (general marginals, eq. grad_hess: w = a for S, 1/a for T).
__device__ __forceinline__ void weights8w(const float T[64], const float w[8], float W[28]) {
#pragma unroll
    for (int j = 0; j < 7; ++j) {
        float c[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) c[i] = T[8 * i + j] * w[i];
#pragma unroll
        for (int k = j + 1; k < 8; ++k) {
            float s = c[0] * T[k];
#pragma unroll
            for (int i = 1; i < 8; ++i) s = __builtin_fmaf(c[i], T[8 * i + k], s);
            W[pw8(j, k)] = s;
        }
    }
}

// Newton direction in log2 units, d = -log2(e) (Lap(W) + lam I)^{-1} g over nodes 0..6
// (node 7 is the ground; lam acts as a conductance from every node to it). Eliminating
// node p joins nodes j, k by W_jp W_pk / piv_p and moves W_jp q_p / piv_p of its ground
// conductance q_p onto node j, piv_p being node p's remaining conductance: every pivot
// is a sum of non-negative terms. A node without conductance gets d = 0.
__device__ __forceinline__ void newton_solve8(const float W[28], const float g[7], float lam, float d[7]) {
    float A[28], q[7], r[7], ip[7];
#pragma unroll
    for (int k = 0; k < 28; ++k) A[k] = W[k];
#pragma unroll
    for (int j = 0; j < 7; ++j) {
        q[j] = W[pw8(j, 7)] + lam;
        r[j] = -kLog2e * g[j];
    }
#pragma unroll
    for (int p = 0; p < 7; ++p) {
        float piv = q[p];
#pragma unroll
        for (int k = p + 1; k < 7; ++k) piv += A[pw8(p, k)];
        ip[p] = rcp(__builtin_fmaxf(piv, kTiny));
#pragma unroll
        for (int j = p + 1; j < 7; ++j) {
            const float f = A[pw8(p, j)] * ip[p];
#pragma unroll
            for (int k = j + 1; k < 7; ++k) A[pw8(j, k)] = __builtin_fmaf(f, A[pw8(p, k)], A[pw8(j, k)]);
            q[j] = __builtin_fmaf(f, q[p], q[j]);
            r[j] = __builtin_fmaf(f, r[p], r[j]);
        }
    }
#pragma unroll
    for (int p = 6; p >= 0; --p) {
        float s = r[p];
#pragma unroll
        for (int k = p + 1; k < 7; ++k) s = __builtin_fmaf(A[pw8(p, k)], d[k], s);
        d[p] = s * ip[p];
    }
}

// max_j v_j - min_j v_j over the 7 free shifts and v_8 = 0
__device__ __forceinline__ float spread8(const float v[7]) {
    float hi = 0.f, lo = 0.f;
#pragma unroll
    for (int j = 0; j < 7; ++j) {
        hi = __builtin_fmaxf(hi, v[j]);
        lo = __builtin_fminf(lo, v[j]);
    }
    return hi - lo;
}

// Trial evaluation in product form (the 4 x 4 kernel's evaluate for 8 columns): column
// j < 7 of T is multiplied by 2^(s_j), rows are renormalised, l receives the log2 row
// sums and g the column sums minus one.
__device__ __forceinline__ void evaluate8(float T[64], const float s[7], float l[8], float g[8]) {
    float S[7];
#pragma unroll
    for (int j = 0; j < 7; ++j) S[j] = ex2(s[j]);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float e[8];
#pragma unroll
        for (int j = 0; j < 7; ++j) e[j] = T[8 * i + j] * S[j];
        e[7] = T[8 * i + 7];
        const float sum = sum8(e);
        const float r = rcp(sum);
        l[i] = lg2(sum);
#pragma unroll
        for (int j = 0; j < 8; ++j) T[8 * i + j] = e[j] * r;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) g[j] = colgrad8(T, j);
}

template <bool WRITE_DUAL, bool WRITE_ITERS>
__device__ __forceinline__ void store_output8(float* __restrict__ P, float* __restrict__ dual,
                                              int32_t* __restrict__ iters, int64_t b, const float T[64],
                                              const float a[8], const float beta[7], int status) {
    v4f* pp = reinterpret_cast<v4f*>(P) + 16 * b;
#pragma unroll
    for (int q = 0; q < 16; ++q) pp[q] = v4f{T[4 * q], T[4 * q + 1], T[4 * q + 2], T[4 * q + 3]};
    if constexpr (WRITE_DUAL) {
        v4f* dp = reinterpret_cast<v4f*>(dual) + 4 * b;
        dp[0] = v4f{-a[0] * kLn2, -a[1] * kLn2, -a[2] * kLn2, -a[3] * kLn2};
        dp[1] = v4f{-a[4] * kLn2, -a[5] * kLn2, -a[6] * kLn2, -a[7] * kLn2};
        dp[2] = v4f{beta[0] * kLn2, beta[1] * kLn2, beta[2] * kLn2, beta[3] * kLn2};
        dp[3] = v4f{beta[4] * kLn2, beta[5] * kLn2, beta[6] * kLn2, beta[0] * 0.f};  // beta_8 = 0
    }
    if constexpr (WRITE_ITERS) iters[b] = status;
}

// Raw storage words of four rows of an 8 x 8 problem (16 for bf16, 32 for fp32).
template <int DT>
struct RawWords8 {
    static constexpr int n = (DT == BIRKHOFF4_BF16) ? 16 : 32;
};

// Rows 4 hf .. 4 hf + 3 of problem b, undecoded.
template <int DT>
__device__ __forceinline__ void load_half8(const void* base, int64_t b, int hf, uint32_t w[RawWords8<DT>::n]) {
    constexpr int NQ = RawWords8<DT>::n / 4;
    const v4u* p = reinterpret_cast<const v4u*>(base) + NQ * (2 * b + hf);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const v4u r = p[q];
        w[4 * q + 0] = r.x;
        w[4 * q + 1] = r.y;
        w[4 * q + 2] = r.z;
        w[4 * q + 3] = r.w;
    }
}

// Row r (0..3) of the four held in raw words, decoded.
template <int DT>
__device__ __forceinline__ void decode_row8(const uint32_t w[RawWords8<DT>::n], int r, float h[8]) {
    if constexpr (DT == BIRKHOFF4_BF16) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            h[2 * k] = __uint_as_float(w[4 * r + k] << 16);
            h[2 * k + 1] = __uint_as_float(w[4 * r + k] & 0xffff0000u);
        }
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) h[k] = __uint_as_float(w[8 * r + k]);
    }
}

// Sum over the two lanes of a pair (2k, 2k + 1); both receive the same value (the add
// commutes, and contraction is off so that it is not fused into the caller's product).
__device__ __forceinline__ float psum(float x) {
#pragma clang fp contract(off)
    return x + __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, true));
}

// The OT stopping test: |c_j - b_j| <= tol max(1, sum a / 8, b_j) for every column: absolute
// for unit-sized marginals (the Birkhoff test), relative above, where the fp32 resolution of
// the column sums grows with the masses. The last column, whose potential is fixed, also
// absorbs |sum a - sum b|, which marginals given in fp32 cannot make exactly zero.
__device__ __forceinline__ bool ot_within_tol8(const float g[8], const float b[8], float tol, float sa, float sb) {
    const float slack = __builtin_fabsf(sa - sb), ms = __builtin_fmaxf(1.f, 0.125f * sa);
    float x = -1.f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        x = __builtin_fmaxf(x, __builtin_fabsf(g[j]) - tol * __builtin_fmaxf(ms, b[j]) - (j == 7 ? slack : 0.f));
    return x <= 0.f;
}

__device__ __forceinline__ float sum8v(const float v[8]) {
    return ((v[0] + v[1]) + (v[2] + v[3])) + ((v[4] + v[5]) + (v[6] + v[7]));
}

// Output of one 8 x 8 OT problem: T = diag(a) S, dual alpha_i = eta (ln a_i - lse_i), beta_j =
// eta x_j (natural units, beta_8 = 0), and the status word.
template <bool WRITE_DUAL, bool WRITE_ITERS>
__device__ __forceinline__ void store_output8_ot(float* __restrict__ P, float* __restrict__ dual,
                                                 int32_t* __restrict__ iters, int64_t b, const float S[64],
                                                 const float la[8], const float x[7], const float ma[8], float eta,
                                                 int status) {
    v4f* pp = reinterpret_cast<v4f*>(P) + 16 * b;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        const float m = ma[q >> 1];
        pp[q] = v4f{m * S[4 * q], m * S[4 * q + 1], m * S[4 * q + 2], m * S[4 * q + 3]};
    }
    if constexpr (WRITE_DUAL) {
        const float e2 = eta * kLn2;
        v4f* dp = reinterpret_cast<v4f*>(dual) + 4 * b;
        dp[0] = v4f{e2 * (lg2(ma[0]) - la[0]), e2 * (lg2(ma[1]) - la[1]), e2 * (lg2(ma[2]) - la[2]),
                    e2 * (lg2(ma[3]) - la[3])};
        dp[1] = v4f{e2 * (lg2(ma[4]) - la[4]), e2 * (lg2(ma[5]) - la[5]), e2 * (lg2(ma[6]) - la[6]),
                    e2 * (lg2(ma[7]) - la[7])};
        dp[2] = v4f{e2 * x[0], e2 * x[1], e2 * x[2], e2 * x[3]};
        dp[3] = v4f{e2 * x[4], e2 * x[5], e2 * x[6], x[0] * 0.f};
    }
    if constexpr (WRITE_ITERS) iters[b] = status;
}

// With OT the kernel solves general entropic OT (eq. entropic) instead: H is the cost M
// (fp32), av and bv the marginals, eta the regulariser; the state is S = diag(a)^-1 T in
// product form (the 4 x 4 OT kernel's substitution), the gradient sum_i a_i S_ij - b_j, the
// weights sum_i a_i S_ij S_ik and the f change sum_i a_i l_i - sum_j b_j s_j.
template <int DT, bool WRITE_DUAL, bool WRITE_ITERS, bool OT>
__global__ __launch_bounds__(kB8Block, 2) void newton8_fwd_kernel(const void* __restrict__ H, float* __restrict__ P,
                                                                float* __restrict__ dual,
                                                                int32_t* __restrict__ iters, int64_t B, float tol,
                                                                int max_iter,
                                                                const float* __restrict__ av,
                                                                const float* __restrict__ bv, float eta) {
    constexpr int NW = RawWords8<DT>::n;
    constexpr int SLOT = OT ? kB8SlotOT : kB8Slot;
    const float hsc = OT ? -kLog2e / eta : kLog2e;  // log2-unit logits per unit of H (or of M)
    const int lane = threadIdx.x & 63;
    const int hf = lane & 1;  // half of the problem this lane initialises (rows 4 hf .. 4 hf + 3)
    const int pb = lane >> 1;  // its position in an initialisation batch
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    // Per-wave ring: slot p holds the initial point of position p of the last batch: row
    // 4 h + r of T in v4f 4 r + 2 h and 4 r + 2 h + 1 (the two lanes of a pair write
    // different banks), a (16..17), beta_1..4 (18), beta_5..7 and the offset (19), g
    // (20..21), with OT the marginals a (22..23) and b (24..25); order[0 .. nfresh) lists the
    // positions whose problems still need steps. With OT each lane also keeps the marginals of
    // its current problem in LDS (a in v4f 0..1, b in 2..3 of its four).
    __shared__ v4f ring_all[kB8Waves][kB8Ring * SLOT];
    __shared__ int32_t order_all[kB8Waves][kB8Ring];
    __shared__ v4f marg_all[OT ? kB8Waves : 1][OT ? 64 * 4 : 1];
    v4f* const ring = ring_all[wv];
    int32_t* const order = order_all[wv];
    v4f* const marg = marg_all[OT ? wv : 0] + (OT ? 4 * lane : 0);
    // The grid is the resident waves. Wave gw of the grid's nwv takes the batches of kB8Ring
    // problems gw, gw + nwv, gw + 2 nwv, ...: it refills its lanes from one batch after the
    // other without draining in between, and all waves run out of batches together.
    const int64_t gw = static_cast<int64_t>(blockIdx.x) * kB8Waves + wv;
    const int64_t nwv = static_cast<int64_t>(gridDim.x) * kB8Waves;
    if (gw * kB8Ring >= B) return;  // uniform across the wave
    // A problem is named by kB8Ring k + p for position p of the wave's k-th batch.
    auto problem = [&](int32_t id) -> int64_t {
        return (static_cast<int64_t>(id / kB8Ring) * nwv + gw) * kB8Ring + id % kB8Ring;
    };

    // Raw words of the batch to initialise next (two lanes per problem), one batch ahead.
    uint32_t raw[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) raw[q] = 0u;
    int64_t bnext = gw * kB8Ring;  // first problem of that batch (uniform)
    int32_t knext = 0;             // its index in the wave's sequence
    v4f pa = {1.f, 1.f, 1.f, 1.f}, pb0 = pa, pb1 = pa;  // OT: its marginals (this lane's four a_i, all b_j)
    auto prefetch = [&]() {
        if (bnext + pb < B) {
            load_half8<DT>(H, bnext + pb, hf, raw);
            if constexpr (OT) {
                const v4f* a4 = reinterpret_cast<const v4f*>(av) + 2 * (bnext + pb);
                const v4f* b4 = reinterpret_cast<const v4f*>(bv) + 2 * (bnext + pb);
                pa = a4[hf];
                pb0 = b4[0];
                pb1 = b4[1];
            }
        }
    };
    prefetch();
    int nfresh = 0, icur = 0;  // order[icur .. nfresh) not yet taken

    bool active = false;  // holds an unfinished problem
    bool setup = false;   // its Newton system must be formed at the current point
    int32_t rel = 0;      // its name (see problem())
    float T[64], a[8], beta[7], g[8], W[28], ga[7], o[7];
#pragma unroll
    for (int q = 0; q < 64; ++q) T[q] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = g[j] = 0.f;
#pragma unroll
    for (int j = 0; j < 7; ++j) beta[j] = ga[j] = o[j] = 0.f;
#pragma unroll
    for (int k = 0; k < 28; ++k) W[k] = 0.f;
    float lam = 0.f, gn2 = 0.f, t = 1.f, fofs = 0.f, gsum = 0.f;
    // rounding-noise threshold of f and floor of the Levenberg-Marquardt shift (OT: scaled by
    // the problem's mass / 8, so that unit marginals give the Birkhoff values)
    float fnoise = kFNoise, lmfloor = kLMFloor;
    int cnt = 0;  // bits 0-15: trial steps; bits 16-18: log2 of the initial trial step

    // Initialise the loaded batch with the whole wave, two lanes per problem: column means
    // and the finiteness test are combined over the pair, each lane forms the row softmax
    // of its four rows straight into the problem's ring slot, and the column sums are
    // combined again. Problems already within tol there (or non-finite, or max_iter = 0)
    // are written out from the slot; the others are listed for the lanes to take.
    auto init_batch = [&]() {
#pragma unroll
        for (int q = 0; q < NW; ++q) asm volatile("" : "+v"(raw[q])::"memory");
        const int64_t bp = bnext + pb;
        const bool valid = bp < B;
        float cm[8];
        bool fin = true;
        // OT: this lane's four row masses and all eight column masses
        const float ma[4] = {pa.x, pa.y, pa.z, pa.w};
        const float mb[8] = {pb0.x, pb0.y, pb0.z, pb0.w, pb1.x, pb1.y, pb1.z, pb1.w};
        if constexpr (OT) {
#pragma unroll
            for (int r = 0; r < 4; ++r) fin = fin && __builtin_isfinite(ma[r]) && ma[r] > 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) fin = fin && __builtin_isfinite(mb[j]) && mb[j] > 0.f;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) cm[j] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float h[8];
            decode_row8<DT>(raw, r, h);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                fin = fin && __builtin_isfinite(h[j]);
                cm[j] += h[j] * hsc;
            }
        }
        fin = fin && __builtin_amdgcn_mov_dpp(static_cast<int>(fin), 0xB1, 0xF, 0xF, true);
        const float poison = fin ? 0.f : __builtin_nanf("");
#pragma unroll
        for (int j = 0; j < 8; ++j) cm[j] = psum(cm[j]);
        float bi[7];
#pragma unroll
        for (int j = 0; j < 7; ++j) bi[j] = 0.125f * (cm[7] - cm[j]) + poison;
        if constexpr (OT) {  // x_j + log2(b_j / b_8): exact for separable costs
            const float ib7 = rcp(mb[7]);
#pragma unroll
            for (int j = 0; j < 7; ++j) bi[j] += lg2(mb[j] * ib7);
        }
        v4f* const sl = ring + pb * SLOT;
        float ai[4], gi[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) gi[j] = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float u[8];
            decode_row8<DT>(raw, r, u);
#pragma unroll
            for (int j = 0; j < 8; ++j) u[j] = __builtin_fmaf(u[j], hsc, j < 7 ? bi[j] : poison);
            float m = u[0];
#pragma unroll
            for (int j = 1; j < 8; ++j) m = __builtin_fmaxf(m, u[j]);
            m += poison;
#pragma unroll
            for (int j = 0; j < 8; ++j) u[j] = ex2(u[j] - m);
            const float sum = sum8(u);
            const float rc = rcp(sum);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                u[j] *= rc;
                if constexpr (OT)
                    gi[j] = __builtin_fmaf(ma[r], u[j], gi[j]);
                else
                    gi[j] += u[j];
            }
            ai[r] = m + lg2(sum);
            sl[4 * r + 2 * hf] = v4f{u[0], u[1], u[2], u[3]};
            sl[4 * r + 2 * hf + 1] = v4f{u[4], u[5], u[6], u[7]};
        }
        float gmax = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            gi[j] = psum(gi[j]) - (OT ? mb[j] : 1.0f);
            gmax = __builtin_fmaxf(gmax, __builtin_fabsf(gi[j]));
        }
        sl[16 + hf] = v4f{ai[0], ai[1], ai[2], ai[3]};
        if constexpr (OT) {
            sl[22 + hf] = pa;
            sl[24 + hf] = hf ? pb1 : pb0;
        }
        sl[18 + hf] = hf ? v4f{bi[4], bi[5], bi[6], __int_as_float(knext * kB8Ring + pb)}
                         : v4f{bi[0], bi[1], bi[2], bi[3]};
        sl[20 + hf] = hf ? v4f{gi[4], gi[5], gi[6], gi[7]} : v4f{gi[0], gi[1], gi[2], gi[3]};
        bool conv = gmax <= tol;
        if constexpr (OT) {
            const float sa = psum((ma[0] + ma[1]) + (ma[2] + ma[3]));
            const float sb = ((mb[0] + mb[1]) + (mb[2] + mb[3])) + ((mb[4] + mb[5]) + (mb[6] + mb[7]));
            conv = ot_within_tol8(gi, mb, tol, sa, sb);
        }
        const bool done = valid && (!fin || conv || max_iter == 0);
        const bool fresh = valid && !done;
        const uint64_t fm = __ballot(fresh && hf == 0);
        if (fresh && hf == 0) order[__popcll(fm & below)] = pb;
        nfresh = __popcll(fm);
        icur = 0;
        if (done) {
            v4f* pp = reinterpret_cast<v4f*>(P) + 16 * bp + 8 * hf;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const v4f u = sl[4 * (q >> 1) + 2 * hf + (q & 1)];
                pp[q] = OT ? u * ma[q >> 1] : u;
            }
            if constexpr (WRITE_DUAL) {
                v4f* dp = reinterpret_cast<v4f*>(dual) + 4 * bp;
                if constexpr (OT) {
                    const float e2 = eta * kLn2;
                    dp[hf] = v4f{e2 * (lg2(ma[0]) - ai[0]), e2 * (lg2(ma[1]) - ai[1]), e2 * (lg2(ma[2]) - ai[2]),
                                 e2 * (lg2(ma[3]) - ai[3])};
                    dp[2 + hf] = hf ? v4f{bi[4] * e2, bi[5] * e2, bi[6] * e2, bi[0] * 0.f}
                                    : v4f{bi[0] * e2, bi[1] * e2, bi[2] * e2, bi[3] * e2};
                } else {
                    dp[hf] = v4f{-ai[0] * kLn2, -ai[1] * kLn2, -ai[2] * kLn2, -ai[3] * kLn2};
                    dp[2 + hf] = hf ? v4f{bi[4] * kLn2, bi[5] * kLn2, bi[6] * kLn2, bi[0] * 0.f}  // beta_8 = 0
                                    : v4f{bi[0] * kLn2, bi[1] * kLn2, bi[2] * kLn2, bi[3] * kLn2};
                }
            }
            if constexpr (WRITE_ITERS)
                if (hf == 0) iters[bp] = !fin ? BIRKHOFF4_NON_FINITE : (conv ? 0 : BIRKHOFF4_NOT_CONVERGED);
        }
        bnext += nwv * kB8Ring;
        ++knext;
        prefetch();
    };

    // OT: the marginals of this lane's current problem, from its LDS side slot
    auto load_marg = [&](float ma8[8], float mb8[8]) {
        const v4f a0 = marg[0], a1 = marg[1], b0 = marg[2], b1 = marg[3];
        ma8[0] = a0.x; ma8[1] = a0.y; ma8[2] = a0.z; ma8[3] = a0.w;
        ma8[4] = a1.x; ma8[5] = a1.y; ma8[6] = a1.z; ma8[7] = a1.w;
        mb8[0] = b0.x; mb8[1] = b0.y; mb8[2] = b0.z; mb8[3] = b0.w;
        mb8[4] = b1.x; mb8[5] = b1.y; mb8[6] = b1.z; mb8[7] = b1.w;
    };

    for (;;) {
        if (active) {
            float d[7], s[7], l[8];
            newton_solve8(W, ga, lam, d);
            t = __builtin_fminf(t, kCap2 * rcp(__builtin_fmaxf(spread8(d), kTiny)));
#pragma unroll
            for (int j = 0; j < 7; ++j) s[j] = __builtin_fmaf(t, d[j], -o[j]);
            evaluate8(T, s, l, g);
            float ls = 0.f, ss = 0.f;
            bool within = false;  // OT: every column within its tolerance
            if constexpr (OT) {  // gradient sum_i a_i S_ij - b_j, f change sum_i a_i l_i - sum_j b_j s_j
                float ma8[8], mb8[8];
                load_marg(ma8, mb8);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    float c = ma8[0] * T[j];
#pragma unroll
                    for (int i = 1; i < 8; ++i) c = __builtin_fmaf(ma8[i], T[8 * i + j], c);
                    g[j] = c - mb8[j];
                }
                within = ot_within_tol8(g, mb8, tol, sum8v(ma8), sum8v(mb8));
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    a[i] += l[i];
                    ls = __builtin_fmaf(ma8[i], l[i], ls);
                }
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    beta[j] += s[j];
                    o[j] += s[j];
                    ss = __builtin_fmaf(mb8[j], s[j], ss);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    a[i] += l[i];
                    ls += l[i];
                }
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    beta[j] += s[j];
                    o[j] += s[j];
                    ss += s[j];
                }
            }
            const float df = fofs + (ls - ss);
            fofs = df;
            gsum += spread8(s);
            ++cnt;
            float gmax = 0.f, gn2t = 0.f, slope = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                gmax = __builtin_fmaxf(gmax, __builtin_fabsf(g[j]));
                gn2t = __builtin_fmaf(g[j], g[j], gn2t);
            }
#pragma unroll
            for (int j = 0; j < 7; ++j) slope = __builtin_fmaf(ga[j], d[j], slope);
            const bool accept = (df <= kArmijo * t * slope) || (__builtin_fabsf(df) < fnoise && gn2t < gn2);
            const int evals = cnt & 0xffff;
            const bool conv = accept && (OT ? within : gmax <= tol);
            if (!conv && evals < max_iter) {
                if (gsum >= kReviveBits) {
                    gsum = 0.f;
                    float tmin = T[0];
#pragma unroll
                    for (int q = 1; q < 64; ++q) tmin = __builtin_fminf(tmin, T[q]);
                    if (tmin == 0.f) {
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            float h[8];
                            load_row8<DT>(H, problem(rel), i, h);
#pragma unroll
                            for (int j = 0; j < 8; ++j)
                                if (T[8 * i + j] == 0.f)
                                    T[8 * i + j] = ex2(__builtin_fmaf(h[j], hsc, j < 7 ? beta[j] : 0.f) - a[i]);
                        }
                    }
                }
                if (accept) {
                    float dd = 0.f;
#pragma unroll
                    for (int j = 0; j < 7; ++j) dd = __builtin_fmaf(g[j], d[j], dd);
                    const int ts = cnt >> 16;
                    const bool grow = t >= 0.999f * __builtin_ldexpf(1.f, ts) && dd < 0.25f * slope;
                    cnt = evals | ((grow ? (ts < kMaxExpandLog2 ? ts + 1 : ts) : 0) << 16);
                    fofs = 0.f;
#pragma unroll
                    for (int j = 0; j < 7; ++j) o[j] = 0.f;
                    t = __builtin_ldexpf(1.f, cnt >> 16);
                    setup = true;
                } else {
                    t *= 0.5f;
                    cnt = evals;
                    lam = __builtin_fminf(16.f * lam, kMaxShift);
                }
            } else {
                if (!accept) {  // max_iter reached on a rejected trial: back to the accepted point
                    float back[7];
#pragma unroll
                    for (int j = 0; j < 7; ++j) back[j] = -o[j];
                    evaluate8(T, back, l, g);
#pragma unroll
                    for (int i = 0; i < 8; ++i) a[i] += l[i];
#pragma unroll
                    for (int j = 0; j < 7; ++j) beta[j] -= o[j];
                }
                if constexpr (OT) {
                    float ma8[8], mb8[8];
                    load_marg(ma8, mb8);
                    store_output8_ot<WRITE_DUAL, WRITE_ITERS>(P, dual, iters, problem(rel), T, a, beta, ma8, eta,
                                                              conv ? evals : BIRKHOFF4_NOT_CONVERGED);
                } else {
                    store_output8<WRITE_DUAL, WRITE_ITERS>(P, dual, iters, problem(rel), T, a, beta,
                                                           conv ? evals : BIRKHOFF4_NOT_CONVERGED);
                }
                active = false;
            }
        }
        // Hand-off: every idle lane takes the next listed problem of the ring; batches are
        // initialised as the list runs out.
        uint64_t wm = __ballot(!active);
        while (wm != 0) {
            const int k = __popcll(wm);
            const int rank = __popcll(wm & below);
            const int avail = nfresh - icur;
            if (!active && rank < avail) {
                const v4f* sl = ring + order[icur + rank] * SLOT;
#pragma unroll
                for (int q = 0; q < 16; ++q) {  // v4f q holds half (q & 1) of row 4 ((q >> 1) & 1) + (q >> 2)
                    const v4f r = sl[q];
                    const int e = 8 * (4 * ((q >> 1) & 1) + (q >> 2)) + 4 * (q & 1);
                    T[e] = r.x; T[e + 1] = r.y; T[e + 2] = r.z; T[e + 3] = r.w;
                }
                const v4f a0 = sl[16], a1 = sl[17], b0 = sl[18], b1 = sl[19], g0 = sl[20], g1 = sl[21];
                a[0] = a0.x; a[1] = a0.y; a[2] = a0.z; a[3] = a0.w;
                a[4] = a1.x; a[5] = a1.y; a[6] = a1.z; a[7] = a1.w;
                beta[0] = b0.x; beta[1] = b0.y; beta[2] = b0.z; beta[3] = b0.w;
                beta[4] = b1.x; beta[5] = b1.y; beta[6] = b1.z;
                rel = __float_as_int(b1.w);
                g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w;
                g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
                if constexpr (OT) {
                    const v4f m0 = sl[22], m1 = sl[23], m2 = sl[24], m3 = sl[25];
                    marg[0] = m0;
                    marg[1] = m1;
                    marg[2] = m2;
                    marg[3] = m3;
                    const float mass = ((m0.x + m0.y) + (m0.z + m0.w)) + ((m1.x + m1.y) + (m1.z + m1.w));
                    fnoise = kFNoise * 0.125f * mass;
                    lmfloor = kLMFloor * 0.125f * mass;
                }
#pragma unroll
                for (int j = 0; j < 7; ++j) o[j] = 0.f;
                t = 1.f;
                fofs = gsum = 0.f;
                cnt = 0;
                active = true;
                setup = true;
            }
            if (k <= avail) {
                icur += k;
                break;
            }
            icur = nfresh;
            if (bnext >= B) break;  // nothing left to initialise
            init_batch();
            wm = __ballot(!active);
        }
        // Newton system at the new accepted point, for lanes that accepted a trial and
        // lanes that took a fresh problem alike.
        if (setup) {
            if constexpr (OT) {
                float ma8[8], mb8[8];
                load_marg(ma8, mb8);
                weights8w(T, ma8, W);
            } else {
                weights8(T, W);
            }
            float gmax = 0.f, s2 = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                gmax = __builtin_fmaxf(gmax, __builtin_fabsf(g[j]));
                s2 = __builtin_fmaf(g[j], g[j], s2);
            }
#pragma unroll
            for (int j = 0; j < 7; ++j) ga[j] = g[j];
            gn2 = s2;
            lam = __builtin_fmaxf(kLM * gmax, lmfloor);
            setup = false;
        }
        if (__ballot(active) == 0) break;
    }
}

// Backward for n = 8 (eq. derivative, a = b = 1, eta = 1), the flow form of the 4 x 4
// kernel: W_jk = sum_i T_ij T_ik and antisymmetric flows F_jk = sum_i T_ij T_ik
// (G_ij - G_ik); eliminating node p adds W_jp W_pk / piv to edge (j, k) and
// (W_pk F_jp + W_jp F_pk) / piv to its flow, piv = sum_{k > p} W_pk (ground = node 8);
// back-substitution gives the potentials w (w_8 = 0), and dH_ij = T_ij (psi_ij -
// sum_k T_ik psi_ik) with psi = G - 1 w^T. Products are formed ratio-first so that a
// term underflows only when its value does. Memory traffic is coalesced: a wave moves
// the 64 problems of a chunk between HBM and an LDS tile (one problem per 17 x 16 bytes,
// so that lanes reading their own problem hit distinct banks) with whole-wave
// non-temporal accesses, and each lane works on its own problem from the tile.
constexpr int kB8Stride = 17;  // v4f per problem in the LDS tile

// With OT it is the backward of 8 x 8 entropic OT (eq. derivative): P is the solution T, av
// the row marginal, dP = dL/dT (fp32) and dH = dL/dM; weights and flows carry 1/a_i, and
// dM_ij = -T_ij (psi_ij - sum_k T_ik psi_ik / a_i) / eta.
// IN_PLACE: dP and dH are the same memory (the 8-stream mixing backward forms dP in dH's
// buffer); they are then not declared non-aliasing. Each wave reads a chunk's dP whole into
// LDS before it writes that chunk's dH, so the in-place update is safe.
template <bool IN_PLACE, typename T>
using MaybeRestrict = std::conditional_t<IN_PLACE, T*, T* __restrict__>;

template <int DT, bool OT, bool IN_PLACE = false>
__global__ __launch_bounds__(kB8Block, 2) void implicit8_bwd_kernel(const float* __restrict__ P,
                                                                     MaybeRestrict<IN_PLACE, const void> dP,
                                                                     MaybeRestrict<IN_PLACE, float> dH, int64_t B,
                                                                     const float* __restrict__ av, float eta) {
    __shared__ v4f tile_all[kB8Waves][64 * kB8Stride];
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    v4f* const tile = tile_all[wv];
    v4u* const tileu = reinterpret_cast<v4u*>(tile);
    const v4f* P4 = reinterpret_cast<const v4f*>(P);
    const v4u* G4 = reinterpret_cast<const v4u*>(dP);
    v4f* dH4 = reinterpret_cast<v4f*>(dH);
    constexpr int GP = (DT == BIRKHOFF4_BF16) ? 8 : 16;  // 16-byte pieces of dP per problem
    const int64_t nchunk = (B + 63) / 64;
    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kB8Waves + wv; c < nchunk;
         c += static_cast<int64_t>(gridDim.x) * kB8Waves) {
        const int64_t base = c * 64;
        const int n = (B - base < 64) ? static_cast<int>(B - base) : 64;  // problems in this chunk
        // P: 16 pieces per problem, piece k of the chunk goes to problem k / 16, slot k % 16
        {
            v4f pc[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int k = 64 * q + lane;
                pc[q] = k < 16 * n ? __builtin_nontemporal_load(P4 + 16 * base + k) : v4f{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const int k = 64 * q + lane;
                tile[(k >> 4) * kB8Stride + (k & 15)] = pc[q];
            }
        }
        __builtin_amdgcn_wave_barrier();
        float T[64];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const v4f t = tile[lane * kB8Stride + r];
            T[4 * r] = t.x; T[4 * r + 1] = t.y; T[4 * r + 2] = t.z; T[4 * r + 3] = t.w;
        }
        __builtin_amdgcn_wave_barrier();
        // dP: GP pieces per problem, kept in the tile (read twice below)
        {
            v4u gc[GP];
#pragma unroll
            for (int q = 0; q < GP; ++q) {
                const int k = 64 * q + lane;
                gc[q] = k < GP * n ? __builtin_nontemporal_load(G4 + GP * base + k) : v4u{0u, 0u, 0u, 0u};
            }
#pragma unroll
            for (int q = 0; q < GP; ++q) {
                const int k = 64 * q + lane;
                tileu[(k / GP) * kB8Stride + (k % GP)] = gc[q];
            }
        }
        __builtin_amdgcn_wave_barrier();
        // row i of this lane's G from the tile
        auto grow = [&](int i, float G[8]) {
            if constexpr (DT == BIRKHOFF4_BF16) {
                const v4u r = tileu[lane * kB8Stride + i];
                const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    G[2 * k] = __uint_as_float(w[k] << 16);
                    G[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
                }
            } else {
                const v4f r0 = tile[lane * kB8Stride + 2 * i], r1 = tile[lane * kB8Stride + 2 * i + 1];
                G[0] = r0.x; G[1] = r0.y; G[2] = r0.z; G[3] = r0.w;
                G[4] = r1.x; G[5] = r1.y; G[6] = r1.z; G[7] = r1.w;
            }
        };
        float W[28], F[28], w[8], ip[7], ia[8];
        if constexpr (OT) {
            const v4f* a4 = reinterpret_cast<const v4f*>(av) + 2 * (base + lane);
            const v4f A0 = lane < n ? a4[0] : v4f{1.f, 1.f, 1.f, 1.f};
            const v4f A1 = lane < n ? a4[1] : v4f{1.f, 1.f, 1.f, 1.f};
            ia[0] = rcp(A0.x); ia[1] = rcp(A0.y); ia[2] = rcp(A0.z); ia[3] = rcp(A0.w);
            ia[4] = rcp(A1.x); ia[5] = rcp(A1.y); ia[6] = rcp(A1.z); ia[7] = rcp(A1.w);
            weights8w(T, ia, W);
        } else {
            weights8(T, W);
        }
#pragma unroll
        for (int k = 0; k < 28; ++k) F[k] = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float G[8];
            grow(i, G);
#pragma unroll
            for (int j = 0; j < 8; ++j)
#pragma unroll
                for (int k = j + 1; k < 8; ++k) {
                    const float q = OT ? T[8 * i + j] * (T[8 * i + k] * ia[i]) : T[8 * i + j] * T[8 * i + k];
                    F[pw8(j, k)] = __builtin_fmaf(q, G[j] - G[k], F[pw8(j, k)]);
                }
        }
#pragma unroll
        for (int p = 0; p < 7; ++p) {
            float piv = 0.f;
#pragma unroll
            for (int k = p + 1; k < 8; ++k) piv += W[pw8(p, k)];
            ip[p] = (piv > kPivMin) ? rcp(piv) : 0.f;
#pragma unroll
            for (int j = p + 1; j < 8; ++j)
#pragma unroll
                for (int k = j + 1; k < 8; ++k) {
                    const float fj = W[pw8(p, j)] * ip[p], fk = W[pw8(p, k)] * ip[p];
                    // F_jp = -F_pj, F_pk as stored (p < j < k)
                    F[pw8(j, k)] = __builtin_fmaf(fj, F[pw8(p, k)], __builtin_fmaf(-fk, F[pw8(p, j)], F[pw8(j, k)]));
                    W[pw8(j, k)] = __builtin_fmaf(fj, W[pw8(p, k)], W[pw8(j, k)]);
                }
        }
        w[7] = 0.f;
#pragma unroll
        for (int p = 6; p >= 0; --p) {
            float s = 0.f;
#pragma unroll
            for (int k = p + 1; k < 8; ++k) s += __builtin_fmaf(W[pw8(p, k)], w[k], F[pw8(p, k)]);
            w[p] = s * ip[p];
        }
        // dH row i replaces tile slots 2i, 2i+1 of this lane's problem; going down from the
        // last row, those slots hold only dP rows already read (bf16 rows are 16 bytes)
#pragma unroll
        for (int i = 7; i >= 0; --i) {
            float G[8], psi[8];
            grow(i, G);
            float mu = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                psi[j] = G[j] - w[j];
                mu = __builtin_fmaf(T[8 * i + j], psi[j], mu);
            }
            float o[8];
            if constexpr (OT) {
                mu *= ia[i];
                const float nie = -1.f / eta;
#pragma unroll
                for (int j = 0; j < 8; ++j) o[j] = T[8 * i + j] * (psi[j] - mu) * nie;
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) o[j] = T[8 * i + j] * (psi[j] - mu);
            }
            tile[lane * kB8Stride + 2 * i] = v4f{o[0], o[1], o[2], o[3]};
            tile[lane * kB8Stride + 2 * i + 1] = v4f{o[4], o[5], o[6], o[7]};
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int k = 64 * q + lane;
            const v4f o = tile[(k >> 4) * kB8Stride + (k & 15)];
            if (k < 16 * n) __builtin_nontemporal_store(o, dH4 + 16 * base + k);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// General entropic OT for 4 x 4 (eq. entropic): cost M, marginals a > 0 and b > 0 with
// equal sums, regulariser eta > 0. With h = -M / eta (log2 units: h log2(e)) and x = beta /
// eta, T_ij = a_i S_ij where S is the row softmax of h + 1 x^T; the reduced dual over
// x_{-4} has gradient c - b with c = T^T 1, and Hessian the Laplacian of the column graph
// with weights W_jk = sum_i a_i S_ij S_ik = sum_i T_ij T_ik / a_i (eq. grad_hess), so the
// Birkhoff iteration carries over with the row masses and column targets: the same
// product-form trials (S updated in place), spread cap, Armijo test on
// f = sum_i a_i lse_i - sum_j b_j x_j, Levenberg-Marquardt shift and re-derivation of
// flushed entries. One problem per lane; each wave owns a range of problems, initialises
// them 64 at a time with all its lanes into an LDS ring, and a lane whose problem finishes
// takes the next one from the ring at once.
// ---------------------------------------------------------------------------
constexpr int kOtBlock = 256;
constexpr int kOtWaves = kOtBlock / 64;
constexpr int kOtSlot = 8;  // v4f per ring slot
#ifndef OT_RANGES
#define OT_RANGES 16384
#endif
constexpr int64_t kOtRanges = OT_RANGES;  // wave ranges per launch

__device__ __forceinline__ v4f load4(const float* base, int64_t b) { return reinterpret_cast<const v4f*>(base)[b]; }

// Initial point: x_j = mean_i h_i4 - mean_i h_ij + log2(b_j / b_4) (exact for separable
// h), S the row softmax of h + 1 x^T, la the log2 row normalisers. Returns false for a
// NaN, infinite or non-positive input (S, la, x are then NaN).
__device__ __forceinline__ bool ot_init(const float* M, const float* av, const float* bv, int64_t p, float rsc,
                                        float S[16], float la[4], float x[3], float a[4], float bb[4]) {
    float h[16];
    load16_f32(M, p, h);
    const v4f A = load4(av, p), Bm = load4(bv, p);
    a[0] = A.x; a[1] = A.y; a[2] = A.z; a[3] = A.w;
    bb[0] = Bm.x; bb[1] = Bm.y; bb[2] = Bm.z; bb[3] = Bm.w;
    bool ok = true;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        ok = ok && __builtin_isfinite(h[q]);
        h[q] *= rsc;  // -log2(e) / eta
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) ok = ok && __builtin_isfinite(a[k]) && a[k] > 0.f && __builtin_isfinite(bb[k]) && bb[k] > 0.f;
    const float poison = ok ? 0.f : __builtin_nanf("");
    float cm[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) cm[j] = 0.25f * ((h[j] + h[4 + j]) + (h[8 + j] + h[12 + j]));
#pragma unroll
    for (int j = 0; j < 3; ++j) x[j] = (cm[3] - cm[j]) + lg2(bb[j] * rcp(bb[3])) + poison;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float u[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) u[j] = h[4 * i + j] + (j < 3 ? x[j] : poison);
        const float m = __builtin_fmaxf(__builtin_fmaxf(u[0], u[1]), __builtin_fmaxf(u[2], u[3])) + poison;
        float e[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) e[j] = ex2(u[j] - m);
        const float sum = (e[0] + e[1]) + (e[2] + e[3]);
        const float r = rcp(sum);
#pragma unroll
        for (int j = 0; j < 4; ++j) S[4 * i + j] = e[j] * r;
        la[i] = m + lg2(sum);
    }
    return ok;
}

// The OT stopping test: |c_j - b_j| <= tol max(1, sum a / 4, b_j) for every column: absolute
// for unit-sized marginals (the Birkhoff test), relative above, where the fp32 resolution of
// the column sums grows with the masses. The last column, whose potential is fixed, also
// absorbs |sum a - sum b|, which marginals given in fp32 cannot make exactly zero.
__device__ __forceinline__ bool ot_within_tol4(const float g[4], const float a[4], const float b[4], float tol) {
    const float sa = (a[0] + a[1]) + (a[2] + a[3]);
    const float slack = __builtin_fabsf(sa - ((b[0] + b[1]) + (b[2] + b[3]))), ms = __builtin_fmaxf(1.f, 0.25f * sa);
    float x = -1.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
        x = __builtin_fmaxf(x, __builtin_fabsf(g[j]) - tol * __builtin_fmaxf(ms, b[j]) - (j == 3 ? slack : 0.f));
    return x <= 0.f;
}

// c_j - b_j with c = sum_i a_i S_ij
__device__ __forceinline__ void ot_grad(const float S[16], const float a[4], const float bb[4], float g[4]) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
        g[j] = (__builtin_fmaf(a[0], S[j], a[1] * S[4 + j]) + __builtin_fmaf(a[2], S[8 + j], a[3] * S[12 + j])) - bb[j];
}

__device__ __forceinline__ Weights ot_weights(const float S[16], const float a[4]) {
    Weights W = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float t0 = a[i] * S[4 * i], t1 = S[4 * i + 1], t2 = S[4 * i + 2], t3 = S[4 * i + 3];
        const float t1a = a[i] * t1, t2a = a[i] * t2;
        W.w01 = __builtin_fmaf(t0, t1, W.w01);
        W.w02 = __builtin_fmaf(t0, t2, W.w02);
        W.w03 = __builtin_fmaf(t0, t3, W.w03);
        W.w12 = __builtin_fmaf(t1a, t2, W.w12);
        W.w13 = __builtin_fmaf(t1a, t3, W.w13);
        W.w23 = __builtin_fmaf(t2a, t3, W.w23);
    }
    return W;
}

template <bool WRITE_DUAL, bool WRITE_ITERS>
__device__ __forceinline__ void ot_store(float* __restrict__ T, float* __restrict__ dual, int32_t* __restrict__ iters,
                                         int64_t p, const float S[16], const float la[4], const float x[3],
                                         const float a[4], float eta, int status) {
    v4f* tp = reinterpret_cast<v4f*>(T) + 4 * p;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        tp[i] = v4f{a[i] * S[4 * i], a[i] * S[4 * i + 1], a[i] * S[4 * i + 2], a[i] * S[4 * i + 3]};
    if constexpr (WRITE_DUAL) {
        // alpha_i = eta (ln a_i - lse_i), beta_j = eta x_j (natural units; beta_4 = 0)
        const float e2 = eta * kLn2;
        v4f* dp = reinterpret_cast<v4f*>(dual) + 2 * p;
        dp[0] = v4f{e2 * (lg2(a[0]) - la[0]), e2 * (lg2(a[1]) - la[1]), e2 * (lg2(a[2]) - la[2]),
                    e2 * (lg2(a[3]) - la[3])};
        dp[1] = v4f{e2 * x[0], e2 * x[1], e2 * x[2], x[0] * 0.f};
    }
    if constexpr (WRITE_ITERS) iters[p] = status;
}

template <bool WRITE_DUAL, bool WRITE_ITERS>
__global__ __launch_bounds__(kOtBlock) void ot4_fwd_kernel(const float* __restrict__ M, const float* __restrict__ av,
                                                          const float* __restrict__ bv, float eta,
                                                          float* __restrict__ T, float* __restrict__ dual,
                                                          int32_t* __restrict__ iters, int64_t B, float tol,
                                                          int max_iter, int64_t per_wave) {
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    // Per-wave ring of 64 slots: S rows (v4f 0..3), la (4), x and the problem's offset (5),
    // a (6), b (7) of a problem not finished at its initial point.
    __shared__ v4f ring_all[kOtWaves][64 * kOtSlot];
    v4f* const ring = ring_all[wv];
    const int64_t r0 = (static_cast<int64_t>(blockIdx.x) * kOtWaves + wv) * per_wave;
    if (r0 >= B) return;  // uniform across the wave
    const int64_t r1 = (r0 + per_wave < B) ? r0 + per_wave : B;
    int64_t bnext = r0;        // first problem of the next batch to initialise (uniform)
    int nfresh = 0, icur = 0;  // ring slots [icur, nfresh) not yet taken
    const float rsc = -kLog2e / eta;

    bool active = false;  // holds an unfinished problem
    bool setup = false;   // its Newton system must be formed at the current point
    int32_t rel = 0;      // problem offset from r0
    float S[16], la[4], x[3], a[4], bb[4], g[4], ga[3], o[3];
#pragma unroll
    for (int q = 0; q < 16; ++q) S[q] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) la[j] = a[j] = bb[j] = g[j] = 0.f;
#pragma unroll
    for (int j = 0; j < 3; ++j) x[j] = ga[j] = o[j] = 0.f;
    Weights W = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float lam = 0.f, gn2 = 0.f, t = 1.f, fofs = 0.f, gsum = 0.f, fnoise = 0.f, lmfloor = 0.f;
    int cnt = 0;

    // Initialise the next 64 problems with the whole wave (one per lane). Those already
    // within tol (or invalid, or max_iter = 0) are written out; the others are compacted
    // into ring slots 0 .. nfresh - 1.
    auto init_batch = [&]() {
        const int64_t p = bnext + lane;
        const bool valid = p < r1;
        float Si[16], lai[4], xi[3], ai[4], bi[4], gi[4];
#pragma unroll
        for (int q = 0; q < 16; ++q) Si[q] = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) lai[j] = ai[j] = bi[j] = 0.f;
#pragma unroll
        for (int j = 0; j < 3; ++j) xi[j] = 0.f;
        bool ok = false;
        if (valid) ok = ot_init(M, av, bv, p, rsc, Si, lai, xi, ai, bi);
        ot_grad(Si, ai, bi, gi);
        const bool within = ot_within_tol4(gi, ai, bi, tol);
        const bool done = valid && (!ok || within || max_iter == 0);
        const bool fresh = valid && !done;
        const uint64_t fm = __ballot(fresh);
        if (fresh) {
            v4f* sl = ring + __popcll(fm & below) * kOtSlot;
            sl[0] = v4f{Si[0], Si[1], Si[2], Si[3]};
            sl[1] = v4f{Si[4], Si[5], Si[6], Si[7]};
            sl[2] = v4f{Si[8], Si[9], Si[10], Si[11]};
            sl[3] = v4f{Si[12], Si[13], Si[14], Si[15]};
            sl[4] = v4f{lai[0], lai[1], lai[2], lai[3]};
            sl[5] = v4f{xi[0], xi[1], xi[2], __int_as_float(static_cast<int32_t>(p - r0))};
            sl[6] = v4f{ai[0], ai[1], ai[2], ai[3]};
            sl[7] = v4f{bi[0], bi[1], bi[2], bi[3]};
        }
        if (done)
            ot_store<WRITE_DUAL, WRITE_ITERS>(T, dual, iters, p, Si, lai, xi, ai, eta,
                                              !ok ? BIRKHOFF4_NON_FINITE : (within ? 0 : BIRKHOFF4_NOT_CONVERGED));
        nfresh = __popcll(fm);
        icur = 0;
        bnext += 64;
    };

    for (;;) {
        if (active) {
            float d0, d1, d2;
            newton_solve(W, ga[0], ga[1], ga[2], lam, d0, d1, d2);
            t = __builtin_fminf(t, kCap2 * rcp(__builtin_fmaxf(spread(d0, d1, d2), kTiny)));
            const float s0 = __builtin_fmaf(t, d0, -o[0]), s1 = __builtin_fmaf(t, d1, -o[1]),
                        s2 = __builtin_fmaf(t, d2, -o[2]);
            float l[4], gu[4];
            evaluate(S, s0, s1, s2, l, gu);  // S renormalised; gu unused (unit-mass sums)
            ot_grad(S, a, bb, g);
#pragma unroll
            for (int i = 0; i < 4; ++i) la[i] += l[i];
            x[0] += s0; x[1] += s1; x[2] += s2;
            o[0] += s0; o[1] += s1; o[2] += s2;
            const float df = fofs + (__builtin_fmaf(a[0], l[0], a[1] * l[1]) + __builtin_fmaf(a[2], l[2], a[3] * l[3])) -
                             __builtin_fmaf(bb[0], s0, __builtin_fmaf(bb[1], s1, bb[2] * s2));
            fofs = df;
            gsum += spread(s0, s1, s2);
            ++cnt;
            const float gn2t = g[0] * g[0] + g[1] * g[1] + g[2] * g[2] + g[3] * g[3];
            const float slope = ga[0] * d0 + ga[1] * d1 + ga[2] * d2;
            const bool accept = (df <= kArmijo * t * slope) || (__builtin_fabsf(df) < fnoise && gn2t < gn2);
            const int evals = cnt & 0xffff;
            const bool conv = accept && ot_within_tol4(g, a, bb, tol);
            if (!conv && evals < max_iter) {
                if (gsum >= kReviveBits) {
                    gsum = 0.f;
                    float smin = S[0];
#pragma unroll
                    for (int q = 1; q < 16; ++q) smin = __builtin_fminf(smin, S[q]);
                    if (smin == 0.f) {
                        float h[16];
                        load16_f32(M, r0 + rel, h);
#pragma unroll
                        for (int i = 0; i < 4; ++i)
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                if (S[4 * i + j] == 0.f)
                                    S[4 * i + j] = ex2(__builtin_fmaf(h[4 * i + j], rsc, j < 3 ? x[j] : 0.f) - la[i]);
                    }
                }
                if (accept) {
                    const float dd = g[0] * d0 + g[1] * d1 + g[2] * d2;
                    const int ts = cnt >> 16;
                    const bool grow = t >= 0.999f * __builtin_ldexpf(1.f, ts) && dd < 0.25f * slope;
                    cnt = evals | ((grow ? (ts < kMaxExpandLog2 ? ts + 1 : ts) : 0) << 16);
                    fofs = 0.f;
                    o[0] = o[1] = o[2] = 0.f;
                    t = __builtin_ldexpf(1.f, cnt >> 16);
                    setup = true;
                } else {
                    t *= 0.5f;
                    cnt = evals;
                    lam = __builtin_fminf(16.f * lam, kMaxShift);
                }
            } else {
                if (!accept) {  // max_iter reached on a rejected trial: back to the accepted point
                    float l2[4], gu2[4];
                    evaluate(S, -o[0], -o[1], -o[2], l2, gu2);
#pragma unroll
                    for (int i = 0; i < 4; ++i) la[i] += l2[i];
                    x[0] -= o[0]; x[1] -= o[1]; x[2] -= o[2];
                }
                ot_store<WRITE_DUAL, WRITE_ITERS>(T, dual, iters, r0 + rel, S, la, x, a, eta,
                                                  conv ? evals : BIRKHOFF4_NOT_CONVERGED);
                active = false;
            }
        }
        // Hand-off: every idle lane takes the next problem of the ring; batches are
        // initialised as the ring runs out.
        uint64_t wm = __ballot(!active);
        while (wm != 0) {
            const int k = __popcll(wm);
            const int rank = __popcll(wm & below);
            const int avail = nfresh - icur;
            if (!active && rank < avail) {
                const v4f* sl = ring + (icur + rank) * kOtSlot;
                const v4f q0 = sl[0], q1 = sl[1], q2 = sl[2], q3 = sl[3], lv = sl[4], xv = sl[5], av4 = sl[6],
                          bv4 = sl[7];
                S[0] = q0.x; S[1] = q0.y; S[2] = q0.z; S[3] = q0.w;
                S[4] = q1.x; S[5] = q1.y; S[6] = q1.z; S[7] = q1.w;
                S[8] = q2.x; S[9] = q2.y; S[10] = q2.z; S[11] = q2.w;
                S[12] = q3.x; S[13] = q3.y; S[14] = q3.z; S[15] = q3.w;
                la[0] = lv.x; la[1] = lv.y; la[2] = lv.z; la[3] = lv.w;
                x[0] = xv.x; x[1] = xv.y; x[2] = xv.z;
                rel = __float_as_int(xv.w);
                a[0] = av4.x; a[1] = av4.y; a[2] = av4.z; a[3] = av4.w;
                bb[0] = bv4.x; bb[1] = bv4.y; bb[2] = bv4.z; bb[3] = bv4.w;
                ot_grad(S, a, bb, g);
                const float mass = (a[0] + a[1]) + (a[2] + a[3]);
                fnoise = kFNoise * mass;
                lmfloor = kLMFloor * 0.25f * mass;
                o[0] = o[1] = o[2] = 0.f;
                t = 1.f;
                fofs = gsum = 0.f;
                cnt = 0;
                active = true;
                setup = true;
            }
            if (k <= avail) {
                icur += k;
                break;
            }
            icur = nfresh;
            if (bnext >= r1) break;  // nothing left to initialise
            init_batch();
            wm = __ballot(!active);
        }
        // Newton system at the new accepted point, for lanes that accepted a trial and
        // lanes that took a fresh problem alike.
        if (setup) {
            W = ot_weights(S, a);
            const float gmax = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(g[0]), __builtin_fabsf(g[1])),
                                               __builtin_fmaxf(__builtin_fabsf(g[2]), __builtin_fabsf(g[3])));
            gn2 = g[0] * g[0] + g[1] * g[1] + g[2] * g[2] + g[3] * g[3];
            ga[0] = g[0]; ga[1] = g[1]; ga[2] = g[2];
            lam = __builtin_fmaxf(kLM * gmax, lmfloor);
            setup = false;
        }
        if (__ballot(active) == 0) break;
    }
}

// Backward of the OT solution (eq. derivative): with W_jk = sum_i T_ij T_ik / a_i and
// flows F_jk = sum_i T_ij T_ik (G_ij - G_ik) / a_i the potentials w solve the grounded
// Laplacian system by the edge-flow elimination of the Birkhoff backward, and
// dL/dM_ij = -T_ij (psi_ij - sum_k T_ik psi_ik / a_i) / eta with psi = G - 1 w^T.
// dL/dM for one problem from its solution t, the marginal a and dL/dT = G.
__device__ __forceinline__ void ot_vjp(const float t[16], const float G[16], const v4f A, float ie, float out[16]) {
    const float ia[4] = {rcp(A.x), rcp(A.y), rcp(A.z), rcp(A.w)};
    float W[4][4], F[4][4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int k = j + 1; k < 4; ++k) {
            float sw = 0.f, sf = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float q = t[4 * i + j] * (t[4 * i + k] * ia[i]);
                sw += q;
                sf = __builtin_fmaf(q, G[4 * i + j] - G[4 * i + k], sf);
            }
            W[j][k] = W[k][j] = sw;
            F[j][k] = sf;
            F[k][j] = -sf;
        }
    float ip[3], w[4];
#pragma unroll
    for (int pn = 0; pn < 3; ++pn) {
        float piv = 0.f;
#pragma unroll
        for (int k = pn + 1; k < 4; ++k) piv += W[pn][k];
        ip[pn] = (piv > kPivMin) ? rcp(piv) : 0.f;
#pragma unroll
        for (int j = pn + 1; j < 4; ++j)
#pragma unroll
            for (int k = j + 1; k < 4; ++k) {
                const float fj = W[j][pn] * ip[pn], fk = W[pn][k] * ip[pn];
                const float Fn = __builtin_fmaf(fk, F[j][pn], __builtin_fmaf(fj, F[pn][k], F[j][k]));
                const float Wn = __builtin_fmaf(fj, W[pn][k], W[j][k]);
                W[j][k] = W[k][j] = Wn;
                F[j][k] = Fn;
                F[k][j] = -Fn;
            }
    }
    w[3] = 0.f;
#pragma unroll
    for (int pn = 2; pn >= 0; --pn) {
        float s = 0.f;
#pragma unroll
        for (int k = pn + 1; k < 4; ++k) s += __builtin_fmaf(W[pn][k], w[k], F[pn][k]);
        w[pn] = s * ip[pn];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        float psi[4], mu = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            psi[j] = G[4 * i + j] - w[j];
            mu = __builtin_fmaf(t[4 * i + j], psi[j], mu);
        }
        mu *= ia[i];
#pragma unroll
        for (int j = 0; j < 4; ++j) out[4 * i + j] = -t[4 * i + j] * (psi[j] - mu) * ie;
    }
}

// One 64-problem chunk per wave; T, dT and dM move between HBM and registers in
// wave-contiguous 16-byte pieces transposed through a per-wave LDS buffer (the 4 x 4
// backward's memory path), a as one 16-byte piece per lane.
__global__ __launch_bounds__(kOtBlock) void ot4_bwd_kernel(const float* __restrict__ T, const float* __restrict__ av,
                                                          const float* __restrict__ dT, float eta,
                                                          float* __restrict__ dM, int64_t B) {
    __shared__ v4f buf_all[kOtWaves][64 * kBwdStride];
    const int lane = threadIdx.x & 63;
    const int wv = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    v4f* const buf = buf_all[wv];
    const v4f* T4 = reinterpret_cast<const v4f*>(T);
    const v4f* G4 = reinterpret_cast<const v4f*>(dT);
    const v4f* A4 = reinterpret_cast<const v4f*>(av);
    v4f* dM4 = reinterpret_cast<v4f*>(dM);
    const float ie = 1.f / eta;
    const int cpos = (lane >> 2) * kBwdStride + (lane & 3);
    const int64_t nchunk = (B + 63) / 64;
    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kOtWaves + wv; c < nchunk;
         c += static_cast<int64_t>(gridDim.x) * kOtWaves) {
        const int64_t base = c * 64;
        const int n = (B - base < 64) ? static_cast<int>(B - base) : 64;
        v4f tc[4], gc[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = 64 * q + lane;
            tc[q] = k < 4 * n ? __builtin_nontemporal_load(T4 + 4 * base + k) : v4f{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = 64 * q + lane;
            gc[q] = k < 4 * n ? __builtin_nontemporal_load(G4 + 4 * base + k) : v4f{0.f, 0.f, 0.f, 0.f};
        }
        const v4f A = lane < n ? __builtin_nontemporal_load(A4 + base + lane) : v4f{1.f, 1.f, 1.f, 1.f};
        float t[16], G[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) buf[16 * q * kBwdStride + cpos] = tc[q];
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const v4f u = buf[lane * kBwdStride + r];
            t[4 * r + 0] = u.x; t[4 * r + 1] = u.y; t[4 * r + 2] = u.z; t[4 * r + 3] = u.w;
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < 4; ++q) buf[16 * q * kBwdStride + cpos] = gc[q];
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const v4f u = buf[lane * kBwdStride + r];
            G[4 * r + 0] = u.x; G[4 * r + 1] = u.y; G[4 * r + 2] = u.z; G[4 * r + 3] = u.w;
        }
        __builtin_amdgcn_wave_barrier();
        float out[16];
        ot_vjp(t, G, A, ie, out);
#pragma unroll
        for (int r = 0; r < 4; ++r)
            buf[lane * kBwdStride + r] = v4f{out[4 * r], out[4 * r + 1], out[4 * r + 2], out[4 * r + 3]};
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int k = 64 * q + lane;
            const v4f o = buf[16 * q * kBwdStride + cpos];
            if (k < 4 * n) __builtin_nontemporal_store(o, dM4 + 4 * base + k);
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
constexpr int kMaxDevices = 64;
int g_cus[kMaxDevices];  // cached compute-unit counts (0 = not queried yet)

// Compute units of the device that `stream` belongs to (the null stream: the current device).
int device_cus(hipStream_t stream, int* cus, int* dev_out = nullptr) {
    hipDevice_t dev = 0;
    if (hipStreamGetDevice(stream, &dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return BIRKHOFF4_ERR_DEVICE;
    if (g_cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            return BIRKHOFF4_ERR_DEVICE;
        g_cus[dev] = n;
    }
    *cus = g_cus[dev];
    if (dev_out) *dev_out = dev;
    return BIRKHOFF4_OK;
}

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    if (!a || !b || na == 0 || nb == 0) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

size_t dtype_bytes(int dt) { return dt == BIRKHOFF4_BF16 ? 2 : 4; }
bool dtype_ok(int dt) { return dt == BIRKHOFF4_F32 || dt == BIRKHOFF4_BF16; }

// Status of the launches made by this thread since the last call: taken from each launch's
// own return value, so an error left pending by someone else's earlier launch is neither
// reported as ours nor cleared.
thread_local int t_launch = BIRKHOFF4_OK;

template <typename... KArgs, typename... Args>
void launch_kernel(void (*kern)(KArgs...), dim3 grid, dim3 block, unsigned lds, hipStream_t stream, Args... args) {
    static_assert(sizeof...(KArgs) == sizeof...(Args), "kernel argument count");
    std::tuple<KArgs...> vals(args...);
    void* ptrs[sizeof...(KArgs)];
    std::apply([&](auto&... v) {
        int k = 0;
        ((ptrs[k++] = static_cast<void*>(&v)), ...);
    }, vals);
    if (hipLaunchKernel(reinterpret_cast<const void*>(kern), grid, block, ptrs, lds, stream) != hipSuccess &&
        t_launch == BIRKHOFF4_OK)
        t_launch = BIRKHOFF4_ERR_LAUNCH;
}

int launch_status() {
    const int r = t_launch;
    t_launch = BIRKHOFF4_OK;
    return r;
}

// Blocks of the forward kernel resident at once on one CU (VGPR-limited),
// from the occupancy calculator; queried once per instantiation.
template <int DT, bool WD, bool WI, bool WH>
int fwd_blocks_per_cu(int dev) {
    static int cached[kMaxDevices];
    if (cached[dev] == 0) {
        int nb = 0, cur = 0;
        // the occupancy calculator answers for the current device
        if (hipGetDevice(&cur) != hipSuccess || cur != dev ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, newton_fwd_kernel<DT, WD, WI, WH>, kFwdBlock, 0) !=
                hipSuccess || nb <= 0)
            nb = 1;
        cached[dev] = nb;
    }
    return cached[dev];
}

// Launch one resident workgroup per CU (as many as the occupancy calculator allows),
// each owning a contiguous range of whole 64-problem batches that its waves share.
template <int DT, bool WD, bool WI, bool WH = false>
int launch_fwd(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol,
               int max_iter, hipStream_t stream, int cus, int dev, float* hess = nullptr) {
    const int64_t batches = (B + 63) / 64;
    int64_t blocks = static_cast<int64_t>(cus) * fwd_blocks_per_cu<DT, WD, WI, WH>(dev);
    if (blocks > batches) blocks = batches;
    const int64_t chunk = ((batches + blocks - 1) / blocks) * 64;
    if (chunk > INT32_MAX / 2) return BIRKHOFF4_ERR_SIZE;  // problems are 32-bit offsets in a range
    blocks = (B + chunk - 1) / chunk;
    launch_kernel((newton_fwd_kernel<DT, WD, WI, WH>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kFwdBlock), 0, stream, H, P, dual, iters, hess, B, chunk, tol, max_iter);
    return launch_status();
}

// Four lanes per problem, one problem per quad, 64 problems per 256-thread block.
template <int DT, bool WD, bool WI>
int launch_fwd_quad(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol,
                    int max_iter, hipStream_t stream) {
    const int64_t blocks = (B + 63) / 64;
    if (blocks > INT32_MAX) return BIRKHOFF4_ERR_SIZE;
    launch_kernel((newton_fwd_quad_kernel<DT, WD, WI>), dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                       stream, H, P, dual, iters, B, tol, max_iter);
    return launch_status();
}

template <int DT>
int dispatch_fwd_quad(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol,
                      int max_iter, hipStream_t stream) {
    if (dual && iters) return launch_fwd_quad<DT, true, true>(H, P, dual, iters, B, tol, max_iter, stream);
    if (dual) return launch_fwd_quad<DT, true, false>(H, P, dual, iters, B, tol, max_iter, stream);
    if (iters) return launch_fwd_quad<DT, false, true>(H, P, dual, iters, B, tol, max_iter, stream);
    return launch_fwd_quad<DT, false, false>(H, P, dual, iters, B, tol, max_iter, stream);
}

template <int DT>
int dispatch_fwd(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol,
                 int max_iter, hipStream_t stream, int cus, int dev) {
    if (dual && iters) return launch_fwd<DT, true, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
    if (dual) return launch_fwd<DT, true, false>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
    if (iters) return launch_fwd<DT, false, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
    return launch_fwd<DT, false, false>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
}

template <int DT>
int dispatch_fwd_hess(const void* H, float* P, float* dual, int32_t* iters, float* hess, int64_t B, float tol,
                      int max_iter, hipStream_t stream, int cus, int dev) {
    if (dual && iters) return launch_fwd<DT, true, true, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev, hess);
    if (dual) return launch_fwd<DT, true, false, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev, hess);
    if (iters) return launch_fwd<DT, false, true, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev, hess);
    return launch_fwd<DT, false, false, true>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev, hess);
}

// Blocks of the n = 8 forward resident at once on one CU, from the occupancy calculator;
// queried once per instantiation and device.
template <int DT, bool WD, bool WI, bool OT>
int fwd8_blocks_per_cu(int dev) {
    static int cached[kMaxDevices];
    if (cached[dev] == 0) {
        int nb = 0, cur = 0;
        if (hipGetDevice(&cur) != hipSuccess || cur != dev ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, newton8_fwd_kernel<DT, WD, WI, OT>, kB8Block, 0) !=
                hipSuccess || nb <= 0)
            nb = 1;
        cached[dev] = nb;
    }
    return cached[dev];
}

// n = 8: the grid is the resident waves (fewer for small B), each taking every nwv-th batch.
template <int DT, bool WD, bool WI, bool OT = false>
int launch_fwd8(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol, int max_iter,
                hipStream_t stream, const float* a = nullptr, const float* b = nullptr, float eta = 1.f) {
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    const int64_t batches = (B + kB8Ring - 1) / kB8Ring;
    int64_t grid = static_cast<int64_t>(cus) * fwd8_blocks_per_cu<DT, WD, WI, OT>(dev);
    const int64_t needed = (batches + kB8Waves - 1) / kB8Waves;
    if (grid > needed) grid = needed;
    // a problem is named in 32 bits by its wave's batch count and its position in the batch
    const int64_t per_wave = (batches + grid * kB8Waves - 1) / (grid * kB8Waves);
    if (per_wave > INT32_MAX / kB8Ring) return BIRKHOFF4_ERR_SIZE;
    launch_kernel((newton8_fwd_kernel<DT, WD, WI, OT>), dim3(static_cast<unsigned>(grid)), dim3(kB8Block), 0,
                  stream, H, P, dual, iters, B, tol, max_iter, a, b, eta);
    return launch_status();
}

template <int DT>
int dispatch_fwd8(const void* H, float* P, float* dual, int32_t* iters, int64_t B, float tol, int max_iter,
                  hipStream_t stream) {
    if (dual && iters) return launch_fwd8<DT, true, true>(H, P, dual, iters, B, tol, max_iter, stream);
    if (dual) return launch_fwd8<DT, true, false>(H, P, dual, iters, B, tol, max_iter, stream);
    if (iters) return launch_fwd8<DT, false, true>(H, P, dual, iters, B, tol, max_iter, stream);
    return launch_fwd8<DT, false, false>(H, P, dual, iters, B, tol, max_iter, stream);
}

int dispatch_ot8_fwd(const float* M, const float* a, const float* b, float eta, float* T, float* dual,
                     int32_t* iters, int64_t B, float tol, int max_iter, hipStream_t stream) {
    constexpr int F = BIRKHOFF4_F32;
    if (dual && iters) return launch_fwd8<F, true, true, true>(M, T, dual, iters, B, tol, max_iter, stream, a, b, eta);
    if (dual) return launch_fwd8<F, true, false, true>(M, T, dual, iters, B, tol, max_iter, stream, a, b, eta);
    if (iters) return launch_fwd8<F, false, true, true>(M, T, dual, iters, B, tol, max_iter, stream, a, b, eta);
    return launch_fwd8<F, false, false, true>(M, T, dual, iters, B, tol, max_iter, stream, a, b, eta);
}

// General OT: one range of problems per wave, blocks scheduled by the hardware (its problems
// take few trials and its ranges are small, so the strided batches of the n = 8 forward do
// not pay here).
template <bool WD, bool WI>
int launch_ot_fwd(const float* M, const float* a, const float* b, float eta, float* T, float* dual, int32_t* iters,
                  int64_t B, float tol, int max_iter, hipStream_t stream) {
    const int64_t waves_min = (B + kMaxGrid * kOtWaves - 1) / (kMaxGrid * kOtWaves);
    int64_t per_wave = (B + kOtRanges - 1) / kOtRanges;
    if (per_wave < 64) per_wave = 64;
    if (per_wave < waves_min) per_wave = waves_min;
    const int64_t waves = (B + per_wave - 1) / per_wave;
    const int64_t grid = (waves + kOtWaves - 1) / kOtWaves;
    launch_kernel((ot4_fwd_kernel<WD, WI>), dim3(static_cast<unsigned>(grid)), dim3(kOtBlock), 0, stream, M, a,
                       b, eta, T, dual, iters, B, tol, max_iter, per_wave);
    return launch_status();
}

int64_t grid_for(int64_t B, int block, int cus, int per_cu) {
    int64_t blocks = (B + block - 1) / block;
    const int64_t cap = static_cast<int64_t>(cus) * per_cu;
    return blocks < cap ? blocks : cap;
}

// Residual mixing, grid-stride over the tokens: one token per wave at a time for n = 4, and
// for n = 8 one token per block of kMix8Wpt waves once every row has at least one chunk per
// wave, nc >= 64 kMix8Wpt, which the backward's per-token barrier needs. Both layouts size
// the grid for the same number of waves per CU.
template <int N>
bool mix_block_per_token(int64_t nc) {
    return N == 8 && nc >= 64 * kMix8Wpt;
}

struct MixLaunch {
    int64_t grid;
    unsigned threads;
};

template <int N>
MixLaunch mix_launch(int64_t B, int64_t nc, int cus) {
    if (mix_block_per_token<N>(nc))
        return {grid_for(B, 1, cus, kMixPerCu * kMixWaves / kMix8Wpt), MixWalk<kMix8Wpt>::kBlockThreads};
    return {grid_for(B, kMixWaves, cus, kMixPerCu), kMixBlock};
}

template <int DX, int N = 4>
int launch_mix_fwd(const float* P, const void* X, void* Y, int64_t B, int64_t nc, hipStream_t stream, int cus) {
    const MixLaunch l = mix_launch<N>(B, nc, cus);
    auto kern = mix_block_per_token<N>(nc) ? mix_fwd_kernel<DX, N, N == 8 ? kMix8Wpt : 1> : mix_fwd_kernel<DX, N, 1>;
    launch_kernel(kern, dim3(static_cast<unsigned>(l.grid)), dim3(l.threads), 0, stream, P,
                  static_cast<const v4u*>(X), static_cast<v4u*>(Y), B, nc);
    return launch_status();
}

template <int DX, int N = 4>
int launch_mix_bwd(const float* P, const void* X, const void* dY, void* dX, float* dH, int64_t B, int64_t nc,
                   hipStream_t stream, int cus) {
    const MixLaunch l = mix_launch<N>(B, nc, cus);
    auto kern = mix_block_per_token<N>(nc) ? mix_bwd_kernel<DX, N, N == 8 ? kMix8Wpt : 1> : mix_bwd_kernel<DX, N, 1>;
    launch_kernel(kern, dim3(static_cast<unsigned>(l.grid)), dim3(l.threads), 0, stream, P,
                  static_cast<const v4u*>(X), static_cast<const v4u*>(dY), static_cast<v4u*>(dX), dH, B, nc);
    return launch_status();
}

}  // namespace

extern "C" {

int birkhoff4_fwd_ex2(const void* H, int h_dtype, float* P, float* dual, int32_t* iters, int64_t B,
                      float tol, int max_iter, int variant, hipStream_t stream) {
    if (variant < BIRKHOFF4_AUTO || variant > BIRKHOFF4_LATENCY) return BIRKHOFF4_ERR_VARIANT;
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(P) || misaligned(dual) || misaligned(iters)) return BIRKHOFF4_ERR_ALIGN;
    const size_t nh = static_cast<size_t>(B) * 16 * dtype_bytes(h_dtype);
    const size_t np = static_cast<size_t>(B) * 64, nd = dual ? static_cast<size_t>(B) * 32 : 0,
                 ni = iters ? static_cast<size_t>(B) * 4 : 0;
    if (overlaps(H, nh, P, np) || overlaps(H, nh, dual, nd) || overlaps(H, nh, iters, ni) ||
        overlaps(P, np, dual, nd) || overlaps(P, np, iters, ni) || overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    if (variant == BIRKHOFF4_LATENCY || (variant == BIRKHOFF4_AUTO && B <= kLatencyMaxB)) {
        if (h_dtype == BIRKHOFF4_BF16)
            return dispatch_fwd_quad<BIRKHOFF4_BF16>(H, P, dual, iters, B, tol, max_iter, stream);
        return dispatch_fwd_quad<BIRKHOFF4_F32>(H, P, dual, iters, B, tol, max_iter, stream);
    }
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    if (h_dtype == BIRKHOFF4_BF16)
        return dispatch_fwd<BIRKHOFF4_BF16>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
    return dispatch_fwd<BIRKHOFF4_F32>(H, P, dual, iters, B, tol, max_iter, stream, cus, dev);
}

int birkhoff4_fwd_hess(const void* H, int h_dtype, float* P, float* dual, float* hess, int32_t* iters,
                       int64_t B, float tol, int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P || !hess) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(P) || misaligned(dual) || misaligned(hess) || misaligned(iters))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t nh = static_cast<size_t>(B) * 16 * dtype_bytes(h_dtype);
    const size_t np = static_cast<size_t>(B) * 64, nd = dual ? static_cast<size_t>(B) * 32 : 0,
                 nw = static_cast<size_t>(B) * 32, ni = iters ? static_cast<size_t>(B) * 4 : 0;
    if (overlaps(H, nh, P, np) || overlaps(H, nh, dual, nd) || overlaps(H, nh, iters, ni) ||
        overlaps(H, nh, hess, nw) || overlaps(P, np, dual, nd) || overlaps(P, np, iters, ni) ||
        overlaps(P, np, hess, nw) || overlaps(dual, nd, iters, ni) || overlaps(dual, nd, hess, nw) ||
        overlaps(hess, nw, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    if (h_dtype == BIRKHOFF4_BF16)
        return dispatch_fwd_hess<BIRKHOFF4_BF16>(H, P, dual, iters, hess, B, tol, max_iter, stream, cus, dev);
    return dispatch_fwd_hess<BIRKHOFF4_F32>(H, P, dual, iters, hess, B, tol, max_iter, stream, cus, dev);
}

int birkhoff4_fwd_ex(const void* H, int h_dtype, float* P, float* dual, int32_t* iters, int64_t B,
                     float tol, int max_iter, hipStream_t stream) {
    return birkhoff4_fwd_ex2(H, h_dtype, P, dual, iters, B, tol, max_iter, BIRKHOFF4_AUTO, stream);
}

int birkhoff4_fwd(const float* H, float* P, float* dual, int64_t B, float tol, int max_iter,
                  hipStream_t stream) {
    return birkhoff4_fwd_ex2(H, BIRKHOFF4_F32, P, dual, nullptr, B, tol, max_iter, BIRKHOFF4_AUTO, stream);
}

int birkhoff4_ot_fwd(const float* M, const float* a, const float* b, float eta, float* T, float* dual,
                     int32_t* iters, int64_t B, float tol, int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!(eta > 0.f) || !(eta <= 3.0e38f)) return BIRKHOFF4_ERR_ETA;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!M || !a || !b || !T) return BIRKHOFF4_ERR_NULL;
    if (misaligned(M) || misaligned(a) || misaligned(b) || misaligned(T) || misaligned(dual) || misaligned(iters))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t nm = static_cast<size_t>(B) * 64, nv = static_cast<size_t>(B) * 16,
                 nd = dual ? static_cast<size_t>(B) * 32 : 0, ni = iters ? static_cast<size_t>(B) * 4 : 0;
    const void* ins[3] = {M, a, b};
    const size_t nins[3] = {nm, nv, nv};
    for (int k = 0; k < 3; ++k)
        if (overlaps(ins[k], nins[k], T, nm) || overlaps(ins[k], nins[k], dual, nd) ||
            overlaps(ins[k], nins[k], iters, ni))
            return BIRKHOFF4_ERR_OVERLAP;
    if (overlaps(T, nm, dual, nd) || overlaps(T, nm, iters, ni) || overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    if (dual && iters) return launch_ot_fwd<true, true>(M, a, b, eta, T, dual, iters, B, tol, max_iter, stream);
    if (dual) return launch_ot_fwd<true, false>(M, a, b, eta, T, dual, iters, B, tol, max_iter, stream);
    if (iters) return launch_ot_fwd<false, true>(M, a, b, eta, T, dual, iters, B, tol, max_iter, stream);
    return launch_ot_fwd<false, false>(M, a, b, eta, T, dual, iters, B, tol, max_iter, stream);
}

int birkhoff4_ot_bwd(const float* T, const float* a, const float* dT, float eta, float* dM, int64_t B,
                     hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!(eta > 0.f) || !(eta <= 3.0e38f)) return BIRKHOFF4_ERR_ETA;
    if (B == 0) return BIRKHOFF4_OK;
    if (!T || !a || !dT || !dM) return BIRKHOFF4_ERR_NULL;
    if (misaligned(T) || misaligned(a) || misaligned(dT) || misaligned(dM)) return BIRKHOFF4_ERR_ALIGN;
    const size_t nm = static_cast<size_t>(B) * 64, nv = static_cast<size_t>(B) * 16;
    if (overlaps(dM, nm, T, nm) || overlaps(dM, nm, dT, nm) || overlaps(dM, nm, a, nv)) return BIRKHOFF4_ERR_OVERLAP;
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kOtWaves - 1) / kOtWaves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    launch_kernel(ot4_bwd_kernel, dim3(static_cast<unsigned>(grid)), dim3(kOtBlock), 0, stream, T, a, dT, eta,
                       dM, B);
    return launch_status();
}

int birkhoff8_ot_fwd(const float* M, const float* a, const float* b, float eta, float* T, float* dual,
                     int32_t* iters, int64_t B, float tol, int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!(eta > 0.f) || !(eta <= 3.0e38f)) return BIRKHOFF4_ERR_ETA;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!M || !a || !b || !T) return BIRKHOFF4_ERR_NULL;
    if (misaligned(M) || misaligned(a) || misaligned(b) || misaligned(T) || misaligned(dual) || misaligned(iters))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t nm = static_cast<size_t>(B) * 256, nv = static_cast<size_t>(B) * 32,
                 nd = dual ? static_cast<size_t>(B) * 64 : 0, ni = iters ? static_cast<size_t>(B) * 4 : 0;
    const void* ins[3] = {M, a, b};
    const size_t nins[3] = {nm, nv, nv};
    for (int k = 0; k < 3; ++k)
        if (overlaps(ins[k], nins[k], T, nm) || overlaps(ins[k], nins[k], dual, nd) ||
            overlaps(ins[k], nins[k], iters, ni))
            return BIRKHOFF4_ERR_OVERLAP;
    if (overlaps(T, nm, dual, nd) || overlaps(T, nm, iters, ni) || overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    return dispatch_ot8_fwd(M, a, b, eta, T, dual, iters, B, tol, max_iter, stream);
}

int birkhoff8_ot_bwd(const float* T, const float* a, const float* dT, float eta, float* dM, int64_t B,
                     hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!(eta > 0.f) || !(eta <= 3.0e38f)) return BIRKHOFF4_ERR_ETA;
    if (B == 0) return BIRKHOFF4_OK;
    if (!T || !a || !dT || !dM) return BIRKHOFF4_ERR_NULL;
    if (misaligned(T) || misaligned(a) || misaligned(dT) || misaligned(dM)) return BIRKHOFF4_ERR_ALIGN;
    const size_t nm = static_cast<size_t>(B) * 256, nv = static_cast<size_t>(B) * 32;
    if (overlaps(dM, nm, T, nm) || overlaps(dM, nm, dT, nm) || overlaps(dM, nm, a, nv)) return BIRKHOFF4_ERR_OVERLAP;
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kB8Waves - 1) / kB8Waves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    launch_kernel((implicit8_bwd_kernel<BIRKHOFF4_F32, true>), dim3(static_cast<unsigned>(grid)),
                       dim3(kB8Block), 0, stream, T, dT, dM, B, a, eta);
    return launch_status();
}

int birkhoff8_fwd(const void* H, int h_dtype, float* P, float* dual, int32_t* iters, int64_t B, float tol,
                  int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(P) || misaligned(dual) || misaligned(iters)) return BIRKHOFF4_ERR_ALIGN;
    const size_t nh = static_cast<size_t>(B) * 64 * dtype_bytes(h_dtype);
    const size_t np = static_cast<size_t>(B) * 256, nd = dual ? static_cast<size_t>(B) * 64 : 0,
                 ni = iters ? static_cast<size_t>(B) * 4 : 0;
    if (overlaps(H, nh, P, np) || overlaps(H, nh, dual, nd) || overlaps(H, nh, iters, ni) ||
        overlaps(P, np, dual, nd) || overlaps(P, np, iters, ni) || overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    if (h_dtype == BIRKHOFF4_BF16) return dispatch_fwd8<BIRKHOFF4_BF16>(H, P, dual, iters, B, tol, max_iter, stream);
    return dispatch_fwd8<BIRKHOFF4_F32>(H, P, dual, iters, B, tol, max_iter, stream);
}

int birkhoff8_bwd(const float* P, const void* dP, int dp_dtype, float* dH, int64_t B, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(dp_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (B == 0) return BIRKHOFF4_OK;
    if (!P || !dP || !dH) return BIRKHOFF4_ERR_NULL;
    if (misaligned(P) || misaligned(dP) || misaligned(dH)) return BIRKHOFF4_ERR_ALIGN;
    const size_t n = static_cast<size_t>(B) * 256, ng = static_cast<size_t>(B) * 64 * dtype_bytes(dp_dtype);
    if (overlaps(dH, n, P, n) || overlaps(dH, n, dP, ng)) return BIRKHOFF4_ERR_OVERLAP;
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kB8Waves - 1) / kB8Waves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    if (dp_dtype == BIRKHOFF4_BF16)
        launch_kernel((implicit8_bwd_kernel<BIRKHOFF4_BF16, false>), dim3(static_cast<unsigned>(grid)),
                           dim3(kB8Block), 0, stream, P, dP, dH, B, nullptr, 1.f);
    else
        launch_kernel((implicit8_bwd_kernel<BIRKHOFF4_F32, false>), dim3(static_cast<unsigned>(grid)),
                           dim3(kB8Block), 0, stream, P, dP, dH, B, nullptr, 1.f);
    return launch_status();
}

int birkhoff4_bwd_ex(const float* P, const void* dP, int dp_dtype, float* dH, int64_t B,
                     hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(dp_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (B == 0) return BIRKHOFF4_OK;
    if (!P || !dP || !dH) return BIRKHOFF4_ERR_NULL;
    if (misaligned(P) || misaligned(dP) || misaligned(dH)) return BIRKHOFF4_ERR_ALIGN;
    const size_t n = static_cast<size_t>(B) * 64, ng = static_cast<size_t>(B) * 16 * dtype_bytes(dp_dtype);
    if (overlaps(dH, n, P, n) || overlaps(dH, n, dP, ng)) return BIRKHOFF4_ERR_OVERLAP;
    // One 64-problem chunk per wave; batches beyond kMaxGrid blocks loop.
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kBwdWaves - 1) / kBwdWaves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    if (dp_dtype == BIRKHOFF4_BF16)
        launch_kernel(implicit_bwd_kernel<BIRKHOFF4_BF16>, dim3(static_cast<unsigned>(grid)), dim3(kBwdBlock),
                           0, stream, P, dP, dH, B, nullptr);
    else
        launch_kernel(implicit_bwd_kernel<BIRKHOFF4_F32>, dim3(static_cast<unsigned>(grid)), dim3(kBwdBlock),
                           0, stream, P, dP, dH, B, nullptr);
    return launch_status();
}

int birkhoff4_bwd_hess(const float* P, const float* hess, const void* dP, int dp_dtype, float* dH, int64_t B,
                       hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(dp_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (B == 0) return BIRKHOFF4_OK;
    if (!P || !hess || !dP || !dH) return BIRKHOFF4_ERR_NULL;
    if (misaligned(P) || misaligned(hess) || misaligned(dP) || misaligned(dH)) return BIRKHOFF4_ERR_ALIGN;
    const size_t n = static_cast<size_t>(B) * 64, ng = static_cast<size_t>(B) * 16 * dtype_bytes(dp_dtype),
                 nw = static_cast<size_t>(B) * 32;
    if (overlaps(dH, n, P, n) || overlaps(dH, n, dP, ng) || overlaps(dH, n, hess, nw)) return BIRKHOFF4_ERR_OVERLAP;
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kBwdWaves - 1) / kBwdWaves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    if (dp_dtype == BIRKHOFF4_BF16)
        launch_kernel((implicit_bwd_kernel<BIRKHOFF4_BF16, true>), dim3(static_cast<unsigned>(grid)),
                           dim3(kBwdBlock), 0, stream, P, dP, dH, B, hess);
    else
        launch_kernel((implicit_bwd_kernel<BIRKHOFF4_F32, true>), dim3(static_cast<unsigned>(grid)),
                           dim3(kBwdBlock), 0, stream, P, dP, dH, B, hess);
    return launch_status();
}

int birkhoff4_bwd(const float* P, const float* dual, const float* dP, float* dH, int64_t B,
                  hipStream_t stream) {
    (void)dual;  // the 4x4 backward needs only T* and G (Sec. 4.2)
    return birkhoff4_bwd_ex(P, dP, BIRKHOFF4_F32, dH, B, stream);
}

int birkhoff4_sk_fwd(const void* H, int h_dtype, float* P, int64_t B, int n_steps, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (n_steps < 1 || n_steps > kMaxSkSteps) return BIRKHOFF4_ERR_STEPS;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(P)) return BIRKHOFF4_ERR_ALIGN;
    if (overlaps(H, static_cast<size_t>(B) * 16 * dtype_bytes(h_dtype), P, static_cast<size_t>(B) * 64))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    const int64_t grid = grid_for(B, 256, cus, 64);
    if (h_dtype == BIRKHOFF4_BF16)
        launch_kernel(sk_fwd_kernel<BIRKHOFF4_BF16>, dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                           stream, H, P, B, n_steps);
    else
        launch_kernel(sk_fwd_kernel<BIRKHOFF4_F32>, dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                           stream, H, P, B, n_steps);
    return launch_status();
}

int birkhoff4_sk_bwd(const void* H, int h_dtype, const void* dP, int dp_dtype, float* dH, int64_t B,
                     int n_steps, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype) || !dtype_ok(dp_dtype)) return BIRKHOFF4_ERR_DTYPE;
    if (n_steps < 1 || n_steps > kMaxSkSteps) return BIRKHOFF4_ERR_STEPS;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !dP || !dH) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(dP) || misaligned(dH)) return BIRKHOFF4_ERR_ALIGN;
    const size_t n = static_cast<size_t>(B) * 64;
    if (overlaps(dH, n, H, static_cast<size_t>(B) * 16 * dtype_bytes(h_dtype)) ||
        overlaps(dH, n, dP, static_cast<size_t>(B) * 16 * dtype_bytes(dp_dtype)))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    if (n_steps == kSkRegSteps) {
        const int64_t grid = grid_for(B, 256, cus, 64);
        const dim3 g(static_cast<unsigned>(grid)), blk(256);
        if (h_dtype == BIRKHOFF4_BF16) {
            if (dp_dtype == BIRKHOFF4_BF16)
                launch_kernel((sk_bwd_reg_kernel<BIRKHOFF4_BF16, BIRKHOFF4_BF16, kSkRegSteps>), g, blk, 0, stream, H, dP, dH, B);
            else
                launch_kernel((sk_bwd_reg_kernel<BIRKHOFF4_BF16, BIRKHOFF4_F32, kSkRegSteps>), g, blk, 0, stream, H, dP, dH, B);
        } else {
            if (dp_dtype == BIRKHOFF4_BF16)
                launch_kernel((sk_bwd_reg_kernel<BIRKHOFF4_F32, BIRKHOFF4_BF16, kSkRegSteps>), g, blk, 0, stream, H, dP, dH, B);
            else
                launch_kernel((sk_bwd_reg_kernel<BIRKHOFF4_F32, BIRKHOFF4_F32, kSkRegSteps>), g, blk, 0, stream, H, dP, dH, B);
        }
        return launch_status();
    }
    const int64_t grid = grid_for(B, 64, cus, 64);
    const size_t lds = static_cast<size_t>(n_steps + 1) * 4 * 64 * sizeof(float);
    const dim3 g(static_cast<unsigned>(grid)), blk(64);
    if (h_dtype == BIRKHOFF4_BF16) {
        if (dp_dtype == BIRKHOFF4_BF16)
            launch_kernel((sk_bwd_kernel<BIRKHOFF4_BF16, BIRKHOFF4_BF16>), g, blk, lds, stream, H, dP, dH, B, n_steps);
        else
            launch_kernel((sk_bwd_kernel<BIRKHOFF4_BF16, BIRKHOFF4_F32>), g, blk, lds, stream, H, dP, dH, B, n_steps);
    } else {
        if (dp_dtype == BIRKHOFF4_BF16)
            launch_kernel((sk_bwd_kernel<BIRKHOFF4_F32, BIRKHOFF4_BF16>), g, blk, lds, stream, H, dP, dH, B, n_steps);
        else
            launch_kernel((sk_bwd_kernel<BIRKHOFF4_F32, BIRKHOFF4_F32>), g, blk, lds, stream, H, dP, dH, B, n_steps);
    }
    return launch_status();
}

int birkhoff4_mix_fwd(const void* H, int h_dtype, const void* X, int x_dtype, void* Y, float* P, float* dual,
                      int32_t* iters, int64_t B, int64_t C, float tol, int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype) || !dtype_ok(x_dtype)) return BIRKHOFF4_ERR_DTYPE;
    const int64_t E = x_dtype == BIRKHOFF4_BF16 ? 8 : 4;
    if (C < 0 || C % E != 0) return BIRKHOFF4_ERR_CHANNELS;
    const int64_t nc = C / E;  // 16-byte chunks per row
    if (B > 0 && nc > INT64_MAX / 64 / B) return BIRKHOFF4_ERR_SIZE;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P || (nc > 0 && (!X || !Y))) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(X) || misaligned(Y) || misaligned(P) || misaligned(dual) || misaligned(iters))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t nh = static_cast<size_t>(B) * 16 * dtype_bytes(h_dtype), nx = static_cast<size_t>(B) * 64 * nc;
    const size_t np = static_cast<size_t>(B) * 64, nd = dual ? static_cast<size_t>(B) * 32 : 0,
                 ni = iters ? static_cast<size_t>(B) * 4 : 0;
    if (overlaps(Y, nx, H, nh) || overlaps(Y, nx, X, nx) || overlaps(Y, nx, P, np) || overlaps(Y, nx, dual, nd) ||
        overlaps(Y, nx, iters, ni) || overlaps(P, np, X, nx) || overlaps(dual, nd, X, nx) ||
        overlaps(iters, ni, X, nx) || overlaps(H, nh, P, np) || overlaps(H, nh, dual, nd) ||
        overlaps(H, nh, iters, ni) || overlaps(P, np, dual, nd) || overlaps(P, np, iters, ni) ||
        overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    // the projection checks and queues P first; the mixing kernel then reads it
    if (int e = birkhoff4_fwd_ex2(H, h_dtype, P, dual, iters, B, tol, max_iter, BIRKHOFF4_AUTO, stream)) return e;
    if (nc == 0) return BIRKHOFF4_OK;
    if (x_dtype == BIRKHOFF4_BF16) return launch_mix_fwd<BIRKHOFF4_BF16>(P, X, Y, B, nc, stream, cus);
    return launch_mix_fwd<BIRKHOFF4_F32>(P, X, Y, B, nc, stream, cus);
}

int birkhoff4_mix_bwd(const float* P, const void* X, const void* dY, int x_dtype, void* dX, float* dH, int64_t B,
                      int64_t C, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 64)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(x_dtype)) return BIRKHOFF4_ERR_DTYPE;
    const int64_t E = x_dtype == BIRKHOFF4_BF16 ? 8 : 4;
    if (C < 0 || C % E != 0) return BIRKHOFF4_ERR_CHANNELS;
    const int64_t nc = C / E;
    if (B > 0 && nc > INT64_MAX / 64 / B) return BIRKHOFF4_ERR_SIZE;
    if (B == 0) return BIRKHOFF4_OK;
    if (!P || !dH || (nc > 0 && (!X || !dY || !dX))) return BIRKHOFF4_ERR_NULL;
    if (misaligned(P) || misaligned(X) || misaligned(dY) || misaligned(dX) || misaligned(dH))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t np = static_cast<size_t>(B) * 64, nx = static_cast<size_t>(B) * 64 * nc;
    if (overlaps(dX, nx, P, np) || overlaps(dX, nx, X, nx) || overlaps(dX, nx, dY, nx) || overlaps(dX, nx, dH, np) ||
        overlaps(dH, np, P, np) || overlaps(dH, np, X, nx) || overlaps(dH, np, dY, nx))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    if (x_dtype == BIRKHOFF4_BF16) return launch_mix_bwd<BIRKHOFF4_BF16>(P, X, dY, dX, dH, B, nc, stream, cus);
    return launch_mix_bwd<BIRKHOFF4_F32>(P, X, dY, dX, dH, B, nc, stream, cus);
}

int birkhoff8_mix_fwd(const void* H, int h_dtype, const void* X, int x_dtype, void* Y, float* P, float* dual,
                      int32_t* iters, int64_t B, int64_t C, float tol, int max_iter, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(h_dtype) || !dtype_ok(x_dtype)) return BIRKHOFF4_ERR_DTYPE;
    const int64_t E = x_dtype == BIRKHOFF4_BF16 ? 8 : 4;
    if (C < 0 || C % E != 0) return BIRKHOFF4_ERR_CHANNELS;
    const int64_t nc = C / E;  // 16-byte chunks per row
    if (B > 0 && nc > INT64_MAX / 128 / B) return BIRKHOFF4_ERR_SIZE;
    if (!(tol >= 0.f)) return BIRKHOFF4_ERR_TOL;
    if (max_iter < 0 || max_iter > kMaxIterCap) return BIRKHOFF4_ERR_MAX_ITER;
    if (B == 0) return BIRKHOFF4_OK;
    if (!H || !P || (nc > 0 && (!X || !Y))) return BIRKHOFF4_ERR_NULL;
    if (misaligned(H) || misaligned(X) || misaligned(Y) || misaligned(P) || misaligned(dual) || misaligned(iters))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t nh = static_cast<size_t>(B) * 64 * dtype_bytes(h_dtype), nx = static_cast<size_t>(B) * 128 * nc;
    const size_t np = static_cast<size_t>(B) * 256, nd = dual ? static_cast<size_t>(B) * 64 : 0,
                 ni = iters ? static_cast<size_t>(B) * 4 : 0;
    if (overlaps(Y, nx, H, nh) || overlaps(Y, nx, X, nx) || overlaps(Y, nx, P, np) || overlaps(Y, nx, dual, nd) ||
        overlaps(Y, nx, iters, ni) || overlaps(P, np, X, nx) || overlaps(dual, nd, X, nx) ||
        overlaps(iters, ni, X, nx) || overlaps(H, nh, P, np) || overlaps(H, nh, dual, nd) ||
        overlaps(H, nh, iters, ni) || overlaps(P, np, dual, nd) || overlaps(P, np, iters, ni) ||
        overlaps(dual, nd, iters, ni))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    if (int e = birkhoff8_fwd(H, h_dtype, P, dual, iters, B, tol, max_iter, stream)) return e;
    if (nc == 0) return BIRKHOFF4_OK;
    if (x_dtype == BIRKHOFF4_BF16) return launch_mix_fwd<BIRKHOFF4_BF16, 8>(P, X, Y, B, nc, stream, cus);
    return launch_mix_fwd<BIRKHOFF4_F32, 8>(P, X, Y, B, nc, stream, cus);
}

int birkhoff8_mix_bwd(const float* P, const void* X, const void* dY, int x_dtype, void* dX, float* dH, int64_t B,
                      int64_t C, hipStream_t stream) {
    if (B < 0 || B > (INT64_MAX / 256)) return BIRKHOFF4_ERR_SIZE;
    if (!dtype_ok(x_dtype)) return BIRKHOFF4_ERR_DTYPE;
    const int64_t E = x_dtype == BIRKHOFF4_BF16 ? 8 : 4;
    if (C < 0 || C % E != 0) return BIRKHOFF4_ERR_CHANNELS;
    const int64_t nc = C / E;
    if (B > 0 && nc > INT64_MAX / 128 / B) return BIRKHOFF4_ERR_SIZE;
    if (B == 0) return BIRKHOFF4_OK;
    if (!P || !dH || (nc > 0 && (!X || !dY || !dX))) return BIRKHOFF4_ERR_NULL;
    if (misaligned(P) || misaligned(X) || misaligned(dY) || misaligned(dX) || misaligned(dH))
        return BIRKHOFF4_ERR_ALIGN;
    const size_t np = static_cast<size_t>(B) * 256, nx = static_cast<size_t>(B) * 128 * nc;
    if (overlaps(dX, nx, P, np) || overlaps(dX, nx, X, nx) || overlaps(dX, nx, dY, nx) || overlaps(dX, nx, dH, np) ||
        overlaps(dH, np, P, np) || overlaps(dH, np, X, nx) || overlaps(dH, np, dY, nx))
        return BIRKHOFF4_ERR_OVERLAP;
    int cus = 0, dev = 0;
    if (int e = device_cus(stream, &cus, &dev)) return e;
    // dX, and dP into dH's memory; then the 8 x 8 backward turns dP into dH in place (each of
    // its waves reads a chunk's dP whole before it writes that chunk's dH)
    const int e = x_dtype == BIRKHOFF4_BF16 ? launch_mix_bwd<BIRKHOFF4_BF16, 8>(P, X, dY, dX, dH, B, nc, stream, cus)
                                            : launch_mix_bwd<BIRKHOFF4_F32, 8>(P, X, dY, dX, dH, B, nc, stream, cus);
    if (e) return e;
    const int64_t chunks = (B + 63) / 64;
    const int64_t want = (chunks + kB8Waves - 1) / kB8Waves;
    const int64_t grid = want < kMaxGrid ? want : kMaxGrid;
    launch_kernel((implicit8_bwd_kernel<BIRKHOFF4_F32, false, true>), dim3(static_cast<unsigned>(grid)),
                  dim3(kB8Block), 0, stream, P, dH, dH, B, nullptr, 1.f);
    return launch_status();
}

const char* birkhoff4_strerror(int code) {
    switch (code) {
        case BIRKHOFF4_OK: return "ok";
        case BIRKHOFF4_ERR_NULL: return "a required pointer is NULL";
        case BIRKHOFF4_ERR_SIZE: return "batch size out of range";
        case BIRKHOFF4_ERR_TOL: return "tol must be >= 0";
        case BIRKHOFF4_ERR_MAX_ITER: return "max_iter must be in [0, 10000]";
        case BIRKHOFF4_ERR_DTYPE: return "unknown dtype code";
        case BIRKHOFF4_ERR_ALIGN: return "arrays must be 16-byte aligned";
        case BIRKHOFF4_ERR_OVERLAP: return "an output overlaps another argument";
        case BIRKHOFF4_ERR_STEPS: return "Sinkhorn step count must be in [1, 48]";
        case BIRKHOFF4_ERR_DEVICE: return "HIP device query failed";
        case BIRKHOFF4_ERR_LAUNCH: return "kernel launch failed";
        case BIRKHOFF4_ERR_VARIANT: return "unknown forward variant";
        case BIRKHOFF4_ERR_ETA: return "eta must be positive and finite";
        case BIRKHOFF4_ERR_CHANNELS: return "C must be >= 0 and a multiple of 8 (bf16 streams) or 4 (fp32)";
        default: return "unknown error";
    }
}

int birkhoff4_version(void) { return 100; }

}  // extern "C"
