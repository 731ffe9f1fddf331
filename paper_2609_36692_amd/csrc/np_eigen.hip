// Dense symmetric eigensolver on the GPU, for the interaction matrix
// Gamma = Psi Psi^T of one active orientation (n = active rows, up to a few
// thousand):
//   * Householder reduction to tridiagonal form (working matrix stored in
//     fp32, all arithmetic and the vectors in fp64): up to n = 192 one
//     launch with the matrix in LDS; above, one reflector per step: a
//     one-block kernel forms the reflector of column j, and one streaming
//     pass over the trailing rows applies the previous step's rank-2 update
//     and forms the next product p = tau A v in the same read;
//   * eigenvalues of the tridiagonal matrix by multisection on Sturm counts
//     (16 lanes per eigenvalue, any subset of indices);
//   * eigenvectors of the selected eigenvalues by inverse iteration with a
//     partially pivoted tridiagonal LU, Gram-Schmidt inside clusters of
//     close eigenvalues, and back-transformation through the reflectors.
// Used by the exact variant of NormPre-L (App. B, exact eigenspace
// extraction: the leading eigenvectors of Gamma span the selected modes), by
// the Rayleigh-Ritz problems of the sketch wider than the Jacobi's limit,
// and by the spectral diagnostics of the normalized and unnormalized Grams
// (App. A, spectral dynamics).  Matrices of one launch share n (grid y).
#include "np_internal.h"

#include <algorithm>
#include <cfloat>

namespace np {
namespace {

constexpr int kHouseThreads = 1024;
constexpr int kRowWaves = 4;          // rows per block of the update pass
constexpr int kVecThreads = 256;      // Gram-Schmidt / back-transformation

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Sum over the block in a fixed order (every thread returns the same value).
template <int NT>
__device__ double block_sum_d(double v, double* red) {
    v = wave_sum_d(v);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    double t = 0.0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) t += red[i];
    return t;
}

// Gamma fp32 (GEMM output, ld ldg) -> symmetrized n x n (ld n).
__global__ void gamma_sym_kernel(const float* g, int64_t ldg, int64_t strideg, int n, float* A,
                                 int64_t strideA) {
    const int z = blockIdx.y;
    const float* gz = g + (int64_t)z * strideg;
    float* Az = A + (int64_t)z * strideA;
    const int64_t nn = (int64_t)n * n;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < nn; idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = idx / n, k = idx - i * n;
        Az[idx] = (float)(0.5 * ((double)gz[i * ldg + k] + (double)gz[k * ldg + i]));
    }
}

// Reflector of step j.  vec holds per matrix [v (2 ping-pong slots) | w | p],
// n doubles each; slot j & 1 receives v_j, slot (j + 1) & 1 holds v_{j-1}.
// With j > 0 it first completes step j - 1: w = p - (tau/2)(p^T v) v, and
// takes column j of the current matrix as row j of A (not yet updated by
// step j - 1) minus that step's rank-2 term.  v_j (v_j[j + 1] = 1, zero at
// indices <= j) is also stored in row j of A for the back-transformation.
__global__ void __launch_bounds__(kHouseThreads) tri_house_kernel(float* A, int64_t strideA, int n, int j,
                                                                  double* vec, int64_t stride_vec, double* dd,
                                                                  double* ee, double* tau, int64_t stride_n) {
    __shared__ double red[kHouseThreads / 64];
    const int z = blockIdx.x, tid = threadIdx.x;
    float* Az = A + (int64_t)z * strideA;
    double* V = vec + (int64_t)z * stride_vec;
    double* vprev = V + (int64_t)((j + 1) & 1) * n;
    double* vcur = V + (int64_t)(j & 1) * n;
    double* W = V + 2 * (int64_t)n;
    const double* P = V + 3 * (int64_t)n;
    float* row = Az + (int64_t)j * n;
    double wj = 0.0, vj = 0.0;
    if (j > 0) {
        const double tp = tau[(int64_t)z * stride_n + j - 1];
        double s = 0.0;
        for (int i = j + tid; i < n; i += kHouseThreads) s += P[i] * vprev[i];
        s = block_sum_d<kHouseThreads>(s, red);
        const double K = 0.5 * tp * s;
        for (int i = j + tid; i < n; i += kHouseThreads) W[i] = P[i] - K * vprev[i];
        __syncthreads();
        wj = W[j];
        vj = vprev[j];
    }
    auto col = [&](int i) -> double {
        const double r = row[i];
        return j > 0 ? r - vprev[i] * wj - W[i] * vj : r;
    };
    const double dj = col(j);
    const double alpha = j + 1 < n ? col(j + 1) : 0.0;
    double sig = 0.0;
    for (int i = j + 2 + tid; i < n; i += kHouseThreads) {
        const double c = col(i);
        sig += c * c;
    }
    sig = block_sum_d<kHouseThreads>(sig, red);   // also orders the reads above before the writes below
    double beta = alpha, t = 0.0, scal = 0.0;
    if (sig > 0.0) {
        beta = -copysign(sqrt(alpha * alpha + sig), alpha);
        t = (beta - alpha) / beta;
        scal = 1.0 / (alpha - beta);
    }
    for (int i = tid; i < n; i += kHouseThreads) {
        const double v = i <= j ? 0.0 : (i == j + 1 ? 1.0 : col(i) * scal);
        vcur[i] = v;
        if (i > j) row[i] = (float)v;
    }
    if (tid == 0) {
        dd[(int64_t)z * stride_n + j] = dj;
        ee[(int64_t)z * stride_n + j] = beta;
        tau[(int64_t)z * stride_n + j] = t;
    }
}

// Rows i > j: A[i, k] -= v_{j-1}[i] w[k] + w[i] v_{j-1}[k] for k > j (step
// j - 1's update, skipped for j = 0), then p[i] = tau_j sum_k A[i, k] v_j[k]
// over the updated row.  One wave per row.
__global__ void __launch_bounds__(kRowWaves * 64) tri_update_kernel(float* A, int64_t strideA, int n, int j,
                                                                    double* vec, int64_t stride_vec,
                                                                    const double* tau, int64_t stride_n) {
    const int z = blockIdx.y, lane = threadIdx.x & 63;
    const int i = j + 1 + blockIdx.x * kRowWaves + (threadIdx.x >> 6);
    if (i >= n) return;
    double* V = vec + (int64_t)z * stride_vec;
    const double* vprev = V + (int64_t)((j + 1) & 1) * n;
    const double* vcur = V + (int64_t)(j & 1) * n;
    const double* W = V + 2 * (int64_t)n;
    double* P = V + 3 * (int64_t)n;
    float* Ar = A + (int64_t)z * strideA + (int64_t)i * n;
    const bool upd = j > 0;
    const double vi = upd ? vprev[i] : 0.0, wi = upd ? W[i] : 0.0;
    double dot = 0.0;
    for (int k = j + 1 + lane; k < n; k += 64) {
        double a = Ar[k];
        if (upd) {
            a -= vi * W[k] + wi * vprev[k];
            Ar[k] = (float)a;
        }
        dot += a * vcur[k];
    }
    dot = wave_sum_d(dot);
    if (lane == 0) P[i] = tau[(int64_t)z * stride_n + j] * dot;
}

// Householder tridiagonalization of the trailing m x m block (m = n - j0 <=
// kTriLdsMax) of one matrix per block, in one launch with the block in LDS:
// per column the reflector from the current column (two block sums),
// p = tau M v over the trailing rows (one wave per row),
// w = p - (tau/2)(p^T v) v, and the eager rank-2 update M -= v w^T + w v^T.
// fp32 storage with fp64 arithmetic, as in the multi-launch reduction, whose
// outputs (d, e, tau and the reflectors in rows of A) it reproduces.  With
// j0 > 0 the multi-launch reduction has done columns 0 .. j0 - 1 and left the
// rank-2 update of column j0 - 1 pending (its reflector and p = tau A v in
// `vec`): the block is loaded with that update applied.  Larger trailing
// blocks stay with the multi-launch reduction: one CU's LDS holds neither the
// square nor, from about m = 200 on, beats the many-CU launches with the
// packed triangle.
constexpr int kTriLdsMax = 192;
constexpr int kTriThreads = 1024;

__global__ void __launch_bounds__(kTriThreads) tri_small_kernel(float* A, int64_t strideA, int n, int j0,
                                                                const double* vec, int64_t stride_vec, double* dd,
                                                                double* ee, double* tau, int64_t stride_n) {
    extern __shared__ float M[];
    __shared__ double v[kTriLdsMax], w[kTriLdsMax], red[kTriThreads / 64];
    constexpr int NW = kTriThreads / 64;
    const int z = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m = n - j0;
    float* Ag = A + (int64_t)z * strideA;
    if (j0 == 0) {
        for (int q = tid; q < m * m; q += kTriThreads) M[q] = Ag[q];
    } else {
        const double* V = vec + (int64_t)z * stride_vec;
        const double* vp = V + (int64_t)((j0 - 1) & 1) * n;
        const double* P = V + 3 * (int64_t)n;
        const double tp = tau[(int64_t)z * stride_n + j0 - 1];
        double s = 0.0;
        for (int i = j0 + tid; i < n; i += kTriThreads) s += P[i] * vp[i];
        const double K = 0.5 * tp * block_sum_d<kTriThreads>(s, red);
        for (int i = tid; i < m; i += kTriThreads) {
            v[i] = vp[j0 + i];
            w[i] = P[j0 + i] - K * vp[j0 + i];
        }
        __syncthreads();
        for (int q = tid; q < m * m; q += kTriThreads) {
            const int ii = q / m, kk = q - (q / m) * m;
            M[q] = (float)((double)Ag[(int64_t)(j0 + ii) * n + j0 + kk] - v[ii] * w[kk] - w[ii] * v[kk]);
        }
    }
    __syncthreads();
    for (int jj = 0; jj < m; ++jj) {
        const int j = j0 + jj;
        const float* row = M + jj * m;   // column jj by symmetry
        const double dj = row[jj];
        const double alpha = jj + 1 < m ? (double)row[jj + 1] : 0.0;
        double sig = 0.0;
        for (int i = jj + 2 + tid; i < m; i += kTriThreads) {
            const double c = row[i];
            sig += c * c;
        }
        sig = block_sum_d<kTriThreads>(sig, red);
        double beta = alpha, t = 0.0, scal = 0.0;
        if (sig > 0.0) {
            beta = -copysign(sqrt(alpha * alpha + sig), alpha);
            t = (beta - alpha) / beta;
            scal = 1.0 / (alpha - beta);
        }
        if (tid == 0) {
            dd[(int64_t)z * stride_n + j] = dj;
            ee[(int64_t)z * stride_n + j] = beta;
            tau[(int64_t)z * stride_n + j] = t;
        }
        if (t == 0.0) continue;   // H_j = I (uniform across the block)
        for (int i = jj + 1 + tid; i < m; i += kTriThreads) {
            const double vi = i == jj + 1 ? 1.0 : (double)row[i] * scal;
            v[i] = vi;
            Ag[(int64_t)j * n + j0 + i] = (float)vi;
        }
        __syncthreads();
        // p = t M v, rows i > jj, one wave per row.
        for (int i = jj + 1 + wave; i < m; i += NW) {
            const float* mi = M + i * m;
            double dot = 0.0;
            for (int k = jj + 1 + lane; k < m; k += 64) dot += (double)mi[k] * v[k];
            dot = wave_sum_d(dot);
            if (lane == 0) w[i] = t * dot;
        }
        __syncthreads();
        double pv = 0.0;
        for (int i = jj + 1 + tid; i < m; i += kTriThreads) pv += w[i] * v[i];
        const double K = 0.5 * t * block_sum_d<kTriThreads>(pv, red);
        for (int i = jj + 1 + tid; i < m; i += kTriThreads) w[i] -= K * v[i];
        __syncthreads();
        for (int i = jj + 1 + wave; i < m; i += NW) {
            float* mi = M + i * m;
            const double vi = v[i], wi = w[i];
            for (int k = jj + 1 + lane; k < m; k += 64) mi[k] = (float)((double)mi[k] - vi * w[k] - wi * v[k]);
        }
        __syncthreads();
    }
}

// Number of eigenvalues of the tridiagonal (d, e) below x (Sturm count of
// the LDL^T pivots; a pivot below pivmin in magnitude is set to -pivmin).
// e^2 / q uses the hardware reciprocal refined by two Newton steps (within an
// ulp or two of the quotient, a relative perturbation of each pivot that the
// backward-stable count absorbs), keeping the dependent chain per step short.
__device__ __forceinline__ double recip(double q) {
    double r = __builtin_amdgcn_rcp(q);
    r = fma(r, fma(-q, r, 1.0), r);
    return fma(r, fma(-q, r, 1.0), r);
}

__device__ int sturm_count(const double* __restrict__ d, const double* __restrict__ e, int n, double x,
                           double pivmin) {
    double q = d[0] - x;
    if (fabs(q) < pivmin) q = -pivmin;
    int c = q < 0.0;
#pragma unroll 8
    for (int i = 1; i < n; ++i) {
        const double ei = e[i - 1];
        q = (d[i] - x) - ei * ei * recip(q);
        if (fabs(q) < pivmin) q = -pivmin;
        c += q < 0.0;
    }
    return c;
}

// Multisection: kMsLanes lanes per eigenvalue, (first + t)-th largest for
// group t.  Each round the lanes count at kMsLanes interior points of the
// group's bracket [lo, hi] (splitting it into kMsLanes + 1 equal parts); the
// bracket becomes the part where the count crosses the eigenvalue's index.
// Stops at a width of 2 eps max(|lo|, |hi|) + pivmin, or when the points no
// longer split the bracket.
constexpr int kMsLanes = 16;

__global__ void __launch_bounds__(64) tri_bisect_kernel(const double* dd, const double* ee, int64_t stride_n, int n,
                                                        int first, int nvals, double* out, int64_t stride_out) {
    const int z = blockIdx.y, lane = threadIdx.x, grp = lane / kMsLanes, sub = lane % kMsLanes;
    const int t = blockIdx.x * (64 / kMsLanes) + grp;
    const double* d = dd + (int64_t)z * stride_n;
    const double* e = ee + (int64_t)z * stride_n;
    // Gershgorin interval, the wave's lanes splitting the rows.
    double lo = DBL_MAX, hi = -DBL_MAX, emax = 0.0;
    for (int i = lane; i < n; i += 64) {
        const double r = (i > 0 ? fabs(e[i - 1]) : 0.0) + (i + 1 < n ? fabs(e[i]) : 0.0);
        lo = fmin(lo, d[i] - r);
        hi = fmax(hi, d[i] + r);
        if (i + 1 < n) emax = fmax(emax, e[i] * e[i]);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        lo = fmin(lo, __shfl_xor(lo, o, 64));
        hi = fmax(hi, __shfl_xor(hi, o, 64));
        emax = fmax(emax, __shfl_xor(emax, o, 64));
    }
    const double pivmin = DBL_MIN * fmax(1.0, emax);
    const double span = fmax(fabs(lo), fabs(hi));
    lo -= 2.0 * DBL_EPSILON * span + pivmin;
    hi += 2.0 * DBL_EPSILON * span + pivmin;
    if (t >= nvals) return;
    // smallest x with count(x) > idx, idx counted from the bottom
    const int idx = n - 1 - (first + t);
    constexpr double kInv = 1.0 / (kMsLanes + 1);
    for (int it = 0; it < 100; ++it) {
        const double w = hi - lo;
        if (w <= 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin) break;
        auto pt = [&](int k) { return lo + (w * (double)k) * kInv; };
        const bool above = sturm_count(d, e, n, pt(sub + 1), pivmin) > idx;
        const unsigned mask =
            (unsigned)(__ballot(above) >> (grp * kMsLanes)) & ((1u << kMsLanes) - 1u);
        // First point whose count exceeds idx (kMsLanes: none does).
        const int s = mask ? __builtin_ctz(mask) : kMsLanes;
        const double nlo = s > 0 ? pt(s) : lo;
        const double nhi = s < kMsLanes ? pt(s + 1) : hi;
        if (!(nlo > lo) && !(nhi < hi)) break;
        lo = nlo;
        hi = nhi;
    }
    if (sub == 0) out[(int64_t)z * stride_out + t] = 0.5 * (lo + hi);
}

// Inverse iteration, one thread per eigenvalue k of matrix z: partially
// pivoted LU of T - lambda_k I, then `solves` solves of y (start: a fixed
// pseudo-random vector when init is set, else y as left by the previous
// launch), each followed by scaling to max |y_i| = 1.  The factors
// [dl | 1/d | du | du2 | pivot flag] and the working vector live in `lu`,
// interleaved across the eigenvalues of a matrix (entry i of vector k at
// [i nvals + k]) so each load and store of a wave is contiguous; the values
// a step carries to the next stay in registers.  y (one contiguous row per
// vector) is read at the start when init is clear and written at the end.
__global__ void __launch_bounds__(64) tri_inverse_kernel(const double* dd, const double* ee, int64_t stride_n, int n,
                                                         const double* lam, int64_t stride_lam, int nvals, double* lu,
                                                         double* y, int solves, int init) {
    const int z = blockIdx.y, k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= nvals) return;
    const double* __restrict__ d0 = dd + (int64_t)z * stride_n;
    const double* __restrict__ e0 = ee + (int64_t)z * stride_n;
    const int64_t nv = nvals, an = (int64_t)n * nv;
    double* base = lu + (int64_t)z * 6 * an + k;
    double* __restrict__ dl = base;
    double* __restrict__ ig = base + an;
    double* __restrict__ du = base + 2 * an;
    double* __restrict__ du2 = base + 3 * an;
    double* __restrict__ pv = base + 4 * an;
    double* __restrict__ yw = base + 5 * an;
    double* __restrict__ yk = y + ((int64_t)z * nvals + k) * (int64_t)n;
    const double lk = lam[(int64_t)z * stride_lam + k];
    if (init) {
        // Scale of T for the pivot floor.
        double tn = 0.0;
        for (int i = 0; i < n; ++i)
            tn = fmax(tn, fabs(d0[i]) + (i > 0 ? fabs(e0[i - 1]) : 0.0) + (i + 1 < n ? fabs(e0[i]) : 0.0));
        const double floor_piv = fmax(tn, DBL_MIN) * DBL_EPSILON;
        auto floored = [&](double g) { return fabs(g) < floor_piv ? (g < 0.0 ? -floor_piv : floor_piv) : g; };
        // g, u: the current diagonal and superdiagonal entries of row i (row
        // i + 1 of the matrix is still untouched when step i starts).
        double g = d0[0] - lk, u = n > 1 ? e0[0] : 0.0;
#pragma unroll 4
        for (int i = 0; i + 1 < n; ++i) {
            const double l = e0[i], gn = d0[i + 1] - lk, un = i + 2 < n ? e0[i + 1] : 0.0;
            const int64_t o = (int64_t)i * nv;
            if (fabs(g) >= fabs(l)) {
                const double f = g != 0.0 ? l / g : 0.0;
                dl[o] = f;
                ig[o] = 1.0 / floored(g);
                du[o] = u;
                du2[o] = 0.0;
                pv[o] = 0.0;
                g = gn - f * u;
                u = un;
            } else {
                const double f = g / l;
                dl[o] = f;
                ig[o] = 1.0 / floored(l);
                du[o] = gn;
                du2[o] = un;
                pv[o] = 1.0;
                g = u - f * gn;
                u = -f * un;
            }
        }
        ig[(int64_t)(n - 1) * nv] = 1.0 / floored(g);
        // Start vector: a fixed pseudo-random sequence in [-1, 1], distinct per k.
        uint32_t h = 0x9e3779b9u * (uint32_t)(k + 1);
        for (int i = 0; i < n; ++i) {
            h ^= h << 13; h ^= h >> 17; h ^= h << 5;
            yw[(int64_t)i * nv] = ((double)(h >> 8) * (1.0 / 8388608.0)) - 1.0;
        }
    } else {
#pragma unroll 8
        for (int i = 0; i < n; ++i) yw[(int64_t)i * nv] = yk[i];
    }
    // Both sweeps load eight steps' operands before the first of their stores
    // (the loads of the working vector would otherwise wait on the stores).
    constexpr int B = 8;
    double scale = 1.0;
    for (int sv = 0; sv < solves; ++sv) {
        // Forward: P L, the running entry c = y[i] in a register.
        double c = yw[0] * scale;
        for (int i0 = 0; i0 + 1 < n; i0 += B) {
            double nx[B], fl[B], pf[B];
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int64_t o = (int64_t)(i0 + j) * nv;
                const bool in = i0 + j + 1 < n;
                nx[j] = in ? yw[o + nv] * scale : 0.0;
                fl[j] = in ? dl[o] : 0.0;
                pf[j] = in ? pv[o] : 0.0;
            }
#pragma unroll
            for (int j = 0; j < B; ++j) {
                if (i0 + j + 1 >= n) break;
                const int64_t o = (int64_t)(i0 + j) * nv;
                if (pf[j] == 0.0) {
                    yw[o] = c;
                    c = nx[j] - fl[j] * c;
                } else {
                    yw[o] = nx[j];
                    c = c - fl[j] * nx[j];
                }
            }
        }
        // Backward: U with two superdiagonals, y[i + 1] and y[i + 2] carried.
        double y1 = c * ig[(int64_t)(n - 1) * nv], y2 = 0.0, mx = fabs(y1);
        yw[(int64_t)(n - 1) * nv] = y1;
        for (int i0 = n - 2; i0 >= 0; i0 -= B) {
            double yv[B], uu[B], u2[B], gi[B];
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int i = i0 - j;
                const int64_t o = (int64_t)(i < 0 ? 0 : i) * nv;
                yv[j] = i >= 0 ? yw[o] : 0.0;
                uu[j] = i >= 0 ? du[o] : 0.0;
                u2[j] = i >= 0 && i + 2 < n ? du2[o] : 0.0;
                gi[j] = i >= 0 ? ig[o] : 0.0;
            }
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int i = i0 - j;
                if (i < 0) break;
                const double y0 = (yv[j] - uu[j] * y1 - u2[j] * y2) * gi[j];
                yw[(int64_t)i * nv] = y0;
                mx = fmax(mx, fabs(y0));
                y2 = y1;
                y1 = y0;
            }
        }
        scale = mx > 0.0 ? 1.0 / mx : 1.0;
    }
#pragma unroll 8
    for (int i = 0; i < n; ++i) yk[i] = yw[(int64_t)i * nv] * scale;
}

// Modified Gram-Schmidt inside clusters (eigenvalues, descending, closer
// than ortol = 1e-9 * max |lambda| to their neighbour), then unit norm.  With
// shifts accurate to a few ulps, two solves leave a neighbour at gap g with a
// weight of about (eps ||T|| / g)^2, so only near-degenerate eigenvalues (the
// same shift from bisection) need the explicit orthogonalization.  Block k
// owns the cluster that starts at eigenvalue k (other blocks return), so
// clusters, mostly single vectors, run in parallel.
__global__ void __launch_bounds__(kVecThreads) vec_cluster_mgs_kernel(const double* lam, int64_t stride_lam, int n,
                                                                     int nvals, double* y) {
    __shared__ double red[kVecThreads / 64];
    const int z = blockIdx.y, k0 = blockIdx.x, tid = threadIdx.x;
    const double* lz = lam + (int64_t)z * stride_lam;
    const double ortol = 1e-9 * fmax(fabs(lz[0]), fabs(lz[nvals - 1]));
    if (k0 > 0 && !(lz[k0 - 1] - lz[k0] > ortol)) return;
    int k1 = k0 + 1;
    while (k1 < nvals && !(lz[k1 - 1] - lz[k1] > ortol)) ++k1;
    double* yz = y + (int64_t)z * nvals * n;
    for (int k = k0; k < k1; ++k) {
        double* yk = yz + (int64_t)k * n;
        for (int q = k0; q < k; ++q) {
            const double* yq = yz + (int64_t)q * n;
            double s = 0.0;
            for (int i = tid; i < n; i += kVecThreads) s += yk[i] * yq[i];
            s = block_sum_d<kVecThreads>(s, red);
            for (int i = tid; i < n; i += kVecThreads) yk[i] -= s * yq[i];
            __syncthreads();
        }
        double s = 0.0;
        for (int i = tid; i < n; i += kVecThreads) s += yk[i] * yk[i];
        s = block_sum_d<kVecThreads>(s, red);
        const double inv = s > 0.0 ? 1.0 / sqrt(s) : 0.0;
        for (int i = tid; i < n; i += kVecThreads) yk[i] *= inv;
        __syncthreads();
    }
}

// u = H_0 H_1 ... H_{n-1} y_k (reflector j in row j of A, v_j[j + 1] = 1),
// in place in y; then written as row k of the fp32 output (ld, zero padded
// to ld), rows nvals .. rows_out - 1 zero.
__global__ void __launch_bounds__(kVecThreads) tri_backtransform_kernel(const float* A, int64_t strideA, int n,
                                                                       const double* tau, int64_t stride_n,
                                                                       double* y, int nvals, float* out,
                                                                       int64_t ld_out, int64_t stride_out) {
    __shared__ double red[kVecThreads / 64];
    const int z = blockIdx.y, k = blockIdx.x, tid = threadIdx.x;
    float* o = out + (int64_t)z * stride_out + (int64_t)k * ld_out;
    if (k >= nvals) {
        for (int64_t i = tid; i < ld_out; i += kVecThreads) o[i] = 0.f;
        return;
    }
    double* u = y + ((int64_t)z * nvals + k) * (int64_t)n;
    const float* Az = A + (int64_t)z * strideA;
    const double* tz = tau + (int64_t)z * stride_n;
    for (int j = n - 1; j >= 0; --j) {
        const double t = tz[j];
        if (t == 0.0) continue;
        const float* v = Az + (int64_t)j * n;
        double s = 0.0;
        for (int i = j + 1 + tid; i < n; i += kVecThreads) s += v[i] * u[i];
        s = block_sum_d<kVecThreads>(s, red);
        const double f = t * s;
        for (int i = j + 1 + tid; i < n; i += kVecThreads) u[i] -= f * v[i];
        __syncthreads();
    }
    for (int64_t i = tid; i < ld_out; i += kVecThreads) o[i] = i < n ? (float)u[i] : 0.f;
}

// Summed fp64 Gram partials (upper 32 x 32 tiles, chunks x l_pad x l_pad)
// -> symmetric n x n fp32 matrix.
__global__ void gram_to_mat_kernel(const double* partial, int chunks, int ell_pad, int n, float* A) {
    const int z = blockIdx.y;
    const double* part = partial + (int64_t)z * chunks * ell_pad * ell_pad;
    float* Az = A + (int64_t)z * n * n;
    for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < n * n; idx += gridDim.x * blockDim.x) {
        const int c = idx / n, d = idx - (idx / n) * n;
        Az[idx] = (float)gram_at(part, ell_pad, c, d);
    }
}

// Selection of the top eigenpairs (lam descending, z rows) above one, Ritz
// values and |C|; K = Z_C diag(lambda^-1/2 - 1) Z_C^T (l_pad x l_pad, zero
// outside n x n), 256 entries per block.
__global__ void __launch_bounds__(256) select_k_kernel(const double* lam, int top, const float* zbuf, int n,
                                                       int ell_pad, float* kmat, float* ritz, int ritz_stride,
                                                       int* nsel) {
    const int z = blockIdx.y;
    const double* lz = lam + (int64_t)z * top;
    const float* Z = zbuf + (int64_t)z * top * n;
    int ns = 0;
    while (ns < top && lz[ns] > 1.0) ++ns;      // descending: the selected ones lead
    if (blockIdx.x == 0) {
        for (int t = threadIdx.x; t < top; t += 256) ritz[(int64_t)z * ritz_stride + t] = (float)lz[t];
        if (threadIdx.x == 0) nsel[z] = ns;
    }
    const int q = blockIdx.x * 256 + threadIdx.x;
    if (q >= ell_pad * ell_pad) return;
    const int c = q / ell_pad, d = q - (q / ell_pad) * ell_pad;
    double sacc = 0.0;
    if (c < n && d < n)
        for (int t = 0; t < ns; ++t) sacc += (double)Z[t * n + c] * (1.0 / sqrt(lz[t]) - 1.0) * (double)Z[t * n + d];
    kmat[(int64_t)z * ell_pad * ell_pad + q] = (float)sacc;
}

}  // namespace

hipError_t launch_gamma_sym(const float* g, int64_t ldg, int64_t strideg, int n, float* A, int batch,
                            hipStream_t s) {
    const int64_t nn = (int64_t)n * n;
    const unsigned blocks = (unsigned)std::min<int64_t>(4096, (nn + 255) / 256);
    hipLaunchKernelGGL(gamma_sym_kernel, dim3(blocks, batch), dim3(256), 0, s, g, ldg, strideg, n, A, nn);
    return hipGetLastError();
}

hipError_t launch_tridiagonalize(const TriWork& w, int n, int batch, hipStream_t s) {
    if (n < 1) return hipErrorInvalidValue;
    // Columns 0 .. j0 - 1 two launches each, then the trailing block of at
    // most kTriLdsMax in one launch.
    const int j0 = std::max(0, n - kTriLdsMax);
    for (int j = 0; j < j0; ++j) {
        hipLaunchKernelGGL(tri_house_kernel, dim3(batch), dim3(kHouseThreads), 0, s, w.A, (int64_t)n * n, n, j,
                           w.vec, 4 * (int64_t)n, w.d, w.e, w.tau, (int64_t)n);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int rows = n - j - 1;
        hipLaunchKernelGGL(tri_update_kernel, dim3((rows + kRowWaves - 1) / kRowWaves, batch),
                           dim3(kRowWaves * 64), 0, s, w.A, (int64_t)n * n, n, j, w.vec, 4 * (int64_t)n, w.tau,
                           (int64_t)n);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int m = n - j0;
    hipLaunchKernelGGL(tri_small_kernel, dim3(batch), dim3(kTriThreads), (size_t)m * m * sizeof(float), s, w.A,
                       (int64_t)n * n, n, j0, w.vec, 4 * (int64_t)n, w.d, w.e, w.tau, (int64_t)n);
    return hipGetLastError();
}

hipError_t launch_tri_eigvals(const TriWork& w, int n, int first, int nvals, double* out, int64_t stride_out,
                              int batch, hipStream_t s) {
    if (nvals < 1) return hipSuccess;
    constexpr int per_block = 64 / kMsLanes;
    hipLaunchKernelGGL(tri_bisect_kernel, dim3((nvals + per_block - 1) / per_block, batch), dim3(64), 0, s, w.d,
                       w.e, (int64_t)n, n, first, nvals, out, stride_out);
    return hipGetLastError();
}

hipError_t launch_tri_eigvecs(const TriWork& w, int n, const double* lam, int nvals, float* out, int64_t ld_out,
                              int rows_out, int64_t stride_out, int batch, hipStream_t s) {
    if (nvals < 1 || nvals > rows_out) return hipErrorInvalidValue;
    const dim3 g((nvals + 63) / 64, batch);
    hipLaunchKernelGGL(tri_inverse_kernel, g, dim3(64), 0, s, w.d, w.e, (int64_t)n, n, lam, (int64_t)nvals, nvals,
                       w.lu, w.y, 2, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(vec_cluster_mgs_kernel, dim3(nvals, batch), dim3(kVecThreads), 0, s, lam, (int64_t)nvals, n,
                       nvals, w.y);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(tri_inverse_kernel, g, dim3(64), 0, s, w.d, w.e, (int64_t)n, n, lam, (int64_t)nvals, nvals,
                       w.lu, w.y, 1, 0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(vec_cluster_mgs_kernel, dim3(nvals, batch), dim3(kVecThreads), 0, s, lam, (int64_t)nvals, n,
                       nvals, w.y);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(tri_backtransform_kernel, dim3(rows_out, batch), dim3(kVecThreads), 0, s, w.A, (int64_t)n * n,
                       n, w.tau, (int64_t)n, w.y, nvals, out, ld_out, stride_out);
    return hipGetLastError();
}

}  // namespace np

namespace np {

hipError_t launch_eig_select_dense(const EigArgs& a, const TriWork& w, double* lam, float* zbuf, int batch,
                                   hipStream_t s) {
    const int n = a.ell, lp = a.ell_pad, top = std::min(a.rank, n);
    if (a.chunks != kGramChunks || n < 1 || n > lp) return hipErrorInvalidValue;
    const unsigned gb = (unsigned)std::min<int64_t>(1024, ((int64_t)n * n + 255) / 256);
    hipLaunchKernelGGL(gram_to_mat_kernel, dim3(gb, batch), dim3(256), 0, s, a.partial, a.chunks, lp, n, w.A);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_tridiagonalize(w, n, batch, s);
    if (e != hipSuccess) return e;
    e = launch_tri_eigvals(w, n, 0, top, lam, top, batch, s);
    if (e != hipSuccess) return e;
    e = launch_tri_eigvecs(w, n, lam, top, zbuf, n, top, (int64_t)top * n, batch, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(select_k_kernel, dim3((unsigned)(((int64_t)lp * lp + 255) / 256), batch), dim3(256), 0, s,
                       lam, top, zbuf, n, lp, a.kmat, a.ritz, a.ritz_stride, a.nsel);
    return hipGetLastError();
}

}  // namespace np
