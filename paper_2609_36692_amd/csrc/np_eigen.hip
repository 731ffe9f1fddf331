// Dense symmetric eigensolver on the GPU, for the interaction matrix
// Gamma = Psi Psi^T of one active orientation (n = active rows, up to a few
// thousand):
//   * Householder reduction to tridiagonal form (working matrix stored in
//     fp32, all arithmetic and the vectors in fp64), one reflector per step:
//     a one-block kernel forms the reflector of column j, and one streaming
//     pass over the trailing rows applies the previous step's rank-2 update
//     and forms the next product p = tau A v in the same read;
//   * eigenvalues of the tridiagonal matrix by bisection on Sturm counts
//     (one thread per eigenvalue, any subset of indices);
//   * eigenvectors of the selected eigenvalues by inverse iteration with a
//     partially pivoted tridiagonal LU, Gram-Schmidt inside clusters of
//     close eigenvalues, and back-transformation through the reflectors.
// Used by the exact variant of NormPre-L (App. B, exact eigenspace
// extraction: the leading eigenvectors of Gamma span the selected modes) and
// by the spectral diagnostics of the normalized and unnormalized Grams
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

// Number of eigenvalues of the tridiagonal (d, e) below x (Sturm count of
// the LDL^T pivots; a pivot below pivmin in magnitude is set to -pivmin).
__device__ int sturm_count(const double* d, const double* e, int n, double x, double pivmin) {
    double q = d[0] - x;
    if (fabs(q) < pivmin) q = -pivmin;
    int c = q < 0.0;
    for (int i = 1; i < n; ++i) {
        q = d[i] - x - e[i - 1] * e[i - 1] / q;
        if (fabs(q) < pivmin) q = -pivmin;
        c += q < 0.0;
    }
    return c;
}

// Thread t finds the (first + t)-th largest eigenvalue.
__global__ void tri_bisect_kernel(const double* dd, const double* ee, int64_t stride_n, int n, int first, int nvals,
                                  double* out, int64_t stride_out) {
    const int z = blockIdx.y, t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= nvals) return;
    const double* d = dd + (int64_t)z * stride_n;
    const double* e = ee + (int64_t)z * stride_n;
    double lo = DBL_MAX, hi = -DBL_MAX, emax = 0.0;
    for (int i = 0; i < n; ++i) {
        const double r = (i > 0 ? fabs(e[i - 1]) : 0.0) + (i + 1 < n ? fabs(e[i]) : 0.0);
        lo = fmin(lo, d[i] - r);
        hi = fmax(hi, d[i] + r);
        if (i + 1 < n) emax = fmax(emax, e[i] * e[i]);
    }
    const double pivmin = DBL_MIN * fmax(1.0, emax);
    const double span = fmax(fabs(lo), fabs(hi));
    lo -= 2.0 * DBL_EPSILON * span + pivmin;
    hi += 2.0 * DBL_EPSILON * span + pivmin;
    // smallest x with count(x) > idx, idx counted from the bottom
    const int idx = n - 1 - (first + t);
    for (int it = 0; it < 200; ++it) {
        const double mid = 0.5 * (lo + hi);
        if (hi - lo <= 2.0 * DBL_EPSILON * fmax(fabs(lo), fabs(hi)) + pivmin || mid <= lo || mid >= hi) break;
        if (sturm_count(d, e, n, mid, pivmin) > idx) hi = mid;
        else lo = mid;
    }
    out[(int64_t)z * stride_out + t] = 0.5 * (lo + hi);
}

// Partially pivoted LU of T - lambda I (per matrix z, eigenvalue k), stored
// as 5 arrays of n doubles [dl | d | du | du2 | piv], then `solves`
// inverse-iteration solves of y (start: a fixed pseudo-random vector when
// init is set), each followed by scaling to max |y_i| = 1.
__global__ void tri_inverse_kernel(const double* dd, const double* ee, int64_t stride_n, int n, const double* lam,
                                   int64_t stride_lam, int nvals, double* lu, double* y, int solves, int init) {
    const int z = blockIdx.y, k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= nvals) return;
    const double* d0 = dd + (int64_t)z * stride_n;
    const double* e0 = ee + (int64_t)z * stride_n;
    double* L = lu + ((int64_t)z * nvals + k) * 5 * (int64_t)n;
    double* dl = L;
    double* dg = L + n;
    double* du = L + 2 * (int64_t)n;
    double* du2 = L + 3 * (int64_t)n;
    double* pv = L + 4 * (int64_t)n;
    double* yk = y + ((int64_t)z * nvals + k) * (int64_t)n;
    const double lk = lam[(int64_t)z * stride_lam + k];
    // Scale of T for the pivot floor.
    double tn = 0.0;
    for (int i = 0; i < n; ++i)
        tn = fmax(tn, fabs(d0[i]) + (i > 0 ? fabs(e0[i - 1]) : 0.0) + (i + 1 < n ? fabs(e0[i]) : 0.0));
    const double floor_piv = fmax(tn, DBL_MIN) * DBL_EPSILON;
    if (init) {
        for (int i = 0; i < n; ++i) {
            dg[i] = d0[i] - lk;
            if (i + 1 < n) { dl[i] = e0[i]; du[i] = e0[i]; }
        }
        for (int i = 0; i + 1 < n; ++i) {
            if (fabs(dg[i]) >= fabs(dl[i])) {
                const double f = dg[i] != 0.0 ? dl[i] / dg[i] : 0.0;
                dl[i] = f;
                dg[i + 1] -= f * du[i];
                if (i + 2 < n) du2[i] = 0.0;
                pv[i] = 0.0;
            } else {
                const double f = dg[i] / dl[i];
                dg[i] = dl[i];
                dl[i] = f;
                const double tmp = du[i];
                du[i] = dg[i + 1];
                dg[i + 1] = tmp - f * dg[i + 1];
                if (i + 2 < n) {
                    du2[i] = du[i + 1];
                    du[i + 1] = -f * du[i + 1];
                }
                pv[i] = 1.0;
            }
        }
        for (int i = 0; i < n; ++i)
            if (fabs(dg[i]) < floor_piv) dg[i] = dg[i] < 0.0 ? -floor_piv : floor_piv;
        // Start vector: a fixed pseudo-random sequence in [-1, 1], distinct per k.
        uint32_t h = 0x9e3779b9u * (uint32_t)(k + 1);
        for (int i = 0; i < n; ++i) {
            h ^= h << 13; h ^= h >> 17; h ^= h << 5;
            yk[i] = ((double)(h >> 8) * (1.0 / 8388608.0)) - 1.0;
        }
    }
    for (int sv = 0; sv < solves; ++sv) {
        for (int i = 0; i + 1 < n; ++i) {
            if (pv[i] == 0.0) {
                yk[i + 1] -= dl[i] * yk[i];
            } else {
                const double tmp = yk[i];
                yk[i] = yk[i + 1];
                yk[i + 1] = tmp - dl[i] * yk[i];
            }
        }
        yk[n - 1] /= dg[n - 1];
        if (n > 1) yk[n - 2] = (yk[n - 2] - du[n - 2] * yk[n - 1]) / dg[n - 2];
        for (int i = n - 3; i >= 0; --i) yk[i] = (yk[i] - du[i] * yk[i + 1] - du2[i] * yk[i + 2]) / dg[i];
        double mx = 0.0;
        for (int i = 0; i < n; ++i) mx = fmax(mx, fabs(yk[i]));
        const double inv = mx > 0.0 ? 1.0 / mx : 1.0;
        for (int i = 0; i < n; ++i) yk[i] *= inv;
    }
}

// Modified Gram-Schmidt inside clusters (eigenvalues, descending, closer
// than ortol = 1e-9 * max |lambda| to their neighbour), then unit norm.  With
// shifts accurate to a few ulps, two solves leave a neighbour at gap g with a
// weight of about (eps ||T|| / g)^2, so only near-degenerate eigenvalues (the
// same shift from bisection) need the explicit orthogonalization.
__global__ void __launch_bounds__(kVecThreads) vec_cluster_mgs_kernel(const double* lam, int64_t stride_lam, int n,
                                                                     int nvals, double* y) {
    __shared__ double red[kVecThreads / 64];
    const int z = blockIdx.x, tid = threadIdx.x;
    const double* lz = lam + (int64_t)z * stride_lam;
    double* yz = y + (int64_t)z * nvals * n;
    const double ortol = 1e-9 * fmax(fabs(lz[0]), fabs(lz[nvals - 1]));
    int cstart = 0;
    for (int k = 0; k < nvals; ++k) {
        if (k > 0 && lz[k - 1] - lz[k] > ortol) cstart = k;
        double* yk = yz + (int64_t)k * n;
        for (int q = cstart; q < k; ++q) {
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
    for (int j = 0; j < n; ++j) {
        hipLaunchKernelGGL(tri_house_kernel, dim3(batch), dim3(kHouseThreads), 0, s, w.A, (int64_t)n * n, n, j,
                           w.vec, 4 * (int64_t)n, w.d, w.e, w.tau, (int64_t)n);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (j + 1 < n) {
            const int rows = n - j - 1;
            hipLaunchKernelGGL(tri_update_kernel, dim3((rows + kRowWaves - 1) / kRowWaves, batch),
                               dim3(kRowWaves * 64), 0, s, w.A, (int64_t)n * n, n, j, w.vec, 4 * (int64_t)n, w.tau,
                               (int64_t)n);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

hipError_t launch_tri_eigvals(const TriWork& w, int n, int first, int nvals, double* out, int64_t stride_out,
                              int batch, hipStream_t s) {
    if (nvals < 1) return hipSuccess;
    hipLaunchKernelGGL(tri_bisect_kernel, dim3((nvals + 63) / 64, batch), dim3(64), 0, s, w.d, w.e, (int64_t)n, n,
                       first, nvals, out, stride_out);
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
    hipLaunchKernelGGL(vec_cluster_mgs_kernel, dim3(batch), dim3(kVecThreads), 0, s, lam, (int64_t)nvals, n, nvals,
                       w.y);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(tri_inverse_kernel, g, dim3(64), 0, s, w.d, w.e, (int64_t)n, n, lam, (int64_t)nvals, nvals,
                       w.lu, w.y, 1, 0);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(vec_cluster_mgs_kernel, dim3(batch), dim3(kVecThreads), 0, s, lam, (int64_t)nvals, n, nvals,
                       w.y);
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
