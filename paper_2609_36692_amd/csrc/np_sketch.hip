// Small and latency-bound kernels of the NormPre-L randomized interaction
// sketch (Alg. 2, App. B) for gfx950:
//   * the Gaussian test matrix Omega (Philox4x32-10 of Salmon et al., SC'11,
//     with the Box-Muller transform),
//   * the deterministic reduction of K-split partial products,
//   * fp64 Gram matrices of l-major skinny matrices (for the orthogonal
//     basis Q = qr(Y) and for the Rayleigh-Ritz matrix Gamma_Q = B B^T),
//   * Cholesky-QR: Cholesky of the Gram with dropping of numerically
//     dependent columns, and the triangular inverse,
//   * small products M^T V with an l x l matrix M,
//   * a parallel cyclic Jacobi eigensolver for Gamma_Q followed by the
//     selection of the top-min(r, l) Ritz values above one and the l x l
//     matrix K = Z_C diag(lambda_C^{-1/2} - 1) Z_C^T.
#include "np_internal.h"

#include <algorithm>

namespace np {
namespace {

// ------------------------------------------------------------- Philox ---
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
        const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    }
    return c;
}

// Normal variate number e of the stream keyed by (seed, step, id).
__device__ __forceinline__ float omega_value(uint64_t seed, int64_t step, uint32_t id, int64_t e) {
    const uint4 ctr = make_uint4((uint32_t)(e >> 2), id, (uint32_t)((uint64_t)step & 0xffffffffu),
                                 (uint32_t)((uint64_t)step >> 32));
    const uint4 x = philox4x32_10(ctr, (uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32));
    const int lane = (int)(e & 3);
    const uint32_t a = lane < 2 ? x.x : x.z;
    const uint32_t b = lane < 2 ? x.y : x.w;
    const float u1 = (float)((a >> 8) + 1u) * 0x1p-24f;
    const float u2 = (float)(b >> 8) * 0x1p-24f;
    const float rad = sqrtf(-2.f * logf(u1));
    float s, c;
    sincospif(2.f * u2, &s, &c);
    return (lane & 1) ? rad * s : rad * c;
}

__global__ void omega_f16_kernel(OmegaArgs a) {
    const int z = blockIdx.y;
    const int64_t total = (int64_t)a.ell_pad * a.ld;
    half_t* out = a.out + (int64_t)z * a.stride;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int c = (int)(idx / a.ld);
        const int64_t i = idx - (int64_t)c * a.ld;
        float v = 0.f;
        if (c < a.ell && i < a.b) v = omega_value(a.seed, a.step, (uint32_t)a.ids[z], (int64_t)c * a.b + i);
        out[idx] = (half_t)v;
    }
}

__global__ void omega_f32_kernel(uint64_t seed, int64_t step, uint32_t id, int64_t b, int ell, float* out) {
    const int64_t total = b * ell;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        // out is b x l row-major: out[i*l + j] = Omega_ij, e = j*b + i.
        const int64_t i = idx / ell, j = idx - i * ell;
        out[idx] = omega_value(seed, step, id, j * b + i);
    }
}

// ------------------------------------------------------ split reduction ---
// Partial sums of one split-K product: out = sum over splits in split order
// (fp32), to fp32 and/or fp16 (times scale16).
__device__ __forceinline__ void reduce_splits_one(const float4* p, int splits, int64_t split4, int64_t i,
                                                  float* out32, half_t* out16, float scale16) {
    float4 s = p[i];
    for (int k = 1; k < splits; ++k) {
        const float4 q = p[i + k * split4];
        s.x += q.x; s.y += q.y; s.z += q.z; s.w += q.w;
    }
    if (out32) reinterpret_cast<float4*>(out32)[i] = s;
    if (out16) {
        half_t h[4] = {(half_t)(s.x * scale16), (half_t)(s.y * scale16), (half_t)(s.z * scale16),
                       (half_t)(s.w * scale16)};
        reinterpret_cast<uint2*>(out16)[i] = *reinterpret_cast<const uint2*>(h);
    }
}

__global__ void reduce_splits_kernel(const float* part, int splits, int64_t stride_split, int64_t stride_mat,
                                     int64_t n4, float* out32, half_t* out16, float scale16, int64_t stride_out) {
    const int z = blockIdx.y;
    const float4* p = reinterpret_cast<const float4*>(part + (int64_t)z * stride_mat);
    float* o32 = out32 ? out32 + (int64_t)z * stride_out : nullptr;
    half_t* o16 = out16 ? out16 + (int64_t)z * stride_out : nullptr;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += (int64_t)gridDim.x * blockDim.x)
        reduce_splits_one(p, splits, stride_split / 4, i, o32, o16, scale16);
}

// The split sums of several sketch products, matrix z of the launch in the
// group whose range holds it.
__global__ void reduce_splits_grouped_kernel(ReduceGroups g) {
    const int z = blockIdx.y;
    int gi = 0;
    while (gi + 1 < g.n && z >= g.zbeg[gi + 1]) ++gi;
    const int lz = z - g.zbeg[gi];
    const float4* p = reinterpret_cast<const float4*>(g.part[gi] + (int64_t)lz * g.stride_mat[gi]);
    float* o32 = g.out32[gi] ? g.out32[gi] + (int64_t)lz * g.stride_out[gi] : nullptr;
    half_t* o16 = g.out16[gi] ? g.out16[gi] + (int64_t)lz * g.stride_out[gi] : nullptr;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < g.n4[gi];
         i += (int64_t)gridDim.x * blockDim.x)
        reduce_splits_one(p, g.splits[gi], g.stride_split[gi] / 4, i, o32, o16, g.scale16[gi]);
}

// ------------------------------------------------------------ fp64 Gram ---
// Item of launch matrix z in a grouped launch (few items: a linear scan).
template <class T>
__device__ __forceinline__ int item_of(const T& t, int z) {
    int g = 0;
    while (g + 1 < t.n && z >= t.zbeg[g + 1]) ++g;
    return g;
}

// 64 x 64 output tile (tc <= td) over one chunk of the length dimension, in
// 4 x 4 register blocks, one per thread, only those with rows and columns
// below l, and on a diagonal tile only the upper ones (written to both
// triangles): waves without a block skip the products, so padding and
// symmetry cost no fp64 FMAs.  The tile's rows stream through LDS 64 columns
// at a time (columns major, so a thread reads its four rows as one float4).
// Every entry sums in a fixed order; chunks past the item's length write
// zeros.  Lengths and chunk lengths are multiples of 64.
__global__ void __launch_bounds__(256) gram64_kernel(Gram64Items t, int ell_pad, double* partial) {
    const int z = blockIdx.z, chunk = blockIdx.y;
    const int g = item_of(t, z);
    const int64_t ld = t.ld[g], len = t.len[g];
    const int chunk_len = t.chunk_len[g], ell = t.ell;
    const int tiles = ell_pad / 64;
    int tc = 0, left = blockIdx.x;
    while (left >= tiles - tc) { left -= tiles - tc; ++tc; }
    const int td = tc + left;
    const bool diag = tc == td;
    __shared__ float sc[64][68], sd[64][68];
    float (*sb)[68] = diag ? sc : sd;
    const int tid = threadIdx.x;
    // This thread's block (bi, bj): row blocks of 4 below l in each tile.
    // When the tile has few blocks (small l), `split` adjacent lanes share a
    // block, each taking every split-th column of a slab, and their sums are
    // combined by shuffles at the end (a fixed order).
    const int nbc = min(16, (ell - 64 * tc + 3) / 4), nbd = min(16, (ell - 64 * td + 3) / 4);
    const int nact = diag ? nbc * (nbc + 1) / 2 : nbc * nbd;
    int split = 1;
    while (split < 8 && nact * split * 2 <= 256) split *= 2;
    const int blk = tid / split, part = tid - blk * split;
    int bi = -1, bj = -1;
    if (diag) {
        int w = blk, r = 0;
        while (r < nbc && w >= nbc - r) { w -= nbc - r; ++r; }
        if (r < nbc) { bi = r; bj = r + w; }
    } else if (blk < nact) {
        bi = blk / nbd;
        bj = blk - bi * nbd;
    }
    const float* vz = t.v[g] + (int64_t)(z - t.zbeg[g]) * t.stride[g];
    double acc[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[u][e] = 0.0;
    const int64_t j0 = (int64_t)chunk * chunk_len, j1 = min(len, j0 + chunk_len);
    const int lr = tid >> 2, lc = (tid & 3) * 16;
    const bool rc = 64 * tc + lr < ell, rd = 64 * td + lr < ell;
    // The next slab's global loads are in flight during this slab's FMAs.
    float4 a[4], b[4];
    auto gload = [&](int64_t jb) {
        const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            a[u] = rc ? *(const float4*)(vz + (int64_t)(64 * tc + lr) * ld + jb + lc + 4 * u) : zero;
            b[u] = !diag && rd ? *(const float4*)(vz + (int64_t)(64 * td + lr) * ld + jb + lc + 4 * u) : zero;
        }
    };
    if (j0 < j1) gload(j0);
    for (int64_t jb = j0; jb < j1; jb += 64) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sc[lc + 4 * u][lr] = a[u].x;
            sc[lc + 4 * u + 1][lr] = a[u].y;
            sc[lc + 4 * u + 2][lr] = a[u].z;
            sc[lc + 4 * u + 3][lr] = a[u].w;
            if (!diag) {
                sd[lc + 4 * u][lr] = b[u].x;
                sd[lc + 4 * u + 1][lr] = b[u].y;
                sd[lc + 4 * u + 2][lr] = b[u].z;
                sd[lc + 4 * u + 3][lr] = b[u].w;
            }
        }
        __syncthreads();
        if (jb + 64 < j1) gload(jb + 64);
        if (bi >= 0) {
#pragma unroll 4
            for (int jj = part; jj < 64; jj += split) {
                const float4 xa = *(const float4*)&sc[jj][4 * bi];
                const float4 xb = *(const float4*)&sb[jj][4 * bj];
                const double av[4] = {xa.x, xa.y, xa.z, xa.w}, bv[4] = {xb.x, xb.y, xb.z, xb.w};
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[u][e] = fma(av[u], bv[e], acc[u][e]);
            }
        }
        __syncthreads();
    }
    // The split lanes of a block are adjacent in one wave (split divides 64).
    for (int o = 1; o < split; o <<= 1)
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[u][e] += __shfl_xor(acc[u][e], o, 64);
    if (bi < 0 || part != 0) return;
    double* out = partial + ((int64_t)z * kGramChunks + chunk) * ell_pad * ell_pad;
    const int r0 = 64 * tc + 4 * bi, c0 = 64 * td + 4 * bj;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[(int64_t)(r0 + u) * ell_pad + c0 + e] = acc[u][e];
            if (diag) out[(int64_t)(c0 + e) * ell_pad + r0 + u] = acc[u][e];
        }
}

// -------------------------------------------------------- Cholesky + inverse
// One block per matrix.  G = R^T R with R upper triangular; a pivot below
// kDropTol * G_kk (relative to the column's own squared norm) marks the
// column as numerically dependent: its row of R and of R^{-1} is zero, so the
// matching column of Q = Y R^{-1} is zero and it never reaches the selection.
constexpr double kDropTol = 1e-12;
// fp64 1/sqrt(x) and 1/x for x > 0: the hardware estimates refined by two
// Newton steps, accurate to fp64 rounding with a much shorter dependent chain
// than the IEEE square-root and division sequences (which sit on the
// per-pivot critical path of the factorizations below).
__device__ __forceinline__ double rsqrt_f64(double x) {
    double y = __builtin_amdgcn_rsq(x);
    const double h = 0.5 * x;
    y = y * fma(-h * y, y, 1.5);
    return y * fma(-h * y, y, 1.5);
}
__device__ __forceinline__ double rcp_f64(double x) {
    double y = __builtin_amdgcn_rcp(x);
    y = fma(y, fma(-x, y, 1.0), y);
    return fma(y, fma(-x, y, 1.0), y);
}

constexpr int kCholLdsMax = 96;
constexpr int kSmallThreads = 512;

constexpr int kCholThreads = 1024;
// Upper-triangle entries (i <= j) owned per thread: l (l + 1) / 2 entries for
// l <= kCholLdsMax over NT threads.
template <int NT>
constexpr int chol_own() { return (kCholLdsMax * (kCholLdsMax + 1) / 2 + NT - 1) / NT; }
// Threads of the LDS kernel (measured: 512 a little ahead of 256 and 1024).
constexpr int kCholLdsThreads = 512;

// l <= kCholLdsMax: the whole matrix lives in LDS (fp64, row stride l + 1);
// R^{-1} overwrites R in place.
template <int NT>
__global__ void __launch_bounds__(NT) chol_inv_kernel(const double* partial, int chunks, int ell, int ell_pad,
                                                      float* rinv) {
    constexpr int kCholOwn = chol_own<NT>();
    extern __shared__ double dynd[];
    const int z = blockIdx.x, tid = threadIdx.x;
    const double* p = partial + (int64_t)z * chunks * ell_pad * ell_pad;
    const int ld = ell + 1;
    // One square buffer.  Step k reads the updated upper row k, leaves the
    // finished row k of R in the lower triangle (R(k, j) at [j][k]) and
    // updates the upper trailing block, so it never reads what it writes and
    // one barrier per step suffices.  R^{-1} then fills the upper triangle,
    // one column per thread, reading R from the lower triangle.
    double* R = dynd;
    float* out = rinv + (int64_t)z * ell_pad * ell_pad;
    __shared__ double diag0[kCholLdsMax];
    __shared__ double inv_diag[kCholLdsMax];
    for (int q = tid; q < ell * ell; q += NT) {
        const int c = q / ell, d = q - (q / ell) * ell;
        if (d >= c) {
            const double g = gram_at(p, ell_pad, c, d);
            R[c * ld + d] = g;
            if (c == d) diag0[c] = g;
        }
    }
    __syncthreads();
    {
        // The trailing updates of this thread's fixed entries, no index
        // arithmetic in the step loop.
        int own[kCholOwn];
        const int ne = ell * (ell + 1) / 2;
#pragma unroll
        for (int m = 0; m < kCholOwn; ++m) {
            int e = tid + m * NT, i = 0;
            if (e < ne) {
                while (e >= ell - i) { e -= ell - i; ++i; }
                own[m] = (i << 16) | (i + e);
            } else {
                own[m] = -1;
            }
        }
        for (int k = 0; k < ell; ++k) {
            const double piv = R[k * ld + k];
            const bool keep = diag0[k] > 0.0 && piv > kDropTol * diag0[k];
            const double irk = keep ? rsqrt_f64(piv) : 0.0;
            const double ipiv = irk * irk;
            if (tid == 0) inv_diag[k] = irk;
            for (int j = k + 1 + tid; j < ell; j += NT) R[j * ld + k] = R[k * ld + j] * irk;
#pragma unroll
            for (int m = 0; m < kCholOwn; ++m) {
                if (own[m] < 0) break;
                const int i = own[m] >> 16, j = own[m] & 0xffff;
                if (i > k) R[i * ld + j] -= R[k * ld + i] * R[k * ld + j] * ipiv;
            }
            __syncthreads();
        }
    }
    // X = R^{-1}: X(i, j) = -(sum_{i < k <= j} R(i, k) X(k, j)) / R(i, i),
    // X(i, i) = 1 / R(i, i); rows of dropped columns are zero.  One column per
    // thread, bottom up, no barriers.
    auto x_entry = [&](int i, int j) {
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
        int k = i + 1;
        for (; k + 3 <= j; k += 4) {
            s0 += R[k * ld + i] * R[k * ld + j];
            s1 += R[(k + 1) * ld + i] * R[(k + 1) * ld + j];
            s2 += R[(k + 2) * ld + i] * R[(k + 2) * ld + j];
            s3 += R[(k + 3) * ld + i] * R[(k + 3) * ld + j];
        }
        for (; k <= j; ++k) s0 += R[k * ld + i] * R[k * ld + j];
        return -((s0 + s1) + (s2 + s3)) * inv_diag[i];
    };
    for (int j = tid; j < ell; j += NT) {
        R[j * ld + j] = inv_diag[j];
        for (int i = j - 1; i >= 0; --i) R[i * ld + j] = x_entry(i, j);
    }
    __syncthreads();
    for (int q = tid; q < ell_pad * ell_pad; q += NT) {
        const int i = q / ell_pad, j = q - (q / ell_pad) * ell_pad;
        out[q] = (i < ell && j < ell && j >= i) ? (float)R[i * ld + j] : 0.f;
    }
}

// l > kCholLdsMax (the whole matrix fits in LDS up to l = 138, but one pivot
// per barrier over the whole trailing matrix is slower from about l = 100 on):
// R and X = R^{-1} live in a global scratch slice (two l_pad^2 fp64 squares,
// upper triangles only, L2-resident at these sizes) and the work runs in row
// panels staged through LDS, so the global traffic is one read and write of
// the trailing triangle per panel rather than per pivot.
//   Cholesky (right-looking), panel of kPanelC rows k0..: factor the panel
//   rows in LDS (one barrier per pivot), scale them into rows of R, then
//   subtract their outer products from the trailing upper triangle in 4x4
//   register tiles.
//   Inverse, row panels of kPanelI rows bottom up: with rows below the panel
//   of X final, T = R(I, below) X(below, :) per column (a column and four
//   panel rows per thread), then X(I, j) = R(I, I)^{-1} (e_j - T(:, j)) by
//   back substitution, one column per thread in registers.
constexpr int kPanelC = 32;
constexpr int kPanelI = 16;

// Copies src[c] -> dst[c] for c in [c0, c1), lane-strided, with eight loads
// in flight per lane before the first store (one L2 latency per 512 entries).
__device__ __forceinline__ void row_to_lds(double* dst, const double* src, int c0, int c1, int lane) {
    for (int c = c0 + lane; c < c1; c += 512) {
        double v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = c + 64 * u < c1 ? src[c + 64 * u] : 0.0;
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (c + 64 * u < c1) dst[c + 64 * u] = v[u];
    }
}

__global__ void __launch_bounds__(kCholThreads) chol_inv_panel_kernel(const double* partial, int chunks, int ell,
                                                                      int ell_pad, double* scratch, float* rinv) {
    constexpr int NT = kCholThreads;
    extern __shared__ double dynd[];
    const int z = blockIdx.x, tid = threadIdx.x, lane = tid & 63, grp = tid >> 6;
    constexpr int NG = NT / 64;
    const double* p = partial + (int64_t)z * chunks * ell_pad * ell_pad;
    const int ld = ell_pad, pst = ell + 1;
    double* W = scratch + (int64_t)z * 2 * ell_pad * ell_pad;
    double* X = W + (int64_t)ell_pad * ell_pad;
    float* out = rinv + (int64_t)z * ell_pad * ell_pad;
    __shared__ double diag0[384];
    __shared__ double pivot[384];
    __shared__ double inv_diag[384];
    // Entries of the output outside the upper triangle of the l x l block
    // are zero; the inverse writes the rest.
    for (int i = grp; i < ell_pad; i += NG)
        for (int j = lane; j < ell_pad; j += 64)
            if (!(i < ell && j < ell && j >= i)) out[(int64_t)i * ell_pad + j] = 0.f;
    for (int i = grp; i < ell; i += NG)
        for (int j0 = i + lane; j0 < ell; j0 += 256) {
            double g[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) g[u] = j0 + 64 * u < ell ? gram_at(p, ell_pad, i, j0 + 64 * u) : 0.0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int j = j0 + 64 * u;
                if (j < ell) {
                    W[(int64_t)i * ld + j] = g[u];
                    if (i == j) diag0[i] = g[u];
                }
            }
        }
    __syncthreads();

    double* P = dynd;  // kPanelC x pst
    for (int k0 = 0; k0 < ell; k0 += kPanelC) {
        const int kb = min(kPanelC, ell - k0), w = ell - k0;
        for (int r = grp; r < kb; r += NG) row_to_lds(P + r * pst, W + (int64_t)(k0 + r) * ld + k0, r, w, lane);
        __syncthreads();
        for (int r = 0; r < kb; ++r) {
            const int k = k0 + r;
            const double piv = P[r * pst + r];
            const bool keep = diag0[k] > 0.0 && piv > kDropTol * diag0[k];
            const double ipiv = keep ? rcp_f64(piv) : 0.0;
            if (tid == 0) pivot[k] = keep ? piv : 0.0;
            const double* pr = P + r * pst;
            for (int rr = r + 1 + grp; rr < kb; rr += NG) {
                const double f = pr[rr] * ipiv;
                double* prr = P + rr * pst;
#pragma unroll 4
                for (int c = rr + lane; c < w; c += 64) prr[c] -= f * pr[c];
            }
            __syncthreads();
        }
        // Rows of R: the pivot rows scaled by 1 / sqrt(pivot) (zero when dropped).
        for (int r = grp; r < kb; r += NG) {
            const double pv = pivot[k0 + r];
            const double s = pv > 0.0 ? rsqrt_f64(pv) : 0.0;
            if (lane == 0) inv_diag[k0 + r] = s;
            for (int c = r + lane; c < w; c += 64) {
                const double v = P[r * pst + c] * s;
                P[r * pst + c] = v;
                W[(int64_t)(k0 + r) * ld + k0 + c] = v;
            }
        }
        __syncthreads();
        const int t0 = kb, t = w - kb, nbk = (t + 3) >> 2;
        for (int b = tid; b < nbk * nbk; b += NT) {
            const int bi = b / nbk, bj = b - bi * nbk;
            if (bi > bj) continue;
            const int ci = t0 + 4 * bi, cj = t0 + 4 * bj;
            double acc[4][4];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = ci + a, j = cj + e;
                    acc[a][e] = (j < w && i <= j) ? W[(int64_t)(k0 + i) * ld + k0 + j] : 0.0;
                }
#pragma unroll 4
            for (int r = 0; r < kb; ++r) {
                double vi[4], vj[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    vi[a] = ci + a < w ? P[r * pst + ci + a] : 0.0;
                    vj[a] = cj + a < w ? P[r * pst + cj + a] : 0.0;
                }
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[a][e] -= vi[a] * vj[e];
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int i = ci + a, j = cj + e;
                    if (j < w && i <= j) W[(int64_t)(k0 + i) * ld + k0 + j] = acc[a][e];
                }
        }
        __syncthreads();
    }

    double* Rp = dynd;                  // kPanelI x pst: rows of R from column i0
    double* T = dynd + kPanelI * pst;   // kPanelI x pst: R(I, below) X(below, :)
    for (int i0 = ((ell - 1) / kPanelI) * kPanelI; i0 >= 0; i0 -= kPanelI) {
        const int kb = min(kPanelI, ell - i0), w = ell - i0, nc = w - kb;
        for (int r = grp; r < kPanelI; r += NG) {
            double* dst = Rp + r * pst;
            const int c0 = r < kb ? r : w;
            for (int c = lane; c < c0; c += 64) dst[c] = 0.0;
            row_to_lds(dst, W + (int64_t)(i0 + r) * ld + i0, c0, w, lane);
        }
        __syncthreads();
        for (int q = tid; q < (kPanelI / 4) * nc; q += NT) {
            const int g = q / nc, jc = q - g * nc;
            const double* r0 = Rp + 4 * g * pst + kb;
            const double* xc = X + (int64_t)(i0 + kb) * ld + i0 + kb + jc;  // X(i0 + kb + u, j) = xc[u ld]
            double acc[4] = {0.0, 0.0, 0.0, 0.0};
            // Eight independent loads in flight per thread: the column of X
            // comes from L2, one latency per eight rows.
            int u = 0;
            for (; u + 8 <= jc + 1; u += 8) {
                double xv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) xv[e] = xc[(int64_t)(u + e) * ld];
#pragma unroll
                for (int e = 0; e < 8; ++e)
#pragma unroll
                    for (int a = 0; a < 4; ++a) acc[a] += r0[a * pst + u + e] * xv[e];
            }
            for (; u <= jc; ++u) {
                const double x = xc[(int64_t)u * ld];
#pragma unroll
                for (int a = 0; a < 4; ++a) acc[a] += r0[a * pst + u] * x;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) T[(4 * g + a) * pst + jc] = acc[a];
        }
        __syncthreads();
        for (int jc = tid; jc < w; jc += NT) {
            double x[kPanelI];
#pragma unroll
            for (int r = kPanelI - 1; r >= 0; --r) {
                double s = 0.0;
                if (r < kb) {
                    s = (jc == r ? 1.0 : 0.0) - (jc >= kb ? T[r * pst + jc - kb] : 0.0);
#pragma unroll
                    for (int r2 = r + 1; r2 < kPanelI; ++r2) s -= Rp[r * pst + r2] * x[r2];
                    s *= inv_diag[i0 + r];
                }
                x[r] = s;
            }
#pragma unroll
            for (int r = 0; r < kPanelI; ++r)
                if (r < kb && r <= jc) {
                    X[(int64_t)(i0 + r) * ld + i0 + jc] = x[r];
                    out[(int64_t)(i0 + r) * ell_pad + i0 + jc] = (float)x[r];
                }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------- M^T V ----
// out(c, j) = sum_d M(d, c) V(d, j), d < l, c < l_pad, j < len.  Block: a
// 64 (c) x 128 (j) output tile, 256 threads of 4 c x 8 j each (j in two runs
// of four, 64 apart, so a row of the tile is 16 threads x 16 B contiguous).
// The l dimension runs in chunks of 16 staged through LDS, the next chunk's
// global loads in flight during the current chunk's FMAs.  Every d sums in
// increasing order, one fp32 FMA per term.  len and the row strides of V and
// the outputs are multiples of 128 (the 256-padded matrix sides), l_pad of 64.
constexpr int kSmBM = 64, kSmBN = 128, kSmBK = 16;

__global__ void __launch_bounds__(256) small_mul_kernel(SmallMulArgs args) {
    const int z = blockIdx.z;
    const int g = item_of(args, z), lz = z - args.zbeg[g];
    const SmallMulItem& a = args.it[g];
    const int64_t j0 = (int64_t)blockIdx.x * kSmBN;
    if (j0 >= a.len_pad) return;
    const int c0 = blockIdx.y * kSmBM;
    const int ell = args.ell, ell_pad = args.ell_pad;
    const int tid = threadIdx.x, tc = tid >> 4, tj = tid & 15;
    const float* M = a.mat + (int64_t)lz * ell_pad * ell_pad;
    const float* V = a.v + (int64_t)lz * a.stride_v;
    __shared__ float4 sm[kSmBK][kSmBM / 4];
    __shared__ float4 sv[kSmBK][kSmBN / 4];
    // Global -> register staging: one float4 of M, two of V per thread.
    const int mr = tid >> 4, mc = tid & 15;           // M: row, float4 column
    const int vr = tid >> 5, vc = tid & 31;           // V: rows vr, vr + 8
    float4 rm, rv0, rv1;
    auto load = [&](int d0) {
        const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
        const int dm = d0 + mr, dv0 = d0 + vr, dv1 = d0 + vr + 8;
        rm = dm < ell ? *(const float4*)(M + (int64_t)dm * ell_pad + c0 + 4 * mc) : zero;
        rv0 = dv0 < ell ? *(const float4*)(V + (int64_t)dv0 * a.ld_v + j0 + 4 * vc) : zero;
        rv1 = dv1 < ell ? *(const float4*)(V + (int64_t)dv1 * a.ld_v + j0 + 4 * vc) : zero;
    };
    auto stage = [&]() {
        sm[mr][mc] = rm;
        sv[vr][vc] = rv0;
        sv[vr + 8][vc] = rv1;
    };
    float acc[4][8];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[u][e] = 0.f;
    load(0);
    stage();
    __syncthreads();
    for (int d0 = 0; d0 < ell; d0 += kSmBK) {
        const bool more = d0 + kSmBK < ell;
        if (more) load(d0 + kSmBK);
#pragma unroll 4
        for (int dd = 0; dd < kSmBK; ++dd) {
            const float4 m4 = sm[dd][tc];
            const float4 va = sv[dd][tj], vb = sv[dd][16 + tj];
            const float mv[4] = {m4.x, m4.y, m4.z, m4.w};
            const float vv[8] = {va.x, va.y, va.z, va.w, vb.x, vb.y, vb.z, vb.w};
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[u][e] = fmaf(mv[u], vv[e], acc[u][e]);
        }
        if (more) {
            __syncthreads();
            stage();
            __syncthreads();
        }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int c = c0 + 4 * tc + u;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int64_t j = j0 + 64 * h + 4 * tj;
            const float* q = acc[u] + 4 * h;
            if (a.out32)
                *(float4*)(a.out32 + (int64_t)lz * a.stride_out32 + (int64_t)c * a.ld_v + j) =
                    make_float4(q[0], q[1], q[2], q[3]);
            if (a.out16) {
                half_t* o = a.out16 + (int64_t)lz * a.stride_out16 + (int64_t)c * a.ld_v + j;
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = (half_t)q[e];
            }
        }
    }
    if (a.out16t) {
        // len-major: row j holds l_pad consecutive c; four of them per store.
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int64_t j = j0 + 64 * h + 4 * tj + e;
                half_t* o = a.out16t + (int64_t)lz * a.stride_out16t + j * ell_pad + c0 + 4 * tc;
#pragma unroll
                for (int u = 0; u < 4; ++u) o[u] = (half_t)acc[u][4 * h + e];
            }
    }
}

// ------------------------------------------------------ Jacobi + select --
// Two-sided cyclic Jacobi with the round-robin pairing: every round rotates
// l/2 disjoint (p, q) pairs at once.  A round is one data-parallel phase: the
// 2 x 2 block of A on rows (p1, q1) and columns (p2, q2) becomes
// J1^T block J2 for every pair of pairs, and columns (p, q) of Z become Z J.
// A and Z live in LDS (row stride l + 1) when they fit, else in a global
// scratch slice.
constexpr int kEigLdsMax = 138;
// Packed mode: the upper triangle of A (rows packed) in LDS, Z^T in a global
// scratch slice; used above kEigLdsMax while l (l + 1) / 2 floats fit.
constexpr int kEigPackedMax = 278;

// Stopping rule of every Jacobi kernel, tested on the squared off-diagonal
// mass `off` against the squared Frobenius norm `tot`: converged below
// 1e-13 relative, or stalled at the fp32 rounding floor (already below 1e-9
// relative and less than a 4x drop over the last sweep; the quadratic phase
// drops it far more per sweep until rounding dominates).
__device__ __forceinline__ bool jacobi_done(float off, float tot, float prev_off) {
    return !(off > 1e-13f * tot) || (off <= 1e-9f * tot && off >= 0.25f * prev_off);
}

__device__ __forceinline__ void rr_pair(int round, int k, int n2, int& p, int& q) {
    const int n1 = n2 - 1;
    if (k == 0) { p = n1; q = round; }
    else { p = (round + k) % n1; q = (round - k + n1) % n1; }
    if (p > q) { const int t = p; p = q; q = t; }
}

template <int NT>
__device__ __forceinline__ float block_sum_f(float v, float* red) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) t += red[w];
    return t;
}

template <bool IN_LDS>
__global__ void __launch_bounds__(kSmallThreads) eig_select_kernel(EigArgs a) {
    constexpr int NT = kSmallThreads;
    extern __shared__ float dyn[];
    const int z = blockIdx.x, tid = threadIdx.x;
    const int n = a.ell, lp = a.ell_pad;
    const int ld = IN_LDS ? n + 1 : n;
    float* A;
    if constexpr (IN_LDS) A = dyn;
    else A = a.scratch + (int64_t)z * 2 * lp * lp;
    float* Z = A + n * ld;
    __shared__ float cs[192], sn[192];
    __shared__ int pp[192], qq[192];
    __shared__ float red[NT / 64];
    __shared__ float lam[384], fcoef[384];
    __shared__ int rnk[384];
    __shared__ int stop_flag;
    const double* part = a.partial + (int64_t)z * a.chunks * lp * lp;
    for (int q = tid; q < n * n; q += NT) {
        const int c = q / n, d = q - (q / n) * n;
        A[c * ld + d] = (float)gram_at(part, lp, c, d);
        Z[c * ld + d] = c == d ? 1.f : 0.f;
    }
    __syncthreads();
    const int n2 = n + (n & 1);
    const int npairs = n2 / 2;
    const int nblk = npairs * npairs;
    float prev_off = INFINITY;
    for (int sweep = 0; sweep < a.max_sweeps; ++sweep) {
        float off = 0.f, tot = 0.f;
        for (int q = tid; q < n * n; q += NT) {
            const int c = q / n, d = q - (q / n) * n;
            const float v = A[c * ld + d] * A[c * ld + d];
            tot += v;
            if (c != d) off += v;
        }
        off = block_sum_f<NT>(off, red);
        tot = block_sum_f<NT>(tot, red);
        if (tid == 0) stop_flag = jacobi_done(off, tot, prev_off);
        prev_off = off;
        __syncthreads();
        if (stop_flag) break;
        for (int round = 0; round < n2 - 1; ++round) {
            for (int k = tid; k < npairs; k += NT) {
                int p, q;
                rr_pair(round, k, n2, p, q);
                float c = 1.f, s = 0.f;
                if (q < n) {
                    const float apq = A[p * ld + q];
                    const float app = A[p * ld + p], aqq = A[q * ld + q];
                    if (fabsf(apq) > 1e-30f && fabsf(apq) > 1e-9f * sqrtf(fabsf(app * aqq))) {
                        const float theta = (aqq - app) / (2.f * apq);
                        float t;
                        if (fabsf(theta) > 1e15f) t = 0.5f / theta;
                        else t = copysignf(1.f, theta) / (fabsf(theta) + sqrtf(theta * theta + 1.f));
                        c = 1.f / sqrtf(t * t + 1.f);
                        s = t * c;
                    }
                }
                cs[k] = c; sn[k] = s; pp[k] = p; qq[k] = q;
            }
            __syncthreads();
            // A <- J^T A J, one 2 x 2 block per work item.
            for (int w = tid; w < nblk; w += NT) {
                const int k1 = w / npairs, k2 = w - k1 * npairs;
                const int p1 = pp[k1], q1 = qq[k1], p2 = pp[k2], q2 = qq[k2];
                const float c1 = cs[k1], s1 = sn[k1], c2 = cs[k2], s2 = sn[k2];
                const bool r1 = q1 < n, r2 = q2 < n;
                const float a00 = A[p1 * ld + p2];
                const float a01 = r2 ? A[p1 * ld + q2] : 0.f;
                const float a10 = r1 ? A[q1 * ld + p2] : 0.f;
                const float a11 = (r1 && r2) ? A[q1 * ld + q2] : 0.f;
                // rows: J1^T
                const float b00 = c1 * a00 - s1 * a10, b01 = c1 * a01 - s1 * a11;
                const float b10 = s1 * a00 + c1 * a10, b11 = s1 * a01 + c1 * a11;
                // columns: J2
                A[p1 * ld + p2] = c2 * b00 - s2 * b01;
                if (r2) A[p1 * ld + q2] = s2 * b00 + c2 * b01;
                if (r1) A[q1 * ld + p2] = c2 * b10 - s2 * b11;
                if (r1 && r2) A[q1 * ld + q2] = s2 * b10 + c2 * b11;
            }
            for (int w = tid; w < npairs * n; w += NT) {
                const int k = w / n, i = w - (w / n) * n;
                const int p = pp[k], q = qq[k];
                if (q >= n) continue;
                const float c = cs[k], s = sn[k];
                const float zp = Z[i * ld + p], zq = Z[i * ld + q];
                Z[i * ld + p] = c * zp - s * zq;
                Z[i * ld + q] = s * zp + c * zq;
            }
            __syncthreads();
        }
    }
    // Ritz values, descending order with ties to the lower index.
    for (int i = tid; i < n; i += NT) lam[i] = A[i * ld + i];
    __syncthreads();
    const int top = min(a.rank, n);
    for (int i = tid; i < n; i += NT) {
        const float li = lam[i];
        int r = 0;
        for (int j = 0; j < n; ++j) r += (lam[j] > li) || (lam[j] == li && j < i);
        rnk[i] = r;
        const bool sel = r < top && li > 1.f;
        fcoef[i] = sel ? (1.f / sqrtf(li) - 1.f) : 0.f;
        if (r < top) a.ritz[(int64_t)z * a.ritz_stride + r] = li;
    }
    __syncthreads();
    // K = Z diag(f) Z^T over the selected modes.
    float* K = a.kmat + (int64_t)z * lp * lp;
    for (int q = tid; q < lp * lp; q += NT) {
        const int c = q / lp, d = q - (q / lp) * lp;
        float s = 0.f;
        if (c < n && d < n)
            for (int i = 0; i < n; ++i)
                if (fcoef[i] != 0.f) s = fmaf(Z[c * ld + i] * fcoef[i], Z[d * ld + i], s);
        K[q] = s;
    }
    if (tid == 0) {
        int cnt = 0;
        for (int i = 0; i < n; ++i) cnt += (rnk[i] < top && lam[i] > 1.f);
        a.nsel[z] = cnt;
    }
}

// Index of (r, c) in the packed upper triangle of an n x n symmetric matrix.
__device__ __forceinline__ int pk(int r, int c, int n) {
    if (r > c) { const int t = r; r = c; c = t; }
    return r * n - (r * (r - 1)) / 2 + (c - r);
}

// The same Jacobi sweep, selection and K as eig_select_kernel, with A packed
// in LDS and Z stored transposed (row i = Ritz vector i) in global memory, so
// the rotation of columns p, q of Z updates two contiguous rows.  Only the
// pair-blocks (k1 <= k2) of the upper triangle are rotated; the diagonal
// block keeps its three distinct entries.
__global__ void __launch_bounds__(kSmallThreads) eig_select_packed_kernel(EigArgs a) {
    constexpr int NT = kSmallThreads;
    extern __shared__ float A[];
    const int z = blockIdx.x, tid = threadIdx.x;
    const int n = a.ell, lp = a.ell_pad;
    float* Zt = a.scratch + (int64_t)z * 2 * lp * lp;
    __shared__ float cs[192], sn[192];
    __shared__ int pp[192], qq[192];
    __shared__ float red[NT / 64];
    __shared__ float lam[384], fcoef[384];
    __shared__ int rnk[384];
    __shared__ int stop_flag;
    const double* part = a.partial + (int64_t)z * a.chunks * lp * lp;
    for (int q = tid; q < n * n; q += NT) {
        const int c = q / n, d = q - (q / n) * n;
        if (c <= d) A[pk(c, d, n)] = (float)gram_at(part, lp, c, d);
        Zt[(int64_t)c * lp + d] = c == d ? 1.f : 0.f;
    }
    __syncthreads();
    const int n2 = n + (n & 1);
    const int npairs = n2 / 2;
    float prev_off = INFINITY;
    for (int sweep = 0; sweep < a.max_sweeps; ++sweep) {
        float off = 0.f, tot = 0.f;
        for (int q = tid; q < n * n; q += NT) {
            const int c = q / n, d = q - (q / n) * n;
            if (c > d) continue;
            const float v = A[pk(c, d, n)] * A[pk(c, d, n)];
            tot += c == d ? v : 2.f * v;
            if (c != d) off += 2.f * v;
        }
        off = block_sum_f<NT>(off, red);
        tot = block_sum_f<NT>(tot, red);
        if (tid == 0) stop_flag = jacobi_done(off, tot, prev_off);
        prev_off = off;
        __syncthreads();
        if (stop_flag) break;
        for (int round = 0; round < n2 - 1; ++round) {
            for (int k = tid; k < npairs; k += NT) {
                int p, q;
                rr_pair(round, k, n2, p, q);
                float c = 1.f, s = 0.f;
                if (q < n) {
                    const float apq = A[pk(p, q, n)];
                    const float app = A[pk(p, p, n)], aqq = A[pk(q, q, n)];
                    if (fabsf(apq) > 1e-30f && fabsf(apq) > 1e-9f * sqrtf(fabsf(app * aqq))) {
                        const float theta = (aqq - app) / (2.f * apq);
                        float t;
                        if (fabsf(theta) > 1e15f) t = 0.5f / theta;
                        else t = copysignf(1.f, theta) / (fabsf(theta) + sqrtf(theta * theta + 1.f));
                        c = 1.f / sqrtf(t * t + 1.f);
                        s = t * c;
                    }
                }
                cs[k] = c; sn[k] = s; pp[k] = p; qq[k] = q;
            }
            __syncthreads();
            for (int w = tid; w < npairs * npairs; w += NT) {
                const int k1 = w / npairs, k2 = w - k1 * npairs;
                if (k1 > k2) continue;
                const int p1 = pp[k1], q1 = qq[k1], p2 = pp[k2], q2 = qq[k2];
                const float c1 = cs[k1], s1 = sn[k1], c2 = cs[k2], s2 = sn[k2];
                const bool r1 = q1 < n, r2 = q2 < n;
                const float a00 = A[pk(p1, p2, n)];
                const float a01 = r2 ? A[pk(p1, q2, n)] : 0.f;
                const float a10 = r1 ? A[pk(q1, p2, n)] : 0.f;
                const float a11 = (r1 && r2) ? A[pk(q1, q2, n)] : 0.f;
                const float b00 = c1 * a00 - s1 * a10, b01 = c1 * a01 - s1 * a11;
                const float b10 = s1 * a00 + c1 * a10, b11 = s1 * a01 + c1 * a11;
                A[pk(p1, p2, n)] = c2 * b00 - s2 * b01;
                if (r2) A[pk(p1, q2, n)] = s2 * b00 + c2 * b01;
                // (q1, p2) is the same stored entry as (p1, q2) on the diagonal block
                if (r1 && k1 != k2) A[pk(q1, p2, n)] = c2 * b10 - s2 * b11;
                if (r1 && r2) A[pk(q1, q2, n)] = s2 * b10 + c2 * b11;
            }
            // Z^T rows p, q <- rotated; ZB items per thread per batch keep
            // several global loads in flight.
            constexpr int ZB = 8;
            const int zitems = npairs * n;
            for (int w0 = tid; w0 < zitems; w0 += NT * ZB) {
                float vp[ZB], vq[ZB];
                int64_t op[ZB], oq[ZB];
                float cz[ZB], sz[ZB];
#pragma unroll
                for (int b = 0; b < ZB; ++b) {
                    const int w = w0 + b * NT;
                    op[b] = -1;
                    if (w < zitems) {
                        const int k = w / n, i = w - (w / n) * n;
                        if (qq[k] < n) {
                            op[b] = (int64_t)pp[k] * lp + i;
                            oq[b] = (int64_t)qq[k] * lp + i;
                            cz[b] = cs[k];
                            sz[b] = sn[k];
                            vp[b] = Zt[op[b]];
                            vq[b] = Zt[oq[b]];
                        }
                    }
                }
#pragma unroll
                for (int b = 0; b < ZB; ++b) {
                    if (op[b] < 0) continue;
                    Zt[op[b]] = cz[b] * vp[b] - sz[b] * vq[b];
                    Zt[oq[b]] = sz[b] * vp[b] + cz[b] * vq[b];
                }
            }
            __syncthreads();
        }
    }
    for (int i = tid; i < n; i += NT) lam[i] = A[pk(i, i, n)];
    __syncthreads();
    const int top = min(a.rank, n);
    for (int i = tid; i < n; i += NT) {
        const float li = lam[i];
        int r = 0;
        for (int j = 0; j < n; ++j) r += (lam[j] > li) || (lam[j] == li && j < i);
        rnk[i] = r;
        const bool sel = r < top && li > 1.f;
        fcoef[i] = sel ? (1.f / sqrtf(li) - 1.f) : 0.f;
        if (r < top) a.ritz[(int64_t)z * a.ritz_stride + r] = li;
    }
    __syncthreads();
    // K = sum_i f_i z_i z_i^T, with the rows of Z^T staged through the LDS that
    // held A, CH rows at a time (K accumulated in place across chunks).
    float* K = a.kmat + (int64_t)z * lp * lp;
    const int CH = (n + 1) / 2;
    for (int i0 = 0; i0 < n; i0 += CH) {
        const int cnt = min(CH, n - i0);
        for (int q = tid; q < cnt * n; q += NT) {
            const int i = q / n, c = q - (q / n) * n;
            A[q] = Zt[(int64_t)(i0 + i) * lp + c];
        }
        __syncthreads();
        for (int q = tid; q < lp * lp; q += NT) {
            const int c = q / lp, d = q - (q / lp) * lp;
            float s = i0 == 0 ? 0.f : K[q];
            if (c < n && d < n)
                for (int i = 0; i < cnt; ++i) {
                    const float f = fcoef[i0 + i];
                    if (f != 0.f) s = fmaf(A[i * n + c] * f, A[i * n + d], s);
                }
            K[q] = s;
        }
        __syncthreads();
    }
    if (tid == 0) {
        int cnt = 0;
        for (int i = 0; i < n; ++i) cnt += (rnk[i] < top && lam[i] > 1.f);
        a.nsel[z] = cnt;
    }
}

// Round-robin Jacobi for l <= kEigRRMax with A double-buffered in LDS: a
// round reads the current A and writes J^T A J into the other buffer, and
// each thread derives the rotations of its own pair-blocks from the current
// A with the same arithmetic the pair's diagonal block uses, so a round
// needs one barrier instead of two.  The columns of Z take round r's
// rotations during round r + 1 (published by the diagonal blocks, double
// buffered by round parity).  The off-diagonal mass is summed while the last
// round of a sweep is written, so the stopping test costs no extra pass.
// Arithmetic per rotation, the stopping rule, selection and K are those of
// eig_select_kernel.
constexpr int kEigRRMax = 104;

__device__ __forceinline__ void rr_pair_fast(int round, int k, int n1, int& p, int& q) {
    if (k == 0) {
        p = n1; q = round;
    } else {
        p = round + k;
        if (p >= n1) p -= n1;
        q = round - k;
        if (q < 0) q += n1;
    }
    if (p > q) { const int t = p; p = q; q = t; }
}

// Rotation (c, s) that zeroes a_pq (Rutishauser's tangent form), or the
// identity below the same threshold as the other Jacobi kernels.  Hardware
// reciprocal / square-root approximations: the rotation only has to be
// orthogonal to fp32 precision, which rsq keeps (c^2 + s^2 = 1 to ~1 ulp),
// and every thread that needs a pair's rotation computes it with the same
// instructions from the same operands.
__device__ __forceinline__ void jacobi_rotation_fast(float app, float aqq, float apq, bool real, float& c, float& s) {
    const float aa = fabsf(apq);
    const bool rot = real && aa > 1e-30f && aa > 1e-9f * __builtin_amdgcn_sqrtf(fabsf(app * aqq));
    const float theta = (aqq - app) * 0.5f * __builtin_amdgcn_rcpf(apq);
    const float at = fabsf(theta);
    const float t = copysignf(__builtin_amdgcn_rcpf(at + __builtin_amdgcn_sqrtf(fmaf(at, at, 1.f))), theta);
    const float cc = __builtin_amdgcn_rsqf(fmaf(t, t, 1.f));
    c = rot ? cc : 1.f;
    s = rot ? t * cc : 0.f;
}

template <int NT, int NB, int NZ>
__global__ void __launch_bounds__(NT) eig_select_rr_kernel(EigArgs a) {
    extern __shared__ float dyn[];
    const int z = blockIdx.x, tid = threadIdx.x;
    const int n = a.ell, lp = a.ell_pad, ld = n + 1;
    // Two n x (n + 1) buffers for A and one for Z; the padding column n
    // absorbs the phantom index of odd n (reads there are masked, writes
    // are identity rotations).
    float* Ac = dyn;
    float* An = dyn + n * ld;
    float* Z = dyn + 2 * n * ld;
    // Rotation of each pair, published by its diagonal block: (c, s, p, q).
    __shared__ float4 rec[2][kEigRRMax / 2 + 1];
    __shared__ float red[2][2][NT / 64];
    __shared__ float lam[kEigRRMax], fcoef[kEigRRMax];
    __shared__ int rnk[kEigRRMax];
    const double* part = a.partial + (int64_t)z * a.chunks * lp * lp;
    for (int q = tid; q < n * ld; q += NT) {
        const int c = q / ld, d = q - (q / ld) * ld;
        Ac[q] = d < n ? (float)gram_at(part, lp, c, d) : 0.f;
        Z[q] = c == d ? 1.f : 0.f;
    }
    const int n2 = n + (n & 1), n1 = n2 - 1, npairs = n2 / 2;
    const int ub = npairs * (npairs + 1) / 2;
    // This thread's pair-blocks (k1 <= k2) and Z items (pair k, row i).
    int bk1[NB], bk2[NB], zk[NZ], zi[NZ];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        int w = tid + j * NT, k1 = -1, k2 = -1;
        if (w < ub) {
            k1 = 0;
            while (w >= npairs - k1) { w -= npairs - k1; ++k1; }
            k2 = k1 + w;
        }
        bk1[j] = k1;
        bk2[j] = k2;
    }
#pragma unroll
    for (int j = 0; j < NZ; ++j) {
        const int w = tid + j * NT;
        zk[j] = w < npairs * n ? w / n : -1;
        zi[j] = w < npairs * n ? w - (w / n) * n : 0;
    }
    __syncthreads();
    int gr = 0;             // rounds done (parity of the published rotations)
    const int lane = tid & 63, wave = tid >> 6;
    // Columns p, q of Z take the rotations published in round gr - 1.
    auto rotate_z = [&](int par) {
#pragma unroll
        for (int j = 0; j < NZ; ++j) {
            if (zk[j] < 0) break;
            const float4 r = rec[par][zk[j]];
            const int p = __float_as_int(r.z), q = __float_as_int(r.w), i = zi[j];
            const float za = Z[i * ld + p], zb = Z[i * ld + q];
            Z[i * ld + p] = r.x * za - r.y * zb;
            Z[i * ld + q] = r.y * za + r.x * zb;
        }
    };
    float prev_off = INFINITY;
    for (int sweep = 0; sweep < a.max_sweeps; ++sweep) {
        float off = 0.f, tot = 0.f;
        for (int round = 0; round < n1; ++round, ++gr) {
            const bool last = round == n1 - 1;
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int k1 = bk1[j], k2 = bk2[j];
                if (k1 < 0) break;
                int p1, q1, p2, q2;
                rr_pair_fast(round, k1, n1, p1, q1);
                rr_pair_fast(round, k2, n1, p2, q2);
                const bool r1 = q1 < n, r2 = q2 < n;
                const int u1 = min(q1, n - 1), u2 = min(q2, n - 1);
                // Every read of the block first, then the rotations.
                const float x0 = Ac[p1 * ld + p1], x1 = Ac[u1 * ld + u1], x2 = Ac[p1 * ld + u1];
                const float x3 = Ac[p2 * ld + p2], x4 = Ac[u2 * ld + u2], x5 = Ac[p2 * ld + u2];
                const float x6 = Ac[p1 * ld + p2], x7 = Ac[p1 * ld + u2];
                const float x8 = Ac[u1 * ld + p2], x9 = Ac[u1 * ld + u2];
                if (j == 0 && gr > 0) rotate_z((gr - 1) & 1);
                float c1, s1, c2, s2;
                jacobi_rotation_fast(x0, x1, x2, r1, c1, s1);
                jacobi_rotation_fast(x3, x4, x5, r2, c2, s2);
                if (k2 == k1) rec[gr & 1][k1] = make_float4(c1, s1, __int_as_float(p1), __int_as_float(q1));
                const float a00 = x6, a01 = r2 ? x7 : 0.f;
                const float a10 = r1 ? x8 : 0.f, a11 = (r1 && r2) ? x9 : 0.f;
                const float b00 = c1 * a00 - s1 * a10, b01 = c1 * a01 - s1 * a11;
                const float b10 = s1 * a00 + c1 * a10, b11 = s1 * a01 + c1 * a11;
                const float d00 = c2 * b00 - s2 * b01, d01 = s2 * b00 + c2 * b01;
                const float d10 = c2 * b10 - s2 * b11, d11 = s2 * b10 + c2 * b11;
                An[p1 * ld + p2] = d00;
                if (r2) An[p1 * ld + q2] = d01;
                if (r1) An[q1 * ld + p2] = d10;
                if (r1 && r2) An[q1 * ld + q2] = d11;
                if (k2 != k1) {
                    An[p2 * ld + p1] = d00;
                    if (r2) An[q2 * ld + p1] = d01;
                    if (r1) An[p2 * ld + q1] = d10;
                    if (r1 && r2) An[q2 * ld + q1] = d11;
                }
                if (last) {
                    const float e00 = d00 * d00, e01 = r2 ? d01 * d01 : 0.f;
                    const float e10 = r1 ? d10 * d10 : 0.f, e11 = (r1 && r2) ? d11 * d11 : 0.f;
                    if (k2 != k1) {
                        const float m = 2.f * (e00 + e01 + e10 + e11);
                        off += m;
                        tot += m;
                    } else {
                        off += e01 + e10;
                        tot += e00 + e01 + e10 + e11;
                    }
                }
            }
            // Threads without a pair-block still rotate their Z items.
            if (bk1[0] < 0 && gr > 0) rotate_z((gr - 1) & 1);
            if (last) {
#pragma unroll
                for (int o = 32; o >= 1; o >>= 1) {
                    off += __shfl_xor(off, o, 64);
                    tot += __shfl_xor(tot, o, 64);
                }
                if (lane == 0) {
                    red[sweep & 1][0][wave] = off;
                    red[sweep & 1][1][wave] = tot;
                }
            }
            __syncthreads();
            float* t = Ac; Ac = An; An = t;
        }
        float so = 0.f, st = 0.f;
#pragma unroll
        for (int w = 0; w < NT / 64; ++w) {
            so += red[sweep & 1][0][w];
            st += red[sweep & 1][1][w];
        }
        if (jacobi_done(so, st, prev_off)) break;
        prev_off = so;
    }
    if (gr > 0) rotate_z((gr - 1) & 1);
    // Ritz values, descending order with ties to the lower index.
    for (int i = tid; i < n; i += NT) lam[i] = Ac[i * ld + i];
    __syncthreads();
    const int top = min(a.rank, n);
    for (int i = tid; i < n; i += NT) {
        const float li = lam[i];
        int r = 0;
        for (int j = 0; j < n; ++j) r += (lam[j] > li) || (lam[j] == li && j < i);
        rnk[i] = r;
        const bool sel = r < top && li > 1.f;
        fcoef[i] = sel ? (1.f / sqrtf(li) - 1.f) : 0.f;
        if (r < top) a.ritz[(int64_t)z * a.ritz_stride + r] = li;
    }
    __syncthreads();
    // K = Z diag(f) Z^T over the selected modes.
    float* K = a.kmat + (int64_t)z * lp * lp;
    for (int q = tid; q < lp * lp; q += NT) {
        const int c = q / lp, d = q - (q / lp) * lp;
        float s = 0.f;
        if (c < n && d < n)
            for (int i = 0; i < n; ++i)
                if (fcoef[i] != 0.f) s = fmaf(Z[c * ld + i] * fcoef[i], Z[d * ld + i], s);
        K[q] = s;
    }
    if (tid == 0) {
        int cnt = 0;
        for (int i = 0; i < n; ++i) cnt += (rnk[i] < top && lam[i] > 1.f);
        a.nsel[z] = cnt;
    }
}

}  // namespace

hipError_t launch_omega_f16(const OmegaArgs& a, int batch, hipStream_t s) {
    const int64_t total = (int64_t)a.ell_pad * a.ld;
    const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(omega_f16_kernel, dim3(blocks, batch), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_omega_f32(uint64_t seed, int64_t step, int id, int64_t b, int ell, float* out, hipStream_t s) {
    const int64_t total = b * ell;
    const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
    hipLaunchKernelGGL(omega_f32_kernel, dim3(blocks), dim3(256), 0, s, seed, step, (uint32_t)id, b, ell, out);
    return hipGetLastError();
}

hipError_t launch_reduce_splits(const float* part, int splits, int64_t stride_split, int64_t stride_mat, int rows,
                                int64_t len, float* out32, half_t* out16, float scale16, int64_t stride_out,
                                int batch, hipStream_t s) {
    if (len % 4 || stride_split % 4) return hipErrorInvalidValue;
    const int64_t n4 = (int64_t)rows * len / 4;
    const unsigned blocks = (unsigned)std::min<int64_t>((n4 + 255) / 256, 2048);
    hipLaunchKernelGGL(reduce_splits_kernel, dim3(blocks, batch), dim3(256), 0, s, part, splits, stride_split,
                       stride_mat, n4, out32, out16, scale16, stride_out);
    return hipGetLastError();
}

hipError_t launch_reduce_splits_grouped(const ReduceGroups& g, hipStream_t s) {
    if (g.n < 1 || g.n > kMaxItems || g.zbeg[0] != 0) return hipErrorInvalidValue;
    int64_t n4 = 0;
    for (int i = 0; i < g.n; ++i) {
        if (g.zbeg[i + 1] <= g.zbeg[i] || g.splits[i] < 1 || g.stride_split[i] % 4 || g.n4[i] < 1)
            return hipErrorInvalidValue;
        n4 = std::max(n4, g.n4[i]);
    }
    const unsigned blocks = (unsigned)std::min<int64_t>((n4 + 255) / 256, 2048);
    hipLaunchKernelGGL(reduce_splits_grouped_kernel, dim3(blocks, g.zbeg[g.n]), dim3(256), 0, s, g);
    return hipGetLastError();
}

int gram64_chunks(int64_t len, int chunk_len) { return (int)((len + chunk_len - 1) / chunk_len); }

hipError_t launch_gram64(const Gram64Items& t, int ell_pad, double* partial, hipStream_t s) {
    if (ell_pad % 64 || t.ell < 1 || t.ell > ell_pad || t.n < 1 || t.n > kMaxItems || t.zbeg[0] != 0)
        return hipErrorInvalidValue;
    for (int g = 0; g < t.n; ++g)
        if (t.chunk_len[g] % 64 || t.len[g] % 64 || t.ld[g] % 4 ||
            gram64_chunks(t.len[g], t.chunk_len[g]) > kGramChunks || t.zbeg[g + 1] <= t.zbeg[g])
            return hipErrorInvalidValue;
    const int tiles = ell_pad / 64;
    dim3 grid(tiles * (tiles + 1) / 2, kGramChunks, t.zbeg[t.n]);
    hipLaunchKernelGGL(gram64_kernel, grid, dim3(256), 0, s, t, ell_pad, partial);
    return hipGetLastError();
}

hipError_t launch_chol_inv(const double* partial, int chunks, int ell, int ell_pad, double* scratch, float* rinv,
                           int batch, hipStream_t s) {
    if (ell < 1 || ell > 384 || ell_pad < ell || ell_pad > 384 || chunks != kGramChunks) return hipErrorInvalidValue;
    if (ell <= kCholLdsMax) {
        const size_t lds = (size_t)(ell + 1) * (ell + 1) * sizeof(double);
        hipLaunchKernelGGL(chol_inv_kernel<kCholLdsThreads>, dim3(batch), dim3(kCholLdsThreads), lds, s, partial,
                           chunks, ell, ell_pad, rinv);
    } else {
        const size_t lds = (size_t)std::max(kPanelC, 2 * kPanelI) * (ell + 1) * sizeof(double);
        hipLaunchKernelGGL(chol_inv_panel_kernel, dim3(batch), dim3(kCholThreads), lds, s, partial, chunks, ell,
                           ell_pad, scratch, rinv);
    }
    return hipGetLastError();
}

hipError_t launch_small_mul(const SmallMulArgs& a, hipStream_t s) {
    if (a.n < 1 || a.n > kMaxItems || a.zbeg[0] != 0) return hipErrorInvalidValue;
    if (a.ell < 1 || a.ell > a.ell_pad || a.ell_pad % kSmBM) return hipErrorInvalidValue;
    int64_t len_pad = 0;
    for (int g = 0; g < a.n; ++g) {
        const SmallMulItem& m = a.it[g];
        if (a.zbeg[g + 1] <= a.zbeg[g] || m.len_pad % kSmBN || m.ld_v % kSmBN || m.ld_v < m.len_pad)
            return hipErrorInvalidValue;
        len_pad = std::max(len_pad, m.len_pad);
    }
    dim3 grid((unsigned)(len_pad / kSmBN), (unsigned)(a.ell_pad / kSmBM), a.zbeg[a.n]);
    hipLaunchKernelGGL(small_mul_kernel, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_eig_select(const EigArgs& a, int batch, hipStream_t s) {
    if (a.ell > 384 || a.ell_pad > 384 || a.chunks != kGramChunks) return hipErrorInvalidValue;
    if (a.ell <= kEigRRMax) {
        const size_t lds = (size_t)3 * a.ell * (a.ell + 1) * sizeof(float);
        if (a.ell <= 64)
            hipLaunchKernelGGL((eig_select_rr_kernel<1024, 1, 2>), dim3(batch), dim3(1024), lds, s, a);
        else
            hipLaunchKernelGGL((eig_select_rr_kernel<1024, 2, 6>), dim3(batch), dim3(1024), lds, s, a);
    } else if (a.ell <= kEigLdsMax) {
        const size_t lds = (size_t)2 * a.ell * (a.ell + 1) * sizeof(float);
        hipLaunchKernelGGL((eig_select_kernel<true>), dim3(batch), dim3(kSmallThreads), lds, s, a);
    } else if (a.ell <= kEigPackedMax) {
        const size_t lds = (size_t)a.ell * (a.ell + 1) / 2 * sizeof(float);
        hipLaunchKernelGGL(eig_select_packed_kernel, dim3(batch), dim3(kSmallThreads), lds, s, a);
    } else {
        hipLaunchKernelGGL((eig_select_kernel<false>), dim3(batch), dim3(kSmallThreads), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace np
