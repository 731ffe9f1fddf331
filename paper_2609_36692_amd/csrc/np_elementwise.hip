// Streaming (HBM-bound) kernels of the NormPre step for gfx950:
//   * momentum + relaxed tangent + diagonal-Gram normalization (Alg. 1;
//     Sec. 3.1 for the tangent, Eq. 2 for Psi = D(X)^{-1} X), in the
//     row-active (k = 0) and column-active (k = 1) orientations;
//   * the Newton-Schulz pre-scale 1 / (||Psi||_F + eps);
//   * the NormPre-G RMS-matched weight update (Sec. 3.1, "Consistent
//     Update RMS", and the last line of Alg. 1).
//
// x = m - c w with c = <m, w> (the relaxed tangent of Sec. 3.1; the ablation
// modes of App. A.4 use c = 0, no tangent, or c = <m, w> / ||w||^2, the strict
// tangent projection) is formed in fp64 from the fp32 values, so a nearly
// radial momentum (m close to a multiple of w) loses no accuracy beyond the
// fp32 rounding of the stored M.  Row-active: the row stays in registers;
// one pass gives <m, w> and ||w||^2, a second one ||x||^2 from the formed x,
// a third writes Psi.  Column-active: one streaming pass gives ||m||^2,
// <m, w>, ||w||^2 per column (fp64), ||x||^2 follows from
//   ||x||^2 = ||m||^2 - 2 c <m, w> + c^2 ||w||^2
// (relative error about u64 K ||m||^2 / ||x||^2 for K summed terms, far
// below the fp32 rounding of M unless ||x|| < 1e-6 ||m||), and a second,
// cache-friendly pass writes Psi.
//
// Also the input of the Muon reference step (Sec. 2.1): momentum update with
// per-block sums of M^2, then X0 = M / (||M||_F + eps) cast to fp16.
#include "np_internal.h"

namespace np {
namespace {

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}
__device__ __forceinline__ float wave_sum_f(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Coefficient c of x = m - c w for the momentum-processing mode.
__device__ __forceinline__ double tangent_coef(int mode, double smw, double sww) {
    if (mode == kTangentNone) return 0.0;
    if (mode == kTangentStrict) return sww > 0.0 ? smw / sww : 0.0;
    return smw;
}

// Block-wide sums (fixed order); results valid in every thread.  The two
// helpers own separate LDS arrays, so one may follow the other without a
// barrier in between.
template <int NT>
__device__ __forceinline__ void block_sum2(double& a, double& b) {
    __shared__ double red2[2][NT / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    a = wave_sum_d(a);
    b = wave_sum_d(b);
    if (lane == 0) { red2[0][wave] = a; red2[1][wave] = b; }
    __syncthreads();
    a = b = 0.0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) { a += red2[0][w]; b += red2[1][w]; }
}
template <int NT>
__device__ __forceinline__ void block_sum1(double& a) {
    __shared__ double red1[NT / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    a = wave_sum_d(a);
    if (lane == 0) red1[wave] = a;
    __syncthreads();
    a = 0.0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) a += red1[w];
}

// x = m - c w in fp64.
__device__ __forceinline__ double tangent_x(float m, float w, double c) { return fma(-c, (double)w, (double)m); }

// Finite check: a non-finite value counts as zero, and is counted.
__device__ __forceinline__ float finite_or_zero(float v, int& bad) {
    const bool ok = __builtin_isfinite(v);
    bad += ok ? 0 : 1;
    return ok ? v : 0.f;
}

// One VW-wide piece of a row: M <- mu M_prev + G (stored), the new m and w
// kept for the statistics.  With the finite check, non-finite M_prev and G
// entries count as zero (and the stored M is finite), non-finite W entries
// count as zero in the tangent; `bad` counts all three.
template <int VW>
__device__ __forceinline__ void load_row_piece(const NormArgs& a, float* M, const float* G, const float* W, int idx,
                                               float (&mv)[VW], float (&wv)[VW], int& bad, int64_t base = 0) {
    M += base;
    G += base;
    W += base;
    float mp[VW], g[VW], w[VW];
    if constexpr (VW == 4) {
        const float4 mp4 = *reinterpret_cast<const float4*>(M + idx);
        const float4 g4 = *reinterpret_cast<const float4*>(G + idx);
        const float4 w4 = *reinterpret_cast<const float4*>(W + idx);
        mp[0] = mp4.x; mp[1] = mp4.y; mp[2] = mp4.z; mp[3] = mp4.w;
        g[0] = g4.x; g[1] = g4.y; g[2] = g4.z; g[3] = g4.w;
        w[0] = w4.x; w[1] = w4.y; w[2] = w4.z; w[3] = w4.w;
    } else {
        mp[0] = M[idx];
        g[0] = G[idx];
        w[0] = W[idx];
    }
    if (a.nfin) {
#pragma unroll
        for (int e = 0; e < VW; ++e) {
            mp[e] = finite_or_zero(mp[e], bad);
            g[e] = finite_or_zero(g[e], bad);
            w[e] = finite_or_zero(w[e], bad);
        }
    }
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        mv[e] = fmaf(a.mu, mp[e], g[e]);
        wv[e] = w[e];
    }
    if constexpr (VW == 4) *reinterpret_cast<float4*>(M + idx) = make_float4(mv[0], mv[1], mv[2], mv[3]);
    else M[idx] = mv[0];
}

// ---------------------------------------------------------------------------
// Row-active orientation: one block per row of W; the row of M and W stays in
// registers between the statistics and the Psi store.  VW = vector width
// (4 when cols % 4 == 0), NV = vectors per thread.
template <int NT, int VW, int NV, bool DBG>
__global__ void __launch_bounds__(NT) normalize_rows_kernel(NormArgs a) {
    const int z = blockIdx.y, row = blockIdx.x, tid = threadIdx.x;
    half_t* prow = a.psi + (int64_t)z * a.stride_psi + (int64_t)row * a.ld_psi;
    if (row >= a.rows) {
        for (int64_t j = tid; j < a.ld_psi; j += NT) prow[j] = (half_t)0.f;
        return;
    }
    const int64_t off = (int64_t)row * a.cols;
    float* W = a.ptrs.w[z] + off;
    float* M = a.ptrs.m[z] + off;
    const float* G = a.ptrs.g[z] + off;
    float mv[NV][VW], wv[NV][VW];
    double smw = 0.0, sww = 0.0;
    int bad = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int idx = (v * NT + tid) * VW;
        if (idx < a.cols) {
            load_row_piece<VW>(a, M, G, W, idx, mv[v], wv[v], bad);
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                const double md = mv[v][e], wd = wv[v][e];
                smw = fma(md, wd, smw);
                sww = fma(wd, wd, sww);
            }
        }
    }
    if (a.nfin) {
        double b = bad;
        block_sum1<NT>(b);
        if (tid == 0) a.nfin[(int64_t)z * a.stride_nfin + row] = (int)b;
        __syncthreads();   // the second block_sum1 below reuses its LDS
    }
    block_sum2<NT>(smw, sww);
    const double d = tangent_coef(a.tangent, smw, sww);
    // x replaces m in the registers (rounded to fp32 after it is formed, so
    // its relative error is u32 whatever the cancellation was).
    double nrm2 = 0.0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
        if ((v * NT + tid) * VW < a.cols) {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                const double x = tangent_x(mv[v][e], wv[v][e], d);
                nrm2 = fma(x, x, nrm2);
                mv[v][e] = (float)x;
            }
        }
    block_sum1<NT>(nrm2);
    const double inv = 1.0 / fmax(sqrt(nrm2), (double)a.eps);
    const float invf = (float)inv;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int idx = (v * NT + tid) * VW;
        if (idx < a.cols) {
            float p[VW];
#pragma unroll
            for (int e = 0; e < VW; ++e) p[e] = mv[v][e] * invf;
            if constexpr (VW == 4) {
                half_t h[4] = {(half_t)p[0], (half_t)p[1], (half_t)p[2], (half_t)p[3]};
                *reinterpret_cast<uint2*>(prow + idx) = *reinterpret_cast<const uint2*>(h);
                if constexpr (DBG)
                    *reinterpret_cast<float4*>(a.psi32 + (int64_t)z * a.stride_psi32 + off + idx) =
                        make_float4(p[0], p[1], p[2], p[3]);
            } else {
                prow[idx] = (half_t)p[0];
                if constexpr (DBG) a.psi32[(int64_t)z * a.stride_psi32 + off + idx] = p[0];
            }
        }
    }
    for (int64_t j = a.cols + tid; j < a.ld_psi; j += NT) prow[j] = (half_t)0.f;
    if (tid == 0) {
        a.psisq[(int64_t)z * a.stride_psisq + row] = (float)(nrm2 * inv * inv);
        if (a.xsq) a.xsq[(int64_t)z * a.stride_psisq + row] = (float)nrm2;
    }
}

// ---------------------------------------------------------------------------
// Row-active orientation, rows of at most 64 * VW * NV elements: one wave per
// row, four rows per block; the row stays in registers and the statistics are
// reduced with wave shuffles only (no LDS, no block barrier).
template <int VW, int NV, bool DBG>
__global__ void __launch_bounds__(256) normalize_rows_wave_kernel(NormArgs a) {
    const int z = blockIdx.y, lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= a.rows_pad) return;
    half_t* prow = a.psi + (int64_t)z * a.stride_psi + (int64_t)row * a.ld_psi;
    if (row >= a.rows) {
        for (int64_t j = lane * 4; j < a.ld_psi; j += 256)
            *reinterpret_cast<uint2*>(prow + j) = make_uint2(0u, 0u);
        return;
    }
    const int64_t off = (int64_t)row * a.cols;
    float* W = a.ptrs.w[z] + off;
    float* M = a.ptrs.m[z] + off;
    const float* G = a.ptrs.g[z] + off;
    float mv[NV][VW], wv[NV][VW];
    double smw = 0.0, sww = 0.0;
    int bad = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int idx = (v * 64 + lane) * VW;
        if (idx < a.cols) {
            load_row_piece<VW>(a, M, G, W, idx, mv[v], wv[v], bad);
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                const double md = mv[v][e], wd = wv[v][e];
                smw = fma(md, wd, smw);
                sww = fma(wd, wd, sww);
            }
        }
    }
    if (a.nfin) {
        const double b = wave_sum_d((double)bad);
        if (lane == 0) a.nfin[(int64_t)z * a.stride_nfin + row] = (int)b;
    }
    smw = wave_sum_d(smw);
    sww = wave_sum_d(sww);
    const double d = tangent_coef(a.tangent, smw, sww);
    // x replaces m in the registers (rounded to fp32 after it is formed, so
    // its relative error is u32 whatever the cancellation was).
    double nrm2 = 0.0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
        if ((v * 64 + lane) * VW < a.cols) {
#pragma unroll
            for (int e = 0; e < VW; ++e) {
                const double x = tangent_x(mv[v][e], wv[v][e], d);
                nrm2 = fma(x, x, nrm2);
                mv[v][e] = (float)x;
            }
        }
    nrm2 = wave_sum_d(nrm2);
    const double inv = 1.0 / fmax(sqrt(nrm2), (double)a.eps);
    const float invf = (float)inv;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
        const int idx = (v * 64 + lane) * VW;
        if (idx < a.cols) {
            float p[VW];
#pragma unroll
            for (int e = 0; e < VW; ++e) p[e] = mv[v][e] * invf;
            if constexpr (VW == 4) {
                half_t h[4] = {(half_t)p[0], (half_t)p[1], (half_t)p[2], (half_t)p[3]};
                *reinterpret_cast<uint2*>(prow + idx) = *reinterpret_cast<const uint2*>(h);
                if constexpr (DBG)
                    *reinterpret_cast<float4*>(a.psi32 + (int64_t)z * a.stride_psi32 + off + idx) =
                        make_float4(p[0], p[1], p[2], p[3]);
            } else {
                prow[idx] = (half_t)p[0];
                if constexpr (DBG) a.psi32[(int64_t)z * a.stride_psi32 + off + idx] = p[0];
            }
        }
    }
    // zero padding of the row (ld_psi is a multiple of 256)
    if constexpr (VW == 4) {
        for (int64_t j = a.cols + lane * 4; j < a.ld_psi; j += 256)
            *reinterpret_cast<uint2*>(prow + j) = make_uint2(0u, 0u);
    } else {
        for (int64_t j = a.cols + lane; j < a.ld_psi; j += 64) prow[j] = (half_t)0.f;
    }
    if (lane == 0) {
        a.psisq[(int64_t)z * a.stride_psisq + row] = (float)(nrm2 * inv * inv);
        if (a.xsq) a.xsq[(int64_t)z * a.stride_psisq + row] = (float)nrm2;
    }
}

// ---------------------------------------------------------------------------
// Column-active orientation.  Block = (64 * VW) columns x 4 row lanes over a
// chunk of rows; each thread owns VW adjacent columns (one 16-byte access per
// row when VW = 4).  Pass 1 updates M and writes fp64 partial column sums;
// pass 2 combines the partials in a fixed order and writes Psi.
constexpr int kColThreads = 256;
constexpr int kColBatch = 4;   // rows whose loads a stats-pass thread issues together

template <int VW>
__global__ void __launch_bounds__(kColThreads) normalize_cols_stats(NormArgs a, double* partials, int row_chunk) {
    const int z = blockIdx.z, chunk = blockIdx.y;
    const int cx = threadIdx.x & 63, ry = threadIdx.x >> 6;
    const int col0 = (blockIdx.x * 64 + cx) * VW;
    const int r0 = chunk * row_chunk, r1 = min(a.rows, r0 + row_chunk);
    double smm[VW], smw[VW], sww[VW];
#pragma unroll
    for (int e = 0; e < VW; ++e) smm[e] = smw[e] = sww[e] = 0.0;
    int bad = 0;
    if (col0 < a.cols) {
        float* W = a.ptrs.w[z];
        float* M = a.ptrs.m[z];
        const float* G = a.ptrs.g[z];
        int i = r0 + ry;
        if constexpr (VW == 4) {
            // kColBatch rows per step: every load of the batch is issued before
            // the first M store, so a wave keeps 12 16-byte loads per lane in
            // flight.  Rows are still accumulated in ascending order.
            for (; i + 4 * (kColBatch - 1) < r1; i += 4 * kColBatch) {
                float4 mp[kColBatch], g[kColBatch], w[kColBatch];
#pragma unroll
                for (int u = 0; u < kColBatch; ++u) {
                    const int64_t o = (int64_t)(i + 4 * u) * a.cols + col0;
                    mp[u] = *reinterpret_cast<const float4*>(M + o);
                    g[u] = *reinterpret_cast<const float4*>(G + o);
                    w[u] = *reinterpret_cast<const float4*>(W + o);
                }
#pragma unroll
                for (int u = 0; u < kColBatch; ++u) {
                    const int64_t o = (int64_t)(i + 4 * u) * a.cols + col0;
                    float pv[4] = {mp[u].x, mp[u].y, mp[u].z, mp[u].w}, gv[4] = {g[u].x, g[u].y, g[u].z, g[u].w};
                    float wv[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
                    if (a.nfin) {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            pv[e] = finite_or_zero(pv[e], bad);
                            gv[e] = finite_or_zero(gv[e], bad);
                            wv[e] = finite_or_zero(wv[e], bad);
                        }
                    }
                    const float m[4] = {fmaf(a.mu, pv[0], gv[0]), fmaf(a.mu, pv[1], gv[1]), fmaf(a.mu, pv[2], gv[2]),
                                        fmaf(a.mu, pv[3], gv[3])};
                    *reinterpret_cast<float4*>(M + o) = make_float4(m[0], m[1], m[2], m[3]);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const double md = m[e], wd = wv[e];
                        smm[e] = fma(md, md, smm[e]);
                        smw[e] = fma(md, wd, smw[e]);
                        sww[e] = fma(wd, wd, sww[e]);
                    }
                }
            }
        }
        for (; i < r1; i += 4) {
            const int64_t o = (int64_t)i * a.cols + col0;
            float m[VW], wv[VW];
            load_row_piece<VW>(a, M, G, W, (int)0, m, wv, bad, o);
            if constexpr (VW == 4) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double md = m[e], wd = wv[e];
                    smm[e] = fma(md, md, smm[e]);
                    smw[e] = fma(md, wd, smw[e]);
                    sww[e] = fma(wd, wd, sww[e]);
                }
            } else {
                const double md = m[0], wd = wv[0];
                smm[0] = fma(md, md, smm[0]);
                smw[0] = fma(md, wd, smw[0]);
                sww[0] = fma(wd, wd, sww[0]);
            }
        }
    }
    __shared__ double red[3][4][64 * VW];
    __shared__ int redbad[kColThreads / 64];
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        red[0][ry][cx * VW + e] = smm[e];
        red[1][ry][cx * VW + e] = smw[e];
        red[2][ry][cx * VW + e] = sww[e];
    }
    if (a.nfin) {
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) bad += __shfl_xor(bad, o, 64);
        if ((threadIdx.x & 63) == 0) redbad[threadIdx.x >> 6] = bad;
    }
    __syncthreads();
    if (a.nfin && threadIdx.x == 0) {
        int t = 0;
        for (int q = 0; q < kColThreads / 64; ++q) t += redbad[q];
        a.nfin[(int64_t)z * a.stride_nfin + (int64_t)chunk * gridDim.x + blockIdx.x] = t;
    }
    const int64_t cols_pad = a.ld_psi;
    const int nchunks = gridDim.y;
    double* p = partials + ((int64_t)z * nchunks + chunk) * 3 * cols_pad;
    for (int c = threadIdx.x; c < 3 * 64 * VW; c += kColThreads) {
        const int q = c / (64 * VW), cc = c - q * (64 * VW);
        const int64_t col = (int64_t)blockIdx.x * 64 * VW + cc;
        if (col < cols_pad) p[q * cols_pad + col] = red[q][0][cc] + red[q][1][cc] + red[q][2][cc] + red[q][3][cc];
    }
}

// Sums the row-chunk partials of each column once, in a fixed order, and
// stores the tangent coefficient c and 1 / max(||x||, eps) in the chunk-0
// slots.
__global__ void __launch_bounds__(256) normalize_cols_finalize(NormArgs a, double* partials, int nchunks) {
    const int z = blockIdx.y;
    const int col = blockIdx.x * 256 + threadIdx.x;
    if (col >= a.cols) return;
    const int64_t cols_pad = a.ld_psi;
    double* p = partials + (int64_t)z * nchunks * 3 * cols_pad;
    double smm = 0.0, smw = 0.0, sww = 0.0;
    for (int c = 0; c < nchunks; ++c) {
        smm += p[(c * 3 + 0) * cols_pad + col];
        smw += p[(c * 3 + 1) * cols_pad + col];
        sww += p[(c * 3 + 2) * cols_pad + col];
    }
    const double d = tangent_coef(a.tangent, smw, sww);
    const double nrm2 = fmax(smm - 2.0 * d * smw + d * d * sww, 0.0);
    const double inv = 1.0 / fmax(sqrt(nrm2), (double)a.eps);
    p[col] = d;
    p[cols_pad + col] = inv;
    a.psisq[(int64_t)z * a.stride_psisq + col] = (float)(nrm2 * inv * inv);
    if (a.xsq) a.xsq[(int64_t)z * a.stride_psisq + col] = (float)nrm2;
}

template <int VW, bool DBG>
__global__ void __launch_bounds__(kColThreads) normalize_cols_apply(NormArgs a, const double* partials, int row_chunk) {
    const int z = blockIdx.z, chunk = blockIdx.y;
    const int cx = threadIdx.x & 63, ry = threadIdx.x >> 6;
    const int col0 = (blockIdx.x * 64 + cx) * VW;
    const int64_t cols_pad = a.ld_psi;
    const int nchunks = (a.rows + row_chunk - 1) / row_chunk;
    half_t* P = a.psi + (int64_t)z * a.stride_psi;
    const int r0 = chunk * row_chunk, r1 = min((int)a.rows_pad, r0 + row_chunk);
    if (col0 >= cols_pad) return;
    double df[VW], inv[VW];
    const double* p = partials + (int64_t)z * nchunks * 3 * cols_pad;
#pragma unroll
    for (int e = 0; e < VW; ++e) {
        const int col = col0 + e;
        df[e] = col < a.cols ? p[col] : 0.0;
        inv[e] = col < a.cols ? p[cols_pad + col] : 0.0;
    }
    const float* W = a.ptrs.w[z];
    const float* M = a.ptrs.m[z];
    for (int i = r0 + ry; i < r1; i += 4) {
        half_t* prow = P + (int64_t)i * cols_pad + col0;
        if constexpr (VW == 4) {
            float v[4] = {0.f, 0.f, 0.f, 0.f};
            if (i < a.rows && col0 < a.cols) {
                const int64_t o = (int64_t)i * a.cols + col0;
                const float4 m = *reinterpret_cast<const float4*>(M + o);
                float4 w = *reinterpret_cast<const float4*>(W + o);
                if (a.nfin) {
                    int unused = 0;
                    w.x = finite_or_zero(w.x, unused); w.y = finite_or_zero(w.y, unused);
                    w.z = finite_or_zero(w.z, unused); w.w = finite_or_zero(w.w, unused);
                }
                v[0] = (float)(tangent_x(m.x, w.x, df[0]) * inv[0]);
                v[1] = (float)(tangent_x(m.y, w.y, df[1]) * inv[1]);
                v[2] = (float)(tangent_x(m.z, w.z, df[2]) * inv[2]);
                v[3] = (float)(tangent_x(m.w, w.w, df[3]) * inv[3]);
                if constexpr (DBG)
                    *reinterpret_cast<float4*>(a.psi32 + (int64_t)z * a.stride_psi32 + o) = make_float4(v[0], v[1], v[2], v[3]);
            }
            half_t h[4] = {(half_t)v[0], (half_t)v[1], (half_t)v[2], (half_t)v[3]};
            *reinterpret_cast<uint2*>(prow) = *reinterpret_cast<const uint2*>(h);
        } else {
            float v = 0.f;
            if (i < a.rows && col0 < a.cols) {
                const int64_t o = (int64_t)i * a.cols + col0;
                int unused = 0;
                const float wo = a.nfin ? finite_or_zero(W[o], unused) : W[o];
                v = (float)(tangent_x(M[o], wo, df[0]) * inv[0]);
                if constexpr (DBG) a.psi32[(int64_t)z * a.stride_psi32 + o] = v;
            }
            prow[0] = (half_t)v;
        }
    }
}

// ---------------------------------------------------------------------------
// Column-active orientation in one pass, for padded columns of at most
// kFusedNR * 4096 / SW rows: one block of kFusedThreads threads per strip of
// SW columns (SW / 4 threads per row, 16 bytes each, at most kFusedNR rows
// per thread).  The strip of the new M (in registers) and of W (in LDS)
// stays on the CU between the column sums and the Psi store, so G, M_prev
// and W are read once: 18 bytes per element, as in the row-active kernels,
// against the 26 of the two-pass path.  As there, <m, w> and ||w||^2 give c,
// x is formed in fp64 and rounded to fp32 in the registers, and ||x||^2 is
// summed from the formed x.
constexpr int kFusedThreads = 1024, kFusedNR = 8;

// Sums NQ per-column quantities (four adjacent columns per thread) over the
// rows of the block in a fixed order: lanes of a wave first, then the waves.
// On return tot[q][c] holds the strip's sum for column c in every thread.
template <int SW, int NQ>
__device__ __forceinline__ void strip_col_sums(double (&v)[NQ][4], double (*part)[NQ][SW], double (*tot)[SW]) {
    constexpr int TPR = SW / 4;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int o = TPR; o < 64; o <<= 1) v[q][e] += __shfl_xor(v[q][e], o, 64);
    if (lane < TPR) {
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) part[wave][q][lane * 4 + e] = v[q][e];
    }
    __syncthreads();
    if (threadIdx.x < NQ * SW) {
        const int q = threadIdx.x / SW, c = threadIdx.x % SW;
        double t = 0.0;
        for (int w = 0; w < kFusedThreads / 64; ++w) t += part[w][q][c];
        tot[q][c] = t;
    }
    __syncthreads();
}

template <int SW, bool DBG>
__global__ void __launch_bounds__(kFusedThreads) normalize_cols_fused(NormArgs a, int nr) {
    constexpr int TPR = SW / 4, RPI = kFusedThreads / TPR, WAVES = kFusedThreads / 64;
    // Workgroups are dispatched round-robin over the 8 XCDs; each XCD takes
    // one contiguous run of strips instead, so neighbouring strips (which
    // share 128-byte lines) meet in the same L2.  The ragged tail keeps its
    // order.
    int lin = blockIdx.x + gridDim.x * blockIdx.y;
    const int per = (int)(gridDim.x * gridDim.y) >> 3;
    if (lin < (per << 3)) lin = (lin & 7) * per + (lin >> 3);
    const int strip = lin % gridDim.x, z = lin / gridDim.x;
    const int tid = threadIdx.x, cx = tid % TPR, ry = tid / TPR;
    const int col0 = strip * SW + cx * 4;
    const bool live = col0 < a.cols;   // cols % 4 == 0: all four columns are real
    float* W = a.ptrs.w[z];
    float* M = a.ptrs.m[z];
    const float* G = a.ptrs.g[z];
    // W of row slot r of this thread: wl[r][tid] (consecutive threads,
    // consecutive 16 bytes).
    __shared__ float4 wl[kFusedNR][kFusedThreads];
    float mv[kFusedNR][4];
    double s2[2][4] = {};   // <m, w>, ||w||^2 per column
    int bad = 0;
#pragma unroll
    for (int r0 = 0; r0 < kFusedNR; r0 += kColBatch) {
        float4 mp[kColBatch], g[kColBatch], w[kColBatch];
#pragma unroll
        for (int u = 0; u < kColBatch; ++u) {
            const int r = r0 + u, i = ry + r * RPI;
            mp[u] = g[u] = w[u] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (r < nr && i < a.rows && live) {
                const int64_t o = (int64_t)i * a.cols + col0;
                mp[u] = *reinterpret_cast<const float4*>(M + o);
                g[u] = *reinterpret_cast<const float4*>(G + o);
                w[u] = *reinterpret_cast<const float4*>(W + o);
            }
        }
#pragma unroll
        for (int u = 0; u < kColBatch; ++u) {
            const int r = r0 + u, i = ry + r * RPI;
            float pv[4] = {mp[u].x, mp[u].y, mp[u].z, mp[u].w}, gv[4] = {g[u].x, g[u].y, g[u].z, g[u].w};
            float wq[4] = {w[u].x, w[u].y, w[u].z, w[u].w};
            if (a.nfin) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    pv[e] = finite_or_zero(pv[e], bad);
                    gv[e] = finite_or_zero(gv[e], bad);
                    wq[e] = finite_or_zero(wq[e], bad);
                }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) mv[r][e] = fmaf(a.mu, pv[e], gv[e]);
            if (r < nr) wl[r][tid] = make_float4(wq[0], wq[1], wq[2], wq[3]);
            if (r < nr && i < a.rows && live) {
                *reinterpret_cast<float4*>(M + (int64_t)i * a.cols + col0) =
                    make_float4(mv[r][0], mv[r][1], mv[r][2], mv[r][3]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const double md = mv[r][e], wd = wq[e];
                    s2[0][e] = fma(md, wd, s2[0][e]);
                    s2[1][e] = fma(wd, wd, s2[1][e]);
                }
            }
        }
    }
    __shared__ double part2[WAVES][2][SW], tot2[2][SW];
    __shared__ double part1[WAVES][1][SW], tot1[1][SW];
    strip_col_sums<SW, 2>(s2, part2, tot2);
    double cf[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) cf[e] = tangent_coef(a.tangent, tot2[0][cx * 4 + e], tot2[1][cx * 4 + e]);
    // x replaces m in the registers (rounded to fp32 after it is formed, so
    // its relative error is u32 whatever the cancellation was).
    double s1[1][4] = {};
#pragma unroll
    for (int r = 0; r < kFusedNR; ++r) {
        const int i = ry + r * RPI;
        if (r < nr && i < a.rows && live) {
            const float4 w4 = wl[r][tid];
            const float wq[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double x = tangent_x(mv[r][e], wq[e], cf[e]);
                s1[0][e] = fma(x, x, s1[0][e]);
                mv[r][e] = (float)x;
            }
        }
    }
    strip_col_sums<SW, 1>(s1, part1, tot1);
    float invf[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) invf[e] = (float)(1.0 / fmax(sqrt(tot1[0][cx * 4 + e]), (double)a.eps));
    if (tid < SW && strip * SW + tid < a.cols) {
        const int64_t col = (int64_t)strip * SW + tid;
        const double n2 = tot1[0][tid], inv = 1.0 / fmax(sqrt(n2), (double)a.eps);
        a.psisq[(int64_t)z * a.stride_psisq + col] = (float)(n2 * inv * inv);
        if (a.xsq) a.xsq[(int64_t)z * a.stride_psisq + col] = (float)n2;
    }
    if (a.nfin) {
        __shared__ int redbad[WAVES];
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) bad += __shfl_xor(bad, o, 64);
        if ((tid & 63) == 0) redbad[tid >> 6] = bad;
        __syncthreads();
        if (tid == 0 && strip * SW < a.cols) {
            int t = 0;
            for (int q = 0; q < WAVES; ++q) t += redbad[q];
            a.nfin[(int64_t)z * a.stride_nfin + strip] = t;
        }
    }
    half_t* P = a.psi + (int64_t)z * a.stride_psi;
#pragma unroll
    for (int r = 0; r < kFusedNR; ++r) {
        const int i = ry + r * RPI;
        if (r < nr && i < a.rows_pad) {
            float p[4] = {0.f, 0.f, 0.f, 0.f};
            if (i < a.rows && live) {
#pragma unroll
                for (int e = 0; e < 4; ++e) p[e] = mv[r][e] * invf[e];
                if constexpr (DBG)
                    *reinterpret_cast<float4*>(a.psi32 + (int64_t)z * a.stride_psi32 + (int64_t)i * a.cols + col0) =
                        make_float4(p[0], p[1], p[2], p[3]);
            }
            half_t h[4] = {(half_t)p[0], (half_t)p[1], (half_t)p[2], (half_t)p[3]};
            *reinterpret_cast<uint2*>(P + (int64_t)i * a.ld_psi + col0) = *reinterpret_cast<const uint2*>(h);
        }
    }
}

// ---------------------------------------------------------------------------
// Muon input, pass 1: M <- mu M + G over the whole matrix, with the block's
// sum of M^2 (fp64 in each thread, fixed-order block reduction) written to
// part[z * stride_part + block].
template <int VW>
__global__ void __launch_bounds__(256) momentum_sumsq_kernel(NormArgs a, float* part, int64_t stride_part) {
    const int z = blockIdx.y;
    float* M = a.ptrs.m[z];
    const float* G = a.ptrs.g[z];
    const int64_t nv = (int64_t)a.rows * a.cols / VW;
    double s = 0.0;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < nv; v += (int64_t)gridDim.x * 256) {
        if constexpr (VW == 4) {
            const float4 mp = reinterpret_cast<const float4*>(M)[v];
            const float4 g = reinterpret_cast<const float4*>(G)[v];
            float4 m;
            m.x = fmaf(a.mu, mp.x, g.x); m.y = fmaf(a.mu, mp.y, g.y);
            m.z = fmaf(a.mu, mp.z, g.z); m.w = fmaf(a.mu, mp.w, g.w);
            reinterpret_cast<float4*>(M)[v] = m;
            s = fma((double)m.x, (double)m.x, s); s = fma((double)m.y, (double)m.y, s);
            s = fma((double)m.z, (double)m.z, s); s = fma((double)m.w, (double)m.w, s);
        } else {
            const float m = fmaf(a.mu, M[v], G[v]);
            M[v] = m;
            s = fma((double)m, (double)m, s);
        }
    }
    s = wave_sum_d(s);
    __shared__ double red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) part[(int64_t)z * stride_part + blockIdx.x] = (float)(red[0] + red[1] + red[2] + red[3]);
}

// Muon input, pass 2: X0 = M * scale[2z] in fp16 over the whole zero-padded
// W-layout workspace (rows_pad x ld_psi); optional fp32 copy of X0.
template <int VW, bool DBG>
__global__ void __launch_bounds__(256) scaled_cast_kernel(NormArgs a, const float* scale) {
    const int z = blockIdx.y;
    const float sc = scale[2 * z];
    const float* M = a.ptrs.m[z];
    half_t* P = a.psi + (int64_t)z * a.stride_psi;
    const int64_t vpr = a.ld_psi / VW;
    const int64_t nv = a.rows_pad * vpr;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < nv; v += (int64_t)gridDim.x * 256) {
        const int64_t row = v / vpr;
        const int64_t col = (v - row * vpr) * VW;
        float x[VW];
#pragma unroll
        for (int e = 0; e < VW; ++e) x[e] = 0.f;
        if (row < a.rows && col < a.cols) {
            const int64_t o = row * a.cols + col;
            if constexpr (VW == 4) {
                const float4 m = *reinterpret_cast<const float4*>(M + o);
                x[0] = m.x * sc; x[1] = m.y * sc; x[2] = m.z * sc; x[3] = m.w * sc;
                if constexpr (DBG)
                    *reinterpret_cast<float4*>(a.psi32 + (int64_t)z * a.stride_psi32 + o) = make_float4(x[0], x[1], x[2], x[3]);
            } else {
                x[0] = M[o] * sc;
                if constexpr (DBG) a.psi32[(int64_t)z * a.stride_psi32 + o] = x[0];
            }
        }
        half_t* dst = P + row * a.ld_psi + col;
        if constexpr (VW == 4) {
            half_t h[4] = {(half_t)x[0], (half_t)x[1], (half_t)x[2], (half_t)x[3]};
            *reinterpret_cast<uint2*>(dst) = *reinterpret_cast<const uint2*>(h);
        } else {
            dst[0] = (half_t)x[0];
        }
    }
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) psi_scale_kernel(const float* psisq, int64_t stride, int active_rows,
                                                        float eps, float* out) {
    const int z = blockIdx.x;
    const float* p = psisq + (int64_t)z * stride;
    float s = 0.f;
    for (int i = threadIdx.x; i < active_rows; i += 256) s += p[i];
    s = wave_sum_f(s);
    __shared__ float red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        const float tot = red[0] + red[1] + red[2] + red[3];
        out[2 * z] = 1.f / (sqrtf(tot) + eps);
        out[2 * z + 1] = tot;
    }
}

// ---------------------------------------------------------------------------
template <int VW, bool DBG>
__global__ void __launch_bounds__(256) g_update_kernel(GUpdateArgs a) {
    const int z = blockIdx.y;
    float scale = a.fixed_scale;
    if (!(scale > 0.f)) {
        const float t2 = a.tnorm2[(int64_t)z * a.tnorm2_stride];
        scale = t2 > 0.f ? a.target_rms * sqrtf((float)a.rows * (float)a.cols) / sqrtf(t2) : 0.f;
    }

    float* W = a.ptrs.w[z];
    const half_t* T = a.t + (int64_t)z * a.stride_t;
    const int64_t n_vec = (int64_t)a.rows * a.cols / VW;
    const int vec_per_row = a.cols / VW;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < n_vec; v += (int64_t)gridDim.x * 256) {
        const int row = (int)(v / vec_per_row);
        const int c0 = (int)(v - (int64_t)row * vec_per_row) * VW;
        const half_t* tp = T + (int64_t)row * a.ld_t + c0;
        float* wp = W + (int64_t)row * a.cols + c0;
        if constexpr (VW == 4) {
            const uint2 hraw = *reinterpret_cast<const uint2*>(tp);
            const half_t* h = reinterpret_cast<const half_t*>(&hraw);
            float4 w = *reinterpret_cast<float4*>(wp);
            const float t0 = (float)h[0], t1 = (float)h[1], t2v = (float)h[2], t3 = (float)h[3];
            w.x = w.x - a.lr * (scale * t0 + a.wd * w.x);
            w.y = w.y - a.lr * (scale * t1 + a.wd * w.y);
            w.z = w.z - a.lr * (scale * t2v + a.wd * w.z);
            w.w = w.w - a.lr * (scale * t3 + a.wd * w.w);
            *reinterpret_cast<float4*>(wp) = w;
            if constexpr (DBG)
                *reinterpret_cast<float4*>(a.t32 + (int64_t)z * a.stride_t32 + (int64_t)row * a.cols + c0) =
                    make_float4(t0, t1, t2v, t3);
        } else {
            const float t = (float)tp[0];
            const float w = *wp;
            *wp = w - a.lr * (scale * t + a.wd * w);
            if constexpr (DBG) a.t32[(int64_t)z * a.stride_t32 + (int64_t)row * a.cols + c0] = t;
        }
    }
}

// One block per matrix; fixed-order (deterministic) sum of n partials.
__global__ void __launch_bounds__(256) sum_partials_kernel(const float* in, int n, float* out, const int* need) {
    const int z = blockIdx.x;
    if (need && need[z] == 0) return;   // the whole block
    const float* p = in + (int64_t)z * n;
    float s = 0.f;
    for (int i = threadIdx.x; i < n; i += 256) s += p[i];
    s = wave_sum_f(s);
    __shared__ float red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[z] = red[0] + red[1] + red[2] + red[3];
}

// One wave per matrix: the closed-form ||T||_F^2 of NormPre-L and whether it
// cancels (see LNormGroups).  The sums over the selected modes are in fp64.
__global__ void __launch_bounds__(64) l_norm_closed_kernel(LNormGroups g) {
    const int zl = blockIdx.x, lane = threadIdx.x;
    int gi = 0;
    while (gi + 1 < g.n && zl >= g.zbeg[gi + 1]) ++gi;
    const int z = zl - g.zbeg[gi];
    const int n = g.nsel[gi][z];
    const float* r = g.ritz[gi] + (int64_t)z * g.ritz_stride[gi];
    double sl = 0.0, sc = 0.0;
    for (int i = lane; i < n; i += 64) {
        const double l = r[i];
        sl += l;
        sc += l - 1.0;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        sl += __shfl_xor(sl, o, 64);
        sc += __shfl_xor(sc, o, 64);
    }
    if (lane == 0) {
        const double p2 = g.psi2[gi][2 * (int64_t)z];
        const double t2 = p2 - sc;
        const bool need = !(sl <= (double)g.frac * p2) || !(t2 > 0.0);
        g.need[gi][z] = need ? 1 : 0;
        if (!need) g.tn2[gi][z] = (float)t2;
    }
}

// Q <- Q + a I in place for a batch of sp x sp fp16 matrices: one thread per
// diagonal entry.
__global__ void __launch_bounds__(256) add_diag_kernel(half_t* q, int64_t sp, int64_t n, float a) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t z = i / sp, d = i - z * sp;
    half_t* e = q + z * sp * sp + d * (sp + 1);
    *e = (half_t)((float)*e + a);
}

__global__ void fill_zero_kernel(uint4* p, int64_t n16) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = make_uint4(0, 0, 0, 0);
}

// Descent alignment, pass 1: block b of matrix z sums g phi, g^2 and phi^2
// over a grid-stride slice (fp64), phi = (wb - wa) / lr - wd wb.
__global__ void __launch_bounds__(256) alignment_partials_kernel(AlignChunk c, double inv_lr, double wd,
                                                                 double* part) {
    const int z = blockIdx.y;
    const float* g = c.g[z];
    const float* wb = c.wb[z];
    const float* wa = c.wa[z];
    const int64_t n = c.n[z];
    double sgp = 0.0, sgg = 0.0, spp = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
        const double b = wb[i], gv = g[i];
        const double phi = (b - (double)wa[i]) * inv_lr - wd * b;
        sgp = fma(gv, phi, sgp);
        sgg = fma(gv, gv, sgg);
        spp = fma(phi, phi, spp);
    }
    sgp = wave_sum_d(sgp);
    sgg = wave_sum_d(sgg);
    spp = wave_sum_d(spp);
    __shared__ double red[3][4];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) { red[0][wave] = sgp; red[1][wave] = sgg; red[2][wave] = spp; }
    __syncthreads();
    if (threadIdx.x < 3) {
        const int q = threadIdx.x;
        part[((int64_t)z * kAlignBlocks + blockIdx.x) * 3 + q] = red[q][0] + red[q][1] + red[q][2] + red[q][3];
    }
}

// Pass 2 (one block): cos[z] from the partials of matrix z in block order;
// the mean of the cosines in matrix order.
__global__ void __launch_bounds__(256) alignment_finalize_kernel(const double* part, int num_mats, double* cos_out,
                                                                 double* mean_out) {
    for (int z = threadIdx.x; z < num_mats; z += 256) {
        double sgp = 0.0, sgg = 0.0, spp = 0.0;
        for (int b = 0; b < kAlignBlocks; ++b) {
            const double* p = part + ((int64_t)z * kAlignBlocks + b) * 3;
            sgp += p[0];
            sgg += p[1];
            spp += p[2];
        }
        const double den = sqrt(sgg) * sqrt(spp);
        cos_out[z] = den > 0.0 ? sgp / den : 0.0;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double m = 0.0;
        for (int z = 0; z < num_mats; ++z) m += cos_out[z];
        *mean_out = num_mats > 0 ? m / num_mats : 0.0;
    }
}

template <int NT, int VW, int NV>
hipError_t rows_launch(const NormArgs& a, int batch, hipStream_t s, bool dbg) {
    dim3 grid((unsigned)a.rows_pad, batch);
    if (dbg) hipLaunchKernelGGL((normalize_rows_kernel<NT, VW, NV, true>), grid, dim3(NT), 0, s, a);
    else hipLaunchKernelGGL((normalize_rows_kernel<NT, VW, NV, false>), grid, dim3(NT), 0, s, a);
    return hipGetLastError();
}

template <int NT, int VW>
hipError_t rows_pick_nv(const NormArgs& a, int batch, hipStream_t s, bool dbg) {
    const int nv = (a.cols + NT * VW - 1) / (NT * VW);
    if (nv <= 1) return rows_launch<NT, VW, 1>(a, batch, s, dbg);
    if (nv <= 2) return rows_launch<NT, VW, 2>(a, batch, s, dbg);
    if (nv <= 4) return rows_launch<NT, VW, 4>(a, batch, s, dbg);
    if (nv <= 8) return rows_launch<NT, VW, 8>(a, batch, s, dbg);
    return hipErrorInvalidValue;
}

}  // namespace

template <int VW, int NV>
hipError_t rows_wave_launch(const NormArgs& a, int batch, hipStream_t s, bool dbg) {
    dim3 grid((unsigned)((a.rows_pad + 3) / 4), batch);
    if (dbg) hipLaunchKernelGGL((normalize_rows_wave_kernel<VW, NV, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((normalize_rows_wave_kernel<VW, NV, false>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_normalize_rows(const NormArgs& a, int batch, hipStream_t s) {
    const bool dbg = a.psi32 != nullptr;
    const bool vec = a.vec_ok && (a.cols % 4) == 0;
    // Rows up to 4096 elements (vectorized) or 1024 (scalar): a wave per row.
    if (vec && a.cols <= 64 * 4 * 16) {
        const int nv = (a.cols + 255) / 256;
        if (nv <= 4) return rows_wave_launch<4, 4>(a, batch, s, dbg);
        if (nv <= 8) return rows_wave_launch<4, 8>(a, batch, s, dbg);
        if (nv <= 12) return rows_wave_launch<4, 12>(a, batch, s, dbg);
        return rows_wave_launch<4, 16>(a, batch, s, dbg);
    }
    if (!vec && a.cols <= 64 * 16) return rows_wave_launch<1, 16>(a, batch, s, dbg);
    if (vec) {
        if (a.cols <= 256 * 4 * 8) return rows_pick_nv<256, 4>(a, batch, s, dbg);
        if (a.cols <= 1024 * 4 * 8) return rows_pick_nv<1024, 4>(a, batch, s, dbg);
    } else {
        if (a.cols <= 256 * 8) return rows_pick_nv<256, 1>(a, batch, s, dbg);
        if (a.cols <= 1024 * 8) return rows_pick_nv<1024, 1>(a, batch, s, dbg);
    }
    return hipErrorInvalidValue;
}

// ------------------------------------------ interaction source X (L only) --
// X_s = c D Psi with c = sqrt(a / ||X||_F^2): recovers the update before
// normalization from Psi and the active norms, trace-matched so that
// X_s X_s^T has trace a.  Covers the padded W layout (zeros there).
__global__ void __launch_bounds__(256) source_x_kernel(const half_t* psi, int64_t ld, int64_t stride, int rows,
                                                       int cols, int rows_pad, int k, int active, const float* xsq,
                                                       int64_t stride_xsq, const float* xtot, half_t* xs) {
    const int z = blockIdx.y;
    const float tot = xtot[2 * z + 1];
    const float c = tot > 0.f ? sqrtf((float)active / tot) : 0.f;
    const float* q = xsq + (int64_t)z * stride_xsq;
    const int64_t total = (int64_t)rows_pad * ld;
    const half_t* p = psi + (int64_t)z * stride;
    half_t* o = xs + (int64_t)z * stride;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        const int r = (int)(e / ld), j = (int)(e - (int64_t)r * ld);
        float v = 0.f;
        if (r < rows && j < cols) v = (float)p[e] * c * sqrtf(q[k == 0 ? r : j]);
        o[e] = (half_t)v;
    }
}

// ------------------------------------- both axes: column pass over fp16 Psi --
// Pass 1: partial sums of squares per (row chunk, column), fp32, fixed order.
__global__ void __launch_bounds__(256) psi_colstats_kernel(const half_t* psi, int64_t ld, int64_t stride, int rows,
                                                           int cols, int row_chunk, float* part, int64_t stride_part,
                                                           int64_t cols_pad) {
    const int z = blockIdx.z, chunk = blockIdx.y;
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (j >= cols) return;
    const half_t* p = psi + (int64_t)z * stride + j;
    const int r0 = chunk * row_chunk, r1 = min(rows, r0 + row_chunk);
    float s = 0.f;
    for (int r = r0; r < r1; ++r) {
        const float v = (float)p[(int64_t)r * ld];
        s = fmaf(v, v, s);
    }
    part[(int64_t)z * stride_part + (int64_t)chunk * cols_pad + j] = s;
}

// Pass 2: per column f_j = 1 / max(||psi_j||, eps) and the new squared norm.
__global__ void __launch_bounds__(256) psi_colfactor_kernel(float* part, int64_t stride_part, int nchunks, int cols,
                                                            int64_t cols_pad, float eps, float* psisq,
                                                            int64_t stride_psisq) {
    const int z = blockIdx.y;
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (j >= cols) return;
    float* pz = part + (int64_t)z * stride_part;
    float s = 0.f;
    for (int c = 0; c < nchunks; ++c) s += pz[(int64_t)c * cols_pad + j];
    const float f = 1.f / fmaxf(sqrtf(s), eps);
    pz[(int64_t)nchunks * cols_pad + j] = f;
    psisq[(int64_t)z * stride_psisq + j] = s * f * f;
}

// Pass 3: psi_ij *= f_j over the real region (fp16 and the fp32 debug copy).
__global__ void __launch_bounds__(256) psi_colscale_kernel(half_t* psi, int64_t ld, int64_t stride, int rows,
                                                           int cols, const float* part, int64_t stride_part,
                                                           int nchunks, int64_t cols_pad, float* psi32,
                                                           int64_t stride_psi32) {
    const int z = blockIdx.y;
    const float* f = part + (int64_t)z * stride_part + (int64_t)nchunks * cols_pad;
    const int64_t total = (int64_t)rows * cols;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
        const int r = (int)(e / cols), j = (int)(e - (int64_t)r * cols);
        half_t* q = psi + (int64_t)z * stride + (int64_t)r * ld + j;
        *q = (half_t)((float)*q * f[j]);
        if (psi32) psi32[(int64_t)z * stride_psi32 + e] *= f[j];
    }
}

// Count slots per matrix, as the launches write them: one per real row in the
// row-active kernels, one per stats block (row chunk x column block) in the
// column-active stats pass (its vector width as launch_normalize_cols picks).
int cols_fused_width(const NormArgs& a) {
    if (!(a.vec_ok && a.cols % 4 == 0 && a.ld_psi % 64 == 0)) return 0;
    for (int sw = 64; sw >= 16; sw >>= 1)
        if (a.rows_pad * sw <= (int64_t)kFusedNR * kFusedThreads * 4) return sw;
    return 0;
}

int64_t nonfinite_slots(const NormArgs& a, bool row_active, int row_chunk) {
    if (row_active) return a.rows;
    if (const int sw = cols_fused_width(a)) return (a.cols + sw - 1) / sw;
    const int nchunks = (a.rows + row_chunk - 1) / row_chunk;
    const int vw = (a.vec_ok && a.cols % 4 == 0 && a.ld_psi % 4 == 0) ? 4 : 1;
    return (int64_t)nchunks * ((a.cols + 64 * vw - 1) / (64 * vw));
}

// One block per matrix: the sum of its count slots, written to the caller's
// position of the matrix.
__global__ void __launch_bounds__(256) count_reduce_kernel(const int* nfin, int64_t slots, int64_t stride,
                                                           IdxChunk idx, long long* status) {
    const int z = blockIdx.x;
    long long t = 0;
    for (int64_t i = threadIdx.x; i < slots; i += 256) t += nfin[(int64_t)z * stride + i];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) t += __shfl_xor(t, o, 64);
    __shared__ long long red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = t;
    __syncthreads();
    if (threadIdx.x == 0) status[idx.idx[z]] = red[0] + red[1] + red[2] + red[3];
}

hipError_t launch_count_reduce(const int* nfin, int64_t slots, int64_t stride, const IdxChunk& idx, int count,
                               long long* status, hipStream_t s) {
    if (count < 1 || count > kChunk) return hipErrorInvalidValue;
    hipLaunchKernelGGL(count_reduce_kernel, dim3(count), dim3(256), 0, s, nfin, slots, stride, idx, status);
    return hipGetLastError();
}

int64_t normalize_cols_partials(int rows, int cols_pad, int row_chunk) {
    const int nchunks = (rows + row_chunk - 1) / row_chunk;
    return (int64_t)nchunks * 3 * cols_pad;
}

hipError_t launch_source_x(const half_t* psi, int64_t ld, int64_t stride, int rows, int cols, int rows_pad, int k,
                           int active, const float* xsq, int64_t stride_xsq, const float* xtot, half_t* xs,
                           int batch, hipStream_t s) {
    const int64_t total = (int64_t)rows_pad * ld;
    const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 2048));
    hipLaunchKernelGGL(source_x_kernel, dim3(blocks, batch), dim3(256), 0, s, psi, ld, stride, rows, cols, rows_pad,
                       k, active, xsq, stride_xsq, xtot, xs);
    return hipGetLastError();
}

hipError_t launch_psi_col_normalize(const NormArgs& a, int batch, float* part, int64_t part_floats, int row_chunk,
                                    hipStream_t s) {
    const int nchunks = (a.rows + row_chunk - 1) / row_chunk;
    const int64_t cols_pad = a.ld_psi;
    if ((int64_t)(nchunks + 1) * cols_pad > part_floats || a.cols > cols_pad) return hipErrorInvalidValue;
    const unsigned cb = (unsigned)((a.cols + 255) / 256);
    hipLaunchKernelGGL(psi_colstats_kernel, dim3(cb, nchunks, batch), dim3(256), 0, s, a.psi, a.ld_psi, a.stride_psi,
                       a.rows, a.cols, row_chunk, part, part_floats, cols_pad);
    hipLaunchKernelGGL(psi_colfactor_kernel, dim3(cb, batch), dim3(256), 0, s, part, part_floats, nchunks, a.cols,
                       cols_pad, a.eps, a.psisq, a.stride_psisq);
    const int64_t total = (int64_t)a.rows * a.cols;
    const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 2048));
    hipLaunchKernelGGL(psi_colscale_kernel, dim3(blocks, batch), dim3(256), 0, s, a.psi, a.ld_psi, a.stride_psi,
                       a.rows, a.cols, part, part_floats, nchunks, cols_pad, a.psi32, a.stride_psi32);
    return hipGetLastError();
}

template <int VW>
hipError_t cols_launch(const NormArgs& a, int batch, double* partials, int row_chunk, hipStream_t s) {
    const int nchunks = (a.rows + row_chunk - 1) / row_chunk;
    const int pad_chunks = (int)((a.rows_pad + row_chunk - 1) / row_chunk);
    const unsigned stat_blocks = (unsigned)((a.cols + 64 * VW - 1) / (64 * VW));
    // The stats pass writes partials for every padded column block it covers;
    // padded columns beyond the last real block are never read.
    hipLaunchKernelGGL((normalize_cols_stats<VW>), dim3(stat_blocks, nchunks, batch), dim3(kColThreads), 0, s, a,
                       partials, row_chunk);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(normalize_cols_finalize, dim3((unsigned)((a.cols + 255) / 256), batch), dim3(256), 0, s, a,
                       partials, nchunks);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const unsigned app_blocks = (unsigned)((a.ld_psi + 64 * VW - 1) / (64 * VW));
    if (a.psi32)
        hipLaunchKernelGGL((normalize_cols_apply<VW, true>), dim3(app_blocks, pad_chunks, batch), dim3(kColThreads), 0,
                           s, a, (const double*)partials, row_chunk);
    else
        hipLaunchKernelGGL((normalize_cols_apply<VW, false>), dim3(app_blocks, pad_chunks, batch), dim3(kColThreads), 0,
                           s, a, (const double*)partials, row_chunk);
    return hipGetLastError();
}

template <int SW>
hipError_t cols_fused_launch(const NormArgs& a, int batch, hipStream_t s) {
    constexpr int rpi = kFusedThreads / (SW / 4);
    const int nr = (int)((a.rows_pad + rpi - 1) / rpi);
    if (nr > kFusedNR || a.ld_psi % SW) return hipErrorInvalidValue;
    const dim3 grid((unsigned)(a.ld_psi / SW), batch);
    if (a.psi32) hipLaunchKernelGGL((normalize_cols_fused<SW, true>), grid, dim3(kFusedThreads), 0, s, a, nr);
    else hipLaunchKernelGGL((normalize_cols_fused<SW, false>), grid, dim3(kFusedThreads), 0, s, a, nr);
    return hipGetLastError();
}

hipError_t launch_normalize_cols(const NormArgs& a, int batch, double* partials, int row_chunk, hipStream_t s) {
    switch (cols_fused_width(a)) {
        case 64: return cols_fused_launch<64>(a, batch, s);
        case 32: return cols_fused_launch<32>(a, batch, s);
        case 16: return cols_fused_launch<16>(a, batch, s);
        default: break;
    }
    if (a.vec_ok && a.cols % 4 == 0 && a.ld_psi % 4 == 0) return cols_launch<4>(a, batch, partials, row_chunk, s);
    return cols_launch<1>(a, batch, partials, row_chunk, s);
}

int momentum_sumsq_blocks(int64_t elems) {
    return (int)std::max<int64_t>(1, std::min<int64_t>(256, (elems + 4095) / 4096));
}

hipError_t launch_momentum_sumsq(const NormArgs& a, int batch, float* part, int64_t stride_part, hipStream_t s) {
    const int64_t n = (int64_t)a.rows * a.cols;
    const bool vec = a.vec_ok && n % 4 == 0;
    dim3 grid((unsigned)momentum_sumsq_blocks(n), batch);
    if (vec) hipLaunchKernelGGL((momentum_sumsq_kernel<4>), grid, dim3(256), 0, s, a, part, stride_part);
    else hipLaunchKernelGGL((momentum_sumsq_kernel<1>), grid, dim3(256), 0, s, a, part, stride_part);
    return hipGetLastError();
}

hipError_t launch_scaled_cast(const NormArgs& a, int batch, const float* scale, hipStream_t s) {
    const bool vec = a.vec_ok && a.cols % 4 == 0 && a.ld_psi % 4 == 0;
    const int64_t nv = a.rows_pad * a.ld_psi / (vec ? 4 : 1);
    dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>((nv + 255) / 256, 2048)), batch);
    const bool dbg = a.psi32 != nullptr;
    if (vec) {
        if (dbg) hipLaunchKernelGGL((scaled_cast_kernel<4, true>), grid, dim3(256), 0, s, a, scale);
        else hipLaunchKernelGGL((scaled_cast_kernel<4, false>), grid, dim3(256), 0, s, a, scale);
    } else {
        if (dbg) hipLaunchKernelGGL((scaled_cast_kernel<1, true>), grid, dim3(256), 0, s, a, scale);
        else hipLaunchKernelGGL((scaled_cast_kernel<1, false>), grid, dim3(256), 0, s, a, scale);
    }
    return hipGetLastError();
}

hipError_t launch_psi_scale(const float* psisq, int64_t stride, int active_rows, float eps, float* out,
                            int batch, hipStream_t s) {
    hipLaunchKernelGGL(psi_scale_kernel, dim3(batch), dim3(256), 0, s, psisq, stride, active_rows, eps, out);
    return hipGetLastError();
}

hipError_t launch_g_update(const GUpdateArgs& a, int batch, hipStream_t s) {
    const int64_t n = (int64_t)a.rows * a.cols;
    const bool vec = a.vec_ok && (a.cols % 4) == 0;
    const int64_t work = vec ? n / 4 : n;
    unsigned blocks = (unsigned)std::min<int64_t>((work + 255) / 256, 2048);
    if (blocks == 0) blocks = 1;
    dim3 grid(blocks, batch);
    const bool dbg = a.t32 != nullptr;
    if (vec) {
        if (dbg) hipLaunchKernelGGL((g_update_kernel<4, true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((g_update_kernel<4, false>), grid, dim3(256), 0, s, a);
    } else {
        if (dbg) hipLaunchKernelGGL((g_update_kernel<1, true>), grid, dim3(256), 0, s, a);
        else hipLaunchKernelGGL((g_update_kernel<1, false>), grid, dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_sum_partials(const float* in, int n, float* out, int batch, hipStream_t s, const int* need) {
    hipLaunchKernelGGL(sum_partials_kernel, dim3(batch), dim3(256), 0, s, in, n, out, need);
    return hipGetLastError();
}

hipError_t launch_l_norm_closed(const LNormGroups& g, hipStream_t s) {
    if (g.n < 1 || g.n > kMaxItems || g.zbeg[0] != 0) return hipErrorInvalidValue;
    for (int i = 0; i < g.n; ++i)
        if (g.zbeg[i + 1] <= g.zbeg[i] || !g.psi2[i] || !g.ritz[i] || !g.nsel[i] || !g.tn2[i] || !g.need[i])
            return hipErrorInvalidValue;
    hipLaunchKernelGGL(l_norm_closed_kernel, dim3(g.zbeg[g.n]), dim3(64), 0, s, g);
    return hipGetLastError();
}

hipError_t launch_add_diag(half_t* q, int64_t sp, int count, float a, hipStream_t s) {
    if (count < 1 || sp < 1) return hipErrorInvalidValue;
    const int64_t n = (int64_t)count * sp;
    hipLaunchKernelGGL(add_diag_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, q, sp, n, a);
    return hipGetLastError();
}

hipError_t launch_alignment_partials(const AlignChunk& c, int cnt, double lr, double wd, double* part,
                                     hipStream_t s) {
    if (cnt < 1 || cnt > kChunk || !(lr > 0.0)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(alignment_partials_kernel, dim3(kAlignBlocks, cnt), dim3(256), 0, s, c, 1.0 / lr, wd, part);
    return hipGetLastError();
}

hipError_t launch_alignment_finalize(const double* part, int num_mats, double* cos_out, double* mean_out,
                                     hipStream_t s) {
    hipLaunchKernelGGL(alignment_finalize_kernel, dim3(1), dim3(256), 0, s, part, num_mats, cos_out, mean_out);
    return hipGetLastError();
}

// Each thread moves kProbeU 16-byte vectors per iteration, every load of the
// iteration issued before the first store.
constexpr int kProbeU = 4;
template <int MIX>
__global__ void __launch_bounds__(256) stream_probe_kernel(const float4* a, const float4* b, const float4* c,
                                                           float4* o32, uint2* o16, int64_t n4) {
    const int64_t step = (int64_t)gridDim.x * 256 * kProbeU;
    for (int64_t base = (int64_t)blockIdx.x * 256 * kProbeU + threadIdx.x; base < n4; base += step) {
        float4 x[kProbeU], y[kProbeU], z[kProbeU];
#pragma unroll
        for (int u = 0; u < kProbeU; ++u) {
            const int64_t i = base + u * 256;
            if (i < n4) {
                x[u] = a[i];
                if constexpr (MIX != 3) y[u] = b[i];
                if constexpr (MIX <= 1) z[u] = c[i];
            }
        }
#pragma unroll
        for (int u = 0; u < kProbeU; ++u) {
            const int64_t i = base + u * 256;
            if (i >= n4) break;
            if constexpr (MIX == 3) {
                o32[i] = x[u];
            } else if constexpr (MIX == 2) {
                half_t h[4] = {(half_t)(x[u].x - y[u].x), (half_t)(x[u].y - y[u].y), (half_t)(x[u].z - y[u].z),
                               (half_t)(x[u].w - y[u].w)};
                o16[i] = *reinterpret_cast<const uint2*>(h);
            } else {
                float4 m;
                m.x = fmaf(0.95f, x[u].x, y[u].x); m.y = fmaf(0.95f, x[u].y, y[u].y);
                m.z = fmaf(0.95f, x[u].z, y[u].z); m.w = fmaf(0.95f, x[u].w, y[u].w);
                if constexpr (MIX == 1) {
                    m.x += z[u].x; m.y += z[u].y; m.z += z[u].z; m.w += z[u].w;
                    o32[i] = m;
                } else {
                    o32[i] = m;
                    half_t h[4] = {(half_t)z[u].x, (half_t)z[u].y, (half_t)z[u].z, (half_t)z[u].w};
                    o16[i] = *reinterpret_cast<const uint2*>(h);
                }
            }
        }
    }
}

hipError_t launch_stream_probe(int mix, int64_t n, const float* a, const float* b, const float* c, float* o32,
                               half_t* o16, hipStream_t s) {
    if (n < 4 || n % 4 || mix < 0 || mix > 3) return hipErrorInvalidValue;
    const int64_t n4 = n / 4;
    const unsigned blocks = (unsigned)std::min<int64_t>((n4 + 256 * kProbeU - 1) / (256 * kProbeU), 4096);
    auto A = reinterpret_cast<const float4*>(a);
    auto B = reinterpret_cast<const float4*>(b);
    auto C = reinterpret_cast<const float4*>(c);
    auto O = reinterpret_cast<float4*>(o32);
    auto H = reinterpret_cast<uint2*>(o16);
    switch (mix) {
        case 0: hipLaunchKernelGGL(stream_probe_kernel<0>, dim3(blocks), dim3(256), 0, s, A, B, C, O, H, n4); break;
        case 1: hipLaunchKernelGGL(stream_probe_kernel<1>, dim3(blocks), dim3(256), 0, s, A, B, C, O, H, n4); break;
        case 2: hipLaunchKernelGGL(stream_probe_kernel<2>, dim3(blocks), dim3(256), 0, s, A, B, C, O, H, n4); break;
        default: hipLaunchKernelGGL(stream_probe_kernel<3>, dim3(blocks), dim3(256), 0, s, A, B, C, O, H, n4); break;
    }
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, int64_t bytes, hipStream_t s) {
    if (bytes <= 0) return hipSuccess;
    if (bytes % 16 || (reinterpret_cast<uintptr_t>(p) & 15)) return hipErrorInvalidValue;
    const int64_t n16 = bytes / 16;
    const unsigned blocks = (unsigned)std::min<int64_t>((n16 + 255) / 256, 4096);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, s, reinterpret_cast<uint4*>(p), n16);
    return hipGetLastError();
}

}  // namespace np
