// Spectral and rank-normalised Frobenius norms of a stack of r x r matrices
// (gfx950): the interface-Jacobian statistics of the appendix "Interface
// Jacobian Structure" (local ||J_k||_2, suffix ||P_k||_2 = ||J_k^T ...
// J_{K-1}^T||_2, local ||J_k||_F / sqrt(r)).
//
// Per matrix M (fp32 or bf16 storage):
//  1. M is read once; m = max |M_ij| is reduced and Ms = M 2^-e, with
//     2^e <= m < 2^(e+1) (an exact scaling), is kept transposed in LDS.
//  2. H_0 = Ms^T Ms on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).
//  3. T times: H <- (H / tr H)(H / tr H)^T.  H stays symmetric positive
//     semidefinite with every entry in [-1, 1]; after T steps it is a
//     multiple of (Ms^T Ms)^(2^T).
//  4. v = the row of H with the largest diagonal entry; the Rayleigh quotient
//     ||Ms v||^2 / ||v||^2 of Ms^T Ms gives sigma_1(M) = 2^e sqrt(quotient).
// A zero matrix gives 0 and 0; a matrix with a NaN or infinite entry NaN and NaN.
// Error of step 4 in exact arithmetic, with no spectral gap assumed: with
// x_k = sigma_k^2 / sigma_1^2 and weights c_k of v's row on the eigenvectors,
// 1 - quotient / sigma_1^2 <= max_x x^(2^T) (1 - x) / (row's diagonal)
// <= r / (exp(1) 2^T) (the diagonal is at least 1/r of the trace); T = 24
// puts it at 2.8e-6 for r = 128 (1.4e-6 for sigma).
//
// Work split: one wavefront per matrix for r <= 64 (four matrices per
// 256-thread workgroup), the whole workgroup for r = 128.  H lives in LDS,
// rows padded by 4 floats so that the 16 rows a b128 read touches fall in
// distinct banks.  The contraction index of the matrix-core steps is
// permuted (lane group q takes k = q r/4 + t at step t) so that each lane's
// operands for four steps are one 16-byte LDS read.

#include "lbi_device.hpp"
#include "lbi_internal.h"

namespace lbi {
namespace {

constexpr int kThreads = 256;
constexpr int kSquarings = 24;

template <int R> struct NormGeo {
    static constexpr int WPM = R == 128 ? 4 : 1;       // waves per matrix
    static constexpr int MPW = 4 / WPM;                // matrices per workgroup
    static constexpr int LD = R + 4;                   // LDS row stride (floats)
    static constexpr int NB = R / 16;                  // 16-row blocks
    static constexpr int LANES = 64 * WPM;             // lanes per matrix
    static constexpr int VPL = R * R / LANES;          // matrix entries per lane
    static_assert(VPL % 4 == 0, "norm geometry");
};

__device__ __forceinline__ float wave_sum(float x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ float wave_max(float x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

// Four consecutive entries of a matrix in storage dtype, widened to fp32.
template <bool BF16> __device__ __forceinline__ f4 load4(const void *p, int64_t idx)
{
    if constexpr (BF16) {
        const u2 w = *(const u2 *)((const uint16_t *)p + idx);
        return f4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & kHighHalf),
                  __uint_as_float(w[1] << 16), __uint_as_float(w[1] & kHighHalf)};
    } else {
        return *(const f4 *)((const float *)p + idx);
    }
}

// Sum (or max) over the lanes of one matrix: the wave, or the workgroup
// through the four-float exchange area red (every lane gets the result).
template <int WPM, bool MAX>
__device__ __forceinline__ float matrix_reduce(float x, float *red)
{
    x = MAX ? wave_max(x) : wave_sum(x);
    if constexpr (WPM > 1) {
        const int w = threadIdx.x / 64;
        __syncthreads();  // red free (earlier readers done)
        if (threadIdx.x % 64 == 0)
            red[w] = x;
        __syncthreads();
        x = MAX ? fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))
                : (red[0] + red[1]) + (red[2] + red[3]);
    }
    return x;
}

// acc = scale * H H^T for this wave's output tiles, written back over H.
// Every wave of the workgroup calls it the same number of times.
template <int R>
__device__ __forceinline__ void gram_step(float *H, float scale)
{
    using G = NormGeo<R>;
    const int lane = threadIdx.x % 64, q = lane / 16, l16 = lane % 16;
    const int wm = G::WPM > 1 ? (int)(threadIdx.x / 64) : 0;  // wave within matrix
    // wave wm owns row blocks [wm * NB / WPM, (wm + 1) * NB / WPM), all column blocks
    constexpr int RB = G::NB / G::WPM;
    f4 acc[RB][G::NB];
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < G::NB; ++j)
            acc[i][j] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const float *Hq = H + q * (R / 4);
#pragma unroll 2
    for (int s = 0; s < R / 16; ++s) {
        f4 a[RB], b[G::NB];
#pragma unroll
        for (int i = 0; i < RB; ++i)
            a[i] = *(const f4 *)&Hq[((wm * RB + i) * 16 + l16) * G::LD + 4 * s];
#pragma unroll
        for (int j = 0; j < G::NB; ++j)
            b[j] = *(const f4 *)&Hq[(j * 16 + l16) * G::LD + 4 * s];
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int i = 0; i < RB; ++i)
#pragma unroll
                for (int j = 0; j < G::NB; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][e], b[j][e], acc[i][j],
                                                                     0, 0, 0);
    }
    __syncthreads();  // every read of H done
#pragma unroll
    for (int i = 0; i < RB; ++i)
#pragma unroll
        for (int j = 0; j < G::NB; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                H[((wm * RB + i) * 16 + 4 * q + v) * G::LD + j * 16 + l16] = acc[i][j][v] * scale;
    __syncthreads();
}

// 1 / tr H (0 for a zero H), the same in every lane of the matrix.
template <int R> __device__ __forceinline__ float inv_trace(const float *H)
{
    using G = NormGeo<R>;
    const int lane = threadIdx.x % 64;
    float d = 0.0f;
#pragma unroll
    for (int i = lane; i < R; i += 64)
        d += H[i * G::LD + i];
    const float tr = wave_sum(d);
    return tr > 0.0f ? 1.0f / tr : 0.0f;
}

template <int R, bool BF16>
__global__ __launch_bounds__(kThreads) void norms_kernel(const void *M, int64_t n, float *spec,
                                                        float *fro)
{
    using G = NormGeo<R>;
    __shared__ __attribute__((aligned(16))) float lds[G::MPW * R * G::LD];
    __shared__ float red[4];
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int slot = wave / G::WPM;                  // matrix within the workgroup
    const int ml = (wave % G::WPM) * 64 + lane;      // lane within the matrix
    const int64_t g = (int64_t)blockIdx.x * G::MPW + slot;
    const bool live = g < n;
    float *H = lds + slot * (R * G::LD);
    const int64_t base = g * R * R;

    // 1. read M: entries 4 (ml + LANES u) + 0..3, u < VPL / 4
    f4 x[G::VPL / 4];
    float mx = 0.0f, poison = 0.0f;  // poison: NaN once any entry is not finite
#pragma unroll
    for (int u = 0; u < G::VPL / 4; ++u) {
        x[u] = live ? load4<BF16>(M, base + 4 * (ml + G::LANES * u)) : f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            mx = fmaxf(mx, fabsf(x[u][c]));
            poison += x[u][c] * 0.0f;
        }
    }
    const float m = matrix_reduce<G::WPM, true>(mx, red);
    poison = matrix_reduce<G::WPM, false>(poison, red);
    // Ms = M 2^-e with 2^e <= m < 2^(e+1), scaled exactly in two halves (a
    // single factor would overflow for subnormal m)
    const int e = (m > 0.0f && m <= 3.0e38f) ? ilogbf(m) : 0;
    const float s1 = ldexpf(1.0f, -(e / 2)), s2 = ldexpf(1.0f, -(e - e / 2));
#pragma unroll
    for (int u = 0; u < G::VPL / 4; ++u)
#pragma unroll
        for (int c = 0; c < 4; ++c)
            x[u][c] = (x[u][c] * s1) * s2;
    // sum of Ms^2 (the Frobenius norm without overflow or underflow)
    float ssn = 0.0f;
#pragma unroll
    for (int u = 0; u < G::VPL / 4; ++u)
#pragma unroll
        for (int c = 0; c < 4; ++c)
            ssn += x[u][c] * x[u][c];
    const float fro2 = matrix_reduce<G::WPM, false>(ssn, red);
    // Ms^T into LDS: entry (row, col) of M goes to H[col][row]
#pragma unroll
    for (int u = 0; u < G::VPL / 4; ++u) {
        const int idx = 4 * (ml + G::LANES * u);
        const int row = idx / R, col = idx % R;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            H[(col + c) * G::LD + row] = x[u][c];
    }
    __syncthreads();

    // 2-3. H_0 = Ms^T Ms, then T normalised squarings
    gram_step<R>(H, 1.0f);
#pragma unroll 1
    for (int t = 0; t < kSquarings; ++t) {
        const float it = inv_trace<R>(H);
        gram_step<R>(H, it * it);
    }

    // 4. v = row i* of H (largest diagonal entry; the lowest index on ties)
    float best = -1.0f;
    int bi = 0;
#pragma unroll
    for (int i = lane; i < R; i += 64) {
        const float d = H[i * G::LD + i];
        if (d > best) {
            best = d;
            bi = i;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ob = __shfl_xor(best, o);
        const int oi = __shfl_xor(bi, o);
        if (ob > best || (ob == best && oi < bi)) {
            best = ob;
            bi = oi;
        }
    }
    const float *v = H + bi * G::LD;
    float vv = 0.0f;
#pragma unroll
    for (int k = lane; k < R; k += 64)
        vv += v[k] * v[k];
    vv = wave_sum(vv);
    // w = Ms v: R rows over the matrix's lanes (LANES / R lanes per row)
    constexpr int LPR = G::LANES / R >= 1 ? G::LANES / R : 1;  // lanes per row
    constexpr int RPL = R / G::LANES >= 1 ? R / G::LANES : 1;  // rows per lane
    constexpr int CPL = R / LPR;                               // columns per lane
    float ww = 0.0f;
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) {
        const int row = (ml / LPR) + (G::LANES / LPR) * rr;
        const int c0 = (ml % LPR) * CPL;
        float acc = 0.0f;
        if (live && row < R) {
#pragma unroll 4
            for (int c = 0; c < CPL; c += 4) {
                f4 a = load4<BF16>(M, base + (int64_t)row * R + c0 + c);
                a = (a * s1) * s2;
                const f4 vv4 = *(const f4 *)&v[c0 + c];
                acc += a[0] * vv4[0] + a[1] * vv4[1] + a[2] * vv4[2] + a[3] * vv4[3];
            }
        }
        // lanes of one row are adjacent: add the partners' parts
#pragma unroll
        for (int o = 1; o < LPR; o <<= 1)
            acc += __shfl_xor(acc, o);
        if (ml % LPR == 0 && row < R) {
            ww += acc * acc;
        }
    }
    ww = matrix_reduce<G::WPM, false>(ww, red);
    if (live && ml == 0) {
        if (spec)
            spec[g] = (vv > 0.0f ? ldexpf(sqrtf(ww / vv), e) : 0.0f) + poison;
        if (fro)
            fro[g] = ldexpf(sqrtf(fro2 / (float)R), e) + poison;
    }
}

template <int R>
hipError_t norms_r(const void *M, bool bf16, int64_t n, float *spec, float *fro, hipStream_t st)
{
    using G = NormGeo<R>;
    const unsigned grid = (unsigned)((n + G::MPW - 1) / G::MPW);
    if (bf16)
        hipLaunchKernelGGL((norms_kernel<R, true>), dim3(grid), dim3(kThreads), 0, st, M, n, spec,
                           fro);
    else
        hipLaunchKernelGGL((norms_kernel<R, false>), dim3(grid), dim3(kThreads), 0, st, M, n, spec,
                           fro);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_norms(const void *M, bool bf16, int64_t n, int32_t r, float *spec, float *fro,
                        hipStream_t stream)
{
    switch (r) {
    case 16: return norms_r<16>(M, bf16, n, spec, fro, stream);
    case 32: return norms_r<32>(M, bf16, n, spec, fro, stream);
    case 64: return norms_r<64>(M, bf16, n, spec, fro, stream);
    default: return norms_r<128>(M, bf16, n, spec, fro, stream);
    }
}

}  // namespace lbi
