// Interface-adjoint suffix scan of LBI on gfx950 (MI355X).
//
// Computes, for B independent chains of K slots,
//     (P_j, c_j) = (A_j, b_j) o (A_{j+1}, b_{j+1}) o ... o (A_{K-1}, b_{K-1}),
//     lambda_j   = P_j lambda_K + c_j,
// with the combine (A, b) o (A', b') = (A A', A b' + b) of the scan
// formulation (Proposition "Scan Formulation of Backpropagation"; Theorem
// "Bounded-Interface Backpropagation" gives lambda_j = mbar_j when b = 0), and
// Phase 2 of Algorithm "Bounded-Interface Backpropagation" (apply the suffix
// products to mbar_K, every slot in parallel).
//
// Kernel design (one workgroup per chain, NW waves):
//   * The running suffix composite P (R x R, fp32) is split by 16-column
//     blocks across the waves; wave w keeps column blocks w, w+NW, ... in the
//     accumulator layout of v_mfma_f32_16x16x*: lane l holds rows
//     16*I + 4*(l/16) + v (v = 0..3) of column 16*cb + l%16.  That layout is
//     also the B-operand layout of the next MFMA (k taken from the lane's row
//     set), so P_{j} = A_j * P_{j+1} chains from accumulator to operand with no
//     shuffles; A_j is the A operand, read from LDS with the k-order permuted
//     to match.  Each combine costs R^3 MACs on the matrix cores.
//   * Work is the algorithmic minimum: the K-1 combines of a right-to-left
//     inclusive scan, and batch parallelism over chains fills the GPU.
//   * A_j tiles stream HBM -> registers (prefetched NPF slots ahead,
//     coalesced 16-byte loads) -> LDS (padded rows, conflict-free MFMA reads)
//     with one barrier per slot.
//   * c_j = A_j c_{j+1} + b_j runs on the VALU (rows split over the
//     workgroup); the apply P_j lambda_K reduces each wave's column slice with
//     a DPP butterfly, then across waves through LDS, and lambda_j is stored
//     once, coalesced.
//   * bf16: A tiles are bf16 MFMA operands; the fp32 composite is fed back as
//     bf16 hi + lo (two MFMAs), so the only bf16 rounding is the inputs'.
//
// All HIP code here is built with packed fp32 math disabled.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "lbi.h"

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned int u4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

enum : int { kF32 = 0, kBF16 = 1 };

template <int DT> struct Elem;
template <> struct Elem<kF32> {
    typedef float T;
    static constexpr int kPad = 4;  // LDS row pitch R + 4 floats
};
template <> struct Elem<kBF16> {
    typedef __bf16 T;
    static constexpr int kPad = 8;  // LDS row pitch R + 8 bf16
};

constexpr int waves_for(int R) { return R == 16 ? 1 : (R == 32 ? 2 : 4); }

struct ScanArgs {
    const void *A;
    const void *b;
    const void *lamK;
    float *lam;
    int64_t K;
    int32_t hinted;       // widths hint present
    int32_t ncol_active;  // column blocks of P that can be nonzero: ceil(r_K/16)
    // nibble k (k = 0..K): ceil(r_k / 16), read only when hinted
    uint8_t wcode[(LBI_MAX_HINT_K + 2) / 2];
};

__device__ __forceinline__ int width_blocks(const ScanArgs &a, int64_t k, int full)
{
    if (!a.hinted)
        return full;
    const uint8_t byte = a.wcode[k >> 1];
    return (k & 1) ? (byte >> 4) : (byte & 15);
}

// DPP lane permutations within a 16-lane row (GFX9 encodings).
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppXor7 = 0x141;       // row_half_mirror: lane i <- i ^ 7
constexpr int kDppXor8 = 0x128;       // row_ror:8:       lane i <- i ^ 8

template <int CTRL> __device__ __forceinline__ float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}

// One butterfly stage over N live values: lanes whose bit BIT is 0 keep the
// lower half (summed with the partner's lower half), the others the upper.
template <int N, int CTRL, int BIT, int V>
__device__ __forceinline__ void bfly_split(float (&q)[V], int li)
{
    const bool upper = (li >> BIT) & 1;
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
        const float keep = upper ? q[i + N / 2] : q[i];
        const float send = upper ? q[i] : q[i + N / 2];
        q[i] = keep + dpp<CTRL>(send);
    }
}

// Sum V values per lane over the 16 lanes of a row.  The partner masks
// 8, 7, 2, 1 span GF(2)^4, so after the four stages lane li holds the full
// sums of original indices (li >> SHIFT) * VF + e, e < VF, where
// VF = max(1, V / 16) and SHIFT = log2(16 / V) for V < 16.
template <int V> __device__ __forceinline__ void row_reduce(float (&q)[V], int li)
{
    static_assert(V == 4 || V == 8 || V == 16 || V == 32, "unsupported width");
    if constexpr (V >= 2) bfly_split<V, kDppXor8, 3>(q, li);
    if constexpr (V >= 4) bfly_split<V / 2, kDppXor7, 2>(q, li);
    else q[0] += dpp<kDppXor7>(q[0]);
    if constexpr (V >= 8) bfly_split<V / 4, kDppXor2, 1>(q, li);
    else q[0] += dpp<kDppXor2>(q[0]);
    if constexpr (V >= 16) bfly_split<V / 8, kDppXor1, 0>(q, li);
    else q[0] += dpp<kDppXor1>(q[0]);
}

template <typename T> __device__ __forceinline__ float to_f32(T x) { return (float)x; }

template <int R, int DT, bool AFF>
__global__ __launch_bounds__(64 * waves_for(R)) void scan_chain_kernel(const ScanArgs args)
{
    constexpr int NW = waves_for(R);
    constexpr int T = 64 * NW;
    constexpr int NRB = R / 16;       // 16-row blocks
    constexpr int CB = NRB / NW;      // column blocks per wave
    constexpr int V = 4 * NRB;        // values per lane in the apply
    constexpr int VF = V >= 16 ? V / 16 : 1;
    constexpr int SHIFT = V >= 16 ? 0 : (V == 8 ? 1 : 2);
    using E = typename Elem<DT>::T;
    constexpr int ESZ = sizeof(E);
    constexpr int PITCH = R + Elem<DT>::kPad;
    constexpr int EPC = 16 / ESZ;                  // elements per 16-byte chunk
    constexpr int TILE_CHUNKS = R * R / EPC;
    constexpr int CPT = (TILE_CHUNKS + T - 1) / T; // chunks per thread
    constexpr int BCH = R / EPC;                   // chunks of one b row
    constexpr int TPR = T / R;                     // threads per row (c update)
    constexpr int CPR = R / TPR;                   // columns per thread
    constexpr int NPF = 2;                         // slots prefetched ahead
    static_assert(NRB % NW == 0 && (TPR == 2 || TPR == 4), "tile geometry");

    __shared__ __attribute__((aligned(16))) E sA[2][R * PITCH];
    __shared__ __attribute__((aligned(16))) float sB[AFF ? 2 : 1][R];
    __shared__ __attribute__((aligned(16))) float sC[AFF ? 2 : 1][R];
    __shared__ __attribute__((aligned(16))) float sPart[2][NW][R];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int g = lane >> 4;
    const int li = lane & 15;
    const int64_t K = args.K;
    const int64_t beta = blockIdx.x;
    const E *A = (const E *)args.A + beta * K * (int64_t)(R * R);
    const E *bv = AFF ? (const E *)args.b + beta * K * (int64_t)R : nullptr;
    float *lam = args.lam + beta * K * (int64_t)R;
    const int ncol = args.ncol_active;

    // ---- staging helpers --------------------------------------------------
    auto load_tile = [&](u4 (&dst)[CPT], int64_t j) {
        const int rows = 16 * width_blocks(args, j, NRB);
        const int cols = 16 * width_blocks(args, j + 1, NRB);
        const u4 *src = (const u4 *)(A + j * (int64_t)(R * R));
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = i * T + tid;
            const int e = c * EPC;
            const int row = e / R, col = e % R;
            u4 z = {0u, 0u, 0u, 0u};
            if (c < TILE_CHUNKS && row < rows && col < cols)
                z = src[c];
            dst[i] = z;
        }
    };
    auto store_tile = [&](const u4 (&src)[CPT], int buf) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = i * T + tid;
            if (c < TILE_CHUNKS) {
                const int e = c * EPC;
                const int row = e / R, col = e % R;
                *(u4 *)&sA[buf][row * PITCH + col] = src[i];
            }
        }
    };
    auto load_b = [&](u4 &dst, int64_t j) {
        u4 z = {0u, 0u, 0u, 0u};
        if (AFF && tid < BCH)
            z = ((const u4 *)(bv + j * (int64_t)R))[tid];
        dst = z;
    };
    auto store_b = [&](const u4 &src, int buf) {
        if (AFF && tid < BCH) {
            const E *x = (const E *)&src;
#pragma unroll
            for (int e = 0; e < EPC; ++e)
                sB[buf][tid * EPC + e] = to_f32(x[e]);
        }
    };

    // ---- per-lane constants -----------------------------------------------
    float lk[CB];
#pragma unroll
    for (int t = 0; t < CB; ++t) {
        const int cb = w + NW * t;
        lk[t] = to_f32(((const E *)args.lamK)[beta * R + 16 * cb + li]);
    }
    auto col_active = [&](int t) { return (w + NW * t) < ncol; };

    // ---- the apply: partial P lambda_K over this wave's columns -----------
    auto apply_partial = [&](const f4 (&P)[NRB][CB], int buf) {
        float q[V];
#pragma unroll
        for (int I = 0; I < NRB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float s = 0.0f;
#pragma unroll
                for (int t = 0; t < CB; ++t)
                    s += P[I][t][v] * lk[t];
                q[4 * I + v] = s;
            }
        row_reduce<V>(q, li);
        if ((li & ((1 << SHIFT) - 1)) == 0) {
#pragma unroll
            for (int e = 0; e < VF; ++e) {
                const int idx = (li >> SHIFT) * VF + e;  // = 4*I + v
                const int row = 16 * (idx >> 2) + 4 * g + (idx & 3);
                sPart[buf][w][row] = q[e];
            }
        }
    };
    // ---- lambda_j = sum of the wave partials + c_j --------------------------
    auto finalize = [&](int64_t j, int buf) {
        if (tid < R) {
            float s = sPart[buf][0][tid];
#pragma unroll
            for (int ww = 1; ww < NW; ++ww)
                s += sPart[buf][ww][tid];
            if constexpr (AFF)
                s += sC[buf][tid];
            lam[j * R + tid] = s;
        }
    };
    // ---- c_j = A_j c_{j+1} + b_j ------------------------------------------
    auto affine_update = [&](int buf, int prv) {
        if constexpr (AFF) {
            const int m = tid / TPR, qq = tid % TPR;
            const E *arow = &sA[buf][m * PITCH + qq * CPR];
            const float *cprev = &sC[prv][qq * CPR];
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < CPR; ++k)
                acc += to_f32(arow[k]) * cprev[k];
            acc += dpp<kDppXor1>(acc);
            if constexpr (TPR == 4)
                acc += dpp<kDppXor2>(acc);
            if (qq == 0)
                sC[buf][m] = acc + sB[buf][m];
        }
    };

    // ---- one combine on the matrix cores: Pn = A_j * P ----------------------
    auto combine = [&](f4 (&Pn)[NRB][CB], const f4 (&P)[NRB][CB], int buf, int64_t j) {
        const int nrb = width_blocks(args, j, NRB);
        const int nkb = width_blocks(args, j + 1, NRB);
#pragma unroll
        for (int I = 0; I < NRB; ++I)
#pragma unroll
            for (int t = 0; t < CB; ++t)
                Pn[I][t] = f4{0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (DT == kF32) {
#pragma unroll
            for (int Ik = 0; Ik < NRB; ++Ik) {
                if (Ik >= nkb)
                    continue;
                f4 a[NRB];
#pragma unroll
                for (int I = 0; I < NRB; ++I)
                    a[I] = *(const f4 *)&sA[buf][(16 * I + li) * PITCH + 16 * Ik + 4 * g];
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int t = 0; t < CB; ++t) {
                        if (!col_active(t))
                            continue;
#pragma unroll
                        for (int I = 0; I < NRB; ++I)
                            if (I < nrb)
                                Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    a[I][v], P[Ik][t][v], Pn[I][t], 0, 0, 0);
                    }
            }
        } else {
            // k runs over pairs of 16-row blocks of P; a missing second block
            // (R = 16) is zero in both operands.
            constexpr int NKP = (NRB + 1) / 2;
#pragma unroll
            for (int p = 0; p < NKP; ++p) {
                if (2 * p >= nkb)
                    continue;
                constexpr bool kFull = (NRB % 2) == 0;
                bf16x8 bh[CB], bl[CB];
#pragma unroll
                for (int t = 0; t < CB; ++t) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float x0 = P[2 * p][t][v];
                        const float x1 = (kFull || 2 * p + 1 < NRB) ? P[kFull ? 2 * p + 1 : 2 * p][t][v] : 0.0f;
                        const __bf16 h0 = (__bf16)x0, h1 = (__bf16)x1;
                        bh[t][v] = h0;
                        bh[t][v + 4] = h1;
                        bl[t][v] = (__bf16)(x0 - (float)h0);
                        bl[t][v + 4] = (__bf16)(x1 - (float)h1);
                    }
                }
#pragma unroll
                for (int I = 0; I < NRB; ++I) {
                    if (I >= nrb)
                        continue;
                    const E *rowp = &sA[buf][(16 * I + li) * PITCH + 32 * p + 4 * g];
                    const bf16x4 a0 = *(const bf16x4 *)rowp;
                    bf16x4 a1 = {};
                    if (kFull || 2 * p + 1 < NRB)
                        a1 = *(const bf16x4 *)(rowp + 16);
                    const bf16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
                    for (int t = 0; t < CB; ++t) {
                        if (!col_active(t))
                            continue;
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh[t], Pn[I][t], 0, 0, 0);
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl[t], Pn[I][t], 0, 0, 0);
                    }
                }
            }
        }
    };

    // ---- slot K-1: P = A_{K-1}, c = b_{K-1} ---------------------------------
    u4 pf[NPF][CPT];
    u4 pfb[NPF];
    {
        u4 first[CPT];
        u4 firstb;
        load_tile(first, K - 1);
        load_b(firstb, K - 1);
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            if (K - 2 - s >= 0) {
                load_tile(pf[s], K - 2 - s);
                load_b(pfb[s], K - 2 - s);
            }
        }
        store_tile(first, 0);
        store_b(firstb, 0);
    }
    __syncthreads();

    f4 P[NRB][CB];
    {
        const int nrb = width_blocks(args, K - 1, NRB);
#pragma unroll
        for (int I = 0; I < NRB; ++I)
#pragma unroll
            for (int t = 0; t < CB; ++t)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int row = 16 * I + 4 * g + v;
                    const int col = 16 * (w + NW * t) + li;
                    P[I][t][v] = (I < nrb && col_active(t)) ? to_f32(sA[0][row * PITCH + col]) : 0.0f;
                }
        if constexpr (AFF) {
            if (tid < R)
                sC[0][tid] = sB[0][tid];
        }
        apply_partial(P, 0);
    }

    // ---- slots K-2 .. 0 -------------------------------------------------------
    for (int64_t base = K - 2; base >= 0; base -= NPF) {
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            const int64_t j = base - s;
            if (j < 0)
                break;
            const int cur = (int)((K - 1 - j) & 1), prv = cur ^ 1;
            store_tile(pf[s], cur);
            store_b(pfb[s], cur);
            if (j - NPF >= 0) {
                load_tile(pf[s], j - NPF);
                load_b(pfb[s], j - NPF);
            }
            __syncthreads();
            finalize(j + 1, prv);
            f4 Pn[NRB][CB];
            combine(Pn, P, cur, j);
            affine_update(cur, prv);
            apply_partial(Pn, cur);
#pragma unroll
            for (int I = 0; I < NRB; ++I)
#pragma unroll
                for (int t = 0; t < CB; ++t)
                    P[I][t] = Pn[I][t];
        }
    }
    __syncthreads();
    finalize(0, (int)((K - 1) & 1));
}

// ---- host side ------------------------------------------------------------

bool supported_r(int32_t r) { return r == 16 || r == 32 || r == 64 || r == 128; }

template <int R, int DT, bool AFF>
hipError_t launch(const ScanArgs &a, int64_t B, hipStream_t stream)
{
    void *params[] = {(void *)&a};
    return hipLaunchKernel((const void *)&scan_chain_kernel<R, DT, AFF>, dim3((unsigned)B),
                           dim3(64 * waves_for(R)), params, 0, stream);
}

template <int DT, bool AFF>
hipError_t dispatch_r(int32_t r, const ScanArgs &a, int64_t B, hipStream_t s)
{
    switch (r) {
    case 16: return launch<16, DT, AFF>(a, B, s);
    case 32: return launch<32, DT, AFF>(a, B, s);
    case 64: return launch<64, DT, AFF>(a, B, s);
    default: return launch<128, DT, AFF>(a, B, s);
    }
}

bool overlaps(const void *p, size_t pn, const void *q, size_t qn)
{
    if (!p || !q || pn == 0 || qn == 0)
        return false;
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + qn && b < a + pn;
}

bool misaligned(const void *p) { return p && ((uintptr_t)p & 15u); }

lbi_status scan_impl(const void *A, const void *b, const void *lamK, float *lam, int64_t B,
                     int64_t K, int32_t r, lbi_dtype dt, void *ws, size_t ws_bytes,
                     lbi_stream_t stream, const int32_t *widths)
{
    if (dt != LBI_F32 && dt != LBI_BF16)
        return LBI_ERR_DTYPE;
    if (!supported_r(r))
        return LBI_ERR_UNSUPPORTED_R;
    if (B < 0 || K < 1)
        return LBI_ERR_SHAPE;
    // sizes must fit comfortably in 64 bits and the launch grid
    const int64_t kMax = (int64_t)1 << 40;
    if (B > (int64_t)INT32_MAX || K > kMax / ((int64_t)r * r) || B > kMax / (K * (int64_t)r * r))
        return LBI_ERR_SHAPE;
    if (B == 0)
        return LBI_OK;
    if (!A || !lamK || !lam)
        return LBI_ERR_NULL;
    if (misaligned(A) || misaligned(b) || misaligned(lamK) || misaligned(lam))
        return LBI_ERR_ALIGN;
    const size_t esz = dt == LBI_F32 ? 4 : 2;
    const size_t nA = (size_t)B * K * r * r * esz, nb = b ? (size_t)B * K * r * esz : 0;
    const size_t nl = (size_t)B * r * esz, nout = (size_t)B * K * r * sizeof(float);
    if (overlaps(lam, nout, A, nA) || overlaps(lam, nout, b, nb) || overlaps(lam, nout, lamK, nl))
        return LBI_ERR_ALIAS;
    const size_t need = lbi_scan_backward_workspace_bytes(B, K, r, dt);
    if (need > 0 && (!ws || ws_bytes < need))
        return LBI_ERR_WORKSPACE;

    ScanArgs a;
    memset(&a, 0, sizeof a);
    a.A = A;
    a.b = b;
    a.lamK = lamK;
    a.lam = lam;
    a.K = K;
    a.hinted = 0;
    a.ncol_active = r / 16;
    if (widths) {
        for (int64_t k = 0; k <= K; ++k)
            if (widths[k] < 1 || widths[k] > r)
                return LBI_ERR_SHAPE;
        if (K <= LBI_MAX_HINT_K) {
            a.hinted = 1;
            for (int64_t k = 0; k <= K; ++k) {
                const int code = (widths[k] + 15) / 16;
                a.wcode[k >> 1] |= (uint8_t)((k & 1) ? (code << 4) : code);
            }
            a.ncol_active = (widths[K] + 15) / 16;
        }
    }
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (dt == LBI_F32)
        e = b ? dispatch_r<kF32, true>(r, a, B, s) : dispatch_r<kF32, false>(r, a, B, s);
    else
        e = b ? dispatch_r<kBF16, true>(r, a, B, s) : dispatch_r<kBF16, false>(r, a, B, s);
    return e == hipSuccess ? LBI_OK : LBI_ERR_HIP;
}

}  // namespace

extern "C" {

size_t lbi_scan_backward_workspace_bytes(int64_t B, int64_t K, int32_t r, lbi_dtype dt)
{
    (void)B;
    (void)K;
    (void)r;
    (void)dt;
    return 0;  // the single-level chain scan needs no scratch
}

lbi_status lbi_scan_backward(const void *A, const void *b, const void *lambda_K, float *lambda,
                             int64_t B, int64_t K, int32_t r, lbi_dtype dt, void *workspace,
                             size_t workspace_bytes, lbi_stream_t stream)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, workspace, workspace_bytes, stream,
                     nullptr);
}

lbi_status lbi_scan_backward_widths(const void *A, const void *b, const void *lambda_K,
                                    float *lambda, int64_t B, int64_t K, int32_t r, lbi_dtype dt,
                                    void *workspace, size_t workspace_bytes, lbi_stream_t stream,
                                    const int32_t *widths_host)
{
    return scan_impl(A, b, lambda_K, lambda, B, K, r, dt, workspace, workspace_bytes, stream,
                     widths_host);
}

const char *lbi_status_string(lbi_status s)
{
    switch (s) {
    case LBI_OK: return "LBI_OK";
    case LBI_ERR_NULL: return "LBI_ERR_NULL: a required pointer is NULL";
    case LBI_ERR_SHAPE: return "LBI_ERR_SHAPE: bad B, K, size or widths";
    case LBI_ERR_DTYPE: return "LBI_ERR_DTYPE: unknown dtype";
    case LBI_ERR_UNSUPPORTED_R: return "LBI_ERR_UNSUPPORTED_R: r must be 16, 32, 64 or 128";
    case LBI_ERR_WORKSPACE: return "LBI_ERR_WORKSPACE: workspace missing or too small";
    case LBI_ERR_HIP: return "LBI_ERR_HIP: the HIP runtime refused the launch";
    case LBI_ERR_ALIGN: return "LBI_ERR_ALIGN: a pointer is not 16-byte aligned";
    case LBI_ERR_ALIAS: return "LBI_ERR_ALIAS: lambda overlaps an input";
    }
    return "unknown lbi_status";
}

int lbi_abi_version(void) { return LBI_ABI_VERSION; }

}  // extern "C"
