// Interface-adjoint suffix scan of LBI on gfx950 (MI355X).
//
// Computes, for B independent chains of K slots,
//     (P_j, c_j) = (A_j, b_j) o (A_{j+1}, b_{j+1}) o ... o (A_{K-1}, b_{K-1}),
//     lambda_j   = P_j lambda_K + c_j,
// with the combine (A, b) o (A', b') = (A A', A b' + b) of the scan
// formulation (Proposition "Scan Formulation of Backpropagation"; Theorem
// "Bounded-Interface Backpropagation" gives lambda_j = mbar_j when b = 0), and
// Phase 2 of Algorithm "Bounded-Interface Backpropagation" (apply the suffix
// products to mbar_K, every slot).
//
// Kernel design (one workgroup per chain, NW waves):
//   * The running suffix composite P (R x R, fp32) is split by 16-column
//     blocks across the waves; wave w keeps column blocks w, w+NW, ... in the
//     accumulator layout of v_mfma_f32_16x16x*: lane l holds rows
//     16*I + 4*(l/16) + v (v = 0..3) of column 16*cb + l%16.  That layout is
//     also the B-operand layout of the next MFMA (k taken from the lane's row
//     set), so P_j = A_j * P_{j+1} chains from accumulator to operand with no
//     shuffles; A_j is the A operand, read from LDS with the k order permuted
//     to match.  Each combine costs R^3 MACs on the matrix cores.
//   * Work is the algorithmic minimum: the K-1 combines of a right-to-left
//     inclusive scan; the B independent chains fill the GPU.
//   * A_j tiles stream HBM -> registers (buffer loads NPF slots ahead, 16
//     bytes per lane, branch-free) -> LDS (padded rows: conflict-free MFMA
//     operand reads), one barrier per slot.
//   * The apply of slot j+1 (P_{j+1} lambda_K: per-wave partial sums reduced
//     by a DPP butterfly, then across waves through LDS) is issued between
//     the MFMAs that form P_j, so VALU and matrix-core work overlap;
//     c_j = A_j c_{j+1} + b_j runs on the VALU with rows split over the
//     workgroup; lambda_j is stored once, coalesced, by one wave in turn.
//   * bf16: A tiles are bf16 MFMA operands; the fp32 composite is fed back as
//     bf16 hi + lo (two MFMAs), so the only bf16 rounding is the inputs'.
//   * Widths hint: loads of all-zero tile regions are skipped (out-of-range
//     buffer offsets return zero without touching memory) and the combine
//     runs a shape specialised to the slot's row and k blocks.
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

// Buffer resource word 3 for raw (untyped) buffer loads on gfx9-family GPUs.
constexpr int kBufferWord3 = 0x00020000;
// A per-lane offset past every tile: the load returns zero, no memory access.
constexpr int kOutOfRange = 0x40000000;

struct ScanArgs {
    const void *A;
    const void *b;
    const void *lamK;
    float *lam;
    int64_t K;
    // ceil(r_k / 16) for k = 0..K as 4-bit fields, 8 per word (hinted launches)
    uint32_t wcode[(LBI_MAX_HINT_K + 1 + 7) / 8];
};

__device__ __forceinline__ int width_blocks(const ScanArgs &a, int64_t k)
{
    return (int)((a.wcode[k >> 3] >> ((k & 7) * 4)) & 15u);
}

__device__ __forceinline__ int pow2_at_least(int x)
{
    return x <= 1 ? 1 : (x <= 2 ? 2 : (x <= 4 ? 4 : 8));
}

// DPP lane permutations within a 16-lane row (GFX9 encodings).
constexpr int kDppXor1 = 0xB1;   // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;   // quad_perm [2,3,0,1]
constexpr int kDppXor7 = 0x141;  // row_half_mirror: lane i <- i ^ 7
constexpr int kDppXor8 = 0x128;  // row_ror:8:       lane i <- i ^ 8

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
    bfly_split<V, kDppXor8, 3>(q, li);
    if constexpr (V >= 4) bfly_split<V / 2, kDppXor7, 2>(q, li);
    else q[0] += dpp<kDppXor7>(q[0]);
    if constexpr (V >= 8) bfly_split<V / 4, kDppXor2, 1>(q, li);
    else q[0] += dpp<kDppXor2>(q[0]);
    if constexpr (V >= 16) bfly_split<V / 8, kDppXor1, 0>(q, li);
    else q[0] += dpp<kDppXor1>(q[0]);
}

template <typename T> __device__ __forceinline__ float to_f32(T x) { return (float)x; }

// Geometry shared by the kernel and its pieces.
template <int R, int DT, int NCA> struct Geo {
    static constexpr int NW = waves_for(R);
    static constexpr int T = 64 * NW;
    static constexpr int NRB = R / 16;    // 16-row blocks
    static constexpr int CB = NCA / NW;   // column blocks per wave
    static constexpr int V = 4 * NRB;     // values per lane in the apply
    static constexpr int VF = V >= 16 ? V / 16 : 1;
    static constexpr int SHIFT = V >= 16 ? 0 : (V == 8 ? 1 : 2);
    using E = typename Elem<DT>::T;
    static constexpr int ESZ = sizeof(E);
    static constexpr int PITCH = R + Elem<DT>::kPad;
    static constexpr int EPC = 16 / ESZ;                   // elements per 16-byte chunk
    static constexpr int TILE_CHUNKS = R * R / EPC;
    static constexpr int CPT = (TILE_CHUNKS + T - 1) / T;  // chunks per thread
    static constexpr int BCH = R / EPC;                    // chunks of one b row
    static constexpr int TPR = T / R;                      // threads per row (c update)
    static constexpr int CPR = R / TPR;                    // columns per thread
    static constexpr int NPF = (DT == kBF16 && R <= 64) ? 3 : 2;  // slots prefetched
    static constexpr int WPF = R > 64 ? R / 64 : 1;        // waves per finalize
    static constexpr int NWF = NW / WPF;                   // finalizing wave groups
    static_assert(NCA % NW == 0 && CB >= 1 && (TPR == 2 || TPR == 4), "tile geometry");
};

// Pn = A_j * P on the matrix cores, for the first NR row blocks and NK k blocks
// (the rest of A_j is zero); rows past NR come out zero.
template <int R, int DT, int NCA, int NR, int NK>
__device__ __forceinline__ void combine(f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                        const f4 (&P)[R / 16][NCA / waves_for(R)],
                                        const typename Elem<DT>::T *sAbuf, int li, int g)
{
    using G = Geo<R, DT, NCA>;
    constexpr int NRB = G::NRB, CB = G::CB, PITCH = G::PITCH;
#pragma unroll
    for (int I = 0; I < NRB; ++I)
#pragma unroll
        for (int t = 0; t < CB; ++t)
            Pn[I][t] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    if constexpr (DT == kF32) {
#pragma unroll
        for (int Ik = 0; Ik < NK; ++Ik) {
            f4 a[NR];
#pragma unroll
            for (int I = 0; I < NR; ++I)
                a[I] = *(const f4 *)&sAbuf[(16 * I + li) * PITCH + 16 * Ik + 4 * g];
#pragma unroll
            for (int v = 0; v < 4; ++v)
#pragma unroll
                for (int t = 0; t < CB; ++t)
#pragma unroll
                    for (int I = 0; I < NR; ++I)
                        Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[I][v], P[Ik][t][v],
                                                                         Pn[I][t], 0, 0, 0);
        }
    } else {
        // k runs over pairs of 16-row blocks of P; a missing second block
        // (one 16-block only) is zero in both operands.
        constexpr int NKP = (NK + 1) / 2;
#pragma unroll
        for (int p = 0; p < NKP; ++p) {
            constexpr bool kPairs = NRB >= 2;
            bf16x8 bh[CB], bl[CB];
#pragma unroll
            for (int t = 0; t < CB; ++t) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float x0 = P[2 * p][t][v];
                    const float x1 = kPairs ? P[kPairs ? 2 * p + 1 : 0][t][v] : 0.0f;
                    const __bf16 h0 = (__bf16)x0, h1 = (__bf16)x1;
                    bh[t][v] = h0;
                    bh[t][v + 4] = h1;
                    bl[t][v] = (__bf16)(x0 - (float)h0);
                    bl[t][v + 4] = (__bf16)(x1 - (float)h1);
                }
            }
#pragma unroll
            for (int I = 0; I < NR; ++I) {
                const typename Elem<DT>::T *rowp = &sAbuf[(16 * I + li) * PITCH + 32 * p + 4 * g];
                const bf16x4 a0 = *(const bf16x4 *)rowp;
                bf16x4 a1 = {};
                if constexpr (kPairs)
                    a1 = *(const bf16x4 *)(rowp + 16);
                const bf16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
                for (int t = 0; t < CB; ++t) {
                    Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bh[t], Pn[I][t], 0, 0, 0);
                    Pn[I][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bl[t], Pn[I][t], 0, 0, 0);
                }
            }
        }
    }
}

// Runtime (row blocks, k blocks) of a hinted slot -> the specialised combine
// for the next powers of two (extra blocks multiply zeros).
template <int R, int DT, int NCA, int NR>
__device__ __forceinline__ void combine_k(int nk, f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                          const f4 (&P)[R / 16][NCA / waves_for(R)],
                                          const typename Elem<DT>::T *sAbuf, int li, int g)
{
    constexpr int NRB = R / 16;
    if (nk <= 1 || NRB == 1) { combine<R, DT, NCA, NR, 1>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 2) if (nk <= 2) { combine<R, DT, NCA, NR, 2>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 4) if (nk <= 4) { combine<R, DT, NCA, NR, 4>(Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 8) combine<R, DT, NCA, NR, 8>(Pn, P, sAbuf, li, g);
}

template <int R, int DT, int NCA>
__device__ __forceinline__ void combine_shape(int nr, int nk, f4 (&Pn)[R / 16][NCA / waves_for(R)],
                                              const f4 (&P)[R / 16][NCA / waves_for(R)],
                                              const typename Elem<DT>::T *sAbuf, int li, int g)
{
    constexpr int NRB = R / 16;
    if (nr <= 1 || NRB == 1) { combine_k<R, DT, NCA, 1>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 2) if (nr <= 2) { combine_k<R, DT, NCA, 2>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 4) if (nr <= 4) { combine_k<R, DT, NCA, 4>(nk, Pn, P, sAbuf, li, g); return; }
    if constexpr (NRB >= 8) combine_k<R, DT, NCA, 8>(nk, Pn, P, sAbuf, li, g);
}

template <int R, int DT, bool AFF, bool HINT, int NCA>
__global__ __launch_bounds__(64 * waves_for(R)) void scan_chain_kernel(const ScanArgs args)
{
    using G = Geo<R, DT, NCA>;
    using E = typename G::E;
    constexpr int NW = G::NW, T = G::T, NRB = G::NRB, CB = G::CB, V = G::V, VF = G::VF;
    constexpr int SHIFT = G::SHIFT, PITCH = G::PITCH, EPC = G::EPC, CPT = G::CPT;
    constexpr int TILE_CHUNKS = G::TILE_CHUNKS, BCH = G::BCH, TPR = G::TPR, CPR = G::CPR;
    static_assert(BCH <= T, "b row fits one chunk per thread");
    constexpr int NPF = G::NPF, WPF = G::WPF, NWF = G::NWF;
    constexpr int TILE_BYTES = R * R * G::ESZ;

    __shared__ __attribute__((aligned(16))) E sA[2][R * PITCH];
    // b_j as loaded: one raw 16-byte chunk per thread (threads < BCH hold b),
    // stored unconditionally so the store needs no branch
    __shared__ __attribute__((aligned(16))) u4 sB[AFF ? 2 : 1][T];
    __shared__ __attribute__((aligned(16))) float sC[AFF ? 3 : 1][R];
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

    // ---- staging: HBM -> registers -> LDS -------------------------------------
    // Loads are issued unconditionally (a slot that does not exist gets only
    // out-of-range offsets), so the compiler can count outstanding loads
    // exactly and wait only for the slot being stored.
    auto load_tile = [&](u4 (&dst)[CPT], int64_t j, bool valid) {
        const int64_t jj = valid ? j : 0;
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(A + jj * (int64_t)(R * R)), 0, TILE_BYTES, kBufferWord3);
        int rows = valid ? R : 0, cols = R;
        if constexpr (HINT) {
            rows = valid ? 16 * width_blocks(args, jj) : 0;
            cols = 16 * width_blocks(args, jj + 1);
        }
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = i * T + tid;
            const int e = c * EPC;
            const bool ok = c < TILE_CHUNKS && (e / R) < rows && (e % R) < cols;
            dst[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, ok ? c * 16 : kOutOfRange, 0, 0);
        }
    };
    auto store_tile = [&](const u4 (&src)[CPT], int buf) {
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int c = i * T + tid;
            if (TILE_CHUNKS % T == 0 || c < TILE_CHUNKS) {
                const int e = c * EPC;
                *(u4 *)&sA[buf][(e / R) * PITCH + (e % R)] = src[i];
            }
        }
    };
    auto load_b = [&](u4 &dst, int64_t j, bool valid) {
        if constexpr (AFF) {
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(bv + (valid ? j : 0) * (int64_t)R), 0, R * G::ESZ, kBufferWord3);
            dst = __builtin_amdgcn_raw_buffer_load_b128(
                rs, (valid && tid < BCH) ? tid * 16 : kOutOfRange, 0, 0);
        }
    };
    auto store_b = [&](const u4 &src, int buf) {
        if constexpr (AFF)
            sB[buf][tid] = src;
    };
    auto b_at = [&](int buf, int m) { return to_f32(((const E *)&sB[buf][0])[m]); };

    // ---- per-lane constants ---------------------------------------------------
    float lk[CB];
#pragma unroll
    for (int t = 0; t < CB; ++t)
        lk[t] = to_f32(((const E *)args.lamK)[beta * R + 16 * (w + NW * t) + li]);

    // ---- the apply: partial P lambda_K over this wave's columns ---------------
    auto apply_partial = [&](const f4 (&P)[NRB][CB], int pbuf) {
        float q[V];
#pragma unroll
        for (int I = 0; I < NRB; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float s = P[I][0][v] * lk[0];
#pragma unroll
                for (int t = 1; t < CB; ++t)
                    s += P[I][t][v] * lk[t];
                q[4 * I + v] = s;
            }
        row_reduce<V>(q, li);
        if ((li & ((1 << SHIFT) - 1)) == 0) {
#pragma unroll
            for (int e = 0; e < VF; ++e) {
                const int idx = (li >> SHIFT) * VF + e;  // = 4*I + v
                const int row = 16 * (idx >> 2) + 4 * g + (idx & 3);
                sPart[pbuf][w][row] = q[e];
            }
        }
    };
    // ---- lambda_s = sum of the wave partials + c_s, stored by one wave group ---
    // Branch-free: lanes with nothing to store (and calls with valid = false)
    // get an out-of-range offset, which the buffer store drops; every wave
    // then issues the same memory instructions, which keeps the compiler's
    // count of outstanding loads exact.
    auto finalize = [&](int64_t s, bool valid, int pbuf, int cring) {
        const int64_t ss = valid ? s : 0;
        const int fw = (int)((uint64_t)ss % NWF);
        const int ft = tid - fw * 64 * WPF;
        const bool mine = valid && ft >= 0 && ft < R;
        const int fi = mine ? ft : 0;
        float acc = sPart[pbuf][0][fi];
#pragma unroll
        for (int ww = 1; ww < NW; ++ww)
            acc += sPart[pbuf][ww][fi];
        if constexpr (AFF)
            acc += sC[cring][fi];
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(lam + ss * R), 0, R * (int)sizeof(float), kBufferWord3);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc), rs,
                                              mine ? fi * (int)sizeof(float) : kOutOfRange, 0, 0);
    };
    // ---- c_j = A_j c_{j+1} + b_j ------------------------------------------------
    auto affine_update = [&](int buf, int cprev, int ccur) {
        if constexpr (AFF) {
            const int m = tid / TPR, qq = tid % TPR;
            const E *arow = &sA[buf][m * PITCH + qq * CPR];
            const float *cp = &sC[cprev][qq * CPR];
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < CPR; ++k)
                acc += to_f32(arow[k]) * cp[k];
            acc += dpp<kDppXor1>(acc);
            if constexpr (TPR == 4)
                acc += dpp<kDppXor2>(acc);
            if (qq == 0)
                sC[ccur][m] = acc + b_at(buf, m);
        }
    };

    // ---- slot K-1: P = A_{K-1}, c = b_{K-1} -----------------------------------
    u4 pf[NPF][CPT];
    u4 pfb[NPF];
    {
        u4 first[CPT];
        u4 firstb;
        load_b(firstb, K - 1, true);
        load_tile(first, K - 1, true);
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            load_b(pfb[s], K - 2 - s, K - 2 - s >= 0);
            load_tile(pf[s], K - 2 - s, K - 2 - s >= 0);
        }
        store_tile(first, 0);
        store_b(firstb, 0);
    }
    __syncthreads();

    f4 P[NRB][CB];
#pragma unroll
    for (int I = 0; I < NRB; ++I)
#pragma unroll
        for (int t = 0; t < CB; ++t)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                P[I][t][v] = to_f32(sA[0][(16 * I + 4 * g + v) * PITCH + 16 * (w + NW * t) + li]);
    if constexpr (AFF) {
        if (tid < R)
            sC[0][tid] = b_at(0, tid);
    }

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Iteration j: stage A_j, then [finalize slot j+2 | MFMA P_j = A_j P_{j+1} |
    // apply slot j+1 | c_j].  Buffers: A, b by slot parity; partials by slot
    // parity; c in a ring of 3.
    for (int64_t base = K - 2; base >= 0; base -= NPF) {
#pragma unroll
        for (int s = 0; s < NPF; ++s) {
            const int64_t j = base - s;
            if (j < 0)
                break;
            const uint32_t step = (uint32_t)(K - 1 - j);  // slots done before j
            const int buf = (int)(step & 1);
            const int cc = (int)(step % 3), cp = (int)((step + 2) % 3), cf = (int)((step + 1) % 3);
            store_tile(pf[s], buf);
            store_b(pfb[s], buf);
            load_b(pfb[s], j - NPF, j - NPF >= 0);
            load_tile(pf[s], j - NPF, j - NPF >= 0);
            __syncthreads();
            finalize(j + 2, j + 2 <= K - 1, (int)((j + 2) & 1), cf);
            f4 Pn[NRB][CB];
            if constexpr (HINT) {
                const int nr = pow2_at_least(width_blocks(args, j));
                const int nk = pow2_at_least(width_blocks(args, j + 1));
                combine_shape<R, DT, NCA>(nr, nk, Pn, P, sA[buf], li, g);
            } else {
                combine<R, DT, NCA, NRB, NRB>(Pn, P, sA[buf], li, g);
            }
            apply_partial(P, (int)((j + 1) & 1));
            affine_update(buf, cp, cc);
#pragma unroll
            for (int I = 0; I < NRB; ++I)
#pragma unroll
                for (int t = 0; t < CB; ++t)
                    P[I][t] = Pn[I][t];
        }
    }
    // slot 0's partials reuse the buffer finalize(2) read in the last iteration
    __syncthreads();
    apply_partial(P, 0);
    __syncthreads();
    {
        // c_0 sits at ring index (K-1) % 3 and c_1 at (K-2) % 3
        const uint32_t last = (uint32_t)(K - 1);
        finalize(1, K >= 2, 1, (int)((last + 2) % 3));
        finalize(0, true, 0, (int)(last % 3));
    }
}

// ---- host side ------------------------------------------------------------

bool supported_r(int32_t r) { return r == 16 || r == 32 || r == 64 || r == 128; }

template <int R, int DT, bool AFF, bool HINT, int NCA>
hipError_t launch(const ScanArgs &a, int64_t B, hipStream_t stream)
{
    void *params[] = {(void *)&a};
    return hipLaunchKernel((const void *)&scan_chain_kernel<R, DT, AFF, HINT, NCA>,
                           dim3((unsigned)B), dim3(64 * waves_for(R)), params, 0, stream);
}

template <int DT, bool AFF, bool HINT>
hipError_t dispatch_r(int32_t r, int ncol, const ScanArgs &a, int64_t B, hipStream_t s)
{
    switch (r) {
    case 16: return launch<16, DT, AFF, HINT, 1>(a, B, s);
    case 32: return launch<32, DT, AFF, HINT, 2>(a, B, s);
    case 64: return launch<64, DT, AFF, HINT, 4>(a, B, s);
    default:
        // With a hint whose r_K <= 64 only the first four column blocks of P
        // can be nonzero.
        if (HINT && ncol <= 4)
            return launch<128, DT, AFF, HINT, 4>(a, B, s);
        return launch<128, DT, AFF, HINT, 8>(a, B, s);
    }
}

template <int DT>
hipError_t dispatch(bool aff, bool hint, int32_t r, int ncol, const ScanArgs &a, int64_t B,
                    hipStream_t s)
{
    if (aff)
        return hint ? dispatch_r<DT, true, true>(r, ncol, a, B, s)
                    : dispatch_r<DT, true, false>(r, ncol, a, B, s);
    return hint ? dispatch_r<DT, false, true>(r, ncol, a, B, s)
                : dispatch_r<DT, false, false>(r, ncol, a, B, s);
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
    bool hinted = false;
    int ncol = r / 16;
    if (widths) {
        for (int64_t k = 0; k <= K; ++k)
            if (widths[k] < 1 || widths[k] > r)
                return LBI_ERR_SHAPE;
        if (K <= LBI_MAX_HINT_K) {
            hinted = true;
            for (int64_t k = 0; k <= K; ++k) {
                const uint32_t code = (uint32_t)(widths[k] + 15) / 16;
                a.wcode[k >> 3] |= code << ((k & 7) * 4);
            }
            ncol = (widths[K] + 15) / 16;
        }
    }
    hipStream_t s = (hipStream_t)stream;
    const hipError_t e = dt == LBI_F32 ? dispatch<kF32>(b != nullptr, hinted, r, ncol, a, B, s)
                                       : dispatch<kBF16>(b != nullptr, hinted, r, ncol, a, B, s);
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
    return 0;  // the chain scan keeps its state in registers and LDS
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
