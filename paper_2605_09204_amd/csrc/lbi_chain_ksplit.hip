// The chain scan for batches too small to give every SIMD two chains, for
// fp32 storage in the split arithmetic at r = 64: sixteen waves per chain, of
// which eight form the products and eight move data.
//
// It computes what the workgroup chain kernel computes (the suffix composites
// P_j = A_j P_{j+1} of the scan formulation, Proposition "Scan Formulation of
// Backpropagation"; c_j = A_j c_{j+1} + b_j; lambda_j = P_j lambda_K + c_j,
// the apply of Algorithm "Bounded-Interface Backpropagation", Phase 2).  With
// one chain or less per CU, a chain's time is K times the latency of one slot,
// and most of that latency is instruction issue: one wave issues a VALU
// instruction about every five cycles, and a slot of the four-wave kernel has
// about 250 per wave.  This kernel shortens the chain of dependent work per
// slot in two ways.
//
//   * Split contraction.  Matrix wave w = (cb, kh) = (w % 4, w / 4), w < 8,
//     owns column block cb of P and the k half kh: rows 32 kh .. 32 kh + 31
//     of P_{j+1}, which are exactly the k pair kh of P's B-operand layout
//     (lane l holds rows 16 I + 4 (l/16) + v of column 16 cb + l%16).  Its
//     MFMAs form, for all 64 rows, what those rows contribute to A_j P_{j+1}:
//     24 MFMAs of the six-product split arithmetic instead of 48, and half the
//     split of P.  The two partial products of a column block are summed
//     through LDS: each wave keeps the two row blocks it owns and hands the
//     other two to its partner.  The wave reads A_j's row blocks rotated by
//     2 kh, so its own blocks are always accumulators 0 and 1 and every
//     register index is static.
//   * Specialised waves.  The matrix waves do only what depends on P: the
//     exchange, the split, the MFMAs and the apply of slot j+1 (own rows of
//     P_{j+1} times lambda_K over the column block, in the MFMAs' shadow).
//     Eight staging waves load A_{j-1} NPF slots ahead (16-byte buffer loads),
//     split it into three bf16 planes in LDS, form c_{j-1} = A_{j-1} c_j +
//     b_{j-1} from the same registers, and store lambda_{j+2}, summed over the
//     four column blocks.
//   * One barrier per slot.  Each role runs its own slot loop with the same
//     barriers, so neither role's loop-carried registers are live in the
//     other's loop (121 VGPRs: four waves per SIMD).  The partial sums of
//     consecutive slots alternate between two LDS buffers.  83 KB of LDS: one
//     chain per CU.
//
// All HIP code here is built with packed fp32 math disabled.

#include "lbi_chain.hpp"

namespace lbi {
namespace {

template <bool AFF>
__global__ __launch_bounds__(1024) void scan_ksplit_kernel(const ScanArgs args)
{
    constexpr int R = 64;
    constexpr int NMW = 8;                   // matrix waves
    constexpr int NSW = 8;                   // staging waves
    constexpr int TH = 64 * NSW;             // staging threads
    using G = Geo<R, kF32X, 4>;              // the LDS plane layout of the chain kernel
    constexpr int PLANE = G::PLANE, PITCH = G::PITCH;
    constexpr int NPF = 2;                   // slots prefetched
    constexpr int CPT = R * R / 4 / TH;      // 16-byte chunks of a tile per staging thread
    constexpr int LPR = R / 4;               // staging lanes per tile row
    constexpr int RPI = TH / LPR;            // tile rows per chunk index
    constexpr int TILE_BYTES = R * R * 4;
    constexpr int SHIFT = ilog2(LPR) - ilog2(CPT);  // staging reduce layout
    static_assert(G::SWZ && G::PERM && PLANE == R * R && CPT * TH * 4 == R * R && CPT <= LPR,
                  "tile layout");

    __shared__ __attribute__((aligned(16))) __bf16 sA[2][3 * PLANE];
    // partial sums handed over: [slot parity][column block][receiving k half][row block][lane]
    __shared__ __attribute__((aligned(16))) f4 sX[2][4][2][2][64];
    // c_s in a ring of four, indexed (K - s) mod 4
    __shared__ __attribute__((aligned(16))) float sC[AFF ? 4 : 1][R];
    // apply partials of lambda_s: [s parity][column block][row]
    __shared__ __attribute__((aligned(16))) float sPart[2][4][R];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const bool mw = w < NMW;
    const int g = lane >> 4;
    const int li = lane & 15;
    const int cb = w & 3, kh = (w >> 2) & 1;
    const int64_t beta = blockIdx.x;
    const int64_t K = args.K;
    const float *A = (const float *)args.A + beta * K * (int64_t)(R * R);
    const float *bv = AFF ? (const float *)args.b + beta * K * (int64_t)R : nullptr;
    float *lam = args.lam + beta * K * (int64_t)R;
    auto ring = [&](int64_t s) { return (int)((K - s) & 3); };

    // staging roles (staging waves): chunk i of thread ht covers tile row
    // i * RPI + srow, columns scol .. scol + 3; after the row reduce, lane
    // sgi = i 2^SHIFT owns the affine sum of row i * RPI + srow
    const int ht = mw ? 0 : tid - 64 * NMW;
    const int sgi = ht % LPR;
    const int srow = ht / LPR;
    const int scol = 4 * sgi;
    const int orow = (sgi >> SHIFT) * RPI + srow;
    const bool oown = (sgi & ((1 << SHIFT) - 1)) == 0;

    // ---- loads (branch-free: a slot outside the chain gets out-of-range
    // offsets, which read zeros without touching memory) --------------------
    auto load_tile = [&](u4 (&dst)[CPT], int64_t j, bool valid) {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(A + (valid ? j : 0) * (int64_t)(R * R)), 0, TILE_BYTES, kBufferWord3);
#pragma unroll
        for (int i = 0; i < CPT; ++i)
            dst[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, valid ? (i * TH + ht) * 16 : kOutOfRange,
                                                           0, 0);
    };
    auto load_b = [&](int64_t j, bool valid) -> uint32_t {
        if constexpr (AFF) {
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                (void *)(bv + (valid ? j : 0) * (int64_t)R), 0, R * 4, kBufferWord3);
            return __builtin_amdgcn_raw_buffer_load_b32(rs, valid && oown ? orow * 4 : kOutOfRange, 0, 0);
        } else {
            return 0u;
        }
    };

    // ---- staging: registers -> three bf16 planes in LDS; c_j ----------------
    auto stage = [&](const u4 (&src)[CPT], int buf, uint32_t braw, int64_t j, bool first) {
        float cv[4];
        if constexpr (AFF) {
            const f4 c4 = first ? f4{0.0f, 0.0f, 0.0f, 0.0f} : *(const f4 *)&sC[ring(j + 1)][scol];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                cv[u] = c4[u];
        }
        float part[CPT];
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            const int row = i * RPI + srow;
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                x[e] = bitsf(src[i][e]);
            if constexpr (AFF) {
                float sum = x[0] * cv[0];
#pragma unroll
                for (int e = 1; e < 4; ++e)
                    sum += x[e] * cv[e];
                part[i] = sum;
            }
            const Split2 s01 = split_pair(x[0], x[1]);
            const Split2 s23 = split_pair(x[2], x[3]);
            const int pos = swz_pos<R>(row, lds_col<true>(scol));
            __bf16 *dst = sA[buf];
            *(u2 *)&dst[pos] = u2{s01.h, s23.h};
            *(u2 *)&dst[PLANE + pos] = u2{s01.m, s23.m};
            *(u2 *)&dst[2 * PLANE + pos] = u2{s01.l, s23.l};
        }
        if constexpr (AFF) {
            group_reduce<LPR, CPT>(part, sgi);
            if (oown)
                sC[ring(j)][orow] = part[0] + bitsf(braw);
        }
    };

    // ---- the apply (matrix waves): own rows of P times lambda_K over cb -------
    const float lk = mw ? ((const float *)args.lamK)[beta * R + 16 * cb + li] : 0.0f;
    auto apply = [&](const f4 (&Po)[2], int pbuf) {
        float q[8];
#pragma unroll
        for (int I = 0; I < 2; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                q[4 * I + v] = Po[I][v] * lk;
        group_reduce<16, 8>(q, li);
        // lane li (even) holds the 16-lane sum of value li / 2 = 4 I + v
        if ((li & 1) == 0) {
            const int idx = li >> 1;
            sPart[pbuf][cb][16 * (2 * kh + (idx >> 2)) + 4 * g + (idx & 3)] = q[0];
        }
    };
    // ---- lambda_s = sum of the column-block partials + c_s (staging waves;
    // one of them stores, in turn) ------------------------------------------
    auto finalize = [&](int64_t s, bool valid, int pbuf) {
        const int64_t ss = valid ? s : 0;
        const int ft = ht - 64 * (int)((uint64_t)ss % NSW);
        const bool mine = valid && ft >= 0 && ft < R;
        const int fi = mine ? ft : 0;
        float acc = ((sPart[pbuf][0][fi] + sPart[pbuf][1][fi]) + sPart[pbuf][2][fi]) + sPart[pbuf][3][fi];
        if constexpr (AFF)
            acc += sC[ring(ss)][fi];
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(lam + ss * R), 0, R * (int)sizeof(float), kBufferWord3);
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc), rs,
                                              mine ? fi * (int)sizeof(float) : kOutOfRange, 0, 0);
    };

    // ---- slot K-1: P = A_{K-1}, c = b_{K-1}; then stage slot K-2 --------------
    // Slot x is prefetched into register set (K-1-x) mod NPF and staged into
    // LDS buffer (K-1-x) mod 2.
    u4 pf[NPF][CPT];
    uint32_t pfb[NPF];
    if (!mw) {
        u4 first[CPT];
        const uint32_t firstb = load_b(K - 1, true);
        load_tile(first, K - 1, true);
#pragma unroll
        for (int q = 1; q <= NPF; ++q) {
            pfb[q % NPF] = load_b(K - 1 - q, K - 1 - q >= 0);
            load_tile(pf[q % NPF], K - 1 - q, K - 1 - q >= 0);
        }
        stage(first, 0, firstb, K - 1, true);
    }
    __syncthreads();

    // own rows of the running composite (matrix waves): row blocks 2 kh, 2 kh + 1
    f4 Po[2];
    if (mw) {
#pragma unroll
        for (int I = 0; I < 2; ++I)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * (2 * kh + I) + 4 * g + v, col = 16 * cb + li;
                const int pos = swz_pos<R>(row, lds_col<true>(col & ~3) + (col & 3));
                Po[I][v] = (to_f32(sA[0][pos]) + to_f32(sA[0][PLANE + pos])) +
                           to_f32(sA[0][2 * PLANE + pos]);
            }
    } else if (K >= 2) {
        stage(pf[1 % NPF], 1, pfb[1 % NPF], K - 2, false);
        pfb[1 % NPF] = load_b(K - 2 - NPF, K - 2 - NPF >= 0);
        load_tile(pf[1 % NPF], K - 2 - NPF, K - 2 - NPF >= 0);
    }

    // ---- slots K-2 .. 0 ---------------------------------------------------------
    // Iteration j (A_j and c_j staged before its barrier).  Matrix waves:
    // complete the own rows of P_{j+1} with the partner's partial sums, split
    // them, the MFMAs of the partial A_j P_{j+1} with the apply of slot j+1 in
    // their shadow, then the partner's row blocks to LDS.  Staging waves:
    // lambda_{j+2}, then slot j-1 into the other LDS buffer, then the loads of
    // slot j-1-NPF.  The buffers each side writes in iteration j were last
    // read before this barrier.
    f4 Pk[2];  // own row blocks of the last partial product
    const int rot = 2 * kh;
    // (each role in its own loop, with the same barriers)
    if (mw) {
        for (int64_t base = K - 2; base >= 0; base -= NPF) {
#pragma unroll
            for (int s = 0; s < NPF; ++s) {
                const int64_t j = base - s;
                if (j < 0)
                    break;
                const int buf = (int)((uint32_t)(K - 1 - j) & 1);
                __syncthreads();
                if (j < K - 2) {
#pragma unroll
                    for (int I = 0; I < 2; ++I)
                        Po[I] = Pk[I] + sX[(j + 1) & 1][cb][kh][I][lane];
                }
                const __bf16 *sAb = sA[buf];
                bf16x8 ah[4], am[4], al[4];
#pragma unroll
                for (int I = 0; I < 4; ++I) {
                    const int rb = (I + rot) & 3;
                    ah[I] = a_operand<R, PITCH>(sAb, rb, kh, li, g);
                    am[I] = a_operand<R, PITCH>(sAb + PLANE, rb, kh, li, g);
                    al[I] = a_operand<R, PITCH>(sAb + 2 * PLANE, rb, kh, li, g);
                }
                // B operand: own rows of P_{j+1} (k pair kh), in three parts
                bf16x8 bh, bm, bl;
                {
                    u4 hh, mm, ll;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const Split2 sp = split_pair_keep(Po[e >> 1][2 * (e & 1)], Po[e >> 1][2 * (e & 1) + 1]);
                        hh[e] = sp.h;
                        mm[e] = sp.m;
                        ll[e] = sp.l;
                    }
                    bh = __builtin_bit_cast(bf16x8, hh);
                    bm = __builtin_bit_cast(bf16x8, mm);
                    bl = __builtin_bit_cast(bf16x8, ll);
                }
                f4 Pn[4];
#pragma unroll
                for (int I = 0; I < 4; ++I)
                    Pn[I] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#define LBI_KS_GROUP(AOP, BOP)                                                             \
    _Pragma("unroll") for (int I = 0; I < 4; ++I) Pn[I] =                                  \
        __builtin_amdgcn_mfma_f32_16x16x32_bf16(AOP[I], BOP, Pn[I], 0, 0, 0);
                // the six partial products that reach 2^-16 of the leading one
                LBI_KS_GROUP(ah, bh)
                LBI_KS_GROUP(ah, bm)
                __builtin_amdgcn_sched_barrier(0);
                apply(Po, (int)((j + 1) & 1));
                __builtin_amdgcn_sched_barrier(0);
                LBI_KS_GROUP(am, bh)
                LBI_KS_GROUP(ah, bl)
                LBI_KS_GROUP(al, bh)
                LBI_KS_GROUP(am, bm)
#undef LBI_KS_GROUP
#pragma unroll
                for (int I = 0; I < 2; ++I) {
                    sX[j & 1][cb][kh ^ 1][I][lane] = Pn[2 + I];
                    Pk[I] = Pn[I];
                }
            }
        }
    } else {
        for (int64_t base = K - 2; base >= 0; base -= NPF) {
#pragma unroll
            for (int s = 0; s < NPF; ++s) {
                const int64_t j = base - s;
                if (j < 0)
                    break;
                const int buf = (int)((uint32_t)(K - 1 - j) & 1);
                __syncthreads();
                finalize(j + 2, j + 2 <= K - 1, (int)((j + 2) & 1));
                const int nx = (s + 2) % NPF;  // register set of slot j-1
                stage(pf[nx], buf ^ 1, pfb[nx], j - 1, false);
                pfb[nx] = load_b(j - 1 - NPF, j - 1 - NPF >= 0);
                load_tile(pf[nx], j - 1 - NPF, j - 1 - NPF >= 0);
            }
        }
    }
    // slot 0's partials (written in the last iteration) and the last two
    // adjoints
    __syncthreads();
    if (mw) {
        if (K >= 2) {
#pragma unroll
            for (int I = 0; I < 2; ++I)
                Po[I] = Pk[I] + sX[0][cb][kh][I][lane];
        }
        apply(Po, 0);
    } else if (K >= 2) {
        finalize(1, true, 1);
    }
    __syncthreads();
    if (!mw)
        finalize(0, true, 0);
}

template <bool AFF> hipError_t launch_ks(const ChainLaunch &c)
{
    void *params[] = {(void *)&c.args};
    return hipLaunchKernel((const void *)&scan_ksplit_kernel<AFF>, dim3((unsigned)c.B), dim3(1024),
                           params, 0, c.stream);
}

}  // namespace

bool chain_ksplit_supported(const ChainLaunch &c)
{
    return c.out == kOutLambda && !c.args.progress && !c.args.compact && !c.hint && c.args.S == 1 &&
           c.r == 64;
}

hipError_t launch_chain_ksplit_f32x(const ChainLaunch &c)
{
    if (!chain_ksplit_supported(c))
        return hipErrorInvalidValue;
    return c.aff ? launch_ks<true>(c) : launch_ks<false>(c);
}

}  // namespace lbi
